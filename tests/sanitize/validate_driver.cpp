// Host-side argument checks and workspace sizing of librbq.so, run under
// AddressSanitizer and UndefinedBehaviorSanitizer on the CPU (built by
// tests/test_host_sanitizers.py with g++ from csrc/validate.cpp and this file;
// no HIP runtime, no GPU). It replays the invalid-argument cases the ABI tests
// send through the exported calls, a sweep of valid shapes, and the size
// functions at the extremes of their int32 arguments, so that an
// out-of-bounds access or a signed overflow in the host code aborts the run.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <initializer_list>
#include <limits>

#include "../../paper_2606_31519_amd/csrc/rbq_internal.h"

using namespace rbq;

namespace {
int failures = 0;
void expect(bool ok, const char* what, int line) {
  if (!ok) {
    std::printf("FAILED line %d: %s\n", line, what);
    ++failures;
  }
}
#define EXPECT(x) expect((x), #x, __LINE__)

// aligned fake device pointers: never dereferenced by the host checks
const void* const P16 = reinterpret_cast<const void*>(uintptr_t(1) << 40);
const void* const P4 = reinterpret_cast<const void*>((uintptr_t(1) << 40) + 4);
template <class T> const T* fp(const void* p) { return static_cast<const T*>(p); }
}  // namespace

int main() {
  const float* F = fp<float>(P16);
  const uint32_t* U = fp<uint32_t>(P16);
  const int32_t* I = fp<int32_t>(P16);
  const size_t big = size_t(1) << 40;
  const int32_t imax = std::numeric_limits<int32_t>::max();

  // ---- heads
  EXPECT(check_heads(1, 32, 8, 128) == RBQ_OK);
  EXPECT(check_heads(1, 32, 8, 64) == RBQ_OK);
  EXPECT(check_heads(0, 32, 8, 128) == RBQ_EINVAL);
  EXPECT(check_heads(1, 6, 4, 128) == RBQ_EINVAL);
  EXPECT(check_heads(1, 32, 8, 100) == RBQ_EINVAL);
  EXPECT(check_heads(1, 32, 8, 96) == RBQ_EUNSUPPORTED);
  EXPECT(check_heads(1, 64, 2, 128) == RBQ_EUNSUPPORTED);
  EXPECT(check_heads(imax, imax, imax, imax) == RBQ_EINVAL);
  EXPECT(check_heads(-imax - 1, 1, 1, 128) == RBQ_EINVAL);

  // ---- encode (the ABI test's cases, then extremes)
  auto enc = [&](int B, int H, int D, int dt, int64_t ld, int n, int off, int cap, const void* P, unsigned flags,
                 const void* ws, size_t wsb) {
    return check_encode(B, H, D, P16, dt, ld, n, off, cap, fp<float>(P), F, U, P16, flags, ws, wsb);
  };
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, P16, 0, P16, 1 << 20) == RBQ_OK);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 1, 10, P16, 0, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, nullptr, 0, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, P16, 4, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 0, 0, 10, P16, 1, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, P16, 1, nullptr, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, P16, 1, P16, 16) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 7, 10, 10, 0, 10, P16, 0, P16, 1 << 20) == RBQ_EUNSUPPORTED);
  EXPECT(enc(1, 1, 96, 1, 10, 10, 0, 10, P16, 0, P16, 1 << 20) == RBQ_EUNSUPPORTED);
  EXPECT(enc(1, 1, 128, 1, 5, 10, 0, 10, P16, 0, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, 10, 10, 0, 10, P4, 0, P16, 1 << 20) == RBQ_EINVAL);
  EXPECT(enc(1, 1, 128, 1, imax, imax, imax, imax, P16, 0, P16, big) == RBQ_EINVAL);   // offset + n beyond cap
  EXPECT(enc(8, 8, 128, 1, imax, imax, 0, imax, P16, 1, P16, big) == RBQ_OK);
  EXPECT(enc(1, 1, 128, 1, int64_t(1) << 40, 10, 0, 10, P16, 0, P16, big) == RBQ_EINVAL);
  for (int n : {1, 1023, 1024, 1025, 1 << 20, imax})
    EXPECT(encode_workspace_bytes(65535, 1, 128, n) >= size_t(65535) * 128 * 4);

  // ---- quantize and score
  EXPECT(check_quantize(1, 8, 4, 128, F, F, F, U, F) == RBQ_OK);
  EXPECT(check_quantize(1, 8, 4, 128, fp<float>(P4), F, F, U, F) == RBQ_EINVAL);
  EXPECT(check_quantize(1, 8, 4, 128, F, F, nullptr, U, F) == RBQ_EINVAL);
  EXPECT(check_score(1, 8, 4, 128, 10, 10, U, P16, U, P16, P16) == RBQ_OK);
  EXPECT(check_score(1, 8, 4, 128, 11, 10, U, P16, U, P16, P16) == RBQ_EINVAL);
  EXPECT(check_score(1, 8, 4, 128, -1, 10, U, P16, U, P16, P16) == RBQ_EINVAL);
  EXPECT(check_score(1, 8, 4, 128, 0, 0, nullptr, nullptr, nullptr, nullptr, nullptr) == RBQ_OK);
  EXPECT(check_score(1, 8, 4, 128, 10, 10, fp<uint32_t>(P4), P16, U, P16, P16) == RBQ_EINVAL);
  for (int32_t n : {0, 1, 4096, 1 << 20, imax})
    for (int32_t bk : {1, 8, 65535}) {
      const int k = score_keys_per_lane(bk, 1, n);
      EXPECT(k == 1 || k == 2 || k == 4);
    }

  // ---- top-p
  auto tp = [&](int B, int H, int n, float p, float s, size_t wsb) {
    return check_topp(B, H, n, F, p, s, I, I, P16, wsb);
  };
  EXPECT(tp(1, 8, 100, 0.9f, 0.1f, big) == RBQ_OK);
  EXPECT(tp(1, 8, 100, 0.0f, 0.1f, big) == RBQ_EINVAL);
  EXPECT(tp(1, 8, 100, 1.5f, 0.1f, big) == RBQ_EINVAL);
  EXPECT(tp(1, 8, 100, std::nanf(""), 0.1f, big) == RBQ_EINVAL);
  EXPECT(tp(1, 8, 100, 0.9f, INFINITY, big) == RBQ_EINVAL);
  EXPECT(tp(1, 8, 100, 0.9f, -1.0f, big) == RBQ_EINVAL);
  EXPECT(tp(1, 8, 100, 0.9f, 0.1f, 8) == RBQ_EINVAL);
  EXPECT(tp(1, 1, 1 << 24, 0.9f, 0.1f, big) == RBQ_EUNSUPPORTED);
  EXPECT(tp(1, 1, imax, 0.9f, 0.1f, big) == RBQ_EUNSUPPORTED);
  EXPECT(tp(1, 65536, 10, 0.9f, 0.1f, big) == RBQ_EINVAL);
  EXPECT(tp(1, 65535, (1 << 24) - 1, 0.9f, 0.1f, big) == RBQ_OK);
  for (int32_t n : {0, 1, kSelSub - 1, kSelSub, kSelSub + 1, kSelSub * kSelMaxParts, kSelSub * kSelMaxParts + 1,
                    (1 << 24) - 1, imax}) {
    const ToppPlan pl = topp_plan(n);
    EXPECT(pl.spb >= 1 && pl.parts >= 1 && pl.parts <= kSelMaxParts);
    EXPECT(int64_t(pl.parts) * pl.spb * kSelSub >= n);
    EXPECT(int64_t(pl.parts - 1) * pl.spb * kSelSub < (n > 0 ? n : 1));
    EXPECT(int64_t(topp_mask_words(n)) * 64 >= n);
    EXPECT(topp_workspace(nullptr, 65535, n).bytes >= size_t(65535) * pl.parts * kSelPart1Bytes);
  }

  // ---- decode
  auto dec = [&](int Hq, int Hkv, int dt, int cap, int n, bool sparse, const void* kl, int64_t ld, int w, float sc,
                 size_t wsb) {
    return check_decode(1, Hq, Hkv, 128, F, P16, P16, dt, cap, n, sparse, I, I, kl, P16, ld, w, sc, F, P16, wsb);
  };
  EXPECT(dec(8, 4, 1, 100, 100, true, P16, 300, 10, 0.1f, big) == RBQ_OK);
  EXPECT(dec(8, 4, 1, 100, 100, true, P16, 5000, 5000, 0.1f, big) == RBQ_EINVAL);
  EXPECT(dec(8, 4, 1, 100, 100, true, nullptr, 300, 10, 0.1f, big) == RBQ_EINVAL);
  EXPECT(dec(8, 4, 1, 100, 100, true, P16, 5, 10, 0.1f, big) == RBQ_EINVAL);
  EXPECT(dec(8, 4, 1, 100, 101, true, P16, 300, 10, 0.1f, big) == RBQ_EINVAL);
  EXPECT(dec(12, 4, 1, 100, 100, true, P16, 300, 10, 0.1f, big) == RBQ_EUNSUPPORTED);
  EXPECT(dec(8, 4, 3, 100, 100, false, nullptr, 0, 0, 0.1f, big) == RBQ_EUNSUPPORTED);
  EXPECT(dec(8, 4, 1, 100, 100, true, P4, 300, 10, 0.1f, big) == RBQ_EINVAL);
  EXPECT(dec(8, 4, 1, imax, imax, true, P16, 300, 10, 0.1f, big) == RBQ_EINVAL);   // 32-bit row offsets
  EXPECT(dec(8, 4, 1, 100, 100, true, P16, 300, 10, 0.1f, 16) == RBQ_EINVAL);
  for (int32_t n : {0, 1, 255, 256, 1023, 1024, 1025, 130816, 1 << 22, imax})
    for (int32_t w : {0, 1, 256, 257, RBQ_MAX_WINDOW, imax}) {
      for (bool tail : {false, true})
        for (bool sparse : {false, true})
          for (bool ragged : {false, true}) {
            const DecodeSplits s = decode_splits(4, 8, n, w, tail, sparse, ragged);
            EXPECT(s.chunk >= 256 && s.chunk <= kDecodeChunk && s.total() >= 1);
          }
      EXPECT(decode_workspace_bytes(4, 32, 8, 128, n, w) > 0);
      EXPECT(rbq_workspace_bytes(RBQ_OP_DECODE_STEP, 4, 32, 8, 128, n, w) > 0);
    }

  // ---- exported sizes and strings
  EXPECT(rbq_workspace_bytes(99, 1, 32, 8, 128, 100, 0) == 0);
  EXPECT(rbq_workspace_bytes(RBQ_OP_TOPP, 0, 32, 8, 128, 100, 0) == 0);
  EXPECT(rbq_workspace_bytes(RBQ_OP_DECODE_STEP, 1, 6, 4, 128, 100, 0) == 0);
  for (int op = RBQ_OP_ENCODE; op <= RBQ_OP_DECODE_STEP; ++op)
    for (int32_t n : {0, 1, 4096, imax}) (void)rbq_workspace_bytes(op, 65535, 16, 1, 128, n, RBQ_MAX_WINDOW);
  EXPECT(rbq_index_bytes(4, 8, 128, 131072) == size_t(4) * 8 * 131072 * 24);
  EXPECT(rbq_index_bytes(65535, 65535, 128, imax) > 0);
  EXPECT(rbq_index_bytes(1, 1, 100, 10) == 0);
  for (int st = -1; st <= 4; ++st) EXPECT(rbq_status_string(rbq_status(st)) != nullptr);
  EXPECT(rbq_version() >= 100);

  if (failures) {
    std::printf("%d checks failed\n", failures);
    return 1;
  }
  std::printf("all host checks passed\n");
  return 0;
}
