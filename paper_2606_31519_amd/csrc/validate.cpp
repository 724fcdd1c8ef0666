// Host-side argument checks and workspace sizing. No HIP calls: everything
// here runs (and is tested) without a GPU.
#include <cmath>
#include <cstdint>

#include "rbq_internal.h"

namespace rbq {

namespace {
constexpr int64_t kMaxRows = int64_t(1) << 31;
// a required device pointer: present, and 16-byte aligned (the kernels use 16-byte vector loads)
bool bad_ptr(const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }
}  // namespace

rbq_status check_heads(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim) {
  if (batch <= 0 || heads_q <= 0 || heads_kv <= 0 || head_dim <= 0) return RBQ_EINVAL;
  if (heads_q % heads_kv != 0) return RBQ_EINVAL;
  if (head_dim % 32 != 0) return RBQ_EINVAL;
  if (int64_t(batch) * heads_q > 65535 * int64_t(1024)) return RBQ_EINVAL;
  if (int64_t(batch) * heads_kv > 65535) return RBQ_EINVAL;   // grid.y of the per-(b, kv-head) kernels
  if (heads_q / heads_kv > 16) return RBQ_EUNSUPPORTED;       // GQA group size handled by the kernels
  if (head_dim != kHeadDim && head_dim != 64) return RBQ_EUNSUPPORTED;   // D = 128, and 64 for the uniform calls
  return RBQ_OK;
}

size_t encode_workspace_bytes(int32_t batch, int32_t heads_kv, int32_t head_dim, int32_t n_new) {
  if (batch <= 0 || heads_kv <= 0 || head_dim <= 0 || n_new < 0) return 0;
  const int64_t chunks = (int64_t(n_new) + kCentroidChunk - 1) / kCentroidChunk;
  return align_up(size_t(batch) * heads_kv * (chunks > 0 ? chunks : 1) * head_dim * sizeof(float), 256);
}

rbq_status check_encode(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys, int32_t keys_dtype,
                        int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap, const float* P,
                        const float* c_k, const uint32_t* codes, const void* kfac, uint32_t flags,
                        const void* ws, size_t ws_bytes) {
  rbq_status s = check_heads(batch, heads_kv, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if (keys_dtype != RBQ_F32 && keys_dtype != RBQ_BF16) return RBQ_EUNSUPPORTED;
  if (n_new < 0 || offset < 0 || cap < 0 || keys_ld < n_new || keys_ld >= kMaxRows) return RBQ_EINVAL;
  if (int64_t(offset) + n_new > cap) return RBQ_EINVAL;
  if (flags & ~RBQ_ENCODE_SET_CENTROID) return RBQ_EINVAL;
  if ((flags & RBQ_ENCODE_SET_CENTROID) && n_new == 0) return RBQ_EINVAL;   // the mean of no keys
  if (bad_ptr(P) || bad_ptr(c_k) || bad_ptr(codes) || bad_ptr(kfac)) return RBQ_EINVAL;
  if (n_new > 0 && bad_ptr(keys)) return RBQ_EINVAL;
  if (flags & RBQ_ENCODE_SET_CENTROID) {
    if (bad_ptr(ws) || ws_bytes < encode_workspace_bytes(batch, heads_kv, head_dim, n_new)) return RBQ_EINVAL;
  }
  return RBQ_OK;
}

rbq_status check_quantize(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                          const float* P, const float* c_k, const uint32_t* qplanes, const float* qscal) {
  rbq_status s = check_heads(batch, heads_q, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if (bad_ptr(q) || bad_ptr(P) || bad_ptr(c_k) || bad_ptr(qplanes) || bad_ptr(qscal)) return RBQ_EINVAL;
  return RBQ_OK;
}

rbq_status check_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                       const uint32_t* codes, const void* kfac, const uint32_t* qplanes, const void* qscal,
                       const void* out) {
  rbq_status s = check_heads(batch, heads_q, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if (n < 0 || cap < 0 || n > cap) return RBQ_EINVAL;
  if (n > 0 && (bad_ptr(codes) || bad_ptr(kfac) || bad_ptr(qplanes) || bad_ptr(qscal) || bad_ptr(out)))
    return RBQ_EINVAL;
  return RBQ_OK;
}

ToppPlan topp_plan(int32_t n) {
  const int64_t subs = n > 0 ? (int64_t(n) + kSelSub - 1) / kSelSub : 1;
  ToppPlan pl;
  pl.spb = int32_t((subs + kSelMaxParts - 1) / kSelMaxParts);
  pl.parts = int32_t((subs + pl.spb - 1) / pl.spb);
  return pl;
}

ToppWorkspace topp_workspace(void* base, int64_t rows, int32_t n) {
  const ToppPlan pl = topp_plan(n);
  ToppWorkspace w{};
  size_t off = 0;
  char* b = static_cast<char*>(base);
  w.part1 = reinterpret_cast<unsigned char*>(b + off);
  off = align_up(off + size_t(rows) * pl.parts * kSelPart1Bytes, 256);
  w.part2 = reinterpret_cast<unsigned char*>(b + off);
  off = align_up(off + size_t(rows) * pl.parts * kSelPart2Bytes, 256);
  w.state = reinterpret_cast<uint32_t*>(b + off);
  off = align_up(off + size_t(rows) * kSelStateWords * sizeof(uint32_t), 256);
  w.bytes = off;
  return w;
}

rbq_status check_topp(int32_t batch, int32_t heads_q, int32_t n, const float* scores, float p, float sm_scale,
                      const int32_t* sel_idx, const int32_t* sel_count, const void* ws, size_t ws_bytes) {
  if (batch <= 0 || heads_q <= 0 || n < 0) return RBQ_EINVAL;
  if (int64_t(batch) * heads_q > 65535) return RBQ_EINVAL;
  // a row's softmax masses are summed as 2^-40 fixed-point integers of at most
  // 2^40 each in 64 bits: exact only below 2^24 keys per row
  if (n >= kToppMaxKeys) return RBQ_EUNSUPPORTED;
  if (!(p > 0.0f) || !(p <= 1.0f)) return RBQ_EINVAL;                  // also rejects NaN
  if (!std::isfinite(sm_scale) || !(sm_scale > 0.0f)) return RBQ_EINVAL;
  if (bad_ptr(sel_count)) return RBQ_EINVAL;
  if (n > 0 && (bad_ptr(scores) || bad_ptr(sel_idx))) return RBQ_EINVAL;
  if (n > 0 && p < 1.0f) {
    if (bad_ptr(ws) || ws_bytes < topp_workspace(nullptr, int64_t(batch) * heads_q, n).bytes) return RBQ_EINVAL;
  }
  return RBQ_OK;
}

DecodeSplits decode_splits(int32_t batch, int32_t heads_kv, int32_t n, int32_t w, bool tail_window, bool sparse,
                           bool ragged) {
  DecodeSplits s;
  s.fold_s0 = 0;
  s.fold_wq = 0;
  // halve the chunk until the grid has kDecodeMinBlocks blocks or the chunk is 256
  const int64_t groups = int64_t(batch) * heads_kv;
  s.chunk = kDecodeChunk;
  while (s.chunk > 256 && groups * ((int64_t(n) + s.chunk - 1) / s.chunk) < kDecodeMinBlocks) s.chunk /= 2;
  s.idx_splits = n > 0 ? int32_t((int64_t(n) + s.chunk - 1) / s.chunk) : 0;
  s.win_splits = w > 0 ? int32_t((int64_t(w) + kDecodeWinChunk - 1) / kDecodeWinChunk) : 0;
  if (tail_window && s.idx_splits > 0 && w > 0) {
    if (ragged) {
      const int cap = kDecodeListCap - s.chunk;   // window rows a split's list can still take
      if ((int64_t(w) + cap - 1) / cap <= s.idx_splits) {
        s.fold_wq = cap;
        s.win_splits = 0;
      }
    } else if (sparse) {
      const int64_t wq = (int64_t(w) + s.idx_splits - 1) / s.idx_splits;
      if (wq <= kDecodeFoldMax) {
        s.fold_wq = int32_t(wq);
        s.win_splits = 0;
      }
    } else if (int64_t(n) - int64_t(s.idx_splits - 1) * s.chunk + w <= s.chunk) {
      s.fold_s0 = s.idx_splits - 1;
      s.fold_wq = w;
      s.win_splits = 0;
    }
  }
  if (s.total() == 0) s.win_splits = 1;   // one empty split keeps the combine step uniform
  return s;
}

size_t decode_workspace_bytes(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n,
                              int32_t w) {
  if (batch <= 0 || heads_q <= 0 || heads_kv <= 0 || head_dim <= 0 || n < 0 || w < 0) return 0;
  const DecodeSplits s = decode_splits(batch, heads_kv, n, w);
  return align_up(size_t(batch) * heads_q * s.total() * (head_dim + 2) * sizeof(float), 256);
}

rbq_status check_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                        const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, bool sparse,
                        const int32_t* sel_idx, const int32_t* sel_count, const void* K_loc, const void* V_loc,
                        int64_t loc_ld, int32_t w, float sm_scale, const float* out, const void* ws,
                        size_t ws_bytes) {
  rbq_status s = check_heads(batch, heads_q, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if (kv_dtype != RBQ_F32 && kv_dtype != RBQ_BF16) return RBQ_EUNSUPPORTED;
  const int32_t G = heads_q / heads_kv;
  if (G & (G - 1)) return RBQ_EUNSUPPORTED;   // the decode kernels are built for G in {1, 2, 4, 8, 16}
  if (n < 0 || cap < 0 || n > cap || w < 0 || w > RBQ_MAX_WINDOW) return RBQ_EINVAL;
  if (!std::isfinite(sm_scale) || !(sm_scale > 0.0f)) return RBQ_EINVAL;
  if (bad_ptr(q) || bad_ptr(out)) return RBQ_EINVAL;
  if (n > 0 && (bad_ptr(K) || bad_ptr(V))) return RBQ_EINVAL;
  if (sparse && (bad_ptr(sel_count) || (n > 0 && bad_ptr(sel_idx)))) return RBQ_EINVAL;
  if (w > 0 && (bad_ptr(K_loc) || bad_ptr(V_loc) || loc_ld < w || loc_ld >= kMaxRows)) return RBQ_EINVAL;
  // rows of one (sequence, KV head) are addressed with 32-bit byte offsets
  const int64_t row_bytes = int64_t(head_dim) * (kv_dtype == RBQ_BF16 ? 2 : 4);
  if (int64_t(n) * row_bytes >= (int64_t(1) << 31) || int64_t(w) * row_bytes >= (int64_t(1) << 31)) return RBQ_EINVAL;
  if (bad_ptr(ws) || ws_bytes < decode_workspace_bytes(batch, heads_q, heads_kv, head_dim, n, w)) return RBQ_EINVAL;
  return RBQ_OK;
}

// Keys per lane of the score kernel: enough blocks to cover the 256 CUs
// several times over, as many keys in flight per lane as that allows.
int score_keys_per_lane(int32_t batch, int32_t heads_kv, int32_t n) {
  const int64_t kv_keys = int64_t(batch) * heads_kv * n;
  if (kv_keys >= int64_t(kScoreThreads) * 4 * 2048) return 4;
  if (kv_keys >= int64_t(kScoreThreads) * 2 * 1024) return 2;
  return 1;
}
int topp_mask_words(int32_t n) {
  return n > 0 ? int((int64_t(n) + kSelSub - 1) / kSelSub * (kSelSub / 64)) : 0;
}

StepWorkspace step_workspace(void* base, int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                             int32_t n, int32_t w) {
  StepWorkspace s{};
  const int64_t rows = int64_t(batch) * heads_q;
  char* b = static_cast<char*>(base);
  size_t off = 0;
  s.decode = b + off;
  off = align_up(off + decode_workspace_bytes(batch, heads_q, heads_kv, head_dim, n, w), 256);
  s.topp = b + off;
  s.topp_bytes = topp_workspace(nullptr, rows, n).bytes;
  off = align_up(off + s.topp_bytes, 256);
  s.masks = reinterpret_cast<unsigned long long*>(b + off);
  off = align_up(off + size_t(rows) * topp_mask_words(n) * sizeof(unsigned long long), 256);
  s.bytes = off;
  return s;
}

}  // namespace rbq

extern "C" {

size_t rbq_workspace_bytes(int32_t op, int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                           int32_t n, int32_t w) {
  if (batch <= 0 || heads_q <= 0 || heads_kv <= 0 || head_dim <= 0 || n < 0 || w < 0) return 0;
  switch (op) {
    case RBQ_OP_ENCODE:
      return rbq::encode_workspace_bytes(batch, heads_kv, head_dim, n);
    case RBQ_OP_TOPP:
      return rbq::topp_workspace(nullptr, int64_t(batch) * heads_q, n).bytes;
    case RBQ_OP_SPARSE_DECODE:
    case RBQ_OP_DENSE_DECODE:
      return rbq::decode_workspace_bytes(batch, heads_q, heads_kv, head_dim, n, w);
    case RBQ_OP_DECODE_STEP:
      if (heads_q % heads_kv != 0) return 0;
      return rbq::step_workspace(nullptr, batch, heads_q, heads_kv, head_dim, n, w).bytes;
    default:
      return 0;
  }
}

size_t rbq_index_bytes(int32_t batch, int32_t heads_kv, int32_t head_dim, int32_t cap) {
  if (batch <= 0 || heads_kv <= 0 || head_dim <= 0 || cap < 0 || head_dim % 32 != 0) return 0;
  return size_t(batch) * heads_kv * size_t(cap) * (size_t(head_dim) / 8 + 2 * sizeof(float));
}

const char* rbq_status_string(rbq_status s) {
  switch (s) {
    case RBQ_OK: return "ok";
    case RBQ_EINVAL: return "invalid argument";
    case RBQ_EUNSUPPORTED: return "unsupported shape, dtype or size";
    case RBQ_EDEVICE: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t rbq_version(void) { return 100; }

}  // extern "C"
