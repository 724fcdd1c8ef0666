// Exported C entry points: validate on the host, then enqueue on `stream`.
#include <hip/hip_runtime.h>

#include <mutex>

#include "rbq_internal.h"

using namespace rbq;

namespace {
// rbq_decode_step over either index form: kfac (f, g in fp32) or, when
// kfac16 is non-NULL, the compact index's fp16 factors (kfac unused)
rbq_status decode_step(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                       const float* P, const float* c_q, const float* c_k, const void* K, const void* V,
                       int32_t kv_dtype, int32_t cap, int32_t n, int32_t w, uint32_t* codes, float* kfac,
                       uint16_t* kfac16, int32_t flush, float p, float sm_scale, uint32_t* qplanes, float* qscal,
                       float* scores, int32_t* sel_idx, int32_t* sel_count, float* out, float* lse, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  const void* fac = kfac16 != nullptr ? static_cast<const void*>(kfac16) : kfac;
  rbq_status s = check_heads(batch, heads_q, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if (n < 0 || w < 0 || cap < 0 || int64_t(n) + w > cap) return RBQ_EINVAL;
  const StepWorkspace sw = step_workspace(ws, batch, heads_q, heads_kv, head_dim, n, w);
  if (ws == nullptr || ws_bytes < sw.bytes) return RBQ_EINVAL;
  const size_t elem = kv_dtype == RBQ_BF16 ? 2 : 4;
  const void* K_loc = K ? static_cast<const char*>(K) + size_t(n) * head_dim * elem : nullptr;
  const void* V_loc = V ? static_cast<const char*>(V) + size_t(n) * head_dim * elem : nullptr;
  const size_t dec_bytes = decode_workspace_bytes(batch, heads_q, heads_kv, head_dim, n, w);
  const bool do_flush = flush != 0 && w > 0;
  if ((s = check_quantize(batch, heads_q, heads_kv, head_dim, q, P, c_k, qplanes, qscal)) != RBQ_OK) return s;
  if ((s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, fac, qplanes, qscal, scores)) != RBQ_OK)
    return s;
  if ((s = check_topp(batch, heads_q, n, scores, p, sm_scale, sel_idx, sel_count, sw.topp, sw.topp_bytes)) != RBQ_OK)
    return s;
  if ((s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, true, sel_idx, sel_count,
                        K_loc, V_loc, cap, w, sm_scale, out, sw.decode, dec_bytes)) != RBQ_OK)
    return s;
  if (do_flush && (s = check_encode(batch, heads_kv, head_dim, K_loc, kv_dtype, cap, w, n, cap, P, c_k, codes, fac,
                                    0u, nullptr, 0)) != RBQ_OK)
    return s;

  const int64_t rows = int64_t(batch) * heads_q;
  if (do_flush)
    s = launch_quantize_flush(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, K_loc, kv_dtype, cap, w, n,
                              cap, codes, kfac, stream, nullptr, nullptr, 0, kfac16, head_dim);
  else
    s = launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, nullptr, stream, 4, head_dim);
  if (s != RBQ_OK) return s;
  s = launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes, qscal, scores, nullptr, nullptr, stream,
                   nullptr, kfac16, 4, head_dim);
  if (s != RBQ_OK) return s;
  s = launch_topp(int32_t(rows), n, scores, p, sm_scale, sel_idx, sel_count, sw.topp, stream, sw.masks);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, sel_idx, sel_count, K_loc, V_loc, cap, w,
                       sm_scale, out, lse, sw.decode, true, stream, sw.masks, topp_mask_words(n), nullptr, nullptr,
                       head_dim);
}

// The scratch memory of rbq_decode_step_noalloc: a static device array, one
// copy per GPU at its own address. Host code never passes `scratch` itself (on
// the host the name is only a stand-in for the symbol): the address of the
// current device's copy is looked up once per device and kept in scratch_ptr.
__device__ __align__(256) unsigned char scratch[RBQ_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices];

rbq_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return RBQ_EDEVICE;
  }
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
      (void)hipGetLastError();   // leave no error behind for the next call
      return RBQ_EDEVICE;
    }
    scratch_ptr[dev] = ptr;
  }
  *out = scratch_ptr[dev];
  return RBQ_OK;
}

}  // namespace

extern "C" {

rbq_status rbq_mapped_device_pointer(const void* host_ptr, void** device_ptr) {
  if (host_ptr == nullptr || device_ptr == nullptr) return RBQ_EINVAL;
  *device_ptr = nullptr;
  void* d = nullptr;
  if (hipHostGetDevicePointer(&d, const_cast<void*>(host_ptr), 0) != hipSuccess || d == nullptr) {
    (void)hipGetLastError();   // leave no error behind for the next call
    return RBQ_EDEVICE;
  }
  *device_ptr = d;
  return RBQ_OK;
}

rbq_status rbq_encode_keys_debug(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys,
                                 int32_t keys_dtype, int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap,
                                 const float* P, const float* c_q, float* c_k, uint32_t* codes, float* kfac,
                                 uint32_t flags, float* alpha_out, void* ws, size_t ws_bytes, float* rot_out,
                                 hipStream_t stream) {
  const rbq_status s = check_encode(batch, heads_kv, head_dim, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_k,
                                    codes, kfac, flags, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_encode(batch, heads_kv, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac,
                       flags, alpha_out, ws, rot_out, stream, nullptr, head_dim);
}

rbq_status rbq_encode_keys(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys, int32_t keys_dtype,
                           int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap, const float* P,
                           const float* c_q, float* c_k, uint32_t* codes, float* kfac, uint32_t flags,
                           float* alpha_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  return rbq_encode_keys_debug(batch, heads_kv, head_dim, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_q, c_k,
                               codes, kfac, flags, alpha_out, ws, ws_bytes, nullptr, stream);
}

rbq_status rbq_quantize_query_debug(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                    const float* q, const float* P, const float* c_q, const float* c_k,
                                    uint32_t* qplanes, float* qscal, float* qrot_out, hipStream_t stream) {
  const rbq_status s = check_quantize(batch, heads_q, heads_kv, head_dim, q, P, c_k, qplanes, qscal);
  if (s != RBQ_OK) return s;
  return launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, qrot_out, stream, 4, head_dim);
}

rbq_status rbq_quantize_query(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                              const float* P, const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal,
                              hipStream_t stream) {
  return rbq_quantize_query_debug(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, qplanes, qscal, nullptr,
                                  stream);
}

rbq_status rbq_quantize_query_bits(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                   const float* q, const float* P, const float* c_q, const float* c_k, int32_t bits,
                                   uint32_t* qplanes, float* qscal, hipStream_t stream) {
  if (bits < 1 || bits > 8) return RBQ_EINVAL;
  const rbq_status s = check_quantize(batch, heads_q, heads_kv, head_dim, q, P, c_k, qplanes, qscal);
  if (s != RBQ_OK) return s;
  return launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, nullptr, stream, bits, head_dim);
}

rbq_status rbq_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                     const uint32_t* codes, const float* kfac, const uint32_t* qplanes, const float* qscal,
                     float* scores, hipStream_t stream) {
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes, qscal, scores);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes, qscal, scores, nullptr, nullptr,
                      stream, nullptr, nullptr, 4, head_dim);
}

rbq_status rbq_encode_keys_f16(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys,
                               int32_t keys_dtype, int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap,
                               const float* P, float* c_k, uint32_t* codes, uint16_t* kfac16, uint32_t flags,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  const rbq_status s = check_encode(batch, heads_kv, head_dim, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_k,
                                    codes, kfac16, flags, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_encode(batch, heads_kv, keys, keys_dtype, keys_ld, n_new, offset, cap, P, nullptr, c_k, codes,
                       nullptr, flags, nullptr, ws, nullptr, stream, kfac16, head_dim);
}

rbq_status rbq_score_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                         const uint32_t* codes, const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal,
                         float* scores, hipStream_t stream) {
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac16, qplanes, qscal, scores);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, nullptr, qplanes, qscal, scores, nullptr, nullptr,
                      stream, nullptr, kfac16, 4, head_dim);
}

rbq_status rbq_score_q8(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                        const uint32_t* codes, const float* kfac, const uint32_t* qplanes8, const float* qscal,
                        float* scores, hipStream_t stream) {
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes8, qscal, scores);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes8, qscal, scores, nullptr, nullptr,
                      stream, nullptr, nullptr, 8, head_dim);
}

rbq_status rbq_score_ints_q8(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n,
                             int32_t cap, const uint32_t* codes, const uint32_t* qplanes8, int32_t* ip_out,
                             int32_t* pc_out, hipStream_t stream) {
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, ip_out, qplanes8, pc_out,
                                   ip_out);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, nullptr, qplanes8, nullptr, nullptr, ip_out, pc_out,
                      stream, nullptr, nullptr, 8, head_dim);
}

rbq_status rbq_score_ints(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                          const uint32_t* codes, const uint32_t* qplanes, int32_t* ip_out, int32_t* pc_out,
                          hipStream_t stream) {
  // the integer path reads neither the factors nor the scalars
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, ip_out, qplanes, pc_out, ip_out);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, nullptr, qplanes, nullptr, nullptr, ip_out, pc_out,
                      stream, nullptr, nullptr, 4, head_dim);
}

rbq_status rbq_topp_select(int32_t batch, int32_t heads_q, int32_t n, const float* scores, float p, float sm_scale,
                           int32_t* sel_idx, int32_t* sel_count, void* ws, size_t ws_bytes, hipStream_t stream) {
  const rbq_status s = check_topp(batch, heads_q, n, scores, p, sm_scale, sel_idx, sel_count, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_topp(batch * heads_q, n, scores, p, sm_scale, sel_idx, sel_count, ws, stream);
}

rbq_status rbq_sparse_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                             const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n,
                             const int32_t* sel_idx, const int32_t* sel_count, const void* K_loc, const void* V_loc,
                             int64_t loc_ld, int32_t w, float sm_scale, float* out, float* lse, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  const rbq_status s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, true, sel_idx,
                                    sel_count, K_loc, V_loc, loc_ld, w, sm_scale, out, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, sel_idx, sel_count, K_loc, V_loc, loc_ld,
                       w, sm_scale, out, lse, ws, true, stream, nullptr, 0, nullptr, nullptr, head_dim);
}

rbq_status rbq_dense_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                            const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, const void* K_loc,
                            const void* V_loc, int64_t loc_ld, int32_t w, float sm_scale, float* out, float* lse,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  const rbq_status s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, false, nullptr,
                                    nullptr, K_loc, V_loc, loc_ld, w, sm_scale, out, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, nullptr, nullptr, K_loc, V_loc, loc_ld, w,
                       sm_scale, out, lse, ws, false, stream, nullptr, 0, nullptr, nullptr, head_dim);
}

rbq_status rbq_decode_step(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                           const float* P, const float* c_q, const float* c_k, const void* K, const void* V,
                           int32_t kv_dtype, int32_t cap, int32_t n, int32_t w, uint32_t* codes, float* kfac,
                           int32_t flush, float p, float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                           int32_t* sel_idx, int32_t* sel_count, float* out, float* lse, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  return decode_step(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, kv_dtype, cap, n, w, codes, kfac,
                     nullptr, flush, p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws, ws_bytes,
                     stream);
}

rbq_status rbq_decode_step_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                               const float* P, const float* c_k, const void* K, const void* V, int32_t kv_dtype,
                               int32_t cap, int32_t n, int32_t w, uint32_t* codes, uint16_t* kfac16, int32_t flush,
                               float p, float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                               int32_t* sel_idx, int32_t* sel_count, float* out, float* lse, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  return decode_step(batch, heads_q, heads_kv, head_dim, q, P, nullptr, c_k, K, V, kv_dtype, cap, n, w, codes,
                     nullptr, kfac16, flush, p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws,
                     ws_bytes, stream);
}

rbq_status rbq_decode_step_noalloc(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                   const float* q, const float* P, const float* c_q, const float* c_k, const void* K,
                                   const void* V, int32_t kv_dtype, int32_t cap, int32_t n, int32_t w,
                                   uint32_t* codes, float* kfac, int32_t flush, float p, float sm_scale,
                                   uint32_t* qplanes, float* qscal, float* scores, int32_t* sel_idx,
                                   int32_t* sel_count, float* out, float* lse, hipStream_t stream) {
  const size_t need = rbq_workspace_bytes(RBQ_OP_DECODE_STEP, batch, heads_q, heads_kv, head_dim, n, w);
  if (need > size_t(RBQ_NOALLOC_SCRATCH_BYTES)) return RBQ_EUNSUPPORTED;   // (0: invalid sizes, rejected below)
  void* ws = nullptr;
  const rbq_status s = scratch_address(&ws);
  if (s != RBQ_OK) return s;
  return decode_step(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, kv_dtype, cap, n, w, codes, kfac,
                     nullptr, flush, p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws,
                     size_t(RBQ_NOALLOC_SCRATCH_BYTES), stream);
}

}  // extern "C"

namespace {

// the checks of a ragged call beyond the uniform call's: the per-sequence
// arrays, and room for every sequence's window at its cache tail
rbq_status check_ragged(int32_t n, int32_t w, int32_t cap, const int32_t* seq_n, const int32_t* seq_w) {
  auto misaligned = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; };
  if (seq_n == nullptr || misaligned(seq_n) || (seq_w != nullptr && misaligned(seq_w))) return RBQ_EINVAL;
  if (n < 0 || w < 0 || cap < 0 || int64_t(n) + w > cap) return RBQ_EINVAL;
  return RBQ_OK;
}

rbq_status decode_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                         const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, int32_t w,
                         const int32_t* seq_n, const int32_t* seq_w, bool sparse, const int32_t* sel_idx,
                         const int32_t* sel_count, float sm_scale, float* out, float* lse, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
  rbq_status s = check_ragged(n, w, cap, seq_n, seq_w);
  if (s != RBQ_OK) return s;
  s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, sparse, sel_idx, sel_count, K, V,
                   cap, w, sm_scale, out, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, sel_idx, sel_count, K, V, cap, w,
                       sm_scale, out, lse, ws, sparse, stream, nullptr, 0, seq_n, seq_w, head_dim);
}


// rbq_decode_step_varlen over either index form (kfac16 non-NULL: the compact index)
rbq_status decode_step_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                              const float* P, const float* c_q, const float* c_k, const void* K, const void* V,
                              int32_t kv_dtype, int32_t cap, int32_t n, int32_t w, const int32_t* seq_n,
                              const int32_t* seq_w, uint32_t* codes, float* kfac, uint16_t* kfac16, int32_t flush,
                              const float* seq_p, float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                              int32_t* sel_idx, int32_t* sel_count, float* out, float* lse, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  const void* fac = kfac16 != nullptr ? static_cast<const void*>(kfac16) : kfac;
  rbq_status s = check_heads(batch, heads_q, heads_kv, head_dim);
  if (s != RBQ_OK) return s;
  if ((s = check_ragged(n, w, cap, seq_n, seq_w)) != RBQ_OK) return s;
  if (seq_p == nullptr || (reinterpret_cast<uintptr_t>(seq_p) & 15u) != 0) return RBQ_EINVAL;
  const StepWorkspace sw = step_workspace(ws, batch, heads_q, heads_kv, head_dim, n, w);
  if (ws == nullptr || ws_bytes < sw.bytes) return RBQ_EINVAL;
  const size_t dec_bytes = decode_workspace_bytes(batch, heads_q, heads_kv, head_dim, n, w);
  const bool do_flush = flush != 0 && w > 0;
  if ((s = check_quantize(batch, heads_q, heads_kv, head_dim, q, P, c_k, qplanes, qscal)) != RBQ_OK) return s;
  if ((s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, fac, qplanes, qscal, scores)) != RBQ_OK)
    return s;
  if ((s = check_topp(batch, heads_q, n, scores, 0.5f, sm_scale, sel_idx, sel_count, sw.topp, sw.topp_bytes)) !=
      RBQ_OK)
    return s;
  if ((s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, true, sel_idx, sel_count, K, V,
                        cap, w, sm_scale, out, sw.decode, dec_bytes)) != RBQ_OK)
    return s;
  if (do_flush && (s = check_encode(batch, heads_kv, head_dim, K, kv_dtype, cap, w, n, cap, P, c_k, codes, fac, 0u,
                                    nullptr, 0)) != RBQ_OK)
    return s;

  const int64_t rows = int64_t(batch) * heads_q;
  if (do_flush)   // window rows [seq_n[b], + seq_w[b]) of K into the same index rows
    s = launch_quantize_flush(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, K, kv_dtype, cap, w, 0, cap,
                              codes, kfac, stream, seq_n, seq_w, n, kfac16, head_dim);
  else
    s = launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, nullptr, stream, 4, head_dim);
  if (s != RBQ_OK) return s;
  s = launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes, qscal, scores, nullptr, nullptr, stream,
                   seq_n, kfac16, 4, head_dim);
  if (s != RBQ_OK) return s;
  s = launch_topp(int32_t(rows), n, scores, 0.5f, sm_scale, sel_idx, sel_count, sw.topp, stream, sw.masks,
                  seq_n, seq_p, heads_q);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, sel_idx, sel_count, K, V, cap, w,
                       sm_scale, out, lse, sw.decode, true, stream, sw.masks, topp_mask_words(n), seq_n, seq_w,
                       head_dim);
}

}  // namespace

extern "C" {

rbq_status rbq_score_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n,
                            int32_t cap, const int32_t* seq_n, const uint32_t* codes, const float* kfac,
                            const uint32_t* qplanes, const float* qscal, float* scores, hipStream_t stream) {
  rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes, qscal, scores);
  if (s != RBQ_OK) return s;
  if ((s = check_ragged(n, 0, cap, seq_n, nullptr)) != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes, qscal, scores, nullptr, nullptr,
                      stream, seq_n, nullptr, 4, head_dim);
}

rbq_status rbq_score_varlen_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n,
                                int32_t cap, const int32_t* seq_n, const uint32_t* codes, const uint16_t* kfac16,
                                const uint32_t* qplanes, const float* qscal, float* scores, hipStream_t stream) {
  rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac16, qplanes, qscal, scores);
  if (s != RBQ_OK) return s;
  if ((s = check_ragged(n, 0, cap, seq_n, nullptr)) != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, nullptr, qplanes, qscal, scores, nullptr, nullptr,
                      stream, seq_n, kfac16, 4, head_dim);
}

rbq_status rbq_topp_select_varlen(int32_t batch, int32_t heads_q, int32_t n, const int32_t* seq_n,
                                  const float* scores, const float* seq_p, float sm_scale, int32_t* sel_idx,
                                  int32_t* sel_count, void* ws, size_t ws_bytes, hipStream_t stream) {
  // (p = 0.5 stands for the device values: the workspace is needed whatever they are)
  rbq_status s = check_topp(batch, heads_q, n, scores, 0.5f, sm_scale, sel_idx, sel_count, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  if ((s = check_ragged(n, 0, n, seq_n, nullptr)) != RBQ_OK) return s;
  if (seq_p == nullptr || (reinterpret_cast<uintptr_t>(seq_p) & 15u) != 0) return RBQ_EINVAL;
  return launch_topp(batch * heads_q, n, scores, 0.5f, sm_scale, sel_idx, sel_count, ws, stream, nullptr, seq_n,
                     seq_p, heads_q);
}

rbq_status rbq_sparse_decode_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                                    const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, int32_t w,
                                    const int32_t* seq_n, const int32_t* seq_w, const int32_t* sel_idx,
                                    const int32_t* sel_count, float sm_scale, float* out, float* lse, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  return decode_varlen(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, w, seq_n, seq_w, true, sel_idx,
                       sel_count, sm_scale, out, lse, ws, ws_bytes, stream);
}

rbq_status rbq_dense_decode_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                                   const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, int32_t w,
                                   const int32_t* seq_n, const int32_t* seq_w, float sm_scale, float* out, float* lse,
                                   void* ws, size_t ws_bytes, hipStream_t stream) {
  return decode_varlen(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, w, seq_n, seq_w, false, nullptr,
                       nullptr, sm_scale, out, lse, ws, ws_bytes, stream);
}

rbq_status rbq_decode_step_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                                  const float* P, const float* c_q, const float* c_k, const void* K, const void* V,
                                  int32_t kv_dtype, int32_t cap, int32_t n, int32_t w, const int32_t* seq_n,
                                  const int32_t* seq_w, uint32_t* codes, float* kfac, int32_t flush,
                                  const float* seq_p, float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                                  int32_t* sel_idx, int32_t* sel_count, float* out, float* lse, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  return decode_step_varlen(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, kv_dtype, cap, n, w, seq_n, seq_w,
                            codes, kfac, nullptr, flush, seq_p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count,
                            out, lse, ws, ws_bytes, stream);
}

rbq_status rbq_decode_step_varlen_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                      const float* q, const float* P, const float* c_k, const void* K, const void* V,
                                      int32_t kv_dtype, int32_t cap, int32_t n, int32_t w, const int32_t* seq_n,
                                      const int32_t* seq_w, uint32_t* codes, uint16_t* kfac16, int32_t flush,
                                      const float* seq_p, float sm_scale, uint32_t* qplanes, float* qscal,
                                      float* scores, int32_t* sel_idx, int32_t* sel_count, float* out, float* lse,
                                      void* ws, size_t ws_bytes, hipStream_t stream) {
  return decode_step_varlen(batch, heads_q, heads_kv, head_dim, q, P, nullptr, c_k, K, V, kv_dtype, cap, n, w, seq_n,
                            seq_w, codes, nullptr, kfac16, flush, seq_p, sm_scale, qplanes, qscal, scores, sel_idx,
                            sel_count, out, lse, ws, ws_bytes, stream);
}

}  // extern "C"
