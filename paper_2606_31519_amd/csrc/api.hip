// Exported C entry points: validate on the host, then enqueue on `stream`.
#include <hip/hip_runtime.h>

#include "rbq_internal.h"

using namespace rbq;

extern "C" {

rbq_status rbq_encode_keys_debug(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys,
                                 int32_t keys_dtype, int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap,
                                 const float* P, const float* c_q, float* c_k, uint32_t* codes, float* kfac,
                                 uint32_t flags, float* alpha_out, void* ws, size_t ws_bytes, float* rot_out,
                                 hipStream_t stream) {
  const rbq_status s = check_encode(batch, heads_kv, head_dim, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_k,
                                    codes, kfac, flags, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_encode(batch, heads_kv, keys, keys_dtype, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac,
                       flags, alpha_out, ws, rot_out, stream);
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
  return launch_quantize(batch, heads_q, heads_kv, q, P, c_q, c_k, qplanes, qscal, qrot_out, stream);
}

rbq_status rbq_quantize_query(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                              const float* P, const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal,
                              hipStream_t stream) {
  return rbq_quantize_query_debug(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, qplanes, qscal, nullptr,
                                  stream);
}

rbq_status rbq_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                     const uint32_t* codes, const float* kfac, const uint32_t* qplanes, const float* qscal,
                     float* scores, hipStream_t stream) {
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes, qscal, scores);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, kfac, qplanes, qscal, scores, nullptr, nullptr,
                      stream);
}

rbq_status rbq_score_ints(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                          const uint32_t* codes, const uint32_t* qplanes, int32_t* ip_out, int32_t* pc_out,
                          hipStream_t stream) {
  // the integer path reads neither the factors nor the scalars
  const rbq_status s = check_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, ip_out, qplanes, pc_out, ip_out);
  if (s != RBQ_OK) return s;
  return launch_score(batch, heads_q, heads_kv, n, cap, codes, nullptr, qplanes, nullptr, nullptr, ip_out, pc_out,
                      stream);
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
                       w, sm_scale, out, lse, ws, true, stream);
}

rbq_status rbq_dense_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                            const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, const void* K_loc,
                            const void* V_loc, int64_t loc_ld, int32_t w, float sm_scale, float* out, float* lse,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  const rbq_status s = check_decode(batch, heads_q, heads_kv, head_dim, q, K, V, kv_dtype, cap, n, false, nullptr,
                                    nullptr, K_loc, V_loc, loc_ld, w, sm_scale, out, ws, ws_bytes);
  if (s != RBQ_OK) return s;
  return launch_decode(batch, heads_q, heads_kv, q, K, V, kv_dtype, cap, n, nullptr, nullptr, K_loc, V_loc, loc_ld, w,
                       sm_scale, out, lse, ws, false, stream);
}

}  // extern "C"
