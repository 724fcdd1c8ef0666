/*
 * rbq_testing.h -- test hooks of librbq.so, kept apart from the product ABI
 * of rbq.h (which this header includes for its types).
 *
 * The paper's score is exact integer arithmetic on sign codes and INT4 codes
 * that come from floating-point rotations (Section 3.2, Section 3.3). These
 * entry points run the same kernels as the calls of rbq.h and also expose the
 * intermediate values, so that a test can check every integer and sign
 * decision exactly against an independent implementation given the same
 * floating-point inputs. They follow rbq.h's conventions (device pointers
 * owned by the caller, host validation with the same errors, enqueue on
 * `stream`); a serving caller has no use for them.
 *
 *   rbq_encode_keys_debug: as rbq_encode_keys, plus rot_out [B][Hkv][n_new][D]
 *     float = the fp32 rotated centred keys whose signs became the codes.
 *   rbq_quantize_query_debug: as rbq_quantize_query, plus qrot_out [B][Hq][D]
 *     float = the fp32 rotated unit query that was quantised.
 *   rbq_score_ints: ip_out [B][Hq][n] int32 = <c_b, q_u>, pc_out [B][Hkv][n]
 *     int32 = popcount(c_b), computed by the score kernel's integer path;
 *     rbq_score_ints_q8 the same from 8-plane queries (rbq_score_q8's path).
 */
#ifndef RBQ_TESTING_H
#define RBQ_TESTING_H

#include "rbq.h"

#ifdef __cplusplus
extern "C" {
#endif

rbq_status rbq_encode_keys_debug(int32_t batch, int32_t heads_kv, int32_t head_dim,
                                 const void* keys, int32_t keys_dtype, int64_t keys_ld,
                                 int32_t n_new, int32_t offset, int32_t cap,
                                 const float* P, const float* c_q, float* c_k,
                                 uint32_t* codes, float* kfac, uint32_t flags,
                                 float* alpha_out, void* ws, size_t ws_bytes,
                                 float* rot_out, hipStream_t stream);
rbq_status rbq_quantize_query_debug(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                    const float* q, const float* P, const float* c_q, const float* c_k,
                                    uint32_t* qplanes, float* qscal, float* qrot_out,
                                    hipStream_t stream);
rbq_status rbq_score_ints(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                          int32_t n, int32_t cap, const uint32_t* codes, const uint32_t* qplanes,
                          int32_t* ip_out, int32_t* pc_out, hipStream_t stream);
rbq_status rbq_score_ints_q8(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                             int32_t n, int32_t cap, const uint32_t* codes, const uint32_t* qplanes8,
                             int32_t* ip_out, int32_t* pc_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RBQ_TESTING_H */
