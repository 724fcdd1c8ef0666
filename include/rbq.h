/*
 * rbq.h -- RaBitQCache decode hot path on AMD MI355X (gfx950), C ABI.
 *
 * RaBitQCache ("Rotated Binary Quantization for KVCache in Long Context LLM
 * Inference") estimates the attention score of every cached key from a
 * randomly rotated 1-bit key code and a 4-bit rotated query, keeps the
 * smallest set of keys holding a fraction p of the estimated attention
 * (adaptive Top-p), and runs exact attention over those keys plus a local
 * window of recent keys.
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers owned by the caller unless marked (host),
 *     16-byte aligned (RBQ_EINVAL otherwise).
 *     The library never allocates, frees or synchronises: each call checks
 *     its arguments on the host, enqueues kernels on `stream` and returns.
 *   - Shapes: B = batch, Hq = query heads, Hkv = KV heads (Hq % Hkv == 0,
 *     G = Hq / Hkv; query head h reads KV head h / G), D = head_dim.
 *     Every call takes D = 128 or D = 64; any other D: RBQ_EUNSUPPORTED.
 *   - Layouts are row-major and contiguous:
 *       codes [B][Hkv][cap][D/32] uint32: dimension d of a key's sign code is
 *             bit d % 32 of word d / 32; the bit is 1 iff the d-th component
 *             of P^T (k - c_k) is > 0 (Section 3.2, Appendix A.2).
 *       kfac  [B][Hkv][cap][2] float: { f = ||k - c_k|| / alpha', g = <c_q, k - c_k> }
 *             where alpha' = sum_j |(P^T (k - c_k))_j| / ||k - c_k|| is the
 *             correction factor <c_bar', P^T k_c> of Appendix A.2 (the paper-
 *             unit alpha is alpha' / sqrt(D)); f = 0 when k == c_k.
 *       c_k, c_q [B][Hkv][D] float: key and query centroids per KV group.
 *       P     [D][D] float: the random orthogonal rotation; r = P^T x is the
 *             row vector x * P (Section 3.1).
 *   - The rotation is applied as r[j] = sum_d P[d][j] x[d] for keys and queries.
 *   - Errors: RBQ_EINVAL for a bad shape, a null required pointer, n > cap,
 *     offset + n_new > cap, p outside (0, 1], a non-finite or non-positive
 *     scale, or a workspace smaller than rbq_workspace_bytes(); nothing is
 *     enqueued then. RBQ_EDEVICE when the HIP runtime reports an error after
 *     the launch (the queue may then hold part of the call's kernels).
 *   - Calls are stateless and thread-safe. Results are bitwise identical run
 *     to run (no floating-point atomics on any output path).
 */
#ifndef RBQ_H
#define RBQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;
typedef struct ihipStream_t* hipStream_t;

typedef enum rbq_status {
  RBQ_OK = 0,
  RBQ_EINVAL = 1,
  RBQ_EUNSUPPORTED = 2,
  RBQ_EDEVICE = 3
} rbq_status;

typedef enum rbq_dtype { RBQ_F32 = 0, RBQ_BF16 = 1 } rbq_dtype;

/* flags of rbq_encode_keys */
#define RBQ_ENCODE_SET_CENTROID 1u

/* op ids of rbq_workspace_bytes */
#define RBQ_OP_ENCODE 1
#define RBQ_OP_TOPP 2
#define RBQ_OP_SPARSE_DECODE 3
#define RBQ_OP_DENSE_DECODE 4
#define RBQ_OP_DECODE_STEP 5

#define RBQ_QSCAL_STRIDE 8   /* floats per query head in qscal */
#define RBQ_MAX_WINDOW 4096  /* largest local window accepted by the decode calls */

/*
 * rbq_encode_keys -- index construction, Algorithm 1 (Section 3.2) and
 * Appendix A.2.
 *
 * Encodes n_new keys per (b, kv-head): keys[b][h][i][:] for i in [0, n_new),
 * where `keys` holds blocks of `keys_ld` rows per (b, kv-head) (keys_ld >= n_new)
 * in dtype `keys_dtype` (RBQ_F32 or RBQ_BF16). The codes and factors are
 * written at rows [offset, offset + n_new) of `codes` / `kfac` (capacity cap
 * rows per (b, kv-head)).
 *   flags & RBQ_ENCODE_SET_CENTROID: c_k[b][h] is first set to the mean of
 *     these keys (the prefill centroid); otherwise the existing c_k is read
 *     and reused (the lazy update of Section 3.4 appends with the prefill
 *     centroid).
 *   c_q: query centroid per KV group, or NULL for zeros.
 *   alpha_out: NULL, or [B][Hkv][n_new] floats receiving the paper-unit alpha.
 *   ws: workspace of at least rbq_workspace_bytes(RBQ_OP_ENCODE, B, Hkv, Hkv, D, n_new, 0)
 *     bytes (only used with RBQ_ENCODE_SET_CENTROID; may be NULL otherwise).
 */
rbq_status rbq_encode_keys(int32_t batch, int32_t heads_kv, int32_t head_dim,
                           const void* keys, int32_t keys_dtype, int64_t keys_ld,
                           int32_t n_new, int32_t offset, int32_t cap,
                           const float* P, const float* c_q, float* c_k,
                           uint32_t* codes, float* kfac, uint32_t flags,
                           float* alpha_out, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/*
 * rbq_quantize_query -- query pre-processing and INT4 quantisation,
 * Algorithm 2 step 1, Section 3.3 (Query Quantization) and Appendix A.3.2.
 *
 * Per query head: y = q - c_q, A = ||y||, u = y / A (0 if A == 0),
 * q' = P^T u, [q_l, q_r] = range of q', Delta = (q_r - q_l) / 15,
 * q_u = clamp(floor((q' - q_l) / Delta + 1/2), 0, 15) (all 0 if Delta == 0),
 * evaluated in IEEE fp32 with correctly rounded division.
 *   q       [B][Hq][D] float
 *   c_q     [B][Hkv][D] float or NULL (zeros); c_k [B][Hkv][D] float
 *   qplanes [B][Hq][4][D/32] uint32 out: bit-plane j holds bit j of every
 *           code, packed like the key codes.
 *   qscal   [B][Hq][8] float out: { q_l, Delta, S_u = sum q_u, A, B0 = <q, c_k>, q_r, 0, 0 }.
 */
rbq_status rbq_quantize_query(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                              const float* q, const float* P, const float* c_q, const float* c_k,
                              uint32_t* qplanes, float* qscal, hipStream_t stream);

/*
 * rbq_quantize_query_bits -- rbq_quantize_query with B_q = `bits` quantisation
 * bits instead of 4 (Theorem A.2 bounds the estimator's error for any B_q;
 * Section 3.3 uses 4): Delta = (q_r - q_l) / (2^bits - 1), codes in
 * [0, 2^bits - 1], bit-planes j >= bits zero. bits in [1, 8], RBQ_EINVAL
 * otherwise.
 *   bits 1..4: qplanes [B][Hq][4][D/32] as rbq_quantize_query writes it; the
 *     output feeds rbq_score (and every call that reads qplanes) unchanged;
 *     bits = 4 gives rbq_quantize_query's results bitwise.
 *   bits 5..8: qplanes [B][Hq][8][D/32], eight bit-planes per head, read by
 *     rbq_score_q8.
 */
rbq_status rbq_quantize_query_bits(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                   const float* q, const float* P, const float* c_q, const float* c_k,
                                   int32_t bits, uint32_t* qplanes, float* qscal, hipStream_t stream);

/*
 * rbq_score -- the binary x INT4 score estimate for every indexed key,
 * Algorithm 2 step 2 with Eq. estimator_core, Eqs. kc_bar_dot_q_c2 /
 * estk_cq_c (Appendix A.3.2) and Eq. decomposition (Section 3.1).
 *
 * For query head h (row r = b*Hq + h) and key i < n of KV head h / G:
 *   ip = <c_b, q_u> = sum_j 2^j popcount(code_i AND plane_j),  pc = popcount(code_i)
 *   X  = 2 Delta ip + 2 q_l pc - Delta S_u - D q_l           (= <c_bar', q_bar>)
 *   S  = A * f_i * X + B0 + g_i                               (the estimate of <q, k_i>)
 *   scores [B][Hq][n] float out (row stride n).
 * The integer parts are exact; S is fp32.
 */
rbq_status rbq_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                     int32_t n, int32_t cap, const uint32_t* codes, const float* kfac,
                     const uint32_t* qplanes, const float* qscal, float* scores,
                     hipStream_t stream);

/*
 * rbq_score_q8 -- rbq_score for queries quantised to up to 8 bits
 * (rbq_quantize_query_bits with bits 5..8, Theorem A.2): qplanes8 is
 * [B][Hq][8][D/32], ip = sum_{j < 8} 2^j popcount(code_i AND plane_j), the
 * rest as in rbq_score. (The fused step and the ragged calls read 4-bit
 * queries only.)
 */
rbq_status rbq_score_q8(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                        int32_t n, int32_t cap, const uint32_t* codes, const float* kfac,
                        const uint32_t* qplanes8, const float* qscal, float* scores,
                        hipStream_t stream);

/*
 * rbq_topp_select -- adaptive Top-p selection, Algorithm 2 step 3 and
 * Section 4.1 (the function of Algorithm 3, computed by a radix threshold
 * select instead of a ternary search).
 *
 * For each row r of scores [B*Hq][n]: pi = softmax(scores[r] * sm_scale);
 * the selected set is the smallest prefix of the keys ranked by score whose
 * mass is >= p, extended to every key whose score equals the last one's.
 * p == 1 selects every key. Masses are accumulated in 2^-40 fixed point from
 * fp32 exponentials, so the set may differ from an exact-arithmetic one only
 * where the cumulative mass passes p within ~1e-6.
 *   p (host) in (0, 1]; sm_scale (host) > 0, usually 1/sqrt(D).
 *   n < 2^24 (16,777,216) keys per row: the masses of a row are summed as
 *     64-bit integers of up to 2^40 each; a longer row gives RBQ_EUNSUPPORTED.
 *   sel_idx   [B][Hq][n] int32 out: the first sel_count[r] entries of row r are
 *             the selected key indices in ascending order; the rest is unspecified.
 *   sel_count [B][Hq] int32 out.
 *   ws: at least rbq_workspace_bytes(RBQ_OP_TOPP, B, Hq, Hkv, D, n, 0) bytes.
 */
rbq_status rbq_topp_select(int32_t batch, int32_t heads_q, int32_t n, const float* scores,
                           float p, float sm_scale, int32_t* sel_idx, int32_t* sel_count,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * rbq_sparse_decode -- hybrid sparse attention, Algorithm 2 step 4 and
 * Section 3.4 (Lazy Decode Updates).
 *
 * For query head h: T = { indexed rows sel_idx[r][0 .. sel_count[r]) } u { all w
 * window rows }; out = sum_t softmax(<q, k_t> * sm_scale)_t v_t over T,
 * accumulated in fp32 (outputs are fp32).
 *   q        [B][Hq][D] float
 *   K, V     [B][Hkv][cap][D] in kv_dtype (RBQ_BF16 or RBQ_F32); rows < n indexed
 *   sel_idx, sel_count: as written by rbq_topp_select (row stride n)
 *   K_loc, V_loc: the local window, blocks of loc_ld rows per (b, kv-head),
 *            rows [0, w) used, same dtype (NULL allowed when w == 0). The tail
 *            of the cache is passed as K_loc = K + n*D with loc_ld = cap.
 *   out      [B][Hq][D] float; lse [B][Hq] float or NULL: natural-log
 *            log-sum-exp of the scaled logits over T (-inf and out = 0 if T is empty).
 *   ws: at least rbq_workspace_bytes(RBQ_OP_SPARSE_DECODE, B, Hq, Hkv, D, n, w) bytes.
 */
rbq_status rbq_sparse_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                             const float* q, const void* K, const void* V, int32_t kv_dtype,
                             int32_t cap, int32_t n, const int32_t* sel_idx, const int32_t* sel_count,
                             const void* K_loc, const void* V_loc, int64_t loc_ld, int32_t w,
                             float sm_scale, float* out, float* lse,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * rbq_dense_decode -- full attention over all n indexed rows plus the w window
 * rows, the baseline the paper compares decode latency against (Section 5.3).
 * Same arguments and outputs as rbq_sparse_decode without the selection.
 *   ws: at least rbq_workspace_bytes(RBQ_OP_DENSE_DECODE, B, Hq, Hkv, D, n, w) bytes.
 */
rbq_status rbq_dense_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                            const float* q, const void* K, const void* V, int32_t kv_dtype,
                            int32_t cap, int32_t n, const void* K_loc, const void* V_loc,
                            int64_t loc_ld, int32_t w, float sm_scale, float* out, float* lse,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * rbq_decode_step -- one decode step of Algorithm 2 (steps 1 to 4) followed by
 * the lazy index update of Section 3.4, in one call. The local window is the
 * tail of the cache: rows [n, n + w) of K and V (n + w <= cap). The outputs
 * are bitwise identical to those of the sequence
 *   rbq_quantize_query(B, Hq, Hkv, D, q, P, c_q, c_k, qplanes, qscal)
 *   rbq_score(B, Hq, Hkv, D, n, cap, codes, kfac, qplanes, qscal, scores)
 *   rbq_topp_select(B, Hq, n, scores, p, sm_scale, sel_idx, sel_count)
 *   rbq_sparse_decode(B, Hq, Hkv, D, q, K, V, kv_dtype, cap, n, sel_idx, sel_count,
 *                     K + n*D, V + n*D, cap, w, sm_scale, out, lse)
 *   if (flush) rbq_encode_keys(B, Hkv, D, K + n*D, kv_dtype, cap, w, n, cap,
 *                              P, c_q, c_k, codes, kfac, 0, NULL)
 * (K + n*D: row n of every (b, kv-head) block, rows `cap` apart), with fewer
 * launches: the query quantisation and the window encode share one launch
 * (the encode writes index rows [n, n + w), which nothing else in the step
 * reads), and the selection also writes per-head bitmaps of the selected
 * keys, from which the sparse attention builds its row lists without
 * searching sel_idx. Every argument means what it means in those calls; qplanes, qscal,
 * scores, sel_idx and sel_count are written as they would be.
 *   flush: nonzero to run the window encode (codes / kfac rows [n, n + w)).
 *   ws: at least rbq_workspace_bytes(RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, n, w) bytes.
 */
rbq_status rbq_decode_step(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                           const float* q, const float* P, const float* c_q, const float* c_k,
                           const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n,
                           int32_t w, uint32_t* codes, float* kfac, int32_t flush, float p,
                           float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                           int32_t* sel_idx, int32_t* sel_count, float* out, float* lse,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Ragged batches -- the score, selection, attention and fused-step calls for a
 * batch whose sequences hold different numbers of keys and use different p,
 * as a serving batch does (Algorithm 2 run per sequence; Section 3.4 for the
 * window). Every layout is the uniform call's, with n and w the LARGEST counts:
 * n is the row stride of scores and sel_idx, and n and w size the launches.
 * Sequence b (query heads b*Hq .. b*Hq + Hq - 1) uses
 *   seq_n [B] int32 (device): its indexed keys, rows [0, seq_n[b]) of the index
 *         and of K / V, clamped to [0, n];
 *   seq_w [B] int32 (device) or NULL: its window rows, which are its cache
 *         tail, rows [seq_n[b], seq_n[b] + seq_w[b]) of K / V, clamped to
 *         [0, w]; NULL gives every sequence w rows;
 *   seq_p [B] float (device): its p. A value >= 1 selects every key; a value
 *         <= 0 or NaN acts as the smallest positive p (the top key and its ties).
 * The results for sequence b are those of the uniform call with B = 1, n =
 * seq_n[b], w = seq_w[b] and p = seq_p[b] (bitwise for scores and selections).
 * Entries of scores and sel_idx past a sequence's count are unspecified. The
 * device counts are not checked on the host: n + w <= cap keeps every row in
 * the cache. Workspaces: as for the uniform op with the same n and w.
 */
rbq_status rbq_score_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                            int32_t n, int32_t cap, const int32_t* seq_n, const uint32_t* codes,
                            const float* kfac, const uint32_t* qplanes, const float* qscal, float* scores,
                            hipStream_t stream);
rbq_status rbq_topp_select_varlen(int32_t batch, int32_t heads_q, int32_t n, const int32_t* seq_n,
                                  const float* scores, const float* seq_p, float sm_scale,
                                  int32_t* sel_idx, int32_t* sel_count, void* ws, size_t ws_bytes,
                                  hipStream_t stream);
/* ws: rbq_workspace_bytes(RBQ_OP_SPARSE_DECODE / RBQ_OP_DENSE_DECODE, B, Hq, Hkv, D, n, w). */
rbq_status rbq_sparse_decode_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                    const float* q, const void* K, const void* V, int32_t kv_dtype,
                                    int32_t cap, int32_t n, int32_t w, const int32_t* seq_n,
                                    const int32_t* seq_w, const int32_t* sel_idx, const int32_t* sel_count,
                                    float sm_scale, float* out, float* lse, void* ws, size_t ws_bytes,
                                    hipStream_t stream);
rbq_status rbq_dense_decode_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                   const float* q, const void* K, const void* V, int32_t kv_dtype,
                                   int32_t cap, int32_t n, int32_t w, const int32_t* seq_n,
                                   const int32_t* seq_w, float sm_scale, float* out, float* lse,
                                   void* ws, size_t ws_bytes, hipStream_t stream);
/* The fused step of a ragged batch: rbq_decode_step with the calls above; the
 * flush encodes each sequence's window rows into index rows [seq_n[b],
 * seq_n[b] + seq_w[b]). ws: rbq_workspace_bytes(RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, n, w). */
rbq_status rbq_decode_step_varlen(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                  const float* q, const float* P, const float* c_q, const float* c_k,
                                  const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n,
                                  int32_t w, const int32_t* seq_n, const int32_t* seq_w, uint32_t* codes,
                                  float* kfac, int32_t flush, const float* seq_p, float sm_scale,
                                  uint32_t* qplanes, float* qscal, float* scores, int32_t* sel_idx,
                                  int32_t* sel_count, float* out, float* lse, void* ws, size_t ws_bytes,
                                  hipStream_t stream);

/*
 * The compact index -- the paper's storage of the per-key scalar in FP16
 * (Appendix C, storage overhead: D/8 + 2 bytes per key and head, 18 at D = 128,
 * about 3.5 % of a 16-bit KV cache), in place of kfac's two fp32 factors.
 *   kfac16 [B][Hkv][cap] uint16: f = ||k - c_k|| / alpha' as IEEE binary16,
 *          rounded to nearest (ties to even) from the fp32 value, and
 *          saturated to 65504 (the largest finite value) above it.
 * The compact index has no room for g = <c_q, k - c_k>, so it is built and
 * read with the query centroid at zero: these calls take no c_q, and the
 * query must be quantised with c_q = NULL. The score is then
 *   S = A * f16_i * X + B0
 * (rbq_score with g = 0 and f rounded to fp16). Each call behaves as its
 * full-index form otherwise (same arguments, layouts, checks and errors);
 * kfac16 must be 16-byte aligned like every other buffer.
 */
rbq_status rbq_encode_keys_f16(int32_t batch, int32_t heads_kv, int32_t head_dim,
                               const void* keys, int32_t keys_dtype, int64_t keys_ld,
                               int32_t n_new, int32_t offset, int32_t cap, const float* P, float* c_k,
                               uint32_t* codes, uint16_t* kfac16, uint32_t flags,
                               void* ws, size_t ws_bytes, hipStream_t stream);
rbq_status rbq_score_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                         int32_t n, int32_t cap, const uint32_t* codes, const uint16_t* kfac16,
                         const uint32_t* qplanes, const float* qscal, float* scores, hipStream_t stream);
/* rbq_decode_step on the compact index: its outputs are bitwise those of
 * rbq_quantize_query (c_q = NULL), rbq_score_f16, rbq_topp_select,
 * rbq_sparse_decode and (flush) rbq_encode_keys_f16 of the window rows. */
rbq_status rbq_decode_step_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                               const float* q, const float* P, const float* c_k,
                               const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n,
                               int32_t w, uint32_t* codes, uint16_t* kfac16, int32_t flush, float p,
                               float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                               int32_t* sel_idx, int32_t* sel_count, float* out, float* lse,
                               void* ws, size_t ws_bytes, hipStream_t stream);
/* The ragged-batch forms on the compact index (semantics of rbq_score_varlen
 * and rbq_decode_step_varlen). */
rbq_status rbq_score_varlen_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                int32_t n, int32_t cap, const int32_t* seq_n, const uint32_t* codes,
                                const uint16_t* kfac16, const uint32_t* qplanes, const float* qscal,
                                float* scores, hipStream_t stream);
rbq_status rbq_decode_step_varlen_f16(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                      const float* q, const float* P, const float* c_k,
                                      const void* K, const void* V, int32_t kv_dtype, int32_t cap,
                                      int32_t n, int32_t w, const int32_t* seq_n, const int32_t* seq_w,
                                      uint32_t* codes, uint16_t* kfac16, int32_t flush, const float* seq_p,
                                      float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                                      int32_t* sel_idx, int32_t* sel_count, float* out, float* lse,
                                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * rbq_decode_step_noalloc -- rbq_decode_step without a workspace argument, for
 * callers that cannot allocate device memory: code under stream capture,
 * serving loops with a fixed memory plan, harnesses that forbid allocation.
 * The step's scratch memory is a static device array of
 * RBQ_NOALLOC_SCRATCH_BYTES bytes inside the library, one per GPU, held until
 * the process ends; the address of the current device's copy is looked up on
 * the first call made with that device current. Arguments, layouts, results
 * (bitwise) and errors are those of rbq_decode_step, plus:
 *   RBQ_EUNSUPPORTED when rbq_workspace_bytes(RBQ_OP_DECODE_STEP, B, Hq, Hkv,
 *     D, n, w) exceeds RBQ_NOALLOC_SCRATCH_BYTES (one sequence of 32 query
 *     heads over 8 KV heads at D = 128 fits up to n = 128K, w = 256);
 *   RBQ_EDEVICE when the array's address cannot be looked up.
 * No kernel depends on what an earlier call left in the array, but every call
 * on one GPU uses the same array: calls that may overlap in time on one GPU
 * (other streams, other host threads) race, and the caller must order them.
 */
#define RBQ_NOALLOC_SCRATCH_BYTES (16u << 20)
rbq_status rbq_decode_step_noalloc(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                                   const float* q, const float* P, const float* c_q, const float* c_k,
                                   const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n,
                                   int32_t w, uint32_t* codes, float* kfac, int32_t flush, float p,
                                   float sm_scale, uint32_t* qplanes, float* qscal, float* scores,
                                   int32_t* sel_idx, int32_t* sel_count, float* out, float* lse,
                                   hipStream_t stream);

/*
 * rbq_mapped_device_pointer -- the device address of pinned host memory
 * (hipHostGetDevicePointer), for a K/V cache kept in host memory while the
 * index stays in HBM (Appendix C: the small index on the GPU, the full cache
 * offloaded). Every call that takes K / V (or K_loc / V_loc) accepts such an
 * address; the kernels then read the rows they touch over PCIe.
 *   host_ptr (host): memory allocated pinned (hipHostMalloc, or a pinned
 *     allocator); device_ptr (host) out: its device address, NULL on error.
 * RBQ_EINVAL for a NULL argument; RBQ_EDEVICE when the runtime cannot map the
 * pointer (not pinned, or not visible to the current device).
 */
rbq_status rbq_mapped_device_pointer(const void* host_ptr, void** device_ptr);

/* Workspace bytes needed by `op` (one of RBQ_OP_*) for these sizes; 0 for an
 * unknown op or invalid sizes. Host-only, never touches the device. */
size_t rbq_workspace_bytes(int32_t op, int32_t batch, int32_t heads_q, int32_t heads_kv,
                           int32_t head_dim, int32_t n, int32_t w);

/* Bytes of codes + kfac for an index of `cap` keys per (b, kv-head): the index
 * footprint of Appendix C (here D/8 + 8 bytes per key and head). Host-only. */
size_t rbq_index_bytes(int32_t batch, int32_t heads_kv, int32_t head_dim, int32_t cap);

const char* rbq_status_string(rbq_status s);
int32_t rbq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RBQ_H */
