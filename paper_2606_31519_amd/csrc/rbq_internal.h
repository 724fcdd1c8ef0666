// Internal declarations shared by the library's translation units.
// Host-side argument checks live in validate.cpp (plain C++, no HIP calls);
// each *.hip file holds one stage's kernels and its launcher.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/rbq.h"
#include "../../include/rbq_testing.h"

namespace rbq {

constexpr int kHeadDim = 128;        // the head dimension of every call (64: the uniform calls, a template argument)
constexpr int kWords = kHeadDim / 32;

// ---------------------------------------------------------------- validation
rbq_status check_heads(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim);
rbq_status check_encode(int32_t batch, int32_t heads_kv, int32_t head_dim, const void* keys, int32_t keys_dtype,
                        int64_t keys_ld, int32_t n_new, int32_t offset, int32_t cap, const float* P,
                        const float* c_k, const uint32_t* codes, const void* kfac, uint32_t flags,
                        const void* ws, size_t ws_bytes);
rbq_status check_quantize(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                          const float* P, const float* c_k, const uint32_t* qplanes, const float* qscal);
rbq_status check_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n, int32_t cap,
                       const uint32_t* codes, const void* kfac, const uint32_t* qplanes, const void* qscal,
                       const void* out);
rbq_status check_topp(int32_t batch, int32_t heads_q, int32_t n, const float* scores, float p, float sm_scale,
                      const int32_t* sel_idx, const int32_t* sel_count, const void* ws, size_t ws_bytes);
rbq_status check_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, const float* q,
                        const void* K, const void* V, int32_t kv_dtype, int32_t cap, int32_t n, bool sparse,
                        const int32_t* sel_idx, const int32_t* sel_count, const void* K_loc, const void* V_loc,
                        int64_t loc_ld, int32_t w, float sm_scale, const float* out, const void* ws,
                        size_t ws_bytes);

// ---------------------------------------------------------------- workspace layouts
// Top-p: each row of scores is cut into parts of spb sub-chunks of kSelSub
// keys; one block of kSelThreads threads per (row, part) in each of three
// passes (per-part histograms, candidate gathering, final select + write).
constexpr int kSelThreads = 1024;
constexpr int kSelPerThread = 16;
constexpr int kSelSub = kSelThreads * kSelPerThread;   // 16384 keys per sub-chunk
constexpr int kSelMaxParts = 64;                       // parts per row (longer rows take more sub-chunks per part)
constexpr int kSelBins = 4096;                         // 12-bit radix levels (key bits 31..20, then 19..8)
constexpr int kSelBins3 = 256;                         // last level (key bits 7..0)
constexpr int kSelCoarse = 64;                         // coarse bins of 64 first-level bins each
constexpr int kSelCandCap = 4096;                      // candidate keys one part hands to the final pass
constexpr int kSelCandLds = 16384;                     // candidate keys of a row the final pass holds in LDS
constexpr int32_t kToppMaxKeys = int32_t(1) << 24;     // keys per row the fixed-point sums hold
// per-part records (bytes): the first pass's exact histogram (the part's
// maximum and total, 64 coarse sums, the directory of non-empty coarse bins
// and their 64-bin sections; 64-bit fixed-point masses relative to the part's
// maximum) and the second pass's counts and candidate keys
constexpr size_t kSelP1Coarse = 16, kSelP1Dir = 16 + 8 * kSelCoarse, kSelP1Sec = 1024;
constexpr size_t kSelPart1Bytes = kSelP1Sec + size_t(8) * kSelCoarse * 64;
constexpr size_t kSelP2Cand = 64;
constexpr size_t kSelPart2Bytes = kSelP2Cand + size_t(4) * kSelCandCap;
constexpr int kSelStateWords = 8;   // per row: row maximum, b1, mass needed inside b1, target (fp64)

struct ToppPlan {
  int32_t spb;     // sub-chunks per part
  int32_t parts;   // parts per row
};
ToppPlan topp_plan(int32_t n);
struct ToppWorkspace {
  unsigned char* part1;   // [rows][parts] kSelPart1Bytes
  unsigned char* part2;   // [rows][parts] kSelPart2Bytes
  uint32_t* state;        // [rows][kSelStateWords]
  size_t bytes;
};
ToppWorkspace topp_workspace(void* base, int64_t rows, int32_t n);

// Decode: split-K over chunks of the indexed rows and of the window.
constexpr int kDecodeChunk = 1024;        // indexed positions per block (at most)
constexpr int kDecodeMinBlocks = 1024;    // the chunk is halved (down to 256) until the grid has this many blocks
constexpr int kCombSlices = 4;            // combine blocks per query head (32 output dimensions each)
constexpr int kDecodeWinChunk = 256;      // window rows per block
struct DecodeSplits {
  int32_t chunk;            // indexed positions per split (<= kDecodeChunk)
  int32_t idx_splits;
  int32_t win_splits;
  int32_t fold_s0;          // window rows folded into the indexed splits: split s >= fold_s0
  int32_t fold_wq;          // takes window rows [(s - fold_s0) * fold_wq, +fold_wq) (0: window splits)
  int32_t total() const { return idx_splits + win_splits; }
};
constexpr int kDecodeFoldMax = 64;        // window rows a sparse split may take beside its indexed rows
constexpr int kDecodeListCap = 1280;      // row-list positions of a sparse split (indexed + folded window)
// tail_window: the window rows are rows [n, n + w) of K / V (the cache tail).
// Then they are folded into the indexed splits instead of splits of their own
// (a grid of whole waves of resident blocks for the usual shapes): spread over
// every split for the sparse call (they are dense, the indexed rows are not),
// given to the last split, beside its rows, for the dense call.
// ragged: each sequence's window is spread on the device over that sequence's
// own splits, fold_wq then being the most a split may take (the list room left
// by the chunk), provided every sequence's window fits its splits that way.
DecodeSplits decode_splits(int32_t batch, int32_t heads_kv, int32_t n, int32_t w, bool tail_window = false,
                           bool sparse = false, bool ragged = false);
size_t decode_workspace_bytes(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim, int32_t n,
                              int32_t w);

// Score: blocks of kScoreThreads lanes, 1, 2 or 4 keys per lane.
constexpr int kScoreThreads = 256;
int score_keys_per_lane(int32_t batch, int32_t heads_kv, int32_t n);
int topp_mask_words(int32_t n);   // 64-key words of a row's selection bitmap

// Placement of blocks on the 8 XCDs (each with its own L2). A launch hands
// workgroup id p to XCD p % 8. The work of a launch is a set of tiles (KV group
// g, Top-p part j) of `slots` workgroups each, placed in one of two ways:
//   kPlaceStream: tile after tile in workgroup order, so the whole GPU streams
//     neighbouring keys at any moment (the fastest order for a scan alone);
//   kPlaceGroup: every kernel that touches the scores of a tile -- the scan
//     that writes them and the Top-p passes that read them and each other's
//     per-part records -- runs that tile on the same XCD: all the parts of a
//     group on XCD g % 8 when there are at least 8 groups, otherwise each group
//     spread over 8 / groups XCDs (part j on the (j % spread)-th of them) so
//     that every XCD still gets work. The passes then read the scores and a
//     row's records from their own L2.
// tile_grid() is the launch size.
constexpr int kXcds = 8;
enum TileMode : int32_t { kPlaceStream = 0, kPlaceGroup = 1 };
struct TilePlace {
  int32_t groups;    // KV groups (B * Hkv; for a call without groups, its rows)
  int32_t parts;     // Top-p parts per row
  int32_t spread;    // XCDs per group (kPlaceGroup)
  int32_t per_xcd;   // tiles per XCD (kPlaceGroup), all tiles (kPlaceStream)
  int32_t mode;
};
inline TilePlace tile_place(int32_t groups, int32_t parts, int32_t mode) {
  TilePlace t;
  t.groups = groups;
  t.parts = parts;
  t.mode = mode;
  t.spread = groups >= kXcds ? 1 : kXcds / groups;
  if (mode == kPlaceStream)
    t.per_xcd = groups * parts;
  else
    t.per_xcd =
        t.spread == 1 ? int32_t((int64_t(groups) + kXcds - 1) / kXcds * parts) : (parts + t.spread - 1) / t.spread;
  return t;
}
inline int64_t tile_grid(const TilePlace& t, int64_t slots) {
  return t.mode == kPlaceStream ? int64_t(t.per_xcd) * slots : int64_t(t.per_xcd) * slots * kXcds;
}

// Fused decode step: the workspaces of its stages side by side.
struct StepWorkspace {
  void* decode;                     // decode_workspace_bytes()
  void* topp;                       // topp_workspace().bytes
  unsigned long long* masks;        // [B * Hq][topp_mask_words(n)]
  size_t topp_bytes;
  size_t bytes;
};
StepWorkspace step_workspace(void* base, int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t head_dim,
                             int32_t n, int32_t w);

// Encode: centroid partial sums over chunks of kCentroidChunk keys.
constexpr int kCentroidChunk = 1024;
size_t encode_workspace_bytes(int32_t batch, int32_t heads_kv, int32_t head_dim, int32_t n_new);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------- launchers (HIP)
rbq_status launch_encode(int32_t batch, int32_t heads_kv, const void* keys, int32_t keys_dtype, int64_t keys_ld,
                         int32_t n_new, int32_t offset, int32_t cap, const float* P, const float* c_q, float* c_k,
                         uint32_t* codes, float* kfac, uint32_t flags, float* alpha_out, void* ws,
                         float* rot_out, hipStream_t stream, uint16_t* kfac16 = nullptr,
                         int32_t head_dim = kHeadDim);
// (kfac16: the compact index's fp16 factors, written instead of kfac when non-NULL)
// bits: B_q, the query's quantisation bits (1..8; 4 bit-planes per head up to 4 bits, 8 above)
rbq_status launch_quantize(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const float* P,
                           const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal, float* qrot_out,
                           hipStream_t stream, int32_t bits = 4, int32_t head_dim = kHeadDim);
// query quantisation and, in the same launch, the lazy encode of n_new window
// keys into index rows [offset, offset + n_new) with the existing c_k (ragged,
// seq_off != NULL: sequence b encodes min(seq_cnt[b], n_new) keys (n_new without
// seq_cnt) from row min(seq_off[b], off_max) of its block of `keys` into index
// rows offset + that row onwards)
rbq_status launch_quantize_flush(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const float* P,
                                 const float* c_q, const float* c_k, uint32_t* qplanes, float* qscal,
                                 const void* keys, int32_t keys_dtype, int64_t keys_ld, int32_t n_new, int32_t offset,
                                 int32_t cap, uint32_t* codes, float* kfac, hipStream_t stream,
                                 const int32_t* seq_off = nullptr, const int32_t* seq_cnt = nullptr,
                                 int32_t off_max = 0, uint16_t* kfac16 = nullptr, int32_t head_dim = kHeadDim);
// seq_n (ragged batches): [B] indexed keys per sequence, clamped to [0, n]; n is the row stride
rbq_status launch_score(int32_t batch, int32_t heads_q, int32_t heads_kv, int32_t n, int32_t cap,
                        const uint32_t* codes, const float* kfac, const uint32_t* qplanes, const float* qscal,
                        float* scores, int32_t* ip_out, int32_t* pc_out, hipStream_t stream,
                        const int32_t* seq_n = nullptr, const uint16_t* kfac16 = nullptr, int32_t planes = 4,
                        int32_t head_dim = kHeadDim);
// (kfac16: the compact index's fp16 factors [B][Hkv][cap], read instead of kfac when non-NULL; g = 0.
//  planes: query bit-planes per head, 4 or 8 (8: B_q up to 8; uniform, unfused calls only))
// masks: optional [rows][topp_mask_words(n)] selection bitmaps (bit i of word k = key 64 k + i); seq_n / seq_p (ragged
// batches): [B] keys and p per sequence, row r of sequence r / heads_q
rbq_status launch_topp(int32_t rows, int32_t n, const float* scores, float p, float sm_scale, int32_t* sel_idx,
                       int32_t* sel_count, void* ws, hipStream_t stream, unsigned long long* masks = nullptr, const int32_t* seq_n = nullptr,
                       const float* seq_p = nullptr, int32_t heads_q = 1);
rbq_status launch_decode(int32_t batch, int32_t heads_q, int32_t heads_kv, const float* q, const void* K,
                         const void* V, int32_t kv_dtype, int32_t cap, int32_t n, const int32_t* sel_idx,
                         const int32_t* sel_count, const void* K_loc, const void* V_loc, int64_t loc_ld, int32_t w,
                         float sm_scale, float* out, float* lse, void* ws, bool sparse, hipStream_t stream,
                         const unsigned long long* sel_mask = nullptr, int32_t mask_words = 0,
                         const int32_t* seq_n = nullptr, const int32_t* seq_w = nullptr,
                         int32_t head_dim = kHeadDim);
// (ragged: seq_n / seq_w [B] indexed and window rows per sequence, the window
// being the sequence's cache tail; K_loc, V_loc and loc_ld are then ignored)

}  // namespace rbq
