// Internal interface between the host scheduler (topk_api.hip) and the kernels
// (topk_kernels.hip). Nothing here is part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace topk {

enum Act { ACT_SOFTMAX = 0, ACT_RELU = 1 };
enum ElemType { T_F32 = 0, T_BF16 = 1 };

// Sampling modes of the fused scan: ALL keeps every valid score as a candidate;
// SAMPLE first estimates a per-query threshold from a strided subset of key tiles.
// THRESH takes each query's threshold from the filtered path's sample (PassBufs::thr).
enum ScanMode { MODE_ALL = 0, MODE_SAMPLE = 1, MODE_THRESH = 2 };

constexpr int REDO_CAP = 1024;          // redo rows recomputed by the wide fallback kernels
constexpr int REDO_SPLIT = 512;         // keys per work item of the wide fallback
constexpr int REDO_SCORE_BLOCKS = 1024; // workgroups of the wide fallback's score kernel
constexpr int64_t FINALIZE_SLICE_BYTES = (int64_t)8 << 20;  // value matrices above this gather in column slices
constexpr int REDO_BLOCKS = 64;         // workgroups of the fallback for rows beyond REDO_CAP
constexpr int MAX_SELECT_K = 2048;  // largest k the workgroup select / finalize handle

// One call's problem. Attention: BH heads; the FFN is one head whose keys/values
// are W1/W2 (kv_head_stride = 0). Rows of Q/out are (bh * Lq + i); keys (bh, j) sit
// at K + bh * kv_head_stride + j * d.
struct Problem {
  const void* Q;
  const void* K;
  const void* V;
  void* out;
  int64_t BH, Lq, Lk, d, k, C;   // C = query chunk size; Lq = query rows per head in memory
  int64_t q0, q1;                // the rows this problem processes: [q0, q1) of every head
  int tile_only;                 // run on the chunk-tile path whatever the shape
  int64_t kv_head_stride;
  int causal;
  float scale;
  int dtype;
  int act;
  int32_t* idx_out;
  float* score_out;
};

// A pass covers chunk ids [c0, c0 + nc); chunk id = bh * nchunk + c covers query
// rows [q0 + c*C, min(q0 + (c+1)*C, q1)) of head bh. Pass-local row p = (id - c0) * C + r.
struct Pass {
  int64_t c0, nc, nchunk;
};

// Filtered chunk-tile path: every FILTER_KSTRIDE-th key is scored first; the R-th
// largest of a row's valid samples is its threshold, and the tile GEMM keeps only
// scores at or above it.
constexpr int FILTER_KSTRIDE = 16;
constexpr int64_t FILTER_MAX_LK = 65536;  // at most 4096 samples per row
// Bytes of padding after the sample buffer: the per-row threshold kernel loads up to
// 1024 samples from a row's start whatever the row's length, and discards the rest.
constexpr size_t FILTER_SAMP_PAD = 4096;

// The filtered path scores its candidates with the scan kernel (direct mode, one
// candidate list per row and half-wave) for bf16 keys of d = 128; with the MFMA tile
// GEMM (one list per row) otherwise.
inline bool filter_scan_ok(const Problem& pb) { return pb.dtype == T_BF16 && pb.d == 128; }

// Workspace pointers of one pass.
struct PassBufs {
  uint64_t* sel;      // [rows, k] selected keys, (score desc, index asc); 0 pads
  int32_t* redo_list; // [rows]
  int32_t* redo_count;
  float* scores;      // chunk-tile path: [rows, Lk]; fused path: redo rows [REDO_CAP + REDO_BLOCKS, Lk]
  uint64_t* cand;     // fused and filtered paths: [rows, 2, caph]
  int32_t* cnt;       // fused and filtered paths: [rows, 2]
  int64_t caph;
  int cand_single;    // one list of up to 2 caph per row, its length in cnt[2p] (fused scan,
                      // filtered tile GEMM); 0: two lists of caph, lengths cnt[2p], cnt[2p + 1]
  float* samp;        // filtered path: [rows, ceil(Lk / FILTER_KSTRIDE)] sampled scores
  float* thr;         // filtered path: [rows] thresholds
};

struct ScanCfg {
  int mode;           // ScanMode
  int stride;         // SAMPLE: one key tile in `stride` is sampled
  int R;              // SAMPLE: block maxima kept per lane, sorted (11 or 12)
  int groups;         // 32-query groups per wave (2)
  int score_only;     // the scan's score-core ablation (no filter, no candidates)
  int union_rank;     // SAMPLE: J > 0: the threshold is the J-th largest of both half-waves'
                      // lists together (13 or 20); 0: the smaller of their R-th
};

hipError_t launch_init(const PassBufs& b, hipStream_t st);
hipError_t launch_tile_scores(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);
hipError_t launch_tile_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);
hipError_t launch_fused_scan(const Problem& pb, const Pass& ps, const PassBufs& b, const ScanCfg& cfg,
                             hipStream_t st);
hipError_t launch_cand_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);
hipError_t launch_redo(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);
hipError_t launch_finalize(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);
hipError_t launch_mfma_probe(int32_t* rows, int32_t* cols, hipStream_t st);
hipError_t launch_mfma_rate(float* sink, uint64_t* clocks, int blocks, hipStream_t st);
// checked builds (TOPK_CHECK_INDICES): out-of-range selected indices seen by the
// finalize since the last read (the count is reset), -1 in other builds
int64_t read_bad_indices();
int mfma_rate_iters();
// Query chunking without top-k (every valid key, softmax): bf16, d in {64, 128}.
hipError_t launch_dense(const Problem& pb, const Pass& ps, hipStream_t st);

// Backward pass with input checkpointing. Rows of Q / dQ / d_out / idx / dots are
// (bh * Lq + i); keys (bh, j) of K, V, dK, dV sit at (bh * kv_head_stride + j * d)
// (the FFN is one head with kv_head_stride = 0 and X, W1, W2 as Q, K, V).
struct BwdProblem {
  const void* Q;
  const void* K;
  const void* V;
  const int32_t* idx;   // [rows, k] selected keys, entries outside [0, Lk) are padding
  const float* dots;    // [rows, k] their raw scores
  const void* dout;     // [rows, d]
  void* dQ;
  void* dK;
  void* dV;
  int64_t BH, Lq, Lk, d, k, kv_head_stride;
  float scale;
  int dtype;
  int act;
  int list_mode;  // how pairs are grouped by key, fixed for the whole call
};

// How the backward pass groups the selected pairs by key. Heads of up to 2^19 keys
// take a two-level stable bucket sort in LDS (keys in buckets of 1 << shift, at most
// BK_MAXB buckets per head, the pairs of a head in tiles of BK_TILE); the lists come
// out in increasing pair order. Larger heads count pairs with atomics on global
// counters and sort each list before summing.
constexpr int BK_TILE = 4096;
constexpr int BK_MAXB = 256;
constexpr int BK_MAXSHIFT = 11;         // at most 2048 keys per bucket
constexpr int BK_LIST_LDS = 40 * 1024;  // LDS of a list workgroup: 4 waves' counters + staged lists
struct BwdLayout {
  bool bucketed;
  int shift;        // keys per bucket = 1 << shift
  int lcap;         // list entries a bucket may stage in LDS (larger buckets write directly)
  int64_t nb;       // buckets per head
  int64_t tiles;    // tiles per head
  int64_t nhist;    // BH * nb * tiles tile counts
};
// list_mode: 0 automatic, 1 bucket sort, 2 atomic counters (as TOPK_LISTS_*)
inline BwdLayout bwd_layout(int64_t BH, int64_t Lq, int64_t Lk, int64_t k, int list_mode) {
  BwdLayout L{};
  int s = 0;
  while (((Lk + (int64_t(1) << s) - 1) >> s) > BK_MAXB) ++s;
  L.bucketed = list_mode != 2 && s <= BK_MAXSHIFT;
  L.shift = s;
  L.lcap = (BK_LIST_LDS - 4 * 4 * (1 << (s < BK_MAXSHIFT ? s : BK_MAXSHIFT))) / 4;
  L.nb = (Lk + (int64_t(1) << s) - 1) >> s;
  L.tiles = (Lq * k + BK_TILE - 1) / BK_TILE;
  L.nhist = L.bucketed ? BH * L.nb * L.tiles : 0;
  return L;
}

struct BwdBufs {
  BwdLayout L;
  float2* pair;         // [rows * k]: (activation weight, score gradient)
  int32_t* count;       // [BH * Lk + 1]: exclusive offsets of the per-key lists
  int32_t* list;        // [rows * k]: pair ids grouped by key
  int32_t* block_sums;  // scan scratch, one entry per 1024 scanned values
  int32_t* rank;        // atomic path, [rows * k]: each pair's place among its key's pairs
  uint64_t* stage;      // bucketed path, [rows * k]: pairs grouped by bucket
  int32_t* hist;        // bucketed path, [nhist + 1]: per-tile bucket counts, then offsets
};

hipError_t launch_backward(const BwdProblem& bp, const BwdBufs& b, hipStream_t st);
hipError_t launch_filter(const Problem& pb, const Pass& ps, const PassBufs& b, int stage, hipStream_t st);
hipError_t launch_filter_scan(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st);

}  // namespace topk
