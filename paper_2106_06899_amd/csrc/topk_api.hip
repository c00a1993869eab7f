// Host side of the C ABI declared in include/topk_attn.h: argument validation,
// path choice, the chunk scheduler (how many query chunks are in flight per pass
// under the workspace budget) and the kernel sequence of each pass.
#include "topk_attn.h"
#include "topk_internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

namespace topk {
namespace {

thread_local std::string g_err;
thread_local void* g_ws = nullptr;
thread_local size_t g_ws_bytes = 0;
thread_local int64_t g_fallback_rows = -1;  // rows a fallback selected in the last debug call

// Optional per-stage timing (topk_profile_begin/end): an event pair around every
// launch group of the calling thread's calls, on the call's own stream.
enum Stage { ST_SCORE = 0, ST_SELECT = 1, ST_REDO = 2, ST_FINAL = 3, ST_BWD = 4, N_STAGES = 5 };
struct Mark {
  hipEvent_t a, b;
  int stage;
};
thread_local bool g_prof = false;
thread_local std::vector<Mark> g_marks;

struct StageTimer {
  hipStream_t st;
  Mark m;
  bool on;
  StageTimer(hipStream_t s, int stage) : st(s), on(g_prof) {
    if (!on) return;
    m.stage = stage;
    if (hipEventCreate(&m.a) != hipSuccess || hipEventCreate(&m.b) != hipSuccess) {
      on = false;
      return;
    }
    hipEventRecord(m.a, st);
  }
  ~StageTimer() {
    if (!on) return;
    hipEventRecord(m.b, st);
    g_marks.push_back(m);
  }
};

constexpr size_t ALIGN = 256;
constexpr size_t DEFAULT_BUDGET = size_t(8) << 30;  // workspace cap when the library allocates
std::atomic<size_t> g_budget{DEFAULT_BUDGET};        // process-wide, set by topk_set_memory_budget
constexpr int64_t DEFAULT_CHUNK = 1024;
constexpr int64_t FUSED_CAPH = 512;                   // candidates kept per (query, half-wave)

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

enum Path { PATH_FUSED = 1, PATH_TILE = 2, PATH_FILTER = 4 };

struct Plan {
  int path;
  ScanCfg scan;
  int64_t nchunk, total_chunks, per_pass;
  size_t per_chunk, fixed;
};

// ---------------------------------------------------------------- validation
int check_ptr(const void* p, const char* name) {
  if (!p) return fail(TOPK_E_NULL, "%s is NULL", name);
  if (((uintptr_t)p) % 16) return fail(TOPK_E_ALIGN, "%s is not 16-byte aligned", name);
  return TOPK_OK;
}

int validate_shape(int64_t BH_a, int64_t BH_b, int64_t Lq, int64_t Lk, int64_t d, int64_t k, int64_t chunk,
                   int causal, float scale, int dtype, bool attn) {
  if (BH_a < 1 || BH_b < 1 || Lq < 1 || Lk < 1 || d < 1)
    return fail(TOPK_E_INVAL, "sizes must be >= 1 (got %lld, %lld, %lld, %lld, %lld)", (long long)BH_a,
                (long long)BH_b, (long long)Lq, (long long)Lk, (long long)d);
  if (k < 1 || k > Lk) return fail(TOPK_E_INVAL, "need 1 <= k <= %lld keys (got k = %lld)", (long long)Lk, (long long)k);
  if (chunk < 0) return fail(TOPK_E_INVAL, "chunk must be >= 0 (0 = default), got %lld", (long long)chunk);
  if (attn && causal != 0 && causal != 1) return fail(TOPK_E_INVAL, "causal must be 0 or 1");
  if (attn && !(isfinite(scale) && scale > 0.f)) return fail(TOPK_E_INVAL, "scale must be finite and > 0");
  if (dtype != TOPK_F32 && dtype != TOPK_BF16) return fail(TOPK_E_INVAL, "dtype must be TOPK_F32 or TOPK_BF16");
  if (d % 8 != 0 || d > 1024)
    return fail(TOPK_E_UNSUPPORTED, "feature size %lld: the library needs a multiple of 8, at most 1024", (long long)d);
  if (k > MAX_SELECT_K) return fail(TOPK_E_UNSUPPORTED, "k = %lld exceeds the library's limit %d", (long long)k, MAX_SELECT_K);
  if (Lk > 0x7FFFFFFFLL) return fail(TOPK_E_UNSUPPORTED, "more than 2^31 - 1 keys");
  return TOPK_OK;
}

// ---------------------------------------------------------------- planning
int order_stat_for(int64_t k) { return k <= 32 ? 3 : (k <= 64 ? 6 : 12); }

// The fused scan's per-query threshold, from the 16-key block maxima of a strided
// sample of key tiles. d = 64, k <= 64: a 1-in-8 sample, each half-wave keeps its 11
// largest, and the threshold is the J-th largest of both lists together (J = 13 for
// k <= 32, 20 for k <= 64: about 2.8 k candidates per row on Gaussian-like scores,
// about one row in 20000 below k). Otherwise (d = 128, whose registers hold fewer
// sorted maxima, or k > 64): a 1-in-16 sample and the smaller of the two half-waves'
// R-th largest, R = order_stat_for(k) (about 4 k candidates).
ScanCfg sample_rule(int64_t k, int64_t d, int groups) {
  if (d == 64 && k <= 32) return {MODE_SAMPLE, 8, 11, groups, 0, 13};
  if (d == 64 && k <= 64) return {MODE_SAMPLE, 8, 11, groups, 0, 20};
  return {MODE_SAMPLE, 16, order_stat_for(k), groups, 0, 0};
}
// Valid keys a row needs for its threshold: twice the rank taken, in sampled blocks of
// the pool it is taken from (a sampled 64-key tile gives each half-wave two blocks).
int64_t sample_rows_needed(const ScanCfg& sc) {
  return sc.union_rank ? (int64_t)2 * sc.union_rank * 64 * sc.stride / 4 : (int64_t)2 * sc.R * 64 * sc.stride / 2;
}

// Filtered chunk-tile path: bf16 MFMA tiles (d % 32 == 0) whose rows are long
// enough for a sampled threshold and at most 4096 samples, k <= 512 (its
// candidates, about 16 R per row, stay within the 1024 the select holds for
// k <= 256, within 2048 for larger k).
bool filter_ok(const Problem& pb) {
  return pb.dtype == T_BF16 && pb.d % 32 == 0 && pb.d <= 1024 && pb.k <= 512 && pb.Lk > 2048 &&
         pb.Lk <= FILTER_MAX_LK;
}
// candidates kept per (row, half) of the list buffers
int64_t caph_for(const Problem& pb, int path) { return path == PATH_FILTER && pb.k > 256 ? 2 * FUSED_CAPH : FUSED_CAPH; }

void choose_path(const Problem& pb, Plan* pl) {
  pl->path = PATH_TILE;
  pl->scan = {MODE_ALL, 16, 8, 2, 0, 0};
  if (pb.tile_only) {
    if (filter_ok(pb)) pl->path = PATH_FILTER;
    return;
  }
  // 64 queries per wave: measured faster than 128 once the filter runs (the LDS
  // staging, not the K operand reads, bounds the scan)
  const int groups = 2;
  // Causal rows (Eq. 2) take the fused path only when the keys are long against k:
  // short rows have so few keys per selected one that most score blocks would
  // beat the threshold and the on-chip filter would stage nearly all of them.
  const bool shape_ok = pb.dtype == T_BF16 && (pb.d == 64 || pb.d == 128) && pb.k <= 128 &&
                        pb.Lk < (int64_t(1) << 25) && (!pb.causal || pb.Lk >= 256 * pb.k);
  if (!shape_ok) {
    if (filter_ok(pb)) pl->path = PATH_FILTER;
    return;
  }
  if (pb.Lk <= 2 * FUSED_CAPH) {  // every key fits the candidate buffers
    pl->path = PATH_FUSED;
    pl->scan = sample_rule(pb.k, pb.d, groups);  // its kernel instantiation; no sample is taken
    pl->scan.mode = MODE_ALL;
    return;
  }
  // Threshold mode, see sample_rule: needs at least 2R sampled 16-key blocks in the
  // pool the order statistic is taken from.
  const ScanCfg sc = sample_rule(pb.k, pb.d, groups);
  const int64_t kt = 64;  // key tile of the scan kernel
  const int64_t sampled_tiles = ((pb.Lk + kt - 1) / kt + sc.stride - 1) / sc.stride;
  if (sampled_tiles * (sc.union_rank ? 4 : 2) >= 2 * (sc.union_rank ? sc.union_rank : sc.R)) {
    pl->path = PATH_FUSED;
    pl->scan = sc;
  } else if (filter_ok(pb)) {
    pl->path = PATH_FILTER;
  }
}

size_t row_bytes(const Problem& pb, const Plan& pl) {
  size_t b = (size_t)pb.k * 8 + 4;  // selection + redo list entry
  if (pl.path == PATH_TILE)
    b += (size_t)pb.Lk * 4;
  else
    b += 2 * (size_t)caph_for(pb, pl.path) * 8 + 8;
  if (pl.path == PATH_FILTER) b += (size_t)((pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE) * 4 + 4;
  return b;
}

void plan_sizes(const Problem& pb, Plan* pl, size_t budget) {
  pl->nchunk = (pb.q1 - pb.q0 + pb.C - 1) / pb.C;
  pl->total_chunks = pb.BH * pl->nchunk;
  pl->per_chunk = row_bytes(pb, *pl) * (size_t)pb.C + 6 * ALIGN;
  pl->fixed = 2 * ALIGN + (pl->path != PATH_TILE ? up((size_t)(REDO_CAP + REDO_BLOCKS) * pb.Lk * 4) : 0) +
              (pl->path == PATH_FILTER ? FILTER_SAMP_PAD : 0);
  int64_t n = 1;
  if (budget > pl->fixed + pl->per_chunk) n = (int64_t)((budget - pl->fixed) / pl->per_chunk);
  if (n > pl->total_chunks) n = pl->total_chunks;
  if (n < 1) n = 1;
  // keep every grid within the launch limits (rows * 256 threads < 2^32, z <= 65535)
  const int64_t max_rows = int64_t(1) << 23;
  if (n * pb.C > max_rows) n = max_rows / pb.C > 0 ? max_rows / pb.C : 1;
  if (n > 65535) n = 65535;
  // equal passes: the last pass must not run a handful of chunks on an idle GPU
  const int64_t passes = (pl->total_chunks + n - 1) / n;
  pl->per_pass = (pl->total_chunks + passes - 1) / passes;
}

size_t plan_total(const Plan& pl, const Problem& pb) {
  (void)pb;
  return pl.fixed + (size_t)pl.per_pass * pl.per_chunk;
}

PassBufs carve(const Problem& pb, const Plan& pl, char* ws) {
  const size_t rows = (size_t)pl.per_pass * pb.C;
  PassBufs b = {};
  size_t off = 0;
  b.redo_count = (int32_t*)(ws + off);
  off += ALIGN;
  b.redo_list = (int32_t*)(ws + off);
  off += up(rows * 4);
  b.sel = (uint64_t*)(ws + off);
  off += up(rows * (size_t)pb.k * 8);
  if (pl.path == PATH_TILE) {
    b.scores = (float*)(ws + off);
    off += up(rows * (size_t)pb.Lk * 4);
  } else {
    b.caph = caph_for(pb, pl.path);
    b.cand = (uint64_t*)(ws + off);
    off += up(rows * 2 * (size_t)b.caph * 8);
    b.cnt = (int32_t*)(ws + off);
    off += up(rows * 8);
    b.scores = (float*)(ws + off);
    off += up((size_t)(REDO_CAP + REDO_BLOCKS) * pb.Lk * 4);
    // one list per row, which the fused scan and the filtered tile GEMM append to; the
    // filtered path's scan keeps one list per row and half-wave
    b.cand_single = pl.path == PATH_FILTER && filter_scan_ok(pb) ? 0 : 1;
    if (pl.path == PATH_FILTER) {
      b.samp = (float*)(ws + off);
      off += up(rows * (size_t)((pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE) * 4 + FILTER_SAMP_PAD);
      b.thr = (float*)(ws + off);
      off += up(rows * 4);
    }
  }
  return b;
}

// Causal rows on the fused path: a row needs twice the rank its threshold takes in
// valid sampled blocks (sample_rows_needed valid keys: 3328, 5120 and 12288 for k <=
// 32, 64 and 128 at d = 64; 3072, 6144 and 12288 at d = 128). The first such rows of every head therefore run on the
// chunk-tile path, the rest fused. Each row's path, and so its result, does not
// depend on the chunk size.
int split_rows(const Problem& pb, Problem* parts) {
  parts[0] = pb;
  Plan pl;
  choose_path(pb, &pl);
  if (!pb.causal || pl.path != PATH_FUSED || pl.scan.mode != MODE_SAMPLE) return 1;
  const int64_t T = sample_rows_needed(pl.scan);
  if (T <= pb.q0) return 1;
  parts[0].q1 = pb.q1 < T ? pb.q1 : T;
  parts[0].tile_only = 1;
  if (T >= pb.q1) return 1;
  parts[1] = pb;
  parts[1].q0 = T;
  return 2;
}

// ---------------------------------------------------------------- execution
// report: read back the rows a fallback selected (waits for the stream; debug calls)
// fixed_ws / fixed_bytes: a workspace the call must run in (no allocation, no
// registered workspace); the plan then fits its passes into fixed_bytes.
int run(Problem whole, hipStream_t st, bool report, void* fixed_ws = nullptr, size_t fixed_bytes = 0) {
  Problem parts[2];
  Plan plans[2];
  const int np = split_rows(whole, parts);
  void* const ws_given = fixed_ws ? fixed_ws : g_ws;
  const size_t ws_given_bytes = fixed_ws ? fixed_bytes : g_ws_bytes;
  size_t budget = ws_given ? ws_given_bytes : g_budget.load(std::memory_order_relaxed), need = 0;
  for (int q = 0; q < np; ++q) {
    choose_path(parts[q], &plans[q]);
    plan_sizes(parts[q], &plans[q], budget);
    const size_t n = plan_total(plans[q], parts[q]);
    need = n > need ? n : need;
  }
  char* ws = (char*)ws_given;
  bool own = false;
  if (fixed_ws) {
    if (need > fixed_bytes)
      return fail(TOPK_E_NOMEM, "one query chunk needs %zu bytes of workspace, above the %zu bytes of the fixed "
                  "device scratch", need, fixed_bytes);
  } else if (g_ws) {
    if (need > g_ws_bytes)
      return fail(TOPK_E_NOMEM, "registered workspace of %zu bytes is below the %zu bytes one query chunk needs",
                  g_ws_bytes, need);
  } else {
    if (hipMallocAsync((void**)&ws, need, st) != hipSuccess)
      return fail(TOPK_E_NOMEM, "could not allocate %zu bytes of workspace", need);
    own = true;
  }
  hipError_t e = hipSuccess;
  int64_t fallback = 0;
  if (report) g_fallback_rows = -1;
  for (int q = 0; q < np; ++q)
  for (int64_t c0 = 0; c0 < plans[q].total_chunks && e == hipSuccess; c0 += plans[q].per_pass) {
    const Problem& pb = parts[q];
    const Plan& pl = plans[q];
    Pass ps;
    ps.c0 = c0;
    ps.nc = pl.total_chunks - c0 < pl.per_pass ? pl.total_chunks - c0 : pl.per_pass;
    ps.nchunk = pl.nchunk;
    PassBufs b = carve(pb, pl, ws);
    if (pl.path == PATH_FILTER) {
      if (e == hipSuccess) e = launch_init(b, st);
      if (e == hipSuccess) e = launch_filter(pb, ps, b, 0, st);
      if (e == hipSuccess) {
        StageTimer t(st, ST_SCORE);
        e = launch_filter(pb, ps, b, 1, st);
        if (e == hipSuccess) e = launch_filter(pb, ps, b, 2, st);
        if (e == hipSuccess) e = launch_filter(pb, ps, b, 3, st);
      }
      if (e == hipSuccess) {
        StageTimer t(st, ST_SELECT);
        e = launch_cand_select(pb, ps, b, st);
      }
      if (e == hipSuccess) {
        StageTimer t(st, ST_REDO);
        e = launch_redo(pb, ps, b, st);
      }
    } else if (pl.path == PATH_TILE) {
      if (e == hipSuccess) e = launch_init(b, st);
      if (e == hipSuccess) {
        StageTimer t(st, ST_SCORE);
        e = launch_tile_scores(pb, ps, b, st);
      }
      if (e == hipSuccess) {
        StageTimer t(st, ST_SELECT);
        e = launch_tile_select(pb, ps, b, st);
      }
    } else {
      if (e == hipSuccess) e = launch_init(b, st);
      if (e == hipSuccess) {
        StageTimer t(st, ST_SCORE);
        e = launch_fused_scan(pb, ps, b, pl.scan, st);
      }
      if (e == hipSuccess) {
        StageTimer t(st, ST_SELECT);
        e = launch_cand_select(pb, ps, b, st);
      }
      if (e == hipSuccess) {
        StageTimer t(st, ST_REDO);
        e = launch_redo(pb, ps, b, st);
      }
    }
    if (e == hipSuccess) {
      StageTimer t(st, ST_FINAL);
      e = launch_finalize(pb, ps, b, st);
    }
    if (e == hipSuccess && report) {  // debug calls report the fallback rows (synchronously)
      int32_t h = 0;
      e = hipMemcpyAsync(&h, b.redo_count, sizeof(h), hipMemcpyDeviceToHost, st);
      if (e == hipSuccess) e = hipStreamSynchronize(st);
      fallback += h;
    }
  }
  if (report) g_fallback_rows = e == hipSuccess ? fallback : -1;
  if (own) hipFreeAsync(ws, st);
  if (e != hipSuccess) return fail(TOPK_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
#ifdef TOPK_CHECK_INDICES
  // checked builds wait for the call, so that an error the kernels raise while running
  // is returned by this call (and topk_last_error) instead of a later one
  e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) return fail(TOPK_E_HIP, "the call's kernels failed: %s", hipGetErrorString(e));
#endif
  return TOPK_OK;
}

int attn_problem(Problem* pb, const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H,
                 int64_t Lq, int64_t Lk, int64_t d, int64_t k, int64_t chunk, int causal, float scale, int dtype,
                 int32_t* idx_out, float* score_out, bool check_ptrs) {
  int rc = validate_shape(B, H, Lq, Lk, d, k, chunk, causal, scale, dtype, true);
  if (rc) return rc;
  if (B > (int64_t(1) << 31) / H) return fail(TOPK_E_INVAL, "B*H too large");
  if (check_ptrs) {
    if ((rc = check_ptr(Q, "Q")) || (rc = check_ptr(K, "K")) || (rc = check_ptr(V, "V")) ||
        (rc = check_ptr(out, "out")))
      return rc;
  }
  pb->Q = Q;
  pb->K = K;
  pb->V = V;
  pb->out = out;
  pb->BH = B * H;
  pb->Lq = Lq;
  pb->q0 = 0;
  pb->q1 = Lq;
  pb->tile_only = 0;
  pb->Lk = Lk;
  pb->d = d;
  pb->k = k;
  pb->C = chunk == 0 ? (Lq < DEFAULT_CHUNK ? Lq : DEFAULT_CHUNK) : (chunk < Lq ? chunk : Lq);
  pb->kv_head_stride = Lk * d;
  pb->causal = causal;
  pb->scale = scale;
  pb->dtype = dtype == TOPK_BF16 ? T_BF16 : T_F32;
  pb->act = ACT_SOFTMAX;
  pb->idx_out = idx_out;
  pb->score_out = score_out;
  return TOPK_OK;
}

int ffn_problem(Problem* pb, const void* X, const void* W1, const void* W2, void* out, int64_t N, int64_t d_model,
                int64_t d_ff, int64_t k, int64_t chunk, int dtype, int32_t* idx_out, float* score_out,
                bool check_ptrs) {
  int rc = validate_shape(1, 1, N, d_ff, d_model, k, chunk, 0, 1.f, dtype, false);
  if (rc) return rc;
  if (check_ptrs) {
    if ((rc = check_ptr(X, "X")) || (rc = check_ptr(W1, "W1")) || (rc = check_ptr(W2, "W2")) ||
        (rc = check_ptr(out, "out")))
      return rc;
  }
  pb->Q = X;
  pb->K = W1;
  pb->V = W2;
  pb->out = out;
  pb->BH = 1;
  pb->Lq = N;
  pb->q0 = 0;
  pb->q1 = N;
  pb->tile_only = 0;
  pb->Lk = d_ff;
  pb->d = d_model;
  pb->k = k;
  pb->C = chunk == 0 ? (N < DEFAULT_CHUNK ? N : DEFAULT_CHUNK) : (chunk < N ? chunk : N);
  pb->kv_head_stride = 0;
  pb->causal = 0;
  pb->scale = 1.f;
  pb->dtype = dtype == TOPK_BF16 ? T_BF16 : T_F32;
  pb->act = ACT_RELU;
  pb->idx_out = idx_out;
  pb->score_out = score_out;
  return TOPK_OK;
}

int debug_ptrs(int32_t* idx_out, float* score_out) {
  if (idx_out && ((uintptr_t)idx_out) % 4) return fail(TOPK_E_ALIGN, "idx_out is not 4-byte aligned");
  if (score_out && ((uintptr_t)score_out) % 4) return fail(TOPK_E_ALIGN, "score_out is not 4-byte aligned");
  return TOPK_OK;
}

size_t workspace_for(const Problem& whole) {
  Problem parts[2];
  const int np = split_rows(whole, parts);
  const size_t budget = g_budget.load(std::memory_order_relaxed);
  size_t need = 0;
  for (int q = 0; q < np; ++q) {
    Plan pl;
    choose_path(parts[q], &pl);
    plan_sizes(parts[q], &pl, budget);
    const size_t n = plan_total(pl, parts[q]);
    need = n > need ? n : need;
  }
  return need;
}

// ---------------------------------------------------------------- backward
std::atomic<int> g_list_mode{TOPK_LISTS_AUTO};  // process-wide, set by topk_set_backward_lists

size_t bwd_bytes(const BwdProblem& bp) {
  const int64_t nkeys = bp.BH * bp.Lk, npairs = bp.BH * bp.Lq * bp.k;
  const BwdLayout L = bwd_layout(bp.BH, bp.Lq, bp.Lk, bp.k, bp.list_mode);
  const int64_t scanned = std::max(nkeys + 1, L.nhist + 1), nb = (scanned + 1023) / 1024;
  size_t total = up((size_t)npairs * 8) + up((size_t)(nkeys + 1) * 4) + up((size_t)npairs * 4) + up((size_t)nb * 4);
  if (L.bucketed) total += up((size_t)npairs * 8) + up((size_t)(L.nhist + 1) * 4);
  else total += up((size_t)npairs * 4);
  return total;
}

BwdBufs bwd_carve(const BwdProblem& bp, char* ws) {
  const int64_t nkeys = bp.BH * bp.Lk, npairs = bp.BH * bp.Lq * bp.k;
  BwdBufs b{};
  b.L = bwd_layout(bp.BH, bp.Lq, bp.Lk, bp.k, bp.list_mode);
  const int64_t scanned = std::max(nkeys + 1, b.L.nhist + 1), nb = (scanned + 1023) / 1024;
  size_t off = 0;
  b.pair = (float2*)(ws + off);
  off += up((size_t)npairs * 8);
  b.count = (int32_t*)(ws + off);
  off += up((size_t)(nkeys + 1) * 4);
  b.list = (int32_t*)(ws + off);
  off += up((size_t)npairs * 4);
  b.block_sums = (int32_t*)(ws + off);
  off += up((size_t)nb * 4);
  if (b.L.bucketed) {
    b.stage = (uint64_t*)(ws + off);
    off += up((size_t)npairs * 8);
    b.hist = (int32_t*)(ws + off);
  } else {
    b.rank = (int32_t*)(ws + off);
  }
  return b;
}

int bwd_problem(BwdProblem* bp, const void* Q, const void* K, const void* V, const int32_t* idx, const float* dots,
                const void* dout, void* dQ, void* dK, void* dV, int64_t BH, int64_t Lq, int64_t Lk, int64_t d,
                int64_t k, int64_t kv_head_stride, float scale, int dtype, int act, bool check_ptrs) {
  int rc = validate_shape(BH, 1, Lq, Lk, d, k, 0, 0, scale, dtype, act == ACT_SOFTMAX);
  if (rc) return rc;
  if (BH * Lq > (int64_t(1) << 31) / k || BH * Lk >= (int64_t(1) << 31) - 1)
    return fail(TOPK_E_UNSUPPORTED, "the backward pass needs rows * k and heads * keys below 2^31");
  const int list_mode = g_list_mode.load(std::memory_order_relaxed);
  if (list_mode == TOPK_LISTS_BUCKET && !bwd_layout(BH, Lq, Lk, k, list_mode).bucketed)
    return fail(TOPK_E_UNSUPPORTED, "bucket-sorted backward lists need at most 2^19 keys per head (got %lld)",
                (long long)Lk);
  if (check_ptrs) {
    if ((rc = check_ptr(Q, "queries")) || (rc = check_ptr(K, "keys")) || (rc = check_ptr(V, "values")) ||
        (rc = check_ptr(dout, "d_out")) || (rc = check_ptr(dQ, "d_queries")) || (rc = check_ptr(dK, "d_keys")) ||
        (rc = check_ptr(dV, "d_values")))
      return rc;
    if (!idx || !dots) return fail(TOPK_E_NULL, "top_idx and top_dots are required");
    if (((uintptr_t)idx) % 4 || ((uintptr_t)dots) % 4) return fail(TOPK_E_ALIGN, "top_idx / top_dots not 4-byte aligned");
  }
  bp->Q = Q;
  bp->K = K;
  bp->V = V;
  bp->idx = idx;
  bp->dots = dots;
  bp->dout = dout;
  bp->dQ = dQ;
  bp->dK = dK;
  bp->dV = dV;
  bp->BH = BH;
  bp->Lq = Lq;
  bp->Lk = Lk;
  bp->d = d;
  bp->k = k;
  bp->kv_head_stride = kv_head_stride;
  bp->scale = scale;
  bp->dtype = dtype == TOPK_BF16 ? T_BF16 : T_F32;
  bp->act = act;
  bp->list_mode = list_mode;
  return TOPK_OK;
}

int run_backward(const BwdProblem& bp, hipStream_t st) {
  const size_t need = bwd_bytes(bp);
  char* ws = (char*)g_ws;
  bool own = false;
  if (g_ws) {
    if (need > g_ws_bytes)
      return fail(TOPK_E_NOMEM, "registered workspace of %zu bytes is below the %zu bytes the backward pass needs",
                  g_ws_bytes, need);
  } else {
    if (hipMallocAsync((void**)&ws, need, st) != hipSuccess)
      return fail(TOPK_E_NOMEM, "could not allocate %zu bytes of workspace", need);
    own = true;
  }
  hipError_t e;
  {
    StageTimer t(st, ST_BWD);
    e = launch_backward(bp, bwd_carve(bp, ws), st);
  }
  if (own) hipFreeAsync(ws, st);
  if (e != hipSuccess) return fail(TOPK_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return TOPK_OK;
}

// ---------------------------------------------------------------- query chunking without top-k
// Every valid key of each query (the k = Lk fixed point): one streaming-softmax launch
// over all query chunks; it needs no workspace, so nothing bounds the chunks in flight.
int run_dense(const Problem& pb, hipStream_t st) {
  if (pb.dtype != T_BF16 || (pb.d != 64 && pb.d != 128))
    return fail(TOPK_E_UNSUPPORTED, "query chunking without top-k runs on bf16 inputs with d = 64 or 128");
  Pass ps;
  ps.nchunk = (pb.Lq + pb.C - 1) / pb.C;
  ps.c0 = 0;
  ps.nc = pb.BH * ps.nchunk;
  hipError_t e;
  {
    StageTimer t(st, ST_SCORE);
    e = launch_dense(pb, ps, st);
  }
  if (e != hipSuccess) return fail(TOPK_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return TOPK_OK;
}

// ---------------------------------------------------------------- fixed device scratch
// The workspace of topk_attn_noalloc: a file-scope device array of TOPK_NOALLOC_SCRATCH_BYTES,
// one copy per GPU, held by the process until it ends. Host code must not pass the
// array's name to a kernel (on the host it only stands for the symbol); the device
// address comes from hipGetSymbolAddress, taken once per device with that device
// current and kept in g_scratch_ptr.
constexpr int MAX_DEVICES = 64;
__device__ __align__(256) unsigned char scratch[TOPK_NOALLOC_SCRATCH_BYTES];
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

int scratch_for_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
    return fail(TOPK_E_HIP, "no current HIP device (or device index above %d)", MAX_DEVICES - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(TOPK_E_HIP, "hipGetSymbolAddress of the fixed scratch failed on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TOPK_OK;
}

}  // namespace
}  // namespace topk

using namespace topk;

extern "C" {

int topk_attn_debug(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H, int64_t Lq,
                    int64_t Lk, int64_t d, int64_t k, int64_t chunk, int causal, float scale, int dtype,
                    void* hip_stream, int32_t* idx_out, float* score_out) {
  g_err.clear();
  Problem pb;
  int rc = attn_problem(&pb, Q, K, V, out, B, H, Lq, Lk, d, k, chunk, causal, scale, dtype, idx_out, score_out, true);
  if (rc) return rc;
  if ((rc = debug_ptrs(idx_out, score_out))) return rc;
  return run(pb, (hipStream_t)hip_stream, idx_out != nullptr || score_out != nullptr);
}

int topk_attn(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H, int64_t Lq, int64_t Lk,
              int64_t d, int64_t k, int64_t chunk, int causal, float scale, int dtype, void* hip_stream) {
  // k = Lk keeps every valid key (Eq. 4 reduces to Eq. 1): beyond the select's limit
  // the streaming-softmax kernel computes it
  if (k == Lk && k > MAX_SELECT_K)
    return topk_attn_dense(Q, K, V, out, B, H, Lq, Lk, d, chunk, causal, scale, dtype, hip_stream);
  return topk_attn_debug(Q, K, V, out, B, H, Lq, Lk, d, k, chunk, causal, scale, dtype, hip_stream, nullptr,
                         nullptr);
}

int topk_attn_noalloc(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H, int64_t Lq,
                      int64_t Lk, int64_t d, int64_t k, int64_t chunk, int causal, float scale, int dtype,
                      void* hip_stream) {
  g_err.clear();
  Problem pb;
  int rc = attn_problem(&pb, Q, K, V, out, B, H, Lq, Lk, d, k, chunk, causal, scale, dtype, nullptr, nullptr, true);
  if (rc) return rc;
  void* ws = nullptr;
  if ((rc = scratch_for_current_device(&ws))) return rc;
  return run(pb, (hipStream_t)hip_stream, false, ws, TOPK_NOALLOC_SCRATCH_BYTES);
}

size_t topk_noalloc_scratch_bytes(void) { return TOPK_NOALLOC_SCRATCH_BYTES; }

int topk_attn_dense(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H, int64_t Lq,
                    int64_t Lk, int64_t d, int64_t chunk, int causal, float scale, int dtype, void* hip_stream) {
  g_err.clear();
  Problem pb;
  // validated as top-k attention with k = 1 (every other check is the same)
  int rc = attn_problem(&pb, Q, K, V, out, B, H, Lq, Lk, d, 1, chunk, causal, scale, dtype, nullptr, nullptr, true);
  if (rc) return rc;
  return run_dense(pb, (hipStream_t)hip_stream);
}

int topk_scan_ablation(const void* Q, const void* K, int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d,
                       int64_t k, int64_t chunk, int score_only, void* hip_stream) {
  g_err.clear();
  Problem pb;
  int rc = attn_problem(&pb, Q, K, K, (void*)Q, B, H, Lq, Lk, d, k, chunk, 0, 1.f, TOPK_BF16, nullptr, nullptr, true);
  if (rc) return rc;
  Plan pl;
  choose_path(pb, &pl);
  if (pl.path != PATH_FUSED || pl.scan.mode != MODE_SAMPLE || pb.d != 64 || pl.scan.union_rank != 20)
    return fail(TOPK_E_UNSUPPORTED, "the scan ablation runs on the sampled fused path with d = 64, 32 < k <= 64");
  pl.scan.score_only = score_only ? 1 : 0;
  plan_sizes(pb, &pl, g_budget.load(std::memory_order_relaxed));
  const size_t need = plan_total(pl, pb);
  hipStream_t st = (hipStream_t)hip_stream;
  char* ws = nullptr;
  if (hipMallocAsync((void**)&ws, need, st) != hipSuccess)
    return fail(TOPK_E_NOMEM, "could not allocate %zu bytes of workspace", need);
  hipError_t e = hipSuccess;
  for (int64_t c0 = 0; c0 < pl.total_chunks && e == hipSuccess; c0 += pl.per_pass) {
    Pass ps;
    ps.c0 = c0;
    ps.nc = pl.total_chunks - c0 < pl.per_pass ? pl.total_chunks - c0 : pl.per_pass;
    ps.nchunk = pl.nchunk;
    PassBufs b = carve(pb, pl, ws);
    e = launch_init(b, st);
    if (e == hipSuccess) {
      StageTimer t(st, ST_SCORE);
      e = launch_fused_scan(pb, ps, b, pl.scan, st);
    }
  }
  hipFreeAsync(ws, st);
  if (e != hipSuccess) return fail(TOPK_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return TOPK_OK;
}

int topk_probe_mfma(double* tflops, double* clock_mhz, void* hip_stream) {
  g_err.clear();
  if (!tflops || !clock_mhz) return fail(TOPK_E_NULL, "tflops and clock_mhz are required");
  hipStream_t st = (hipStream_t)hip_stream;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess)
    return fail(TOPK_E_HIP, "no current HIP device");
  const int blocks = cus * 8;  // two waves per SIMD
  float* sink = nullptr;
  uint64_t* clk = nullptr;
  if (hipMallocAsync((void**)&sink, (size_t)blocks * 256 * 4, st) != hipSuccess ||
      hipMallocAsync((void**)&clk, (size_t)blocks * 16, st) != hipSuccess)
    return fail(TOPK_E_NOMEM, "could not allocate the probe buffers");
  hipEvent_t a, b;
  hipEventCreate(&a);
  hipEventCreate(&b);
  hipError_t e = launch_mfma_rate(sink, clk, blocks, st);  // warm-up
  hipEventRecord(a, st);
  if (e == hipSuccess) e = launch_mfma_rate(sink, clk, blocks, st);
  hipEventRecord(b, st);
  std::vector<uint64_t> h((size_t)blocks * 2);
  if (e == hipSuccess) e = hipMemcpyAsync(h.data(), clk, h.size() * 8, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  hipEventDestroy(a);
  hipEventDestroy(b);
  hipFreeAsync(sink, st);
  hipFreeAsync(clk, st);
  hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(TOPK_E_HIP, "MFMA probe failed: %s", hipGetErrorString(e));
  const double flops = (double)blocks * 4 * mfma_rate_iters() * 8 * 32768.0;
  *tflops = flops / (ms * 1e-3) / 1e12;
  double sum = 0;
  for (int i = 0; i < blocks; ++i) sum += (double)h[2 * i] / (double)(h[2 * i + 1] ? h[2 * i + 1] : 1) * 100.0;
  *clock_mhz = sum / blocks;
  return TOPK_OK;
}

int topk_ffn_debug(const void* X, const void* W1, const void* W2, void* out, int64_t N, int64_t d_model, int64_t d_ff,
                   int64_t k, int64_t chunk, int dtype, void* hip_stream, int32_t* idx_out, float* score_out) {
  g_err.clear();
  Problem pb;
  int rc = ffn_problem(&pb, X, W1, W2, out, N, d_model, d_ff, k, chunk, dtype, idx_out, score_out, true);
  if (rc) return rc;
  if ((rc = debug_ptrs(idx_out, score_out))) return rc;
  return run(pb, (hipStream_t)hip_stream, idx_out != nullptr || score_out != nullptr);
}

int topk_attn_with_cache(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t H, int64_t Lq,
                         int64_t Lk, int64_t d, int64_t k, int64_t chunk, int causal, float scale, int dtype,
                         void* hip_stream, int32_t* top_idx, float* top_dots) {
  g_err.clear();
  if (!top_idx || !top_dots) return fail(TOPK_E_NULL, "top_idx and top_dots are required");
  Problem pb;
  int rc = attn_problem(&pb, Q, K, V, out, B, H, Lq, Lk, d, k, chunk, causal, scale, dtype, top_idx, top_dots, true);
  if (rc) return rc;
  if ((rc = debug_ptrs(top_idx, top_dots))) return rc;
  return run(pb, (hipStream_t)hip_stream, false);
}

int topk_ffn_with_cache(const void* X, const void* W1, const void* W2, void* out, int64_t N, int64_t d_model,
                        int64_t d_ff, int64_t k, int64_t chunk, int dtype, void* hip_stream, int32_t* top_idx,
                        float* top_dots) {
  g_err.clear();
  if (!top_idx || !top_dots) return fail(TOPK_E_NULL, "top_idx and top_dots are required");
  Problem pb;
  int rc = ffn_problem(&pb, X, W1, W2, out, N, d_model, d_ff, k, chunk, dtype, top_idx, top_dots, true);
  if (rc) return rc;
  if ((rc = debug_ptrs(top_idx, top_dots))) return rc;
  return run(pb, (hipStream_t)hip_stream, false);
}

int topk_ffn(const void* X, const void* W1, const void* W2, void* out, int64_t N, int64_t d_model, int64_t d_ff,
             int64_t k, int64_t chunk, int dtype, void* hip_stream) {
  return topk_ffn_debug(X, W1, W2, out, N, d_model, d_ff, k, chunk, dtype, hip_stream, nullptr, nullptr);
}

size_t topk_attn_workspace_bytes(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d, int64_t k, int64_t chunk,
                                 int causal, int dtype) {
  Problem pb;
  if (attn_problem(&pb, nullptr, nullptr, nullptr, nullptr, B, H, Lq, Lk, d, k, chunk, causal, 1.f, dtype, nullptr,
                   nullptr, false))
    return 0;
  return workspace_for(pb);
}

size_t topk_ffn_workspace_bytes(int64_t N, int64_t d_model, int64_t d_ff, int64_t k, int64_t chunk, int dtype) {
  Problem pb;
  if (ffn_problem(&pb, nullptr, nullptr, nullptr, nullptr, N, d_model, d_ff, k, chunk, dtype, nullptr, nullptr, false))
    return 0;
  return workspace_for(pb);
}

int topk_set_workspace(void* dev_ptr, size_t bytes) {
  g_err.clear();
  if (!dev_ptr && bytes > 0) return fail(TOPK_E_NULL, "workspace pointer is NULL");
  if (((uintptr_t)dev_ptr) % ALIGN) return fail(TOPK_E_ALIGN, "workspace must be 256-byte aligned");
  g_ws = bytes ? dev_ptr : nullptr;
  g_ws_bytes = dev_ptr ? bytes : 0;
  return TOPK_OK;
}

int topk_attn_backward(const void* Q, const void* K, const void* V, const int32_t* top_idx, const float* top_dots,
                       const void* d_out, void* d_Q, void* d_K, void* d_V, int64_t B, int64_t H, int64_t Lq,
                       int64_t Lk, int64_t d, int64_t k, float scale, int dtype, void* hip_stream) {
  g_err.clear();
  if (B < 1 || H < 1 || B > (int64_t(1) << 31) / H) return fail(TOPK_E_INVAL, "B and H must be >= 1, B*H < 2^31");
  BwdProblem bp;
  int rc = bwd_problem(&bp, Q, K, V, top_idx, top_dots, d_out, d_Q, d_K, d_V, B * H, Lq, Lk, d, k, Lk * d, scale,
                       dtype, ACT_SOFTMAX, true);
  if (rc) return rc;
  return run_backward(bp, (hipStream_t)hip_stream);
}

int topk_ffn_backward(const void* X, const void* W1, const void* W2, const int32_t* top_idx, const float* top_dots,
                      const void* d_out, void* d_X, void* d_W1, void* d_W2, int64_t N, int64_t d_model, int64_t d_ff,
                      int64_t k, int dtype, void* hip_stream) {
  g_err.clear();
  BwdProblem bp;
  int rc = bwd_problem(&bp, X, W1, W2, top_idx, top_dots, d_out, d_X, d_W1, d_W2, 1, N, d_ff, d_model, k, 0, 1.f,
                       dtype, ACT_RELU, true);
  if (rc) return rc;
  return run_backward(bp, (hipStream_t)hip_stream);
}

size_t topk_attn_backward_workspace_bytes(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d, int64_t k,
                                          int dtype) {
  if (B < 1 || H < 1 || B > (int64_t(1) << 31) / H) return 0;
  BwdProblem bp;
  if (bwd_problem(&bp, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, B * H, Lq,
                  Lk, d, k, Lk * d, 1.f, dtype, ACT_SOFTMAX, false))
    return 0;
  return bwd_bytes(bp);
}

size_t topk_ffn_backward_workspace_bytes(int64_t N, int64_t d_model, int64_t d_ff, int64_t k, int dtype) {
  BwdProblem bp;
  if (bwd_problem(&bp, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 1, N, d_ff,
                  d_model, k, 0, 1.f, dtype, ACT_RELU, false))
    return 0;
  return bwd_bytes(bp);
}

int topk_set_memory_budget(size_t bytes) {
  g_err.clear();
  g_budget.store(bytes ? bytes : DEFAULT_BUDGET, std::memory_order_relaxed);
  return TOPK_OK;
}

int topk_set_backward_lists(int mode) {
  g_err.clear();
  if (mode != TOPK_LISTS_AUTO && mode != TOPK_LISTS_BUCKET && mode != TOPK_LISTS_ATOMIC)
    return fail(TOPK_E_INVAL, "backward list mode must be TOPK_LISTS_AUTO, _BUCKET or _ATOMIC (got %d)", mode);
  g_list_mode.store(mode, std::memory_order_relaxed);
  return TOPK_OK;
}

const char* topk_last_error(void) { return g_err.c_str(); }

int64_t topk_debug_bad_indices(void) { return read_bad_indices(); }

int64_t topk_last_fallback_rows(void) { return g_fallback_rows; }

int topk_attn_path(int64_t B, int64_t H, int64_t Lq, int64_t Lk, int64_t d, int64_t k, int64_t chunk, int causal,
                   int dtype) {
  Problem pb;
  int rc = attn_problem(&pb, nullptr, nullptr, nullptr, nullptr, B, H, Lq, Lk, d, k, chunk, causal, 1.f, dtype,
                        nullptr, nullptr, false);
  if (rc) return rc;
  Problem parts[2];
  if (split_rows(pb, parts) == 2) return 3;
  Plan pl;
  choose_path(parts[0], &pl);
  return pl.path;
}

int topk_ffn_path(int64_t N, int64_t d_model, int64_t d_ff, int64_t k, int64_t chunk, int dtype) {
  Problem pb;
  int rc = ffn_problem(&pb, nullptr, nullptr, nullptr, nullptr, N, d_model, d_ff, k, chunk, dtype, nullptr, nullptr,
                       false);
  if (rc) return rc;
  Plan pl;
  choose_path(pb, &pl);
  return pl.path;
}

int topk_profile_begin(void) {
  g_err.clear();
  for (auto& m : g_marks) {
    hipEventDestroy(m.a);
    hipEventDestroy(m.b);
  }
  g_marks.clear();
  g_prof = true;
  return TOPK_OK;
}

int topk_profile_end(double* stage_ms, int64_t* stage_launches, int n_stages) {
  g_err.clear();
  g_prof = false;
  int rc = TOPK_OK;
  for (int s = 0; s < n_stages; ++s) {
    if (stage_ms) stage_ms[s] = 0.0;
    if (stage_launches) stage_launches[s] = 0;
  }
  for (auto& m : g_marks) {
    float ms = 0.f;
    if (hipEventSynchronize(m.b) != hipSuccess || hipEventElapsedTime(&ms, m.a, m.b) != hipSuccess)
      rc = fail(TOPK_E_HIP, "could not read stage timing events");
    if (m.stage < n_stages) {
      if (stage_ms) stage_ms[m.stage] += ms;
      if (stage_launches) stage_launches[m.stage] += 1;
    }
    hipEventDestroy(m.a);
    hipEventDestroy(m.b);
  }
  g_marks.clear();
  return rc;
}

int topk_selftest_mfma_layout(int32_t* rows_out, int32_t* cols_out, void* hip_stream) {
  g_err.clear();
  int rc;
  if ((rc = check_ptr(rows_out, "rows_out")) || (rc = check_ptr(cols_out, "cols_out"))) return rc;
  hipError_t e = launch_mfma_probe(rows_out, cols_out, (hipStream_t)hip_stream);
  if (e != hipSuccess) return fail(TOPK_E_HIP, "probe launch failed: %s", hipGetErrorString(e));
  return TOPK_OK;
}

}  // extern "C"
