// gfx950 kernels of the top-k attention forward pass (arXiv 2106.06899, Eq. 4).
//
// Two ways to reach each query row's top-k set, both ending in the same
// selection format and the same finalize kernel:
//
//  * chunk-tile path: the chunk's score tile Q_C K^T is written to workspace
//    (the O(C * Lk) memory of the paper's query chunking, Section 2.2), then one
//    workgroup per row runs an exact radix select over it;
//  * fused path: bf16 MFMA score tiles are compared on chip against a per-query
//    threshold, and only the survivors (candidates) leave the chip; a per-row
//    select over the candidates yields the top-k. The threshold comes from a
//    strided sample of key tiles; a row whose candidate set cannot be proven to
//    contain its top-k is recomputed exactly by the fallback kernel.
//
// Selected keys are 64-bit words  (ord(score) << 32) | (0xFFFFFFFF - index)  so
// that one unsigned comparison implements the total order (score desc, index
// asc) used for ties; ord() maps fp32 to an order-preserving u32, with -0 == +0.
#include "topk_internal.h"

#include <math.h>

namespace topk {

typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef float f32x16 __attribute__((__vector_size__(64)));

// ------------------------------------------------------------------ scalar helpers
__device__ __forceinline__ uint32_t ord_u32(float s) {
  uint32_t b = __float_as_uint(s);
  if ((b << 1) == 0u) b = 0u;  // -0 and +0 are the same score
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float ord_to_f32(uint32_t u) {
  uint32_t b = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(b);
}
__device__ __forceinline__ uint64_t make_key(float s, uint32_t j) {
  return ((uint64_t)ord_u32(s) << 32) | (uint64_t)(0xFFFFFFFFu - j);
}
__device__ __forceinline__ float key_score(uint64_t key) { return ord_to_f32((uint32_t)(key >> 32)); }
__device__ __forceinline__ uint32_t key_index(uint64_t key) { return 0xFFFFFFFFu - (uint32_t)key; }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {  // nearest-even, finite inputs
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}
template <typename T> __device__ __forceinline__ float load_elem(const void* p, int64_t e);
template <> __device__ __forceinline__ float load_elem<float>(const void* p, int64_t e) {
  return ((const float*)p)[e];
}
template <> __device__ __forceinline__ float load_elem<uint16_t>(const void* p, int64_t e) {
  return bf16_to_f32(((const uint16_t*)p)[e]);
}
template <typename T> __device__ __forceinline__ void store_elem(void* p, int64_t e, float v);
template <> __device__ __forceinline__ void store_elem<float>(void* p, int64_t e, float v) { ((float*)p)[e] = v; }
template <> __device__ __forceinline__ void store_elem<uint16_t>(void* p, int64_t e, float v) {
  ((uint16_t*)p)[e] = f32_to_bf16(v);
}

// Pass-local row -> (head, query index); false for padding rows of a partial chunk.
struct RowRef {
  int64_t bh, i;
  bool ok;
};
__device__ __forceinline__ RowRef row_of(const Problem& pb, const Pass& ps, int64_t p) {
  int64_t chunk_local = p / pb.C, r = p - chunk_local * pb.C;
  int64_t id = ps.c0 + chunk_local;
  RowRef rr;
  rr.bh = id / ps.nchunk;
  rr.i = (id - rr.bh * ps.nchunk) * pb.C + r;
  rr.ok = chunk_local < ps.nc && rr.i < pb.Lq;
  return rr;
}
__device__ __forceinline__ int64_t valid_keys(const Problem& pb, int64_t i) {
  return pb.causal ? (i + 1 < pb.Lk ? i + 1 : pb.Lk) : pb.Lk;
}

// ------------------------------------------------------------------ team primitives
// A "team" is one workgroup of NT threads (NT = 64 or 256); all sync is __syncthreads.
template <int NT>
__device__ __forceinline__ uint32_t team_excl_scan(uint32_t x, uint32_t* tmp) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint32_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (NT == 64) return incl - x;
  if (lane == 63) tmp[w] = incl;
  __syncthreads();
  uint32_t base = 0;
  for (int q = 0; q < w; ++q) base += tmp[q];
  __syncthreads();
  return base + incl - x;
}

// Exact radix select of the k_eff largest keys among n (distinct) 64-bit keys,
// 8 bits per pass from the top. On return the selected set is exactly
// { key : (key >> shift) >= (prefix >> shift) }.
template <int NT, class GetKey>
__device__ void team_radix_select(const GetKey& getkey, int64_t n, uint32_t k_eff, uint32_t* hist,
                                  uint32_t* misc, int* shift_out, uint64_t* prefix_out) {
  uint64_t prefix = 0;
  int shift = 64;
  uint32_t kr = k_eff;
  for (int pass = 0; pass < 8; ++pass) {
    shift -= 8;
    for (int b = threadIdx.x; b < 256; b += NT) hist[b] = 0;
    __syncthreads();
    for (int64_t e = threadIdx.x; e < n; e += NT) {
      const uint64_t key = getkey(e);
      const bool match = pass == 0 || (key >> (shift + 8)) == (prefix >> (shift + 8));
      if (match) atomicAdd(&hist[(uint32_t)(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    constexpr int BPT = 256 / NT;
    uint32_t c[BPT];
    uint32_t local = 0;
#pragma unroll
    for (int e = 0; e < BPT; ++e) {
      c[e] = hist[255 - (threadIdx.x * BPT + e)];  // bins in descending digit order
      local += c[e];
    }
    uint32_t run = team_excl_scan<NT>(local, misc);
#pragma unroll
    for (int e = 0; e < BPT; ++e) {
      if (run < kr && kr <= run + c[e]) {
        misc[4] = 255u - (uint32_t)(threadIdx.x * BPT + e);
        misc[5] = run;
        misc[6] = c[e];
      }
      run += c[e];
    }
    __syncthreads();
    const uint32_t digit = misc[4], above = misc[5], cnt = misc[6];
    __syncthreads();
    prefix |= (uint64_t)digit << shift;
    kr -= above;
    if (cnt == kr) break;  // every key of this bucket is selected
  }
  *shift_out = shift;
  *prefix_out = prefix;
}

// Bitonic sort of P (power of two) keys in LDS, descending.
template <int NT>
__device__ void team_sort_desc(uint64_t* s, int P) {
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = threadIdx.x; t < (P >> 1); t += NT) {
        const int i = 2 * stride * (t / stride) + (t % stride);
        const int j = i + stride;
        const bool desc = (i & size) == 0;
        const uint64_t a = s[i], b = s[j];
        if ((a < b) == desc) {
          s[i] = b;
          s[j] = a;
        }
      }
      __syncthreads();
    }
  }
}

// Select the k_eff largest of n keys, sort them and write k words to out (0 pads).
// sbuf holds P >= k_eff keys (power of two).
template <int NT, class GetKey>
__device__ void team_topk(const GetKey& getkey, int64_t n, uint32_t k_eff, uint32_t k, uint64_t* sbuf, int P,
                          uint32_t* hist, uint32_t* misc, uint64_t* out) {
  int shift;
  uint64_t prefix;
  team_radix_select<NT>(getkey, n, k_eff, hist, misc, &shift, &prefix);
  const uint64_t lim = prefix >> shift;
  if (threadIdx.x == 0) misc[7] = 0;
  for (int t = threadIdx.x; t < P; t += NT) sbuf[t] = 0;
  __syncthreads();
  for (int64_t e = threadIdx.x; e < n; e += NT) {
    const uint64_t key = getkey(e);
    if ((key >> shift) >= lim) {
      const uint32_t pos = atomicAdd(&misc[7], 1u);
      if (pos < (uint32_t)P) sbuf[pos] = key;
    }
  }
  __syncthreads();
  team_sort_desc<NT>(sbuf, P);
  for (uint32_t t = threadIdx.x; t < k; t += NT) out[t] = t < k_eff ? sbuf[t] : 0ull;
}

__host__ __device__ __forceinline__ int pow2_at_least(int64_t x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// ------------------------------------------------------------------ init
__global__ void k_init(int32_t* redo_count) {
  if (threadIdx.x == 0) *redo_count = 0;
}

// ------------------------------------------------------------------ chunk-tile path: scores
// Block = 64 query rows x 64 keys of one chunk, fp32 FMA from LDS tiles of 16 features.
template <typename T>
__global__ __launch_bounds__(256) void k_tile_scores(Problem pb, Pass ps, float* S) {
  __shared__ float qs[16][65];
  __shared__ float ks[16][65];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int64_t key0 = (int64_t)blockIdx.x * 64, r0 = (int64_t)blockIdx.y * 64, cl = blockIdx.z;
  const int64_t id = ps.c0 + cl, bh = id / ps.nchunk, c = id - bh * ps.nchunk, i0 = c * pb.C;
  if (r0 >= pb.C || i0 + r0 >= pb.Lq) return;
  if (pb.causal) {
    int64_t last = r0 + 63 < pb.C ? r0 + 63 : pb.C - 1;
    if (key0 > i0 + last) return;  // tile entirely above the diagonal: never read
  }
  const int64_t d = pb.d;
  const char* Kh = (const char*)pb.K + bh * pb.kv_head_stride * (int64_t)sizeof(T);
  float acc[4][4] = {};
  for (int64_t d0 = 0; d0 < d; d0 += 16) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int e = tid + 256 * m, rr = e >> 4, cc = e & 15;
      const int64_t lr = r0 + rr, i = i0 + lr, key = key0 + rr, f = d0 + cc;
      qs[cc][rr] = (lr < pb.C && i < pb.Lq && f < d) ? load_elem<T>(pb.Q, (bh * pb.Lq + i) * d + f) : 0.f;
      ks[cc][rr] = (key < pb.Lk && f < d) ? load_elem<T>(Kh, key * d + f) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int cc = 0; cc < 16; ++cc) {
      float qv[4], kv[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        qv[a] = qs[cc][ty * 4 + a];
        kv[a] = ks[cc][tx * 4 + a];
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = fmaf(qv[a], kv[b], acc[a][b]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int64_t lr = r0 + ty * 4 + a, i = i0 + lr;
    if (lr >= pb.C || i >= pb.Lq) continue;
    const int64_t nv = valid_keys(pb, i);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int64_t key = key0 + tx * 4 + b;
      if (key < nv) S[(cl * pb.C + lr) * pb.Lk + key] = acc[a][b];
    }
  }
}

// ------------------------------------------------------------------ chunk-tile path: select
__global__ __launch_bounds__(256) void k_tile_select(Problem pb, Pass ps, const float* S, uint64_t* sel) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  const float* row = S + p * pb.Lk;
  auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
  team_topk<256>(getkey, nv, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc, sel + p * pb.k);
}

// ------------------------------------------------------------------ fused path: scan
// One workgroup = 4 waves x 32 queries of one head. The B operand (32 queries x d)
// stays in registers; key tiles of 64 rows are staged in LDS; each wave computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so lane l holds 16 keys' scores of
// query l % 32 (keys 8*(v/4) + 4*(l/32) + v%4 of the 32-key block, v = 0..15).
// The feature dimension is split between the half-waves: lane half h holds
// features [h*D/2, h*D/2 + D/2) of its row in both operands (the contraction is
// order-free), so every lane loads 2*(D/2) contiguous bytes.
struct ScanArgs {
  const uint16_t* Q;
  const uint16_t* K;
  int64_t Lq, Lk, C, kv_head_stride;
  int64_t c0, nchunk, wgs_per_chunk;
  uint64_t* cand;
  int32_t* cnt;
  int64_t caph;
  int mode, stride;
};

template <int D, int R>
__global__ __launch_bounds__(256) void k_fused_scan(ScanArgs a) {
  constexpr int KT = 64;             // keys per LDS tile (two 32-key MFMA blocks)
  constexpr int ROWB = 2 * D + 16;   // padded LDS row (bytes): conflict-free 16-byte reads
  constexpr int NS = D / 16;         // MFMA steps over the features
  constexpr int CH = 2 * D / 16;     // 16-byte pieces per key row
  __shared__ __attribute__((aligned(16))) unsigned char ks[KT * ROWB];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5, n = lane & 31;
  const int64_t wg = blockIdx.x, cl = wg / a.wgs_per_chunk, blk = wg - cl * a.wgs_per_chunk;
  const int64_t id = a.c0 + cl, bh = id / a.nchunk, c = id - bh * a.nchunk;
  const int64_t local = blk * 128 + wave * 32 + n, i = c * a.C + local;
  const bool row_ok = local < a.C && i < a.Lq;
  const int64_t p = cl * a.C + local;
  const uint16_t* Kh = a.K + bh * a.kv_head_stride;
  const int64_t ntiles = (a.Lk + KT - 1) / KT;

  bf16x8 b[NS];
  {
    const bf16x8 zero8 = {};
    const uint16_t* q = a.Q + (bh * a.Lq + (row_ok ? i : 0)) * D + (D / 2) * half;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      b[s] = *(const bf16x8*)(q + 8 * s);
      if (!row_ok) b[s] = zero8;
    }
  }

  auto load_tile = [&](int64_t t) {
    const int64_t key0 = t * KT;
#pragma unroll
    for (int cidx = tid; cidx < KT * CH; cidx += 256) {
      const int kr = cidx / CH, part = cidx - kr * CH;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (key0 + kr < a.Lk) v = *(const uint4*)(Kh + (key0 + kr) * D + part * 8);
      *(uint4*)(ks + kr * ROWB + part * 16) = v;
    }
  };
  auto block_scores = [&](int rb) {
    f32x16 acc = {};
    const unsigned char* base = ks + (rb * 32 + n) * ROWB + half * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 av = *(const bf16x8*)(base + 16 * s);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, b[s], acc, 0, 0, 0);
    }
    return acc;
  };
  auto mask_tail = [&](f32x16& acc, int64_t jb) {  // keys >= Lk of the last tile -> -inf
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (jb + 8 * (v >> 2) + (v & 3) >= a.Lk) acc[v] = -INFINITY;
  };

  float tau = -INFINITY;
  if (a.mode == MODE_SAMPLE) {
    float top[R];
#pragma unroll
    for (int r = 0; r < R; ++r) top[r] = -INFINITY;
    for (int64_t t = 0; t < ntiles; t += a.stride) {
      __syncthreads();
      load_tile(t);
      __syncthreads();
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        f32x16 acc = block_scores(rb);
        if ((t + 1) * KT > a.Lk) mask_tail(acc, t * KT + rb * 32 + 4 * half);
        float m = acc[0];
#pragma unroll
        for (int v = 1; v < 16; ++v) m = fmaxf(m, acc[v]);
#pragma unroll
        for (int r = 0; r < R; ++r) {  // sorted insert, descending
          const float hi = fmaxf(top[r], m);
          m = fminf(top[r], m);
          top[r] = hi;
        }
      }
    }
    const float mine = top[R - 1];
    tau = fminf(mine, __shfl_xor(mine, 32, 64));
  }
  if (!row_ok) tau = INFINITY;

  uint64_t* mybuf = a.cand + (p * 2 + half) * a.caph;
  int cnt = 0;
  for (int64_t t = 0; t < ntiles; ++t) {
    __syncthreads();
    load_tile(t);
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      f32x16 acc = block_scores(rb);
      const int64_t jb = t * KT + rb * 32 + 4 * half;
      if ((t + 1) * KT > a.Lk) mask_tail(acc, jb);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        if (acc[v] > tau) {
          if (cnt < a.caph) mybuf[cnt] = make_key(acc[v], (uint32_t)(jb + 8 * (v >> 2) + (v & 3)));
          ++cnt;
        }
      }
    }
  }
  if (row_ok) a.cnt[p * 2 + half] = cnt;
}

// ------------------------------------------------------------------ fused path: select
// One wave per row. A row whose candidates overflowed, or (threshold mode) hold
// fewer than k_eff keys, goes to the redo list; otherwise the candidate set is
// proven to contain the row's top-k and an exact select runs over it.
__global__ __launch_bounds__(64) void k_cand_select(Problem pb, Pass ps, PassBufs bufs) {
  __shared__ uint64_t sbuf[256];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  const int64_t c0 = bufs.cnt[2 * p], c1 = bufs.cnt[2 * p + 1];
  if (c0 > bufs.caph || c1 > bufs.caph || c0 + c1 < (int64_t)k_eff || k_eff > 256) {
    if (threadIdx.x == 0) bufs.redo_list[atomicAdd(bufs.redo_count, 1)] = (int32_t)p;
    return;
  }
  const uint64_t* b0 = bufs.cand + (2 * p) * bufs.caph;
  const uint64_t* b1 = b0 + bufs.caph;
  auto getkey = [&](int64_t e) { return e < c0 ? b0[e] : b1[e - c0]; };
  team_topk<64>(getkey, c0 + c1, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc,
                bufs.sel + p * pb.k);
}

// ------------------------------------------------------------------ fused path: fallback
// Exact recomputation of the rows on the redo list: fp32 dot products of the row
// against every valid key into a per-block row buffer, then the same radix select.
template <typename T>
__global__ __launch_bounds__(256) void k_redo(Problem pb, Pass ps, PassBufs bufs) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  __shared__ float qrow[1024];
  float* row = bufs.scores + (int64_t)blockIdx.x * pb.Lk;
  const int32_t total = *bufs.redo_count;
  for (int32_t t = blockIdx.x; t < total; t += gridDim.x) {
    const int64_t p = bufs.redo_list[t];
    const RowRef rr = row_of(pb, ps, p);
    const int64_t nv = valid_keys(pb, rr.i);
    const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
    for (int f = threadIdx.x; f < pb.d; f += 256) qrow[f] = load_elem<T>(pb.Q, (rr.bh * pb.Lq + rr.i) * pb.d + f);
    __syncthreads();
    const char* Kh = (const char*)pb.K + rr.bh * pb.kv_head_stride * (int64_t)sizeof(T);
    for (int64_t j = threadIdx.x; j < nv; j += 256) {
      float s = 0.f;
      for (int64_t f = 0; f < pb.d; ++f) s = fmaf(qrow[f], load_elem<T>(Kh, j * pb.d + f), s);
      row[j] = s;
    }
    __syncthreads();
    auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
    team_topk<256>(getkey, nv, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc, bufs.sel + p * pb.k);
    __syncthreads();
  }
}

// ------------------------------------------------------------------ finalize
// One wave per row: activation over the k_eff survivors (softmax with the Eq. 1
// temperature, or ReLU), then the weighted sum of the selected value rows.
template <typename T>
__global__ __launch_bounds__(64) void k_finalize(Problem pb, Pass ps, const uint64_t* sel) {
  extern __shared__ float fsh[];
  float* w = fsh;
  uint32_t* jj = (uint32_t*)(fsh + pb.k);
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int64_t nv = valid_keys(pb, rr.i);
  const int64_t k_eff = pb.k < nv ? pb.k : nv;
  const int64_t grow = rr.bh * pb.Lq + rr.i;
  const uint64_t* srow = sel + p * pb.k;
  for (int64_t t = threadIdx.x; t < pb.k; t += 64) {
    float s = -INFINITY;
    int32_t j = -1;
    if (t < k_eff) {
      const uint64_t key = srow[t];
      s = key_score(key);
      j = (int32_t)key_index(key);
      w[t] = s;
      jj[t] = (uint32_t)j;
    }
    if (pb.idx_out) pb.idx_out[grow * pb.k + t] = j;
    if (pb.score_out) pb.score_out[grow * pb.k + t] = s;
  }
  __syncthreads();
  float inv = 1.f;
  if (pb.act == ACT_SOFTMAX) {
    const float m = w[0];
    const float c = pb.scale * 1.4426950408889634f;  // exp(x) = exp2(x * log2 e)
    float sum = 0.f;
    for (int64_t t = threadIdx.x; t < k_eff; t += 64) {
      const float e = exp2f((w[t] - m) * c);
      w[t] = e;
      sum += e;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
    inv = 1.f / sum;
  } else {
    for (int64_t t = threadIdx.x; t < k_eff; t += 64) w[t] = fmaxf(w[t], 0.f);
  }
  __syncthreads();
  const char* Vh = (const char*)pb.V + rr.bh * pb.kv_head_stride * (int64_t)sizeof(T);
  const uint32_t jmax = (uint32_t)(pb.Lk - 1);
  for (int64_t col = threadIdx.x; col < pb.d; col += 64) {
    float acc = 0.f;
    for (int64_t t = 0; t < k_eff; ++t) {
      const uint32_t j = jj[t] < jmax ? jj[t] : jmax;  // keeps a bad selection from reading out of bounds
      acc = fmaf(w[t], load_elem<T>(Vh, (int64_t)j * pb.d + col), acc);
    }
    store_elem<T>(pb.out, grow * pb.d + col, acc * inv);
  }
}

// ------------------------------------------------------------------ MFMA layout probe
__global__ void k_mfma_probe(int32_t* rows, int32_t* cols) {
  const int l = threadIdx.x;
  union U {
    bf16x8 v;
    uint16_t h[8];
  };
  U a, b, a1, b1;
  for (int e = 0; e < 8; ++e) a.h[e] = b.h[e] = a1.h[e] = b1.h[e] = 0;
  if (l < 32) {  // only element 0 of the lower half-wave is non-zero: the k = 0 slice
    a.h[0] = f32_to_bf16((float)l);
    b.h[0] = f32_to_bf16(1.f);
    a1.h[0] = f32_to_bf16(1.f);
    b1.h[0] = f32_to_bf16((float)l);
  }
  f32x16 z = {};
  const f32x16 r = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, z, 0, 0, 0);   // D[m][n] = m
  const f32x16 c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1.v, b1.v, z, 0, 0, 0); // D[m][n] = n
  for (int v = 0; v < 16; ++v) {
    rows[l * 16 + v] = (int32_t)r[v];
    cols[l * 16 + v] = (int32_t)c[v];
  }
}

// ------------------------------------------------------------------ launchers
static int64_t pass_rows(const Problem& pb, const Pass& ps) { return ps.nc * pb.C; }

hipError_t launch_init(const PassBufs& b, hipStream_t st) {
  k_init<<<1, 64, 0, st>>>(b.redo_count);
  return hipGetLastError();
}

hipError_t launch_tile_scores(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  dim3 grid((unsigned)((pb.Lk + 63) / 64), (unsigned)((pb.C + 63) / 64), (unsigned)ps.nc);
  if (pb.dtype == T_BF16)
    k_tile_scores<uint16_t><<<grid, 256, 0, st>>>(pb, ps, b.scores);
  else
    k_tile_scores<float><<<grid, 256, 0, st>>>(pb, ps, b.scores);
  return hipGetLastError();
}

hipError_t launch_tile_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const int P = pow2_at_least(pb.k);
  k_tile_select<<<(unsigned)pass_rows(pb, ps), 256, (size_t)P * 8, st>>>(pb, ps, b.scores, b.sel);
  return hipGetLastError();
}

hipError_t launch_fused_scan(const Problem& pb, const Pass& ps, const PassBufs& b, const ScanCfg& cfg,
                             hipStream_t st) {
  ScanArgs a;
  a.Q = (const uint16_t*)pb.Q;
  a.K = (const uint16_t*)pb.K;
  a.Lq = pb.Lq;
  a.Lk = pb.Lk;
  a.C = pb.C;
  a.kv_head_stride = pb.kv_head_stride;
  a.c0 = ps.c0;
  a.nchunk = ps.nchunk;
  a.wgs_per_chunk = (pb.C + 127) / 128;
  a.cand = b.cand;
  a.cnt = b.cnt;
  a.caph = b.caph;
  a.mode = cfg.mode;
  a.stride = cfg.stride;
  const unsigned grid = (unsigned)(ps.nc * a.wgs_per_chunk);
#define TOPK_SCAN(D_, R_) k_fused_scan<D_, R_><<<grid, 256, 0, st>>>(a)
  if (pb.d == 64) {
    if (cfg.R == 4) TOPK_SCAN(64, 4);
    else if (cfg.R == 8) TOPK_SCAN(64, 8);
    else TOPK_SCAN(64, 16);
  } else {
    if (cfg.R == 4) TOPK_SCAN(128, 4);
    else if (cfg.R == 8) TOPK_SCAN(128, 8);
    else TOPK_SCAN(128, 16);
  }
#undef TOPK_SCAN
  return hipGetLastError();
}

hipError_t launch_cand_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  k_cand_select<<<(unsigned)pass_rows(pb, ps), 64, 0, st>>>(pb, ps, b);
  return hipGetLastError();
}

hipError_t launch_redo(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const int P = pow2_at_least(pb.k);
  if (pb.dtype == T_BF16)
    k_redo<uint16_t><<<REDO_BLOCKS, 256, (size_t)P * 8, st>>>(pb, ps, b);
  else
    k_redo<float><<<REDO_BLOCKS, 256, (size_t)P * 8, st>>>(pb, ps, b);
  return hipGetLastError();
}

hipError_t launch_finalize(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const size_t sh = (size_t)pb.k * 8;
  if (pb.dtype == T_BF16)
    k_finalize<uint16_t><<<(unsigned)pass_rows(pb, ps), 64, sh, st>>>(pb, ps, b.sel);
  else
    k_finalize<float><<<(unsigned)pass_rows(pb, ps), 64, sh, st>>>(pb, ps, b.sel);
  return hipGetLastError();
}

hipError_t launch_mfma_probe(int32_t* rows, int32_t* cols, hipStream_t st) {
  k_mfma_probe<<<1, 64, 0, st>>>(rows, cols);
  return hipGetLastError();
}

}  // namespace topk
