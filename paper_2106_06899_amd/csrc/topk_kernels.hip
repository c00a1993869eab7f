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

#include <type_traits>

namespace topk {

typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef float f32x16 __attribute__((__vector_size__(64)));

// s_waitcnt immediate that waits until at most n vector-memory operations are
// outstanding and does not wait on the other counters
#define TOPK_WAIT_VM(n) (((n) & 15) | (7 << 4) | (15 << 8) | (((n) >> 4) << 14))

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
  int64_t chunk_local, r, id, c;
  RowRef rr;
  if (((uint64_t)p | (uint64_t)pb.C | (uint64_t)(ps.c0 + ps.nc) | (uint64_t)ps.nchunk) >> 31 == 0) {
    // the common case: 32-bit divisions (a few instructions instead of a 64-bit routine)
    const uint32_t cl32 = (uint32_t)p / (uint32_t)pb.C, id32 = (uint32_t)ps.c0 + cl32;
    chunk_local = cl32;
    r = (uint32_t)p - cl32 * (uint32_t)pb.C;
    id = id32;
    rr.bh = id32 / (uint32_t)ps.nchunk;
    c = id32 - (uint32_t)rr.bh * (uint32_t)ps.nchunk;
  } else {
    chunk_local = p / pb.C;
    r = p - chunk_local * pb.C;
    id = ps.c0 + chunk_local;
    rr.bh = id / ps.nchunk;
    c = id - rr.bh * ps.nchunk;
  }
  rr.i = pb.q0 + c * pb.C + r;
  rr.ok = chunk_local < ps.nc && rr.i < pb.q1;
  return rr;
}
__device__ __forceinline__ int64_t valid_keys(const Problem& pb, int64_t i) {
  return pb.causal ? (i + 1 < pb.Lk ? i + 1 : pb.Lk) : pb.Lk;
}

// ------------------------------------------------------------------ team primitives
// Orders one wave's LDS accesses around this point for the compiler; the hardware
// runs a wave's LDS instructions in order, so a wave sees its own earlier writes
// and atomics without a workgroup barrier.
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

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

// Digits a sampled threshold resolves: the sign, the exponent and the top 7 bits of the
// mantissa of the R-th largest sample (finer resolution only trims a few candidates).
constexpr int THRESH_PASSES = 2;

// Exact radix select of the k_eff largest keys among n (distinct) 64-bit keys,
// 8 bits per pass from the top. On return the selected set is exactly
// { key : (key >> shift) >= (prefix >> shift) }. With max_passes < 8 it stops early
// and the set holds the k_eff largest keys and possibly more (the rest of the last
// digit's bucket), which is all a threshold needs.
template <int NT, class GetKey>
__device__ void team_radix_select(const GetKey& getkey, int64_t n, uint32_t k_eff, uint32_t* hist,
                                  uint32_t* misc, int* shift_out, uint64_t* prefix_out, int max_passes = 8) {
  uint64_t prefix = 0;
  int shift = 64;
  uint32_t kr = k_eff;
  for (int pass = 0; pass < max_passes; ++pass) {
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
  const int64_t id = ps.c0 + cl, bh = id / ps.nchunk, c = id - bh * ps.nchunk, i0 = pb.q0 + c * pb.C;
  if (r0 >= pb.C || i0 + r0 >= pb.q1) return;
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
      qs[cc][rr] = (lr < pb.C && i < pb.q1 && f < d) ? load_elem<T>(pb.Q, (bh * pb.Lq + i) * d + f) : 0.f;
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
    if (lr >= pb.C || i >= pb.q1) continue;
    const int64_t nv = valid_keys(pb, i);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int64_t key = key0 + tx * 4 + b;
      if (key < nv) S[(cl * pb.C + lr) * pb.Lk + key] = acc[a][b];
    }
  }
}

// ------------------------------------------------------------------ chunk-tile path: MFMA scores
// bf16 inputs with d % 32 == 0: a 128-query x 256-key tile per workgroup, the
// feature dimension consumed 32 at a time. Each slice of Q (128 rows x 64 bytes)
// and K (256 rows x 64 bytes) is loaded straight from global memory into one of
// two LDS buffers (global_load_lds, no register staging); 16-byte part p of row r
// sits at position 4r + (p ^ ((r >> 1) & 3)), so the fragment reads of 8
// consecutive rows hit 8 different bank groups. Each wave owns 64 queries x 128
// keys = 2 x 4 blocks of v_mfma_f32_32x32x16_bf16 with A = K (rows = keys) and
// B = Q^T (columns = queries): per 16 features it reads 6 fragments for 8 MFMAs,
// and lane l holds keys 8*(v/4) + 4*(l/32) + v%4 of a block for query l % 32,
// four consecutive keys of one score row per 16-byte store. Tiles entirely above
// the causal diagonal are skipped (never read by the select).
// MODE 0 writes the tile; MODE 1 scores every FILTER_KSTRIDE-th key only (the
// filtered path's sample, "keys" of the grid are sample slots); MODE 2 appends the
// scores at or above each row's threshold to the row's candidate list instead of
// writing the tile.
constexpr int TSM_TQ = 128, TSM_TK = 256;

template <int MODE>
__global__ __launch_bounds__(256, 2) void k_tile_scores_mfma(Problem pb, Pass ps, PassBufs bufs) {
  constexpr int64_t KSTEP = MODE == 1 ? FILTER_KSTRIDE : 1;  // key index of grid key slot s: s * KSTEP
  constexpr int TQ = TSM_TQ, TK = TSM_TK, KS = 32;  // tile rows, tile keys, features per slice
  constexpr int QBYTES = TQ * KS * 2, KBYTES = TK * KS * 2;
  constexpr int QLPW = QBYTES / 1024 / 4, KLPW = KBYTES / 1024 / 4;  // 1 KB loads per wave
  __shared__ __attribute__((aligned(16))) unsigned char sm[2][QBYTES + KBYTES];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5, n = lane & 31;
  // Workgroup order: query tiles fastest, then key tiles, then chunks, renumbered
  // so each XCD runs a contiguous range. The query tiles of one chunk then read
  // the same K tile at about the same time from their XCD's L2, and the chunk's
  // Q stays in L2 while K streams past once per chunk.
  const int64_t NG = gridDim.x, bid = blockIdx.x;
  const int64_t wg = (NG % 8 == 0) ? (bid % 8) * (NG / 8) + bid / 8 : bid;
  const int64_t Lslots = (pb.Lk + KSTEP - 1) / KSTEP;  // key slots of the grid
  const int64_t nq = (pb.C + TQ - 1) / TQ, nk = (Lslots + TK - 1) / TK;
  const int64_t qt = wg % nq, kt = (wg / nq) % nk, cl = wg / (nq * nk);
  const int64_t key0 = kt * TK, r0 = qt * TQ;
  const int64_t id = ps.c0 + cl, bh = id / ps.nchunk, c = id - bh * ps.nchunk, i0 = pb.q0 + c * pb.C;
  if (r0 >= pb.C || i0 + r0 >= pb.q1) return;
  if (pb.causal) {
    const int64_t last = r0 + TQ - 1 < pb.C ? r0 + TQ - 1 : pb.C - 1;
    if (key0 * KSTEP > i0 + last) return;
  }
  const int64_t d = pb.d;
  const uint16_t* Qb = (const uint16_t*)pb.Q;
  const uint16_t* Kh = (const uint16_t*)pb.K + bh * pb.kv_head_stride;
  // rows past the chunk / sequence load the tile's first row (their scores are
  // never stored); keys past Lk load the last key
  auto issue = [&](int64_t f0, int buf) {
#pragma unroll
    for (int j = 0; j < QLPW; ++j) {
      const int cidx = (wave * QLPW + j) * 64 + lane, r = cidx >> 2, p = (cidx & 3) ^ ((r >> 1) & 3);
      const int64_t lr = r0 + r, i = i0 + lr;
      const int64_t qi = (lr < pb.C && i < pb.q1) ? i : i0 + r0;
      __builtin_amdgcn_global_load_lds((const void*)(Qb + (bh * pb.Lq + qi) * d + f0 + p * 8),
                                       (__attribute__((address_space(3))) void*)&sm[buf][(wave * QLPW + j) * 1024],
                                       16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < KLPW; ++j) {
      const int cidx = (wave * KLPW + j) * 64 + lane, r = cidx >> 2, p = (cidx & 3) ^ ((r >> 1) & 3);
      int64_t key = (key0 + r) * KSTEP;
      key = key < pb.Lk ? key : pb.Lk - 1;
      __builtin_amdgcn_global_load_lds(
          (const void*)(Kh + key * d + f0 + p * 8),
          (__attribute__((address_space(3))) void*)&sm[buf][QBYTES + (wave * KLPW + j) * 1024], 16, 0, 0);
    }
  };
  auto frag = [&](const unsigned char* base, int r, int st) {  // features 16*st + 8*half .. +8 of row r
    const int p = 2 * st + half;
    return *(const bf16x8*)(base + (r * 4 + (p ^ ((r >> 1) & 3))) * 16);
  };
  const int wq = (wave >> 1) * 64, wk = (wave & 1) * 128;  // this wave's 64 x 128 sub-tile
  f32x16 acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = (f32x16){};
  const int64_t nsl = d / KS;
  issue(0, 0);
  for (int64_t sl = 0; sl < nsl; ++sl) {
    const int buf = (int)(sl & 1);
    __builtin_amdgcn_s_waitcnt(TOPK_WAIT_VM(0));  // this wave's loads of slice sl have landed
    __syncthreads();  // ... and every wave's; nobody reads the other buffer any more
    if (sl + 1 < nsl) issue((sl + 1) * KS, buf ^ 1);
    const unsigned char* qsm = &sm[buf][0];
    const unsigned char* ksm = &sm[buf][QBYTES];
#pragma unroll
    for (int st = 0; st < KS / 16; ++st) {
      bf16x8 qf[2], kf[4];
#pragma unroll
      for (int a = 0; a < 2; ++a) qf[a] = frag(qsm, wq + a * 32 + n, st);
#pragma unroll
      for (int b = 0; b < 4; ++b) kf[b] = frag(ksm, wk + b * 32 + n, st);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[b], qf[a], acc[a][b], 0, 0, 0);
    }
  }
  // D[m][n]: m = key 8*(v/4) + 4*half + v%4 of block b, n = query lane%32 of block a
  if (MODE == 2) {
    // candidates: count this lane's passing scores per row, reserve room per row in
    // LDS, then once per row and workgroup in the row's global list
    static_assert(4 * 8192 + 4 * TQ <= 2 * (QBYTES + KBYTES), "stash and row counts fit the operand buffers");
    uint32_t* rc = (uint32_t*)&sm[0][0] + 4 * 2048;  // after the four waves' stashes
    float* stash = (float*)&sm[0][0] + wave * 2048;  // this wave's 32 scores per lane
    __syncthreads();  // every wave is done with the operand buffers
    if (tid < TQ) rc[tid] = 0;
    __syncthreads();
    uint32_t off[2];
    // pass[a][h], bit j = 16 * (b - 2h) + v: score v of block (a, b) is a candidate
    uint32_t pass[2][2];
    // keys of this wave's sub-tile all valid for every row of the tile (no causal
    // diagonal, no tail): the per-key test can go
    const int64_t kend = key0 + wk + 128;
    const bool all_valid = kend <= pb.Lk && (!pb.causal || kend <= i0 + r0 + 1);
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int64_t lr = r0 + wq + a * 32 + n, i = i0 + lr;
      const bool okr = lr < pb.C && i < pb.q1;
      const int64_t nv = okr ? valid_keys(pb, i) : 0;
      const float ts = okr ? bufs.thr[cl * pb.C + lr] : INFINITY;
      uint32_t c = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t m = 0;
        if (all_valid) {
          // highest bit first, m = 2m + pass: an add with the comparison as carry-in
#pragma unroll
          for (int j = 31; j >= 0; --j) m = m + m + (uint32_t)(acc[a][2 * h + (j >> 4)][j & 15] >= ts);
        } else {
#pragma unroll
          for (int bb = 0; bb < 2; ++bb) {
            const int b = 2 * h + bb;
            const int64_t kb = key0 + wk + b * 32 + 4 * half;
#pragma unroll
            for (int v = 0; v < 16; ++v)
              m |= (kb + 8 * (v >> 2) + (v & 3) < nv && acc[a][b][v] >= ts ? 1u : 0u) << (16 * bb + v);
          }
        }
        // rows past the chunk or the sequence hold the tile's first row's scores (and a
        // threshold of +inf, which a +inf score would still meet): they append nothing
        m = okr ? m : 0u;
        pass[a][h] = m;
        c += (uint32_t)__builtin_popcount(m);
      }
      off[a] = c ? atomicAdd(&rc[wq + a * 32 + n], c) : 0u;
    }
    __syncthreads();
    if (tid < TQ) {
      const int64_t lr = r0 + tid, i = i0 + lr;
      const uint32_t total = rc[tid];
      rc[tid] = (total && lr < pb.C && i < pb.q1)
                    ? (uint32_t)atomicAdd(&bufs.cnt[2 * (cl * pb.C + lr)], (int32_t)total) : 0u;
    }
    __syncthreads();
    const uint32_t cap = 2u * (uint32_t)bufs.caph;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int64_t lr = r0 + wq + a * 32 + n;
      uint32_t pos = rc[wq + a * 32 + n] + off[a];
      uint64_t* dst = bufs.cand + 2 * (cl * pb.C + lr) * bufs.caph;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // The 32 scores of blocks (a, 2h) and (a, 2h + 1) go to the wave's LDS stash,
        // score j of the lane at float j * 64 + lane (full-width writes, two scores per
        // instruction); the lane then walks its set bits and reads each passing score
        // back by its index, from its own bank. A wave reads only what its own lanes
        // wrote, and its LDS accesses complete in order: no barrier. The next stash
        // overwrites this one only after every read of this one was issued.
#pragma unroll
        for (int j = 0; j < 32; ++j) stash[j * 64 + lane] = acc[a][2 * h + (j >> 4)][j & 15];
        // bit j is key 8 * (j / 4) + j % 4 = j + (j & ~3) past the lane's first key of
        // block 2h
        const uint32_t nk0 = 0xFFFFFFFFu - (uint32_t)(key0 + wk + 64 * h + 4 * half);
        for (uint32_t m = pass[a][h]; m; m &= m - 1) {
          const uint32_t j = (uint32_t)__builtin_ctz(m);
          const float x = stash[j * 64 + lane];
          if (pos < cap) dst[pos] = ((uint64_t)__float_as_uint(x) << 32) | (uint64_t)(nk0 - (j + (j & ~3u)));
          ++pos;
        }
      }
    }
    return;
  }
  float* S = MODE == 1 ? bufs.samp : bufs.scores;
  const int64_t rowlen = MODE == 1 ? Lslots : pb.Lk;
  const bool vec = (rowlen & 3) == 0;  // rows start 16-byte aligned
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int64_t lr = r0 + wq + a * 32 + n, i = i0 + lr;
    if (lr >= pb.C || i >= pb.q1) continue;
    const int64_t nv = (valid_keys(pb, i) + KSTEP - 1) / KSTEP;  // valid key slots
    float* srow = S + (cl * pb.C + lr) * rowlen;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t key = key0 + wk + b * 32 + 8 * j + 4 * half;
        const f32x16& x = acc[a][b];
        if (vec && key + 3 < nv) {
          *(float4*)(srow + key) = make_float4(x[4 * j], x[4 * j + 1], x[4 * j + 2], x[4 * j + 3]);
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (key + u < nv) srow[key + u] = x[4 * j + u];
        }
      }
    }
  }
}

// ------------------------------------------------------------------ row gather helper
// Appends every element of row[0, nv) whose score is >= ts to cbuf (LDS) as the
// word (raw score bits << 32) | (0xFFFFFFFF - index) (raw_to_key turns it into
// the order key), wave-compacted: reserve(n) returns the base position of this
// wave's next n words (wave-uniform). A batch that would cross cap is counted but
// not written. ts = -inf takes every element. Each lane loads 4 x 16 bytes before
// testing them; rows must start 16-byte aligned when vec.
// (The gathered set {score >= ts} holds the row's top k whenever it holds k keys:
// a key outside it is below every key inside.)
__device__ __forceinline__ uint64_t raw_to_key(uint64_t w) {
  return ((uint64_t)ord_u32(__uint_as_float((uint32_t)(w >> 32))) << 32) | (w & 0xFFFFFFFFull);
}

template <class Reserve>
__device__ __forceinline__ void gather_row(const float* row, int64_t nv, float ts, bool vec, int64_t lane0,
                                           int64_t lanes, uint64_t* cbuf, uint32_t cap, const Reserve& reserve) {
  auto offer = [&](bool take, uint32_t i, float v) {
    const uint64_t bal = __ballot(take);
    if (bal == 0) return;
    const uint32_t cnt = (uint32_t)__popcll(bal);
    const uint32_t base = reserve(cnt);
    if (base + cnt > cap) return;  // wave-uniform: the set overflows, nothing is written
    const uint32_t pos = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
    if (take) cbuf[pos] = ((uint64_t)__float_as_uint(v) << 32) | (uint64_t)(0xFFFFFFFFu - i);
  };
  if (vec) {
    constexpr int U = 4;  // float4 loads in flight per lane
    const int64_t step = 4 * lanes * U;
    int64_t base = 0;
    for (; base + step <= nv; base += step) {  // full steps: every element is in the row
      float4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = *(const float4*)(row + base + 4 * (lane0 + lanes * u));
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i = (uint32_t)(base + 4 * (lane0 + lanes * u));
        offer(v[u].x >= ts, i, v[u].x);
        offer(v[u].y >= ts, i + 1, v[u].y);
        offer(v[u].z >= ts, i + 2, v[u].z);
        offer(v[u].w >= ts, i + 3, v[u].w);
      }
    }
    for (; base < nv; base += step) {  // the last, partial step
      float4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t i = base + 4 * (lane0 + lanes * u);
        v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i + 3 < nv) {
          v[u] = *(const float4*)(row + i);
        } else if (i < nv) {
          v[u].x = row[i];
          if (i + 1 < nv) v[u].y = row[i + 1];
          if (i + 2 < nv) v[u].z = row[i + 2];
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t i = base + 4 * (lane0 + lanes * u);
        offer(i < nv && v[u].x >= ts, (uint32_t)i, v[u].x);
        offer(i + 1 < nv && v[u].y >= ts, (uint32_t)i + 1, v[u].y);
        offer(i + 2 < nv && v[u].z >= ts, (uint32_t)i + 2, v[u].z);
        offer(i + 3 < nv && v[u].w >= ts, (uint32_t)i + 3, v[u].w);
      }
    }
  } else {
    for (int64_t base = 0; base < nv; base += lanes) {
      const int64_t i = base + lane0;
      const float v = i < nv ? row[i] : 0.f;
      offer(i < nv && v >= ts, (uint32_t)i, v);
    }
  }
}

// ------------------------------------------------------------------ chunk-tile path: select
// One workgroup per query row of the score tile. Every key at or above a
// threshold key is gathered into LDS in one streaming pass over the row, and the
// exact select runs on that candidate set in LDS:
//  * rows of at most TS_CAP valid keys take all of them;
//  * longer rows take the R-th largest key of a sample of TS_SAMPLE keys (32
//    blocks of 32 contiguous scores spread over the row), with R a few standard
//    deviations above the sample's expected share of the top k;
//  * the set is proven to hold the row's top k when it has at least k_eff keys
//    and did not overflow; otherwise the row is selected from global memory by the
//    multi-pass radix select (exact for any input).
constexpr int TS_CAP = 4096;
constexpr int TS_SAMPLE = 1024;

// The select of one row of nv fp32 scores by a 256-thread workgroup (see above).
// cand: TS_CAP keys of LDS; sbuf: pow2_at_least(k_eff) keys of LDS.
// fallbacks (optional, may be NULL) counts the rows selected by the multi-pass path.
__device__ void wg_row_select(const float* row, int64_t nv, uint32_t k_eff, int64_t k, bool vec, uint64_t* cand,
                              uint64_t* sbuf, uint32_t* hist, uint32_t* misc, uint32_t* ccount, uint64_t* out,
                              int32_t* fallbacks) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int P = pow2_at_least(k_eff);
  float ts = -INFINITY;  // candidates: scores >= ts
  if (nv > TS_CAP) {
    // sample: block b covers [start_b, start_b + 32), start_b = 32 * floor(b * nv / (32 * 32))
    for (int s = tid; s < TS_SAMPLE; s += 256) {
      const int64_t b = s >> 5, start = ((b * nv) / (32 * 32)) * 32, e = start + (s & 31);
      cand[s] = e < nv ? make_key(row[e], (uint32_t)e) : 0ull;
    }
    __syncthreads();
    // expected sampled keys among the row's top k_eff: mu = k_eff * TS_SAMPLE / nv;
    // R = mu + 6 sqrt(mu) + 8 keeps P(sample rank R below the k-th key) negligible
    const float mu = (float)k_eff * (float)TS_SAMPLE / (float)nv;
    int R = (int)ceilf(mu + 6.0f * sqrtf(mu) + 8.0f);
    R = R < TS_SAMPLE ? R : TS_SAMPLE;
    if (tid < 64) {
      // one wave: the R-th largest sampled score, built bit by bit on the scores'
      // order-preserving keys (a bit stays when at least R samples are at or above the
      // prefix with it set; a missing sample's key is 0, below every score)
      constexpr int E = TS_SAMPLE / 64;
      uint32_t u[E];
#pragma unroll
      for (int e = 0; e < E; ++e) u[e] = (uint32_t)(cand[lane + 64 * e] >> 32);
      uint32_t prefix = 0;
      for (int b = 31; b >= 0; --b) {
        const uint32_t c = prefix | (1u << b);
        uint32_t cnt = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) cnt += (uint32_t)__popcll(__ballot(u[e] >= c));
        if (cnt >= (uint32_t)R) prefix = c;
      }
      if (lane == 0) misc[0] = prefix;
    }
    __syncthreads();
    ts = ord_to_f32(misc[0]);
    __syncthreads();
  }
  if (tid == 0) *ccount = 0;
  __syncthreads();
  // one pass: wave-level compaction, one counter update per wave and step
  auto reserve = [&](uint32_t cnt) {
    uint32_t wbase = 0;
    if (lane == 0) wbase = atomicAdd(ccount, cnt);
    return (uint32_t)__shfl(wbase, 0, 64);
  };
  gather_row(row, nv, ts, vec, tid, 256, cand, (uint32_t)TS_CAP, reserve);
  __syncthreads();
  const uint32_t c = *ccount;
  __syncthreads();
  if (c >= k_eff && c <= (uint32_t)TS_CAP) {
    auto getkey = [&](int64_t e) { return raw_to_key(cand[e]); };
    team_topk<256>(getkey, c, k_eff, (uint32_t)k, sbuf, P, hist, misc, out);
  } else {
    if (fallbacks && tid == 0) atomicAdd(fallbacks, 1);
    auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
    team_topk<256>(getkey, nv, k_eff, (uint32_t)k, sbuf, P, hist, misc, out);
  }
}

__global__ __launch_bounds__(256) void k_tile_select(Problem pb, Pass ps, const float* S, uint64_t* sel,
                                                     int32_t* fallbacks) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint64_t cand[TS_CAP];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  __shared__ uint32_t ccount;
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  wg_row_select(S + p * pb.Lk, nv, k_eff, pb.k, (pb.Lk & 3) == 0, cand, sbuf, hist, misc, &ccount, sel + p * pb.k,
                fallbacks);
}

// ------------------------------------------------------------------ fused path: scan
// One workgroup = 4 waves x 32*G queries of one head (G = 2). Each wave keeps the B operand
// of G 32-query column groups in registers; key tiles of 64 keys stream through two
// LDS buffers that are filled by direct global-to-LDS loads issued one tile ahead
// (no register staging). Each wave computes S^T = K Q^T
// with v_mfma_f32_32x32x16_bf16, so lane l holds 16 keys' scores of query l % 32 of
// a group (keys 8*(v/4) + 4*(l/32) + v%4 of the 32-key block, v = 0..15); one LDS
// read of the K operand feeds all G groups. The feature dimension is split between
// the half-waves: half h holds features [h*D/2, h*D/2 + D/2) of its row in both
// operands (the contraction is order-free). In LDS, 16-byte part p of key row r
// sits at position r*CH + (p ^ (r & 7)), so the 8 rows one LDS cycle serves hit 8
// different bank groups.
//
// Filtering is two-level. Per 16-score lane block, a max tree decides whether any
// score beats the query's threshold; only such "dirty" blocks are copied into a
// per-wave LDS staging ring. When the ring fills, the whole wave drains it: each
// lane takes one staged block, finds its passing scores and appends them as
// 64-bit words  (raw fp32 score bits << 32) | (~key)  to the query's candidate
// list in global memory (one list per query, shared by its two half-waves, so a
// wave keeps half as many partly written lines in flight; one LDS counter update
// per block reserves the positions). The select converts the words to
// order-preserving keys.
struct ScanArgs {
  const uint16_t* Q;
  const uint16_t* K;
  int64_t Lq, Lk, C, kv_head_stride;  // Lq: query rows per head in memory
  int64_t q0, q1;                     // rows processed: [q0, q1) of every head
  int64_t c0, nchunk, wgs_per_chunk;
  uint64_t* cand;
  int32_t* cnt;
  int64_t caph;
  const float* thr;  // MODE_THRESH: per pass-local row, the threshold its candidates beat
  int mode, stride, causal;
};

constexpr int SCAN_KT = 64;  // keys per K tile
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

// Launch shape of the scan: G = 32-query groups per wave, NB = K tile buffers in
// LDS, CAP = staged 8-score half blocks per wave (whole 64-slot rounds drain at
// tile boundaries; a block whose dirty lanes would not fit drains the ring first),
// OCC = waves per SIMD the register and LDS sizes allow (37 KB of LDS per
// workgroup: four workgroups per CU); OCC_CAUSAL = the same under the causal mask,
// whose extra registers would spill at four waves per SIMD (three waves without
// spills measured 20 % faster). For d = 128 (twice the registers for the queries'
// operand, 53 KB of LDS) the kernel asks for two waves per SIMD only, so that the
// compiler never spills to reach more; it gets three where its registers allow.
template <int G>
struct ScanShape;
template <>
struct ScanShape<2> {  // 256 queries per workgroup
  static constexpr int NB = 2, CAP = 128, OCC = 4, OCC_CAUSAL = 3;
};

template <int G>
constexpr int scan_queries_per_wg() { return 4 * 32 * G; }


// SCORE_ONLY: the ablation that keeps the sample phase, the K tile pipeline, the MFMAs
// and each block's maximum, and drops the filter (no staging, no drain, no candidate
// output; the maxima go to cnt so that the work is kept). It measures what the score
// core alone costs at the same launch shape.
// DIRECT: the variant for dense candidates (the filtered path, MODE_THRESH): each
// row's threshold comes from a.thr, and every lane appends its own passing scores of
// each block straight to its own list (one per query and half-wave, the length in
// cnt[2 * row + half]) instead of staging dirty blocks; see `extract`.
template <int D, int R, int G, bool CAUSAL, bool SCORE_ONLY = false, int J = 0, bool DIRECT = false>
__global__ __launch_bounds__(256, D == 64 ? (CAUSAL ? ScanShape<G>::OCC_CAUSAL : ScanShape<G>::OCC) : 2) void k_fused_scan(
    ScanArgs a) {
  static_assert(ScanShape<G>::CAP >= 128, "a ring holds one block's 64 lanes, both halves");
  constexpr int SCAN_NB = ScanShape<G>::NB;
  constexpr int STAGE_CAP = ScanShape<G>::CAP;
  constexpr int KT = SCAN_KT;
  constexpr int NRB = KT / 32;            // 32-key MFMA blocks per tile
  constexpr int NS = D / 16;              // MFMA steps over the features
  constexpr int CH = 2 * D / 16;          // 16-byte parts per key row
  constexpr int TILEB = KT * 2 * D;       // bytes per K tile
  constexpr int LPW = TILEB / 1024 / 4;   // 1 KB direct loads per wave per tile
  constexpr int QB = scan_queries_per_wg<G>();
  static_assert(LPW >= 1 && TILEB % 4096 == 0, "tile must split evenly over the 4 waves");
  // the two K tile buffers, used alternately; as two arrays (not one indexed array) so
  // that every access below names its buffer at compile time
  static_assert(SCAN_NB == 2, "two K tile buffers");
  __shared__ __attribute__((aligned(16))) unsigned char ks0[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char ks1[TILEB];
  // staging slot = 8 scores: one dirty half of a lane block, as two 16-byte chunks
  // held in separate arrays (chunk c of slot s at stage[wave][c][s]), so the writes
  // and reads of consecutive slots by consecutive lanes are free of bank conflicts
  __shared__ __attribute__((aligned(16))) float4 stage[4][2][STAGE_CAP];
  __shared__ uint32_t stage_meta[4][STAGE_CAP];
  __shared__ float tau_lds[4][32 * G];
  __shared__ uint32_t cnt_lds[4][32 * G];

  // the wave index is uniform: kept in a scalar register, so LDS and load addresses
  // that depend on it need no vector arithmetic
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63,
            half = lane >> 5, n = lane & 31;
  // XCD-aware order: the hardware deals workgroups round-robin over the 8 XCDs;
  // renumber so each XCD runs consecutive logical workgroups (same head) and K
  // stays in that XCD's L2. Under the causal mask a workgroup's key tiles grow with
  // its queries' position, so the logical order is reversed: the longest workgroups
  // start first and the last to start are the shortest.
  const int64_t NG = gridDim.x, bid = blockIdx.x;
  int64_t wg = (NG % 8 == 0) ? (bid % 8) * (NG / 8) + bid / 8 : bid;
  if (CAUSAL) wg = NG - 1 - wg;
  const int64_t cl = wg / a.wgs_per_chunk, blk = wg - cl * a.wgs_per_chunk;
  const int64_t id = a.c0 + cl, bh = id / a.nchunk, c = id - bh * a.nchunk;
  const uint16_t* Kh = a.K + bh * a.kv_head_stride;
  // the workgroup's first and last query (index in the head); under the causal mask
  // (Eq. 2) its key tiles end at the one holding its last query
  const int64_t q_first = a.q0 + c * a.C + blk * QB;
  int64_t q_last = a.q0 + c * a.C + (blk * QB + QB < a.C ? blk * QB + QB : a.C) - 1;
  q_last = q_last < a.q1 - 1 ? q_last : a.q1 - 1;
  const int64_t ntiles_all = (a.Lk + KT - 1) / KT;
  const int64_t ntiles = CAUSAL && q_last / KT + 1 < ntiles_all ? q_last / KT + 1 : ntiles_all;
  const bool tail = ntiles * KT > a.Lk;
  const int64_t wave_row0 = cl * a.C + blk * QB + wave * 32 * G;  // pass-local row of the wave's query 0
  const int64_t wave_q0 = q_first + wave * 32 * G;                 // the wave's first query

  bool ok[G];
  bf16x8 b[G][NS];
  {
    const bf16x8 zero8 = {};
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int64_t local = blk * QB + wave * 32 * G + g * 32 + n, i = a.q0 + c * a.C + local;
      ok[g] = local < a.C && i < a.q1;
      const uint16_t* q = a.Q + (bh * a.Lq + (ok[g] ? i : 0)) * D + (D / 2) * half;
#pragma unroll
      for (int s = 0; s < NS; ++s) b[g][s] = ok[g] ? *(const bf16x8*)(q + 8 * s) : zero8;
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g)
    if (half == 0) cnt_lds[wave][g * 32 + n] = 0;

  // direct loads of tile t into buffer dst: lane `lane` of this wave's j-th load
  // fills LDS position cidx = (wave*LPW + j)*64 + lane with part
  // (cidx % CH) ^ (row & 7) of key row cidx / CH (rows past Lk load the last key;
  // their scores are masked)
  // Load number q = wave*LPW + j covers key rows q*RPL .. q*RPL + RPL - 1; within them
  // the lane's element offset depends on q only through q mod NPAT (the swizzle
  // repeats every 8 rows), so the lane keeps NPAT offsets (one at d = 64).
  constexpr int RPL = 64 / CH, NPAT = RPL % 8 == 0 ? 1 : 8 / RPL;
  uint32_t lane_off[NPAT];
#pragma unroll
  for (int e = 0; e < NPAT; ++e) {
    const int r = e * RPL + lane / CH, p = (lane % CH) ^ (r & 7);
    lane_off[e] = (uint32_t)((lane / CH) * D + p * 8);
  }
  auto issue = [&](int64_t t, unsigned char* dst) {
    if ((t + 1) * KT <= a.Lk) {  // whole tile: a uniform base plus the lane's offset
      const uint16_t* base = Kh + t * KT * D;
#pragma unroll
      for (int j = 0; j < LPW; ++j) {
        const int q = wave * LPW + j;
        __builtin_amdgcn_global_load_lds((const void*)(base + q * RPL * D + lane_off[q % NPAT]),
                                         (__attribute__((address_space(3))) void*)&dst[q * 1024], 16, 0, 0);
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int cidx = (wave * LPW + j) * 64 + lane, r = cidx / CH, p = (cidx % CH) ^ (r & 7);
      int64_t key = t * KT + r;
      key = key < a.Lk ? key : a.Lk - 1;
      __builtin_amdgcn_global_load_lds((const void*)(Kh + key * D + p * 8),
                                       (__attribute__((address_space(3))) void*)&dst[(wave * LPW + j) * 1024], 16,
                                       0, 0);
    }
  };
  // Runs step_fn(t, cur, nxt) for t = 0 .. count - 1 with the buffers alternating,
  // unrolled by two so that each call names its buffers at compile time: the
  // compiler then knows that reads of one buffer do not overlap the direct loads
  // into the other, and does not make them wait for those loads.
  auto alternate = [&](int64_t count, auto&& step_fn) {
    for (int64_t t = 0; t < count; t += 2) {
      step_fn(t, ks0, ks1);
      if (t + 1 < count) step_fn(t + 1, ks1, ks0);
    }
  };
  // Runs body(tile, lds) over tiles 0, step, 2*step, ... (count of them) with one
  // tile in flight. Before tile t is read, this wave's loads of t are complete and
  // the barrier publishes every wave's part; the barrier also proves that no wave
  // still reads the buffer the next load overwrites.
  auto pipeline = [&](int64_t count, int64_t step, auto&& body) {
    if (count <= 0) return;
    issue(0, ks0);
    alternate(count, [&](int64_t t, const unsigned char* cur, unsigned char* nxt) {
      __builtin_amdgcn_s_waitcnt(TOPK_WAIT_VM(0));
      __syncthreads();
      if (t + 1 < count) issue((t + 1) * step, nxt);
      body(t * step, cur);
    });
    __syncthreads();
  };
  // scores of 32 keys (block rb of the tile) for all G query groups
  auto block_scores = [&](const unsigned char* kb, int rb, f32x16 (&acc)[G]) {
    const int r = rb * 32 + n;
    bf16x8 av[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) av[s] = *(const bf16x8*)(kb + (r * CH + ((half * NS + s) ^ (r & 7))) * 16);
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = (f32x16){};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[s], b[g][s], acc[g], 0, 0, 0);
  };
  auto mask_keys = [&](f32x16& acc, int64_t jb) {  // keys >= Lk of the last tile -> -inf
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (jb + 8 * (v >> 2) + (v & 3) >= a.Lk) acc[v] = -INFINITY;
  };
  // causal mask: keys j > i of this lane's queries -> -inf; only blocks reaching past
  // the wave's first query need it (offsets within 32-bit range: the block starts
  // at most 63 keys past that query)
  auto mask_future = [&](f32x16 (&acc)[G], int64_t t, int rb) {
    if (!CAUSAL) return;
    const int64_t j0 = t * KT + rb * 32;
    if (j0 + 31 <= wave_q0) return;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int room = (int)(wave_q0 - j0) + g * 32 + n - 4 * half;  // i - (lane's first key)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if (8 * (v >> 2) + (v & 3) > room) acc[g][v] = -INFINITY;
    }
  };
  // the A operand (32 keys of block rb) and one group's 4 MFMAs, for the pipelined scan
  auto read_a = [&](const unsigned char* kb, int rb, bf16x8 (&av)[NS]) {
    const int r = rb * 32 + n;
#pragma unroll
    for (int s = 0; s < NS; ++s) av[s] = *(const bf16x8*)(kb + (r * CH + ((half * NS + s) ^ (r & 7))) * 16);
  };
  auto group_scores = [&](const bf16x8 (&av)[NS], const bf16x8 (&bg)[NS], f32x16& acc) {
    acc = (f32x16){};
#pragma unroll
    for (int s = 0; s < NS; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[s], bg[s], acc, 0, 0, 0);
  };
  // the tail and causal masks of one group's block
  auto mask_group = [&](f32x16& acc, int g, int64_t t, int rb) {
    if (tail && t == ntiles - 1) mask_keys(acc, t * KT + rb * 32 + 4 * half);
    if (!CAUSAL) return;
    const int64_t j0 = t * KT + rb * 32;
    if (j0 + 31 <= wave_q0) return;
    const int room = (int)(wave_q0 - j0) + g * 32 + n - 4 * half;
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if (8 * (v >> 2) + (v & 3) > room) acc[v] = -INFINITY;
  };
  // maxima of finite scores (and -inf): the NaN-propagating maximum, which needs no
  // canonicalising instructions and fuses into three-input maxima
  auto fmax_ = [](float x, float y) { return __builtin_elementwise_maximum(x, y); };
  auto block_max = [&](const f32x16& acc) {
    float m = acc[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) m = fmax_(m, acc[v]);
    return m;
  };

  float tau[G];
#pragma unroll
  for (int g = 0; g < G; ++g) tau[g] = a.mode == MODE_THRESH && ok[g] ? a.thr[wave_row0 + g * 32 + n] : -INFINITY;
  // Causal rows sample the same 1-in-stride tiles; the masked (future) keys of a
  // sampled tile give -inf block maxima, so a row's threshold depends on the row
  // alone. The host sends only rows with enough valid sampled blocks this way.
  if (a.mode == MODE_SAMPLE) {
    float top[G][R];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int r = 0; r < R; ++r) top[g][r] = -INFINITY;
    // sorted insert, descending: entry r becomes the median of the old entries r - 1
    // and r and the new value (entry 0 the larger of it and the value), so the R
    // updates do not wait on each other (a chain of maxima and minima would)
    auto insert = [&](float (&tp)[R], float m) {
#pragma unroll
      for (int r = R - 1; r > 0; --r) tp[r] = __builtin_amdgcn_fmed3f(tp[r - 1], tp[r], m);
      tp[0] = __builtin_elementwise_maximum(tp[0], m);
    };
    const int64_t ns = (ntiles + a.stride - 1) / a.stride;
    pipeline(ns, a.stride, [&](int64_t t, const unsigned char* kb) {
#pragma unroll 1
      for (int rb = 0; rb < NRB; ++rb) {
        f32x16 acc[G];
        block_scores(kb, rb, acc);
        if (tail && t == ntiles - 1) {
          const int64_t jb = t * KT + rb * 32 + 4 * half;
#pragma unroll
          for (int g = 0; g < G; ++g) mask_keys(acc[g], jb);
        }
        mask_future(acc, t, rb);
#pragma unroll
        for (int g = 0; g < G; ++g) insert(top[g], block_max(acc[g]));
      }
    });
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (J > 0) {
        // the J-th largest of the two half-waves' lists together (each holds its R
        // largest block maxima, J <= 2R): the largest, over p + q = J with p, q <= R,
        // of min(p-th of this lane's list, q-th of the partner's), the 0-th entry
        // standing for +inf. Where more than R of the J largest of all sampled blocks
        // fall in one half-wave this is below the exact J-th: still a lower bound.
        static_assert(J <= 2 * R, "the J-th needs R >= J / 2 per list");
        float other[R];
#pragma unroll
        for (int r = 0; r < R; ++r) other[r] = __shfl_xor(top[g][r], 32, 64);
        float t = -INFINITY;
#pragma unroll
        for (int p = (J > R ? J - R : 0); p <= (J < R ? J : R); ++p) {
          const float ap = p > 0 ? top[g][p > 0 ? p - 1 : 0] : INFINITY;
          const float bq = J - p > 0 ? other[J - p > 0 ? J - p - 1 : 0] : INFINITY;
          t = fmaxf(t, fminf(ap, bq));
        }
        tau[g] = t;
      } else {
        const float mine = top[g][R - 1];
        tau[g] = fminf(mine, __shfl_xor(mine, 32, 64));
      }
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (!ok[g]) tau[g] = INFINITY;
    if (half == 0) tau_lds[wave][g * 32 + n] = tau[g];
  }

  // ---- staging ring and its drain (all per wave; LDS ops of one wave execute in order)
  // A slot holds one dirty half (8 scores) of a lane block: scores 8*hb .. 8*hb+7.
  // slot meta = (32-key block index << 8) | (hb << 7) | (group << 6) | lane
  static_assert(G <= 2, "the slot meta holds one group bit");
  // The ring is circular: slots [rhead, rtail) (positions modulo STAGE_CAP) wait for
  // the drain; both counters are wave-uniform.
  static_assert((STAGE_CAP & (STAGE_CAP - 1)) == 0, "ring size must be a power of two");
  int rhead = 0, rtail = 0;
  auto drain_to = [&](int end) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int base = rhead; base < end; base += 64) {
      const int idx = base + lane, slot = idx & (STAGE_CAP - 1);
      uint32_t mask = 0, meta = 0;
      if (idx < end) {
        meta = stage_meta[wave][slot];
        const float t = tau_lds[wave][(meta >> 6 & 1) * 32 + (meta & 31)];
#pragma unroll
        for (uint32_t cc = 0; cc < 2; ++cc) {
          const float4 x = stage[wave][cc][slot];
          const uint32_t m4 = (x.x > t ? 1u : 0u) | (x.y > t ? 2u : 0u) | (x.z > t ? 4u : 0u) | (x.w > t ? 8u : 0u);
          mask |= m4 << (4 * cc);
        }
      }
      if (mask) {
        const uint32_t ql = meta & 63, g = meta >> 6 & 1, h = ql >> 5, hb = meta >> 7 & 1;
        // one counter update per slot reserves room for all its passing scores in the
        // query's list (both half-waves append to the same list)
        uint32_t pos = atomicAdd(&cnt_lds[wave][g * 32 + (ql & 31)], (uint32_t)__builtin_popcount(mask));
        const uint32_t nj = 0xFFFFFFFFu - ((meta >> 8) * 32u + 4u * h);
        uint64_t* dst = a.cand + (wave_row0 + g * 32 + (ql & 31)) * 2 * a.caph;
        do {
          const uint32_t v = __builtin_ctz(mask);
          mask &= mask - 1;
          // score u = 8*hb + v of the block is key 8*(u/4) + u%4 = u + (u & ~3) past the block's first key
          const uint32_t u = 8u * hb + v;
          const float sc = ((const float*)&stage[wave][v >> 2][slot])[v & 3];
          if (pos < (uint32_t)(2 * a.caph))
            dst[pos] = ((uint64_t)__float_as_uint(sc) << 32) | (uint64_t)(nj - (u + (u & 12u)));
          ++pos;
        } while (mask);
      }
    }
    rhead = end;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  auto drain = [&]() { drain_to(rtail); };
  // A lane whose block maximum beats its query's threshold stages its dirty half
  // (the lower one when both are dirty); lanes with both halves dirty stage the
  // upper half in a second, rarely needed, round. Two 16-byte writes per lane and
  // round instead of four.
  auto filter = [&](int g, const f32x16& acc, int64_t t, int rb) {
    float hA = fmax_(acc[0], acc[1]), hB = fmax_(acc[8], acc[9]);
#pragma unroll
    for (int v = 2; v < 8; ++v) {
      hA = fmax_(hA, acc[v]);
      hB = fmax_(hB, acc[8 + v]);
    }
    const bool dA = hA > tau[g], dB = hB > tau[g];
    // the ballots straight from the comparisons (the compare masks themselves), not
    // from a combined predicate that the compiler would turn back into a lane mask
    const uint64_t bA = __builtin_amdgcn_ballot_w64(hA > tau[g]), bB = __builtin_amdgcn_ballot_w64(hB > tau[g]);
    const uint64_t bal = bA | bB;
    if (bal == 0) return;
    const uint64_t bal2 = bA & bB;
    const int n1 = __popcll(bal), n2 = __popcll(bal2);
    if (rtail - rhead + n1 + n2 > STAGE_CAP) drain();
    const uint32_t mb = (uint32_t)((t * KT + rb * 32) / 32) << 8 | (uint32_t)(g << 6) | (uint32_t)lane;
    if (dA || dB) {
      const int slot = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)bal, (uint32_t)rtail)) &
                       (STAGE_CAP - 1);
      // the half to stage, selected in registers (a bitwise mux per score, so the
      // compiler does not turn it into an indexed read of the accumulator)
      const uint32_t sel = dA ? 0xFFFFFFFFu : 0u;
      float x[8];
#pragma unroll
      for (int v = 0; v < 8; ++v)
        x[v] = __uint_as_float((__float_as_uint(acc[v]) & sel) | (__float_as_uint(acc[8 + v]) & ~sel));
      stage[wave][0][slot] = make_float4(x[0], x[1], x[2], x[3]);
      stage[wave][1][slot] = make_float4(x[4], x[5], x[6], x[7]);
      stage_meta[wave][slot] = mb | (dA ? 0u : 128u);
    }
    if (bal2) {
      if (dA && dB) {
        const int slot = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal2 >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)bal2, (uint32_t)(rtail + n1))) &
                         (STAGE_CAP - 1);
        stage[wave][0][slot] = make_float4(acc[8], acc[9], acc[10], acc[11]);
        stage[wave][1][slot] = make_float4(acc[12], acc[13], acc[14], acc[15]);
        stage_meta[wave][slot] = mb | 128u;
      }
    }
    rtail += n1 + n2;
  };
  // DIRECT: the lane's passing scores of one 16-score lane block, as bits (built
  // highest first, m = 2m + pass); the 16 scores go to
  // the wave's stash in LDS (score v of the lane at float v * 64 + lane, full-width
  // writes), and the lane walks its bits, reading each passing score back by its index
  // from its own bank and appending it to its list. A wave reads only what its own
  // lanes wrote and its LDS accesses complete in order, so the stash needs no barrier,
  // and the next block's stash is written only after every read of this one.
  uint32_t dpos[G] = {};
  uint64_t dheld[G] = {};
  float* const dstash = (float*)&stage[wave][0][0];
  static_assert(sizeof(stage[0]) >= 16 * 64 * sizeof(float), "a wave's stash holds 16 scores per lane");
  auto extract = [&](int g, const f32x16& acc, int64_t t, int rb) {
    uint32_t m = 0;
#pragma unroll
    for (int v = 15; v >= 0; --v) m = m + m + (uint32_t)(acc[v] > tau[g]);
    if (__builtin_amdgcn_ballot_w64(m != 0) == 0) return;
#pragma unroll
    for (int v = 0; v < 16; ++v) dstash[v * 64 + lane] = acc[v];
    // score v is key 8 * (v / 4) + v % 4 = v + (v & ~3) past the lane's first key
    const uint32_t nk0 = 0xFFFFFFFFu - (uint32_t)(t * KT + rb * 32 + 4 * half);
    uint64_t* dst = a.cand + ((wave_row0 + g * 32 + n) * 2 + half) * a.caph;
    uint32_t pos = dpos[g];
    for (; m; m &= m - 1) {
      const uint32_t v = (uint32_t)__builtin_ctz(m);
      const float x = dstash[v * 64 + lane];
      const uint64_t w = ((uint64_t)__float_as_uint(x) << 32) | (uint64_t)(nk0 - (v + (v & ~3u)));
      // words go out in pairs (one 16-byte store per two candidates); an even position
      // waits in a register for its partner
      if (pos & 1) {
        if (pos < (uint32_t)a.caph) *(u64x2*)&dst[pos - 1] = (u64x2){dheld[g], w};
      } else {
        dheld[g] = w;
      }
      ++pos;
    }
    dpos[g] = pos;
  };
  // Main scan: tile by tile. A tile's wait and barrier, and the loads of the next
  // tile into the other buffer, come first; then its 32-key blocks.
  float core_sink = -INFINITY;
  if constexpr (SCORE_ONLY) {
    // the ablation keeps the plain order (both groups' MFMAs, then both maxima)
    issue(0, ks0);
    alternate(ntiles, [&](int64_t t, const unsigned char* cur, unsigned char* nxt) {
      __builtin_amdgcn_s_waitcnt(TOPK_WAIT_VM(0));
      __syncthreads();
      if (t + 1 < ntiles) issue(t + 1, nxt);
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        f32x16 x[G];
        block_scores(cur, rb, x);
        if (tail && t == ntiles - 1) {
          const int64_t jb = t * KT + rb * 32 + 4 * half;
#pragma unroll
          for (int g = 0; g < G; ++g) mask_keys(x[g], jb);
        }
        mask_future(x, t, rb);
#pragma unroll
        for (int g = 0; g < G; ++g) core_sink = fmax_(core_sink, block_max(x[g]) - tau[g]);
      }
    });
  } else {
    // Each block's group-0 MFMAs are issued before the previous block's group-1
    // filter, and its group-1 MFMAs before its own group-0 filter, so a wave has a
    // filter (VALU, LDS) to run while its own MFMAs execute. Group 1 of a tile's last
    // block is filtered after the next tile's barrier (its scores are in registers).
    static_assert(G == 2, "the pipelined scan alternates two query groups");
    f32x16 x0, x1;
    int64_t pt = -1;  // tile of the block whose group 1 still awaits its filter
    int prb = 0;
    auto filter1 = [&]() {
      mask_group(x1, 1, pt, prb);
      if constexpr (DIRECT) extract(1, x1, pt, prb);
      else filter(1, x1, pt, prb);
    };
    issue(0, ks0);
    alternate(ntiles, [&](int64_t t, const unsigned char* cur, unsigned char* nxt) {
      __builtin_amdgcn_s_waitcnt(TOPK_WAIT_VM(0));
      __syncthreads();
      // drain whole 64-slot rounds at the tile boundary, before the next tile's loads
      // are issued: the drain's LDS counter updates then have no direct loads to wait
      // for, and its candidate stores complete while this tile is computed instead of
      // delaying a later wait
      if (!DIRECT && t > 0 && rtail - rhead >= 64) drain_to(rhead + ((rtail - rhead) & ~63));
      if (t + 1 < ntiles) issue(t + 1, nxt);
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb) {
        bf16x8 av[NS];
        read_a(cur, rb, av);
        group_scores(av, b[0], x0);
        if (pt >= 0) filter1();
        group_scores(av, b[1], x1);
        mask_group(x0, 0, t, rb);
        if constexpr (DIRECT) extract(0, x0, t, rb);
        else filter(0, x0, t, rb);
        pt = t;
        prb = rb;
      }
    });
    if (pt >= 0) filter1();
  }
  if (SCORE_ONLY) {
    if (ok[0]) a.cnt[(wave_row0 + n) * 2 + half] = (int32_t)__float_as_uint(core_sink);
    return;
  }
  if constexpr (DIRECT) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t pos = dpos[g];
      if ((pos & 1) && pos - 1 < (uint32_t)a.caph) a.cand[((wave_row0 + g * 32 + n) * 2 + half) * a.caph + pos - 1] = dheld[g];
      if (ok[g]) a.cnt[(wave_row0 + g * 32 + n) * 2 + half] = (int32_t)pos;
    }
    return;
  }
  drain();
#pragma unroll
  for (int g = 0; g < G; ++g)
    if (ok[g] && half == 0) a.cnt[(wave_row0 + g * 32 + n) * 2] = (int32_t)cnt_lds[wave][g * 32 + n];
}

// ------------------------------------------------------------------ fused path: select
// One wave per row. A row whose candidates overflowed, or (threshold mode) hold
// fewer than k_eff keys, goes to the redo list; otherwise the candidate set is
// proven to contain the row's top-k and an exact select runs over it:
//  * the candidates (at most 2 * caph <= CAND_REGS * 64) are read once into
//    registers as order-preserving keys;
//  * the key bytes shared by every candidate are skipped (min/max reduction), and
//    radix passes of 8 bits find the k_eff-th largest key; the pass's digit is
//    broadcast with ballot/shuffle, only the histogram lives in LDS;
//  * the selected keys are compacted with mbcnt and sorted (descending) by a
//    bitonic network on registers, E = P/64 keys per lane.
constexpr int CAND_REGS = 16;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)x, m, 64), hi = __shfl_xor((uint32_t)(x >> 32), m, 64);
  return ((uint64_t)hi << 32) | lo;
}
// The value of lane (lane ^ m), m a power of two known at compile time once the
// caller is unrolled: m = 1, 2 by a DPP quad permutation (no LDS traffic), m = 4..16
// by a bit-mode ds_swizzle (xor within 32 lanes), m = 32 by ds_bpermute.
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t x, int m) {
  switch (m) {
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);  // quad [1,0,3,2]
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);  // quad [2,3,0,1]
    case 4: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (4 << 10));
    case 8: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (8 << 10));
    case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (16 << 10));
    default: return (uint32_t)__shfl_xor((int)x, m, 64);
  }
}
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t x, int m) {
  return ((uint64_t)xor_lane_u32((uint32_t)(x >> 32), m) << 32) | xor_lane_u32((uint32_t)x, m);
}
// The minimum or maximum of x over a wave whose lanes are all active, as a
// wave-uniform value: two DPP quad permutations and the half-row and row mirrors
// leave every row of 16 lanes holding its row's extreme, and the four rows' values
// are read into scalar registers (no LDS traffic, unlike a shuffle).
template <bool MAX>
__device__ __forceinline__ uint32_t wave_extreme_u32_full(uint32_t x) {
  auto op = [](uint32_t u, uint32_t v) { return MAX ? max(u, v) : min(u, v); };
  x = op(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false));   // quad [1,0,3,2]
  x = op(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false));   // quad [2,3,0,1]
  x = op(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = op(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, false));  // row_mirror
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 0), r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 16);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 32), r3 = (uint32_t)__builtin_amdgcn_readlane((int)x, 48);
  return op(op(r0, r1), op(r2, r3));
}
// Inclusive prefix sum over the 64 lanes of a wave whose lanes are all active, by
// DPP: row shifts 1, 2, 4, 8 scan each row of 16 lanes, then the broadcasts of lane
// 15 (into rows 1 and 3) and lane 31 (into rows 2 and 3) carry the row totals.
// Lanes without a source add the `old` operand, 0.
__device__ __forceinline__ uint32_t wave_incl_scan_full(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Bitonic sort, descending, of 64*E keys held as r[e] = element (e*64 + lane).
template <int E>
__device__ __forceinline__ void wave_sort_desc(uint64_t (&r)[E]) {
  const int lane = threadIdx.x & 63;
  constexpr int P = 64 * E;
  // fully unrolled: every shuffle distance is a compile-time constant
#pragma unroll
  for (int size = 2; size <= P; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= 64) {  // partners in the same lane, other register
        const int rs = stride / 64;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & rs) == 0) {
            const int i = e * 64 + lane;
            const bool desc = (i & size) == 0;
            const uint64_t x = r[e], y = r[e + rs];
            if ((x < y) == desc) {
              r[e] = y;
              r[e + rs] = x;
            }
          }
        }
      } else {  // partners in another lane, same register
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int i = e * 64 + lane;
          const uint64_t y = xor_lane_u64(r[e], stride);
          const bool desc = (i & size) == 0;
          const bool lower = (lane & stride) == 0;
          // the lower element of a pair keeps the larger key when descending
          const bool keep_max = lower == desc;
          r[e] = keep_max ? (r[e] > y ? r[e] : y) : (r[e] < y ? r[e] : y);
        }
      }
    }
  }
}

template <int E>
__device__ __forceinline__ void wave_sort_store(const uint64_t* sbuf, uint32_t k_eff, int64_t k, uint64_t* out) {
  const int lane = threadIdx.x & 63;
  uint64_t r[E];
#pragma unroll
  for (int e = 0; e < E; ++e) r[e] = (uint32_t)(e * 64 + lane) < k_eff ? sbuf[e * 64 + lane] : 0ull;
  wave_sort_desc<E>(r);
#pragma unroll
  for (int e = 0; e < E; ++e)
    if (e * 64 + lane < k) out[e * 64 + lane] = r[e];
}

// Radix select on n <= E * 64 distinct keys held in registers (key[e] is element
// e*64 + lane; elements >= n are ignored). Returns (shift, prefix): the k_eff
// largest keys are exactly those with (key >> shift) >= (prefix >> shift). One
// wave runs it (hist: 256 words of LDS of its own); it synchronises only itself.
// With max_passes, the select stops after that many digits: the set then holds the
// k_eff largest keys and possibly more (the rest of the last digit's bucket), which
// is all a threshold needs.
template <int E>
__device__ __forceinline__ void wave_radix_select(const uint64_t (&key)[E], int n, uint32_t k_eff, uint32_t* hist,
                                                  int* shift_out, uint64_t* prefix_out, int max_passes = 8) {
  const int lane = threadIdx.x & 63;
  uint64_t kmin = ~0ull, kmax = 0ull;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if (lane + 64 * e < n) {
      kmin = key[e] < kmin ? key[e] : kmin;
      kmax = key[e] > kmax ? key[e] : kmax;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t a0 = xor_lane_u64(kmin, off), a1 = xor_lane_u64(kmax, off);
    kmin = a0 < kmin ? a0 : kmin;
    kmax = a1 > kmax ? a1 : kmax;
  }
  // bits above the highest differing bit are common to every candidate; the first
  // digit starts at that bit (not at a byte boundary), so it splits the candidates
  // over as many bins as 8 bits can (scores above a threshold often share their top
  // byte, which would pile a byte-aligned first pass onto a few bins)
  const uint64_t diff = kmin ^ kmax;
  int shift = diff == 0 ? 1 : 64 - __builtin_clzll(diff);  // bits [0, shift) differ
  uint64_t prefix = (shift >= 64) ? 0 : (kmax >> shift) << shift;
  uint32_t kr = k_eff;
  for (int pass = 0; pass < max_passes && shift > 0 && kr < (uint32_t)n; ++pass) {
    const int top = shift;  // keys still in play share every bit at or above top
    const int width = top < 8 ? top : 8;
    shift = top - width;
    reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0u, 0u, 0u, 0u);
    wave_sync_lds();
    const uint64_t pre_hi = top >= 64 ? 0 : prefix >> top;
    const uint32_t dmask = (1u << width) - 1u;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool match = lane + 64 * e < n && (top >= 64 || (key[e] >> top) == pre_hi);
      if (match) atomicAdd(&hist[(uint32_t)(key[e] >> shift) & dmask], 1u);
    }
    wave_sync_lds();
    const uint4 h4 = reinterpret_cast<const uint4*>(hist)[63 - lane];  // bins 255-4l .. 252-4l
    const uint32_t c4[4] = {h4.w, h4.z, h4.y, h4.x};                   // descending digit order
    const uint32_t local = c4[0] + c4[1] + c4[2] + c4[3];
    uint32_t run = wave_incl_scan_full(local) - local;
    uint32_t digit = 0, above = 0, cnt = 0;
    bool here = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (!here && run < kr && kr <= run + c4[e]) {
        here = true;
        digit = 255u - (uint32_t)(lane * 4 + e);
        above = run;
        cnt = c4[e];
      }
      run += c4[e];
    }
    const uint64_t who = __ballot(here);
    const int src = __builtin_ctzll(who);  // wave-uniform
    digit = (uint32_t)__builtin_amdgcn_readlane((int)digit, src);
    above = (uint32_t)__builtin_amdgcn_readlane((int)above, src);
    cnt = (uint32_t)__builtin_amdgcn_readlane((int)cnt, src);
    wave_sync_lds();  // hist is cleared again by the next pass
    prefix |= (uint64_t)digit << shift;
    kr -= above;
    if (cnt == kr) break;  // every key of this bucket is selected
  }
  *shift_out = shift;
  *prefix_out = prefix;
}

// The k_eff <= 64 * E distinct keys of sbuf, stored in descending order (the first
// 64 * E of k words, 0 pads): each key goes to its rank, the number of larger keys,
// counted against every key through broadcast LDS reads. Two VALU per comparison:
// at E = 1 faster than the bitonic network (measured slower at E = 2).
template <int E>
__device__ __forceinline__ void wave_rank_store(const uint64_t* sbuf, uint32_t k_eff, int64_t k, uint64_t* out) {
  const int lane = threadIdx.x & 63;
  uint64_t x[E];
  uint32_t rank[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    x[e] = (uint32_t)(e * 64 + lane) < k_eff ? sbuf[e * 64 + lane] : 0ull;
    rank[e] = 0;
  }
#pragma unroll 8
  for (uint32_t j = 0; j < k_eff; ++j) {
    const uint64_t y = sbuf[j];
#pragma unroll
    for (int e = 0; e < E; ++e) rank[e] += y > x[e] ? 1u : 0u;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int t = e * 64 + lane;
    if ((uint32_t)t < k_eff) out[rank[e]] = x[e];
    else if (t < k) out[t] = 0ull;
  }
}

// The k_eff (<= KCAP: 256 or 512) largest of n <= E * 64 register keys, sorted
// descending, written as k words to out (0 pads). sbuf: KCAP keys of LDS.
template <int E, int KCAP = 256>
__device__ __forceinline__ void wave_select_store(const uint64_t (&key)[E], int n, uint32_t k_eff, int64_t k,
                                                  uint64_t* sbuf, uint32_t* hist, uint64_t* out) {
  const int lane = threadIdx.x & 63;
  int shift;
  uint64_t prefix;
  wave_radix_select<E>(key, n, k_eff, hist, &shift, &prefix);
  // selected: (key >> shift) >= (prefix >> shift); compact them into sbuf
  const uint64_t lim = prefix >> shift;
  int base = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const bool take = lane + 64 * e < n && (key[e] >> shift) >= lim;
    const uint64_t m = __ballot(take);
    const int pos = base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (take && pos < KCAP) sbuf[pos] = key[e];
    base += __popcll(m);
  }
  wave_sync_lds();
  int sorted;
  if (k_eff <= 64) wave_rank_store<1>(sbuf, k_eff, k, out), sorted = 64;
  else if (k_eff <= 128) wave_sort_store<2>(sbuf, k_eff, k, out), sorted = 128;
  else if (KCAP <= 256 || k_eff <= 256) wave_sort_store<4>(sbuf, k_eff, k, out), sorted = 256;
  else wave_sort_store<(KCAP > 256 ? 8 : 4)>(sbuf, k_eff, k, out), sorted = 512;
  for (int64_t t = lane + sorted; t < k; t += 64) out[t] = 0ull;
}

// Reads a row's n candidate words (c0 from b0, the rest from b1) into E registers
// per lane as order-preserving keys, then selects and stores.
template <int E, int KCAP = 256>
__device__ __forceinline__ void cand_select_regs(const uint64_t* b0, const uint64_t* b1, int c0, int n, uint32_t k_eff,
                                                 int64_t k, uint64_t* sbuf, uint32_t* hist, uint64_t* out) {
  const int lane = threadIdx.x & 63;
  uint64_t key[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = lane + 64 * e;
    uint64_t wd = 0;
    if (i < n) wd = i < c0 ? b0[i] : b1[i - c0];
    key[e] = ((uint64_t)ord_u32(__uint_as_float((uint32_t)(wd >> 32))) << 32) | (wd & 0xFFFFFFFFull);
  }
  wave_select_store<E, KCAP>(key, n, k_eff, k, sbuf, hist, out);
}

// BIG: rows of up to 2048 candidates and k <= 512 (the filtered path's larger lists)
template <bool BIG>
__device__ __forceinline__ void cand_select_row(const Problem& pb, const Pass& ps, const PassBufs& bufs, int64_t p,
                                                uint64_t* sbuf, uint32_t* hist, uint32_t* misc) {
  constexpr int KCAP = BIG ? 512 : 256, NMAX = BIG ? 128 * CAND_REGS : 64 * CAND_REGS;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  int64_t c0 = bufs.cnt[2 * p], c1 = bufs.cnt[2 * p + 1];
  if (bufs.cand_single) {  // one list of c0 entries running on into the second half
    c1 = c0 > bufs.caph ? c0 - bufs.caph : 0;
    c0 = c0 > bufs.caph ? bufs.caph : c0;
  }
  if (c0 > bufs.caph || c1 > bufs.caph || c0 + c1 < (int64_t)k_eff || k_eff > KCAP || c0 + c1 > NMAX) {
    if ((threadIdx.x & 63) == 0) bufs.redo_list[atomicAdd(bufs.redo_count, 1)] = (int32_t)p;
    return;
  }
  const int n = (int)(c0 + c1);
  const uint64_t* b0 = bufs.cand + (2 * p) * bufs.caph;
  uint64_t* out = bufs.sel + p * pb.k;
  if (!BIG) {
    // registers sized to the list in steps of 64 keys
    if (n <= 128) cand_select_regs<2>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 192) cand_select_regs<3>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 256) cand_select_regs<4>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 320) cand_select_regs<5>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 384) cand_select_regs<6>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 448) cand_select_regs<7>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 512) cand_select_regs<8>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else {
      // rare long lists: the exact select over the words where they are (global
      // memory), so that the common short lists keep few registers (more waves)
      auto getkey = [&](int64_t e) { return raw_to_key(e < c0 ? b0[e] : b0[bufs.caph + (e - c0)]); };
      team_topk<64>(getkey, n, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc, out);
    }
  } else {
    if (n <= 512) cand_select_regs<8, KCAP>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else if (n <= 1024) cand_select_regs<CAND_REGS, KCAP>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
    else cand_select_regs<2 * CAND_REGS, KCAP>(b0, b0 + bufs.caph, (int)c0, n, k_eff, pb.k, sbuf, hist, out);
  }
}

template <bool BIG>
__global__ __launch_bounds__(64) void k_cand_select(Problem pb, Pass ps, PassBufs bufs) {
  __shared__ uint64_t sbuf[BIG ? 512 : 256];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  cand_select_row<BIG>(pb, ps, bufs, blockIdx.x, sbuf, hist, misc);
}

// ------------------------------------------------------------------ filtered chunk-tile path
// Per row, the threshold is the R-th largest of its valid sampled scores (every
// FILTER_KSTRIDE-th key), R a few standard deviations above the sample's expected
// share mu of the top k_eff, resolved to a few bits below those all the row's samples
// share (it may lie a little below that sample, never above). About R * FILTER_KSTRIDE scores of the row
// are then at or above it; a row with fewer than R valid samples keeps every valid key. The
// candidate select proves each row's set complete (at least k_eff entries, no
// overflow) or sends the row to the exact fallback.
// The rank R of a row's threshold among its ns valid samples (nv valid keys): mu =
// k_eff * ns / nv is the sample's expected share of the row's top k_eff, and R = mu +
// z sqrt(mu) + z puts the k-th score below the threshold about z standard deviations
// away. A row that misses is recomputed exactly, at a cost of nv * d products: where
// that is small (at most 2^21) z = 3 (about one row in 10^4 recomputed, fewer
// candidates for all the others), else z = 4.
__device__ __forceinline__ int filter_rank(uint32_t k_eff, int64_t ns, int64_t nv, int64_t d) {
  const float mu = (float)k_eff * (float)ns / (float)nv;
  const float z = nv * d <= (int64_t(1) << 21) ? 3.0f : 4.0f;
  return (int)ceilf(mu + z * sqrtf(mu) + z);
}

// One wave per row, four rows per workgroup. Each lane keeps the two largest of its
// samples (a running maximum and median of three, on the scores themselves); the
// R-th largest of those 128 is built bit by bit, high to low, on their
// order-preserving 32-bit keys: a bit is kept when at least R of them are at or above
// the prefix with it set (two ballots per bit, no LDS). Starting below the bits that
// the largest and the smallest of the 128 share, THRESH_BITS bits are resolved; the
// threshold is then the smallest of the 128 at or above the prefix, which is at most
// their R-th largest and so at most the R-th largest sample. The kernel is bound by
// its vector instructions: per sample it spends a range test, a select, a maximum and
// a median, and the row's sample loads run past its end (into the next rows, or the
// padding that ends the sample buffer) instead of being clamped.
constexpr int THRESH_BITS = 16;
static_assert(64 * CAND_REGS * sizeof(float) <= FILTER_SAMP_PAD, "a row's loads stay within the padded buffer");
__global__ __launch_bounds__(256) void k_filter_threshold(Problem pb, Pass ps, PassBufs bufs) {
  const int64_t p = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform
  if (p >= ps.nc * pb.C) return;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int lane = threadIdx.x & 63;
  const int64_t nv = valid_keys(pb, rr.i);
  const int64_t ns = (nv + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE;  // valid samples (<= 64 * CAND_REGS)
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  const int R = filter_rank(k_eff, ns, nv, pb.d);
  float ts = -INFINITY;
  if (R < ns) {
    const float* row = bufs.samp + p * ((pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE);
    const int nsi = (int)ns;
    auto rth = [&](auto tag) {  // the R-th largest of the row's ns samples, or a little less
      constexpr int E = decltype(tag)::value;
      float x[E];
#pragma unroll
      for (int e = 0; e < E; ++e) x[e] = row[lane + 64 * e];  // every load in flight at once
      // this lane's two largest samples, t1 >= t2 (-inf where it has fewer)
      float t1 = -INFINITY, t2 = -INFINITY;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float v = lane + 64 * e < nsi ? x[e] : -INFINITY;
        t2 = __builtin_amdgcn_fmed3f(t1, t2, v);
        t1 = __builtin_elementwise_maximum(t1, v);
      }
      const uint32_t u1 = ord_u32(t1), u2 = ord_u32(t2);
      // the smallest of the 128 that is a sample (t2 is one wherever ns > 128)
      const uint32_t lo = t2 != -INFINITY ? u2 : t1 != -INFINITY ? u1 : 0xFFFFFFFFu;
      const uint32_t kmin = wave_extreme_u32_full<false>(lo), kmax = wave_extreme_u32_full<true>(u1);
      // bits [0, top) differ among them; the ones above are shared by all, so also by
      // their R-th largest
      const int top = kmin == kmax ? 0 : 32 - __builtin_clz(kmin ^ kmax);
      uint32_t prefix = top >= 32 ? 0u : (kmax >> top) << top;
      const int stop = top > THRESH_BITS ? top - THRESH_BITS : 0;
      // (k <= 512 and one sample in 16 keep R near 60 at most, within the 128)
      for (int b = top - 1; b >= stop; --b) {
        const uint32_t cand = prefix | (1u << b);
        const uint32_t cnt = (uint32_t)__popcll(__ballot(u1 >= cand)) + (uint32_t)__popcll(__ballot(u2 >= cand));
        if (cnt >= (uint32_t)R) prefix = cand;
      }
      const uint32_t m = min(u1 >= prefix ? u1 : 0xFFFFFFFFu, u2 >= prefix ? u2 : 0xFFFFFFFFu);
      return ord_to_f32(wave_extreme_u32_full<false>(m));
    };
    if (ns <= 128) ts = rth(std::integral_constant<int, 2>{});
    else if (ns <= 256) ts = rth(std::integral_constant<int, 4>{});
    else if (ns <= 512) ts = rth(std::integral_constant<int, 8>{});
    else ts = rth(std::integral_constant<int, CAND_REGS>{});
  }
  if (lane == 0) bufs.thr[p] = ts;
}

// the same threshold with one workgroup per row, for rows of up to 4096 samples
__global__ __launch_bounds__(256) void k_filter_threshold_wg(Problem pb, Pass ps, PassBufs bufs) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  __shared__ uint32_t lowest;
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;  // whole workgroup
  const int64_t nv = valid_keys(pb, rr.i);
  const int64_t ns = (nv + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE;
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  const int R = filter_rank(k_eff, ns, nv, pb.d);
  float ts = -INFINITY;
  if (R < ns) {
    const float* row = bufs.samp + p * ((pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE);
    auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
    int shift;
    uint64_t prefix;
    team_radix_select<256>(getkey, ns, (uint32_t)R, hist, misc, &shift, &prefix, THRESH_PASSES);
    if (threadIdx.x == 0) lowest = 0xFFFFFFFFu;
    __syncthreads();
    uint32_t m = 0xFFFFFFFFu;  // the smallest selected score: at most the R-th largest sample
    for (int64_t e = threadIdx.x; e < ns; e += 256) {
      const uint64_t key = getkey(e);
      if ((key >> shift) >= (prefix >> shift)) m = min(m, (uint32_t)(key >> 32));
    }
    atomicMin(&lowest, m);
    __syncthreads();
    ts = ord_to_f32(lowest);
  }
  if (threadIdx.x == 0) bufs.thr[p] = ts;
}

__global__ void k_zero_counts(int32_t* p, int64_t n) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    p[e] = 0;
}

// stage 0: zero the candidate counts; 1: sampled scores; 2: thresholds; 3: filtered tile
hipError_t launch_filter(const Problem& pb, const Pass& ps, const PassBufs& b, int stage, hipStream_t st) {
  const int64_t rows = ps.nc * pb.C;
  if (stage == 0) {
    k_zero_counts<<<1024, 256, 0, st>>>(b.cnt, 2 * rows);
  } else if (stage == 1 || stage == 3) {
    const int64_t slots = stage == 1 ? (pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE : pb.Lk;
    const int64_t g = ((slots + TSM_TK - 1) / TSM_TK) * ((pb.C + TSM_TQ - 1) / TSM_TQ) * ps.nc;
    if (g > 0x7FFFFFFF || pb.dtype != T_BF16 || pb.d % 32 != 0 || pb.Lk > FILTER_MAX_LK) return hipErrorInvalidValue;
    if (stage == 1) k_tile_scores_mfma<1><<<(unsigned)g, 256, 0, st>>>(pb, ps, b);
    else if (filter_scan_ok(pb)) return launch_filter_scan(pb, ps, b, st);
    else k_tile_scores_mfma<2><<<(unsigned)g, 256, 0, st>>>(pb, ps, b);
  } else if ((pb.Lk + FILTER_KSTRIDE - 1) / FILTER_KSTRIDE <= 64 * CAND_REGS) {
    k_filter_threshold<<<(unsigned)((rows + 3) / 4), 256, 0, st>>>(pb, ps, b);
  } else {
    k_filter_threshold_wg<<<(unsigned)rows, 256, 0, st>>>(pb, ps, b);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ chunk-tile path: short-row select
// One wave per query row of the score tile, for rows of at most TSW_MAX_N valid
// keys and k <= 256. The row's candidates are gathered into LDS in one pass and
// selected in registers (radix select sized to the candidate count):
//  * rows of at most 64 * CAND_REGS keys take every key;
//  * longer rows take every score >= ts, ts being the R-th largest of
//    64 * CAND_REGS evenly spaced sampled scores, R a few standard deviations
//    above the sample's expected share of the top k, resolved to THRESH_PASSES
//    radix digits (it may lie a little below that sample, never above). For
//    R <= 96 (long rows) ts comes from the per-lane top two of the sample, which
//    leaves at least R sampled scores >= ts at a fraction of the cost;
//  * a row whose gathered set is short of k_eff keys or overflows goes to the
//    redo list (exact fallback from the tile row).
constexpr int TSW_MAX_N = 8192;

template <int E>
__device__ __forceinline__ void lds_select_store(const uint64_t* cbuf, int c, uint32_t k_eff, int64_t k,
                                                 uint64_t* sbuf, uint32_t* hist, uint64_t* out) {
  const int lane = threadIdx.x & 63;
  uint64_t key[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = lane + 64 * e;
    key[e] = i < c ? raw_to_key(cbuf[i]) : 0ull;
  }
  __syncthreads();  // cbuf may alias sbuf
  wave_select_store<E>(key, c, k_eff, k, sbuf, hist, out);
}

__global__ __launch_bounds__(64) void k_tile_select_wave(Problem pb, Pass ps, const float* S, uint64_t* sel,
                                                         int32_t* redo_list, int32_t* redo_count) {
  constexpr int CAPW = 64 * CAND_REGS;
  __shared__ uint64_t cbuf[CAPW];  // gathered keys; the final sort reuses its start
  __shared__ uint32_t hist[256];
  const int64_t p = blockIdx.x;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int lane = threadIdx.x & 63;
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  const float* row = S + p * pb.Lk;
  uint64_t* out = sel + p * pb.k;
  float ts = -INFINITY;
  if (nv > CAPW) {
    // sample s = lane + 64 e sits at position floor(s * nv / CAPW) (distinct: nv > CAPW)
    float smp[CAND_REGS];
    static_assert((int64_t)TSW_MAX_N * CAPW < (int64_t(1) << 31), "sample positions fit 32 bits");
#pragma unroll
    for (int e = 0; e < CAND_REGS; ++e) smp[e] = row[((uint32_t)(lane + 64 * e) * (uint32_t)nv) / CAPW];
    const float mu = (float)k_eff * (float)CAPW / (float)nv;
    int R = (int)ceilf(mu + 6.0f * sqrtf(mu) + 8.0f);
    R = R < CAPW ? R : CAPW;
    int shift;
    uint64_t prefix;
    if (R <= 96) {
      float t1 = -INFINITY, t2 = -INFINITY;  // this lane's two largest samples
#pragma unroll
      for (int e = 0; e < CAND_REGS; ++e) {
        const float hi = fmaxf(t1, smp[e]), lo = fminf(t1, smp[e]);
        t1 = hi;
        t2 = fmaxf(t2, lo);
      }
      uint64_t k2[2] = {make_key(t1, 2u * lane), make_key(t2, 2u * lane + 1u)};
      wave_radix_select<2>(k2, 128, (uint32_t)R, hist, &shift, &prefix, THRESH_PASSES);
      uint32_t m = 0xFFFFFFFFu;
#pragma unroll
      for (int e = 0; e < 2; ++e)
        if ((k2[e] >> shift) >= (prefix >> shift)) m = min(m, (uint32_t)(k2[e] >> 32));
      ts = ord_to_f32(wave_extreme_u32_full<false>(m));
    } else {
      uint64_t key[CAND_REGS];
#pragma unroll
      for (int e = 0; e < CAND_REGS; ++e) key[e] = make_key(smp[e], (uint32_t)(lane + 64 * e));
      wave_radix_select<CAND_REGS>(key, CAPW, (uint32_t)R, hist, &shift, &prefix, THRESH_PASSES);
      uint32_t m = 0xFFFFFFFFu;
#pragma unroll
      for (int e = 0; e < CAND_REGS; ++e)
        if ((key[e] >> shift) >= (prefix >> shift)) m = min(m, (uint32_t)(key[e] >> 32));
      ts = ord_to_f32(wave_extreme_u32_full<false>(m));
    }
  }
  // gather (wave-level compaction; c is wave-uniform)
  uint32_t c = 0;
  auto reserve = [&](uint32_t cnt) {
    const uint32_t b = c;
    c += cnt;
    return b;
  };
  gather_row(row, nv, ts, (pb.Lk & 3) == 0, lane, 64, cbuf, (uint32_t)CAPW, reserve);
  if (c < k_eff || c > (uint32_t)CAPW) {
    if (lane == 0) redo_list[atomicAdd(redo_count, 1)] = (int32_t)p;
    return;
  }
  __syncthreads();
  if (c <= 128) lds_select_store<2>(cbuf, (int)c, k_eff, pb.k, cbuf, hist, out);
  else if (c <= 256) lds_select_store<4>(cbuf, (int)c, k_eff, pb.k, cbuf, hist, out);
  else if (c <= 512) lds_select_store<8>(cbuf, (int)c, k_eff, pb.k, cbuf, hist, out);
  else lds_select_store<CAND_REGS>(cbuf, (int)c, k_eff, pb.k, cbuf, hist, out);
}

// Rows the short-row select could not settle: multi-pass radix select straight
// from the tile row, one workgroup per row, REDO_BLOCKS workgroups in turn.
__global__ __launch_bounds__(256) void k_tile_select_redo(Problem pb, Pass ps, const float* S, uint64_t* sel,
                                                          const int32_t* redo_list, const int32_t* redo_count) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  const int32_t nredo = *redo_count;
  for (int32_t r = blockIdx.x; r < nredo; r += gridDim.x) {
    const int64_t p = redo_list[r];
    const RowRef rr = row_of(pb, ps, p);
    const int64_t nv = valid_keys(pb, rr.i);
    const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
    const float* row = S + p * pb.Lk;
    auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
    team_topk<256>(getkey, nv, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc, sel + p * pb.k);
    __syncthreads();
  }
}

// ------------------------------------------------------------------ fused path: fallback
// Exact recomputation of the rows on the redo list (candidate buffer overflow, or
// a threshold that turned out above the row's k-th score). The first REDO_CAP rows
// are spread over many workgroups: fp32 dot products of each row against every
// valid key (key splits of REDO_SPLIT keys per work item) into a row buffer, then
// one workgroup per row runs the radix select. Rows beyond REDO_CAP (only when the
// threshold fails wholesale, e.g. adversarially ordered scores) take the slower
// one-workgroup-per-row kernel.
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&x)[8]);
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float (&x)[8]) {
  const uint4 v = *(const uint4*)p;
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(w[e] << 16);
    x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
  }
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&x)[8]) {
  const float4 u = *(const float4*)p, v = *(const float4*)(p + 4);
  x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  x[4] = v.x; x[5] = v.y; x[6] = v.z; x[7] = v.w;
}

template <typename T>
__global__ __launch_bounds__(256) void k_redo_scores(Problem pb, Pass ps, PassBufs bufs) {
  __shared__ float qrow[1024];
  const int32_t total = *bufs.redo_count;
  const int64_t rows = total < REDO_CAP ? total : REDO_CAP;
  const int64_t splits = (pb.Lk + REDO_SPLIT - 1) / REDO_SPLIT;
  for (int64_t item = blockIdx.x; item < rows * splits; item += gridDim.x) {
    const int64_t r = item / splits, sp = item - r * splits;
    const int64_t p = bufs.redo_list[r];
    const RowRef rr = row_of(pb, ps, p);
    const int64_t nv = valid_keys(pb, rr.i);
    const T* q = (const T*)pb.Q + (rr.bh * pb.Lq + rr.i) * pb.d;
    for (int f = threadIdx.x; f < pb.d; f += 256) qrow[f] = load_elem<T>(q, f);
    __syncthreads();
    const T* Kh = (const T*)pb.K + rr.bh * pb.kv_head_stride;
    float* row = bufs.scores + r * pb.Lk;
    // two keys per thread, their loads interleaved (REDO_SPLIT = 2 * 256)
    static_assert(REDO_SPLIT == 512, "two keys per thread");
    const int64_t j1 = (sp + 1) * REDO_SPLIT < nv ? (sp + 1) * REDO_SPLIT : nv;
    const int64_t ja = sp * REDO_SPLIT + threadIdx.x, jb = ja + 256;
    const T* ka = Kh + (ja < j1 ? ja : 0) * pb.d;
    const T* kb = Kh + (jb < j1 ? jb : 0) * pb.d;
    float acc_a = 0.f, acc_b = 0.f;
    // unrolled so that several 16-byte loads of both rows are in flight at once
#pragma unroll 4
    for (int64_t f = 0; f < pb.d; f += 8) {
      float xa[8], xb[8];
      load8<T>(ka + f, xa);
      load8<T>(kb + f, xb);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        acc_a = fmaf(qrow[f + e], xa[e], acc_a);
        acc_b = fmaf(qrow[f + e], xb[e], acc_b);
      }
    }
    if (ja < j1) row[ja] = acc_a;
    if (jb < j1) row[jb] = acc_b;
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void k_redo_select(Problem pb, Pass ps, PassBufs bufs) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  const int64_t r = blockIdx.x;
  if (r >= *bufs.redo_count) return;
  const int64_t p = bufs.redo_list[r];
  const RowRef rr = row_of(pb, ps, p);
  const int64_t nv = valid_keys(pb, rr.i);
  const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
  __shared__ uint64_t cand[TS_CAP];
  __shared__ uint32_t ccount;
  wg_row_select(bufs.scores + r * pb.Lk, nv, k_eff, pb.k, (pb.Lk & 3) == 0, cand, sbuf, hist, misc, &ccount,
                bufs.sel + p * pb.k, nullptr);
}

template <typename T>
__global__ __launch_bounds__(256) void k_redo_rest(Problem pb, Pass ps, PassBufs bufs) {
  extern __shared__ uint64_t sbuf[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t misc[8];
  __shared__ float qrow[1024];
  float* row = bufs.scores + ((int64_t)REDO_CAP + blockIdx.x) * pb.Lk;
  const int32_t total = *bufs.redo_count;
  for (int32_t t = REDO_CAP + blockIdx.x; t < total; t += gridDim.x) {
    const int64_t p = bufs.redo_list[t];
    const RowRef rr = row_of(pb, ps, p);
    const int64_t nv = valid_keys(pb, rr.i);
    const uint32_t k_eff = (uint32_t)(pb.k < nv ? pb.k : nv);
    const T* q = (const T*)pb.Q + (rr.bh * pb.Lq + rr.i) * pb.d;
    for (int f = threadIdx.x; f < pb.d; f += 256) qrow[f] = load_elem<T>(q, f);
    __syncthreads();
    const T* Kh = (const T*)pb.K + rr.bh * pb.kv_head_stride;
    for (int64_t j = threadIdx.x; j < nv; j += 256) {
      const T* kr = Kh + j * pb.d;
      float acc = 0.f;
      for (int64_t f = 0; f < pb.d; f += 8) {
        float x[8];
        load8<T>(kr + f, x);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(qrow[f + e], x[e], acc);
      }
      row[j] = acc;
    }
    __syncthreads();
    auto getkey = [&](int64_t e) { return make_key(row[e], (uint32_t)e); };
    team_topk<256>(getkey, nv, k_eff, (uint32_t)pb.k, sbuf, pow2_at_least(k_eff), hist, misc, bufs.sel + p * pb.k);
    __syncthreads();
  }
}

// ------------------------------------------------------------------ finalize
// One wave per row (or per row and column slice): activation over the k_eff
// survivors (softmax with the Eq. 1 temperature, or ReLU), then the weighted sum of
// the selected value rows (Eq. 4; the value rows are W2's rows for Eq. 3). Value
// rows are read as 16-byte vectors: with NV vectors per row (or slice), 64/NV rows
// are gathered per wave instruction (d = 64 bf16: 8 rows), each lane accumulating
// its vector's columns in fp32; the row slots are then reduced across lanes.
// value-row gathers a finalize lane has in flight together: 4 where the value rows sit
// in an XCD's L2 (more measured slower), 8 for column slices of a larger matrix, whose
// gathers the fabric serves (16384 tokens, 65536 value rows of 1024: 1.73 -> 1.57 ms)
template <int NSLICES>
constexpr int fin_unroll() { return NSLICES > 1 ? 8 : 4; }
template <typename T> struct Vec16;
template <> struct Vec16<uint16_t> {
  static constexpr int E = 8;
  static __device__ __forceinline__ uint4 raw(const uint16_t* p) { return *(const uint4*)p; }
  static __device__ __forceinline__ void unpack(const uint4 v, float (&x)[8]) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
  static __device__ __forceinline__ void load(const uint16_t* p, float (&x)[8]) { unpack(raw(p), x); }
  static __device__ __forceinline__ void store(uint16_t* p, const float (&x)[8]) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = (uint32_t)f32_to_bf16(x[2 * e]) | ((uint32_t)f32_to_bf16(x[2 * e + 1]) << 16);
    *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Vec16<float> {
  static constexpr int E = 4;
  static __device__ __forceinline__ uint4 raw(const float* p) { return *(const uint4*)p; }
  static __device__ __forceinline__ void unpack(const uint4 v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y); x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  static __device__ __forceinline__ void load(const float* p, float (&x)[4]) { unpack(raw(p), x); }
  static __device__ __forceinline__ void store(float* p, const float (&x)[4]) {
    *(float4*)p = make_float4(x[0], x[1], x[2], x[3]);
  }
};

// Reorders a row's n <= 64 * E (weight, key index) pairs in LDS by increasing key
// index (the indices are distinct), through the register bitonic network.
template <int E>
__device__ __forceinline__ void sort_by_key_index(float* w, uint32_t* jj, int n) {
  const int lane = threadIdx.x & 63;
  uint64_t r[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int t = e * 64 + lane;  // descending on ~index = ascending on index; pads (0) go last
    r[e] = t < n ? ((uint64_t)(~jj[t]) << 32) | __float_as_uint(w[t]) : 0ull;
  }
  wave_sort_desc<E>(r);
  __syncthreads();
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int t = e * 64 + lane;
    if (t < n) {
      jj[t] = ~(uint32_t)(r[e] >> 32);
      w[t] = __uint_as_float((uint32_t)r[e]);
    }
  }
  __syncthreads();
}

#ifdef TOPK_CHECK_INDICES
// Checked builds count the selected indices that lie outside the value matrix (the
// finalize still clamps them, so that no read leaves it); read with
// topk_debug_bad_indices.
__device__ unsigned long long g_bad_indices = 0;
#endif

template <typename T, int NSLICES>
__device__ __forceinline__ void finalize_row(const Problem& pb, const Pass& ps, const uint64_t* sel, int64_t p,
                                             float* w, uint32_t* jj, int slice) {
  constexpr int E = Vec16<T>::E;
  const RowRef rr = row_of(pb, ps, p);
  if (!rr.ok) return;
  const int lane = threadIdx.x & 63;
  const int64_t nv = valid_keys(pb, rr.i);
  const int64_t k_eff = pb.k < nv ? pb.k : nv;
  const int64_t grow = rr.bh * pb.Lq + rr.i;
  const uint64_t* srow = sel + p * pb.k;
  const uint32_t jmax = (uint32_t)(pb.Lk - 1);
  for (int64_t t = lane; t < pb.k; t += 64) {
    float s = -INFINITY;
    int32_t j = -1;
    if (t < k_eff) {
      const uint64_t key = srow[t];
      s = key_score(key);
      j = (int32_t)key_index(key);
      w[t] = s;
      jj[t] = (uint32_t)j < jmax ? (uint32_t)j : jmax;  // keeps a bad selection from reading out of bounds
#ifdef TOPK_CHECK_INDICES
      if ((uint32_t)j > jmax) atomicAdd(&g_bad_indices, 1ull);
#endif
    }
    if (slice == 0) {
      if (pb.idx_out) pb.idx_out[grow * pb.k + t] = j;
      if (pb.score_out) pb.score_out[grow * pb.k + t] = s;
    }
  }
  __syncthreads();
  float inv = 1.f;
  if (pb.act == ACT_SOFTMAX) {
    const float m = w[0];
    const float c = pb.scale * 1.4426950408889634f;  // exp(x) = exp2(x * log2 e)
    float sum = 0.f;
    for (int64_t t = lane; t < k_eff; t += 64) {
      const float e = exp2f((w[t] - m) * c);
      w[t] = e;
      sum += e;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
    inv = 1.f / sum;
  } else {
    for (int64_t t = lane; t < k_eff; t += 64) w[t] = fmaxf(w[t], 0.f);
  }
  __syncthreads();
  if (NSLICES > 1 && k_eff > 1 && k_eff <= 512) {
    // wide value rows: gather the survivors in increasing key order, so that the
    // waves sharing an XCD walk its slice of the value matrix in the same direction
    if (k_eff <= 64) sort_by_key_index<1>(w, jj, (int)k_eff);
    else if (k_eff <= 128) sort_by_key_index<2>(w, jj, (int)k_eff);
    else if (k_eff <= 256) sort_by_key_index<4>(w, jj, (int)k_eff);
    else sort_by_key_index<8>(w, jj, (int)k_eff);
  }
  const T* Vh = (const T*)pb.V + rr.bh * pb.kv_head_stride;
  const uint32_t d32 = (uint32_t)pb.d;  // row offsets j * d are 32 x 32 -> 64-bit products
  T* orow = (T*)pb.out + grow * pb.d;
  const int nvec = (int)(pb.d / E) / NSLICES;      // 16-byte vectors of this slice per value row
  const int vbeg = slice * nvec, vend = vbeg + nvec;
  int np2 = 1;                                      // lanes per row slot: a power of two >= nvec
  while (np2 < nvec && np2 < 64) np2 <<= 1;
  const int slots = 64 / np2;                       // rows gathered per instruction
  const int vlane = lane % np2, slot = lane / np2;
  for (int v0 = vbeg + vlane; v0 < vend; v0 += 64) {
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    constexpr int FIN_U = fin_unroll<NSLICES>();
    {
      // FIN_U independent gathers: every raw load is issued before the first
      // is unpacked; the sum still runs over t in increasing order
      const T* vcol = Vh + v0 * E;
      int64_t t = slot;
      for (; t + (FIN_U - 1) * slots < k_eff; t += FIN_U * slots) {
        uint4 raw[FIN_U];
#pragma unroll
        for (int q = 0; q < FIN_U; ++q) raw[q] = Vec16<T>::raw(vcol + (uint64_t)jj[t + q * slots] * d32);
        // keep the scheduler from sinking loads below the first unpack (it otherwise
        // waits for each load before issuing the next ones); the sliced gathers, bound
        // by the fabric rather than by latency, measured faster without
        if (NSLICES == 1) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < FIN_U; ++q) {
          float x[E];
          Vec16<T>::unpack(raw[q], x);
          const float wt = w[t + q * slots];
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] = fmaf(wt, x[e], acc[e]);
        }
      }
      for (; t < k_eff; t += slots) {
        float x[E];
        Vec16<T>::load(vcol + (uint64_t)jj[t] * d32, x);
        const float wt = w[t];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(wt, x[e], acc[e]);
      }
    }
    // reduce the row slots: lanes with the same vector index differ by multiples of np2
    for (int off = np2; off < 64; off <<= 1) {
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += __shfl_xor(acc[e], off, 64);
    }
    if (slot == 0) {
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] *= inv;
      Vec16<T>::store(orow + v0 * E, acc);
    }
  }
}

template <typename T, int NSLICES>
__global__ __launch_bounds__(64) void k_finalize(Problem pb, Pass ps, const uint64_t* sel) {
  static_assert(8 % NSLICES == 0, "slices are dealt to the 8 XCDs");
  extern __shared__ float fsh[];
  const int64_t G = gridDim.x, bid = blockIdx.x;
  int64_t p;
  int slice = 0;
  if (NSLICES > 1) {
    // column slices: workgroups are dealt to the XCDs in turn, so slice bid % NSLICES
    // runs only on the XCDs whose L2 holds that slice's columns
    slice = (int)(bid % NSLICES);
    p = bid / NSLICES;
  } else {
    // same XCD-aware renumbering as the scan: neighbouring rows (same head, same
    // value rows) run on one XCD
    p = (G % 8 == 0) ? (bid % 8) * (G / 8) + bid / 8 : bid;
  }
  finalize_row<T, NSLICES>(pb, ps, sel, p, fsh, (uint32_t*)(fsh + pb.k), slice);
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

// ------------------------------------------------------------------ MFMA rate probe
// A register-only stream of independent v_mfma_f32_32x32x16_bf16 (eight accumulators
// per wave, no memory traffic in the loop): the sustained MFMA rate of the chip. Wave 0
// of each workgroup also reads the shader clock counter and the constant 100 MHz
// counter around the loop, so the host can derive the clock the MFMAs ran at.
constexpr int PROBE_ITERS = 4096;
__global__ __launch_bounds__(256) void k_mfma_rate(float* sink, uint64_t* clocks) {
  const int lane = threadIdx.x & 63;
  bf16x8 av, bv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    av[e] = (__bf16)(1.0f + 0.001f * (lane + e));
    bv[e] = (__bf16)(1.0f - 0.001f * (lane + e));
  }
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = (f32x16){};
  uint64_t t0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  for (int it = 0; it < PROBE_ITERS; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j][lane & 15];
  sink[blockIdx.x * 256 + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
    clocks[2 * blockIdx.x] = t1 - t0;
    clocks[2 * blockIdx.x + 1] = r1 - r0;
  }
}

hipError_t launch_mfma_rate(float* sink, uint64_t* clocks, int blocks, hipStream_t st) {
  k_mfma_rate<<<blocks, 256, 0, st>>>(sink, clocks);
  return hipGetLastError();
}
int mfma_rate_iters() { return PROBE_ITERS; }

// ------------------------------------------------------------------ launchers
static int64_t pass_rows(const Problem& pb, const Pass& ps) { return ps.nc * pb.C; }

hipError_t launch_init(const PassBufs& b, hipStream_t st) {
  k_init<<<1, 64, 0, st>>>(b.redo_count);
  return hipGetLastError();
}

hipError_t launch_tile_scores(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  if (pb.dtype == T_BF16 && pb.d % 32 == 0) {
    const int64_t g = ((pb.Lk + TSM_TK - 1) / TSM_TK) * ((pb.C + TSM_TQ - 1) / TSM_TQ) * ps.nc;
    if (g > 0x7FFFFFFF) return hipErrorInvalidValue;
    k_tile_scores_mfma<0><<<(unsigned)g, 256, 0, st>>>(pb, ps, b);
    return hipGetLastError();
  }
  dim3 grid((unsigned)((pb.Lk + 63) / 64), (unsigned)((pb.C + 63) / 64), (unsigned)ps.nc);
  if (pb.dtype == T_BF16)
    k_tile_scores<uint16_t><<<grid, 256, 0, st>>>(pb, ps, b.scores);
  else
    k_tile_scores<float><<<grid, 256, 0, st>>>(pb, ps, b.scores);
  return hipGetLastError();
}

hipError_t launch_tile_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const int P = pow2_at_least(pb.k);
  if (pb.k <= 256 && pb.Lk <= TSW_MAX_N) {
    k_tile_select_wave<<<(unsigned)pass_rows(pb, ps), 64, 0, st>>>(pb, ps, b.scores, b.sel, b.redo_list,
                                                                    b.redo_count);
    k_tile_select_redo<<<REDO_BLOCKS, 256, (size_t)P * 8, st>>>(pb, ps, b.scores, b.sel, b.redo_list, b.redo_count);
  } else {
    k_tile_select<<<(unsigned)pass_rows(pb, ps), 256, (size_t)P * 8, st>>>(pb, ps, b.scores, b.sel, b.redo_count);
  }
  return hipGetLastError();
}

// the scan's arguments for one pass (G = 2 query groups per wave)
ScanArgs scan_args(const Problem& pb, const Pass& ps, const PassBufs& b, int mode, int stride) {
  ScanArgs a;
  a.Q = (const uint16_t*)pb.Q;
  a.K = (const uint16_t*)pb.K;
  a.Lq = pb.Lq;
  a.q0 = pb.q0;
  a.q1 = pb.q1;
  a.Lk = pb.Lk;
  a.C = pb.C;
  a.kv_head_stride = pb.kv_head_stride;
  a.c0 = ps.c0;
  a.nchunk = ps.nchunk;
  a.cand = b.cand;
  a.cnt = b.cnt;
  a.caph = b.caph;
  a.thr = b.thr;
  a.mode = mode;
  a.stride = stride;
  a.causal = pb.causal ? 1 : 0;
  a.wgs_per_chunk = (pb.C + scan_queries_per_wg<2>() - 1) / scan_queries_per_wg<2>();
  return a;
}

// The filtered path's candidates (stage 3) by the scan in its direct mode: thresholds
// from b.thr, one list per row and half-wave (b.cand_single == 0).
hipError_t launch_filter_scan(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  if (!filter_scan_ok(pb) || b.cand_single || !b.thr) return hipErrorInvalidValue;
  const ScanArgs a = scan_args(pb, ps, b, MODE_THRESH, 1);
  const int64_t grid = ps.nc * a.wgs_per_chunk;
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  if (pb.causal) k_fused_scan<128, 3, 2, true, false, 0, true><<<(unsigned)grid, 256, 0, st>>>(a);
  else k_fused_scan<128, 3, 2, false, false, 0, true><<<(unsigned)grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_fused_scan(const Problem& pb, const Pass& ps, const PassBufs& b, const ScanCfg& cfg,
                             hipStream_t st) {
  ScanArgs a = scan_args(pb, ps, b, cfg.mode, cfg.stride);
  const int G = cfg.groups;
  const bool causal = pb.causal != 0;
  const unsigned grid = (unsigned)(ps.nc * a.wgs_per_chunk);
#define TOPK_SCAN(D_, G_, C_)                                                 \
  do {                                                                        \
    if (D_ == 64 && cfg.union_rank == 13) k_fused_scan<D_, 11, G_, C_, false, 13><<<grid, 256, 0, st>>>(a);      \
    else if (D_ == 64 && cfg.union_rank == 20) k_fused_scan<D_, 11, G_, C_, false, 20><<<grid, 256, 0, st>>>(a); \
    else if (D_ == 128 && cfg.R == 3) k_fused_scan<D_, 3, G_, C_><<<grid, 256, 0, st>>>(a);                      \
    else if (D_ == 128 && cfg.R == 6) k_fused_scan<D_, 6, G_, C_><<<grid, 256, 0, st>>>(a);                      \
    else k_fused_scan<D_, 12, G_, C_><<<grid, 256, 0, st>>>(a);                                                 \
  } while (0)
  // the instantiated sample rules (R, J): d = 64: (11, 13), (11, 20), (12, 0); d = 128:
  // (3, 0), (6, 0), (12, 0)
  const bool rule_ok = pb.d == 64 ? (cfg.R == 11 && (cfg.union_rank == 13 || cfg.union_rank == 20)) ||
                                        (cfg.R == 12 && cfg.union_rank == 0)
                                  : cfg.union_rank == 0 && (cfg.R == 3 || cfg.R == 6 || cfg.R == 12);
  if (G != 2 || (cfg.mode == MODE_SAMPLE && !rule_ok)) return hipErrorInvalidValue;
  if (cfg.score_only) {  // the ablation exists for the d = 64, 32 < k <= 64 sampled non-causal shape only
    if (pb.d != 64 || causal || cfg.mode != MODE_SAMPLE || cfg.union_rank != 20) return hipErrorInvalidValue;
    k_fused_scan<64, 11, 2, false, true, 20><<<grid, 256, 0, st>>>(a);
    return hipGetLastError();
  }
  if (pb.d == 64 && !causal) TOPK_SCAN(64, 2, false);
  else if (pb.d == 64) TOPK_SCAN(64, 2, true);
  else if (!causal) TOPK_SCAN(128, 2, false);
  else TOPK_SCAN(128, 2, true);
#undef TOPK_SCAN
  return hipGetLastError();
}

hipError_t launch_cand_select(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  if (b.caph > 512) k_cand_select<true><<<(unsigned)pass_rows(pb, ps), 64, 0, st>>>(pb, ps, b);
  else k_cand_select<false><<<(unsigned)pass_rows(pb, ps), 64, 0, st>>>(pb, ps, b);
  return hipGetLastError();
}

hipError_t launch_redo(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const size_t P8 = (size_t)pow2_at_least(pb.k) * 8;
  if (pb.dtype == T_BF16) {
    k_redo_scores<uint16_t><<<REDO_SCORE_BLOCKS, 256, 0, st>>>(pb, ps, b);
    k_redo_select<<<REDO_CAP, 256, P8, st>>>(pb, ps, b);
    k_redo_rest<uint16_t><<<REDO_BLOCKS, 256, P8, st>>>(pb, ps, b);
  } else {
    k_redo_scores<float><<<REDO_SCORE_BLOCKS, 256, 0, st>>>(pb, ps, b);
    k_redo_select<<<REDO_CAP, 256, P8, st>>>(pb, ps, b);
    k_redo_rest<float><<<REDO_BLOCKS, 256, P8, st>>>(pb, ps, b);
  }
  return hipGetLastError();
}

hipError_t launch_finalize(const Problem& pb, const Pass& ps, const PassBufs& b, hipStream_t st) {
  const size_t sh = (size_t)pb.k * 8;
  // value matrices larger than an L2: up to eight column slices, each a whole number of
  // 128-byte lines (a slice that split a line would fetch it on two XCDs), so each
  // XCD's L2 caches its slice of the matrix only
  const int64_t esz = pb.dtype == T_BF16 ? 2 : 4, row = pb.d * esz;
  int S = 1;
  if (pb.Lk * row > FINALIZE_SLICE_BYTES)
    for (int c = 8; c > 1 && S == 1; c >>= 1)
      if (row % (128 * c) == 0) S = c;
  const int64_t g = pass_rows(pb, ps) * S;
  if (g > 0x7FFFFFFF) return hipErrorInvalidValue;
#define TOPK_FINALIZE(T_)                                                                   \
  do {                                                                                      \
    if (S == 8) k_finalize<T_, 8><<<(unsigned)g, 64, sh, st>>>(pb, ps, b.sel);              \
    else if (S == 4) k_finalize<T_, 4><<<(unsigned)g, 64, sh, st>>>(pb, ps, b.sel);         \
    else if (S == 2) k_finalize<T_, 2><<<(unsigned)g, 64, sh, st>>>(pb, ps, b.sel);         \
    else k_finalize<T_, 1><<<(unsigned)g, 64, sh, st>>>(pb, ps, b.sel);                     \
  } while (0)
  if (pb.dtype == T_BF16) TOPK_FINALIZE(uint16_t);
  else TOPK_FINALIZE(float);
#undef TOPK_FINALIZE
  return hipGetLastError();
}

int64_t read_bad_indices() {
#ifdef TOPK_CHECK_INDICES
  unsigned long long h = 0, zero = 0;
  if (hipMemcpyFromSymbol(&h, HIP_SYMBOL(g_bad_indices), sizeof(h)) != hipSuccess) return -2;
  if (hipMemcpyToSymbol(HIP_SYMBOL(g_bad_indices), &zero, sizeof(zero)) != hipSuccess) return -2;
  return (int64_t)h;
#else
  return -1;
#endif
}

hipError_t launch_mfma_probe(int32_t* rows, int32_t* cols, hipStream_t st) {
  k_mfma_probe<<<1, 64, 0, st>>>(rows, cols);
  return hipGetLastError();
}


// ------------------------------------------------------------------ backward pass
// Input checkpointing (Section 2.2, "Input checkpointing", and the backward
// pseudo-code): the forward caches only its inputs and each row's selected keys
// with their raw scores. The backward pass recomputes the activation on the k
// survivors, backpropagates through it, and forms the three gradients by gathers,
// never an Lq x Lk matrix:
//  0. the pairs grouped by key into per-key lists (see the bucket kernels below;
//     heads of more than 2^19 keys use per-key atomic counters, steps 2-3);
//  1. k_bwd_rows (one wave per query row): d_top_actv[m] = d_out . V[j_m] for the
//     k selected keys; the activation (softmax with temperature, or ReLU)
//     recomputed from the cached scores and backpropagated to d_top_dots;
//     d_Q = sum_m d_top_dots[m] K[j_m]; each pair's (weight, score gradient) is
//     kept (on the atomic path its key's counter also gives the pair its place);
//  2. an exclusive scan of the per-key counts (k_bwd_scan_*);
//  3. k_bwd_fill: each pair's id into its key's list at that place;
//  4. k_bwd_keys (one wave per key): d_V[j] = sum weight * d_out[row] and
//     d_K[j] = sum score gradient * Q[row] over the key's list, in increasing pair
//     order (on the atomic path lists of up to 1024 pairs are sorted first). No
//     floating-point atomics: the sums do not depend on scheduling.

__global__ void k_bwd_zero(int32_t* p, int64_t n) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    p[e] = 0;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

// Rows are read in 16-byte chunks of EPC elements (8 bf16 or 4 fp32). G lanes (the
// smallest power of two >= the row's chunk count CH, at most 64) share one row, lane
// part = lane % G taking chunks part, part + G, ...; one wave step covers S = 64 / G
// rows. A lane holds NCL = ceil(CH / G) chunks: 1, 2 or 4 (d <= 1024).
template <typename T> struct RowChunks {
  static constexpr int EPC = 16 / (int)sizeof(T);
};

struct LaneMap {
  int CH, G, S, slot, part;
};
__device__ __forceinline__ LaneMap lane_map(int64_t d, int bytes, int lane) {
  LaneMap m;
  m.CH = (int)(d * bytes / 16);
  m.G = 1;
  while (m.G < m.CH && m.G < 64) m.G <<= 1;
  m.S = 64 / m.G;
  m.slot = lane / m.G;
  m.part = lane & (m.G - 1);
  return m;
}
inline int lane_chunks(int64_t d, int bytes) {  // NCL for the host's kernel choice
  const int64_t CH = d * bytes / 16;
  int64_t G = 1;
  while (G < CH && G < 64) G <<= 1;
  return (int)((CH + G - 1) / G);
}

// 16 raw bytes at element offset e of a row-major tensor of T
template <typename T> __device__ __forceinline__ uint4 load16(const void* base, int64_t e) {
  return *(const uint4*)((const T*)base + e);
}
template <typename T> __device__ __forceinline__ void unpack(const uint4& v, float (&x)[RowChunks<T>::EPC]);
template <> __device__ __forceinline__ void unpack<uint16_t>(const uint4& v, float (&x)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
template <> __device__ __forceinline__ void unpack<float>(const uint4& v, float (&x)[4]) {
  x[0] = __uint_as_float(v.x), x[1] = __uint_as_float(v.y), x[2] = __uint_as_float(v.z), x[3] = __uint_as_float(v.w);
}
template <typename T> __device__ __forceinline__ void store_chunk(void* base, int64_t e, const float (&x)[RowChunks<T>::EPC]);
template <> __device__ __forceinline__ void store_chunk<uint16_t>(void* base, int64_t e, const float (&x)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f32_to_bf16(x[2 * i]) | ((uint32_t)f32_to_bf16(x[2 * i + 1]) << 16);
  *(uint4*)((uint16_t*)base + e) = make_uint4(w[0], w[1], w[2], w[3]);
}
template <> __device__ __forceinline__ void store_chunk<float>(void* base, int64_t e, const float (&x)[4]) {
  *(float4*)((float*)base + e) = make_float4(x[0], x[1], x[2], x[3]);
}

// sum the S row slots' partial rows: afterwards every lane holds the total of its part
template <int NCL, int EPC>
__device__ __forceinline__ void slot_reduce(float (&acc)[NCL][EPC], const LaneMap& lm) {
  for (int off = lm.G; off < 64; off <<= 1) {
#pragma unroll
    for (int u = 0; u < NCL; ++u)
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[u][e] += __shfl_xor(acc[u][e], off, 64);
  }
}

// XCD-aware renumbering: the hardware deals workgroups round-robin over the 8 XCDs;
// with a grid that is a multiple of 8, each XCD runs a contiguous range of logical
// workgroups (neighbouring rows or keys of one head share that XCD's L2).
__device__ __forceinline__ int64_t xcd_workgroup() {
  const int64_t NG = gridDim.x, bid = blockIdx.x;
  return (NG % 8 == 0) ? (bid % 8) * (NG / 8) + bid / 8 : bid;
}

constexpr int BWD_UNROLL = 4;  // row steps whose gathers are in flight together

template <typename T, int NCL>
__global__ __launch_bounds__(256) void k_bwd_rows(BwdProblem bp, BwdBufs b) {
  constexpr int EPC = RowChunks<T>::EPC, U = BWD_UNROLL;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t r = xcd_workgroup() * 4 + wave;
  if (r >= bp.BH * bp.Lq) return;  // whole wave; the kernel syncs waves only
  const int64_t bh = r / bp.Lq, d = bp.d, k = bp.k;
  const int32_t* idx = bp.idx + r * k;
  const float* dots = bp.dots + r * k;
  float2* pair = b.pair + r * k;
  const int64_t kv0 = bh * bp.kv_head_stride;
  const bool softmax = bp.act == ACT_SOFTMAX;
  auto valid_key = [&](int32_t j) { return j >= 0 && (int64_t)j < bp.Lk; };
  const LaneMap lm = lane_map(d, (int)sizeof(T), lane);

  // this lane's chunks of d_out[r]
  float gout[NCL][EPC];
#pragma unroll
  for (int u = 0; u < NCL; ++u) {
    const int c = lm.part + lm.G * u;
    if (c < lm.CH) unpack<T>(load16<T>(bp.dout, r * d + (int64_t)c * EPC), gout[u]);
    else
#pragma unroll
      for (int e = 0; e < EPC; ++e) gout[u][e] = 0.f;
  }

  // pass 1: the softmax's maximum and normaliser over the survivors' cached scores
  float mx = -INFINITY, z = 0.f;
  if (softmax) {
    for (int64_t m = lane; m < k; m += 64)
      if (valid_key(idx[m])) mx = fmaxf(mx, dots[m]);
    mx = wave_max(mx);
    for (int64_t m = lane; m < k; m += 64)
      if (valid_key(idx[m])) z += __expf(bp.scale * (dots[m] - mx));
    z = wave_sum(z);
  }
  const float inv_z = softmax ? 1.f / z : 0.f;

  // pass 2: d_top_actv[m] = d_out . V[j_m]. 64 pairs at a time sit one per lane;
  // shuffles deal them to the row slots, U steps of gathers in flight together
  float gpart = 0.f;
  for (int64_t c0 = 0; c0 < k; c0 += 64) {
    const int32_t jl = c0 + lane < k ? idx[c0 + lane] : -1;
    const float sl = c0 + lane < k ? dots[c0 + lane] : 0.f;
    const int n = (int)(k - c0 < 64 ? k - c0 : 64);
    for (int e0 = 0; e0 < n; e0 += U * lm.S) {
      uint4 xv[U][NCL];
      int32_t jq[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int e = e0 + q * lm.S + lm.slot;
        jq[q] = __shfl(jl, e & 63, 64);
        // no branches around the gathers (see pass 3): skipped slots and lanes past the
        // row's last chunk read value row 0 / the last chunk, and their products are
        // discarded below
        const int64_t jr = e < n && valid_key(jq[q]) ? jq[q] : 0;
#pragma unroll
        for (int u = 0; u < NCL; ++u) {
          const int c = lm.part + lm.G * u < lm.CH ? lm.part + lm.G * u : lm.CH - 1;
          xv[q][u] = load16<T>(bp.V, kv0 + jr * d + (int64_t)c * EPC);
        }
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int e = e0 + q * lm.S + lm.slot;
        const bool ok = e < n && valid_key(jq[q]);
        float dw = 0.f;  // lanes past the last chunk add x * 0 (gout is 0 there)
#pragma unroll
        for (int u = 0; u < NCL; ++u) {
          float x[EPC];
          unpack<T>(xv[q][u], x);
#pragma unroll
          for (int t = 0; t < EPC; ++t) dw = fmaf(x[t], gout[u][t], dw);
        }
        for (int off = 1; off < lm.G; off <<= 1) dw += __shfl_xor(dw, off, 64);
        const float s = __shfl(sl, e & 63, 64);
        if (ok && lm.part == 0) {
          const float w = softmax ? __expf(bp.scale * (s - mx)) * inv_z : fmaxf(s, 0.f);
          pair[c0 + e] = make_float2(w, dw);
          gpart += w * dw;
        }
      }
    }
  }
  const float g = wave_sum(gpart);
  __threadfence_block();  // this wave's pair writes are visible to its own reads below

  // pass 3: d_top_dots and each pair's place among its key's pairs (one pair per
  // lane), then d_Q = sum_m d_top_dots[m] K[j_m] (pairs dealt to the row slots)
  float acc[NCL][EPC];
#pragma unroll
  for (int u = 0; u < NCL; ++u)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[u][e] = 0.f;
  for (int64_t c0 = 0; c0 < k; c0 += 64) {
    const int64_t m = c0 + lane;
    const int32_t jl = m < k ? idx[m] : -1;
    const bool okl = valid_key(jl);
    float dsl = 0.f;
    int32_t place = 0;
    if (okl) {
      const float2 wdw = pair[m];
      dsl = softmax ? bp.scale * wdw.x * (wdw.y - g) : (dots[m] > 0.f ? wdw.y : 0.f);
      pair[m] = make_float2(wdw.x, dsl);
      if (!b.L.bucketed) place = atomicAdd(&b.count[bh * bp.Lk + jl], 1);
    }
    const int32_t jg = okl && dsl != 0.f ? jl : -1;  // a zero score gradient adds nothing
    const int n = (int)(k - c0 < 64 ? k - c0 : 64);
    for (int e0 = 0; e0 < n; e0 += U * lm.S) {
      uint4 xk[U][NCL];
      int32_t jq[U];
      float dq[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int e = e0 + q * lm.S + lm.slot;
        jq[q] = __shfl(jg, e & 63, 64);
        dq[q] = __shfl(dsl, e & 63, 64);
        // no branch on the entry: skipped slots load key row 0 and are not summed
        // (a load under a data-dependent branch made the compiler wait for every
        // earlier load before it)
        const int64_t jr = e < n && jq[q] >= 0 ? jq[q] : 0;
#pragma unroll
        for (int u = 0; u < NCL; ++u) {
          // lanes past the row's last chunk read its last chunk; their sums are never stored
          const int c = lm.part + lm.G * u < lm.CH ? lm.part + lm.G * u : lm.CH - 1;
          xk[q][u] = load16<T>(bp.K, kv0 + jr * d + (int64_t)c * EPC);
        }
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        // skipped slots add 0 * (a finite key row): no branch, so every load above is
        // consumed on every path and none has to be waited for early
        const int e = e0 + q * lm.S + lm.slot;
        const float dqe = e < n && jq[q] >= 0 ? dq[q] : 0.f;
#pragma unroll
        for (int u = 0; u < NCL; ++u) {
          float x[EPC];
          unpack<T>(xk[q][u], x);
#pragma unroll
          for (int t = 0; t < EPC; ++t) acc[u][t] = fmaf(dqe, x[t], acc[u][t]);
        }
      }
    }
    if (okl && !b.L.bucketed) b.rank[r * k + m] = place;
  }
  slot_reduce(acc, lm);
  if (lm.slot == 0) {
#pragma unroll
    for (int u = 0; u < NCL; ++u) {
      const int c = lm.part + lm.G * u;
      if (c < lm.CH) store_chunk<T>(bp.dQ, r * d + (int64_t)c * EPC, acc[u]);
    }
  }
}

// exclusive scan, in place: 1024 elements per block, block totals to sums
__global__ __launch_bounds__(256) void k_bwd_scan_local(int32_t* a, int64_t n, int32_t* sums) {
  __shared__ uint32_t tmp[4];
  const int64_t base = (int64_t)blockIdx.x * 1024 + threadIdx.x * 4;
  uint32_t v[4], s = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = base + e < n ? (uint32_t)a[base + e] : 0u;
    s += v[e];
  }
  const uint32_t ex = team_excl_scan<256>(s, tmp);
  uint32_t run = ex;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (base + e < n) a[base + e] = (int32_t)run;
    run += v[e];
  }
  if (threadIdx.x == 255) sums[blockIdx.x] = (int32_t)run;
}

// exclusive scan of the nb block totals by one workgroup, 1024 at a time
__global__ __launch_bounds__(256) void k_bwd_scan_sums(int32_t* sums, int64_t nb) {
  __shared__ uint32_t tmp[4];
  __shared__ uint32_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t c0 = 0; c0 < nb; c0 += 1024) {
    const int64_t base = c0 + threadIdx.x * 4;
    uint32_t v[4], s = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = base + e < nb ? (uint32_t)sums[base + e] : 0u;
      s += v[e];
    }
    const uint32_t ex = team_excl_scan<256>(s, tmp);
    const uint32_t c = carry;
    uint32_t run = c + ex;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (base + e < nb) sums[base + e] = (int32_t)run;
      run += v[e];
    }
    __syncthreads();
    if (threadIdx.x == 255) carry = run;
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void k_bwd_scan_add(int32_t* a, int64_t n, const int32_t* sums) {
  const int64_t base = (int64_t)blockIdx.x * 1024 + threadIdx.x * 4;
  const int32_t add = sums[blockIdx.x];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (base + e < n) a[base + e] += add;
}

__global__ __launch_bounds__(256) void k_bwd_fill(BwdProblem bp, BwdBufs b) {
  // pair ids, rows * k and heads * keys are below 2^31 (checked by the host)
  const uint32_t npairs = (uint32_t)(bp.BH * bp.Lq * bp.k), per_head = (uint32_t)(bp.Lq * bp.k);
  for (uint32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < npairs; p += gridDim.x * blockDim.x) {
    const int32_t j = bp.idx[p];
    if (j < 0 || (int64_t)j >= bp.Lk) continue;
    const int64_t key = (int64_t)(p / per_head) * bp.Lk + j;
    b.list[b.count[key] + b.rank[p]] = (int32_t)p;
  }
}

// ---- per-key lists by a two-level stable bucket sort (heads of up to 2^19 keys)
// Level 1 groups each head's pairs by bucket (key >> shift): k_bwd_bucket_count
// counts every tile's pairs per bucket, a scan over (head, bucket, tile) gives each
// tile's run of every bucket, k_bwd_bucket_scatter places the tile's pairs in LDS
// grouped by bucket and writes the runs out. Level 2, k_bwd_bucket_lists (one
// workgroup per bucket), counts the bucket's pairs per key, writes the keys' list
// offsets, and places each pair in its key's list. Ranks within a wave come from
// ballots over the digit bits and pairs are taken in increasing order, so every
// list is in increasing pair order. One wave per workgroup: the order of its LDS
// updates is program order.

// lanes among `active` whose v agrees with this lane's v on the low `bits` bits
__device__ __forceinline__ uint64_t match_low_bits(uint32_t v, int bits, uint64_t active) {
  uint64_t peers = active;
  for (int t = 0; t < bits; ++t) {
    const bool bit = (v >> t) & 1u;
    const uint64_t bal = __ballot(bit);
    peers &= bit ? bal : ~bal;
  }
  return peers;
}
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ int digit_bits(int64_t n) {  // bits that tell apart 0 .. n - 1
  int t = 0;
  while ((int64_t(1) << t) < n) ++t;
  return t;
}
// exclusive scan of a[0 .. n) in LDS by one wave, plus `base`; returns the total
__device__ __forceinline__ uint32_t wave_excl_scan_lds(uint32_t* a, int n, uint32_t base) {
  const int lane = threadIdx.x & 63;
  uint32_t carry = base;
  for (int c0 = 0; c0 < n; c0 += 64) {
    const int i = c0 + lane;
    const uint32_t v = i < n ? a[i] : 0u;
    uint32_t x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    if (i < n) a[i] = carry + x - v;
    carry += __shfl(x, 63, 64);
  }
  wave_sync_lds();
  return carry;
}

constexpr int BK_WAVES = 4;                             // waves per bucket-pass workgroup
constexpr int BK_PER_LANE = BK_TILE / (64 * BK_WAVES);  // a wave's quarter of a tile, per lane
constexpr int BK_BATCH = 8;                             // chunks of 64 stage entries loaded together

__global__ __launch_bounds__(256) void k_bwd_bucket_count(BwdProblem bp, BwdLayout L, int32_t* hist) {
  __shared__ uint32_t cnt[BK_MAXB];
  const int tid = threadIdx.x;
  const int64_t head = blockIdx.x / L.tiles, t = blockIdx.x - head * L.tiles;
  const int64_t per_head = bp.Lq * bp.k, e_beg = t * BK_TILE;
  const int n = (int)(per_head - e_beg < BK_TILE ? per_head - e_beg : BK_TILE);
  const int32_t* idx = bp.idx + head * per_head + e_beg;
  int32_t jj[BK_PER_LANE];
#pragma unroll
  for (int u = 0; u < BK_PER_LANE; ++u) jj[u] = u * 256 + tid < n ? idx[u * 256 + tid] : -1;
  for (int i = tid; i < L.nb; i += 256) cnt[i] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < BK_PER_LANE; ++u)
    if (jj[u] >= 0 && (int64_t)jj[u] < bp.Lk) atomicAdd(&cnt[jj[u] >> L.shift], 1u);
  __syncthreads();
  for (int i = tid; i < L.nb; i += 256) hist[(head * L.nb + i) * L.tiles + t] = (int32_t)cnt[i];
  if (blockIdx.x == 0 && tid == 0) hist[L.nhist] = 0;
}

// stage entry: bits 0..30 pair id, 32..42 key within its bucket, 48..55 bucket.
// Wave w places the w-th quarter of the tile; its cursor in a bucket's run starts
// after the lower waves' pairs of that bucket, so the runs stay in pair order.
__global__ __launch_bounds__(256) void k_bwd_bucket_scatter(BwdProblem bp, BwdLayout L, const int32_t* off,
                                                            uint64_t* stage) {
  __shared__ uint32_t cur[BK_WAVES][BK_MAXB];  // per-wave counts, then per-wave cursors
  __shared__ uint32_t start[BK_MAXB];
  __shared__ int32_t gpos[BK_MAXB];
  __shared__ uint32_t tmp[4], nvalid_s;
  __shared__ uint64_t buf[BK_TILE];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t head = blockIdx.x / L.tiles, t = blockIdx.x - head * L.tiles;
  const int64_t per_head = bp.Lq * bp.k, e_beg = t * BK_TILE, p_beg = head * per_head + e_beg;
  const int n = (int)(per_head - e_beg < BK_TILE ? per_head - e_beg : BK_TILE);
  const int e_w = wave * (BK_TILE / BK_WAVES);
  int32_t jj[BK_PER_LANE];
#pragma unroll
  for (int u = 0; u < BK_PER_LANE; ++u) {
    const int e = e_w + u * 64 + lane;
    jj[u] = e < n ? bp.idx[p_beg + e] : -1;
  }
  for (int i = tid; i < BK_WAVES * BK_MAXB; i += 256) (&cur[0][0])[i] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < BK_PER_LANE; ++u)
    if (jj[u] >= 0 && (int64_t)jj[u] < bp.Lk) atomicAdd(&cur[wave][jj[u] >> L.shift], 1u);
  __syncthreads();
  // tile-local run starts (thread tid takes buckets BPT * tid ...) and each wave's
  // cursor in its run
  constexpr int BPT = BK_MAXB / 256;
  uint32_t tot[BPT], all = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    const int bk = tid * BPT + q;
    tot[q] = 0;
    if (bk < L.nb)
      for (int w = 0; w < BK_WAVES; ++w) tot[q] += cur[w][bk];
    all += tot[q];
  }
  uint32_t st = team_excl_scan<256>(all, tmp);
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    const int bk = tid * BPT + q;
    if (bk < L.nb) {
      start[bk] = st;
      gpos[bk] = off[(head * L.nb + bk) * L.tiles + t];
      uint32_t c = st;
      for (int w = 0; w < BK_WAVES; ++w) {
        const uint32_t x = cur[w][bk];
        cur[w][bk] = c;
        c += x;
      }
    }
    st += tot[q];
  }
  if (tid == 255) nvalid_s = st;
  __syncthreads();
  const int bbits = digit_bits(L.nb);
  const uint32_t kmask = (1u << L.shift) - 1u;
#pragma unroll
  for (int u = 0; u < BK_PER_LANE; ++u) {
    const int32_t j = jj[u];
    const bool ok = j >= 0 && (int64_t)j < bp.Lk;
    const uint32_t bk = ok ? (uint32_t)j >> L.shift : 0u;
    const uint64_t peers = match_low_bits(bk, bbits, __ballot(ok));
    const uint32_t prior = ok ? cur[wave][bk] : 0u;
    const uint32_t rank = lanes_below(peers);
    if (ok) {
      buf[prior + rank] = ((uint64_t)bk << 48) | ((uint64_t)((uint32_t)j & kmask) << 32) |
                          (uint64_t)(p_beg + e_w + u * 64 + lane);
      if (rank == 0) cur[wave][bk] = prior + (uint32_t)__popcll(peers);
    }
    wave_sync_lds();
  }
  __syncthreads();
  // write the runs: consecutive threads write consecutive entries of a run
  const uint32_t nvalid = nvalid_s;
  for (uint32_t i = tid; i < nvalid; i += 256) {
    const uint64_t v = buf[i];
    const uint32_t bk = (uint32_t)(v >> 48);
    stage[gpos[bk] + (i - start[bk])] = v;
  }
}

// One workgroup per bucket; wave w takes the w-th quarter of the bucket's pairs
// (cursors after the lower waves' pairs of each key, as in the scatter).
__global__ __launch_bounds__(256) void k_bwd_bucket_lists(BwdProblem bp, BwdLayout L, const int32_t* off,
                                                          const uint64_t* stage, BwdBufs b) {
  // [BK_WAVES][1 << shift] per-wave counts, then cursors; then up to lcap list entries
  extern __shared__ uint32_t cur[];
  __shared__ uint32_t tmp[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t head = blockIdx.x / L.nb, bk = blockIdx.x - head * L.nb, hb = head * L.nb + bk;
  const int32_t beg = off[hb * L.tiles], end = off[(hb + 1) * L.tiles];
  const int KB = 1 << L.shift;
  const int64_t key0 = bk * KB;
  const int nkb = (int)(bp.Lk - key0 < KB ? bp.Lk - key0 : KB);
  const uint32_t kmask = (uint32_t)KB - 1u;
  // a bucket whose lists fit in LDS is placed there and written out contiguously
  const bool staged = end - beg <= L.lcap;
  int32_t* lds_list = (int32_t*)(cur + (BK_WAVES << L.shift));
  const int32_t share = ((end - beg + BK_WAVES - 1) / BK_WAVES + 63) / 64 * 64;
  const int32_t wb = beg + wave * share, we = wb + share < end ? wb + share : end;
  uint32_t* wc = cur + wave * KB;
  for (int i = tid; i < BK_WAVES * KB; i += 256) cur[i] = 0;
  __syncthreads();
  // this wave's pairs per key; BK_BATCH chunks of loads in flight
  for (int32_t e0 = wb; e0 < we; e0 += 64 * BK_BATCH) {
    uint32_t kq[BK_BATCH];
    // loads without a branch (lanes past the end re-read the last entry), so that the
    // compiler issues all of them before the first wait
#pragma unroll
    for (int u = 0; u < BK_BATCH; ++u) {
      const int32_t e = e0 + u * 64 + lane;
      const uint32_t hi = (uint32_t)(stage[e < we ? e : we - 1] >> 32);
      kq[u] = e < we ? hi & kmask : 0xFFFFFFFFu;
    }
#pragma unroll
    for (int u = 0; u < BK_BATCH; ++u)
      if (kq[u] != 0xFFFFFFFFu) atomicAdd(&wc[kq[u]], 1u);
  }
  __syncthreads();
  // list starts (keys in order) and each wave's cursor; thread tid takes `per` keys
  const int per = (KB + 255) / 256, kq0 = tid * per;
  uint32_t tot = 0;
  for (int i = 0; i < per; ++i)
    if (kq0 + i < KB)
      for (int w = 0; w < BK_WAVES; ++w) tot += cur[w * KB + kq0 + i];
  uint32_t c = (uint32_t)beg + team_excl_scan<256>(tot, tmp);
  for (int i = 0; i < per; ++i) {
    const int key = kq0 + i;
    if (key < KB) {
      if (key < nkb) b.count[head * bp.Lk + key0 + key] = (int32_t)c;
      for (int w = 0; w < BK_WAVES; ++w) {
        const uint32_t x = cur[w * KB + key];
        cur[w * KB + key] = c;
        c += x;
      }
    }
  }
  if (hb == bp.BH * L.nb - 1 && tid == 0) b.count[bp.BH * bp.Lk] = end;
  __syncthreads();
  // each of this wave's pairs into its key's list, in increasing pair order
  for (int32_t e0 = wb; e0 < we; e0 += 64 * BK_BATCH) {
    uint64_t vq[BK_BATCH];
#pragma unroll
    for (int u = 0; u < BK_BATCH; ++u) {
      const int32_t e = e0 + u * 64 + lane;
      vq[u] = stage[e < we ? e : we - 1];  // lanes past the end: not ok below
    }
#pragma unroll
    for (int u = 0; u < BK_BATCH; ++u) {
      const bool ok = e0 + u * 64 + lane < we;
      const uint32_t key = (uint32_t)(vq[u] >> 32) & kmask;
      const uint64_t peers = match_low_bits(key, L.shift, __ballot(ok));
      const uint32_t prior = ok ? wc[key] : 0u;
      const uint32_t rank = lanes_below(peers);
      if (ok) {
        const int32_t p = (int32_t)(vq[u] & 0x7FFFFFFFull);
        if (staged) lds_list[prior + rank - (uint32_t)beg] = p;
        else b.list[prior + rank] = p;
        if (rank == 0) wc[key] = prior + (uint32_t)__popcll(peers);
      }
      wave_sync_lds();
    }
  }
  if (staged) {
    __syncthreads();
    for (int32_t i = tid; i < end - beg; i += 256) b.list[beg + i] = lds_list[i];
  }
}

// SORTED: the lists come from the atomic counters (unordered), and lists of up to 1024
// pairs are sorted first; the bucket-sorted lists need no sort, and their kernel then
// carries none of the sort's registers.
template <typename T, int NCL, bool SORTED>
__global__ __launch_bounds__(256) void k_bwd_keys(BwdProblem bp, BwdBufs b) {
  constexpr int EPC = RowChunks<T>::EPC, U = BWD_UNROLL;
  __shared__ int32_t lst[4][1024];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t key = xcd_workgroup() * 4 + wave;
  if (key >= bp.BH * bp.Lk) return;  // whole wave
  const int64_t bh = key / bp.Lk, j = key - bh * bp.Lk, d = bp.d;
  const uint32_t kk = (uint32_t)bp.k;
  const int32_t beg = b.count[key], n = b.count[key + 1] - beg;
  const LaneMap lm = lane_map(d, (int)sizeof(T), lane);
  float dv[NCL][EPC], dk[NCL][EPC];
#pragma unroll
  for (int u = 0; u < NCL; ++u)
#pragma unroll
    for (int e = 0; e < EPC; ++e) dv[u][e] = dk[u][e] = 0.f;
  // one listed pair per row slot: slot s sums entries s, s + S, ... of the list,
  // U steps of gathers in flight together
  auto accumulate = [&](auto get) {
    for (int e0 = 0; e0 < n; e0 += U * lm.S) {
      uint4 xo[U][NCL], xq[U][NCL];
      float2 c[U];
      // the U list entries first, then every gather, without branches (slots past the
      // list repeat its last entry and are skipped below): a wait for one entry inside
      // a branch became a wait for every gather issued before it
      int32_t pq[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int e = e0 + q * lm.S + lm.slot;
        pq[q] = get(e < n ? e : n - 1);
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int32_t p = pq[q];
        c[q] = b.pair[p];
        const int64_t row = (int64_t)((uint32_t)p / kk) * d;
#pragma unroll
        for (int u = 0; u < NCL; ++u) {
          const int ch = lm.part + lm.G * u;
          if (ch < lm.CH) {
            xo[q][u] = load16<T>(bp.dout, row + (int64_t)ch * EPC);
            xq[q][u] = load16<T>(bp.Q, row + (int64_t)ch * EPC);
          }
        }
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int e = e0 + q * lm.S + lm.slot;
        if (e < n) {
#pragma unroll
          for (int u = 0; u < NCL; ++u) {
            const int ch = lm.part + lm.G * u;
            if (ch < lm.CH) {
              float x[EPC], y[EPC];
              unpack<T>(xo[q][u], x);
              unpack<T>(xq[q][u], y);
#pragma unroll
              for (int t = 0; t < EPC; ++t) {
                dv[u][t] = fmaf(c[q].x, x[t], dv[u][t]);
                dk[u][t] = fmaf(c[q].y, y[t], dk[u][t]);
              }
            }
          }
        }
      }
    }
  };
  // increasing pair order: a fixed summation order whatever order the places took
  auto sorted = [&](auto tag) {
    constexpr int E = decltype(tag)::value;
    uint64_t r[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = e * 64 + lane;
      r[e] = i < n ? (uint64_t)(0xFFFFFFFFu - (uint32_t)b.list[beg + i]) : 0ull;
    }
    wave_sort_desc<E>(r);  // descending in 0xFFFFFFFF - p: ascending p
#pragma unroll
    for (int e = 0; e < E; ++e) lst[wave][e * 64 + lane] = (int32_t)(0xFFFFFFFFu - (uint32_t)r[e]);
    wave_sync_lds();
    accumulate([&](int e) { return lst[wave][e]; });
  };
  if (!SORTED) accumulate([&](int e) { return b.list[beg + e]; });
  else if (n <= 64) sorted(std::integral_constant<int, 1>{});
  else if (n <= 128) sorted(std::integral_constant<int, 2>{});
  else if (n <= 256) sorted(std::integral_constant<int, 4>{});
  else if (n <= 512) sorted(std::integral_constant<int, 8>{});
  else if (n <= 1024) sorted(std::integral_constant<int, 16>{});
  else accumulate([&](int e) { return b.list[beg + e]; });
  slot_reduce(dv, lm);
  slot_reduce(dk, lm);
  if (lm.slot == 0) {
    const int64_t o = bh * bp.kv_head_stride + j * d;
#pragma unroll
    for (int u = 0; u < NCL; ++u) {
      const int ch = lm.part + lm.G * u;
      if (ch < lm.CH) {
        store_chunk<T>(bp.dV, o + (int64_t)ch * EPC, dv[u]);
        store_chunk<T>(bp.dK, o + (int64_t)ch * EPC, dk[u]);
      }
    }
  }
}

// exclusive scan of a[0 .. n) in place; sums holds ceil(n / 1024) entries
static void scan_in_place(int32_t* a, int64_t n, int32_t* sums, hipStream_t st) {
  const int64_t nb = (n + 1023) / 1024;
  k_bwd_scan_local<<<(unsigned)nb, 256, 0, st>>>(a, n, sums);
  k_bwd_scan_sums<<<1, 256, 0, st>>>(sums, nb);
  k_bwd_scan_add<<<(unsigned)nb, 256, 0, st>>>(a, n, sums);
}

hipError_t launch_backward(const BwdProblem& bp, const BwdBufs& b, hipStream_t st) {
  const int64_t nkeys = bp.BH * bp.Lk, rows = bp.BH * bp.Lq, npairs = rows * bp.k;
  const BwdLayout& L = b.L;
  if (L.bucketed) {
    k_bwd_bucket_count<<<(unsigned)(bp.BH * L.tiles), 256, 0, st>>>(bp, L, b.hist);
    scan_in_place(b.hist, L.nhist + 1, b.block_sums, st);
    k_bwd_bucket_scatter<<<(unsigned)(bp.BH * L.tiles), 256, 0, st>>>(bp, L, b.hist, b.stage);
    k_bwd_bucket_lists<<<(unsigned)(bp.BH * L.nb), 256, BK_LIST_LDS, st>>>(bp, L, b.hist, b.stage, b);
  } else {
    k_bwd_zero<<<1024, 256, 0, st>>>(b.count, nkeys + 1);
  }
  // grids rounded up to a multiple of 8 for the XCD-aware renumbering
  const unsigned grid_rows = (unsigned)(((rows + 3) / 4 + 7) / 8 * 8);
  const unsigned grid_keys = (unsigned)(((nkeys + 3) / 4 + 7) / 8 * 8);
  const int ncl = lane_chunks(bp.d, bp.dtype == T_BF16 ? 2 : 4);
#define TOPK_BWD(KERNEL, GRID)                                                                  \
  if (bp.dtype == T_BF16 && ncl == 1) KERNEL<uint16_t, 1><<<GRID, 256, 0, st>>>(bp, b);          \
  else if (bp.dtype == T_BF16 && ncl == 2) KERNEL<uint16_t, 2><<<GRID, 256, 0, st>>>(bp, b);     \
  else if (bp.dtype == T_F32 && ncl == 1) KERNEL<float, 1><<<GRID, 256, 0, st>>>(bp, b);         \
  else if (bp.dtype == T_F32 && ncl == 2) KERNEL<float, 2><<<GRID, 256, 0, st>>>(bp, b);         \
  else if (bp.dtype == T_F32 && ncl == 4) KERNEL<float, 4><<<GRID, 256, 0, st>>>(bp, b);         \
  else return hipErrorInvalidValue;
  TOPK_BWD(k_bwd_rows, grid_rows)
  if (!L.bucketed) {
    scan_in_place(b.count, nkeys + 1, b.block_sums, st);
    const int64_t gf = (npairs + 255) / 256;
    k_bwd_fill<<<(unsigned)(gf < 65536 ? gf : 65536), 256, 0, st>>>(bp, b);
  }
#define TOPK_BWD_KEYS(SORTED)                                                                             \
  if (bp.dtype == T_BF16 && ncl == 1) k_bwd_keys<uint16_t, 1, SORTED><<<grid_keys, 256, 0, st>>>(bp, b);      \
  else if (bp.dtype == T_BF16 && ncl == 2) k_bwd_keys<uint16_t, 2, SORTED><<<grid_keys, 256, 0, st>>>(bp, b); \
  else if (bp.dtype == T_F32 && ncl == 1) k_bwd_keys<float, 1, SORTED><<<grid_keys, 256, 0, st>>>(bp, b);     \
  else if (bp.dtype == T_F32 && ncl == 2) k_bwd_keys<float, 2, SORTED><<<grid_keys, 256, 0, st>>>(bp, b);     \
  else if (bp.dtype == T_F32 && ncl == 4) k_bwd_keys<float, 4, SORTED><<<grid_keys, 256, 0, st>>>(bp, b);     \
  else return hipErrorInvalidValue;
  if (L.bucketed) {
    TOPK_BWD_KEYS(false)
  } else {
    TOPK_BWD_KEYS(true)
  }
#undef TOPK_BWD_KEYS
#undef TOPK_BWD
  return hipGetLastError();
}

}  // namespace topk
