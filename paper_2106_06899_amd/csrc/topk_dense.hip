// Query chunking with the top-k disabled: the paper's comparison baseline
// (Section 2.2, "Query chunking"; Section 3 compares top-k attention against it).
// Every valid key of a query contributes: out_i = sum_j softmax_j(scale * q_i.k_j) v_j
// (Eq. 1, with the causal mask of Eq. 2), the k = Lk fixed point of Eq. 4.
//
// gfx950 kernel, bf16 inputs, fp32 accumulation, d in {64, 128}: a streaming
// softmax over key tiles, so no [C, Lk] score tile is ever written. One workgroup
// = 4 waves x 32 queries of one query chunk of one head. Per 64-key tile:
//   * scores S^T = K Q^T by v_mfma_f32_32x32x16_bf16 (K tile from LDS as the A
//     operand, the wave's 32 queries in registers as B): lane l holds 16 keys'
//     scores of query l % 32 per 32-key block, keys 8*(v/4) + 4*(l/32) + v%4;
//   * the running row maximum and sum are per query (the two lanes of a query,
//     l and l + 32, exchange their maxima), the accumulator is rescaled when the
//     maximum grows;
//   * O^T += V^T P^T by the same MFMA: the B operand is the lane's own 8 softmax
//     weights of a 16-key step, in the order the score layout holds them, and the
//     A operand reads V^T from LDS in that same key order, so each lane keeps the
//     output rows (features) of its own query and rescales them alone.
// V tiles are transposed into LDS on the way in (V^T[feature][key], 8-byte key
// groups XOR-swizzled by feature row).
#include "topk_internal.h"

#include <math.h>

namespace topk {

typedef __bf16 dbf16x8 __attribute__((__vector_size__(16)));
typedef __bf16 dbf16x4 __attribute__((__vector_size__(8)));
typedef float df32x16 __attribute__((__vector_size__(64)));

#define DENSE_WAIT_VM(n) (((n) & 15) | (7 << 4) | (15 << 8) | (((n) >> 4) << 14))

constexpr int DN_KT = 64;   // keys per tile
constexpr int DN_QW = 32;   // queries per wave
constexpr int DN_QB = 4 * DN_QW;

struct DenseArgs {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  uint16_t* out;
  int64_t Lq, Lk, C, kv_head_stride;  // Lq: query rows per head in memory
  int64_t c0, nchunk, wgs_per_chunk;
  float scale_log2e;                  // scale * log2(e)
};

// LDS position (in bf16 units) of V^T[f][j] inside one tile buffer: row f holds the
// 64 keys of the tile; the 16 groups of 4 keys are permuted by (f & 15).
__device__ __forceinline__ int vt_pos(int f, int j) { return f * DN_KT + ((((j >> 2) ^ (f & 15))) << 2) + (j & 3); }

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void k_dense_attn(DenseArgs a) {
  constexpr int NS = D / 16;         // MFMA steps over the features (scores)
  constexpr int CH = 2 * D / 16;     // 16-byte parts per key row
  constexpr int TILEB = DN_KT * 2 * D;
  constexpr int LPW = TILEB / 1024 / 4;
  constexpr int NDB = D / 32;        // 32-feature blocks of the output
  constexpr int VLD = DN_KT * D / 8 / 256;  // 16-byte V loads per thread per tile
  __shared__ __attribute__((aligned(16))) unsigned char ks0[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char ks1[TILEB];
  __shared__ __attribute__((aligned(16))) uint16_t vt0[D * DN_KT];
  __shared__ __attribute__((aligned(16))) uint16_t vt1[D * DN_KT];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5, n = lane & 31;
  const int64_t NG = gridDim.x, bid = blockIdx.x;
  const int64_t wg = (NG % 8 == 0) ? (bid % 8) * (NG / 8) + bid / 8 : bid;
  const int64_t cl = wg / a.wgs_per_chunk, blk = wg - cl * a.wgs_per_chunk;
  const int64_t id = a.c0 + cl, bh = id / a.nchunk, c = id - bh * a.nchunk;
  const uint16_t* Kh = a.K + bh * a.kv_head_stride;
  const uint16_t* Vh = a.V + bh * a.kv_head_stride;
  const int64_t q_first = c * a.C + blk * DN_QB;
  int64_t q_last = c * a.C + (blk * DN_QB + DN_QB < a.C ? blk * DN_QB + DN_QB : a.C) - 1;
  q_last = q_last < a.Lq - 1 ? q_last : a.Lq - 1;
  const int64_t ntiles_all = (a.Lk + DN_KT - 1) / DN_KT;
  const int64_t ntiles = CAUSAL && q_last / DN_KT + 1 < ntiles_all ? q_last / DN_KT + 1 : ntiles_all;

  const int64_t local = blk * DN_QB + wave * DN_QW + n;  // the lane's query within the chunk
  const int64_t qi = c * a.C + local;                      // its index within the head
  const bool ok = local < a.C && qi < a.Lq;
  dbf16x8 b[NS];
  {
    const uint16_t* q = a.Q + (bh * a.Lq + (ok ? qi : 0)) * D + (D / 2) * half;
#pragma unroll
    for (int s = 0; s < NS; ++s) b[s] = ok ? *(const dbf16x8*)(q + 8 * s) : (dbf16x8){};
  }

  // K tile t -> LDS (direct loads, XOR swizzle of 16-byte parts as the fused scan);
  // rows past Lk load the last key, their scores are masked
  auto issue_k = [&](int64_t t, unsigned char* dst) {
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int cidx = (wave * LPW + j) * 64 + tid % 64, r = cidx / CH, p = (cidx % CH) ^ (r & 7);
      int64_t key = t * DN_KT + r;
      key = key < a.Lk ? key : a.Lk - 1;
      __builtin_amdgcn_global_load_lds((const void*)(Kh + key * D + p * 8),
                                       (__attribute__((address_space(3))) void*)&dst[(wave * LPW + j) * 1024], 16,
                                       0, 0);
    }
  };
  // V tile t -> registers (thread: key tid % 64, feature groups of 8)
  uint4 vreg[VLD];
  auto load_v = [&](int64_t t) {
    const int j = tid & 63;
    int64_t key = t * DN_KT + j;
    key = key < a.Lk ? key : a.Lk - 1;
#pragma unroll
    for (int e = 0; e < VLD; ++e) {
      const int f0 = ((tid >> 6) + 4 * e) * 8;
      vreg[e] = *(const uint4*)(Vh + key * D + f0);
    }
  };
  auto store_vt = [&](uint16_t* vt) {
    const int j = tid & 63;
#pragma unroll
    for (int e = 0; e < VLD; ++e) {
      const int f0 = ((tid >> 6) + 4 * e) * 8;
      const uint32_t w[4] = {vreg[e].x, vreg[e].y, vreg[e].z, vreg[e].w};
#pragma unroll
      for (int i = 0; i < 8; ++i) vt[vt_pos(f0 + i, j)] = (uint16_t)(w[i >> 1] >> (16 * (i & 1)));
    }
  };

  df32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) o[db] = (df32x16){};
  float m_run = -INFINITY, l_run = 0.f;
  const float cexp = a.scale_log2e;

  // scores of the 32-key block rb of tile t for the lane's query
  auto block_scores = [&](const unsigned char* kb, int rb) {
    const int r = rb * 32 + n;
    dbf16x8 av[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) av[s] = *(const dbf16x8*)(kb + (r * CH + ((half * NS + s) ^ (r & 7))) * 16);
    df32x16 acc = {};
#pragma unroll
    for (int s = 0; s < NS; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[s], b[s], acc, 0, 0, 0);
    return acc;
  };
  auto mask = [&](df32x16& acc, int64_t jb) {  // jb: key of register 0 of this lane
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t j = jb + 8 * (v >> 2) + (v & 3);
      if (j >= a.Lk || (CAUSAL && j > qi)) acc[v] = -INFINITY;
    }
  };
  auto tile = [&](int64_t t, const unsigned char* kb, const uint16_t* vt) {
    df32x16 s[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      s[rb] = block_scores(kb, rb);
      const int64_t jb = t * DN_KT + rb * 32 + 4 * half;
      if (t * DN_KT + DN_KT > a.Lk || (CAUSAL && t * DN_KT + DN_KT - 1 > q_first + wave * DN_QW)) mask(s[rb], jb);
    }
    // running maximum of the query (both of its lanes)
    float mt = s[0][0];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, s[rb][v]);
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;  // all keys masked so far: weights stay 0
    const float alpha = exp2f((m_run - m_use) * cexp);     // m_run = -inf -> 0
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
    const float off = m_use * cexp;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {  // the weights replace the scores
        s[rb][v] = exp2f(fmaf(s[rb][v], cexp, -off));
        l_run += s[rb][v];
      }
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        // B: the lane's 8 weights of keys 16 st + {4h..4h+3, 8+4h..8+4h+3} of the block
        dbf16x8 pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[rb][8 * st + e];
        const int k0 = rb * 32 + 16 * st + 4 * half;  // first key of each 4-key group
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const int f = db * 32 + n;  // A row: output feature
          const dbf16x4 lo = *(const dbf16x4*)(vt + vt_pos(f, k0));
          const dbf16x4 hi = *(const dbf16x4*)(vt + vt_pos(f, k0 + 8));
          const dbf16x8 av = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, o[db], 0, 0, 0);
        }
      }
    }
  };

  // Pipeline, one tile of lookahead: during tile t the loads of K tile t+1 (direct to
  // LDS) and of V tile t+2 (to registers) are in flight; V tile t+1 was written to
  // V^T LDS at the start of tile t. Loads are issued V first, then K, so that the
  // K tile can be awaited without waiting for the younger V loads.
  if (ntiles > 0) {
    load_v(0);
    issue_k(0, ks0);
    __builtin_amdgcn_s_waitcnt(DENSE_WAIT_VM(LPW));  // V tile 0 is in registers
    store_vt(vt0);
    if (ntiles > 1) load_v(1);
  }
  for (int64_t t = 0; t < ntiles; t += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t tt = t + u;
      if (tt >= ntiles) break;
      const unsigned char* kcur = u ? ks1 : ks0;
      unsigned char* knxt = u ? ks0 : ks1;
      const uint16_t* vcur = u ? vt1 : vt0;
      uint16_t* vnxt = u ? vt0 : vt1;
      // in flight: K tile tt, then V tile tt+1 (if any); wait for K tile tt
      if (tt + 1 < ntiles) __builtin_amdgcn_s_waitcnt(DENSE_WAIT_VM(VLD));
      else __builtin_amdgcn_s_waitcnt(DENSE_WAIT_VM(0));
      // publishes every wave's K tile tt parts and V^T tile tt stores, and ends every
      // wave's reads of tile tt-1, whose buffers are refilled below
      __syncthreads();
      if (tt + 1 < ntiles) {
        __builtin_amdgcn_s_waitcnt(DENSE_WAIT_VM(0));  // V tile tt+1 is in registers
        store_vt(vnxt);
        if (tt + 2 < ntiles) load_v(tt + 2);
        issue_k(tt + 1, knxt);
      }
      tile(tt, kcur, vcur);
    }
  }
  if (!ok) return;
  const float l = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l > 0.f ? 1.f / l : 0.f;
  uint16_t* dst = a.out + (bh * a.Lq + qi) * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      // features db*32 + 8g + 4h .. +3 of the lane's query
      dbf16x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (__bf16)(o[db][4 * g + e] * inv);
      *(dbf16x4*)(dst + db * 32 + 8 * g + 4 * half) = w;
    }
}

hipError_t launch_dense(const Problem& pb, const Pass& ps, hipStream_t st) {
  DenseArgs a;
  a.Q = (const uint16_t*)pb.Q;
  a.K = (const uint16_t*)pb.K;
  a.V = (const uint16_t*)pb.V;
  a.out = (uint16_t*)pb.out;
  a.Lq = pb.Lq;
  a.Lk = pb.Lk;
  a.C = pb.C;
  a.kv_head_stride = pb.kv_head_stride;
  a.c0 = ps.c0;
  a.nchunk = ps.nchunk;
  a.wgs_per_chunk = (pb.C + DN_QB - 1) / DN_QB;
  a.scale_log2e = pb.scale * 1.4426950408889634f;
  const int64_t g = ps.nc * a.wgs_per_chunk;
  if (g > 0x7FFFFFFF) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)g;
  if (pb.d == 64 && !pb.causal) k_dense_attn<64, false><<<grid, 256, 0, st>>>(a);
  else if (pb.d == 64) k_dense_attn<64, true><<<grid, 256, 0, st>>>(a);
  else if (pb.d == 128 && !pb.causal) k_dense_attn<128, false><<<grid, 256, 0, st>>>(a);
  else if (pb.d == 128) k_dense_attn<128, true><<<grid, 256, 0, st>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace topk
