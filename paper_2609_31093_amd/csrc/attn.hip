// Selected sparse attention (Sec. 3.1 eq. selected_sparse_attention; App. B
// masks future tokens inside the selected blocks).
//
// attn_rows_kernel: a team (one wavefront, or a 256-thread workgroup for few
// rows) owns one (query row, query head).  Its 16-lane groups stride over the
// selected tokens; each group keeps an online softmax state (running max,
// running sum, running output slice) in registers, 16-byte loads bring one key
// row and one value row per group, and the groups' states are merged at the
// end.  Outputs: o in the input dtype (round to nearest even for bf16), lse in
// natural log.
#include <algorithm>
#include <atomic>

#include "common.h"
#include "kernels.h"

namespace pisa {

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* idx;
  void* o;
  float* lse;
  int H, Hkv, G, Nq, N, C, K, causal;
  float qscale2;
  int Nkv;  // rows per (batch, KV head) in k and v
};

template <typename T, int DPL>
__device__ __forceinline__ void store_row_part(T* p, const float (&x)[DPL]);

template <>
__device__ __forceinline__ void store_row_part<uint16_t, 8>(uint16_t* p, const float (&x)[8]) {
  uint4 r;
  r.x = pack2_bf16(x[0], x[1]);
  r.y = pack2_bf16(x[2], x[3]);
  r.z = pack2_bf16(x[4], x[5]);
  r.w = pack2_bf16(x[6], x[7]);
  *reinterpret_cast<uint4*>(p) = r;
}
template <>
__device__ __forceinline__ void store_row_part<uint16_t, 4>(uint16_t* p, const float (&x)[4]) {
  uint2 r;
  r.x = pack2_bf16(x[0], x[1]);
  r.y = pack2_bf16(x[2], x[3]);
  *reinterpret_cast<uint2*>(p) = r;
}
template <>
__device__ __forceinline__ void store_row_part<float, 8>(float* p, const float (&x)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
template <>
__device__ __forceinline__ void store_row_part<float, 4>(float* p, const float (&x)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}

template <int DPL>
__device__ __forceinline__ void merge_state(float& m, float& s, float (&o)[DPL], float m2, float s2,
                                            const float (&o2)[DPL]) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  const float a1 = fast_exp2(m - mn), a2 = fast_exp2(m2 - mn);
  s = s * a1 + s2 * a2;
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = o[e] * a1 + o2[e] * a2;
  m = mn;
}

template <typename T, int D, int TEAM>
__global__ __launch_bounds__(256) void attn_rows_kernel(AttnArgs a) {
  constexpr int DPL = D / 16;
  constexpr int NGRP = TEAM / 16;
  constexpr int ROWS = 256 / TEAM;
  constexpr int NW = TEAM / 64;
  __shared__ float red[ROWS][NW][2 + D];

  const int team = threadIdx.x / TEAM;
  const int tid = threadIdx.x % TEAM;
  const int lane = threadIdx.x & 63;
  const int wave_in_team = tid >> 6;
  const int grp = tid >> 4;
  const int sub = tid & 15;
  const int row = blockIdx.x * ROWS + team;
  if (row >= a.Nq) return;
  const int hq = blockIdx.y % a.H;
  const int b = blockIdx.y / a.H;
  const int hk = hq / a.G;
  const int bh = b * a.Hkv + hk;
  const int t = a.N - a.Nq + row;

  float qv[DPL];
  const T* qp = static_cast<const T*>(a.q) + ((static_cast<int64_t>(b) * a.H + hq) * a.Nq + row) * D + sub * DPL;
  load_row_part<T, DPL>(qp, qv);
#pragma unroll
  for (int e = 0; e < DPL; ++e) qv[e] *= a.qscale2;

  const T* kb = static_cast<const T*>(a.k) + static_cast<int64_t>(bh) * a.Nkv * D + sub * DPL;
  const T* vb = static_cast<const T*>(a.v) + static_cast<int64_t>(bh) * a.Nkv * D + sub * DPL;
  const int32_t* sel = a.idx + (static_cast<int64_t>(bh) * a.Nq + row) * a.K;

  float m = -INFINITY, s = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;

  const int total = a.K * a.C;
  const int nblk = (a.N + a.C - 1) / a.C;
  for (int i = grp; i < total; i += NGRP) {
    const int slot = i / a.C;
    const int blk = sel[slot];
    if (blk < 0 || blk >= nblk) continue;  // padding
    const int tok = blk * a.C + (i - slot * a.C);
    if (tok >= a.N || (a.causal && tok > t)) continue;
    float x[DPL], y[DPL];
    load_row_part<T, DPL>(kb + static_cast<int64_t>(tok) * D, x);
    load_row_part<T, DPL>(vb + static_cast<int64_t>(tok) * D, y);
    float z = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) z = fmaf(qv[e], x[e], z);
    z = sum16(z);
    const float mn = fmaxf(m, z);
    const float corr = fast_exp2(m - mn);
    const float p = fast_exp2(z - mn);
    s = s * corr + p;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] = fmaf(p, y[e], o[e] * corr);
    m = mn;
  }
  // Merge the four lane groups of each wavefront.
#pragma unroll
  for (int msk = 16; msk <= 32; msk <<= 1) {
    float o2[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) o2[e] = __shfl_xor(o[e], msk);
    const float m2 = __shfl_xor(m, msk), s2 = __shfl_xor(s, msk);
    merge_state<DPL>(m, s, o, m2, s2, o2);
  }
  if constexpr (NW > 1) {
    if (lane < 16) {
      if (lane == 0) {
        red[team][wave_in_team][0] = m;
        red[team][wave_in_team][1] = s;
      }
#pragma unroll
      for (int e = 0; e < DPL; ++e) red[team][wave_in_team][2 + sub * DPL + e] = o[e];
    }
    __syncthreads();
    if (wave_in_team != 0) return;
    for (int w = 1; w < NW; ++w) {
      float o2[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) o2[e] = red[team][w][2 + sub * DPL + e];
      merge_state<DPL>(m, s, o, red[team][w][0], red[team][w][1], o2);
    }
  }
  if (lane < 16) {
    const int64_t orow = (static_cast<int64_t>(b) * a.H + hq) * a.Nq + row;
    float res[DPL];
    const float inv = s > 0.f ? 1.0f / s : 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) res[e] = o[e] * inv;
    store_row_part<T, DPL>(static_cast<T*>(a.o) + orow * D + sub * DPL, res);
    if (a.lse && lane == 0) a.lse[orow] = s > 0.f ? (m + fast_log2(s)) * kLn2 : -INFINITY;
  }
}


// ----------------------------------------------------------------------------
// Block-centric attention for many rows (bf16).
//
// attn_block16_kernel: one workgroup per chunk of up to kAttnChunk (row,
// slot) pairs of one (batch x KV head, key block) cluster, taken as
// kClusterTile-pair tiles.  The block's C
// keys are staged in LDS row-major and its values transposed (V^T, two keys
// per 32-bit word, so that the PV product reads contiguous 8-byte runs);
// the pairs are processed 16 per wavefront tile on v_mfma_f32_16x16x32_bf16
// (A lane l: row l%16, k 8*(l/16)..+7; B lane l: k 8*(l/16)..+7, column
// l%16; D lane l: rows 4*(l/16)..+3, column l%16): S^T = K q^T (keys along
// M, queries along N), the causal mask, the block-local max, P = 2^(S - m)
// in bf16, then O^T = V^T P with the key order of P's operand reproduced in
// the V^T reads.  Each pair leaves a partial: o normalised by its own sum
// (bf16) and its log2-sum (fp32).  attn_local_kernel (causal) or
// attn_combine_kernel merges the partials of each (row, head) with the usual
// log-sum-exp weights.
// ----------------------------------------------------------------------------

typedef __bf16 bf16x8a __attribute__((ext_vector_type(8)));
typedef float f32x4a __attribute__((ext_vector_type(4)));

struct AttnBlockArgs {
  int H, Hkv, G, Nq, N, C, K, causal, M1;
  int row0, nrows;  // row chunk handled by this launch
  float qscale2;
  int Nkv;          // rows per (batch, KV head) in k and v
  // rows attended by the row-tile union kernel (flag per tile of
  // 1 << skip_shift rows); the block-centric kernels leave them alone
  const uint8_t* skip = nullptr;
  int skip_shift = 0, skip_tiles = 0;
};

__device__ __forceinline__ bool union_row(const AttnBlockArgs& a, int bh, int row) {
  return a.skip && a.skip[static_cast<int64_t>(bh) * a.skip_tiles + (row >> a.skip_shift)];
}

__device__ __forceinline__ bf16x8a u4_as_bf16x8(uint4 r) { return __builtin_bit_cast(bf16x8a, r); }

constexpr int kAttnChunk = 1024;  // pairs of one selected-block cluster per workgroup (key block staged once)
constexpr int kAttnBlockWaves = 8;  // wavefronts per workgroup of attn_block16_kernel

template <int D, int CT, int NW>
__global__ __launch_bounds__(NW * 64, (CT >= 3 ? 1 : NW == 8 ? 4 : 3)) void attn_block16_kernel(AttnBlockArgs a, const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ offs,
                                                           const int32_t* __restrict__ toffs, int64_t ncl,
                                                           const int32_t* __restrict__ pairs,
                                                           uint16_t* __restrict__ part_o,
                                                           float* __restrict__ part_lse) {
  constexpr int KS = D / 32;       // k-steps of QK^T (32 dims each)
  constexpr int LDK = D + 8;       // padded K row (bf16 elements)
  constexpr int C = CT * 32;       // keys per block
  constexpr int MT = C / 16;       // 16-key tiles of S
  constexpr int LDV = C + 4;       // padded V^T row
  constexpr int DT = D / 16;       // 16-row d tiles of O
  constexpr int TBS = D + 8;       // padded row of the partial transposition buffer
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* klds = lds;
  uint16_t* vt = lds + C * LDK;
  uint32_t* vt32 = reinterpret_cast<uint32_t*>(vt);
  uint16_t* tbuf = vt + D * LDV;   // [NW wavefronts][16][TBS]
  constexpr int NT = 16 / NW;      // 16-pair tiles of a 256-pair tile per wavefront

  int64_t cl;
  int cbeg, cend;
  if (!cluster_chunk(offs, toffs, ncl, blockIdx.x, kAttnChunk, cl, cbeg, cend)) return;
  const int bh = static_cast<int>(cl / a.M1);
  const int blk = static_cast<int>(cl - static_cast<int64_t>(bh) * a.M1);
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = blk * C;
  const int nkeys = min(C, a.N - r0);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;   // query column
  const int grp = lane >> 4;   // 0..3: k slice of the operands, row group of the results

  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  const uint16_t* vb = v + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  for (int e = threadIdx.x; e < C * (D / 8); e += NW * 64) {
    const int r = e / (D / 8), c8 = (e - r * (D / 8)) * 8;
    uint4 kv = make_uint4(0, 0, 0, 0);
    if (r < nkeys) kv = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D + c8);
    *reinterpret_cast<uint4*>(klds + r * LDK + c8) = kv;
  }
  for (int e = threadIdx.x; e < (C / 2) * (D / 8); e += NW * 64) {
    const int kp = e % (C / 2), c8 = (e / (C / 2)) * 8;
    uint4 v0 = make_uint4(0, 0, 0, 0), v1 = make_uint4(0, 0, 0, 0);
    if (2 * kp < nkeys) v0 = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(2 * kp) * D + c8);
    if (2 * kp + 1 < nkeys) v1 = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(2 * kp + 1) * D + c8);
    const uint32_t w0[4] = {v0.x, v0.y, v0.z, v0.w};
    const uint32_t w1[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      vt32[(c8 + 2 * i) * (LDV / 2) + kp] = (w0[i] & 0xFFFFu) | (w1[i] << 16);
      vt32[(c8 + 2 * i + 1) * (LDV / 2) + kp] = (w0[i] >> 16) | (w1[i] & 0xFFFF0000u);
    }
  }
  __syncthreads();

  // The chunk's pairs in 256-pair tiles.  This wavefront's 16-pair tiles of
  // a tile are wave, wave + NW, ... (at most NT); iteration it covers tile
  // it / G and query head it % G.  The pair words of all of them are read up
  // front, and the query operand of the next iteration is gathered while the
  // current one computes.
  static_assert(kClusterTile == 256 && NT * NW == 16, "sixteen 16-pair tiles per 256-pair tile");
  for (int beg = cbeg; beg < cend; beg += kClusterTile) {
  const int end = min(cend, beg + kClusterTile);
  const int ntile = (end - beg + 15) / 16;
  const int nmine = ntile > wave ? (ntile - wave + NW - 1) / NW : 0;
  const int nit = nmine * a.G;
  int prw[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int p = beg + (wave + NW * j) * 16 + col;
    prw[j] = (j < nmine && p < end) ? pairs[p] : -1;
  }
  auto pair_of = [&](int j) {
    if constexpr (NT == 4) {
      return j == 0 ? prw[0] : j == 1 ? prw[1] : j == 2 ? prw[2] : prw[3];
    } else {
      int r = prw[0];
#pragma unroll
      for (int jj = 1; jj < NT; ++jj) r = j == jj ? prw[jj] : r;
      return r;
    }
  };
  auto gather = [&](int it, bf16x8a (&dst)[KS]) {
    const int j = it / a.G, hh = it - j * a.G;
    const int pr = pair_of(j);
    const int row = a.row0 + (pr >= 0 ? (pr >> 8) : 0);
    const uint16_t* qrow = q + ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + row) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (pr >= 0) u = *reinterpret_cast<const uint4*>(qrow + ks * 32);
      dst[ks] = u4_as_bf16x8(u);
    }
  };
  bf16x8a qn[KS];
  if (nit > 0) gather(0, qn);

  for (int it = 0; it < nit; ++it) {
    bf16x8a qb[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qb[ks] = qn[ks];
    if (it + 1 < nit) gather(it + 1, qn);
    const int j = it / a.G, hh = it - j * a.G;
    const int pr = pair_of(j);
    const bool valid = pr >= 0;
    const int rr = valid ? pr >> 8 : 0, slot = pr & 255;
    const int row = a.row0 + rr;
    const int t = a.N - a.Nq + row;
    const int kmax = a.causal ? min(nkeys, t - r0 + 1) : nkeys;
    {
      // S^T tile mt holds the logits of keys mt*16 + 4*grp + i (i = 0..3) of
      // query `col`; keys at or past the query's causal limit become -inf.
      // Blocks of up to 64 keys keep their S tiles in registers (raw logits;
      // the causal mask applied only when some pair of the tile needs it, the
      // scale folded into the exponent); larger blocks recompute the scaled,
      // masked tiles in the second pass.
      constexpr bool kKeepS = MT <= 4;
      const bool masked = !kKeepS || __ballot(kmax < C) != 0;
      const float sscale = kKeepS ? 1.f : a.qscale2;
      auto s_tile = [&](int mt) {
        f32x4a acc = {0.f, 0.f, 0.f, 0.f};
        const uint16_t* arow = klds + (mt * 16 + col) * LDK + grp * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8a av = u4_as_bf16x8(*reinterpret_cast<const uint4*>(arow + ks * 32));
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qb[ks], acc, 0, 0, 0);
        }
        if (masked) {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = mt * 16 + 4 * grp + i < kmax ? acc[i] * sscale : -INFINITY;
        }
        return acc;
      };
      // The block-local maximum m (scaled, log2 units), then P = 2^(S - m)
      // per 32-key step and O^T += V^T P.  The P operand k = 8*grp + i holds
      // key 32s + 4*grp + i (i < 4) or 32s + 16 + 4*grp + (i - 4) (i >= 4);
      // the V^T operand reads the same keys.
      f32x4a st[kKeepS ? MT : 1];
      float m = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const f32x4a sa = s_tile(mt);
        if constexpr (kKeepS) st[mt] = sa;
        m = fmaxf(m, fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])));
      }
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      const float msafe = (m == -INFINITY) ? 0.f : (kKeepS ? m * a.qscale2 : m);
      m = msafe;
      if constexpr (!kKeepS) asm volatile("" ::: "memory");  // recompute rather than hold the tiles
      const float pscale = kKeepS ? a.qscale2 : 1.f;
      f32x4a oacc[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4a{0.f, 0.f, 0.f, 0.f};
      float l = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < MT / 2; ++s2) {
        f32x4a sa, sb;
        if constexpr (kKeepS) {
          sa = st[2 * s2];
          sb = st[2 * s2 + 1];
        } else {
          sa = s_tile(2 * s2);
          sb = s_tile(2 * s2 + 1);
        }
        float pv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pv[i] = fast_exp2(fmaf(sa[i], pscale, -msafe));
          pv[4 + i] = fast_exp2(fmaf(sb[i], pscale, -msafe));
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) l += pv[i];
        uint4 u;
        u.x = pack2_bf16(pv[0], pv[1]);
        u.y = pack2_bf16(pv[2], pv[3]);
        u.z = pack2_bf16(pv[4], pv[5]);
        u.w = pack2_bf16(pv[6], pv[7]);
        const bf16x8a pb = u4_as_bf16x8(u);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const uint16_t* vrow = vt + (dt * 16 + col) * LDV + 4 * grp + 32 * s2;
          const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
          const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
          const bf16x8a av = u4_as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
          oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb, oacc[dt], 0, 0, 0);
        }
      }
      l += __shfl_xor(l, 16);
      l += __shfl_xor(l, 32);
      const float inv = l > 0.f ? 1.0f / l : 0.f;
      const int64_t pidx = ((static_cast<int64_t>(bh) * a.nrows + rr) * a.K + slot) * a.G + hh;
      // oacc[dt][i] = O[d = dt*16 + 4*grp + i][query col]: the tile's 16
      // partial rows go through LDS so that each store writes whole rows
      // (16 lanes x 16 bytes per row, four rows per instruction).
      uint16_t* tb = tbuf + wave * (16 * TBS);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        uint2 w;
        w.x = pack2_bf16(oacc[dt][0] * inv, oacc[dt][1] * inv);
        w.y = pack2_bf16(oacc[dt][2] * inv, oacc[dt][3] * inv);
        *reinterpret_cast<uint2*>(tb + col * TBS + dt * 16 + 4 * grp) = w;
      }
      if (valid && grp == 0) part_lse[pidx] = l > 0.f ? m + fast_log2(l) : -INFINITY;
      wave_sync();
#pragma unroll
      for (int j = 0; j < 16 * D / 8 / 64; ++j) {
        const int e = j * 64 + lane;           // 16-byte chunk of the tile
        const int r = e / (D / 8), c8 = (e - r * (D / 8)) * 8;
        const int64_t pr_idx = __shfl(pidx, r);  // lane r (grp 0) holds column r's pair
        const bool pv_ok = __shfl(static_cast<int>(valid), r) != 0;
        const uint4 u = *reinterpret_cast<const uint4*>(tb + r * TBS + c8);
        if (pv_ok) *reinterpret_cast<uint4*>(part_o + pr_idx * D + c8) = u;
      }
      wave_sync();
    }
  }
  }
}

// ----------------------------------------------------------------------------
// Causal attention over the blocks that every row of a leaf block selects by
// construction (App. B: the first block, the previous one and the row's own),
// for all rows of that leaf block at once, merged with the partials that
// attn_block16_kernel left for each row's other selected blocks.
//
// One workgroup per (batch x KV head, query leaf block c).  For each query
// head and each of the distinct blocks {0, c-1, c}, the block is staged in
// LDS as in attn_block16_kernel and every wavefront advances an online
// softmax for 16 query rows on v_mfma_f32_16x16x32_bf16 (S^T = K q^T, the
// causal mask, O^T += V^T P); a block enters a row's sum only if it is in
// that row's index list.  The wavefront then folds in the row's partials of
// its other slots (o normalised by its own sum, log2-sum) and writes o (bf16)
// and lse (natural log).  The rows' shared blocks never become partials, and
// each is read once per leaf block instead of once per row.
// ----------------------------------------------------------------------------
constexpr int kMergeBatch = 4;  // partials of a row requested together by attn_local_kernel

// NWL wavefronts per workgroup, each owning 16-row query groups NWL apart.
template <int D, int CT, int NWL>
__global__ __launch_bounds__(NWL * 64, NWL == 8 ? 2 : 3) void attn_local_kernel(AttnBlockArgs a, const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ k,
                                                         const uint16_t* __restrict__ v,
                                                         const int32_t* __restrict__ idx,
                                                         const uint16_t* __restrict__ part_o,
                                                         const float* __restrict__ part_lse,
                                                         uint16_t* __restrict__ o, float* __restrict__ lse) {
  constexpr int KS = D / 32;
  constexpr int LDK = D + 8;
  constexpr int C = CT * 32;
  constexpr int MT = C / 16;
  constexpr int LDV = C + 4;
  constexpr int DT = D / 16;
  constexpr int QG = C / 16;             // 16-row query groups of a leaf block
  constexpr int NPASS = (QG + NWL - 1) / NWL;  // groups per wavefront
  constexpr int DPL = D / 16;            // merge: elements per lane
  constexpr int SROW = D + 4;            // merge: padded state row (floats)
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* klds = lds;
  uint16_t* vt = lds + C * LDK;
  uint32_t* vt32 = reinterpret_cast<uint32_t*>(vt);

  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int tq0 = a.N - a.Nq;  // absolute position of query row 0
  const int c = (tq0 + a.row0) / C + static_cast<int>(blockIdx.x);
  const int p_lo = max(c * C, tq0 + a.row0), p_hi = min((c + 1) * C, tq0 + a.row0 + a.nrows);
  if (p_lo >= p_hi) return;
  // rows attended by the row-tile union kernel: bit t - t_lo of umask for
  // the block's tiles t_lo.. (at most C / 16 + 1 <= 9 of them)
  uint32_t umask = 0;
  int t_lo = 0;
  if (a.skip) {
    t_lo = (p_lo - tq0) >> a.skip_shift;
    const int t_hi = (p_hi - 1 - tq0) >> a.skip_shift;
    for (int t = t_lo; t <= t_hi; ++t)
      umask |= (a.skip[static_cast<int64_t>(bh) * a.skip_tiles + t] ? 1u : 0u) << (t - t_lo);
    if (umask == (2u << (t_hi - t_lo)) - 1u) return;  // every row of the block
  }
  auto urow = [&](int row) { return ((umask >> ((row >> a.skip_shift) - t_lo)) & 1u) != 0u; };
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  int sb[3];
  int nsb = 0;
  sb[nsb++] = 0;
  if (c - 1 > 0) sb[nsb++] = c - 1;
  if (c > 0) sb[nsb++] = c;

  for (int it = 0; it < NPASS * a.G; ++it) {
    const int hh = it / NPASS, qg = (it - hh * NPASS) * NWL + wave;
    const int p = c * C + qg * 16 + col;  // this lane's query position
    const bool vq = qg < QG && p >= p_lo && p < p_hi && !urow(p - tq0);
    const int rowq = vq ? p - tq0 : p_lo - tq0;  // a row of the tile for lanes without a query
    const int32_t* sel = idx + (static_cast<int64_t>(bh) * a.Nq + rowq) * a.K;
    // which shared blocks this row selected (each of the 4 lanes of a column
    // reads a quarter of the list)
    int has = 0;
    for (int s = grp; s < a.K; s += 4) {
      const int x = sel[s];
      has |= (x == 0 ? 1 : 0) | (x == c - 1 && c - 1 > 0 ? 2 : 0) | (x == c && c > 0 ? 4 : 0);
    }
    has |= __shfl_xor(has, 16);
    has |= __shfl_xor(has, 32);
    bf16x8a qb[KS];
    {
      const uint16_t* qrow = q + ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + rowq) * D + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qb[ks] = u4_as_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 32));
    }
    float m = -INFINITY, l = 0.f;
    f32x4a oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4a{0.f, 0.f, 0.f, 0.f};

    for (int j = 0; j < nsb; ++j) {
      const int blk = sb[j];
      const int r0 = blk * C;
      const int nkeys = min(C, a.N - r0);
      __syncthreads();  // the previous block's readers are done
      const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
      const uint16_t* vb = v + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
      for (int e = threadIdx.x; e < C * (D / 8); e += NWL * 64) {
        const int r = e / (D / 8), c8 = (e - r * (D / 8)) * 8;
        uint4 kv = make_uint4(0, 0, 0, 0);
        if (r < nkeys) kv = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D + c8);
        *reinterpret_cast<uint4*>(klds + r * LDK + c8) = kv;
      }
      for (int e = threadIdx.x; e < (C / 2) * (D / 8); e += NWL * 64) {
        const int kp = e % (C / 2), c8 = (e / (C / 2)) * 8;
        uint4 v0 = make_uint4(0, 0, 0, 0), v1 = make_uint4(0, 0, 0, 0);
        if (2 * kp < nkeys) v0 = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(2 * kp) * D + c8);
        if (2 * kp + 1 < nkeys) v1 = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(2 * kp + 1) * D + c8);
        const uint32_t w0[4] = {v0.x, v0.y, v0.z, v0.w};
        const uint32_t w1[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          vt32[(c8 + 2 * i) * (LDV / 2) + kp] = (w0[i] & 0xFFFFu) | (w1[i] << 16);
          vt32[(c8 + 2 * i + 1) * (LDV / 2) + kp] = (w0[i] >> 16) | (w1[i] & 0xFFFF0000u);
        }
      }
      __syncthreads();
      if (qg >= QG) continue;
      const int bit = blk == 0 ? 1 : blk == c ? 4 : 2;
      const int kmax = (!vq || !(has & bit)) ? 0 : (a.causal ? min(nkeys, p - r0 + 1) : nkeys);
      // S^T tiles: tile mt holds keys mt*16 + 4*grp + i of query `col`
      f32x4a sa[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4a acc = {0.f, 0.f, 0.f, 0.f};
        const uint16_t* arow = klds + (mt * 16 + col) * LDK + grp * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8a av = u4_as_bf16x8(*reinterpret_cast<const uint4*>(arow + ks * 32));
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qb[ks], acc, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = mt * 16 + 4 * grp + i;
          acc[i] = key < kmax ? acc[i] * a.qscale2 : -INFINITY;
        }
        sa[mt] = acc;
      }
      float bm = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) bm = fmaxf(bm, fmaxf(fmaxf(sa[mt][0], sa[mt][1]), fmaxf(sa[mt][2], sa[mt][3])));
      bm = fmaxf(bm, __shfl_xor(bm, 16));
      bm = fmaxf(bm, __shfl_xor(bm, 32));
      const float mn = fmaxf(m, bm);
      const float msafe = mn == -INFINITY ? 0.f : mn;  // nothing visible yet: P = 0, the state stays empty
      const float sc = fast_exp2(m - msafe);            // m = -inf: 0
      l *= sc;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= sc;
      // P operand k = 8*grp + i: key 32 s2 + 4 grp + i (i < 4) or 32 s2 + 16 + 4 grp + i - 4
#pragma unroll
      for (int s2 = 0; s2 < MT / 2; ++s2) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pv[i] = fast_exp2(sa[2 * s2][i] - msafe);
          pv[4 + i] = fast_exp2(sa[2 * s2 + 1][i] - msafe);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) l += pv[i];
        uint4 u;
        u.x = pack2_bf16(pv[0], pv[1]);
        u.y = pack2_bf16(pv[2], pv[3]);
        u.z = pack2_bf16(pv[4], pv[5]);
        u.w = pack2_bf16(pv[6], pv[7]);
        const bf16x8a pb = u4_as_bf16x8(u);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const uint16_t* vrow = vt + (dt * 16 + col) * LDV + 4 * grp + 32 * s2;
          const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
          const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
          const bf16x8a av = u4_as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
          oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb, oacc[dt], 0, 0, 0);
        }
      }
      m = mn;
    }
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    // The wavefront's 16 states go to LDS (row-major, over the staging area
    // once every wavefront is done with it) so that the merge reads each
    // partial with 16 lanes x 16 bytes, like attn_combine_kernel.
    __syncthreads();
    if (qg >= QG) continue;
    float* st = reinterpret_cast<float*>(lds) + wave * (16 * SROW + 32);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(st + col * SROW + dt * 16 + 4 * grp) =
          make_float4(oacc[dt][0], oacc[dt][1], oacc[dt][2], oacc[dt][3]);
    if (grp == 0) {
      st[16 * SROW + col] = m;
      st[16 * SROW + 16 + col] = l;
    }
    wave_sync();
    // Merge: 16 lanes per row, four rows at a time; every row's index list
    // and partial log-sums are requested before any partial is read.
    const int sub = lane & 15;
    int selA[4], selB[4];
    float lsA[4], lsB[4];
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int pr = c * C + qg * 16 + r4 * 4 + grp;
      const bool v4 = pr >= p_lo && pr < p_hi && !urow(pr - tq0);
      const int32_t* sl = idx + (static_cast<int64_t>(bh) * a.Nq + (v4 ? pr - tq0 : p_lo - tq0)) * a.K;
      selA[r4] = (v4 && sub < a.K) ? sl[sub] : -1;
      selB[r4] = (v4 && sub + 16 < a.K) ? sl[sub + 16] : -1;
    }
    auto far = [&](int x) { return x >= 0 && x < a.M1 && !(a.causal && (x == 0 || x == c || x == c - 1)); };
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int pr = c * C + qg * 16 + r4 * 4 + grp;
      const int64_t pb = (static_cast<int64_t>(bh) * a.nrows + (pr - tq0 - a.row0)) * a.K;
      lsA[r4] = far(selA[r4]) ? part_lse[(pb + sub) * a.G + hh] : -INFINITY;
      lsB[r4] = far(selB[r4]) ? part_lse[(pb + sub + 16) * a.G + hh] : -INFINITY;
    }
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int rl = r4 * 4 + grp;  // row of the wavefront's 16
      const int pr = c * C + qg * 16 + rl;
      const bool v4 = pr >= p_lo && pr < p_hi && !urow(pr - tq0);
      const int rowm = v4 ? pr - tq0 : p_lo - tq0;
      const int64_t pb = (static_cast<int64_t>(bh) * a.nrows + (rowm - a.row0)) * a.K;
      float mm = st[16 * SROW + rl], ll = st[16 * SROW + 16 + rl];
      float acc[DPL];
      {
        const float* sr = st + rl * SROW + sub * DPL;
#pragma unroll
        for (int e = 0; e < DPL; e += 4) {
          const float4 x4 = *reinterpret_cast<const float4*>(sr + e);
          acc[e] = x4.x;
          acc[e + 1] = x4.y;
          acc[e + 2] = x4.z;
          acc[e + 3] = x4.w;
        }
      }
      const uint16_t* prow = part_o + (pb * a.G + hh) * D + sub * DPL;  // slot s at prow + s * G * D
      // Slots 0..31 (lane sub holds the words of slots sub and sub + 16);
      // attn_combine_kernel<D, true> takes in any further slots afterwards.
      const int k32 = min(a.K, 32);
      for (int s0 = 0; s0 < k32; s0 += kMergeBatch) {
        float ls[kMergeBatch];
        int off[kMergeBatch];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
          const int s = s0 + u;
          const float la = __shfl(lsA[r4], (lane & 48) | (s & 15)), lb = __shfl(lsB[r4], (lane & 48) | (s & 15));
          ls[u] = s < k32 ? (s < 16 ? la : lb) : -INFINITY;
          off[u] = (ls[u] != -INFINITY ? s : 0) * a.G * D;
        }
        float x[kMergeBatch][DPL];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) load_row_part<uint16_t, DPL>(prow + off[u], x[u]);
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
          if (ls[u] == -INFINITY) continue;
          const float mn = fmaxf(mm, ls[u]);
          const float c0 = fast_exp2(mm - mn), c1 = fast_exp2(ls[u] - mn);
          ll = ll * c0 + c1;
#pragma unroll
          for (int e = 0; e < DPL; ++e) acc[e] = acc[e] * c0 + x[u][e] * c1;
          mm = mn;
        }
      }
      if (!v4) continue;
      const int64_t orow = (static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + rowm;
      const float inv = ll > 0.f ? 1.0f / ll : 0.f;
      float res[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) res[e] = acc[e] * inv;
      store_row_part<uint16_t, DPL>(o + orow * D + sub * DPL, res);
      if (lse && sub == 0) lse[orow] = ll > 0.f ? (mm + fast_log2(ll)) * kLn2 : -INFINITY;
    }
  }
}

// One wavefront per (row of the chunk, query head): merge the row's K
// partials.  16 lanes cover one partial (8 bf16 each for d = 128).  TAIL:
// causal budgets above 32, after attn_local_kernel has merged slots 0..31
// into o and lse: the row's state restarts from (o, lse) and takes in the
// partials of its other slots (not its first, previous or own block, which
// never have partials).
template <int D, bool TAIL>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnBlockArgs a, const int32_t* __restrict__ idx,
                                                           const uint16_t* __restrict__ part_o,
                                                           const float* __restrict__ part_lse,
                                                           uint16_t* __restrict__ o, float* __restrict__ lse) {
  constexpr int DPL = D / 16;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = lane >> 4, sub = lane & 15;
  const int rr = blockIdx.x * 4 + wave;
  if (rr >= a.nrows) return;
  const int hq = blockIdx.y % a.H;
  const int b = blockIdx.y / a.H;
  const int hk = hq / a.G, hh = hq - hk * a.G;
  const int bh = b * a.Hkv + hk;
  const int row = a.row0 + rr;
  if (union_row(a, bh, row)) return;  // written by the row-tile union kernel
  const int32_t* sel = idx + (static_cast<int64_t>(bh) * a.Nq + row) * a.K;
  const int64_t orow = (static_cast<int64_t>(b) * a.H + hq) * a.Nq + row;
  float m = -INFINITY, s = 0.f, acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
  int slot0 = 0;
  const int c = (a.N - a.Nq + row) / a.C;
  if constexpr (TAIL) {
    slot0 = 32;
    if (grp == 0) {
      const float l0 = lse[orow];
      if (l0 != -INFINITY) {
        m = l0 * kLog2e;
        s = 1.f;
        load_row_part<uint16_t, DPL>(o + orow * D + sub * DPL, acc);
      }
    }
  }
  // The group takes slots grp, grp + 4, ...: SPL of them at a time, their
  // block indices, then their log-sums, then their partials each requested
  // together.
  constexpr int SPL = 4;
  const int64_t pbase = (static_cast<int64_t>(bh) * a.nrows + rr) * a.K;
  for (int s0 = slot0 + grp; s0 < a.K; s0 += 4 * SPL) {
    int blk[SPL];
    float ls[SPL];
#pragma unroll
    for (int i = 0; i < SPL; ++i) blk[i] = s0 + 4 * i < a.K ? sel[s0 + 4 * i] : -1;
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      // padding (no partial was written); TAIL: the blocks merged before
      const bool take = blk[i] >= 0 && blk[i] < a.M1 && !(TAIL && (blk[i] == 0 || blk[i] == c || blk[i] == c - 1));
      ls[i] = take ? part_lse[(pbase + s0 + 4 * i) * a.G + hh] : -INFINITY;
    }
    float x[SPL][DPL];
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      if (ls[i] != -INFINITY) {
        load_row_part<uint16_t, DPL>(part_o + ((pbase + s0 + 4 * i) * a.G + hh) * D + sub * DPL, x[i]);
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) x[i][e] = 0.f;
      }
    }
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      if (ls[i] == -INFINITY) continue;
      const float mn = fmaxf(m, ls[i]);
      const float c0 = fast_exp2(m - mn), c1 = fast_exp2(ls[i] - mn);
      s = s * c0 + c1;
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] = acc[e] * c0 + x[i][e] * c1;
      m = mn;
    }
  }
#pragma unroll
  for (int msk = 16; msk <= 32; msk <<= 1) {
    float o2[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) o2[e] = __shfl_xor(acc[e], msk);
    const float m2 = __shfl_xor(m, msk), s2 = __shfl_xor(s, msk);
    merge_state<DPL>(m, s, acc, m2, s2, o2);
  }
  if (grp == 0) {
    float res[DPL];
    const float inv = s > 0.f ? 1.0f / s : 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) res[e] = acc[e] * inv;
    store_row_part<uint16_t, DPL>(o + orow * D + sub * DPL, res);
    if (lse && sub == 0) lse[orow] = s > 0.f ? (m + fast_log2(s)) * kLn2 : -INFINITY;
  }
}

// ----------------------------------------------------------------------------
// Row-tile union attention, for selections where neighbouring query rows pick
// mostly the same blocks (slowly drifting queries and keys).  A tile is
// T = 256 / G consecutive rows of one (batch, KV head); its columns are the
// (row, head) pairs, 16 per v_mfma_f32_16x16x32_bf16 column group, two groups
// per wavefront, eight wavefronts per workgroup.  attn_union_plan_kernel
// counts the distinct blocks the tile selects (its union U) and flags the
// tile when |U| <= ulimit.  attn_union_kernel then walks U (ascending) once
// per flagged tile: each block's keys and values are staged in LDS (the next
// block's are loaded into registers meanwhile) and every column group one of
// whose rows selected the block runs the online softmax over it (a column
// masks the block off when its row did not select it, and the keys after its
// position when causal).  o and lse are written directly: no partials.  The
// block-centric kernels skip the rows of flagged tiles.
// ----------------------------------------------------------------------------
constexpr int kUnionWaves = 8;
constexpr int kUnionGroups = 2;   // 16-column groups per wavefront
constexpr int kUnionCols = kUnionWaves * kUnionGroups * 16;
constexpr int kUnionMaxU = 256;   // union limit: at most min(3K, 256) blocks
constexpr float kUnionSlack = 8.f;  // log2 units the running maximum may lag behind
constexpr size_t kUnionMaxLds = 160 * 1024;  // LDS of one CU
constexpr int kUnionMergeBatch = 4;  // LOCAL: partials requested together
constexpr int kLocalWaves = 4;       // LOCAL: wavefronts per workgroup (several workgroups per CU)
constexpr int kDeviceCUs = 256;
// LDS byte address of a pointer into dynamic shared memory, made wave-uniform.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char*)p)));
}
// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane.
// Issued from inline assembly so that the compiler does not make the next
// LDS read wait for it (it cannot tell the two stages apart); the consumer
// waits for it with an explicit vmcnt wait and a barrier.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds) : "memory", "m0");
}
// Chunk-position swizzle of a staged key row (NCH 16-byte chunks per row):
// the 16 rows of a K operand read get 16 distinct bank positions.
template <int NCH>
__device__ __forceinline__ int union_swz(int r) {
  return NCH == 16 ? (r & 15) : ((r >> 1) & 7);
}
// Fewest flagged tiles the union kernel takes: four per CU of the 256-CU
// device, so that its persistent grid (two workgroups per CU) runs at least
// two rounds of tiles.
constexpr int kUnionMinTiles = 1024;
// Process-wide threshold (pisa_attn_union_min_tiles); negative: union kernel off.
static std::atomic<int> g_union_min_tiles{kUnionMinTiles};

// One workgroup of 256 threads per tile: |U| against ulimit.  The union of
// four rows spread over the tile is counted first: when it already exceeds
// ulimit, so does U, and the other rows are not read.
__global__ __launch_bounds__(256) void attn_union_plan_kernel(AttnBlockArgs a, const int32_t* __restrict__ idx,
                                                              uint8_t* __restrict__ flag, int T, int ulimit) {
  extern __shared__ __align__(16) uint32_t bits[];  // [ceil(M1 / 32)]
  __shared__ int s_cnt[2];
  const int tid = threadIdx.x, tile = blockIdx.x, bh = blockIdx.y;
  const int MW = (a.M1 + 31) / 32;
  for (int e = tid; e < MW; e += 256) bits[e] = 0;
  if (tid < 2) s_cnt[tid] = 0;
  __syncthreads();
  const int r0 = tile * T;
  const int nr = min(T, a.Nq - r0);
  const int32_t* lst = idx + (static_cast<int64_t>(bh) * a.Nq + r0) * a.K;
  auto mark = [&](int e) {
    const int x = lst[e];
    if (x >= 0 && x < a.M1) atomicOr(&bits[x >> 5], 1u << (x & 31));
  };
  auto count = [&](int* dst) {
    int c = 0;
    for (int e = tid; e < MW; e += 256) c += __builtin_popcount(bits[e]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
    if ((tid & 63) == 0) atomicAdd(dst, c);
    __syncthreads();
    return *dst;
  };
  // rows 0, nr/3, 2nr/3 and nr-1 (repeats are harmless: the bits are idempotent)
  for (int e = tid; e < 4 * a.K; e += 256) {
    const int j = e / a.K, row = j == 3 ? nr - 1 : j * nr / 3;
    mark(row * a.K + e - j * a.K);
  }
  __syncthreads();
  int u = count(&s_cnt[0]);
  if (u <= ulimit) {
    for (int e = tid; e < nr * a.K; e += 256) mark(e);
    __syncthreads();
    u = count(&s_cnt[1]);
  }
  if (tid == 0) flag[static_cast<int64_t>(bh) * a.skip_tiles + tile] = u <= ulimit ? 1 : 0;
}

// One workgroup of 1024 threads, four flags per thread per pass.  Fewer than
// min_tiles flagged tiles would leave most of the chip idle behind a few
// long tiles: their flags are cleared (the block-centric kernels then take
// those rows) and the count is zero.  Otherwise the flagged tiles' ids
// (bh * tiles + tile), ascending, and their count, for the union kernel's
// persistent grid.
__global__ __launch_bounds__(1024) void attn_union_compact_kernel(uint8_t* __restrict__ flag, int n, int min_tiles,
                                                                  int32_t* __restrict__ list,
                                                                  int32_t* __restrict__ count) {
  __shared__ int wsum[16];
  __shared__ int s_total;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  auto flags4 = [&](int i) -> uint32_t {  // flags i..i+3 as bytes (flag is 256-byte aligned)
    if (i + 3 < n) return *reinterpret_cast<const uint32_t*>(flag + i);
    uint32_t x = 0;
    for (int j = 0; j < 4 && i + j < n; ++j) x |= static_cast<uint32_t>(flag[i + j]) << (8 * j);
    return x;
  };
  int c = 0;
  for (int i = 4 * tid; i < n; i += 4096) c += __builtin_popcount(flags4(i));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
  if (tid == 0) s_total = 0;
  __syncthreads();
  if (lane == 0) atomicAdd(&s_total, c);
  __syncthreads();
  const int total = s_total;
  if (total < min_tiles) {
    for (int i = 4 * tid; i < n; i += 4096) {
      if (i + 3 < n) *reinterpret_cast<uint32_t*>(flag + i) = 0u;
      else for (int j = 0; i + j < n; ++j) flag[i + j] = 0;
    }
    if (tid == 0) *count = 0;
    return;
  }
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += 4096) {
    const int i = c0 + 4 * tid;
    const uint32_t x = i < n ? flags4(i) : 0u;
    const int mine = __builtin_popcount(x);
    int inc = mine;  // inclusive scan over the wavefront
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(inc, off);
      if (lane >= off) inc += y;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int pre = 0, tot = 0;
    for (int j = 0; j < 16; ++j) {
      pre += j < w ? wsum[j] : 0;
      tot += wsum[j];
    }
    int pos = base + pre + inc - mine;
    for (int j = 0; j < 4; ++j)
      if ((x >> (8 * j)) & 1u) list[pos++] = i + j;
    base += tot;
    __syncthreads();  // wsum is rewritten by the next chunk
  }
  if (tid == 0) *count = base;
}

// LOCAL (causal, block-centric path): the tiles of the chunk [a.row0,
// a.row0 + a.nrows) that the union kernel did not take, each over the union
// of its rows' first, previous and own blocks only (the ones they selected);
// every column then merges the partials the block-centric kernel wrote for
// its row's other slots before o and lse are written.  ltiles: tiles per
// (batch, KV head) in the chunk, lcount: ltiles times the groups.
template <int D, int CT, int G, bool LOCAL>
__global__ __launch_bounds__((LOCAL ? kLocalWaves : kUnionWaves) * 64, 2) void attn_union_kernel(
    AttnBlockArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ idx, uint16_t* __restrict__ o, float* __restrict__ lse,
    const int32_t* __restrict__ tile_list, const int32_t* __restrict__ tile_count,
    const uint16_t* __restrict__ part_o, const float* __restrict__ part_lse, int ltiles, int lcount) {
  constexpr int NW = LOCAL ? kLocalWaves : kUnionWaves, NG = kUnionGroups;
  constexpr int RW = 16 * NG / G, T = NW * RW;  // rows per wavefront, per tile
  constexpr int KS = D / 32;
  constexpr int C = CT * 32;
  constexpr int MT = C / 16;
  constexpr int MC = (D == 128 && MT > 4) ? 2 : (MT <= 6 ? MT : 4);  // 16-key tiles per softmax chunk
  static_assert(MT % MC == 0 && MC % 2 == 0, "blocks of 32, 64, 96 or 128 keys");
  constexpr int DT = D / 16;
  constexpr int MWU = kUnionMaxU / 32;  // row-mask words
  constexpr int NCH = D / 8;            // 16-byte chunks per key row
  constexpr int RPI = 64 / NCH;         // key rows per direct-to-LDS load instruction
  constexpr int BLK = C * D;            // elements of one staged K (or V) block
  static_assert(D == 64 || D == 128, "head dimension 64 or 128");
  // Two stages of [K block, V block], both row-major with the 16-byte chunks
  // of row r stored at chunk position c ^ union_swz<NCH>(r): the K operand
  // reads (16 rows x one chunk per 16 lanes) and the transposing V reads
  // (16 rows x 32 bytes per wavefront) then spread over all banks.
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* stage = lds;
  uint32_t* bitmap = reinterpret_cast<uint32_t*>(lds + 4 * BLK);  // [ceil(M1 / 32)]
  const int MW = (a.M1 + 31) / 32;
  int* wpre = reinterpret_cast<int*>(bitmap + MW);                // [MW] set bits before word w
  int* ulist = wpre + MW;                                         // [kUnionMaxU] union, ascending
  uint32_t* rmask = reinterpret_cast<uint32_t*>(ulist + kUnionMaxU);  // [T][MWU] row j selected U[u]
  __shared__ int s_nu;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ntile = LOCAL ? lcount : *tile_count;
  const int rend = LOCAL ? min(a.Nq, a.row0 + a.nrows) : a.Nq;  // rows of this launch end here
  // persistent workgroups over the tiles
  for (int li = blockIdx.x; li < ntile; li += gridDim.x) {
  int bh, tile;
  if constexpr (LOCAL) {
    bh = li / ltiles;
    tile = a.row0 / T + (li - bh * ltiles);
    // the union kernel's tiles (T divides its tile rows)
    if (a.skip && a.skip[static_cast<int64_t>(bh) * a.skip_tiles + ((tile * T) >> a.skip_shift)]) continue;
  } else {
    const int id = tile_list[li];
    bh = id / a.skip_tiles;
    tile = id - bh * a.skip_tiles;
  }
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = tile * T;
  const int32_t* lst = idx + static_cast<int64_t>(bh) * a.Nq * a.K;
  // LOCAL: only a row's first, previous and own blocks (App. B's forced set)
  auto take = [&](int row, int x) {
    if (x < 0 || x >= a.M1) return false;
    if constexpr (LOCAL) {
      const int cr = (a.N - a.Nq + row) / C;
      return x == 0 || x == cr || x == cr - 1;
    }
    return true;
  };

  __syncthreads();  // the previous tile's readers of the LDS are done
  for (int e = tid; e < MW; e += NW * 64) bitmap[e] = 0;
  for (int e = tid; e < T * MWU; e += NW * 64) rmask[e] = 0;
  __syncthreads();
  for (int e = tid; e < T * a.K; e += NW * 64) {
    const int row = r0 + e / a.K;
    if (row >= rend) continue;
    const int x = lst[static_cast<int64_t>(row) * a.K + e % a.K];
    if (take(row, x)) atomicOr(&bitmap[x >> 5], 1u << (x & 31));
  }
  __syncthreads();
  if (wave == 0) {
    const int per = (MW + 63) / 64;
    const int w0 = min(MW, lane * per), w1 = min(MW, w0 + per);
    int cnt = 0;
    for (int w = w0; w < w1; ++w) cnt += __builtin_popcount(bitmap[w]);
    int x = cnt;  // inclusive scan over the wavefront
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(x, off);
      if (lane >= off) x += y;
    }
    int run = x - cnt;
    for (int w = w0; w < w1; ++w) {
      wpre[w] = run;
      run += __builtin_popcount(bitmap[w]);
    }
    if (lane == 63) s_nu = min(x, kUnionMaxU);  // the plan kernel flagged |U| <= ulimit <= kUnionMaxU
  }
  __syncthreads();
  const int nu = s_nu;
  for (int w = tid; w < MW; w += NW * 64) {
    uint32_t bm = bitmap[w];
    int pos = wpre[w];
    while (bm && pos < kUnionMaxU) {
      ulist[pos++] = w * 32 + __builtin_ctz(bm);
      bm &= bm - 1;
    }
  }
  for (int e = tid; e < T * a.K; e += NW * 64) {
    const int j = e / a.K, row = r0 + j;
    if (row >= rend) continue;
    const int x = lst[static_cast<int64_t>(row) * a.K + e % a.K];
    if (!take(row, x)) continue;
    const int u = wpre[x >> 5] + __builtin_popcount(bitmap[x >> 5] & ((1u << (x & 31)) - 1u));
    if (u < kUnionMaxU) atomicOr(&rmask[j * MWU + (u >> 5)], 1u << (u & 31));
  }

  // this lane's columns: group cg holds row j = wave * RW + (cg * 16 + col) / G,
  // head (cg * 16 + col) % G
  const int col = lane & 15, grp = lane >> 4;
  int jr[NG], tq[NG];
  bool vrow[NG];
  bf16x8a qb[NG][KS];
  float m[NG], l[NG];
  f32x4a oacc[NG][DT];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    const int cc = cg * 16 + col;
    jr[cg] = wave * RW + cc / G;
    const int row = r0 + jr[cg];
    vrow[cg] = row < rend;
    const int rowc = vrow[cg] ? row : r0;
    tq[cg] = a.N - a.Nq + rowc;
    const uint16_t* qrow = q + ((static_cast<int64_t>(b) * a.H + h * G + cc % G) * a.Nq + rowc) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qb[cg][ks] = u4_as_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 32));
    m[cg] = -INFINITY;
    l[cg] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[cg][dt] = f32x4a{0.f, 0.f, 0.f, 0.f};
  }

  // Block blk's keys and values straight from global memory into stage buf:
  // each instruction fills RPI rows (lane L: row L / NCH, chunk position
  // L % NCH, which holds logical chunk (L % NCH) ^ swz(row)).  Rows past the
  // sequence's end repeat its last row (finite values; their keys are masked).
  auto issue = [&](int blk, int buf) __attribute__((always_inline)) {
    const int rb = blk * C;
    const int last = min(C, a.N - rb) - 1;
    const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + rb) * D;
    const uint16_t* vb = v + (static_cast<int64_t>(bh) * a.Nkv + rb) * D;
    uint16_t* kd = stage + buf * 2 * BLK;
    for (int ins = wave; ins < C / RPI; ins += NW) {
      const int row = ins * RPI + lane / NCH;
      const int64_t src = static_cast<int64_t>(min(row, last)) * D + ((lane % NCH) ^ union_swz<NCH>(row)) * 8;
      const uint32_t dk = lds_addr(kd + ins * RPI * D);
      lds_dma16(kb + src, dk);
      lds_dma16(vb + src, dk + BLK * 2);
    }
  };
  // this lane's K operand offsets (elements within a block): row tile*16 + col,
  // logical chunk 4 ks + grp
  int koff[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = col * D + ((4 * ks + grp) ^ union_swz<NCH>(col)) * 8;
  // V operand (transposing reads): lane i = col of group grp reads 8 bytes of
  // row 4 grp + i / 4 (+16 for the second half of a 32-key step) at column
  // 16 dt + 4 (i % 4)
  const int vr0 = 4 * grp + col / 4;
  int voff[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
    voff[dt] = vr0 * D + ((2 * dt + (col & 3) / 2) ^ union_swz<NCH>(vr0)) * 8 + (col & 1) * 4;

  __syncthreads();  // ulist and rmask complete
  if (nu > 0) issue(ulist[0], 0);
  for (int u = 0; u < nu; ++u) {
    const int blk = ulist[u];
    const int rb = blk * C;
    const int nkeys = min(C, a.N - rb);
    __builtin_amdgcn_s_waitcnt(0);  // this wavefront's loads of block u have landed
    __syncthreads();                // every wavefront's have, and block u - 1 is done
    if (u + 1 < nu) issue(ulist[u + 1], (u + 1) & 1);
    const uint16_t* klds = stage + (u & 1) * 2 * BLK;
    const uint16_t* vlds = klds + BLK;
    // Both column groups take every staged operand read: K and V^T tiles are
    // read from LDS once per wavefront and feed one product per group.
    int kmax[NG];
    bool any = false, full = true;
#pragma unroll
    for (int cg = 0; cg < NG; ++cg) {
      const bool sel = vrow[cg] && ((rmask[jr[cg] * MWU + (u >> 5)] >> (u & 31)) & 1u);
      // keys the column sees (0 also for a selected block after its position)
      kmax[cg] = !sel ? 0 : (a.causal ? max(0, min(nkeys, tq[cg] - rb + 1)) : nkeys);
      any = any || kmax[cg] > 0;
      full = full && kmax[cg] == C;
    }
    if (__ballot(any) == 0) continue;  // no column of the wavefront sees a key of the block
    // every column of the wavefront sees every key of the block: no masking
    const bool wfull = __ballot(!full) == 0;
    // keys in chunks of 64 (online softmax per chunk) to bound the registers
#pragma unroll
    for (int k0 = 0; k0 < MT; k0 += MC) {
      f32x4a sa[NG][MC];
#pragma unroll
      for (int mt = 0; mt < MC; ++mt) {
        f32x4a acc[NG];
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) acc[cg] = f32x4a{0.f, 0.f, 0.f, 0.f};
        const uint16_t* arow = klds + (k0 + mt) * 16 * D;
        bf16x8a av[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) av[ks] = u4_as_bf16x8(*reinterpret_cast<const uint4*>(arow + koff[ks]));
        __builtin_amdgcn_sched_barrier(0);  // the reads leave together; the products wait for them in turn
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int cg = 0; cg < NG; ++cg)
            acc[cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[ks], qb[cg][ks], acc[cg], 0, 0, 0);
        // raw logits (the log2e / sqrt(d) scale is applied in the exponent)
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) {
          if (!wfull) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int key = (k0 + mt) * 16 + 4 * grp + i;
              acc[cg][i] = key < kmax[cg] ? acc[cg][i] : -INFINITY;
            }
          }
          sa[cg][mt] = acc[cg];
        }
      }
      // Online softmax with a lazily raised reference: m only moves (and
      // the accumulators are rescaled) when the chunk's maximum exceeds it
      // by more than kUnionSlack, so the exponentials stay below
      // 2^kUnionSlack; in most chunks no column of the wavefront moves.
      // Each lane tests its own logits first; only when one of them exceeds
      // its column's reference does the wavefront reduce the column maxima
      // across lanes and move the references.
      float lm[NG];
      bool over = false;
#pragma unroll
      for (int cg = 0; cg < NG; ++cg) {
        float bm = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < MC; ++mt)
          bm = fmaxf(bm, fmaxf(fmaxf(sa[cg][mt][0], sa[cg][mt][1]), fmaxf(sa[cg][mt][2], sa[cg][mt][3])));
        lm[cg] = bm * a.qscale2;
        over = over || lm[cg] > m[cg] + kUnionSlack;
      }
      if (__ballot(over) != 0) {
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) {
          float bm = lm[cg];
          bm = fmaxf(bm, __shfl_xor(bm, 16));
          bm = fmaxf(bm, __shfl_xor(bm, 32));
          const float nm = bm > m[cg] + kUnionSlack ? bm : m[cg];
          const float scl = nm != m[cg] ? fast_exp2(m[cg] - nm) : 1.f;
          l[cg] *= scl;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) oacc[cg][dt] *= scl;
          m[cg] = nm;
        }
      }
      float nms[NG];  // -m, or 0 while no key was seen (then every logit is -inf)
#pragma unroll
      for (int cg = 0; cg < NG; ++cg) nms[cg] = m[cg] == -INFINITY ? 0.f : -m[cg];
#pragma unroll
      for (int s2 = 0; s2 < MC / 2; ++s2) {
        bf16x8a pb[NG];
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) {
          float pv[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pv[i] = fast_exp2(fmaf(sa[cg][2 * s2][i], a.qscale2, nms[cg]));
            pv[4 + i] = fast_exp2(fmaf(sa[cg][2 * s2 + 1][i], a.qscale2, nms[cg]));
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) l[cg] += pv[i];
          uint4 uu;
          uu.x = pack2_bf16(pv[0], pv[1]);
          uu.y = pack2_bf16(pv[2], pv[3]);
          uu.z = pack2_bf16(pv[4], pv[5]);
          uu.w = pack2_bf16(pv[6], pv[7]);
          pb[cg] = u4_as_bf16x8(uu);
        }
        bf16x8a avv[DT];
        const uint16_t* vr = vlds + (k0 + 2 * s2) * 16 * D;  // keys of tiles 2 s2, 2 s2 + 1 of the chunk
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const v4s16 lo = lds_read_tr16x4(vr + voff[dt]);
          const v4s16 hi = lds_read_tr16x4(vr + 16 * D + voff[dt]);
          avv[dt] = __builtin_bit_cast(bf16x8a, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int cg = 0; cg < NG; ++cg)
            oacc[cg][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(avv[dt], pb[cg], oacc[cg][dt], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    float ll = l[cg];
    ll += __shfl_xor(ll, 16);
    ll += __shfl_xor(ll, 32);
    float mm = m[cg];
    const int cc = cg * 16 + col;
    if constexpr (LOCAL) {
      // merge the partials (o normalised, log2-sum) of the row's other
      // slots.  The four lanes of a column request the slot indices, then
      // the log-sums, of slots grp, grp + 4, ... (the first 32) all at once;
      // the partials (each lane the 4 values of each 16-wide d tile it
      // holds) follow in batches of four slots.
      const int row = tq[cg] - (a.N - a.Nq);
      const int cr = tq[cg] / C;
      const int hq = cc % G;
      const int32_t* sl = lst + static_cast<int64_t>(row) * a.K;
      const int64_t pb = (static_cast<int64_t>(bh) * a.nrows + (row - a.row0)) * a.K;
      auto far = [&](int x) { return x >= 0 && x < a.M1 && x != 0 && x != cr && x != cr - 1; };
      constexpr int KB = 8;  // the first 4 * KB slots: KB per lane
      int xs[KB];
      float lsv[KB];
#pragma unroll
      for (int i = 0; i < KB; ++i) xs[i] = 4 * i + grp < a.K ? sl[4 * i + grp] : -1;
#pragma unroll
      for (int i = 0; i < KB; ++i) lsv[i] = far(xs[i]) ? part_lse[(pb + 4 * i + grp) * G + hq] : -INFINITY;
      const uint16_t* pcol = part_o + (pb * G + hq) * D + 4 * grp;  // slot s at pcol + s * G * D
      auto merge = [&](const float (&ls)[kUnionMergeBatch], const uint2 (&xo)[kUnionMergeBatch][DT])
                       __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kUnionMergeBatch; ++u) {
          if (ls[u] == -INFINITY) continue;
          const float mn = fmaxf(mm, ls[u]);
          const float c0 = fast_exp2(mm - mn), c1 = fast_exp2(ls[u] - mn);
          ll = ll * c0 + c1;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            oacc[cg][dt][0] = oacc[cg][dt][0] * c0 + __uint_as_float(xo[u][dt].x << 16) * c1;
            oacc[cg][dt][1] = oacc[cg][dt][1] * c0 + __uint_as_float(xo[u][dt].x & 0xFFFF0000u) * c1;
            oacc[cg][dt][2] = oacc[cg][dt][2] * c0 + __uint_as_float(xo[u][dt].y << 16) * c1;
            oacc[cg][dt][3] = oacc[cg][dt][3] * c0 + __uint_as_float(xo[u][dt].y & 0xFFFF0000u) * c1;
          }
          mm = mn;
        }
      };
      static_assert(kUnionMergeBatch == 4, "a batch is the four slots of one register of lsv");
      // batch i = slots 4 i .. 4 i + 3; slot 4 i + u is held by lane col + 16 u
      auto fetch = [&](int i, float (&ls)[kUnionMergeBatch], uint2 (&xo)[kUnionMergeBatch][DT])
                       __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kUnionMergeBatch; ++u) {
          ls[u] = __shfl(lsv[i], col | (u << 4));
          const uint16_t* pr = pcol + static_cast<int64_t>(ls[u] != -INFINITY ? 4 * i + u : 0) * G * D;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) xo[u][dt] = *reinterpret_cast<const uint2*>(pr + dt * 16);
        }
      };
      const int nb = min(a.K, 4 * KB);
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        if (4 * i >= nb) break;
        float ls[kUnionMergeBatch];
        uint2 xo[kUnionMergeBatch][DT];
        fetch(i, ls, xo);
        merge(ls, xo);
      }
      // slots 32 and up (budgets above 32), a batch at a time
      for (int s0 = 4 * KB; s0 < a.K; s0 += kUnionMergeBatch) {
        float ls[kUnionMergeBatch];
        uint2 xo[kUnionMergeBatch][DT];
#pragma unroll
        for (int u = 0; u < kUnionMergeBatch; ++u) {
          const int sx = s0 + u;
          const int x = sx < a.K ? sl[sx] : -1;
          ls[u] = far(x) ? part_lse[(pb + sx) * G + hq] : -INFINITY;
        }
#pragma unroll
        for (int u = 0; u < kUnionMergeBatch; ++u) {
          const uint16_t* pr = pcol + static_cast<int64_t>(ls[u] != -INFINITY ? s0 + u : 0) * G * D;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) xo[u][dt] = *reinterpret_cast<const uint2*>(pr + dt * 16);
        }
        merge(ls, xo);
      }
    }
    if (!vrow[cg]) continue;
    // oacc[cg][dt][i] = O[d = dt*16 + 4*grp + i][this column]
    const int64_t orow = (static_cast<int64_t>(b) * a.H + h * G + cc % G) * a.Nq + r0 + jr[cg];
    const float inv = ll > 0.f ? 1.0f / ll : 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      uint2 w;
      w.x = pack2_bf16(oacc[cg][dt][0] * inv, oacc[cg][dt][1] * inv);
      w.y = pack2_bf16(oacc[cg][dt][2] * inv, oacc[cg][dt][3] * inv);
      *reinterpret_cast<uint2*>(o + orow * D + dt * 16 + 4 * grp) = w;
    }
    if (lse && grp == 0) lse[orow] = ll > 0.f ? (mm + fast_log2(ll)) * kLn2 : -INFINITY;
  }
  }
}

// Attention for few rows (decode): one workgroup per (row, slot) attends the
// slot's key block for the G query heads of the KV head and leaves the same
// partial as attn_block16_kernel (o normalised by its own sum in bf16, the
// log2-sum in fp32); attn_combine_kernel merges the K partials of each row.
// The block's keys and values are staged in LDS with every load in flight
// at once, so a step costs a few memory round trips whatever the row count.
template <int D, int GMAX>
__global__ __launch_bounds__(256) void attn_slot_kernel(AttnBlockArgs a, const uint16_t* __restrict__ q,
                                                        const uint16_t* __restrict__ k,
                                                        const uint16_t* __restrict__ v,
                                                        const int32_t* __restrict__ idx,
                                                        uint16_t* __restrict__ part_o,
                                                        float* __restrict__ part_lse) {
  constexpr int DPL = D / 16;
  constexpr int NPART = 256 / D;  // key subsets summed separately in the PV product
  extern __shared__ __align__(16) uint16_t lds[];
  const int C = a.C;
  uint16_t* ks = lds;                                          // [C][D]
  uint16_t* vs = lds + C * D;                                  // [C][D]
  float* z = reinterpret_cast<float*>(lds + 2 * C * D);        // [C][G] logits, then weights
  float* red = z + C * GMAX;                                   // [256] PV partial sums
  float* ml = red + 256;                                       // [GMAX][2] max, sum

  const int slot = blockIdx.x;
  const int rr = blockIdx.y % a.nrows;
  const int bh = blockIdx.y / a.nrows;
  const int row = a.row0 + rr;
  const int blk = idx[(static_cast<int64_t>(bh) * a.Nq + row) * a.K + slot];
  if (blk < 0 || blk >= a.M1) return;  // padding: the combine skips these slots
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int G = a.G;
  const int t = a.N - a.Nq + row;
  const int r0 = blk * C;
  const int nkeys = min(C, a.N - r0);
  const int kmax = a.causal ? min(nkeys, t - r0 + 1) : nkeys;
  const int tid = threadIdx.x;

  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  const uint16_t* vb = v + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  for (int e = tid; e < C * (D / 8); e += 256) {
    const int r = e / (D / 8);
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (r < nkeys) {
      kv = reinterpret_cast<const uint4*>(kb)[e];
      vv = reinterpret_cast<const uint4*>(vb)[e];
    }
    reinterpret_cast<uint4*>(ks)[e] = kv;
    reinterpret_cast<uint4*>(vs)[e] = vv;
  }
  const int grp = tid >> 4, sub = tid & 15;
  float qv[GMAX][DPL];
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) {
    if (hh < G) {
      const int64_t off = ((static_cast<int64_t>(b) * a.H + h * G + hh) * a.Nq + row) * D + sub * DPL;
      load_row_part<uint16_t, DPL>(q + off, qv[hh]);
#pragma unroll
      for (int e = 0; e < DPL; ++e) qv[hh][e] *= a.qscale2;
    } else {
#pragma unroll
      for (int e = 0; e < DPL; ++e) qv[hh][e] = 0.f;
    }
  }
  __syncthreads();
  // logits of the visible keys (16 lanes per key)
  for (int r = grp; r < C; r += 16) {
    float x[DPL];
    load_row_part<uint16_t, DPL>(ks + r * D + sub * DPL, x);
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < G) {
        float d0 = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) d0 = fmaf(qv[hh][e], x[e], d0);
        d0 = sum16(d0);
        if (sub == 0) z[r * G + hh] = r < kmax ? d0 : -INFINITY;
      }
    }
  }
  __syncthreads();
  // per head: block-local max and sum, z turned into weights 2^(z - m)
  const int wave = tid >> 6, lane = tid & 63;
  for (int hh = wave; hh < G; hh += 4) {
    float m = -INFINITY;
    for (int r = lane; r < C; r += 64) m = fmaxf(m, z[r * G + hh]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const float msafe = m == -INFINITY ? 0.f : m;
    float sm = 0.f;
    for (int r = lane; r < C; r += 64) {
      const float p = fast_exp2(z[r * G + hh] - msafe);
      z[r * G + hh] = p;
      sm += p;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sm += __shfl_xor(sm, o);
    if (lane == 0) {
      ml[2 * hh] = m;
      ml[2 * hh + 1] = sm;
    }
  }
  __syncthreads();
  // O[hh][d] = sum_r w[r][hh] V[r][d] / l: thread (part, d) sums keys part, part + NPART, ...
  const int dcol = tid % D, part = tid / D;
  for (int hh = 0; hh < G; ++hh) {
    float acc = 0.f;
    for (int r = part; r < kmax; r += NPART) acc = fmaf(z[r * G + hh], bf16_to_f32(vs[r * D + dcol]), acc);
    red[tid] = acc;
    __syncthreads();
    if (tid < D) {
      float o = red[tid];
#pragma unroll
      for (int pp = 1; pp < NPART; ++pp) o += red[tid + pp * D];
      const float m = ml[2 * hh], l = ml[2 * hh + 1];
      const int64_t pidx = ((static_cast<int64_t>(bh) * a.nrows + rr) * a.K + slot) * G + hh;
      part_o[pidx * D + tid] = f32_to_bf16_rne(l > 0.f ? o / l : 0.f);
      if (tid == 0) part_lse[pidx] = l > 0.f ? m + fast_log2(l) : -INFINITY;
    }
    __syncthreads();
  }
}

template <typename T, int D, int TEAM>
static void launch_rows(const Shape& s, const AttnArgs& a, hipStream_t st) {
  constexpr int ROWS = 256 / TEAM;
  dim3 grid((s.Nq + ROWS - 1) / ROWS, s.B * s.H);
  attn_rows_kernel<T, D, TEAM><<<grid, 256, 0, st>>>(a);
}

template <typename T, int D>
static void launch_rows_team(const Shape& s, const AttnArgs& a, hipStream_t st) {
  if (static_cast<int64_t>(s.B) * s.H * s.Nq <= 2048)
    launch_rows<T, D, 256>(s, a, st);
  else
    launch_rows<T, D, 64>(s, a, st);
}

// Block-centric path: bf16, many rows, cluster histogram fits in LDS.
static bool use_block_path(const Shape& s, const Geo& geo) {
  return s.bf16 && static_cast<int64_t>(s.BH()) * s.Nq >= 4096 && geo.M[1] <= 16384 && s.C <= 128;
}

// Rows per chunk: the partials of a chunk (K slots x G heads x (d bf16 + lse))
// are bounded by kPartialBudget bytes.
constexpr size_t kPartialBudget = size_t(6) << 30;

static int attn_chunk_rows(const Shape& s) {
  const size_t per_row = static_cast<size_t>(s.BH()) * s.K * s.G * (s.D * 2 + 4);
  size_t rows = kPartialBudget / per_row;
  // several chunks: whole 256-row tiles each, so that the row-tile kernels'
  // tiles line up with every chunk
  if (rows < static_cast<size_t>(s.Nq) && rows >= 256) rows = rows / 256 * 256;
  return static_cast<int>(std::min<size_t>(s.Nq, std::max<size_t>(rows, 1)));
}

// Split path for few rows: bf16, a workgroup per (row, slot), partials for
// every row at once (rows * K * G of them).
static bool use_split_path(const Shape& s, const Geo& geo) {
  return s.bf16 && !use_block_path(s, geo) && static_cast<int64_t>(s.BH()) * s.Nq <= 2048;
}

struct AttnWs {
  size_t part_o, part_lse, cl, row_lse, uflag, ulist, total;
};

// The row-tile union kernel serves groups of 1, 2, 4, 8 or 16 heads.
static bool union_ok(const Shape& s) {
  return s.G == 1 || s.G == 2 || s.G == 4 || s.G == 8 || s.G == 16;
}
static int union_tile_rows(const Shape& s) { return kUnionCols / s.G; }

static AttnWs attn_layout(const Shape& s, const Geo& geo) {
  const size_t ch = attn_chunk_rows(s);
  const size_t np = static_cast<size_t>(s.BH()) * ch * s.K;  // pairs per chunk
  AttnWs w{};
  size_t o = 0;
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  w.part_o = o;   o += al(np * s.G * s.D * 2);
  w.part_lse = o; o += al(np * s.G * 4);
  w.cl = o;       o += al(cluster_ws(s.BH(), geo.M[1], static_cast<int64_t>(np), static_cast<int>(ch)));
  // causal budgets above 32: the rows' log-sums between the per-leaf-block
  // merge and the tail merge, for callers that pass no lse
  w.row_lse = o;
  if (s.causal && s.K > 32) o += al(static_cast<size_t>(s.B) * s.H * s.Nq * 4);
  // one flag per (batch, KV head, row tile) of the row-tile union kernel
  const size_t ntile = union_ok(s) ? static_cast<size_t>(s.BH()) * ((s.Nq + union_tile_rows(s) - 1) / union_tile_rows(s)) : 0;
  w.uflag = o;
  o += al(ntile);
  // the flagged tiles' ids and their count
  w.ulist = o;
  if (ntile) o += al((ntile + 1) * 4);
  w.total = o;
  return w;
}

static AttnWs split_attn_layout(const Shape& s) {
  const size_t np = static_cast<size_t>(s.BH()) * s.Nq * s.K;
  AttnWs w{};
  size_t o = 0;
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  w.part_o = o;   o += al(np * s.G * s.D * 2);
  w.part_lse = o; o += al(np * s.G * 4);
  w.cl = o;
  w.total = o;
  return w;
}

size_t attn_ws(const Shape& s, const Geo& geo) {
  if (use_block_path(s, geo)) return attn_layout(s, geo).total;
  if (use_split_path(s, geo)) return split_attn_layout(s).total;
  return 0;
}

template <int D>
static hipError_t launch_split_path(const Shape& s, const void* q, const void* k, const void* v,
                                    const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st) {
  const AttnWs w = split_attn_layout(s);
  char* base = static_cast<char*>(ws);
  uint16_t* part_o = reinterpret_cast<uint16_t*>(base + w.part_o);
  float* part_lse = reinterpret_cast<float*>(base + w.part_lse);
  AttnBlockArgs a{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, (s.N + s.C - 1) / s.C, 0, s.Nq,
                  kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv};
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  {
    ProfScope ps("attn_slot", st);
    dim3 grid(s.K, static_cast<unsigned>(static_cast<int64_t>(s.BH()) * s.Nq));
    auto go = [&](auto kern, int gmax) {
      const size_t lds = static_cast<size_t>(2) * s.C * D * 2 + (static_cast<size_t>(s.C) * gmax + 256 + 2 * gmax) * 4;
      if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      kern<<<grid, 256, lds, st>>>(a, qq, kk, vv, idx, part_o, part_lse);
    };
    if (s.G == 1)
      go(attn_slot_kernel<D, 1>, 1);
    else if (s.G <= 4)
      go(attn_slot_kernel<D, 4>, 4);
    else
      go(attn_slot_kernel<D, 16>, 16);
  }
  {
    ProfScope ps("attn_combine", st);
    dim3 grid((s.Nq + 3) / 4, s.B * s.H);
    attn_combine_kernel<D, false><<<grid, 256, 0, st>>>(a, idx, part_o, part_lse, static_cast<uint16_t*>(o), lse);
  }
  return hipGetLastError();
}

template <int D>
static hipError_t launch_block_path(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                                    const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st) {
  const AttnWs w = attn_layout(s, geo);
  char* base = static_cast<char*>(ws);
  uint16_t* part_o = reinterpret_cast<uint16_t*>(base + w.part_o);
  float* part_lse = reinterpret_cast<float*>(base + w.part_lse);
  if (!lse && s.causal && s.K > 32) lse = reinterpret_cast<float*>(base + w.row_lse);
  const int ch = attn_chunk_rows(s);
  hipError_t e;
  // Row tiles whose selections share blocks: attended whole by the union
  // kernel first; the block-centric kernels below skip their rows.
  const uint8_t* skip = nullptr;
  int skip_shift = 0, skip_tiles = 0;
  const int union_min = g_union_min_tiles.load(std::memory_order_relaxed);
  const int mw = (geo.M[1] + 31) / 32;
  // the union kernel's LDS: two stages of a K and a V block, then the
  // union's bookkeeping (block bitmap, its prefix counts, the union, the
  // rows' masks over it); beyond the device's LDS the block-centric path
  // takes every row
  const size_t ulds = static_cast<size_t>(4) * s.C * D * 2 +
                      (static_cast<size_t>(2) * mw + kUnionMaxU +
                       static_cast<size_t>(union_ok(s) ? union_tile_rows(s) : 0) * (kUnionMaxU / 32)) * 4;
  const bool union_lds_ok = ulds <= kUnionMaxLds;
  if (union_ok(s) && union_min >= 0 && union_lds_ok) {
    const int T = union_tile_rows(s);
    skip_tiles = (s.Nq + T - 1) / T;
    while ((1 << skip_shift) < T) ++skip_shift;
    uint8_t* flag = reinterpret_cast<uint8_t*>(base + w.uflag);
    int32_t* tlist = reinterpret_cast<int32_t*>(base + w.ulist);
    int32_t* tcount = tlist + static_cast<int64_t>(s.BH()) * skip_tiles;
    skip = flag;
    AttnBlockArgs ua{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], 0, s.Nq,
                     kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv, nullptr, skip_shift, skip_tiles};
    const int ulimit = std::min(3 * s.K, kUnionMaxU);
    dim3 grid(static_cast<unsigned>(skip_tiles), s.BH());
    {
      ProfScope ps("attn_union_plan", st);
      attn_union_plan_kernel<<<grid, 256, static_cast<size_t>(mw) * 4, st>>>(ua, idx, flag, T, ulimit);
      attn_union_compact_kernel<<<1, 1024, 0, st>>>(flag, s.BH() * skip_tiles, union_min, tlist, tcount);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    ProfScope ps("attn_union", st);
    auto go = [&](auto kern) {
      if (ulds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                  hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(ulds));
      // persistent workgroups: as many as are resident at once
      int per_cu = 0;
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kUnionWaves * 64, ulds) != hipSuccess ||
          per_cu < 1)
        per_cu = 1;
      const unsigned ugrid = static_cast<unsigned>(std::min(s.BH() * skip_tiles, per_cu * kDeviceCUs));
      kern<<<ugrid, kUnionWaves * 64, ulds, st>>>(ua, static_cast<const uint16_t*>(q),
                                                  static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), idx,
                                                  static_cast<uint16_t*>(o), lse, tlist, tcount, nullptr, nullptr, 0, 0);
    };
    auto by_g = [&](auto k1, auto k2, auto k4, auto k8, auto k16) {
      switch (s.G) {
        case 1: go(k1); break;
        case 2: go(k2); break;
        case 4: go(k4); break;
        case 8: go(k8); break;
        default: go(k16); break;
      }
    };
#define PISA_UNION(CT) \
    by_g(attn_union_kernel<D, CT, 1, false>, attn_union_kernel<D, CT, 2, false>, attn_union_kernel<D, CT, 4, false>, \
         attn_union_kernel<D, CT, 8, false>, attn_union_kernel<D, CT, 16, false>)
    if (s.C == 32) PISA_UNION(1);
    else if (s.C == 64) PISA_UNION(2);
    else if (s.C == 96) PISA_UNION(3);
    else PISA_UNION(4);
#undef PISA_UNION
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  for (int row0 = 0; row0 < s.Nq; row0 += ch) {
    const int nrows = std::min(ch, s.Nq - row0);
    // Causal: each row's first, previous and own block are attended per leaf
    // block by attn_local_kernel, which also merges the other partials.
    const bool local = s.causal != 0;
    ClusterArgs ca{idx, nullptr, s.K, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], local ? kClusterAttnFar : kClusterAttn,
                   row0, nrows, s.g, skip, skip_shift, skip_tiles};
    ClusterOut co{};
    if ((e = launch_cluster(ca, s.BH(), base + w.cl, &co, st, kAttnChunk)) != hipSuccess) return e;
    AttnBlockArgs a{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], row0, nrows,
                    kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv, skip, skip_shift, skip_tiles};
    {
      ProfScope ps("attn_block", st);
      dim3 grid(static_cast<unsigned>(
          cluster_max_chunks(s.BH(), geo.M[1], static_cast<int64_t>(s.BH()) * nrows * s.K, kAttnChunk)));
      const uint16_t* qq = static_cast<const uint16_t*>(q);
      const uint16_t* kk = static_cast<const uint16_t*>(k);
      const uint16_t* vv = static_cast<const uint16_t*>(v);
      // Eight wavefronts share the staged block: with blocks of up to 64 keys
      // two workgroups (16 wavefronts) fit a CU, with larger blocks one.
      auto go = [&](auto kern, int nw) {
        const size_t lds = (static_cast<size_t>(s.C) * (D + 8) + static_cast<size_t>(D) * (s.C + 4) +
                            static_cast<size_t>(nw) * 16 * (D + 8)) * 2;
        if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        kern<<<grid, nw * 64, lds, st>>>(a, qq, kk, vv, co.offs, co.toffs, co.ncl, co.pairs, part_o, part_lse);
      };
      if (s.C == 32)
        go(attn_block16_kernel<D, 1, kAttnBlockWaves>, kAttnBlockWaves);
      else if (s.C == 64)
        go(attn_block16_kernel<D, 2, kAttnBlockWaves>, kAttnBlockWaves);
      else if (s.C == 96)
        go(attn_block16_kernel<D, 3, kAttnBlockWaves>, kAttnBlockWaves);
      else
        go(attn_block16_kernel<D, 4, kAttnBlockWaves>, kAttnBlockWaves);
    }
    // With several heads per KV head, the row tiles of this chunk that the
    // union kernel did not take go through its LOCAL mode: the forced blocks
    // staged once per tile for every head, then the far partials merged.
    const int lT = union_ok(s) ? kLocalWaves * kUnionGroups * 16 / s.G : 0;
    const size_t llds = static_cast<size_t>(4) * s.C * D * 2 +
                        (static_cast<size_t>(2) * mw + kUnionMaxU + static_cast<size_t>(lT) * (kUnionMaxU / 32)) * 4;
    if (local && s.G > 1 && union_ok(s) && llds <= kUnionMaxLds && row0 % lT == 0) {
      ProfScope ps("attn_local", st);
      const int ltiles = (row0 + nrows + lT - 1) / lT - row0 / lT;
      const int lcount = s.BH() * ltiles;
      const uint16_t* qq = static_cast<const uint16_t*>(q);
      const uint16_t* kk = static_cast<const uint16_t*>(k);
      const uint16_t* vv = static_cast<const uint16_t*>(v);
      auto go = [&](auto kern) {
        if (llds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                    hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(llds));
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kLocalWaves * 64, llds) != hipSuccess ||
            per_cu < 1)
          per_cu = 1;
        const unsigned lgrid = static_cast<unsigned>(std::min(lcount, per_cu * kDeviceCUs));
        kern<<<lgrid, kLocalWaves * 64, llds, st>>>(a, qq, kk, vv, idx, static_cast<uint16_t*>(o), lse, nullptr,
                                                    nullptr, part_o, part_lse, ltiles, lcount);
      };
      auto by_g = [&](auto k2, auto k4, auto k8, auto k16) {
        switch (s.G) {
          case 2: go(k2); break;
          case 4: go(k4); break;
          case 8: go(k8); break;
          default: go(k16); break;
        }
      };
#define PISA_LOCAL(CT) \
      by_g(attn_union_kernel<D, CT, 2, true>, attn_union_kernel<D, CT, 4, true>, attn_union_kernel<D, CT, 8, true>, \
           attn_union_kernel<D, CT, 16, true>)
      if (s.C == 32) PISA_LOCAL(1);
      else if (s.C == 64) PISA_LOCAL(2);
      else if (s.C == 96) PISA_LOCAL(3);
      else PISA_LOCAL(4);
#undef PISA_LOCAL
    } else if (local) {
      ProfScope ps("attn_local", st);
      const int tq0 = s.N - s.Nq;
      const int nblk = (tq0 + row0 + nrows - 1) / s.C - (tq0 + row0) / s.C + 1;
      dim3 grid(static_cast<unsigned>(nblk), s.BH());
      // one key block staged, or (later) the wavefronts' 16 row states; blocks
      // of 128 keys give every one of eight wavefronts one 16-row group, so
      // that each shared block is staged once per query head
      const int nwl = s.C == 128 ? 8 : 4;
      const size_t lds = std::max((static_cast<size_t>(s.C) * (D + 8) + static_cast<size_t>(D) * (s.C + 4)) * 2,
                                  static_cast<size_t>(nwl) * (16 * (D + 4) + 32) * 4);
      const uint16_t* qq = static_cast<const uint16_t*>(q);
      const uint16_t* kk = static_cast<const uint16_t*>(k);
      const uint16_t* vv = static_cast<const uint16_t*>(v);
      auto go = [&](auto kern) {
        if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        kern<<<grid, nwl * 64, lds, st>>>(a, qq, kk, vv, idx, part_o, part_lse, static_cast<uint16_t*>(o), lse);
      };
      if (s.C == 32)
        go(attn_local_kernel<D, 1, 4>);
      else if (s.C == 64)
        go(attn_local_kernel<D, 2, 4>);
      else if (s.C == 96)
        go(attn_local_kernel<D, 3, 4>);
      else
        go(attn_local_kernel<D, 4, 8>);
      if (s.K > 32) {  // attn_local_kernel merges the first 32 slots
        if ((e = hipGetLastError()) != hipSuccess) return e;
        dim3 tgrid((nrows + 3) / 4, s.B * s.H);
        attn_combine_kernel<D, true><<<tgrid, 256, 0, st>>>(a, idx, part_o, part_lse, static_cast<uint16_t*>(o), lse);
      }
    } else {
      ProfScope ps("attn_combine", st);
      dim3 grid((nrows + 3) / 4, s.B * s.H);
      attn_combine_kernel<D, false><<<grid, 256, 0, st>>>(a, idx, part_o, part_lse, static_cast<uint16_t*>(o), lse);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attention(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                            const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st) {
  if (use_block_path(s, geo)) {
    return s.D == 128 ? launch_block_path<128>(s, geo, q, k, v, idx, o, lse, ws, st)
                      : launch_block_path<64>(s, geo, q, k, v, idx, o, lse, ws, st);
  }
  if (use_split_path(s, geo)) {
    return s.D == 128 ? launch_split_path<128>(s, q, k, v, idx, o, lse, ws, st)
                      : launch_split_path<64>(s, q, k, v, idx, o, lse, ws, st);
  }
  AttnArgs a{q, k, v, idx, o, lse, s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal,
             kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv};
  ProfScope ps("attn_rows", st);
  if (s.bf16) {
    if (s.D == 128)
      launch_rows_team<uint16_t, 128>(s, a, st);
    else
      launch_rows_team<uint16_t, 64>(s, a, st);
  } else {
    if (s.D == 128)
      launch_rows_team<float, 128>(s, a, st);
    else
      launch_rows_team<float, 64>(s, a, st);
  }
  return hipGetLastError();
}

}  // namespace pisa

extern "C" int pisa_attn_union_min_tiles(int32_t n) {
  return pisa::g_union_min_tiles.exchange(n < 0 ? -1 : n);
}
