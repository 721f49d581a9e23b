// Mean pyramid construction (Sec. 3.2, eq. mean_pyramid).
//
// pool_leaf_kernel streams K once: a workgroup owns a run of LPB = g^s
// consecutive leaf blocks of one (batch, KV head), computes their level-1
// means with 16-byte coalesced loads (16 lanes cover one key row), then the
// s coarser levels whose nodes lie inside that run, from LDS.  pool_top_kernel
// finishes the few remaining levels (at most M_1 / LPB rows) with one
// workgroup per (batch, KV head).  All accumulation is float32; every node is
// the mean of its existing children (the last node of a level may be short).
#include "common.h"
#include "kernels.h"

namespace pisa {

template <typename T, int D>
__global__ __launch_bounds__(256) void pool_leaf_kernel(const T* __restrict__ k, float* __restrict__ pyr,
                                                        Geo geo, int s_levels, int lpb) {
  constexpr int DPL = D / 16;
  extern __shared__ float lds[];  // two buffers of LPB * D floats
  float* buf0 = lds;
  float* buf1 = lds + lpb * D;

  const int bh = blockIdx.y;
  const int leaf0 = blockIdx.x * lpb;
  const int nleaf = min(lpb, geo.M[1] - leaf0);
  const T* kb = k + static_cast<int64_t>(bh) * geo.N * D;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int sub = lane & 15;   // column slice of the row
  const int rg = lane >> 4;    // row group 0..3

  for (int lf = wave; lf < nleaf; lf += 4) {
    const int leaf = leaf0 + lf;
    const int64_t row0 = static_cast<int64_t>(leaf) * geo.C;
    const int nrows = min(geo.C, geo.N - static_cast<int>(row0));
    float acc[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
    const T* base = kb + row0 * D + sub * DPL;
    int r = rg;
    for (; r + 12 < nrows; r += 16) {
      float x0[DPL], x1[DPL], x2[DPL], x3[DPL];
      load_row_part<T, DPL>(base + static_cast<int64_t>(r) * D, x0);
      load_row_part<T, DPL>(base + static_cast<int64_t>(r + 4) * D, x1);
      load_row_part<T, DPL>(base + static_cast<int64_t>(r + 8) * D, x2);
      load_row_part<T, DPL>(base + static_cast<int64_t>(r + 12) * D, x3);
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] += (x0[e] + x1[e]) + (x2[e] + x3[e]);
    }
    for (; r < nrows; r += 4) {
      float x0[DPL];
      load_row_part<T, DPL>(base + static_cast<int64_t>(r) * D, x0);
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] += x0[e];
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      acc[e] += __shfl_xor(acc[e], 16);
      acc[e] += __shfl_xor(acc[e], 32);
    }
    if (rg == 0) {
      const float inv = 1.0f / static_cast<float>(nrows);
      float m[DPL];
#pragma unroll
      for (int e = 0; e < DPL; ++e) m[e] = acc[e] * inv;
      float* dst = pb + (geo.off[1] + leaf) * D + sub * DPL;
      float* ldst = buf0 + lf * D + sub * DPL;
#pragma unroll
      for (int e = 0; e < DPL; e += 4) {
        float4 v4 = make_float4(m[e], m[e + 1], m[e + 2], m[e + 3]);
        *reinterpret_cast<float4*>(dst + e) = v4;
        *reinterpret_cast<float4*>(ldst + e) = v4;
      }
    }
  }
  __syncthreads();

  // Coarser levels whose nodes lie inside this run of leaves.
  const int top = min(s_levels + 1, geo.Lstore);
  float* src = buf0;
  float* dstb = buf1;
  for (int lv = 2; lv <= top; ++lv) {
    const int g = geo.g;
    const int first = anc_at(geo, leaf0, lv);  // node index of the run start
    const int below_first = anc_at(geo, leaf0, lv - 1);
    const int nnode = min(lpb / geo.gp[lv], geo.M[lv] - first);
    for (int e = threadIdx.x; e < nnode * D; e += blockDim.x) {
      const int j = e / D, col = e - j * D;
      const int node = first + j;
      const int c0 = node * g;
      const int c1 = min(c0 + g, geo.M[lv - 1]);
      float s = 0.f;
      for (int ch = c0; ch < c1; ++ch) s += src[(ch - below_first) * D + col];
      const float mval = s / static_cast<float>(c1 - c0);
      dstb[j * D + col] = mval;
      pb[(geo.off[lv] + node) * D + col] = mval;
    }
    __syncthreads();
    float* tmp = src;
    src = dstb;
    dstb = tmp;
  }
}

// Levels from `first_level` to Lstore, one workgroup per (batch, KV head).
// Each level reads the level below from global memory written by this same
// workgroup (or by pool_leaf_kernel earlier on the stream).
__global__ __launch_bounds__(256) void pool_top_kernel(float* __restrict__ pyr, Geo geo, int first_level, int D) {
  const int bh = blockIdx.x;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;
  for (int lv = first_level; lv <= geo.Lstore; ++lv) {
    const int n = geo.M[lv] * D;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
      const int node = e / D, col = e - node * D;
      const int c0 = node * geo.g;
      const int c1 = min(c0 + geo.g, geo.M[lv - 1]);
      float s = 0.f;
      for (int ch = c0; ch < c1; ++ch) s += pb[(geo.off[lv - 1] + ch) * D + col];
      pb[(geo.off[lv] + node) * D + col] = s / static_cast<float>(c1 - c0);
    }
    __syncthreads();
  }
}

// s = number of coarser levels computed inside pool_leaf_kernel: the largest
// s with g^s <= 16.
static int pool_s_levels(int g) {
  int s = 0;
  int64_t p = 1;
  while (p * g <= 16) { p *= g; ++s; }
  return s;
}

hipError_t launch_build_pyramid(const Geo& geo, int BH, int D, bool bf16, const void* k, float* pyr,
                                hipStream_t st) {
  const int s = pool_s_levels(geo.g);
  int lpb = 1;
  for (int i = 0; i < s; ++i) lpb *= geo.g;
  dim3 grid((geo.M[1] + lpb - 1) / lpb, BH);
  const size_t lds = 2 * static_cast<size_t>(lpb) * D * sizeof(float);
  {
  ProfScope ps("pool_leaf", st);
  if (bf16) {
    if (D == 128)
      pool_leaf_kernel<uint16_t, 128><<<grid, 256, lds, st>>>(static_cast<const uint16_t*>(k), pyr, geo, s, lpb);
    else
      pool_leaf_kernel<uint16_t, 64><<<grid, 256, lds, st>>>(static_cast<const uint16_t*>(k), pyr, geo, s, lpb);
  } else {
    if (D == 128)
      pool_leaf_kernel<float, 128><<<grid, 256, lds, st>>>(static_cast<const float*>(k), pyr, geo, s, lpb);
    else
      pool_leaf_kernel<float, 64><<<grid, 256, lds, st>>>(static_cast<const float*>(k), pyr, geo, s, lpb);
  }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (geo.Lstore >= s + 2) {
    ProfScope ps("pool_top", st);
    pool_top_kernel<<<BH, 256, 0, st>>>(pyr, geo, s + 2, D);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace pisa
