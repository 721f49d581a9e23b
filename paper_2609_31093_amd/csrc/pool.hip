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

// Mean of leaf block `leaf` (rows [leaf*C, min((leaf+1)*C, N))) computed by
// one wavefront: 16 lanes cover a key row, the 4 row groups take every 4th
// row; lanes of row group 0 return the D/16 means of their column slice.
// Both the full build and the decode-cache update use this, so their leaf
// means agree bit for bit.
template <typename T, int D>
__device__ __forceinline__ void leaf_mean(const T* __restrict__ kb, const Geo& geo, int leaf, int sub, int rg,
                                          float (&m)[D / 16]) {
  constexpr int DPL = D / 16;
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
  const float inv = 1.0f / static_cast<float>(nrows);
#pragma unroll
  for (int e = 0; e < DPL; ++e) m[e] = acc[e] * inv;
}

// Node `node` of level lv (>= 2): the mean of its existing children, summed
// in index order; `child(ch, col)` reads column col of child ch.
template <typename F>
__device__ __forceinline__ float node_mean(const Geo& geo, int lv, int node, int col, F child) {
  const int c0 = node * geo.g;
  const int c1 = min(c0 + geo.g, geo.M[lv - 1]);
  float s = 0.f;
  for (int ch = c0; ch < c1; ++ch) s += child(ch, col);
  return s / static_cast<float>(c1 - c0);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void pool_leaf_kernel(const T* __restrict__ k, float* __restrict__ pyr,
                                                        Geo geo, int s_levels, int lpb) {
  constexpr int DPL = D / 16;
  extern __shared__ __align__(16) float lds[];  // two buffers of LPB * D floats
  float* buf0 = lds;
  float* buf1 = lds + lpb * D;

  const int bh = blockIdx.y;
  const int leaf0 = blockIdx.x * lpb;
  const int nleaf = min(lpb, geo.M[1] - leaf0);
  const T* kb = k + static_cast<int64_t>(bh) * geo.Nkv * D;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int sub = lane & 15;   // column slice of the row
  const int rg = lane >> 4;    // row group 0..3

  for (int lf = wave; lf < nleaf; lf += 4) {
    const int leaf = leaf0 + lf;
    float m[DPL];
    leaf_mean<T, D>(kb, geo, leaf, sub, rg, m);
    if (rg == 0) {
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
    const int first = anc_at(geo, leaf0, lv);  // node index of the run start
    const int below_first = anc_at(geo, leaf0, lv - 1);
    const int nnode = min(lpb / geo.gp[lv], geo.M[lv] - first);
    for (int e = threadIdx.x; e < nnode * D; e += blockDim.x) {
      const int j = e / D, col = e - j * D;
      const int node = first + j;
      const float mval = node_mean(geo, lv, node, col, [&](int ch, int cc) { return src[(ch - below_first) * D + cc]; });
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
      pb[(geo.off[lv] + node) * D + col] =
          node_mean(geo, lv, node, col, [&](int ch, int cc) { return pb[(geo.off[lv - 1] + ch) * D + cc]; });
    }
    __syncthreads();
  }
}

// The same levels with the level below first_level read into LDS once (every
// load in flight together) and each coarser level computed from LDS, so that
// the level-by-level chain does not wait on global memory; used when the two
// largest levels fit the dynamic LDS.  Same arithmetic, same results.
__global__ __launch_bounds__(1024) void pool_top_lds_kernel(float* __restrict__ pyr, Geo geo, int first_level, int D) {
  extern __shared__ __align__(16) float lds[];
  const int bh = blockIdx.x;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;
  float* src = lds;
  float* dst = lds + static_cast<int64_t>(geo.M[first_level - 1]) * D;
  {
    const int n4 = geo.M[first_level - 1] * D / 4;
    const float4* g4 = reinterpret_cast<const float4*>(pb + static_cast<int64_t>(geo.off[first_level - 1]) * D);
    for (int e = threadIdx.x; e < n4; e += blockDim.x) reinterpret_cast<float4*>(src)[e] = g4[e];
  }
  __syncthreads();
  for (int lv = first_level; lv <= geo.Lstore; ++lv) {
    const int n = geo.M[lv] * D;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
      const int node = e / D, col = e - node * D;
      const float mval = node_mean(geo, lv, node, col, [&](int ch, int cc) { return src[ch * D + cc]; });
      dst[e] = mval;
      pb[(geo.off[lv] + node) * D + col] = mval;
    }
    __syncthreads();
    float* t = src;
    src = dst;
    dst = t;
  }
}

// Decode-cache update (App. B): one workgroup per (batch, KV head).  The
// leaf blocks from c_first (the block holding row n_old) to the end are
// recomputed, then level by level the nodes from the ancestor of c_first to
// the end of the level (exactly the ancestors of the recomputed leaves), or
// the whole level where it did not exist at n_old (l > old_lstore).  Same
// arithmetic as the full build, so the result equals it bit for bit.
template <typename T, int D>
__global__ __launch_bounds__(256) void pool_append_kernel(const T* __restrict__ k, float* __restrict__ pyr, Geo geo,
                                                          int c_first, int old_lstore) {
  constexpr int DPL = D / 16;
  const int bh = blockIdx.x;
  const T* kb = k + static_cast<int64_t>(bh) * geo.Nkv * D;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane & 15, rg = lane >> 4;
  for (int leaf = c_first + wave; leaf < geo.M[1]; leaf += 4) {
    float m[DPL];
    leaf_mean<T, D>(kb, geo, leaf, sub, rg, m);
    if (rg == 0) {
      float* dst = pb + (geo.off[1] + leaf) * D + sub * DPL;
#pragma unroll
      for (int e = 0; e < DPL; e += 4)
        *reinterpret_cast<float4*>(dst + e) = make_float4(m[e], m[e + 1], m[e + 2], m[e + 3]);
    }
  }
  __syncthreads();
  for (int lv = 2; lv <= geo.Lstore; ++lv) {
    const int first = lv > old_lstore ? 0 : anc_at(geo, c_first, lv);
    const int n = (geo.M[lv] - first) * D;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
      const int node = first + e / D, col = e % D;
      pb[(geo.off[lv] + node) * D + col] =
          node_mean(geo, lv, node, col, [&](int ch, int cc) { return pb[(geo.off[lv - 1] + ch) * D + cc]; });
    }
    __syncthreads();
  }
}

// The decode case of the update: only the last leaf block changed and no
// level is new, so the changed nodes are the last node of every level and
// each one's changed child is its last child.  While wavefront 0 recomputes
// the leaf mean, the other wavefronts fetch every ancestor's unchanged
// children into LDS; then thread d walks column d up all levels on its own
// (children summed in index order, as in the full build), with no barrier
// and no dependent memory round trip per level.
template <typename T, int D>
__global__ __launch_bounds__(256) void pool_append_path_kernel(const T* __restrict__ k, float* __restrict__ pyr,
                                                               Geo geo) {
  constexpr int DPL = D / 16;
  extern __shared__ __align__(16) float lds[];  // [D] changed child, then per level (g - 1) x D siblings
  float* val = lds;
  float* sib = lds + D;
  const int bh = blockIdx.x;
  const T* kb = k + static_cast<int64_t>(bh) * geo.Nkv * D;
  float* pb = pyr + static_cast<int64_t>(bh) * geo.R * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = geo.g;
  const int leaf = geo.M[1] - 1;
  if (wave == 0) {
    const int sub = lane & 15, rg = lane >> 4;
    float m[DPL];
    leaf_mean<T, D>(kb, geo, leaf, sub, rg, m);
    if (rg == 0) {
      float* dst = pb + (geo.off[1] + leaf) * D + sub * DPL;
#pragma unroll
      for (int e = 0; e < DPL; e += 4) {
        const float4 v4 = make_float4(m[e], m[e + 1], m[e + 2], m[e + 3]);
        *reinterpret_cast<float4*>(dst + e) = v4;
        *reinterpret_cast<float4*>(val + sub * DPL + e) = v4;
      }
    }
  } else {
    // siblings of level lv's last node: children c0 .. M[lv-1]-2 at level lv-1
    for (int lv = 2; lv <= geo.Lstore; ++lv) {
      const int c0 = (geo.M[lv] - 1) * g;
      const int ns = geo.M[lv - 1] - 1 - c0;
      float* dst = sib + (lv - 2) * (g - 1) * D;
      for (int e = tid - 64; e < ns * D; e += 192) dst[e] = pb[(geo.off[lv - 1] + c0) * D + e];
    }
  }
  __syncthreads();
  if (tid < D) {
    float x = val[tid];
    for (int lv = 2; lv <= geo.Lstore; ++lv) {
      const int c0 = (geo.M[lv] - 1) * g;
      const int ns = geo.M[lv - 1] - 1 - c0;
      const float* sv = sib + (lv - 2) * (g - 1) * D + tid;
      float sum = 0.f;
      for (int j = 0; j < ns; ++j) sum += sv[j * D];
      sum += x;
      x = sum / static_cast<float>(ns + 1);
      pb[(geo.off[lv] + geo.M[lv] - 1) * D + tid] = x;
    }
  }
}

hipError_t launch_pyramid_append(const Geo& geo, const Geo& geo_old, int BH, int D, bool bf16, const void* k,
                                 float* pyr, int n_old, hipStream_t st) {
  const int c_first = n_old / geo.C;
  const int old_lstore = n_old > 0 ? geo_old.Lstore : 0;
  ProfScope ps("pool_append", st);
  if (n_old > 0 && c_first == geo.M[1] - 1 && old_lstore == geo.Lstore) {
    const size_t lds = (static_cast<size_t>(D) + static_cast<size_t>(geo.Lstore) * (geo.g - 1) * D) * sizeof(float);
    if (bf16) {
      if (D == 128)
        pool_append_path_kernel<uint16_t, 128><<<BH, 256, lds, st>>>(static_cast<const uint16_t*>(k), pyr, geo);
      else
        pool_append_path_kernel<uint16_t, 64><<<BH, 256, lds, st>>>(static_cast<const uint16_t*>(k), pyr, geo);
    } else {
      if (D == 128)
        pool_append_path_kernel<float, 128><<<BH, 256, lds, st>>>(static_cast<const float*>(k), pyr, geo);
      else
        pool_append_path_kernel<float, 64><<<BH, 256, lds, st>>>(static_cast<const float*>(k), pyr, geo);
    }
    return hipGetLastError();
  }
  if (bf16) {
    if (D == 128)
      pool_append_kernel<uint16_t, 128><<<BH, 256, 0, st>>>(static_cast<const uint16_t*>(k), pyr, geo, c_first, old_lstore);
    else
      pool_append_kernel<uint16_t, 64><<<BH, 256, 0, st>>>(static_cast<const uint16_t*>(k), pyr, geo, c_first, old_lstore);
  } else {
    if (D == 128)
      pool_append_kernel<float, 128><<<BH, 256, 0, st>>>(static_cast<const float*>(k), pyr, geo, c_first, old_lstore);
    else
      pool_append_kernel<float, 64><<<BH, 256, 0, st>>>(static_cast<const float*>(k), pyr, geo, c_first, old_lstore);
  }
  return hipGetLastError();
}

// Decode-cache capacity growth (App. B): per (batch, KV head) one stream of
// 16-byte units -- the rows of every stored level, moved from that level's
// offset in the old layout to its offset in the new one, then the first N
// rows of k and of v -- copied with coalesced vector loads and stores.
__global__ __launch_bounds__(256) void cache_grow_kernel(GrowArgs a, const uint4* __restrict__ pyr_old,
                                                         uint4* __restrict__ pyr_new, const uint4* __restrict__ k_old,
                                                         uint4* __restrict__ k_new, const uint4* __restrict__ v_old,
                                                         uint4* __restrict__ v_new) {
  const int64_t bh = blockIdx.y;
  const int64_t total = a.pyr_units + 2 * a.kv_units;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * 256) {
    if (e < a.pyr_units) {
      int l = 0;
      while (e >= a.lev_end[l]) ++l;
      const int64_t local = e - (l > 0 ? a.lev_end[l - 1] : 0);
      pyr_new[bh * a.pyr_new_stride + a.off_new[l] + local] = pyr_old[bh * a.pyr_old_stride + a.off_old[l] + local];
    } else if (e < a.pyr_units + a.kv_units) {
      const int64_t local = e - a.pyr_units;
      k_new[bh * a.kv_new_stride + local] = k_old[bh * a.kv_old_stride + local];
    } else {
      const int64_t local = e - a.pyr_units - a.kv_units;
      v_new[bh * a.kv_new_stride + local] = v_old[bh * a.kv_old_stride + local];
    }
  }
}

hipError_t launch_cache_grow(const GrowArgs& a, int BH, const float* pyr_old, float* pyr_new, const void* k_old,
                             void* k_new, const void* v_old, void* v_new, hipStream_t st) {
  const int64_t total = a.pyr_units + 2 * a.kv_units;
  // enough workgroups for ~4 units per thread, at most 65535 per head
  const int64_t per_head = (total + 1023) / 1024;
  dim3 grid(static_cast<unsigned>(per_head < 1 ? 1 : (per_head > 65535 ? 65535 : per_head)), BH);
  ProfScope ps("cache_grow", st);
  cache_grow_kernel<<<grid, 256, 0, st>>>(a, reinterpret_cast<const uint4*>(pyr_old), reinterpret_cast<uint4*>(pyr_new),
                                          static_cast<const uint4*>(k_old), static_cast<uint4*>(k_new),
                                          static_cast<const uint4*>(v_old), static_cast<uint4*>(v_new));
  return hipGetLastError();
}

constexpr size_t kPoolTopLds = 160 * 1024;  // dynamic LDS of one workgroup on a CDNA4 CU

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
    // levels s+1 (read) and s+2 (the largest computed) in LDS, the coarser
    // ones reuse the two buffers
    const size_t tlds = static_cast<size_t>(geo.M[s + 1] + geo.M[s + 2]) * D * sizeof(float);
    bool fits = tlds <= kPoolTopLds;
    if (fits && tlds > 65536) {
      fits = hipFuncSetAttribute(reinterpret_cast<const void*>(pool_top_lds_kernel),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(tlds)) == hipSuccess;
      if (!fits) (void)hipGetLastError();  // the refusal is not the caller's error
    }
    if (fits) {
      pool_top_lds_kernel<<<BH, 1024, tlds, st>>>(pyr, geo, s + 2, D);
    } else {
      pool_top_kernel<<<BH, 256, 0, st>>>(pyr, geo, s + 2, D);
    }
    e = hipGetLastError();
  }
  return e;
}

}  // namespace pisa
