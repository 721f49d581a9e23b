// Grouping of (query row, slot) pairs by key block, the "query clustering"
// step of the two-stage design (Sec. 3.3, Stage 2), shared by the leaf
// scorer and the block-centric attention.
//
// A workgroup owns a chunk of rows of one (batch, KV head) and builds an LDS
// histogram of the blocks its pairs reference; only the non-zero bins reach
// global memory: one atomic per bin per chunk adds the chunk's count to the
// bin's total and returns the chunk's offset inside the bin, which is kept
// (one row of bins per chunk).  An exclusive scan turns the totals into
// cluster offsets; the scatter pass starts each bin at its cluster offset
// plus the chunk's offset and places each pair with an LDS atomic inside that
// range.  The order of pairs inside a cluster is therefore not fixed, which
// no consumer depends on (every pair is processed on its own).
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pisa {

constexpr int kClusterThreads = 1024;
constexpr int kClusterRows = 1024;  // rows per workgroup chunk

__device__ __forceinline__ bool cluster_pair(const ClusterArgs& a, int bh, int r, int slot, int& blk) {
  const int64_t rg = static_cast<int64_t>(bh) * a.Nq + a.row0 + r;
  const int32_t* lst = a.list + rg * a.S;
  blk = lst[slot];
  if (blk < 0) return false;
  // attention lists come from the caller: entries past the last leaf block
  // are padding, like negative ones (the bins cover blocks 0 .. M1-1 only)
  if ((a.mode == kClusterAttn || a.mode == kClusterAttnFar) && blk >= a.M1) return false;
  if (a.skip && a.skip[static_cast<int64_t>(bh) * a.skip_tiles + ((a.row0 + r) >> a.skip_shift)]) return false;
  if (a.mode == kClusterAttnFar) {
    const int c = (a.N - a.Nq + a.row0 + r) / a.C;
    return !(a.causal && (blk == 0 || blk == c || blk == c - 1));
  }
  if (a.mode == kClusterLeaf || a.mode == kClusterLeafParent) {
    const int n = a.cnt[rg];
    if (slot >= n || n <= a.K) return false;
    const int c = (a.N - a.Nq + a.row0 + r) / a.C;
    auto forced = [&](int x) { return a.causal && (x == 0 || x == c || x == c - 1); };
    if (forced(blk)) return false;
    if (a.mode == kClusterLeafParent) {
      // the candidate list is ascending, so siblings are adjacent: emit only
      // at the first non-forced child of the parent
      const int par = blk / a.g;
      for (int i = 1; i < a.g && slot - i >= 0; ++i) {
        const int o = lst[slot - i];
        if (o / a.g != par) break;
        if (!forced(o)) return false;
      }
      blk = par;
    }
  }
  return true;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(int32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < n; i += 256LL * gridDim.x) p[i] = 0;
}

__global__ __launch_bounds__(kClusterThreads) void cluster_hist_kernel(ClusterArgs a, int32_t* __restrict__ hist,
                                                                       int32_t* __restrict__ chunk_base) {
  extern __shared__ __align__(16) int32_t h[];
  const int bh = blockIdx.y;
  const int r0 = blockIdx.x * kClusterRows;
  const int nr = min(kClusterRows, a.nrows - r0);
  for (int i = threadIdx.x; i < a.M1; i += kClusterThreads) h[i] = 0;
  __syncthreads();
  const int npairs = nr * a.S;
  for (int e = threadIdx.x; e < npairs; e += kClusterThreads) {
    const int r = r0 + e / a.S, slot = e % a.S;
    int blk;
    if (cluster_pair(a, bh, r, slot, blk)) atomicAdd(&h[blk], 1);
  }
  __syncthreads();
  int32_t* gh = hist + static_cast<int64_t>(bh) * a.M1;
  int32_t* cb = chunk_base + (static_cast<int64_t>(bh) * gridDim.x + blockIdx.x) * a.M1;
  for (int i = threadIdx.x; i < a.M1; i += kClusterThreads) {
    const int n = h[i];
    cb[i] = n ? atomicAdd(&gh[i], n) : 0;  // this chunk's offset inside bin i
  }
}

// Exclusive scans of the n counts into offs[0..n] (pair offsets) and of
// their tile counts ceil(count / tile) into toffs[0..n].
// Each thread owns a contiguous run of the counts; runs of up to kScanRun
// are read into registers with independent loads.
constexpr int kScanRun = 32;

__global__ __launch_bounds__(1024) void cluster_scan_kernel(const int32_t* __restrict__ hist,
                                                            int32_t* __restrict__ offs,
                                                            int32_t* __restrict__ toffs, int64_t n, int tile) {
  __shared__ int wsum[16], wtile[16];
  const int tid = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t i0 = min(n, tid * per), i1 = min(n, i0 + per);
  const int cnt = static_cast<int>(i1 - i0);
  const bool inreg = per <= kScanRun;
  int v[kScanRun];
  int local = 0, ltile = 0;
  if (inreg) {
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) v[j] = j < cnt ? hist[i0 + j] : 0;
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) {
      local += v[j];
      ltile += (v[j] + tile - 1) / tile;
    }
  } else {
    for (int64_t i = i0; i < i1; ++i) {
      const int c = hist[i];
      local += c;
      ltile += (c + tile - 1) / tile;
    }
  }
  const int lane = tid & 63, w = tid >> 6;
  int x = local, y = ltile;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int xs = __shfl_up(x, o), ys = __shfl_up(y, o);
    if (lane >= o) {
      x += xs;
      y += ys;
    }
  }
  if (lane == 63) {
    wsum[w] = x;
    wtile[w] = y;
  }
  __syncthreads();
  int pre = 0, tot = 0, tpre = 0, ttot = 0;
  for (int i = 0; i < 16; ++i) {
    pre += (i < w) ? wsum[i] : 0;
    tot += wsum[i];
    tpre += (i < w) ? wtile[i] : 0;
    ttot += wtile[i];
  }
  int run = pre + x - local, trun = tpre + y - ltile;
  if (inreg) {
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) {
      if (j < cnt) {
        offs[i0 + j] = run;
        toffs[i0 + j] = trun;
      }
      run += v[j];
      trun += (v[j] + tile - 1) / tile;
    }
  } else {
    for (int64_t i = i0; i < i1; ++i) {
      const int c = hist[i];
      offs[i] = run;
      toffs[i] = trun;
      run += c;
      trun += (c + tile - 1) / tile;
    }
  }
  if (tid == 0) {
    offs[n] = tot;
    toffs[n] = ttot;
  }
}

// The same scans with the counts staged through LDS (n <= kScanLdsMax): the
// counts are read and the offsets written with coalesced accesses, and each
// thread's run is read from LDS (one pad word per 16 keeps the runs on
// distinct banks) instead of as strided global loads.
constexpr int kScanLdsMax = 17408;
__host__ __device__ __forceinline__ int scan_pad(int i) { return i + (i >> 4); }

__global__ __launch_bounds__(1024) void cluster_scan_lds_kernel(const int32_t* __restrict__ hist,
                                                                int32_t* __restrict__ offs,
                                                                int32_t* __restrict__ toffs, int n, int tile) {
  extern __shared__ __align__(16) int32_t sh[];
  __shared__ int wsum[16], wtile[16];
  int32_t* ho = sh;                       // counts, then offsets (padded)
  int32_t* ht = sh + scan_pad(n) + 1;     // tile offsets (padded)
  const int tid = threadIdx.x;
  for (int e = tid; e < n; e += 1024) ho[scan_pad(e)] = hist[e];
  __syncthreads();
  const int per = (n + 1023) / 1024;
  const int i0 = min(n, tid * per), i1 = min(n, i0 + per);
  const int cnt = i1 - i0;
  int v[kScanRun];
  int local = 0, ltile = 0;
#pragma unroll
  for (int j = 0; j < kScanRun; ++j) {
    v[j] = j < cnt ? ho[scan_pad(i0 + j)] : 0;
    local += v[j];
    ltile += (v[j] + tile - 1) / tile;
  }
  const int lane = tid & 63, w = tid >> 6;
  int x = local, y = ltile;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int xs = __shfl_up(x, o), ys = __shfl_up(y, o);
    if (lane >= o) {
      x += xs;
      y += ys;
    }
  }
  if (lane == 63) {
    wsum[w] = x;
    wtile[w] = y;
  }
  __syncthreads();
  int pre = 0, tot = 0, tpre = 0, ttot = 0;
  for (int i = 0; i < 16; ++i) {
    pre += (i < w) ? wsum[i] : 0;
    tot += wsum[i];
    tpre += (i < w) ? wtile[i] : 0;
    ttot += wtile[i];
  }
  int run = pre + x - local, trun = tpre + y - ltile;
#pragma unroll
  for (int j = 0; j < kScanRun; ++j) {
    if (j < cnt) {
      ho[scan_pad(i0 + j)] = run;
      ht[scan_pad(i0 + j)] = trun;
    }
    run += v[j];
    trun += (v[j] + tile - 1) / tile;
  }
  __syncthreads();
  for (int e = tid; e < n; e += 1024) {
    offs[e] = ho[scan_pad(e)];
    toffs[e] = ht[scan_pad(e)];
  }
  if (tid == 0) {
    offs[n] = tot;
    toffs[n] = ttot;
  }
}

__global__ __launch_bounds__(kClusterThreads) void cluster_scatter_kernel(ClusterArgs a, const int32_t* __restrict__ offs,
                                                                          const int32_t* __restrict__ chunk_base,
                                                                          int32_t* __restrict__ pairs) {
  extern __shared__ __align__(16) int32_t h[];
  const int bh = blockIdx.y;
  const int r0 = blockIdx.x * kClusterRows;
  const int nr = min(kClusterRows, a.nrows - r0);
  // bin i of this chunk starts at its cluster's offset plus the chunk's
  // offset inside the cluster (reserved by cluster_hist_kernel)
  const int32_t* go = offs + static_cast<int64_t>(bh) * a.M1;
  const int32_t* cb = chunk_base + (static_cast<int64_t>(bh) * gridDim.x + blockIdx.x) * a.M1;
  for (int i = threadIdx.x; i < a.M1; i += kClusterThreads) h[i] = go[i] + cb[i];
  __syncthreads();
  const int npairs = nr * a.S;
  for (int e = threadIdx.x; e < npairs; e += kClusterThreads) {
    const int r = r0 + e / a.S, slot = e % a.S;
    int blk;
    if (cluster_pair(a, bh, r, slot, blk)) {
      const int pos = atomicAdd(&h[blk], 1);
      pairs[pos] = (r << 8) | slot;
    }
  }
}

size_t cluster_ws(int BH, int M1, int64_t max_pairs, int max_rows) {
  const size_t ncl = static_cast<size_t>(BH) * M1;
  const size_t nchunk = static_cast<size_t>(BH) * ((max_rows + kClusterRows - 1) / kClusterRows);
  return 3 * ((ncl + 1) * 4 + 256) + (nchunk * M1 * 4 + 256) + static_cast<size_t>(max_pairs) * 4 + 256;
}

int64_t cluster_max_chunks(int BH, int M1, int64_t max_pairs, int tile) {
  return (max_pairs + tile - 1) / tile + static_cast<int64_t>(BH) * M1;
}

static size_t al(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

hipError_t launch_cluster(const ClusterArgs& a, int BH, void* ws, ClusterOut* out, hipStream_t st, int tile) {
  // the rows read are [row0, row0 + nrows) of [0, Nq): refuse anything else
  if (a.row0 < 0 || a.nrows < 1 || a.row0 + a.nrows > a.Nq || a.M1 < 1 || tile < 1 ||
      (a.mode == kClusterLeafParent && a.g < 2))
    return hipErrorInvalidValue;
  const int64_t ncl = static_cast<int64_t>(BH) * a.M1;
  const int nchunk = (a.nrows + kClusterRows - 1) / kClusterRows;  // row chunks per (batch, KV head)
  char* base = static_cast<char*>(ws);
  int32_t* hist = reinterpret_cast<int32_t*>(base);
  int32_t* offs = reinterpret_cast<int32_t*>(base + al((ncl + 1) * 4));
  int32_t* toffs = reinterpret_cast<int32_t*>(base + 2 * al((ncl + 1) * 4));
  int32_t* chunk_base = reinterpret_cast<int32_t*>(base + 3 * al((ncl + 1) * 4));
  int32_t* pairs = reinterpret_cast<int32_t*>(base + 3 * al((ncl + 1) * 4) +
                                              al(static_cast<size_t>(BH) * nchunk * a.M1 * 4));
  out->offs = offs;
  out->toffs = toffs;
  out->pairs = pairs;
  out->ncl = ncl;
  ProfScope ps("cluster_build", st);
  fill_zero_kernel<<<static_cast<unsigned>(std::min<int64_t>((ncl + 255) / 256, 4096)), 256, 0, st>>>(hist, ncl);
  dim3 grid(nchunk, BH);
  const size_t lds = static_cast<size_t>(a.M1) * 4;
  cluster_hist_kernel<<<grid, kClusterThreads, lds, st>>>(a, hist, chunk_base);
  if (ncl <= kScanLdsMax) {
    const size_t slds = 2 * (static_cast<size_t>(scan_pad(static_cast<int>(ncl))) + 1) * sizeof(int32_t);
    if (slds > 65536)
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(cluster_scan_lds_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(slds));
    cluster_scan_lds_kernel<<<1, 1024, slds, st>>>(hist, offs, toffs, static_cast<int>(ncl), tile);
  } else {
    cluster_scan_kernel<<<1, 1024, 0, st>>>(hist, offs, toffs, ncl, tile);
  }
  cluster_scatter_kernel<<<grid, kClusterThreads, lds, st>>>(a, offs, chunk_base, pairs);
  return hipGetLastError();
}

}  // namespace pisa
