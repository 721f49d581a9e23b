// Block-selection quality diagnostic (Sec. 4 "Block-selection quality", eq.
// oracle_metrics; App. C "Block-selection diagnostic", eq. oracle_block_mass).
//
// quality_mass_kernel: the log mass a(B) = log sum_{j in B, j <= t}
// exp(q.k_j / sqrt(d)) of every eligible leaf block B for every listed query
// row and query head, from the raw keys.  A workgroup owns 64 (row, head)
// columns and a chunk of key blocks; each block's keys are staged in LDS
// once and every wavefront scores its 16 columns against them on
// v_mfma_f32_16x16x32_bf16 (S^T = K q^T, as in the attention kernels), then
// reduces each column's masked logits to their log-sum-exp.
//
// quality_rank_kernel: one workgroup per (KV head, listed row).  P(B) is the
// mean over the group's heads of each head's softmax of a(B) over the
// eligible blocks; the reference set is the forced blocks plus the eligible
// blocks of highest P (ties to the smaller index), found by repeated
// workgroup arg-max; the selection's Recall@K, captured mass and mass ratio
// follow.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pisa {

typedef __bf16 bf16x8q __attribute__((ext_vector_type(8)));
typedef float f32x4q __attribute__((ext_vector_type(4)));

constexpr int kQualCols = 64;     // (row, head) columns per workgroup of the mass kernel
constexpr int kQualBlocks = 32;   // key blocks per workgroup of the mass kernel
constexpr int kQualMaxM1 = 16384; // leaf blocks the rank kernel holds in LDS

__device__ __forceinline__ bf16x8q u4_as_bf16x8q(uint4 r) { return __builtin_bit_cast(bf16x8q, r); }

template <int D, int CT>
__global__ __launch_bounds__(256) void quality_mass_kernel(QualityArgs a, const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const int32_t* __restrict__ rows,
                                                           float* __restrict__ mass) {
  constexpr int KS = D / 32;
  constexpr int LDK = D + 8;
  constexpr int C = CT * 32;
  constexpr int MT = C / 16;
  __shared__ __align__(16) uint16_t klds[C * LDK];
  __shared__ int cmax_w[4];

  const int bh = blockIdx.z;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int64_t ncols = static_cast<int64_t>(a.n_rows) * a.G;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * kQualCols + wave * 16 + col;  // this lane's column
  const bool vj = j < ncols;
  const int ri = vj ? static_cast<int>(j / a.G) : 0;
  const int hh = vj ? static_cast<int>(j - static_cast<int64_t>(ri) * a.G) : 0;
  const int r = vj ? rows[ri] : 0;
  const bool vr = vj && r >= 0 && r < a.Nq;  // rows outside [0, Nq) are skipped (their output stays NaN)
  const int t = a.N - a.Nq + (vr ? r : 0);
  const int nE = !vr ? 0 : (a.causal ? min(t / a.C + 1, a.M1) : a.M1);  // eligible blocks of the column

  // the largest eligible count among the workgroup's columns bounds the blocks visited
  int ne = nE;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ne = max(ne, __shfl_xor(ne, o));
  if (lane == 0) cmax_w[wave] = ne;
  __syncthreads();
  const int ne_wg = max(max(cmax_w[0], cmax_w[1]), max(cmax_w[2], cmax_w[3]));
  const int blk0 = blockIdx.y * kQualBlocks;
  const int blk1 = min(blk0 + kQualBlocks, ne_wg);

  bf16x8q qb[KS];
  {
    const uint16_t* qrow =
        q + ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + (vr ? r : 0)) * D + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qb[ks] = u4_as_bf16x8q(*reinterpret_cast<const uint4*>(qrow + ks * 32));
  }
  float* out = mass + (static_cast<int64_t>(bh) * ncols + (vj ? j : 0)) * a.M1;

  for (int blk = blk0; blk < blk1; ++blk) {
    const int r0 = blk * C;
    const int nkeys = min(C, a.N - r0);
    __syncthreads();  // the previous block's readers are done
    const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
    for (int e = threadIdx.x; e < C * (D / 8); e += 256) {
      const int rr = e / (D / 8), c8 = (e - rr * (D / 8)) * 8;
      uint4 kv = make_uint4(0, 0, 0, 0);
      if (rr < nkeys) kv = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(rr) * D + c8);
      *reinterpret_cast<uint4*>(klds + rr * LDK + c8) = kv;
    }
    __syncthreads();
    const int kmax = blk >= nE ? 0 : (a.causal ? min(nkeys, t - r0 + 1) : nkeys);
    float sv[MT][4];
    float m = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      f32x4q acc = {0.f, 0.f, 0.f, 0.f};
      const uint16_t* arow = klds + (mt * 16 + col) * LDK + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8q av = u4_as_bf16x8q(*reinterpret_cast<const uint4*>(arow + ks * 32));
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qb[ks], acc, 0, 0, 0);
      }
      // acc[i]: key mt*16 + 4*grp + i of column `col`
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = mt * 16 + 4 * grp + i;
        sv[mt][i] = key < kmax ? acc[i] * a.qscale2 : -INFINITY;
        m = fmaxf(m, sv[mt][i]);
      }
    }
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    const float msafe = m == -INFINITY ? 0.f : m;
    float s = 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s += fast_exp2(sv[mt][i] - msafe);
    s += __shfl_xor(s, 16);
    s += __shfl_xor(s, 32);
    if (vr && grp == 0 && blk < nE) out[blk] = (m + fast_log2(s)) * kLn2;
  }
}

// Workgroup arg-max of (value desc, index asc) over the 256 threads.
__device__ __forceinline__ void wg_argmax(float& v, int& i, float* sv, int* si) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float v2 = __shfl_xor(v, o);
    const int i2 = __shfl_xor(i, o);
    if (v2 > v || (v2 == v && i2 < i)) {
      v = v2;
      i = i2;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = v;
    si[wave] = i;
  }
  __syncthreads();
  v = sv[0];
  i = si[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) {
    if (sv[w] > v || (sv[w] == v && si[w] < i)) {
      v = sv[w];
      i = si[w];
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(256) void quality_rank_kernel(QualityArgs a, const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ rows,
                                                           const float* __restrict__ mass,
                                                           float* __restrict__ metrics, int32_t* __restrict__ ref) {
  extern __shared__ __align__(16) float P[];                                  // [M1] grouped mass
  uint8_t* taken = reinterpret_cast<uint8_t*>(P + a.M1);        // [M1] in the reference set
  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ int kept[64];
  const int ri = blockIdx.x;
  const int bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t orow = static_cast<int64_t>(bh) * a.n_rows + ri;
  const int r = rows[ri];
  if (r < 0 || r >= a.Nq) {  // not a query row: NaN metrics, empty reference
    if (tid < 3) metrics[orow * 3 + tid] = __builtin_nanf("");
    if (ref)
      for (int s = tid; s < a.K; s += 256) ref[orow * a.K + s] = -1;
    return;
  }
  const int t = a.N - a.Nq + r;
  const int c = t / a.C;
  const int nE = a.causal ? min(c + 1, a.M1) : a.M1;
  for (int B = tid; B < nE; B += 256) {
    P[B] = 0.f;
    taken[B] = 0;
  }
  __syncthreads();
  const int64_t ncols = static_cast<int64_t>(a.n_rows) * a.G;
  for (int hh = 0; hh < a.G; ++hh) {
    const float* am = mass + (static_cast<int64_t>(bh) * ncols + static_cast<int64_t>(ri) * a.G + hh) * a.M1;
    float mx = -INFINITY;
    int dummy = 0;
    for (int B = tid; B < nE; B += 256) mx = fmaxf(mx, am[B]);
    wg_argmax(mx, dummy, sv, si);
    const float msafe = mx == -INFINITY ? 0.f : mx;
    float sm = 0.f;
    for (int B = tid; B < nE; B += 256) sm += expf(am[B] - msafe);
    float tot = sm;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) tot += __shfl_xor(tot, o);
    if ((tid & 63) == 0) sv[tid >> 6] = tot;
    __syncthreads();
    tot = sv[0] + sv[1] + sv[2] + sv[3];
    __syncthreads();
    const float inv = tot > 0.f ? 1.f / (tot * a.G) : 0.f;
    for (int B = tid; B < nE; B += 256) P[B] += expf(am[B] - msafe) * inv;
    __syncthreads();
  }
  // Reference set: every eligible block when at most K, else the forced
  // blocks and the best of the rest by P.
  int nref = 0;
  if (nE <= a.K) {
    for (int B = tid; B < nE; B += 256) taken[B] = 1;
    if (tid < nE) kept[tid] = tid;
    nref = nE;
  } else {
    int nf = 0;
    if (a.causal) {
      const int f[3] = {0, c - 1, c};
      for (int x = 0; x < 3; ++x) {
        const int B = f[x];
        if (B < 0 || B >= nE) continue;
        bool dup = false;
        for (int y = 0; y < x; ++y) dup |= f[y] == B;
        if (dup) continue;
        if (tid == 0) {
          taken[B] = 1;
          kept[nf] = B;
        }
        ++nf;
      }
    }
    __syncthreads();
    nref = a.K;
    for (int n = nf; n < a.K; ++n) {
      float v = -INFINITY;
      int bi = 0x7fffffff;
      for (int B = tid; B < nE; B += 256) {
        const float x = taken[B] ? -INFINITY : P[B];
        if (!taken[B] && (x > v || (x == v && B < bi))) {
          v = x;
          bi = B;
        }
      }
      wg_argmax(v, bi, sv, si);
      if (tid == 0) {
        taken[bi] = 1;
        kept[n] = bi;
      }
      __syncthreads();
    }
  }
  __syncthreads();
  if (tid == 0) {
    // the selection's captured mass and overlap with the reference
    const int32_t* sel = idx + (static_cast<int64_t>(bh) * a.Nq + r) * a.K;
    float cap = 0.f, refm = 0.f;
    int hit = 0;
    for (int s = 0; s < a.K; ++s) {
      const int B = sel[s];
      if (B < 0 || B >= nE) continue;
      bool dup = false;
      for (int y = 0; y < s; ++y) dup |= sel[y] == B;
      if (dup) continue;
      cap += P[B];
      hit += taken[B];
    }
    for (int n = 0; n < nref; ++n) refm += P[kept[n]];
    metrics[orow * 3 + 0] = static_cast<float>(hit) / static_cast<float>(a.K);
    metrics[orow * 3 + 1] = cap;
    metrics[orow * 3 + 2] = refm > 0.f ? cap / refm : 0.f;
    if (ref) {
      // ascending (insertion sort of at most K entries)
      for (int x = 1; x < nref; ++x) {
        const int v = kept[x];
        int y = x - 1;
        while (y >= 0 && kept[y] > v) {
          kept[y + 1] = kept[y];
          --y;
        }
        kept[y + 1] = v;
      }
      for (int s = 0; s < a.K; ++s) ref[orow * a.K + s] = s < nref ? kept[s] : -1;
    }
  }
}

size_t quality_ws(const Shape& s, int n_rows) {
  const size_t m1 = static_cast<size_t>((s.N + s.C - 1) / s.C);
  return static_cast<size_t>(s.BH()) * n_rows * s.G * m1 * 4;
}

bool quality_supported(const Shape& s) {
  const int m1 = (s.N + s.C - 1) / s.C;
  return s.bf16 && (s.C == 32 || s.C == 64 || s.C == 96 || s.C == 128) && m1 <= kQualMaxM1 && s.K <= 64;
}

hipError_t launch_quality(const Shape& s, const void* q, const void* k, const int32_t* idx, const int32_t* rows,
                          int n_rows, float* metrics, int32_t* ref, void* ws, hipStream_t st) {
  float* mass = static_cast<float*>(ws);
  QualityArgs a{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, (s.N + s.C - 1) / s.C, n_rows,
                kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv};
  // never-written entries (blocks past a row's eligible range) are never read
  const int64_t ncols = static_cast<int64_t>(n_rows) * s.G;
  {
    ProfScope ps("quality_mass", st);
    dim3 grid(static_cast<unsigned>((ncols + kQualCols - 1) / kQualCols),
              static_cast<unsigned>((a.M1 + kQualBlocks - 1) / kQualBlocks), s.BH());
    const uint16_t* qq = static_cast<const uint16_t*>(q);
    const uint16_t* kk = static_cast<const uint16_t*>(k);
    auto go = [&](auto kern) { kern<<<grid, 256, 0, st>>>(a, qq, kk, rows, mass); };
    if (s.D == 128) {
      if (s.C == 32) go(quality_mass_kernel<128, 1>);
      else if (s.C == 64) go(quality_mass_kernel<128, 2>);
      else if (s.C == 96) go(quality_mass_kernel<128, 3>);
      else go(quality_mass_kernel<128, 4>);
    } else {
      if (s.C == 32) go(quality_mass_kernel<64, 1>);
      else if (s.C == 64) go(quality_mass_kernel<64, 2>);
      else if (s.C == 96) go(quality_mass_kernel<64, 3>);
      else go(quality_mass_kernel<64, 4>);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    ProfScope ps("quality_rank", st);
    const size_t lds = static_cast<size_t>(a.M1) * 5;
    if (lds > 65536)
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(quality_rank_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    dim3 grid(static_cast<unsigned>(n_rows), s.BH());
    quality_rank_kernel<<<grid, 256, lds, st>>>(a, idx, rows, mass, metrics, ref);
  }
  return hipGetLastError();
}

}  // namespace pisa
