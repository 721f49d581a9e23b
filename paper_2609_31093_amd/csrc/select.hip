// Pyramid Top-K block selection (Sec. 3.2 eqs. hierarchical_topk,
// direct_child_lse; Sec. 3.3 eq. kernel_grouped_score and the two kernel
// designs; App. B causal policy).
//
// select_kernel<..., FUSED>: a "team" (one wavefront, or a whole 256-thread
// workgroup for latency-bound decode) owns one (query row, KV head).  It keeps
// the candidate set A in LDS and walks the levels from the root down:
//   * |A| <= K: keep everything, no scores;
//   * otherwise score each non-forced candidate: 16-lane groups compute the
//     scaled child logits (16-byte loads of one fp32 summary row or one raw
//     key row per group, wave-shuffle dot reduction), the group's heads' LSEs
//     are summed, candidates are ranked by (score desc, index asc) and the
//     forced ones plus the best K - |F| survive;
//   * survivors expand to their eligible children (team prefix sum).
// FUSED = true continues to the leaf level (raw keys, online LSE) and writes
// the final indices; FUSED = false stops after level 2 and stores A^(1).
//
// Two-stage remainder (bf16): cluster_* kernels group the (query, candidate
// leaf) pairs by leaf block (histogram, scan, scatter); leaf_score_kernel
// stages one key block in LDS and scores 32 queries per MFMA tile
// (v_mfma_f32_32x32x16_bf16, keys along M, queries along N, fp32 accumulate);
// final_topk_kernel ranks each row's scored leaf candidates.
//
// Scores are kept in log2 units internally (q pre-scaled by log2(e)/sqrt(d),
// hardware exp2/log2); the ranking is unchanged and exported scores are
// converted back to natural log.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pisa {

struct SelArgs {
  Geo geo;
  const void* q;
  const void* k;
  const float* pyr;
  int32_t* idx;     // fused: [BH, Nq, K]
  float* score;     // fused: [BH, Nq, K] or null
  int32_t* a1;      // stage 1: [BH, Nq, gK]
  int32_t* a1cnt;   // stage 1: [BH, Nq]
  int H, Hkv, G, Nq, K, causal, gK;
  float qscale2;    // log2(e) / sqrt(d)
};

template <int TEAM>
__device__ __forceinline__ void team_sync() {
  if constexpr (TEAM == 64) {
    wave_sync();
  } else {
    __syncthreads();
  }
}

// Exclusive prefix sum of one int per team thread; returns the prefix and the
// team total.  `scratch` needs TEAM/64 ints.
template <int TEAM>
__device__ __forceinline__ int team_scan(int v, int* scratch, int& total) {
  const int lane = threadIdx.x & 63;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if constexpr (TEAM == 64) {
    total = __shfl(x, 63);
    return x - v;
  } else {
    const int w = (threadIdx.x % TEAM) >> 6;
    if (lane == 63) scratch[w] = x;
    __syncthreads();
    int pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < TEAM / 64; ++i) {
      const int s = scratch[i];
      pre += (i < w) ? s : 0;
      tot += s;
    }
    __syncthreads();
    total = tot;
    return pre + x - v;
  }
}

struct Forced {
  int causal, f1, f2;  // ancestors of leaf c-1 (or -1) and of leaf c; node 0 always
  __device__ __forceinline__ bool is(int node) const {
    return causal && (node == 0 || node == f1 || node == f2);
  }
  __device__ __forceinline__ int count() const {
    if (!causal) return 0;
    int n = 1;
    if (f2 != 0) ++n;
    if (f1 >= 0 && f1 != 0 && f1 != f2) ++n;
    return n;
  }
};

__device__ __forceinline__ Forced forced_at(const Geo& geo, int lev, int c, int causal) {
  Forced f;
  f.causal = causal;
  f.f2 = static_cast<int>(c / geo.gpow[lev]);
  f.f1 = (c >= 1) ? static_cast<int>((c - 1) / geo.gpow[lev]) : -1;
  return f;
}

// Online LSE merge of (m, s) pairs in log2 units; s is the sum of 2^(z - m).
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) {
    m = mn;
    s = 0.f;
    return;
  }
  s = s * fast_exp2(m - mn) + s2 * fast_exp2(m2 - mn);
  m = mn;
}

template <typename T, int D, int TEAM, int GMAX, bool FUSED>
__global__ __launch_bounds__(256) void select_kernel(SelArgs a, int lds_words) {
  constexpr int DPL = D / 16;
  constexpr int NGRP = TEAM / 16;
  constexpr int NW = TEAM / 64;
  constexpr int ROWS = 256 / TEAM;
  extern __shared__ int lds_i[];
  const Geo& geo = a.geo;
  const int gK = a.gK;
  const int g = geo.g;
  const int G = a.G;

  const int team = threadIdx.x / TEAM;
  const int tid = threadIdx.x % TEAM;
  const int lane = threadIdx.x & 63;
  const int wave_in_team = tid >> 6;
  const int grp = tid >> 4;        // lane group within the team
  const int grp_in_wave = lane >> 4;
  const int sub = tid & 15;

  int* L = lds_i + team * lds_words;
  int* cand = L;
  int* cand2 = L + gK;
  float* score = reinterpret_cast<float*>(L + 2 * gK);
  int* flag = L + 3 * gK;
  int* misc = L + 4 * gK;
  float* zbuf = reinterpret_cast<float*>(L + 4 * gK + 8);

  const int row = blockIdx.x * ROWS + team;
  if (row >= a.Nq) return;  // the whole team leaves together
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = geo.N - a.Nq + row;
  const int c = t / geo.C;

  // Query slices of the group's heads, pre-scaled to log2 units.
  float qv[GMAX][DPL];
  {
    const T* qb = static_cast<const T*>(a.q);
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < G) {
        const int64_t off = ((static_cast<int64_t>(b) * a.H + h * G + hh) * a.Nq + row) * D + sub * DPL;
        load_row_part<T, DPL>(qb + off, qv[hh]);
#pragma unroll
        for (int e = 0; e < DPL; ++e) qv[hh][e] *= a.qscale2;
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) qv[hh][e] = 0.f;
      }
    }
  }

  if (tid == 0) cand[0] = 0;
  int nA = 1;
  team_sync<TEAM>();

  const int last_level = FUSED ? 1 : 2;
  bool ranked = false;
  for (int lev = geo.L; lev >= last_level; --lev) {
    const Forced fz = forced_at(geo, lev, c, a.causal);
    ranked = nA > a.K;
    if (ranked) {
      if (lev >= 2) {
        // Child logits of every (candidate, child) pair into zbuf.
        const int Mb = geo.M[lev - 1];
        const float* pbase = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * D + sub * DPL;
        const int npairs = nA * g;
        for (int p = grp; p < npairs; p += NGRP) {
          const int ci = p / g;
          const int node = cand[ci];
          const int r = node * g + (p - ci * g);
          const bool valid = r < Mb && !fz.is(node);
          float x[DPL];
          if (valid) {
            load_row_part<float, DPL>(pbase + static_cast<int64_t>(r) * D, x);
          } else {
#pragma unroll
            for (int e = 0; e < DPL; ++e) x[e] = 0.f;
          }
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) {
            if (hh < G) {
              float d0 = 0.f;
#pragma unroll
              for (int e = 0; e < DPL; ++e) d0 = fmaf(qv[hh][e], x[e], d0);
              d0 = sum16(d0);
              if (sub == 0) zbuf[p * G + hh] = valid ? d0 : -INFINITY;
            }
          }
        }
        team_sync<TEAM>();
        for (int ci = tid; ci < nA; ci += TEAM) {
          const int node = cand[ci];
          float u = 0.f;
          if (!fz.is(node)) {
            const int nch = min(g, Mb - node * g);
            for (int hh = 0; hh < G; ++hh) {
              float m = -INFINITY;
              for (int j = 0; j < nch; ++j) m = fmaxf(m, zbuf[(ci * g + j) * G + hh]);
              float s = 0.f;
              for (int j = 0; j < nch; ++j) s += fast_exp2(zbuf[(ci * g + j) * G + hh] - m);
              u += m + fast_log2(s);
            }
          }
          score[ci] = u;
        }
      } else if constexpr (FUSED) {
        // Leaf level: exact LSE over each candidate block's raw keys.
        const T* kb = static_cast<const T*>(a.k) + static_cast<int64_t>(bh) * geo.N * D + sub * DPL;
        for (int ci = wave_in_team; ci < nA; ci += NW) {
          const int node = cand[ci];
          if (fz.is(node)) {
            if (lane == 0) score[ci] = 0.f;
            continue;
          }
          const int r0 = node * geo.C;
          const int nrows = min(geo.C, geo.N - r0);
          float m[GMAX], s[GMAX];
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) {
            m[hh] = -INFINITY;
            s[hh] = 0.f;
          }
          for (int r = grp_in_wave; r < nrows; r += 4) {
            float x[DPL];
            load_row_part<T, DPL>(kb + static_cast<int64_t>(r0 + r) * D, x);
#pragma unroll
            for (int hh = 0; hh < GMAX; ++hh) {
              if (hh < G) {
                float d0 = 0.f;
#pragma unroll
                for (int e = 0; e < DPL; ++e) d0 = fmaf(qv[hh][e], x[e], d0);
                d0 = sum16(d0);
                const float mn = fmaxf(m[hh], d0);
                s[hh] = s[hh] * fast_exp2(m[hh] - mn) + fast_exp2(d0 - mn);
                m[hh] = mn;
              }
            }
          }
          float u = 0.f;
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) {
            if (hh < G) {
              float m2 = __shfl_xor(m[hh], 16), s2 = __shfl_xor(s[hh], 16);
              lse_merge(m[hh], s[hh], m2, s2);
              m2 = __shfl_xor(m[hh], 32);
              s2 = __shfl_xor(s[hh], 32);
              lse_merge(m[hh], s[hh], m2, s2);
              u += m[hh] + fast_log2(s[hh]);
            }
          }
          if (lane == 0) score[ci] = u;
        }
      }
      team_sync<TEAM>();
      // Rank the non-forced candidates; keep forced + the best K - |F|.
      const int keepn = a.K - fz.count();
      for (int ci = tid; ci < nA; ci += TEAM) {
        const int node = cand[ci];
        int keep = 1;
        if (!fz.is(node)) {
          const float sc = score[ci];
          int rank = 0;
          for (int cj = 0; cj < nA; ++cj) {
            const int o = cand[cj];
            rank += (!fz.is(o) && ranks_before(score[cj], o, sc, node)) ? 1 : 0;
          }
          keep = rank < keepn;
        }
        flag[ci] = keep;
      }
    } else {
      for (int ci = tid; ci < nA; ci += TEAM) flag[ci] = 1;
    }
    team_sync<TEAM>();

    if (lev > last_level || (!FUSED && lev == 2)) {
      // Expand kept nodes to their eligible children at level lev-1.
      const int Mb = geo.M[lev - 1];
      const int64_t span_below = geo.gpow[lev - 1] * geo.C;
      const int rmax = a.causal ? static_cast<int>(min<int64_t>(t / span_below, Mb - 1)) : Mb - 1;
      const int E = (nA + TEAM - 1) / TEAM;
      const int i0 = tid * E, i1 = min(nA, i0 + E);
      int mine = 0;
      for (int ci = i0; ci < i1; ++ci) {
        if (flag[ci]) {
          const int c0 = cand[ci] * g;
          mine += max(0, min(c0 + g - 1, rmax) - c0 + 1);
        }
      }
      int total;
      int pos = team_scan<TEAM>(mine, misc, total);
      for (int ci = i0; ci < i1; ++ci) {
        if (flag[ci]) {
          const int c0 = cand[ci] * g;
          const int n = max(0, min(c0 + g - 1, rmax) - c0 + 1);
          for (int j = 0; j < n; ++j) cand2[pos + j] = c0 + j;
          pos += n;
        }
      }
      team_sync<TEAM>();
      for (int ci = tid; ci < total; ci += TEAM) cand[ci] = cand2[ci];
      nA = total;
      team_sync<TEAM>();
    }
  }

  const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row;
  if constexpr (FUSED) {
    // Final leaf set: kept candidates, already ascending.
    const int E = (nA + TEAM - 1) / TEAM;
    const int i0 = tid * E, i1 = min(nA, i0 + E);
    int mine = 0;
    for (int ci = i0; ci < i1; ++ci) mine += flag[ci];
    int total;
    int pos = team_scan<TEAM>(mine, misc, total);
    const Forced f1 = forced_at(geo, 1, c, a.causal);
    for (int ci = i0; ci < i1; ++ci) {
      if (flag[ci]) {
        const int node = cand[ci];
        a.idx[orow * a.K + pos] = node;
        if (a.score) {
          a.score[orow * a.K + pos] = (ranked && !f1.is(node)) ? score[ci] * kLn2 : INFINITY;
        }
        ++pos;
      }
    }
    for (int j = total + tid; j < a.K; j += TEAM) {
      a.idx[orow * a.K + j] = -1;
      if (a.score) a.score[orow * a.K + j] = -INFINITY;
    }
  } else {
    if (geo.L == 1 && tid == 0) {  // single leaf block: nothing was expanded
      cand[0] = 0;
    }
    for (int ci = tid; ci < gK; ci += TEAM) a.a1[orow * gK + ci] = ci < nA ? cand[ci] : -1;
    if (tid == 0) a.a1cnt[orow] = nA;
  }
}

// ----------------------------------------------------------------------------
// Two-stage remainder: cluster build, MFMA leaf scoring, final Top-K.
// ----------------------------------------------------------------------------

struct PairArgs {
  int Nq, N, C, K, gK, M1, causal;
  int64_t rows;  // BH * Nq
};

__device__ __forceinline__ bool pair_needs_score(const PairArgs& a, const int32_t* a1, const int32_t* a1cnt,
                                                 int64_t gid, int& bh, int& row, int& slot, int& blk) {
  const int64_t rg = gid / a.gK;
  slot = static_cast<int>(gid - rg * a.gK);
  const int n = a1cnt[rg];
  if (slot >= n || n <= a.K) return false;
  blk = a1[gid];
  bh = static_cast<int>(rg / a.Nq);
  row = static_cast<int>(rg - static_cast<int64_t>(bh) * a.Nq);
  const int c = (a.N - a.Nq + row) / a.C;
  if (a.causal && (blk == 0 || blk == c || blk == c - 1)) return false;
  return true;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(int32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < n; i += 256LL * gridDim.x) p[i] = 0;
}

__global__ __launch_bounds__(256) void cluster_count_kernel(PairArgs a, const int32_t* __restrict__ a1,
                                                            const int32_t* __restrict__ a1cnt,
                                                            int32_t* __restrict__ hist) {
  const int64_t gid = blockIdx.x * 256LL + threadIdx.x;
  if (gid >= a.rows * a.gK) return;
  int bh, row, slot, blk;
  if (!pair_needs_score(a, a1, a1cnt, gid, bh, row, slot, blk)) return;
  atomicAdd(&hist[static_cast<int64_t>(bh) * a.M1 + blk], 1);
}

// Exclusive scan of n counts into offs[0..n] and cursor[0..n), one workgroup.
__global__ __launch_bounds__(1024) void cluster_scan_kernel(const int32_t* __restrict__ hist,
                                                            int32_t* __restrict__ offs,
                                                            int32_t* __restrict__ cursor, int64_t n) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t i0 = tid * per, i1 = min(n, i0 + per);
  int local = 0;
  for (int64_t i = i0; i < i1; ++i) local += hist[i];
  const int lane = tid & 63, w = tid >> 6;
  int x = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int pre = 0, tot = 0;
  for (int i = 0; i < 16; ++i) {
    pre += (i < w) ? wsum[i] : 0;
    tot += wsum[i];
  }
  int run = pre + x - local;
  for (int64_t i = i0; i < i1; ++i) {
    offs[i] = run;
    cursor[i] = run;
    run += hist[i];
  }
  if (tid == 0) offs[n] = tot;
}

__global__ __launch_bounds__(256) void cluster_scatter_kernel(PairArgs a, const int32_t* __restrict__ a1,
                                                              const int32_t* __restrict__ a1cnt,
                                                              int32_t* __restrict__ cursor,
                                                              int32_t* __restrict__ pairs) {
  const int64_t gid = blockIdx.x * 256LL + threadIdx.x;
  if (gid >= a.rows * a.gK) return;
  int bh, row, slot, blk;
  if (!pair_needs_score(a, a1, a1cnt, gid, bh, row, slot, blk)) return;
  const int pos = atomicAdd(&cursor[static_cast<int64_t>(bh) * a.M1 + blk], 1);
  pairs[pos] = (row << 8) | slot;
}

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef float f32x16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8v as_bf16x8(uint4 r) {
  return __builtin_bit_cast(bf16x8v, r);
}

struct LeafArgs {
  int H, Hkv, G, Nq, N, C, M1, gK;
  float qscale2;
};

// One workgroup per (leaf block, batch x KV head): the C x D key block is
// staged in LDS once (rows padded by 16 B against bank conflicts) and every
// (query, slot) pair of the block's cluster is scored against it, 32 pairs
// per wavefront tile.
template <int D>
__global__ __launch_bounds__(256) void leaf_score_kernel(LeafArgs a, const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ k,
                                                         const int32_t* __restrict__ offs,
                                                         const int32_t* __restrict__ pairs,
                                                         float* __restrict__ u1) {
  constexpr int LDR = D + 8;  // padded LDS row, in bf16 elements
  constexpr int KS = D / 16;
  extern __shared__ uint16_t klds[];
  const int blk = blockIdx.x;
  const int bh = blockIdx.y;
  const int64_t cl = static_cast<int64_t>(bh) * a.M1 + blk;
  const int beg = offs[cl], end = offs[cl + 1];
  if (beg == end) return;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = blk * a.C;
  const int nrows = min(a.C, a.N - r0);

  // Stage the key block (zero rows past the end of the sequence).
  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.N + r0) * D;
  for (int e = threadIdx.x; e < a.C * (D / 8); e += 256) {
    const int r = e / (D / 8), cidx = (e - r * (D / 8)) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < nrows) v = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D + cidx);
    *reinterpret_cast<uint4*>(klds + r * LDR + cidx) = v;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 31;   // query column of this lane
  const int half = lane >> 5;  // which 8-wide k slice / which 4-row key group
  const int ntile = (end - beg + 31) / 32;
  for (int tile = wave; tile < ntile; tile += 4) {
    const int p = beg + tile * 32 + col;
    const bool valid = p < end;
    const int pr = valid ? pairs[p] : 0;
    const int row = pr >> 8, slot = pr & 255;
    float u = 0.f;
    for (int hh = 0; hh < a.G; ++hh) {
      const uint16_t* qrow = q + ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + row) * D + half * 8;
      bf16x8v qb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 v = make_uint4(0, 0, 0, 0);
        if (valid) v = *reinterpret_cast<const uint4*>(qrow + ks * 16);
        qb[ks] = as_bf16x8(v);
      }
      float m = -INFINITY, s = 0.f;
      for (int kt = 0; kt < a.C / 32; ++kt) {
        f32x16v acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        const uint16_t* arow = klds + (kt * 32 + col) * LDR + half * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8v av = as_bf16x8(*reinterpret_cast<const uint4*>(arow + ks * 16));
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qb[ks], acc, 0, 0, 0);
        }
        // acc[r] is the logit of key kt*32 + 8*(r/4) + 4*half + r%4 for query `col`.
        float tm = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          acc[r] = key < nrows ? acc[r] * a.qscale2 : -INFINITY;
          tm = fmaxf(tm, acc[r]);
        }
        float ts = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) ts += fast_exp2(acc[r] - tm);
        lse_merge(m, s, tm, ts);
      }
      const float m2 = __shfl_xor(m, 32), s2 = __shfl_xor(s, 32);
      lse_merge(m, s, m2, s2);
      u += m + fast_log2(s);
    }
    if (valid && half == 0) u1[(static_cast<int64_t>(bh) * a.Nq + row) * a.gK + slot] = u;
  }
}

struct TopkArgs {
  int Nq, N, C, K, gK, causal;
  int64_t rows;
};

// One wavefront per (batch x KV head, row): rank the scored leaf candidates.
__global__ __launch_bounds__(256) void final_topk_kernel(TopkArgs a, const int32_t* __restrict__ a1,
                                                         const int32_t* __restrict__ a1cnt,
                                                         const float* __restrict__ u1,
                                                         int32_t* __restrict__ idx, float* __restrict__ score) {
  __shared__ int s_node[4][kMaxCand];
  __shared__ float s_u[4][kMaxCand];
  __shared__ int s_keep[4][kMaxCand];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t rg = blockIdx.x * 4LL + wave;
  if (rg >= a.rows) return;
  const int row = static_cast<int>(rg % a.Nq);
  const int t = a.N - a.Nq + row;
  const int c = t / a.C;
  const int n = a1cnt[rg];
  const int32_t* cand = a1 + rg * a.gK;
  const float* uu = u1 + rg * a.gK;
  int* nodes = s_node[wave];
  float* us = s_u[wave];
  int* keep = s_keep[wave];
  auto forced = [&](int node) { return a.causal && (node == 0 || node == c || node == c - 1); };
  const bool ranked = n > a.K;
  int nF = 0;
  if (a.causal) nF = 1 + (c != 0) + (c - 1 > 0);
  for (int i = lane; i < n; i += 64) {
    nodes[i] = cand[i];
    us[i] = (ranked && !forced(cand[i])) ? uu[i] : 0.f;
  }
  wave_sync();
  const int keepn = a.K - nF;
  for (int i = lane; i < n; i += 64) {
    const int node = nodes[i];
    int kp = 1;
    if (ranked && !forced(node)) {
      int rank = 0;
      for (int j = 0; j < n; ++j) rank += (!forced(nodes[j]) && ranks_before(us[j], nodes[j], us[i], node)) ? 1 : 0;
      kp = rank < keepn;
    }
    keep[i] = kp;
  }
  wave_sync();
  // Compact in order (candidates are ascending).
  const int E = (n + 63) / 64;
  const int i0 = lane * E, i1 = min(n, i0 + E);
  int mine = 0;
  for (int i = i0; i < i1; ++i) mine += keep[i];
  int x = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  const int total = __shfl(x, 63);
  int pos = x - mine;
  for (int i = i0; i < i1; ++i) {
    if (keep[i]) {
      idx[rg * a.K + pos] = nodes[i];
      if (score) score[rg * a.K + pos] = (ranked && !forced(nodes[i])) ? us[i] * kLn2 : INFINITY;
      ++pos;
    }
  }
  for (int j = total + lane; j < a.K; j += 64) {
    idx[rg * a.K + j] = -1;
    if (score) score[rg * a.K + j] = -INFINITY;
  }
}

// ----------------------------------------------------------------------------
// Host launchers.
// ----------------------------------------------------------------------------

static int sel_lds_words(const Shape& s) {
  const int gK = s.gK();
  int w = 4 * gK + 8 + gK * s.g * s.G;
  return (w + 3) & ~3;
}

static SelArgs make_sel_args(const Shape& s, const Geo& geo, const void* q, const void* k, const float* pyr) {
  SelArgs a{};
  a.geo = geo;
  a.q = q;
  a.k = k;
  a.pyr = pyr;
  a.H = s.H;
  a.Hkv = s.Hkv;
  a.G = s.G;
  a.Nq = s.Nq;
  a.K = s.K;
  a.causal = s.causal;
  a.gK = s.gK();
  a.qscale2 = kLog2e / sqrtf(static_cast<float>(s.D));
  return a;
}

template <typename T, int D, int TEAM, bool FUSED>
static void launch_sel_g(const Shape& s, const SelArgs& a, hipStream_t st) {
  constexpr int ROWS = 256 / TEAM;
  const int words = sel_lds_words(s);
  dim3 grid((s.Nq + ROWS - 1) / ROWS, s.BH());
  const size_t lds = static_cast<size_t>(ROWS) * words * sizeof(int);
  if (s.G == 1)
    select_kernel<T, D, TEAM, 1, FUSED><<<grid, 256, lds, st>>>(a, words);
  else if (s.G <= 4)
    select_kernel<T, D, TEAM, 4, FUSED><<<grid, 256, lds, st>>>(a, words);
  else
    select_kernel<T, D, TEAM, 16, FUSED><<<grid, 256, lds, st>>>(a, words);
}

template <typename T, int TEAM, bool FUSED>
static void launch_sel_d(const Shape& s, const SelArgs& a, hipStream_t st) {
  if (s.D == 128)
    launch_sel_g<T, 128, TEAM, FUSED>(s, a, st);
  else
    launch_sel_g<T, 64, TEAM, FUSED>(s, a, st);
}

hipError_t launch_select_fused(const Shape& s, const Geo& geo, const void* q, const void* k, const float* pyr,
                               int32_t* idx, float* score, hipStream_t st) {
  SelArgs a = make_sel_args(s, geo, q, k, pyr);
  a.idx = idx;
  a.score = score;
  // Few rows: a whole workgroup per row to cut latency; many rows: a wave per row.
  const bool wide = static_cast<int64_t>(s.BH()) * s.Nq <= 2048;
  if (s.bf16) {
    if (wide)
      launch_sel_d<uint16_t, 256, true>(s, a, st);
    else
      launch_sel_d<uint16_t, 64, true>(s, a, st);
  } else {
    if (wide)
      launch_sel_d<float, 256, true>(s, a, st);
    else
      launch_sel_d<float, 64, true>(s, a, st);
  }
  return hipGetLastError();
}

static size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct TwoStageWs {
  size_t a1, a1cnt, u1, hist, offs, cursor, pairs, total;
};

static TwoStageWs two_stage_layout(const Shape& s, const Geo& geo) {
  const size_t rows = static_cast<size_t>(s.BH()) * s.Nq;
  const size_t ncl = static_cast<size_t>(s.BH()) * geo.M[1];
  TwoStageWs w{};
  size_t o = 0;
  w.a1 = o;     o += align256(rows * s.gK() * 4);
  w.a1cnt = o;  o += align256(rows * 4);
  w.u1 = o;     o += align256(rows * s.gK() * 4);
  w.hist = o;   o += align256(ncl * 4);
  w.offs = o;   o += align256((ncl + 1) * 4);
  w.cursor = o; o += align256(ncl * 4);
  w.pairs = o;  o += align256(rows * s.gK() * 4);
  w.total = o;
  return w;
}

size_t select_two_stage_ws(const Shape& s, const Geo& geo) { return two_stage_layout(s, geo).total; }

hipError_t launch_select_two_stage(const Shape& s, const Geo& geo, const void* q, const void* k,
                                   const float* pyr, int32_t* idx, float* score, void* ws, hipStream_t st) {
  const TwoStageWs w = two_stage_layout(s, geo);
  char* base = static_cast<char*>(ws);
  int32_t* a1 = reinterpret_cast<int32_t*>(base + w.a1);
  int32_t* a1cnt = reinterpret_cast<int32_t*>(base + w.a1cnt);
  float* u1 = reinterpret_cast<float*>(base + w.u1);
  int32_t* hist = reinterpret_cast<int32_t*>(base + w.hist);
  int32_t* offs = reinterpret_cast<int32_t*>(base + w.offs);
  int32_t* cursor = reinterpret_cast<int32_t*>(base + w.cursor);
  int32_t* pairs = reinterpret_cast<int32_t*>(base + w.pairs);
  hipError_t e;

  // Stage 1: intermediate levels, one wavefront per (row, KV head).
  SelArgs a = make_sel_args(s, geo, q, k, pyr);
  a.a1 = a1;
  a.a1cnt = a1cnt;
  launch_sel_d<uint16_t, 64, false>(s, a, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // Cluster the (row, slot) pairs by leaf block.
  const int64_t rows = static_cast<int64_t>(s.BH()) * s.Nq;
  const int64_t ncl = static_cast<int64_t>(s.BH()) * geo.M[1];
  PairArgs pa{s.Nq, s.N, s.C, s.K, s.gK(), geo.M[1], s.causal, rows};
  fill_zero_kernel<<<static_cast<unsigned>(std::min<int64_t>((ncl + 255) / 256, 4096)), 256, 0, st>>>(hist, ncl);
  const unsigned pgrid = static_cast<unsigned>((rows * s.gK() + 255) / 256);
  cluster_count_kernel<<<pgrid, 256, 0, st>>>(pa, a1, a1cnt, hist);
  cluster_scan_kernel<<<1, 1024, 0, st>>>(hist, offs, cursor, ncl);
  cluster_scatter_kernel<<<pgrid, 256, 0, st>>>(pa, a1, a1cnt, cursor, pairs);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // Stage 2: leaf scoring against each key block once per cluster.
  LeafArgs la{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, geo.M[1], s.gK(), kLog2e / sqrtf(static_cast<float>(s.D))};
  dim3 lgrid(geo.M[1], s.BH());
  const size_t llds = static_cast<size_t>(s.C) * (s.D + 8) * 2;
  if (s.D == 128)
    leaf_score_kernel<128><<<lgrid, 256, llds, st>>>(la, static_cast<const uint16_t*>(q),
                                                     static_cast<const uint16_t*>(k), offs, pairs, u1);
  else
    leaf_score_kernel<64><<<lgrid, 256, llds, st>>>(la, static_cast<const uint16_t*>(q),
                                                    static_cast<const uint16_t*>(k), offs, pairs, u1);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // Final Top-K per row.
  TopkArgs ta{s.Nq, s.N, s.C, s.K, s.gK(), s.causal, rows};
  final_topk_kernel<<<static_cast<unsigned>((rows + 3) / 4), 256, 0, st>>>(ta, a1, a1cnt, u1, idx, score);
  return hipGetLastError();
}

}  // namespace pisa
