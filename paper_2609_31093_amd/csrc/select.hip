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
  int score_kind;   // kScoreLse / kScoreMean / kScoreMeanVar
  float qscale2;    // log2(e) / sqrt(d)
};

struct TopkArgsP {
  int Nq, N, C, K, gK, causal;
  int64_t rows;
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
  f.f2 = anc_at(geo, c, lev);
  f.f1 = (c >= 1) ? anc_at(geo, c - 1, lev) : -1;
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

// ----------------------------------------------------------------------------
// Score reducers over the logits of one candidate and query head (log2 units):
// the LSE of eq. direct_child_lse (PISA) and its first- and second-order
// truncations of App. A "First- and second-order approximations": the mean
// (PISA-1) and the mean plus half the population variance (PISA-2; ln 2
// rescales the variance of log2-unit logits so that the score is the natural-
// log one times log2(e), which ranks identically).
// ----------------------------------------------------------------------------
constexpr int kScoreLse = 0, kScoreMean = 1, kScoreMeanVar = 2;

// LSE: (max, sum of 2^(v - max)); moments: (count, mean, sum of squared
// deviations from the mean).
struct ScoreAcc {
  float x, y, z;
};

__device__ __forceinline__ ScoreAcc acc_empty(int kind) {
  return kind == kScoreLse ? ScoreAcc{-INFINITY, 0.f, 0.f} : ScoreAcc{0.f, 0.f, 0.f};
}

// Merge two states (the moments by Chan et al.'s pairwise update).
__device__ __forceinline__ void acc_merge(int kind, ScoreAcc& a, const ScoreAcc& b) {
  if (kind == kScoreLse) {
    lse_merge(a.x, a.y, b.x, b.y);
    return;
  }
  if (b.x == 0.f) return;
  if (a.x == 0.f) {
    a = b;
    return;
  }
  const float n = a.x + b.x;
  const float d = b.y - a.y;
  a.y += d * (b.x / n);
  a.z += b.z + d * d * (a.x * b.x / n);
  a.x = n;
}

__device__ __forceinline__ void acc_push(int kind, ScoreAcc& a, float v) {
  acc_merge(kind, a, kind == kScoreLse ? ScoreAcc{v, 1.f, 0.f} : ScoreAcc{1.f, v, 0.f});
}

// State of NV register values; -inf marks an absent value.
template <int NV>
__device__ __forceinline__ ScoreAcc acc_of(int kind, const float (&v)[NV]) {
  if (kind == kScoreLse) {
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) m = fmaxf(m, v[i]);
    if (m == -INFINITY) return ScoreAcc{-INFINITY, 0.f, 0.f};
    float sm = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) sm += fast_exp2(v[i] - m);
    return ScoreAcc{m, sm, 0.f};
  }
  float n = 0.f, sum = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const bool ok = v[i] != -INFINITY;
    n += ok ? 1.f : 0.f;
    sum += ok ? v[i] : 0.f;
  }
  if (n == 0.f) return ScoreAcc{0.f, 0.f, 0.f};
  const float mean = sum / n;
  float m2 = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const float dv = v[i] - mean;
    m2 += v[i] != -INFINITY ? dv * dv : 0.f;
  }
  return ScoreAcc{n, mean, m2};
}

// The score state of NV raw logits (unscaled, -inf = no key) times a
// positive scale: for the LSE the scale enters the exponent's FMA, since the
// maximum of the raw logits scales to the maximum of the scaled ones.
template <int KIND, int NV>
__device__ __forceinline__ ScoreAcc acc_of_scaled(float (&v)[NV], float scale) {
  if constexpr (KIND == kScoreLse) {
    float m = v[0];
#pragma unroll
    for (int i = 1; i < NV; ++i) m = fmaxf(m, v[i]);
    if (m == -INFINITY) return ScoreAcc{-INFINITY, 0.f, 0.f};
    const float ms = m * scale;
    float sm = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) sm += fast_exp2(fmaf(v[i], scale, -ms));
    return ScoreAcc{ms, sm, 0.f};
  } else {
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] *= scale;
    return acc_of(KIND, v);
  }
}

__device__ __forceinline__ ScoreAcc acc_shfl_xor(const ScoreAcc& a, int mask) {
  return ScoreAcc{__shfl_xor(a.x, mask), __shfl_xor(a.y, mask), __shfl_xor(a.z, mask)};
}

__device__ __forceinline__ float acc_value(int kind, const ScoreAcc& a) {
  if (kind == kScoreLse) return a.x + fast_log2(a.y);
  if (kind == kScoreMean) return a.y;
  return a.y + 0.5f * kLn2 * (a.z / a.x);
}

// Score of the n >= 1 logits z[0], z[stride], ... (two passes).
__device__ __forceinline__ float reduce_logits(int kind, const float* z, int n, int stride) {
  if (kind == kScoreLse) {
    float m = -INFINITY;
    for (int j = 0; j < n; ++j) m = fmaxf(m, z[j * stride]);
    float sm = 0.f;
    for (int j = 0; j < n; ++j) sm += fast_exp2(z[j * stride] - m);
    return m + fast_log2(sm);
  }
  float sum = 0.f;
  for (int j = 0; j < n; ++j) sum += z[j * stride];
  const float mean = sum / static_cast<float>(n);
  if (kind == kScoreMean) return mean;
  float m2 = 0.f;
  for (int j = 0; j < n; ++j) {
    const float dv = z[j * stride] - mean;
    m2 += dv * dv;
  }
  return mean + 0.5f * kLn2 * (m2 / static_cast<float>(n));
}

// Rank order (key desc, pack asc) as one ascending 64-bit integer: the high
// word maps the float key to an unsigned value that decreases as the key
// grows (total order, -inf last), the low word is the non-negative pack.
__device__ __forceinline__ uint32_t desc_bits(float key) {
  const uint32_t u = __float_as_uint(key + 0.0f);  // -0 ranks as +0
  const uint32_t m = static_cast<uint32_t>(static_cast<int32_t>(u) >> 31);
  return u ^ (~m & 0x7FFFFFFFu);
}
__device__ __forceinline__ float desc_bits_inv(uint32_t d) {
  const uint32_t m = static_cast<uint32_t>(static_cast<int32_t>(d) >> 31);
  return __uint_as_float(d ^ (~m & 0x7FFFFFFFu));
}

// Bitonic sort of 128 (key, pack) entries held two per lane (entry lane and
// lane + 64) into rank order (key desc, pack asc); packs are non-negative.
// Step (K2, J) of entry e keeps the smaller of e and e ^ J where
// (e & K2 == 0) == (e & J == 0); that direction is a lane mask per entry
// half, known at compile time.
template <int K2, int J, int S>
constexpr uint64_t sort128_want_small() {
  uint64_t m = 0;
  for (int l = 0; l < 64; ++l) {
    const int e = l + 64 * S;
    if (((e & K2) == 0) == ((e & J) == 0)) m |= uint64_t(1) << l;
  }
  return m;
}

template <int K2, int J, int S>
__device__ __forceinline__ void sort128_half_step(uint32_t& hi, uint32_t& lo) {
  uint32_t ohi, olo;
  if constexpr (J < 32) {
    ohi = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(hi)));
    olo = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(lo)));
  } else {
    ohi = static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), 32));
    olo = static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), 32));
  }
  const uint64_t mine = (static_cast<uint64_t>(hi) << 32) | lo;
  const uint64_t other = (static_cast<uint64_t>(ohi) << 32) | olo;
  constexpr uint64_t kWant = sort128_want_small<K2, J, S>();
  const bool take = (other < mine) == __builtin_amdgcn_inverse_ballot_w64(kWant);
  hi = take ? ohi : hi;
  lo = take ? olo : lo;
}

// The steps J = J0, J0 / 2, ..., 1 of stage K2.
template <int K2, int J>
__device__ __forceinline__ void sort128_stage(uint32_t (&hi)[2], uint32_t (&lo)[2]) {
  if constexpr (J == 64) {  // the two entries of a lane: the lower index keeps the smaller
    const uint64_t x = (static_cast<uint64_t>(hi[0]) << 32) | lo[0];
    const uint64_t y = (static_cast<uint64_t>(hi[1]) << 32) | lo[1];
    const bool sw = y < x;
    const uint32_t h0 = sw ? hi[1] : hi[0], l0 = sw ? lo[1] : lo[0];
    hi[1] = sw ? hi[0] : hi[1];
    lo[1] = sw ? lo[0] : lo[1];
    hi[0] = h0;
    lo[0] = l0;
  } else {
    sort128_half_step<K2, J, 0>(hi[0], lo[0]);
    sort128_half_step<K2, J, 1>(hi[1], lo[1]);
  }
  if constexpr (J > 1) sort128_stage<K2, J / 2>(hi, lo);
}

__device__ __forceinline__ void sort128(uint32_t (&hi)[2], uint32_t (&lo)[2], int lane) {
  (void)lane;
  sort128_stage<2, 1>(hi, lo);
  sort128_stage<4, 2>(hi, lo);
  sort128_stage<8, 4>(hi, lo);
  sort128_stage<16, 8>(hi, lo);
  sort128_stage<32, 16>(hi, lo);
  sort128_stage<64, 32>(hi, lo);
  sort128_stage<128, 64>(hi, lo);
}

template <typename T, int D, int TEAM, int GMAX, bool FUSED>
__global__ __launch_bounds__(256) void select_kernel(SelArgs a, int lds_words) {
  constexpr int DPL = D / 16;
  constexpr int NGRP = TEAM / 16;
  constexpr int NW = TEAM / 64;
  constexpr int ROWS = 256 / TEAM;
  extern __shared__ __align__(16) int lds_i[];
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
  // Per-candidate strides padded by one word so that lanes owning
  // consecutive candidates hit different LDS banks.
  const int CS = g * G + 1;           // zbuf stride per candidate
  const int SS = G + 1;               // zself stride per candidate
  float* zbuf = reinterpret_cast<float*>(L + 4 * gK + 8);
  float* zself = zbuf + gK * CS;      // logit of each candidate (per head), NaN if unknown
  float* zself2 = zself + gK * SS;

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
  for (int hh = tid; hh < G; hh += TEAM) zself[hh] = __builtin_nanf("");
  int nA = 1;
  team_sync<TEAM>();

  const int last_level = FUSED ? 1 : 2;
  bool ranked = false;
  for (int lev = geo.L; lev >= last_level; --lev) {
    const Forced fz = forced_at(geo, lev, c, a.causal);
    ranked = nA > a.K;
    if (ranked) {
      if (lev >= 2) {
        // Child logits of every (candidate, child) pair into zbuf, UNR loads in
        // flight per lane group.  A candidate whose own logit is known from
        // the level above (zself) skips its last child: the mean pyramid
        // makes the node logit the mean of its children's logits, so that
        // child's logit is nch * z_node - (sum of the others).
        const int Mb = geo.M[lev - 1];
        const float* pbase = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * D + sub * DPL;
        const int npairs = nA * g;
        constexpr int UNR = 4;
        for (int p0 = grp; p0 < npairs; p0 += NGRP * UNR) {
          float x[UNR][DPL];
          bool ld[UNR];
#pragma unroll
          for (int u = 0; u < UNR; ++u) {
            const int p = p0 + u * NGRP;
            ld[u] = false;
            int r = 0;
            if (p < npairs) {
              const int ci = p / g, j = p - ci * g;
              const int node = cand[ci];
              const int nch = min(g, Mb - node * g);
              const bool derived = j == nch - 1 && !__builtin_isnan(zself[ci * SS]);
              r = node * g + j;
              ld[u] = j < nch && !fz.is(node) && !derived;
            }
            if (ld[u]) {
              load_row_part<float, DPL>(pbase + static_cast<int64_t>(r) * D, x[u]);
            } else {
#pragma unroll
              for (int e = 0; e < DPL; ++e) x[u][e] = 0.f;
            }
          }
#pragma unroll
          for (int u = 0; u < UNR; ++u) {
            const int p = p0 + u * NGRP;
#pragma unroll
            for (int hh = 0; hh < GMAX; ++hh) {
              if (hh < G) {
                float d0 = 0.f;
#pragma unroll
                for (int e = 0; e < DPL; ++e) d0 = fmaf(qv[hh][e], x[u][e], d0);
                d0 = rowsum16_to15(d0);  // DPP row reduction: the total lands in the group's lane 15
                if (sub == 15 && p < npairs) zbuf[(p / g) * CS + (p % g) * G + hh] = ld[u] ? d0 : -INFINITY;
              }
            }
          }
        }
        team_sync<TEAM>();
        for (int ci = tid; ci < nA; ci += TEAM) {
          const int node = cand[ci];
          float u = 0.f;
          if (!fz.is(node)) {
            const int nch = min(g, Mb - node * g);
            const bool has_self = !__builtin_isnan(zself[ci * SS]);
            for (int hh = 0; hh < G; ++hh) {
              float* zc = zbuf + ci * CS + hh;
              if (has_self) {
                float others = 0.f;
                for (int j = 0; j < nch - 1; ++j) others += zc[j * G];
                zc[(nch - 1) * G] = static_cast<float>(nch) * zself[ci * SS + hh] - others;
              }
              u += reduce_logits(a.score_kind, zc, nch, G);
            }
          }
          score[ci] = u;
        }
      } else if constexpr (FUSED) {
        // Leaf level: exact LSE over each candidate block's raw keys.
        const T* kb = static_cast<const T*>(a.k) + static_cast<int64_t>(bh) * geo.Nkv * D + sub * DPL;
        for (int ci = wave_in_team; ci < nA; ci += NW) {
          const int node = cand[ci];
          if (fz.is(node)) {
            if (lane == 0) score[ci] = 0.f;
            continue;
          }
          const int r0 = node * geo.C;
          const int nrows = min(geo.C, geo.N - r0);
          ScoreAcc st[GMAX];
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) st[hh] = acc_empty(a.score_kind);
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
                acc_push(a.score_kind, st[hh], d0);
              }
            }
          }
          float u = 0.f;
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) {
            if (hh < G) {
              acc_merge(a.score_kind, st[hh], acc_shfl_xor(st[hh], 16));
              acc_merge(a.score_kind, st[hh], acc_shfl_xor(st[hh], 32));
              u += acc_value(a.score_kind, st[hh]);
            }
          }
          if (lane == 0) score[ci] = u;
        }
      }
      team_sync<TEAM>();
      // Rank the non-forced candidates; keep forced + the best K - |F|.
      const int keepn = a.K - fz.count();
      bool sorted = false;
      if constexpr (TEAM == 64) {
        if (nA <= 128) {  // one wavefront, two candidates per lane: a bitonic rank sort
          // Forced candidates sort first (key word 0), then score descending,
          // ties by candidate index (candidates are ascending node ids), then
          // the empty slots.
          uint32_t hi[2], lo[2];
          int nforced = 0;
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const int ci = lane + 64 * s2;
            const bool v = ci < nA;
            const bool f = v && fz.is(cand[ci]);
            hi[s2] = !v ? 0xFFFFFFFFu : (f ? 0u : desc_bits(score[ci]));
            lo[s2] = static_cast<uint32_t>(ci);
            nforced += __popcll(__ballot(f));
          }
          sort128(hi, lo, lane);
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const int r = lane + 64 * s2;  // rank among all candidates
            if (static_cast<int>(lo[s2]) < nA) flag[lo[s2]] = (r < nforced || r - nforced < keepn) ? 1 : 0;
          }
          sorted = true;
        }
      }
      for (int ci = tid; !sorted && ci < nA; ci += TEAM) {
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
      const int rmax = a.causal ? min(anc_at(geo, c, lev - 1), Mb - 1) : Mb - 1;
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
      const bool logits_known = ranked && lev >= 2;
      for (int ci = i0; ci < i1; ++ci) {
        if (flag[ci]) {
          const int c0 = cand[ci] * g;
          const int n = max(0, min(c0 + g - 1, rmax) - c0 + 1);
          const bool known = logits_known && !fz.is(cand[ci]);
          for (int j = 0; j < n; ++j) {
            cand2[pos + j] = c0 + j;
            for (int hh = 0; hh < G; ++hh)
              zself2[(pos + j) * SS + hh] = known ? zbuf[ci * CS + j * G + hh] : __builtin_nanf("");
          }
          pos += n;
        }
      }
      team_sync<TEAM>();
      for (int ci = tid; ci < total; ci += TEAM) {
        cand[ci] = cand2[ci];
        for (int hh = 0; hh < G; ++hh) zself[ci * SS + hh] = zself2[ci * SS + hh];
      }
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
// Stage 1 for g*K <= 32: two query rows per wavefront, one candidate per lane.
//
// Lanes 0-31 own row 2w and lanes 32-63 row 2w+1 (lane hl of a half holds
// candidate hl).  Per ranked level: the candidates needing child logits build
// a compact load list (a candidate whose own logit is known loads one child
// fewer, see select_kernel), the lane groups of each half (4, 8 or 16 lanes
// per dot) compute the listed dots, each lane turns its children's logits
// into its LSE score, and a 32-lane bitonic sort on (score desc, node asc) with forced nodes keyed
// +inf ranks the half: the first K survive.  Survivors expand through an LDS
// staging list.  The leaf candidate set is sorted ascending before it is
// stored.
// ----------------------------------------------------------------------------

// The lanes of a wavefront whose entry e (= lane & 31 for the 32-lane
// sorts) keeps the smaller of itself and its partner in the bitonic step
// (K2, J), as a lane mask known at compile time.
template <int K2, int J>
constexpr uint64_t sort32_want_small() {
  uint64_t m = 0;
  for (int l = 0; l < 64; ++l) {
    const int e = l & 31;
    if (((e & K2) == 0) == ((e & J) == 0)) m |= uint64_t(1) << l;
  }
  return m;
}

// One compare-exchange stage of the bitonic network, without branches: the
// lane keeps the smaller of (itself, partner) where the stage wants the
// smaller, else the larger.  hl = lane & 31 (the stage's direction comes
// from a constant lane mask).
template <int K2, int J>
__device__ __forceinline__ void sort32_step(uint32_t& hi, uint32_t& lo, int hl) {
  (void)hl;
  const uint32_t ohi = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(hi)));
  const uint32_t olo = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(lo)));
  const uint64_t mine = (static_cast<uint64_t>(hi) << 32) | lo;
  const uint64_t other = (static_cast<uint64_t>(ohi) << 32) | olo;
  constexpr uint64_t kWant = sort32_want_small<K2, J>();
  const bool want_small = __builtin_amdgcn_inverse_ballot_w64(kWant);
  const bool take = (other < mine) == want_small;
  hi = take ? ohi : hi;
  lo = take ? olo : lo;
}

// Bitonic sort of the 32 lanes of each wavefront half into rank order
// (key desc, pack asc); packs are non-negative.
__device__ __forceinline__ void sort32(float& key, int& pack, int hl) {
  uint32_t hi = desc_bits(key), lo = static_cast<uint32_t>(pack);
  sort32_step<2, 1>(hi, lo, hl);
  sort32_step<4, 2>(hi, lo, hl);
  sort32_step<4, 1>(hi, lo, hl);
  sort32_step<8, 4>(hi, lo, hl);
  sort32_step<8, 2>(hi, lo, hl);
  sort32_step<8, 1>(hi, lo, hl);
  sort32_step<16, 8>(hi, lo, hl);
  sort32_step<16, 4>(hi, lo, hl);
  sort32_step<16, 2>(hi, lo, hl);
  sort32_step<16, 1>(hi, lo, hl);
  sort32_step<32, 16>(hi, lo, hl);
  sort32_step<32, 8>(hi, lo, hl);
  sort32_step<32, 4>(hi, lo, hl);
  sort32_step<32, 2>(hi, lo, hl);
  sort32_step<32, 1>(hi, lo, hl);
  key = desc_bits_inv(hi);
  pack = static_cast<int>(lo);
}

// The best 16 of each wavefront half (key desc, pack asc) in its lanes 0-15,
// in no particular order, when only that set matters: the network's last
// merge stops after its first step (each 16-lane run is sorted, in opposite
// directions, and lane i keeps the better of i and i ^ 16); `full` finishes
// the sort (rank order in every lane), as sort32.
__device__ __forceinline__ void sort32_top16(float& key, int& pack, int hl, bool full) {
  uint32_t hi = desc_bits(key), lo = static_cast<uint32_t>(pack);
  sort32_step<2, 1>(hi, lo, hl);
  sort32_step<4, 2>(hi, lo, hl);
  sort32_step<4, 1>(hi, lo, hl);
  sort32_step<8, 4>(hi, lo, hl);
  sort32_step<8, 2>(hi, lo, hl);
  sort32_step<8, 1>(hi, lo, hl);
  sort32_step<16, 8>(hi, lo, hl);
  sort32_step<16, 4>(hi, lo, hl);
  sort32_step<16, 2>(hi, lo, hl);
  sort32_step<16, 1>(hi, lo, hl);
  sort32_step<32, 16>(hi, lo, hl);
  if (full) {
    sort32_step<32, 8>(hi, lo, hl);
    sort32_step<32, 4>(hi, lo, hl);
    sort32_step<32, 2>(hi, lo, hl);
    sort32_step<32, 1>(hi, lo, hl);
  }
  key = desc_bits_inv(hi);
  pack = static_cast<int>(lo);
}

// Inclusive prefix sum over the 32 lanes of a wavefront half.
__device__ __forceinline__ int scan32(int v, int) { return scan32_incl(v); }

// ----------------------------------------------------------------------------
// Stage 1 on the matrix cores (bf16 queries, fan-out 2 or 4, at most 16 heads
// per KV head, g*K <= 128; used for g*K > 32 or 8+ heads per KV head): one
// wavefront per query row.
//
// Each ranked level scores its candidates' children as one product per
// 16-child tile on v_mfma_f32_16x16x32_bf16: A = 16 child summary rows (lane
// l: child row l%16, dims 8*(l/16)..+7 of each 32-dim step), B = the group's
// query heads as columns (lane l: head l%16, zero past G).  The fp32
// summaries enter as a bf16 pair hi + lo (hi = the rounded value, lo = the
// rounded remainder: about 16 mantissa bits) with two products per step; the
// bf16 queries are exact.  In the result lane l holds tile rows 4*(l/16)+i
// (i = 0..3) of head l%16, i.e. all children of 4/g candidates, so each
// lane reduces its candidates' children to per-head scores in registers and
// a 16-lane row sum adds the heads.  Ranking is a 32-lane bitonic sort for
// up to 32 candidates, else the 128-entry register sort of the wavefront;
// expansion and the stored leaf candidate set are as in select_kernel.
// ----------------------------------------------------------------------------

typedef __bf16 bf16x8m __attribute__((ext_vector_type(8)));
typedef float f32x4m __attribute__((ext_vector_type(4)));

// Score of the first n of a lane's child logits (n >= 1).
template <int KIND, int NC>
__device__ __forceinline__ float lane_children_score(const float (&z)[NC], int n) {
  if constexpr (KIND == kScoreLse) {
    float m = z[0];
#pragma unroll
    for (int i = 1; i < NC; ++i) m = i < n ? fmaxf(m, z[i]) : m;
    float sm = 0.f;
#pragma unroll
    for (int i = 0; i < NC; ++i) sm += i < n ? fast_exp2(z[i] - m) : 0.f;
    return m + fast_log2(sm);
  } else {
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < NC; ++i) sum += i < n ? z[i] : 0.f;
    const float mean = sum / static_cast<float>(n);
    if constexpr (KIND == kScoreMean) {
      return mean;
    } else {
      float m2 = 0.f;
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const float dv = z[i] - mean;
        m2 += i < n ? dv * dv : 0.f;
      }
      return mean + 0.5f * kLn2 * (m2 / static_cast<float>(n));
    }
  }
}

constexpr int kMfmaSelRows = 4;  // rows (wavefronts) per workgroup

template <int D, int GC, int KIND>
__global__ __launch_bounds__(kMfmaSelRows * 64) void stage1_mfma_kernel(SelArgs a, const uint16_t* __restrict__ hilo) {
  constexpr int KS = D / 32;      // 32-dim steps
  constexpr int CPL = 4 / GC;     // candidates per lane in the result layout
  constexpr int CPT = 16 / GC;    // candidates per 16-row tile
  __shared__ int s_cand[kMfmaSelRows][128];
  __shared__ int s_cand2[kMfmaSelRows][128];
  __shared__ int s_flag[kMfmaSelRows][128];
  __shared__ float s_score[kMfmaSelRows][128];
  const Geo& geo = a.geo;
  const int G = a.G, K = a.K, gK = a.gK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = blockIdx.x * kMfmaSelRows + wave;
  if (row >= a.Nq) return;  // the whole wavefront leaves; only wavefront-level syncs follow
  int* cand = s_cand[wave];
  int* cand2 = s_cand2[wave];
  int* flag = s_flag[wave];
  float* score = s_score[wave];
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = geo.N - a.Nq + row;
  const int c = t / geo.C;
  const int col = lane & 15, quad = lane >> 4;

  bf16x8m qB[KS];
  {
    const bool hv = col < G;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) +
                           ((static_cast<int64_t>(b) * a.H + h * G + (hv ? col : 0)) * a.Nq + row) * D + 8 * quad;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (hv) u = *reinterpret_cast<const uint4*>(qrow + ks * 32);
      qB[ks] = __builtin_bit_cast(bf16x8m, u);
    }
  }

  if (lane == 0) cand[0] = 0;
  int nA = 1;
  wave_sync();
  for (int lev = geo.L; lev >= 2; --lev) {
    const Forced fz = forced_at(geo, lev, c, a.causal);
    const bool ranked = nA > K;
    if (ranked) {
      const int Mb = geo.M[lev - 1];
      const uint16_t* pb = hilo + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * (2 * D) + 16 * quad;
      const int ntile = (nA * GC + 15) / 16;
      for (int tile = 0; tile < ntile; ++tile) {
        // A operand: tile row r = (candidate r / GC, child r % GC)
        const int r = tile * 16 + col;
        const int ci = r / GC, j = r % GC;
        bool ok = false;
        int crow = 0;
        if (ci < nA) {
          const int node = cand[ci];
          crow = node * GC + j;
          ok = crow < Mb && !fz.is(node);
        }
        const uint16_t* ar = pb + static_cast<int64_t>(ok ? crow : 0) * (2 * D);
        uint4 hi[KS], lo[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          hi[ks] = make_uint4(0, 0, 0, 0);
          lo[ks] = make_uint4(0, 0, 0, 0);
          if (ok) {
            hi[ks] = *reinterpret_cast<const uint4*>(ar + ks * 64);
            lo[ks] = *reinterpret_cast<const uint4*>(ar + ks * 64 + 8);
          }
        }
        f32x4m acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8m, hi[ks]), qB[ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8m, lo[ks]), qB[ks], acc, 0, 0, 0);
        }
        // This lane: tile rows 4*quad + i of head col; candidate(s) tile*CPT + CPL*quad + k.
#pragma unroll
        for (int k2 = 0; k2 < CPL; ++k2) {
          const int cj = tile * CPT + CPL * quad + k2;
          float z[GC];
#pragma unroll
          for (int i = 0; i < GC; ++i) z[i] = acc[k2 * GC + i] * a.qscale2;
          int n = 1;
          if (cj < nA) n = max(1, min(GC, Mb - cand[cj] * GC));
          float u = col < G ? lane_children_score<KIND, GC>(z, n) : 0.f;
          u = rowsum16_to15(u);
          if (col == 15 && cj < nA) score[cj] = u;
        }
      }
      wave_sync();
      // Forced candidates first, then score descending, ties by candidate
      // index (candidates are ascending node ids), then empty slots.
      const int keepn = K - fz.count();
      if (nA <= 32) {  // one 32-lane sort (the upper half sorts nothing of use)
        const bool v = lane < nA;
        const bool f = v && fz.is(cand[lane]);
        float key = !v ? -INFINITY : (f ? INFINITY : score[lane]);
        int pack = lane;
        const int nforced = __popcll(__ballot(f));
        sort32(key, pack, lane & 31);
        if (lane < nA) flag[pack] = (lane < nforced || lane - nforced < keepn) ? 1 : 0;
      } else {  // two candidates per lane: the 128-entry sort (forced keyed below every score)
        uint32_t khi[2], klo[2];
        int nforced = 0;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int ci = lane + 64 * s2;
          const bool v = ci < nA;
          const bool f = v && fz.is(cand[ci]);
          khi[s2] = !v ? 0xFFFFFFFFu : (f ? 0u : desc_bits(score[ci]));
          klo[s2] = static_cast<uint32_t>(ci);
          nforced += __popcll(__ballot(f));
        }
        sort128(khi, klo, lane);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int rk = lane + 64 * s2;
          if (static_cast<int>(klo[s2]) < nA) flag[klo[s2]] = (rk < nforced || rk - nforced < keepn) ? 1 : 0;
        }
      }
    } else {
      for (int ci = lane; ci < nA; ci += 64) flag[ci] = 1;
    }
    wave_sync();
    // Expand kept nodes to their eligible children at level lev-1.
    const int Mb = geo.M[lev - 1];
    const int rmax = a.causal ? min(anc_at(geo, c, lev - 1), Mb - 1) : Mb - 1;
    const int i0 = lane * 2, i1 = min(nA, i0 + 2);
    int mine = 0;
    for (int ci = i0; ci < i1; ++ci) {
      if (flag[ci]) {
        const int c0 = cand[ci] * GC;
        mine += max(0, min(c0 + GC - 1, rmax) - c0 + 1);
      }
    }
    int total;
    int pos = team_scan<64>(mine, nullptr, total);
    for (int ci = i0; ci < i1; ++ci) {
      if (flag[ci]) {
        const int c0 = cand[ci] * GC;
        const int n = max(0, min(c0 + GC - 1, rmax) - c0 + 1);
        for (int jj = 0; jj < n; ++jj) cand2[pos + jj] = c0 + jj;
        pos += n;
      }
    }
    wave_sync();
    for (int ci = lane; ci < total; ci += 64) cand[ci] = cand2[ci];
    nA = total;
    wave_sync();
  }

  const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row;
  for (int ci = lane; ci < gK; ci += 64) a.a1[orow * gK + ci] = ci < nA ? cand[ci] : -1;
  if (lane == 0) a.a1cnt[orow] = nA;
}

// Stage 1 on the matrix cores for kUnionRows consecutive query rows per
// wavefront (G = 1, 2 or 4 heads per KV head, so that the rows' heads fill at
// most the 16 columns of a tile): each ranked level scores the union of the
// rows' candidate sets once, column r*G + h of the tile being head h of row
// r, so that rows whose candidates coincide (neighbouring queries mostly
// select the same nodes) share every summary load; each row then ranks its
// own candidates with the union's scores.  The union is built through a
// bitmap over the level's nodes, so it comes out ascending, and a node's
// place in it is the population count below its bit.  Products, scores,
// ranking and expansion are otherwise those of stage1_mfma_kernel.
constexpr int kUnionRows = 4;   // query rows per wavefront
constexpr int kUnionWaves = 4;  // wavefronts per workgroup

// LDS words of one wavefront of stage1_union_kernel.
__host__ __device__ constexpr int union_wave_words(int bm_words) {
  return kUnionRows * 128 * 3 + kUnionRows * 128 + kUnionRows * 128 * kUnionRows + 2 * (bm_words + 1);
}

template <int D, int GC, int KIND>
__global__ __launch_bounds__(kUnionWaves * 64) void stage1_union_kernel(SelArgs a, const uint16_t* __restrict__ hilo,
                                                                       int bm_words) {
  constexpr int KS = D / 32;
  constexpr int CPL = 4 / GC;   // union candidates per lane in the result layout
  constexpr int CPT = 16 / GC;  // union candidates per 16-row tile
  constexpr int R = kUnionRows;
  constexpr int UMAX = R * 128;
  extern __shared__ __align__(16) int lds_u[];
  const Geo& geo = a.geo;
  const int G = a.G, K = a.K, gK = a.gK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = (blockIdx.x * kUnionWaves + wave) * R;
  if (row0 >= a.Nq) return;  // the whole wavefront leaves; only wavefront-level syncs follow
  int* L = lds_u + wave * union_wave_words(bm_words);
  int* cand = L;                     // [R][128]
  int* cand2 = cand + R * 128;       // [R][128]
  int* flag = cand2 + R * 128;       // [R][128]
  int* U = flag + R * 128;           // [UMAX] union, ascending
  float* us = reinterpret_cast<float*>(U + UMAX);  // [UMAX][R] scores of the union for each row
  uint32_t* bm = reinterpret_cast<uint32_t*>(us + UMAX * R);  // [bm_words + 1]
  int* pre = reinterpret_cast<int*>(bm + bm_words + 1);       // [bm_words + 1]
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int col = lane & 15, quad = lane >> 4;
  const int crow_r = col / G, chh = col - crow_r * G;  // this lane's column: row crow_r, head chh
  const bool cvalid = col < R * G && row0 + crow_r < a.Nq;

  bf16x8m qB[KS];
  {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) +
                           ((static_cast<int64_t>(b) * a.H + h * G + (cvalid ? chh : 0)) * a.Nq +
                            (cvalid ? row0 + crow_r : 0)) * D + 8 * quad;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (cvalid) u = *reinterpret_cast<const uint4*>(qrow + ks * 32);
      qB[ks] = __builtin_bit_cast(bf16x8m, u);
    }
  }

  int nAr[R], cr[R];
  bool rv[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    rv[r] = row0 + r < a.Nq;
    nAr[r] = 1;
    cr[r] = (geo.N - a.Nq + row0 + r) / geo.C;
    if (lane == 0) cand[r * 128] = 0;
  }
  wave_sync();
  for (int lev = geo.L; lev >= 2; --lev) {
    const int Mb = geo.M[lev - 1];
    bool rk[R];
    bool any = false;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      rk[r] = rv[r] && nAr[r] > K;
      any = any || rk[r];
    }
    if (any) {
      // 1) the union of the ranked rows' candidates
      const int nw = (geo.M[lev] + 31) / 32;
      for (int w = lane; w < nw; w += 64) bm[w] = 0u;
      wave_sync();
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (!rk[r]) continue;
        for (int ci = lane; ci < nAr[r]; ci += 64) {
          const int node = cand[r * 128 + ci];
          atomicOr(&bm[node >> 5], 1u << (node & 31));
        }
      }
      wave_sync();
      const int wpl = (nw + 63) / 64;
      const int w0 = min(nw, lane * wpl), w1 = min(nw, w0 + wpl);
      int mine = 0;
      for (int w = w0; w < w1; ++w) mine += __popc(bm[w]);
      int nU;
      int pos = team_scan<64>(mine, nullptr, nU);
      for (int w = w0; w < w1; ++w) {
        pre[w] = pos;
        uint32_t bits = bm[w];
        while (bits) {
          U[pos++] = w * 32 + __ffs(bits) - 1;
          bits &= bits - 1;
        }
      }
      wave_sync();
      // 2) the union's child logits, tile by tile, every row's heads as columns
      const uint16_t* pb = hilo + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * (2 * D) + 16 * quad;
      const int ntile = (nU * GC + 15) / 16;
      for (int tile = 0; tile < ntile; ++tile) {
        const int rr = tile * 16 + col;
        const int ui = rr / GC, j = rr % GC;
        bool ok = false;
        int crow = 0;
        if (ui < nU) {
          crow = U[ui] * GC + j;
          ok = crow < Mb;
        }
        const uint16_t* ar = pb + static_cast<int64_t>(ok ? crow : 0) * (2 * D);
        uint4 hi[KS], lo[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          hi[ks] = make_uint4(0, 0, 0, 0);
          lo[ks] = make_uint4(0, 0, 0, 0);
          if (ok) {
            hi[ks] = *reinterpret_cast<const uint4*>(ar + ks * 64);
            lo[ks] = *reinterpret_cast<const uint4*>(ar + ks * 64 + 8);
          }
        }
        f32x4m acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8m, hi[ks]), qB[ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8m, lo[ks]), qB[ks], acc, 0, 0, 0);
        }
#pragma unroll
        for (int k2 = 0; k2 < CPL; ++k2) {
          const int cj = tile * CPT + CPL * quad + k2;
          float z[GC];
#pragma unroll
          for (int i = 0; i < GC; ++i) z[i] = acc[k2 * GC + i] * a.qscale2;
          int n = 1;
          if (cj < nU) n = max(1, min(GC, Mb - U[cj] * GC));
          float u = cvalid ? lane_children_score<KIND, GC>(z, n) : 0.f;
          // the G heads of a row sit in G neighbouring lanes of the 16-lane row
          for (int o = 1; o < G; o <<= 1) u += __shfl_xor(u, o);
          if (cvalid && chh == 0 && cj < nU) us[cj * R + crow_r] = u;
        }
      }
      wave_sync();
      // 3) each ranked row ranks its own candidates with the union's scores:
      // forced first, then score descending, ties by candidate index
      // (ascending nodes), then empty slots
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (!rk[r]) continue;
        const Forced fz = forced_at(geo, lev, cr[r], a.causal);
        const int keepn = K - fz.count();
        const int nA = nAr[r];
        const int* cr_ = cand + r * 128;
        auto score_of = [&](int node) {
          const int w = node >> 5;
          const int ui = pre[w] + __popc(bm[w] & ((1u << (node & 31)) - 1u));
          return us[ui * R + r];
        };
        int* fl = flag + r * 128;
        if (nA <= 32) {
          const bool v = lane < nA;
          const int node = v ? cr_[lane] : 0;
          const bool f = v && fz.is(node);
          float key = !v ? -INFINITY : (f ? INFINITY : score_of(node));
          int pack = lane;
          const int nforced = __popcll(__ballot(f));
          sort32(key, pack, lane & 31);
          if (lane < nA) fl[pack] = (lane < nforced || lane - nforced < keepn) ? 1 : 0;
        } else {
          uint32_t khi[2], klo[2];
          int nforced = 0;
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const int ci = lane + 64 * s2;
            const bool v = ci < nA;
            const int node = v ? cr_[ci] : 0;
            const bool f = v && fz.is(node);
            khi[s2] = !v ? 0xFFFFFFFFu : (f ? 0u : desc_bits(score_of(node)));
            klo[s2] = static_cast<uint32_t>(ci);
            nforced += __popcll(__ballot(f));
          }
          sort128(khi, klo, lane);
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const int rk2 = lane + 64 * s2;
            if (static_cast<int>(klo[s2]) < nA) fl[klo[s2]] = (rk2 < nforced || rk2 - nforced < keepn) ? 1 : 0;
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (rv[r] && !rk[r])
        for (int ci = lane; ci < nAr[r]; ci += 64) flag[r * 128 + ci] = 1;
    }
    wave_sync();
    // 4) each row expands its kept nodes to their eligible children
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!rv[r]) continue;
      const int rmax = a.causal ? min(anc_at(geo, cr[r], lev - 1), Mb - 1) : Mb - 1;
      const int* cr_ = cand + r * 128;
      const int* fl = flag + r * 128;
      int* c2 = cand2 + r * 128;
      const int i0 = lane * 2, i1 = min(nAr[r], i0 + 2);
      int mine = 0;
      for (int ci = i0; ci < i1; ++ci) {
        if (fl[ci]) {
          const int c0 = cr_[ci] * GC;
          mine += max(0, min(c0 + GC - 1, rmax) - c0 + 1);
        }
      }
      int total;
      int pos = team_scan<64>(mine, nullptr, total);
      for (int ci = i0; ci < i1; ++ci) {
        if (fl[ci]) {
          const int c0 = cr_[ci] * GC;
          const int n = max(0, min(c0 + GC - 1, rmax) - c0 + 1);
          for (int jj = 0; jj < n; ++jj) c2[pos + jj] = c0 + jj;
          pos += n;
        }
      }
      nAr[r] = total;
    }
    wave_sync();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!rv[r]) continue;
      for (int ci = lane; ci < nAr[r]; ci += 64) cand[r * 128 + ci] = cand2[r * 128 + ci];
    }
    wave_sync();
  }

#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (!rv[r]) continue;
    const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row0 + r;
    for (int ci = lane; ci < gK; ci += 64) a.a1[orow * gK + ci] = ci < nAr[r] ? cand[r * 128 + ci] : -1;
    if (lane == 0) a.a1cnt[orow] = nAr[r];
  }
}

// Summaries as bf16 pairs for stage1_mfma_kernel: each group of 8 fp32
// values becomes 8 rounded values (hi) followed by 8 rounded remainders (lo).
__global__ __launch_bounds__(256) void pyr_hilo_kernel(const float* __restrict__ pyr, uint16_t* __restrict__ hilo,
                                                       int64_t ngroups) {
  const int64_t i = blockIdx.x * 256LL + threadIdx.x;
  if (i >= ngroups) return;
  const float4 x0 = reinterpret_cast<const float4*>(pyr)[2 * i];
  const float4 x1 = reinterpret_cast<const float4*>(pyr)[2 * i + 1];
  const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
  uint32_t hw[4], lw[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hw[e] = pack2_bf16(x[2 * e], x[2 * e + 1]);
    const float h0 = __uint_as_float(hw[e] << 16), h1 = __uint_as_float(hw[e] & 0xFFFF0000u);
    lw[e] = pack2_bf16(x[2 * e] - h0, x[2 * e + 1] - h1);
  }
  uint4* out = reinterpret_cast<uint4*>(hilo) + 2 * i;
  out[0] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
  out[1] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
}


// Total of a 32-lane half from an inclusive scan.
__device__ __forceinline__ int half_total(int incl, int lane) {
  const int t0 = __builtin_amdgcn_readlane(incl, 31);
  const int t1 = __builtin_amdgcn_readlane(incl, 63);
  return lane < 32 ? t0 : t1;
}

// Sum over each aligned group of LPE lanes (LPE in {4, 8, 16}); the total
// lands in the group's last lane.
template <int LPE>
__device__ __forceinline__ float group_sum_to_last(float v) {
  v += dpp_f<0x111>(v);
  v += dpp_f<0x112>(v);
  if constexpr (LPE >= 8) v += dpp_f<0x114>(v);
  if constexpr (LPE >= 16) v += dpp_f<0x118>(v);
  return v;
}

// LPE lanes share one child dot; lane s of a group holds the 16-byte chunks
// s, s + LPE, s + 2 LPE, ... of the row, so each load instruction reads
// whole 128-byte lines.
template <int D, int GMAX, int LPE>
__global__ __launch_bounds__(256) void stage1_pair_kernel(SelArgs a, int row_words) {
  constexpr int DPL = D / LPE;      // floats per lane
  constexpr int NCH = DPL / 4;      // 16-byte chunks per lane
  constexpr int NG = 32 / LPE;      // lane groups per half
  constexpr int UNR = DPL >= 32 ? 1 : (32 / DPL > 4 ? 4 : 32 / DPL);
  extern __shared__ __align__(16) int lds_i[];
  const Geo& geo = a.geo;
  const int g = geo.g, G = a.G, K = a.K, gK = a.gK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, hl = lane & 31;
  const int gr = hl / LPE;  // lane group within the half
  const int sub = hl % LPE;
  int* L = lds_i + (wave * 2 + half) * row_words;
  int* lst_r = L;                                   // [gK*g] child row to load
  int* lst_s = lst_r + gK * g;                      // [gK*g] zbuf slot of that child
  int* cand2 = lst_s + gK * g;                      // [gK]
  float* zbuf = reinterpret_cast<float*>(cand2 + gK);  // [gK*g*G]
  float* zs2 = zbuf + gK * g * G;                   // [gK*G]

  const int row = (blockIdx.x * 4 + wave) * 2 + half;
  const bool live = row < a.Nq;
  const int rowc = live ? row : a.Nq - 1;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = geo.N - a.Nq + rowc;
  const int c = t / geo.C;

  float qv[GMAX][DPL];
  {
    const uint16_t* qb = static_cast<const uint16_t*>(a.q);
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < G) {
        const int64_t off = ((static_cast<int64_t>(b) * a.H + h * G + hh) * a.Nq + rowc) * D + sub * 4;
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
          float x4[4];
          load_row_part<uint16_t, 4>(qb + off + ch * 4 * LPE, x4);
#pragma unroll
          for (int e = 0; e < 4; ++e) qv[hh][ch * 4 + e] = x4[e] * a.qscale2;
        }
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) qv[hh][e] = 0.f;
      }
    }
  }

  // Levels whose eligible nodes number at most K keep everything, so the
  // candidate set of the first level that can hold more than K is simply
  // all its eligible nodes: each row starts there (the root level when none
  // can, i.e. the whole set reaches the leaf level unpruned).
  auto n_eligible = [&](int lev) { return a.causal ? min(anc_at(geo, c, lev) + 1, geo.M[lev]) : geo.M[lev]; };
  int start = 1;
  for (int lev = geo.L; lev >= 2; --lev) {
    if (n_eligible(lev) > K) {
      start = lev;
      break;
    }
  }
  // start == 1: fewer than K+1 eligible leaves; start >= 2: first ranked level.
  const int wave_start = max(start, __shfl_xor(start, 32));

  int node = -1;  // candidate of this lane (-1: none)
  float zs[GMAX];  // its logit per head, NaN if unknown
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) zs[hh] = __builtin_nanf("");
  int nA = 0;

  for (int lev = wave_start; lev >= 2; --lev) {
    if (lev == start) {
      nA = n_eligible(lev);
      node = hl < nA ? hl : -1;
    }
    const bool active = lev <= start;
    const Forced fz = forced_at(geo, lev, c, a.causal);
    const bool ranked = active && nA > K;
    const int Mb = geo.M[lev - 1];
    const bool valid = node >= 0;
    const bool isf = valid && fz.is(node);
    const int nch = valid ? min(g, Mb - node * g) : 0;
    float key = valid ? INFINITY : -INFINITY;
    if (ranked) {
      // 1) compact list of the child rows to load
      const bool has_self = !__builtin_isnan(zs[0]);
      const int nl = (valid && !isf) ? (has_self ? nch - 1 : nch) : 0;
      const int incl = scan32(nl, hl);
      const int T = half_total(incl, lane);
      int pos = incl - nl;
      for (int j = 0; j < nl; ++j) {
        lst_r[pos + j] = node * g + j;
        lst_s[pos + j] = hl * g + j;
      }
      wave_sync();
      // 2) child logits, UNR loads in flight per 16-lane group (loads past the
      //    list end fetch row 0 and are discarded)
      const float* pbase = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * D + sub * 4;
      for (int e0 = gr; e0 < T; e0 += NG * UNR) {
        float x[UNR][DPL];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int e = e0 + NG * u;
          const int r = e < T ? lst_r[e] : 0;
#pragma unroll
          for (int ch = 0; ch < NCH; ++ch) {
            const float4 v4 = *reinterpret_cast<const float4*>(pbase + static_cast<int64_t>(r) * D + ch * 4 * LPE);
            x[u][ch * 4 + 0] = v4.x;
            x[u][ch * 4 + 1] = v4.y;
            x[u][ch * 4 + 2] = v4.z;
            x[u][ch * 4 + 3] = v4.w;
          }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int e = e0 + NG * u;
#pragma unroll
          for (int hh = 0; hh < GMAX; ++hh) {
            if (hh < G) {
              float d0 = 0.f;
#pragma unroll
              for (int i = 0; i < DPL; ++i) d0 = fmaf(qv[hh][i], x[u][i], d0);
              d0 = group_sum_to_last<LPE>(d0);
              if (sub == LPE - 1 && e < T) zbuf[lst_s[e] * G + hh] = d0;
            }
          }
        }
      }
      wave_sync();
      // 3) this lane's candidate score
      if (valid && !isf) {
        float u = 0.f;
#pragma unroll
        for (int hh = 0; hh < GMAX; ++hh) {
          if (hh < G) {
            float* zc = zbuf + hl * g * G + hh;
            if (has_self) {
              float others = 0.f;
              for (int j = 0; j < nch - 1; ++j) others += zc[j * G];
              zc[(nch - 1) * G] = static_cast<float>(nch) * zs[hh] - others;
            }
            u += reduce_logits(a.score_kind, zc, nch, G);
          }
        }
        key = u;
      }
    }
    // 4) rank: the first K in (key desc, node asc) order survive
    int knode = node, korig = hl;
    bool kept = active && valid;
    if (__ballot(ranked) != 0) {
      int pack = valid ? (node << 6) | hl : 0x7FFFFFC0 | hl;
      float skey = key;
      sort32(skey, pack, hl);
      if (ranked) {
        kept = hl < K && skey != -INFINITY;
        knode = pack >> 6;
        korig = pack & 63;
      }
    }
    const bool known = ranked && kept && !fz.is(knode);
    wave_sync();  // zbuf reads of step 3 are done before cand2/zs2 are written
    // 5) expand survivors to their eligible children
    const int rmax = a.causal ? min(anc_at(geo, c, lev - 1), Mb - 1) : Mb - 1;
    const int c0 = knode * g;
    const int nk = kept ? max(0, min(c0 + g - 1, rmax) - c0 + 1) : 0;
    const int incl = scan32(nk, hl);
    const int nA2 = half_total(incl, lane);
    int pos = incl - nk;
    for (int j = 0; j < nk; ++j) {
      cand2[pos + j] = c0 + j;
      for (int hh = 0; hh < G; ++hh)
        zs2[(pos + j) * G + hh] = known ? zbuf[(korig * g + j) * G + hh] : __builtin_nanf("");
    }
    wave_sync();
    if (active) {
      node = hl < nA2 ? cand2[hl] : -1;
#pragma unroll
      for (int hh = 0; hh < GMAX; ++hh) zs[hh] = (hh < G && hl < nA2) ? zs2[hl * G + hh] : __builtin_nanf("");
      nA = nA2;
    }
    wave_sync();
  }
  if (start == 1) {  // every eligible leaf survives unranked
    nA = n_eligible(1);
    node = hl < nA ? hl : -1;
  }

  // Leaf candidate set ascending.
  float akey = node >= 0 ? -static_cast<float>(node) : -INFINITY;
  int apack = node >= 0 ? node : 0x7FFFFFC0 | hl;
  sort32(akey, apack, hl);
  if (live) {
    const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row;
    if (hl < gK) a.a1[orow * gK + hl] = hl < nA ? apack : -1;
    if (hl == 0) a.a1cnt[orow] = nA;
  }
}

// ----------------------------------------------------------------------------
// Stage 1 for fan-out 2 and K <= 16: two query rows per wavefront, lane hl of
// a half owns candidate slot hl, with no LDS lists.
//
//   * Child logits: the LPE lanes of a dot group compute the dots of their
//     own LPE slots (each lane loads 16-byte chunks sub, sub+LPE, ... of every
//     row) and a reduce-scatter leaves slot j's logit in lane j of the group.
//     Every valid slot, forced or not, gets both child logits: child 0 by a
//     dot, child 1 derived from the node's own logit (a summary is the mean of
//     its two children, so z1 = 2 z - z0), except on the row's first ranked
//     level, where own logits are unknown and child 1 is a dot as well.
//   * Rank: key = score (scored), +inf (forced, or every valid slot of an
//     unranked level), -inf (empty slot); a 32-lane bitonic sort puts the
//     survivors in lanes 0 .. min(K, #valid) - 1.
//   * Expand: slot s of the next level is child s & 1 of survivor s >> 1; its
//     node and its own logit come from the survivor's lanes by lane permutes.
// ----------------------------------------------------------------------------

// Broadcast lane j of each LPE-lane group to the whole group.
template <int LPE>
__device__ __forceinline__ int group_bcast(int v, int j, int lane) {
  if constexpr (LPE == 4) {
    switch (j) {
      case 0: return dpp_i<0x00>(v);
      case 1: return dpp_i<0x55>(v);
      case 2: return dpp_i<0xAA>(v);
      default: return dpp_i<0xFF>(v);
    }
  } else {
    return __shfl(v, (lane & ~(LPE - 1)) | j);
  }
}

// One reduce-scatter step over partner lane ^ M: of each pair (k, k | M) the
// lane keeps the entry whose bit M matches its own and adds the partner's copy.
template <int M>
__device__ __forceinline__ void rs_step(float* w, int sub) {
  const bool up = (sub & M) != 0;
#pragma unroll
  for (int k = 0; k < M; ++k) {
    const float send = up ? w[k] : w[k | M];
    const float mine = up ? w[k | M] : w[k];
    w[k] = mine + xor32_f<M>(send);
  }
}

// Lane sub of an LPE-lane group ends with the group total of w[sub].
template <int LPE>
__device__ __forceinline__ float reduce_scatter(float (&w)[LPE], int sub) {
  if constexpr (LPE >= 16) rs_step<8>(w, sub);
  if constexpr (LPE >= 8) rs_step<4>(w, sub);
  if constexpr (LPE >= 4) rs_step<2>(w, sub);
  rs_step<1>(w, sub);
  return w[0];
}

// Logits of pyramid row `ri` (this lane's slot) against every head's query:
// the group's LPE rows are loaded together, lane sub reading chunks
// sub, sub + LPE, ... of each.  `base` (row 0 of the level, the same for the
// whole wavefront) plus a 32-bit byte offset per row keeps the address
// arithmetic to one instruction per row.
template <int D, int GMAX, int LPE, int INFLIGHT, int RS = D>
__device__ __forceinline__ void slot_dots(const float* __restrict__ base, int ri, const float (&qv)[GMAX][D / LPE],
                                          int sub, int lane, float (&z)[GMAX]) {
  constexpr int NCH = D / LPE / 4;
  constexpr int UNR = INFLIGHT < LPE ? INFLIGHT : LPE;  // rows whose loads are issued together
  float w[GMAX][LPE];
#pragma unroll
  for (int j0 = 0; j0 < LPE; j0 += UNR) {
    float4 x[UNR][NCH];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int rj = group_bcast<LPE>(ri, j0 + u, lane);
      const uint32_t boff = (__umul24(static_cast<uint32_t>(rj), RS) + static_cast<uint32_t>(sub) * 4u) * 4u;
      const char* rp = reinterpret_cast<const char*>(base) + boff;
#pragma unroll
      for (int i = 0; i < NCH; ++i) x[u][i] = *reinterpret_cast<const float4*>(rp + i * LPE * 16);
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
#pragma unroll
      for (int hh = 0; hh < GMAX; ++hh) {  // heads past G have zero queries
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
          acc = fmaf(qv[hh][4 * i + 0], x[u][i].x, acc);
          acc = fmaf(qv[hh][4 * i + 1], x[u][i].y, acc);
          acc = fmaf(qv[hh][4 * i + 2], x[u][i].z, acc);
          acc = fmaf(qv[hh][4 * i + 3], x[u][i].w, acc);
        }
        w[hh][j0 + u] = acc;
      }
    }
  }
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) z[hh] = reduce_scatter<LPE>(w[hh], sub);
}

// Score of a node from its two child logits (z1 = -inf: a single child).
template <int KIND>
__device__ __forceinline__ float pair_score(float z0, float z1) {
  if constexpr (KIND == kScoreLse) {
    const float m = fmaxf(z0, z1), n = fminf(z0, z1);
    return m + fast_log2(1.f + fast_exp2(n - m));
  } else {
    const bool two = z1 != -INFINITY;
    const float mean = two ? 0.5f * (z0 + z1) : z0;
    if constexpr (KIND == kScoreMean) {
      return mean;
    } else {
      const float h = two ? 0.5f * (z0 - z1) : 0.f;
      return mean + 0.5f * kLn2 * (h * h);
    }
  }
}

// One level of the fan-out-2 walk for the two rows of a wavefront: rank the
// slots (first K in (key desc, node asc) order survive; scored slots keyed by
// their summed score, forced slots and every slot of an unranked level +inf,
// empty slots -inf) and expand the survivors: slot s of the next level is
// child s & 1 of survivor s >> 1, its own logits taken from the survivor's
// child logits.  A half idle on this level (lev above its start) stays idle.
template <int GMAX, int KIND>
__device__ __forceinline__ void g2_rank_expand(const Geo& geo, int lev, int c, int causal, int K, int G, int start,
                                               int hl, int hbase, int& node, const float (&z0)[GMAX],
                                               const float (&z1)[GMAX], float (&zs)[GMAX]) {
  const int lb = lev - 1;
  const int Mb = geo.M[lb];
  const bool valid = node >= 0;
  const int nvalid = __builtin_popcount(static_cast<uint32_t>(__ballot(valid) >> hbase));
  const bool ranked = nvalid > K;  // more candidates than the budget
  const Forced fz = forced_at(geo, lev, c, causal);
  float key = -INFINITY;
  if (valid) {
    if (ranked && !fz.is(node)) {
      float u = 0.f;
#pragma unroll
      for (int hh = 0; hh < GMAX; ++hh) {
        const float sc = pair_score<KIND>(z0[hh], z1[hh]);
        u += hh < G ? sc : 0.f;
      }
      key = u;
    } else {
      key = INFINITY;
    }
  }
  int pack = valid ? (node << 6) | hl : 0x7FFFFFC0 | hl;
  // With K = 16 only the set of the best 16 matters (a survivor's place
  // among the next level's slots does not), so the sort stops early; the
  // survivors then sit in lanes 0-15 in any order, empty slots among them.
  sort32_top16(key, pack, hl, K != 16);
  const int nkept = K == 16 ? 16 : min(K, nvalid);

  const int r = hl >> 1;
  const int pr = __shfl(pack, hbase | r);
  const int korig = pr & 63;
  const int rmax = causal ? min(anc_at(geo, c, lb), Mb - 1) : Mb - 1;
  const int cn = 2 * (pr >> 6) + (hl & 1);
  const bool cvalid = r < nkept && pr < 0x7FFFFFC0 && cn <= rmax;
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) {
    const float a0 = __shfl(z0[hh], hbase | korig);
    const float a1v = __shfl(z1[hh], hbase | korig);
    zs[hh] = (hl & 1) ? a1v : a0;
  }
  if (lev <= start) node = cvalid ? cn : -1;
}

// Store a half's leaf candidate set in ascending order, -1 padded to g*K.
__device__ __forceinline__ void g2_store_leaves(const SelArgs& a, int bh, int row, bool live, int hl, int hbase,
                                                int node) {
  const int nA = __builtin_popcount(static_cast<uint32_t>(__ballot(node >= 0) >> hbase));
  float akey = node >= 0 ? -static_cast<float>(node) : -INFINITY;
  int apack = node >= 0 ? node : 0x7FFFFFC0 | hl;
  sort32(akey, apack, hl);
  if (live) {
    const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row;
    if (hl < a.gK) a.a1[orow * a.gK + hl] = hl < nA ? apack : -1;
    if (hl == 0) a.a1cnt[orow] = nA;
  }
}

// Stage-1 coarse levels kept in LDS by a workgroup (fp32 rows padded to
// D + 4 floats): the budget in floats.
constexpr int kStageFloats = 16384;  // 64 KiB: two workgroups of 8 wavefronts per CU

template <int D, int GMAX, int LPE, int KIND, int NWAVE, bool STAGE>
__global__ __launch_bounds__(NWAVE * 64) void stage1_g2_kernel(SelArgs a) {
  constexpr int DPL = D / LPE;
  constexpr int NCH = DPL / 4;
  constexpr int SROW = D + 4;
  const Geo& geo = a.geo;
  const int G = a.G, K = a.K, gK = a.gK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, hl = lane & 31, hbase = lane & 32;
  const int sub = hl % LPE;
  const int row = (blockIdx.x * NWAVE + wave) * 2 + half;
  const bool live = row < a.Nq;
  const int rowc = live ? row : a.Nq - 1;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = geo.N - a.Nq + rowc;
  const int c = t / geo.C;

  float qv[GMAX][DPL];
  {
    const uint16_t* qb = static_cast<const uint16_t*>(a.q);
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < G) {
        const int64_t off = ((static_cast<int64_t>(b) * a.H + h * G + hh) * a.Nq + rowc) * D + sub * 4;
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
          float x4[4];
          load_row_part<uint16_t, 4>(qb + off + ch * 4 * LPE, x4);
#pragma unroll
          for (int e = 0; e < 4; ++e) qv[hh][ch * 4 + e] = x4[e] * a.qscale2;
        }
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) qv[hh][e] = 0.f;
      }
    }
  }

  auto n_eligible = [&](int lev) { return a.causal ? min(anc_at(geo, c, lev) + 1, geo.M[lev]) : geo.M[lev]; };
  int start = 1;  // first level holding more than K eligible nodes (1: none)
  for (int lev = geo.L; lev >= 2; --lev) {
    if (n_eligible(lev) > K) {
      start = lev;
      break;
    }
  }
  // the same in every lane; readfirstlane lets the compiler keep the level
  // loop, and every per-level address, in scalar registers
  const int wave_start = __builtin_amdgcn_readfirstlane(max(start, __shfl_xor(start, 32)));

  // Coarse levels in LDS: every level read by the workgroup's rows, from the
  // coarsest down, whose eligible prefix (for the last row, plus one row for
  // the second child of the last eligible node) still fits the budget; each
  // row then reads them from LDS instead of through the L1 data path.
  extern __shared__ __align__(16) float stg[];
  int stage_lo = 1 << 30, stage_hi = -1;  // staged levels [stage_lo, stage_hi]
  auto stage_rows = [&](int cl, int lb) {
    const int e = a.causal ? anc_at(geo, cl, lb) + 2 : geo.M[lb];
    return min(e, geo.M[lb]);
  };
  int c_last = c;
  if constexpr (STAGE) {
    const int last = min(static_cast<int>(blockIdx.x + 1) * NWAVE * 2, a.Nq) - 1;
    c_last = (geo.N - a.Nq + last) / geo.C;
    int tstart = 1;
    for (int lev = geo.L; lev >= 2; --lev) {
      if ((a.causal ? min(anc_at(geo, c_last, lev) + 1, geo.M[lev]) : geo.M[lev]) > K) {
        tstart = lev;
        break;
      }
    }
    int used = 0;
    for (int lb = tstart - 1; lb >= 1; --lb) {
      const int need = stage_rows(c_last, lb) * SROW;
      if (used + need > kStageFloats) break;
      if (stage_hi < 0) stage_hi = lb;
      stage_lo = lb;
      used += need;
    }
    int off = 0;
    for (int lb = stage_hi; lb >= stage_lo && stage_hi >= 0; --lb) {
      const int nr = stage_rows(c_last, lb);
      const float* src = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lb]) * D;
      for (int e = threadIdx.x; e < nr * (D / 4); e += NWAVE * 64) {
        const int r = e / (D / 4), c4 = (e - r * (D / 4)) * 4;
        *reinterpret_cast<float4*>(stg + off + r * SROW + c4) =
            *reinterpret_cast<const float4*>(src + static_cast<int64_t>(r) * D + c4);
      }
      off += nr * SROW;
    }
    __syncthreads();
  }
  // LDS offset of staged level lb (levels stacked from stage_hi down)
  auto stage_off = [&](int lb) {
    int off = 0;
    for (int l = stage_hi; l > lb; --l) off += stage_rows(c_last, l) * SROW;
    return off;
  };

  int node = -1;  // a half is idle (no valid slot) on the levels above its start
  float zs[GMAX];
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) zs[hh] = 0.f;

  for (int lev = wave_start; lev >= 2; --lev) {
    if (lev == start) node = hl < n_eligible(lev) ? hl : -1;
    const bool fresh = lev == start;
    const int lb = lev - 1;
    const int Mb = geo.M[lb];
    const bool valid = node >= 0;
    const int nch = valid ? min(2, Mb - 2 * node) : 0;
    float z0[GMAX], z1[GMAX];
    const bool two = __ballot(fresh && nch == 2) != 0;
    if (STAGE && lb >= stage_lo && lb <= stage_hi) {
      const float* sbase = stg + stage_off(lb);
      slot_dots<D, GMAX, LPE, 4, SROW>(sbase, valid ? 2 * node : 0, qv, sub, lane, z0);
      if (two) slot_dots<D, GMAX, LPE, 4, SROW>(sbase, nch == 2 ? 2 * node + 1 : 0, qv, sub, lane, z1);
    } else {
      const float* pbase = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lb]) * D;
      slot_dots<D, GMAX, LPE, 4>(pbase, valid ? 2 * node : 0, qv, sub, lane, z0);
      if (two) slot_dots<D, GMAX, LPE, 4>(pbase, nch == 2 ? 2 * node + 1 : 0, qv, sub, lane, z1);
    }
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) z1[hh] = nch < 2 ? -INFINITY : (fresh ? z1[hh] : 2.f * zs[hh] - z0[hh]);

    g2_rank_expand<GMAX, KIND>(geo, lev, c, a.causal, K, G, start, hl, hbase, node, z0, z1, zs);
  }
  if (start == 1) node = hl < n_eligible(1) ? hl : -1;  // every eligible leaf, unranked
  g2_store_leaves(a, bh, row, live, hl, hbase, node);
}

// Final Top-K for g*K <= 32: a row per 32-lane half of a wavefront (RP such
// pairs of rows per wavefront), one candidate per lane (the candidates
// arrive in ascending block order).  sort32 ranks them
// (forced and unranked rows keyed +inf); the rank of each lane's own
// candidate comes back through LDS and the kept ones are compacted in their
// original, ascending order with a prefix sum.
template <int RP>
__global__ __launch_bounds__(256) void final_topk_pair_kernel(TopkArgsP a, const int32_t* __restrict__ a1,
                                                              const int32_t* __restrict__ a1cnt,
                                                              const float* __restrict__ u1,
                                                              int32_t* __restrict__ idx, float* __restrict__ score) {
  __shared__ int s_rank[4][RP][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, hl = lane & 31;
  // RP pairs of rows per wavefront, processed side by side (independent
  // chains whose memory and lane-exchange latencies overlap)
  int64_t rg[RP];
  bool live[RP];
  int n[RP], node_raw[RP], c[RP];
  float u_raw[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    rg[p] = ((blockIdx.x * 4LL + wave) * RP + p) * 2 + half;
    live[p] = rg[p] < a.rows;
    const int64_t rgc = live[p] ? rg[p] : a.rows - 1;
    const int row = static_cast<int>(rgc % a.Nq);
    c[p] = (a.N - a.Nq + row) / a.C;
    // the three loads of a row are independent (slots past the count hold
    // stale workspace values that are masked below)
    const int slot = min(hl, a.gK - 1);
    n[p] = a1cnt[rgc];
    node_raw[p] = a1[rgc * a.gK + slot];
    u_raw[p] = u1[rgc * a.gK + slot];
  }
  float key[RP], own[RP];
  int pack[RP], node[RP];
  bool valid[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const bool ranked = n[p] > a.K;
    valid[p] = hl < n[p];
    node[p] = valid[p] ? node_raw[p] : -1;
    const bool isf = a.causal && valid[p] && (node[p] == 0 || node[p] == c[p] || node[p] == c[p] - 1);
    key[p] = -INFINITY;
    if (valid[p]) key[p] = (ranked && !isf) ? u_raw[p] : INFINITY;
    own[p] = key[p];
    pack[p] = valid[p] ? (node[p] << 6) | hl : 0x7FFFFFC0 | hl;
  }
  // lane q of the sorted half holds rank q (with K = 16 only the best 16 are
  // separated from the rest); send it back to the source lane
#pragma unroll
  for (int p = 0; p < RP; ++p) sort32_top16(key[p], pack[p], hl, a.K != 16);
#pragma unroll
  for (int p = 0; p < RP; ++p) s_rank[wave][p][(lane & 32) + (pack[p] & 63)] = hl;
  wave_sync();
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const bool kept = valid[p] && s_rank[wave][p][lane] < a.K;
    const int incl = scan32(kept ? 1 : 0, hl);
    if (live[p]) {
      const int total = half_total(incl, lane);
      if (kept) {
        idx[rg[p] * a.K + incl - 1] = node[p];
        if (score) score[rg[p] * a.K + incl - 1] = (own[p] == INFINITY) ? INFINITY : own[p] * kLn2;
      }
      if (hl >= total && hl < a.K) {
        idx[rg[p] * a.K + hl] = -1;
        if (score) score[rg[p] * a.K + hl] = -INFINITY;
      }
    }
  }
}

// ----------------------------------------------------------------------------
// Two-stage remainder: cluster build, MFMA leaf scoring, final Top-K.
// ----------------------------------------------------------------------------

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef float f32x16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8v as_bf16x8(uint4 r) {
  return __builtin_bit_cast(bf16x8v, r);
}

constexpr int kLeafChunk = 1024;  // pairs (or (row, parent) entries) per workgroup of the leaf scorers

struct LeafArgs {
  int H, Hkv, G, Nq, N, C, M1, gK;
  float qscale2;
  int Nkv;  // rows per (batch, KV head) in k
};

// One workgroup per chunk of up to kLeafChunk pairs of one (batch x KV head,
// leaf block) cluster: the C x D key block is staged in LDS once (rows padded
// by 16 B against bank conflicts) and the chunk's (query, slot) pairs are
// scored against it, 32 pairs per wavefront MFMA tile.
template <int D, int KIND>
__global__ __launch_bounds__(256) void leaf_score_kernel(LeafArgs a, const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ k,
                                                         const int32_t* __restrict__ offs,
                                                         const int32_t* __restrict__ toffs, int64_t ncl,
                                                         const int32_t* __restrict__ pairs,
                                                         float* __restrict__ u1) {
  constexpr int LDR = D + 8;  // padded LDS row, in bf16 elements
  constexpr int KS = D / 16;
  extern __shared__ __align__(16) uint16_t klds[];
  int64_t cl;
  int beg, end;
  if (!cluster_chunk(offs, toffs, ncl, blockIdx.x, kLeafChunk, cl, beg, end)) return;
  const int bh = static_cast<int>(cl / a.M1);
  const int blk = static_cast<int>(cl - static_cast<int64_t>(bh) * a.M1);
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = blk * a.C;
  const int nrows = min(a.C, a.N - r0);

  // Stage the key block (zero rows past the end of the sequence).
  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
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
      ScoreAcc st = acc_empty(KIND);
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
        // acc[r] is the logit of key kt*32 + 8*(r/4) + 4*half + r%4 for query `col`
        // (-inf past the end of the sequence; a tile may hold no key at all).
        float zv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) zv[r] = acc[r];
        if (kt * 32 + 32 > nrows) {  // a partial tile: keys past the end of the sequence drop out
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
            zv[r] = key < nrows ? zv[r] : -INFINITY;
          }
        }
        acc_merge(KIND, st, acc_of_scaled<KIND, 16>(zv, a.qscale2));
      }
      acc_merge(KIND, st, acc_shfl_xor(st, 32));
      u += acc_value(KIND, st);
    }
    if (valid && half == 0) u1[(static_cast<int64_t>(bh) * a.Nq + row) * a.gK + slot] = u;
  }
}

struct LeafParentArgs {
  int H, Hkv, G, Nq, N, C, g, M1, M2, gK, K, causal;
  float qscale2;
  int Nkv;  // rows per (batch, KV head) in k
};


// Leaf scoring grouped by parent node (g*C <= 128 keys): one workgroup per
// chunk of up to kLeafChunk (row, first-child slot) entries of one parent;
// the parent's children key blocks are staged in LDS together and each query
// row is gathered once for all of them; every 32-key MFMA tile belongs to
// one child, whose LSE is accumulated separately.
template <int D, int KIND>
__global__ __launch_bounds__(256, KIND == kScoreLse ? 5 : 1) void leaf_parent_kernel(LeafParentArgs a, const uint16_t* __restrict__ q,
                                                          const uint16_t* __restrict__ k,
                                                          const int32_t* __restrict__ a1,
                                                          const int32_t* __restrict__ a1cnt,
                                                          const int32_t* __restrict__ offs,
                                                          const int32_t* __restrict__ toffs, int64_t ncl,
                                                          const int32_t* __restrict__ pairs,
                                                          float* __restrict__ u1) {
  constexpr int LDR = D + 8;
  constexpr int KS = D / 16;
  extern __shared__ __align__(16) uint16_t klds[];
  int64_t cl;
  int beg, end;
  if (!cluster_chunk(offs, toffs, ncl, blockIdx.x, kLeafChunk, cl, beg, end)) return;
  const int bh = static_cast<int>(cl / a.M2);
  const int par = static_cast<int>(cl - static_cast<int64_t>(bh) * a.M2);
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = par * a.g * a.C;                  // first key of the parent
  const int nkeys = min(a.g * a.C, a.N - r0);      // keys of its existing children
  const int nkt = (nkeys + 31) / 32;

  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  for (int e = threadIdx.x; e < nkt * 32 * (D / 8); e += 256) {
    const int r = e / (D / 8), cidx = (e - r * (D / 8)) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < nkeys) v = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D + cidx);
    *reinterpret_cast<uint4*>(klds + r * LDR + cidx) = v;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 31;
  const int half = lane >> 5;
  const int ntile = (end - beg + 31) / 32;
  const int kt_per_child = a.C / 32;
  for (int tile = wave; tile < ntile; tile += 4) {
    const int p = beg + tile * 32 + col;
    const bool valid = p < end;
    const int pr = valid ? pairs[p] : 0;
    const int row = pr >> 8, slot0 = pr & 255;
    float uc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int hh = 0; hh < a.G; ++hh) {
      const uint16_t* qrow = q + ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + row) * D + half * 8;
      bf16x8v qb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 v = make_uint4(0, 0, 0, 0);
        if (valid) v = *reinterpret_cast<const uint4*>(qrow + ks * 16);
        qb[ks] = as_bf16x8(v);
      }
      ScoreAcc stc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) stc[j] = acc_empty(KIND);
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        if (kt >= nkt) break;
        f32x16v acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        const uint16_t* arow = klds + (kt * 32 + col) * LDR + half * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8v av = as_bf16x8(*reinterpret_cast<const uint4*>(arow + ks * 16));
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qb[ks], acc, 0, 0, 0);
        }
        float zv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) zv[r] = acc[r];
        if (kt * 32 + 32 > nkeys) {  // a partial tile: keys past the parent's end drop out
          // (for the LSE reducer the limit is re-read here so that its per-lane
          // compares are not hoisted out of the loop and held in scalar
          // registers throughout, which spilled them)
          int nk = nkeys;
          if constexpr (KIND == kScoreLse) asm volatile("" : "+s"(nk));
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
            zv[r] = key < nk ? zv[r] : -INFINITY;
          }
        }
        const ScoreAcc ts = acc_of_scaled<KIND, 16>(zv, a.qscale2);
        const int j = kt / kt_per_child;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          if (jj == j) acc_merge(KIND, stc[jj], ts);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc_merge(KIND, stc[j], acc_shfl_xor(stc[j], 32));
        uc[j] += acc_value(KIND, stc[j]);
      }
    }
    if (valid && half == 0) {
      // the row's children of this parent sit at consecutive slots from slot0
      const int64_t rgi = static_cast<int64_t>(bh) * a.Nq + row;
      const int n = a1cnt[rgi];
      const int c = (a.N - a.Nq + row) / a.C;
      for (int i = 0; i < a.g && slot0 + i < n; ++i) {
        const int node = a1[rgi * a.gK + slot0 + i];
        if (node / a.g != par) break;
        if (a.causal && (node == 0 || node == c || node == c - 1)) continue;
        const int j = node - par * a.g;
        float uj = uc[0];
#pragma unroll
        for (int jj = 1; jj < 4; ++jj)
          if (jj == j) uj = uc[jj];
        u1[rgi * a.gK + slot0 + i] = uj;
      }
    }
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
  if (ranked && n <= 128) {
    // Up to 128 candidates: the 128-entry register sort, forced candidates
    // keyed below every score, ties by candidate index (ascending nodes).
    uint32_t khi[2], klo[2];
    int nforced = 0;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int ci = lane + 64 * s2;
      const bool v = ci < n;
      const bool f = v && forced(nodes[ci]);
      khi[s2] = !v ? 0xFFFFFFFFu : (f ? 0u : desc_bits(us[ci]));
      klo[s2] = static_cast<uint32_t>(ci);
      nforced += __popcll(__ballot(f));
    }
    sort128(khi, klo, lane);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int rk = lane + 64 * s2;
      if (static_cast<int>(klo[s2]) < n) keep[klo[s2]] = (rk < nforced || rk - nforced < keepn) ? 1 : 0;
    }
  } else {
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
// Stage 1 for few rows (decode) and g*K <= 64: one workgroup per row.
//
// Latency is the cost here, so each ranked level is one memory round trip
// and no more: the row starts at its first ranked level (every coarser level
// keeps all of its eligible nodes, so that level's candidates are simply its
// eligible nodes), all 256 threads fetch every child row of the level at
// once (16 lanes per row) and leave the logits in LDS, and wavefront 0 holds
// one candidate per lane, forms the LSE scores, ranks them with a 64-lane
// bitonic sort (forced nodes keyed +inf), keeps the first K and expands them
// to their eligible children through a lane scan.
// ----------------------------------------------------------------------------
template <int K2, int J>
__device__ __forceinline__ void sort64_step(uint32_t& hi, uint32_t& lo, int lane) {
  uint32_t ohi, olo;
  if constexpr (J == 32) {
    ohi = static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), 32));
    olo = static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), 32));
  } else {
    ohi = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(hi)));
    olo = static_cast<uint32_t>(xor32_i<J>(static_cast<int>(lo)));
  }
  const uint64_t mine = (static_cast<uint64_t>(hi) << 32) | lo;
  const uint64_t other = (static_cast<uint64_t>(ohi) << 32) | olo;
  const bool want_small = ((lane & K2) == 0) == ((lane & J) == 0);
  const bool take = (other < mine) == want_small;
  hi = take ? ohi : hi;
  lo = take ? olo : lo;
}

// Bitonic sort of the 64 lanes of a wavefront into rank order (key desc,
// pack asc); packs are non-negative.
__device__ __forceinline__ void sort64(float& key, int& pack, int lane) {
  uint32_t hi = desc_bits(key), lo = static_cast<uint32_t>(pack);
  sort64_step<2, 1>(hi, lo, lane);
  sort64_step<4, 2>(hi, lo, lane);
  sort64_step<4, 1>(hi, lo, lane);
  sort64_step<8, 4>(hi, lo, lane);
  sort64_step<8, 2>(hi, lo, lane);
  sort64_step<8, 1>(hi, lo, lane);
  sort64_step<16, 8>(hi, lo, lane);
  sort64_step<16, 4>(hi, lo, lane);
  sort64_step<16, 2>(hi, lo, lane);
  sort64_step<16, 1>(hi, lo, lane);
  sort64_step<32, 16>(hi, lo, lane);
  sort64_step<32, 8>(hi, lo, lane);
  sort64_step<32, 4>(hi, lo, lane);
  sort64_step<32, 2>(hi, lo, lane);
  sort64_step<32, 1>(hi, lo, lane);
  sort64_step<64, 32>(hi, lo, lane);
  sort64_step<64, 16>(hi, lo, lane);
  sort64_step<64, 8>(hi, lo, lane);
  sort64_step<64, 4>(hi, lo, lane);
  sort64_step<64, 2>(hi, lo, lane);
  sort64_step<64, 1>(hi, lo, lane);
  key = desc_bits_inv(hi);
  pack = static_cast<int>(lo);
}

// Inclusive prefix sum over the 64 lanes of a wavefront.
__device__ __forceinline__ int scan64_incl(int v, int lane) {
  const int x = scan32_incl(v);
  return x + (lane >= 32 ? __builtin_amdgcn_readlane(x, 31) : 0);
}

template <typename T, int D, int GMAX>
__global__ __launch_bounds__(256) void stage1_row_kernel(SelArgs a) {
  constexpr int DPL = D / 16;
  constexpr int UNR = 4;  // child rows per 16-lane group in flight: 64 per round
  __shared__ int s_cand[64];
  __shared__ int s_n;
  extern __shared__ __align__(16) float s_z[];  // [candidate * g + child][head], g*K*g*G floats
  const Geo& geo = a.geo;
  const int g = geo.g, G = a.G, K = a.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = tid >> 4, sub = tid & 15;
  const int row = blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = geo.N - a.Nq + row;
  const int c = t / geo.C;

  auto n_eligible = [&](int lev) { return a.causal ? min(anc_at(geo, c, lev) + 1, geo.M[lev]) : geo.M[lev]; };
  int start = 1;
  for (int lev = geo.L; lev >= 2; --lev) {
    if (n_eligible(lev) > K) {
      start = lev;
      break;
    }
  }
  // wavefront 0 keeps the candidate of each lane in a register
  int node = -1, nA = n_eligible(start);
  if (wave == 0) {
    node = lane < nA ? lane : -1;
    if (lane < nA) s_cand[lane] = lane;
    if (lane == 0) s_n = nA;
  }
  __syncthreads();
  // q is requested with the first level's child rows (a barrier waits for
  // every outstanding load, and scaling q right after its load would too)
  float qv[GMAX][DPL];
  bool need_q = true;
  auto load_q = [&]() __attribute__((always_inline)) {
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
    need_q = false;
  };

  for (int lev = start; lev >= 2; --lev) {
    nA = s_n;
    const int Mb = geo.M[lev - 1];
    const int nch_all = nA * g;
    // 1) logits of every child row of every candidate (non-existent children
    //    past the level's end are skipped)
    const float* pbase = a.pyr + (static_cast<int64_t>(bh) * geo.R + geo.off[lev - 1]) * D + sub * DPL;
    for (int e0 = grp; e0 < nch_all; e0 += 16 * UNR) {
      float x[UNR][DPL];
      bool ok[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + 16 * u;
        const int r = e < nch_all ? s_cand[e / g] * g + (e % g) : Mb;
        ok[u] = r < Mb;
        if (ok[u]) {
          load_row_part<float, DPL>(pbase + static_cast<int64_t>(r) * D, x[u]);
        } else {
#pragma unroll
          for (int i = 0; i < DPL; ++i) x[u][i] = 0.f;
        }
      }
      if (need_q) load_q();
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = e0 + 16 * u;
#pragma unroll
        for (int hh = 0; hh < GMAX; ++hh) {
          if (hh < G) {
            float d0 = 0.f;
#pragma unroll
            for (int i = 0; i < DPL; ++i) d0 = fmaf(qv[hh][i], x[u][i], d0);
            d0 = rowsum16_to15(d0);
            if (sub == 15 && e < nch_all) s_z[e * G + hh] = ok[u] ? d0 : -INFINITY;
          }
        }
      }
    }
    __syncthreads();
    if (wave == 0) {
      // 2) scores, rank, keep
      const Forced fz = forced_at(geo, lev, c, a.causal);
      const bool valid = node >= 0;
      const bool isf = valid && fz.is(node);
      const bool ranked = nA > K;
      float key = valid ? INFINITY : -INFINITY;
      if (ranked && valid && !isf) {
        const int nch = min(g, Mb - node * g);
        float u = 0.f;
        for (int hh = 0; hh < G; ++hh) {
          u += reduce_logits(a.score_kind, s_z + lane * g * G + hh, nch, G);
        }
        key = u;
      }
      int knode = node;
      bool kept = valid;
      if (ranked) {
        int pack = valid ? node : 0x7FFFFFC0 | lane;
        // at most 32 candidates (g*K <= 32) sit in lanes 0-31: a 32-lane
        // sort (with K = 16 only the best 16 separated from the rest) ranks them
        if (a.gK <= 32)
          sort32_top16(key, pack, lane & 31, K != 16);
        else
          sort64(key, pack, lane);
        kept = lane < K && key != -INFINITY;
        knode = pack;
      }
      // 3) expand the kept nodes to their eligible children
      const int rmax = a.causal ? min(anc_at(geo, c, lev - 1), Mb - 1) : Mb - 1;
      const int c0 = knode * g;
      const int nk = kept ? max(0, min(c0 + g - 1, rmax) - c0 + 1) : 0;
      const int incl = scan64_incl(nk, lane);
      const int n2 = __builtin_amdgcn_readlane(incl, 63);
      for (int j = 0; j < nk; ++j) s_cand[incl - nk + j] = c0 + j;
      wave_sync();
      node = lane < n2 ? s_cand[lane] : -1;
      if (lane == 0) s_n = n2;
    }
    __syncthreads();
  }
  if (wave == 0) {
    if (start == 1) node = lane < nA ? lane : -1;
    nA = start == 1 ? nA : s_n;
    // leaf candidate set, ascending
    float akey = node >= 0 ? -static_cast<float>(node) : -INFINITY;
    int apack = node >= 0 ? node : 0x7FFFFFC0 | lane;
    if (a.gK <= 32)
      sort32(akey, apack, lane & 31);
    else
      sort64(akey, apack, lane);
    const int64_t orow = static_cast<int64_t>(bh) * a.Nq + row;
    if (lane < a.gK) a.a1[orow * a.gK + lane] = lane < nA ? apack : -1;
    if (lane == 0) a.a1cnt[orow] = nA;
  }
}

// ----------------------------------------------------------------------------
// Leaf scoring for few rows (decode): one workgroup per (row, candidate slot)
// computes the exact LSE over the candidate block's raw keys for the G query
// heads of the KV head (Sec. 3.3 leaf level; the same u as the clustered
// scorers, in log2 units).  Up to 64 key rows are requested at once, so a
// step costs a few memory round trips whatever the number of rows; key-block
// reuse across queries, the reason for clustering, does not arise here.
// ----------------------------------------------------------------------------
template <typename T, int D, int GMAX>
__global__ __launch_bounds__(256) void leaf_slot_kernel(SelArgs a, const int32_t* __restrict__ a1,
                                                        const int32_t* __restrict__ a1cnt, float* __restrict__ u1) {
  constexpr int DPL = D / 16;
  constexpr int UNR = 4;  // rounds of 16 key rows in flight
  __shared__ float z[kMaxLeafKeys * GMAX];
  __shared__ float lse_h[GMAX];
  const Geo& geo = a.geo;
  const int slot = blockIdx.x;
  const int64_t rg = blockIdx.y;  // bh * Nq + row
  const int bh = static_cast<int>(rg / a.Nq), row = static_cast<int>(rg - static_cast<int64_t>(bh) * a.Nq);
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int G = a.G;
  const int tid = threadIdx.x, grp = tid >> 4, sub = tid & 15;
  // the candidate count, the slot's node (in bounds: slot < g*K) and q are
  // requested together
  const int n = a1cnt[rg];
  const int node = a1[rg * a.gK + slot];
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
  if (slot >= n || n <= a.K) return;
  const int c = (geo.N - a.Nq + row) / geo.C;
  if (a.causal && (node == 0 || node == c || node == c - 1)) return;  // forced: never scored
  const int r0 = node * geo.C;
  const int nrows = min(geo.C, geo.N - r0);
  const T* kb = static_cast<const T*>(a.k) + (static_cast<int64_t>(bh) * geo.Nkv + r0) * D + sub * DPL;
  for (int base = 0; base < nrows; base += 16 * UNR) {
    float x[UNR][DPL];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int r = base + grp + 16 * u;
      if (r < nrows) {
        load_row_part<T, DPL>(kb + static_cast<int64_t>(r) * D, x[u]);
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) x[u][e] = 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int r = base + grp + 16 * u;
#pragma unroll
      for (int hh = 0; hh < GMAX; ++hh) {
        if (hh < G) {
          float d0 = 0.f;
#pragma unroll
          for (int e = 0; e < DPL; ++e) d0 = fmaf(qv[hh][e], x[u][e], d0);
          d0 = sum16(d0);
          if (sub == 0 && r < nrows) z[r * G + hh] = d0;
        }
      }
    }
  }
  __syncthreads();
  // LSE per head: wave w takes heads w, w + 4, ...
  const int wave = tid >> 6, lane = tid & 63;
  for (int hh = wave; hh < G; hh += 4) {
    ScoreAcc st = acc_empty(a.score_kind);
    for (int r = lane; r < nrows; r += 64) acc_push(a.score_kind, st, z[r * G + hh]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc_merge(a.score_kind, st, acc_shfl_xor(st, o));
    if (lane == 0) lse_h[hh] = acc_value(a.score_kind, st);
  }
  __syncthreads();
  if (tid == 0) {
    float u = 0.f;
    for (int hh = 0; hh < G; ++hh) u += lse_h[hh];
    u1[rg * a.gK + slot] = u;
  }
}

// ----------------------------------------------------------------------------
// Host launchers.
// ----------------------------------------------------------------------------

static int sel_lds_words(const Shape& s) {
  const int gK = s.gK();
  int w = 4 * gK + 8 + gK * (s.g * s.G + 1) + 2 * gK * (s.G + 1);
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
  a.score_kind = s.score;
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
  ProfScope ps("select_fused", st);
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
  size_t a1, a1cnt, u1, cl, hilo, total;
};

// Stage 1 on the matrix cores: bf16 queries, fan-out 2 or 4, up to 16 heads
// per KV head, within the 128-entry rank sort, and either candidate sets
// wider than one wavefront half (g*K > 32) or groups of 8 or more heads
// (enough columns of the 16-wide tile do work to beat the vector ALUs).
static bool stage1_mfma_ok(const Shape& s) {
  return s.bf16 && (s.g == 2 || s.g == 4) && s.G <= 16 && (s.gK() > 32 || s.G >= 8) && s.gK() <= 128 &&
         (s.D == 64 || s.D == 128);
}

static TwoStageWs two_stage_layout(const Shape& s, const Geo& geo) {
  const size_t rows = static_cast<size_t>(s.BH()) * s.Nq;
  TwoStageWs w{};
  size_t o = 0;
  w.a1 = o;     o += align256(rows * s.gK() * 4);
  w.a1cnt = o;  o += align256(rows * 4);
  w.u1 = o;     o += align256(rows * s.gK() * 4);
  w.cl = o;     o += align256(cluster_ws(s.BH(), geo.M[1], static_cast<int64_t>(rows) * s.gK(), s.Nq));
  w.hilo = o;
  if (stage1_mfma_ok(s)) o += align256(static_cast<size_t>(s.BH()) * geo.R * s.D * 4);  // bf16 hi + lo per value
  w.total = o;
  return w;
}

size_t select_two_stage_ws(const Shape& s, const Geo& geo) { return two_stage_layout(s, geo).total; }

// Final Top-K per row over the scored leaf candidates.
static hipError_t launch_final_topk(const Shape& s, const int32_t* a1, const int32_t* a1cnt, const float* u1,
                                    int32_t* idx, float* score, hipStream_t st) {
  const int64_t rows = static_cast<int64_t>(s.BH()) * s.Nq;
  ProfScope ps("final_topk", st);
  if (s.gK() <= 32) {
    TopkArgsP ta{s.Nq, s.N, s.C, s.K, s.gK(), s.causal, rows};
    if (rows >= 65536)  // two row pairs per wavefront once the grid fills the GPU several times over
      final_topk_pair_kernel<2><<<static_cast<unsigned>((rows + 15) / 16), 256, 0, st>>>(ta, a1, a1cnt, u1, idx,
                                                                                        score);
    else
      final_topk_pair_kernel<1><<<static_cast<unsigned>((rows + 7) / 8), 256, 0, st>>>(ta, a1, a1cnt, u1, idx,
                                                                                       score);
  } else {
    TopkArgs ta{s.Nq, s.N, s.C, s.K, s.gK(), s.causal, rows};
    final_topk_kernel<<<static_cast<unsigned>((rows + 3) / 4), 256, 0, st>>>(ta, a1, a1cnt, u1, idx, score);
  }
  return hipGetLastError();
}

static hipError_t launch_two_stage_heads(const Shape& s, const Geo& geo, const void* q, const void* k,
                                        const float* pyr, int32_t* idx, float* score, void* ws, hipStream_t st) {
  const TwoStageWs w = two_stage_layout(s, geo);
  char* base = static_cast<char*>(ws);
  int32_t* a1 = reinterpret_cast<int32_t*>(base + w.a1);
  int32_t* a1cnt = reinterpret_cast<int32_t*>(base + w.a1cnt);
  float* u1 = reinterpret_cast<float*>(base + w.u1);
  hipError_t e;

  // Stage 1: intermediate levels.
  SelArgs a = make_sel_args(s, geo, q, k, pyr);
  a.a1 = a1;
  a.a1cnt = a1cnt;
  const bool narrow = s.gK() <= 32 && !stage1_mfma_ok(s);
  {
    ProfScope ps("select_stage1", st);
    if (narrow) {
      const int gK = s.gK();
      const int words = gK * s.g * 2 + gK + gK * s.g * s.G + gK * s.G;
      dim3 grid((s.Nq + 7) / 8, s.BH());
      const size_t lds = static_cast<size_t>(8) * words * sizeof(int);
      auto go = [&](auto kern) { kern<<<grid, 256, lds, st>>>(a, words); };
      // One head per KV head: 16 rows per workgroup with the coarse levels
      // staged in LDS.  Several heads: 8 rows per workgroup (the query
      // registers of four heads leave no room for the staged variant).
      dim3 grid2((s.Nq + 15) / 16, s.BH());
      const size_t slds = static_cast<size_t>(kStageFloats) * 4;
      auto go2 = [&](auto kern) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(slds));
        kern<<<grid2, 512, slds, st>>>(a);
      };
      auto go4 = [&](auto kern) { kern<<<grid, 256, 0, st>>>(a); };
      auto by_kind4 = [&](auto k0, auto k1, auto k2) {
        if (s.score == kScoreLse) go4(k0);
        else if (s.score == kScoreMean) go4(k1);
        else go4(k2);
      };
      auto by_kind = [&](auto k0, auto k1, auto k2) {
        if (s.score == kScoreLse) go2(k0);
        else if (s.score == kScoreMean) go2(k1);
        else go2(k2);
      };
      if (s.g == 2 && s.G <= 4) {
        if (s.D == 128) {
          if (s.G == 1)
            by_kind(stage1_g2_kernel<128, 1, 16, kScoreLse, 8, true>, stage1_g2_kernel<128, 1, 16, kScoreMean, 8, true>,
                    stage1_g2_kernel<128, 1, 16, kScoreMeanVar, 8, true>);
          else
            by_kind4(stage1_g2_kernel<128, 4, 8, kScoreLse, 4, false>, stage1_g2_kernel<128, 4, 8, kScoreMean, 4, false>,
                     stage1_g2_kernel<128, 4, 8, kScoreMeanVar, 4, false>);
        } else {
          if (s.G == 1)
            by_kind(stage1_g2_kernel<64, 1, 16, kScoreLse, 8, true>, stage1_g2_kernel<64, 1, 16, kScoreMean, 8, true>,
                    stage1_g2_kernel<64, 1, 16, kScoreMeanVar, 8, true>);
          else
            by_kind4(stage1_g2_kernel<64, 4, 8, kScoreLse, 4, false>, stage1_g2_kernel<64, 4, 8, kScoreMean, 4, false>,
                     stage1_g2_kernel<64, 4, 8, kScoreMeanVar, 4, false>);
        }
      } else if (s.D == 128) {
        if (s.G == 1) go(stage1_pair_kernel<128, 1, 4>);
        else if (s.G <= 4) go(stage1_pair_kernel<128, 4, 16>);
        else go(stage1_pair_kernel<128, 16, 16>);
      } else {
        if (s.G == 1) go(stage1_pair_kernel<64, 1, 4>);
        else if (s.G <= 4) go(stage1_pair_kernel<64, 4, 16>);
        else go(stage1_pair_kernel<64, 16, 16>);
      }
    } else if (stage1_mfma_ok(s)) {
      uint16_t* hilo = reinterpret_cast<uint16_t*>(base + w.hilo);
      const int64_t ngroups = static_cast<int64_t>(s.BH()) * geo.R * s.D / 8;
      pyr_hilo_kernel<<<static_cast<unsigned>((ngroups + 255) / 256), 256, 0, st>>>(pyr, hilo, ngroups);
      dim3 grid((s.Nq + kMfmaSelRows - 1) / kMfmaSelRows, s.BH());
      auto go = [&](auto k0, auto k1, auto k2) {
        if (s.score == kScoreLse) k0<<<grid, kMfmaSelRows * 64, 0, st>>>(a, hilo);
        else if (s.score == kScoreMean) k1<<<grid, kMfmaSelRows * 64, 0, st>>>(a, hilo);
        else k2<<<grid, kMfmaSelRows * 64, 0, st>>>(a, hilo);
      };
      // 1, 2 or 4 heads per KV head: kUnionRows rows per wavefront share the
      // union of their candidates (their heads fill at most 16 columns)
      const int bm_words = (geo.L >= 2 ? (geo.M[2] + 31) / 32 : 1);
      dim3 ugrid((s.Nq + kUnionRows * kUnionWaves - 1) / (kUnionRows * kUnionWaves), s.BH());
      const size_t ulds = static_cast<size_t>(kUnionWaves) * union_wave_words(bm_words) * 4;
      auto gu = [&](auto k0, auto k1, auto k2) {
        auto run = [&](auto kern) {
          if (ulds > 65536)
            (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(ulds));
          kern<<<ugrid, kUnionWaves * 64, ulds, st>>>(a, hilo, bm_words);
        };
        if (s.score == kScoreLse) run(k0);
        else if (s.score == kScoreMean) run(k1);
        else run(k2);
      };
      const bool union_rows = s.G == 1 || s.G == 2 || s.G == 4;
      if (union_rows && s.D == 128) {
        if (s.g == 4)
          gu(stage1_union_kernel<128, 4, kScoreLse>, stage1_union_kernel<128, 4, kScoreMean>,
             stage1_union_kernel<128, 4, kScoreMeanVar>);
        else
          gu(stage1_union_kernel<128, 2, kScoreLse>, stage1_union_kernel<128, 2, kScoreMean>,
             stage1_union_kernel<128, 2, kScoreMeanVar>);
      } else if (union_rows) {
        if (s.g == 4)
          gu(stage1_union_kernel<64, 4, kScoreLse>, stage1_union_kernel<64, 4, kScoreMean>,
             stage1_union_kernel<64, 4, kScoreMeanVar>);
        else
          gu(stage1_union_kernel<64, 2, kScoreLse>, stage1_union_kernel<64, 2, kScoreMean>,
             stage1_union_kernel<64, 2, kScoreMeanVar>);
      } else if (s.D == 128) {
        if (s.g == 4)
          go(stage1_mfma_kernel<128, 4, kScoreLse>, stage1_mfma_kernel<128, 4, kScoreMean>,
             stage1_mfma_kernel<128, 4, kScoreMeanVar>);
        else
          go(stage1_mfma_kernel<128, 2, kScoreLse>, stage1_mfma_kernel<128, 2, kScoreMean>,
             stage1_mfma_kernel<128, 2, kScoreMeanVar>);
      } else {
        if (s.g == 4)
          go(stage1_mfma_kernel<64, 4, kScoreLse>, stage1_mfma_kernel<64, 4, kScoreMean>,
             stage1_mfma_kernel<64, 4, kScoreMeanVar>);
        else
          go(stage1_mfma_kernel<64, 2, kScoreLse>, stage1_mfma_kernel<64, 2, kScoreMean>,
             stage1_mfma_kernel<64, 2, kScoreMeanVar>);
      }
    } else {
      launch_sel_d<uint16_t, 64, false>(s, a, st);
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // Cluster the (row, slot) pairs by leaf block, or by parent node when a
  // parent's children fit one tile (each query row is then gathered once per
  // parent instead of once per child).
  const int64_t rows = static_cast<int64_t>(s.BH()) * s.Nq;
  const bool by_parent = geo.L >= 2 && s.g * s.C <= 128;
  const int M2 = geo.L >= 2 ? geo.M[2] : 1;
  ClusterArgs ca{a1, a1cnt, s.gK(), s.Nq, s.N, s.C, s.K, s.causal, by_parent ? M2 : geo.M[1],
                 by_parent ? kClusterLeafParent : kClusterLeaf, 0, s.Nq, s.g};
  ClusterOut co{};
  if ((e = launch_cluster(ca, s.BH(), base + w.cl, &co, st, kLeafChunk)) != hipSuccess) return e;
  if (by_parent) {
    LeafParentArgs lp{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.g, geo.M[1], M2, s.gK(), s.K, s.causal,
                      kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv};
    dim3 pgrid(static_cast<unsigned>(cluster_max_chunks(s.BH(), M2, rows * s.gK(), kLeafChunk)));
    const size_t plds = static_cast<size_t>(128) * (s.D + 8) * 2;
    {
      ProfScope ps("leaf_score", st);
      auto go = [&](auto kern) {
        kern<<<pgrid, 256, plds, st>>>(lp, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), a1,
                                       a1cnt, co.offs, co.toffs, co.ncl, co.pairs, u1);
      };
      if (s.D == 128) {
        if (s.score == kScoreLse) go(leaf_parent_kernel<128, kScoreLse>);
        else if (s.score == kScoreMean) go(leaf_parent_kernel<128, kScoreMean>);
        else go(leaf_parent_kernel<128, kScoreMeanVar>);
      } else {
        if (s.score == kScoreLse) go(leaf_parent_kernel<64, kScoreLse>);
        else if (s.score == kScoreMean) go(leaf_parent_kernel<64, kScoreMean>);
        else go(leaf_parent_kernel<64, kScoreMeanVar>);
      }
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else {
    // Stage 2: leaf scoring against each key block once per cluster.
    LeafArgs la{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, geo.M[1], s.gK(), kLog2e / sqrtf(static_cast<float>(s.D)), s.Nkv};
    dim3 lgrid(static_cast<unsigned>(cluster_max_chunks(s.BH(), geo.M[1], rows * s.gK(), kLeafChunk)));
    const size_t llds = static_cast<size_t>(s.C) * (s.D + 8) * 2;
    {
      ProfScope ps("leaf_score", st);
      auto go = [&](auto kern) {
        if (llds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                    hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(llds));
        kern<<<lgrid, 256, llds, st>>>(la, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                       co.offs, co.toffs, co.ncl, co.pairs, u1);
      };
      if (s.D == 128) {
        if (s.score == kScoreLse) go(leaf_score_kernel<128, kScoreLse>);
        else if (s.score == kScoreMean) go(leaf_score_kernel<128, kScoreMean>);
        else go(leaf_score_kernel<128, kScoreMeanVar>);
      } else {
        if (s.score == kScoreLse) go(leaf_score_kernel<64, kScoreLse>);
        else if (s.score == kScoreMean) go(leaf_score_kernel<64, kScoreMean>);
        else go(leaf_score_kernel<64, kScoreMeanVar>);
      }
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }

  return launch_final_topk(s, a1, a1cnt, u1, idx, score, st);
}

// The cluster builder counts and places (row, slot) pairs with 32-bit
// offsets, so one pass may hold at most kMaxPairsPerPass pairs: larger
// problems run as passes over consecutive (batch, KV head) slices, each a
// problem of its own (B = 1, the slice's heads) with the same workspace
// layout, shrunk.  One slice holds Nq * g * K < 2^23 * 2^8 pairs, so every
// problem the ABI accepts splits.
constexpr int64_t kMaxPairsPerPass = (int64_t(1) << 31) - 1;

static int two_stage_heads_per_pass(const Shape& s) {
  const int64_t per_bh = static_cast<int64_t>(s.Nq) * s.gK();
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(s.BH(), kMaxPairsPerPass / per_bh)));
}

hipError_t launch_select_two_stage(const Shape& s, const Geo& geo, const void* q, const void* k,
                                   const float* pyr, int32_t* idx, float* score, void* ws, hipStream_t st) {
  const int per = two_stage_heads_per_pass(s);
  if (per >= s.BH()) return launch_two_stage_heads(s, geo, q, k, pyr, idx, score, ws, st);
  for (int bh0 = 0; bh0 < s.BH(); bh0 += per) {
    Shape sub = s;
    sub.B = 1;
    sub.Hkv = std::min(per, s.BH() - bh0);
    sub.H = sub.Hkv * s.G;
    const int64_t qoff = static_cast<int64_t>(bh0) * s.G * s.Nq * s.D;  // bf16 elements
    const int64_t koff = static_cast<int64_t>(bh0) * s.Nkv * s.D;
    const int64_t poff = static_cast<int64_t>(bh0) * geo.R * s.D;
    const int64_t ioff = static_cast<int64_t>(bh0) * s.Nq * s.K;
    const hipError_t e = launch_two_stage_heads(
        sub, geo, static_cast<const uint16_t*>(q) + qoff, static_cast<const uint16_t*>(k) + koff, pyr + poff,
        idx + ioff, score ? score + ioff : nullptr, ws, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Split schedule: stage 1 with a workgroup per row, every scored leaf
// candidate on a workgroup of its own, then the final Top-K.
struct SplitWs {
  size_t a1, a1cnt, u1, total;
};

static SplitWs split_layout(const Shape& s) {
  const size_t rows = static_cast<size_t>(s.BH()) * s.Nq;
  SplitWs w{};
  size_t o = 0;
  w.a1 = o;     o += align256(rows * s.gK() * 4);
  w.a1cnt = o;  o += align256(rows * 4);
  w.u1 = o;     o += align256(rows * s.gK() * 4);
  w.total = o;
  return w;
}

size_t select_split_ws(const Shape& s) { return split_layout(s).total; }

template <typename T, int D>
static void launch_leaf_slot(const Shape& s, const SelArgs& a, const int32_t* a1, const int32_t* a1cnt, float* u1,
                             hipStream_t st) {
  dim3 grid(s.gK(), static_cast<unsigned>(static_cast<int64_t>(s.BH()) * s.Nq));
  if (s.G == 1)
    leaf_slot_kernel<T, D, 1><<<grid, 256, 0, st>>>(a, a1, a1cnt, u1);
  else if (s.G <= 4)
    leaf_slot_kernel<T, D, 4><<<grid, 256, 0, st>>>(a, a1, a1cnt, u1);
  else
    leaf_slot_kernel<T, D, 16><<<grid, 256, 0, st>>>(a, a1, a1cnt, u1);
}

hipError_t launch_select_split(const Shape& s, const Geo& geo, const void* q, const void* k, const float* pyr,
                               int32_t* idx, float* score, void* ws, hipStream_t st) {
  const SplitWs w = split_layout(s);
  char* base = static_cast<char*>(ws);
  int32_t* a1 = reinterpret_cast<int32_t*>(base + w.a1);
  int32_t* a1cnt = reinterpret_cast<int32_t*>(base + w.a1cnt);
  float* u1 = reinterpret_cast<float*>(base + w.u1);
  hipError_t e;
  SelArgs a = make_sel_args(s, geo, q, k, pyr);
  a.a1 = a1;
  a.a1cnt = a1cnt;
  {
    ProfScope ps("select_stage1", st);
    if (s.gK() <= 64) {
      dim3 grid(s.Nq, s.BH());
      const size_t lds = static_cast<size_t>(s.gK()) * s.g * s.G * sizeof(float);
      auto go = [&](auto tag) {
        using T = decltype(tag);
        auto run = [&](auto kern) {
          if (lds > 60000)  // beyond the default dynamic limit once the static arrays are added
            (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
          kern<<<grid, 256, lds, st>>>(a);
        };
        if (s.D == 128) {
          if (s.G == 1) run(stage1_row_kernel<T, 128, 1>);
          else if (s.G <= 4) run(stage1_row_kernel<T, 128, 4>);
          else run(stage1_row_kernel<T, 128, 16>);
        } else {
          if (s.G == 1) run(stage1_row_kernel<T, 64, 1>);
          else if (s.G <= 4) run(stage1_row_kernel<T, 64, 4>);
          else run(stage1_row_kernel<T, 64, 16>);
        }
      };
      if (s.bf16)
        go(uint16_t{});
      else
        go(float{});
    } else if (s.bf16) {
      launch_sel_d<uint16_t, 256, false>(s, a, st);
    } else {
      launch_sel_d<float, 256, false>(s, a, st);
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  {
    ProfScope ps("leaf_score", st);
    if (s.bf16) {
      if (s.D == 128)
        launch_leaf_slot<uint16_t, 128>(s, a, a1, a1cnt, u1, st);
      else
        launch_leaf_slot<uint16_t, 64>(s, a, a1, a1cnt, u1, st);
    } else {
      if (s.D == 128)
        launch_leaf_slot<float, 128>(s, a, a1, a1cnt, u1, st);
      else
        launch_leaf_slot<float, 64>(s, a, a1, a1cnt, u1, st);
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_final_topk(s, a1, a1cnt, u1, idx, score, st);
}

}  // namespace pisa
