// Flat block selection baseline (Sec. 3.1 eqs. bsa_block_scores, bsa_topk;
// per-head normalisation before the head sum, App. C.1; forced blocks App. B).
//
// bsa_rows_kernel: one wavefront per (query row, KV head).  Its 16-lane groups
// stride over the eligible leaf summaries (16-byte loads of fp32 pyramid
// level-1 rows), computing the scaled logit of every head of the group.  With
// G > 1 a first pass collects each head's softmax normaliser over the
// eligible non-forced blocks and a second pass sums the heads' probabilities;
// with G = 1 the logit itself ranks.  Scores go to LDS and the best K - |F|
// are extracted by repeated wavefront arg-max (score desc, index asc).
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pisa {

struct BsaArgs {
  const void* q;
  const float* pyr;
  int32_t* idx;
  int H, Hkv, G, Nq, N, C, K, causal, M1;
  int64_t R;
  float qscale2;
};

template <typename T, int D, int GMAX>
__global__ __launch_bounds__(64) void bsa_rows_kernel(BsaArgs a) {
  constexpr int DPL = D / 16;
  extern __shared__ __align__(16) float sc[];  // [M1] scores, then [K] output scratch (as int)
  int* outl = reinterpret_cast<int*>(sc + a.M1);
  const int lane = threadIdx.x;
  const int grp = lane >> 4, sub = lane & 15;
  const int row = blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int t = a.N - a.Nq + row;
  const int c = t / a.C;
  const int E = a.causal ? min(c + 1, a.M1) : a.M1;
  int32_t* out = a.idx + (static_cast<int64_t>(bh) * a.Nq + row) * a.K;
  if (E <= a.K) {
    for (int j = lane; j < a.K; j += 64) out[j] = j < E ? j : -1;
    return;
  }
  auto forced = [&](int i) { return a.causal && (i == 0 || i == c || i == c - 1); };
  const int nF = a.causal ? 1 + (c != 0) + (c - 1 > 0) : 0;

  float qv[GMAX][DPL];
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) {
    if (hh < a.G) {
      const T* qp = static_cast<const T*>(a.q) +
                    ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + row) * D + sub * DPL;
      load_row_part<T, DPL>(qp, qv[hh]);
#pragma unroll
      for (int e = 0; e < DPL; ++e) qv[hh][e] *= a.qscale2;
    }
  }
  const float* pbase = a.pyr + static_cast<int64_t>(bh) * a.R * D + sub * DPL;

  // Pass 1 (G > 1): per-head normaliser (log2 units) over eligible non-forced blocks.
  float hm[GMAX], hs[GMAX];
#pragma unroll
  for (int hh = 0; hh < GMAX; ++hh) {
    hm[hh] = -INFINITY;
    hs[hh] = 0.f;
  }
  if (a.G > 1) {
    for (int i = grp; i < E; i += 4) {
      if (forced(i)) continue;
      float x[DPL];
      load_row_part<float, DPL>(pbase + static_cast<int64_t>(i) * D, x);
#pragma unroll
      for (int hh = 0; hh < GMAX; ++hh) {
        if (hh < a.G) {
          float z = 0.f;
#pragma unroll
          for (int e = 0; e < DPL; ++e) z = fmaf(qv[hh][e], x[e], z);
          z = sum16(z);
          const float mn = fmaxf(hm[hh], z);
          hs[hh] = hs[hh] * fast_exp2(hm[hh] - mn) + fast_exp2(z - mn);
          hm[hh] = mn;
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < a.G) {
#pragma unroll
        for (int msk = 16; msk <= 32; msk <<= 1) {
          const float m2 = __shfl_xor(hm[hh], msk), s2 = __shfl_xor(hs[hh], msk);
          const float mn = fmaxf(hm[hh], m2);
          hs[hh] = (mn == -INFINITY) ? 0.f : hs[hh] * fast_exp2(hm[hh] - mn) + s2 * fast_exp2(m2 - mn);
          hm[hh] = mn;
        }
        hm[hh] += fast_log2(hs[hh]);  // log2 of the normaliser
      }
    }
  }
  // Pass 2: the ranking score of every eligible block.
  for (int i = grp; i < E; i += 4) {
    float x[DPL];
    load_row_part<float, DPL>(pbase + static_cast<int64_t>(i) * D, x);
    float u = 0.f;
#pragma unroll
    for (int hh = 0; hh < GMAX; ++hh) {
      if (hh < a.G) {
        float z = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) z = fmaf(qv[hh][e], x[e], z);
        z = sum16(z);
        u += (a.G > 1) ? fast_exp2(z - hm[hh]) : z;
      }
    }
    if (sub == 0) sc[i] = forced(i) ? -INFINITY : u;
  }
  wave_sync();
  // Extract the best K - |F| by repeated arg-max.
  const int keepn = a.K - nF;
  for (int r = 0; r < keepn; ++r) {
    float best = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = lane; i < E; i += 64) {
      const float v = sc[i];
      if (!forced(i) && v != -INFINITY && ranks_before(v, i, best, bi)) {
        best = v;
        bi = i;
      }
    }
#pragma unroll
    for (int msk = 1; msk < 64; msk <<= 1) {
      const float b2 = __shfl_xor(best, msk);
      const int i2 = __shfl_xor(bi, msk);
      if (ranks_before(b2, i2, best, bi)) {
        best = b2;
        bi = i2;
      }
    }
    if (lane == 0) {
      outl[r] = bi;
      sc[bi] = -INFINITY;
    }
    wave_sync();
  }
  // Forced blocks join, then sort ascending.
  if (lane == 0) {
    int n = keepn;
    if (a.causal) {
      outl[n++] = 0;
      if (c >= 1 && c - 1 != 0) outl[n++] = c - 1;
      if (c != 0) outl[n++] = c;
    }
  }
  wave_sync();
  for (int j = lane; j < a.K; j += 64) {
    const int v = outl[j];
    int rank = 0;
    for (int i = 0; i < a.K; ++i) rank += outl[i] < v ? 1 : 0;
    out[rank] = v;
  }
}

// ----------------------------------------------------------------------------
// MFMA flat selection (bf16 q).  One workgroup of four wavefronts per tile of
// 64 consecutive query rows of one (batch, KV head).  The leaf means are
// split once per call into bf16 hi + lo planes (bsa_hilo_kernel; hi + lo
// reproduces the fp32 mean to ~2^-17 relative) and streamed through LDS in
// chunks of 64 blocks, scored on v_mfma_f32_32x32x16_bf16 (wave w: queries
// (w&1)*32.., blocks (w>>1)*32.. of the chunk).  The chunk's scores go to an
// LDS tile [64 queries][64 blocks]; then each wavefront takes 16 queries in
// turn, one block per lane, and keeps every query's running top list (KP
// entries, best first, ties to the smaller block) in LDS: a chunk's blocks
// that beat the list's last entry are found with one ballot; a few are
// inserted one by one (position = popcount of the entries ranking before it,
// the tail shifted down one lane), many are merged by a 64-lane bitonic sort
// and a bitonic merge with the list.  With G > 1 a first pass over the chunks
// gathers each head's normaliser (online max / sum of 2^z over eligible
// non-forced blocks) and the second pass ranks by the sum of the heads'
// probabilities.
// ----------------------------------------------------------------------------

typedef __bf16 bf16x8b __attribute__((ext_vector_type(8)));
typedef float f32x16b __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8b u4_bf16x8(uint4 r) { return __builtin_bit_cast(bf16x8b, r); }

// The leaf level of the pyramid as bf16 hi and lo planes, [BH][M1][D] each.
__global__ __launch_bounds__(256) void bsa_hilo_kernel(const float* __restrict__ pyr, int64_t R, int M1, int D,
                                                       int64_t n4, uint16_t* __restrict__ hi,
                                                       uint16_t* __restrict__ lo) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;  // group of 4 values
  if (e >= n4) return;
  const int64_t per_bh = static_cast<int64_t>(M1) * D / 4;
  const int64_t bh = e / per_bh, rem = e - bh * per_bh;
  const float4 x = *reinterpret_cast<const float4*>(pyr + bh * R * D + rem * 4);
  const uint32_t h01 = pack2_bf16(x.x, x.y), h23 = pack2_bf16(x.z, x.w);
  const float hx = __uint_as_float(h01 << 16), hy = __uint_as_float(h01 & 0xFFFF0000u);
  const float hz = __uint_as_float(h23 << 16), hw = __uint_as_float(h23 & 0xFFFF0000u);
  *reinterpret_cast<uint2*>(hi + e * 4) = make_uint2(h01, h23);
  *reinterpret_cast<uint2*>(lo + e * 4) =
      make_uint2(pack2_bf16(x.x - hx, x.y - hy), pack2_bf16(x.z - hz, x.w - hw));
}

// Sorted best-first list of KP (score, block) entries; blocks arrive in
// ascending order, so a new entry goes after equal scores, and an entry
// pushed down keeps its place before equal scores of larger blocks.
template <int KP>
struct TopList {
  float s[KP];
  int i[KP];
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      s[j] = -INFINITY;
      i[j] = 0x7fffffff;
    }
  }
  __device__ __forceinline__ void insert(float v, int idx) {
    if (!(v > s[KP - 1])) return;
    float cur = v;
    int ci = idx;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const bool sw = cur > s[j] || (cur == s[j] && ci < i[j]);
      const float ts = s[j];
      const int ti = i[j];
      s[j] = sw ? cur : ts;
      i[j] = sw ? ci : ti;
      cur = sw ? ts : cur;
      ci = sw ? ti : ci;
    }
  }
};

// (score desc, block asc): does (sa, ia) rank before (sb, ib)?
__device__ __forceinline__ bool bsa_better(float sa, int ia, float sb, int ib) {
  return (sa > sb) | ((sa == sb) & (ia < ib));  // bitwise: no branches
}

// One compare-exchange of a bitonic network over the wavefront: lanes with
// bit j clear keep the better entry of the pair when `asc` holds, the worse
// otherwise (equal sentinel entries may go either way).
__device__ __forceinline__ void bsa_cx(float& s, int& i, int lane, int j, bool asc) {
  const float ps = __shfl_xor(s, j);
  const int pi = __shfl_xor(i, j);
  const bool lower = (lane & j) == 0;
  const bool pbetter = bsa_better(ps, pi, s, i);
  const bool take = (lower == asc) ? pbetter : (!pbetter & !((ps == s) & (pi == i)));
  s = take ? ps : s;
  i = take ? pi : i;
}

template <int D, int KP, int GM>
__global__ __launch_bounds__(256, 2) void bsa_mfma_kernel(BsaArgs a, const uint16_t* __restrict__ phi,
                                                          const uint16_t* __restrict__ plo) {
  constexpr int KS = D / 16;
  constexpr int LDS_ROW = D + 8;
  constexpr int CAP = 32;                      // blocks collected per query in the second scan
  constexpr int PRE = 2 * 64 * (D / 8) / 256;  // 16-byte staging loads per thread per chunk
  extern __shared__ __align__(16) uint16_t lds[];
  uint16_t* shi = lds;                   // [64][LDS_ROW]
  uint16_t* slo = lds + 64 * LDS_ROW;    // [64][LDS_ROW]
  float* hred = reinterpret_cast<float*>(lds);  // pass-1 merge (over the chunk area and beyond)
  // After the chunk area, reused phase by phase: the 64 class bests of every
  // query (threshold search), then the collected blocks, or the exact
  // method's holder lists and merged lists; after those, T, the counts and
  // the output scratch.
  float* work = reinterpret_cast<float*>(lds + 2 * 64 * LDS_ROW);
  constexpr int kSmall = (8 * KP * 64 + 64 * KP) > 8192 ? (8 * KP * 64 + 64 * KP) : 8192;
  float* tsc = work + kSmall;                              // [64] T score
  int* tix = reinterpret_cast<int*>(tsc + 64);             // [64] T block
  int* cntq = tix + 64;                                    // [64] blocks collected per query
  int* sel = cntq + 64;                                    // [64][32] output scratch
  __shared__ int any_over;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 31, half = lane >> 5;
  const int qh = wave & 1, bhalf = wave >> 1;
  const int q64 = qh * 32 + col, holder = bhalf * 2 + half;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int row0 = blockIdx.x * 64;
  const int rowc = min(row0 + q64, a.Nq - 1);
  const int c = (a.N - a.Nq + rowc) / a.C;
  const int elig = a.causal ? min(c + 1, a.M1) : a.M1;  // blocks [0, elig) are eligible
  const int t_last = a.N - a.Nq + min(row0 + 63, a.Nq - 1);
  const int nblk = a.causal ? min(t_last / a.C + 1, a.M1) : a.M1;
  const int nchunk = (nblk + 63) / 64;
  // a block counts for the ranking: eligible and not forced (bitwise, no branches)
  const bool cz = a.causal != 0;
  auto rankable = [&](int i) __attribute__((always_inline)) {
    return (i < elig) & !(cz & ((i == 0) | (i == c) | (i == c - 1)));
  };
  const uint16_t* hbase = phi + static_cast<int64_t>(bh) * a.M1 * D;
  const uint16_t* lbase = plo + static_cast<int64_t>(bh) * a.M1 * D;
  auto block_off = [&](int r) __attribute__((always_inline)) { return bhalf * 32 + 8 * (r >> 2) + 4 * half + (r & 3); };
  // queries with at most K eligible blocks keep them all (no ranking); the
  // others keep K minus the forced ones
  auto keep_of = [&](int rowm) __attribute__((always_inline)) {
    const int cm = (a.N - a.Nq + rowm) / a.C;
    const int E = a.causal ? min(cm + 1, a.M1) : a.M1;
    return E <= a.K ? 0 : a.K - (a.causal ? 1 + (cm != 0) + (cm - 1 > 0) : 0);
  };

  // Staging with the next chunk's rows prefetched into registers while the
  // current one is scored: a chunk costs two barriers and no exposed load.
  uint4 pre[PRE];
  auto prefetch = [&](int ch) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
      const int e = threadIdx.x + k * 256;
      const int pl = e / (64 * (D / 8)), rem = e - pl * 64 * (D / 8);
      const int r = rem / (D / 8), c8 = (rem - r * (D / 8)) * 8;
      const int blk = ch * 64 + r;
      pre[k] = blk < nblk ? *reinterpret_cast<const uint4*>((pl ? lbase : hbase) + static_cast<int64_t>(blk) * D + c8)
                          : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_pre = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
      const int e = threadIdx.x + k * 256;
      const int pl = e / (64 * (D / 8)), rem = e - pl * 64 * (D / 8);
      const int r = rem / (D / 8), c8 = (rem - r * (D / 8)) * 8;
      *reinterpret_cast<uint4*>((pl ? slo : shi) + r * LDS_ROW + c8) = pre[k];
    }
  };
  // logits (log2 units) of this lane's 16 blocks of the staged chunk for head hh
  auto logits = [&](int hh, f32x16b& acc) __attribute__((always_inline)) {
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) +
                           ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + rowc) * D + half * 8;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const int arow = (bhalf * 32 + col) * LDS_ROW + half * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8b qb = u4_bf16x8(*reinterpret_cast<const uint4*>(qrow + ks * 16));
      const bf16x8b ah = u4_bf16x8(*reinterpret_cast<const uint4*>(shi + arow + ks * 16));
      const bf16x8b al = u4_bf16x8(*reinterpret_cast<const uint4*>(slo + arow + ks * 16));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, qb, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, qb, acc, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] *= a.qscale2;
  };
  // every chunk: stage it, then per_lane(ch, acc-derived values)
  auto scan = [&](auto&& per_lane) __attribute__((always_inline)) {
    __syncthreads();
    prefetch(0);
    store_pre();
    if (nchunk > 1) prefetch(1);
    __syncthreads();
    for (int ch = 0; ch < nchunk; ++ch) {
      per_lane(ch, true);   // the MFMA part, reading the staged chunk
      __syncthreads();      // every wavefront has read the staged chunk
      if (ch + 1 < nchunk) {
        store_pre();
        if (ch + 2 < nchunk) prefetch(ch + 2);
      }
      per_lane(ch, false);  // the per-lane part
      __syncthreads();      // the next chunk is staged
    }
  };

  // Pass 1 (G > 1): each head's log2 normaliser over eligible non-forced blocks.
  float lnorm[GM];
#pragma unroll
  for (int hh = 0; hh < GM; ++hh) lnorm[hh] = 0.f;
  if constexpr (GM > 1) {
    float hm[GM], hs[GM];
#pragma unroll
    for (int hh = 0; hh < GM; ++hh) {
      hm[hh] = -INFINITY;
      hs[hh] = 0.f;
    }
    scan([&](int ch, bool mfma) __attribute__((always_inline)) {
      if (!mfma) return;
#pragma unroll
      for (int hh = 0; hh < GM; ++hh) {
        if (hh < a.G) {
          f32x16b acc;
          logits(hh, acc);
          float m = hm[hh];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int blk = ch * 64 + block_off(r);
            if (rankable(blk)) m = fmaxf(m, acc[r]);
          }
          float sacc = (m == -INFINITY) ? 0.f : hs[hh] * fast_exp2(hm[hh] - m);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int blk = ch * 64 + block_off(r);
            if (rankable(blk)) sacc += fast_exp2(acc[r] - m);
          }
          hm[hh] = m;
          hs[hh] = sacc;
        }
      }
    });
    // merge the four holders of each query through LDS
#pragma unroll
    for (int hh = 0; hh < GM; ++hh) {
      if (hh < a.G) {
        hred[((q64 * GM + hh) * 4 + holder) * 2 + 0] = hm[hh];
        hred[((q64 * GM + hh) * 4 + holder) * 2 + 1] = hs[hh];
      }
    }
    __syncthreads();
#pragma unroll
    for (int hh = 0; hh < GM; ++hh) {
      if (hh >= a.G) continue;
      float m = -INFINITY, sacc = 0.f;
      for (int k2 = 0; k2 < 4; ++k2) {
        const float m2 = hred[((q64 * GM + hh) * 4 + k2) * 2 + 0];
        const float s2 = hred[((q64 * GM + hh) * 4 + k2) * 2 + 1];
        const float mn = fmaxf(m, m2);
        sacc = (mn == -INFINITY) ? 0.f : sacc * fast_exp2(m - mn) + s2 * fast_exp2(m2 - mn);
        m = mn;
      }
      lnorm[hh] = m + fast_log2(sacc);
    }
  }
  // the ranking score of this lane's 16 blocks of the staged chunk
  auto scores = [&](float (&u)[16]) {
    if constexpr (GM == 1) {
      f32x16b acc;
      logits(0, acc);
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = acc[r];
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = 0.f;
#pragma unroll
      for (int hh = 0; hh < GM; ++hh) {
        if (hh < a.G) {
          f32x16b acc;
          logits(hh, acc);
#pragma unroll
          for (int r = 0; r < 16; ++r) u[r] += fast_exp2(acc[r] - lnorm[hh]);
        }
      }
    }
  };

  // With several heads per KV head every scan costs G products per chunk,
  // and with few chunks the threshold search does not pay: the two-scan
  // threshold method below then gives way to the one-scan exact list method
  // (single head, MI355X: 1.09 vs 0.84 ms at 32K tokens, 8.6 vs 9.1 ms at 128K).
  const bool kThreshold = GM == 1 && nchunk >= 8;
  // Pass 2a: the blocks of a query fall into 64 classes (the 16 output
  // positions of each of its 4 holder lanes); every class's best block.  The
  // keepn-th best of those 64 class bests (T) has at least keepn blocks
  // ranking at or before it, so the keepn best blocks all rank at or before T.
  float bs[16];
  int bi[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    bs[r] = -INFINITY;
    bi[r] = 0x7fffffff;
  }
  if (kThreshold) {
    float u[16];
    scan([&](int ch, bool mfma) __attribute__((always_inline)) {
      if (mfma) {
        scores(u);
        return;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int blk = ch * 64 + block_off(r);
        const bool take = rankable(blk) & bsa_better(u[r], blk, bs[r], bi[r]);
        bs[r] = take ? u[r] : bs[r];
        bi[r] = take ? blk : bi[r];
      }
    });
  }
  bool fallback = !kThreshold;
  float* bq = work;                                       // [64 queries][CAP] scores
  int* bqi = reinterpret_cast<int*>(work + 64 * CAP);     // [64 queries][CAP] blocks
  if (kThreshold) {
  float* part = work;                                    // [64 queries][64 classes] scores, then blocks
  int* parti = reinterpret_cast<int*>(part + 64 * 64);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    part[q64 * 64 + holder * 16 + r] = bs[r];
    parti[q64 * 64 + holder * 16 + r] = bi[r];
  }
  __syncthreads();
  for (int qq = 0; qq < 16; ++qq) {
    const int qw = wave * 16 + qq;
    float v = part[qw * 64 + lane];
    int vb = parti[qw * 64 + lane];
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
      for (int j = k >> 1; j > 0; j >>= 1) bsa_cx(v, vb, lane, j, (lane & k) == 0);
    }
    const int kq = max(keep_of(min(row0 + qw, a.Nq - 1)), 1);
    const float tv = __shfl(v, kq - 1);
    const int tb = __shfl(vb, kq - 1);
    if (lane == 0) {
      tsc[qw] = tv;
      tix[qw] = tb;
      cntq[qw] = 0;
    }
  }
  __syncthreads();
  const float my_ts = tsc[q64];
  const int my_ti = tix[q64];
  // Pass 2b: collect every block ranking at or before T (at most CAP per query).
  {
    float u[16];
    scan([&](int ch, bool mfma) __attribute__((always_inline)) {
      if (mfma) {
        scores(u);
        return;
      }
      uint32_t msk = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int blk = ch * 64 + block_off(r);
        const bool in = rankable(blk) & !bsa_better(my_ts, my_ti, u[r], blk);
        msk |= in ? (1u << r) : 0u;
      }
      if (msk) {
        int off = atomicAdd(&cntq[q64], __builtin_popcount(msk));
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (msk & (1u << r)) {
            if (off < CAP) {
              bq[q64 * CAP + off] = u[r];
              bqi[q64 * CAP + off] = ch * 64 + block_off(r);
            }
            ++off;
          }
        }
      }
    });
  }
  // a query with more than CAP such blocks (many equal or clustered scores)
  // is ranked again by the exact list method
  if (threadIdx.x == 0) any_over = 0;
  __syncthreads();
  if (threadIdx.x < 64 && keep_of(min(row0 + threadIdx.x, a.Nq - 1)) > 0 && cntq[threadIdx.x] > CAP) any_over = 1;
  __syncthreads();
  fallback = any_over != 0;
  }
  int* ml = reinterpret_cast<int*>(work) + 8 * KP * 64;   // [64 queries][KP] merged lists (exact method)
  if (fallback) {
    // every lane keeps the best KP blocks of its 16 classes (sorted, ties to
    // the smaller block); the four holders' lists of a query are merged by
    // one thread
    TopList<KP> top;
    top.init();
    {
      float u[16];
      scan([&](int ch, bool mfma) __attribute__((always_inline)) {
        if (mfma) {
          scores(u);
          return;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int blk = ch * 64 + block_off(r);
          if (rankable(blk)) top.insert(u[r], blk);
        }
      });
    }
    float* ms = work;                                   // [holder][KP][64 queries]
    int* mi = reinterpret_cast<int*>(ms + 4 * KP * 64);
#pragma unroll
    for (int jj = 0; jj < KP; ++jj) {
      ms[(holder * KP + jj) * 64 + q64] = top.s[jj];
      mi[(holder * KP + jj) * 64 + q64] = top.i[jj];
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int qm = threadIdx.x;
      const int kn = keep_of(min(row0 + qm, a.Nq - 1));
      int ptr[4] = {0, 0, 0, 0};
      for (int r = 0; r < kn; ++r) {
        int bh4 = -1;
        float bsv = -INFINITY;
        int biv = 0x7fffffff;
#pragma unroll
        for (int hd = 0; hd < 4; ++hd) {
          if (ptr[hd] >= KP) continue;
          const float sv = ms[(hd * KP + ptr[hd]) * 64 + qm];
          const int iv = mi[(hd * KP + ptr[hd]) * 64 + qm];
          if (iv != 0x7fffffff && (bh4 < 0 || bsa_better(sv, iv, bsv, biv))) {
            bh4 = hd;
            bsv = sv;
            biv = iv;
          }
        }
        ml[qm * KP + r] = biv;
#pragma unroll
        for (int hd = 0; hd < 4; ++hd) ptr[hd] += hd == bh4 ? 1 : 0;
      }
    }
    __syncthreads();
  }
  // Output: each wavefront ranks and writes its 16 queries' selections.
  for (int qq = 0; qq < 16; ++qq) {
    const int qw = wave * 16 + qq;
    const int rowm = row0 + qw;
    if (rowm >= a.Nq) break;
    const int tm = a.N - a.Nq + rowm;
    const int cm = tm / a.C;
    const int E = a.causal ? min(cm + 1, a.M1) : a.M1;
    int32_t* out = a.idx + (static_cast<int64_t>(bh) * a.Nq + rowm) * a.K;
    if (E <= a.K) {
      if (lane < a.K) out[lane] = lane < E ? lane : -1;
      continue;
    }
    const int keepn = keep_of(rowm);
    int xb;  // lane j < keepn: the j-th best block
    if (!fallback) {
      const int n = cntq[qw];
      float v = lane < n ? bq[qw * CAP + lane] : -INFINITY;
      xb = lane < n ? bqi[qw * CAP + lane] : 0x7fffffff;
#pragma unroll
      for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) bsa_cx(v, xb, lane, j, (lane & k) == 0);
      }
    } else {
      xb = lane < keepn ? ml[qw * KP + lane] : 0x7fffffff;
    }
    // the keepn ranked blocks, then the forced ones, ascending
    int x = lane < keepn ? xb : 0x7fffffff;
    if (a.causal) {
      if (lane == keepn) x = 0;
      if (cm >= 1 && cm - 1 != 0 && lane == keepn + 1) x = cm - 1;
      if (cm != 0 && lane == keepn + (cm >= 1 && cm - 1 != 0 ? 2 : 1)) x = cm;
    }
    int* sq = sel + wave * 32;
    if (lane < a.K) sq[lane] = x;
    wave_sync();
    int rank = 0;
    for (int y = 0; y < a.K; ++y) rank += sq[y] < x ? 1 : 0;
    if (lane < a.K) out[rank] = x == 0x7fffffff ? -1 : x;
    wave_sync();
  }
}

static bool bsa_mfma_path(const Shape& s) { return s.bf16 && s.K <= 32; }

size_t bsa_ws(const Shape& s, const Geo& geo) {
  if (!bsa_mfma_path(s)) return 0;
  return 2 * ((static_cast<size_t>(s.BH()) * geo.M[1] * s.D * 2 + 255) & ~static_cast<size_t>(255));
}

template <typename T, int D>
static void launch_bsa_g(const Shape& s, const BsaArgs& a, hipStream_t st) {
  dim3 grid(s.Nq, s.BH());
  const size_t lds = (static_cast<size_t>(a.M1) + s.K) * 4;
  if (s.G == 1)
    bsa_rows_kernel<T, D, 1><<<grid, 64, lds, st>>>(a);
  else if (s.G <= 4)
    bsa_rows_kernel<T, D, 4><<<grid, 64, lds, st>>>(a);
  else
    bsa_rows_kernel<T, D, 16><<<grid, 64, lds, st>>>(a);
}

hipError_t launch_flat_bsa(const Shape& s, const Geo& geo, const void* q, const float* pyr, int32_t* idx,
                           void* ws, hipStream_t st) {
  (void)ws;
  BsaArgs a{q, pyr, idx, s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], geo.R,
            kLog2e / sqrtf(static_cast<float>(s.D))};
  if (bsa_mfma_path(s)) {
    const size_t plane = (static_cast<size_t>(s.BH()) * geo.M[1] * s.D * 2 + 255) & ~static_cast<size_t>(255);
    uint16_t* phi = static_cast<uint16_t*>(ws);
    uint16_t* plo = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + plane);
    {
      ProfScope ps("bsa_hilo", st);
      const int64_t n4 = static_cast<int64_t>(s.BH()) * geo.M[1] * s.D / 4;
      bsa_hilo_kernel<<<static_cast<unsigned>((n4 + 255) / 256), 256, 0, st>>>(pyr, geo.R, geo.M[1], s.D, n4, phi,
                                                                              plo);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    ProfScope ps("bsa_mfma", st);
    dim3 grid((s.Nq + 63) / 64, s.BH());
    const int KP = s.K <= 16 ? 16 : 32;
    // staged chunk (hi + lo rows), the score tile and the lists; the pass-1
    // merge reuses the chunk area
    const int GM = s.G == 1 ? 1 : (s.G <= 4 ? 4 : 16);
    const size_t small = std::max<size_t>(static_cast<size_t>(8) * KP * 64 + 64 * KP, 8192) + 3 * 64 + 4 * 32;
    const size_t lds = std::max<size_t>(static_cast<size_t>(2) * 64 * (s.D + 8) * 2 + small * 4,
                                        static_cast<size_t>(64) * GM * 4 * 2 * 4);
    auto go = [&](auto kern) {
      if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      kern<<<grid, 256, lds, st>>>(a, phi, plo);
    };
    auto by_g = [&](auto k1, auto k4, auto k16) {
      if (GM == 1) go(k1); else if (GM == 4) go(k4); else go(k16);
    };
    if (s.D == 128) {
      if (KP == 16)
        by_g(bsa_mfma_kernel<128, 16, 1>, bsa_mfma_kernel<128, 16, 4>, bsa_mfma_kernel<128, 16, 16>);
      else
        by_g(bsa_mfma_kernel<128, 32, 1>, bsa_mfma_kernel<128, 32, 4>, bsa_mfma_kernel<128, 32, 16>);
    } else {
      if (KP == 16)
        by_g(bsa_mfma_kernel<64, 16, 1>, bsa_mfma_kernel<64, 16, 4>, bsa_mfma_kernel<64, 16, 16>);
      else
        by_g(bsa_mfma_kernel<64, 32, 1>, bsa_mfma_kernel<64, 32, 4>, bsa_mfma_kernel<64, 32, 16>);
    }
    return hipGetLastError();
  }
  ProfScope ps("bsa_rows", st);
  if (s.bf16) {
    if (s.D == 128)
      launch_bsa_g<uint16_t, 128>(s, a, st);
    else
      launch_bsa_g<uint16_t, 64>(s, a, st);
  } else {
    if (s.D == 128)
      launch_bsa_g<float, 128>(s, a, st);
    else
      launch_bsa_g<float, 64>(s, a, st);
  }
  return hipGetLastError();
}

}  // namespace pisa
