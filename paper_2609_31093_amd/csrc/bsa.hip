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
  extern __shared__ float sc[];  // [M1] scores, then [K] output scratch (as int)
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
// MFMA flat selection (bf16 q).  One workgroup per tile of 64 consecutive
// query rows of one (batch, KV head).  Leaf means are streamed in chunks of
// 64 blocks, split once into bf16 hi + lo parts in LDS (hi + lo reproduces
// the fp32 mean to ~2^-17 relative), and scored with
// v_mfma_f32_32x32x16_bf16: wave w covers queries (w&1)*32.. and blocks
// (w>>1)*32.. of the chunk, so each query's blocks are spread over four
// "holders" (two lanes of two waves).  Every holder keeps its own top list
// of the best non-forced eligible blocks in registers (insertion in block
// order, so equal scores keep the smaller index first); the four lists of a
// query are merged at the end.  With G > 1 a first pass over the chunks
// gathers each head's normaliser (online max / sum of 2^z over eligible
// non-forced blocks) and the second pass ranks by the sum of the heads'
// probabilities.
// ----------------------------------------------------------------------------

typedef __bf16 bf16x8b __attribute__((ext_vector_type(8)));
typedef float f32x16b __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8b u4_bf16x8(uint4 r) { return __builtin_bit_cast(bf16x8b, r); }

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
  // v arrives with a larger block index than every entry already held.
  __device__ __forceinline__ void insert(float v, int idx) {
    if (!(v > s[KP - 1])) return;
    float cur = v;
    int ci = idx;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      const bool sw = cur > s[j];
      const float ts = s[j];
      const int ti = i[j];
      s[j] = sw ? cur : ts;
      i[j] = sw ? ci : ti;
      cur = sw ? ts : cur;
      ci = sw ? ti : ci;
    }
  }
};

template <int D, int KP>
__global__ __launch_bounds__(256) void bsa_mfma_kernel(BsaArgs a) {
  constexpr int KS = D / 16;
  constexpr int LDS_ROW = D + 8;
  extern __shared__ uint16_t lds[];
  uint16_t* shi = lds;                   // [64][LDS_ROW]
  uint16_t* slo = lds + 64 * LDS_ROW;    // [64][LDS_ROW]
  float* hred = reinterpret_cast<float*>(lds);  // pass-1 merge, reuses the chunk area after the loop

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 31, half = lane >> 5;
  const int qh = wave & 1, bhalf = wave >> 1;
  const int bh = blockIdx.y;
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int row0 = blockIdx.x * 64;
  const int row = row0 + qh * 32 + col;
  const bool live = row < a.Nq;
  const int rowc = live ? row : a.Nq - 1;
  const int t = a.N - a.Nq + rowc;
  const int c = t / a.C;
  const int elig = a.causal ? min(c + 1, a.M1) : a.M1;  // blocks [0, elig) are eligible
  const int t_last = a.N - a.Nq + min(row0 + 63, a.Nq - 1);
  const int nblk = a.causal ? min(t_last / a.C + 1, a.M1) : a.M1;
  const int nchunk = (nblk + 63) / 64;
  auto forced = [&](int i) { return a.causal && (i == 0 || i == c || i == c - 1); };
  const float* pbase = a.pyr + static_cast<int64_t>(bh) * a.R * D;

  auto stage_chunk = [&](int ch) {
    for (int e = threadIdx.x; e < 64 * (D / 4); e += 256) {
      const int r = e / (D / 4), c4 = (e - r * (D / 4)) * 4;
      const int blk = ch * 64 + r;
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (blk < nblk) x = *reinterpret_cast<const float4*>(pbase + static_cast<int64_t>(blk) * D + c4);
      const uint32_t h01 = pack2_bf16(x.x, x.y), h23 = pack2_bf16(x.z, x.w);
      const float hx = __uint_as_float(h01 << 16), hy = __uint_as_float(h01 & 0xFFFF0000u);
      const float hz = __uint_as_float(h23 << 16), hw = __uint_as_float(h23 & 0xFFFF0000u);
      const uint32_t l01 = pack2_bf16(x.x - hx, x.y - hy), l23 = pack2_bf16(x.z - hz, x.w - hw);
      *reinterpret_cast<uint2*>(shi + r * LDS_ROW + c4) = make_uint2(h01, h23);
      *reinterpret_cast<uint2*>(slo + r * LDS_ROW + c4) = make_uint2(l01, l23);
    }
  };
  // logits (log2 units) of this lane's 16 blocks of the chunk for head hh
  auto chunk_logits = [&](int hh, f32x16b& acc) {
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
  auto block_of = [&](int ch, int r) { return ch * 64 + bhalf * 32 + 8 * (r >> 2) + 4 * half + (r & 3); };

  // Pass 1 (G > 1): each head's log2 normaliser over eligible non-forced blocks.
  float lnorm[16];
#pragma unroll
  for (int hh = 0; hh < 16; ++hh) lnorm[hh] = 0.f;
  if (a.G > 1) {
    float hm[16], hs[16];
#pragma unroll
    for (int hh = 0; hh < 16; ++hh) {
      hm[hh] = -INFINITY;
      hs[hh] = 0.f;
    }
    for (int ch = 0; ch < nchunk; ++ch) {
      __syncthreads();
      stage_chunk(ch);
      __syncthreads();
#pragma unroll
      for (int hh = 0; hh < 16; ++hh) {
        if (hh < a.G) {
          f32x16b acc;
          chunk_logits(hh, acc);
          float m = hm[hh];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int blk = block_of(ch, r);
            if (blk < elig && !forced(blk)) m = fmaxf(m, acc[r]);
          }
          float sacc = (m == -INFINITY) ? 0.f : hs[hh] * fast_exp2(hm[hh] - m);
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int blk = block_of(ch, r);
            if (blk < elig && !forced(blk)) sacc += fast_exp2(acc[r] - m);
          }
          hm[hh] = m;
          hs[hh] = sacc;
        }
      }
    }
    __syncthreads();
    // merge the four holders of each query through LDS
    const int q64 = qh * 32 + col, holder = bhalf * 2 + half;
#pragma unroll
    for (int hh = 0; hh < 16; ++hh) {
      if (hh < a.G) {
        hred[((q64 * 16 + hh) * 4 + holder) * 2 + 0] = hm[hh];
        hred[((q64 * 16 + hh) * 4 + holder) * 2 + 1] = hs[hh];
      }
    }
    __syncthreads();
#pragma unroll
    for (int hh = 0; hh < 16; ++hh) {
      if (hh >= a.G) continue;
      float m = -INFINITY, sacc = 0.f;
      for (int k2 = 0; k2 < 4; ++k2) {
        const float m2 = hred[((q64 * 16 + hh) * 4 + k2) * 2 + 0];
        const float s2 = hred[((q64 * 16 + hh) * 4 + k2) * 2 + 1];
        const float mn = fmaxf(m, m2);
        sacc = (mn == -INFINITY) ? 0.f : sacc * fast_exp2(m - mn) + s2 * fast_exp2(m2 - mn);
        m = mn;
      }
      lnorm[hh] = m + fast_log2(sacc);
    }
  }

  // Pass 2: rank.
  TopList<KP> top;
  top.init();
  for (int ch = 0; ch < nchunk; ++ch) {
    __syncthreads();
    stage_chunk(ch);
    __syncthreads();
    float u[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) u[r] = 0.f;
    if (a.G == 1) {
      f32x16b acc;
      chunk_logits(0, acc);
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = acc[r];
    } else {
#pragma unroll
      for (int hh = 0; hh < 16; ++hh) {
        if (hh < a.G) {
          f32x16b acc;
          chunk_logits(hh, acc);
#pragma unroll
          for (int r = 0; r < 16; ++r) u[r] += fast_exp2(acc[r] - lnorm[hh]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int blk = block_of(ch, r);
      if (blk < elig && !forced(blk)) top.insert(u[r], blk);
    }
  }
  __syncthreads();
  // Merge the four holders' lists of each query: LDS [64 queries][4 holders][KP].
  float* ms = reinterpret_cast<float*>(lds);
  int* mi = reinterpret_cast<int*>(ms + 64 * 4 * KP);
  {
    const int q64 = qh * 32 + col, holder = bhalf * 2 + half;
#pragma unroll
    for (int j = 0; j < KP; ++j) {
      ms[(q64 * 4 + holder) * KP + j] = top.s[j];
      mi[(q64 * 4 + holder) * KP + j] = top.i[j];
    }
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int q64 = threadIdx.x;
    const int rowm = row0 + q64;
    if (rowm < a.Nq) {
      const int tm = a.N - a.Nq + rowm;
      const int cm = tm / a.C;
      const int E = a.causal ? min(cm + 1, a.M1) : a.M1;
      int32_t* out = a.idx + (static_cast<int64_t>(bh) * a.Nq + rowm) * a.K;
      if (E <= a.K) {
        for (int j = 0; j < a.K; ++j) out[j] = j < E ? j : -1;
      } else {
        const int nF = a.causal ? 1 + (cm != 0) + (cm - 1 > 0) : 0;
        const int keepn = a.K - nF;
        int* sel = mi + 64 * 4 * KP + q64 * 32;  // LDS scratch of this query (K <= 32)
        int n = 0;
        // pick the best keepn among the 4*KP entries (score desc, index asc)
        float* qs = ms + q64 * 4 * KP;
        int* qi = mi + q64 * 4 * KP;
        for (int r = 0; r < keepn; ++r) {
          int bj = -1;
          for (int j = 0; j < 4 * KP; ++j) {
            if (qi[j] == 0x7fffffff) continue;
            if (bj < 0 || ranks_before(qs[j], qi[j], qs[bj], qi[bj])) bj = j;
          }
          sel[n++] = qi[bj];
          qi[bj] = 0x7fffffff;
        }
        if (a.causal) {
          sel[n++] = 0;
          if (cm >= 1 && cm - 1 != 0) sel[n++] = cm - 1;
          if (cm != 0) sel[n++] = cm;
        }
        // ascending insertion sort of the K entries
        for (int x = 1; x < n; ++x) {
          const int v = sel[x];
          int y = x - 1;
          while (y >= 0 && sel[y] > v) {
            sel[y + 1] = sel[y];
            --y;
          }
          sel[y + 1] = v;
        }
        for (int j = 0; j < a.K; ++j) out[j] = j < n ? sel[j] : -1;
      }
    }
  }
}

size_t bsa_ws(const Shape&, const Geo&) { return 0; }

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
  if (s.bf16 && s.K <= 32) {
    ProfScope ps("bsa_mfma", st);
    dim3 grid((s.Nq + 63) / 64, s.BH());
    const int KP = s.K <= 16 ? 16 : 32;
    const size_t chunk = static_cast<size_t>(2) * 64 * (s.D + 8) * 2;
    const size_t merge = static_cast<size_t>(64) * 4 * KP * 8 + static_cast<size_t>(64) * 32 * 4;
    const size_t hred = static_cast<size_t>(64) * 16 * 4 * 2 * 4;
    const size_t lds = std::max(chunk, std::max(merge, s.G > 1 ? hred : size_t(0)));
    auto go = [&](auto kern) {
      if (lds > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
      kern<<<grid, 256, lds, st>>>(a);
    };
    if (s.D == 128) {
      if (KP == 16) go(bsa_mfma_kernel<128, 16>); else go(bsa_mfma_kernel<128, 32>);
    } else {
      if (KP == 16) go(bsa_mfma_kernel<64, 16>); else go(bsa_mfma_kernel<64, 32>);
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
