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
