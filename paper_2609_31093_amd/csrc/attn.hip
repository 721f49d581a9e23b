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
};

template <typename T, int DPL>
__device__ __forceinline__ void store_row_part(T* p, const float (&x)[DPL]);

template <>
__device__ __forceinline__ void store_row_part<uint16_t, 8>(uint16_t* p, const float (&x)[8]) {
  uint4 r;
  r.x = f32_to_bf16_rne(x[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[1])) << 16);
  r.y = f32_to_bf16_rne(x[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[3])) << 16);
  r.z = f32_to_bf16_rne(x[4]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[5])) << 16);
  r.w = f32_to_bf16_rne(x[6]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[7])) << 16);
  *reinterpret_cast<uint4*>(p) = r;
}
template <>
__device__ __forceinline__ void store_row_part<uint16_t, 4>(uint16_t* p, const float (&x)[4]) {
  uint2 r;
  r.x = f32_to_bf16_rne(x[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[1])) << 16);
  r.y = f32_to_bf16_rne(x[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(x[3])) << 16);
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

  const T* kb = static_cast<const T*>(a.k) + static_cast<int64_t>(bh) * a.N * D + sub * DPL;
  const T* vb = static_cast<const T*>(a.v) + static_cast<int64_t>(bh) * a.N * D + sub * DPL;
  const int32_t* sel = a.idx + (static_cast<int64_t>(bh) * a.Nq + row) * a.K;

  float m = -INFINITY, s = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;

  const int total = a.K * a.C;
  for (int i = grp; i < total; i += NGRP) {
    const int slot = i / a.C;
    const int blk = sel[slot];
    if (blk < 0) continue;
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

size_t attn_ws(const Shape&, const Geo&) { return 0; }

hipError_t launch_attention(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                            const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st) {
  (void)geo;
  (void)ws;
  AttnArgs a{q, k, v, idx, o, lse, s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal,
             kLog2e / sqrtf(static_cast<float>(s.D))};
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
