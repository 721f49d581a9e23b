// Device-side helpers shared by the PISA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pisa {

constexpr int kMaxLevels = 32;
constexpr int kMaxCand = 256;     // fanout * K upper bound (candidates per level)
constexpr int kMaxLeafKeys = 256;  // leaf block size C upper bound
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Hierarchy geometry of one problem (identical for every batch and KV head).
// Level l (1-based) has M[l] nodes; node i of level l covers leaf blocks
// [i*gpow[l], (i+1)*gpow[l]) where gpow[l] = fanout^(l-1); stored levels
// 1..Lstore start at pyramid row off[l].  Level sizes follow N; the row
// offsets and R follow the capacity the pyramid is laid out for (>= N).
struct Geo {
  int32_t N, C, g, L, Lstore;
  int32_t Nkv;  // rows per (batch, KV head) in k and v (row stride), >= N
  int32_t lg;  // log2(g) when g is a power of two, else -1
  int32_t M[kMaxLevels + 1];
  int32_t gp[kMaxLevels + 1];  // g^(l-1), saturated at 2^30 (exact wherever it matters: <= g*M_1)
  int64_t gpow[kMaxLevels + 1];
  int64_t off[kMaxLevels + 2];
  int64_t R;  // rows per (batch, KV head)
};

struct bf16x8_t {
  uint4 raw;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) {  // inf or nan: keep, quiet nan
    return static_cast<uint16_t>((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  }
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// x / g^(l-1) for 0 <= x < 2^31 (leaf-block index -> its level-l ancestor).
__device__ __forceinline__ int anc_at(const Geo& geo, int x, int l) {
  if (geo.lg >= 0) return x >> min(geo.lg * (l - 1), 31);
  return static_cast<int>(static_cast<uint32_t>(x) / static_cast<uint32_t>(geo.gp[l]));
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

typedef short v4s16 __attribute__((ext_vector_type(4)));

// Transposing LDS read (ds_read_b64_tr_b16): in each group of 16 lanes, lane
// i receives element i % 4 of the 8-byte reads of lanes 4j + i / 4, j = 0..3.
// With lane s reading 4 consecutive bf16 of row s / 4 at column 4 (s % 4),
// lane i gets column i of those 4 rows: an MFMA operand's 4 consecutive
// k-elements from a row-major tile whose rows are the k index.
__device__ __forceinline__ v4s16 lds_read_tr16x4(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s16*)(p));
}

// Two floats to packed bf16 (round to nearest even, hardware conversion).
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Load DPL consecutive elements (DPL in {4, 8}) of a bf16 or f32 row as floats.
template <typename T, int DPL>
__device__ __forceinline__ void load_row_part(const T* __restrict__ p, float (&x)[DPL]);

template <>
__device__ __forceinline__ void load_row_part<uint16_t, 8>(const uint16_t* __restrict__ p, float (&x)[8]) {
  uint4 r = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

template <>
__device__ __forceinline__ void load_row_part<uint16_t, 4>(const uint16_t* __restrict__ p, float (&x)[4]) {
  uint2 r = *reinterpret_cast<const uint2*>(p);
  x[0] = __uint_as_float(r.x << 16);
  x[1] = __uint_as_float(r.x & 0xFFFF0000u);
  x[2] = __uint_as_float(r.y << 16);
  x[3] = __uint_as_float(r.y & 0xFFFF0000u);
}

template <>
__device__ __forceinline__ void load_row_part<float, 8>(const float* __restrict__ p, float (&x)[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

template <>
__device__ __forceinline__ void load_row_part<float, 4>(const float* __restrict__ p, float (&x)[4]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
}

// Sum over the 16 lanes of a lane group (lanes 16j .. 16j+15).
__device__ __forceinline__ float sum16(float v) {
  v += __shfl_xor(v, 8, 16);
  v += __shfl_xor(v, 4, 16);
  v += __shfl_xor(v, 2, 16);
  v += __shfl_xor(v, 1, 16);
  return v;
}

// ---- cross-lane moves on the VALU (DPP) or the LDS swizzle unit -------------
// dpp_ctrl encodings: quad_perm 0x00-0xFF, row_shr:n 0x110+n, row_ror:n
// 0x120+n, row_bcast15 0x142.  Lanes without a source (or masked rows) read 0.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROW_MASK, 0xF, true);
}
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, dpp_i<CTRL, ROW_MASK>(__builtin_bit_cast(int, v)));
}

// Sum over each 16-lane row; the total lands in lane 15 of the row.
__device__ __forceinline__ float rowsum16_to15(float v) {
  v += dpp_f<0x111>(v);
  v += dpp_f<0x112>(v);
  v += dpp_f<0x114>(v);
  v += dpp_f<0x118>(v);
  return v;
}

// Inclusive prefix sum within each 32-lane half of the wavefront.
__device__ __forceinline__ int scan32_incl(int v) {
  v += dpp_i<0x111>(v);
  v += dpp_i<0x112>(v);
  v += dpp_i<0x114>(v);
  v += dpp_i<0x118>(v);
  v += dpp_i<0x142, 0xA>(v);  // row_bcast15 into rows 1 and 3
  return v;
}

// Value of lane (j XOR lane) within a 32-lane half, for j in {1,2,4,8,16}.
template <int J>
__device__ __forceinline__ int xor32_i(int v) {
  if constexpr (J == 1) return dpp_i<0xB1>(v);        // quad_perm [1,0,3,2]
  else if constexpr (J == 2) return dpp_i<0x4E>(v);   // quad_perm [2,3,0,1]
  else if constexpr (J == 8) return dpp_i<0x128>(v);  // row_ror:8
  else return __builtin_amdgcn_ds_swizzle(v, (J << 10) | 0x1F);
}
template <int J>
__device__ __forceinline__ float xor32_f(float v) {
  return __builtin_bit_cast(float, xor32_i<J>(__builtin_bit_cast(int, v)));
}

// Orders LDS traffic among the lanes of one wavefront (no cross-wave effect).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Base-2 exponent / logarithm on the hardware transcendental unit.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// (score desc, index asc) strict ordering: does (sa, ia) rank before (sb, ib)?
__device__ __forceinline__ bool ranks_before(float sa, int ia, float sb, int ib) {
  return sa > sb || (sa == sb && ia < ib);
}

}  // namespace pisa
