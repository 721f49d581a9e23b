// Host-side launchers of the PISA kernels (internal to libpisa).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace pisa {

// Problem shape as the kernels see it (validated by the ABI layer).
struct Shape {
  int B, H, Hkv, G, Nq, N, D, C, g, K, causal;
  bool bf16;
  int BH() const { return B * Hkv; }
  int gK() const { return g * K; }
};

hipError_t launch_build_pyramid(const Geo& geo, int BH, int D, bool bf16, const void* k, float* pyr,
                                hipStream_t st);

// Fused single-stage selector (all levels, raw leaf keys scored per query).
hipError_t launch_select_fused(const Shape& s, const Geo& geo, const void* q, const void* k,
                               const float* pyr, int32_t* idx, float* score, hipStream_t st);

// Two-stage selector: workspace layout is computed by select_two_stage_ws().
size_t select_two_stage_ws(const Shape& s, const Geo& geo);
hipError_t launch_select_two_stage(const Shape& s, const Geo& geo, const void* q, const void* k,
                                   const float* pyr, int32_t* idx, float* score, void* ws,
                                   hipStream_t st);

// Sparse attention.
size_t attn_ws(const Shape& s, const Geo& geo);
hipError_t launch_attention(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                            const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st);

// Flat block selection baseline.
size_t bsa_ws(const Shape& s, const Geo& geo);
hipError_t launch_flat_bsa(const Shape& s, const Geo& geo, const void* q, const float* pyr, int32_t* idx,
                           void* ws, hipStream_t st);

}  // namespace pisa
