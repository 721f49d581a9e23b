// Host-side launchers of the PISA kernels (internal to libpisa).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace pisa {

// Brackets the kernel launches of its scope with timing events when
// per-kernel profiling is enabled (pisa_profile_enable); otherwise inert.
class ProfScope {
 public:
  ProfScope(const char* name, hipStream_t st);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  const char* name_;
  hipStream_t st_;
  void* a_;
};

// Problem shape as the kernels see it (validated by the ABI layer).
struct Shape {
  int B, H, Hkv, G, Nq, N, D, C, g, K, causal;
  int Nkv;    // rows per (batch, KV head) in k and v (row stride), >= N
  int score;  // PISA_SCORE_* reducer of the selection
  bool bf16;
  int BH() const { return B * Hkv; }
  int gK() const { return g * K; }
};

// Pair clustering by key block (cluster.hip).
constexpr int kClusterLeaf = 0;  // leaf scoring: rows with more than K candidates, forced blocks skipped
constexpr int kClusterAttn = 1;  // attention: every non-negative slot
constexpr int kClusterLeafParent = 2;  // leaf scoring grouped by parent node: one entry per
                                       // (row, parent) at the slot of its first non-forced child
constexpr int kClusterAttnFar = 3;     // causal attention: every non-negative slot except the row's first,
                                       // previous and own leaf block (those are attended per leaf block)
struct ClusterArgs {
  const int32_t* list;  // [BH, Nq, S] block per slot, -1 = none
  const int32_t* cnt;   // [BH, Nq] candidates per row (leaf mode only)
  int S, Nq, N, C, K, causal, M1, mode;  // M1: number of bins (leaf blocks, or parents)
  int row0, nrows;      // rows [row0, row0 + nrows) of every (batch, KV head)
  int g;                // fan-out (parent mode)
  // attention modes: rows whose tile flag is set (skip[bh * skip_tiles +
  // (row >> skip_shift)]) were attended by the row-tile union kernel
  const uint8_t* skip = nullptr;
  int skip_shift = 0, skip_tiles = 0;
};
constexpr int kClusterTile = 256;  // pairs per inner tile of the block attention's workgroup chunks
struct ClusterOut {
  const int32_t* offs;   // [BH*M1 + 1] cluster start offsets into pairs
  const int32_t* toffs;  // [BH*M1 + 1] first chunk of each cluster (the `tile` of launch_cluster pairs per chunk)
  const int32_t* pairs;  // (row - row0) << 8 | slot, grouped by (bh, block)
  int64_t ncl;           // BH*M1
};
// workspace of launch_cluster for up to max_pairs pairs and max_rows rows per
// (batch, KV head) in one launch
size_t cluster_ws(int BH, int M1, int64_t max_pairs, int max_rows);

// Chunk w of the cluster list when the consumer takes up to `tile` pairs per
// workgroup (the tile offsets of launch_cluster(..., tile)): its cluster (the
// largest cl with toffs[cl] <= w) and pair range; false past the last chunk.
__device__ __forceinline__ bool cluster_chunk(const int32_t* __restrict__ offs, const int32_t* __restrict__ toffs,
                                              int64_t ncl, int64_t w, int tile, int64_t& cl, int& beg, int& end) {
  if (w >= toffs[ncl]) return false;
  int64_t lo = 0, hi = ncl - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (toffs[mid] <= w) lo = mid; else hi = mid - 1;
  }
  cl = lo;
  beg = offs[cl] + static_cast<int>(w - toffs[cl]) * tile;
  end = min(offs[cl + 1], beg + tile);
  return true;
}
// Groups the pairs by block; toffs counts `tile`-pair chunks per cluster.
hipError_t launch_cluster(const ClusterArgs& a, int BH, void* ws, ClusterOut* out, hipStream_t st, int tile);
int64_t cluster_max_chunks(int BH, int M1, int64_t max_pairs, int tile);

hipError_t launch_build_pyramid(const Geo& geo, int BH, int D, bool bf16, const void* k, float* pyr,
                                hipStream_t st);
// Recompute the leaves holding rows [n_old, N), their ancestors, and whole
// levels absent at n_old (geo_old: the geometry at n_old, same layout).
hipError_t launch_pyramid_append(const Geo& geo, const Geo& geo_old, int BH, int D, bool bf16, const void* k,
                                 float* pyr, int n_old, hipStream_t st);

// Decode-cache growth: the stored levels' rows and the first N rows of k and
// v moved into a layout for a larger capacity.  All counts and offsets are in
// 16-byte units; lev_end[l] is the end of stored level l+1 within a head's
// stream (levels in order), off_old/off_new that level's first unit in the
// old / new pyramid of one head.  kv_units = 0 copies no keys or values.
struct GrowArgs {
  int64_t pyr_units, kv_units;
  int64_t pyr_old_stride, pyr_new_stride;  // units per head
  int64_t kv_old_stride, kv_new_stride;    // units per head
  int64_t lev_end[kMaxLevels];
  int64_t off_old[kMaxLevels], off_new[kMaxLevels];
};
hipError_t launch_cache_grow(const GrowArgs& a, int BH, const float* pyr_old, float* pyr_new, const void* k_old,
                             void* k_new, const void* v_old, void* v_new, hipStream_t st);

// Fused single-stage selector (all levels, raw leaf keys scored per query).
hipError_t launch_select_fused(const Shape& s, const Geo& geo, const void* q, const void* k,
                               const float* pyr, int32_t* idx, float* score, hipStream_t st);

// Split selector for few rows (decode): workspace of select_split_ws().
size_t select_split_ws(const Shape& s);
hipError_t launch_select_split(const Shape& s, const Geo& geo, const void* q, const void* k, const float* pyr,
                               int32_t* idx, float* score, void* ws, hipStream_t st);

// Two-stage selector: workspace layout is computed by select_two_stage_ws().
size_t select_two_stage_ws(const Shape& s, const Geo& geo);
hipError_t launch_select_two_stage(const Shape& s, const Geo& geo, const void* q, const void* k,
                                   const float* pyr, int32_t* idx, float* score, void* ws,
                                   hipStream_t st);

// Backward of the sparse attention with the selection held fixed (attn_bwd.hip).
size_t attn_bwd_ws(const Shape& s, const Geo& geo);
bool attn_bwd_supported(const Shape& s);
hipError_t launch_attention_bwd(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                                const int32_t* idx, const void* o, const float* lse, const void* d_o, void* dq,
                                void* dk, void* dv, void* ws, hipStream_t st);

// Sparse attention.
size_t attn_ws(const Shape& s, const Geo& geo);
hipError_t launch_attention(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                            const int32_t* idx, void* o, float* lse, void* ws, hipStream_t st);

// Block-selection quality diagnostic (quality.hip).
struct QualityArgs {
  int H, Hkv, G, Nq, N, C, K, causal, M1, n_rows;
  float qscale2;
  int Nkv;  // rows per (batch, KV head) in k
};
size_t quality_ws(const Shape& s, int n_rows);
bool quality_supported(const Shape& s);
hipError_t launch_quality(const Shape& s, const void* q, const void* k, const int32_t* idx, const int32_t* rows,
                          int n_rows, float* metrics, int32_t* ref, void* ws, hipStream_t st);

// Flat block selection baseline.
size_t bsa_ws(const Shape& s, const Geo& geo);
hipError_t launch_flat_bsa(const Shape& s, const Geo& geo, const void* q, const float* pyr, int32_t* idx,
                           void* ws, hipStream_t st);

}  // namespace pisa
