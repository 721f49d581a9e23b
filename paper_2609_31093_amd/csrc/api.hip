// C ABI of libpisa: argument validation, hierarchy geometry, workspace sizing
// and dispatch to the kernels.  Nothing is enqueued before every argument has
// been checked; no call allocates device memory or synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "../../include/pisa.h"
#include "common.h"
#include "kernels.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Level sizes M[1..L] of an N-token hierarchy (Sec. 3.2 eq. key_hierarchy);
// returns L or a negative status.
int level_sizes(int64_t N, int32_t C, int32_t g, int32_t* M) {
  int64_t m = (N + C - 1) / C;
  int L = 1;
  M[1] = static_cast<int32_t>(m);
  while (m > 1) {
    m = (m + g - 1) / g;
    ++L;
    if (L > pisa::kMaxLevels) return PISA_ERR_UNSUPPORTED;
    M[L] = static_cast<int32_t>(m);
  }
  return L;
}

// Geometry of an N-token problem whose pyramid (and k/v rows) are laid out
// for cap >= N tokens.
int compute_geo(int32_t N, int32_t C, int32_t g, pisa::Geo* geo, int32_t cap = 0) {
  if (N < 1 || C < 1 || g < 2) return PISA_ERR_INVALID_ARG;
  if (cap == 0) cap = N;
  if (cap < N) return PISA_ERR_INVALID_ARG;
  pisa::Geo G{};
  G.N = N;
  G.Nkv = cap;
  G.C = C;
  G.g = g;
  const int L = level_sizes(N, C, g, G.M);
  if (L < 0) return L;
  int32_t Mc[pisa::kMaxLevels + 1] = {};
  const int Lc = level_sizes(cap, C, g, Mc);
  if (Lc < 0) return Lc;
  G.L = L;
  G.Lstore = L > 1 ? L - 1 : 1;
  G.lg = -1;
  for (int b = 0; b < 31; ++b)
    if ((1 << b) == g) G.lg = b;
  G.gpow[1] = 1;
  G.gp[1] = 1;
  for (int l = 2; l <= pisa::kMaxLevels; ++l)
    G.gp[l] = G.gp[l - 1] > (1 << 26) ? (1 << 30) : G.gp[l - 1] * g;
  for (int l = 2; l <= pisa::kMaxLevels; ++l)  // saturate beyond the root
    G.gpow[l] = G.gpow[l - 1] > (int64_t(1) << 40) ? G.gpow[l - 1] : G.gpow[l - 1] * g;
  // Row offsets of the capacity layout: levels 1 .. max(1, Lc - 1) of a
  // cap-token hierarchy (which contain the stored levels of N).
  const int Lcs = Lc > 1 ? Lc - 1 : 1;
  G.off[1] = 0;
  for (int l = 1; l <= pisa::kMaxLevels; ++l) G.off[l + 1] = G.off[l] + (l <= Lcs ? Mc[l] : 0);
  G.R = G.off[Lcs + 1];
  if (geo) *geo = G;
  return L;
}

// Leaf blocks of the capacity (Ncap tokens) a problem may reserve.
constexpr int32_t kMaxLeafBlocks = 65535;

// Full validation of a problem; fills the kernel view on success.
int check_problem(const pisa_problem* p, pisa::Shape* s, pisa::Geo* geo) {
  if (!p) return fail(PISA_ERR_INVALID_ARG, "problem is NULL");
  if (p->B < 1 || p->H < 1 || p->Hkv < 1)
    return fail(PISA_ERR_INVALID_ARG, "B, H and Hkv must be >= 1 (got %d, %d, %d)", p->B, p->H, p->Hkv);
  if (p->H % p->Hkv != 0)
    return fail(PISA_ERR_INVALID_ARG, "H (%d) must be a multiple of Hkv (%d)", p->H, p->Hkv);
  if (p->N < 1 || p->Nq < 1 || p->Nq > p->N)
    return fail(PISA_ERR_INVALID_ARG, "need 1 <= Nq <= N (got Nq=%d, N=%d)", p->Nq, p->N);
  if (p->C < 1 || p->fanout < 2 || p->K < 1)
    return fail(PISA_ERR_INVALID_ARG, "need C >= 1, fanout >= 2, K >= 1 (got %d, %d, %d)", p->C, p->fanout,
                p->K);
  if (p->causal != 0 && p->causal != 1) return fail(PISA_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (p->causal && p->K < 3)
    return fail(PISA_ERR_INVALID_ARG, "causal selection keeps the first, previous and current blocks: K >= 3");
  if (p->dtype != PISA_DTYPE_F32 && p->dtype != PISA_DTYPE_BF16)
    return fail(PISA_ERR_INVALID_ARG, "unknown dtype %d", p->dtype);
  if (p->schedule < PISA_SCHEDULE_AUTO || p->schedule > PISA_SCHEDULE_SPLIT)
    return fail(PISA_ERR_INVALID_ARG, "unknown schedule %d", p->schedule);
  if (p->d != 64 && p->d != 128) return fail(PISA_ERR_UNSUPPORTED, "head dim %d (supported: 64, 128)", p->d);
  if (p->C % 32 != 0 || p->C > pisa::kMaxLeafKeys)
    return fail(PISA_ERR_UNSUPPORTED, "block size %d (supported: multiples of 32 up to 256)", p->C);
  if (p->fanout > 16) return fail(PISA_ERR_UNSUPPORTED, "fanout %d (supported: 2..16)", p->fanout);
  const int G = p->H / p->Hkv;
  if (G > 16) return fail(PISA_ERR_UNSUPPORTED, "group size H/Hkv = %d (supported: <= 16)", G);
  if (static_cast<int64_t>(p->fanout) * p->K > pisa::kMaxCand)
    return fail(PISA_ERR_UNSUPPORTED, "fanout*K = %lld exceeds %d", static_cast<long long>(p->fanout) * p->K,
                pisa::kMaxCand);
  if (static_cast<int64_t>(p->fanout) * p->fanout * p->K * G > 2048)
    return fail(PISA_ERR_UNSUPPORTED, "fanout^2*K*G = %lld exceeds 2048",
                static_cast<long long>(p->fanout) * p->fanout * p->K * G);
  if (p->Nq >= (1 << 23)) return fail(PISA_ERR_UNSUPPORTED, "Nq %d exceeds 2^23-1", p->Nq);
  if (static_cast<int64_t>(p->B) * p->Hkv > 65535 || static_cast<int64_t>(p->B) * p->H > 65535)
    return fail(PISA_ERR_UNSUPPORTED, "B*H must be <= 65535");
  if (p->score < PISA_SCORE_LSE || p->score > PISA_SCORE_MEAN_VAR)
    return fail(PISA_ERR_INVALID_ARG, "unknown score %d", p->score);
  if (p->Ncap != 0 && p->Ncap < p->N)
    return fail(PISA_ERR_INVALID_ARG, "Ncap (%d) must be 0 or >= N (%d)", p->Ncap, p->N);
  pisa::Geo g{};
  const int L = compute_geo(p->N, p->C, p->fanout, &g, p->Ncap);
  if (L < 0) return fail(L, "hierarchy too deep");
  if ((static_cast<int64_t>(g.Nkv) + p->C - 1) / p->C > kMaxLeafBlocks)
    return fail(PISA_ERR_UNSUPPORTED, "more than %d leaf blocks", kMaxLeafBlocks);
  if (s) {
    s->B = p->B;
    s->H = p->H;
    s->Hkv = p->Hkv;
    s->G = G;
    s->Nq = p->Nq;
    s->N = p->N;
    s->D = p->d;
    s->C = p->C;
    s->g = p->fanout;
    s->K = p->K;
    s->causal = p->causal;
    s->Nkv = g.Nkv;
    s->score = p->score;
    s->bf16 = p->dtype == PISA_DTYPE_BF16;
  }
  if (geo) *geo = g;
  return PISA_OK;
}

int check_ptr(const void* ptr, const char* name, bool nullable = false) {
  if (!ptr) return nullable ? PISA_OK : fail(PISA_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(ptr)) return fail(PISA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return PISA_OK;
}

int check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return PISA_OK;
  if (ws_bytes < need)
    return fail(PISA_ERR_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, need);
  if (!ws) return fail(PISA_ERR_WORKSPACE, "workspace is NULL, need %zu bytes", need);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(PISA_ERR_INVALID_ARG, "workspace not 256-byte aligned");
  return PISA_OK;
}

int device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return PISA_OK;
  return fail(PISA_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// The cluster histogram of the two-stage schedule lives in LDS (one int per
// leaf block).
constexpr int kMaxClusterBins = 16384;

// Rows (query rows x batch x KV heads) up to which the automatic schedule
// spreads each row's leaf candidates over workgroups of their own.
constexpr int64_t kSplitMaxRows = 2048;

int pick_schedule(const pisa_problem* p, const pisa::Shape& s, const pisa::Geo& g) {
  if (p->schedule != PISA_SCHEDULE_AUTO) return p->schedule;
  const int64_t rows = static_cast<int64_t>(s.Nq) * s.BH();
  // Key-block reuse pays once many queries share the key blocks (Sec. 3.3).
  if (s.bf16 && rows >= 4096 && g.M[1] <= kMaxClusterBins) return PISA_SCHEDULE_TWO_STAGE;
  return rows <= kSplitMaxRows ? PISA_SCHEDULE_SPLIT : PISA_SCHEDULE_FUSED;
}

size_t select_ws(int sched, const pisa::Shape& s, const pisa::Geo& g) {
  if (sched == PISA_SCHEDULE_TWO_STAGE) return pisa::select_two_stage_ws(s, g);
  if (sched == PISA_SCHEDULE_SPLIT) return pisa::select_split_ws(s);
  return 0;
}

#define PISA_TRY(x)           \
  do {                        \
    const int _st = (x);      \
    if (_st != PISA_OK) return _st; \
  } while (0)

// Argument checks of pisa_select and pisa_select_static (everything except
// the workspace); fills the kernel view and the schedule.
int check_select(const pisa_problem* p, const void* q, const void* k, const float* pyramid, const int32_t* block_idx,
                 const float* block_score, pisa::Shape* s, pisa::Geo* g, int* sched) {
  PISA_TRY(check_problem(p, s, g));
  PISA_TRY(check_ptr(q, "q"));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(pyramid, "pyramid"));
  PISA_TRY(check_ptr(block_idx, "block_idx"));
  PISA_TRY(check_ptr(block_score, "block_score", true));
  *sched = pick_schedule(p, *s, *g);
  const bool two = *sched == PISA_SCHEDULE_TWO_STAGE;
  if (two && !s->bf16)
    return fail(PISA_ERR_UNSUPPORTED, "the two-stage schedule runs on bf16 inputs (use the fused schedule)");
  if (two && g->M[1] > kMaxClusterBins)
    return fail(PISA_ERR_UNSUPPORTED, "the two-stage schedule needs N/C <= %d", kMaxClusterBins);
  return PISA_OK;
}

int run_select(const pisa::Shape& s, const pisa::Geo& g, int sched, const void* q, const void* k,
               const float* pyramid, int32_t* block_idx, float* block_score, void* ws, hipStream_t st,
               const char* who) {
  hipError_t e;
  if (sched == PISA_SCHEDULE_TWO_STAGE)
    e = pisa::launch_select_two_stage(s, g, q, k, pyramid, block_idx, block_score, ws, st);
  else if (sched == PISA_SCHEDULE_SPLIT)
    e = pisa::launch_select_split(s, g, q, k, pyramid, block_idx, block_score, ws, st);
  else
    e = pisa::launch_select_fused(s, g, q, k, pyramid, block_idx, block_score, st);
  return device_status(e, who);
}

// Per-device address of the static scratch of pisa_select_static, taken once
// per device (with that device current) on its first call there.
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

}  // namespace

namespace pisa {
// Scratch of pisa_select_static: one copy per device, held while the library
// is loaded.  Host code never passes this name to a kernel or a copy (on the
// host it only names the symbol); it uses the device address from
// hipGetSymbolAddress instead.
__device__ __align__(256) unsigned char scratch[PISA_STATIC_SCRATCH_BYTES];
}  // namespace pisa

namespace {

int static_scratch(void** out) {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(PISA_ERR_UNSUPPORTED, "device %d (supported: < %d)", dev, kMaxDevices);
  std::call_once(g_scratch_once[dev], [dev] {
    void* ptr = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&ptr, HIP_SYMBOL(pisa::scratch));
    g_scratch_ptr[dev] = ptr;
  });
  if (g_scratch_err[dev] != hipSuccess) return device_status(g_scratch_err[dev], "hipGetSymbolAddress(scratch)");
  if ((reinterpret_cast<uintptr_t>(g_scratch_ptr[dev]) & 255u) != 0)
    return fail(PISA_ERR_DEVICE, "static scratch is not 256-byte aligned");
  *out = g_scratch_ptr[dev];
  return PISA_OK;
}

}  // namespace

extern "C" {

int pisa_num_levels(int32_t N, int32_t C, int32_t fanout) {
  const int L = compute_geo(N, C, fanout, nullptr);
  if (L < 0) return fail(L, "invalid N, C or fanout");
  return L;
}

int pisa_pyramid_layout(const pisa_problem* p, int64_t* level_row_offset, int64_t* rows_R) {
  pisa::Geo g{};
  PISA_TRY(check_problem(p, nullptr, &g));
  if (!level_row_offset || !rows_R) return fail(PISA_ERR_INVALID_ARG, "output pointers must be non-NULL");
  for (int l = 1; l <= g.L; ++l) level_row_offset[l - 1] = l <= g.Lstore ? g.off[l] : g.R;
  *rows_R = g.R;
  return g.L;
}

size_t pisa_pyramid_bytes(const pisa_problem* p) {
  pisa::Geo g{};
  if (check_problem(p, nullptr, &g) != PISA_OK) return 0;
  return static_cast<size_t>(p->B) * p->Hkv * g.R * p->d * sizeof(float);
}

size_t pisa_select_workspace_bytes(const pisa_problem* p) {
  pisa::Shape s{};
  pisa::Geo g{};
  if (check_problem(p, &s, &g) != PISA_OK) return 0;
  return select_ws(pick_schedule(p, s, g), s, g);
}

size_t pisa_bsa_workspace_bytes(const pisa_problem* p) {
  pisa::Shape s{};
  pisa::Geo g{};
  if (check_problem(p, &s, &g) != PISA_OK) return 0;
  return pisa::bsa_ws(s, g);
}

size_t pisa_attn_workspace_bytes(const pisa_problem* p) {
  pisa::Shape s{};
  pisa::Geo g{};
  if (check_problem(p, &s, &g) != PISA_OK) return 0;
  return pisa::attn_ws(s, g);
}

int pisa_build_pyramid(const pisa_problem* p, const void* k, float* pyramid, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(pyramid, "pyramid"));
  return device_status(pisa::launch_build_pyramid(g, s.BH(), s.D, s.bf16, k, pyramid,
                                                  static_cast<hipStream_t>(stream)),
                       "pisa_build_pyramid");
}

int pisa_pyramid_append(const pisa_problem* p, const void* k, float* pyramid, int32_t n_old, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(pyramid, "pyramid"));
  if (n_old < 0 || n_old > p->N) return fail(PISA_ERR_INVALID_ARG, "need 0 <= n_old <= N (got %d, N=%d)", n_old, p->N);
  if (n_old == p->N) return PISA_OK;
  pisa::Geo g_old{};
  if (n_old > 0) compute_geo(n_old, p->C, p->fanout, &g_old, g.Nkv);
  return device_status(pisa::launch_pyramid_append(g, g_old, s.BH(), s.D, s.bf16, k, pyramid, n_old,
                                                   static_cast<hipStream_t>(stream)),
                       "pisa_pyramid_append");
}

int32_t pisa_cache_capacity(int32_t cap, int32_t need, int32_t C) {
  if (cap < 0 || need < 1 || C < 1) return fail(PISA_ERR_INVALID_ARG, "need cap >= 0, need >= 1, C >= 1");
  if (need <= cap) return cap;
  const int64_t grown = std::max<int64_t>(need, static_cast<int64_t>(cap) + (static_cast<int64_t>(cap) + 1) / 2);
  const int64_t rounded = (grown + C - 1) / C * C;
  const int64_t limit = static_cast<int64_t>(kMaxLeafBlocks) * C;
  if (rounded <= limit && rounded <= INT32_MAX) return static_cast<int32_t>(rounded);
  if (need <= limit && need <= INT32_MAX) return static_cast<int32_t>(std::min<int64_t>(limit, INT32_MAX));
  return fail(PISA_ERR_UNSUPPORTED, "a cache of %d tokens exceeds %d leaf blocks of %d", need, kMaxLeafBlocks, C);
}

int pisa_cache_grow(const pisa_problem* p, int32_t new_cap, const float* pyr_old, float* pyr_new, const void* k_old,
                    void* k_new, const void* v_old, void* v_new, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  if (new_cap < g.Nkv)
    return fail(PISA_ERR_INVALID_ARG, "new_cap (%d) is below the current capacity (%d)", new_cap, g.Nkv);
  pisa_problem pn = *p;
  pn.Ncap = new_cap;
  pisa::Geo gn{};
  PISA_TRY(check_problem(&pn, nullptr, &gn));
  PISA_TRY(check_ptr(pyr_old, "pyr_old"));
  PISA_TRY(check_ptr(pyr_new, "pyr_new"));
  const bool kv = k_old || k_new || v_old || v_new;
  if (kv) {
    PISA_TRY(check_ptr(k_old, "k_old"));
    PISA_TRY(check_ptr(k_new, "k_new"));
    PISA_TRY(check_ptr(v_old, "v_old"));
    PISA_TRY(check_ptr(v_new, "v_new"));
  }
  const int64_t BH = s.BH();
  const size_t esz = s.bf16 ? 2 : 4;
  auto overlap = [](const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
  };
  const size_t pyr_old_bytes = static_cast<size_t>(BH) * g.R * s.D * 4;
  const size_t pyr_new_bytes = static_cast<size_t>(BH) * gn.R * s.D * 4;
  if (overlap(pyr_old, pyr_old_bytes, pyr_new, pyr_new_bytes))
    return fail(PISA_ERR_INVALID_ARG, "pyr_old and pyr_new overlap");
  if (kv) {
    const size_t kv_old_bytes = static_cast<size_t>(BH) * g.Nkv * s.D * esz;
    const size_t kv_new_bytes = static_cast<size_t>(BH) * gn.Nkv * s.D * esz;
    if (overlap(k_old, kv_old_bytes, k_new, kv_new_bytes) || overlap(v_old, kv_old_bytes, v_new, kv_new_bytes) ||
        overlap(k_new, kv_new_bytes, v_new, kv_new_bytes) || overlap(k_old, kv_old_bytes, v_new, kv_new_bytes) ||
        overlap(v_old, kv_old_bytes, k_new, kv_new_bytes))
      return fail(PISA_ERR_INVALID_ARG, "old and new key/value buffers overlap");
  }
  // 16-byte units: a summary row is D floats (16 or 32 units), a key row D
  // elements of esz bytes (8/16 units in bf16, 16/32 in fp32)
  const int64_t pu = s.D / 4, ku = s.D * static_cast<int64_t>(esz) / 16;
  pisa::GrowArgs a{};
  int64_t end = 0;
  for (int l = 1; l <= g.Lstore; ++l) {
    end += static_cast<int64_t>(g.M[l]) * pu;
    a.lev_end[l - 1] = end;
    a.off_old[l - 1] = g.off[l] * pu;
    a.off_new[l - 1] = gn.off[l] * pu;
  }
  a.pyr_units = end;
  a.kv_units = kv ? static_cast<int64_t>(s.N) * ku : 0;
  a.pyr_old_stride = g.R * pu;
  a.pyr_new_stride = gn.R * pu;
  a.kv_old_stride = static_cast<int64_t>(g.Nkv) * ku;
  a.kv_new_stride = static_cast<int64_t>(gn.Nkv) * ku;
  return device_status(pisa::launch_cache_grow(a, static_cast<int>(BH), pyr_old, pyr_new, k_old, k_new, v_old, v_new,
                                               static_cast<hipStream_t>(stream)),
                       "pisa_cache_grow");
}

int pisa_select(const pisa_problem* p, const void* q, const void* k, const float* pyramid, int32_t* block_idx,
                float* block_score, void* ws, size_t ws_bytes, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  int sched = 0;
  PISA_TRY(check_select(p, q, k, pyramid, block_idx, block_score, &s, &g, &sched));
  PISA_TRY(check_ws(ws, ws_bytes, select_ws(sched, s, g)));
  return run_select(s, g, sched, q, k, pyramid, block_idx, block_score, ws, static_cast<hipStream_t>(stream),
                    "pisa_select");
}

int pisa_select_static(const pisa_problem* p, const void* q, const void* k, const float* pyramid,
                       int32_t* block_idx, float* block_score, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  int sched = 0;
  PISA_TRY(check_select(p, q, k, pyramid, block_idx, block_score, &s, &g, &sched));
  const size_t need = select_ws(sched, s, g);
  if (need > PISA_STATIC_SCRATCH_BYTES)
    return fail(PISA_ERR_WORKSPACE,
                "pisa_select_static: this selection needs %zu bytes of scratch, the static scratch holds %zu "
                "(call pisa_select with a workspace instead)",
                need, static_cast<size_t>(PISA_STATIC_SCRATCH_BYTES));
  void* ws = nullptr;
  if (need > 0) PISA_TRY(static_scratch(&ws));
  return run_select(s, g, sched, q, k, pyramid, block_idx, block_score, ws, static_cast<hipStream_t>(stream),
                    "pisa_select_static");
}

int pisa_select_flat_bsa(const pisa_problem* p, const void* q, const float* pyramid, int32_t* block_idx, void* ws,
                         size_t ws_bytes, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(q, "q"));
  PISA_TRY(check_ptr(pyramid, "pyramid"));
  PISA_TRY(check_ptr(block_idx, "block_idx"));
  const bool mfma_bsa = s.bf16 && s.K <= 32;
  if (!mfma_bsa && (static_cast<int64_t>(g.M[1]) + s.K) * 4 > 65536)
    return fail(PISA_ERR_UNSUPPORTED, "flat BSA on fp32 or K > 32 keeps one score per leaf block in LDS: N/C < 16384");
  PISA_TRY(check_ws(ws, ws_bytes, pisa::bsa_ws(s, g)));
  return device_status(pisa::launch_flat_bsa(s, g, q, pyramid, block_idx, ws, static_cast<hipStream_t>(stream)),
                       "pisa_select_flat_bsa");
}

int pisa_sparse_attn_fwd(const pisa_problem* p, const void* q, const void* k, const void* v,
                         const int32_t* block_idx, void* o, float* lse, void* ws, size_t ws_bytes,
                         pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(q, "q"));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(v, "v"));
  PISA_TRY(check_ptr(block_idx, "block_idx"));
  PISA_TRY(check_ptr(o, "o"));
  PISA_TRY(check_ptr(lse, "lse", true));
  PISA_TRY(check_ws(ws, ws_bytes, pisa::attn_ws(s, g)));
  return device_status(
      pisa::launch_attention(s, g, q, k, v, block_idx, o, lse, ws, static_cast<hipStream_t>(stream)),
      "pisa_sparse_attn_fwd");
}

size_t pisa_attn_bwd_workspace_bytes(const pisa_problem* p) {
  pisa::Shape s{};
  pisa::Geo g{};
  if (check_problem(p, &s, &g) != PISA_OK || !pisa::attn_bwd_supported(s)) return 0;
  return pisa::attn_bwd_ws(s, g);
}

int pisa_sparse_attn_bwd(const pisa_problem* p, const void* q, const void* k, const void* v,
                         const int32_t* block_idx, const void* o, const float* lse, const void* d_o, void* dq,
                         void* dk, void* dv, void* ws, size_t ws_bytes, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(q, "q"));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(v, "v"));
  PISA_TRY(check_ptr(block_idx, "block_idx"));
  PISA_TRY(check_ptr(o, "o"));
  PISA_TRY(check_ptr(lse, "lse"));
  PISA_TRY(check_ptr(d_o, "d_o"));
  PISA_TRY(check_ptr(dq, "dq"));
  PISA_TRY(check_ptr(dk, "dk"));
  PISA_TRY(check_ptr(dv, "dv"));
  if (!pisa::attn_bwd_supported(s))
    return fail(PISA_ERR_UNSUPPORTED, "the attention backward runs on bf16 with d in {64,128} and C in {32,64,96,128}");
  PISA_TRY(check_ws(ws, ws_bytes, pisa::attn_bwd_ws(s, g)));
  return device_status(pisa::launch_attention_bwd(s, g, q, k, v, block_idx, o, lse, d_o, dq, dk, dv, ws,
                                                  static_cast<hipStream_t>(stream)),
                       "pisa_sparse_attn_bwd");
}

size_t pisa_quality_workspace_bytes(const pisa_problem* p, int32_t n_rows) {
  pisa::Shape s{};
  pisa::Geo g{};
  if (check_problem(p, &s, &g) != PISA_OK || n_rows < 1) return 0;
  return pisa::quality_ws(s, n_rows);
}

int pisa_selection_quality(const pisa_problem* p, const void* q, const void* k, const int32_t* block_idx,
                           const int32_t* rows, int32_t n_rows, float* metrics, int32_t* ref_idx, void* ws,
                           size_t ws_bytes, pisa_stream_t stream) {
  pisa::Shape s{};
  pisa::Geo g{};
  PISA_TRY(check_problem(p, &s, &g));
  PISA_TRY(check_ptr(q, "q"));
  PISA_TRY(check_ptr(k, "k"));
  PISA_TRY(check_ptr(block_idx, "block_idx"));
  PISA_TRY(check_ptr(rows, "rows"));
  PISA_TRY(check_ptr(metrics, "metrics"));
  PISA_TRY(check_ptr(ref_idx, "ref_idx", true));
  if (n_rows < 1 || n_rows > (1 << 24)) return fail(PISA_ERR_INVALID_ARG, "n_rows %d out of [1, 2^24]", n_rows);
  if (!pisa::quality_supported(s))
    return fail(PISA_ERR_UNSUPPORTED, "the quality diagnostic runs on bf16 with C in {32,64,96,128}, N/C <= 16384, K <= 64");
  PISA_TRY(check_ws(ws, ws_bytes, pisa::quality_ws(s, n_rows)));
  return device_status(pisa::launch_quality(s, q, k, block_idx, rows, n_rows, metrics, ref_idx, ws,
                                            static_cast<hipStream_t>(stream)),
                       "pisa_selection_quality");
}

const char* pisa_status_string(int status) {
  switch (status) {
    case PISA_OK: return "ok";
    case PISA_ERR_INVALID_ARG: return "invalid argument";
    case PISA_ERR_UNSUPPORTED: return "unsupported shape";
    case PISA_ERR_WORKSPACE: return "workspace too small";
    case PISA_ERR_DEVICE: return "device error";
    default: return "unknown status";
  }
}

const char* pisa_last_error(void) { return g_last_error; }

}  // extern "C"
