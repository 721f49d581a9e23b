/*
 * pisa.h -- C ABI of the PISA hot path for AMD Instinct MI355X (gfx950).
 *
 * PISA ("Block Sparse Attention with Log-Linear Complexity") selects, for
 * every query position, K key blocks of C tokens by a coarse-to-fine search
 * over a mean-pooled key pyramid, then runs softmax attention over the
 * original keys and values of the selected blocks.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every buffer pointer is a DEVICE pointer unless stated otherwise and must
 *   be 16-byte aligned.  The caller allocates and owns every buffer,
 *   including workspaces; the library never allocates device memory, never
 *   synchronises and never creates streams.
 * - Every compute call is asynchronous on `stream` (a hipStream_t; 0 is the
 *   legacy default stream).
 * - Indices are 0-based (the paper counts from 1).
 * - Layouts are contiguous and row-major:
 *     q, o      [B, H,   Nq, d]   (dtype of the problem)
 *     k, v      [B, Hkv, Ncap, d] (dtype of the problem; Ncap = N unless
 *               the problem reserves more rows, see pisa_problem.Ncap)
 *     pyramid   [B, Hkv, R,  d]   float32: summary levels 1 .. max(1, L-1)
 *               concatenated (level 1 = leaf blocks first), each level laid
 *               out for Ncap tokens; R and the level offsets come from
 *               pisa_pyramid_layout().  The root (level L) is never scored
 *               and is not stored.
 *     block_idx [B, Hkv, Nq, K]   int32, ascending, padded with -1
 *     lse       [B, H,   Nq]      float32, natural log
 * - Query row i sits at absolute position t = N - Nq + i (end-aligned), so
 *   Nq = N is prefill and Nq = 1 is one decode step.
 * - Query head h' reads KV head h' / (H / Hkv) (grouped-query attention);
 *   the G = H / Hkv heads of a group share one selected block set.
 * - Logits are scaled by 1/sqrt(d); scores and lse use the natural log.
 * - Errors: every call validates all arguments before anything is enqueued.
 *   On error it returns a negative status, launches nothing and leaves the
 *   outputs untouched; pisa_last_error() then describes the problem (per
 *   thread).  PISA_ERR_DEVICE means a HIP launch reported a failure.
 *
 * Supported shapes: d in {64, 128}; C a multiple of 32 in [32, 256];
 * 2 <= fanout <= 16; 1 <= K with fanout*K <= 256 (K >= 3 when causal);
 * G = H/Hkv <= 16 with fanout*fanout*K*G <= 2048; Nq <= N < 2^31,
 * Nq < 2^23; B*Hkv <= 65535.
 */
#ifndef PISA_H
#define PISA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* pisa_stream_t;

typedef enum { PISA_DTYPE_F32 = 0, PISA_DTYPE_BF16 = 1 } pisa_dtype;

enum {
  PISA_OK = 0,
  PISA_ERR_INVALID_ARG = -1, /* malformed problem, null or misaligned pointer */
  PISA_ERR_UNSUPPORTED = -2, /* well-formed but outside the supported shapes */
  PISA_ERR_WORKSPACE = -3,   /* workspace smaller than the *_workspace_bytes */
  PISA_ERR_DEVICE = -4       /* a HIP call or kernel launch failed */
};

/* Selection schedules (pisa_problem.schedule). */
enum {
  PISA_SCHEDULE_AUTO = 0,      /* library picks from the problem size */
  PISA_SCHEDULE_TWO_STAGE = 1, /* Sec. 3.3 prefill design: intermediate
                                  levels per query, then leaf blocks scored
                                  once per key block for a tile of queries,
                                  then a final Top-K (bf16 only) */
  PISA_SCHEDULE_FUSED = 2,     /* Sec. 3.3 decode design: one program per
                                  (query, KV head) walks every level down to
                                  the raw leaf keys */
  PISA_SCHEDULE_SPLIT = 3      /* few rows (decode): intermediate levels with
                                  a workgroup per (query, KV head), then each
                                  leaf candidate scored by a workgroup of its
                                  own, then the final Top-K; the same
                                  selection as the other schedules, spread
                                  over the whole GPU */
};

/* Block scores of pisa_select (pisa_problem.score): for one candidate and
 * query head with child logits z_1..z_m (child summaries above the leaf
 * level, raw keys at it), summed over the group's query heads. */
enum {
  PISA_SCORE_LSE = 0,      /* PISA, eq. direct_child_lse: log sum_j exp(z_j) */
  PISA_SCORE_MEAN = 1,     /* PISA-1, App. A: the mean of the z_j             */
  PISA_SCORE_MEAN_VAR = 2  /* PISA-2, App. A: the mean plus half the
                              population variance of the z_j                   */
};

/* The problem statement of Sec. 3.1-3.2: q/k/v, N, head dim d, block size C,
 * fan-out g (the paper fixes g = 2; any 2..16 is accepted), budget K. */
typedef struct {
  int32_t B, H, Hkv; /* batch, query heads, KV heads (H % Hkv == 0)         */
  int32_t Nq, N;     /* query rows and key rows, 1 <= Nq <= N               */
  int32_t d;         /* head dimension                                      */
  int32_t C;         /* leaf block size (tokens per leaf block)             */
  int32_t fanout;    /* g: children per node above the leaf level           */
  int32_t K;         /* block budget per (query, KV head) at every level    */
  int32_t causal;    /* 1: App. B eligibility + forced first/previous/current
                        blocks and masked future tokens; 0: plain method    */
  int32_t dtype;     /* pisa_dtype of q, k, v and o                         */
  int32_t schedule;  /* PISA_SCHEDULE_* for pisa_select; ignored elsewhere  */
  int32_t Ncap;      /* rows reserved per (batch, KV head): k and v are
                        [B,Hkv,Ncap,d] of which the first N rows are used,
                        and the pyramid is laid out for Ncap tokens, so a
                        decode loop grows N in place (App. B decode cache);
                        0 means N, otherwise N <= Ncap                       */
  int32_t score;     /* PISA_SCORE_* reducer of pisa_select (ignored by flat
                        BSA and everywhere else)                            */
} pisa_problem;

/* Number of hierarchy levels L (Sec. 3.2 eq. key_hierarchy: M_1 = ceil(N/C),
 * M_{l+1} = ceil(M_l / fanout) until M_L = 1), or a negative status. */
int pisa_num_levels(int32_t N, int32_t C, int32_t fanout);

/* Row layout of the stored pyramid.  Writes level_row_offset[l-1] = first row
 * of level l for l = 1..L (host array with room for L entries; the root's
 * entry equals R) and *rows_R = R.  Returns L or a negative status. */
int pisa_pyramid_layout(const pisa_problem* p, int64_t* level_row_offset, int64_t* rows_R);

/* Bytes of the pyramid buffer (B*Hkv*R*d*4), or 0 if the problem is invalid. */
size_t pisa_pyramid_bytes(const pisa_problem* p);

/* Workspace bytes each call needs (0 is a valid answer); 0 also for invalid
 * problems, which the call itself then rejects. */
size_t pisa_select_workspace_bytes(const pisa_problem* p);
size_t pisa_bsa_workspace_bytes(const pisa_problem* p);
size_t pisa_attn_workspace_bytes(const pisa_problem* p);

/* Mean pyramid (Sec. 3.2 eq. mean_pyramid): level 1 = mean of each leaf
 * block's raw keys (the last block may be short), level l+1 = mean of the
 * existing children at level l.  Accumulates in float32; writes `pyramid`. */
int pisa_build_pyramid(const pisa_problem* p, const void* k, float* pyramid, pisa_stream_t stream);

/* Decode cache update (App. B "decode cache": each new token updates the
 * mean of its leaf block and of that block's ancestors).  `pyramid` holds
 * the pyramid of the first n_old keys, as left by pisa_build_pyramid or an
 * earlier append with the same C, fanout and Ncap; k holds the first p->N
 * keys.  The leaf blocks containing rows [n_old, N) and all of their
 * ancestors are recomputed, and levels that did not exist at n_old are
 * computed whole, with the arithmetic of pisa_build_pyramid: the result
 * equals a full build at N bit for bit.  0 <= n_old <= N (n_old = 0 rebuilds
 * every block, on one workgroup per (batch, KV head)); one launch, no
 * workspace. */
int pisa_pyramid_append(const pisa_problem* p, const void* k, float* pyramid, int32_t n_old,
                        pisa_stream_t stream);

/* Capacity rule of the decode cache (App. B "Decode cache": when the cache
 * needs room, each level's capacity grows by a fixed fraction, so a level is
 * re-laid a constant number of times per doubling of the length and the
 * copying through length N stays within O((N/C) d log N) per KV head).
 * Returns the capacity (in tokens) for a cache that reserves `cap` tokens and
 * must hold `need`: cap when need <= cap, otherwise the smallest multiple of
 * C that is >= need and >= cap + cap/2 (the fraction is 1/2), clamped to the
 * largest supported capacity (65535 leaf blocks); a negative status if need
 * itself exceeds it or an argument is invalid (cap >= 0, need >= 1, C >= 1).
 * Host only. */
int32_t pisa_cache_capacity(int32_t cap, int32_t need, int32_t C);

/* Decode cache growth (App. B "Decode cache"): re-lays a cache of p->N tokens
 * held in buffers reserved for p->Ncap tokens (0 means N) into caller-
 * allocated buffers reserved for new_cap >= max(N, Ncap) tokens.  Per (batch,
 * KV head), the rows of every stored level of pyr_old (the layout of
 * pisa_pyramid_layout for Ncap) move to that level's offset in pyr_new (the
 * layout for new_cap), and, when the four key/value pointers are non-NULL,
 * the first N rows of k_old, v_old [B,Hkv,Ncap,d] go to k_new, v_new
 * [B,Hkv,new_cap,d].  Afterwards pyr_new equals pisa_build_pyramid of the
 * problem with Ncap = new_cap bit for bit, and pisa_pyramid_append continues
 * from it with that Ncap.  Rows past N in the new buffers are not written.
 * The key/value pointers are all NULL (pyramid only) or all non-NULL; old and
 * new buffers must not overlap (PISA_ERR_INVALID_ARG otherwise).  One launch,
 * no workspace, no allocation. */
int pisa_cache_grow(const pisa_problem* p, int32_t new_cap, const float* pyr_old, float* pyr_new, const void* k_old,
                    void* k_new, const void* v_old, void* v_new, pisa_stream_t stream);

/* Pyramid Top-K selection (Sec. 3.2 eqs. hierarchical_topk and
 * direct_child_lse; grouped heads Sec. 3.3 eq. kernel_grouped_score; causal
 * policy App. B).  From the root, each level keeps all candidates when there
 * are at most K, otherwise keeps the forced ones plus the best by the sum over
 * the group's heads of the LSE of the children's scaled logits (child
 * summaries above the leaf level, raw keys at the leaf level); kept blocks
 * expand to their eligible children.  Ties go to the smaller block index.
 * Writes block_idx.  block_score (nullable, float32 [B,Hkv,Nq,K]) receives the
 * leaf score of each kept block, +inf for blocks kept without a score, -inf
 * for padding.  `pyramid` must come from pisa_build_pyramid on the same k. */
int pisa_select(const pisa_problem* p, const void* q, const void* k, const float* pyramid,
                int32_t* block_idx, float* block_score, void* ws, size_t ws_bytes,
                pisa_stream_t stream);

/* Bytes of the static scratch that pisa_select_static uses instead of a
 * caller workspace (one copy per device, held while the library is loaded). */
#define PISA_STATIC_SCRATCH_BYTES (32u << 20)

/* pisa_select without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that must not
 * call hipMalloc, harnesses that forbid it).  Same arguments, validation,
 * kernels and results as pisa_select; the scratch it needs comes from a
 * static device array of PISA_STATIC_SCRATCH_BYTES bytes instead of `ws`.
 * A problem whose pisa_select_workspace_bytes() exceeds that size is refused
 * with PISA_ERR_WORKSPACE (nothing is launched; use pisa_select).  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine);
 * its first call on a device looks up that device's copy of the array.
 * Every call on a device shares that device's one array, so calls that
 * overlap on one device (concurrent streams, or host threads) race and give
 * undefined results: serialise them.  The array keeps the last call's
 * contents; every call writes what it reads. */
int pisa_select_static(const pisa_problem* p, const void* q, const void* k, const float* pyramid,
                       int32_t* block_idx, float* block_score, pisa_stream_t stream);

/* Flat block selection baseline (Sec. 3.1 eqs. bsa_block_scores, bsa_topk):
 * every eligible leaf summary (pyramid level 1) is scored; with G > 1 the
 * scores are turned into per-head softmax probabilities over the eligible
 * non-forced blocks and summed over the group (App. C.1); the forced blocks
 * of App. B are kept inside the budget.  Same block_idx layout as
 * pisa_select. */
int pisa_select_flat_bsa(const pisa_problem* p, const void* q, const float* pyramid,
                         int32_t* block_idx, void* ws, size_t ws_bytes, pisa_stream_t stream);

/* Selected sparse attention (Sec. 3.1 eq. selected_sparse_attention): for
 * every query row and head, softmax over the tokens of its KV head's selected
 * blocks (future tokens masked when causal, App. B) applied to the original
 * values.  block_idx entries outside [0, ceil(N/C)) -- negative ones and
 * ones past the last leaf block -- are padding and contribute nothing; in
 * causal mode a block that starts after the query contributes nothing either
 * (all of its tokens are masked).  The entries of a row need not be sorted
 * but must be distinct (pisa_select writes them so): a block listed twice is
 * attended once or twice depending on the kernel that takes the row (the
 * row-tile kernels, and a row's first, previous and own blocks, count it
 * once).  Writes o (problem dtype) and lse (nullable); a row with no visible
 * token gets o = 0 and lse = -inf. */
int pisa_sparse_attn_fwd(const pisa_problem* p, const void* q, const void* k, const void* v,
                         const int32_t* block_idx, void* o, float* lse, void* ws,
                         size_t ws_bytes, pisa_stream_t stream);

/* Tuning of pisa_sparse_attn_fwd's row-tile path (same results either way, up
 * to fp32 rounding order).  A row tile is 256/G consecutive query rows of one
 * (batch, KV head); when the blocks its rows select number at most
 * min(3K, 256), the whole tile can be attended by one workgroup that walks
 * those blocks once, instead of by the block-centric kernels.  That path is
 * taken, on calls with G in {1, 2, 4, 8, 16}, only when at least n tiles of
 * the call qualify (so that it fills the device); n < 0 turns it off.
 * Process-wide, read at each call's launch; default 1024.  Returns the
 * previous value.  Host only: no device work. */
int pisa_attn_union_min_tiles(int32_t n);

/* Backward of the selected sparse attention with the block indices held
 * fixed (App. B: during backpropagation gradients flow through the attention
 * over the selected entries, not through the selection).  For every row and
 * query head, with z = q.k / sqrt(d) over the selected visible tokens,
 * p = exp(z - lse) and D = d_o . o:
 *   dv_j += p_j d_o,  ds_j = p_j (d_o . v_j - D),  dq = sum_j ds_j k_j / sqrt(d),
 *   dk_j += ds_j q / sqrt(d)
 * (dk, dv summed over every row and query head that reaches token j).
 * o and lse are the forward's outputs (pisa_sparse_attn_fwd on the same
 * block_idx); d_o has o's layout.  Writes dq [B,H,Nq,d] and dk, dv in k's
 * layout [B,Hkv,N,d] (row stride Ncap; every stored row is written, rows no
 * query reaches get 0), all in the problem dtype; sums run in fp32.  bf16
 * with d in {64,128} and C in {32,64,96,128}, else PISA_ERR_UNSUPPORTED.
 * Workspace: pisa_attn_bwd_workspace_bytes(p). */
size_t pisa_attn_bwd_workspace_bytes(const pisa_problem* p);
int pisa_sparse_attn_bwd(const pisa_problem* p, const void* q, const void* k, const void* v,
                         const int32_t* block_idx, const void* o, const float* lse, const void* d_o, void* dq,
                         void* dk, void* dv, void* ws, size_t ws_bytes, pisa_stream_t stream);

/* Block-selection quality diagnostic (Sec. 4 "Block-selection quality", eq.
 * oracle_metrics; App. C "Block-selection diagnostic", eq. oracle_block_mass).
 * For each (batch, KV head) and each listed query row: the full attention's
 * log mass of every eligible leaf block, a(B) = log of the sum over B's
 * tokens (future ones masked when causal) of exp(q.k / sqrt(d)), per query
 * head; P(B) = mean over the KV head's query heads of each head's softmax of
 * a over the eligible blocks.  The reference set holds the forced blocks of
 * App. B (causal) and the eligible blocks of highest P up to K (ties to the
 * smaller index); with at most K eligible blocks it is all of them.  For the
 * selection in block_idx:
 *   metrics[..., 0] = |selection & reference| / K         (Recall@K)
 *   metrics[..., 1] = sum of P over the selection          (captured mass)
 *   metrics[..., 2] = metrics[..., 1] / sum of P over the reference
 *                                                          (attention mass ratio)
 * rows: device int32 [n_rows], query-row indices; a row outside [0, Nq)
 * gets NaN metrics and an empty reference.  block_idx: [B,Hkv,Nq,K] as
 * pisa_select writes it (negative entries are padding; repeats count once).
 * metrics: device float32 [B,Hkv,n_rows,3]; ref_idx: nullable device int32
 * [B,Hkv,n_rows,K], the reference set ascending, -1 padded.  The work is dense
 * over every visible key of every listed row (n_rows x N x d per head): meant
 * for sampled rows.  bf16 inputs, C in {32, 64, 96, 128}, N/C <= 16384, K <= 64;
 * otherwise PISA_ERR_UNSUPPORTED.  Workspace: pisa_quality_workspace_bytes(p,
 * n_rows) bytes (the log masses, B*Hkv*n_rows*G*ceil(N/C) floats). */
size_t pisa_quality_workspace_bytes(const pisa_problem* p, int32_t n_rows);
int pisa_selection_quality(const pisa_problem* p, const void* q, const void* k, const int32_t* block_idx,
                           const int32_t* rows, int32_t n_rows, float* metrics, int32_t* ref_idx, void* ws,
                           size_t ws_bytes, pisa_stream_t stream);

/* Per-kernel timing for benchmarks (not needed for computing anything).
 * pisa_profile_enable(1) makes every later call bracket each kernel it
 * launches with two hipEvents recorded on that call's stream (host-side
 * bookkeeping only; no device memory).  pisa_profile_report() waits for the
 * recorded events, writes one line "kernel_name launches total_ms" per kernel
 * into buf (host, NUL-terminated, truncated to cap) and clears the totals; it
 * returns the untruncated text length. */
int pisa_profile_enable(int on);
int pisa_profile_report(char* buf, size_t cap);

/* Static text for a status code. */
const char* pisa_status_string(int status);

/* Detail of the last failing call on this thread ("" if none). */
const char* pisa_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PISA_H */
