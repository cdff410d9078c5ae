/*
 * refcache.h -- C ABI of librefcache: block-masked multi-head attention for
 * exact reference caching in in-context diffusion transformers
 * (arXiv 2608.21229, "Anchoring Instruction Outside Mask").
 *
 * The sequence is a list of segments in order (Sec. 3.1, Eq. 1; Sec. 3.3):
 *   ST  static text anchors   (kind RC_SEG_ANCHOR)
 *   LT  live text             (kind RC_SEG_TEXT)
 *   X   denoising target      (kind RC_SEG_TARGET)
 *   R^k reference k           (kind RC_SEG_REF)
 * ST and R are the static subgraph: fixed for a whole request.  LT and X are
 * live: their Q/K/V change at every denoising step.
 *
 * Three entry points (App. C, derivation paragraph):
 *   rc_ref_kv_prefill         once per request and layer: the static rows
 *                             attend within the static subgraph, and the K/V
 *                             of every static segment that a live query reads
 *                             are written to the reference K/V cache (Eq. 2).
 *   rc_step_masked_attention  every denoising step: the live rows attend to
 *                             fresh LT/X K/V plus the cached K/V.
 *   rc_full_attention         the recompute baseline: all rows over the whole
 *                             sequence under any mask (dense over [LT,X,R] is
 *                             the paper's full-attention Base).
 * The prefill and step also exist over a cache stored as e4m3 codes
 * (rc_ref_kv_prefill_fp8, rc_step_masked_attention_fp8), and rc_linear is the
 * dense projection of the chained synthetic layer built around them.
 *
 * Common conventions
 *   Element type   bf16 for Q, K, V, O and the cache (passed as raw bits;
 *                  the FP8 entries store the cache as e4m3 codes with fp32
 *                  scales); fp32 for LSE and workspace.  Arithmetic: bf16 products,
 *                  fp32 accumulation and softmax, O rounded to bf16 (RNE).
 *   Token layout   Q/K/V are [B, N, H, D] with D contiguous and head stride D;
 *                  `tok_stride` (elements, >= H*D, multiple of 8, <= 2^24) separates
 *                  consecutive tokens so views into a fused QKV buffer work;
 *                  batch stride is N * tok_stride.  O is contiguous
 *                  [B, N, H, D].  LSE is contiguous [B, H, N] (natural log).
 *   Cache layout   [B, H, N_cached, D] contiguous, one buffer for K and one
 *                  for V; rows are the cached segments in sequence order.
 *   Pointers       device pointers, 16-byte aligned; `stream` is a
 *                  hipStream_t passed as void* (NULL = default stream).
 *   Ownership      the caller allocates every buffer; the library allocates
 *                  nothing and keeps no device state.  An rc_layout is read
 *                  only during the call.
 *   Asynchrony     calls enqueue kernels on `stream` and return without
 *                  synchronising.  Results are deterministic: fixed
 *                  reduction order; the only atomic (the FP8 cache's
 *                  per-head maximum) is order-independent.
 *   Errors         every function validates all arguments before any HIP
 *                  call and returns an rc_status; on error nothing is
 *                  launched and rc_last_error() (thread-local) describes it.
 *   head_dim       D in {64, 128}.
 */
#ifndef REFCACHE_H
#define REFCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RC_MAX_SEGMENTS 32

/* `splits` value of rc_step_masked_attention for the balanced schedule: one
 * round of 256 work-groups (one per CU), each taking an equal contiguous share
 * of all (query tile, key tile) work; query tiles cut between work-groups are
 * merged from fp32 partials in work-group order.  Needs a workspace of
 * 2 * 256 * 256 * (D + 2) * 4 bytes whatever the problem size. */
#define RC_SPLITS_BALANCED (-1)

/* `splits` value of rc_step_masked_attention for the tail split: two key
 * splits per query tile, a long one (the first f of its key tiles) and a short
 * one (the rest).  The long pieces are dispatched first, one work-group per
 * CU; the short ones run on the CUs the query tiles leave free, several in
 * turn, so that both finish together: with Q query tiles (Q < 256) every CU
 * but Q runs R = ceil(Q / (256 - Q)) short pieces and f = R / (R + 1).  The
 * two partials of each row are merged in split order.  Workspace as for
 * splits = 2.  rc_step_auto_splits returns it when the query tiles alone
 * fill more than half the CUs and R <= 3 (Q <= 192). */
#define RC_SPLITS_TAIL (-2)

/* `splits` value of rc_step_masked_attention for the last-round split: when
 * the query tiles (one work-group each) outnumber the 256 CUs and the last
 * round of T tiles leaves 256 - T of them idle, those T tiles run as a long
 * and a short piece of their keys as in RC_SPLITS_TAIL (R = ceil(T / (256 -
 * T)) <= 3 rounds of short pieces on the idle CUs; every split tile has at
 * least 16 key tiles), and the other tiles run whole, written directly.
 * Workspace 2 * T * 512 * (D + 2) * 4 bytes (rc_step_workspace_bytes); where
 * it does not apply the step runs unsplit and needs none.
 * rc_step_auto_splits returns it for such grids. */
#define RC_SPLITS_LAST_ROUND (-3)

typedef enum {
  RC_OK = 0,
  RC_ERR_ARG = -1,                 /* null/misaligned pointer, bad size or stride */
  RC_ERR_UNSUPPORTED = -2,         /* head_dim not 64/128, schedule too fragmented */
  RC_ERR_MASK_NOT_CACHEABLE = -3,  /* a static query reads a live segment */
  RC_ERR_WORKSPACE = -4,           /* split-KV workspace missing or too small */
  RC_ERR_HIP = -5                  /* a HIP launch failed */
} rc_status;

typedef enum {
  RC_SEG_ANCHOR = 0,  /* ST: static text anchors, timestep fixed at 0 (Sec. 3.3) */
  RC_SEG_TEXT = 1,    /* LT: live text (Sec. 3.1) */
  RC_SEG_TARGET = 2,  /* X_t: denoising target (Sec. 3.1) */
  RC_SEG_REF = 3      /* R^(k): one reference image's tokens (Sec. 3.1, Eq. 1) */
} rc_seg_kind;

typedef enum {
  /* Sec. 3.3: ST <-> R see each other (all references form one R block);
   * neither reads LT or X; LT and X read LT, X and R but not ST. */
  RC_MASK_PAPER = 0,
  /* Per-reference anchored mask of the synthetic workloads: R^(k) reads
   * ST and itself, ST reads ST, LT and X read every segment. */
  RC_MASK_PERREF = 1,
  /* Prior-work isolated cache (Sec. 1, Sec. 2): R reads R, LT and X read
   * LT, X, R; anchor segments are detached (no keys, read by nobody). */
  RC_MASK_ISOLATED = 2,
  /* Full attention: every segment reads every segment (App. C Base). */
  RC_MASK_DENSE = 3
} rc_mask_preset;

typedef enum { RC_ENTRY_PREFILL = 0, RC_ENTRY_STEP = 1, RC_ENTRY_FULL = 2 } rc_entry;

typedef enum {
  RC_ROWS_STATIC = 0,  /* tokens of ST and R segments */
  RC_ROWS_LIVE = 1,    /* tokens of LT and X segments */
  RC_ROWS_CACHED = 2,  /* tokens of the cached segments */
  RC_ROWS_ALL = 3      /* all tokens */
} rc_rows_kind;

typedef struct {
  int32_t kind;  /* rc_seg_kind */
  int32_t len;   /* tokens, >= 1 */
} rc_segment;

/* Segment table + segment-level block mask.  visible[q] bit k set means the
 * tokens of query segment q attend to the tokens of key segment k (query
 * first; App. A writes the transpose, M[b',b] = 1 for "b attends b'"). */
typedef struct {
  int32_t n_seg;
  rc_segment seg[RC_MAX_SEGMENTS];
  uint32_t visible[RC_MAX_SEGMENTS];
} rc_layout;

/* Fill L->visible from the segment kinds for one rc_mask_preset.  n_seg and
 * seg[] must already be set.  RC_ERR_ARG on a bad table or preset. */
rc_status rc_layout_preset(rc_layout* L, int32_t preset);

/* Check a layout for one entry (rc_entry): 1 <= n_seg <= 32, every len >= 1,
 * known kinds, no visible bit beyond n_seg; for PREFILL and STEP also the
 * caching condition (no static query segment reads LT or X; App. A,
 * StructCacheable for a layer-shared mask) -> RC_ERR_MASK_NOT_CACHEABLE. */
rc_status rc_layout_validate(const rc_layout* L, int32_t entry);

/* Visible query-key pairs per (batch, head) for the rows of `entry`
 * (App. C: one unit per query-key interaction).  Useful FLOPs of a call are
 * 4 * D * H * B * pairs.  Returns < 0 (an rc_status) on an invalid layout. */
int64_t rc_pairs(const rc_layout* L, int32_t entry);

/* Token count of a row class (rc_rows_kind); < 0 on an invalid layout. */
int64_t rc_rows(const rc_layout* L, int32_t which);

/* Bytes of fp32 workspace rc_step_masked_attention needs for `splits`
 * key splits (0 when splits == 1): splits * B * H * N_live * (D + 2) * 4,
 * two splits' worth for RC_SPLITS_TAIL, the last round's pieces for
 * RC_SPLITS_LAST_ROUND (above), and the fixed size given above for
 * RC_SPLITS_BALANCED.  splits = 0 resolves the automatic choice first.
 * 0 on invalid input. */
size_t rc_step_workspace_bytes(const rc_layout* L, int32_t B, int32_t H, int32_t D, int32_t splits);

/* The split count rc_step_masked_attention uses when passed splits = 0:
 * RC_SPLITS_LAST_ROUND when the query tiles outnumber the 256 CUs and that
 * split applies, 1 when they fill more than 192 CUs otherwise,
 * RC_SPLITS_TAIL when they fill more than half, otherwise as many even splits
 * as keep one round of work-groups (at most one per 8 key tiles and 32 in
 * all). */
int32_t rc_step_auto_splits(const rc_layout* L, int32_t B, int32_t H, int32_t D);

/* Launch shape of the step's attention kernel for `splits` (0 = automatic)
 * with the bf16 cache (fp8 = 0) or the FP8 cache (fp8 = 1), for occupancy
 * reports: *work_groups over all its launches (one per query tile and split;
 * the whole tiles plus two per split tile for RC_SPLITS_LAST_ROUND; 256 for
 * RC_SPLITS_BALANCED), *rows_per_wg the query rows per work-group,
 * *splits_used the split count it resolves to (2 for the tail split,
 * RC_SPLITS_LAST_ROUND when that split applies and 1 when it does not,
 * RC_SPLITS_BALANCED for the balanced schedule).
 * Host only; RC_ERR_ARG on bad arguments or null outputs, RC_ERR_UNSUPPORTED
 * for head_dim other than 64/128 and for the balanced schedule with the FP8
 * cache. */
rc_status rc_step_launch_shape(const rc_layout* L, int32_t B, int32_t H, int32_t D, int32_t splits, int32_t fp8,
                               int64_t* work_groups, int32_t* rows_per_wg, int32_t* splits_used);

/* Launch plan of rc_ref_kv_prefill (bf16 cache), for reports and tests:
 * *attn_wgs attention work-groups over all launches (one per query tile),
 * *copy_wgs copy work-groups appended to the (last) attention launch, and
 * *copy_rows the flat cache rows (b, h, row) [0, *copy_rows) that they
 * copy; the store kernel copies the other B * H * N_cached - *copy_rows rows
 * after the attention.  The copy work-groups run on the CUs that the
 * attention grid leaves free before it ends (its partial last round, and
 * CUs whose work-groups end early), and take as many rows as a dispatch
 * model of the grid says fit there.  Host only; RC_ERR_ARG on
 * bad arguments or null outputs, RC_ERR_MASK_NOT_CACHEABLE as the
 * prefill. */
rc_status rc_prefill_launch_plan(const rc_layout* L, int32_t B, int32_t H, int32_t D, int64_t* attn_wgs,
                                 int32_t* copy_wgs, int64_t* copy_rows);

/* Static-subgraph prefill (Sec. 3.3; App. C, Eq. cost-pre).
 *   q_static, k_static, v_static  [B, N_static, H, D]: the ST and R tokens in
 *                                 sequence order (RC_ROWS_STATIC rows).
 *   o_static                      [B, N_static, H, D] out, every static row
 *                                 (anchor rows included: later layers of the
 *                                 prefill read them; the caller drops them).
 *   lse_static                    [B, H, N_static] fp32 out, nullable.
 *   k_cache, v_cache              [B, H, N_cached, D] out: bit copies of the
 *                                 K/V rows of the cached segments (Eq. 2).
 * Rows with no visible key get O = 0 and LSE = -inf. */
rc_status rc_ref_kv_prefill(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                            const void* q_static, const void* k_static, const void* v_static,
                            int64_t tok_stride, void* o_static, float* lse_static,
                            void* k_cache, void* v_cache, void* stream);

/* Per-denoising-step masked attention (App. C, Eq. cost-step).
 *   q_live, k_live, v_live  [B, N_live, H, D]: LT and X tokens in sequence order.
 *   k_cache, v_cache        [B, H, N_cached, D] as written by rc_ref_kv_prefill.
 *   o_live                  [B, N_live, H, D] out;  lse_live [B, H, N_live] fp32, nullable.
 *   splits                  key splits per query tile (split-KV); 0 = automatic,
 *                           1 = none, 2..32 even splits, RC_SPLITS_TAIL,
 *                           RC_SPLITS_BALANCED, RC_SPLITS_LAST_ROUND.  Any
 *                           choice with a nonzero rc_step_workspace_bytes needs
 *                           `workspace` (device, 16-byte aligned) of
 *                           rc_step_workspace_bytes bytes; partials are merged
 *                           in a fixed order. */
rc_status rc_step_masked_attention(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                   const void* q_live, const void* k_live, const void* v_live,
                                   int64_t tok_stride, const void* k_cache, const void* v_cache,
                                   void* o_live, float* lse_live, int32_t splits,
                                   void* workspace, size_t ws_bytes, void* stream);

/* Full-recompute baseline: every row of the sequence under L's mask.
 *   q, k, v [B, N, H, D] with N = all tokens;  o [B, N, H, D];  lse [B, H, N] nullable. */
rc_status rc_full_attention(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                            const void* q, const void* k, const void* v, int64_t tok_stride,
                            void* o, float* lse, void* stream);

/* The same recompute (App. C's Base when L is dense over [LT, X, R]) with a
 * workspace for the last-round split: when the grid of whole query tiles
 * (one work-group each) fills more than the 256 CUs and its partial last
 * round leaves enough of them idle, that round's T query tiles run as a long
 * piece and a short piece of their keys each, and a merge kernel combines
 * the two pieces' fp32 partials in a fixed order (the other tiles are
 * computed whole, as rc_full_attention computes them).
 *   workspace  device, 16-byte aligned, rc_full_workspace_bytes bytes, or
 *              NULL: then the call is rc_full_attention.
 * RC_ERR_WORKSPACE when a non-null workspace is misaligned or smaller than
 * that size; other errors as rc_full_attention. */
rc_status rc_full_attention_ws(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                               const void* q, const void* k, const void* v, int64_t tok_stride,
                               void* o, float* lse, void* workspace, size_t ws_bytes, void* stream);

/* Bytes of workspace rc_full_attention_ws uses: 2 * T * 512 * (D + 2) * 4 for
 * the T query tiles of the partial last round it splits, 0 when it splits
 * none (the grid fits one round or fills whole rounds, the idle CUs would
 * run more than three rounds of short pieces, or a tile has fewer than 16 key
 * tiles).  0 on invalid input. */
size_t rc_full_workspace_bytes(const rc_layout* L, int32_t B, int32_t H, int32_t D);

/* FP8 reference cache (the paper calls caching complementary to other
 * accelerations, Sec. 1 and Sec. 4.2; storing the cache in e4m3 halves its bytes,
 * its residency and the step's cached-key traffic).
 *   k_cache8, v_cache8  [B, H, N_cached, D] e4m3fn codes (bytes), the rows of the
 *              bf16 cache in the same order.
 *   kv_scale   [B, H, 2] fp32: the scales s_K, s_V of each (batch, head).
 * Quantisation, per (b, h) and tensor X in {K, V} over the cached rows:
 *   amax = max |x|;  s = 2^e with e the smallest integer such that amax / s <= 448
 *   (s = 1 when amax = 0);  code = e4m3fn(x / s), round to nearest even (x / s is
 *   exact);  the step reads code * s, exact in bf16.
 * rc_ref_kv_prefill_fp8 computes the same static-row attention as
 * rc_ref_kv_prefill (o_static, lse_static) and writes the FP8 cache instead of the
 * bf16 one.  rc_step_masked_attention_fp8 is rc_step_masked_attention with the
 * cached K/V read from the FP8 cache (fresh LT/X K/V stay bf16); splits and
 * workspace as there, except that RC_SPLITS_BALANCED is not supported
 * (RC_ERR_UNSUPPORTED).  N_cached at most 16 776 960 (65 535 x 256).  Cache pointers
 * 16-byte aligned; kv_scale 4-byte aligned (written by the prefill, read by the
 * step).  Errors as the bf16 entries. */
rc_status rc_ref_kv_prefill_fp8(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                const void* q_static, const void* k_static, const void* v_static,
                                int64_t tok_stride, void* o_static, float* lse_static, void* k_cache8,
                                void* v_cache8, float* kv_scale, void* stream);
rc_status rc_step_masked_attention_fp8(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                       const void* q_live, const void* k_live, const void* v_live,
                                       int64_t tok_stride, const void* k_cache8, const void* v_cache8,
                                       const float* kv_scale, void* o_live, float* lse_live, int32_t splits,
                                       void* workspace, size_t ws_bytes, void* stream);

/* Dense bf16 projection of the chained synthetic layer (Sec. 3.1, Eq. 2:
 * per layer K = h W_K, V = h W_V, and the output projection plus residual
 * that feeds the next layer):
 *   out[m, n] = bf16( sum_k a[m, k] * w[n, k]  (+ r[m, n]) )
 * fp32 accumulation in a fixed order, one RNE rounding.  Each output row
 * depends only on its own input row: a row's result is the same whatever M
 * is, so projecting the live rows alone reproduces the rows of a projection of
 * the whole sequence bit for bit.
 *   a    [M, K] bf16, row stride lda (elements)      w [N, K] bf16, contiguous
 *   r    [M, N] bf16, row stride ldr, nullable        out [M, N] bf16, row stride ldo
 * Requirements: N a multiple of 128, K a multiple of 64, K <= 2^22; lda >= K,
 * ldr >= N, ldo >= N, all multiples of 8 and <= 2^22; pointers 16-byte
 * aligned; 0 <= M <= 2^40.  `out` may not overlap `a` or `w` (it may be `r`).  M = 0 is a no-op.
 * RC_ERR_UNSUPPORTED for N or K off those multiples, RC_ERR_ARG otherwise. */
rc_status rc_linear(int64_t M, int32_t N, int32_t K, const void* a, int64_t lda, const void* w,
                    const void* r, int64_t ldr, void* out, int64_t ldo, void* stream);

/* Bytes of the static device array (per GPU) behind
 * rc_step_masked_attention_noalloc: 128 MiB, enough for the balanced schedule
 * at D = 128 (65 MiB) and for two splits over 24 heads x 4608 live rows. */
#define RC_NOALLOC_SCRATCH_BYTES (128u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * rc_step_masked_attention with its split partials in a static device array
 * of RC_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on,
 * from that GPU's first call until the process ends.  Allocates nothing and
 * calls no allocating routine.  Arguments, layouts and results as for
 * rc_step_masked_attention, on the current device; the caller still owns and
 * passes the inputs and outputs.  A split choice whose workspace
 * (rc_step_workspace_bytes) exceeds RC_NOALLOC_SCRATCH_BYTES returns
 * RC_ERR_WORKSPACE.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (several streams or host threads) race, so
 * serialise them.  The array's earlier contents never matter (every partial
 * a merge reads is written by the same call). */
rc_status rc_step_masked_attention_noalloc(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                           const void* q_live, const void* k_live, const void* v_live,
                                           int64_t tok_stride, const void* k_cache, const void* v_cache,
                                           void* o_live, float* lse_live, int32_t splits, void* stream);

/* Static description of a status code. */
const char* rc_status_string(rc_status s);

/* Message for the last error on the calling thread ("" if none). */
const char* rc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* REFCACHE_H */
