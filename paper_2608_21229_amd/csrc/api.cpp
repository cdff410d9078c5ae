// extern "C" entry points of librefcache: argument validation, planning and
// kernel launches.  Every check runs before the first HIP call, so a failing
// call launches nothing and needs no GPU.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "rc_internal.h"

namespace rc {
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

rc_status check_dims(int32_t B, int32_t H, int32_t D, float scale) {
  if (B < 1 || H < 1 || B > 65535 || H > 65535) {
    set_error("B = %d, H = %d: each must be in [1, 65535]", B, H);
    return RC_ERR_ARG;
  }
  if (D != 64 && D != 128) {
    set_error("head_dim %d is not supported (64 or 128)", D);
    return RC_ERR_UNSUPPORTED;
  }
  if (!(scale > 0.f) || !isfinite(scale)) {
    set_error("softmax scale must be finite and > 0 (got %g)", (double)scale);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_ptr(const void* p, const char* name) {
  if (!p) {
    set_error("%s is null", name);
    return RC_ERR_ARG;
  }
  if (!aligned16(p)) {
    set_error("%s is not 16-byte aligned", name);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_lse(const float* p, const char* name) {
  if (p && (reinterpret_cast<uintptr_t>(p) & 3u)) {
    set_error("%s is not 4-byte aligned", name);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_stride(int64_t tok_stride, int32_t H, int32_t D) {
  if (tok_stride < int64_t(H) * D || (tok_stride & 7)) {
    set_error("tok_stride %lld must be >= H*D = %d and a multiple of 8", (long long)tok_stride, H * D);
    return RC_ERR_ARG;
  }
  // a 64-token tile of the source spans 128 * tok_stride bytes, addressed
  // with 32-bit buffer offsets
  if (tok_stride > (int64_t(1) << 24)) {
    set_error("tok_stride %lld is too large (at most 2^24 elements)", (long long)tok_stride);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_blocks(int64_t blocks, const char* what) {
  if (blocks >= (int64_t(1) << 31)) {
    set_error("%s launch of %lld work-groups exceeds the grid limit", what, (long long)blocks);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_grid(const Params& p) {
  return check_blocks(int64_t(p.B) * p.H * p.n_qtiles * p.splits, "attention");
}

#define RC_TRY(x)                  \
  do {                             \
    rc_status _s = (x);            \
    if (_s != RC_OK) return _s;    \
  } while (0)

rc_status hip_status(int err, const char* what) {
  if (err != 0) {
    set_error("%s: HIP error %d", what, err);
    return RC_ERR_HIP;
  }
  return RC_OK;
}

size_t balanced_workspace_bytes(int32_t D) {
  return size_t(2) * kBalancedWGs * rows_per_wg(kQBBalanced) * size_t(D + 2) * sizeof(float);
}

// A bf16 key source from element strides (batch, head, token) shared by K and V.
KeySrc bf16_source(const void* k, const void* v, int64_t sb, int64_t sh, int64_t st) {
  return KeySrc{static_cast<const char*>(k), static_cast<const char*>(v), 2 * sb, 2 * sh, 2 * st, 2 * sb, 2 * sh,
                2 * st};
}

void fill_common(Params& p, int32_t B, int32_t H, float scale) {
  p.B = B;
  p.H = H;
  p.splits = 1;
  p.scale_log2 = scale * 1.4426950408889634f;
  p.lse = nullptr;
  p.ws_o = nullptr;
  p.ws_ml = nullptr;
  p.src[1] = KeySrc{nullptr, nullptr, 0, 0, 0, 0, 0, 0};
}

}  // namespace
}  // namespace rc

namespace rc {
namespace {

// The prefill of both cache formats: static-row attention, then the bf16 cache
// store or the FP8 quantising store.
rc_status prefill_impl(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale, const void* q_static,
                       const void* k_static, const void* v_static, int64_t tok_stride, void* o_static,
                       float* lse_static, bool fp8, void* k_cache, void* v_cache, float* kv_scale, void* stream) {
  RC_TRY(check_layout(L, RC_ENTRY_PREFILL));
  RC_TRY(check_dims(B, H, D, scale));
  RC_TRY(check_stride(tok_stride, H, D));
  const int64_t n_static = count_rows(L, RowSet::Static);
  const int64_t n_cached = count_cached_rows(L);
  if (n_static == 0) return RC_OK;  // no ST/R segment: nothing to prefill
  RC_TRY(check_ptr(q_static, "q_static"));
  RC_TRY(check_ptr(k_static, "k_static"));
  RC_TRY(check_ptr(v_static, "v_static"));
  RC_TRY(check_ptr(o_static, "o_static"));
  RC_TRY(check_lse(lse_static, "lse_static"));
  if (fp8) {
    // the scales are required whatever the cache size, so that a caller's
    // missing buffer is caught here rather than on the device
    if (!kv_scale) {
      set_error("kv_scale is null");
      return RC_ERR_ARG;
    }
    RC_TRY(check_lse(kv_scale, "kv_scale"));
  }
  if (n_cached > 0) {
    RC_TRY(check_ptr(k_cache, fp8 ? "k_cache8" : "k_cache"));
    RC_TRY(check_ptr(v_cache, fp8 ? "v_cache8" : "v_cache"));
    if (fp8 && n_cached > kFp8MaxKeys) {
      set_error("FP8 cache of %lld keys per (batch, head) exceeds %lld", (long long)n_cached,
                (long long)kFp8MaxKeys);
      return RC_ERR_ARG;
    }
  }
  Params p;
  memset(&p, 0, sizeof p);
  fill_common(p, B, H, scale);
  p.bm = rows_per_wg(kQBPlain);
  RC_TRY(plan(L, RC_ENTRY_PREFILL, p));
  RC_TRY(check_grid(p));
  p.q = static_cast<const uint16_t*>(q_static);
  p.q_st = tok_stride;
  p.q_sb = tok_stride * n_static;
  p.o = static_cast<uint16_t*>(o_static);
  p.o_st = int64_t(H) * D;
  p.o_sb = p.o_st * n_static;
  p.lse = lse_static;
  p.src[0] = bf16_source(k_static, v_static, tok_stride * n_static, D, tok_stride);

  // the cached segments' rows inside the static buffers and their cache
  // positions
  CopySeg seg[RC_MAX_SEGMENTS];
  int n_copy = 0;
  {
    const uint32_t cm = cached_mask(L);
    int32_t srow = 0, drow = 0;
    for (int i = 0; i < L->n_seg; ++i) {
      if (!is_static_kind(L->seg[i].kind)) continue;
      if (cm >> i & 1u) {
        seg[n_copy++] = CopySeg{srow, L->seg[i].len, drow};
        drow += L->seg[i].len;
      }
      srow += L->seg[i].len;
    }
  }
  if (!fp8) {
    CacheStoreParams c;
    memset(&c, 0, sizeof c);
    if (n_cached > 0) {
      c.k_src = static_cast<const uint16_t*>(k_static);
      c.v_src = static_cast<const uint16_t*>(v_static);
      c.k_dst = static_cast<uint16_t*>(k_cache);
      c.v_dst = static_cast<uint16_t*>(v_cache);
      c.src_st = tok_stride;
      c.src_sb = tok_stride * n_static;
      c.B = B;
      c.H = H;
      c.D = D;
      c.n_cached = int32_t(n_cached);
      c.n_copy = n_copy;
      for (int i = 0; i < n_copy; ++i) c.seg[i] = seg[i];
      c.total_rows = int32_t(n_cached);
    }
    // Copy work-groups at the end of the attention grid take the cache rows
    // that fit on the CUs its partial last round leaves free; the store
    // kernel (one thread per 16-byte granule, 256 per work-group) the rest.
    const CopyPlan cpl = plan_copy_tail(p, n_cached);
    if (cpl.blocks > 0) {
      CopyTail& t = p.cp;
      t.k_src = c.k_src;
      t.v_src = c.v_src;
      t.k_dst = c.k_dst;
      t.v_dst = c.v_dst;
      t.src_sb = c.src_sb;
      t.src_st = c.src_st;
      t.B = B;
      t.H = H;
      t.n_cached = c.n_cached;
      t.n_copy = c.n_copy;
      for (int i = 0; i < n_copy; ++i) t.seg[i] = seg[i];
      t.blocks = cpl.blocks;
      t.rows = int32_t(cpl.rows);
      RC_TRY(check_blocks(int64_t(B) * H * p.n_qtiles + cpl.blocks, "prefill attention"));
    }
    c.row0 = cpl.rows;
    const int64_t rest = int64_t(B) * H * n_cached - cpl.rows;
    RC_TRY(check_blocks((rest * (D / 8) + 255) / 256, "cache store"));
    RC_TRY(hip_status(launch_attention(p, D, stream), "prefill attention launch"));
    if (rest > 0) RC_TRY(hip_status(launch_cache_store(c, stream), "cache store launch"));
    return RC_OK;
  }
  CacheStore8Params c;
  memset(&c, 0, sizeof c);
  c.k_src = static_cast<const uint16_t*>(k_static);
  c.v_src = static_cast<const uint16_t*>(v_static);
  c.k_dst = static_cast<uint8_t*>(k_cache);
  c.v_dst = static_cast<uint8_t*>(v_cache);
  c.kv_scale = kv_scale;
  c.src_st = tok_stride;
  c.src_sb = tok_stride * n_static;
  c.B = B;
  c.H = H;
  c.D = D;
  c.n_cached = int32_t(n_cached);
  c.n_copy = n_copy;
  for (int i = 0; i < n_copy; ++i) c.seg[i] = seg[i];
  // the quantising store's grids: (B H) x row blocks (amax), one thread per
  // 16-byte granule of K and of V
  RC_TRY(check_blocks(int64_t(B) * H, "FP8 cache store"));
  RC_TRY(check_blocks((int64_t(B) * H * n_cached * (D / 8) + 255) / 256, "FP8 cache store"));
  RC_TRY(hip_status(launch_attention(p, D, stream), "prefill attention launch"));
  if (n_cached > 0) RC_TRY(hip_status(launch_cache_store_fp8(c, stream), "FP8 cache store launch"));
  return RC_OK;
}

// The step's schedule for a split choice (0 = automatic): query tiles, key
// ranges and the resolved split count, in p (p.B and p.H set by the caller).
rc_status plan_step(const rc_layout* L, int32_t D, bool fp8, int32_t splits, Params& p) {
  // the automatic choice is the one rc_step_auto_splits reports (for either
  // cache format)
  if (splits == 0) splits = rc_step_auto_splits(L, p.B, p.H, D);
  const bool balanced = splits == kSplitsBalanced;
  p.bm = rows_per_wg(fp8 ? kQBFp8 : balanced ? kQBBalanced : kQBPlain);
  RC_TRY(plan(L, RC_ENTRY_STEP, p, fp8));
  if (splits == kSplitsTail) {
    p.splits = 2;
    p.tail_num = tail_num(p);
  } else if (splits == kSplitsLastRound) {
    p.lr_tiles = last_round_tiles(p);
    p.splits = p.lr_tiles > 0 ? 2 : 1;
  } else {
    p.splits = splits;
  }
  if (balanced) {
    p.units = int64_t(p.B) * p.H * p.units_bh;
    p.bal_wgs = kBalancedWGs;
    return RC_OK;
  }
  return check_grid(p);
}

// The per-step attention over either cache format (bf16, or FP8: K8 and V8
// with their scales).
rc_status step_impl(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale, const void* q_live,
                    const void* k_live, const void* v_live, int64_t tok_stride, bool fp8, const void* k_cache,
                    const void* v_cache, const float* kv_scale, void* o_live, float* lse_live, int32_t splits,
                    void* workspace, size_t ws_bytes, void* stream) {
  RC_TRY(check_layout(L, RC_ENTRY_STEP));
  RC_TRY(check_dims(B, H, D, scale));
  RC_TRY(check_stride(tok_stride, H, D));
  if (splits < kSplitsLastRound || splits > kMaxSplits) {
    set_error("splits = %d must be RC_SPLITS_LAST_ROUND (-3), RC_SPLITS_TAIL (-2), RC_SPLITS_BALANCED (-1) or in "
              "[0, %d]",
              splits, kMaxSplits);
    return RC_ERR_ARG;
  }
  const int64_t n_live = count_rows(L, RowSet::Live);
  const int64_t n_cached = count_cached_rows(L);
  if (fp8 && splits == kSplitsBalanced) {
    set_error("the balanced schedule is not available with the FP8 cache");
    return RC_ERR_UNSUPPORTED;
  }
  if (fp8) {
    // required whatever the cache size (see the prefill)
    if (!kv_scale) {
      set_error("kv_scale is null");
      return RC_ERR_ARG;
    }
    RC_TRY(check_lse(kv_scale, "kv_scale"));
  }
  if (n_live == 0) return RC_OK;  // no LT/X segment: nothing to attend
  RC_TRY(check_ptr(q_live, "q_live"));
  RC_TRY(check_ptr(k_live, "k_live"));
  RC_TRY(check_ptr(v_live, "v_live"));
  RC_TRY(check_ptr(o_live, "o_live"));
  RC_TRY(check_lse(lse_live, "lse_live"));
  if (n_cached > 0) {
    RC_TRY(check_ptr(k_cache, fp8 ? "k_cache8" : "k_cache"));
    RC_TRY(check_ptr(v_cache, fp8 ? "v_cache8" : "v_cache"));
    if (fp8) {
      if (n_cached > kFp8MaxKeys) {
        set_error("FP8 cache of %lld keys per (batch, head) exceeds %lld", (long long)n_cached,
                  (long long)kFp8MaxKeys);
        return RC_ERR_ARG;
      }
    }
  }
  Params p;
  memset(&p, 0, sizeof p);
  fill_common(p, B, H, scale);
  RC_TRY(plan_step(L, D, fp8, splits, p));
  const bool balanced = p.splits == kSplitsBalanced;
  p.q = static_cast<const uint16_t*>(q_live);
  p.q_st = tok_stride;
  p.q_sb = tok_stride * n_live;
  p.o = static_cast<uint16_t*>(o_live);
  p.o_st = int64_t(H) * D;
  p.o_sb = p.o_st * n_live;
  p.lse = lse_live;
  p.src[0] = bf16_source(k_live, v_live, tok_stride * n_live, D, tok_stride);
  if (fp8) {
    p.fp8 = 1;
    p.kv_scale = kv_scale;
    p.src[1] = KeySrc{static_cast<const char*>(k_cache), static_cast<const char*>(v_cache), int64_t(H) * n_cached * D,
                      n_cached * D, D, int64_t(H) * n_cached * D, n_cached * D, D};
  } else {
    p.src[1] = bf16_source(k_cache, v_cache, int64_t(H) * n_cached * D, n_cached * D, D);
  }
  if (balanced) {
    const size_t need = balanced_workspace_bytes(D);
    if (!workspace || !aligned16(workspace) || ws_bytes < need) {
      set_error("the balanced schedule needs a 16-byte aligned workspace of %zu bytes (got %zu)", need,
                workspace ? ws_bytes : size_t(0));
      return RC_ERR_WORKSPACE;
    }
    p.ws_o = static_cast<float*>(workspace);
    p.ws_ml = p.ws_o + size_t(2) * kBalancedWGs * rows_per_wg(kQBBalanced) * D;
    RC_TRY(check_blocks((int64_t(B) * H * n_live * (D / 4) + 255) / 256, "balanced merge"));
    RC_TRY(hip_status(launch_attention_balanced(p, D, stream), "step attention launch"));
    RC_TRY(hip_status(launch_combine_balanced(p, D, stream), "balanced merge launch"));
    return RC_OK;
  }
  CombineParams c;
  memset(&c, 0, sizeof c);
  if (p.splits > 1) {
    const size_t need = rc_step_workspace_bytes(L, B, H, D, splits);
    if (!workspace || !aligned16(workspace) || ws_bytes < need) {
      set_error("split-KV with %d splits needs a 16-byte aligned workspace of %zu bytes (got %zu)", p.splits,
                need, workspace ? ws_bytes : size_t(0));
      return RC_ERR_WORKSPACE;
    }
    p.ws_o = static_cast<float*>(workspace);
    p.ws_ml = p.lr_tiles > 0 ? p.ws_o + size_t(2) * p.lr_tiles * p.bm * D
                             : p.ws_o + size_t(p.splits) * B * H * n_live * D;
    c.ws_o = p.ws_o;
    c.ws_ml = p.ws_ml;
    c.o = p.o;
    c.lse = lse_live;
    c.o_sb = p.o_sb;
    c.o_st = p.o_st;
    c.B = B;
    c.H = H;
    c.D = D;
    c.n_rows = int32_t(n_live);
    c.splits = p.splits;
  }
  // combine: one thread per 4 output elements, 256 per work-group
  if (p.splits > 1) RC_TRY(check_blocks((int64_t(B) * H * n_live * (D / 4) + 255) / 256, "split-KV combine"));
  if (p.lr_tiles > 0) RC_TRY(check_blocks(int64_t(B) * H * p.n_qtiles + p.lr_tiles, "step attention"));
  RC_TRY(hip_status(launch_attention(p, D, stream), "step attention launch"));
  if (p.lr_tiles > 0) RC_TRY(hip_status(launch_combine_last_round(p, D, stream), "last-round merge launch"));
  else if (p.splits > 1) RC_TRY(hip_status(launch_combine(c, stream), "split-KV combine launch"));
  return RC_OK;
}

}  // namespace
}  // namespace rc

using namespace rc;

extern "C" {

rc_status rc_ref_kv_prefill(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                            const void* q_static, const void* k_static, const void* v_static,
                            int64_t tok_stride, void* o_static, float* lse_static, void* k_cache,
                            void* v_cache, void* stream) {
  return prefill_impl(L, B, H, D, scale, q_static, k_static, v_static, tok_stride, o_static, lse_static, false,
                      k_cache, v_cache, nullptr, stream);
}

rc_status rc_ref_kv_prefill_fp8(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                const void* q_static, const void* k_static, const void* v_static,
                                int64_t tok_stride, void* o_static, float* lse_static, void* k_cache8,
                                void* v_cache8, float* kv_scale, void* stream) {
  return prefill_impl(L, B, H, D, scale, q_static, k_static, v_static, tok_stride, o_static, lse_static, true,
                      k_cache8, v_cache8, kv_scale, stream);
}

int32_t rc_step_auto_splits(const rc_layout* L, int32_t B, int32_t H, int32_t D) {
  if (check_layout(L, RC_ENTRY_STEP) != RC_OK) return 1;
  if (B < 1 || H < 1 || (D != 64 && D != 128)) return 1;
  Params p;
  memset(&p, 0, sizeof p);
  p.B = B;
  p.H = H;
  p.bm = rows_per_wg(kQBPlain);
  if (plan(L, RC_ENTRY_STEP, p) != RC_OK) return 1;
  return auto_splits(p);
}

rc_status rc_prefill_launch_plan(const rc_layout* L, int32_t B, int32_t H, int32_t D, int64_t* attn_wgs,
                                 int32_t* copy_wgs, int64_t* copy_rows) {
  using namespace rc;
  RC_TRY(check_layout(L, RC_ENTRY_PREFILL));
  if (!attn_wgs || !copy_wgs || !copy_rows) {
    set_error("rc_prefill_launch_plan: null output pointer");
    return RC_ERR_ARG;
  }
  RC_TRY(check_dims(B, H, D, 1.0f));
  Params p;
  memset(&p, 0, sizeof p);
  fill_common(p, B, H, 1.0f);
  p.bm = rows_per_wg(kQBPlain);
  RC_TRY(plan(L, RC_ENTRY_PREFILL, p));
  const CopyPlan c = plan_copy_tail(p, count_cached_rows(L));
  *attn_wgs = int64_t(B) * H * p.n_qtiles;
  *copy_wgs = c.blocks;
  *copy_rows = c.rows;
  return RC_OK;
}

rc_status rc_step_launch_shape(const rc_layout* L, int32_t B, int32_t H, int32_t D, int32_t splits, int32_t fp8,
                               int64_t* work_groups, int32_t* rows_per_wg, int32_t* splits_used) {
  using namespace rc;
  RC_TRY(check_layout(L, RC_ENTRY_STEP));
  if (!work_groups || !rows_per_wg || !splits_used) {
    set_error("rc_step_launch_shape: null output pointer");
    return RC_ERR_ARG;
  }
  RC_TRY(check_dims(B, H, D, 1.0f));
  if (splits < kSplitsLastRound || splits > kMaxSplits || (fp8 != 0 && fp8 != 1)) {
    set_error("rc_step_launch_shape: splits = %d or fp8 = %d out of range", splits, fp8);
    return RC_ERR_ARG;
  }
  if (fp8 && splits == kSplitsBalanced) {
    set_error("the balanced schedule is not available with the FP8 cache");
    return RC_ERR_UNSUPPORTED;
  }
  Params p;
  memset(&p, 0, sizeof p);
  p.B = B;
  p.H = H;
  RC_TRY(plan_step(L, D, fp8 != 0, splits, p));
  *rows_per_wg = p.bm;
  *splits_used = p.splits;
  if (p.lr_tiles > 0) *splits_used = kSplitsLastRound;
  *work_groups = p.splits == kSplitsBalanced ? int64_t(p.bal_wgs)
                 : p.lr_tiles > 0            ? int64_t(B) * H * p.n_qtiles + p.lr_tiles
                                             : int64_t(B) * H * p.n_qtiles * p.splits;
  return RC_OK;
}

size_t rc_step_workspace_bytes(const rc_layout* L, int32_t B, int32_t H, int32_t D, int32_t splits) {
  if (check_layout(L, RC_ENTRY_STEP) != RC_OK) return 0;
  if (B < 1 || H < 1 || (D != 64 && D != 128) || splits < kSplitsLastRound || splits > kMaxSplits) return 0;
  if (splits == 0) splits = rc_step_auto_splits(L, B, H, D);
  if (splits == kSplitsBalanced) return balanced_workspace_bytes(D);
  if (splits == kSplitsLastRound) {
    Params p;
    memset(&p, 0, sizeof p);
    p.B = B;
    p.H = H;
    p.bm = rows_per_wg(kQBPlain);
    if (plan(L, RC_ENTRY_STEP, p) != RC_OK) return 0;
    return size_t(2) * last_round_tiles(p) * p.bm * size_t(D + 2) * sizeof(float);
  }
  if (splits == kSplitsTail) splits = 2;
  if (splits <= 1) return 0;
  const int64_t n_live = count_rows(L, RowSet::Live);
  return size_t(splits) * size_t(B) * size_t(H) * size_t(n_live) * size_t(D + 2) * sizeof(float);
}

rc_status rc_step_masked_attention(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                   const void* q_live, const void* k_live, const void* v_live,
                                   int64_t tok_stride, const void* k_cache, const void* v_cache,
                                   void* o_live, float* lse_live, int32_t splits, void* workspace,
                                   size_t ws_bytes, void* stream) {
  return step_impl(L, B, H, D, scale, q_live, k_live, v_live, tok_stride, false, k_cache, v_cache, nullptr, o_live,
                   lse_live, splits, workspace, ws_bytes, stream);
}

rc_status rc_step_masked_attention_noalloc(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                           const void* q_live, const void* k_live, const void* v_live,
                                           int64_t tok_stride, const void* k_cache, const void* v_cache,
                                           void* o_live, float* lse_live, int32_t splits, void* stream) {
  using namespace rc;
  // the workspace the split choice needs (0 for none, or for invalid input,
  // which step_impl then reports)
  const size_t need = rc_step_workspace_bytes(L, B, H, D, splits);
  if (need > size_t(RC_NOALLOC_SCRATCH_BYTES)) {
    set_error("the no-allocation step holds %zu bytes of scratch; splits = %d needs %zu",
              size_t(RC_NOALLOC_SCRATCH_BYTES), splits, need);
    return RC_ERR_WORKSPACE;
  }
  void* ws = nullptr;
  if (need > 0) RC_TRY(hip_status(scratch_address(&ws), "scratch lookup"));
  return step_impl(L, B, H, D, scale, q_live, k_live, v_live, tok_stride, false, k_cache, v_cache, nullptr, o_live,
                   lse_live, splits, ws, need > 0 ? size_t(RC_NOALLOC_SCRATCH_BYTES) : 0, stream);
}

rc_status rc_step_masked_attention_fp8(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale,
                                       const void* q_live, const void* k_live, const void* v_live,
                                       int64_t tok_stride, const void* k_cache8, const void* v_cache8,
                                       const float* kv_scale, void* o_live, float* lse_live, int32_t splits,
                                       void* workspace, size_t ws_bytes, void* stream) {
  return step_impl(L, B, H, D, scale, q_live, k_live, v_live, tok_stride, true, k_cache8, v_cache8, kv_scale,
                   o_live, lse_live, splits, workspace, ws_bytes, stream);
}

size_t rc_full_workspace_bytes(const rc_layout* L, int32_t B, int32_t H, int32_t D) {
  using namespace rc;
  if (B < 1 || H < 1 || (D != 64 && D != 128)) return 0;
  if (check_layout(L, RC_ENTRY_FULL) != RC_OK) return 0;
  Params p;
  memset(&p, 0, sizeof p);
  fill_common(p, B, H, 1.0f);
  p.bm = rows_per_wg(kQBPlain);
  if (plan(L, RC_ENTRY_FULL, p) != RC_OK) return 0;
  return size_t(2) * last_round_tiles(p) * p.bm * size_t(D + 2) * sizeof(float);
}

rc_status rc_full_attention_ws(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale, const void* q,
                               const void* k, const void* v, int64_t tok_stride, void* o, float* lse,
                               void* workspace, size_t ws_bytes, void* stream) {
  RC_TRY(check_layout(L, RC_ENTRY_FULL));
  RC_TRY(check_dims(B, H, D, scale));
  RC_TRY(check_stride(tok_stride, H, D));
  RC_TRY(check_ptr(q, "q"));
  RC_TRY(check_ptr(k, "k"));
  RC_TRY(check_ptr(v, "v"));
  RC_TRY(check_ptr(o, "o"));
  RC_TRY(check_lse(lse, "lse"));
  const int64_t n = count_rows(L, RowSet::All);
  Params p;
  memset(&p, 0, sizeof p);
  fill_common(p, B, H, scale);
  p.bm = rows_per_wg(kQBPlain);
  RC_TRY(plan(L, RC_ENTRY_FULL, p));
  RC_TRY(check_grid(p));
  p.q = static_cast<const uint16_t*>(q);
  p.q_st = tok_stride;
  p.q_sb = tok_stride * n;
  p.o = static_cast<uint16_t*>(o);
  p.o_st = int64_t(H) * D;
  p.o_sb = p.o_st * n;
  p.lse = lse;
  p.src[0] = bf16_source(k, v, tok_stride * n, D, tok_stride);
  if (workspace) {
    const int32_t T = last_round_tiles(p);
    const size_t need = size_t(2) * T * p.bm * size_t(D + 2) * sizeof(float);
    if (!aligned16(workspace) || ws_bytes < need) {
      set_error("the last-round split needs a 16-byte aligned workspace of %zu bytes (got %zu)", need, ws_bytes);
      return RC_ERR_WORKSPACE;
    }
    if (T > 0) {
      p.splits = 2;
      p.lr_tiles = T;
      p.ws_o = static_cast<float*>(workspace);
      p.ws_ml = p.ws_o + size_t(2) * T * p.bm * D;
      RC_TRY(check_blocks(int64_t(B) * H * p.n_qtiles + T, "full attention"));
      RC_TRY(hip_status(launch_attention(p, D, stream), "full attention launch"));
      RC_TRY(hip_status(launch_combine_last_round(p, D, stream), "last-round merge launch"));
      return RC_OK;
    }
    p.tail_num = 0;
  }
  RC_TRY(hip_status(launch_attention(p, D, stream), "full attention launch"));
  return RC_OK;
}

rc_status rc_full_attention(const rc_layout* L, int32_t B, int32_t H, int32_t D, float scale, const void* q,
                            const void* k, const void* v, int64_t tok_stride, void* o, float* lse,
                            void* stream) {
  return rc_full_attention_ws(L, B, H, D, scale, q, k, v, tok_stride, o, lse, nullptr, 0, stream);
}

rc_status rc_linear(int64_t M, int32_t N, int32_t K, const void* a, int64_t lda, const void* w, const void* r,
                    int64_t ldr, void* out, int64_t ldo, void* stream) {
  if (M < 0 || M > (int64_t(1) << 40) || N <= 0 || K <= 0) {
    set_error("linear: M = %lld, N = %d, K = %d must be in [0, 2^40], > 0, > 0", (long long)M, N, K);
    return RC_ERR_ARG;
  }
  if (N % 128 != 0 || K % 64 != 0 || K > (1 << 22)) {
    set_error("linear: N = %d must be a multiple of 128 and K = %d a multiple of 64 up to 2^22", N, K);
    return RC_ERR_UNSUPPORTED;
  }
  const auto bad_ld = [](int64_t ld, int64_t lo) { return ld < lo || ld % 8 != 0 || ld > (int64_t(1) << 22); };
  if (bad_ld(lda, K) || bad_ld(ldo, N) || (r && bad_ld(ldr, N))) {
    set_error("linear: strides lda = %lld, ldr = %lld, ldo = %lld must be >= K / N, multiples of 8, <= 2^22",
              (long long)lda, (long long)ldr, (long long)ldo);
    return RC_ERR_ARG;
  }
  if (M == 0) return RC_OK;
  RC_TRY(check_ptr(a, "a"));
  RC_TRY(check_ptr(w, "w"));
  RC_TRY(check_ptr(out, "out"));
  if (r) RC_TRY(check_ptr(r, "r"));
  RC_TRY(check_blocks((M + 127) / 128 * (N / 128), "linear"));
  LinearParams q;
  q.a = static_cast<const uint16_t*>(a);
  q.w = static_cast<const uint16_t*>(w);
  q.r = static_cast<const uint16_t*>(r);
  q.out = static_cast<uint16_t*>(out);
  q.M = M;
  q.N = N;
  q.K = K;
  q.lda = lda;
  q.ldr = r ? ldr : 0;
  q.ldo = ldo;
  RC_TRY(hip_status(launch_linear(q, stream), "linear launch"));
  return RC_OK;
}

}  // extern "C"
