// Internal schedule shared by the host planner (layout.cpp, api.cpp) and the
// HIP kernels (attn_fwd.hip).  Not part of the public ABI.
//
// The planner turns an rc_layout plus an entry point into:
//   * query segments: which rows of the Q/O buffers one segment occupies and
//     how many BM-row tiles it splits into (a tile never straddles segments);
//   * key ranges: for each query segment, the visible key segments merged into
//     contiguous runs inside one key source, in sequence order.  Invisible
//     segments never appear, so masked blocks cost no loads and no MFMA.
// Two key sources exist: source 0 is the entry's own K/V buffer ([B,N,H,D]),
// source 1 is the reference K/V cache ([B,H,N_cached,D]).
#pragma once
#include <stdint.h>

#include "refcache.h"

namespace rc {

constexpr int kCUs = 256;         // compute units of the MI355X
constexpr int kWaves = 8;         // waves per work-group (two per SIMD)
constexpr int kStages = 2;        // K/V tiles resident in LDS in the one-block ring
// 32-row query blocks per wave.  The step over either cache, the prefill
// and the full recompute give each wave two blocks (BM = 512 rows per
// work-group); the balanced schedule keeps one (BM = 256), which its
// registers allow.
constexpr int kQBPlain = 2;
constexpr int kQBFp8 = 2;
constexpr int kQBBalanced = 1;
constexpr int rows_per_wg(int qb) { return 32 * qb * kWaves; }
constexpr int kBN = 64;           // keys per K/V tile
constexpr int kMaxRanges = 96;    // merged key ranges over all query segments
constexpr int kMaxSplits = 32;
// Balanced step schedule: one round of work-groups (one per CU of the 256),
// each taking an equal contiguous share of all (query tile, key tile) units.
constexpr int kBalancedWGs = 256;
constexpr int32_t kSplitsBalanced = RC_SPLITS_BALANCED;
constexpr int32_t kSplitsTail = RC_SPLITS_TAIL;
constexpr int32_t kSplitsLastRound = RC_SPLITS_LAST_ROUND;

struct KeyRange {
  int32_t start;   // first key token inside its source
  int32_t len;     // tokens
  int32_t src;     // 0 = entry buffer, 1 = cache
  int32_t ntiles;  // ceil(len / kBN)
};

struct QSeg {
  int64_t unit0;   // key-tile units of the earlier query segments, per (batch, head)
  int32_t row0;    // first row inside the Q/O buffers
  int32_t len;     // rows
  int32_t tile0;   // index of this segment's first query tile
  int32_t r0;      // first key range
  int32_t nr;      // number of key ranges
  int32_t ktiles;  // key tiles over all its ranges
};

// A run of cached rows: static-buffer rows [src_row0, src_row0 + len) go to
// cache rows [dst_row0, dst_row0 + len).
struct CopySeg {
  int32_t src_row0, len, dst_row0;
};

// The bf16 cache store carried by the prefill's attention launch: `blocks`
// work-groups after the attention work-groups copy the cached rows, on the
// CUs that the attention grid's partial last round leaves idle.
struct CopyTail {
  const uint16_t* k_src;
  const uint16_t* v_src;
  uint16_t* k_dst;
  uint16_t* v_dst;
  int64_t src_sb, src_st;  // element strides of the static K/V: batch, token
  int32_t B, H, n_cached, n_copy;
  int32_t blocks;          // copy work-groups at the end of the grid (0: none)
  int32_t rows;            // flat cache rows (b, h, row) [0, rows) that they copy
  CopySeg seg[RC_MAX_SEGMENTS];
};

// A key source, addressed in bytes.  bf16 sources hold K and V as
// [B, N, H, D] with one token stride; the FP8 cache holds K8 and V8 as
// [B, H, N_cached, D] bytes.
struct KeySrc {
  const char* k;
  const char* v;
  int64_t k_sb, k_sh, k_st;  // byte strides of K: batch, head, token
  int64_t v_sb, v_sh, v_st;  // byte strides of V: batch, head, token
};

struct Params {
  const uint16_t* q;
  int64_t q_sb, q_st;  // element strides of Q: batch, token (head stride = D)
  uint16_t* o;
  int64_t o_sb, o_st;
  float* lse;          // [B, H, n_rows] or null
  float* ws_o;         // split partials [splits, B, H, n_rows, D] (unnormalised)
  float* ws_ml;        // split partials [splits, B, H, n_rows, 2] (max in log2 units, sum)
  KeySrc src[2];
  int32_t B, H, n_rows, n_qseg, n_qtiles, splits;  // splits: kSplitsBalanced = balanced schedule
  int32_t bm;          // query rows per work-group tile (rows_per_wg of the kernel that runs)
  int32_t tail_num;    // tail split (splits = 2): split 0 takes floor(ktiles * tail_num / 1024) key tiles; 0 = even
  int32_t lr_tiles;    // last-round split (splits = 2, tail_num > 0): only the last lr_tiles query tiles
                       // (logical order) run as a long and a short piece; the others whole, written directly
  int32_t fp8;         // key source 1 is the FP8 cache
  const float* kv_scale;  // FP8 cache: [B, H, 2] power-of-two scales of K and V
  int64_t units_bh;    // key-tile units (query tile x key tile) per (batch, head)
  int64_t units;       // B * H * units_bh
  int32_t bal_wgs;     // work-groups of the balanced schedule
  float scale_log2;    // softmax scale * log2(e)
  QSeg qseg[RC_MAX_SEGMENTS];
  KeyRange range[kMaxRanges];
  CopyTail cp;         // prefill only; cp.blocks = 0 elsewhere
};

// Cache store: copy rows of the cached segments from the static K/V buffers
// ([B, N_static, H, D], token stride) into the cache ([B, H, N_cached, D]).
struct CacheStoreParams {
  const uint16_t* k_src;
  const uint16_t* v_src;
  uint16_t* k_dst;
  uint16_t* v_dst;
  int64_t src_sb, src_st;
  int64_t row0;        // first flat cache row (b, h, row) this launch copies
  int32_t B, H, D, n_cached, n_copy, total_rows;
  CopySeg seg[RC_MAX_SEGMENTS];
};

// FP8 cache store: quantise the cached segments' K/V rows (bf16, [B, N_static,
// H, D]) into K8 and V8 [B, H, N_cached, D] (the bf16 cache's rows, one byte
// per value).
// The amax pass runs one work-group row per 256 cached keys (grid y at most
// 65535).
constexpr int64_t kFp8MaxKeys = int64_t(65535) * 256;
struct CacheStore8Params {
  const uint16_t* k_src;
  const uint16_t* v_src;
  uint8_t* k_dst;
  uint8_t* v_dst;
  float* kv_scale;     // [B, H, 2]: amax while quantising, the scales afterwards
  int64_t src_sb, src_st;
  int32_t B, H, D, n_cached, n_copy;
  CopySeg seg[RC_MAX_SEGMENTS];
};

// Dense projection out = A W^T (+ R) of the chained synthetic layer.
struct LinearParams {
  const uint16_t* a;   // [M, K], row stride lda
  const uint16_t* w;   // [N, K], contiguous
  const uint16_t* r;   // [M, N], row stride ldr, or null
  uint16_t* out;       // [M, N], row stride ldo
  int64_t M;
  int32_t N, K;
  int64_t lda, ldr, ldo;
};

struct CombineParams {
  const float* ws_o;
  const float* ws_ml;
  uint16_t* o;
  float* lse;
  int64_t o_sb, o_st;
  int32_t B, H, D, n_rows, splits;
};

// Host-side planning (layout.cpp).
enum class RowSet { Static, Live, All };
bool is_static_kind(int32_t kind);
bool is_live_kind(int32_t kind);
rc_status check_layout(const rc_layout* L, int32_t entry);  // sets the thread error on failure
uint32_t cached_mask(const rc_layout* L);                  // bit i: segment i is cached
int64_t count_rows(const rc_layout* L, RowSet set);
int64_t count_cached_rows(const rc_layout* L);
// Fill p.qseg / p.range / n_qseg / n_qtiles / n_rows for an entry, with
// query tiles of p.bm rows (set by the caller).
rc_status plan(const rc_layout* L, int32_t entry, Params& p, bool fresh_first = false);
int32_t auto_splits(const Params& p);
int32_t tail_num(const Params& p);  // the long split's share of the key tiles, in 1/1024
// The full recompute's last-round split: the query tiles of an unsplit grid's
// partial last round (0 when none pays), with p.tail_num set for them.
int32_t last_round_tiles(Params& p);
// The prefill's bf16 cache store: the copy work-groups appended to the
// attention grid and the flat cache rows [0, rows) they take; the store
// kernel copies the rest.
struct CopyPlan {
  int32_t blocks;
  int64_t rows;
};
CopyPlan plan_copy_tail(const Params& p, int64_t n_cached);

void set_error(const char* fmt, ...);

// Kernel launchers (attn_fwd.hip).  Return a hipError_t as int.
// Unsplit multi-batch grids that run one launch per batch entry (each entry
// alone fills more than half the CUs).
bool per_batch_launches(const Params& p);
int launch_attention(const Params& p, int D, void* stream);
int launch_combine(const CombineParams& c, void* stream);
int launch_combine_last_round(const Params& p, int D, void* stream);  // the lr_tiles tiles' partials
int launch_attention_balanced(const Params& p, int D, void* stream);
int launch_combine_balanced(const Params& p, int D, void* stream);
int launch_cache_store(const CacheStoreParams& c, void* stream);
int launch_cache_store_fp8(const CacheStore8Params& c, void* stream);
int launch_linear(const LinearParams& q, void* stream);  // linear.hip
// Device address of the current GPU's static scratch array
// (RC_NOALLOC_SCRATCH_BYTES), looked up once per device.  hipError_t as int.
int scratch_address(void** ptr);

}  // namespace rc
