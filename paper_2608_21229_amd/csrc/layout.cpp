// Host-side layout logic: mask presets, validation, pair counts and the
// work schedule (query tiles + merged visible key ranges) for each entry.
//
// Segment semantics follow Sec. 3.1 (Eq. 1) and Sec. 3.3: ST and R form the
// static subgraph evaluated once per request; LT and X are live.  The caching
// condition is App. A's StructCacheable for a layer-shared mask: no static
// query segment may read a live key segment, otherwise target information
// reaches R through some layer (Sec. 3.2, Eq. 3).
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <queue>
#include <vector>

#include "rc_internal.h"

namespace rc {

static thread_local char g_err[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
}

const char* last_error() { return g_err; }

bool is_static_kind(int32_t kind) { return kind == RC_SEG_ANCHOR || kind == RC_SEG_REF; }
bool is_live_kind(int32_t kind) { return kind == RC_SEG_TEXT || kind == RC_SEG_TARGET; }

static rc_status check_table(const rc_layout* L) {
  if (!L) {
    set_error("layout is null");
    return RC_ERR_ARG;
  }
  if (L->n_seg < 1 || L->n_seg > RC_MAX_SEGMENTS) {
    set_error("n_seg = %d, must be in [1, %d]", L->n_seg, RC_MAX_SEGMENTS);
    return RC_ERR_ARG;
  }
  int64_t total = 0;
  for (int i = 0; i < L->n_seg; ++i) {
    if (L->seg[i].kind < RC_SEG_ANCHOR || L->seg[i].kind > RC_SEG_REF) {
      set_error("segment %d has unknown kind %d", i, L->seg[i].kind);
      return RC_ERR_ARG;
    }
    if (L->seg[i].len < 1) {
      set_error("segment %d has length %d, must be >= 1", i, L->seg[i].len);
      return RC_ERR_ARG;
    }
    total += L->seg[i].len;
  }
  if (total > (int64_t(1) << 24)) {
    set_error("sequence of %lld tokens exceeds the 2^24 limit", (long long)total);
    return RC_ERR_ARG;
  }
  return RC_OK;
}

rc_status check_layout(const rc_layout* L, int32_t entry) {
  rc_status s = check_table(L);
  if (s != RC_OK) return s;
  if (entry < RC_ENTRY_PREFILL || entry > RC_ENTRY_FULL) {
    set_error("unknown entry %d", entry);
    return RC_ERR_ARG;
  }
  const uint32_t valid = (L->n_seg == 32) ? 0xffffffffu : ((1u << L->n_seg) - 1u);
  for (int q = 0; q < L->n_seg; ++q) {
    if (L->visible[q] & ~valid) {
      set_error("visible[%d] = 0x%x has bits beyond n_seg = %d", q, L->visible[q], L->n_seg);
      return RC_ERR_ARG;
    }
  }
  if (entry == RC_ENTRY_FULL) return RC_OK;
  for (int q = 0; q < L->n_seg; ++q) {
    if (!is_static_kind(L->seg[q].kind)) continue;
    for (int k = 0; k < L->n_seg; ++k) {
      if ((L->visible[q] >> k & 1u) && is_live_kind(L->seg[k].kind)) {
        set_error("static segment %d reads live segment %d: reference K/V would depend on the "
                  "denoising target, so they are not exactly cacheable",
                  q, k);
        return RC_ERR_MASK_NOT_CACHEABLE;
      }
    }
  }
  return RC_OK;
}

uint32_t cached_mask(const rc_layout* L) {
  uint32_t m = 0;
  for (int k = 0; k < L->n_seg; ++k) {
    if (!is_static_kind(L->seg[k].kind)) continue;
    for (int q = 0; q < L->n_seg; ++q)
      if (is_live_kind(L->seg[q].kind) && (L->visible[q] >> k & 1u)) m |= 1u << k;
  }
  return m;
}

static bool in_set(const rc_layout* L, int i, RowSet set) {
  switch (set) {
    case RowSet::Static: return is_static_kind(L->seg[i].kind);
    case RowSet::Live: return is_live_kind(L->seg[i].kind);
    default: return true;
  }
}

int64_t count_rows(const rc_layout* L, RowSet set) {
  int64_t n = 0;
  for (int i = 0; i < L->n_seg; ++i)
    if (in_set(L, i, set)) n += L->seg[i].len;
  return n;
}

int64_t count_cached_rows(const rc_layout* L) {
  const uint32_t m = cached_mask(L);
  int64_t n = 0;
  for (int i = 0; i < L->n_seg; ++i)
    if (m >> i & 1u) n += L->seg[i].len;
  return n;
}

static RowSet rows_of(int32_t entry) {
  return entry == RC_ENTRY_PREFILL ? RowSet::Static : entry == RC_ENTRY_STEP ? RowSet::Live : RowSet::All;
}

rc_status plan(const rc_layout* L, int32_t entry, Params& p, bool fresh_first) {
  const RowSet rset = rows_of(entry);
  // Position of every segment inside each key source.
  int32_t src_of[RC_MAX_SEGMENTS], pos_of[RC_MAX_SEGMENTS], row_of[RC_MAX_SEGMENTS];
  const uint32_t cmask = cached_mask(L);
  int32_t pos_entry = 0, pos_cache = 0, pos_rows = 0;
  for (int i = 0; i < L->n_seg; ++i) {
    src_of[i] = -1;
    pos_of[i] = 0;
    row_of[i] = -1;
    const bool row_member = in_set(L, i, rset);
    if (row_member) {
      row_of[i] = pos_rows;
      pos_rows += L->seg[i].len;
    }
    if (entry == RC_ENTRY_FULL || entry == RC_ENTRY_PREFILL ? row_member : is_live_kind(L->seg[i].kind)) {
      src_of[i] = 0;
      pos_of[i] = pos_entry;
      pos_entry += L->seg[i].len;
    } else if (entry == RC_ENTRY_STEP && (cmask >> i & 1u)) {
      src_of[i] = 1;
      pos_of[i] = pos_cache;
      pos_cache += L->seg[i].len;
    }
  }
  p.n_rows = pos_rows;
  p.n_qseg = 0;
  p.n_qtiles = 0;
  p.units_bh = 0;
  int nranges = 0;
  for (int q = 0; q < L->n_seg; ++q) {
    if (row_of[q] < 0) continue;
    KeyRange tmp[RC_MAX_SEGMENTS];
    int nr = 0;
    for (int k = 0; k < L->n_seg; ++k) {
      if (!(L->visible[q] >> k & 1u)) continue;
      if (src_of[k] < 0) {
        // validated layouts never get here: a static row reading a live key
        set_error("internal: segment %d has no key source for entry %d", k, entry);
        return RC_ERR_ARG;
      }
      if (nr > 0 && tmp[nr - 1].src == src_of[k] && tmp[nr - 1].start + tmp[nr - 1].len == pos_of[k]) {
        tmp[nr - 1].len += L->seg[k].len;
      } else {
        tmp[nr].start = pos_of[k];
        tmp[nr].len = L->seg[k].len;
        tmp[nr].src = src_of[k];
        ++nr;
      }
    }
    if (fresh_first) {
      // FP8 cache: fresh (bf16) ranges first, then cache ranges, so that the
      // kernel runs one ring over each tile kind (softmax is order-free)
      KeyRange part[RC_MAX_SEGMENTS];
      int np = 0;
      for (int pass = 0; pass < 2; ++pass)
        for (int r = 0; r < nr; ++r)
          if (tmp[r].src == pass) part[np++] = tmp[r];
      for (int r = 0; r < nr; ++r) tmp[r] = part[r];
    }
    int ktiles = 0;
    for (int r = 0; r < nr; ++r) {
      tmp[r].ntiles = (tmp[r].len + kBN - 1) / kBN;
      ktiles += tmp[r].ntiles;
    }
    // Reuse an identical range list of an earlier query segment.
    int r0 = -1;
    for (int e = 0; e < p.n_qseg && r0 < 0; ++e) {
      const QSeg& o = p.qseg[e];
      if (o.nr != nr) continue;
      bool same = true;
      for (int r = 0; r < nr && same; ++r) {
        const KeyRange& a = p.range[o.r0 + r];
        same = a.start == tmp[r].start && a.len == tmp[r].len && a.src == tmp[r].src;
      }
      if (same) r0 = o.r0;
    }
    if (r0 < 0) {
      if (nranges + nr > kMaxRanges) {
        set_error("schedule needs more than %d merged key ranges", kMaxRanges);
        return RC_ERR_UNSUPPORTED;
      }
      r0 = nranges;
      for (int r = 0; r < nr; ++r) p.range[nranges++] = tmp[r];
    }
    QSeg& s = p.qseg[p.n_qseg++];
    s.row0 = row_of[q];
    s.len = L->seg[q].len;
    s.tile0 = p.n_qtiles;
    s.r0 = r0;
    s.nr = nr;
    s.ktiles = ktiles;
    s.unit0 = p.units_bh;
    const int ntiles = (s.len + p.bm - 1) / p.bm;
    p.n_qtiles += ntiles;
    p.units_bh += int64_t(ntiles) * ktiles;
  }
  return RC_OK;
}

int32_t auto_splits(const Params& p) {
  // Beyond one round of query tiles, the last-round split (when it applies).
  // Otherwise split the keys only when the query tiles alone leave CUs idle.  When they
  // fill more than half of the 256 CUs, the tail split uses the rest: every
  // query tile keeps one work-group for most of its keys and the short
  // remainders run on the idle CUs, R = ceil(Q / (256 - Q)) in turn.  Each
  // short piece pays a Q load, a partial write and its share of the combine,
  // so beyond R = 3 (Q > 192) the split measured slower than none.  Below
  // half, split evenly, as far as one round of work-groups still fits: a
  // partial second round measured cheaper than the extra splits' overheads.
  // Keep >= 8 key tiles per split.
  const int64_t wgs = int64_t(p.B) * p.H * p.n_qtiles;
  const int64_t slots = 256;  // one work-group per CU
  if (wgs <= 0) return 1;
  if (wgs >= slots) {
    // more tiles than CUs: split only the partial last round's tiles
    Params q = p;
    return last_round_tiles(q) > 0 ? kSplitsLastRound : 1;
  }
  int max_kt = 0;
  for (int i = 0; i < p.n_qseg; ++i)
    if (p.qseg[i].ktiles > max_kt) max_kt = p.qseg[i].ktiles;
  if (2 * wgs > slots) {
    const int64_t rounds = (wgs + (slots - wgs) - 1) / (slots - wgs);
    return (rounds <= 3 && max_kt >= 16) ? kSplitsTail : 1;
  }
  int64_t s = slots / wgs;
  const int64_t cap = max_kt / 8;
  if (s > cap) s = cap;
  if (s > kMaxSplits) s = kMaxSplits;
  return s < 1 ? 1 : int32_t(s);
}

bool per_batch_launches(const Params& p) {
  return p.B > 1 && p.splits == 1 && 2 * int64_t(p.H) * p.n_qtiles > kCUs;
}

// Dispatch model of one unsplit attention launch: work-group i goes to XCD
// i mod 8 and there, in order, to the first of the XCD's 32 CUs to become
// free; a work-group lasts its query tile's key tiles plus kTileOverhead
// tile times.  The copy work-groups come after the last attention
// work-group, at most one on each CU that becomes free before the attention
// ends (short work-groups, such as one-key-tile anchor rows, free theirs
// early), and may run until the attention ends, each counted on for
// kCopyRowsPerTile cache rows (K and V of one token and head) per tile time:
// a conservative figure (a copy work-group next to the attention measured
// 100 or more at D = 128 with 512-row tiles, and larger settings were no
// better overall).  The model stops at kMaxModelWGs work-groups, where the
// store is a small part of the launch.
namespace {
constexpr int64_t kCopyRowsPerTile = 64;
constexpr int64_t kTileOverhead = 2;
constexpr int64_t kCopyMinRows = 64;  // per copy work-group
constexpr int64_t kMaxModelWGs = int64_t(1) << 16;
}  // namespace

CopyPlan plan_copy_tail(const Params& p, int64_t n_cached) {
  const CopyPlan none{0, 0};
  if (n_cached <= 0 || p.splits != 1 || p.fp8) return none;
  const int64_t R = int64_t(p.B) * p.H * n_cached;
  if (R >= (int64_t(1) << 31)) return none;  // the copy work-groups index rows in 32 bits
  const int64_t A = per_batch_launches(p) ? int64_t(p.H) * p.n_qtiles : int64_t(p.B) * p.H * p.n_qtiles;
  if (A <= 0 || A > kMaxModelWGs) return none;
  // candidates: one copy work-group per CU, placed in dispatch order; the
  // ones the model sees start only when the attention ends drop out below
  const int64_t C = kCUs;
  constexpr int kXcds = 8, kPerXcd = kCUs / kXcds;
  typedef std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> FreeAt;
  std::vector<FreeAt> cu(kXcds);
  for (auto& q : cu)
    for (int i = 0; i < kPerXcd; ++i) q.push(0);
  // the kernel's block -> (query tile) mapping: consecutive logical blocks
  // on one XCD
  const int64_t per = A >> 3, rem = A & 7;
  int64_t end = 0;
  for (int64_t bid = 0; bid < A; ++bid) {
    const int64_t x = bid & 7, kx = bid >> 3;
    const int64_t w = x < rem ? x * (per + 1) + kx : rem * (per + 1) + (x - rem) * per + kx;
    const int t = int(w % p.n_qtiles);
    int qi = 0;
    while (qi + 1 < p.n_qseg && p.qseg[qi + 1].tile0 <= t) ++qi;
    FreeAt& q = cu[size_t(x)];
    const int64_t fin = q.top() + p.qseg[qi].ktiles + kTileOverhead;
    q.pop();
    q.push(fin);
    end = std::max(end, fin);
  }
  // Copy work-groups take equal row counts, so the one with the shortest
  // window sets the pace: keep the first c of them (those placed earliest)
  // with the largest c x (shortest window among them), no more than give
  // each kCopyMinRows rows, and no more than take every row.
  std::vector<int64_t> win(static_cast<size_t>(C), 0);
  int64_t window = end, best_c = 0;
  for (int64_t j = 0; j < C; ++j) {
    FreeAt& q = cu[size_t((A + j) & 7)];
    window = std::min(window, end - q.top());
    q.pop();  // the copy keeps its CU
    win[size_t(j)] = window;
    if ((j + 1) * window > (best_c ? best_c * win[size_t(best_c - 1)] : 0)) best_c = j + 1;
  }
  int64_t c = std::min(best_c, R / kCopyMinRows);
  if (c <= 0) return none;
  // When they can take every row, as few as can: each busy CU lowers the
  // clock of the attention work-groups still running.
  if (c * kCopyRowsPerTile * win[size_t(c - 1)] >= R) {
    int64_t m = 1;
    while (m < c && m * kCopyRowsPerTile * win[size_t(m - 1)] < R) ++m;
    c = m;
  }
  const int64_t rows = std::min(R, c * kCopyRowsPerTile * win[size_t(c - 1)]);
  return CopyPlan{int32_t(c), rows};
}

int32_t last_round_tiles(Params& p) {
  // An unsplit grid of A > 256 whole query tiles leaves 256 - T CUs idle in
  // its last round of T tiles.  Those T tiles run as a long piece (on the CUs
  // the earlier rounds free) and a short piece (on the idle CUs, R rounds of
  // them): the long piece takes R / (R + 1) of the keys so both end together,
  // and the round shrinks to R / (R + 1) of a tile.  Kept to R <= 3 and to
  // tiles of >= 16 key tiles, as the step's tail split (each piece pays a Q
  // load, a partial write and its share of the merge).
  const int64_t A = int64_t(p.B) * p.H * p.n_qtiles;
  const int64_t T = A % kCUs, idle = kCUs - T;
  if (A <= kCUs || T == 0) return 0;
  const int64_t r = (T + idle - 1) / idle;
  if (r > 3) return 0;
  for (int64_t w = A - T; w < A; ++w) {
    const int t = int(w % p.n_qtiles);
    int qi = 0;
    while (qi + 1 < p.n_qseg && p.qseg[qi + 1].tile0 <= t) ++qi;
    if (p.qseg[qi].ktiles < 16) return 0;
  }
  p.tail_num = int32_t(1024 * r / (r + 1));
  return int32_t(T);
}

int32_t tail_num(const Params& p) {
  // Q query tiles on Q CUs; 256 - Q CUs run the short pieces, R rounds each:
  // the long piece takes R / (R + 1) of the keys so both end together.
  const int64_t q = int64_t(p.B) * p.H * p.n_qtiles;
  const int64_t free_cus = 256 - q;
  if (q <= 0 || free_cus <= 0) return 512;
  const int64_t r = (q + free_cus - 1) / free_cus;
  return int32_t(1024 * r / (r + 1));
}

}  // namespace rc

extern "C" {

rc_status rc_layout_preset(rc_layout* L, int32_t preset) {
  rc_status s = rc::check_table(L);
  if (s != RC_OK) return s;
  if (preset < RC_MASK_PAPER || preset > RC_MASK_DENSE) {
    rc::set_error("unknown mask preset %d", preset);
    return RC_ERR_ARG;
  }
  for (int q = 0; q < RC_MAX_SEGMENTS; ++q) L->visible[q] = 0;
  for (int q = 0; q < L->n_seg; ++q) {
    const int32_t qk = L->seg[q].kind;
    uint32_t row = 0;
    for (int k = 0; k < L->n_seg; ++k) {
      const int32_t kk = L->seg[k].kind;
      bool v = false;
      switch (preset) {
        case RC_MASK_PAPER:
          // ST <-> R both ways; LT, X read LT, X, R (not ST)
          v = rc::is_static_kind(qk) ? rc::is_static_kind(kk) : kk != RC_SEG_ANCHOR;
          break;
        case RC_MASK_PERREF:
          // ST reads ST; R^(k) reads ST and itself; LT, X read everything
          if (qk == RC_SEG_ANCHOR) v = kk == RC_SEG_ANCHOR;
          else if (qk == RC_SEG_REF) v = kk == RC_SEG_ANCHOR || k == q;
          else v = true;
          break;
        case RC_MASK_ISOLATED:
          // anchors detached; R reads R; LT, X read LT, X, R
          if (qk == RC_SEG_ANCHOR) v = false;
          else if (qk == RC_SEG_REF) v = kk == RC_SEG_REF;
          else v = kk != RC_SEG_ANCHOR;
          break;
        default:
          v = true;
      }
      if (v) row |= 1u << k;
    }
    L->visible[q] = row;
  }
  return RC_OK;
}

rc_status rc_layout_validate(const rc_layout* L, int32_t entry) { return rc::check_layout(L, entry); }

int64_t rc_pairs(const rc_layout* L, int32_t entry) {
  rc_status s = rc::check_layout(L, entry);
  if (s != RC_OK) return s;
  const rc::RowSet set = rc::rows_of(entry);
  int64_t pairs = 0;
  for (int q = 0; q < L->n_seg; ++q) {
    if (!rc::in_set(L, q, set)) continue;
    int64_t keys = 0;
    for (int k = 0; k < L->n_seg; ++k)
      if (L->visible[q] >> k & 1u) keys += L->seg[k].len;
    pairs += int64_t(L->seg[q].len) * keys;
  }
  return pairs;
}

int64_t rc_rows(const rc_layout* L, int32_t which) {
  rc_status s = rc::check_layout(L, RC_ENTRY_FULL);
  if (s != RC_OK) return s;
  switch (which) {
    case RC_ROWS_STATIC: return rc::count_rows(L, rc::RowSet::Static);
    case RC_ROWS_LIVE: return rc::count_rows(L, rc::RowSet::Live);
    case RC_ROWS_CACHED: return rc::count_cached_rows(L);
    case RC_ROWS_ALL: return rc::count_rows(L, rc::RowSet::All);
    default:
      rc::set_error("unknown row class %d", which);
      return RC_ERR_ARG;
  }
}

const char* rc_status_string(rc_status s) {
  switch (s) {
    case RC_OK: return "ok";
    case RC_ERR_ARG: return "invalid argument";
    case RC_ERR_UNSUPPORTED: return "unsupported configuration";
    case RC_ERR_MASK_NOT_CACHEABLE: return "mask is not cacheable";
    case RC_ERR_WORKSPACE: return "workspace missing or too small";
    case RC_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* rc_last_error(void) { return rc::last_error(); }

}  // extern "C"
