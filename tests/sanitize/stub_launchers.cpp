// Stand-ins for the kernel launchers, linked with the host planner
// (layout.cpp, api.cpp) into a CPU-only library built with AddressSanitizer
// and UndefinedBehaviorSanitizer.  Test infrastructure only: no GPU code runs.
//
// Every launcher checks the schedule it is handed against the invariants the
// kernels rely on (segments and key ranges inside their tables, tile and unit
// counts that add up, rows inside the buffers, the pointers a launch reads)
// and aborts with a message on the first violation; a clean call returns
// hipSuccess (0) and counts the launch.
#include <stdio.h>
#include <stdlib.h>

#include <cmath>

#include "rc_internal.h"

namespace {

long g_launches = 0;

[[noreturn]] void fail(const char* what, long a, long b) {
  fprintf(stderr, "stub launcher: broken schedule: %s (%ld, %ld)\n", what, a, b);
  fflush(stderr);
  abort();
}

#define REQUIRE(cond, a, b) \
  do {                      \
    if (!(cond)) fail(#cond, long(a), long(b)); \
  } while (0)

void check_params(const rc::Params& p, int D, bool balanced) {
  using namespace rc;
  REQUIRE(D == 64 || D == 128, D, 0);
  REQUIRE(p.B >= 1 && p.H >= 1, p.B, p.H);
  REQUIRE(p.bm == rows_per_wg(1) || p.bm == rows_per_wg(2), p.bm, 0);
  REQUIRE(p.n_qseg >= 1 && p.n_qseg <= RC_MAX_SEGMENTS, p.n_qseg, 0);
  REQUIRE(p.q && p.o, 0, 0);
  REQUIRE(std::isfinite(p.scale_log2) && p.scale_log2 > 0.f, 0, 0);
  REQUIRE(p.fp8 == 0 || p.fp8 == 1, p.fp8, 0);
  REQUIRE(!p.fp8 || p.kv_scale, p.fp8, 0);
  int64_t tiles = 0, units = 0, prev_end = 0;
  bool reads[2] = {false, false};
  for (int i = 0; i < p.n_qseg; ++i) {
    const QSeg& s = p.qseg[i];
    REQUIRE(s.len >= 1 && s.row0 >= prev_end, i, s.row0);
    REQUIRE(int64_t(s.row0) + s.len <= p.n_rows, i, p.n_rows);
    prev_end = s.row0 + s.len;
    REQUIRE(s.tile0 == tiles, i, s.tile0);
    REQUIRE(s.unit0 == units, i, s.unit0);
    REQUIRE(s.r0 >= 0 && s.nr >= 0 && s.r0 + s.nr <= kMaxRanges, s.r0, s.nr);
    int64_t kt = 0;
    for (int r = s.r0; r < s.r0 + s.nr; ++r) {
      const KeyRange& k = p.range[r];
      REQUIRE(k.len >= 1 && k.start >= 0, r, k.len);
      REQUIRE(k.src == 0 || k.src == 1, r, k.src);
      REQUIRE(k.ntiles == (k.len + kBN - 1) / kBN, r, k.ntiles);
      reads[k.src] = true;
      kt += k.ntiles;
    }
    REQUIRE(kt == s.ktiles, i, kt);
    const int64_t nt = (s.len + p.bm - 1) / p.bm;
    tiles += nt;
    units += nt * s.ktiles;
  }
  REQUIRE(tiles == p.n_qtiles, tiles, p.n_qtiles);
  REQUIRE(units == p.units_bh, units, p.units_bh);
  for (int s = 0; s < 2; ++s)
    if (reads[s]) REQUIRE(p.src[s].k && p.src[s].v && p.src[s].k_st > 0 && p.src[s].v_st > 0, s, 0);
  // a tile's byte record count (64 tokens x token stride) stays below 2^32
  for (int s = 0; s < 2; ++s)
    if (reads[s]) REQUIRE(int64_t(kBN) * p.src[s].k_st <= (int64_t(1) << 32), s, p.src[s].k_st);
  if (balanced) {
    REQUIRE(p.splits == kSplitsBalanced && p.bal_wgs == kBalancedWGs, p.splits, p.bal_wgs);
    REQUIRE(p.units == int64_t(p.B) * p.H * p.units_bh, p.units, 0);
    REQUIRE(p.ws_o && p.ws_ml, 0, 0);
  } else {
    REQUIRE(p.splits >= 1 && p.splits <= kMaxSplits, p.splits, 0);
    REQUIRE(p.splits == 1 || (p.ws_o && p.ws_ml), p.splits, 0);
    REQUIRE(p.tail_num == 0 || (p.splits == 2 && p.tail_num > 0 && p.tail_num < 1024), p.tail_num, p.splits);
    REQUIRE(int64_t(p.B) * p.H <= 65535 * int64_t(65535), p.B, p.H);
  }
}

void check_copy(const rc::CopySeg* seg, int n_copy, int32_t n_cached) {
  REQUIRE(n_copy >= 1 && n_copy <= RC_MAX_SEGMENTS, n_copy, 0);
  int64_t dst = 0;
  for (int i = 0; i < n_copy; ++i) {
    REQUIRE(seg[i].len >= 1 && seg[i].src_row0 >= 0, i, seg[i].len);
    REQUIRE(seg[i].dst_row0 == dst, i, seg[i].dst_row0);
    dst += seg[i].len;
  }
  REQUIRE(dst == n_cached, dst, n_cached);
}

}  // namespace

namespace rc {

int launch_attention(const Params& p, int D, void*) {
  check_params(p, D, false);
  REQUIRE(p.lr_tiles >= 0 && p.lr_tiles < kCUs, p.lr_tiles, 0);
  if (p.lr_tiles > 0) {
    REQUIRE(p.splits == 2 && p.tail_num > 0 && p.cp.blocks == 0, p.splits, p.tail_num);
    REQUIRE(p.lr_tiles <= int64_t(p.B) * p.H * p.n_qtiles, p.lr_tiles, p.n_qtiles);
  }
  const CopyTail& c = p.cp;
  REQUIRE(c.blocks >= 0 && c.blocks <= kCUs, c.blocks, 0);
  if (c.blocks > 0) {
    REQUIRE(p.splits == 1 && !p.fp8, p.splits, p.fp8);
    REQUIRE(c.k_src && c.v_src && c.k_dst && c.v_dst, 0, 0);
    REQUIRE(c.B == p.B && c.H == p.H, c.B, c.H);
    REQUIRE(int64_t(c.B) * c.H * c.n_cached < (int64_t(1) << 31), c.n_cached, 0);
    REQUIRE(c.rows >= c.blocks && c.rows <= int64_t(c.B) * c.H * c.n_cached, c.rows, c.blocks);
    check_copy(c.seg, c.n_copy, c.n_cached);
  }
  ++g_launches;
  return 0;
}

int launch_attention_balanced(const Params& p, int D, void*) {
  check_params(p, D, true);
  ++g_launches;
  return 0;
}

int launch_combine_balanced(const Params& p, int D, void*) {
  check_params(p, D, true);
  ++g_launches;
  return 0;
}

int launch_combine_last_round(const Params& p, int D, void*) {
  check_params(p, D, false);
  REQUIRE(p.lr_tiles > 0 && p.splits == 2 && p.ws_o && p.ws_ml, p.lr_tiles, p.splits);
  ++g_launches;
  return 0;
}

int launch_combine(const CombineParams& c, void*) {
  REQUIRE(c.ws_o && c.ws_ml && c.o, 0, 0);
  REQUIRE(c.splits >= 2 && c.splits <= kMaxSplits, c.splits, 0);
  REQUIRE(c.n_rows >= 1 && (c.D == 64 || c.D == 128), c.n_rows, c.D);
  ++g_launches;
  return 0;
}

int launch_cache_store(const CacheStoreParams& c, void*) {
  REQUIRE(c.k_src && c.v_src && c.k_dst && c.v_dst, 0, 0);
  REQUIRE(c.total_rows == c.n_cached, c.total_rows, c.n_cached);
  REQUIRE(c.row0 >= 0 && c.row0 < int64_t(c.B) * c.H * c.n_cached, c.row0, c.n_cached);
  check_copy(c.seg, c.n_copy, c.n_cached);
  ++g_launches;
  return 0;
}

int launch_cache_store_fp8(const CacheStore8Params& c, void*) {
  REQUIRE(c.k_src && c.v_src && c.k_dst && c.v_dst && c.kv_scale, 0, 0);
  REQUIRE(c.n_cached <= kFp8MaxKeys, c.n_cached, 0);
  check_copy(c.seg, c.n_copy, c.n_cached);
  ++g_launches;
  return 0;
}

int launch_linear(const LinearParams& q, void*) {
  REQUIRE(q.a && q.w && q.out, 0, 0);
  REQUIRE(q.M >= 1 && q.N >= 1 && q.K >= 1, q.M, q.N);
  REQUIRE(q.lda >= q.K && q.ldo >= q.N && (!q.r || q.ldr >= q.N), q.lda, q.ldo);
  ++g_launches;
  return 0;
}

// a fake, never dereferenced device address of the scratch array
int scratch_address(void** ptr) {
  *ptr = reinterpret_cast<void*>(uintptr_t(0x7f0000100000));
  ++g_launches;
  return 0;
}

}  // namespace rc

extern "C" long rc_stub_launches(void) { return g_launches; }
