// Block-masked flash attention forward for gfx950 (CDNA4), plus the split-KV
// combine and the reference K/V cache store.
//
// Method: softmax(scale * Q K^T) V over the visible key segments of each
// query segment (Sec. 3.3 mask; App. C interaction counts).  The planner
// hands every work-group a BM-row query tile inside one segment and the list
// of visible key ranges; invisible segments are never loaded.
//
// Work-group = 8 waves of 64 lanes, one work-group and two waves per SIMD on
// each CU.  A wave owns QB blocks of 32 query rows (two in the step over
// either cache, the prefill and the full recompute: BM = 512; one in the
// balanced schedule: BM = 256).
// Per 64-key tile:
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = the
//                   wave's Q rows held in registers for the whole kernel; each
//                   K fragment feeds one MFMA per query block.  The 32x32
//                   accumulator puts one query per lane (lane % 32) and 16
//                   keys per lane, so row reductions stay in the lane plus
//                   one exchange between the two 32-lane halves.
//   online softmax  exp2 with scale*log2(e) folded into one FMA; the running
//                   max is refreshed lazily (only when a row's weights would
//                   grow past a bound), which is exact because the same stale
//                   max scales both the sum and the accumulator.
//   O^T += V^T P^T  A = V^T read from row-major V in LDS with the gfx950
//                   transpose read ds_read_b64_tr_b16, B = P^T straight from
//                   the S^T accumulator registers (bf16), so the output also
//                   has one query per lane and the softmax statistics never
//                   leave their lane.
// K/V tiles arrive by direct global->LDS buffer loads (16 bytes per lane, 16
// lanes per 256-byte row), placed with an XOR swizzle at 16-byte granularity
// that keeps both the 128-bit K reads and the transpose V reads free of bank
// conflicts.  The tile cursor keeps the current key range's pointers in
// scalar registers, so issuing a tile needs no reads of the range table.
//
// With two query blocks per wave a tile is computed as two 32-key sub-tiles,
// and the two waves of each SIMD run half a phase apart (the ping-pong ring):
// one issues MFMAs while the other does its softmax.  With one block per wave
// every wave loads and computes whole tiles behind one barrier per tile.
//
// Over the FP8 cache (the kF8 instantiation) the fresh key ranges run through
// the ping-pong ring and the cached ranges through a second pass of it whose
// tiles arrive as 8-bit codes and are widened to bf16 in LDS, exactly (the
// scales are powers of two), one tile ahead of their compute.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "rc_internal.h"

namespace rc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) const char lds_cchar;
typedef __attribute__((address_space(3))) const bf16x8 lds_cbf16x8;

constexpr float kLazyThreshold = 8.0f;  // log2 units: rescale when a row max grows by > 2^8

// 16-byte-granule XOR swizzle of a K/V tile row.  Bits 0-1 of the row move to
// bits 2-3 of the granule and bits 2-3 of the row to bits 0-1: any 16
// consecutive rows at one granule hit 16 distinct granule slots (128-bit K
// reads), and 4 consecutive rows x 4 consecutive granules hit 16 distinct
// slots (transpose V reads of two 16-lane groups), so neither access pattern
// conflicts in the 64-bank LDS.
__device__ __forceinline__ int swz(int row, int g, int gr) {
  return g ^ ((((row & 3) << 2) | ((row >> 2) & 3)) & (gr - 1));
}

__device__ __forceinline__ float max_halves(float x) {
  // max of this lane and lane ^ 32 (the two halves hold different keys of the same query)
  auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(pr[0]), __uint_as_float(pr[1]));
}

__device__ __forceinline__ float sum_halves(float x) {
  auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(pr[0]) + __uint_as_float(pr[1]);
}

// Cursor over the key tiles of one query segment.  It keeps the current key
// range's source pointers, stride and remaining key count in (scalar)
// registers and steps from tile to tile by pointer arithmetic; the range and
// source descriptors in the kernel arguments are read again only when the
// cursor crosses into the next range.
struct Cursor {
  const char* k;      // K / V of the current tile's first key, batch and head applied (bytes)
  const char* v;
  int64_t kstep;      // bytes between consecutive tiles of the range, K and V
  int64_t vstep;
  int32_t st;         // K token stride of the key source (bytes)
  int32_t rem;        // keys of the range from the current tile on
  int32_t src;        // key source of the range
  int32_t r, t, ntiles, r_end;
  int32_t b, h;
};

__device__ __forceinline__ void cursor_load(const Params& p, Cursor& c, int r, int t) {
  const KeyRange rg = p.range[r];
  const KeySrc s = p.src[rg.src];
  c.r = r;
  c.t = t;
  c.ntiles = rg.ntiles;
  c.src = rg.src;
  c.st = int32_t(s.k_st);
  c.rem = rg.len - t * kBN;
  c.kstep = int64_t(kBN) * s.k_st;
  c.vstep = int64_t(kBN) * s.v_st;
  const int64_t key = rg.start + t * kBN;
  c.k = s.k + int64_t(c.b) * s.k_sb + int64_t(c.h) * s.k_sh + key * s.k_st;
  c.v = s.v + int64_t(c.b) * s.v_sb + int64_t(c.h) * s.v_sh + key * s.v_st;
}

__device__ __forceinline__ Cursor cursor_at(const Params& p, const QSeg& qs, int kt, int b, int h) {
  Cursor c;
  c.b = b;
  c.h = h;
  c.r_end = qs.r0 + qs.nr;
  if (qs.nr == 0) {  // a query segment that reads no key: no tile, and no range entry to read
    c.k = c.v = nullptr;
    c.kstep = c.vstep = 0;
    c.st = c.rem = c.src = 0;
    c.r = qs.r0;
    c.t = c.ntiles = 0;
    return c;
  }
  int r = qs.r0;
  for (int i = 0; i + 1 < qs.nr; ++i) {
    const int n = p.range[r].ntiles;
    if (kt < n) break;
    kt -= n;
    ++r;
  }
  cursor_load(p, c, r, kt);
  return c;
}

__device__ __forceinline__ void cursor_next(const Params& p, Cursor& c) {
  if (++c.t < c.ntiles) {
    c.k += c.kstep;
    c.v += c.vstep;
    c.rem -= kBN;
  } else if (c.r + 1 < c.r_end) {
    cursor_load(p, c, c.r + 1, 0);
  }
}

typedef __attribute__((address_space(3))) void lds_void;

constexpr int kThreads = 64 * kWaves;
constexpr int kTileElems = kBN * 128;  // LDS elements reserved per K or V tile (D <= 128)

// The K/V ring in LDS.  Separate objects per stage (selected at compile time)
// let the compiler see that a DMA into one stage never aliases reads of
// another, so it inserts no conservative vector-memory waits before them.
__shared__ __attribute__((aligned(1024))) uint16_t g_k0[kTileElems];
__shared__ __attribute__((aligned(1024))) uint16_t g_v0[kTileElems];
__shared__ __attribute__((aligned(1024))) uint16_t g_k1[kTileElems];
__shared__ __attribute__((aligned(1024))) uint16_t g_v1[kTileElems];
__shared__ __attribute__((aligned(1024))) uint16_t g_k2[kTileElems];  // third stage: ping-pong ring only
__shared__ __attribute__((aligned(1024))) uint16_t g_v2[kTileElems];

template <int S>
__device__ __forceinline__ uint16_t* kbuf() {
  if constexpr (S == 0) return g_k0;
  else if constexpr (S == 1) return g_k1;
  else return g_k2;
}
template <int S>
__device__ __forceinline__ uint16_t* vbuf() {
  if constexpr (S == 0) return g_v0;
  else if constexpr (S == 1) return g_v1;
  else return g_v2;
}

// Work-group barrier without the memory fences of __syncthreads(): every
// wave first waits for its own LDS reads; the tile DMA is waited for
// explicitly (wait_tiles_in_flight) so that later tiles stay in flight.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

// 32-bit LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const uint16_t* ptr) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void*)ptr));
}

// One 16-byte-per-lane buffer load straight into LDS: lane l's bytes land at
// M0 + 16 l; offsets past the buffer's record count read as zeros.  Written
// as inline assembly so the compiler does no alias tracking of its own for
// these LDS writes (it would otherwise wait for every in-flight tile before
// unrelated LDS reads); the kernel waits for the loads explicitly with
// vmcnt.  M0 needs one wait state before the load.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, __amdgpu_buffer_rsrc_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}

// Issue the direct global->LDS loads of one K/V tile.  The tile is
// kBN rows x D/8 16-byte granules; wave w's instruction i fills the 1 KB LDS
// chunk c = i * kWaves + w, lane l writing granule position p = 64 c + l (the
// hardware puts lane l's 16 bytes at chunk base + 16 l).  Position p holds
// row p / (D/8), swizzled slot p % (D/8); the per-lane byte offsets `voff`
// are fixed for the whole kernel.  Rows past the range end lie beyond the
// buffer record count and arrive as zeros.
template <int D>
__device__ __forceinline__ void issue_tile(const Cursor& c, int wave, const uint32_t* voff0, const uint32_t* voff1,
                                           uint16_t* ks, uint16_t* vs) {
  constexpr int kLoads = kBN * (D / 8) / kThreads;
  // record count: at most 64 tokens of at most 2^25 bytes (the stride limit
  // the API enforces), i.e. at most 2^31, which fits the unsigned 32-bit field
  const uint32_t nrec = uint32_t(min(kBN, c.rem)) * uint32_t(c.st);
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.k, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.v, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  // the lane offsets are passed straight from the long-lived per-source
  // registers (a uniform branch, not a select into a temporary)
  if (c.src == 0) {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int chunk = i * kWaves + wave;
      dma16(lds_addr(ks + chunk * 512), voff0[i], rk);
      dma16(lds_addr(vs + chunk * 512), voff0[i], rv);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int chunk = i * kWaves + wave;
      dma16(lds_addr(ks + chunk * 512), voff1[i], rk);
      dma16(lds_addr(vs + chunk * 512), voff1[i], rv);
    }
  }
}

__device__ __forceinline__ int tile_valid(const Cursor& c) { return min(kBN, c.rem); }

// ---------------------------------------------------------------- tile compute
// A wave owns QB blocks of 32 query rows.  Every K or V^T fragment it reads
// from LDS feeds one MFMA per block, so two blocks halve the LDS bytes per
// MFMA.  With two blocks the score accumulators of both must fit next to the
// output accumulators within the register budget of two waves per SIMD, so a
// 64-key tile is computed as two 32-key sub-tiles (QK^T, softmax, PV each).
template <int QB>
struct Blk {
  static constexpr int kSub = QB == 1 ? kBN : 32;  // keys per sub-tile
  static constexpr int kKB = kSub / 32;            // 32-key blocks per sub-tile
  static constexpr int kPF = 3;                    // fragment reads in flight ahead of their MFMAs
  static constexpr int kRows = 32 * QB * kWaves;   // query rows per work-group
};

// Scheduling fence: the compiler moves no instruction across it, so the
// software-pipelined order below (reads issued kPF fragments ahead) stays.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Per-lane LDS byte offsets of the fragment reads inside a tile.  The swizzle
// XORs granule bits with row bits, so a fragment's address is the lane's base
// XOR a compile-time constant (the XOR touches only in-row bits), plus a
// constant row offset that the LDS instruction's offset field absorbs.
struct FragBase {
  uint32_t k;       // K fragment: row lane%32, granule lane/32
  uint32_t v0, v1;  // V^T fragment: the two transpose reads (rows r0 and r0 + 8)
};

template <int D>
__device__ __forceinline__ FragBase frag_base(int lane) {
  constexpr int GR = D / 8;
  const int hh = lane >> 5, li = lane & 15;
  FragBase fb;
  {
    const int row = lane & 31;
    const int x = (((row & 3) << 2) | ((row >> 2) & 3)) & (GR - 1);
    fb.k = uint32_t(row * D * 2 + 16 * (x ^ hh));  // granule 2 dc + hh = (2 dc) ^ hh
  }
  // V^T: rows r0 = 4 hh + li/4 (+ 8), d = 16 ((lane/16)&1) + 4 (li%4) inside a
  // 32-wide block: granule c = 2 ((lane/16)&1) + (li%4)/2, element 4 (li%2)
  const int c = 2 * ((lane >> 4) & 1) + ((li & 3) >> 1);
  const int r0 = 4 * hh + (li >> 2), r1 = r0 + 8;
  const int x0 = (((r0 & 3) << 2) | ((r0 >> 2) & 3)) & (GR - 1);
  const int x1 = (((r1 & 3) << 2) | ((r1 >> 2) & 3)) & (GR - 1);
  fb.v0 = uint32_t(r0 * D * 2 + 16 * (c ^ x0) + 8 * (li & 1));
  fb.v1 = uint32_t(r1 * D * 2 + 16 * (c ^ x1) + 8 * (li & 1));
  return fb;
}

// The fragment bases of one compute phase.  They are hidden from
// loop-invariant code motion, so each phase recomputes its fragment addresses
// (one XOR per read) instead of keeping all of them live in registers.
template <int D>
__device__ __forceinline__ FragBase phase_base(int lane) {
  FragBase fb = frag_base<D>(lane);
  asm volatile("" : "+v"(fb.k), "+v"(fb.v0), "+v"(fb.v1));
  return fb;
}

// K fragment f = kb * NDC + dc of S^T = K Q^T: rows kb*32 + lane%32 of the
// tile, granule 2 dc + lane/32.
template <int D>
__device__ __forceinline__ bf16x8 k_frag(const uint16_t* ks, const FragBase& fb, int f) {
  constexpr int NDC = D / 16;
  const int kb = f / NDC, dc = f % NDC;
  const char* p = reinterpret_cast<const char*>(ks) + (fb.k ^ uint32_t(32 * dc)) + kb * 32 * D * 2;
  return *reinterpret_cast<const bf16x8*>(p);
}

// S^T = K Q^T for sub-tile j (kKB 32x32 accumulators per query block);
// src.k(f) reads K fragment f of the stage.
template <int D, int QB, class Src>
__device__ __forceinline__ void s_part(const Src& src, int j, const bf16x8 (&qf)[QB][D / 16],
                                       f32x16 (&sacc)[QB][Blk<QB>::kKB]) {
  constexpr int KB = Blk<QB>::kKB;
  constexpr int NDC = D / 16;
  constexpr int NF = KB * NDC;
  constexpr int PF = Blk<QB>::kPF;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[qb][kb][r] = 0.f;
  bf16x8 a[PF + 1];
#pragma unroll
  for (int f = 0; f < PF && f < NF; ++f) a[f] = src.k(j * NF + f);
  sched_fence();
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int kb = f / NDC, dc = f % NDC;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
      sacc[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[f % (PF + 1)], qf[qb][dc], sacc[qb][kb], 0, 0, 0);
    if (f + PF < NF) a[(f + PF) % (PF + 1)] = src.k(j * NF + f + PF);
    sched_fence();
  }
}

// Online softmax of one S^T sub-tile, in three parts per query block (row =
// this lane's query): the tile's row max, the lazy rescale, and P^T = exp2 in
// bf16 with the row sum.
//
// Row max of one block's sub-tile in log2 units (c: the factor from
// accumulator units to log2 units).  Keys past the end of the range (valid:
// keys of the sub-tile inside the range) score -inf first: slot r of half hh
// holds key kb*32 + 8 (r/4) + 4 hh + r%4, so the lane-independent part is
// compared against valid - 4 hh.
template <int KB>
__device__ __forceinline__ float tile_max(int lane, int valid, f32x16 (&sacc)[KB], float c) {
  if (valid < 32 * KB) {
    const int lim = valid - 4 * (lane >> 5);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + 8 * (r >> 2) + (r & 3);
        if (key >= lim) sacc[kb][r] = -INFINITY;
      }
  }
  float mx = sacc[0][0];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
  return max_halves(mx) * c;
}

// Move the running max to max(m_used, mt): exact, since the same factor
// scales the row sum and the accumulator.
template <int D>
__device__ __forceinline__ void rescale(f32x16 (&oacc)[D / 32], float& m_used, float& lsum, float mt) {
  const float m_new = fmaxf(m_used, mt);
  const float alpha = __builtin_amdgcn_exp2f(m_used - m_new);
  lsum *= alpha;
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[nb][r] *= alpha;
  m_used = m_new;
}

// p = 2^(s c - m_used) into P^T (bf16, the B operand of the P V MFMAs) and
// the unrounded sum.
template <int KB>
__device__ __forceinline__ void exp_part(const f32x16 (&sacc)[KB], bf16x8 (&pf)[2 * KB], float m_used, float& lsum,
                                         float c) {
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][r], c, -m_used));
      lsum += e;
      pf[kb * 2 + (r >> 3)][r & 7] = (__bf16)e;
    }
}

// All query blocks of a sub-tile.  The running max is refreshed lazily, only
// when some row's tile max exceeds it by more than 2^8; one wave-uniform
// branch covers all blocks (a block whose max did not grow is rescaled too,
// by 1 or by the exact factor).  A sub-tile whose keys all lie past the range
// end (valid <= 0) contributes p = 0 once the running max is finite, which
// the first sub-tile of a segment's keys (valid >= 1) guarantees.
template <int D, int QB>
__device__ __forceinline__ void softmax_part(int lane, int valid, f32x16 (&sacc)[QB][Blk<QB>::kKB],
                                             bf16x8 (&pf)[QB][2 * Blk<QB>::kKB], f32x16 (&oacc)[QB][D / 32],
                                             float (&m_used)[QB], float (&lsum)[QB], const float (&c)[QB]) {
  float mt[QB];
  bool grow = false;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    mt[qb] = tile_max(lane, valid, sacc[qb], c[qb]);
    grow = grow || mt[qb] > m_used[qb] + kLazyThreshold;
  }
  if (__any(grow)) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) rescale<D>(oacc[qb], m_used[qb], lsum[qb], mt[qb]);
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) exp_part(sacc[qb], pf[qb], m_used[qb], lsum[qb], c[qb]);
}

// Optimistic online softmax of one 32-key sub-tile for both query blocks of
// a wave, used by the ping-pong ring.  Its VALU work issues while the other
// wave of the SIMD runs its MFMAs, provided it holds no instruction that
// waits for the matrix unit: v_dot2_f32_bf16 is one (it does not issue while
// an MFMA is in flight, so a stream of the other wave's MFMAs stalls it), so
// the row sums use plain fp32 adds.  The common case does no max reduction:
// the arguments a = s c - m_used for both blocks (in place), then p = 2^a
// packed to bf16 P^T, and the row sum of the fp32 weights in four
// independent chains.  If some lane's partial sum leaves [0, 2^16] or is not a
// number, the running max moves up by max(0, max a) and the weights are
// recomputed from the shifted arguments (exact up to one fp32 rounding of the
// argument).  So every weight stays below 2^16 and the fp32 accumulators
// cannot overflow.  The first sub-tile of a query tile (m_used = -inf) takes
// the exact path up front: tile max, then the weights.
constexpr float kSumLimit = 65536.f;

// p = 2^a for one block into P^T (bf16); returns the per-lane fp32 sum of p
// in four independent chains of plain adds.  (v_dot2_f32_bf16 would sum the
// rounded values in half the instructions, but it does not issue while an
// MFMA of the SIMD is in flight.)
__device__ __forceinline__ float pack_sum(const f32x16& arg, bf16x8 (&pf)[2]) {
  float e[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    e[r] = __builtin_amdgcn_exp2f(arg[r]);
    pf[r >> 3][r & 7] = (__bf16)e[r];
  }
  float a[4] = {e[0], e[1], e[2], e[3]};
#pragma unroll
  for (int r = 4; r < 16; ++r) a[r & 3] += e[r];
  return (a[0] + a[1]) + (a[2] + a[3]);
}

template <int D>
__device__ __forceinline__ void softmax_pp(int lane, int valid, bool first, f32x16 (&sacc)[2][1],
                                           bf16x8 (&pf)[2][2], f32x16 (&oacc)[2][D / 32], float (&m_used)[2],
                                           float (&lsum)[2], const float (&c)[2]) {
  if (valid < 32) {  // keys past the range end score -inf (see tile_max)
    const int lim = valid - 4 * (lane >> 5);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (8 * (r >> 2) + (r & 3) >= lim) sacc[qb][0][r] = -INFINITY;
  }
  if (first) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) rescale<D>(oacc[qb], m_used[qb], lsum[qb], tile_max(lane, 32, sacc[qb], c[qb]));
  }
  // the arguments of both blocks first (independent), then one block at a
  // time, so that a block's arguments die at its check
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[qb][0][r] = __builtin_fmaf(sacc[qb][0][r], c[qb], -m_used[qb]);
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float ts = pack_sum(sacc[qb][0], pf[qb]);
    if (__any(!(ts <= kSumLimit))) {
      float mx = 0.f;  // the shift: max(0, max a) over the row
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[qb][0][r]);
      mx = max_halves(mx);
      rescale<D>(oacc[qb], m_used[qb], lsum[qb], m_used[qb] + mx);
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[qb][0][r] -= mx;
      ts = pack_sum(sacc[qb][0], pf[qb]);
    }
    lsum[qb] += ts;
  }
}

// V^T fragment f = cc * NB + nb of O^T += V^T P^T: two transpose reads of V
// rows 16 cc + 4 (lane/32) + (lane%16)/4 (and 8 rows further) at
// d = 32 nb + 16 ((lane/16)&1) + 4 (lane%4) .. +3, matching the key order of
// P^T in the S^T accumulator.  Granule 4 nb + c = (4 nb) ^ c, so block nb is
// the base XOR 64 nb bytes.
template <int D>
__device__ __forceinline__ bf16x8 v_frag(const uint16_t* vs, const FragBase& fb, int f) {
  constexpr int NB = D / 32;
  const int cc = f / NB, nb = f % NB;
  const char* base = reinterpret_cast<const char*>(vs) + cc * 16 * D * 2;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + (fb.v0 ^ uint32_t(64 * nb))));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + (fb.v1 ^ uint32_t(64 * nb))));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Fragments of one ring stage from its pointers and the lane's per-phase
// bases (the two-block kernels).
template <int D>
struct PtrFrags {
  const uint16_t* ks;
  const uint16_t* vs;
  FragBase fb;
  __device__ __forceinline__ bf16x8 k(int f) const { return k_frag<D>(ks, fb, f); }
  __device__ __forceinline__ bf16x8 v(int f) const { return v_frag<D>(vs, fb, f); }
};

// Absolute LDS byte addresses of one stage's fragment reads for one lane:
// K fragment of d chunk dc at k[dc] (+ 32 D 2 bytes per 32-key block), the
// two V^T reads of d block nb at v0[nb] and v1[nb] (+ 16 D 2 bytes per 16
// keys).  The one-block rings compute them once per ring and keep them in
// registers, which they have to spare; every remaining offset (at most
// 12 KB) then fits the LDS read's 16-bit offset field wherever the stage lies.
template <int D>
struct StageAddr {
  uint32_t k[D / 16];
  uint32_t v0[D / 32], v1[D / 32];
};

template <int D>
__device__ __forceinline__ StageAddr<D> stage_addr(int lane, const uint16_t* ks, const uint16_t* vs) {
  const FragBase fb = frag_base<D>(lane);
  StageAddr<D> a;
#pragma unroll
  for (int dc = 0; dc < D / 16; ++dc) a.k[dc] = lds_addr(ks) + (fb.k ^ uint32_t(32 * dc));
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb) {
    a.v0[nb] = lds_addr(vs) + (fb.v0 ^ uint32_t(64 * nb));
    a.v1[nb] = lds_addr(vs) + (fb.v1 ^ uint32_t(64 * nb));
  }
  // opaque to the optimiser, which would otherwise split the stage base back
  // out and fold it with the fragment offset (past the offset field's range
  // for stages high in LDS)
#pragma unroll
  for (int dc = 0; dc < D / 16; ++dc) asm volatile("" : "+v"(a.k[dc]));
#pragma unroll
  for (int nb = 0; nb < D / 32; ++nb) asm volatile("" : "+v"(a.v0[nb]), "+v"(a.v1[nb]));
  return a;
}

template <int D>
struct AddrFrags {
  const StageAddr<D>& a;
  __device__ __forceinline__ bf16x8 k(int f) const {
    constexpr int NDC = D / 16;
    const int kb = f / NDC, dc = f % NDC;
    return *reinterpret_cast<lds_cbf16x8*>(reinterpret_cast<lds_cchar*>(uintptr_t(a.k[dc])) + kb * 32 * D * 2);
  }
  __device__ __forceinline__ bf16x8 v(int f) const {
    constexpr int NB = D / 32;
    const int cc = f / NB, nb = f % NB;
    const int off = cc * 16 * D * 2;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(reinterpret_cast<lds_cchar*>(uintptr_t(a.v0[nb])) + off));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(reinterpret_cast<lds_cchar*>(uintptr_t(a.v1[nb])) + off));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }
};

// O^T += V^T P^T for sub-tile j: 16 keys per MFMA, 32 d-rows per MFMA;
// src.v(f) reads V^T fragment f of the stage.
template <int D, int QB, class Src>
__device__ __forceinline__ void pv_part(const Src& src, int j, const bf16x8 (&pf)[QB][2 * Blk<QB>::kKB],
                                        f32x16 (&oacc)[QB][D / 32]) {
  constexpr int NB = D / 32;
  constexpr int NF = 2 * Blk<QB>::kKB * NB;
  constexpr int PF = Blk<QB>::kPF;
  bf16x8 a[PF + 1];
#pragma unroll
  for (int f = 0; f < PF && f < NF; ++f) a[f] = src.v(j * NF + f);
  sched_fence();
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int cc = f / NB, nb = f % NB;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
      oacc[qb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[f % (PF + 1)], pf[qb][cc], oacc[qb][nb], 0, 0, 0);
    if (f + PF < NF) a[(f + PF) % (PF + 1)] = src.v(j * NF + f + PF);
    sched_fence();
  }
}

// One 64-key tile for one wave, all phases back to back: per sub-tile
// S^T = K Q^T, online softmax, O^T += V^T P^T.  A sub-tile wholly past the
// range end is skipped (valid is wave-uniform).
template <int D, int QB>
__device__ __forceinline__ void tile_compute(const StageAddr<D>& sa, int lane, int valid,
                                             const bf16x8 (&qf)[QB][D / 16], f32x16 (&oacc)[QB][D / 32],
                                             float (&m_used)[QB], float (&lsum)[QB], const float (&c)[QB]) {
  constexpr int SUB = Blk<QB>::kSub, KB = Blk<QB>::kKB;
  const AddrFrags<D> src{sa};
#pragma unroll
  for (int j = 0; j < kBN / SUB; ++j) {
    if (j > 0 && valid <= j * SUB) break;
    f32x16 sacc[QB][KB];
    bf16x8 pf[QB][2 * KB];
    s_part<D, QB>(src, j, qf, sacc);
    softmax_part<D, QB>(lane, valid - j * SUB, sacc, pf, oacc, m_used, lsum, c);
    pv_part<D, QB>(src, j, pf, oacc);
  }
}

// ---------------------------------------------------------------- FP8 cache tiles
// Staging slots for the codes of a cache tile of the FP8 cache (64 key rows of
// D e4m3fn codes each for K8 and V8), which the ping-pong ring widens into
// its bf16 stages (see the ring below).
constexpr int kTile8Bytes = kBN * 128;  // bytes per K8 or V8 staging tile (D <= 128)
__shared__ __attribute__((aligned(1024))) char g_k8r[2][kTile8Bytes];
__shared__ __attribute__((aligned(1024))) char g_v8_0[kTile8Bytes];
__shared__ __attribute__((aligned(1024))) char g_v8_1[kTile8Bytes];

__device__ __forceinline__ uint32_t lds_addr8(const char* ptr) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void*)ptr));
}

// 16 codes (one 8-bit granule: d = 16 g .. 16 g + 15 of key row `row`) times
// the scale into bf16 granules 2 g and 2 g + 1 of that row of the bf16 tile.
template <int D>
__device__ __forceinline__ void widen_granule(const char* src8, uint16_t* dst, int p, float s) {
  constexpr int GR8 = D / 16, GR = D / 8;
  const u32x4 w = *reinterpret_cast<const u32x4*>(src8 + p * 16);
  uint32_t e[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    e[2 * j] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[j], s, false));
    e[2 * j + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[j], s, true));
  }
  const int row = p / GR8, g = p % GR8;
  *reinterpret_cast<u32x4*>(dst + row * D + swz(row, 2 * g, GR) * 8) = u32x4{e[0], e[1], e[2], e[3]};
  *reinterpret_cast<u32x4*>(dst + row * D + swz(row, 2 * g + 1, GR) * 8) = u32x4{e[4], e[5], e[6], e[7]};
}

// ---------------------------------------------------------------- one-block ring
// Every wave loads its share of each tile and computes it whole: per tile one
// barrier, then the refill of the stage the previous tile freed, then the
// tile's QK^T, softmax and PV.  Used with one query block per wave.

// Wait until at most `n` tiles of this wave's loads are still in flight
// (each tile is `per_tile` vector-memory instructions per wave).
template <int per_tile>
__device__ __forceinline__ void wait_tiles_in_flight(int n) {
  static_assert(2 * per_tile <= 63, "vmcnt range");
  if (n <= 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else if (n == 1) {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(per_tile) : "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * per_tile) : "memory");
  }
}

// State a wave carries through the K/V ring.
struct RingState {
  Cursor icur, ccur;  // next tile to issue, next tile to compute
  int issued;         // tiles issued so far (absolute key-tile index)
};

// Tile k (in stage S): wait for its DMA, barrier, refill the stage that
// became free with tile k + kStages - 1, then compute tile k.
template <int S, int D, int QB>
__device__ __forceinline__ void ring_step(const Params& p, int k, int kt_end, int wave, int lane, bool wave_active,
                                          const uint32_t* voff0, const uint32_t* voff1, const StageAddr<D>& sa,
                                          RingState& rs,
                                          const bf16x8 (&qf)[QB][D / 16], f32x16 (&oacc)[QB][D / 32],
                                          float (&m_used)[QB], float (&lsum)[QB], const float (&c)[QB]) {
  constexpr int kLoads = kBN * (D / 8) / kThreads;
  constexpr int F = (S + kStages - 1) % kStages;  // stage freed by the previous tile
  wait_tiles_in_flight<2 * kLoads>(rs.issued - 1 - k);
  ring_barrier();
  if (rs.issued < kt_end) {
    issue_tile<D>(rs.icur, wave, voff0, voff1, kbuf<F>(), vbuf<F>());
    ++rs.issued;
    if (rs.issued < kt_end) cursor_next(p, rs.icur);
  }
  const int valid = tile_valid(rs.ccur);
  if (wave_active) tile_compute<D, QB>(sa, lane, valid, qf, oacc, m_used, lsum, c);
  if (k + 1 < kt_end) cursor_next(p, rs.ccur);
}

// The K/V ring over key tiles [kt_begin, kt_end) of query segment qs: tile kt
// lives in stage (kt - kt_begin) % kStages; tiles up to kStages - 1 ahead are in
// flight while one is computed.
template <int D, int QB>
__device__ __forceinline__ void run_ring(const Params& p, const QSeg& qs, int b, int h, int kt_begin, int kt_end,
                                         int wave, int lane, bool wave_active, const uint32_t* voff0,
                                         const uint32_t* voff1, const bf16x8 (&qf)[QB][D / 16],
                                         f32x16 (&oacc)[QB][D / 32], float (&m_used)[QB], float (&lsum)[QB],
                                         const float (&c)[QB]) {
  if (kt_begin >= kt_end) return;
  const StageAddr<D> sa0 = stage_addr<D>(lane, kbuf<0>(), vbuf<0>());
  const StageAddr<D> sa1 = stage_addr<D>(lane, kbuf<1>(), vbuf<1>());
  RingState rs;
  rs.icur = cursor_at(p, qs, kt_begin, b, h);
  rs.ccur = rs.icur;
  rs.issued = kt_begin;
  if (rs.issued < kt_end) {
    issue_tile<D>(rs.icur, wave, voff0, voff1, kbuf<0>(), vbuf<0>());
    if (++rs.issued < kt_end) cursor_next(p, rs.icur);
  }
  for (int kt = kt_begin; kt < kt_end; kt += kStages) {
    ring_step<0, D, QB>(p, kt, kt_end, wave, lane, wave_active, voff0, voff1, sa0, rs, qf, oacc, m_used, lsum, c);
    if (kt + 1 >= kt_end) break;
    ring_step<1, D, QB>(p, kt + 1, kt_end, wave, lane, wave_active, voff0, voff1, sa1, rs, qf, oacc, m_used, lsum,
                        c);
  }
}

// ---------------------------------------------------------------- ping-pong ring
// With two query blocks per wave the two waves of each SIMD (waves w and w + 4
// of the work-group share a SIMD) run half a phase apart: a wave alternates
// an MFMA phase (P V of sub-tile u, then S^T of sub-tile u + 1) and a softmax
// phase (sub-tile u + 1), with a work-group barrier between phases, and group
// 1 (waves 4-7) starts one phase after group 0 (waves 0-3).  So while one
// wave of a SIMD issues MFMAs the other one does its exp2/max/sum work, and
// the two streams share the SIMD instead of taking turns.
//
// Group 1 alone loads the tiles (during its softmax phases), into a ring of
// three stages: tile t + 2 is issued at the first softmax phase of tile t
// (the stage of tile t - 1 is free by then for both groups), and group 1
// waits for tile t + 1 at the end of the MFMA phase that precedes group 0's
// first read of it.  Sub-tiles past the range end are computed with every
// key masked, so that both groups pass the same barriers.
constexpr int kLoaders = 4;  // waves of group 1

// The lane index computed afresh (v_mbcnt over a full mask) where it is
// needed: written as inline assembly so that the compiler neither hoists it
// out of the tile loop nor keeps it live across the phases, where a register
// is only to be had by spilling (a spilled lane index costs a scratch reload,
// a full memory latency, in the phase that issues the tile loads).
__device__ __forceinline__ int fresh_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Issue the loads of one K/V tile from the loader wave lw of group 1: its
// instruction i fills the 1 KB chunk c = i * 4 + lw of each tensor, lane l
// the granule position p = 64 c + l (row p / (D/8), swizzled slot).
template <int D>
__device__ __forceinline__ void issue_tile_pp(const Cursor& c, int lw, uint16_t* ks, uint16_t* vs) {
  constexpr int GR = D / 8;
  constexpr int kLoads = kBN * GR / (kLoaders * 64);
  const uint32_t nrec = uint32_t(min(kBN, c.rem)) * uint32_t(c.st);  // at most 2^31 (see issue_tile)
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.k, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.v, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  const uint32_t lane = uint32_t(fresh_lane());
#pragma unroll
  for (int i = 0; i < kLoads; ++i) {
    const int chunk = i * kLoaders + lw;
    const uint32_t pos = uint32_t(chunk * 64) + lane;
    const uint32_t row = pos / GR, slot = pos % GR;
    const uint32_t voff = row * uint32_t(c.st) + (slot ^ ((((row & 3u) << 2) | ((row >> 2) & 3u)) & (GR - 1))) * 16u;
    dma16(lds_addr(ks + chunk * 512), voff, rk);
    dma16(lds_addr(vs + chunk * 512), voff, rv);
  }
}

template <int D>
__device__ __forceinline__ void wait_tiles_pp(int n) {
  constexpr int kPerTile = 2 * (kBN * (D / 8) / (kLoaders * 64));
  static_assert(2 * kPerTile <= 63, "vmcnt range");
  if (n <= 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else if (n == 1) {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kPerTile) : "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kPerTile) : "memory");
  }
}

// Pin a phase's results before the barrier that ends it: the empty asm
// statement reads and rewrites the registers, so the compiler can neither sink
// their computation into the next phase nor start it early.
template <int QB, int KB>
__device__ __forceinline__ void pin_scores(f32x16 (&sacc)[QB][KB]) {
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) asm volatile("" : "+v"(sacc[qb][kb]));
}
template <int QB, int N>
__device__ __forceinline__ void pin_probs(bf16x8 (&pf)[QB][N], float (&m_used)[QB], float (&lsum)[QB]) {
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int i = 0; i < N; ++i) asm volatile("" : "+v"(pf[qb][i]));
    asm volatile("" : "+v"(m_used[qb]), "+v"(lsum[qb]));
  }
}

// The MFMA phase of the ping-pong ring as one stream of fragment reads: the
// 2 NB V^T fragments of sub-tile jv (O^T += V^T P^T), then the NDC K
// fragments of sub-tile jk of ks (S^T = K Q^T), each read kPF fragments ahead
// of its MFMAs, so that the first K reads are in flight during the last P V
// MFMAs.  The first kPF V^T fragments arrive in a[] (v_prefetch), read at the
// end of the softmax phase before, so that the phase's first MFMAs do not wait
// for the LDS.
template <int D>
__device__ __forceinline__ void v_prefetch(const uint16_t* vs, const FragBase& fb, int jv, bf16x8 (&a)[4]) {
  constexpr int NV = D / 16;  // 2 NB
#pragma unroll
  for (int f = 0; f < Blk<2>::kPF; ++f) a[f] = v_frag<D>(vs, fb, jv * NV + f);
}

template <int D>
__device__ __forceinline__ void mfma_phase(const uint16_t* vs, const uint16_t* ks, const FragBase& fb, int jv, int jk,
                                           bf16x8 (&a)[4], const bf16x8 (&pf)[2][2], const bf16x8 (&qf)[2][D / 16],
                                           f32x16 (&oacc)[2][D / 32], f32x16 (&sacc)[2][1]) {
  constexpr int NB = D / 32, NDC = D / 16, NV = 2 * NB, NF = NV + NDC;
  constexpr int PF = Blk<2>::kPF;
  static_assert(PF + 1 == 4 && NV >= PF, "fragment ring of four");
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    if (f < NV) {
      const int cc = f / NB, nb = f % NB;
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        oacc[qb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[f % 4], pf[qb][cc], oacc[qb][nb], 0, 0, 0);
    } else {
      const int dc = f - NV;
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        sacc[qb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[f % 4], qf[qb][dc], dc == 0 ? f32x16{} : sacc[qb][0],
                                                              0, 0, 0);
    }
    const int g = f + PF;
    if (g < NV) a[g % 4] = v_frag<D>(vs, fb, jv * NV + g);
    else if (g < NF) a[g % 4] = k_frag<D>(ks, fb, jk * NDC + g - NV);
    sched_fence();
  }
}

// Barrier that starts an MFMA phase of the ping-pong ring.  The wave's LDS
// reads still in flight are the phase's first V^T fragments, of the tile
// being computed, which no load issued after this barrier overwrites (the
// loads after a barrier refill the stage of the tile before), so unlike
// ring_barrier it does not wait for them.  The empty asm statement keeps the
// reads before the barrier.
__device__ __forceinline__ void mfma_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

struct PPState {
  Cursor icur;  // next tile to load (group 1)
  Cursor ccur;  // tile being computed
  int issued;   // tiles loaded so far (group 1), counted from the first
  int n;        // tiles of the range
  float sk, sv; // FP8 cache ring: the (batch, head)'s K and V scales
};

// ------------------------------------------------ FP8 cache tiles in the ping-pong ring
// A cache tile (64 rows of D e4m3 codes each for K8 and V8, rows D bytes
// apart) reaches the ring in two steps, both by group 1: its codes are loaded
// into one of two staging slots, and one tile later widened (times the
// power-of-two scales: exact) into the tile's bf16 ring stage, in the layout a
// fresh tile has, at the end of group 1's first softmax phase of the tile two
// before it.  From there on it is a bf16 tile.  Tile t + 3 loads into the slot
// tile t + 1 left, while tile t + 2 is widened out of the other one.
template <int D>
constexpr int kChunks8pp = kBN * D / 1024;  // 1 KB chunks of a K8 or V8 tile
template <int D>
constexpr int kLoads8pp = 2 * kChunks8pp<D> / kLoaders;  // loads per wave per tile (K8 and V8)

// The FP8 ring's wait: at most n tiles' 8-bit loads of this wave in flight.
template <int D>
__device__ __forceinline__ void wait_tiles_pp8(int n) {
  static_assert(kLoads8pp<D> <= 63, "vmcnt range");
  if (n <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLoads8pp<D>) : "memory");
}

template <int D>
__device__ __forceinline__ void issue_tile8_pp(const Cursor& c, int lw, int slot) {
  static_assert(kChunks8pp<D> % kLoaders == 0, "chunks divide over the loader waves");
  const uint32_t nrec = uint32_t(min(kBN, c.rem)) * uint32_t(c.st);  // c.st = D bytes: at most 2^13
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.k, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void*)c.v, (short)0, __builtin_bit_cast(int, nrec), 0x00020000);
  char* k8 = g_k8r[slot];
  char* v8 = slot ? g_v8_1 : g_v8_0;
  const uint32_t lane = uint32_t(fresh_lane());
#pragma unroll
  for (int i = 0; i < kChunks8pp<D> / kLoaders; ++i) {
    const int ch = i * kLoaders + lw;
    const uint32_t voff = uint32_t(ch * 1024) + lane * 16u;
    dma16(lds_addr8(k8 + ch * 1024), voff, rk);
    dma16(lds_addr8(v8 + ch * 1024), voff, rv);
  }
}

// Widen staging slot `slot` into bf16 stage S: lane l of loader wave lw takes
// the 8-bit granules lw * 64 + l + 256 i of K8 and of V8.
template <int S, int D>
__device__ __forceinline__ void widen_tile_pp(int lw, int slot, float sk, float sv) {
  constexpr int NG = kBN * (D / 16);
  static_assert(NG % (kLoaders * 64) == 0, "granules divide over the loader lanes");
  const char* k8 = g_k8r[slot];
  const char* v8 = slot ? g_v8_1 : g_v8_0;
  const int lane = fresh_lane();
#pragma unroll
  for (int i = 0; i < NG / (kLoaders * 64); ++i) {
    const int pos = i * kLoaders * 64 + lw * 64 + lane;
    widen_granule<D>(k8, kbuf<S>(), pos, sk);
    sched_fence();
    widen_granule<D>(v8, vbuf<S>(), pos, sv);
    sched_fence();
  }
}

// The four phases of tile t (stage S): softmax of sub-tile 2t, MFMA phase
// (P V of 2t, S^T of 2t + 1), softmax of 2t + 1, MFMA phase (P V of 2t + 1,
// S^T of sub-tile 0 of tile t + 1 in stage (S + 1) % 3).  A wave raises its issue
// priority for its MFMA phases, so that the other wave's softmax instructions
// fill the gaps between its MFMAs rather than delay them (measured 1-2.5%
// faster than equal priorities or a raised softmax phase).  In the FP8 ring
// each phase takes the lane index afresh (fresh_lane): with the widening's
// registers it would otherwise be spilled and reloaded once per tile.
template <int S, int D, bool kF8>
__device__ __forceinline__ void pp_tile(const Params& p, int t, PPState& st, int grp, int lw, int lane,
                                        const bf16x8 (&qf)[2][D / 16], f32x16 (&oacc)[2][D / 32],
                                        float (&m_used)[2], float (&lsum)[2], const float (&c)[2],
                                        f32x16 (&sacc)[2][1], bf16x8 (&pf)[2][2]) {
  constexpr int SN = (S + 1) % 3;  // stage of tile t + 1
  constexpr int SL = (S + 2) % 3;  // stage of tile t - 1, refilled with tile t + 2
  const int valid = tile_valid(st.ccur);
  // softmax of sub-tile 2t; group 1 loads tile t + 2
  ring_barrier();
  __builtin_amdgcn_s_setprio(0);
  if constexpr (kF8) {
    // the codes of tile t + 3 into the slot tile t + 1 left
    if (grp == 1 && t + 3 < st.n) {
      issue_tile8_pp<D>(st.icur, lw, (t + 3) & 1);
      if (t + 4 < st.n) cursor_next(p, st.icur);
    }
  } else if (grp == 1 && t >= 1 && t + 2 < st.n) {
    issue_tile_pp<D>(st.icur, lw, kbuf<SL>(), vbuf<SL>());
    ++st.issued;
    if (t + 3 < st.n) cursor_next(p, st.icur);
  }
  softmax_pp<D>(kF8 ? fresh_lane() : lane, valid, t == 0, sacc, pf, oacc, m_used, lsum, c);
  pin_probs(pf, m_used, lsum);
  if constexpr (kF8) {
    // tile t + 2 (its codes landed; tile t + 3's may be in flight) widened into
    // the stage of tile t - 1, which no wave reads any more
    if (grp == 1 && t + 2 < st.n) {
      if (t + 3 < st.n) wait_tiles_pp8<D>(1);
      else wait_tiles_pp8<D>(0);
      sched_fence();
      widen_tile_pp<SL, D>(lw, (t + 2) & 1, st.sk, st.sv);
    }
  }
  // P V of sub-tile 2t, S^T of sub-tile 2t + 1; group 1 then waits for tile t + 1
  {
    sched_fence();
    const FragBase fb = phase_base<D>(kF8 ? fresh_lane() : lane);
    bf16x8 a[4];
    v_prefetch<D>(vbuf<S>(), fb, 0, a);
    sched_fence();
    mfma_barrier();
    __builtin_amdgcn_s_setprio(3);
    mfma_phase<D>(vbuf<S>(), kbuf<S>(), fb, 0, 1, a, pf, qf, oacc, sacc);
    pin_scores(sacc);
  }
  if (!kF8 && grp == 1 && t + 1 < st.n) wait_tiles_pp<D>(st.issued - (t + 2));
  // softmax of sub-tile 2t + 1
  ring_barrier();
  __builtin_amdgcn_s_setprio(0);
  softmax_pp<D>(kF8 ? fresh_lane() : lane, valid - 32, false, sacc, pf, oacc, m_used, lsum, c);
  pin_probs(pf, m_used, lsum);
  // P V of sub-tile 2t + 1, S^T of the next tile's first sub-tile (after the
  // last tile it reads a stage that holds no new tile and the scores go
  // unused; computing it anyway keeps the old scores from living across this
  // phase)
  {
    sched_fence();
    const FragBase fb = phase_base<D>(kF8 ? fresh_lane() : lane);
    bf16x8 a[4];
    v_prefetch<D>(vbuf<S>(), fb, 1, a);
    sched_fence();
    mfma_barrier();
    __builtin_amdgcn_s_setprio(3);
    mfma_phase<D>(vbuf<S>(), kbuf<SN>(), fb, 1, 0, a, pf, qf, oacc, sacc);
    pin_scores(sacc);
  }
  if (t + 1 < st.n) cursor_next(p, st.ccur);
}

template <int D, bool kF8 = false>
__device__ __forceinline__ void run_ring_pp(const Params& p, const QSeg& qs, int b, int h, int kt_begin, int kt_end,
                                            int wave, int lane, const bf16x8 (&qf)[2][D / 16],
                                            f32x16 (&oacc)[2][D / 32], float (&m_used)[2], float (&lsum)[2],
                                            const float (&c)[2], float sk = 1.f, float sv = 1.f) {
  const int n = kt_end - kt_begin;  // the same for every wave of the work-group
  if (n <= 0) return;
  const int grp = wave >> 2, lw = wave & 3;
  PPState st;
  st.n = n;
  st.ccur = cursor_at(p, qs, kt_begin, b, h);
  st.icur = st.ccur;
  st.issued = 0;
  st.sk = sk;
  st.sv = sv;
  if (kF8 && grp == 1) {
    // tiles 0 and 1 loaded and widened into stages 0 and 1; tile 2's codes
    // then load into slot 0, whose widening reads are done
    issue_tile8_pp<D>(st.icur, lw, 0);
    if (n > 1) {
      cursor_next(p, st.icur);
      issue_tile8_pp<D>(st.icur, lw, 1);
      wait_tiles_pp8<D>(1);
    } else {
      wait_tiles_pp8<D>(0);
    }
    widen_tile_pp<0, D>(lw, 0, sk, sv);
    if (n > 1) {
      wait_tiles_pp8<D>(0);
      widen_tile_pp<1, D>(lw, 1, sk, sv);
    }
    if (n > 2) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      cursor_next(p, st.icur);
      issue_tile8_pp<D>(st.icur, lw, 0);
      if (n > 3) cursor_next(p, st.icur);
    }
  } else if (grp == 1) {
    issue_tile_pp<D>(st.icur, lw, kbuf<0>(), vbuf<0>());
    st.issued = 1;
    if (n > 1) {
      cursor_next(p, st.icur);
      issue_tile_pp<D>(st.icur, lw, kbuf<1>(), vbuf<1>());
      st.issued = 2;
      if (n > 2) {
        cursor_next(p, st.icur);
        issue_tile_pp<D>(st.icur, lw, kbuf<2>(), vbuf<2>());
        st.issued = 3;
        if (n > 3) cursor_next(p, st.icur);
      }
    }
    wait_tiles_pp<D>(st.issued - 1);  // tile 0 landed
  }
  ring_barrier();
  if (grp == 1) ring_barrier();  // group 1 runs one phase behind group 0
  f32x16 sacc[2][1];
  bf16x8 pf[2][2];
  s_part<D, 2>(PtrFrags<D>{kbuf<0>(), vbuf<0>(), phase_base<D>(lane)}, 0, qf, sacc);
  pin_scores(sacc);
  for (int t = 0; t < n; t += 3) {
    pp_tile<0, D, kF8>(p, t, st, grp, lw, lane, qf, oacc, m_used, lsum, c, sacc, pf);
    if (t + 1 >= n) break;
    pp_tile<1, D, kF8>(p, t + 1, st, grp, lw, lane, qf, oacc, m_used, lsum, c, sacc, pf);
    if (t + 2 >= n) break;
    pp_tile<2, D, kF8>(p, t + 2, st, grp, lw, lane, qf, oacc, m_used, lsum, c, sacc, pf);
  }
  if (grp == 0) ring_barrier();  // the barrier group 1 passed at the start
}

// Logical work-group index: the hardware deals blocks round-robin to the 8
// XCDs; remap so that each XCD receives a contiguous run of logical indices,
// i.e. neighbouring work items (the query tiles of one head, which stream the
// same K/V) share one XCD's L2.
__device__ __forceinline__ int xcd_logical_block(int bid, int nblk) {
  const int xcd = bid & 7, kx = bid >> 3, per = nblk >> 3, rem = nblk & 7;
  return (xcd < rem) ? xcd * (per + 1) + kx : rem * (per + 1) + (xcd - rem) * per + kx;
}

// One query tile t of segment qs, batch b, head h, over the segment's key
// tiles [kt_begin, kt_end).  part_row < 0: final output (bf16 O and LSE);
// otherwise unnormalised fp32 partials (O, running max in log2 units, row
// sum) at workspace row part_row + (row inside the tile).  Wave w owns rows
// w * 32 QB .. + 32 QB - 1 of the tile, block qb of it rows
// w * 32 QB + 32 qb + lane % 32.
template <int D, bool kF8, int QB>
__device__ __forceinline__ void attend_tile(const Params& p, const QSeg& qs, int t, int b, int h, int kt_begin,
                                            int kt_end, int64_t part_row, int wave, int lane) {
  constexpr int GR = D / 8;
  constexpr int NDC = D / 16;  // 16-wide d chunks of the QK^T contraction
  constexpr int NB = D / 32;   // 32-wide d blocks of the output
  constexpr int kLoads = kBN * GR / kThreads;
  constexpr int BM = Blk<QB>::kRows;
  constexpr int RW = 32 * QB;  // query rows per wave
  constexpr bool kPingPong = QB == 2;
  static_assert(kLoads >= 1 && kBN * GR % kThreads == 0, "tile granules must divide over the threads");
  static_assert(!kPingPong || kWaves == 2 * kLoaders, "ping-pong pairs waves w and w + 4 on one SIMD");
  const int hh = lane >> 5;  // which 32-lane half

  const int seg_row0 = (t - qs.tile0) * BM;
  const int rows_valid = min(BM, qs.len - seg_row0);
  const int row0 = qs.row0 + seg_row0;  // first row of the tile in the Q/O buffers
  const bool wave_active = wave * RW < rows_valid;  // wave-uniform

  // ---- Q fragments (B operand of S^T = K Q^T): in block qb, lane holds
  // query (lane % 32), d = 16*dc + 8*hh .. +7.
  int my_row[QB];
  bool row_ok[QB];
  bf16x8 qf[QB][NDC];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    my_row[qb] = wave * RW + 32 * qb + (lane & 31);
    row_ok[qb] = my_row[qb] < rows_valid;
    const uint16_t* qp =
        p.q + int64_t(b) * p.q_sb + int64_t(row0 + my_row[qb]) * p.q_st + int64_t(h) * D + hh * 8;
#pragma unroll
    for (int dc = 0; dc < NDC; ++dc) {
      u32x4 raw = row_ok[qb] ? *reinterpret_cast<const u32x4*>(qp + dc * 16) : u32x4{0u, 0u, 0u, 0u};
      qf[qb][dc] = __builtin_bit_cast(bf16x8, raw);
    }
  }
  // Q in registers before any tile DMA is counted; a compiler-visible wait
  // (gfx9 encoding of vmcnt(0) with expcnt/lgkmcnt left at their maxima) so
  // that no further waits for these loads are inserted inside the loop
  __builtin_amdgcn_s_waitcnt(0x0F70);

  f32x16 oacc[QB][NB];
  float m_used[QB], lsum[QB], cb[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[qb][nb][r] = 0.f;
    m_used[qb] = -INFINITY;  // running max in log2 units
    lsum[qb] = 0.f;          // this half's partial row sum
    cb[qb] = p.scale_log2;
  }

  if constexpr (kPingPong) {
    // every wave computes (a wave past the tile's rows holds zero queries and
    // stores nothing): keeping the phases unconditional lets the score and
    // P registers die at each phase instead of living across the next one
    if constexpr (kF8) {
      // the planner puts this segment's fresh (bf16) key ranges before its
      // FP8 cache ranges: the bf16 ring over the first, the widening ring over
      // the rest
      int kt_split = 0;
      for (int r = qs.r0; r < qs.r0 + qs.nr && p.range[r].src == 0; ++r) kt_split += p.range[r].ntiles;
      const int mid = min(max(kt_split, kt_begin), kt_end);
      run_ring_pp<D>(p, qs, b, h, kt_begin, mid, wave, lane, qf, oacc, m_used, lsum, cb);
      if (mid < kt_end) {
        if (kt_begin < mid) ring_barrier();  // the first ring's stages are read no more
        const float sk = p.kv_scale[(int64_t(b) * p.H + h) * 2];
        const float sv = p.kv_scale[(int64_t(b) * p.H + h) * 2 + 1];
        run_ring_pp<D, true>(p, qs, b, h, mid, kt_end, wave, lane, qf, oacc, m_used, lsum, cb, sk, sv);
      }
    } else {
      run_ring_pp<D>(p, qs, b, h, kt_begin, kt_end, wave, lane, qf, oacc, m_used, lsum, cb);
    }
  } else {
    // per-lane byte offsets of this lane's granules inside a tile, per key source
    uint32_t voff0[kLoads], voff1[kLoads];
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int pos = (i * kWaves + wave) * 64 + lane;
      const int row = pos / GR, slot = pos % GR;
      const uint32_t g16 = uint32_t(slot ^ ((((row & 3) << 2) | ((row >> 2) & 3)) & (GR - 1))) * 16u;
      voff0[i] = uint32_t(row) * uint32_t(p.src[0].k_st) + g16;
      voff1[i] = uint32_t(row) * uint32_t(p.src[1].k_st) + g16;
    }
    static_assert(!kF8, "the FP8 cache runs on the ping-pong ring");
    run_ring<D, QB>(p, qs, b, h, kt_begin, kt_end, wave, lane, wave_active, voff0, voff1, qf, oacc, m_used, lsum, cb);
  }

  // ---- epilogue (the half-sum exchange runs on every lane before any lane leaves)
  float l_tot[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) l_tot[qb] = sum_halves(lsum[qb]);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if (!row_ok[qb]) continue;
    if (part_row >= 0) {
      const int64_t prow = part_row + my_row[qb];
      float* op = p.ws_o + prow * D;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = nb * 32 + 8 * q4 + 4 * hh;
          float4 v4 = make_float4(oacc[qb][nb][4 * q4], oacc[qb][nb][4 * q4 + 1], oacc[qb][nb][4 * q4 + 2],
                                  oacc[qb][nb][4 * q4 + 3]);
          *reinterpret_cast<float4*>(op + d) = v4;
        }
      if (hh == 0) {
        p.ws_ml[prow * 2] = m_used[qb];
        p.ws_ml[prow * 2 + 1] = l_tot[qb];
      }
    } else {
      const int grow = row0 + my_row[qb];
      const float inv = l_tot[qb] > 0.f ? 1.f / l_tot[qb] : 0.f;
      uint16_t* op = p.o + int64_t(b) * p.o_sb + int64_t(grow) * p.o_st + int64_t(h) * D;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int d = nb * 32 + 8 * q4 + 4 * hh;
          __bf16 o4[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) o4[j] = (__bf16)(oacc[qb][nb][4 * q4 + j] * inv);
          *reinterpret_cast<u32x2*>(op + d) = __builtin_bit_cast(u32x2, o4);
        }
      if (p.lse && hh == 0)
        p.lse[(int64_t(b) * p.H + h) * p.n_rows + grow] =
            l_tot[qb] > 0.f ? m_used[qb] * 0.69314718055994531f + __logf(l_tot[qb]) : -INFINITY;
    }
  }
}

// Copy work-group j of the prefill's cache store: rows [j R / C, (j + 1) R /
// C) of the first R = c.rows flat cache rows ([B, H, n_cached] rows of D
// values), D / 8 lanes per row, eight rows per lane in flight before their
// stores.  Work-groups are dispatched in order, so these start when the last
// attention work-groups have been placed and take the CUs that the partial
// last round leaves free.  Loads and stores bypass the caches' retention
// (the attention work-groups still running read their keys through L2).
template <int D>
__device__ __forceinline__ void copy_tail(const CopyTail& c, int j, int tid) {
  constexpr int GR = D / 8, RPP = kThreads / GR, U = 8;
  const uint32_t H = uint32_t(c.H);
  const uint32_t R = uint32_t(c.rows);  // <= B H n_cached < 2^31 (host check)
  const uint32_t r0 = uint32_t(uint64_t(R) * uint32_t(j) / uint32_t(c.blocks));
  const uint32_t r1 = uint32_t(uint64_t(R) * uint32_t(j + 1) / uint32_t(c.blocks));
  const int g8 = (tid % GR) * 8;
  for (uint32_t base = r0 + uint32_t(tid / GR); base < r1; base += uint32_t(RPP * U)) {
    u32x4 kx[U], vx[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t r = base + uint32_t(u * RPP);
      if (r < r1) {
        const uint32_t bh = r / uint32_t(c.n_cached), drow = r - bh * uint32_t(c.n_cached);
        const uint32_t b = bh / H, h = bh - b * H;
        // the run holding drow, by a loop over the whole table: its index is
        // wave-uniform, so the table comes in through scalar loads (a per-lane
        // index would read it with vector loads, whose waits also wait for the
        // copy loads already in flight)
        int64_t delta = 0;
        for (int k = 0; k < c.n_copy; ++k)
          if (drow >= uint32_t(c.seg[k].dst_row0)) delta = int64_t(c.seg[k].src_row0) - c.seg[k].dst_row0;
        const int64_t srow = int64_t(drow) + delta;
        const int64_t so = int64_t(b) * c.src_sb + srow * c.src_st + int64_t(h) * D + g8;
        kx[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(c.k_src + so));
        vx[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(c.v_src + so));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t r = base + uint32_t(u * RPP);
      if (r < r1) {
        const int64_t dof = int64_t(r) * D + g8;
        __builtin_nontemporal_store(kx[u], reinterpret_cast<u32x4*>(c.k_dst + dof));
        __builtin_nontemporal_store(vx[u], reinterpret_cast<u32x4*>(c.v_dst + dof));
      }
    }
  }
}

// One work-group per (batch, head, query tile, key split), then p.cp.blocks
// copy work-groups (the prefill's cache store; unsplit bf16 launches only).
// The host plans the query tiles with p.bm = rows_per_wg of the kernel's
// block count.
template <int D, bool kSplit, bool kF8>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const Params p) {
  constexpr int QB = kF8 ? kQBFp8 : kQBPlain;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int n_attn = gridDim.x;
  if constexpr (!kSplit && !kF8) {
    n_attn -= p.cp.blocks;
    if (int(blockIdx.x) >= n_attn) {
      copy_tail<D>(p.cp, blockIdx.x - n_attn, tid);
      return;
    }
  }
  int split, rest;
  if (kSplit && p.lr_tiles > 0) {
    // last-round split: blocks [0, U) are whole query tiles (logical tiles
    // [0, U)), then the long pieces of logical tiles [U, U + T), then their
    // short pieces, which the CUs idle in the last round take first
    const int T = p.lr_tiles, U = n_attn - 2 * T;
    if (int(blockIdx.x) < U) {
      split = -1;
      rest = xcd_logical_block(blockIdx.x, U);
    } else {
      const int i = blockIdx.x - U;
      split = i >= T;
      rest = U + xcd_logical_block(i - split * T, T);
    }
  } else if (kSplit && p.tail_num > 0) {
    // tail split: blocks [0, Q) are the long pieces, dispatched first; blocks
    // [Q, 2 Q) the short ones.  Both halves map to query tiles the same way,
    // so (for Q a multiple of 8) a tile's short piece runs on the XCD of its
    // long piece, where the other short pieces of the head share its keys.
    const int q = n_attn / 2;
    split = blockIdx.x >= q;
    rest = xcd_logical_block(blockIdx.x - split * q, q);
  } else {
    const int w = xcd_logical_block(blockIdx.x, n_attn);
    split = w % p.splits;
    rest = w / p.splits;
  }
  const int w = rest;  // logical query tile
  const int t = rest % p.n_qtiles;
  rest /= p.n_qtiles;
  const int h = rest % p.H, b = rest / p.H;

  int qi = 0;
  while (qi + 1 < p.n_qseg && p.qseg[qi + 1].tile0 <= t) ++qi;
  const QSeg qs = p.qseg[qi];
  int kt_begin, kt_end;
  if (kSplit && p.tail_num > 0) {
    const int mid = int((int64_t(qs.ktiles) * p.tail_num) >> 10);
    kt_begin = split > 0 ? mid : 0;
    kt_end = split == 0 ? mid : qs.ktiles;
  } else {
    kt_begin = int(int64_t(qs.ktiles) * split / p.splits);
    kt_end = int(int64_t(qs.ktiles) * (split + 1) / p.splits);
  }
  int64_t part_row = -1;
  if constexpr (kSplit) {
    if (p.lr_tiles > 0) {
      // piece s of last-round tile i: workspace rows (s T + i) BM + row
      if (split >= 0) part_row = (int64_t(split) * p.lr_tiles + (w - (n_attn - 2 * p.lr_tiles))) * Blk<QB>::kRows;
    } else {
      part_row = ((int64_t(split) * p.B + b) * p.H + h) * p.n_rows + qs.row0 + (t - qs.tile0) * Blk<QB>::kRows;
    }
  }
  attend_tile<D, kF8, QB>(p, qs, t, b, h, kt_begin, kt_end, part_row, wave, lane);
}

// Balanced schedule: work-group g of G takes the key-tile units
// [g W / G, (g + 1) W / G) of the W units, ordered by (batch, head, query
// segment, query tile, key tile).  A query tile wholly inside one range is
// written directly; a cut one leaves partials: the work-group's first piece
// in workspace slot 2 g, its last piece (when not also its first) in 2 g + 1.
template <int D, bool kF8>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_balanced_kernel(const Params p) {
  constexpr int QB = kQBBalanced;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = xcd_logical_block(blockIdx.x, gridDim.x);
  const int64_t G = gridDim.x;
  int64_t u = int64_t(g) * p.units / G;
  const int64_t hi = int64_t(g + 1) * p.units / G;
  bool first = true;
  while (u < hi) {
    const int64_t bh = u / p.units_bh;
    int64_t r = u - bh * p.units_bh;
    int qi = 0;
    while (qi + 1 < p.n_qseg && p.qseg[qi + 1].unit0 <= r) ++qi;
    const QSeg qs = p.qseg[qi];
    r -= qs.unit0;
    const int tl = int(r / qs.ktiles);
    const int kt0 = int(r - int64_t(tl) * qs.ktiles);
    const int kt1 = int(min(int64_t(qs.ktiles), int64_t(kt0) + (hi - u)));
    const bool whole = kt0 == 0 && kt1 == qs.ktiles;
    const int64_t part_row = whole ? -1 : int64_t(first ? 2 * g : 2 * g + 1) * Blk<QB>::kRows;
    if (!first) ring_barrier();  // every wave is done with the previous piece's LDS stages
    attend_tile<D, kF8, QB>(p, qs, qs.tile0 + tl, int(bh / p.H), int(bh % p.H), kt0, kt1, part_row, wave, lane);
    u += kt1 - kt0;
    first = false;
  }
}

// Merge of the balanced schedule, one thread per (row, 4 consecutive d):
// rows of a query tile that lies inside one work-group's range were written by
// the attention kernel and are skipped; a cut tile merges the partials of the
// work-groups g_first .. g_last that cover it, in that order (the key order);
// rows that read no key get O = 0 and LSE = -inf.
__global__ __launch_bounds__(256) void combine_balanced_kernel(const Params p, int D) {
  const int dq = D / 4;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = int64_t(p.B) * p.H * p.n_rows * dq;
  if (idx >= total) return;
  const int d4 = int(idx % dq);
  const int64_t bhr = idx / dq;  // (b*H + h)*n_rows + row
  const int row = int(bhr % p.n_rows);
  const int64_t bh = bhr / p.n_rows;
  const int h = int(bh % p.H), b = int(bh / p.H);
  int qi = 0;
  while (qi + 1 < p.n_qseg && p.qseg[qi + 1].row0 <= row) ++qi;
  const QSeg& qs = p.qseg[qi];
  const int tl = (row - qs.row0) / p.bm, rin = (row - qs.row0) % p.bm;
  uint16_t* op = p.o + int64_t(b) * p.o_sb + int64_t(row) * p.o_st + int64_t(h) * D + 4 * d4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float M = -INFINITY, l = 0.f;
  if (qs.ktiles > 0) {
    const int64_t W = p.units, G = p.bal_wgs;
    const int64_t s = bh * p.units_bh + qs.unit0 + int64_t(tl) * qs.ktiles;
    const int64_t e = s + qs.ktiles;
    // work-group holding unit x: the largest g with floor(g W / G) <= x
    const int64_t gf = ((s + 1) * G - 1) / W, gl = (e * G - 1) / W;
    if (gf == gl) return;
    // work-groups with an empty range (more work-groups than units) write nothing
    for (int64_t g = gf; g <= gl; ++g) {
      const int64_t lo = g * W / G;
      if (lo == (g + 1) * W / G) continue;
      const int64_t slot = (g == gf && lo < s) ? 2 * g + 1 : 2 * g;
      const int64_t prow = slot * p.bm + rin;
      if (p.ws_ml[prow * 2 + 1] > 0.f) M = fmaxf(M, p.ws_ml[prow * 2]);
    }
    if (M != -INFINITY) {
      for (int64_t g = gf; g <= gl; ++g) {
        const int64_t lo = g * W / G;
        if (lo == (g + 1) * W / G) continue;
        const int64_t slot = (g == gf && lo < s) ? 2 * g + 1 : 2 * g;
        const int64_t prow = slot * p.bm + rin;
        const float ls = p.ws_ml[prow * 2 + 1];
        if (!(ls > 0.f)) continue;
        const float wgt = __builtin_amdgcn_exp2f(p.ws_ml[prow * 2] - M);
        const float4 o = *reinterpret_cast<const float4*>(p.ws_o + prow * D + 4 * d4);
        acc.x += wgt * o.x;
        acc.y += wgt * o.y;
        acc.z += wgt * o.z;
        acc.w += wgt * o.w;
        l += wgt * ls;
      }
    }
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  __bf16 o4[4] = {(__bf16)(acc.x * inv), (__bf16)(acc.y * inv), (__bf16)(acc.z * inv), (__bf16)(acc.w * inv)};
  *reinterpret_cast<u32x2*>(op) = __builtin_bit_cast(u32x2, o4);
  if (p.lse && d4 == 0) p.lse[bhr] = l > 0.f ? M * 0.69314718055994531f + __logf(l) : -INFINITY;
}


// Split-KV merge: O = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s, in split order.
// One thread per (row, 4 consecutive d).
// Merge of one output row's split partials, in split order: partial s of the
// row sits at workspace row r0 + s * stride (D floats of O, then max and sum
// in the (max, sum) plane).  Writes 4 bf16 of O (columns 4 d4..) and, for
// d4 = 0, the LSE when lse is not null.
__device__ __forceinline__ void merge_partials(const float* ws_o, const float* ws_ml, int64_t r0, int64_t stride,
                                               int splits, int D, int d4, uint16_t* op, float* lse) {
  float M = -INFINITY;
  for (int s = 0; s < splits; ++s) {
    const float ls = ws_ml[(s * stride + r0) * 2 + 1];
    if (ls > 0.f) M = fmaxf(M, ws_ml[(s * stride + r0) * 2]);
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float l = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < splits; ++s) {
      const float ls = ws_ml[(s * stride + r0) * 2 + 1];
      if (!(ls > 0.f)) continue;
      const float wgt = __builtin_amdgcn_exp2f(ws_ml[(s * stride + r0) * 2] - M);
      const float4 o = *reinterpret_cast<const float4*>(ws_o + (s * stride + r0) * D + 4 * d4);
      acc.x += wgt * o.x;
      acc.y += wgt * o.y;
      acc.z += wgt * o.z;
      acc.w += wgt * o.w;
      l += wgt * ls;
    }
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  __bf16 o4[4] = {(__bf16)(acc.x * inv), (__bf16)(acc.y * inv), (__bf16)(acc.z * inv), (__bf16)(acc.w * inv)};
  *reinterpret_cast<u32x2*>(op) = __builtin_bit_cast(u32x2, o4);
  if (lse && d4 == 0) *lse = l > 0.f ? M * 0.69314718055994531f + __logf(l) : -INFINITY;
}

__global__ __launch_bounds__(256) void combine_kernel(const CombineParams c) {
  const int dq = c.D / 4;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = int64_t(c.B) * c.H * c.n_rows * dq;
  if (idx >= total) return;
  const int d4 = int(idx % dq);
  const int64_t bhr = idx / dq;  // (b*H + h)*n_rows + row
  const int row = int(bhr % c.n_rows);
  const int64_t bh = bhr / c.n_rows;
  const int h = int(bh % c.H), b = int(bh / c.H);
  const int64_t plane = int64_t(c.B) * c.H * c.n_rows;
  uint16_t* op = c.o + int64_t(b) * c.o_sb + int64_t(row) * c.o_st + int64_t(h) * c.D + 4 * d4;
  merge_partials(c.ws_o, c.ws_ml, bhr, plane, c.splits, c.D, d4, op, c.lse ? c.lse + bhr : nullptr);
}

// Merge of the last-round split: one thread per 4 output elements of the
// p.lr_tiles last query tiles (logical order); piece s of tile i holds row r
// at workspace row (s T + i) BM + r.
__global__ __launch_bounds__(256) void combine_last_round_kernel(const Params p, int D) {
  const int dq = D / 4;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int T = p.lr_tiles;
  if (idx >= int64_t(T) * p.bm * dq) return;
  const int d4 = int(idx % dq);
  const int64_t ir = idx / dq;
  const int r = int(ir % p.bm), i = int(ir / p.bm);
  const int64_t w = int64_t(p.B) * p.H * p.n_qtiles - T + i;
  const int t = int(w % p.n_qtiles);
  const int64_t bh = w / p.n_qtiles;
  const int h = int(bh % p.H), b = int(bh / p.H);
  int qi = 0;
  while (qi + 1 < p.n_qseg && p.qseg[qi + 1].tile0 <= t) ++qi;
  const int in_seg = (t - p.qseg[qi].tile0) * p.bm + r;
  if (in_seg >= p.qseg[qi].len) return;
  const int row = p.qseg[qi].row0 + in_seg;
  uint16_t* op = p.o + int64_t(b) * p.o_sb + int64_t(row) * p.o_st + int64_t(h) * D + 4 * d4;
  merge_partials(p.ws_o, p.ws_ml, int64_t(i) * p.bm + r, int64_t(T) * p.bm, 2, D, d4, op,
                 p.lse ? p.lse + bh * p.n_rows + row : nullptr);
}

// Cache store: one thread per 16-byte granule of one cached (b, h, row),
// from flat row c.row0 on.
__global__ __launch_bounds__(256) void cache_store_kernel(const CacheStoreParams c) {
  const int gr = c.D / 8;
  const int64_t idx = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) + c.row0 * gr;
  const int64_t total = int64_t(c.B) * c.H * c.total_rows * gr;
  if (idx >= total) return;
  const int g = int(idx % gr);
  int64_t rest = idx / gr;
  const int drow = int(rest % c.total_rows);
  rest /= c.total_rows;
  const int h = int(rest % c.H), b = int(rest / c.H);
  int delta = 0;  // uniform loop over the run table: scalar loads
  for (int k = 0; k < c.n_copy; ++k)
    if (drow >= c.seg[k].dst_row0) delta = c.seg[k].src_row0 - c.seg[k].dst_row0;
  const int srow = drow + delta;
  const int64_t so = int64_t(b) * c.src_sb + int64_t(srow) * c.src_st + int64_t(h) * c.D + g * 8;
  const int64_t dof = ((int64_t(b) * c.H + h) * c.n_cached + drow) * c.D + g * 8;
  *reinterpret_cast<u32x4*>(c.k_dst + dof) = *reinterpret_cast<const u32x4*>(c.k_src + so);
  *reinterpret_cast<u32x4*>(c.v_dst + dof) = *reinterpret_cast<const u32x4*>(c.v_src + so);
}

}  // namespace

template <int D, bool kF8>
void launch_grid(const Params& p, int64_t blocks, hipStream_t s) {
  if (p.splits > 1) hipLaunchKernelGGL((attn_fwd_kernel<D, true, kF8>), dim3(blocks), dim3(kThreads), 0, s, p);
  else hipLaunchKernelGGL((attn_fwd_kernel<D, false, kF8>), dim3(blocks), dim3(kThreads), 0, s, p);
}

// Split partials of the no-allocation step entry.  In host code `scratch`
// names a host-side stand-in: kernels get the device address that
// scratch_address looks up once per device.
static __device__ __align__(256) unsigned char scratch[RC_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

int scratch_address(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return int(e);
  if (dev < 0 || dev >= kMaxDevices) return int(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return int(e);
    g_scratch_ptr[dev] = a;
  }
  *ptr = g_scratch_ptr[dev];
  return int(hipSuccess);
}

int launch_attention(const Params& p, int D, void* stream) {
  const int64_t per_batch = int64_t(p.H) * p.n_qtiles * p.splits;
  // the last-round split adds one short piece per split tile
  const int64_t blocks =
      p.lr_tiles > 0 ? int64_t(p.B) * p.H * p.n_qtiles + p.lr_tiles : int64_t(p.B) * per_batch;
  if (blocks == 0) return 0;
  if (p.lr_tiles < 0 ||
      (p.lr_tiles > 0 && (p.splits != 2 || p.tail_num <= 0 || p.lr_tiles > int64_t(p.B) * p.H * p.n_qtiles)))
    return int(hipErrorInvalidValue);
  // copy work-groups ride on unsplit bf16 grids only (the other kernels have
  // no copy path)
  if (p.cp.blocks < 0 || (p.cp.blocks > 0 && (p.splits != 1 || p.fp8))) return int(hipErrorInvalidValue);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const auto launch = [&](const Params& q, int64_t nb) {
    nb += q.cp.blocks;
    if (D == 128) q.fp8 ? launch_grid<128, true>(q, nb, s) : launch_grid<128, false>(q, nb, s);
    else q.fp8 ? launch_grid<64, true>(q, nb, s) : launch_grid<64, false>(q, nb, s);
  };
  // When one batch entry alone fills more than half the CUs, the entries run
  // as consecutive launches: the partial last round of one combined grid
  // costs more than the idle CUs of the separate ones (five references,
  // 216 work-groups per entry: B = 2 2.33 vs 2.35-2.59 ms, B = 3 3.53 vs
  // 3.67 ms).  Split-KV partials are laid out per batch entry, so only
  // unsplit grids do this.
  if (per_batch_launches(p)) {
    Params q = p;
    q.B = 1;
    for (int b = 0; b < p.B; ++b) {
      q.cp.blocks = b == p.B - 1 ? p.cp.blocks : 0;  // the copy rides on the last launch
      q.q = p.q + int64_t(b) * p.q_sb;
      q.o = p.o + int64_t(b) * p.o_sb;
      q.lse = p.lse ? p.lse + int64_t(b) * p.H * p.n_rows : nullptr;
      for (int i = 0; i < 2; ++i) {
        q.src[i].k = p.src[i].k ? p.src[i].k + int64_t(b) * p.src[i].k_sb : nullptr;
        q.src[i].v = p.src[i].v ? p.src[i].v + int64_t(b) * p.src[i].v_sb : nullptr;
      }
      q.kv_scale = p.kv_scale ? p.kv_scale + int64_t(b) * p.H * 2 : nullptr;
      launch(q, per_batch);
    }
  } else {
    launch(p, blocks);
  }
  return int(hipGetLastError());
}

int launch_attention_balanced(const Params& p, int D, void* stream) {
  if (p.units == 0) return 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // bf16 caches only (the API refuses the balanced schedule with the FP8 cache)
  const dim3 g(p.bal_wgs), t(kThreads);
  if (D == 128) hipLaunchKernelGGL((attn_fwd_balanced_kernel<128, false>), g, t, 0, s, p);
  else hipLaunchKernelGGL((attn_fwd_balanced_kernel<64, false>), g, t, 0, s, p);
  return int(hipGetLastError());
}

int launch_combine_balanced(const Params& p, int D, void* stream) {
  const int64_t total = int64_t(p.B) * p.H * p.n_rows * (D / 4);
  if (total == 0) return 0;
  hipLaunchKernelGGL(combine_balanced_kernel, dim3((total + 255) / 256), dim3(256), 0,
                     static_cast<hipStream_t>(stream), p, D);
  return int(hipGetLastError());
}

int launch_combine_last_round(const Params& p, int D, void* stream) {
  const int64_t total = int64_t(p.lr_tiles) * p.bm * (D / 4);
  if (total == 0) return 0;
  hipLaunchKernelGGL(combine_last_round_kernel, dim3((total + 255) / 256), dim3(256), 0,
                     static_cast<hipStream_t>(stream), p, D);
  return int(hipGetLastError());
}

int launch_combine(const CombineParams& c, void* stream) {
  const int64_t total = int64_t(c.B) * c.H * c.n_rows * (c.D / 4);
  if (total == 0) return 0;
  hipLaunchKernelGGL(combine_kernel, dim3((total + 255) / 256), dim3(256), 0, static_cast<hipStream_t>(stream), c);
  return int(hipGetLastError());
}

int launch_cache_store(const CacheStoreParams& c, void* stream) {
  const int64_t total = (int64_t(c.B) * c.H * c.total_rows - c.row0) * (c.D / 8);
  if (total == 0) return 0;
  hipLaunchKernelGGL(cache_store_kernel, dim3((total + 255) / 256), dim3(256), 0, static_cast<hipStream_t>(stream), c);
  return int(hipGetLastError());
}

}  // namespace rc
