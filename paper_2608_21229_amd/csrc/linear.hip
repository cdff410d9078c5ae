// Dense bf16 projection for the chained synthetic layer: out = A W^T (+ R).
//
// The layer around the attention (Sec. 3.1, Eq. 2: K_R = R W_K, V_R = R W_V
// per layer; the output projection and residual feed the next layer) is a
// plain GEMM per token: out[m, n] = sum_k A[m, k] W[n, k] (+ R[m, n]), fp32
// accumulation, one bf16 rounding (RNE) at the end.
//
// Two kernels: 256 x 256 output tiles with 8 waves when N is a multiple of
// 256 (the layer's projections), 128 x 128 tiles with 4 waves otherwise.  K
// advances in steps of 64; each wave owns a block of v_mfma_f32_32x32x16_bf16
// accumulators.  A and W tiles (64 k per row, 128-byte rows) stream through
// a two-stage LDS ring with direct global->LDS loads; 16-byte granule g of
// row r is stored at slot g ^ ((r >> 1) & 7), so the 128-bit fragment reads
// of 16 consecutive rows hit 16 distinct bank groups.  Every output row
// depends only on its own input row, with a fixed reduction order: a row's
// result does not depend on how many rows the call has.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rc_internal.h"

namespace rc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kLinBM = 128, kLinBN = 128, kLinBK = 64;
constexpr int kLinThreads = 256;
constexpr int kTileBytes = kLinBM * kLinBK * 2;  // 16 KB per A or W tile

__shared__ __attribute__((aligned(1024))) char g_a0[kTileBytes];
__shared__ __attribute__((aligned(1024))) char g_w0[kTileBytes];
__shared__ __attribute__((aligned(1024))) char g_a1[kTileBytes];
__shared__ __attribute__((aligned(1024))) char g_w1[kTileBytes];

template <int S>
__device__ __forceinline__ char* abuf() {
  if constexpr (S == 0) return g_a0;
  else return g_a1;
}
template <int S>
__device__ __forceinline__ char* wbuf() {
  if constexpr (S == 0) return g_w0;
  else return g_w1;
}

__device__ __forceinline__ uint32_t lds_u32(const char* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_void*)p));
}

// 16 bytes per lane straight into LDS at M0 + 16 lane; offsets past the
// record count read as zeros (see the attention kernel for the wait rules).
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, __amdgpu_buffer_rsrc_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}

__device__ __forceinline__ int lin_swz(int row, int g) { return g ^ ((row >> 1) & 7); }

// Wave w loads the 1 KB chunks w, w + 4, w + 8, w + 12 of a 16 KB tile; lane l
// of chunk c fills LDS slot p = 64 c + l: row p / 8, slot p % 8, holding the
// row's granule slot ^ ((row >> 1) & 7).  `ld` is the row stride in elements.
__device__ __forceinline__ uint32_t lin_off(int chunk, int lane, int64_t ld) {
  const int p = chunk * 64 + lane;
  const int row = p >> 3, slot = p & 7;
  return uint32_t(row) * uint32_t(ld) * 2u + uint32_t(lin_swz(row, slot)) * 16u;
}

template <int S>
__device__ __forceinline__ void issue_k_step(const LinearParams& q, int m0, int n0, int k0, int wave,
                                             const uint32_t (&aoff)[4], const uint32_t (&woff)[4]) {
  // rows past M (A) lie beyond the record count and load zeros
  const int a_rows = min(kLinBM, int(q.M - m0));
  const int nrec_a = a_rows > 0 ? int(int64_t(a_rows - 1) * q.lda * 2 + kLinBK * 2) : 0;
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(q.a + int64_t(m0) * q.lda + k0), (short)0, nrec_a, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(q.w + int64_t(n0) * q.K + k0), (short)0, int(int64_t(kLinBN - 1) * q.K * 2 + kLinBK * 2),
      0x00020000);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int chunk = i * 4 + wave;
    dma16(lds_u32(abuf<S>() + chunk * 1024), aoff[i], ra);
    dma16(lds_u32(wbuf<S>() + chunk * 1024), woff[i], rw);
  }
}

// 128-bit fragment of rows r0 + lane % 32, k = 16 kk + 8 (lane / 32) .. +7.
__device__ __forceinline__ bf16x8 lin_frag(const char* t, int r0, int lane, int kk) {
  const int row = r0 + (lane & 31);
  const int g = 2 * kk + (lane >> 5);
  return *reinterpret_cast<const bf16x8*>(t + row * (kLinBK * 2) + lin_swz(row, g) * 16);
}

template <int S>
__device__ __forceinline__ void mma_k_step(int lane, int wm, int wn, f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int kk = 0; kk < kLinBK / 16; ++kk) {
    bf16x8 af[2], wf[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) af[i] = lin_frag(abuf<S>(), wm * 64 + i * 32, lane, kk);
#pragma unroll
    for (int j = 0; j < 2; ++j) wf[j] = lin_frag(wbuf<S>(), wn * 64 + j * 32, lane, kk);
    // C^T block (n rows, m columns): A = W fragment, B = A fragment, so the
    // accumulator holds one output row m per lane (lane % 32)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[j], af[i], acc[i][j], 0, 0, 0);
  }
}

__device__ __forceinline__ void lin_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
}

__global__ __launch_bounds__(kLinThreads, 2) void linear_kernel(const LinearParams q) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;  // this wave's 64 x 64 block of the tile
  const int n_tiles = q.N / kLinBN;
  const int64_t tile = blockIdx.x;
  const int64_t m0 = (tile / n_tiles) * kLinBM;
  const int n0 = int(tile % n_tiles) * kLinBN;

  uint32_t aoff[4], woff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    aoff[i] = lin_off(i * 4 + wave, lane, q.lda);
    woff[i] = lin_off(i * 4 + wave, lane, q.K);
  }
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = q.K / kLinBK;
  issue_k_step<0>(q, int(m0), n0, 0, wave, aoff, woff);
  for (int ks = 0; ks < nk; ks += 2) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lin_barrier();
    if (ks + 1 < nk) issue_k_step<1>(q, int(m0), n0, (ks + 1) * kLinBK, wave, aoff, woff);
    mma_k_step<0>(lane, wm, wn, acc);
    if (ks + 1 >= nk) break;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lin_barrier();
    if (ks + 2 < nk) issue_k_step<0>(q, int(m0), n0, (ks + 2) * kLinBK, wave, aoff, woff);
    mma_k_step<1>(lane, wm, wn, acc);
  }

  // epilogue: lane holds output row m = m0 + wm*64 + i*32 + lane%32 and, in
  // accumulator slot r, column n = n0 + wn*64 + j*32 + 8 (r/4) + 4 (lane/32) + r%4
  const int hh = lane >> 5;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t m = m0 + wm * 64 + i * 32 + (lane & 31);
    if (m >= q.M) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn * 64 + j * 32 + 8 * q4 + 4 * hh;
        float v4[4] = {acc[i][j][4 * q4], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3]};
        if (q.r) {
          const u32x2 rr = *reinterpret_cast<const u32x2*>(q.r + m * q.ldr + n);
          const __bf16* rb = reinterpret_cast<const __bf16*>(&rr);
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] += float(rb[e]);
        }
        __bf16 o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (__bf16)v4[e];
        *reinterpret_cast<u32x2*>(q.out + m * q.ldo + n) = __builtin_bit_cast(u32x2, o4);
      }
  }
}

// ---------------------------------------------------------------------------
// 256 x 256 output tiles (N a multiple of 256): 8 waves, one work-group per
// CU, each wave a 128 (m) x 64 (n) block of 4 x 2 accumulators.  Per K step
// of 64 a wave reads 24 KB of fragments for 32 MFMAs (the 128 x 128 kernel:
// 16 KB for 16), and the work-group stages 64 KB for 256 MFMAs (32 KB for 64),
// so the LDS reads and fills per MFMA halve.  Tiles are ordered in groups of
// kGroupM m-tiles (m fastest inside a group), so the 32 work-groups an XCD
// runs together share 4 A tiles and 8 W tiles in its L2.  (Measured on these
// projections: one wave per SIMD with 128 x 128 blocks, register-staged tile
// loads, and K steps of 32 through a 4-stage ring were each 6-10% slower.)
constexpr int kL2BM = 256, kL2BN = 256;
constexpr int kL2Waves = 8;                    // 2 x 4 waves of 128 x 64
constexpr int kL2Threads = kL2Waves * 64;
constexpr int kL2WN = kL2BN / (kL2Waves / 2);  // n width of a wave's block
constexpr int kL2NJ = kL2WN / 32;              // 32-wide n blocks per wave
constexpr int kL2TileBytes = kL2BM * kLinBK * 2;  // 32 KB per A or W tile
constexpr int kL2Chunks = kL2TileBytes / 1024 / kL2Waves;  // 1 KB chunks per wave per tile
constexpr int kGroupM = 4;

__shared__ __attribute__((aligned(1024))) char g2_a0[kL2TileBytes];
__shared__ __attribute__((aligned(1024))) char g2_w0[kL2TileBytes];
__shared__ __attribute__((aligned(1024))) char g2_a1[kL2TileBytes];
__shared__ __attribute__((aligned(1024))) char g2_w1[kL2TileBytes];

template <int S>
__device__ __forceinline__ char* a2buf() {
  if constexpr (S == 0) return g2_a0;
  else return g2_a1;
}
template <int S>
__device__ __forceinline__ char* w2buf() {
  if constexpr (S == 0) return g2_w0;
  else return g2_w1;
}

// Wave w loads the 1 KB chunks w, w + 8, w + 16, w + 24 of the A and the W tile.
template <int S>
__device__ __forceinline__ void issue_k_step256(const LinearParams& q, int64_t m0, int n0, int k0, int wave,
                                                const uint32_t (&aoff)[kL2Chunks], const uint32_t (&woff)[kL2Chunks]) {
  const int a_rows = int(min(int64_t(kL2BM), q.M - m0));
  const int nrec_a = a_rows > 0 ? int(int64_t(a_rows - 1) * q.lda * 2 + kLinBK * 2) : 0;
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(q.a + m0 * q.lda + k0), (short)0, nrec_a, 0x00020000);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(q.w + int64_t(n0) * q.K + k0), (short)0, int(int64_t(kL2BN - 1) * q.K * 2 + kLinBK * 2),
      0x00020000);
#pragma unroll
  for (int i = 0; i < kL2Chunks; ++i) {
    const int chunk = i * kL2Waves + wave;
    dma16(lds_u32(a2buf<S>() + chunk * 1024), aoff[i], ra);
    dma16(lds_u32(w2buf<S>() + chunk * 1024), woff[i], rw);
  }
}

// Scheduling fence: the compiler moves no instruction across it.
__device__ __forceinline__ void lin_fence() { __builtin_amdgcn_sched_barrier(0); }

// Fragment t (0..5) of 16-wide k chunk kk: A rows wm*128 + 32 t for t < 4,
// W rows wn*64 + 32 (t - 4) otherwise.
template <int S>
__device__ __forceinline__ bf16x8 frag256(int lane, int wm, int wn, int kk, int t) {
  return t < 4 ? lin_frag(a2buf<S>(), wm * 128 + t * 32, lane, kk)
               : lin_frag(w2buf<S>(), wn * kL2WN + (t - 4) * 32, lane, kk);
}

// One K step: 4 chunks of 16 x 8 MFMAs.  The six fragments of chunk kk + 1
// are read while chunk kk's MFMAs run (two register sets), one read after
// each of the first six MFMAs.
template <int S>
__device__ __forceinline__ void mma_k_step256(int lane, int wm, int wn, f32x16 (&acc)[4][kL2NJ]) {
  constexpr int NF = 4 + kL2NJ;   // fragments per 16-wide k chunk
  constexpr int NM = 4 * kL2NJ;   // MFMAs per chunk
  bf16x8 fr[2][NF];
#pragma unroll
  for (int t = 0; t < NF; ++t) fr[0][t] = frag256<S>(lane, wm, wn, 0, t);
#pragma unroll
  for (int kk = 0; kk < kLinBK / 16; ++kk) {
    const int c = kk & 1;
    lin_fence();
#pragma unroll
    for (int t = 0; t < NM; ++t) {
      const int i = t / kL2NJ, j = t % kL2NJ;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[c][4 + j], fr[c][i], acc[i][j], 0, 0, 0);
      if (kk + 1 < kLinBK / 16 && t < NF) fr[c ^ 1][t] = frag256<S>(lane, wm, wn, kk + 1, t);
      lin_fence();
    }
  }
}

// The hardware deals work-groups round-robin to the 8 XCDs; give each XCD a
// contiguous run of logical tiles.
__device__ __forceinline__ int64_t lin_xcd_block(int64_t bid, int64_t nblk) {
  const int64_t xcd = bid & 7, kx = bid >> 3, per = nblk >> 3, rem = nblk & 7;
  return (xcd < rem) ? xcd * (per + 1) + kx : rem * (per + 1) + (xcd - rem) * per + kx;
}

__global__ __launch_bounds__(kL2Threads, 1) void linear256_kernel(const LinearParams q) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / (kL2Waves / 2), wn = wave % (kL2Waves / 2);  // this wave's 128 x kL2WN block
  const int64_t n_tiles = q.N / kL2BN;
  const int64_t m_tiles = (q.M + kL2BM - 1) / kL2BM;
  const int64_t w = lin_xcd_block(blockIdx.x, gridDim.x);
  const int64_t per_group = int64_t(kGroupM) * n_tiles;
  const int64_t first_m = (w / per_group) * kGroupM;
  const int64_t group_m = min(int64_t(kGroupM), m_tiles - first_m);
  const int64_t in_group = w % per_group;
  const int64_t m0 = (first_m + in_group % group_m) * kL2BM;
  const int n0 = int(in_group / group_m) * kL2BN;

  uint32_t aoff[kL2Chunks], woff[kL2Chunks];
#pragma unroll
  for (int i = 0; i < kL2Chunks; ++i) {
    aoff[i] = lin_off(i * kL2Waves + wave, lane, q.lda);
    woff[i] = lin_off(i * kL2Waves + wave, lane, q.K);
  }
  f32x16 acc[4][kL2NJ];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < kL2NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // two K steps per iteration (stage 0, then stage 1); an odd last step after
  // the loop, so the loop has a single exit
  const int nk = q.K / kLinBK;
  issue_k_step256<0>(q, m0, n0, 0, wave, aoff, woff);
  int ks = 0;
  for (; ks + 1 < nk; ks += 2) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lin_barrier();
    issue_k_step256<1>(q, m0, n0, (ks + 1) * kLinBK, wave, aoff, woff);
    mma_k_step256<0>(lane, wm, wn, acc);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lin_barrier();
    if (ks + 2 < nk) issue_k_step256<0>(q, m0, n0, (ks + 2) * kLinBK, wave, aoff, woff);
    mma_k_step256<1>(lane, wm, wn, acc);
  }
  if (ks < nk) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lin_barrier();
    mma_k_step256<0>(lane, wm, wn, acc);
  }

  // epilogue: lane holds output row m = m0 + wm*128 + i*32 + lane%32 and, in
  // accumulator slot r, column n = n0 + wn*64 + j*32 + 8 (r/4) + 4 (lane/32) + r%4
  const int hh = lane >> 5;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + wm * 128 + i * 32 + (lane & 31);
    if (m >= q.M) continue;
#pragma unroll
    for (int j = 0; j < kL2NJ; ++j)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn * kL2WN + j * 32 + 8 * q4 + 4 * hh;
        float v4[4] = {acc[i][j][4 * q4], acc[i][j][4 * q4 + 1], acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3]};
        if (q.r) {
          const u32x2 rr = *reinterpret_cast<const u32x2*>(q.r + m * q.ldr + n);
          const __bf16* rb = reinterpret_cast<const __bf16*>(&rr);
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] += float(rb[e]);
        }
        __bf16 o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (__bf16)v4[e];
        *reinterpret_cast<u32x2*>(q.out + m * q.ldo + n) = __builtin_bit_cast(u32x2, o4);
      }
  }
}

}  // namespace

int launch_linear(const LinearParams& q, void* stream) {
  if (q.N % kL2BN == 0) {
    const int64_t blocks = ((q.M + kL2BM - 1) / kL2BM) * (q.N / kL2BN);
    if (blocks == 0) return 0;
    hipLaunchKernelGGL(linear256_kernel, dim3(blocks), dim3(kL2Threads), 0, static_cast<hipStream_t>(stream), q);
    return int(hipGetLastError());
  }
  const int64_t blocks = ((q.M + kLinBM - 1) / kLinBM) * (q.N / kLinBN);
  if (blocks == 0) return 0;
  hipLaunchKernelGGL(linear_kernel, dim3(blocks), dim3(kLinThreads), 0, static_cast<hipStream_t>(stream), q);
  return int(hipGetLastError());
}

}  // namespace rc
