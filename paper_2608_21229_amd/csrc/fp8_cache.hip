// FP8 (e4m3fn) reference cache store: quantise the cached segments' K/V rows
// of the static buffers into K8 and V8 [B, H, N_cached, D] (the rows of the
// bf16 cache, one byte per value) with one power-of-two scale per (batch,
// head) and tensor.
//
// Per (b, h) and tensor X: amax = max |x| over the cached rows; the scale is
// s = 2^e with e the smallest integer such that amax / s <= 448 (the largest
// finite e4m3fn value), s = 1 when amax = 0; the code of x is the nearest
// e4m3fn value of x / s (ties to even), which the hardware conversion
// computes.  Dividing by a power of two is exact, so a code depends on x alone,
// and code * s is exact in bf16.
//
// Four launches on the stream: amax accumulators cleared, per-(b, h) amax
// (work-group maxima, then one atomic max per work-group and tensor: the
// result does not depend on the order), the quantising store of K and V,
// and the scales written over the amax values.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rc_internal.h"

namespace rc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kRowsPerBlock = 256;

// e: the smallest integer with amax * 2^-e <= 448 (amax = m 2^k, 0.5 <= m < 1;
// 448 = 0.875 * 2^9).
__device__ __forceinline__ int fp8_exponent(float amax) {
  if (!(amax > 0.f)) return 0;
  int k;
  const float m = frexpf(amax, &k);
  return m <= 0.875f ? k - 9 : k - 8;
}

// Source row (in the static buffers) of cache position pos: a loop over the
// whole run table with a wave-uniform index, so the table comes in through
// scalar loads (a per-lane index would read it with vector loads, whose
// waits also wait for the data loads in flight).
__device__ __forceinline__ int source_row(const CacheStore8Params& c, int pos) {
  int delta = 0;
  for (int k = 0; k < c.n_copy; ++k)
    if (pos >= c.seg[k].dst_row0) delta = c.seg[k].src_row0 - c.seg[k].dst_row0;
  return pos + delta;
}

__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ float amax8(u32x4 g) {
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m = fmaxf(m, fabsf(bf16_bits_to_float(g[i] & 0xffffu)));
    m = fmaxf(m, fabsf(bf16_bits_to_float(g[i] >> 16)));
  }
  return m;
}

// 8 bf16 values (one 16-byte granule) times 2^-e to 8 e4m3fn codes.
__device__ __forceinline__ u32x2 quant8(u32x4 g, int e) {
  u32x2 out;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float a = ldexpf(bf16_bits_to_float(g[2 * i] & 0xffffu), -e);
    const float b = ldexpf(bf16_bits_to_float(g[2 * i] >> 16), -e);
    const float cc = ldexpf(bf16_bits_to_float(g[2 * i + 1] & 0xffffu), -e);
    const float d = ldexpf(bf16_bits_to_float(g[2 * i + 1] >> 16), -e);
    int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    w = __builtin_amdgcn_cvt_pk_fp8_f32(cc, d, w, true);
    out[i] = uint32_t(w);
  }
  return out;
}

__global__ void fill_zero_kernel(float* a, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) a[i] = 0.f;
}

// Grid (B * H, ceil(n_cached / kRowsPerBlock)); 256 threads stride over the
// block's rows x D/8 granules of K and V, four granules of each in flight.
__global__ __launch_bounds__(256) void amax_kernel(const CacheStore8Params c) {
  const int bh = blockIdx.x, b = bh / c.H, h = bh % c.H;
  const int gr = c.D / 8;
  const int row0 = blockIdx.y * kRowsPerBlock;
  const int n = min(kRowsPerBlock, c.n_cached - row0) * gr;
  float mk = 0.f, mv = 0.f;
  for (int g0 = threadIdx.x; g0 < n; g0 += 4 * blockDim.x) {
    u32x4 kx[4], vx[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int g = g0 + u * blockDim.x;
      kx[u] = vx[u] = u32x4{0u, 0u, 0u, 0u};
      if (g < n) {
        const int srow = source_row(c, row0 + g / gr);
        const int64_t off = int64_t(b) * c.src_sb + int64_t(srow) * c.src_st + int64_t(h) * c.D + (g % gr) * 8;
        kx[u] = *reinterpret_cast<const u32x4*>(c.k_src + off);
        vx[u] = *reinterpret_cast<const u32x4*>(c.v_src + off);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      mk = fmaxf(mk, amax8(kx[u]));
      mv = fmaxf(mv, amax8(vx[u]));
    }
  }
  __shared__ float red[2][256];
  red[0][threadIdx.x] = mk;
  red[1][threadIdx.x] = mv;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      red[0][threadIdx.x] = fmaxf(red[0][threadIdx.x], red[0][threadIdx.x + w]);
      red[1][threadIdx.x] = fmaxf(red[1][threadIdx.x], red[1][threadIdx.x + w]);
    }
    __syncthreads();
  }
  // non-negative floats order like their bit patterns
  if (threadIdx.x == 0) {
    atomicMax(reinterpret_cast<unsigned int*>(c.kv_scale + bh * 2), __float_as_uint(red[0][0]));
    atomicMax(reinterpret_cast<unsigned int*>(c.kv_scale + bh * 2 + 1), __float_as_uint(red[1][0]));
  }
}

// K8 and V8: one thread per (b, h, cached row, granule of 8 elements) of
// both tensors.
__global__ __launch_bounds__(256) void quant_kernel(const CacheStore8Params c) {
  const int gr = c.D / 8;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = int64_t(c.B) * c.H * c.n_cached * gr;
  if (idx >= total) return;
  const int g = int(idx % gr);
  int64_t rest = idx / gr;
  const int pos = int(rest % c.n_cached);
  const int64_t bh = rest / c.n_cached;
  const int b = int(bh / c.H), h = int(bh % c.H);
  const int srow = source_row(c, pos);
  const int64_t off = int64_t(b) * c.src_sb + int64_t(srow) * c.src_st + int64_t(h) * c.D + g * 8;
  const u32x4 kx = *reinterpret_cast<const u32x4*>(c.k_src + off);
  const u32x4 vx = *reinterpret_cast<const u32x4*>(c.v_src + off);
  const int64_t dof = (bh * c.n_cached + pos) * c.D + g * 8;
  *reinterpret_cast<u32x2*>(c.k_dst + dof) = quant8(kx, fp8_exponent(c.kv_scale[bh * 2]));
  *reinterpret_cast<u32x2*>(c.v_dst + dof) = quant8(vx, fp8_exponent(c.kv_scale[bh * 2 + 1]));
}

__global__ void finalize_scale_kernel(float* a, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) a[i] = ldexpf(1.f, fp8_exponent(a[i]));
}

}  // namespace

int launch_cache_store_fp8(const CacheStore8Params& c, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nsc = c.B * c.H * 2;
  if (nsc == 0 || c.n_cached == 0) return 0;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((nsc + 255) / 256), dim3(256), 0, s, c.kv_scale, nsc);
  hipLaunchKernelGGL(amax_kernel, dim3(c.B * c.H, (c.n_cached + kRowsPerBlock - 1) / kRowsPerBlock), dim3(256), 0, s,
                     c);
  const int64_t tk = int64_t(c.B) * c.H * c.n_cached * (c.D / 8);
  hipLaunchKernelGGL(quant_kernel, dim3((tk + 255) / 256), dim3(256), 0, s, c);
  hipLaunchKernelGGL(finalize_scale_kernel, dim3((nsc + 255) / 256), dim3(256), 0, s, c.kv_scale, nsc);
  return int(hipGetLastError());
}

}  // namespace rc
