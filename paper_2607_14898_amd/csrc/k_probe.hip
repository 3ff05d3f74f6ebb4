// Sustained dense MFMA throughput of the GPU this library runs on.
//
// The datasheet MFMA peak assumes the 2.4 GHz peak engine clock; under a dense
// MFMA load the chip's power and current management lowers the clock, and the
// throughput that load actually sustains is what the decoder's GEMMs and
// attention are measured against beside the datasheet figure. Every wave of
// two 4-wave workgroups per CU issues 32x32x16 MFMAs back to back on eight
// accumulators, with operands that change every instruction (pseudo-random
// values in [-1, 1), like real activations and weights), and records its
// shader-clock cycles and wall-clock ticks. A second probe measures how many
// bytes per clock the LDS of a compute unit delivers to ds_read_b128, and a
// third how far a wave's MFMAs and its vector instructions (exponentials,
// fused multiply-adds) overlap.
#include "fd_kernels.h"

#include <hip/hip_bf16.h>

namespace fd {
namespace {

typedef _Float16 h16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 b16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16p __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float hash_unit(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return (float)(x & 0xFFFFu) * (1.f / 32768.f) - 1.f;
}

template <typename V, typename E>
__device__ __forceinline__ f32x16p mfma_op(V a, V b, f32x16p c);
template <>
__device__ __forceinline__ f32x16p mfma_op<h16x8, _Float16>(h16x8 a, h16x8 b, f32x16p c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x16p mfma_op<b16x8, __bf16>(b16x8 a, b16x8 b, f32x16p c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

template <typename V, typename E>
__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, unsigned long long* clk, float* sink) {
  const uint32_t gid = blockIdx.x * 256 + threadIdx.x;
  V a[8], b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[i][e] = (E)hash_unit(gid * 131u + i * 8u + e);
      b[i][e] = (E)hash_unit(gid * 131u + 64u + i * 8u + e);
    }
  f32x16p acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  const unsigned long long c0 = clock64(), w0 = wall_clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k % 8] = mfma_op<V, E>(a[(k / 2) % 8], b[k % 8], acc[k % 8]);
  }
  const unsigned long long c1 = clock64(), w1 = wall_clock64();
  float z = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) z += acc[i][r];
  sink[gid] = z;
  if (threadIdx.x == 0) {
    clk[2 * blockIdx.x] = c1 - c0;
    clk[2 * blockIdx.x + 1] = w1 - w0;
  }
}

// LDS read bandwidth: every wave reads 16 bytes per lane per ds_read_b128 from
// a 64 KB block of LDS, consecutive lanes reading consecutive 16-byte chunks
// (no bank conflicts), 8 independent reads in flight per step; the values are
// folded into one register so the reads stay live.
__global__ __launch_bounds__(512) void lds_read_kernel(int iters, unsigned long long* clk, unsigned* sink) {
  __shared__ uint4 buf[4096];  // 64 KB
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 4096; i += blockDim.x) buf[i] = make_uint4(i, i * 3u, i * 5u, i * 7u);
  __syncthreads();
  uint32_t acc = 0;
  int base = (wave * 512 + lane) & 4095;
  const unsigned long long c0 = clock64(), w0 = wall_clock64();
  for (int it = 0; it < iters; ++it) {
    uint4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = buf[(base + 64 * k) & 4095];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
    base = (base + 512 + (acc & 1)) & 4095;
  }
  const unsigned long long c1 = clock64(), w1 = wall_clock64();
  sink[blockIdx.x * blockDim.x + tid] = acc;
  if (tid == 0) {
    clk[2 * blockIdx.x] = c1 - c0;
    clk[2 * blockIdx.x + 1] = w1 - w0;
  }
}

// Issue overlap: per iteration 4 slots, each one 32x32x16 MFMA on its own
// accumulator (MODE bit 0), then NEXP exponentials each followed by a multiply
// (bit 1), then NVALU fused multiply-adds (bit 2), in this order (scheduling
// barriers keep it); every vector instruction works on one of 16 independent
// registers, so no slot waits on another slot's result.
template <int MODE, int NEXP, int NVALU>
__global__ __launch_bounds__(512) void overlap_kernel(int iters, unsigned long long* clk, float* sink) {
  const int tid = threadIdx.x;
  const float seed = 0.37f;
  h16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(seed * (tid + e));
    b[e] = (_Float16)(seed * (tid - e));
  }
  f32x16p c[4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) c[m][r] = 0.f;
  float x[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = seed * (tid + i) * 1e-3f;
  // the workgroup's time: from a common start until its last wave is done
  // (waves sharing a SIMD do not progress at the same rate)
  __syncthreads();
  const unsigned long long c0 = clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (MODE & 1) c[m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c[m], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (MODE & 2) {
#pragma unroll
        for (int e = 0; e < NEXP; ++e) x[(m * NEXP + e) & 15] = __builtin_amdgcn_exp2f(x[(m * NEXP + e) & 15]) * -0.5f;
      }
      if (MODE & 4) {
#pragma unroll
        for (int e = 0; e < NVALU; ++e) x[(m * NVALU + e + 7) & 15] = x[(m * NVALU + e + 7) & 15] * 0.999f + 0.001f;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  float z = 0.f;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int r = 0; r < 16; ++r) z += c[m][r];
#pragma unroll
  for (int i = 0; i < 16; ++i) z += x[i];
  sink[blockIdx.x * blockDim.x + tid] = z;
  __syncthreads();
  const unsigned long long c1 = clock64();
  if (tid == 0) clk[blockIdx.x] = c1 - c0;
}

}  // namespace

hipError_t issue_overlap_probe(int mode, int blocks, int waves_per_simd, int iters, unsigned long long* clk,
                               float* sink, hipStream_t s) {
  if (blocks <= 0 || iters <= 0 || waves_per_simd < 1 || waves_per_simd > 2) return hipErrorInvalidValue;
  const dim3 b(256 * waves_per_simd);
  switch (mode) {
    case 0: hipLaunchKernelGGL((overlap_kernel<1, 0, 0>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    case 1: hipLaunchKernelGGL((overlap_kernel<2, 4, 0>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    case 2: hipLaunchKernelGGL((overlap_kernel<3, 4, 0>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    case 3: hipLaunchKernelGGL((overlap_kernel<4, 0, 8>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    case 4: hipLaunchKernelGGL((overlap_kernel<5, 0, 8>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    case 5: hipLaunchKernelGGL((overlap_kernel<7, 4, 4>), dim3(blocks), b, 0, s, iters, clk, sink); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t lds_read_probe(int blocks, int iters, unsigned long long* clk, unsigned* sink, hipStream_t s) {
  if (blocks <= 0 || iters <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lds_read_kernel, dim3(blocks), dim3(512), 0, s, iters, clk, sink);
  return hipGetLastError();
}

hipError_t mfma_peak(Act16 t, int blocks, int iters, unsigned long long* clk, float* sink, hipStream_t s) {
  if (blocks <= 0 || iters <= 0) return hipErrorInvalidValue;
  if (t == Act16::F16)
    hipLaunchKernelGGL((mfma_peak_kernel<h16x8, _Float16>), dim3(blocks), dim3(256), 0, s, iters, clk, sink);
  else
    hipLaunchKernelGGL((mfma_peak_kernel<b16x8, __bf16>), dim3(blocks), dim3(256), 0, s, iters, clk, sink);
  return hipGetLastError();
}

}  // namespace fd
