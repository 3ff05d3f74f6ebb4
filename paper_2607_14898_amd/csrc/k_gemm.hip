// Dense projections of the decoder: C = A W^T + b with fused epilogues.
//
// Every Linear layer of the decoder goes through here: the latent projection
// (Eq. projection), the QKV / output / MLP projections of each block (Sec. 3.2),
// the temporal upsampling Linear D -> r_t D (Eq. temporal_upsample) and the
// 2-layer pixel head (Sec. 3.4 Step 3). The epilogues fuse what follows each
// projection: bias, residual add into the fp32 stream, SiLU / GELU / SwiGLU,
// the channel -> sub-frame reshape of Step 1 and the PixelShuffle store.
//
// 16-bit path: one workgroup of 4 wave64s computes a BM x BN tile with the
// gfx950 32x32x16 MFMA (fp32 accumulate). A and W are both K-contiguous, so
// both operands are read from LDS with 16-byte ds_read_b128 per lane; tiles of
// 64 K-columns are double-buffered in LDS with a per-row XOR swizzle of the
// 16-byte chunks (conflict-free for 8 consecutive rows).
#include "fd_kernels.h"

#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>

namespace fd {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + __expf(-x)); }
__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

template <typename T> __device__ __forceinline__ T to_act(float v);
template <> __device__ __forceinline__ _Float16 to_act<_Float16>(float v) { return (_Float16)v; }
template <> __device__ __forceinline__ __hip_bfloat16 to_act<__hip_bfloat16>(float v) { return __float2bfloat16(v); }
template <> __device__ __forceinline__ float to_act<float>(float v) { return v; }

// One output element of an unpaired epilogue. `TA` is the activation type of
// EPI_STORE_* destinations.
template <int EPI, typename TA>
__device__ __forceinline__ void epi_one(const EpiParams& p, int row, int col, float c) {
  c += p.bias[col];
  if constexpr (EPI == EPI_STORE_F32) {
    p.out_f[(int64_t)row * p.ld_out + col] = c;
  } else if constexpr (EPI == EPI_RESID_ADD) {
    p.out_f[(int64_t)row * p.ld_out + col] += c;
  } else if constexpr (EPI == EPI_STORE_ACT) {
    ((TA*)p.out_a)[(int64_t)row * p.ld_out + col] = to_act<TA>(c);
  } else if constexpr (EPI == EPI_STORE_SILU) {
    ((TA*)p.out_a)[(int64_t)row * p.ld_out + col] = to_act<TA>(silu_f(c));
  } else if constexpr (EPI == EPI_STORE_GELU) {
    ((TA*)p.out_a)[(int64_t)row * p.ld_out + col] = to_act<TA>(gelu_f(c));
  } else if constexpr (EPI == EPI_TUP) {
    // row = frame * L + n, col = j * D + d  ->  refinement row (frame * r_t + j) * L + n
    const int f = row / p.L, n = row - f * p.L;
    const int j = col / p.dim, d = col - j * p.dim;
    p.out_f[((int64_t)(f * p.r_t + j) * p.L + n) * p.ld_out + d] = c;
  } else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
    int bo, n, ch;
    if constexpr (EPI == EPI_PIXEL) {
      // row = (b * frames_out + fo) * L + n, col = c s^2 + i1 s + i2
      bo = row / p.L;
      n = row - bo * p.L;
      ch = col;
    } else {
      // row = (b * frames_in + f) * L + n, col = j C s^2 + c s^2 + i1 s + i2
      const int bf = row / p.L;
      n = row - bf * p.L;
      const int cs2 = p.C * p.s * p.s;
      const int j = col / cs2;
      ch = col - j * cs2;
      const int b = bf / p.frames_in, f = bf - b * p.frames_in;
      bo = b * p.frames_out + f * p.r_t + j;
    }
    const int b = bo / p.frames_out, fo = bo - b * p.frames_out;
    const int s2 = p.s * p.s;
    const int c3 = ch / s2, rem = ch - c3 * s2;
    const int i1 = rem / p.s, i2 = rem - i1 * p.s;
    const int h = n / p.grid_w, w = n - h * p.grid_w;
    const int OW = p.grid_w * p.s, OH = p.grid_h * p.s;
    if (p.clamp) c = fminf(1.f, fmaxf(-1.f, c));
    p.out_f[(((int64_t)(b * p.C + c3) * p.frames_out + fo) * OH + (p.s * h + i1)) * OW +
            p.s * w + i2] = c;
  }
}

// ---------------------------------------------------------------------------
// 16-bit MFMA GEMM
// ---------------------------------------------------------------------------

template <typename T> struct Mfma;
template <> struct Mfma<_Float16> {
  using V = f16x8;
  static __device__ __forceinline__ f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<__hip_bfloat16> {
  using V = bf16x8;
  static __device__ __forceinline__ f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

constexpr int BK = 64;   // K-columns per LDS tile: 8 chunks of 16 bytes per row

// Physical 16-byte chunk of (row, chunk) inside a [rows][8 chunks] LDS tile.
__device__ __forceinline__ int swz(int row, int chunk) { return row * 8 + (chunk ^ (row & 7)); }

// Raw buffer resource over `bytes` bytes at `base`: loads at offsets past the
// end return zeros, which covers the ragged M / N edges of a tile.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t soff) {
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0);
  return *reinterpret_cast<uint4*>(&v);
}

template <typename T, int BM, int BN, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_mfma_kernel(const T* __restrict__ A,
                                                           const T* __restrict__ W, int M, int N,
                                                           int K, int lda, int ldw, EpiParams ep,
                                                           int tiles_n) {
  constexpr int WM = BM / 2, WN = BN / 2;       // wave tile (2 x 2 waves)
  constexpr int FM = WM / 32, FN = WN / 32;     // 32x32 MFMA blocks per wave
  constexpr int CA = BM * 8 / 256, CB = BN * 8 / 256;  // 16-byte chunks per thread
  using V = typename Mfma<T>::V;

  extern __shared__ uint4 lds[];
  // buffer b: A tile at lds + b (BM + BN) 8, W tile right after it
  auto As = [&](int b) { return lds + b * (BM + BN) * 8; };
  auto Bs = [&](int b) { return lds + b * (BM + BN) * 8 + BM * 8; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tile = blockIdx.x;
  const int tm = tile / tiles_n, tn = tile - tm * tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;

  // global -> register staging through buffer loads; chunk i of this thread is
  // row (tid / 8) + 32 i, 16-byte column (tid % 8) of the tile
  const __amdgpu_buffer_rsrc_t rA =
      make_rsrc(A + (int64_t)m0 * lda, (uint32_t)min(BM, M - m0) * lda * (uint32_t)sizeof(T));
  const __amdgpu_buffer_rsrc_t rB =
      make_rsrc(W + (int64_t)n0 * ldw, (uint32_t)min(BN, N - n0) * ldw * (uint32_t)sizeof(T));
  const uint32_t offA = ((tid >> 3) * lda + (tid & 7) * 8) * (uint32_t)sizeof(T);
  const uint32_t offB = ((tid >> 3) * ldw + (tid & 7) * 8) * (uint32_t)sizeof(T);
  const uint32_t stepA = 32u * lda * (uint32_t)sizeof(T), stepB = 32u * ldw * (uint32_t)sizeof(T);
  uint4 ra[CA], rb[CB];
  auto gload = [&](int kt) {
    const uint32_t koff = kt * BK * (uint32_t)sizeof(T);
#pragma unroll
    for (int i = 0; i < CA; ++i) ra[i] = buf_load16(rA, offA + i * stepA, koff);
#pragma unroll
    for (int i = 0; i < CB; ++i) rb[i] = buf_load16(rB, offB + i * stepB, koff);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + i * 256;
      As(buf)[swz(c >> 3, c & 7)] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * 256;
      Bs(buf)[swz(c >> 3, c & 7)] = rb[i];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int lr = lane & 31, lk = lane >> 5;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      V a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint4 v = As(cur)[swz(wm0 + i * 32 + lr, 2 * ks + lk)];
        a[i] = *reinterpret_cast<const V*>(&v);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint4 v = Bs(cur)[swz(wn0 + j * 32 + lr, 2 * ks + lk)];
        b[j] = *reinterpret_cast<const V*>(&v);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < KT) lstore(cur ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds column (lane & 31) of each 32x32 block and rows
  // 8 (r / 4) + 4 (lane / 32) + r % 4
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + wm0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
      if (row >= M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int pc = n0 + wn0 + j * 32 + lr;  // packed gate column; up is +32
          if (pc >= N) continue;
          const float g = acc[i][j][r] + ep.bias[pc];
          const float u = acc[i][j + 1][r] + ep.bias[pc + 32];
          const int oc = (n0 + wn0 + j * 32) / 2 + lr;
          ((T*)ep.out_a)[(int64_t)row * ep.ld_out + oc] = to_act<T>(silu_f(g) * u);
        }
      } else {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = n0 + wn0 + j * 32 + lr;
          if (col < N) epi_one<EPI, T>(ep, row, col, acc[i][j][r]);
        }
      }
    }
  }
}

template <typename T, int BM, int BN, int EPI>
hipError_t launch_mfma(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
  constexpr int lds_bytes = 2 * (BM + BN) * 8 * 16;
  static bool attr_set = false;  // raise the dynamic LDS limit once per instantiation
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_mfma_kernel<T, BM, BN, EPI>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((gemm_mfma_kernel<T, BM, BN, EPI>), dim3(tm * tn), dim3(256), lds_bytes, s,
                     (const T*)g.A, (const T*)g.W, g.M, g.N, g.K, g.lda, g.ldw, g.ep, tn);
  return hipGetLastError();
}

// Tile choice: estimated time = waves of workgroups x per-tile cost, where a
// 256x256 tile is the most efficient per flop and smaller tiles trade that for
// filling the 256 CUs when the grid would be short.
template <typename T, int EPI>
hipError_t dispatch_tiles(const GemmArgs& g, hipStream_t s) {
  struct Cand { int bm, bn; double cost; };
  const Cand cands[3] = {{256, 256, 1.0}, {256, 128, 1.12}, {128, 128, 1.3}};
  int best = 0;
  double best_t = 1e300;
  for (int c = 0; c < 3; ++c) {
    if (EPI == EPI_SWIGLU && cands[c].bn < 128) continue;
    const double tiles = (double)((g.M + cands[c].bm - 1) / cands[c].bm) *
                         ((g.N + cands[c].bn - 1) / cands[c].bn);
    const double per_cu = (cands[c].bm * cands[c].bn == 65536) ? 1.0 : 2.0;  // tiles resident per CU
    const double waves = __builtin_ceil(tiles / (256.0 * per_cu));
    const double t = waves * per_cu * cands[c].bm * cands[c].bn * cands[c].cost;
    if (t < best_t - 1e-9) { best_t = t; best = c; }
  }
  switch (best) {
    case 0: return launch_mfma<T, 256, 256, EPI>(g, s);
    case 1: return launch_mfma<T, 256, 128, EPI>(g, s);
    default: return launch_mfma<T, 128, 128, EPI>(g, s);
  }
}

template <typename T>
hipError_t dispatch_epi(const GemmArgs& g, hipStream_t s) {
  switch (g.epi) {
    case EPI_STORE_F32: return dispatch_tiles<T, EPI_STORE_F32>(g, s);
    case EPI_RESID_ADD: return dispatch_tiles<T, EPI_RESID_ADD>(g, s);
    case EPI_STORE_ACT: return dispatch_tiles<T, EPI_STORE_ACT>(g, s);
    case EPI_STORE_SILU: return dispatch_tiles<T, EPI_STORE_SILU>(g, s);
    case EPI_STORE_GELU: return dispatch_tiles<T, EPI_STORE_GELU>(g, s);
    case EPI_SWIGLU: return dispatch_tiles<T, EPI_SWIGLU>(g, s);
    case EPI_TUP: return dispatch_tiles<T, EPI_TUP>(g, s);
    case EPI_PIXEL: return dispatch_tiles<T, EPI_PIXEL>(g, s);
    case EPI_LINEAR_PIXEL: return dispatch_tiles<T, EPI_LINEAR_PIXEL>(g, s);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------------------
// fp32 GEMM (fp32 compute path): 64x64 tiles, 4x4 outputs per thread
// ---------------------------------------------------------------------------

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ W, int M, int N,
                                                       int K, int lda, int ldw, EpiParams ep) {
  constexpr int T = 64, TK = 16;
  __shared__ float As[TK][T + 1];
  __shared__ float Ws[TK][T + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += TK) {
    for (int e = tid; e < T * TK; e += 256) {
      const int r = e / TK, kk = e % TK;
      const int gm = m0 + r, gn = n0 + r, gk = k0 + kk;
      As[kk][r] = (gm < M && gk < K) ? A[(int64_t)gm * lda + gk] : 0.f;
      Ws[kk][r] = (gn < N && gk < K) ? W[(int64_t)gn * ldw + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = Ws[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx + 16 * j;
      if (col < N) epi_one<EPI, float>(ep, row, col, acc[i][j]);
    }
  }
}

template <int EPI>
hipError_t launch_f32(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
  hipLaunchKernelGGL((gemm_f32_kernel<EPI>), grid, dim3(256), 0, s, (const float*)g.A,
                     (const float*)g.W, g.M, g.N, g.K, g.lda, g.ldw, g.ep);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_mfma(Act16 t, const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.K % BK || g.lda % 8 || g.ldw % 8) return hipErrorInvalidValue;
  if (g.epi == EPI_SWIGLU && g.N % 64) return hipErrorInvalidValue;
  return t == Act16::F16 ? dispatch_epi<_Float16>(g, s) : dispatch_epi<__hip_bfloat16>(g, s);
}

hipError_t gemm_f32(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  switch (g.epi) {
    case EPI_STORE_F32: return launch_f32<EPI_STORE_F32>(g, s);
    case EPI_RESID_ADD: return launch_f32<EPI_RESID_ADD>(g, s);
    case EPI_STORE_ACT: return launch_f32<EPI_STORE_ACT>(g, s);
    case EPI_STORE_SILU: return launch_f32<EPI_STORE_SILU>(g, s);
    case EPI_STORE_GELU: return launch_f32<EPI_STORE_GELU>(g, s);
    case EPI_TUP: return launch_f32<EPI_TUP>(g, s);
    case EPI_PIXEL: return launch_f32<EPI_PIXEL>(g, s);
    case EPI_LINEAR_PIXEL: return launch_f32<EPI_LINEAR_PIXEL>(g, s);
    default: return hipErrorInvalidValue;  // SwiGLU: raw store + swiglu_f32 on this path
  }
}

}  // namespace fd
