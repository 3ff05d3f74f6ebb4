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
// 16-byte chunks (conflict-free for the 16 rows a ds_read_b128 serves at once).
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

// Every epilogue stores to out[row_off(row) + col_off(col)]: the destination
// offset splits into a part that depends only on the output row and a part
// that depends only on the column, so the per-element cost is one add. The
// reshapes of the temporal upsampling (Eq. temporal_upsample) and of the
// PixelShuffle store (Sec. 3.4 Step 3) are expressed this way.
template <int EPI>
__device__ __forceinline__ int64_t row_off(const EpiParams& p, int row) {
  if constexpr (EPI == EPI_TUP) {
    // row = frame L + n  ->  refinement rows (frame r_t + j) L + n
    const int f = row / p.L, n = row - f * p.L;
    return ((int64_t)f * p.r_t * p.L + n) * p.ld_out;
  } else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
    const int bo = row / p.L, n = row - bo * p.L;
    const int h = n / p.grid_w, w = n - h * p.grid_w;
    const int OW = p.grid_w * p.s;
    const int64_t OHW = (int64_t)p.grid_h * p.s * OW;
    int b, fo;
    if constexpr (EPI == EPI_PIXEL) {      // row block bo = b frames_out + fo
      b = bo / p.frames_out;
      fo = bo - b * p.frames_out;
    } else {                               // row block bo = b frames_in + f; sub-frame in col
      b = bo / p.frames_in;
      fo = (bo - b * p.frames_in) * p.r_t;
    }
    return ((int64_t)b * p.C * p.frames_out + fo) * OHW + (int64_t)p.s * h * OW + p.s * w;
  } else {
    return (int64_t)row * p.ld_out;
  }
}

template <int EPI>
__device__ __forceinline__ int64_t col_off(const EpiParams& p, int col) {
  if constexpr (EPI == EPI_TUP) {
    const int j = col / p.dim, d = col - j * p.dim;
    return (int64_t)j * p.L * p.ld_out + d;
  } else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
    const int OW = p.grid_w * p.s;
    const int64_t OHW = (int64_t)p.grid_h * p.s * OW;
    const int s2 = p.s * p.s;
    int j = 0, ch = col;
    if constexpr (EPI == EPI_LINEAR_PIXEL) {  // col = j C s^2 + c s^2 + i1 s + i2
      j = col / (p.C * s2);
      ch = col - j * p.C * s2;
    }
    const int c3 = ch / s2, rem = ch - c3 * s2;
    const int i1 = rem / p.s, i2 = rem - i1 * p.s;
    return ((int64_t)c3 * p.frames_out + j) * OHW + (int64_t)i1 * OW + i2;
  } else {
    return col;
  }
}

// Store one value (bias already added) at the precomputed offset.
template <int EPI, typename TA>
__device__ __forceinline__ void epi_store(const EpiParams& p, int64_t off, float c) {
  if constexpr (EPI == EPI_STORE_F32 || EPI == EPI_TUP) {
    p.out_f[off] = c;
  } else if constexpr (EPI == EPI_RESID_ADD) {
    p.out_f[off] += c;
  } else if constexpr (EPI == EPI_STORE_ACT) {
    ((TA*)p.out_a)[off] = to_act<TA>(c);
  } else if constexpr (EPI == EPI_STORE_SILU) {
    ((TA*)p.out_a)[off] = to_act<TA>(silu_f(c));
  } else if constexpr (EPI == EPI_STORE_GELU) {
    ((TA*)p.out_a)[off] = to_act<TA>(gelu_f(c));
  } else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
    p.out_f[off] = p.clamp ? fminf(1.f, fmaxf(-1.f, c)) : c;
  }
}

template <int EPI, typename TA>
__device__ __forceinline__ void epi_one(const EpiParams& p, int row, int col, float c) {
  epi_store<EPI, TA>(p, row_off<EPI>(p, row) + col_off<EPI>(p, col), c + p.bias[col]);
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
// gfx950 LDS serves 16 lanes of a ds_read_b128 per cycle from 64 banks, i.e.
// 16 groups of 16 bytes; chunk p of row r sits in group 8 (r % 2) + p. XOR-ing
// the chunk with (r / 2) % 8 puts the 16 consecutive rows a wave reads together
// in 16 different groups (and keeps the row-wise stores conflict-free).
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * 8 + (chunk ^ ((row >> 1) & 7));
}

// Raw buffer resource over `bytes` bytes at `base`: loads at offsets past the
// end return zeros, which covers the ragged M / N edges of a tile.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t soff) {
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0);
  return *reinterpret_cast<uint4*>(&v);
}

// Workgroup -> output tile. The hardware deals workgroups round-robin to the 8
// XCDs (workgroup i runs on XCD i % 8), each with its own L2. Give every XCD a
// contiguous range of tiles, and order tiles in groups of GROUP_M row blocks so
// that the tiles an XCD runs at once cover a compact 2D region: their A row
// blocks and W column blocks are then shared through that XCD's L2.
constexpr int GROUP_M = 8;
__device__ __forceinline__ void tile_of(int bid, int n_tiles, int tiles_m, int tiles_n, int& tm,
                                        int& tn) {
  const int q = n_tiles / 8, r = n_tiles % 8, x = bid % 8, i = bid / 8;
  const int t = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
  const int per_group = GROUP_M * tiles_n;
  const int grp = t / per_group, first_m = grp * GROUP_M;
  const int gm = min(GROUP_M, tiles_m - first_m);
  const int in = t - grp * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

// Tile configuration of the MFMA GEMM: BM x BN output tile, WAVES_M x WAVES_N
// wave64s (each a (BM / WAVES_M) x (BN / WAVES_N) sub-tile of 32x32 MFMA
// blocks), PF = 1 or 2 K-tiles of global loads in flight in registers.
template <int BM_, int BN_, int WAVES_M_, int WAVES_N_, int PF_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, PF = PF_;
  static constexpr int NT = 64 * WAVES_M * WAVES_N;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int CA = BM * 8 / NT, CB = BN * 8 / NT;  // 16-byte chunks per thread
  static constexpr int LDS_BYTES = 2 * (BM + BN) * BK * 2;
  static constexpr int MIN_BLOCKS = (163840 / LDS_BYTES) < 2 ? 1 : 2;
};

template <typename T, class C, int EPI>
__global__ __launch_bounds__(C::NT, C::MIN_BLOCKS) void gemm_mfma_kernel(
    const T* __restrict__ A, const T* __restrict__ W, int M, int N, int K, int lda, int ldw,
    EpiParams ep, int tiles_m, int tiles_n) {
  constexpr int BM = C::BM, BN = C::BN, FM = C::FM, FN = C::FN, CA = C::CA, CB = C::CB;
  constexpr int NT = C::NT;
  using V = typename Mfma<T>::V;

  extern __shared__ uint4 lds[];
  // LDS buffer b: A tile at lds + b (BM + BN) 8, W tile right after it
  auto As = [&](int b) { return lds + b * (BM + BN) * 8; };
  auto Bs = [&](int b) { return lds + b * (BM + BN) * 8 + BM * 8; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm0 = (wave / C::WAVES_N) * C::WM, wn0 = (wave % C::WAVES_N) * C::WN;

  // global -> register staging through buffer loads; chunk i of this thread is
  // row (tid / 8) + (NT / 8) i, 16-byte column (tid % 8) of the tile
  const __amdgpu_buffer_rsrc_t rA =
      make_rsrc(A + (int64_t)m0 * lda, (uint32_t)min(BM, M - m0) * lda * (uint32_t)sizeof(T));
  const __amdgpu_buffer_rsrc_t rB =
      make_rsrc(W + (int64_t)n0 * ldw, (uint32_t)min(BN, N - n0) * ldw * (uint32_t)sizeof(T));
  const uint32_t offA = ((tid >> 3) * lda + (tid & 7) * 8) * (uint32_t)sizeof(T);
  const uint32_t offB = ((tid >> 3) * ldw + (tid & 7) * 8) * (uint32_t)sizeof(T);
  constexpr int RSTEP = NT / 8;  // rows between a thread's chunks
  const uint32_t stepA = RSTEP * lda * (uint32_t)sizeof(T), stepB = RSTEP * ldw * (uint32_t)sizeof(T);
  const int lds_w = swz(tid >> 3, tid & 7);  // + NT i for chunk i
  uint4 ra0[CA], rb0[CB], ra1[C::PF == 2 ? CA : 1], rb1[C::PF == 2 ? CB : 1];
#define FD_GLOAD(RA, RB, KT)                                                   \
  do {                                                                         \
    const uint32_t koff = (KT) * BK * (uint32_t)sizeof(T);                     \
    _Pragma("unroll") for (int i = 0; i < CA; ++i) RA[i] = buf_load16(rA, offA + i * stepA, koff); \
    _Pragma("unroll") for (int i = 0; i < CB; ++i) RB[i] = buf_load16(rB, offB + i * stepB, koff); \
  } while (0)
#define FD_LSTORE(RA, RB, BUF)                                                 \
  do {                                                                         \
    _Pragma("unroll") for (int i = 0; i < CA; ++i) As(BUF)[lds_w + i * NT] = RA[i]; \
    _Pragma("unroll") for (int i = 0; i < CB; ++i) Bs(BUF)[lds_w + i * NT] = RB[i]; \
  } while (0)

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lr = lane & 31, lk = lane >> 5;
  // MFMA operand fragments of one 16-wide k-step, double-buffered so that the
  // LDS reads of step ks + 1 are in flight while the MFMAs of step ks run.
  V fa[2][FM], fb[2][FN];
  auto load_frags = [&](int slot, int buf, int ks) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint4 v = As(buf)[swz(wm0 + i * 32 + lr, 2 * ks + lk)];
      fa[slot][i] = *reinterpret_cast<const V*>(&v);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint4 v = Bs(buf)[swz(wn0 + j * 32 + lr, 2 * ks + lk)];
      fb[slot][j] = *reinterpret_cast<const V*>(&v);
    }
  };
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(fa[slot][i], fb[slot][j], acc[i][j]);
  };
  // One K tile from LDS buffer `buf`; `mid` runs between k-steps 1 and 2.
  auto compute_tile = [&](int buf, auto mid) {
    load_frags(0, buf, 0);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      if (ks + 1 < BK / 16) {
        load_frags((ks + 1) & 1, buf, ks + 1);
        // issue the next step's LDS reads ahead of this step's MFMAs
        __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
      }
      mfmas(ks & 1);
      __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
      if (ks == 1) mid();
    }
  };
  auto compute = [&](int buf) { compute_tile(buf, [] {}); };

  const int KT = K / BK;
  if constexpr (C::PF == 2) {
    // two register stages: tile kt + 2 is in flight while tile kt is computed;
    // two K tiles per trip so that the stages have static names
    FD_GLOAD(ra0, rb0, 0);
    if (KT > 1) FD_GLOAD(ra1, rb1, 1);
    FD_LSTORE(ra0, rb0, 0);
    __syncthreads();
    for (int kt = 0; kt < KT; kt += 2) {
      if (kt + 2 < KT) FD_GLOAD(ra0, rb0, kt + 2);
      compute(0);
      if (kt + 1 < KT) FD_LSTORE(ra1, rb1, 1);
      __syncthreads();
      if (kt + 1 >= KT) break;
      if (kt + 3 < KT) FD_GLOAD(ra1, rb1, kt + 3);
      compute(1);
      if (kt + 2 < KT) FD_LSTORE(ra0, rb0, 0);
      __syncthreads();
    }
  } else {
    // one register stage: tile kt + 1 is loaded while tile kt is computed, and
    // written to the other LDS buffer (free since the last barrier) halfway
    // through and at the end of the MFMA work, so the stores overlap MFMA
    FD_GLOAD(ra0, rb0, 0);
    FD_LSTORE(ra0, rb0, 0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int cur = kt & 1, nxt = cur ^ 1;
      const bool more = kt + 1 < KT;
      if (more) FD_GLOAD(ra0, rb0, kt + 1);
      compute_tile(cur, [&] {
        if (more) {
          _Pragma("unroll") for (int i = 0; i < CA; ++i) As(nxt)[lds_w + i * NT] = ra0[i];
        }
      });
      if (more) {
        _Pragma("unroll") for (int i = 0; i < CB; ++i) Bs(nxt)[lds_w + i * NT] = rb0[i];
      }
      __syncthreads();
    }
  }
#undef FD_GLOAD
#undef FD_LSTORE

  // epilogue: lane holds column (lane & 31) of each 32x32 block and rows
  // 8 (r / 4) + 4 (lane / 32) + r % 4
  if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int pc = n0 + wn0 + j * 32 + lr;  // packed gate column; up is +32
          if (pc >= N) continue;
          const float g = acc[i][j][r] + ep.bias[pc];
          const float u = acc[i][j + 1][r] + ep.bias[pc + 32];
          const int oc = (n0 + wn0 + j * 32) / 2 + lr;
          ((T*)ep.out_a)[(int64_t)row * ep.ld_out + oc] = to_act<T>(silu_f(g) * u);
        }
      }
  } else {
    int64_t coff[FN];
    float cb[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = min(n0 + wn0 + j * 32 + lr, N - 1);
      coff[j] = col_off<EPI>(ep, col);
      cb[j] = ep.bias[col];
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
        if (row >= M) continue;
        const int64_t ro = row_off<EPI>(ep, row);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          if (n0 + wn0 + j * 32 + lr < N) epi_store<EPI, T>(ep, ro + coff[j], acc[i][j][r] + cb[j]);
      }
  }
}

template <typename T, class C, int EPI>
hipError_t launch_mfma(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + C::BM - 1) / C::BM, tn = (g.N + C::BN - 1) / C::BN;
  static bool attr_set = false;  // raise the dynamic LDS limit once per instantiation
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_mfma_kernel<T, C, EPI>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((gemm_mfma_kernel<T, C, EPI>), dim3(tm * tn), dim3(C::NT), C::LDS_BYTES, s,
                     (const T*)g.A, (const T*)g.W, g.M, g.N, g.K, g.lda, g.ldw, g.ep, tm, tn);
  return hipGetLastError();
}

// Tile choice. 256 x 256 tiles load half the bytes per flop of 128 x 128 ones
// (128 vs 64 flop/byte), which keeps the 256 CUs within L2 bandwidth, but the
// decoder's small-M projections (M = 3600 rows per 720p frame, N = 1536 or
// 1920) give only 90-120 such tiles for 256 CUs; there 128 x 128 tiles (two
// workgroups per CU) are faster. Threshold measured on the 480p / 720p shapes.
using TileBig = TileCfg<256, 256, 4, 2, 1>;    // 8 waves of 64 x 128, one workgroup per CU
using TileSmall = TileCfg<128, 128, 2, 2, 2>;  // 4 waves of 64 x 64, two workgroups per CU

template <typename T, int EPI>
hipError_t dispatch_tiles(const GemmArgs& g, hipStream_t s) {
  const int tiles_big = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (tiles_big >= 160) return launch_mfma<T, TileBig, EPI>(g, s);
  return launch_mfma<T, TileSmall, EPI>(g, s);
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
