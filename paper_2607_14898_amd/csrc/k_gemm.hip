// Dense projections of the decoder: C = A W^T + b with fused epilogues.
//
// Every Linear layer of the decoder goes through here: the latent projection
// (Eq. projection), the QKV / output / MLP projections of each block (Sec. 3.2),
// the temporal upsampling Linear D -> r_t D (Eq. temporal_upsample) and the
// 2-layer pixel head (Sec. 3.4 Step 3). The epilogues fuse what follows each
// projection: bias, residual add into the fp32 stream, SiLU / GELU / SwiGLU,
// the channel -> sub-frame reshape of Step 1 and the PixelShuffle store.
//
// 16-bit path: one workgroup of wave64s computes a BM x BN tile with the
// gfx950 32x32x16 MFMA (fp32 accumulate). A and W are both K-contiguous; K
// tiles of 32 columns are copied from memory straight into LDS by the buffer
// unit (buffer_load ... lds, no register staging) several tiles ahead of the
// MFMAs, and read back as MFMA fragments with 16-byte ds_read_b128 per lane
// through a per-row XOR swizzle of the 16-byte chunks that keeps the 16 rows
// one ds_read_b128 serves at once in 16 different bank groups.
#include "fd_kernels.h"

#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>

#include <type_traits>

namespace fd {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// SiLU with the hardware reciprocal (1 ulp) instead of an IEEE division; the
// limits hold: x -> -inf gives x * rcp(inf) = -0.
__device__ __forceinline__ float silu_f(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }
__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

template <typename T> __device__ __forceinline__ T to_act(float v);
template <> __device__ __forceinline__ _Float16 to_act<_Float16>(float v) { return (_Float16)v; }
template <> __device__ __forceinline__ __hip_bfloat16 to_act<__hip_bfloat16>(float v) { return __float2bfloat16(v); }
// bit pattern of a 16-bit value (for packed stores without a stack array)
__device__ __forceinline__ uint32_t bits16(_Float16 x) { return __builtin_bit_cast(uint16_t, x); }
__device__ __forceinline__ uint32_t bits16(__hip_bfloat16 x) { return __bfloat16_as_ushort(x); }
template <> __device__ __forceinline__ float to_act<float>(float v) { return v; }

// A value bound for a 16-bit operand, clamped to the fp16 range when T is
// fp16 (+-65504; NaN passes unchanged), counting the clamped values in n.
template <typename T>
__device__ __forceinline__ float sat16(float v, int& n) {
  if constexpr (std::is_same<T, _Float16>::value) {
    const bool big = fabsf(v) > 65504.f;
    n += big;
    return big ? copysignf(65504.f, v) : v;
  } else {
    return v;
  }
}

// Adds this wave's count of clamped values to *sat (one atomic per wave that
// clamped anything).
__device__ __forceinline__ void count_sat(unsigned* sat, int n) {
  if (!sat || __builtin_amdgcn_ballot_w64(n != 0) == 0) return;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o);
  if ((threadIdx.x & 63) == 0) atomicAdd(sat, (unsigned)n);
}

// Every epilogue stores to out[row_off(row) + col_off(col)]: the destination
// offset splits into a part that depends only on the output row and a part
// that depends only on the column, so the per-element cost is one add. The
// reshapes of the temporal upsampling (Eq. temporal_upsample) and of the
// PixelShuffle store (Sec. 3.4 Step 3) are expressed this way, and so is the
// packed operand layout of 16-bit activations (blocks of 16 rows x 32
// columns: row part (row / 16) 16 ld + (row % 16) 32, column part
// (col / 32) 512 + col % 32).
template <int EPI>
constexpr bool kPackable = EPI == EPI_SWIGLU || EPI == EPI_STORE_ACT || EPI == EPI_STORE_SILU ||
                           EPI == EPI_STORE_GELU;
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
    if constexpr (kPackable<EPI>)
      if (p.out_packed) return (int64_t)(row >> 4) * p.ld_out * 16 + (row & 15) * 32;
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
    if constexpr (kPackable<EPI>)
      if (p.out_packed) return (int64_t)(col >> 5) * 512 + (col & 31);
    return col;
  }
}

// One output pixel: clamped to [-1, 1] if requested, then in the destination
// format (fp32; bf16 rounded to nearest even; uint8 = rint of the fp32 fma
// x 127.5 + 127.5, ties to even, limited to 0..255).
__device__ __forceinline__ float px_clamp(const EpiParams& p, float v) {
  return p.clamp ? fminf(1.f, fmaxf(-1.f, v)) : v;
}
__device__ __forceinline__ uint32_t px_u8(float v) {
  return (uint32_t)fminf(255.f, fmaxf(0.f, rintf(fmaf(v, 127.5f, 127.5f))));
}
// PXF: the format when known at compile time, -1 to read p.out_fmt
template <int PXF>
__device__ __forceinline__ void px_store(const EpiParams& p, int64_t off, float v) {
  const int f = PXF >= 0 ? PXF : p.out_fmt;
  v = px_clamp(p, v);
  if (f == 0) p.out_f[off] = v;
  else if (f == 1) reinterpret_cast<__hip_bfloat16*>(p.out_f)[off] = __float2bfloat16(v);
  else reinterpret_cast<uint8_t*>(p.out_f)[off] = (uint8_t)px_u8(v);
}
// Four consecutive pixels at an offset that is a multiple of 4 (16-, 8- or
// 4-byte store).
template <int PXF>
__device__ __forceinline__ void px_store4(const EpiParams& p, int64_t off, const float (&v)[4]) {
  static_assert(PXF >= 0, "vector pixel stores take a compile-time format");
  float c[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) c[e] = px_clamp(p, v[e]);
  if constexpr (PXF == 0) {
    *reinterpret_cast<float4*>(p.out_f + off) = make_float4(c[0], c[1], c[2], c[3]);
  } else if constexpr (PXF == 1) {  // packed from the bit patterns (no stack array)
    auto bits = [](float x) { return (uint32_t)__bfloat16_as_ushort(__float2bfloat16(x)); };
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p.out_f) + off) =
        make_uint2(bits(c[0]) | (bits(c[1]) << 16), bits(c[2]) | (bits(c[3]) << 16));
  } else {
    *reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(p.out_f) + off) =
        px_u8(c[0]) | (px_u8(c[1]) << 8) | (px_u8(c[2]) << 16) | (px_u8(c[3]) << 24);
  }
}

// Store one value (bias already added) at the precomputed offset.
template <int EPI, typename TA, int PXF = -1>
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
    px_store<PXF>(p, off, c);
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

// Raw buffer resource over `bytes` bytes at `base`: loads at offsets past the
// end return zeros, which covers the ragged M / N edges of a tile.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
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

// Epilogue of one wave's FM x FN blocks of 32 x 32 accumulators whose first
// output row / column are r0 / c0. MFMA accumulator layout: lane (lk, lr) holds
// column lr of each block and rows 8 (r / 4) + 4 lk + r % 4 for r = 0..15.
// Loads of the destination (residual add) are issued for a whole 32-row block
// before any of its stores: interleaved, every load would wait for the store
// before it (the compiler cannot tell the addresses apart) and each element
// would cost a full memory round trip.
// x / d for 0 <= x < 2^23 and 0 < d, given inv = 1.0f / d (float product, then
// one exact integer correction)
__device__ __forceinline__ int div_small(int x, int d, float inv) {
  int q = (int)((float)x * inv);
  const int r = x - q * d;
  return q + (r >= d) - (r < 0);
}

template <int EPI, typename T, int FM, int FN, bool FAST_RMW, int PXF = 0>
__device__ __forceinline__ void store_tile(const EpiParams& ep, const f32x16 (&acc)[FM][FN], int r0,
                                           int c0, int M, int N, int lr, int lk, float* ws) {
  if constexpr (EPI == EPI_QKV) {
    // The QKV projection's post step (Sec. 3.2, Eq. kv_cache): a wave's 64
    // columns are one head vector (head slot c0 / 64: query heads, then key
    // groups, then value groups). Each 32-row block of the wave goes through
    // the wave's share of the stage buffers (free once the K loop is done): 16 lanes then hold
    // 4 columns of one row, so the KV-norm (RMS over the 64 columns) is a
    // 16-lane sum and the 3D-RoPE pairs sit inside a lane. Queries go to the
    // query buffer, keys to their ring slot, values (normalised in LDS, then
    // one lane per column) transposed to the V ring.
    static_assert(FN == 2, "one 64-column head vector per wave");
    const QkvPostArgs& a = ep.qkv;
    const int lane = lk * 32 + lr;
    const int wave = threadIdx.x >> 6;
    const int hs = c0 >> 6;
    const bool is_q = hs < a.N, is_v = hs >= a.N + a.G;
    const float* gn = is_q ? nullptr : (is_v ? a.vnorm_g : a.knorm_g);
    const int kvg = hs - a.N - (is_v ? a.G : 0);  // KV group
    const int cq = 4 * (lane & 15);               // this lane's 4 columns in the second pass
    float4 gq = make_float4(1.f, 1.f, 1.f, 1.f);
    if (gn) gq = *reinterpret_cast<const float4*>(gn + cq);
    const bool rope = a.rope && !is_v;
    const int pa = cq >> 1;  // RoPE pairs pa and pa + 1 of columns cq .. cq + 3
    const int ax0 = rope ? a.rope_axis[pa] : 0, ax1 = rope ? a.rope_axis[pa + 1] : 0;
    const float inv_rpb = 1.f / a.rows_per_batch, inv_L = 1.f / a.L;
    const float inv_gw = 1.f / a.grid_w, inv_U = 1.f / a.U;
    const int slot0 = (int)(a.u0 % a.S);
    const float bias0 = ep.bias[min(c0, N - 64) + lr], bias1 = ep.bias[min(c0, N - 64) + 32 + lr];
    constexpr int LS = 68;  // row stride: rows 4 apart fall in other banks, rows stay 16-byte aligned
    float* wl = ws + wave * (32 * LS);  // [32 rows][64 columns]
    // row of the call -> (stream, unit, position) and (sub-frame, h, w)
    auto split = [&](int row, int& b, int& lu, int& pos, int& fs, int& hh, int& ww) {
      b = div_small(row, a.rows_per_batch, inv_rpb);
      const int rb = row - b * a.rows_per_batch;
      lu = div_small(rb, a.U, inv_U);
      pos = rb - lu * a.U;
      fs = div_small(rb, a.L, inv_L);
      const int tok = rb - fs * a.L;
      hh = div_small(tok, a.grid_w, inv_gw);
      ww = tok - hh * a.grid_w;
    };
    __syncthreads();  // every wave is past its last read of the stage buffers
    if (c0 >= N) return;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int rbase = r0 + i * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rr = 8 * (r >> 2) + 4 * lk + (r & 3);
        wl[rr * LS + lr] = acc[i][0][r] + bias0;
        wl[rr * LS + 32 + lr] = acc[i][1][r] + bias1;
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS writes are done
      for (int it = 0; it < 8; ++it) {
        const int rr = it * 4 + (lane >> 4);
        const int row_t = rbase + rr, row = min(row_t, M - 1);
        float4 v = *reinterpret_cast<const float4*>(wl + rr * LS + cq);
        if (gn) {
          float ss = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
          const float rn = rsqrtf(ss * (1.f / 64.f) + a.eps);
          v = make_float4(v.x * rn * gq.x, v.y * rn * gq.y, v.z * rn * gq.z, v.w * rn * gq.w);
        }
        int b, lu, pos, fs, hh, ww;
        split(row, b, lu, pos, fs, hh, ww);
        if (rope) {
          const float2 c0v = ax0 == 0 ? a.rope_t[fs * 32 + pa] : a.rope_hw[(ax0 == 1 ? hh : ww) * 32 + pa];
          const float2 c1v = ax1 == 0 ? a.rope_t[fs * 32 + pa + 1] : a.rope_hw[(ax1 == 1 ? hh : ww) * 32 + pa + 1];
          v = make_float4(v.x * c0v.x - v.y * c0v.y, v.x * c0v.y + v.y * c0v.x,
                          v.z * c1v.x - v.w * c1v.y, v.z * c1v.y + v.w * c1v.x);
        }
        if (is_v) {  // normalised values back to LDS for the transposed store
          *reinterpret_cast<float4*>(wl + rr * LS + cq) = v;
          continue;
        }
        if (row_t >= M) continue;
        T o4[4] = {to_act<T>(v.x), to_act<T>(v.y), to_act<T>(v.z), to_act<T>(v.w)};
        T* dst;
        if (is_q) {
          dst = (T*)a.q + (int64_t)row * (a.N * 64) + c0 + cq;
        } else {
          const int slot = (slot0 + lu) % a.S;
          dst = (T*)a.k_ring + (((int64_t)(b * a.G + kvg) * a.S + slot) * a.U_pad + pos) * 64 + cq;
        }
        *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(o4);
      }
      if (is_v) {  // V^T[dim][pos] of the block's 32 rows
        // lane l % 16 takes rows 2 (l % 16) and 2 (l % 16) + 1, lane / 16 picks
        // the dimension: each store instruction writes 32 consecutive positions
        // of 4 dimensions (four 64-byte segments), as 4-byte pairs where the
        // two rows are adjacent in one ring slot
        __builtin_amdgcn_s_waitcnt(0xC07F);
        const int l16 = lane & 15, dg = lane >> 4;
        const int ra = rbase + 2 * l16;
        const bool oka = ra < M, okb = ra + 1 < M;
        int b0, lu0, pos0, b1, lu1, pos1, fs, hh, ww;
        split(min(ra, M - 1), b0, lu0, pos0, fs, hh, ww);
        split(min(ra + 1, M - 1), b1, lu1, pos1, fs, hh, ww);
        T* va = (T*)a.vt_ring + ((int64_t)(b0 * a.G + kvg) * a.S + (slot0 + lu0) % a.S) * 64 * a.U_pad + pos0;
        T* vb = (T*)a.vt_ring + ((int64_t)(b1 * a.G + kvg) * a.S + (slot0 + lu1) % a.S) * 64 * a.U_pad + pos1;
        const bool pair = oka && okb && vb == va + 1 && (pos0 & 1) == 0;
#pragma unroll 4
        for (int it = 0; it < 16; ++it) {
          const int d = it * 4 + dg;
          const T x0 = to_act<T>(wl[(2 * l16) * LS + d]), x1 = to_act<T>(wl[(2 * l16 + 1) * LS + d]);
          if (pair) {
            *reinterpret_cast<uint32_t*>(va + (int64_t)d * a.U_pad) = bits16(x0) | (bits16(x1) << 16);
          } else {
            if (oka) va[(int64_t)d * a.U_pad] = x0;
            if (okb) vb[(int64_t)d * a.U_pad] = x1;
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // the block's LDS reads are done before the next block
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    float bg[FN / 2], bu[FN / 2];
#pragma unroll
    for (int j = 0; j < FN; j += 2) {
      const int pc = min(c0 + j * 32 + lr, N - 33);  // packed gate column; up is +32
      bg[j / 2] = ep.bias[pc];
      bu[j / 2] = ep.bias[pc + 32];
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = r0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          if (c0 + j * 32 + lr >= N) continue;
          const float g = acc[i][j][r] + bg[j / 2];
          const float u = acc[i][j + 1][r] + bu[j / 2];
          const int oc = (c0 + j * 32) / 2 + lr;
          ((T*)ep.out_a)[(int64_t)row * ep.ld_out + oc] = to_act<T>(silu_f(g) * u);
        }
      }
  } else {
    int64_t coff[FN];
    float cb[FN];
    bool cok[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int col = min(c0 + j * 32 + lr, N - 1);
      coff[j] = col_off<EPI>(ep, col);
      cb[j] = ep.bias[col];
      cok[j] = c0 + j * 32 + lr < N;
    }
    // interior blocks (the wave's rows and columns all in range) skip the
    // per-element checks; for the residual read-modify-write only where other
    // waves of the CU cover its load latency (measured: slower on a lone
    // 4-wave workgroup per CU)
    const bool interior = (EPI != EPI_RESID_ADD || FAST_RMW) && r0 + FM * 32 <= M && c0 + FN * 32 <= N;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      int64_t ro[16];
      bool rok[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = r0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3);
        rok[r] = row < M;
        ro[r] = row_off<EPI>(ep, min(row, M - 1));
      }
      if (interior) {
        if constexpr (EPI == EPI_RESID_ADD || EPI == EPI_STORE_F32) {
          // row-major destination: column blocks j are 32 floats apart, an
          // immediate offset from one row pointer
          float* rp[16];
#pragma unroll
          for (int r = 0; r < 16; ++r)
            rp[r] = ep.out_f + (int64_t)(r0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3)) * ep.ld_out + c0 + lr;
          if constexpr (EPI == EPI_RESID_ADD) {
            float old[16][FN];
#pragma unroll
            for (int r = 0; r < 16; ++r)
#pragma unroll
              for (int j = 0; j < FN; ++j) old[r][j] = rp[r][32 * j];
#pragma unroll
            for (int r = 0; r < 16; ++r)
#pragma unroll
              for (int j = 0; j < FN; ++j) rp[r][32 * j] = old[r][j] + (acc[i][j][r] + cb[j]);
          } else {
#pragma unroll
            for (int r = 0; r < 16; ++r)
#pragma unroll
              for (int j = 0; j < FN; ++j) rp[r][32 * j] = acc[i][j][r] + cb[j];
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r)
#pragma unroll
            for (int j = 0; j < FN; ++j) epi_store<EPI, T, PXF>(ep, ro[r] + coff[j], acc[i][j][r] + cb[j]);
        }
        continue;
      }
      if constexpr (EPI == EPI_RESID_ADD) {
        float old[16][FN];
#pragma unroll
        for (int r = 0; r < 16; ++r)
#pragma unroll
          for (int j = 0; j < FN; ++j) old[r][j] = rok[r] && cok[j] ? ep.out_f[ro[r] + coff[j]] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            if (rok[r] && cok[j]) ep.out_f[ro[r] + coff[j]] = old[r][j] + (acc[i][j][r] + cb[j]);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            if (rok[r] && cok[j]) epi_store<EPI, T, PXF>(ep, ro[r] + coff[j], acc[i][j][r] + cb[j]);
      }
    }
  }
}

// Epilogue of one wave's blocks computed transposed (acc[i][j] = W block j
// times A block i): lane (lk, lr) holds output row r0 + 32 i + lr and, in
// registers 4 q .. 4 q + 3, the four consecutive columns c0 + 32 j + 8 q +
// 4 lk + 0..3. Every destination access covers those four columns at once (one
// 16-byte fp32 or 8-byte 16-bit access) whenever the four land contiguously;
// vec == false (a ragged or unaligned destination) stores element by element.
template <int EPI, typename T, int FM, int FN, bool SCALED = false, int PXF = 0>
__device__ __forceinline__ void store_tile_t(const EpiParams& ep, const f32x16 (&acc)[FM][FN], int r0,
                                             int c0, int M, int N, int lr, int lk, bool vec) {
  // SCALED (FP8 GEMM, SwiGLU only): each accumulator is multiplied by its
  // column's then its row's dequantisation scale right before use
  static_assert(!SCALED || EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_E4M3, "scaled transposed epilogue: SwiGLU only");
  typedef __attribute__((ext_vector_type(4))) float f4;
  int nsat = 0;  // fp16 values clamped to +-65504 by this lane
  int64_t ro[FM];
  bool rok[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = r0 + i * 32 + lr;
    rok[i] = row < M;
    ro[i] = row_off<EPI>(ep, min(row, M - 1));
  }
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_E4M3) {
    float rs[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      rs[i] = SCALED ? ep.row_scale[min(r0 + i * 32 + lr, M - 1) * ep.row_scale_stride] : 1.f;
    const float q_inv = EPI == EPI_SWIGLU_E4M3 ? ep.out_scale[1] : 1.f;
    // gate block j and up block j + 1 give output columns (c0 + 32 j) / 2 + 0..31
#pragma unroll
    for (int j = 0; j < FN; j += 2)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int lc = 8 * q + 4 * lk, pc = c0 + j * 32 + lc;
        if (pc >= N) continue;  // N % 64 == 0: a group is valid as a whole
        float bg[4], bu[4], sg[4], su[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bg[e] = ep.bias[pc + e];
          bu[e] = ep.bias[pc + 32 + e];
          sg[e] = SCALED ? ep.col_scale[pc + e] : 1.f;
          su[e] = SCALED ? ep.col_scale[pc + 32 + e] : 1.f;
        }
        const int oc = (c0 + j * 32) / 2 + lc;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          if (!rok[i]) continue;
          T o4[4];
          float h4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float g = acc[i][j][4 * q + e], u = acc[i][j + 1][4 * q + e];
            if (SCALED) {
              g = g * sg[e] * rs[i];
              u = u * su[e] * rs[i];
            }
            o4[e] = to_act<T>(sat16<T>(silu_f(g + bg[e]) * (u + bu[e]), nsat));
            h4[e] = (float)o4[e];
          }
          if constexpr (EPI == EPI_SWIGLU_E4M3) {
            // codes of the fp16-rounded hidden value at the static scale (saturating)
            auto cl = [&](float v) { return fminf(448.f, fmaxf(-448.f, v * q_inv)); };
            int w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(h4[0]), cl(h4[1]), 0, false);
            w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(h4[2]), cl(h4[3]), w, true);
            // E4M3 codes: row-major, or the FP8 GEMM's packed operand layout
            // (blocks of 16 rows x 64 bytes)
            const int64_t rr = r0 + i * 32 + lr;
            const int64_t bo = ep.out_packed ? (rr >> 4) * ep.ld_out * 16 + (rr & 15) * 64 +
                                                   (int64_t)(oc >> 6) * 1024 + (oc & 63)
                                             : ro[i] + oc;
            *reinterpret_cast<int*>((uint8_t*)ep.out_a + bo) = w;
            continue;
          }
          *reinterpret_cast<uint2*>((T*)ep.out_a + ro[i] + col_off<EPI>(ep, oc)) =
              *reinterpret_cast<const uint2*>(o4);
        }
      }
  } else {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      int64_t co[4];
      float cb[4][4];
      bool cok[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = c0 + j * 32 + 8 * q + 4 * lk;
        cok[q] = n < N;
        co[q] = col_off<EPI>(ep, min(n, N - 1));
#pragma unroll
        for (int e = 0; e < 4; ++e) cb[q][e] = ep.bias[min(n + e, N - 1)];
      }
      if (!vec) {  // element by element
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int n = c0 + j * 32 + 8 * q + 4 * lk + e;
              if (!(rok[i] && n < N)) continue;
              if constexpr (EPI == EPI_STORE_SILU)
                ((T*)ep.out_a)[ro[i] + col_off<EPI>(ep, n)] = to_act<T>(sat16<T>(silu_f(acc[i][j][4 * q + e] + cb[q][e]), nsat));
              else
                epi_store<EPI, T, PXF>(ep, ro[i] + col_off<EPI>(ep, n), acc[i][j][4 * q + e] + cb[q][e]);
            }
        continue;
      }
      if constexpr (EPI == EPI_RESID_ADD) {
        // the four loads of a row before its stores (the compiler cannot tell
        // the addresses apart and would otherwise serialise each pair)
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          if (!rok[i]) continue;
          f4 old[4];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (cok[q]) old[q] = *reinterpret_cast<const f4*>(ep.out_f + ro[i] + co[q]);
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (cok[q]) {
              f4 v;
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = old[q][e] + (acc[i][j][4 * q + e] + cb[q][e]);
              *reinterpret_cast<f4*>(ep.out_f + ro[i] + co[q]) = v;
            }
        }
      } else {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (!(rok[i] && cok[q])) continue;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e] + cb[q][e];
            const int64_t off = ro[i] + co[q];
            if constexpr (EPI == EPI_STORE_F32 || EPI == EPI_TUP) {
              *reinterpret_cast<f4*>(ep.out_f + off) = f4{v[0], v[1], v[2], v[3]};
            } else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
              px_store4<PXF>(ep, off, v);
            } else {
              T o4[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                if constexpr (EPI == EPI_STORE_SILU) o4[e] = to_act<T>(sat16<T>(silu_f(v[e]), nsat));
                else if constexpr (EPI == EPI_STORE_GELU) o4[e] = to_act<T>(gelu_f(v[e]));
                else o4[e] = to_act<T>(v[e]);
              }
              *reinterpret_cast<uint2*>((T*)ep.out_a + off) = *reinterpret_cast<const uint2*>(o4);
            }
          }
      }
    }
  }
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_E4M3 || EPI == EPI_STORE_SILU) count_sat(ep.sat, nsat);
}

// ---------------------------------------------------------------------------
// 16-bit MFMA GEMM. K tiles of 32 columns go from memory straight into LDS
// with buffer_load_dwordx4 ... lds (no register staging, no LDS store
// instructions), NS tiles deep: while tile t is multiplied, tiles t + 1 ..
// t + NS - 1 are in flight. A DMA instruction writes the 16 bytes of lane l to
// LDS slot l after a wave-uniform base, so the bank swizzle is applied on the
// global side: lane l fetches the chunk that belongs in slot l.
// ---------------------------------------------------------------------------
constexpr int BKD = 32;  // K-columns per stage: 4 chunks of 16 bytes per row

// Tile configuration: BM x BN output tile, WAVES_M x WAVES_N wave64s (each a
// (BM / WAVES_M) x (BN / WAVES_N) sub-tile of 32 x 32 MFMA blocks), NS stages.
template <int BM_, int BN_, int WAVES_M_, int WAVES_N_, int NS_, bool IL_ = false>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, NS = NS_;
  // IL: the stage refill DMAs are spread between the MFMAs instead of issued
  // as one burst between two k-steps
  static constexpr bool IL = IL_;
  static constexpr int NW = WAVES_M * WAVES_N, NT = 64 * NW;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N, FM = WM / 32, FN = WN / 32;
  static constexpr int STAGE = (BM + BN) * 4;                 // 16-byte slots per stage
  static constexpr int QA = BM / 16 / NW, QB = BN / 16 / NW;  // DMAs per thread and stage
  static constexpr int LDS_BYTES = NS * STAGE * 16;
  static constexpr int MIN_BLOCKS = 163840 / LDS_BYTES >= 2 ? 2 : 1;
  static_assert(BM % (16 * NW) == 0 && BN % (16 * NW) == 0, "DMA rows split evenly over waves");
  static_assert(NS >= 3 && LDS_BYTES <= 163840, "at least 3 stages, within 160 KB of LDS");
  static_assert((NS - 2) * (QA + QB) < 64, "vmcnt range");
};

// s_waitcnt immediates (gfx9 encoding): vmcnt(n) with lgkmcnt and expcnt
// untouched, and lgkmcnt(0) alone.
#define FD_VMCNT(n) ((((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8)))
#define FD_LGKMCNT0 (0xF | (0x3 << 14) | (0x7 << 4))

// Stage row r (A rows 0..BM-1, then W rows) holds K-chunk c of that row in
// physical slot 4 r + (c ^ ((r / 4) % 4)): the 16 rows one ds_read_b128 serves
// at once then cover all 16 bank groups.
//
// The DMAs are issued from inline assembly (M0 = LDS destination of the wave),
// so the compiler neither sees nor orders them; every ordering they need is
// explicit: s_waitcnt on the wave's own DMAs, then s_barrier (with compiler
// memory barriers around it) before any wave reads the tile or refills a stage.
// Epilogues with 16-bit destinations take the accumulators transposed: four
// consecutive columns per lane make one 8-byte store and one bias / SiLU pass
// per four values. fp32 destinations keep the direct layout, where the 32 lanes
// of a half-wave write one full 128-byte row segment per store.
template <int EPI> constexpr bool kTransposed = EPI == EPI_SWIGLU || EPI == EPI_SWIGLU_E4M3 ||
    EPI == EPI_STORE_ACT || EPI == EPI_STORE_SILU || EPI == EPI_STORE_GELU;

template <typename T, class C, int EPI>
__global__ __launch_bounds__(C::NT, C::MIN_BLOCKS) void gemm_mfma_kernel(
    const T* __restrict__ A, const T* __restrict__ W, int M, int N, int K, int lda, int ldw,
    EpiParams ep, int tiles_m, int tiles_n, int vec_store, int a_packed) {
  constexpr int BM = C::BM, BN = C::BN, FM = C::FM, FN = C::FN, NS = C::NS, NW = C::NW;
  constexpr int QA = C::QA, Q = C::QA + C::QB, STAGE = C::STAGE;
  using V = typename Mfma<T>::V;
  __shared__ uint4 lds[NS * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  tile_of(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm0 = (wave / C::WAVES_N) * C::WM, wn0 = (wave % C::WAVES_N) * C::WN;

  // W is packed K-tile-major: blocks of 16 rows x 32 K-columns (1 KB), block
  // (row / 16, k / 32) at ((row / 16) (K / 32) + k / 32) KB, rows padded with
  // zeros to a multiple of 16, so each DMA of W reads one contiguous 1 KB
  // block. A is row-major (lda), or packed the same way (lda = K, whole
  // 16-row blocks readable).
  const int KB = K / BKD;  // K tiles
  const bool apk = a_packed != 0;
  const int a_rows = apk ? (min(BM, M - m0) + 15) / 16 * 16 : min(BM, M - m0);
  const __amdgpu_buffer_rsrc_t rA =
      make_rsrc(A + (int64_t)m0 * lda, (uint32_t)a_rows * lda * (uint32_t)sizeof(T));
  const uint32_t a_kstep = apk ? 1024u : (uint32_t)BKD * (uint32_t)sizeof(T);  // bytes per K tile
  const int nrows_w = min(BN, (N + 15) / 16 * 16 - n0);
  const __amdgpu_buffer_rsrc_t rB =
      make_rsrc(W + (int64_t)(n0 / 16) * KB * 512, (uint32_t)(nrows_w / 16) * KB * 1024u);
  (void)ldw;
  // DMA j of this wave fills stage rows 16 q .. 16 q + 15, q = j NW + wave (A
  // rows for j < QA, W rows after); lane l lands in row 16 q + l / 4, physical
  // chunk l % 4, which holds K-chunk (l % 4) ^ ((l / 16) % 4).
  const int lrow = lane >> 2, lchunk = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t voff[Q];
#pragma unroll
  for (int j = 0; j < Q; ++j) {
    const int q = j * NW + wave;
    voff[j] = j >= QA ? (uint32_t)(q - BM / 16) * KB * 1024u + (uint32_t)(lrow * 64 + lchunk * 16)
              : apk   ? (uint32_t)q * KB * 1024u + (uint32_t)(lrow * 64 + lchunk * 16)
                      : (uint32_t)((16 * q + lrow) * lda + lchunk * 8) * (uint32_t)sizeof(T);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)lds;
  // DMA instruction j of the refill of stage st with K tile kt
  auto dma1 = [&](int st, int kt, int j) {
    const uint32_t soff = j < QA ? (uint32_t)kt * a_kstep : (uint32_t)kt * 1024u;
    const uint32_t m0addr = lds0 + (uint32_t)(st * STAGE + 64 * (j * NW + wave)) * 16u;
    // M0 is reserved by the compiler, but nothing else in this kernel reads it
    // (no LDS DMA builtins, interpolation, GWS or message sends).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(m0addr), "v"(voff[j]), "s"(j < QA ? rA : rB), "s"(soff)
                 : "m0");
#pragma clang diagnostic pop
  };
  auto dma = [&](int st, int kt) {
#pragma unroll
    for (int j = 0; j < Q; ++j) dma1(st, kt, j);
  };
  // Every wave waits for its own DMAs of the next tile (all but the (NS - 2) Q
  // youngest, or all of them near the end of K) and for its LDS reads; the
  // barrier then makes the tile visible and frees the stage read before it.
  auto sync = [&](bool drain) {
    if (drain) __builtin_amdgcn_s_waitcnt(FD_VMCNT(0));
    else __builtin_amdgcn_s_waitcnt(FD_VMCNT((NS - 2) * Q));
    __builtin_amdgcn_s_waitcnt(FD_LGKMCNT0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lr = lane & 31, lk = lane >> 5, xr = (lr >> 2) & 3;
  // slot of fragment row (A: wm0 + lr, W: BM + wn0 + lr) at k-step ks: K-chunk 2 ks + lk
  const int ia0 = (wm0 + lr) * 4 + (lk ^ xr), ia1 = (wm0 + lr) * 4 + ((2 + lk) ^ xr);
  const int ib0 = (BM + wn0 + lr) * 4 + (lk ^ xr), ib1 = (BM + wn0 + lr) * 4 + ((2 + lk) ^ xr);
  V fa[2][FM], fb[2][FN];
  auto load_frags = [&](int slot, int st, int ks) {
    const uint4* sb = lds + st * STAGE;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint4 v = sb[(ks ? ia1 : ia0) + i * 128];
      fa[slot][i] = *reinterpret_cast<const V*>(&v);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint4 v = sb[(ks ? ib1 : ib0) + j * 128];
      fb[slot][j] = *reinterpret_cast<const V*>(&v);
    }
  };
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = kTransposed<EPI> ? Mfma<T>::run(fb[slot][j], fa[slot][i], acc[i][j])
                                     : Mfma<T>::run(fa[slot][i], fb[slot][j], acc[i][j]);
  };
  // the MFMAs of a k-step with DMA instructions j0 .. j0 + Q / 2 - 1 of a
  // stage refill between them, evenly spaced, in this order
  auto mfmas_dma = [&](int slot, int st, int kt, int j0) {
    if constexpr (C::IL) {
      constexpr int NM = FM * FN, ND = Q / 2, EVERY = NM / ND;
      static_assert(Q % 2 == 0 && NM % ND == 0, "DMA spacing");
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const int i = m / FN, j = m % FN;
        acc[i][j] = kTransposed<EPI> ? Mfma<T>::run(fb[slot][j], fa[slot][i], acc[i][j])
                                     : Mfma<T>::run(fa[slot][i], fb[slot][j], acc[i][j]);
        if (m % EVERY == EVERY - 1) {
          __builtin_amdgcn_sched_barrier(0);
          dma1(st, kt, j0 + m / EVERY);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Tile t sits in stage t % NS. The loop starts at the barrier (whose
  // explicit lgkmcnt(0) leaves no LDS read pending at the loop header), then
  // reads k-step 0 of tile t + 1, multiplies k-step 1 of tile t, reads k-step 1
  // of tile t + 1, refills the stage of tile t (read by everyone before the
  // barrier) with tile t + NS, and multiplies k-step 0 of tile t + 1.
  const int KT = K / BKD;
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < KT) dma(p, p);
  sync(KT < NS - 1);
  load_frags(0, 0, 0);
  load_frags(1, 0, 1);
  if (NS - 1 < KT) dma(NS - 1, NS - 1);
  mfmas(0);
  int sc = 0;  // stage of tile t
  int t = 0;
  if constexpr (C::IL) {
    for (; t < KT - NS; ++t) {
      const int sn = sc + 1 == NS ? 0 : sc + 1;
      sync(false);
      load_frags(0, sn, 0);
      mfmas_dma(1, sc, t + NS, 0);
      load_frags(1, sn, 1);
      mfmas_dma(0, sc, t + NS, Q / 2);
      sc = sn;
    }
  }
  for (; t < KT - 1; ++t) {
    const int sn = sc + 1 == NS ? 0 : sc + 1;
    sync(t + NS - 1 >= KT);
    load_frags(0, sn, 0);
    mfmas(1);
    load_frags(1, sn, 1);
    if (t + NS < KT) dma(sc, t + NS);
    mfmas(0);
    sc = sn;
  }
  mfmas(1);
  static_assert(EPI != EPI_QKV || NW * 32 * 68 * 4 <= NS * STAGE * 16, "QKV epilogue staging fits the stage buffers");
  if constexpr (kTransposed<EPI>)
    store_tile_t<EPI, T, FM, FN>(ep, acc, m0 + wm0, n0 + wn0, M, N, lr, lk, vec_store != 0);
  else if constexpr (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) {
    // one instantiation per pixel format, chosen once per tile (a format test
    // per store makes the epilogue loops too large to unroll, and the
    // accumulators would go to scratch memory)
    constexpr bool R = !(C::NW == 4 && C::MIN_BLOCKS == 1);
    float* ws = reinterpret_cast<float*>(lds);
    if (ep.out_fmt == 0) store_tile<EPI, T, FM, FN, R, 0>(ep, acc, m0 + wm0, n0 + wn0, M, N, lr, lk, ws);
    else if (ep.out_fmt == 1) store_tile<EPI, T, FM, FN, R, 1>(ep, acc, m0 + wm0, n0 + wn0, M, N, lr, lk, ws);
    else store_tile<EPI, T, FM, FN, R, 2>(ep, acc, m0 + wm0, n0 + wn0, M, N, lr, lk, ws);
  } else {
    store_tile<EPI, T, FM, FN, !(C::NW == 4 && C::MIN_BLOCKS == 1)>(ep, acc, m0 + wm0, n0 + wn0, M, N, lr, lk,
                                                                   reinterpret_cast<float*>(lds));
  }
}

// ---------------------------------------------------------------------------
// E4M3 GEMM (the FP8 MLP of the "-Opt" decoder, Sec. 4.6) on the gfx950
// 32x32x64 FP8 MFMA. The memory path is that of the 16-bit kernel: a 64-byte
// stage row now holds 64 K-values, one MFMA k-step, whose fragment (32
// consecutive K-values of one row per lane, K-half lk) is two 16-byte chunks
// of the swizzled stage row. Fragments are double-buffered across tiles: tile
// t + 1's are read while tile t's MFMAs run (8-wave tiles single-buffer the W
// fragments). The accumulator of (m, n) is multiplied by col_scale[n] and then
// row_scale[m * row_scale_stride] (per-channel weight scales; per-token or, with
// stride 0, static per-tensor activation scales), in the epilogue's layout.
// The matrix instruction sums each aligned group of 8 products after cutting
// them 13 bits below the group's largest exponent sum (measured), so results
// differ from an exact fp32 sum by up to 2^-10 of that magnitude per group.
// ---------------------------------------------------------------------------
typedef int i32x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma_e4m3(i32x8 a, i32x8 b, f32x16 c) {
  // format fields 0 / 0: both operands OCP E4M3; no block scales
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

template <class C, int EPI>
__global__ __launch_bounds__(C::NT, C::MIN_BLOCKS) void gemm_fp8_kernel(
    const uint8_t* __restrict__ A, const uint8_t* __restrict__ W, int M, int N, int K, int lda,
    EpiParams ep, int tiles_m, int tiles_n, int a_packed) {
  constexpr int BM = C::BM, BN = C::BN, FM = C::FM, FN = C::FN, NS = C::NS, NW = C::NW;
  constexpr int QA = C::QA, Q = C::QA + C::QB, STAGE = C::STAGE;
  constexpr bool TR = kTransposed<EPI>;
  __shared__ uint4 lds[NS * STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  tile_of(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm0 = (wave / C::WAVES_N) * C::WM, wn0 = (wave % C::WAVES_N) * C::WN;

  const int KB = K / 64;  // K tiles (64-byte stage rows)
  // A row-major (lda bytes), or packed like W (lda = K, whole 16-row blocks)
  const bool apk = a_packed != 0;
  const int a_rows = apk ? (min(BM, M - m0) + 15) / 16 * 16 : min(BM, M - m0);
  const __amdgpu_buffer_rsrc_t rA = make_rsrc(A + (int64_t)m0 * lda, (uint32_t)a_rows * (uint32_t)lda);
  const int nrows_w = min(BN, (N + 15) / 16 * 16 - n0);
  const __amdgpu_buffer_rsrc_t rB =
      make_rsrc(W + (int64_t)(n0 / 16) * KB * 1024, (uint32_t)(nrows_w / 16) * KB * 1024u);
  const int lrow = lane >> 2, lchunk = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t voff[Q];
#pragma unroll
  for (int j = 0; j < Q; ++j) {
    const int q = j * NW + wave;
    voff[j] = j >= QA ? (uint32_t)(q - BM / 16) * KB * 1024u + (uint32_t)(lrow * 64 + lchunk * 16)
              : apk   ? (uint32_t)q * KB * 1024u + (uint32_t)(lrow * 64 + lchunk * 16)
                      : (uint32_t)((16 * q + lrow) * lda + lchunk * 16);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)lds;
  const uint32_t a_kstep = apk ? 1024u : 64u;  // bytes per K tile
  auto dma = [&](int st, int kt) {
    const uint32_t soffA = (uint32_t)kt * a_kstep, soffB = (uint32_t)kt * 1024u;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const uint32_t m0addr = lds0 + (uint32_t)(st * STAGE + 64 * (j * NW + wave)) * 16u;
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                   :
                   : "s"(m0addr), "v"(voff[j]), "s"(j < QA ? rA : rB), "s"(j < QA ? soffA : soffB)
                   : "m0");
#pragma clang diagnostic pop
    }
  };
  auto sync = [&](bool drain) {
    if (drain) __builtin_amdgcn_s_waitcnt(FD_VMCNT(0));
    else __builtin_amdgcn_s_waitcnt(FD_VMCNT((NS - 2) * Q));
    __builtin_amdgcn_s_waitcnt(FD_LGKMCNT0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lr = lane & 31, lk = lane >> 5, xr = (lr >> 2) & 3;
  // the two chunks of fragment row (A: wm0 + lr, W: BM + wn0 + lr): K-chunks 2 lk, 2 lk + 1
  const int ia0 = (wm0 + lr) * 4 + ((2 * lk) ^ xr), ia1 = (wm0 + lr) * 4 + ((2 * lk + 1) ^ xr);
  const int ib0 = (BM + wn0 + lr) * 4 + ((2 * lk) ^ xr), ib1 = (BM + wn0 + lr) * 4 + ((2 * lk + 1) ^ xr);
  // 8-wave tiles leave 256 registers per lane: double-buffering both operands'
  // fragments (96) beside 128 accumulators would spill, so the W fragments are
  // single-buffered there and each W block is re-read for the next tile as
  // soon as its last MFMA has issued.
  constexpr bool FB1 = NW == 8;
  i32x8 fa[2][FM], fb[FB1 ? 1 : 2][FN];
  auto load_fa1 = [&](int slot, int st, int i) {
    const uint4* sb = lds + st * STAGE;
    const uint4 v0 = sb[ia0 + i * 128], v1 = sb[ia1 + i * 128];
    fa[slot][i] = i32x8{(int)v0.x, (int)v0.y, (int)v0.z, (int)v0.w, (int)v1.x, (int)v1.y, (int)v1.z, (int)v1.w};
  };
  auto load_fa = [&](int slot, int st) {
#pragma unroll
    for (int i = 0; i < FM; ++i) load_fa1(slot, st, i);
  };
  auto load_fb = [&](int slot, int st, int j) {
    const uint4* sb = lds + st * STAGE;
    const uint4 v0 = sb[ib0 + j * 128], v1 = sb[ib1 + j * 128];
    fb[slot][j] = i32x8{(int)v0.x, (int)v0.y, (int)v0.z, (int)v0.w, (int)v1.x, (int)v1.y, (int)v1.z, (int)v1.w};
  };
  // MFMAs of the tile in register slot `slot`; with FB1 and reload, W block j
  // of the tile in stage next_st replaces block j once its MFMAs are issued
  auto mfmas = [&](int slot, int next_st, bool reload) {
    const int bs = FB1 ? 0 : slot;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
        acc[i][j] = TR ? mfma_e4m3(fb[bs][j], fa[slot][i], acc[i][j]) : mfma_e4m3(fa[slot][i], fb[bs][j], acc[i][j]);
      if (FB1 && reload) load_fb(0, next_st, j);
    }
  };

  // Tile t sits in stage t % NS. Iteration t: the barrier publishes tile t + 1
  // (and frees the stage read in iteration t - 1), its fragments are read
  // into register slot (t + 1) & 1, the stage of tile t is refilled with tile
  // t + NS, and tile t's MFMAs run from slot t & 1. The loop runs two
  // iterations per trip so that both slots are compile-time indices (a
  // run-time index would put the fragment arrays in scratch memory).
  const int KT = KB;
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < KT) dma(p, p);
  sync(KT < NS - 1);
  load_fa(0, 0);
#pragma unroll
  for (int j = 0; j < FN; ++j) load_fb(0, 0, j);
  if (NS - 1 < KT) dma(NS - 1, NS - 1);
  int sc = 0;
  auto step = [&](int t, int load_slot, int mfma_slot) {
    const int sn = sc + 1 == NS ? 0 : sc + 1;
    sync(t + NS - 1 >= KT);
    load_fa(load_slot, sn);
    if (!FB1) {
#pragma unroll
      for (int j = 0; j < FN; ++j) load_fb(load_slot, sn, j);
    }
    if (t + NS < KT) dma(sc, t + NS);
    mfmas(mfma_slot, sn, true);
    sc = sn;
  };
  int t = 0;
  for (; t + 2 <= KT - 1; t += 2) {
    step(t, 1, 0);
    step(t + 1, 0, 1);
  }
  if (t < KT - 1) {
    step(t, 1, 0);
    ++t;
  }
  // t == KT - 1: the last tile's fragments move to slot 0 (a branch around the
  // MFMAs instead would merge two copies of the accumulators and spill)
  if (t & 1) {
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[0][i] = fa[1][i];
    if (!FB1) {
#pragma unroll
      for (int j = 0; j < FN; ++j) fb[0][j] = fb[FB1 ? 0 : 1][j];
    }
  }
  mfmas(0, 0, false);

  // dequantisation by column then row scale: inside the transposed SwiGLU store,
  // per element; here, in the accumulator layout, for the residual add
  const int r0 = m0 + wm0, c0 = n0 + wn0;
  if constexpr (TR) {  // lane: row r0 + 32 i + lr; columns c0 + 32 j + 8 q + 4 lk + e
    store_tile_t<EPI, _Float16, FM, FN, true>(ep, acc, r0, c0, M, N, lr, lk, true);
  } else {  // lane: column c0 + 32 j + lr; rows r0 + 32 i + 8 (r / 4) + 4 lk + r % 4
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const float cs = ep.col_scale[min(c0 + j * 32 + lr, N - 1)];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] *= cs;
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float rs = ep.row_scale[min(r0 + i * 32 + 8 * (r >> 2) + 4 * lk + (r & 3), M - 1) * ep.row_scale_stride];
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j][r] *= rs;
      }
    store_tile<EPI, _Float16, FM, FN, !(C::NW == 4 && C::MIN_BLOCKS == 1)>(ep, acc, r0, c0, M, N, lr, lk,
                                                                          reinterpret_cast<float*>(lds));
  }
}

template <typename T, class C, int EPI>
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + C::BM - 1) / C::BM, tn = (g.N + C::BN - 1) / C::BN;
  // four consecutive output columns land contiguously and 16-byte aligned
  // (fp32) / 8-byte aligned (16-bit) in the destination
  bool vec = g.N % 4 == 0 && g.ep.ld_out % 4 == 0;
  if (EPI == EPI_PIXEL || EPI == EPI_LINEAR_PIXEL) vec = vec && g.ep.s % 4 == 0;
  if (EPI == EPI_TUP) vec = vec && g.ep.dim % 4 == 0;
  vec = vec && ((uintptr_t)g.ep.out_f % 16 == 0) && ((uintptr_t)g.ep.out_a % 8 == 0);
  hipLaunchKernelGGL((gemm_mfma_kernel<T, C, EPI>), dim3(tm * tn), dim3(C::NT), 0, s,
                     (const T*)g.A, (const T*)g.W, g.M, g.N, g.K, g.lda, g.ldw, g.ep, tm, tn, vec ? 1 : 0,
                     g.a_packed);
  return hipGetLastError();
}

// Tile choice, measured on the 480p / 720p decoder shapes (random fp16 data).
// - 256 x 256 tiles (8 waves of 128 x 64) read the fewest LDS and L2 bytes
//   per flop and win wherever there are enough of them to fill the 256 CUs,
//   except for residual-add epilogues behind a short K loop.
// - When 192 x 128 tiles come to one nearly full wave (200-256 workgroups,
//   the backbone's M = 3600 x N = 1536 projections), one workgroup per CU with
//   6 stages in flight wins.
// - When even 128 x 128 tiles leave CUs idle (480p backbone), each CU runs a
//   single workgroup, so it gets 6 stages in flight.
// - Otherwise 128 x 128 tiles with 3 stages, several workgroups per CU, so one
//   workgroup's epilogue and barriers overlap another's MFMAs.
using TileL = TileCfg<256, 256, 2, 4, 4, true>;   // 8 waves of 128 x 64, 128 KB LDS
using TileW = TileCfg<256, 192, 2, 2, 5>;         // 4 waves of 128 x 96, 140 KB
using TileM = TileCfg<192, 128, 2, 2, 6>;         // 4 waves of 96 x 64, 120 KB
using TileM4 = TileCfg<192, 128, 2, 2, 4>;        // the same, 80 KB: two per CU
using TileS1 = TileCfg<128, 128, 2, 2, 6, true>;  // 4 waves of 64 x 64, 96 KB
using TileS = TileCfg<128, 128, 2, 2, 3, true>;   // 4 waves of 64 x 64, 48 KB

template <typename T, int EPI>
hipError_t dispatch_tiles(const GemmArgs& g, hipStream_t s) {
  auto tiles = [&](int bm, int bn) { return ((g.M + bm - 1) / bm) * ((g.N + bn - 1) / bn); };
  const bool short_rmw = EPI == EPI_RESID_ADD && g.K <= 2048;
  if (tiles(256, 256) >= 160 && !short_rmw) {
    // a SwiGLU projection of under two rounds of 256 x 256 tiles (the 480p
    // backbone: 336 tiles, 1.3 rounds) runs faster as 128 x 128 tiles, several
    // per CU (measured 1.8% per 480p chunk); so do the QKV and temporal-up
    // projections of the 720p refinement input (456 and 360 tiles)
    if (EPI == EPI_SWIGLU && tiles(256, 256) < 512) return launch_gemm<T, TileS, EPI>(g, s);
    if ((EPI == EPI_QKV || EPI == EPI_TUP) && tiles(256, 256) < 512) return launch_gemm<T, TileS, EPI>(g, s);
    // 256 x 192 tiles where their rounds of 256 CUs, weighted by tile area,
    // are fewer than those of 256 x 256 tiles (for instance 342 -> 456 tiles,
    // 2 -> 1.5 round-equivalents, for 14400 x 1536 outputs). Their 96-column
    // wave blocks suit every epilogue but the paired SwiGLU and the QKV post
    // step (one 64-column head vector per wave); the GELU epilogue's erf needs
    // more registers than a 4-wave 256 x 192 tile leaves.
    if constexpr (EPI != EPI_SWIGLU && EPI != EPI_QKV && EPI != EPI_STORE_GELU) {
      const int rounds_l = (tiles(256, 256) + 255) / 256, rounds_w = (tiles(256, 192) + 255) / 256;
      if (4 * rounds_w * 3 < 4 * rounds_l * 4) return launch_gemm<T, TileW, EPI>(g, s);
    }
    return launch_gemm<T, TileL, EPI>(g, s);
  }
  const int tm = tiles(192, 128);
  if constexpr (EPI == EPI_RESID_ADD) {
    // residual adds: 192 x 128 tiles with 4 stages (two workgroups per CU)
    // behind a long K loop in one round, and wherever 192 x 128 tiles make one
    // round of two per CU (257-512 tiles, the 480p refinement O projection)
    if ((tm >= 200 && tm <= 256 && g.K > 2048) || (tm > 256 && tm <= 512))
      return launch_gemm<T, TileM4, EPI>(g, s);
  }
  if (tm >= 200 && tm <= 256) return launch_gemm<T, TileM, EPI>(g, s);
  if (tiles(128, 128) <= 256) return launch_gemm<T, TileS1, EPI>(g, s);
  return launch_gemm<T, TileS, EPI>(g, s);
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
    case EPI_QKV: return dispatch_tiles<T, EPI_QKV>(g, s);
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

template <class C, int EPI>
hipError_t launch_fp8(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + C::BM - 1) / C::BM, tn = (g.N + C::BN - 1) / C::BN;
  hipLaunchKernelGGL((gemm_fp8_kernel<C, EPI>), dim3(tm * tn), dim3(C::NT), 0, s, (const uint8_t*)g.A,
                     (const uint8_t*)g.W, g.M, g.N, g.K, g.lda, g.ep, tm, tn, g.a_packed);
  return hipGetLastError();
}

template <int EPI>
hipError_t dispatch_fp8(const GemmArgs& g, hipStream_t s) {
  auto tiles = [&](int bm, int bn) { return ((g.M + bm - 1) / bm) * ((g.N + bn - 1) / bn); };
  // (256 x 256 tiles would spill the residual epilogue's registers)
  if constexpr (EPI != EPI_RESID_ADD)
    if (tiles(256, 256) >= 160) return launch_fp8<TileL, EPI>(g, s);
  const int tm = tiles(192, 128);
  if (tm >= 200) return launch_fp8<TileM, EPI>(g, s);
  return launch_fp8<TileS, EPI>(g, s);
}

}  // namespace

hipError_t gemm_fp8(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  // packed A codes need lda = K; only the E4M3 SwiGLU codes can be written packed
  if ((g.a_packed && g.lda != g.K) || (g.ep.out_packed && (g.epi != EPI_SWIGLU_E4M3 || g.ep.ld_out % 64)))
    return hipErrorInvalidValue;
  if (g.K <= 0 || g.K % 64 || g.lda % 16 || !g.ep.row_scale || !g.ep.col_scale) return hipErrorInvalidValue;
  if (g.epi == EPI_SWIGLU) {
    if (g.N % 64 || g.ep.ld_out % 4 || (uintptr_t)g.ep.out_a % 8) return hipErrorInvalidValue;
    return dispatch_fp8<EPI_SWIGLU>(g, s);
  }
  if (g.epi == EPI_SWIGLU_E4M3) {
    if (g.N % 64 || g.ep.ld_out % 4 || (uintptr_t)g.ep.out_a % 4 || !g.ep.out_scale) return hipErrorInvalidValue;
    return dispatch_fp8<EPI_SWIGLU_E4M3>(g, s);
  }
  if (g.epi == EPI_RESID_ADD) return dispatch_fp8<EPI_RESID_ADD>(g, s);
  return hipErrorInvalidValue;
}

hipError_t gemm_mfma(Act16 t, const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.K <= 0 || g.K % BKD || g.lda % 8 || g.ldw != g.K) return hipErrorInvalidValue;
  if (g.a_packed && g.lda != g.K) return hipErrorInvalidValue;
  if (g.ep.out_packed && (g.ep.ld_out % 32 || !(g.epi == EPI_SWIGLU || g.epi == EPI_STORE_ACT ||
                                                g.epi == EPI_STORE_SILU || g.epi == EPI_STORE_GELU)))
    return hipErrorInvalidValue;
  if ((g.epi == EPI_SWIGLU || g.epi == EPI_QKV) && g.N % 64) return hipErrorInvalidValue;
  if (g.epi == EPI_QKV && g.ep.qkv.Dh != 64) return hipErrorInvalidValue;
  return t == Act16::F16 ? dispatch_epi<_Float16>(g, s) : dispatch_epi<__hip_bfloat16>(g, s);
}

hipError_t gemm_f32(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.a_packed || g.ep.out_packed) return hipErrorInvalidValue;  // row-major fp32 operands
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
