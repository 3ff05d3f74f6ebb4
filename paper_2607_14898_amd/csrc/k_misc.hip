// Bandwidth-bound passes of the decoder forward:
//  * norm_rows       pre-sublayer RMSNorm / LayerNorm of the fp32 residual
//                    stream (Sec. 3.2 "Base Architecture") into the operand
//                    format and packed block layout of the next projection;
//  * qkv_post        KV-norm and 3D-RoPE (Sec. 3.2), then the rolling-cache
//                    append of Sec. 3.3 / Algorithm 1 as a write into ring slot
//                    (unit mod S);
//  * unshuffle_latent PixelUnshuffle(p) + raster flatten of latent frames
//                    (Sec. 4.3 and Eq. projection);
//  * swiglu_f32      SwiGLU gate of the fp32 path;
//  * quant_rows_e4m3 per-row E4M3 codes and scales of the FP8 MLP (Sec. 4.6).
#include "fd_kernels.h"

#include <hip/hip_bf16.h>

namespace fd {
namespace {

__device__ __forceinline__ void store_kind(void* out, int64_t i, float v, int kind) {
  if (kind == 0) ((_Float16*)out)[i] = (_Float16)v;
  else if (kind == 1) ((__hip_bfloat16*)out)[i] = __float2bfloat16(v);
  else ((float*)out)[i] = v;
}

// Element (row, k) of a 16-bit [rows, K] activation in the packed operand
// layout of the MFMA GEMM (blocks of 16 rows x 32 columns, block-row major).
__device__ __forceinline__ int64_t pk16(int64_t row, int k, int K) {
  return ((row >> 4) * (K >> 5) + (k >> 5)) * 512 + (row & 15) * 32 + (k & 31);
}
// Byte (row, k) of E4M3 codes [rows, K] in the packed operand layout of the
// FP8 GEMM (blocks of 16 rows x 64 bytes).
__device__ __forceinline__ int64_t pk8(int64_t row, int k, int K) {
  return ((row >> 4) * (K >> 6) + (k >> 6)) * 1024 + (row & 15) * 64 + (k & 63);
}

// Four consecutive values as one 8-byte (16-bit kinds) or 16-byte (fp32) store.
__device__ __forceinline__ void store4(void* out, int64_t i, float4 y, int kind) {
  if (kind == 0) {
    typedef _Float16 h4 __attribute__((ext_vector_type(4)));
    const h4 h = {(_Float16)y.x, (_Float16)y.y, (_Float16)y.z, (_Float16)y.w};
    *reinterpret_cast<h4*>((_Float16*)out + i) = h;
  } else if (kind == 1) {
    __hip_bfloat16 h[4] = {__float2bfloat16(y.x), __float2bfloat16(y.y), __float2bfloat16(y.z),
                           __float2bfloat16(y.w)};
    *reinterpret_cast<uint2*>((__hip_bfloat16*)out + i) = *reinterpret_cast<uint2*>(h);
  } else {
    *reinterpret_cast<float4*>((float*)out + i) = y;
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// E4M3 quantisation of a row whose amplitude (max |v|) is m: inv = 448 / m,
// codes of fp32(v * inv) by the gfx950 conversion (round to nearest even),
// after clamping to +-448 so that the code saturates; scale m / 448. A zero
// row gets scale 1 (and codes 0).
struct E4m3Row {
  float inv, scale;
  __device__ __forceinline__ explicit E4m3Row(float m) {
    const float mm = m > 0.f ? m : 448.f;
    inv = 448.f / mm;
    scale = mm / 448.f;
  }
  // a static (calibrated) scale: {scale, inverse scale}
  __device__ __forceinline__ explicit E4m3Row(const float* sc) : inv(sc[1]), scale(sc[0]) {}
  // four values -> four codes, byte e = value e
  __device__ __forceinline__ uint32_t pack4(float a, float b, float c, float d) const {
    auto cl = [&](float v) { return fminf(448.f, fmaxf(-448.f, v * inv)); };
    int w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(a), cl(b), 0, false);
    w = __builtin_amdgcn_cvt_pk_fp8_f32(cl(c), cl(d), w, true);
    return (uint32_t)w;
  }
};

// One wave per row; rows of D floats (D % 4 == 0).
template <int KIND>
__global__ __launch_bounds__(256) void norm_kernel(const float* __restrict__ x, int M, int D,
                                                   const float* __restrict__ g,
                                                   const float* __restrict__ bta, float eps,
                                                   void* out, int out_kind, float* row_scale,
                                                   const float* __restrict__ static_sc,
                                                   unsigned* __restrict__ amax_out, int packed) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const float4* xr = reinterpret_cast<const float4*>(x + (int64_t)row * D);
  const int nv = D / 4;
  constexpr int MAXV = 8;  // up to D = 2048 held in registers
  float4 v[MAXV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      v[i] = xr[c];
      s += KIND == 0 ? v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w
                     : v[i].x + v[i].y + v[i].z + v[i].w;
    }
  }
  s = wave_sum(s);
  float mu = 0.f, rs;
  if (KIND == 0) {
    rs = rsqrtf(s / D + eps);
  } else {
    mu = s / D;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < MAXV; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        const float a0 = v[i].x - mu, a1 = v[i].y - mu, a2 = v[i].z - mu, a3 = v[i].w - mu;
        q += a0 * a0 + a1 * a1 + a2 * a2 + a3 * a3;
      }
    }
    q = wave_sum(q);
    rs = rsqrtf(q / D + eps);
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      const float4 gv = reinterpret_cast<const float4*>(g)[c];
      float4 y = make_float4((v[i].x - mu) * rs * gv.x, (v[i].y - mu) * rs * gv.y,
                             (v[i].z - mu) * rs * gv.z, (v[i].w - mu) * rs * gv.w);
      if (KIND == 1) {
        const float4 bv = reinterpret_cast<const float4*>(bta)[c];
        y.x += bv.x; y.y += bv.y; y.z += bv.z; y.w += bv.w;
      }
      if (out_kind == 3) {  // E4M3: keep the row for its amplitude
        v[i] = y;
        amax = fmaxf(fmaxf(amax, fmaxf(fabsf(y.x), fabsf(y.y))), fmaxf(fabsf(y.z), fabsf(y.w)));
      } else {
        store4(out, packed ? pk16(row, 4 * c, D) : (int64_t)row * D + 4 * c, y, out_kind);
      }
    }
  }
  if (out_kind == 3) {
    const float m = wave_max(amax);
    if (amax_out && lane == 0) atomicMax(amax_out, __float_as_uint(m));  // non-negative: ordered as bits
    const E4m3Row q = static_sc ? E4m3Row(static_sc) : E4m3Row(m);
#pragma unroll
    for (int i = 0; i < MAXV; ++i) {
      const int c = lane + 64 * i;
      if (c < nv)
        *reinterpret_cast<uint32_t*>((uint8_t*)out + (packed ? pk8(row, 4 * c, D) : (int64_t)row * D + 4 * c)) =
            q.pack4(v[i].x, v[i].y, v[i].z, v[i].w);
    }
    if (!static_sc && lane == 0) row_scale[row] = q.scale;
  }
}

// Per-row E4M3 codes of in [M, K] (fp16 or fp32, K % 8 == 0): one wave per row,
// a first pass for the amplitude, a second (from cache) for the codes.
template <typename TIN>
__global__ __launch_bounds__(256) void quant_rows_kernel(const TIN* __restrict__ in, int64_t M, int K,
                                                         uint8_t* __restrict__ codes,
                                                         float* __restrict__ scale,
                                                         unsigned* __restrict__ amax_out, int packed) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const TIN* r = in + row * K;
  float amax = 0.f;
  for (int c = 8 * lane; c < K; c += 512) {
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)r[c + e]));
  }
  const float m = wave_max(amax);
  if (amax_out && lane == 0) atomicMax(amax_out, __float_as_uint(m));
  const E4m3Row q(m);
  for (int c = 8 * lane; c < K; c += 512) {
    float f[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (float)r[c + e];
    uint2 w;
    w.x = q.pack4(f[0], f[1], f[2], f[3]);
    w.y = q.pack4(f[4], f[5], f[6], f[7]);
    *reinterpret_cast<uint2*>(codes + (packed ? pk8(row, c, K) : row * K + c)) = w;
  }
  if (lane == 0) scale[row] = q.scale;
}

// cos / sin of the RoPE angle of channel pair `pair` for the row (frame-or-
// sub-frame fs of the call, token tok): temporal pairs read the per-call table
// (fs), spatial pairs the table indexed by the token's row h or column w.
__device__ __forceinline__ float2 rope_cs(const QkvPostArgs& a, int pair, int fs, int tok) {
  const int axis = a.rope_axis[pair];
  const int np = a.Dh / 2;
  if (axis == 0) return a.rope_t[fs * np + pair];
  const int p = axis == 1 ? tok / a.grid_w : tok % a.grid_w;
  return a.rope_hw[p * np + pair];
}

// Queries and keys: one thread per 4 consecutive channels of a (row, head slot),
// slots 0..N-1 query heads and N..N+G-1 key groups, so a head vector is 16
// consecutive lanes (D_h = 64; D_h / 4 lanes in general) and consecutive
// threads read consecutive 16-byte chunks of the raw projection.
__global__ __launch_bounds__(256) void qk_post_kernel(QkvPostArgs a, int rows) {
  const int Dh = a.Dh, qpv = Dh / 4;  // threads per head vector
  const int slots = a.N + a.G;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_row = (int64_t)slots * qpv;
  const bool valid = t < (int64_t)rows * per_row;
  const int row = valid ? (int)(t / per_row) : 0;
  const int rem = (int)(t - (int64_t)row * per_row);
  const int hs = rem / qpv, qd = rem - hs * qpv;
  const int width = a.N * Dh + 2 * a.G * Dh;
  float4 x = valid ? *reinterpret_cast<const float4*>(a.raw + (int64_t)row * width + hs * Dh + 4 * qd)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
  const bool is_q = hs < a.N;
  if (!is_q && a.knorm_g) {  // KV-norm: RMSNorm over D_h with a learned gain
    float ss = x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    for (int o = qpv / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    const float r = rsqrtf(ss / Dh + a.eps);
    const float4 gv = reinterpret_cast<const float4*>(a.knorm_g)[qd];
    x = make_float4(x.x * r * gv.x, x.y * r * gv.y, x.z * r * gv.z, x.w * r * gv.w);
  }
  if (!valid) return;
  const int b = row / a.rows_per_batch, rb = row - b * a.rows_per_batch;
  if (a.rope) {
    const int fs = rb / a.L, tok = rb - fs * a.L;
    const float2 c0 = rope_cs(a, 2 * qd, fs, tok), c1 = rope_cs(a, 2 * qd + 1, fs, tok);
    x = make_float4(x.x * c0.x - x.y * c0.y, x.x * c0.y + x.y * c0.x,
                    x.z * c1.x - x.w * c1.y, x.z * c1.y + x.w * c1.x);
  }
  if (is_q) {
    store4(a.q, (int64_t)row * a.N * Dh + hs * Dh + 4 * qd, x, a.out_kind);
    return;
  }
  const int lu = rb / a.U, pos = rb - lu * a.U;
  const int slot = (int)((a.u0 + lu) % a.S);
  const int64_t base = (((int64_t)(b * a.G + hs - a.N) * a.S + slot) * a.U_pad + pos) * Dh;
  store4(a.k_ring, base + 4 * qd, x, a.out_kind);
}

// Values: one workgroup per 64 consecutive positions of one causal unit of one
// stream and one KV group; KV-norm, then written transposed ([D_h][U_pad] per
// slot) through LDS as rows of 64 positions.
constexpr int VP_ROWS = 64;
__global__ __launch_bounds__(256) void v_post_kernel(QkvPostArgs a, int blocks_per_unit) {
  __shared__ float vt[64][VP_ROWS + 1];  // [dim][position]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Dh = a.Dh;
  const bool act = lane < Dh;
  const int g = blockIdx.y;
  const int blk = blockIdx.x % blocks_per_unit, bu = blockIdx.x / blocks_per_unit;
  const int units_per_batch = a.rows_per_batch / a.U;
  const int lu = bu % units_per_batch, b = bu / units_per_batch;
  const int pos0 = blk * VP_ROWS;
  const int npos = min(VP_ROWS, a.U - pos0);
  const int width = a.N * Dh + 2 * a.G * Dh;
  constexpr int RPW = VP_ROWS / 4;
  const int64_t row0 = (int64_t)b * a.rows_per_batch + (int64_t)lu * a.U + pos0 + wave * RPW;
  float x[RPW];
#pragma unroll
  for (int i = 0; i < RPW; ++i)
    x[i] = (act && wave * RPW + i < npos) ? a.raw[(row0 + i) * width + (a.N + a.G + g) * Dh + lane] : 0.f;
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
    float y = x[i];
    if (a.vnorm_g) {
      const float ms = wave_sum(y * y) / Dh;
      y = act ? y * rsqrtf(ms + a.eps) * a.vnorm_g[lane] : 0.f;
    }
    vt[lane][wave * RPW + i] = y;
  }
  __syncthreads();
  const int slot = (int)((a.u0 + lu) % a.S);
  const int64_t vbase = ((int64_t)(b * a.G + g) * a.S + slot) * Dh * a.U_pad + pos0;
  for (int d = wave; d < Dh; d += 4)
    if (lane < npos) store_kind(a.vt_ring, vbase + (int64_t)d * a.U_pad + lane, vt[d][lane], a.out_kind);
}

// Temporal RoPE cos / sin of the call's (sub-)frames: entry (fs, pair) for
// position tau0 + fs; the angle is reduced modulo 2 pi in double precision so
// that long streams keep full accuracy.
__global__ void rope_time_kernel(int64_t tau0, int n_fs, int np, const int* axis,
                                 const double* freq, float2* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_fs * np) return;
  const int fs = i / np, pair = i - fs * np;
  float2 r = make_float2(1.f, 0.f);
  if (axis[pair] == 0) {
    const double ph = (double)(tau0 + fs) * freq[pair];
    const double red = ph - 6.283185307179586 * floor(ph * 0.15915494309189535);
    float sn, cs;
    sincosf((float)red, &sn, &cs);
    r = make_float2(cs, sn);
  }
  out[i] = r;
}

// u[(b F + f) L + h W_t + w, c p^2 + i p + j] = z[b, c, f, p h + i, p w + j]; zero padding to K_pad.
__global__ __launch_bounds__(256) void unshuffle_kernel(const void* z, int z_kind, int B, int C,
                                                        int F, int H, int W, int p, int K_pad,
                                                        void* u, int out_kind, int packed) {
  const int Ht = H / p, Wt = W / p, L = Ht * Wt;
  const int64_t total = (int64_t)B * F * L * K_pad;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int k = (int)(e % K_pad);
    const int64_t row = e / K_pad;
    float v = 0.f;
    if (k < C * p * p) {
      const int n = (int)(row % L);
      const int64_t bf = row / L;
      const int f = (int)(bf % F), b = (int)(bf / F);
      const int c = k / (p * p), rem = k % (p * p), i = rem / p, j = rem % p;
      const int h = n / Wt, w = n % Wt;
      const int64_t zi = ((((int64_t)b * C + c) * F + f) * H + (p * h + i)) * W + p * w + j;
      if (z_kind == 0) v = ((const float*)z)[zi];
      else if (z_kind == 1) v = __bfloat162float(((const __hip_bfloat16*)z)[zi]);
      else v = (float)((const _Float16*)z)[zi];
    }
    store_kind(u, packed ? pk16(row, k, K_pad) : e, v, out_kind);
  }
}

__global__ __launch_bounds__(256) void swiglu_f32_kernel(const float* raw, int M, int H, float* h) {
  const int64_t total = (int64_t)M * H;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = e / H;
    const int j = (int)(e % H);
    const float gt = raw[m * 2 * H + j], up = raw[m * 2 * H + H + j];
    h[e] = gt / (1.f + expf(-gt)) * up;
  }
}

__global__ __launch_bounds__(256) void convert_kernel(const float* src, void* dst, int64_t n,
                                                      int out_kind) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    store_kind(dst, e, src[e], out_kind);
}

int grid_for(int64_t total) {
  int64_t b = (total + 255) / 256;
  return (int)(b < 65536 ? (b > 0 ? b : 1) : 65536);
}

}  // namespace

hipError_t norm_rows(const float* x, int M, int D, const float* g, const float* b, int kind,
                     float eps, void* out, int out_kind, hipStream_t s, float* row_scale,
                     const float* static_sc, unsigned* amax_out, bool packed) {
  if (M <= 0) return hipSuccess;
  if (D % 4 || D > 2048 || (out_kind == 3 && !row_scale && !static_sc)) return hipErrorInvalidValue;
  if (packed && (out_kind == 3 ? D % 64 : (D % 32 || (out_kind != 0 && out_kind != 1))))
    return hipErrorInvalidValue;
  const int grid = (M + 3) / 4;
  if (kind == 0)
    hipLaunchKernelGGL(norm_kernel<0>, dim3(grid), dim3(256), 0, s, x, M, D, g, b, eps, out, out_kind,
                       row_scale, static_sc, amax_out, packed ? 1 : 0);
  else
    hipLaunchKernelGGL(norm_kernel<1>, dim3(grid), dim3(256), 0, s, x, M, D, g, b, eps, out, out_kind,
                       row_scale, static_sc, amax_out, packed ? 1 : 0);
  return hipGetLastError();
}

hipError_t quant_rows_e4m3(const void* in, int in_kind, int64_t M, int K, uint8_t* codes,
                           float* scale, hipStream_t s, unsigned* amax_out, bool packed) {
  if (M <= 0) return hipSuccess;
  if (K <= 0 || K % 8 || (in_kind != 0 && in_kind != 2) || (packed && K % 64)) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((M + 3) / 4);
  if (in_kind == 0)
    hipLaunchKernelGGL(quant_rows_kernel<_Float16>, dim3(grid), dim3(256), 0, s, (const _Float16*)in, M,
                       K, codes, scale, amax_out, packed ? 1 : 0);
  else
    hipLaunchKernelGGL(quant_rows_kernel<float>, dim3(grid), dim3(256), 0, s, (const float*)in, M, K,
                       codes, scale, amax_out, packed ? 1 : 0);
  return hipGetLastError();
}

hipError_t rope_time(const QkvPostArgs& a, hipStream_t s) {
  if (!a.rope || a.rows_per_batch <= 0) return hipSuccess;
  const int n_fs = a.rows_per_batch / a.L, np = a.Dh / 2;
  hipLaunchKernelGGL(rope_time_kernel, dim3((n_fs * np + 255) / 256), dim3(256), 0, s, a.tau0,
                     n_fs, np, a.rope_axis, a.rope_freq, a.rope_t);
  return hipGetLastError();
}

hipError_t qkv_post(const QkvPostArgs& a, hipStream_t s) {
  const int rows = a.B * a.rows_per_batch;
  if (rows <= 0) return hipSuccess;
  if (a.Dh > 64 || a.Dh % 8 || a.rows_per_batch % a.U) return hipErrorInvalidValue;
  const int64_t threads = (int64_t)rows * (a.N + a.G) * (a.Dh / 4);
  hipLaunchKernelGGL(qk_post_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, a, rows);
  const int blocks_per_unit = (a.U + VP_ROWS - 1) / VP_ROWS;
  const int units = a.B * (a.rows_per_batch / a.U);
  hipLaunchKernelGGL(v_post_kernel, dim3(blocks_per_unit * units, a.G), dim3(256), 0, s, a,
                     blocks_per_unit);
  return hipGetLastError();
}

hipError_t unshuffle_latent(const void* z, int z_kind, int B, int C, int F, int H, int W, int p,
                            int K_pad, void* u, int out_kind, hipStream_t s, bool packed) {
  if (packed && (K_pad % 32 || (out_kind != 0 && out_kind != 1))) return hipErrorInvalidValue;
  const int64_t total = (int64_t)B * F * (H / p) * (W / p) * K_pad;
  hipLaunchKernelGGL(unshuffle_kernel, dim3(grid_for(total)), dim3(256), 0, s, z, z_kind, B, C, F,
                     H, W, p, K_pad, u, out_kind, packed ? 1 : 0);
  return hipGetLastError();
}

hipError_t swiglu_f32(const float* raw, int M, int H, float* h, hipStream_t s) {
  hipLaunchKernelGGL(swiglu_f32_kernel, dim3(grid_for((int64_t)M * H)), dim3(256), 0, s, raw, M, H, h);
  return hipGetLastError();
}

hipError_t convert_f32_to_16(const float* src, void* dst, int64_t n, int out_kind, hipStream_t s) {
  hipLaunchKernelGGL(convert_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, dst, n, out_kind);
  return hipGetLastError();
}

}  // namespace fd
