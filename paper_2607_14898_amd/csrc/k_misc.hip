// Bandwidth-bound passes of the decoder forward:
//  * norm_rows       pre-sublayer RMSNorm / LayerNorm of the fp32 residual
//                    stream (Sec. 3.2 "Base Architecture") into the operand
//                    format of the next projection;
//  * qkv_post        KV-norm and 3D-RoPE (Sec. 3.2), then the rolling-cache
//                    append of Sec. 3.3 / Algorithm 1 as a write into ring slot
//                    (unit mod S);
//  * unshuffle_latent PixelUnshuffle(p) + raster flatten of latent frames
//                    (Sec. 4.3 and Eq. projection);
//  * swiglu_f32      SwiGLU gate of the fp32 path.
#include "fd_kernels.h"

#include <hip/hip_bf16.h>

namespace fd {
namespace {

__device__ __forceinline__ void store_kind(void* out, int64_t i, float v, int kind) {
  if (kind == 0) ((_Float16*)out)[i] = (_Float16)v;
  else if (kind == 1) ((__hip_bfloat16*)out)[i] = __float2bfloat16(v);
  else ((float*)out)[i] = v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One wave per row; rows of D floats (D % 4 == 0).
template <int KIND>
__global__ __launch_bounds__(256) void norm_kernel(const float* __restrict__ x, int M, int D,
                                                   const float* __restrict__ g,
                                                   const float* __restrict__ bta, float eps,
                                                   void* out, int out_kind) {
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
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      const float e[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int col = 4 * c + k;
        float y = (e[k] - mu) * rs * g[col];
        if (KIND == 1) y += bta[col];
        store_kind(out, (int64_t)row * D + col, y, out_kind);
      }
    }
  }
}

// One wave per (row, head slot): head slots 0..N-1 are query heads, N..N+G-1
// key groups, N+G..N+2G-1 value groups. Lane d handles channel d (D_h <= 64).
__global__ __launch_bounds__(256) void qkv_post_kernel(QkvPostArgs a, int rows) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int hs = blockIdx.y;
  if (row >= rows) return;
  const int Dh = a.Dh;
  const bool act = lane < Dh;
  const int width = a.N * Dh + 2 * a.G * Dh;
  const float x0 = act ? a.raw[(int64_t)row * width + hs * Dh + lane] : 0.f;
  float x = x0;
  const bool is_q = hs < a.N, is_k = !is_q && hs < a.N + a.G, is_v = hs >= a.N + a.G;

  if (a.knorm_g && (is_k || is_v)) {  // KV-norm: RMSNorm over D_h with a learned gain
    const float ms = wave_sum(x * x) / Dh;
    const float* gg = is_k ? a.knorm_g : a.vnorm_g;
    x = act ? x * rsqrtf(ms + a.eps) * gg[lane] : 0.f;
  }
  const int b = row / a.rows_per_batch, rb = row - b * a.rows_per_batch;
  const int fs = rb / a.L, tok = rb - fs * a.L;  // (sub-)frame of the call, token
  if (a.rope && !is_v) {
    const int pair = lane >> 1;
    const float partner = __shfl_xor(x, 1);
    float ang = 0.f;
    if (act) {
      const int axis = a.rope_axis[pair];
      if (axis == 0) {
        // temporal position can be large: reduce the angle in double precision
        const double ph = (double)(a.tau0 + fs) * a.rope_freq[pair];
        ang = (float)(ph - 6.283185307179586 * floor(ph / 6.283185307179586));
      } else {
        const int pos = axis == 1 ? tok / a.grid_w : tok % a.grid_w;
        ang = (float)((double)pos * a.rope_freq[pair]);
      }
    }
    float sn, cs;
    sincosf(ang, &sn, &cs);
    x = (lane & 1) ? partner * sn + x * cs : x * cs - partner * sn;
  }
  if (!act) return;
  if (is_q) {
    store_kind(a.q, (int64_t)row * a.N * Dh + hs * Dh + lane, x, a.out_kind);
    return;
  }
  const int lu = rb / a.U, pos = rb - lu * a.U;
  const int slot = (int)((a.u0 + lu) % a.S);
  if (is_k) {
    const int gk = hs - a.N;
    const int64_t base = (((int64_t)(b * a.G + gk) * a.S + slot) * a.U_pad + pos) * Dh;
    store_kind(a.k_ring, base + lane, x, a.out_kind);
  } else {
    const int gv = hs - a.N - a.G;
    const int64_t base = (((int64_t)(b * a.G + gv) * a.S + slot) * Dh + lane) * a.U_pad + pos;
    store_kind(a.vt_ring, base, x, a.out_kind);
  }
}

// u[(b F + f) L + h W_t + w, c p^2 + i p + j] = z[b, c, f, p h + i, p w + j]; zero padding to K_pad.
__global__ __launch_bounds__(256) void unshuffle_kernel(const void* z, int z_kind, int B, int C,
                                                        int F, int H, int W, int p, int K_pad,
                                                        void* u, int out_kind) {
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
    store_kind(u, e, v, out_kind);
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
                     float eps, void* out, int out_kind, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (D % 4 || D > 2048) return hipErrorInvalidValue;
  const int grid = (M + 3) / 4;
  if (kind == 0)
    hipLaunchKernelGGL(norm_kernel<0>, dim3(grid), dim3(256), 0, s, x, M, D, g, b, eps, out, out_kind);
  else
    hipLaunchKernelGGL(norm_kernel<1>, dim3(grid), dim3(256), 0, s, x, M, D, g, b, eps, out, out_kind);
  return hipGetLastError();
}

hipError_t qkv_post(const QkvPostArgs& a, hipStream_t s) {
  const int rows = a.B * a.rows_per_batch;
  if (rows <= 0) return hipSuccess;
  if (a.Dh > 64 || a.Dh % 2) return hipErrorInvalidValue;
  dim3 grid((rows + 3) / 4, a.N + 2 * a.G);
  hipLaunchKernelGGL(qkv_post_kernel, grid, dim3(256), 0, s, a, rows);
  return hipGetLastError();
}

hipError_t unshuffle_latent(const void* z, int z_kind, int B, int C, int F, int H, int W, int p,
                            int K_pad, void* u, int out_kind, hipStream_t s) {
  const int64_t total = (int64_t)B * F * (H / p) * (W / p) * K_pad;
  hipLaunchKernelGGL(unshuffle_kernel, dim3(grid_for(total)), dim3(256), 0, s, z, z_kind, B, C, F,
                     H, W, p, K_pad, u, out_kind);
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
