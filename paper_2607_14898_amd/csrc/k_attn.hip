// Windowed GQA attention over the rolling KV ring (Sec. 3.3, Eq. kv_cache).
//
// Queries of causal unit u attend to every key of units max(0, u - W + 1) .. u
// (bidirectional inside a unit, causal across units, window W); query head n
// reads KV group n / (N / G). Keys and values sit in a per-layer ring of S unit
// slots: unit u lives in slot u mod S, K as [U_pad][D_h], V transposed as
// [D_h][U_pad] (U_pad = U rounded up to 64, padding zero-filled once).
//
// 16-bit path (D_h = 64): a workgroup is 4 wave64s x 32 queries of one head.
// Each wave computes S^T = K Q^T with the 32x32x16 MFMA so that a lane owns one
// query and 16 key scores of each 32-key block; the online-softmax max needs a
// single cross-half exchange per tile and the row sums stay lane-local until
// the end. K rows are fed to the MFMA in the order that makes the score
// registers of a lane exactly the B operand of the following P V^T MFMA, so P
// never leaves registers. K and V^T tiles of 64 keys are double-buffered in LDS.
#include "fd_kernels.h"

#include <hip/hip_bf16.h>

namespace fd {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename T> struct AMfma;
template <> struct AMfma<_Float16> {
  using V = f16x8;
  using E = _Float16;
  static __device__ __forceinline__ f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ E cvt(float x) { return (_Float16)x; }
};
template <> struct AMfma<__hip_bfloat16> {
  using V = bf16x8;
  using E = __bf16;
  static __device__ __forceinline__ f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ E cvt(float x) { return (__bf16)x; }
};

// LDS chunk position inside a [64 rows][8 x 16-byte chunks] tile.
// K tiles are read by rows {0-3, 8-11} together, V^T tiles by 8 consecutive rows.
__device__ __forceinline__ int swz_k(int row, int c) {
  return row * 8 + (c ^ ((row & 3) | (((row >> 3) & 1) << 2)));
}
__device__ __forceinline__ int swz_v(int row, int c) { return row * 8 + (c ^ (row & 7)); }

// Key fed to A-operand row i of the S^T MFMA (i = 8a + 4b + c maps to key
// 16 (a / 2) + 8 b + 4 (a % 2) + c): output register r of lane l then holds
// key 16 (r / 8) + 8 (l / 32) + r % 8, the B-operand layout of P V^T.
__device__ __forceinline__ int key_of_row(int i) {
  return 16 * (i >> 4) + 8 * ((i >> 2) & 1) + 4 * ((i >> 3) & 1) + (i & 3);
}

constexpr int QT = 128;  // queries per workgroup
constexpr int KT = 64;   // keys per tile

template <typename T>
__global__ __launch_bounds__(256, 2) void attn_mfma_kernel(AttnArgs a, int q_tiles) {
  using M = AMfma<T>;
  using V = typename M::V;
  __shared__ uint4 sk[2][KT * 8];
  __shared__ uint4 sv[2][KT * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int n = blockIdx.y;
  const int bx = blockIdx.x;
  const int qt = bx % q_tiles, bu = bx / q_tiles;
  const int lu = bu % a.n_units, b = bu / a.n_units;
  const int g = n / (a.N / a.G);
  const int64_t u = a.u0 + lu;
  const int ldq = a.N * 64;

  // queries of this lane (clamped inside the unit; extra rows are not stored)
  const int qi = qt * QT + wave * 32 + lr;
  const int64_t qrow = (int64_t)(b * a.n_units + lu) * a.U + min(qi, a.U - 1);
  const T* qp = (const T*)a.q + qrow * ldq + n * 64;
  V qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const uint4 v = *reinterpret_cast<const uint4*>(qp + 16 * ks + 8 * lh);
    qf[ks] = *reinterpret_cast<const V*>(&v);
  }

  const int64_t u_lo = u - a.window + 1 > 0 ? u - a.window + 1 : 0;
  const int n_units_vis = (int)(u - u_lo + 1);
  const int tiles_per_unit = a.U_pad / KT;
  const int n_it = n_units_vis * tiles_per_unit;

  // global tile loads: thread handles chunks tid and tid + 256 of each tile
  uint4 rk[2], rv[2];
  auto gload = [&](int it) {
    const int ku_i = it / tiles_per_unit, kt = it - ku_i * tiles_per_unit;
    const int slot = (int)((u_lo + ku_i) % a.S);
    const int64_t ring = ((int64_t)(b * a.G + g) * a.S + slot);
    const T* kb = (const T*)a.k_ring + ring * a.U_pad * 64 + (int64_t)kt * KT * 64;
    const T* vb = (const T*)a.vt_ring + ring * 64 * a.U_pad + (int64_t)kt * KT;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256, r = c >> 3, cc = c & 7;
      rk[i] = *reinterpret_cast<const uint4*>(kb + r * 64 + cc * 8);
      rv[i] = *reinterpret_cast<const uint4*>(vb + (int64_t)r * a.U_pad + cc * 8);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + i * 256, r = c >> 3, cc = c & 7;
      sk[buf][swz_k(r, cc)] = rk[i];
      sv[buf][swz_v(r, cc)] = rv[i];
    }
  };

  const float sl2 = a.scale * 1.44269504088896341f;  // scores in log2 units
  float m_run = -1e30f, l_run = 0.f;
  f32x16 acc_o[2];
#pragma unroll
  for (int d = 0; d < 2; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[d][r] = 0.f;

  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < n_it; ++it) {
    const int cur = it & 1;
    if (it + 1 < n_it) gload(it + 1);
    const int kt = it % tiles_per_unit;
    const int valid = a.U - kt * KT;  // keys of this tile that exist

    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
      const int krow = kb * 32 + key_of_row(lr);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 v = sk[cur][swz_k(krow, 2 * ks + lh)];
        s[kb] = M::run(*reinterpret_cast<const V*>(&v), qf[ks], s[kb]);
      }
    }
    float mx = -1e30f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + 16 * (r >> 3) + 8 * lh + (r & 7);
        const float x = key < valid ? s[kb][r] * sl2 : -INFINITY;
        s[kb][r] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
    V pf[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(s[kb][r] - m_new);
        psum += p;
        pf[kb * 2 + (r >> 3)][r & 7] = M::cvt(p);
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_o[d][r] *= alpha;
#pragma unroll
    for (int d = 0; d < 2; ++d) {
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const uint4 v = sv[cur][swz_v(d * 32 + lr, 2 * st + lh)];
        acc_o[d] = M::run(*reinterpret_cast<const V*>(&v), pf[st], acc_o[d]);
      }
    }
    if (it + 1 < n_it) lstore(cur ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  if (qi < a.U) {
    T* op = (T*)a.o + qrow * ldq + n * 64;
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        typedef typename M::E E;
        E o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = M::cvt(acc_o[d][r4 * 4 + e] * inv);
        *reinterpret_cast<uint2*>(op + d * 32 + 8 * r4 + 4 * lh) = *reinterpret_cast<uint2*>(o4);
      }
  }
}

// fp32 path: one thread per query, 64 queries of one head per workgroup.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a, int q_tiles) {
  __shared__ float sk[64][DH + 1];
  __shared__ float sv[DH][65];
  const int tid = threadIdx.x;
  const int n = blockIdx.y;
  const int bx = blockIdx.x;
  const int qt = bx % q_tiles, bu = bx / q_tiles;
  const int lu = bu % a.n_units, b = bu / a.n_units;
  const int g = n / (a.N / a.G);
  const int64_t u = a.u0 + lu;
  const int ldq = a.N * DH;
  const int qi = qt * 64 + tid;
  const int64_t qrow = (int64_t)(b * a.n_units + lu) * a.U + min(qi, a.U - 1);
  float q[DH], o[DH];
  for (int d = 0; d < DH; ++d) {
    q[d] = ((const float*)a.q)[qrow * ldq + n * DH + d];
    o[d] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  const int64_t u_lo = u - a.window + 1 > 0 ? u - a.window + 1 : 0;
  for (int64_t ku = u_lo; ku <= u; ++ku) {
    const int slot = (int)(ku % a.S);
    const int64_t ring = ((int64_t)(b * a.G + g) * a.S + slot);
    const float* kb = (const float*)a.k_ring + ring * a.U_pad * DH;
    const float* vb = (const float*)a.vt_ring + ring * DH * a.U_pad;
    for (int k0 = 0; k0 < a.U; k0 += 64) {
      __syncthreads();
      for (int e = tid; e < 64 * DH; e += 64) {
        const int r = e / DH, d = e % DH;
        sk[r][d] = kb[(int64_t)(k0 + r) * DH + d];
        sv[d][r] = vb[(int64_t)d * a.U_pad + k0 + r];
      }
      __syncthreads();
      const int nk = min(64, a.U - k0);
      float sc[64];
      float mx = m_run;
      for (int j = 0; j < nk; ++j) {
        float acc = 0.f;
        for (int d = 0; d < DH; ++d) acc = fmaf(q[d], sk[j][d], acc);
        sc[j] = acc * a.scale;
        mx = fmaxf(mx, sc[j]);
      }
      const float alpha = expf(m_run - mx);
      for (int d = 0; d < DH; ++d) o[d] *= alpha;
      l_run *= alpha;
      for (int j = 0; j < nk; ++j) {
        const float p = expf(sc[j] - mx);
        l_run += p;
        for (int d = 0; d < DH; ++d) o[d] = fmaf(p, sv[d][j], o[d]);
      }
      m_run = mx;
    }
  }
  if (qi < a.U) {
    for (int d = 0; d < DH; ++d) ((float*)a.o)[qrow * ldq + n * DH + d] = o[d] / l_run;
  }
}

}  // namespace

hipError_t attention_mfma(Act16 t, const AttnArgs& a, hipStream_t s) {
  if (a.Dh != 64 || a.U <= 0 || a.U_pad % 64 || a.N % a.G) return hipErrorInvalidValue;
  const int q_tiles = (a.U + QT - 1) / QT;
  dim3 grid(q_tiles * a.n_units * a.B, a.N);
  if (t == Act16::F16)
    hipLaunchKernelGGL(attn_mfma_kernel<_Float16>, grid, dim3(256), 0, s, a, q_tiles);
  else
    hipLaunchKernelGGL(attn_mfma_kernel<__hip_bfloat16>, grid, dim3(256), 0, s, a, q_tiles);
  return hipGetLastError();
}

hipError_t attention_f32(const AttnArgs& a, hipStream_t s) {
  if (a.U <= 0 || a.U_pad % 64 || a.N % a.G) return hipErrorInvalidValue;
  const int q_tiles = (a.U + 63) / 64;
  dim3 grid(q_tiles * a.n_units * a.B, a.N);
  switch (a.Dh) {
    case 16: hipLaunchKernelGGL(attn_f32_kernel<16>, grid, dim3(64), 0, s, a, q_tiles); break;
    case 32: hipLaunchKernelGGL(attn_f32_kernel<32>, grid, dim3(64), 0, s, a, q_tiles); break;
    case 64: hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a, q_tiles); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fd
