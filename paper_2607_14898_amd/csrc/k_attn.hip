// Windowed GQA attention over the rolling KV ring (Sec. 3.3, Eq. kv_cache).
//
// Queries of causal unit u attend to every key of units max(0, u - W + 1) .. u
// (bidirectional inside a unit, causal across units, window W); query head n
// reads KV group n / (N / G). Keys and values sit in a per-layer ring of S unit
// slots: unit u lives in slot u mod S, K as [U_pad][D_h], V transposed as
// [D_h][U_pad] (U_pad = U rounded up to 64, padding zero-filled once).
//
// 16-bit path (D_h = 64): a workgroup is 4 wave64s; they are 4 query heads of
// one KV group (GQA), so every K / V^T tile staged in LDS serves all four. Each
// wave owns NQB 32-query MFMA blocks (the launch uses one) and computes S^T = K Q^T
// with the 32x32x16 MFMA, so a lane holds one query and 16 key scores per 32-key
// block: the softmax max needs one cross-half exchange per tile and the row
// sums stay lane-local until the end (per tile a packed-f16 sum of the f16
// probabilities for fp16 operands, an fp32 sum for bf16). K
// rows are fed to the MFMA in the order that makes the score registers of a
// lane exactly the B operand of the following O^T += V^T P^T MFMA, so P never
// leaves registers. Queries are pre-scaled by log2(e) / sqrt(D_h), and each
// score accumulator starts from the query's negated running shift (the MFMA's
// C operand), so the MFMA output is the exp2 argument itself. The shift is set
// to the first tile's max and afterwards raised (with O and the row sum
// rescaled) only when some probability of a lane could leave the f16 range;
// only the ragged last tile of a unit is masked. K and V^T tiles of 64 keys
// are double-buffered in LDS.
#include "fd_kernels.h"

#include <hip/hip_bf16.h>
#include <type_traits>

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

// LDS chunk position inside a [64 rows][8 x 16-byte chunks] tile. gfx950 LDS
// serves 16 lanes of a ds_read_b128 per cycle from 16 groups of 16 bytes; chunk
// p of row r sits in group 8 (r % 2) + p. Lanes 0-15 (and 16-31) read 16
// distinct rows of one 16-row block -- in the order of key_of_row for K, in
// order for V^T -- so XOR-ing the chunk with (r / 2) % 8 makes both
// conflict-free, as well as the row-wise tile stores.
__device__ __forceinline__ int swz_k(int row, int c) { return row * 8 + (c ^ ((row >> 1) & 7)); }
__device__ __forceinline__ int swz_v(int row, int c) { return row * 8 + (c ^ ((row >> 1) & 7)); }

// Key fed to A-operand row i of the S^T MFMA (i = 8a + 4b + c maps to key
// 16 (a / 2) + 8 b + 4 (a % 2) + c): output register r of lane l then holds
// key 16 (r / 8) + 8 (l / 32) + r % 8, the B-operand layout of P V^T.
__device__ __forceinline__ int key_of_row(int i) {
  return 16 * (i >> 4) + 8 * ((i >> 2) & 1) + 4 * ((i >> 3) & 1) + (i & 3);
}

constexpr int KT = 64;   // keys per tile

__device__ __forceinline__ __amdgpu_buffer_rsrc_t attn_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// Workgroup: 4 waves = HPB heads of one KV group x (4 / HPB) query sub-tiles of
// 32 NQB queries. K and V^T tiles of 64 keys are shared by the 4 waves through LDS;
// they are copied there by buffer-to-LDS DMA (no register staging), one tile
// ahead. Each wave's Q fragments sit in LDS too, which leaves the registers
// for reading a whole tile's K fragments ahead of the score MFMAs.
template <typename T, int HPB, int NQB>
__global__ __launch_bounds__(256, NQB == 2 ? 2 : 3) void attn_mfma_kernel(AttnArgs a, int q_tiles) {
  using M = AMfma<T>;
  using V = typename M::V;
  constexpr int QW = 32 * NQB;        // queries per wave (NQB 32-query MFMA blocks)
  constexpr int QB = QW * (4 / HPB);  // queries per workgroup
  __shared__ uint4 sk[2][KT * 8];
  __shared__ uint4 sv[2][KT * 8];
  __shared__ uint4 sq[4][NQB * 4 * 64];  // Q fragments of each wave, lane order

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  // Workgroup -> (query tile, head block). The hardware deals workgroups
  // round-robin to the 8 XCDs (workgroup i runs on XCD i % 8), each with its own
  // L2. Every XCD gets a contiguous range of the (head block, query tile) order,
  // so the workgroups one XCD runs together mostly share a KV group, and its K
  // and V^T tiles stream through that XCD's L2 once for all of them.
  const int nbx = gridDim.x, n_wg = nbx * gridDim.y;
  const int lin = blockIdx.y * nbx + blockIdx.x;
  const int xq = n_wg / 8, xr = n_wg % 8, xcd = lin % 8;
  const int wid = (xcd < xr ? xcd * (xq + 1) : xr * (xq + 1) + (xcd - xr) * xq) + lin / 8;
  const int bx = wid % nbx;
  const int qt = bx % q_tiles, bu = bx / q_tiles;
  const int lu = bu % a.n_units, b = bu / a.n_units;
  const int head0 = (wid / nbx) * HPB;
  const int n = head0 + wave % HPB;
  const int g = head0 / (a.N / a.G);
  const int64_t u = a.u0 + lu;
  const int ldq = a.N * 64;
  const int q0 = qt * QB + (wave / HPB) * QW;  // first query (unit-local) of this wave

  // queries pre-scaled by log2(e) / sqrt(D_h): S^T then holds exp2 arguments
  const float c = a.scale * 1.44269504088896341f;
  auto qrow = [&](int qb) {
    return (int64_t)(b * a.n_units + lu) * a.U + min(q0 + qb * 32 + lr, a.U - 1);
  };
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const T* qp = (const T*)a.q + qrow(qb) * ldq + n * 64 + 8 * lh;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = *reinterpret_cast<const uint4*>(qp + 16 * ks);
      const V raw = *reinterpret_cast<const V*>(&v);
      V qv;
#pragma unroll
      for (int e = 0; e < 8; ++e) qv[e] = M::cvt((float)raw[e] * c);
      sq[wave][(qb * 4 + ks) * 64 + lane] = *reinterpret_cast<const uint4*>(&qv);
    }
  }

  const int64_t u_lo = u - a.window + 1 > 0 ? u - a.window + 1 : 0;
  const int tiles_per_unit = a.U_pad / KT;
  const int n_it = (int)(u - u_lo + 1) * tiles_per_unit;
  const int tail_valid = a.U - (tiles_per_unit - 1) * KT;  // keys in a unit's last tile

  // DMA of a tile: wave w moves rows 8 w .. 8 w + 7 and 8 (w + 4) .. of the K
  // tile and of the V^T tile; lane l lands in row base + l / 8, physical chunk
  // l % 8, which holds chunk (l % 8) ^ ((row / 2) % 8) (the swizzle of swz_k /
  // swz_v). The tile walk (ring slot, tile of the unit) advances incrementally.
  int ld_slot = (int)(u_lo % a.S), ld_kt = 0;
  const int64_t ring0 = (int64_t)(b * a.G + g) * a.S;
  const __amdgpu_buffer_rsrc_t rk =
      attn_rsrc((const T*)a.k_ring + ring0 * a.U_pad * 64, (uint32_t)a.S * a.U_pad * 128u);
  const __amdgpu_buffer_rsrc_t rv =
      attn_rsrc((const T*)a.vt_ring + ring0 * 64 * a.U_pad, (uint32_t)a.S * 64u * a.U_pad * 2u);
  const uint32_t ldsk0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)&sk[0][0];
  const uint32_t ldsv0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)&sv[0][0];
  auto dma_tile = [&](int buf) {
    const uint32_t sofk = (uint32_t)(ld_slot * a.U_pad + ld_kt * KT) * 128u;
    const uint32_t sofv = (uint32_t)ld_slot * 64u * (uint32_t)a.U_pad * 2u + (uint32_t)ld_kt * KT * 2u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rb = 8 * (wave + 4 * h);  // first row of this DMA
      int l = __builtin_amdgcn_workitem_id_x() & 63;
      const int row = rb + (l >> 3), ch = (l & 7) ^ ((row >> 1) & 7);
      const uint32_t vk = (uint32_t)(row * 128 + ch * 16);
      const uint32_t vv = (uint32_t)(row * a.U_pad * 2 + ch * 16);
      const uint32_t bo = (uint32_t)buf * KT * 8 * 16 + (uint32_t)rb * 8 * 16;
      // M0 is reserved by the compiler, but nothing else in this kernel reads it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                   :
                   : "s"(ldsk0 + bo), "v"(vk), "s"(rk), "s"(sofk)
                   : "m0");
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                   :
                   : "s"(ldsv0 + bo), "v"(vv), "s"(rv), "s"(sofv)
                   : "m0");
#pragma clang diagnostic pop
    }
    if (++ld_kt == tiles_per_unit) {
      ld_kt = 0;
      if (++ld_slot == a.S) ld_slot = 0;
    }
  };
  // end of a tile: this wave's DMAs and LDS reads are complete, then the
  // barrier publishes the next tile and frees the buffer just read
  auto sync = [&]() {
    __builtin_amdgcn_s_waitcnt(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // Running shift m_q of each query, kept as an f16-representable value. The
  // score MFMAs accumulate onto cinit = -m_q, so they return c q.k - m_q and
  // P = exp2(S^T) needs no VALU work before the exponential. The shift only has
  // to keep P in f16 range: it is set to the first tile's max and raised (and
  // O, l rescaled by the exact exp2 of the change) whenever some p of a lane
  // may exceed 2^15, detected from the lane's partial row sum of the tile.
  float mq[NQB], l_run[NQB];
  f32x16 cinit[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
    for (int r = 0; r < 16; ++r) cinit[qb][r] = 0.f;
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) mq[qb] = l_run[qb] = 0.f;
  f32x16 acc[NQB][2];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[qb][d][r] = 0.f;

  dma_tile(0);
  sync();
  int kt = 0;
  for (int it = 0; it < n_it; ++it) {
    const int cur = it & 1;

    // S^T = K Q^T - m_q: lane holds query lr of each 32-query block, 16 keys per key block
    const bool tail = kt == tiles_per_unit - 1 && tail_valid < KT;
    if (++kt == tiles_per_unit) kt = 0;
    f32x16 s[2][NQB];
    // The MFMA blocks run at raised wave priority: a wave that reaches its MFMAs
    // issues them ahead of the other waves on the SIMD, which meanwhile issue
    // their exp2 / conversion work, so the waves drift into different phases
    // and the matrix and vector units overlap more. The score block with its
    // K fragment reads, which starts a tile's dependency chain, outranks the
    // P V block (3 over 2; measured 1.4% faster per 720p chunk than one level
    // for both MFMA bursts, and 0.9% more with the K reads raised too).
    auto scores = [&](bool with_dma) {
      // all K fragments of the tile are read before the first MFMA, already
      // at the score block's priority
      __builtin_amdgcn_s_setprio(3);
      V kfr[2][4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const uint4 v = sk[cur][swz_k(kb * 32 + key_of_row(lr), 2 * ks + lh)];
          kfr[kb][ks] = *reinterpret_cast<const V*>(&v);
        }
      // the next tile's DMA (main pass only) goes out after the K fragment
      // reads, still at the score block's priority, so their LDS latency
      // overlaps its issue (measured 1.3% faster per 720p chunk than at the
      // loop top)
      if (with_dma && it + 1 < n_it) dma_tile(cur ^ 1);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) {
            const uint4 w = sq[wave][(qb * 4 + ks) * 64 + lane];
            s[kb][qb] = M::run(kfr[kb][ks], *reinterpret_cast<const V*>(&w), ks == 0 ? cinit[qb] : s[kb][qb]);
          }
      __builtin_amdgcn_s_setprio(0);
      // the padding keys of a unit's ragged last tile: register r of a lane
      // holds key 16 (r / 8) + 8 lh + r % 8 of its 32-key block
      if (tail) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (kb * 32 + 16 * (r >> 3) + 8 * lh + (r & 7) >= tail_valid) s[kb][qb][r] = -INFINITY;
      }
    };
    // P = exp2(S^T) in f16, laid out as the B operand of O^T += V^T P^T
    V pf[NQB][4];
    float ls[NQB];
    auto exp_tile = [&]() {
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float t[32];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float p = __builtin_amdgcn_exp2f(s[kb][qb][8 * h + e]);
              pf[qb][kb * 2 + h][e] = M::cvt(p);
              t[(kb * 2 + h) * 8 + e] = p;
            }
          }
        if constexpr (std::is_same<T, _Float16>::value) {
          // row sum of the f16 probabilities the P V MFMA multiplies, by a
          // packed-f16 pairwise tree (16 instructions instead of 31 fp32
          // adds); an overflow to inf raises the shift like any large sum
          typedef _Float16 h2 __attribute__((ext_vector_type(2)));
          h2 u[16];
#pragma unroll
          for (int st = 0; st < 4; ++st)
#pragma unroll
            for (int e = 0; e < 4; ++e) u[st * 4 + e] = h2{pf[qb][st][2 * e], pf[qb][st][2 * e + 1]};
#pragma unroll
          for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
            for (int i = 0; i < w; ++i) u[i] = u[i] + u[i + w];
          ls[qb] = (float)u[0][0] + (float)u[0][1];
        } else {
          // row sum of the fp32 probabilities by a pairwise tree (plain adds
          // overlap the MFMAs; the packed-f16 dot instruction does not)
#pragma unroll
          for (int w = 16; w >= 1; w >>= 1)
#pragma unroll
            for (int i = 0; i < w; ++i) t[i] = t[i] + t[i + w];
          ls[qb] = t[0];
        }
      }
    };
    scores(true);
    exp_tile();
    bool big = false;
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) big = big || !(ls[qb] <= 32768.f);
    if (it == 0 || __builtin_amdgcn_ballot_w64(big) != 0) {
      // On the first tile the shift of every query becomes that tile's max
      // (from the initial 0, so it also drops to a negative max: a row whose
      // logits all lie far below 0 would otherwise underflow to a zero sum);
      // later it is only ever raised. Softmax is invariant to the shift, so
      // any value that keeps P in f16 range is exact. The scores are
      // recomputed from the K tile still in LDS.
      const bool first = it == 0;
      scores(false);
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float m0 = s[0][qb][0], m1 = s[1][qb][0];
#pragma unroll
        for (int r = 1; r < 16; ++r) {
          m0 = fmaxf(m0, s[0][qb][r]);
          m1 = fmaxf(m1, s[1][qb][r]);
        }
        m0 = fmaxf(m0, m1);
        m0 = fmaxf(m0, __shfl_xor(m0, 32));
        // (the first tile's max is bounded below by -65504, the largest f16
        // magnitude, so the shift stays finite in the 16-bit type)
        const float mq_new = (float)M::cvt(mq[qb] + (first ? fmaxf(m0, -65504.f) : fmaxf(m0, 0.f)));
        const float delta = mq_new - mq[qb];  // exact: both are f16 values
        mq[qb] = mq_new;
#pragma unroll
        for (int r = 0; r < 16; ++r) cinit[qb][r] = -mq_new;
        const float alpha = __builtin_amdgcn_exp2f(-delta);
        l_run[qb] *= alpha;
#pragma unroll
        for (int d = 0; d < 2; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[qb][d][r] *= alpha;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][qb][r] -= delta;
      }
      exp_tile();
    }
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) l_run[qb] += ls[qb];

    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int d = 0; d < 2; ++d) {
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const uint4 v = sv[cur][swz_v(d * 32 + lr, 2 * st + lh)];
        const V vf = *reinterpret_cast<const V*>(&v);
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) acc[qb][d] = M::run(vf, pf[qb][st], acc[qb][d]);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    sync();
  }

#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
    const float inv = 1.f / l_tot;
    if (q0 + qb * 32 + lr < a.U) {
      // row-major, or the O projection's packed operand layout (blocks of 16
      // rows x 32 columns; the head's two 32-column halves are blocks 2n, 2n + 1)
      const int64_t orow = qrow(qb);
      T* op = (T*)a.o + (a.o_packed ? (orow >> 4) * ldq * 16 + (orow & 15) * 32 + (int64_t)n * 1024
                                    : orow * ldq + n * 64);
      const int dstep = a.o_packed ? 512 : 32;
#pragma unroll
      for (int d = 0; d < 2; ++d)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          typedef typename M::E E;
          E o4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) o4[e] = M::cvt(acc[qb][d][r4 * 4 + e] * inv);
          *reinterpret_cast<uint2*>(op + d * dstep + 8 * r4 + 4 * lh) = *reinterpret_cast<uint2*>(o4);
        }
    }
  }
}

// fp32 path: one thread per query, 64 queries of one head per workgroup.
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a, int q_tiles) {
  __shared__ float sk[64][DH + 1];
  __shared__ float sv[DH][65];
  __shared__ float ss[64][65];  // scores of a key tile, one column per thread (query)
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
      float mx = m_run;
      for (int j = 0; j < nk; ++j) {
        float acc = 0.f;
        for (int d = 0; d < DH; ++d) acc = fmaf(q[d], sk[j][d], acc);
        const float sc = acc * a.scale;
        ss[j][tid] = sc;
        mx = fmaxf(mx, sc);
      }
      const float alpha = expf(m_run - mx);
      for (int d = 0; d < DH; ++d) o[d] *= alpha;
      l_run *= alpha;
      for (int j = 0; j < nk; ++j) {
        const float p = expf(ss[j][tid] - mx);
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

// Launch shape: 4 heads of a KV group per workgroup when the group has a
// multiple of 4 query heads (GQA), and 32 queries per wave: 143 registers let
// three workgroups share a CU (three waves per SIMD), which hides more of the
// per-tile latency than 64 queries per wave (239 registers, two per CU) saves
// in LDS reads and barriers (measured: 2509 vs 2550 us per 720p refinement
// launch; the same at 480p).
template <typename TT, int HPB>
hipError_t attn_launch(const AttnArgs& a, hipStream_t s) {
  const int q_tiles = (a.U + 32 * (4 / HPB) - 1) / (32 * (4 / HPB));
  dim3 grid(q_tiles * a.n_units * a.B, a.N / HPB);
  hipLaunchKernelGGL((attn_mfma_kernel<TT, HPB, 1>), grid, dim3(256), 0, s, a, q_tiles);
  return hipGetLastError();
}

hipError_t attention_mfma(Act16 t, const AttnArgs& a, hipStream_t s) {
  if (a.Dh != 64 || a.U <= 0 || a.U_pad % 64 || a.N % a.G) return hipErrorInvalidValue;
  const int hpg = a.N / a.G;  // query heads per KV group
  const int hpb = hpg % 4 == 0 ? 4 : (hpg % 2 == 0 ? 2 : 1);
  if (t == Act16::F16) {
    if (hpb == 4) return attn_launch<_Float16, 4>(a, s);
    if (hpb == 2) return attn_launch<_Float16, 2>(a, s);
    return attn_launch<_Float16, 1>(a, s);
  }
  if (hpb == 4) return attn_launch<__hip_bfloat16, 4>(a, s);
  if (hpb == 2) return attn_launch<__hip_bfloat16, 2>(a, s);
  return attn_launch<__hip_bfloat16, 1>(a, s);
}

hipError_t attention_f32(const AttnArgs& a, hipStream_t s) {
  if (a.U <= 0 || a.U_pad % 64 || a.N % a.G || a.o_packed) return hipErrorInvalidValue;
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
