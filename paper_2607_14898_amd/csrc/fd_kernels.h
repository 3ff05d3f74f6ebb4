// Internal interface between the host runtime and the gfx950 kernels.
// Every launcher enqueues on `stream` and returns the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fd {

enum class Act16 : int { F16 = 0, BF16 = 1 };  // 16-bit MFMA operand format

// GEMM epilogues: C = A W^T + bias, then one of these.
enum Epi : int {
  EPI_STORE_F32 = 0,   // out_f[row, col] = c
  EPI_RESID_ADD = 1,   // out_f[row, col] += c           (fp32 residual stream)
  EPI_STORE_ACT = 2,   // out_a[row, col] = act(c)        (operand format of the next GEMM)
  EPI_STORE_SILU = 3,  // out_a = SiLU(c)
  EPI_STORE_GELU = 4,  // out_a = GELU(c), erf form
  EPI_SWIGLU = 5,      // out_a[row, j] = SiLU(c_gate) * c_up, W rows interleaved per 32
  EPI_TUP = 6,         // temporal upsampling reshape into the refinement stream (fp32)
  EPI_PIXEL = 7,       // head output -> PixelShuffle store (+clamp), fp32 pixels
  EPI_LINEAR_PIXEL = 8,// linear head output -> sub-frame + PixelShuffle store
  EPI_QKV = 9,         // KV-norm + 3D-RoPE of the QKV projection: q buffer and K / V^T rings
  EPI_SWIGLU_E4M3 = 10,// SwiGLU as EPI_SWIGLU, rounded to fp16, then E4M3 codes at the static
                       // inverse scale out_scale[1] (FP8 GEMM only)
  EPI_COUNT = 11
};

struct QkvPostArgs {
  const float* raw = nullptr;  // [rows, D + 2 G D_h]
  void* q = nullptr;           // [rows, N D_h]
  void* k_ring = nullptr;
  void* vt_ring = nullptr;
  const float* knorm_g = nullptr;  // [D_h] or null
  const float* vnorm_g = nullptr;
  const int* rope_axis = nullptr;  // [D_h / 2] axis of each pair (0 t, 1 h, 2 w)
  const double* rope_freq = nullptr;// [D_h / 2] angular frequency of each pair
  const float2* rope_hw = nullptr;  // [max(grid_h, grid_w)][D_h / 2] (cos, sin) of spatial pairs
  float2* rope_t = nullptr;         // [(sub-)frames of the call][D_h / 2] temporal (cos, sin), filled here
  int rope = 1;
  float eps = 1e-6f;
  int B = 1, N = 1, G = 1, Dh = 64;
  int rows_per_batch = 0;      // rows of one stream in this call
  int L = 0;                   // tokens per (sub-)frame
  int grid_w = 1;
  int U = 0, U_pad = 0, S = 1; // unit geometry of the ring
  int64_t u0 = 0;              // absolute index of the first unit of the call
  int64_t tau0 = 0;            // temporal position of the call's first (sub-)frame
  int out_kind = 0;            // 0 f16, 1 bf16, 2 fp32
};

struct EpiParams {
  float* out_f = nullptr;   // fp32 destination
  void* out_a = nullptr;    // 16-bit (or fp32 on the fp32 path) activation destination
  int ld_out = 0;           // row stride of the destination in elements
  const float* bias = nullptr;
  // reshape / pixel-store geometry
  int L = 0;                // tokens per frame
  int r_t = 1;              // temporal factor
  int dim = 0;              // D (temporal-up)
  int grid_h = 0, grid_w = 0, s = 1, C = 3;
  int frames_in = 0;        // latent frames in the call
  int frames_out = 0;       // output frames in the call (frames_in * r_t)
  int clamp = 1;
  // pixel stores (EPI_PIXEL, EPI_LINEAR_PIXEL) write out_f's memory as fp32
  // (0), bf16 (1, nearest even) or uint8 (2, rint(fp32(x 127.5 + 127.5))
  // limited to 0..255)
  int out_fmt = 0;
  // FP8 GEMM: the accumulator of (row m, column n) is multiplied by
  // row_scale[m] * col_scale[n] before the bias and the epilogue
  const float* row_scale = nullptr;
  const float* col_scale = nullptr;
  int row_scale_stride = 1;          // 0: one scale for every row (static per-tensor)
  const float* out_scale = nullptr;  // EPI_SWIGLU_E4M3: {scale, inverse scale} of the codes
  QkvPostArgs qkv;          // EPI_QKV geometry and destinations (raw unused)
  // fp16 SwiGLU / SiLU outputs beyond +-65504 are clamped to it; when set,
  // the number of clamped values is added here
  unsigned* sat = nullptr;
  // 16-bit activation epilogues (EPI_STORE_ACT / _SILU / _GELU, EPI_SWIGLU of
  // the 16-bit GEMM) and the E4M3 SwiGLU codes of the FP8 GEMM: write out_a in
  // the packed operand layout (pack_a16_index / pack_a8_index with K = ld_out)
  // instead of row-major
  int out_packed = 0;
};

struct GemmArgs {
  // [M, K] row-major with stride lda, or (16-bit MFMA GEMM, a_packed = 1)
  // packed by pack_a16_index with lda = K over ceil(M / 16) 16 rows
  const void* A = nullptr;
  int a_packed = 0;
  // [N, K]: row-major with stride ldw for the fp32 GEMM; for the 16-bit MFMA
  // GEMM packed K-tile-major (see pack_w16_index), ldw = K
  const void* W = nullptr;
  int M = 0, N = 0, K = 0, lda = 0, ldw = 0;
  Epi epi = EPI_STORE_F32;
  EpiParams ep;
};

// Position of element (row, k) of an [N, K] weight in the packed layout the
// 16-bit MFMA GEMM reads: 1 KB blocks of 16 rows x 32 K-columns, block-row
// major, rows padded with zeros to a multiple of 16 (ceil(N / 16) 16 K
// elements in all).
inline int64_t pack_w16_index(int64_t row, int64_t k, int64_t K) {
  return ((row / 16) * (K / 32) + k / 32) * 512 + (row % 16) * 32 + k % 32;
}
// The same layout for a 16-bit activation [M, K] that is a GEMM's A operand.
// Each DMA of a K tile then reads one contiguous 1 KB block (eight whole
// 128-byte lines) instead of 16 rows of 64 bytes, which halves the L2
// requests of the A side. Producers write it (norm, unshuffle, attention
// output, activation epilogues); the buffer holds ceil(M / 16) 16 rows. The
// GEMM reads the rows past M of the last block, which only reach output rows
// that are not stored.
inline int64_t pack_a16_index(int64_t row, int64_t k, int64_t K) { return pack_w16_index(row, k, K); }
// Position of byte (row, k) of an [N, K] E4M3 weight in the packed layout the
// FP8 MFMA GEMM reads: 1 KB blocks of 16 rows x 64 K-columns, block-row major,
// rows padded with zeros to a multiple of 16.
inline int64_t pack_w8_index(int64_t row, int64_t k, int64_t K) {
  return ((row / 16) * (K / 64) + k / 64) * 1024 + (row % 16) * 64 + k % 64;
}
// The same layout for E4M3 activation codes that are an FP8 GEMM's A operand
// (a_packed; written by the norm, the quantiser and the E4M3 SwiGLU epilogue).
inline int64_t pack_a8_index(int64_t row, int64_t k, int64_t K) { return pack_w8_index(row, k, K); }
// 16-bit operand GEMM on MFMA (K > 0, K % 32 == 0, lda % 8 == 0, 16-byte aligned
// A, row-major or packed; W packed as above).
hipError_t gemm_mfma(Act16 t, const GemmArgs& g, hipStream_t stream);
// fp32 GEMM (any shape) for the fp32 compute path.
hipError_t gemm_f32(const GemmArgs& g, hipStream_t stream);
// E4M3 x E4M3 GEMM on the gfx950 32x32x64 FP8 MFMA: A [M, K] E4M3 bytes
// row-major (lda bytes, lda % 16 == 0) or packed (a_packed, pack_a8_index),
// W packed by pack_w8_index, K % 64 == 0;
// epilogues EPI_SWIGLU (fp16 out_a), EPI_SWIGLU_E4M3 (E4M3 out_a) and
// EPI_RESID_ADD, after the row / column scales of EpiParams.
hipError_t gemm_fp8(const GemmArgs& g, hipStream_t stream);

// Attention over the rolling KV ring.
struct AttnArgs {
  const void* q = nullptr;     // [rows, N * D_h], rows = B * n_units * U
  const void* k_ring = nullptr;// [B][G][S][U_pad][D_h]
  const void* vt_ring = nullptr;// [B][G][S][D_h][U_pad]
  void* o = nullptr;           // [rows, N * D_h]; 16-bit path: packed (pack_a16_index) if o_packed
  int o_packed = 0;
  int B = 1, N = 1, G = 1, Dh = 64;
  int U = 0, U_pad = 0;        // tokens per causal unit, padded to 64
  int S = 1;                   // ring slots
  int n_units = 1;             // units in this call
  int64_t u0 = 0;              // absolute index of the call's first unit
  int window = 1;              // W_frm in units
  float scale = 1.f;           // 1 / sqrt(D_h)
};
hipError_t attention_mfma(Act16 t, const AttnArgs& a, hipStream_t stream);
hipError_t attention_f32(const AttnArgs& a, hipStream_t stream);

// Norm of the fp32 residual stream into the next GEMM's operand format.
// kind 0 = RMSNorm, 1 = LayerNorm. out_kind: 0 f16, 1 bf16, 2 fp32, 3 E4M3
// codes: with static_sc ({scale, inverse scale}) at that fixed scale
// (saturating), else with the per-row scale (rule of fd_quantize_e4m3_rows)
// written to row_scale. amax_out, if set, is raised to the largest |output|
// (fp32 bits; calibration).
// packed: output in the packed operand layout (16-bit: pack_a16_index; E4M3
// codes: pack_a8_index; K = D).
hipError_t norm_rows(const float* x, int M, int D, const float* g, const float* b, int kind,
                     float eps, void* out, int out_kind, hipStream_t stream,
                     float* row_scale = nullptr, const float* static_sc = nullptr,
                     unsigned* amax_out = nullptr, bool packed = false);

// Per-row E4M3 quantisation (rule of fd_quantize_e4m3_rows) of in [M, K]
// (in_kind 0 f16, 2 fp32) into codes [M, K] bytes and scale [M] fp32;
// amax_out as for norm_rows; packed: codes in the FP8 GEMM's packed operand
// layout (pack_a8_index, K % 64 == 0).
hipError_t quant_rows_e4m3(const void* in, int in_kind, int64_t M, int K, uint8_t* codes,
                           float* scale, hipStream_t stream, unsigned* amax_out = nullptr,
                           bool packed = false);

// Split raw qkv (fp32, bias included) into rotated queries and the KV ring
// (KV-norm, RoPE) for rows of one call.
hipError_t qkv_post(const QkvPostArgs& a, hipStream_t stream);
// Temporal (cos, sin) of the call's (sub-)frames into a.rope_t; run once per
// stack and call, before the QKV post step of its layers.
hipError_t rope_time(const QkvPostArgs& a, hipStream_t stream);

// PixelUnshuffle + flatten of latent frames into embedding operands [B F L, K_pad]
// (packed: 16-bit output in the packed operand layout, K = K_pad).
hipError_t unshuffle_latent(const void* z, int z_kind, int B, int C, int F, int H, int W, int p,
                            int K_pad, void* u, int out_kind, hipStream_t stream, bool packed = false);

// h[m, j] = SiLU(raw[m, j]) * raw[m, H + j]  (fp32 path, un-interleaved weights)
hipError_t swiglu_f32(const float* raw, int M, int H, float* h, hipStream_t stream);

// Sustained MFMA throughput probe: `blocks` workgroups of 4 waves issue 16
// 32x32x16 MFMAs per iteration each; clk receives per workgroup the shader
// cycles and wall-clock ticks of its loop ([blocks][2]), sink blocks * 256
// floats.
hipError_t mfma_peak(Act16 t, int blocks, int iters, unsigned long long* clk, float* sink,
                     hipStream_t stream);

// LDS read-bandwidth probe: `blocks` workgroups of 8 waves, each wave issuing
// 8 conflict-free ds_read_b128 per iteration; clk as for mfma_peak, sink
// blocks * 512 words.
hipError_t lds_read_probe(int blocks, int iters, unsigned long long* clk, unsigned* sink,
                          hipStream_t stream);

// MFMA / vector-instruction issue overlap probe: `blocks` workgroups of
// 4 waves_per_simd waves (1 or 2 per SIMD) run mode 0..5 (MFMA only; 4
// exponentials; MFMA + 4 exponentials; 8 FMAs; MFMA + 8 FMAs; MFMA + 4
// exponentials + 4 FMAs per slot, 4 slots per iteration); clk receives each
// workgroup's shader cycles, sink blocks * 256 * waves_per_simd floats.
hipError_t issue_overlap_probe(int mode, int blocks, int waves_per_simd, int iters, unsigned long long* clk,
                               float* sink, hipStream_t stream);

// Convert a host-prepared fp32 array on the device into 16-bit operands.
hipError_t convert_f32_to_16(const float* src, void* dst, int64_t n, int out_kind,
                             hipStream_t stream);

}  // namespace fd

namespace fd {
// fd_decode_chunk_noalloc: size of the fixed per-device workspace, and its
// device address on `device` (looked up once per device; no allocation).
constexpr size_t kNoallocScratchBytes = (size_t)256 << 20;
hipError_t noalloc_scratch(int device, void** ptr);
}  // namespace fd
