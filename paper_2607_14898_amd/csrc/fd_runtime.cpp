// Host runtime behind include/flashdecoder.h: config validation, weight layout
// and upload, ring / workspace allocation, and the per-chunk launch sequence of
// the streaming decoder (Algorithm 1 of FlashDecoder for the frames of a call).
#include "../../include/flashdecoder.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "fd_kernels.h"

namespace {

thread_local std::string g_last_error;

fd_status fail(fd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

#define FD_HIP(expr)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(FD_ERR_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));       \
  } while (0)

struct Derived {
  int Dh, grid_h, grid_w, L, K_in, K_pad, qkv_w, act_bytes;
  bool is16;
  bool mlp8;     // MLP GEMMs on E4M3 operands (FD_MLP_PRECISION_FP8 / _FP8_STATIC)
  bool mlp8s;    // ... with static per-tensor activation scales (FD_MLP_PRECISION_FP8_STATIC)
  fd::Act16 a16;
  int act_kind;  // 0 f16, 1 bf16, 2 fp32
};

bool pos_int(int v) { return v > 0; }

fd_status validate(const fd_config* c, Derived* d) {
  if (!c) return fail(FD_ERR_INVALID_ARGUMENT, "config is NULL");
  if (c->struct_size != sizeof(fd_config))
    return fail(FD_ERR_INVALID_ARGUMENT, "config struct_size %u != %zu", c->struct_size,
                sizeof(fd_config));
  if (c->compute_dtype < 0 || c->compute_dtype > 2)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown compute_dtype %d", c->compute_dtype);
  const int ints[] = {c->latent_channels, c->latent_h, c->latent_w, c->patch, c->dim,
                      c->n_heads, c->n_kv_groups, c->mlp_hidden, c->r_t, c->s_out,
                      c->out_channels, c->window, c->unit_frames, c->max_batch,
                      c->max_frames_per_call};
  for (int v : ints)
    if (!pos_int(v)) return fail(FD_ERR_INVALID_ARGUMENT, "config sizes must be positive");
  if (c->n_backbone_blocks < 0 || c->n_refine_blocks < 0)
    return fail(FD_ERR_INVALID_ARGUMENT, "negative block count");
  if (c->latent_h % c->patch || c->latent_w % c->patch)
    return fail(FD_ERR_INVALID_ARGUMENT, "latent H', W' must be divisible by patch");
  if (c->dim % c->n_heads) return fail(FD_ERR_INVALID_ARGUMENT, "dim %% n_heads != 0");
  if (c->n_heads % c->n_kv_groups)
    return fail(FD_ERR_INVALID_ARGUMENT, "n_heads %% n_kv_groups != 0");
  if (c->mlp_kind != FD_MLP_SWIGLU && c->mlp_kind != FD_MLP_GELU)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown mlp_kind");
  if (c->norm_kind != FD_NORM_RMS && c->norm_kind != FD_NORM_LAYER)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown norm_kind");
  if (c->head_kind != FD_HEAD_TEMPORAL_FIRST && c->head_kind != FD_HEAD_LINEAR)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown head_kind");
  if (c->head_kind == FD_HEAD_TEMPORAL_FIRST && c->head_hidden <= 0)
    return fail(FD_ERR_INVALID_ARGUMENT, "head_hidden must be positive for the temporal-first head");
  if (!(c->norm_eps > 0.f) || !(c->rope_theta > 1.f))
    return fail(FD_ERR_INVALID_ARGUMENT, "norm_eps must be > 0 and rope_theta > 1");
  if (c->max_frames_per_call % c->unit_frames)
    return fail(FD_ERR_INVALID_ARGUMENT, "max_frames_per_call must be a multiple of unit_frames");
  Derived x{};
  x.Dh = c->dim / c->n_heads;
  x.grid_h = c->latent_h / c->patch;
  x.grid_w = c->latent_w / c->patch;
  // widths that index in 32-bit arithmetic inside the kernels
  const int64_t L64 = (int64_t)x.grid_h * x.grid_w;
  const int64_t kin64 = (int64_t)c->latent_channels * c->patch * c->patch;
  const int64_t cs2_64 = (int64_t)c->out_channels * c->s_out * c->s_out * c->r_t;
  if (L64 >= (int64_t)1 << 23 || kin64 > 65536 || cs2_64 > 65536 || c->mlp_hidden > 65536 ||
      c->head_hidden > 65536 || c->r_t > 64)
    return fail(FD_ERR_UNSUPPORTED,
                "sizes beyond the kernels' ranges (tokens per frame < 2^23, C' p^2, C s_out^2 r_t, MLP and "
                "head widths <= 65536, r_t <= 64)");
  x.L = (int)L64;
  x.K_in = (int)kin64;
  x.is16 = c->compute_dtype != FD_DTYPE_F32;
  x.a16 = c->compute_dtype == FD_DTYPE_BF16 ? fd::Act16::BF16 : fd::Act16::F16;
  x.act_kind = c->compute_dtype == FD_DTYPE_F32 ? 2 : (c->compute_dtype == FD_DTYPE_BF16 ? 1 : 0);
  x.act_bytes = x.is16 ? 2 : 4;
  x.K_pad = x.is16 ? (x.K_in + 63) / 64 * 64 : x.K_in;
  x.qkv_w = c->dim + 2 * c->n_kv_groups * x.Dh;
  if (c->rope && (x.Dh % 16))
    return fail(FD_ERR_INVALID_ARGUMENT, "3D-RoPE needs D_h %% 16 == 0 (got %d)", x.Dh);
  if (x.Dh % 2 || x.Dh > 64)
    return fail(FD_ERR_UNSUPPORTED, "head dim %d not supported (even, <= 64)", x.Dh);
  if (c->dim % 4 || c->dim > 2048)
    return fail(FD_ERR_UNSUPPORTED, "dim must be a multiple of 4 and <= 2048");
  if (x.is16) {
    if (x.Dh != 64) return fail(FD_ERR_UNSUPPORTED, "16-bit compute needs D_h == 64");
    if (c->dim % 64 || c->mlp_hidden % 64 ||
        (c->head_kind == FD_HEAD_TEMPORAL_FIRST && c->head_hidden % 64))
      return fail(FD_ERR_UNSUPPORTED, "16-bit compute needs D, MLP and head widths %% 64 == 0");
  } else if (x.Dh != 16 && x.Dh != 32 && x.Dh != 64) {
    return fail(FD_ERR_UNSUPPORTED, "fp32 compute needs D_h in {16, 32, 64}");
  }
  if (c->mlp_precision < FD_MLP_PRECISION_COMPUTE || c->mlp_precision > FD_MLP_PRECISION_FP8_STATIC)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown mlp_precision %d", c->mlp_precision);
  x.mlp8 = c->mlp_precision != FD_MLP_PRECISION_COMPUTE;
  x.mlp8s = c->mlp_precision == FD_MLP_PRECISION_FP8_STATIC;
  if (x.mlp8 && (!x.is16 || c->mlp_kind != FD_MLP_SWIGLU))
    return fail(FD_ERR_UNSUPPORTED, "the FP8 MLP needs a 16-bit compute dtype and the SwiGLU MLP");
  // Index ranges of the kernels. The rows of one call (batch x frames x L_frm,
  // times r_t in the refinement stack) are split into (stream, unit, position,
  // h, w) by a reciprocal multiply that is exact only below 2^23, and the
  // attention reads one stream's ring of one KV group through a buffer
  // descriptor whose size (S slots x U_pad keys x D_h values) is 32-bit.
  const bool tf = c->head_kind == FD_HEAD_TEMPORAL_FIRST;
  const int64_t rows_call = (int64_t)c->max_batch * c->max_frames_per_call * x.L * (tf ? c->r_t : 1);
  if (rows_call >= (int64_t)1 << 23)
    return fail(FD_ERR_UNSUPPORTED,
                "max_batch x max_frames_per_call x tokens per frame%s = %lld rows per call; the kernels "
                "need fewer than 2^23",
                tf ? " x r_t" : "", (long long)rows_call);
  const int64_t slots = (int64_t)c->window - 1 + c->max_frames_per_call / c->unit_frames;
  const int64_t unit_pad = ((int64_t)c->unit_frames * x.L * (tf ? c->r_t : 1) + 63) / 64 * 64;
  const int64_t ring_bytes = slots * unit_pad * x.Dh * x.act_bytes;
  if (ring_bytes >= (int64_t)1 << 32)
    return fail(FD_ERR_UNSUPPORTED,
                "one KV group's ring of one stream takes %lld bytes (window - 1 + max_frames_per_call / "
                "unit_frames slots); the attention needs fewer than 2^32",
                (long long)ring_bytes);
  if (d) *d = x;
  return FD_OK;
}

struct TensorSpec {
  std::string name;
  int ndim;
  int64_t s0, s1;
};

std::vector<TensorSpec> layout(const fd_config* c) {
  const int D = c->dim, H = c->mlp_hidden, Dh = D / c->n_heads, G = c->n_kv_groups;
  const bool ln = c->norm_kind == FD_NORM_LAYER;
  const bool tf = c->head_kind == FD_HEAD_TEMPORAL_FIRST;
  const int cs2 = c->out_channels * c->s_out * c->s_out;
  std::vector<TensorSpec> v;
  auto add1 = [&](const std::string& n, int64_t a) { v.push_back({n, 1, a, 0}); };
  auto add2 = [&](const std::string& n, int64_t a, int64_t b) { v.push_back({n, 2, a, b}); };
  auto norm = [&](const std::string& p) {
    add1(p + ".g", D);
    if (ln) add1(p + ".b", D);
  };
  add2("embed.w", D, c->latent_channels * c->patch * c->patch);
  add1("embed.b", D);
  const char* stacks[2] = {"bb", "rf"};
  const int nblk[2] = {c->n_backbone_blocks, c->n_refine_blocks};
  for (int s = 0; s < (tf ? 2 : 1); ++s) {
    for (int i = 0; i < nblk[s]; ++i) {
      const std::string p = std::string(stacks[s]) + "." + std::to_string(i);
      norm(p + ".norm1");
      add2(p + ".wqkv", D + 2 * G * Dh, D);
      add1(p + ".bqkv", D + 2 * G * Dh);
      if (c->kv_norm) {
        add1(p + ".knorm.g", Dh);
        add1(p + ".vnorm.g", Dh);
      }
      add2(p + ".wo", D, D);
      add1(p + ".bo", D);
      norm(p + ".norm2");
      if (c->mlp_kind == FD_MLP_SWIGLU) {
        add2(p + ".w13", 2 * H, D);
        add1(p + ".b13", 2 * H);
      } else {
        add2(p + ".w1", H, D);
        add1(p + ".b1", H);
      }
      add2(p + ".w2", D, H);
      add1(p + ".b2", D);
    }
    norm(std::string(stacks[s]) + ".norm_f");
    if (s == 0 && tf) {
      add2("tup.w", (int64_t)c->r_t * D, D);
      add1("tup.b", (int64_t)c->r_t * D);
    }
  }
  if (tf) {
    add2("head1.w", c->head_hidden, D);
    add1("head1.b", c->head_hidden);
    add2("head2.w", cs2, c->head_hidden);
    add1("head2.b", cs2);
  } else {
    add2("head.w", (int64_t)c->r_t * cs2, D);
    add1("head.b", (int64_t)c->r_t * cs2);
  }
  return v;
}

float half_bits_to_float(uint16_t h) {
  const uint32_t s = (h >> 15) & 1, e = (h >> 10) & 31, m = h & 1023;
  float v;
  if (e == 0) v = std::ldexp((float)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = std::ldexp((float)(m | 1024), (int)e - 25);
  return s ? -v : v;
}

float bf16_bits_to_float(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

struct LayerW {
  const void *wqkv = nullptr, *wo = nullptr, *w1 = nullptr, *w2 = nullptr;
  const float *n1g = nullptr, *n1b = nullptr, *bqkv = nullptr, *kg = nullptr, *vg = nullptr,
              *bo = nullptr, *n2g = nullptr, *n2b = nullptr, *b1 = nullptr, *b2 = nullptr;
  const float *s1 = nullptr, *s2 = nullptr;  // per-output-channel scales of E4M3 w13 / w2
};

// OCP E4M3 code (bit layout S.EEEE.MMM, exponent bias 7, no infinities) of a
// finite value: the nearest representable value, ties to even, saturating at
// +-448. Normals 2^e (1 + M/8) for e = -6..8; below 2^-6 subnormals M 2^-9.
uint8_t e4m3_encode(float x) {
  const uint8_t sgn = std::signbit(x) ? 0x80 : 0;
  const float a = std::fabs(x);
  if (a >= 448.f) return sgn | 0x7E;
  if (a < 0.015625f) return sgn | (uint8_t)std::nearbyint(a * 512.f);  // 8 is the code of 2^-6
  int e;
  (void)std::frexp(a, &e);
  e -= 1;  // a in [2^e, 2^(e + 1))
  int m = (int)std::nearbyint(std::ldexp(a, -e) * 8.f) - 8;  // 0..8 (8: carry into the exponent)
  if (m == 8) {
    e += 1;
    m = 0;
  }
  return sgn | (uint8_t)(((e + 7) << 3) | m);
}

// Per-row E4M3 quantisation (the rule documented at fd_quantize_e4m3_rows).
bool quantize_rows_e4m3(const float* in, int64_t rows, int64_t cols, uint8_t* codes, float* scales) {
  for (int64_t r = 0; r < rows; ++r) {
    const float* x = in + r * cols;
    float m = 0.f;
    for (int64_t c = 0; c < cols; ++c) {
      if (!std::isfinite(x[c])) return false;
      m = std::max(m, std::fabs(x[c]));
    }
    const float mm = m > 0.f ? m : 448.f;
    const float inv = 448.f / mm;
    for (int64_t c = 0; c < cols; ++c)
      codes[r * cols + c] = e4m3_encode(std::fmin(448.f, std::fmax(-448.f, x[c] * inv)));
    scales[r] = mm / 448.f;
  }
  return true;
}

}  // namespace

struct fd_decoder {
  fd_config cfg{};
  Derived d{};
  int device = 0;
  void* wmem = nullptr;     // compute-type matrices
  float* fmem = nullptr;    // fp32 vectors (biases, gains) and rope tables
  void* tables = nullptr;   // rope axis / frequency tables
  std::vector<LayerW> bb, rf;
  const void *embed_w = nullptr, *tup_w = nullptr, *head1_w = nullptr, *head2_w = nullptr,
             *head_w = nullptr;
  const float *embed_b = nullptr, *bbf_g = nullptr, *bbf_b = nullptr, *rff_g = nullptr,
              *rff_b = nullptr, *tup_b = nullptr, *head1_b = nullptr, *head2_b = nullptr,
              *head_b = nullptr;
  const int* rope_axis = nullptr;
  const double* rope_freq = nullptr;
  const float2* rope_hw = nullptr;
  // FP8 MLP: static activation scales {s_in, 1/s_in, s_hid, 1/s_hid} per block
  // (backbone blocks, then refinement blocks) and the calibration maxima
  // {amax_in, amax_hid} per block (fp32 bits)
  float* act_sc = nullptr;
  unsigned* calib = nullptr;
  bool act_set = false;
};

struct Probe {
  int cls = -1;
  struct Rec {
    hipEvent_t a, b;
    double work;
  };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  double total_ms = 0.0, work = 0.0;
  int64_t launches = 0;
};

struct fd_kv_cache {
  const fd_decoder* dec = nullptr;
  int batch = 1;
  int64_t t = 0;
  int S = 1;
  int U_bb = 0, U_bb_pad = 0, U_rf = 0, U_rf_pad = 0;
  void* ring = nullptr;
  std::vector<void*> k_bb, v_bb, k_rf, v_rf;
  unsigned* sat = nullptr;  // fp16 hidden values clamped to +-65504 (zeroed with the ring)
  void* ws = nullptr;
  float *x_bb = nullptr, *x_rf = nullptr, *raw = nullptr;
  void *a = nullptr, *q = nullptr, *o = nullptr, *h = nullptr, *u = nullptr;
  uint8_t *a8 = nullptr, *h8 = nullptr;  // E4M3 MLP operands (FP8 MLP)
  float *sa = nullptr, *sh = nullptr;     // their per-row scales
  float2* rope_t = nullptr;  // temporal RoPE (cos, sin) of the current call
  Probe probe;
  // fd_decode_chunks: this cache's own stream and its fork / join events
  hipStream_t own = nullptr;
  hipEvent_t fork = nullptr, done = nullptr;
};

namespace {

// ---------------------------------------------------------------- probe

fd_status probe_begin(fd_kv_cache* c, int cls, hipStream_t s, hipEvent_t* ev, int cls2 = -1) {
  *ev = nullptr;
  if (c->probe.cls != cls && (cls2 < 0 || c->probe.cls != cls2)) return FD_OK;
  if (c->probe.pool.size() < 2) {
    for (int i = 0; i < 64; ++i) {
      hipEvent_t e;
      FD_HIP(hipEventCreate(&e));
      c->probe.pool.push_back(e);
    }
  }
  *ev = c->probe.pool.back();
  c->probe.pool.pop_back();
  FD_HIP(hipEventRecord(*ev, s));
  return FD_OK;
}

fd_status probe_end(fd_kv_cache* c, hipStream_t s, hipEvent_t start, double work) {
  if (!start) return FD_OK;
  hipEvent_t e = c->probe.pool.back();
  c->probe.pool.pop_back();
  FD_HIP(hipEventRecord(e, s));
  c->probe.pending.push_back({start, e, work});
  return FD_OK;
}

// ---------------------------------------------------------------- forward

struct Ctx {
  const fd_decoder* dec;
  fd_kv_cache* c;
  hipStream_t s;
  float* trace;
  int64_t trace_off;
  bool calibrate = false;  // FP8 MLP: per-token scales, maxima recorded into dec->calib
};

fd_status run_gemm(Ctx& x, const fd::GemmArgs& g_in, double algo_k) {
  fd::GemmArgs g = g_in;
  if (x.dec->d.is16) {
    // On the 16-bit path every A operand of these GEMMs (norm, unshuffle and
    // attention outputs, the hidden of the activation epilogues) is stored in
    // the packed operand layout, and so is every 16-bit activation output.
    g.a_packed = 1;
    if (g.epi == fd::EPI_SWIGLU || g.epi == fd::EPI_STORE_ACT || g.epi == fd::EPI_STORE_SILU ||
        g.epi == fd::EPI_STORE_GELU)
      g.ep.out_packed = 1;
  }
  hipEvent_t ev;
  fd_status st = probe_begin(x.c, FD_KC_GEMM, x.s, &ev);
  if (st) return st;
  hipError_t e = x.dec->d.is16 ? fd::gemm_mfma(x.dec->d.a16, g, x.s) : fd::gemm_f32(g, x.s);
  if (e != hipSuccess)
    return fail(FD_ERR_DEVICE, "gemm launch (M=%d N=%d K=%d epi=%d) failed: %s", g.M, g.N, g.K,
                (int)g.epi, hipGetErrorString(e));
  return probe_end(x.c, x.s, ev, 2.0 * g.M * (double)g.N * algo_k);
}

fd::GemmArgs gemm_args(const void* A, int lda, const void* W, int M, int N, int K, fd::Epi epi,
                       const float* bias) {
  fd::GemmArgs g;
  g.A = A;
  g.W = W;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldw = K;
  g.epi = epi;
  g.ep.bias = bias;
  return g;
}

// Norm into the operand buffer a (compute type), or, for the FP8 MLP input,
// into E4M3 codes a8 with per-row scales sa.
fd_status run_norm(Ctx& x, const float* src, int M, const float* g, const float* b, bool e4m3 = false,
                   const float* static_sc = nullptr, unsigned* amax_out = nullptr) {
  const fd_decoder* dec = x.dec;
  hipEvent_t ev;
  fd_status st = probe_begin(x.c, FD_KC_NORM, x.s, &ev);
  if (st) return st;
  hipError_t e = e4m3 ? fd::norm_rows(src, M, dec->cfg.dim, g, b, dec->cfg.norm_kind, dec->cfg.norm_eps,
                                      x.c->a8, 3, x.s, x.c->sa, static_sc, amax_out, true)
                      : fd::norm_rows(src, M, dec->cfg.dim, g, b, dec->cfg.norm_kind, dec->cfg.norm_eps,
                                      x.c->a, dec->d.act_kind, x.s, nullptr, nullptr, nullptr, dec->d.is16);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "norm launch failed: %s", hipGetErrorString(e));
  return probe_end(x.c, x.s, ev, (double)M * dec->cfg.dim * (4.0 + (e4m3 ? 1.0 : dec->d.act_bytes)));
}

fd_status run_gemm8(Ctx& x, const fd::GemmArgs& g_in, double algo_k) {
  // the E4M3 A operands (norm and quantiser codes, the E4M3 SwiGLU codes) are
  // stored in the FP8 GEMM's packed operand layout
  fd::GemmArgs g = g_in;
  g.a_packed = 1;
  if (g.epi == fd::EPI_SWIGLU_E4M3) g.ep.out_packed = 1;
  hipEvent_t ev;
  fd_status st = probe_begin(x.c, FD_KC_GEMM, x.s, &ev);
  if (st) return st;
  hipError_t e = fd::gemm_fp8(g, x.s);
  if (e != hipSuccess)
    return fail(FD_ERR_DEVICE, "fp8 gemm launch (M=%d N=%d K=%d epi=%d) failed: %s", g.M, g.N, g.K,
                (int)g.epi, hipGetErrorString(e));
  return probe_end(x.c, x.s, ev, 2.0 * g.M * (double)g.N * algo_k);
}

fd_status trace_copy(Ctx& x, const float* src, int64_t n) {
  if (!x.trace) return FD_OK;
  FD_HIP(hipMemcpyAsync(x.trace + x.trace_off, src, n * sizeof(float), hipMemcpyDeviceToDevice, x.s));
  x.trace_off += n;
  return FD_OK;
}

// One transformer stack (backbone or refinement) over the rows of this call.
fd_status run_stack(Ctx& x, const std::vector<LayerW>& layers, float* xs, int rows_per_batch,
                    int U, int U_pad, int64_t tau0, const std::vector<void*>& kr,
                    const std::vector<void*>& vr, bool refine) {
  const int layer0 = refine ? x.dec->cfg.n_backbone_blocks : 0;  // index of the FP8 scales
  const fd_decoder* dec = x.dec;
  const fd_config& c = dec->cfg;
  const Derived& d = dec->d;
  fd_kv_cache* kc = x.c;
  const int B = kc->batch;
  const int rows = B * rows_per_batch;
  const int D = c.dim, H = c.mlp_hidden;
  const int n_units = rows_per_batch / U;
  const int64_t u0 = kc->t / c.unit_frames;
  // geometry of the QKV post step (KV-norm, 3D-RoPE, ring append), shared by the layers
  fd::QkvPostArgs qa;
  qa.raw = kc->raw;
  qa.q = kc->q;
  qa.rope_axis = dec->rope_axis;
  qa.rope_freq = dec->rope_freq;
  qa.rope_hw = dec->rope_hw;
  qa.rope_t = kc->rope_t;
  qa.rope = c.rope;
  qa.eps = c.norm_eps;
  qa.B = B;
  qa.N = c.n_heads;
  qa.G = c.n_kv_groups;
  qa.Dh = d.Dh;
  qa.rows_per_batch = rows_per_batch;
  qa.L = d.L;
  qa.grid_w = d.grid_w;
  qa.U = U;
  qa.U_pad = U_pad;
  qa.S = kc->S;
  qa.u0 = u0;
  qa.tau0 = tau0;
  qa.out_kind = d.act_kind;
  // temporal RoPE angles of this call's (sub-)frames, once for the whole stack
  hipError_t e = fd::rope_time(qa, x.s);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "rope_time launch failed: %s", hipGetErrorString(e));
  for (size_t l = 0; l < layers.size(); ++l) {
    const LayerW& w = layers[l];
    fd_status st = run_norm(x, xs, rows, w.n1g, w.n1b);
    if (st) return st;
    qa.k_ring = kr[l];
    qa.vt_ring = vr[l];
    qa.knorm_g = c.kv_norm ? w.kg : nullptr;
    qa.vnorm_g = c.kv_norm ? w.vg : nullptr;
    hipEvent_t ev;
    fd::GemmArgs g;
    if (d.is16) {
      // 16-bit path: the post step runs in the projection's epilogue
      g = gemm_args(kc->a, D, w.wqkv, rows, d.qkv_w, D, fd::EPI_QKV, w.bqkv);
      g.ep.qkv = qa;
      if ((st = run_gemm(x, g, D))) return st;
    } else {
      g = gemm_args(kc->a, D, w.wqkv, rows, d.qkv_w, D, fd::EPI_STORE_F32, w.bqkv);
      g.ep.out_f = kc->raw;
      g.ep.ld_out = d.qkv_w;
      if ((st = run_gemm(x, g, D))) return st;
      if ((st = probe_begin(kc, FD_KC_QKV_POST, x.s, &ev))) return st;
      e = fd::qkv_post(qa, x.s);
      if (e != hipSuccess) return fail(FD_ERR_DEVICE, "qkv_post launch failed: %s", hipGetErrorString(e));
      if ((st = probe_end(kc, x.s, ev, (double)rows * d.qkv_w * (4.0 + d.act_bytes)))) return st;
    }

    fd::AttnArgs aa;
    aa.q = kc->q;
    aa.k_ring = kr[l];
    aa.vt_ring = vr[l];
    aa.o = kc->o;
    aa.B = B;
    aa.N = c.n_heads;
    aa.G = c.n_kv_groups;
    aa.Dh = d.Dh;
    aa.U = U;
    aa.U_pad = U_pad;
    aa.S = kc->S;
    aa.n_units = n_units;
    aa.u0 = u0;
    aa.window = c.window;
    aa.scale = 1.0f / std::sqrt((float)d.Dh);
    aa.o_packed = d.is16 ? 1 : 0;  // the O projection's A operand
    double keys = 0.0;  // visible keys summed over the call's query units
    for (int lu = 0; lu < n_units; ++lu) {
      const int64_t u = u0 + lu;
      const int64_t vis = std::min<int64_t>(u + 1, c.window);
      keys += (double)vis * U;
    }
    if ((st = probe_begin(kc, FD_KC_ATTENTION, x.s, &ev, refine ? FD_KC_ATTENTION_REFINE : -1)))
      return st;
    e = d.is16 ? fd::attention_mfma(d.a16, aa, x.s) : fd::attention_f32(aa, x.s);
    if (e != hipSuccess) return fail(FD_ERR_DEVICE, "attention launch failed: %s", hipGetErrorString(e));
    if ((st = probe_end(kc, x.s, ev, 4.0 * B * c.n_heads * (double)U * keys * d.Dh))) return st;

    g = gemm_args(kc->o, D, w.wo, rows, D, D, fd::EPI_RESID_ADD, w.bo);
    g.ep.out_f = xs;
    g.ep.ld_out = D;
    if ((st = run_gemm(x, g, D))) return st;

    if (d.mlp8 && d.mlp8s && !x.calibrate) {
      // static-calibrated FP8 MLP: E4M3 MLP input at the block's fixed scale,
      // w13 with the fused SwiGLU straight into E4M3 codes at the second fixed
      // scale, w2 with the residual add
      const float* sc = dec->act_sc + 4 * (layer0 + (int)l);
      if ((st = run_norm(x, xs, rows, w.n2g, w.n2b, true, sc))) return st;
      g = gemm_args(kc->a8, D, w.w1, rows, 2 * H, D, fd::EPI_SWIGLU_E4M3, w.b1);
      g.ep.sat = kc->sat;
      g.ep.out_a = kc->h8;
      g.ep.ld_out = H;
      g.ep.row_scale = sc;
      g.ep.row_scale_stride = 0;
      g.ep.col_scale = w.s1;
      g.ep.out_scale = sc + 2;
      if ((st = run_gemm8(x, g, D))) return st;
      g = gemm_args(kc->h8, H, w.w2, rows, D, H, fd::EPI_RESID_ADD, w.b2);
      g.ep.out_f = xs;
      g.ep.ld_out = D;
      g.ep.row_scale = sc + 2;
      g.ep.row_scale_stride = 0;
      g.ep.col_scale = w.s2;
      if ((st = run_gemm8(x, g, H))) return st;
      if ((st = trace_copy(x, xs, (int64_t)rows * D))) return st;
      continue;
    }
    if (d.mlp8) {
      // FP8 MLP (Sec. 4.6 "-Opt"): E4M3 MLP input per token, w13 with the fused
      // SwiGLU into fp16, per-token E4M3 codes of that, w2 with the residual
      // add; when calibrating, the maxima of both quantised tensors are recorded
      unsigned* cal = x.calibrate ? dec->calib + 2 * (layer0 + (int)l) : nullptr;
      if ((st = run_norm(x, xs, rows, w.n2g, w.n2b, true, nullptr, cal))) return st;
      g = gemm_args(kc->a8, D, w.w1, rows, 2 * H, D, fd::EPI_SWIGLU, w.b1);
      g.ep.sat = kc->sat;
      g.ep.out_a = kc->h;
      g.ep.ld_out = H;
      g.ep.row_scale = kc->sa;
      g.ep.col_scale = w.s1;
      if ((st = run_gemm8(x, g, D))) return st;
      if ((st = probe_begin(kc, FD_KC_NORM, x.s, &ev))) return st;
      e = fd::quant_rows_e4m3(kc->h, 0, rows, H, kc->h8, kc->sh, x.s, cal ? cal + 1 : nullptr, true);
      if (e != hipSuccess) return fail(FD_ERR_DEVICE, "quantisation launch failed: %s", hipGetErrorString(e));
      if ((st = probe_end(kc, x.s, ev, (double)rows * H * 3.0))) return st;
      g = gemm_args(kc->h8, H, w.w2, rows, D, H, fd::EPI_RESID_ADD, w.b2);
      g.ep.out_f = xs;
      g.ep.ld_out = D;
      g.ep.row_scale = kc->sh;
      g.ep.col_scale = w.s2;
      if ((st = run_gemm8(x, g, H))) return st;
      if ((st = trace_copy(x, xs, (int64_t)rows * D))) return st;
      continue;
    }
    if ((st = run_norm(x, xs, rows, w.n2g, w.n2b))) return st;
    if (c.mlp_kind == FD_MLP_SWIGLU) {
      if (d.is16) {
        g = gemm_args(kc->a, D, w.w1, rows, 2 * H, D, fd::EPI_SWIGLU, w.b1);
        g.ep.sat = kc->sat;
        g.ep.out_a = kc->h;
        g.ep.ld_out = H;
        if ((st = run_gemm(x, g, D))) return st;
      } else {
        g = gemm_args(kc->a, D, w.w1, rows, 2 * H, D, fd::EPI_STORE_F32, w.b1);
        g.ep.out_f = kc->raw;
        g.ep.ld_out = 2 * H;
        if ((st = run_gemm(x, g, D))) return st;
        e = fd::swiglu_f32(kc->raw, rows, H, (float*)kc->h, x.s);
        if (e != hipSuccess) return fail(FD_ERR_DEVICE, "swiglu launch failed: %s", hipGetErrorString(e));
      }
    } else {
      g = gemm_args(kc->a, D, w.w1, rows, H, D, fd::EPI_STORE_GELU, w.b1);
      g.ep.out_a = kc->h;
      g.ep.ld_out = H;
      if ((st = run_gemm(x, g, D))) return st;
    }
    g = gemm_args(kc->h, H, w.w2, rows, D, H, fd::EPI_RESID_ADD, w.b2);
    g.ep.out_f = xs;
    g.ep.ld_out = D;
    if ((st = run_gemm(x, g, H))) return st;
    if ((st = trace_copy(x, xs, (int64_t)rows * D))) return st;
  }
  return FD_OK;
}

// Argument checks of one decode call (no device work).
fd_status check_decode(const fd_decoder* dec, const void* latent, int32_t latent_dtype, int32_t F,
                       const fd_kv_cache* kc, const void* out, int32_t out_fmt) {
  if (!dec || !kc || !latent || !out) return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument");
  if (kc->dec != dec) return fail(FD_ERR_STATE, "cache was created by a different decoder");
  const fd_config& c = dec->cfg;
  if (latent_dtype < 0 || latent_dtype > 2)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown latent dtype %d", latent_dtype);
  if (out_fmt < FD_PIXELS_F32 || out_fmt > FD_PIXELS_U8)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown pixel format %d", out_fmt);
  if (F <= 0 || F > c.max_frames_per_call || F % c.unit_frames)
    return fail(FD_ERR_INVALID_ARGUMENT,
                "n_frames %d must be in 1..%d and a multiple of unit_frames %d", F,
                c.max_frames_per_call, c.unit_frames);
  return FD_OK;
}

fd_status decode(const fd_decoder* dec, const void* latent, int32_t latent_dtype, int32_t F,
                 fd_kv_cache* kc, void* out, int32_t out_fmt, void* stream, float* trace,
                 size_t trace_elems, bool calibrate = false) {
  fd_status cst = check_decode(dec, latent, latent_dtype, F, kc, out, out_fmt);
  if (cst != FD_OK) return cst;
  if (dec->d.mlp8s && !dec->act_set && !calibrate)
    return fail(FD_ERR_STATE, "static FP8 scales are not set (fd_set_fp8_act_amax)");
  const fd_config& c = dec->cfg;
  const Derived& d = dec->d;
  if (trace && trace_elems < fd_trace_elems(dec, kc->batch, F))
    return fail(FD_ERR_INVALID_ARGUMENT, "trace buffer too small");
  hipStream_t s = (hipStream_t)stream;
  int prev_dev = 0;
  FD_HIP(hipGetDevice(&prev_dev));
  if (prev_dev != dec->device) FD_HIP(hipSetDevice(dec->device));
  Ctx x{dec, kc, s, trace, 0, calibrate};
  const int B = kc->batch;
  const int M = B * F * d.L;
  const int D = c.dim;
  fd_status st = FD_OK;
  hipEvent_t ev;
  do {
    if ((st = probe_begin(kc, FD_KC_EMBED_IN, s, &ev))) break;
    hipError_t e = fd::unshuffle_latent(latent, latent_dtype == FD_DTYPE_F32 ? 0 : (latent_dtype == FD_DTYPE_BF16 ? 1 : 2),
                                        B, c.latent_channels, F, c.latent_h, c.latent_w, c.patch,
                                        d.K_pad, kc->u, d.act_kind, s, d.is16);
    if (e != hipSuccess) { st = fail(FD_ERR_DEVICE, "unshuffle launch failed: %s", hipGetErrorString(e)); break; }
    if ((st = probe_end(kc, s, ev, (double)M * d.K_in * (latent_dtype == FD_DTYPE_F32 ? 4 : 2) +
                                       (double)M * d.K_pad * d.act_bytes))) break;
    fd::GemmArgs g = gemm_args(kc->u, d.K_pad, dec->embed_w, M, D, d.K_pad, fd::EPI_STORE_F32, dec->embed_b);
    g.ep.out_f = kc->x_bb;
    g.ep.ld_out = D;
    if ((st = run_gemm(x, g, d.K_in))) break;
    if ((st = trace_copy(x, kc->x_bb, (int64_t)M * D))) break;
    if ((st = run_stack(x, dec->bb, kc->x_bb, F * d.L, c.unit_frames * d.L, kc->U_bb_pad, kc->t,
                        kc->k_bb, kc->v_bb, false))) break;
    if ((st = run_norm(x, kc->x_bb, M, dec->bbf_g, dec->bbf_b))) break;
    if (c.head_kind == FD_HEAD_TEMPORAL_FIRST) {
      const int MR = M * c.r_t;
      g = gemm_args(kc->a, D, dec->tup_w, M, c.r_t * D, D, fd::EPI_TUP, dec->tup_b);
      g.ep.out_f = kc->x_rf;
      g.ep.ld_out = D;
      g.ep.L = d.L;
      g.ep.r_t = c.r_t;
      g.ep.dim = D;
      if ((st = run_gemm(x, g, D))) break;
      if ((st = trace_copy(x, kc->x_rf, (int64_t)MR * D))) break;
      if ((st = run_stack(x, dec->rf, kc->x_rf, F * c.r_t * d.L, c.unit_frames * c.r_t * d.L,
                          kc->U_rf_pad, kc->t * c.r_t, kc->k_rf, kc->v_rf, true))) break;
      if ((st = run_norm(x, kc->x_rf, MR, dec->rff_g, dec->rff_b))) break;
      g = gemm_args(kc->a, D, dec->head1_w, MR, c.head_hidden, D, fd::EPI_STORE_SILU, dec->head1_b);
      g.ep.sat = kc->sat;
      g.ep.out_a = kc->h;
      g.ep.ld_out = c.head_hidden;
      if ((st = run_gemm(x, g, D))) break;
      const int cs2 = c.out_channels * c.s_out * c.s_out;
      g = gemm_args(kc->h, c.head_hidden, dec->head2_w, MR, cs2, c.head_hidden, fd::EPI_PIXEL,
                    dec->head2_b);
      g.ep.out_f = (float*)out;
      g.ep.out_fmt = out_fmt;
      g.ep.L = d.L;
      g.ep.r_t = c.r_t;
      g.ep.grid_h = d.grid_h;
      g.ep.grid_w = d.grid_w;
      g.ep.s = c.s_out;
      g.ep.C = c.out_channels;
      g.ep.frames_in = F;
      g.ep.frames_out = F * c.r_t;
      g.ep.clamp = c.clamp_output;
      if ((st = run_gemm(x, g, c.head_hidden))) break;
    } else {
      const int cs2 = c.out_channels * c.s_out * c.s_out;
      g = gemm_args(kc->a, D, dec->head_w, M, c.r_t * cs2, D, fd::EPI_LINEAR_PIXEL, dec->head_b);
      g.ep.out_f = (float*)out;
      g.ep.out_fmt = out_fmt;
      g.ep.L = d.L;
      g.ep.r_t = c.r_t;
      g.ep.grid_h = d.grid_h;
      g.ep.grid_w = d.grid_w;
      g.ep.s = c.s_out;
      g.ep.C = c.out_channels;
      g.ep.frames_in = F;
      g.ep.frames_out = F * c.r_t;
      g.ep.clamp = c.clamp_output;
      if ((st = run_gemm(x, g, D))) break;
    }
  } while (false);
  if (prev_dev != dec->device) (void)hipSetDevice(prev_dev);
  if (st != FD_OK) return st;
  kc->t += F;
  return FD_OK;
}

fd_status upload_weights(fd_decoder* dec, const void* w, int32_t wdt, size_t n_elems) {
  const fd_config& c = dec->cfg;
  const Derived& d = dec->d;
  const std::vector<TensorSpec> specs = layout(&c);
  size_t total = 0;
  for (auto& t : specs) total += (size_t)t.s0 * (t.ndim == 2 ? t.s1 : 1);
  if (n_elems != total)
    return fail(FD_ERR_INVALID_ARGUMENT, "weight blob has %zu elements, layout needs %zu", n_elems, total);
  // device sizes: matrices in the compute type, vectors in fp32; 16-bit
  // matrices are stored K-tile-major for the MFMA GEMM (fd::pack_w16_index),
  // rows padded to a multiple of 16
  auto mat_k = [&](const TensorSpec& t) -> int64_t { return t.name == "embed.w" ? d.K_pad : t.s1; };
  auto mat_elems = [&](const TensorSpec& t) -> size_t {
    const int64_t rows = d.is16 ? (t.s0 + 15) / 16 * 16 : t.s0;
    return (size_t)rows * mat_k(t);
  };
  auto ends_with = [](const std::string& n, const char* suf) {
    const size_t k = std::strlen(suf);
    return n.size() > k && n.compare(n.size() - k, k, suf) == 0;
  };
  // FP8 MLP: w13 and w2 are stored as E4M3 codes (1 byte) plus per-row scales
  auto is_fp8 = [&](const TensorSpec& t) {
    return d.mlp8 && t.ndim == 2 && (ends_with(t.name, ".w13") || ends_with(t.name, ".w2"));
  };
  size_t wbytes = 0, fbytes = 0;
  for (auto& t : specs) {
    if (t.ndim == 2) wbytes += (mat_elems(t) * (is_fp8(t) ? 1 : d.act_bytes) + 255) / 256 * 256;
    else fbytes += ((size_t)t.s0 * 4 + 255) / 256 * 256;
    if (is_fp8(t)) fbytes += ((size_t)t.s0 * 4 + 255) / 256 * 256;
  }
  if (hipMalloc(&dec->wmem, wbytes) != hipSuccess)
    return fail(FD_ERR_OUT_OF_MEMORY, "weights: hipMalloc(%zu) failed", wbytes);
  if (hipMalloc((void**)&dec->fmem, fbytes) != hipSuccess)
    return fail(FD_ERR_OUT_OF_MEMORY, "vectors: hipMalloc(%zu) failed", fbytes);
  size_t max_mat = 0;
  for (auto& t : specs)
    if (t.ndim == 2) max_mat = std::max(max_mat, mat_elems(t));
  float* stage = nullptr;
  if (d.is16 && hipMalloc((void**)&stage, max_mat * 4) != hipSuccess)
    return fail(FD_ERR_OUT_OF_MEMORY, "staging: hipMalloc failed");

  std::vector<float> host;
  char* wp = (char*)dec->wmem;
  char* fp = (char*)dec->fmem;
  size_t src_off = 0;
  const bool swiglu_pack = d.is16 && c.mlp_kind == FD_MLP_SWIGLU;
  const int H = c.mlp_hidden;
  fd_status st = FD_OK;
  for (auto& t : specs) {
    const size_t n = (size_t)t.s0 * (t.ndim == 2 ? t.s1 : 1);
    std::vector<float> src(n);
    for (size_t i = 0; i < n; ++i) {
      const size_t k = src_off + i;
      if (wdt == FD_DTYPE_F32) src[i] = ((const float*)w)[k];
      else if (wdt == FD_DTYPE_BF16) src[i] = bf16_bits_to_float(((const uint16_t*)w)[k]);
      else src[i] = half_bits_to_float(((const uint16_t*)w)[k]);
    }
    src_off += n;
    const bool is_w13 = t.name.size() > 4 && t.name.compare(t.name.size() - 4, 4, ".w13") == 0;
    const bool is_b13 = t.name.size() > 4 && t.name.compare(t.name.size() - 4, 4, ".b13") == 0;
    // SwiGLU packing for the fused epilogue: rows interleaved per 32 (gate, up)
    auto interleave = [&](const std::vector<float>& v, int64_t rowlen) {
      std::vector<float> o(v.size());
      for (int64_t q = 0; q < H / 32; ++q)
        for (int e = 0; e < 32; ++e) {
          std::memcpy(&o[(64 * q + e) * rowlen], &v[(32 * q + e) * rowlen], rowlen * 4);
          std::memcpy(&o[(64 * q + 32 + e) * rowlen], &v[(H + 32 * q + e) * rowlen], rowlen * 4);
        }
      return o;
    };
    if (swiglu_pack && (is_w13 || is_b13)) src = interleave(src, is_w13 ? t.s1 : 1);
    const void* dptr;
    const float* wscale = nullptr;
    if (is_fp8(t)) {  // per-row E4M3 codes, packed in 16-row x 64-byte blocks
      const int64_t K = t.s1, rows16 = (t.s0 + 15) / 16 * 16;
      std::vector<uint8_t> codes((size_t)t.s0 * K), packed((size_t)rows16 * K, 0);
      std::vector<float> scales(t.s0);
      if (!quantize_rows_e4m3(src.data(), t.s0, K, codes.data(), scales.data())) {
        st = fail(FD_ERR_INVALID_ARGUMENT, "weight %s has a non-finite value", t.name.c_str());
        break;
      }
      for (int64_t r = 0; r < t.s0; ++r)
        for (int64_t k = 0; k < K; k += 64)
          std::memcpy(&packed[fd::pack_w8_index(r, k, K)], &codes[r * K + k], 64);
      if (hipMemcpy(wp, packed.data(), packed.size(), hipMemcpyHostToDevice) != hipSuccess ||
          hipMemcpy(fp, scales.data(), scales.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
        st = fail(FD_ERR_DEVICE, "weight upload of %s failed", t.name.c_str());
        break;
      }
      dptr = wp;
      wscale = (const float*)fp;
      wp += (packed.size() + 255) / 256 * 256;
      fp += (scales.size() * 4 + 255) / 256 * 256;
    } else if (t.ndim == 2) {
      size_t elems = mat_elems(t);
      if (t.name == "embed.w" && d.K_pad != t.s1) {
        host.assign((size_t)t.s0 * d.K_pad, 0.f);
        for (int64_t r = 0; r < t.s0; ++r)
          std::memcpy(&host[r * d.K_pad], &src[r * t.s1], t.s1 * 4);
        src.swap(host);
      }
      if (d.is16) {  // K-tile-major packing (zero rows up to a multiple of 16)
        const int64_t K = mat_k(t);
        host.assign(elems, 0.f);
        for (int64_t r = 0; r < t.s0; ++r)
          for (int64_t k = 0; k < K; k += 32)  // runs of 32 K-columns stay contiguous
            std::memcpy(&host[fd::pack_w16_index(r, k, K)], &src[r * K + k], 32 * sizeof(float));
        src.swap(host);
      }
      if (d.is16) {
        if (hipMemcpy(stage, src.data(), elems * 4, hipMemcpyHostToDevice) != hipSuccess ||
            fd::convert_f32_to_16(stage, wp, elems, d.act_kind, nullptr) != hipSuccess ||
            hipDeviceSynchronize() != hipSuccess) {
          st = fail(FD_ERR_DEVICE, "weight upload of %s failed", t.name.c_str());
          break;
        }
      } else if (hipMemcpy(wp, src.data(), elems * 4, hipMemcpyHostToDevice) != hipSuccess) {
        st = fail(FD_ERR_DEVICE, "weight upload of %s failed", t.name.c_str());
        break;
      }
      dptr = wp;
      wp += (elems * d.act_bytes + 255) / 256 * 256;
    } else {
      if (hipMemcpy(fp, src.data(), n * 4, hipMemcpyHostToDevice) != hipSuccess) {
        st = fail(FD_ERR_DEVICE, "vector upload of %s failed", t.name.c_str());
        break;
      }
      dptr = fp;
      fp += (n * 4 + 255) / 256 * 256;
    }
    // bind
    const std::string& nm = t.name;
    const float* f = (const float*)dptr;
    if (nm == "embed.w") dec->embed_w = dptr;
    else if (nm == "embed.b") dec->embed_b = f;
    else if (nm == "bb.norm_f.g") dec->bbf_g = f;
    else if (nm == "bb.norm_f.b") dec->bbf_b = f;
    else if (nm == "rf.norm_f.g") dec->rff_g = f;
    else if (nm == "rf.norm_f.b") dec->rff_b = f;
    else if (nm == "tup.w") dec->tup_w = dptr;
    else if (nm == "tup.b") dec->tup_b = f;
    else if (nm == "head1.w") dec->head1_w = dptr;
    else if (nm == "head1.b") dec->head1_b = f;
    else if (nm == "head2.w") dec->head2_w = dptr;
    else if (nm == "head2.b") dec->head2_b = f;
    else if (nm == "head.w") dec->head_w = dptr;
    else if (nm == "head.b") dec->head_b = f;
    else {
      const bool isbb = nm.compare(0, 3, "bb.") == 0;
      const size_t dot = nm.find('.', 3);
      const int li = std::stoi(nm.substr(3, dot - 3));
      LayerW& L = isbb ? dec->bb[li] : dec->rf[li];
      const std::string f2 = nm.substr(dot + 1);
      if (f2 == "norm1.g") L.n1g = f;
      else if (f2 == "norm1.b") L.n1b = f;
      else if (f2 == "wqkv") L.wqkv = dptr;
      else if (f2 == "bqkv") L.bqkv = f;
      else if (f2 == "knorm.g") L.kg = f;
      else if (f2 == "vnorm.g") L.vg = f;
      else if (f2 == "wo") L.wo = dptr;
      else if (f2 == "bo") L.bo = f;
      else if (f2 == "norm2.g") L.n2g = f;
      else if (f2 == "norm2.b") L.n2b = f;
      else if (f2 == "w13" || f2 == "w1") {
        L.w1 = dptr;
        L.s1 = wscale;
      } else if (f2 == "b13" || f2 == "b1") L.b1 = f;
      else if (f2 == "w2") {
        L.w2 = dptr;
        L.s2 = wscale;
      }
      else if (f2 == "b2") L.b2 = f;
    }
  }
  if (stage) (void)hipFree(stage);
  if (st) return st;

  // 3D-RoPE tables: axis and angular frequency of every channel pair
  const int Dh = d.Dh, np = Dh / 2;
  std::vector<int> axis(np);
  std::vector<double> freq(np);
  const int sec[3] = {Dh / 4, (3 * Dh) / 8, Dh - Dh / 4 - (3 * Dh) / 8};
  int pidx = 0;
  for (int a = 0; a < 3; ++a)
    for (int i = 0; i < sec[a] / 2; ++i, ++pidx) {
      axis[pidx] = a;
      freq[pidx] = std::pow((double)c.rope_theta, -2.0 * i / sec[a]);
    }
  // spatial (cos, sin) table: entry (p, pair) for coordinate p along the pair's axis
  const int gmax = std::max(d.grid_h, d.grid_w);
  std::vector<float2> hw((size_t)gmax * np);
  for (int p = 0; p < gmax; ++p)
    for (int i = 0; i < np; ++i) {
      const double ang = axis[i] == 0 ? 0.0 : p * freq[i];
      hw[(size_t)p * np + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
    }
  const size_t tbytes = np * sizeof(double) + 256 + np * sizeof(int) + 256 + hw.size() * sizeof(float2);
  if (hipMalloc(&dec->tables, tbytes) != hipSuccess)
    return fail(FD_ERR_OUT_OF_MEMORY, "rope tables: hipMalloc failed");
  double* fd_ = (double*)dec->tables;
  int* ax = (int*)((char*)dec->tables + np * sizeof(double) + 256);
  float2* hwd = (float2*)((char*)ax + np * sizeof(int) + 256);
  FD_HIP(hipMemcpy(fd_, freq.data(), np * sizeof(double), hipMemcpyHostToDevice));
  FD_HIP(hipMemcpy(ax, axis.data(), np * sizeof(int), hipMemcpyHostToDevice));
  FD_HIP(hipMemcpy(hwd, hw.data(), hw.size() * sizeof(float2), hipMemcpyHostToDevice));
  dec->rope_hw = hwd;
  dec->rope_freq = fd_;
  dec->rope_axis = ax;
  return FD_OK;
}

// Activation workspace of a call of M backbone rows (batch x frames x L_frm):
// byte offsets of every buffer, each 256-byte aligned, and the total.
struct WsLayout {
  size_t xbb = 0, xrf = 0, raw = 0, a = 0, q = 0, o = 0, h = 0, u = 0, rt = 0, a8 = 0, h8 = 0, sa = 0,
         sh = 0, total = 0;
  bool has_rf = false, has_raw = false, has_fp8 = false;
};

WsLayout ws_layout(const fd_config& c, const Derived& d, int64_t M) {
  const bool tf = c.head_kind == FD_HEAD_TEMPORAL_FIRST;
  const int64_t MR = tf ? M * c.r_t : M;
  const int64_t D = c.dim;
  const size_t es = d.act_bytes;
  // fp32 raw projections: the fp32 path's QKV post step and SwiGLU read them;
  // the 16-bit path does both in GEMM epilogues
  const int64_t raw_cols = d.is16 ? 0 : std::max<int64_t>(d.qkv_w, 2 * c.mlp_hidden);
  const int64_t hid = std::max<int64_t>(c.mlp_hidden, tf ? c.head_hidden : 0);
  auto al = [](int64_t b) { return (size_t)((b + 255) / 256 * 256); };
  // GEMM operands (a, o, h, u, a8, h8) in the packed layout hold whole 16-row blocks
  const int64_t M16 = (M + 15) / 16 * 16, MR16 = (MR + 15) / 16 * 16;
  const size_t sizes[13] = {
      al(M * D * 4),                                           // x_bb
      tf ? al(MR * D * 4) : 0,                                 // x_rf
      al(MR * raw_cols * 4),                                   // raw
      al(MR16 * D * (int64_t)es),                              // a
      al(MR * D * (int64_t)es),                                // q
      al(MR16 * D * (int64_t)es),                              // o
      al(MR16 * hid * (int64_t)es),                            // h
      al(M16 * d.K_pad * (int64_t)es),                         // u
      al((int64_t)(M / d.L) * c.r_t * (d.Dh / 2) * (int64_t)sizeof(float2)),  // rope_t
      d.mlp8 ? al(MR16 * D) : 0,                               // a8
      d.mlp8 ? al(MR16 * c.mlp_hidden) : 0,                    // h8
      d.mlp8 ? al(MR * 4) : 0,                                 // sa
      d.mlp8 ? al(MR * 4) : 0};                                // sh
  WsLayout w;
  size_t* off[13] = {&w.xbb, &w.xrf, &w.raw, &w.a, &w.q, &w.o, &w.h, &w.u, &w.rt, &w.a8, &w.h8, &w.sa, &w.sh};
  size_t p = 0;
  for (int i = 0; i < 13; ++i) {
    *off[i] = p;
    p += sizes[i];
  }
  w.total = p;
  w.has_rf = tf;
  w.has_raw = raw_cols > 0;
  w.has_fp8 = d.mlp8;
  return w;
}

// The cache's workspace buffer pointers, saved and restored as a set.
struct WsPtrs {
  float *x_bb, *x_rf, *raw;
  void *a, *q, *o, *h, *u;
  float2* rope_t;
  uint8_t *a8, *h8;
  float *sa, *sh;
};

WsPtrs ws_ptrs(const fd_kv_cache* kc) {
  return {kc->x_bb, kc->x_rf, kc->raw, kc->a, kc->q, kc->o, kc->h, kc->u, kc->rope_t, kc->a8, kc->h8,
          kc->sa, kc->sh};
}

void set_ws_ptrs(fd_kv_cache* kc, const WsPtrs& p) {
  kc->x_bb = p.x_bb;
  kc->x_rf = p.x_rf;
  kc->raw = p.raw;
  kc->a = p.a;
  kc->q = p.q;
  kc->o = p.o;
  kc->h = p.h;
  kc->u = p.u;
  kc->rope_t = p.rope_t;
  kc->a8 = p.a8;
  kc->h8 = p.h8;
  kc->sa = p.sa;
  kc->sh = p.sh;
}

// Point the cache's workspace buffers into base (laid out by w).
void carve_workspace(fd_kv_cache* kc, char* base, const WsLayout& w) {
  set_ws_ptrs(kc, {(float*)(base + w.xbb), w.has_rf ? (float*)(base + w.xrf) : nullptr,
                   w.has_raw ? (float*)(base + w.raw) : nullptr, base + w.a, base + w.q, base + w.o,
                   base + w.h, base + w.u, (float2*)(base + w.rt),
                   w.has_fp8 ? (uint8_t*)(base + w.a8) : nullptr,
                   w.has_fp8 ? (uint8_t*)(base + w.h8) : nullptr,
                   w.has_fp8 ? (float*)(base + w.sa) : nullptr,
                   w.has_fp8 ? (float*)(base + w.sh) : nullptr});
}

void free_decoder(fd_decoder* d) {
  if (!d) return;
  if (d->wmem) (void)hipFree(d->wmem);
  if (d->fmem) (void)hipFree(d->fmem);
  if (d->tables) (void)hipFree(d->tables);
  if (d->act_sc) (void)hipFree(d->act_sc);
  if (d->calib) (void)hipFree(d->calib);
  delete d;
}

void free_cache(fd_kv_cache* c) {
  if (!c) return;
  if (c->ring) (void)hipFree(c->ring);
  if (c->ws) (void)hipFree(c->ws);
  for (auto& r : c->probe.pending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : c->probe.pool) (void)hipEventDestroy(e);
  if (c->own) (void)hipStreamDestroy(c->own);
  if (c->fork) (void)hipEventDestroy(c->fork);
  if (c->done) (void)hipEventDestroy(c->done);
  delete c;
}

}  // namespace

extern "C" {

fd_status fd_config_validate(const fd_config* cfg) { return validate(cfg, nullptr); }

fd_status fd_weights_layout(const fd_config* cfg, fd_tensor_desc* descs, size_t capacity,
                            size_t* n_tensors, size_t* n_elements) {
  fd_status st = validate(cfg, nullptr);
  if (st != FD_OK && st != FD_ERR_UNSUPPORTED) return st;
  try {
    const std::vector<TensorSpec> v = layout(cfg);
    uint64_t off = 0;
    for (size_t i = 0; i < v.size(); ++i) {
      if (descs && i < capacity) {
        fd_tensor_desc& t = descs[i];
        std::memset(&t, 0, sizeof t);
        std::snprintf(t.name, sizeof t.name, "%s", v[i].name.c_str());
        t.ndim = v[i].ndim;
        t.shape[0] = v[i].s0;
        t.shape[1] = v[i].ndim == 2 ? v[i].s1 : 0;
        t.offset = off;
      }
      off += (uint64_t)v[i].s0 * (v[i].ndim == 2 ? v[i].s1 : 1);
    }
    if (n_tensors) *n_tensors = v.size();
    if (n_elements) *n_elements = off;
  } catch (...) {
    return fail(FD_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  return FD_OK;
}

fd_status fd_decoder_create(const fd_config* cfg, const void* weights, int32_t weights_dtype,
                            size_t n_elements, fd_decoder** out) {
  if (!out) return fail(FD_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  Derived d;
  fd_status st = validate(cfg, &d);
  if (st) return st;
  if (!weights) return fail(FD_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (weights_dtype < 0 || weights_dtype > 2)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown weights dtype %d", weights_dtype);
  fd_decoder* dec = nullptr;
  try {
    dec = new fd_decoder;
    dec->cfg = *cfg;
    dec->d = d;
    dec->bb.resize(cfg->n_backbone_blocks);
    dec->rf.resize(cfg->head_kind == FD_HEAD_TEMPORAL_FIRST ? cfg->n_refine_blocks : 0);
    if (hipGetDevice(&dec->device) != hipSuccess) {
      free_decoder(dec);
      return fail(FD_ERR_DEVICE, "no HIP device");
    }
    st = upload_weights(dec, weights, weights_dtype, n_elements);
    if (st == FD_OK && d.mlp8) {
      const size_t nl = dec->bb.size() + dec->rf.size();
      if (hipMalloc((void**)&dec->act_sc, nl * 4 * sizeof(float)) != hipSuccess ||
          hipMalloc((void**)&dec->calib, nl * 2 * sizeof(unsigned)) != hipSuccess)
        st = fail(FD_ERR_OUT_OF_MEMORY, "device allocation of the FP8 scales failed");
    }
  } catch (const std::bad_alloc&) {
    st = fail(FD_ERR_OUT_OF_MEMORY, "host allocation failed");
  } catch (...) {
    st = fail(FD_ERR_DEVICE, "unexpected error while creating the decoder");
  }
  if (st) {
    free_decoder(dec);
    return st;
  }
  *out = dec;
  return FD_OK;
}

void fd_decoder_destroy(fd_decoder* dec) { free_decoder(dec); }

const fd_config* fd_decoder_config(const fd_decoder* dec) { return dec ? &dec->cfg : nullptr; }

fd_status fd_kv_cache_create(const fd_decoder* dec, int32_t batch, fd_kv_cache** out) {
  if (!out) return fail(FD_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  if (!dec) return fail(FD_ERR_INVALID_ARGUMENT, "decoder is NULL");
  const fd_config& c = dec->cfg;
  const Derived& d = dec->d;
  if (batch < 1 || batch > c.max_batch)
    return fail(FD_ERR_INVALID_ARGUMENT, "batch %d outside 1..%d", batch, c.max_batch);
  fd_kv_cache* kc = nullptr;
  try {
    kc = new fd_kv_cache;
  } catch (...) {
    return fail(FD_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  kc->dec = dec;
  kc->batch = batch;
  kc->S = c.window - 1 + c.max_frames_per_call / c.unit_frames;
  const bool tf = c.head_kind == FD_HEAD_TEMPORAL_FIRST;
  kc->U_bb = c.unit_frames * d.L;
  kc->U_bb_pad = (kc->U_bb + 63) / 64 * 64;
  kc->U_rf = tf ? c.unit_frames * c.r_t * d.L : 0;
  kc->U_rf_pad = (kc->U_rf + 63) / 64 * 64;
  const int G = c.n_kv_groups, Dh = d.Dh;
  const size_t es = d.act_bytes;
  const size_t ring_bb = (size_t)batch * G * kc->S * kc->U_bb_pad * Dh * es;
  const size_t ring_rf = (size_t)batch * G * kc->S * kc->U_rf_pad * Dh * es;
  const int nb = c.n_backbone_blocks, nr = tf ? c.n_refine_blocks : 0;
  const size_t ring_total = 2 * (nb * ring_bb + nr * ring_rf) + 256;  // + the saturation counter
  {
    if (hipMalloc(&kc->ring, ring_total) != hipSuccess) {
      free_cache(kc);
      return fail(FD_ERR_OUT_OF_MEMORY, "KV ring: hipMalloc(%zu) failed", ring_total);
    }
    if (hipMemset(kc->ring, 0, ring_total) != hipSuccess) {
      free_cache(kc);
      return fail(FD_ERR_DEVICE, "KV ring memset failed");
    }
  }
  char* p = (char*)kc->ring;
  for (int l = 0; l < nb; ++l) {
    kc->k_bb.push_back(p); p += ring_bb;
    kc->v_bb.push_back(p); p += ring_bb;
  }
  for (int l = 0; l < nr; ++l) {
    kc->k_rf.push_back(p); p += ring_rf;
    kc->v_rf.push_back(p); p += ring_rf;
  }
  kc->sat = (unsigned*)p;
  // workspace for the largest call
  const WsLayout w = ws_layout(c, d, (int64_t)batch * c.max_frames_per_call * d.L);
  if (hipMalloc(&kc->ws, w.total) != hipSuccess) {
    free_cache(kc);
    return fail(FD_ERR_OUT_OF_MEMORY, "workspace: hipMalloc(%zu) failed", w.total);
  }
  carve_workspace(kc, (char*)kc->ws, w);
  *out = kc;
  return FD_OK;
}

fd_status fd_kv_cache_reset(fd_kv_cache* cache) {
  if (!cache) return fail(FD_ERR_INVALID_ARGUMENT, "cache is NULL");
  cache->t = 0;
  return FD_OK;
}

int64_t fd_kv_cache_position(const fd_kv_cache* cache) { return cache ? cache->t : -1; }

fd_status fd_kv_cache_fp16_saturations(fd_kv_cache* cache, uint64_t* count) {
  if (!cache || !count) return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument");
  *count = 0;
  int prev = 0;
  FD_HIP(hipGetDevice(&prev));
  const int dev = cache->dec->device;
  if (prev != dev) FD_HIP(hipSetDevice(dev));
  unsigned v = 0;
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(&v, cache->sat, sizeof v, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemset(cache->sat, 0, sizeof v);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (prev != dev) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "reading the saturation counter failed: %s", hipGetErrorString(e));
  *count = v;
  return FD_OK;
}

void fd_kv_cache_destroy(fd_kv_cache* cache) { free_cache(cache); }

fd_status fd_output_shape(const fd_decoder* dec, int32_t batch, int32_t n_frames, int64_t shape[5]) {
  if (!dec || !shape) return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument");
  const fd_config& c = dec->cfg;
  shape[0] = batch;
  shape[1] = c.out_channels;
  shape[2] = (int64_t)n_frames * c.r_t;
  shape[3] = (int64_t)dec->d.grid_h * c.s_out;
  shape[4] = (int64_t)dec->d.grid_w * c.s_out;
  return FD_OK;
}

size_t fd_trace_elems(const fd_decoder* dec, int32_t batch, int32_t n_frames) {
  if (!dec || batch < 1 || n_frames < 1) return 0;
  const fd_config& c = dec->cfg;
  const size_t rows = (size_t)batch * n_frames * dec->d.L;
  size_t n = (1 + (size_t)c.n_backbone_blocks) * rows * c.dim;
  if (c.head_kind == FD_HEAD_TEMPORAL_FIRST)
    n += (1 + (size_t)c.n_refine_blocks) * rows * c.r_t * c.dim;
  return n;
}

fd_status fd_decode_chunk(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                          int32_t n_frames, fd_kv_cache* cache, float* out, void* stream) {
  try {
    return decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32, stream, nullptr, 0);
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_decode_chunk");
  }
}

fd_status fd_decode_chunk_as(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                             int32_t n_frames, fd_kv_cache* cache, void* out, int32_t out_format,
                             void* stream) {
  try {
    return decode(dec, latent, latent_dtype, n_frames, cache, out, out_format, stream, nullptr, 0);
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_decode_chunk_as");
  }
}

fd_status fd_decode_chunks(const fd_decoder* dec, int32_t n, const void* const* latents,
                           int32_t latent_dtype, int32_t n_frames, fd_kv_cache* const* caches,
                           void* const* outs, int32_t out_format, void* stream) {
  if (!dec || n < 1 || !latents || !caches || !outs)
    return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument or n < 1");
  for (int i = 0; i < n; ++i) {
    fd_status st = check_decode(dec, latents[i], latent_dtype, n_frames, caches[i], outs[i], out_format);
    if (st != FD_OK) return st;
    for (int j = 0; j < i; ++j)
      if (caches[j] == caches[i]) return fail(FD_ERR_INVALID_ARGUMENT, "cache %d appears twice", i);
  }
  try {
    int prev_dev = 0;
    FD_HIP(hipGetDevice(&prev_dev));
    if (prev_dev != dec->device) FD_HIP(hipSetDevice(dec->device));
    fd_status st = FD_OK;
    for (int i = 0; i < n && st == FD_OK; ++i) {  // streams and events, once per cache
      fd_kv_cache* kc = caches[i];
      if (!kc->own && hipStreamCreateWithFlags(&kc->own, hipStreamNonBlocking) != hipSuccess)
        st = fail(FD_ERR_DEVICE, "stream creation failed");
      else if (!kc->fork && hipEventCreateWithFlags(&kc->fork, hipEventDisableTiming) != hipSuccess)
        st = fail(FD_ERR_DEVICE, "event creation failed");
      else if (!kc->done && hipEventCreateWithFlags(&kc->done, hipEventDisableTiming) != hipSuccess)
        st = fail(FD_ERR_DEVICE, "event creation failed");
    }
    hipStream_t s = (hipStream_t)stream;
    // fork: every cache's stream starts after the work already on `stream`
    if (st == FD_OK && hipEventRecord(caches[0]->fork, s) != hipSuccess)
      st = fail(FD_ERR_DEVICE, "event record failed");
    for (int i = 0; i < n && st == FD_OK; ++i) {
      fd_kv_cache* kc = caches[i];
      if (hipStreamWaitEvent(kc->own, caches[0]->fork, 0) != hipSuccess) {
        st = fail(FD_ERR_DEVICE, "stream wait failed");
        break;
      }
      st = decode(dec, latents[i], latent_dtype, n_frames, kc, outs[i], out_format, kc->own, nullptr, 0);
      // join: `stream` continues after every cache's decode (also after a
      // failed one, so no work is left unordered)
      if (hipEventRecord(kc->done, kc->own) != hipSuccess || hipStreamWaitEvent(s, kc->done, 0) != hipSuccess)
        if (st == FD_OK) st = fail(FD_ERR_DEVICE, "join failed");
    }
    if (prev_dev != dec->device) (void)hipSetDevice(prev_dev);
    return st;
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_decode_chunks");
  }
}

fd_status fd_decode_chunk_trace(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                                int32_t n_frames, fd_kv_cache* cache, float* out, void* stream,
                                float* trace, size_t trace_elems) {
  if (!trace) return fail(FD_ERR_INVALID_ARGUMENT, "trace is NULL");
  try {
    return decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32, stream, trace,
                  trace_elems);
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_decode_chunk_trace");
  }
}

fd_status fd_decode_chunk_noalloc(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                                  int32_t n_frames, fd_kv_cache* cache, float* out, void* stream) {
  fd_status st = check_decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32);
  if (st != FD_OK) return st;
  if (cache->probe.cls >= 0)
    return fail(FD_ERR_STATE, "the event probe (which creates events) is enabled on this cache");
  if (dec->d.mlp8s && !dec->act_set)
    return fail(FD_ERR_STATE, "static FP8 scales are not set (fd_set_fp8_act_amax)");
  const WsLayout w = ws_layout(dec->cfg, dec->d, (int64_t)cache->batch * n_frames * dec->d.L);
  if (w.total > fd::kNoallocScratchBytes)
    return fail(FD_ERR_UNSUPPORTED,
                "this call needs %zu bytes of workspace; the fixed workspace of fd_decode_chunk_noalloc "
                "holds %zu (fewer frames per call or a smaller batch fit)",
                w.total, fd::kNoallocScratchBytes);
  try {
    void* base = nullptr;
    const hipError_t e = fd::noalloc_scratch(dec->device, &base);
    if (e != hipSuccess)
      return fail(FD_ERR_DEVICE, "address of the fixed workspace: %s", hipGetErrorString(e));
    // the call's buffers point into the fixed array for its duration; the
    // cache's own workspace pointers are restored afterwards
    const WsPtrs own = ws_ptrs(cache);
    carve_workspace(cache, (char*)base, w);
    st = decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32, stream, nullptr, 0);
    set_ws_ptrs(cache, own);
    return st;
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_decode_chunk_noalloc");
  }
}

fd_status fd_probe_enable(fd_kv_cache* cache, int32_t kernel_class) {
  if (!cache) return fail(FD_ERR_INVALID_ARGUMENT, "cache is NULL");
  if (kernel_class >= FD_KC_COUNT) return fail(FD_ERR_INVALID_ARGUMENT, "unknown kernel class");
  Probe& p = cache->probe;
  for (auto& r : p.pending) {
    (void)hipEventSynchronize(r.b);
    p.pool.push_back(r.a);
    p.pool.push_back(r.b);
  }
  p.pending.clear();
  p.cls = kernel_class < 0 ? -1 : kernel_class;
  p.total_ms = 0.0;
  p.work = 0.0;
  p.launches = 0;
  return FD_OK;
}

fd_status fd_probe_read(fd_kv_cache* cache, double* total_ms, int64_t* launches, double* work) {
  if (!cache) return fail(FD_ERR_INVALID_ARGUMENT, "cache is NULL");
  Probe& p = cache->probe;
  for (auto& r : p.pending) {
    FD_HIP(hipEventSynchronize(r.b));
    float ms = 0.f;
    FD_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    p.total_ms += ms;
    p.work += r.work;
    p.launches += 1;
    p.pool.push_back(r.a);
    p.pool.push_back(r.b);
  }
  p.pending.clear();
  if (total_ms) *total_ms = p.total_ms;
  if (launches) *launches = p.launches;
  if (work) *work = p.work;
  return FD_OK;
}

fd_status fd_measure_mfma_peak(int32_t dtype, int32_t iters, void* stream, double* tflops,
                               double* clock_ghz) {
  if (!tflops || !clock_ghz) return fail(FD_ERR_INVALID_ARGUMENT, "output pointer is NULL");
  if (dtype != FD_DTYPE_F16 && dtype != FD_DTYPE_BF16)
    return fail(FD_ERR_INVALID_ARGUMENT, "dtype must be FD_DTYPE_F16 or FD_DTYPE_BF16");
  if (iters < 1 || iters > 10000000) return fail(FD_ERR_INVALID_ARGUMENT, "iters out of range");
  int dev = 0, cus = 0, wclk_khz = 0;
  FD_HIP(hipGetDevice(&dev));
  FD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  FD_HIP(hipDeviceGetAttribute(&wclk_khz, hipDeviceAttributeWallClockRate, dev));
  if (cus <= 0 || wclk_khz <= 0) return fail(FD_ERR_DEVICE, "device attributes unavailable");
  const int blocks = 2 * cus;
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* clk = nullptr;
  float* sink = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  fd_status st = FD_OK;
  std::vector<unsigned long long> h(2 * (size_t)blocks);
  float ms = 0.f;
  do {
    if (hipMalloc(&clk, h.size() * sizeof(unsigned long long)) != hipSuccess ||
        hipMalloc(&sink, (size_t)blocks * 256 * sizeof(float)) != hipSuccess) {
      st = fail(FD_ERR_OUT_OF_MEMORY, "probe buffers");
      break;
    }
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
      st = fail(FD_ERR_DEVICE, "hipEventCreate failed");
      break;
    }
    const fd::Act16 t = dtype == FD_DTYPE_F16 ? fd::Act16::F16 : fd::Act16::BF16;
    hipError_t e = fd::mfma_peak(t, blocks, iters, clk, sink, s);
    if (e == hipSuccess) e = fd::mfma_peak(t, blocks, iters, clk, sink, s);
    if (e == hipSuccess) e = hipEventRecord(e0, s);
    if (e == hipSuccess) e = fd::mfma_peak(t, blocks, iters, clk, sink, s);
    if (e == hipSuccess) e = hipEventRecord(e1, s);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e == hipSuccess)
      e = hipMemcpy(h.data(), clk, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
      st = fail(FD_ERR_DEVICE, "MFMA probe failed: %s", hipGetErrorString(e));
      break;
    }
  } while (false);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (clk) (void)hipFree(clk);
  if (sink) (void)hipFree(sink);
  if (st != FD_OK) return st;
  double cyc = 0.0, ticks = 0.0;
  for (int b = 0; b < blocks; ++b) {
    cyc += (double)h[2 * b];
    ticks += (double)h[2 * b + 1];
  }
  *tflops = (double)blocks * 4.0 * iters * 16.0 * 32768.0 / (ms * 1e-3) / 1e12;
  *clock_ghz = ticks > 0 ? cyc / ticks * wclk_khz * 1e-6 : 0.0;
  return FD_OK;
}

fd_status fd_measure_issue_overlap(int32_t waves_per_simd, int32_t iters, void* stream, double* cycles) {
  if (!cycles) return fail(FD_ERR_INVALID_ARGUMENT, "output pointer is NULL");
  if (iters < 1 || iters > 10000000) return fail(FD_ERR_INVALID_ARGUMENT, "iters out of range");
  if (waves_per_simd < 1 || waves_per_simd > 2) return fail(FD_ERR_INVALID_ARGUMENT, "waves_per_simd must be 1 or 2");
  int dev = 0, cus = 0;
  FD_HIP(hipGetDevice(&dev));
  FD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  if (cus <= 0) return fail(FD_ERR_DEVICE, "device attributes unavailable");
  const int blocks = cus;  // one workgroup of 4 waves_per_simd waves per compute unit
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* clk = nullptr;
  float* sink = nullptr;
  fd_status st = FD_OK;
  std::vector<unsigned long long> h((size_t)blocks);
  do {
    if (hipMalloc(&clk, h.size() * sizeof(unsigned long long)) != hipSuccess ||
        hipMalloc(&sink, (size_t)blocks * 256 * waves_per_simd * sizeof(float)) != hipSuccess) {
      st = fail(FD_ERR_OUT_OF_MEMORY, "probe buffers");
      break;
    }
    for (int mode = 0; mode < 6 && st == FD_OK; ++mode) {
      hipError_t e = fd::issue_overlap_probe(mode, blocks, waves_per_simd, iters, clk, sink, s);
      if (e == hipSuccess) e = hipStreamSynchronize(s);
      if (e == hipSuccess)
        e = hipMemcpy(h.data(), clk, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
      if (e != hipSuccess) {
        st = fail(FD_ERR_DEVICE, "overlap probe failed: %s", hipGetErrorString(e));
        break;
      }
      double sum = 0.0;
      for (int b = 0; b < blocks; ++b) sum += (double)h[b];
      cycles[mode] = sum / blocks / iters / 4.0;  // shader cycles per slot
    }
  } while (false);
  if (clk) (void)hipFree(clk);
  if (sink) (void)hipFree(sink);
  return st;
}

fd_status fd_measure_lds_bandwidth(int32_t iters, void* stream, double* bytes_per_clock_cu,
                                   double* clock_ghz) {
  if (!bytes_per_clock_cu || !clock_ghz) return fail(FD_ERR_INVALID_ARGUMENT, "output pointer is NULL");
  if (iters < 1 || iters > 10000000) return fail(FD_ERR_INVALID_ARGUMENT, "iters out of range");
  int dev = 0, cus = 0, wclk_khz = 0;
  FD_HIP(hipGetDevice(&dev));
  FD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  FD_HIP(hipDeviceGetAttribute(&wclk_khz, hipDeviceAttributeWallClockRate, dev));
  if (cus <= 0 || wclk_khz <= 0) return fail(FD_ERR_DEVICE, "device attributes unavailable");
  const int per_cu = 2, blocks = per_cu * cus;
  hipStream_t s = (hipStream_t)stream;
  unsigned long long* clk = nullptr;
  unsigned* sink = nullptr;
  fd_status st = FD_OK;
  std::vector<unsigned long long> h(2 * (size_t)blocks);
  do {
    if (hipMalloc(&clk, h.size() * sizeof(unsigned long long)) != hipSuccess ||
        hipMalloc(&sink, (size_t)blocks * 512 * sizeof(unsigned)) != hipSuccess) {
      st = fail(FD_ERR_OUT_OF_MEMORY, "probe buffers");
      break;
    }
    hipError_t e = fd::lds_read_probe(blocks, iters, clk, sink, s);
    if (e == hipSuccess) e = fd::lds_read_probe(blocks, iters, clk, sink, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess)
      e = hipMemcpy(h.data(), clk, h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
      st = fail(FD_ERR_DEVICE, "LDS probe failed: %s", hipGetErrorString(e));
      break;
    }
  } while (false);
  if (clk) (void)hipFree(clk);
  if (sink) (void)hipFree(sink);
  if (st != FD_OK) return st;
  // each workgroup: 8 waves x iters x 8 reads x 64 lanes x 16 bytes over its own cycles;
  // per_cu workgroups share a compute unit
  const double bytes_wg = 8.0 * iters * 8.0 * 64.0 * 16.0;
  double rate = 0.0, cyc = 0.0, ticks = 0.0;
  for (int b = 0; b < blocks; ++b) {
    rate += bytes_wg / (double)h[2 * b];
    cyc += (double)h[2 * b];
    ticks += (double)h[2 * b + 1];
  }
  *bytes_per_clock_cu = rate / blocks * per_cu;
  *clock_ghz = ticks > 0 ? cyc / ticks * wclk_khz * 1e-6 : 0.0;
  return FD_OK;
}

fd_status fd_quantize_e4m3_rows(const float* in, int64_t rows, int64_t cols, uint8_t* codes,
                                float* scales) {
  if (rows < 0 || cols < 1) return fail(FD_ERR_INVALID_ARGUMENT, "rows >= 0 and cols >= 1 required");
  if (rows > 0 && (!in || !codes || !scales)) return fail(FD_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (!quantize_rows_e4m3(in, rows, cols, codes, scales))
    return fail(FD_ERR_INVALID_ARGUMENT, "non-finite input");
  return FD_OK;
}

fd_status fd_quantize_e4m3_rows_device(const float* in, int64_t rows, int64_t cols, uint8_t* codes,
                                       float* scales, void* stream) {
  if (rows < 0 || cols < 8 || cols > 65536 || cols % 8)
    return fail(FD_ERR_INVALID_ARGUMENT, "cols must be a multiple of 8 in [8, 65536], rows >= 0");
  if (rows > 0 && (!in || !codes || !scales)) return fail(FD_ERR_INVALID_ARGUMENT, "NULL pointer");
  hipError_t e = fd::quant_rows_e4m3(in, 2, rows, (int)cols, codes, scales, (hipStream_t)stream);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "quantisation launch failed: %s", hipGetErrorString(e));
  return FD_OK;
}

size_t fd_fp8_act_count(const fd_decoder* dec) {
  return dec && dec->d.mlp8 ? 2 * (dec->bb.size() + dec->rf.size()) : 0;
}

fd_status fd_set_fp8_act_amax(fd_decoder* dec, const float* amax, size_t count) {
  if (!dec || !amax) return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument");
  if (!dec->d.mlp8s) return fail(FD_ERR_STATE, "the decoder does not use static FP8 scales");
  if (count != fd_fp8_act_count(dec))
    return fail(FD_ERR_INVALID_ARGUMENT, "expected %zu amplitudes, got %zu", fd_fp8_act_count(dec), count);
  std::vector<float> sc(2 * count);
  for (size_t i = 0; i < count; ++i) {
    const float a = amax[i];
    if (!(a > 0.f) || !std::isfinite(a))
      return fail(FD_ERR_INVALID_ARGUMENT, "amplitude %zu must be finite and > 0", i);
    sc[2 * i] = a / 448.f;      // dequantisation scale
    sc[2 * i + 1] = 448.f / a;  // quantisation multiplier
  }
  int prev = 0;
  FD_HIP(hipGetDevice(&prev));
  if (prev != dec->device) FD_HIP(hipSetDevice(dec->device));
  const hipError_t e = hipMemcpy(dec->act_sc, sc.data(), sc.size() * sizeof(float), hipMemcpyHostToDevice);
  if (prev != dec->device) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "upload of the FP8 scales failed: %s", hipGetErrorString(e));
  dec->act_set = true;
  return FD_OK;
}

fd_status fd_calibrate_chunk(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                             int32_t n_frames, fd_kv_cache* cache, float* out, float* amax,
                             size_t count, void* stream) {
  if (!dec || !amax) return fail(FD_ERR_INVALID_ARGUMENT, "NULL argument");
  if (!dec->d.mlp8) return fail(FD_ERR_STATE, "the decoder has no FP8 MLP");
  if (count != fd_fp8_act_count(dec))
    return fail(FD_ERR_INVALID_ARGUMENT, "expected %zu amplitudes, got %zu", fd_fp8_act_count(dec), count);
  std::vector<unsigned> bits(count);
  for (size_t i = 0; i < count; ++i) {
    if (!(amax[i] >= 0.f) || !std::isfinite(amax[i]))
      return fail(FD_ERR_INVALID_ARGUMENT, "amplitude %zu must be finite and >= 0", i);
    std::memcpy(&bits[i], &amax[i], 4);
  }
  fd_status st = check_decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32);
  if (st != FD_OK) return st;
  try {
    hipStream_t s = (hipStream_t)stream;
    int prev = 0;
    FD_HIP(hipGetDevice(&prev));
    if (prev != dec->device) FD_HIP(hipSetDevice(dec->device));
    if (hipMemcpyAsync(dec->calib, bits.data(), count * 4, hipMemcpyHostToDevice, s) != hipSuccess)
      st = fail(FD_ERR_DEVICE, "calibration upload failed");
    if (st == FD_OK)
      st = decode(dec, latent, latent_dtype, n_frames, cache, out, FD_PIXELS_F32, stream, nullptr, 0, true);
    if (st == FD_OK && (hipMemcpyAsync(bits.data(), dec->calib, count * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
                        hipStreamSynchronize(s) != hipSuccess))
      st = fail(FD_ERR_DEVICE, "calibration readback failed");
    if (prev != dec->device) (void)hipSetDevice(prev);
    if (st != FD_OK) return st;
    for (size_t i = 0; i < count; ++i) std::memcpy(&amax[i], &bits[i], 4);
    return FD_OK;
  } catch (...) {
    return fail(FD_ERR_DEVICE, "unexpected error in fd_calibrate_chunk");
  }
}

fd_status fd_pack_e4m3_weight(const uint8_t* w, int64_t n, int64_t k, uint8_t* packed) {
  if (n < 1 || k < 64 || k % 64) return fail(FD_ERR_INVALID_ARGUMENT, "N >= 1 and K a positive multiple of 64 required");
  if (!w || !packed) return fail(FD_ERR_INVALID_ARGUMENT, "NULL pointer");
  const int64_t rows16 = (n + 15) / 16 * 16;
  std::memset(packed, 0, (size_t)(rows16 * k));
  for (int64_t r = 0; r < n; ++r)
    for (int64_t c = 0; c < k; c += 64) std::memcpy(&packed[fd::pack_w8_index(r, c, k)], &w[r * k + c], 64);
  return FD_OK;
}

fd_status fd_gemm_e4m3_device(const uint8_t* a, int64_t lda, const float* a_scale,
                              const uint8_t* w_packed, const float* w_scale, const float* bias,
                              int32_t m, int32_t n, int32_t k, int32_t epilogue, void* out,
                              int64_t ld_out, void* stream) {
  if (m < 0 || n < 1 || k < 64 || k > 65536 || k % 64)
    return fail(FD_ERR_INVALID_ARGUMENT, "M >= 0, N >= 1 and K a multiple of 64 in [64, 65536] required");
  if (lda < k || lda % 16 || lda >= (1 << 20) || ld_out >= (1 << 20))
    return fail(FD_ERR_INVALID_ARGUMENT, "lda must be a multiple of 16 in [K, 2^20), ld_out below 2^20");
  if (epilogue != FD_GEMM_E4M3_RESID_ADD && epilogue != FD_GEMM_E4M3_SWIGLU_F16)
    return fail(FD_ERR_INVALID_ARGUMENT, "unknown epilogue %d", epilogue);
  const bool swiglu = epilogue == FD_GEMM_E4M3_SWIGLU_F16;
  if (swiglu && (n % 64 || ld_out < n / 2 || ld_out % 4 || (uintptr_t)out % 8))
    return fail(FD_ERR_INVALID_ARGUMENT,
                "SwiGLU needs N % 64 == 0, ld_out >= N / 2 and a multiple of 4, out 8-byte aligned");
  if (!swiglu && ld_out < n) return fail(FD_ERR_INVALID_ARGUMENT, "ld_out >= N required");
  if (m == 0) return FD_OK;
  if (!a || !a_scale || !w_packed || !w_scale || !bias || !out)
    return fail(FD_ERR_INVALID_ARGUMENT, "NULL pointer");
  if ((uintptr_t)a % 16 || (uintptr_t)w_packed % 16 || (!swiglu && (uintptr_t)out % 4))
    return fail(FD_ERR_INVALID_ARGUMENT, "a and w_packed must be 16-byte aligned, out 4-byte aligned");
  fd::GemmArgs g;
  g.A = a;
  g.W = w_packed;
  g.M = m;
  g.N = n;
  g.K = k;
  g.lda = (int)lda;
  g.ldw = k;
  g.epi = swiglu ? fd::EPI_SWIGLU : fd::EPI_RESID_ADD;
  g.ep.bias = bias;
  g.ep.row_scale = a_scale;
  g.ep.col_scale = w_scale;
  g.ep.ld_out = (int)ld_out;
  if (swiglu) g.ep.out_a = out;
  else g.ep.out_f = (float*)out;
  hipError_t e = fd::gemm_fp8(g, (hipStream_t)stream);
  if (e != hipSuccess) return fail(FD_ERR_DEVICE, "E4M3 GEMM launch failed: %s", hipGetErrorString(e));
  return FD_OK;
}

const char* fd_status_string(fd_status s) {
  switch (s) {
    case FD_OK: return "ok";
    case FD_ERR_INVALID_ARGUMENT: return "invalid argument";
    case FD_ERR_UNSUPPORTED: return "unsupported";
    case FD_ERR_OUT_OF_MEMORY: return "out of memory";
    case FD_ERR_DEVICE: return "device error";
    case FD_ERR_STATE: return "invalid state";
  }
  return "unknown status";
}

const char* fd_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
