/*
 * flashdecoder.h -- C ABI of the MI355X (gfx950) FlashDecoder decoder forward.
 *
 * The library decodes video latents into RGB pixels chunk by chunk, as the
 * streaming decoder of FlashDecoder (Kang & Kwak) defines it:
 *   - Sec. 3.1: latent z in R^{B x C' x T' x H' x W'} -> video in R^{B x C x T x H x W};
 *   - Sec. 3.2 / Eq. projection: raster tokens per latent frame, Linear C' -> D
 *     (after PixelUnshuffle(p) for 8x-compressed latents, Sec. 4.3);
 *   - Sec. 3.3 / Eq. kv_cache and Algorithm 1: frame-by-frame processing with a
 *     rolling KV cache of W_frm frames;
 *   - Sec. 3.4 Steps 1-3: temporal upsampling, temporal refinement, 2-layer MLP
 *     head and PixelShuffle.
 *
 * Conventions for every function below:
 *   - Arguments, the configuration and object states are checked before any
 *     device work: a call that fails a check (FD_ERR_INVALID_ARGUMENT,
 *     FD_ERR_UNSUPPORTED, FD_ERR_STATE) enqueues nothing and changes no state.
 *   - A decode call that returns FD_ERR_DEVICE (a kernel launch failed part
 *     way) may already have enqueued the kernels before the failing one: its
 *     output buffer may be partly written and the ring slots of the call's own
 *     frames partly rewritten (slots that hold no frame a later call reads),
 *     while the cache position stays where it was.
 *   - After any non-OK status fd_last_error() holds a message (thread-local).
 *   - No C++ exception crosses this boundary.
 *   - "device pointer" means memory the caller allocated on the GPU the decoder
 *     was created on; "host pointer" means ordinary CPU memory.
 */
#ifndef FLASHDECODER_H
#define FLASHDECODER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fd_status {
  FD_OK = 0,
  FD_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, shape or config value      */
  FD_ERR_UNSUPPORTED = 2,      /* valid per the paper but not built here          */
  FD_ERR_OUT_OF_MEMORY = 3,    /* device allocation failed                        */
  FD_ERR_DEVICE = 4,           /* a HIP runtime call or kernel launch failed      */
  FD_ERR_STATE = 5             /* object used in the wrong state / wrong pairing  */
} fd_status;

/* Element types. Compute types: F32 (all fp32) or F16 / BF16 (16-bit MFMA
 * operands, fp32 accumulation, fp32 residual stream, fp32 norm and softmax
 * statistics). Input types (weights, latents): F32, BF16 or F16. */
typedef enum fd_dtype { FD_DTYPE_F32 = 0, FD_DTYPE_BF16 = 1, FD_DTYPE_F16 = 2 } fd_dtype;

enum { FD_MLP_SWIGLU = 0, FD_MLP_GELU = 1 };
enum { FD_NORM_RMS = 0, FD_NORM_LAYER = 1 };
enum { FD_HEAD_TEMPORAL_FIRST = 0, FD_HEAD_LINEAR = 1 };
/* Operand precision of the two MLP GEMMs of every block. FP8: the "-Opt"
 * decoder of Sec. 4.6 runs its MLP GEMMs in FP8; here both take OCP E4M3
 * operands (round to nearest even, saturating at +-448): the weights quantised
 * per output channel at create (static scales), the MLP input and the SwiGLU
 * output (kept in fp16 between the two GEMMs) per token when produced, with
 * fp32 accumulation and the two scales applied in the epilogue.
 * FP8_STATIC: the paper's "static-calibrated" form: the MLP input and the
 * fp16 SwiGLU output of every block take one fixed scale each, amax / 448,
 * from amplitudes given with fd_set_fp8_act_amax (for instance the maxima
 * fd_calibrate_chunk records); values beyond amax saturate. Decoding before the
 * amplitudes are set gives STATE. Both need a 16-bit compute dtype and the
 * SwiGLU MLP. */
enum { FD_MLP_PRECISION_COMPUTE = 0, FD_MLP_PRECISION_FP8 = 1, FD_MLP_PRECISION_FP8_STATIC = 2 };

/* Decoder shape. Copied by fd_decoder_create; the caller keeps ownership.
 * Field meanings follow the paper's notation (Sec. 3.2-3.4, supplement Table A). */
typedef struct fd_config {
  uint32_t struct_size;      /* must be sizeof(fd_config) (ABI guard)                   */
  int32_t compute_dtype;     /* fd_dtype                                                 */
  int32_t latent_channels;   /* C'                                                       */
  int32_t latent_h, latent_w;/* H', W' of the latent frames                              */
  int32_t patch;             /* PixelUnshuffle factor p (Sec. 4.3); H', W' divisible by p */
  int32_t dim;               /* D                                                        */
  int32_t n_heads;           /* N (query heads); head dim D_h = D / N                    */
  int32_t n_kv_groups;       /* G (GQA key/value groups); N % G == 0                     */
  int32_t n_backbone_blocks; /* blocks of the backbone transformer B                     */
  int32_t n_refine_blocks;   /* blocks of the temporal refinement transformer R          */
  int32_t mlp_hidden;        /* MLP hidden width (4 D in the paper)                      */
  int32_t head_hidden;       /* hidden width of the 2-layer pixel head                   */
  int32_t mlp_kind;          /* FD_MLP_*                                                 */
  int32_t norm_kind;         /* FD_NORM_*                                                */
  int32_t head_kind;         /* FD_HEAD_*                                                */
  int32_t kv_norm;           /* 1: RMS-normalise keys and values over D_h (KV-norm)      */
  int32_t rope;              /* 1: 3D-RoPE on queries and keys                           */
  float rope_theta;          /* RoPE base (10000)                                        */
  float norm_eps;            /* epsilon of every norm                                    */
  int32_t r_t;               /* temporal upsampling factor                               */
  int32_t s_out;             /* output pixels per token side (p x latent spatial factor) */
  int32_t out_channels;      /* C (3)                                                    */
  int32_t window;            /* W_frm, in causal units                                   */
  int32_t unit_frames;       /* latent frames per causal unit (1 in the paper)           */
  int32_t max_batch;         /* largest batch a cache of this decoder may hold           */
  int32_t max_frames_per_call;/* largest n_frames of one fd_decode_chunk call            */
  int32_t clamp_output;      /* 1: clamp pixels to [-1, 1]                               */
  int32_t mlp_precision;     /* FD_MLP_PRECISION_*                                       */
} fd_config;

/* One learned tensor of the canonical weight blob. */
typedef struct fd_tensor_desc {
  char name[48];             /* e.g. "bb.3.wqkv"                                         */
  int32_t ndim;              /* 1 or 2                                                   */
  int64_t shape[2];          /* [out, in] for Linear weights (row-major), [n] otherwise  */
  uint64_t offset;           /* element offset of the tensor in the blob                 */
} fd_tensor_desc;

typedef struct fd_decoder fd_decoder;
typedef struct fd_kv_cache fd_kv_cache;

/* ------------------------------------------------------------------------
 * Decoder, streaming state and the decode call: the problem statement's
 * create(config, weights) / reset / decode_chunk(latent, cache, pixels).
 * ------------------------------------------------------------------------ */

/* Check a config. FD_OK, FD_ERR_INVALID_ARGUMENT (inconsistent values) or
 * FD_ERR_UNSUPPORTED: a 16-bit compute type with D_h != 64, or sizes beyond
 * the kernels' index ranges -- max_batch x max_frames_per_call x L_frm rows
 * per call (x r_t for the temporal-first head) must stay below 2^23, one
 * stream's ring of one KV group ((window - 1 + max_frames_per_call /
 * unit_frames) slots of L_frm unit_frames (x r_t) keys rounded up to 64, of
 * D_h values) below 2^32 bytes, L_frm below 2^23, and C' p^2, C s_out^2 r_t,
 * mlp_hidden and head_hidden at most 65536. Host only. */
fd_status fd_config_validate(const fd_config* cfg);

/* Canonical weight layout of the learned tensors the paper's decoder defines:
 * the latent projection (Sec. 3.2, Eq. projection), the transformer blocks of
 * the backbone and of the temporal refinement stack (Sec. 3.2; Sec. 3.4 Step
 * 2), the temporal upsampling Linear (Sec. 3.4 Step 1, Eq. temporal_upsample)
 * and the pixel head (Sec. 3.4 Step 3). All tensors are concatenated in this
 * order (row-major):
 * embed.w [D, C'p^2], embed.b; per block of B then R: norm1.g (+.b for LayerNorm),
 * wqkv [D + 2 G D_h, D] (rows q | k | v), bqkv, knorm.g [D_h] and vnorm.g [D_h]
 * (if kv_norm), wo [D, D], bo, norm2.g (+.b), w13 [2H, D] (rows gate | up) and
 * b13 (SwiGLU) or w1 [H, D] and b1 (GELU), w2 [D, H], b2; after each stack its
 * final norm (bb.norm_f, rf.norm_f); tup.w [r_t D, D] and tup.b after the
 * backbone; head1.w [head_hidden, D], head1.b, head2.w [C s^2, head_hidden],
 * head2.b (temporal-first head) or head.w [r_t C s^2, D], head.b (linear head).
 * descs (host, may be NULL) receives up to `capacity` entries; *n_tensors and
 * *n_elements (host, may be NULL) receive the totals. Host only. */
fd_status fd_weights_layout(const fd_config* cfg, fd_tensor_desc* descs, size_t capacity,
                            size_t* n_tensors, size_t* n_elements);

/* Create the decoder of Sec. 3.2-3.4 (shape per cfg; the FlashDecoder-XL
 * hyper-parameters are those of the supplement's Table A) on the current HIP
 * device: validates cfg, copies the weight
 * blob (host pointer, canonical layout, n_elements values of weights_dtype) to
 * the device, converting and packing it for the compute type, and builds the
 * RoPE tables. The blob is only read during the call. The decoder owns its
 * device memory; it is immutable afterwards and may be shared by caches used on
 * different streams. Synchronous. */
fd_status fd_decoder_create(const fd_config* cfg, const void* weights, int32_t weights_dtype,
                            size_t n_elements, fd_decoder** out);

/* Free a decoder (NULL is ignored). All caches created from it must be
 * destroyed first and no work using it may be in flight. */
void fd_decoder_destroy(fd_decoder* dec);

/* The decoder's config (host pointer valid while dec lives), or NULL. */
const fd_config* fd_decoder_config(const fd_decoder* dec);

/* Create the streaming state of `batch` independent streams (1..max_batch):
 * per-layer rolling K/V rings (Eq. kv_cache: G x W_frm L_frm x D_h per layer
 * and stream, plus room for the frames of one call) and the activation
 * workspace. Starts at position 0. Synchronous. */
fd_status fd_kv_cache_create(const fd_decoder* dec, int32_t batch, fd_kv_cache** out);

/* Rewind to position 0 (Algorithm 1: caches initialised to empty). O(1): no
 * device work; ring contents are ignored until rewritten. Must not be called
 * while a decode on this cache is in flight. */
fd_status fd_kv_cache_reset(fd_kv_cache* cache);

/* Latent frames decoded since the last reset, or -1 for NULL. */
int64_t fd_kv_cache_position(const fd_kv_cache* cache);

/* fp16 range guard of the 16-bit path with fp16 operands: hidden
 * activations that enter the next GEMM as fp16 (the SwiGLU output of every
 * block and the pixel head's SiLU output) are clamped to +-65504 instead of
 * overflowing to infinity, and the clamped values are counted per cache. The
 * other fp16 operands are bounded by construction (normalised rows, KV-normed
 * keys and values, convex combinations of those values). Writes the number of
 * values clamped since the cache's creation or the previous call and clears
 * it; 0 for the bf16 and fp32 paths. Synchronises the device first. Host
 * pointer `count`; NULL arguments give INVALID_ARGUMENT. */
fd_status fd_kv_cache_fp16_saturations(fd_kv_cache* cache, uint64_t* count);

/* Free a cache (NULL is ignored). No work using it may be in flight. */
void fd_kv_cache_destroy(fd_kv_cache* cache);

/* Shape of the pixels a call of n_frames latent frames produces:
 * [batch, C, n_frames r_t, (H'/p) s_out, (W'/p) s_out]. */
fd_status fd_output_shape(const fd_decoder* dec, int32_t batch, int32_t n_frames,
                          int64_t shape[5]);

/* Decode one chunk (Algorithm 1 for n_frames consecutive latent frames).
 *   latent  device pointer, [batch, C', n_frames, H', W'] contiguous, latent_dtype
 *   n_frames 1..max_frames_per_call, a multiple of unit_frames
 *   out     device pointer, fp32, shape of fd_output_shape(dec, batch, n_frames)
 *   stream  hipStream_t (NULL = default stream)
 * Asynchronous on `stream`: the caller keeps latent and out alive and
 * synchronises before reading out. One call with n_frames frames equals
 * n_frames / unit_frames successive calls with one unit each; outputs of frame
 * t never depend on frames after t. Advances the cache position by n_frames.
 * The cache must not be used by two calls at once. */
fd_status fd_decode_chunk(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                          int32_t n_frames, fd_kv_cache* cache, float* out, void* stream);

/* For callers that cannot allocate device memory while decoding (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * fd_decode_chunk with the call's activation workspace (residual streams,
 * GEMM operands, MLP hidden, per-call RoPE table) taken from a fixed device
 * array of 256 MiB that the library holds once per GPU, instead of the
 * cache's own workspace; the cache still provides the rings and the position.
 * Arguments, layouts, results and asynchrony are those of fd_decode_chunk, bit
 * for bit. It calls no device allocation or free. The first call on a device
 * looks the array's address up (hipGetSymbolAddress) and keeps it; make one
 * call before capturing a graph. A call whose workspace (batch x n_frames
 * x L_frm backbone rows, r_t times as many refinement rows) exceeds the array
 * gives FD_ERR_UNSUPPORTED before any device work (the 480p XL stream fits;
 * the 720p one does not), as does STATE with the event probe enabled on the
 * cache or before static FP8 scales are set. All such calls on one GPU share the
 * array, which keeps the last call's contents (nothing in it has to start at
 * zero): calls that overlap on one GPU race, so order them (one stream, or
 * events). */
fd_status fd_decode_chunk_noalloc(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                                  int32_t n_frames, fd_kv_cache* cache, float* out, void* stream);

/* ------------------------------------------------------------------------
 * Serving: other pixel formats and several streams at once.
 * ------------------------------------------------------------------------ */

/* Pixel formats of fd_decode_chunk_as / fd_decode_chunks. Each pixel is first
 * clamped to [-1, 1] when clamp_output is set, then stored as
 *   FD_PIXELS_F32   fp32;
 *   FD_PIXELS_BF16  bf16, rounded to nearest even;
 *   FD_PIXELS_U8    uint8 = rint(fp32(x * 127.5 + 127.5)), one fp32 rounding of
 *                   the fused multiply-add, ties to even, limited to 0..255
 *                   (so -1 -> 0, 0 -> 128, 1 -> 255; 4x fewer bytes than fp32). */
enum { FD_PIXELS_F32 = 0, FD_PIXELS_BF16 = 1, FD_PIXELS_U8 = 2 };

/* fd_decode_chunk with the pixels in out_format (FD_PIXELS_*): out holds
 * fd_output_shape elements of 4, 2 or 1 bytes. The decode before the pixel
 * store is the same, so an FD_PIXELS_U8 or FD_PIXELS_BF16 call equals the rule
 * above applied to the fp32 pixels of the same call. Unknown formats give
 * INVALID_ARGUMENT. */
fd_status fd_decode_chunk_as(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                             int32_t n_frames, fd_kv_cache* cache, void* out, int32_t out_format,
                             void* stream);

/* Multi-stream serving: one chunk of n_frames frames for each of n independent
 * streams of one decoder, each with its own cache (and so its own position,
 * ring and workspace): caches[i] decodes latents[i] into outs[i] (layouts and
 * rules of fd_decode_chunk_as). The decodes run concurrently, each on a HIP
 * stream owned by its cache (created at the cache's first such call, default
 * priority), after the work already enqueued on `stream`; `stream` waits for
 * all of them, so the call is asynchronous on `stream` like fd_decode_chunk.
 * Each cache's result equals fd_decode_chunk_as on that cache alone. All
 * arguments are checked before any work is enqueued: n >= 1, no NULL, no
 * cache twice, every cache from dec, else INVALID_ARGUMENT / STATE. A cache
 * must not be in use by another call meanwhile. */
fd_status fd_decode_chunks(const fd_decoder* dec, int32_t n, const void* const* latents,
                           int32_t latent_dtype, int32_t n_frames, fd_kv_cache* const* caches,
                           void* const* outs, int32_t out_format, void* stream);

/* ------------------------------------------------------------------------
 * FP8 MLP of the "-Opt" decoder (Sec. 4.6): static activation amplitudes and
 * their calibration.
 * ------------------------------------------------------------------------ */

/* FP8 MLP decoders: the number of activation amplitudes, two per block (the
 * MLP input, then the SwiGLU output), backbone blocks first, then refinement
 * blocks; 0 for other decoders or NULL. */
size_t fd_fp8_act_count(const fd_decoder* dec);

/* FD_MLP_PRECISION_FP8_STATIC: set the static amplitudes amax[count] (host,
 * count = fd_fp8_act_count, each finite and > 0; layout above). The codes of a
 * tensor with amplitude a are e4m3(fp32(x * fp32(448 / a))), its dequantisation
 * scale fp32(a / 448). Synchronous; no decode on this decoder may be in flight.
 * STATE for other decoders, INVALID_ARGUMENT for a wrong count or value. */
fd_status fd_set_fp8_act_amax(fd_decoder* dec, const float* amax, size_t count);

/* Calibration for FD_MLP_PRECISION_FP8_STATIC (also accepted by FP8 decoders):
 * decode one chunk like fd_decode_chunk (fp32 pixels into out, the cache
 * advances) with per-token activation scales, and raise each amax[i] (host,
 * in / out, count = fd_fp8_act_count, finite and >= 0) to the largest |value|
 * of that tensor in this chunk (the fp32 MLP input; the fp16 SwiGLU output).
 * Start from zeros and call it over calibration chunks, then pass the result
 * to fd_set_fp8_act_amax. Blocks until done. Calibrations of one decoder must
 * not overlap. STATE for decoders without an FP8 MLP. */
fd_status fd_calibrate_chunk(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                             int32_t n_frames, fd_kv_cache* cache, float* out, float* amax,
                             size_t count, void* stream);

/* ------------------------------------------------------------------------
 * Diagnostics and kernel-level test hooks. Decoding needs none of these: they
 * expose internal state (the residual stream), time kernel classes inside real
 * decode calls, measure the GPU's sustained MFMA rate, and run single kernels
 * of the FP8 MLP on caller buffers so that tests can check them directly.
 * ------------------------------------------------------------------------ */

/* fd_decode_chunk that also copies the fp32 residual stream into `trace`
 * (device pointer, fp32) after the embedding and after every block: first the
 * backbone ([1 + n_backbone_blocks] x rows x D, rows = batch n_frames L_frm),
 * then, for the temporal-first head, the refinement stream after temporal
 * upsampling and after every refinement block ([1 + n_refine_blocks] x r_t rows
 * x D). trace_elems is the capacity in floats; too small -> INVALID_ARGUMENT. */
fd_status fd_decode_chunk_trace(const fd_decoder* dec, const void* latent, int32_t latent_dtype,
                                int32_t n_frames, fd_kv_cache* cache, float* out, void* stream,
                                float* trace, size_t trace_elems);

/* Number of floats fd_decode_chunk_trace writes for this batch and n_frames. */
size_t fd_trace_elems(const fd_decoder* dec, int32_t batch, int32_t n_frames);

/* Kernel classes for the event probe. FD_KC_ATTENTION_REFINE is the subset of
 * FD_KC_ATTENTION launched by the temporal-refinement stack. */
enum { FD_KC_GEMM = 0, FD_KC_ATTENTION = 1, FD_KC_NORM = 2, FD_KC_QKV_POST = 3,
       FD_KC_EMBED_IN = 4, FD_KC_ATTENTION_REFINE = 5, FD_KC_COUNT = 6 };

/* Event probe for measuring one kernel class inside real decode calls: when
 * enabled on a cache, every launch of that class made by fd_decode_chunk is
 * bracketed by a pair of HIP events on the call's stream. fd_probe_read
 * synchronises on the recorded events and returns the summed device time (ms),
 * the number of launches, and the algorithmic work of those launches (flops
 * for GEMM and attention, bytes moved for the bandwidth passes). Enabling or
 * disabling clears the totals. kernel_class < 0 disables. */
fd_status fd_probe_enable(fd_kv_cache* cache, int32_t kernel_class);
fd_status fd_probe_read(fd_kv_cache* cache, double* total_ms, int64_t* launches,
                        double* work);

/* Sustained dense MFMA throughput of the current device (a measurement aid
 * beside the datasheet peak, which assumes the peak engine clock). Runs two
 * 4-wave workgroups per compute unit, each wave issuing `iters` x 16
 * back-to-back 32x32x16 MFMAs (dtype FD_DTYPE_F16 or FD_DTYPE_BF16) on
 * operands that change every instruction, three launches back to back on
 * `stream` (NULL = default), and times the last with HIP events. Writes the
 * achieved TFLOP/s and the mean shader clock (GHz) of that launch. Blocks until
 * done; allocates and frees its own small device buffers. iters in [1, 10^7],
 * else INVALID_ARGUMENT; HIP failures give DEVICE. */
fd_status fd_measure_mfma_peak(int32_t dtype, int32_t iters, void* stream, double* tflops,
                               double* clock_ghz);

/* LDS read bandwidth of one compute unit (a measurement aid for the GEMM and
 * attention kernels, which read their MFMA operands from LDS): two 8-wave
 * workgroups per compute unit each read 64 KB of LDS with conflict-free
 * 16-byte loads (8 in flight per wave), `iters` rounds, twice back to back on
 * `stream` (NULL = default); the second launch's per-workgroup shader cycles
 * give the bytes per shader clock a compute unit delivers, written with the
 * mean shader clock (GHz). Blocks until done; allocates and frees its own small
 * device buffers. iters in [1, 10^7], else INVALID_ARGUMENT; HIP failures give
 * DEVICE. */
fd_status fd_measure_lds_bandwidth(int32_t iters, void* stream, double* bytes_per_clock_cu,
                                   double* clock_ghz);

/* How far a wave's MFMAs and its vector instructions overlap (a measurement
 * aid for the attention kernel, whose exponentials share the SIMD with its
 * MFMAs): on every compute unit one workgroup with waves_per_simd (1 or 2)
 * waves per SIMD, `iters` iterations of 4 slots on `stream` (NULL = default). A slot is,
 * by mode: 0 one 32x32x16 f16 MFMA; 1 four exponentials (each with a
 * multiply); 2 both; 3 eight fused multiply-adds; 4 MFMA and eight FMAs; 5
 * MFMA, four exponentials and four FMAs; every slot's instructions are
 * independent of the other slots'. cycles[0..5] receive the mean shader cycles
 * per slot and wave. Blocks until done; allocates and frees its own small
 * device buffers. waves_per_simd outside {1, 2} or iters outside [1, 10^7]
 * give INVALID_ARGUMENT; HIP failures give DEVICE. */
fd_status fd_measure_issue_overlap(int32_t waves_per_simd, int32_t iters, void* stream, double* cycles);

/* E4M3 quantisation of rows, the rule the FP8 MLP applies to its weights
 * (FD_MLP_PRECISION_FP8): for each row r of in[rows][cols] (row-major fp32),
 * m = max |in[r][:]|, inv = 448 / m (fp32 division), codes[r][c] = the OCP
 * E4M3 code nearest to fp32(in[r][c] * inv), ties to even, saturating at
 * +-448 (bit layout S.EEEE.MMM, exponent bias 7); scales[r] = m / 448 (fp32),
 * so in ~= decode(codes) * scales. A row of zeros gives codes 0 and scale 1.
 * Host pointers, caller-owned; rows >= 0, cols >= 1, else INVALID_ARGUMENT.
 * NaN or infinite inputs give INVALID_ARGUMENT. */
fd_status fd_quantize_e4m3_rows(const float* in, int64_t rows, int64_t cols, uint8_t* codes,
                                float* scales);

/* The same rule on the GPU (the kernel the FP8 MLP uses for its per-token
 * activation codes), on device pointers in[rows][cols] fp32, codes[rows][cols]
 * bytes and scales[rows] fp32, enqueued on `stream` (NULL = default);
 * asynchronous. cols a multiple of 8 in [8, 65536], rows >= 0, else
 * INVALID_ARGUMENT. */
fd_status fd_quantize_e4m3_rows_device(const float* in, int64_t rows, int64_t cols, uint8_t* codes,
                                       float* scales, void* stream);

/* Packing of an E4M3 weight for fd_gemm_e4m3_device (the layout the FP8 MLP
 * keeps its weights in): w[n][k] (row-major byte codes, host) goes to 1 KB
 * blocks of 16 rows x 64 K-columns, block (n / 16, k / 64) at byte offset
 * ((n / 16) (K / 64) + k / 64) 1024, inside it row n % 16 at 64 (n % 16) and
 * column k % 64; rows up to the next multiple of 16 are zero. packed (host,
 * caller-owned) holds ceil(N / 16) 16 K bytes. N >= 1, K a positive multiple
 * of 64, non-NULL pointers, else INVALID_ARGUMENT. */
fd_status fd_pack_e4m3_weight(const uint8_t* w, int64_t n, int64_t k, uint8_t* packed);

/* Epilogues of fd_gemm_e4m3_device. */
enum {
  /* out is fp32 [M][ld_out]: out[m][c] += C[m][c] for c < N */
  FD_GEMM_E4M3_RESID_ADD = 0,
  /* SwiGLU: W rows interleaved per 32 (rows 64 i .. 64 i + 31 gate, 64 i + 32
   * .. 64 i + 63 up); out is fp16 [M][ld_out]:
   * out[m][32 i + j] = fp16(SiLU(C[m][64 i + j]) C[m][64 i + 32 + j]) */
  FD_GEMM_E4M3_SWIGLU_F16 = 1
};

/* The E4M3 GEMM the FP8 MLP's two projections run on (Sec. 4.6, the "-Opt"
 * decoder's FP8 MLP GEMMs), on the gfx950 FP8 matrix cores:
 *   C[m][n] = (sum_k e4m3(a[m][k]) e4m3(w[n][k])) a_scale[m] w_scale[n] + bias[n]
 * with fp32 accumulation (each product is exact in fp32), then the epilogue.
 * Device pointers: a [M][lda] E4M3 codes (16-byte aligned, lda a multiple of
 * 16, lda >= K), a_scale [M], w_packed as fd_pack_e4m3_weight writes it
 * (16-byte aligned), w_scale [N], bias [N] (fp32), out per the epilogue
 * (SwiGLU: N a multiple of 64, ld_out >= N / 2 and a multiple of 4, out
 * 8-byte aligned; residual add: ld_out >= N). M >= 0, 1 <= N, K a multiple of
 * 64 in [64, 65536], lda and ld_out below 2^20, else INVALID_ARGUMENT.
 * Enqueued on `stream` (NULL = default), asynchronous; a launch failure gives
 * DEVICE. */
fd_status fd_gemm_e4m3_device(const uint8_t* a, int64_t lda, const float* a_scale,
                              const uint8_t* w_packed, const float* w_scale, const float* bias,
                              int32_t m, int32_t n, int32_t k, int32_t epilogue, void* out,
                              int64_t ld_out, void* stream);

const char* fd_status_string(fd_status status);

/* Message of the last failed call on this thread ("" if none). */
const char* fd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLASHDECODER_H */
