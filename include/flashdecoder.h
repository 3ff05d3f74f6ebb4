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
 *   - Nothing is enqueued and no state changes when a call returns a status
 *     other than FD_OK; fd_last_error() then holds a message (thread-local).
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

/* Check a config. FD_OK, FD_ERR_INVALID_ARGUMENT (inconsistent values) or
 * FD_ERR_UNSUPPORTED (e.g. a 16-bit compute type with D_h != 64). Host only. */
fd_status fd_config_validate(const fd_config* cfg);

/* Canonical weight layout: all tensors concatenated in this order (row-major):
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

/* Create a decoder on the current HIP device: validates cfg, copies the weight
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

const char* fd_status_string(fd_status status);

/* Message of the last failed call on this thread ("" if none). */
const char* fd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLASHDECODER_H */
