/*
 * eas_encoder.h -- C ABI of the MI355X Encode-stage encoder library (libeas.so).
 *
 * What the library computes.  The Encode stage runs a modality encoder and a
 * lightweight connector that map raw images, video clips or audio clips to the
 * embedding vectors the LLM consumes (paper Section 2.1).  The encode worker
 * runs that forward pass on a micro-batch of up to B requests at a time
 * (Section 3.2, load-adaptive micro-batching), and each request's embeddings
 * leave the worker as one contiguous block (Section 3.3, envelope transfer).
 * The encoder families are those of Table 3: a CLIP ViT-L image encoder, a
 * dynamic-resolution ViT for images and video, and a Whisper audio encoder.
 *
 * Conventions shared by every call:
 *   - "device" pointers are HIP device memory on the current device; "host"
 *     pointers are ordinary process memory read or written before the call
 *     returns.
 *   - The caller owns every buffer it passes in (inputs, weights, outputs).
 *     The library owns only the workspace that eas_encoder_create allocates.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device work is enqueued on it and the call returns without waiting;
 *     the caller keeps device buffers alive until the stream has consumed
 *     them.  One handle serves one stream at a time: calls that overlap on
 *     one handle share its workspace and race.
 *   - Every call returns an eas_status.  Argument and shape errors are found
 *     on the host before anything is enqueued: nothing is written and the
 *     handle stays usable.  No C++ exception crosses this boundary.
 *   - Matrices are row-major; "bf16" is IEEE bfloat16 stored as 16 bits.
 *     Linear weights are [out, in].
 */
#ifndef EAS_ENCODER_H
#define EAS_ENCODER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EAS_OK = 0,
  EAS_ERR_INVALID_ARG = 1,  /* NULL pointer, unknown enum, bad config field  */
  EAS_ERR_SHAPE = 2,        /* cu_seqlens / grid_thw / item shape rejected    */
  EAS_ERR_CAPACITY = 3,     /* more tokens or sequences than the handle holds */
  EAS_ERR_UNSUPPORTED = 4,  /* valid but not built (e.g. head_dim 48)          */
  EAS_ERR_HIP = 5           /* a HIP runtime call failed; see eas_last_error  */
} eas_status;

/* Encoder families (Table 3).  VIT_ABS: learned absolute positions;
 * VIT_CLS_ABS: CLS token + learned positions + pre-LN (CLIP style);
 * VIT_ROPE: 2D/3D rotary positions on the (t, h, w) patch grid;
 * WHISPER: two kernel-3 conv1d layers + sinusoid positions. */
enum { EAS_KIND_VIT_ABS = 0, EAS_KIND_VIT_CLS_ABS = 1, EAS_KIND_VIT_ROPE = 2, EAS_KIND_WHISPER = 3 };
enum { EAS_FP32 = 0, EAS_BF16 = 1 };
enum { EAS_ACT_GELU = 0 /* exact erf */, EAS_ACT_QUICKGELU = 1 /* x*sigmoid(1.702x) */ };

/* Largest number of requests (sequences) in one micro-batch. */
#define EAS_MAX_SEQS 64

typedef struct {
  int32_t kind;            /* EAS_KIND_*                                         */
  int32_t dtype;           /* EAS_FP32 or EAS_BF16: weights, packed input and    */
                           /* GEMM operands; accumulation is always fp32 and the */
                           /* residual stream is kept in fp32                    */
  int32_t layers, hidden, heads, head_dim, mlp, act;
  int32_t in_chans, patch, temporal_patch;
  int32_t merge;           /* 1: no merger; 2: 2x2 patch merger (VIT_ABS/ROPE)   */
  int32_t out_dim;         /* merger output width (merge == 2), else hidden      */
  float ln_eps;            /* every encoder LayerNorm                            */
  float merger_ln_eps;     /* the merger's LayerNorm                             */
  float rope_theta;        /* VIT_ROPE: base of the rotary frequencies           */
  int32_t rope_sections[3];/* VIT_ROPE: rotation slots for the t, h, w axes;     */
                           /* they sum to head_dim / 2                           */
  int32_t pos_grid[2];     /* VIT_ABS / VIT_CLS_ABS: h, w of the position table  */
  int32_t n_mels, n_frames;/* WHISPER: mel bins, frames per clip (even)          */
  int64_t max_tokens;      /* workspace capacity: tokens per micro-batch          */
  int32_t max_seqs;        /* requests per micro-batch, 1..EAS_MAX_SEQS           */
  int32_t out_dtype;       /* EAS_FP32 or EAS_BF16 for out_embeddings            */
} eas_config;

typedef struct eas_encoder eas_encoder;   /* opaque, library-owned */

typedef struct {
  char name[48];           /* e.g. "layers.3.qkv.w"                              */
  int64_t offset_bytes;    /* from the start of the flat weight buffer (256-B aligned) */
  int32_t ndim;            /* 1 or 2                                             */
  int64_t shape[2];
} eas_tensor_desc;

/* Not from the paper (library plumbing): the handle of one encoder.
 * Validates *cfg and allocates the workspace for cfg->max_tokens tokens and
 * cfg->max_seqs requests on the current device.  *out receives the handle.
 * Errors: INVALID_ARG (NULL, inconsistent fields), UNSUPPORTED (a head_dim or
 * width the kernels are not built for), HIP (allocation failed). */
eas_status eas_encoder_create(const eas_config* cfg, eas_encoder** out);

/* Not from the paper (library plumbing).  Waits for the handle's own pending
 * work -- its last eas_encode_microbatch call on the caller's stream and its
 * second stream, not the whole device -- and frees its workspace.  NULL-safe. */
void eas_encoder_destroy(eas_encoder* enc);

/* Not from the paper (the paper names the encoders but not their weights).
 * Canonical layout of the flat weight buffer for *cfg: one descriptor per
 * tensor, in order -- the embedding (patch.w [hidden, C*tp*p*p] and patch.b,
 * or conv1.w [hidden, n_mels*3], conv1.b, conv2.w [hidden, hidden*3],
 * conv2.b, both flattened in (channel, tap) order), then cls, pos and
 * ln_pre.{g,b} where the kind has them, then per layer ln1.{g,b},
 * qkv.w [3*hidden, hidden] (q, k, v blocks, heads contiguous inside each),
 * qkv.b, o.w, o.b, ln2.{g,b}, fc1.w [mlp, hidden], fc1.b, fc2.w, fc2.b, then
 * ln_q.{g,b}, m1.w [4h, 4h], m1.b, m2.w [out_dim, 4h], m2.b (merge == 2) or
 * ln_post.{g,b} (WHISPER).  Elements are cfg->dtype.  Pass descs == NULL to
 * query the count.  Host only; no HIP calls. */
eas_status eas_weights_layout(const eas_config* cfg, eas_tensor_desc* descs, int32_t capacity,
                              int32_t* n_descs, int64_t* total_bytes);

/* Not from the paper (shape rules of the packed format below).
 * Shape of a micro-batch before it is packed (host only, no HIP calls).
 * tchw: host [n_req, 4] = (frames, channels, height, width) per request; for
 * WHISPER (1, 1, n_mels, n_frames).  Writes cu_seqlens (host [n_req+1]: the
 * prefix sums of the per-request token counts, a CLS token included),
 * grid_thw (host [n_req, 3] patch grid; may be NULL), *packed_elems (elements
 * of the packed input) and *out_rows (rows of out_embeddings). */
eas_status eas_microbatch_shape(const eas_config* cfg, int32_t n_req, const int32_t* tchw,
                                int32_t* cu_seqlens, int32_t* grid_thw, int64_t* packed_elems,
                                int64_t* out_rows);

/* Not from the paper (argument checking).
 * Checks a packed micro-batch description against *cfg (host only, no HIP
 * calls): 1 <= n_seqs <= max_seqs, cu_seqlens[0] == 0, strictly increasing,
 * cu_seqlens[n_seqs] <= max_tokens; per request the token count matches its
 * grid (t*h*w, +1 for the CLS token; n_frames/2 for WHISPER), h and w are even
 * under the 2x2 merger and fit the learned position table.  grid_thw may be
 * NULL only for WHISPER. */
eas_status eas_validate_microbatch(const eas_config* cfg, const int32_t* cu_seqlens,
                                   const int32_t* grid_thw, int32_t n_seqs);

/* Micro-batch packer (Section 3.2: the encode worker runs a micro-batch of
 * up to B queued requests as one encoder pass): concatenates requests
 * without padding.
 * items: host array of n_req device pointers to fp32 inputs -- images and
 * clips [frames, C, H, W], audio [n_mels, n_frames]; tchw as in
 * eas_microbatch_shape.  packed (device, cfg->dtype): vision [N, C*tp*p*p]
 * patch rows in storage order -- merge-window order (the 4 tokens of each 2x2
 * window consecutive) when merge == 2, raster order otherwise, with one zero
 * row reserved for the CLS token at the start of each CLS-model request; the
 * row of patch (ti, hi, wi) holds pixel[ti*tp + tau, c, hi*p + dy, wi*p + dx]
 * at index ((c*tp + tau)*p + dy)*p + dx.  Audio: [n_req, n_frames, n_mels]
 * (time-major).  cu_seqlens / grid_thw (host) receive what
 * eas_microbatch_shape gives. */
eas_status eas_pack_microbatch(eas_encoder* enc, int32_t n_req, const float* const* items,
                               const int32_t* tchw, void* packed, int32_t* cu_seqlens,
                               int32_t* grid_thw, void* stream);

/* The Encode forward pass on one packed micro-batch: the encoder and
 * connector that turn a request's raw input into the embeddings the LLM
 * consumes (Section 2.1), run on one micro-batch (Section 3.2); each
 * request's rows leave as one contiguous block (Section 3.3).
 * packed_in (device, cfg->dtype): as written by eas_pack_microbatch.
 * cu_seqlens (host [n_seqs+1]), grid_thw (host [n_seqs, 3]; NULL for WHISPER).
 * weights (device): flat buffer laid out by eas_weights_layout.
 * out_embeddings (device, cfg->out_dtype): [sum of output rows, out_dim], each
 * request's rows contiguous and in request order -- L_r/4 rows with the 2x2
 * merger, L_r rows otherwise (all 577 CLIP tokens, CLS first).
 * cu_out (host [n_seqs+1], may be NULL): prefix sums of the output rows.
 * Attention is full within each request and never crosses requests; each
 * request's output does not depend on the other requests in the batch.
 * A micro-batch of 8192 tokens or more (not while profiling) is run as two
 * halves split by tokens: the first on `stream`, the second on a stream the
 * handle owns, forked from and joined back into `stream` by events, so work
 * enqueued on `stream` afterwards sees the whole result.  Per-request bits do
 * not change with the split. */
eas_status eas_encode_microbatch(eas_encoder* enc, const void* packed_in, const int32_t* cu_seqlens,
                                 const int32_t* grid_thw, int32_t n_seqs, const void* weights,
                                 void* out_embeddings, int32_t* cu_out, void* stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * Encode pass as eas_encode_microbatch, with the same arguments except that
 * *cfg takes the place of a handle: no eas_encoder_create, and the call makes
 * no hipMalloc / hipFree and no other allocating call.  Its per-token
 * workspace lives in a fixed device array of EAS_NOALLOC_SCRATCH_BYTES that
 * the library holds on every device it runs on until the process ends.
 * A micro-batch whose workspace does not fit is refused with
 * EAS_ERR_CAPACITY before anything is enqueued (256 MiB holds about 11,800
 * CLIP ViT-L tokens, 9,400 Qwen-style ViT tokens -- one 1344 x 1344 image --
 * or six Whisper-large clips).  The micro-batch always runs as one pass on
 * `stream` (no second stream), and profiling does not apply.  Every call on a
 * device shares that device's array and leaves its contents behind; no
 * buffer in it needs to start at zero (every kernel writes what it later
 * reads).  Calls that overlap on one device -- on different streams, or from
 * different threads -- race on the array: the caller orders them.  The
 * output bits equal eas_encode_microbatch's for the same inputs.
 * Errors as eas_encode_microbatch (no handle, so no eas_last_error detail);
 * EAS_ERR_HIP if the array's device address cannot be looked up. */
#define EAS_NOALLOC_SCRATCH_BYTES (256u << 20)
eas_status eas_encode_microbatch_noalloc(const eas_config* cfg, const void* packed_in, const int32_t* cu_seqlens,
                                         const int32_t* grid_thw, int32_t n_seqs, const void* weights,
                                         void* out_embeddings, int32_t* cu_out, void* stream);

/* Not from the paper (measurement).  Kernel timing: while enabled, every
 * launch the handle makes is bracketed by HIP events on its stream.  eas_profile_read waits for the
 * recorded events and returns, per kernel, the number of launches, the summed
 * event time (ms), and the summed algorithmic flops and HBM bytes of those
 * launches; it then clears the record.  Pass stats == NULL to query the count. */
typedef struct {
  char kernel[64];
  int64_t launches;
  double total_ms;
  double flops;
  double bytes;
} eas_kernel_stat;

eas_status eas_profile_enable(eas_encoder* enc, int32_t enable);
eas_status eas_profile_read(eas_encoder* enc, eas_kernel_stat* stats, int32_t capacity, int32_t* n_stats);

/* Not from the paper (measurement).  MFMA issue rate with no memory traffic:
 * one workgroup per CU runs iters x 32 back-to-back v_mfma_f32_32x32x16_bf16 on
 * operands held in registers -- random finite bf16 values, or all zero when
 * zero_operands != 0 -- after one warm-up launch, timed with HIP events on
 * `stream` (synchronised before return).  *tflops: dense bf16 TFLOP/s of the
 * timed launch.  On random operands the board's power limit, not the clock,
 * sets the rate; the gap to the zero-operand rate is what the limit takes from
 * MFMA-bound kernels.  Allocates and frees a small device buffer.  Returns
 * EAS_ERR_INVALID_ARG for a NULL tflops or iters outside [1, 2^20], EAS_ERR_HIP
 * on a failed HIP call. */
eas_status eas_mfma_rate_probe(int32_t zero_operands, int32_t iters, double* tflops, void* stream);

const char* eas_status_string(eas_status s);
/* Detail of the last failing call on this handle ("" if none; NULL-safe). */
const char* eas_last_error(const eas_encoder* enc);

#ifdef __cplusplus
}
#endif
#endif /* EAS_ENCODER_H */
