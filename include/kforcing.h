/*
 * kforcing.h -- C ABI of the MI355X (gfx950) K-Forcing decode library.
 *
 * K-Forcing (paper Sec. 3.1) learns a push-forward map
 *     G_theta : V^t x [0,1]^k -> V^k
 * that turns a context and k i.i.d. uniform noise variables into the next k
 * tokens in one forward pass.  This library runs the inference procedure of
 * Appendix C.1 ("K-Forcing Inference with KV Cache"): a prefill over the
 * prompt plus k noise rows, then decode blocks that each feed the k tokens
 * emitted by the previous block plus k fresh noise rows, keep only the real
 * tokens' K/V, and take the argmax of the head over the last k outputs.  An
 * ordinary autoregressive (k = 1, inverse-CDF) path on the same backbone is
 * included as the baseline the paper compares against (Sec. 4, Table 1).
 *
 * Conventions for every entry point:
 *   - Return 0 (KF_OK) or a negative KF_E* code.  On an error nothing is
 *     launched and the context's state is unchanged; kf_last_error() gives a
 *     message.  No C++ exception crosses this boundary.
 *   - Array arguments are DEVICE pointers unless stated otherwise, and all
 *     work is enqueued asynchronously on the stream given to kf_create();
 *     outputs are valid once that stream has been synchronised.
 *   - The caller owns every buffer it passes (state, inputs, outputs); the
 *     library never allocates or frees device memory.
 *   - A context is bound to one stream and is not thread-safe.
 *   - Matrices are row-major; token ids are int32; noise values are fp32 in
 *     [0, 1).
 */
#ifndef KFORCING_H
#define KFORCING_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ error codes */
#define KF_OK 0
#define KF_EINVAL (-1) /* bad argument: k < 1, k > max_k, B out of range, null pointer, L % k != 0 ... */
#define KF_ESTATE (-2) /* no state bound, no weights loaded, decode before prefill, B mismatch */
#define KF_ECTX (-3)   /* the step would run past n_ctx positions */
#define KF_ENOMEM (-4) /* out of memory: the bound state buffer is smaller than
                          * kf_state_bytes(), the serving KV page pool cannot cover
                          * a call, or kf_create could not allocate the context */
#define KF_EHIP (-5)   /* a HIP runtime call failed (message from hipGetErrorString) */

/* ---------------------------------------------------------- configuration */
#define KF_FP32 0 /* weights, activations and KV cache in fp32 */
#define KF_BF16 1 /* weights, GEMM inputs and KV cache in bf16; fp32 accumulation,
                     fp32 residual stream, fp32 noise sinusoid */

#define KF_FLAG_DEBUG_LOGITS 1u /* reserve room for, and record, the fp32 head logits of
                                   the most recent step (kf_debug_logits) */
#define KF_FLAG_TEACHER 4u      /* reserve the sampling-head workspace of kf_teacher_targets
                                   (min(max_batch * max_prompt, 8192) rows x (Vpad / 128) x
                                   36 bytes) */
#define KF_FLAG_ROLLOUT 8u      /* reserve the workspace of kf_selfforcing_targets: residual
                                   rows for 2 * max_batch * max_prompt * max_k rows and
                                   n_layer x 2 x max_batch x n_head x max_prompt (1 + 2 max_k)
                                   x d_head elements of keys and values */
#define KF_FLAG_RMS_ROPE 16u    /* the paper's backbone (Appendix D model table): RMSNorm
                                   pre-norm and rotary positions (RoFormer pairs (2i, 2i+1)
                                   over d_rot = min(64, d_head), angle p 10000^(-2i/d_rot)),
                                   no learned positions; the blob has header word 9 bit 1
                                   set and still carries the position table and the norm
                                   shifts, which are ignored */
#define KF_FLAG_SERVING 32u     /* continuous batching over a paged KV cache: the
                                   kf_serve_* calls, a page table and per-slot state */
#define KF_FLAG_TEMPERATURE 2u  /* the model has a temperature-conditioned noise encoder
                                   (its weight blob carries the encoder, header word 9 bit 0);
                                   see kf_set_temperature */

typedef struct kf_config {
  int n_layer;    /* Transformer blocks */
  int d_model;    /* hidden size d; multiple of 64 */
  int n_head;     /* heads H; d_model / n_head must be 32, 64 or 128 */
  int d_mlp;      /* MLP hidden size; multiple of 64 */
  int vocab;      /* vocabulary size V (any value >= 2) */
  int n_ctx;      /* positions (learned position table length, KV capacity); multiple of 8 */
  int dtype;      /* KF_FP32 or KF_BF16 */
  int max_batch;  /* largest B any call may use */
  int max_k;      /* largest window k any call may use (k <= max_k) */
  int max_prompt; /* longest prompt N given to a prefill call */
  unsigned flags; /* KF_FLAG_* */
  int kv_pages;   /* KV pool size in pages of 128 positions (KF_FLAG_SERVING only);
                     0 = max_batch * ceil(n_ctx / 128), every slot can reach n_ctx */
} kf_config;
/* A config is also rejected when the rows of its largest step,
 * max_batch * (max(max_prompt, max_k) + max_k), times max(d_mlp, 4 d_model)
 * compute-dtype elements (or times d_model fp32 elements) reach 2 GiB: the
 * GEMMs address their operands with 32-bit byte ranges. */

/* Opaque per-stream context. */
typedef struct kf_ctx kf_ctx;

/* Validate cfg and create a context bound to hip_stream (a hipStream_t; NULL
 * is the default stream).  Touches no device.  *out is set on success. */
int kf_create(const kf_config *cfg, void *hip_stream, kf_ctx **out);

/* Device bytes the caller must provide for cfg: packed weights, the KV cache
 * and the workspace.  The KV cache is a pool of pages of 128 positions of one
 * sequence, each [n_layer][K,V][n_head][128 * d_head] compute-dtype elements
 * (keys slot-major, values transposed); the pool holds kv_pages pages, or
 * max_batch * ceil(n_ctx / 128) when kv_pages is 0.  Returns 0 for an invalid
 * cfg. */
size_t kf_state_bytes(const kf_config *cfg);

/* Hand the context a device buffer of at least kf_state_bytes() bytes,
 * 256-byte aligned.  Re-binding discards weights and sequence state. */
int kf_bind_state(kf_ctx *ctx, void *dev_ptr, size_t bytes);

/* Load the weights of the model the paper's model table defines (Appendix D:
 * a causal Transformer backbone, its token and position embeddings, the
 * noise encoder -- a sinusoid of u and a two-layer GELU MLP -- and, for a
 * temperature-conditioned model, the temperature encoder; the head is tied
 * to the token table) from a flat blob: 16 int32 header words (magic 0x4B465731,
 * version 1, n_layer, d_model, n_head, d_mlp, vocab, n_ctx, dtype, 7 zero
 * words) followed by every tensor as fp32 in a fixed order: token table
 * [V][d] (also the tied output head), position table [n_ctx][d], noise MLP
 * W1 [4d][d], b1 [4d], W2 [d][4d], b2 [d], then per layer: ln1 gain, ln1
 * shift [d], W_qkv [3d][d], b_qkv [3d], W_o [d][d], b_o [d], ln2 gain, ln2
 * shift [d], W_1 [d_mlp][d], b_1 [d_mlp], W_2 [d][d_mlp], b_2 [d]; finally
 * the final-norm gain and shift [d]; with KF_FLAG_TEMPERATURE, then the
 * temperature encoder W_t1 [d][d], b_t1 [d], W_t2 [d][d], b_t2 [d].  Matrices
 * are [out][in].  For KF_BF16 the 2-D tensors are rounded to bf16 (round to
 * nearest even) on load.
 * blob_is_device: 0 = host pointer (copied synchronously), 1 = device
 * pointer (converted on the stream).  The header must match the config. */
int kf_load_weights(kf_ctx *ctx, const void *blob, size_t bytes, int blob_is_device);

/* First step of Appendix C.1: for each of the B sequences, the N prompt
 * tokens (prompt [B][N], positions 0..N-1) followed by k noise rows
 * (noise [B][k], positions N..N+k-1), one causal forward pass, argmax of the
 * head over the k noise rows -> out [B][k] (positions N..N+k-1).  Commits the
 * prompt's K/V (context length C = N) and keeps out as the pending block.
 * 0 <= N <= max_prompt, 1 <= k <= max_k, N + k <= n_ctx.  Token ids outside
 * [0, V) are replaced by 0 and flagged (kf_device_errors). */
int kf_prefill(kf_ctx *ctx, int B, int N, const int32_t *prompt, int k, const float *noise,
               int32_t *out);

/* One decode block (Appendix C.1): the pending tokens from the previous step
 * (positions C..C+p-1) plus k noise rows (noise [B][k], positions
 * C+p..C+p+k-1) attend causally over the cached context; the argmax of the
 * head over the k noise rows -> out [B][k].  The pending tokens' K/V are
 * committed (C += p), the noise K/V are dropped, out becomes pending.
 * B must equal the prefill's B; k may change between calls; C+p+k <= n_ctx. */
int kf_decode_block(kf_ctx *ctx, int B, int k, const float *noise, int32_t *out);

/* kf_decode_block for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same decode block, bit for bit, with the step's partial results -- the
 * attention key-split states, the split-K parts and the head's per-tile
 * argmax partials -- held in a device array of the library instead of the
 * state buffer's workspace.  The array is KF_NOALLOC_SCRATCH_BYTES (about
 * 20 MiB), one copy per GPU the library runs on, kept until the process ends;
 * its address is looked up once per GPU by kf_bind_state.  The call allocates
 * nothing and needs nothing cleared (every partial result is written before it
 * is read within the call).  Every call on one GPU shares that GPU's copy:
 * calls that overlap on one GPU (several contexts or streams at once) race
 * and must be serialised by the caller.
 * Returns what kf_decode_block returns, plus KF_EINVAL when B * k *
 * ceil(V / 128) exceeds KF_NOALLOC_HEAD_ENTRIES, and KF_EHIP when the array's
 * address could not be found for the state buffer's GPU. */
#define KF_NOALLOC_ATTN_ENTRIES 8192        /* attention key-split states, d_head <= 128 */
#define KF_NOALLOC_SPLIT_BYTES (8u << 20)   /* split-K fp32 parts */
#define KF_NOALLOC_HEAD_ENTRIES (1u << 20)  /* head argmax partials (value and index each) */
#define KF_NOALLOC_SCRATCH_BYTES \
  ((size_t)KF_NOALLOC_ATTN_ENTRIES * (2 + 128) * 4 + KF_NOALLOC_SPLIT_BYTES + \
   (size_t)KF_NOALLOC_HEAD_ENTRIES * 8)
int kf_decode_block_noalloc(kf_ctx *ctx, int B, int k, const float *noise, int32_t *out);

/* The whole of Appendix C.1's algorithm "K-Forcing Inference with KV Cache"
 * (its REQUIRE: prompt x_1..x_N, window k, generation length; its ENSURE: the
 * generated tokens): generate L new tokens per sequence (L % k == 0,
 * N + L <= n_ctx) as one prefill and L/k - 1 decode blocks, with noise drawn on the device by
 * Philox4x32-10 (key = seed, counter = (emitted position, sequence, 2, 0),
 * u = (word0 >> 8) * 2^-24).  out [B][L] holds positions N..N+L-1.  Leaves
 * the context decoded up to the last block (pending = last k tokens).
 * L == 0 launches nothing. */
int kf_generate(kf_ctx *ctx, int B, int N, const int32_t *prompt, int L, int k, uint64_t seed,
                int32_t *out);

/* Temperature-controlled generation (Sec. 3.3; Appendix C.2, temperature
 * control at inference): tau [B] (device memory, read during the call) sets the
 * temperature of sequences 0..B-1.  Each tau goes through the noise sinusoid
 * and the encoder's Linear(d, d), GELU, Linear(d, d); the resulting vector is
 * added to every later noise row of that sequence until the next call (the
 * weights are reloaded, or the temperature is set again).  Requires
 * KF_FLAG_TEMPERATURE (else KF_ESTATE) and loaded weights; 1 <= B <= max_batch.
 * With the flag, kf_prefill, kf_decode_block and kf_generate for B sequences
 * return KF_ESTATE until the temperature of at least B sequences is set; the
 * AR calls have no noise rows and do not need it. */
int kf_set_temperature(kf_ctx *ctx, const float *tau, int B);

/* Autoregressive baseline (the AR teacher's decoding, Sec. 4; inverse-CDF map
 * of Appendix B: the smallest token id m with F_m > u, F the CDF of the
 * softmax in token-id order).  Prefill: prompt rows only (N >= 1), the head
 * on the last prompt row, u [B] -> out [B] (position N).  C = N. */
int kf_prefill_ar(kf_ctx *ctx, int B, int N, const int32_t *prompt, const float *u, int32_t *out);

/* One AR step: the pending tokens as real rows, head on the last of them,
 * inverse CDF with u [B] -> out [B]; commits the pending tokens. */
int kf_decode_ar(kf_ctx *ctx, int B, const float *u, int32_t *out);

/* AR generation of L >= 0 tokens with device Philox noise (same stream as
 * kf_generate, so position p uses the same u for every method). */
int kf_generate_ar(kf_ctx *ctx, int B, int N, const int32_t *prompt, int L, uint64_t seed,
                   int32_t *out);

/* Copy the fp32 head logits of the most recent step to out (device,
 * rows x V floats; rows = B*k for a K-Forcing step, B for an AR step).
 * n_floats is the capacity of out.  Requires KF_FLAG_DEBUG_LOGITS. */
int kf_debug_logits(kf_ctx *ctx, float *out, size_t n_floats);

/* Fill out [B][n] with the device generator's u for positions p0..p0+n-1. */
int kf_fill_noise(kf_ctx *ctx, uint64_t seed, int B, int p0, int n, float *out);

/* Replay the decode blocks of kf_generate / kf_generate_ar as one captured
 * HIP graph per argument set (default on).  Every launch of a decode block
 * reads the context length from device memory, so a captured block replays
 * unchanged; the instantiated graph is kept on the context until the
 * arguments, the state buffer or the weights change.  kf_serve_step likewise
 * replays one graph per (sequences, pending count, k), up to 16 of them, with
 * noise and tokens copied through fixed device buffers around the replay.
 * Used only on a non-null stream and while kernel timing is off; results are
 * identical either way. */
int kf_set_graphs(kf_ctx *ctx, int enable);

/* Host view of the sequence state: committed length C, pending count, B. */
int kf_get_state(const kf_ctx *ctx, int *C, int *pending, int *B);

/* Synchronise the stream and return the device-side error flags (bit 0: a
 * token id outside [0, V) was replaced by 0; bit 1: kf_teacher_targets met a
 * temperature outside (0, inf)), then clear them. */
int kf_device_errors(kf_ctx *ctx, int *flags);

/* Distillation targets of the Stage-1 AR teacher (Appendix C.2, forward
 * distillation algorithm, teacher lines): the loaded model runs as an
 * autoregressive teacher, one causal pass over tokens [B][N] (positions
 * 0..N-1), and for every (b, p)
 *     targets[b][p] = smallest m with F_m > u[b][p],
 * F the CDF of softmax(l_{b,p} / tau[b]) over the vocabulary, l_{b,p} the head
 * logits at position p (the teacher's distribution of the token after
 * tokens[b][0..p]).  The inverse CDF is the strict convention of the AR
 * sampler; if rounding leaves F_V <= u it returns the last token with
 * q > 0.  The logits never reach HBM: the head GEMM keeps per-tile maxima and
 * 16-column sums of exp(l / tau) and a selection kernel recomputes only the
 * 16 logits around the crossing point.
 *   tokens int32 [B][N], tau fp32 [B] (> 0), u fp32 [B][N] in [0, 1),
 *   targets int32 [B][N]: device pointers owned by the caller.
 *   Requires KF_FLAG_TEACHER; 1 <= B <= max_batch, 1 <= N <= max_prompt.
 *   A tau outside (0, inf) sets device error bit 1 (kf_device_errors) and
 *   gives target 0 for that sequence's rows.  Token ids outside [0, V) are
 *   replaced by 0 (error bit 0), as in a prefill.
 *   The pass uses the KV cache: any generation in progress ends (a later
 *   decode needs a new prefill).  With KF_FLAG_DEBUG_LOGITS the fp32 logits
 *   of the last head chunk (rows ((B*N - 1) / 8192) * 8192 .. B*N - 1) are
 *   kept for kf_debug_logits. */
int kf_teacher_targets(kf_ctx *ctx, int B, int N, const int32_t *tokens, const float *tau,
                       const float *u, int32_t *targets);

/* Stage-2 self-forcing targets (Appendix C.2, self-forcing distillation, the
 * teacher's lines): the loaded K-Forcing model is the teacher with window k.
 * Round 1 is one SingleForward pass over the N context tokens and, after
 * each context position t = 0..N-1, k noise rows z1[b][t][0..k) (noise j of
 * group t at position t + 1 + j, the position of the token it stands for);
 * x1[b][t][j] is the argmax of noise row (t, j).  Round 2 is one
 * DoubleForward pass: Future-1 rows carry x1 as tokens (positions t + 1 + j),
 * Future-2 rows carry the noise z2 (positions t + 1 + k + j), both attending
 * to round 1's context keys under M_D; x2[b][t][j] is the argmax of Future-2
 * row (t, j).  The 2k targets of context position t are [x1[b][t] ; x2[b][t]].
 *   tokens int32 [B][N]; z1, z2 fp32 [B][N][k] in [0, 1); x1, x2 int32
 *   [B][N][k]: device pointers owned by the caller.
 *   Requires KF_FLAG_ROLLOUT and a bf16 model; 1 <= B <= max_batch,
 *   1 <= N <= max_prompt, 1 <= k <= max_k, N + 2k <= n_ctx (else KF_ECTX).
 *   A temperature-conditioned model uses the temperatures of
 *   kf_set_temperature for both rounds.  The call ends any generation in
 *   progress.  With KF_FLAG_DEBUG_LOGITS, the fp32 logits of the Future-2
 *   rows (B*N*k rows, in x2 order) are kept for kf_debug_logits. */
int kf_selfforcing_targets(kf_ctx *ctx, int B, int N, int k, const int32_t *tokens,
                           const float *z1, const float *z2, int32_t *x1, int32_t *x2);

/* Per-kernel timing with HIP events on the context's stream.  kf_set_timing
 * takes a bit mask over the kernel classes below (bit c = class c; 0 turns
 * timing off; KF_TIMING_ALL brackets every class) and clears earlier records.
 * While a class is selected, each of its launches is bracketed by an event
 * pair.  kf_kernel_time() synchronises and returns the summed milliseconds
 * and the launch count of one class since timing was last set. */
#define KF_KC_EMBED 0    /* real-row embedding (in kf_generate also the noise rows' position add) */
#define KF_KC_NOISE 1    /* noise sinusoid + noise-MLP GEMMs + position add (kf_generate: the
                            sinusoids and GEMMs of whole chunks of passes, computed ahead) */
#define KF_KC_NORM 2     /* standalone LayerNorm (none: every LayerNorm is folded into the GEMM that consumes it) */
#define KF_KC_QKV 3      /* LayerNorm-folded QKV GEMM with KV append */
#define KF_KC_ATTN 4     /* block attention */
#define KF_KC_OPROJ 5    /* attention-out GEMM + residual */
#define KF_KC_MLP_UP 6   /* LayerNorm-folded MLP up GEMM + GELU */
#define KF_KC_MLP_DOWN 7 /* MLP down GEMM + residual */
#define KF_KC_HEAD 8     /* final-LayerNorm-folded head GEMM with argmax partials / logits
                            (the argmax head also commits the step: C += real rows) */
#define KF_KC_SELECT 9   /* argmax reduction, or the AR baseline's inverse-CDF sampler and commit */
#define KF_KC_COUNT 10
#define KF_TIMING_ALL ((1 << KF_KC_COUNT) - 1)
int kf_set_timing(kf_ctx *ctx, int class_mask);
int kf_kernel_time(kf_ctx *ctx, int kernel_class, double *total_ms, int *launches);

/* ------------------------------------------- attention of the training masks
 * Block-sparse attention under the masks that train K-Forcing (Appendix C.2),
 * for N context tokens and k tokens per context position, 0-based group
 * t = 0..N-1 and in-group index j = 0..k-1:
 *   KF_MASK_SINGLE (SingleForward M_S): queries = keys = [context N | noise N*k];
 *     context row i sees context 0..i; noise row N + t*k + j sees context
 *     0..t and noise N + t*k .. N + t*k + j.
 *   KF_MASK_DOUBLE (DoubleForward M_D, its Future-1 and Future-2 query rows):
 *     queries [F1 N*k | F2 N*k], keys [context N | F1 N*k | F2 N*k];
 *     F1 row t*k + j sees context 0..t and F1 keys of group t up to j;
 *     F2 row N*k + t*k + j sees context 0..t, all k F1 keys of group t and F2
 *     keys of group t up to j.
 * O = softmax(scale * Q K^T + mask) V per (sequence, head), fp32 softmax.
 *   Q, O: bf16 [B][H][rows][d_head]; K, V: bf16 [B][H][keys][d_head]; device
 *   pointers, 16-byte aligned, owned by the caller; O must not overlap the
 *   inputs.  rows = N + N*k (single) or 2*N*k (double); keys = N + N*k
 *   (single) or N + 2*N*k (double).  d_head in {32, 64, 128}.
 *   Work is enqueued on hip_stream (null: the default stream); nothing is
 *   allocated.  B, H or N equal to 0 is an empty problem (KF_OK, nothing
 *   launched, pointers unchecked).
 * Returns KF_EINVAL for an unknown mask, k < 1, a negative size, an unsupported
 * d_head, a non-finite scale, a null or misaligned pointer, or a problem whose
 * per-head element count or workgroup count reaches 2^31; KF_EHIP when the
 * launch fails.  There is no context, hence no kf_last_error() message. */
#define KF_MASK_SINGLE 0
#define KF_MASK_DOUBLE 1
int kf_training_attention(void *hip_stream, int mask, int B, int H, int N, int k, int d_head,
                          const void *Q, const void *K, const void *V, void *O, float scale);

/* ----------------------------------------------------- continuous batching
 * Serving of independent sequences that start and end at different steps
 * (the decode of Appendix C.1 per sequence, batched): a context created with
 * KF_FLAG_SERVING has max_batch sequence slots, each with its own committed
 * length C and pending tokens, over a pool of KV pages (kv_pages) handed out
 * as sequences grow and returned when they are released.  Every sequence
 * computes exactly what kf_prefill / kf_decode_block compute for it alone.
 * Slot lists are host arrays of distinct ids in [0, max_batch); the row order
 * of prompts, noise and out follows the list.  Calls of this group end a
 * lock-step generation in progress; the lock-step calls (kf_prefill,
 * kf_generate, the AR calls, kf_teacher_targets) release every slot.
 * A temperature-conditioned model uses the temperature of each slot's index
 * (kf_set_temperature sets slots 0..B-1).
 *
 * kf_serve_admit: start n sequences in free slots: prompt rows prompts [n][N]
 * (device, positions 0..N-1) and k noise rows noise [n][k] (device), one
 * causal pass, argmax tokens -> out [n][k] (device), pending; C = N.
 * 0 <= N <= max_prompt, 1 <= k <= max_k, N + k <= n_ctx (else KF_ECTX).
 * KF_ESTATE if a slot is in use; KF_ENOMEM (nothing changes) if the pool
 * lacks the ceil((N + k) / 128) pages per sequence.
 *
 * kf_serve_step: one decode block for the n listed slots, which must hold
 * sequences with equal pending counts p: pending tokens at positions
 * C..C+p-1 and noise [n][k] rows after them; out [n][k] becomes the slots'
 * pending tokens and C += p.  Per slot C + p + k <= n_ctx (else KF_ECTX);
 * KF_ENOMEM (nothing changes) when the pool cannot cover positions
 * 0..C+p+k-1 of every listed slot.  Slots not listed are untouched.
 *
 * kf_serve_release: end the sequences in the listed slots and return their
 * pages (KF_ESTATE, nothing changes, if one holds no sequence).
 *
 * kf_serve_state: C, pending count and pages of a slot (C = -1 if free).
 * kf_serve_pages: free and total pages of the pool. */
int kf_serve_admit(kf_ctx *ctx, int n, const int32_t *slots, int N, const int32_t *prompts, int k,
                   const float *noise, int32_t *out);
int kf_serve_step(kf_ctx *ctx, int n, const int32_t *slots, int k, const float *noise,
                  int32_t *out);
int kf_serve_release(kf_ctx *ctx, int n, const int32_t *slots);
int kf_serve_state(const kf_ctx *ctx, int slot, int *C, int *pending, int *pages);
int kf_serve_pages(const kf_ctx *ctx, int *free_pages, int *total);

/* Release host resources (device memory belongs to the caller). */
void kf_destroy(kf_ctx *ctx);

/* Last error message of ctx ("" if none); kf_strerror names a code. */
const char *kf_last_error(const kf_ctx *ctx);
const char *kf_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* KFORCING_H */
