/*
 * fp.h -- C ABI of the MI355X fingerprint forward pass.
 *
 * A fingerprint (iServe, arXiv 2501.13111, Sec. 1 and Sec. 5.1, Fig. 2) is an
 * LLM cut down to a few hidden layers that keep the architecture's components.
 * iServe's Profiler deploys it and sends dummy requests to measure the time to
 * first token and the time per output token (Sec. 4.2, Sec. 5.3, Eq. 1):
 * a prefill over the prompt, then one KV-cached decode step per output token.
 * This library runs that forward pass for Llama-style decoder layers on one
 * gfx950 GPU under the compression settings the paper searches over
 * (Sec. 3.2, Table A.1): bf16 weights, int8 per-channel or int4 group-128
 * weight-only quantisation, and a bf16 or int8 KV cache.
 *
 * Conventions shared by every call:
 *  - Device pointers are HIP device addresses; host pointers are plain host
 *    memory.  "stream" is a hipStream_t passed as void* (NULL = the default
 *    stream).  Enqueuing calls return as soon as the work is queued; buffers
 *    must stay valid until the stream has passed them.
 *  - Activations are bf16 bit patterns (uint16), contiguous, row-major.
 *  - Every argument and state check happens on the host before any launch;
 *    on error nothing is modified and a negative fp_status is returned, with
 *    a message available from fp_last_error() (thread-local).
 *  - A handle is not thread-safe: calls on one handle must be serialised.
 *  - The library allocates and owns weights, KV cache and workspace; the
 *    caller owns the x / y buffers it passes.
 */
#ifndef FP_MI355X_H
#define FP_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FP_OK = 0,
    FP_ERR_INVALID_ARG = -1,   /* bad pointer, shape, size or enum */
    FP_ERR_STATE = -2,         /* call not allowed in the handle's state (decode before prefill) */
    FP_ERR_CAPACITY = -3,      /* batch / prompt / sequence beyond what the handle was created for */
    FP_ERR_OOM = -4,           /* device allocation failed */
    FP_ERR_HIP = -5,           /* HIP runtime error (no device, launch failure, ...) */
    FP_ERR_UNSUPPORTED = -6    /* valid request the library does not implement */
} fp_status;

/* Weight compression (Sec. 3.2). */
typedef enum {
    FP_WQ_BF16 = 0,          /* unquantised 16-bit weights */
    FP_WQ_INT8_CHANNEL = 1,  /* symmetric int8, one fp16 scale per output row */
    FP_WQ_INT4_G128 = 2,     /* asymmetric int4, fp16 scale and integer zero per 128 inputs */
    FP_WQ_BF16_2OF4 = 3      /* 2:4 semi-structured sparse bf16 (pruning, Sec. 3.3, Table A.1):
                                in every 4 consecutive inputs of a row the 2 weights of largest
                                magnitude are kept (the lower input first among equal ones);
                                runs on the sparse matrix cores */
} fp_weight_quant;

/* KV-cache compression (Sec. 3.2, "KV-cache quantization"). */
typedef enum {
    FP_KV_BF16 = 0,
    FP_KV_INT8 = 1           /* int8 codes, one fp16 scale per (sequence, position, kv head) */
} fp_kv_quant;

/* Layer-stack shape and capacity, fixed at creation.
 * Requirements (checked by fp_layer_create on the host):
 *  - every field > 0, rms_eps > 0, rope_theta > 0                 (else FP_ERR_INVALID_ARG)
 *  - n_heads % n_kv_heads == 0                                      (FP_ERR_INVALID_ARG)
 *  - hidden, n_heads*head_dim and ffn multiples of 16, of 128 for int4 weights (their
 *    groups run along every projection's input dimension)          (FP_ERR_INVALID_ARG)
 *  - max_seq >= max_prompt (max_seq == max_prompt leaves no room for a decode step
 *    after a full-length prompt)                                    (FP_ERR_INVALID_ARG)
 *  - vocab >= 0 and a multiple of 16                              (FP_ERR_INVALID_ARG)
 *  - 2:4 sparse weights: hidden, n_heads*head_dim and ffn multiples of 64 (FP_ERR_INVALID_ARG)
 *  - head_dim 64 or 128; query group n_heads / n_kv_heads from 1 to 16;
 *    max_batch <= 64; max_batch * max_prompt <= 2^24               (FP_ERR_UNSUPPORTED) */
typedef struct {
    int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn;
    int32_t max_batch, max_prompt, max_seq;
    float rms_eps;      /* RMSNorm epsilon, inside the square root (1e-5) */
    float rope_theta;   /* rotary base (1e4) */
    int32_t vocab;      /* 0: hidden layers only (requests on hidden states); > 0 (a multiple
                           of 16): the fingerprint also keeps the token embedding, the final
                           norm and the LM head (Sec. 5.1, Fig. 2) for requests on token ids */
} fp_shape;

typedef struct fp_layer fp_layer;   /* opaque: weights, KV cache, workspace, position */

/* Tensor ids (weights of layer l are synthesised from (seed, l, id)). */
enum {
    FP_T_ATTN_NORM = 0, FP_T_Q = 1, FP_T_K = 2, FP_T_V = 3, FP_T_O = 4,
    FP_T_MLP_NORM = 5, FP_T_GATE = 6, FP_T_UP = 7, FP_T_DOWN = 8,
    FP_T_INPUT = 15,     /* prompt hidden states, layer id -1 */
    /* the blocks outside the hidden layers (layer id -1), present when vocab > 0; all
     * bf16 under every weight format (the weight-only quantisation of Sec. 3.2 applies
     * to the hidden layers' projections) */
    FP_T_EMBED = 16,     /* token embedding [vocab, hidden], ~N(0, 0.02) */
    FP_T_FINAL_NORM = 17,/* final RMSNorm gain [hidden], 1 + N(0, 0.02) */
    FP_T_LM_HEAD = 18    /* LM head [vocab, hidden], ~N(0, 0.02) */
};

/*
 * Build a fingerprint: allocate weights, KV cache and workspace on the current
 * device and synthesise the weights from `seed` (the Generator of Sec. 5.1
 * reads a checkpoint; here weights ~N(0, 0.02) and norm gains 1 + N(0, 0.02)
 * come from the counter-based generator of fp_fill_normal), then quantise them
 * on the device.  Synchronous.  *out receives the handle (NULL on error).
 */
fp_status fp_layer_create(const fp_shape* shape, fp_weight_quant wq, fp_kv_quant kvq,
                          uint64_t seed, fp_layer** out);

/*
 * Validation-only handle with no device storage: fp_prefill / fp_decode_step
 * check their arguments and advance the host-side state exactly as a real
 * handle does, but enqueue no work; export calls return FP_ERR_STATE.  Needs
 * no GPU (host-side tests of the argument and state checks).
 */
fp_status fp_layer_create_unbacked(const fp_shape* shape, fp_weight_quant wq, fp_kv_quant kvq,
                                   uint64_t seed, fp_layer** out);

/* Free everything the handle owns: weights, KV cache, workspace and captured decode
 * graphs (synchronises the device first).  NULL is a no-op.  The handle is the
 * fingerprint the Profiler deploys (Sec. 4.2, Sec. 5.1); destroying it ends its
 * deployment. */
fp_status fp_layer_destroy(fp_layer* layer);

/*
 * Prefill (time to first token, Sec. 5.3): run the layer stack over a prompt.
 * x: device bf16 [B, P, hidden], y: device bf16 [B, P, hidden] (may not alias x).
 * Resets the KV cache of the B sequences and sets the position to P.
 * 1 <= B <= max_batch, 1 <= P <= max_prompt.  A prefill with a batch other than
 * the previous one drops the decode graphs captured for that batch (it waits for
 * the device to finish their replays first).
 */
fp_status fp_prefill(fp_layer* layer, const void* x, int32_t B, int32_t P, void* y, void* stream);

/*
 * One decode step (time per output token, Sec. 5.3): the B sequences of the
 * last prefill each take one token's hidden state at the current position,
 * append its K/V to the cache, attend over the whole prefix and produce the
 * layer stack's output; the position then advances by one.
 * x: device bf16 [B, hidden] (normally the previous output fed back), y: device
 * bf16 [B, hidden], no aliasing.  FP_ERR_STATE before a prefill,
 * FP_ERR_CAPACITY when the position has reached max_seq.
 */
fp_status fp_decode_step(fp_layer* layer, const void* x, void* y, void* stream);

/*
 * n consecutive decode steps, each step's output fed back as the next step's input
 * (the fingerprint generating n tokens, Sec. 5.3).  Step 1 reads x and writes y,
 * step 2 reads y and writes x, and so on: the last step's output ends in y when n
 * is odd and in x when n is even.  x and y: device bf16 [B, hidden] each, both
 * written, no aliasing.  With the decode graph on (fp_set_decode_graph), the n
 * steps are captured once per (x, y, n) and replayed as one graph, which saves a
 * graph launch per step; the results equal n calls of fp_decode_step.  The
 * position advances by n.  FP_ERR_INVALID_ARG for n < 1, NULL or overlapping
 * buffers; FP_ERR_STATE before a prefill; FP_ERR_CAPACITY when fewer than n
 * positions remain before max_seq (nothing runs).
 */
fp_status fp_decode_steps(fp_layer* layer, void* x, void* y, int32_t n, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): one decode step exactly as
 * fp_decode_step computes it (same kernels, same results bit for bit), launched
 * kernel by kernel with no graph instantiation and no allocation of any kind.  The
 * step's split-K partials, attention partials and row-norm sums live in a static
 * 64 MiB device region per GPU (held from the first call on that GPU until the
 * process ends) instead of the handle's workspace.  Every call on one GPU shares that
 * GPU's region: calls that overlap on one GPU (other streams, other threads, other
 * handles) race, so serialise them.  FP_ERR_CAPACITY, with nothing launched, when
 * the step at the active batch needs more than 64 MiB of scratch (the message gives
 * the size); otherwise the same argument and state errors as fp_decode_step.
 */
fp_status fp_decode_step_noalloc(fp_layer* layer, const void* x, void* y, void* stream);

/*
 * Replay decode steps as a captured HIP graph (1, the default) or launch the
 * kernels one by one (0).  Results are identical.  Graphs are captured on first
 * use per (x, y, active batch) for fp_decode_step and per (x, y, n, active batch)
 * for fp_decode_steps; each cache holds at most 16 graphs and is emptied (after a
 * device synchronisation) when a new capture would exceed that.
 */
fp_status fp_set_decode_graph(fp_layer* layer, int32_t enable);

/*
 * Synthetic data on the device: dst[i] = bf16(mean + sigma * z_i), i < n, where
 * z_i is element i of the Irwin-Hall-12 stream of (seed, layer, tensor):
 *   key = mix64(mix64(seed) + G*(((layer+1) << 8) | tensor)),
 *   words mix64(key + G*(c+1)) for c = 3i..3i+2, z_i = (sum of their twelve
 *   16-bit lanes - 393210) * 2^-16, with mix64 the SplitMix64 finaliser
 *   (Steele, Lea & Flood, OOPSLA 2014) and G = 0x9E3779B97F4A7C15.
 * Prompts use layer -1, tensor FP_T_INPUT, mean 0, sigma 1.  dst: device bf16 [n].
 */
fp_status fp_fill_normal(void* dst, int64_t n, uint64_t seed, int32_t layer, int32_t tensor,
                         float mean, float sigma, void* stream);

/*
 * The fingerprint's blocks outside the hidden layers (Sec. 5.1, Fig. 2), for handles
 * created with vocab > 0 (FP_ERR_STATE otherwise).  Their time is the "other" share
 * of TTFT and TPOT in Eq. 2 and Eq. 3 (Sec. 5.3).
 *
 * fp_embed: x[m] = row ids[m] of the embedding table, m < M.  ids: device int32 [M];
 * x: device bf16 [M, hidden].  An id outside [0, vocab) gives a row of zeros.
 */
fp_status fp_embed(fp_layer* layer, const int32_t* ids, int64_t M, void* x, void* stream);

/*
 * fp_head: final RMSNorm and LM head of the last position of each of B sequences, then
 * greedy decoding.  y: device bf16 [B, T, hidden] (a decode step's output has T = 1, a
 * prefill's T = P); the head reads position T - 1 of each sequence:
 *   yn = bf16(y * rsqrt(mean(y^2) + eps) * g_final),  logits = yn W_lm^T (fp32),
 *   next_ids[b] = argmax_v logits[b, v], the lowest v among equal maxima.
 * logits: device fp32 [B, vocab], or NULL; next_ids: device int32 [B].
 * 1 <= B <= max_batch, T >= 1.
 */
fp_status fp_head(fp_layer* layer, const void* y, int32_t B, int32_t T, float* logits, int32_t* next_ids,
                  void* stream);

/*
 * fp_generate: one dummy request on token ids (the Profiler's request, Sec. 4.2 and
 * Sec. 5.3): embed the prompt, prefill, head -> token 0 (the first token); then n_out
 * decode steps, step i embedding token i - 1 and producing token i.  Output length
 * n_out is the number of decode steps (Eq. 1: latency = TTFT + n_out * TPOT).
 *   prompt_ids: device int32 [B, P];  out_ids: device int32 [n_out + 1, B];
 *   logits: device fp32 [n_out + 1, B, vocab], or NULL;
 *   force_ids: NULL, or device int32 [n_out, B]: step i embeds force_ids[i - 1] instead
 *     of its own token i - 1 (teacher forcing, for parity checks); out_ids still
 *     receives the generated tokens;
 *   elapsed_ms: NULL, or receives the request's device time (events recorded on
 *     `stream` around it; the call then synchronises the stream).
 * Resets the cache of the B sequences like fp_prefill; the position ends at P + n_out.
 * The n_out decode steps replay as one captured graph per (out_ids, logits, force_ids,
 * n_out, B) while the decode graph is on.  1 <= B <= max_batch, 1 <= P <= max_prompt,
 * n_out >= 0, P + n_out <= max_seq (FP_ERR_CAPACITY).
 */
fp_status fp_generate(fp_layer* layer, const int32_t* prompt_ids, int32_t B, int32_t P, int32_t n_out,
                      int32_t* out_ids, float* logits, const int32_t* force_ids, float* elapsed_ms,
                      void* stream);

/*
 * Latency and memory estimation from fingerprints (host arithmetic, no device).
 *
 * Eq. 1 (Sec. 5.3): latency = TTFT + output_length * TPOT.  fp_fit_ttft_tpot solves the
 * 2x2 system of Eq. 1 at two output lengths.  L2: two fingerprints with layers[0] and
 * layers[1] hidden layers, each timed at the output lengths n_out[0] and n_out[1]
 * (latency[2*i + j]: fingerprint i at length j, any time unit); fp_fit_latency_l2
 * solves each fingerprint's 2x2, then the 4x4 system of Eq. 2 and Eq. 3
 *   TTFT = num_layers * TTFT_layer + TTFT_other,  TPOT = num_layers * TPOT_layer + TPOT_other.
 * fp_predict_latency evaluates Eq. 1-3 for any layer count and output length (NULL
 * outputs skipped).  FP_ERR_INVALID_ARG for NULL inputs or a singular system (equal
 * lengths or equal layer counts).
 */
typedef struct {
    double ttft_layer, tpot_layer, ttft_other, tpot_other;
} fp_latency_model;

fp_status fp_fit_ttft_tpot(const int32_t n_out[2], const double latency[2], double* ttft, double* tpot);
fp_status fp_fit_latency_l2(const int32_t layers[2], const int32_t n_out[2], const double latency[4],
                            fp_latency_model* model);
fp_status fp_predict_latency(const fp_latency_model* model, int32_t n_layers, int32_t n_out, double* ttft,
                             double* tpot, double* latency);

/*
 * M2's layer extrapolation (Sec. 5.2): the value (e.g. a memory footprint) on the straight
 * line through (layers[0], values[0]) and (layers[1], values[1]) at n_layers; footprints
 * grow linearly with the number of hidden layers (Sec. 5, Fig. 7).  FP_ERR_INVALID_ARG
 * for equal layer counts.
 */
fp_status fp_extrapolate_layers(const int32_t layers[2], const double values[2], int32_t n_layers,
                                double* value);

/* Device memory in use on the current device (total - free, hipMemGetInfo) and its
 * total; the observed footprint M2 profiles (Sec. 5.2).  Either pointer may be NULL. */
fp_status fp_device_memory(size_t* used, size_t* total);

/*
 * Copy one weight tensor to host memory in its canonical layout (synchronous).
 * For parity checks of the quantised formats of Sec. 3.2 / Table A.1 (INT8 per
 * channel, INT4 group-128) against an independent implementation:
 *  bf16:  codes = bf16 [N, K] (scales, zeros unused, may be NULL)
 *  int8:  codes = int8 [N, K], scales = fp16 [N]
 *  int4:  codes = int32 [N, K/8] with nibble j of word w holding column 8w+j,
 *         scales = fp16 [N, K/128], zeros = fp16 [N, K/128] (integer values)
 *  2:4:   codes = bf16 [N, K], dense, the pruned weights zero (scales, zeros unused)
 * Norm gains (FP_T_ATTN_NORM, FP_T_MLP_NORM): codes = bf16 [hidden].
 * With vocab > 0 and l = -1: FP_T_EMBED and FP_T_LM_HEAD codes = bf16 [vocab, hidden],
 * FP_T_FINAL_NORM codes = bf16 [hidden].
 * [N, K] is (out, in): q [nh*d, hidden], k/v [nkv*d, hidden], o [hidden, nh*d],
 * gate/up [ffn, hidden], down [hidden, ffn].
 */
fp_status fp_export_weight(fp_layer* layer, int32_t l, int32_t tensor, void* codes, void* scales,
                           void* zeros);

/*
 * Copy layer l's KV cache (the cache that keeps per-token decode cost constant,
 * Sec. 5.3; int8 per Table A.1's KV-cache quantisation) for the active batch to
 * host memory (synchronous).  FP_ERR_STATE before a prefill:
 * k, v: [B, n_kv_heads, max_seq, head_dim] of bf16 or int8; k_scales, v_scales:
 * fp16 [B, n_kv_heads, max_seq] (int8 cache only, else may be NULL).
 */
fp_status fp_export_kv(fp_layer* layer, int32_t l, void* k, void* v, void* k_scales, void* v_scales);

/*
 * Debug: when dev_f32 is non-NULL, every later prefill / decode step also
 * writes the float32 K (after the rotary embedding) and V that enter the KV
 * store of every layer into dev_f32, laid out [n_layers, 2, B, T, n_kv_heads,
 * head_dim] with T the step's token count (P for prefill, 1 for decode);
 * the buffer must hold n_layers*2*max_batch*max_prompt*n_kv_heads*head_dim
 * floats.  NULL switches it off.  Disables graph replay while set.
 */
fp_status fp_set_debug_kv_dump(fp_layer* layer, void* dev_f32);

/*
 * Debug: when dev_bf16 is non-NULL, every later prefill / decode step also
 * copies each layer's output (the bf16 hidden states it hands to the next
 * layer, Sec. 5.1's stack of decoder layers) into dev_bf16, laid out
 * [n_layers, B, T, hidden] with T as above; the buffer must hold
 * n_layers*max_batch*max_prompt*hidden bf16 values and stay valid while set.
 * Lets a test compare each layer against a reference fed that layer's own
 * input.  NULL switches it off.  Disables graph replay while set.
 */
fp_status fp_set_debug_layer_dump(fp_layer* layer, void* dev_bf16);

/*
 * Per-kernel timing (the Profiler of Sec. 4.2 measures latency with dummy
 * requests; this breaks one request's step down by kernel).  Runs one prefill
 * or one decode step exactly as fp_prefill / fp_decode_step do, but launches
 * kernel by kernel with a HIP event recorded on `stream` before each launch and
 * after the last; synchronises, then writes one record per launch into out[]
 * (at most cap records; *count receives the number written).  State changes as
 * for the plain call.
 */
typedef enum {
    FP_K_RMSNORM = 0, FP_K_QKV = 1, FP_K_ROPE_KV = 2, FP_K_ATTN = 3, FP_K_O = 4,
    FP_K_RESID_NORM = 5, FP_K_GATE_UP = 6, FP_K_SWIGLU = 7, FP_K_DOWN = 8, FP_K_POS = 9
} fp_kernel_kind;

typedef struct {
    int32_t kind;    /* fp_kernel_kind */
    int32_t layer;   /* layer index, -1 for step-level kernels */
    float ms;        /* event-to-event device time of the launch */
} fp_kernel_time;

fp_status fp_profile_prefill(fp_layer* layer, const void* x, int32_t B, int32_t P, void* y,
                             void* stream, fp_kernel_time* out, int32_t cap, int32_t* count);
fp_status fp_profile_decode_step(fp_layer* layer, const void* x, void* y, void* stream,
                                 fp_kernel_time* out, int32_t cap, int32_t* count);

/*
 * Bytes of device memory the handle holds for weights (W), KV cache and workspace
 * (the activations A of the memory breakdown mem_base = W + A, Sec. 5.2).  On an
 * unbacked handle: the bytes a real handle of the same shape and formats holds.
 * Weight bytes count the fragment-major codes (K padded to a whole 1 KiB block
 * row-slice), the fp16 scales and zeros, the packed int4 scale/zero words and the
 * bf16 norm gains.  Any output pointer may be NULL.
 */
fp_status fp_memory_bytes(const fp_layer* layer, size_t* weights, size_t* kv, size_t* workspace);

/* Current position (tokens in the cache, Sec. 5.3) and active batch of the handle;
 * both 0 before the first prefill.  Any output pointer may be NULL. */
fp_status fp_get_position(const fp_layer* layer, int32_t* pos, int32_t* batch);

const char* fp_status_str(fp_status status);
const char* fp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FP_MI355X_H */
