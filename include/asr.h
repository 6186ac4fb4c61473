/*
 * asr.h - C ABI of the MI355X (gfx950) batched Whisper-shaped ASR step behind
 * a duration-aware waiting queue.
 *
 * What the calls compute (paper: "Duration Aware Scheduling for ASR Serving
 * Under Workload Drift"):
 *   - asr_submit records a request; its job length is the audio duration
 *     (Section 3.2: duration is used directly as the job-length proxy) or the
 *     Eq. 1 token estimate max(1, floor(d * kappa)) (Appendix A.4 endpoint).
 *   - asr_rank / asr_pop_batch order the waiting requests by FCFS, SJF
 *     (shortest first, earlier arrival then lower id on ties; Section 3.2 and
 *     the SJF key of Appendix A.4) or HRRN (highest (wait + job) / job first,
 *     recomputed at every pop; Section 3.2, Appendix A.4).
 *   - asr_step runs one batched Whisper step (the work the scheduler
 *     dispatches, Section 3.1): for newly admitted clips the log-mel
 *     front-end, the conv stem, the encoder layers and the cross-attention K/V
 *     of every decoder layer; for running sequences one decoder step with
 *     causal self-attention over the per-slot cache, cross-attention over the
 *     1500 cached encoder positions, and the vocabulary projection fused with
 *     argmax.
 *
 * Conventions
 *   - Every call returns asr_status and never throws or aborts; on failure a
 *     thread-local message is available from asr_last_error().
 *   - Time is never read from a clock: callers pass now_us / arrival_us, so
 *     every ordering is reproducible.
 *   - Host buffers belong to the caller.  Device memory is ONE caller-provided
 *     block (asr_bind) that the library sub-allocates and never frees; the
 *     library itself never allocates device memory.
 *   - GPU work is enqueued on the stream given to asr_bind.  A prefill may
 *     fork onto streams the context owns (default priority): its clip groups
 *     (asr_set_encoder_streams) and, with overlapped prefill, the whole
 *     prefill; every fork waits on an event of the bound stream and is joined
 *     back into it (or synchronised) before the call returns.  asr_step and
 *     the debug readers synchronise only to copy results to the host.
 *   - A context is not thread-safe; calls on one context must be serialised.
 */
#ifndef ASR_H
#define ASR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ASR_OK = 0,
  ASR_EINVAL = 1,    /* bad argument (message says which) */
  ASR_ENOMEM = 2,    /* bound block smaller than asr_workspace_size */
  ASR_EFULL = 3,     /* queue at max_queue, or no free decode slot */
  ASR_ENOTFOUND = 4, /* unknown request id or slot */
  ASR_ESTATE = 5,    /* call out of order (e.g. step before bind/load) */
  ASR_ENODEV = 6,    /* GPU call on a queue-only context (device = -1) */
  ASR_EDEVICE = 7    /* HIP runtime error, or a NaN logit */
} asr_status;

typedef enum { ASR_FCFS = 0, ASR_SJF = 1, ASR_HRRN = 2 } asr_policy;

typedef enum { ASR_F32 = 0, ASR_BF16 = 1 } asr_dtype;

/* Model and capacity.  Whisper shapes: d_model = 64 * n_head; the encoder
 * always sees 30-s segments (480000 samples at 16 kHz -> 3000 mel frames ->
 * 1500 positions); the decoder context is 448 positions (Section 4.1: at most
 * 448 output tokens).  n_enc = 0 builds a decoder-only context (cross K/V then
 * come from asr_debug_set_encoder_out); n_dec = 0 an encoder-only one.
 * dtype ASR_BF16 stores matrices, caches and activations between kernels in
 * bfloat16 (round to nearest even) with float32 accumulation, float32
 * residual stream, LayerNorm and softmax; ASR_F32 keeps everything float32. */
typedef struct {
  int32_t n_mels;      /* multiple of 8, at most 128 (Whisper: 80 or 128) */
  int32_t d_model;     /* multiple of 64 (of 128 for bf16), at most 2048 */
  int32_t n_enc;       /* encoder layers (>= 0) */
  int32_t n_dec;       /* decoder layers (>= 0) */
  int32_t n_head;      /* d_model / 64 */
  int32_t d_ffn;       /* MLP width, multiple of 64 */
  int32_t vocab;       /* vocabulary size (tied output projection) */
  int32_t dtype;       /* asr_dtype */
  int32_t max_slots;   /* decode slots, each with its own self and cross cache */
  int32_t max_prefill; /* clips per prefill batch */
  int32_t max_decode;  /* rows per decode step (<= max_slots) */
  int32_t max_queue;   /* waiting requests */
} asr_model_cfg;

typedef struct asr_ctx asr_ctx;

/* Creates a context.  device >= 0 selects a HIP device; device = -1 creates a
 * queue-only context (no HIP call is ever made; GPU calls return ASR_ENODEV).
 * Errors: EINVAL for inconsistent shapes. */
asr_status asr_create(const asr_model_cfg* cfg, int32_t device, asr_ctx** out);
asr_status asr_destroy(asr_ctx* ctx);
const char* asr_last_error(void);

/* Device bytes the context needs: weights, per-slot caches and scratch. */
asr_status asr_workspace_size(const asr_ctx* ctx, size_t* bytes);

/* Hands the library a device block of at least asr_workspace_size bytes
 * (256-byte aligned) and the hipStream_t to enqueue on (NULL = default
 * stream).  The caller keeps the block alive until asr_destroy.  Uploads the
 * library's own constant tables (window, twiddles, mel filterbank,
 * sinusoidal positions).  Errors: ENODEV, ENOMEM, EINVAL (alignment). */
asr_status asr_bind(asr_ctx* ctx, void* dev_block, size_t bytes, void* stream);

/* Parameter tensors, in the fixed load order (n = asr_n_params):
 * encoder (n_enc > 0): conv1.w [d][n_mels][3], conv1.b [d], conv2.w [d][d][3],
 *   conv2.b [d]; per layer: attn_ln.g, attn_ln.b, q.w [d][d], q.b, k.w, v.w,
 *   v.b, o.w, o.b, mlp_ln.g, mlp_ln.b, fc1.w [ffn][d], fc1.b, fc2.w [d][ffn],
 *   fc2.b; then ln_post.g, ln_post.b.
 * decoder (n_dec > 0): tok_emb [vocab][d], pos_emb [448][d]; per layer:
 *   attn_ln.g/b, q.w, q.b, k.w, v.w, v.b, o.w, o.b, xattn_ln.g/b, xq.w, xq.b,
 *   xk.w, xv.w, xv.b, xo.w, xo.b, mlp_ln.g/b, fc1.w, fc1.b, fc2.w, fc2.b;
 *   then ln.g, ln.b.
 * Linear weights are [out][in]; conv weights [out][in][tap]. */
asr_status asr_n_params(const asr_ctx* ctx, int32_t* n);
asr_status asr_param_numel(const asr_ctx* ctx, int32_t index, int64_t* numel);

/* Loads all parameters from float32 tensors in the order above (host
 * pointers, or device pointers when on_device != 0).  The library repacks
 * them (fused QKV, per-tap conv layout, all layers' cross K/V in one matrix)
 * and rounds matrices to bfloat16 (round to nearest even) on bf16 contexts.
 * Synchronous.  Errors: ESTATE before bind, EINVAL on a NULL tensor. */
asr_status asr_load_weights(asr_ctx* ctx, const float* const* tensors, int32_t n,
                            int32_t on_device);

/* Scheduling policy (Section 3.2).  kappa_den == 0: the job length is the
 * duration in microseconds; otherwise it is the Eq. 1 estimate
 * max(1, floor(n_samples * kappa_num / (sample_rate * kappa_den))) tokens,
 * falling back to max_tokens for a request without audio (Appendix A.4).
 * Takes effect for the next rank/pop.  Errors: EINVAL. */
asr_status asr_set_policy(asr_ctx* ctx, int32_t policy, int32_t kappa_num, int32_t kappa_den);

/* Records a waiting request.  pcm: n_samples float32 samples at 16 kHz
 * (n_samples <= 480000: one 30-s segment).  pcm_on_device = 0: the samples
 * are copied before return.  pcm_on_device = 1: pcm is a device pointer the
 * caller keeps valid until the request has been prefilled.  pcm may be NULL
 * (with n_samples giving the length) for a request whose encoder output will
 * be supplied through asr_debug_set_encoder_out.  duration_us <= 0 derives
 * floor(n_samples * 1e6 / sample_rate).  max_tokens <= 0 means 448.
 * Errors: EINVAL (duplicate id, sample_rate != 16000, n_samples out of
 * [1, 480000], max_tokens > 448), EFULL (max_queue reached). */
asr_status asr_submit(asr_ctx* ctx, int64_t id, const float* pcm, int64_t n_samples,
                      int32_t sample_rate, int64_t duration_us, int64_t arrival_us,
                      int32_t max_tokens, int32_t pcm_on_device);

/* Waiting requests with arrival_us <= now_us, in service order, without
 * removing them.  Writes min(cap, eligible) ids; *n_out = that count. */
asr_status asr_rank(const asr_ctx* ctx, int64_t now_us, int64_t* out_ids, int32_t cap,
                    int32_t* n_out);

/* Removes and returns the first max_n eligible requests in service order (one
 * now_us for the whole batch).  Popped requests stay known to the context
 * until they are prefilled by asr_step (or their slot is filled by
 * asr_debug_set_encoder_out). */
asr_status asr_pop_batch(asr_ctx* ctx, int64_t now_us, int32_t max_n, int64_t* out_ids,
                         int32_t* n_out);
asr_status asr_queue_len(const asr_ctx* ctx, int32_t* n);

typedef struct {
  int32_t n_prefill;           /* popped requests to encode this step (<= max_prefill) */
  const int64_t* prefill_ids;  /* [n_prefill] */
  int32_t n_decode;            /* running sequences to advance (<= max_decode) */
  const int32_t* slots;        /* [n_decode] distinct occupied slots */
  const int32_t* tokens;       /* [n_decode] input token ids (teacher forcing) */
  float* logits;               /* optional host [n_decode][vocab] float32 */
} asr_step_in;

typedef struct {
  int32_t* slot_of;  /* [n_prefill] slot given to each prefilled request */
  int32_t* argmax;   /* [n_decode] argmax of each row's logits, lowest index on ties */
  int32_t* done;     /* [n_decode] 1 when the row's slot has no steps left */
} asr_step_out;

/* One batched step on the bound stream: prefill (mel -> stem -> encoder ->
 * cross K/V into a free slot per request, positions reset to 0, steps left =
 * min(max_tokens, round-half-up(2.7 tokens per audio-second)), then decode
 * (each row writes its self K/V at the slot's position, attends over
 * position + 1 keys, produces its argmax; the position then advances).
 * Prefill happens before decode, so a slot prefilled here may be decoded in
 * the same call.  Errors: ESTATE, ENODEV, EINVAL (bad id/slot/token,
 * duplicate slot, position at 448), EFULL (no free slot), EDEVICE. */
asr_status asr_step(asr_ctx* ctx, const asr_step_in* in, asr_step_out* out);

/* Frees a slot for reuse. */
asr_status asr_release_slot(asr_ctx* ctx, int32_t slot);
/* State of a slot: occupied flag, request id, position, steps left. */
asr_status asr_slot_info(const asr_ctx* ctx, int32_t slot, int32_t* occupied, int64_t* id,
                         int32_t* position, int32_t* steps_left);

/* ---- per-kernel timing (HIP events around every launch on the bound stream) */
typedef enum {
  ASR_K_MEL = 0,        /* log-mel front-end (+ normalise) */
  ASR_K_GEMM = 1,       /* encoder and stem MFMA GEMMs */
  ASR_K_ATTN = 2,       /* encoder flash attention */
  ASR_K_LN = 3,         /* LayerNorms */
  ASR_K_DGEMM = 4,      /* decode GEMMs (+ split-K reduce) */
  ASR_K_DATTN = 5,      /* decode self + cross attention */
  ASR_K_VOCAB = 6,      /* vocabulary GEMM + argmax */
  ASR_K_OTHER = 7,
  ASR_K_PREFILL = 8,    /* whole prefill phase of asr_step (mel .. cross K/V) */
  ASR_K_DECODE = 9,     /* whole decode phase of asr_step (embed .. argmax) */
  ASR_K_ENCODE = 10,    /* encoder part of a prefill (mel .. ln_post, without cross K/V):
                           from its start to the last clip group's ln_post */
  ASR_K_XKV = 11,       /* the cross K/V product of a prefill (all decoder layers, one
                           MFMA GEMM after the encoder's clip groups have joined) */
  ASR_K_COUNT = 12
} asr_kernel_class;

/* ---------------------------------------------------------------------------
 * Continuous batching with preemption (the serving loop the scheduling policy
 * runs in: Section 4.1's engine setup, and the preemption rule of the
 * implementation appendix).
 *
 * Each engine step at now_us: (1) every running request is about to decode
 * one token; while the KV pool cannot hold that, a running request is
 * preempted -- SJF the one with the largest job key, HRRN the one with the
 * lowest current response ratio (wait + job) / job, FCFS the most recently
 * admitted -- and goes back to the waiting queue with its arrival time and
 * keys (its tokens are dropped: it is recomputed when admitted again);
 * (2) free slots are refilled from the queue in the policy's order, each
 * admitted request being prefilled and producing its first token in this
 * step, until max_admit, no free slot, or the first request the pool cannot
 * hold; (3) all running requests decode one token (greedy: the argmax becomes
 * the next input) and those that reach their token count finish.
 *
 * A request produces round-half-up(duration * tok_num / tok_den) tokens,
 * clamped to [1, min(448, max_tokens)].  The pool counts token positions: a
 * running request holds cross_tokens plus one per generated token.
 * ------------------------------------------------------------------------- */
typedef struct {
  int64_t kv_capacity;  /* pool size in token positions; <= 0: slots are the only bound.
                           Every request must fit on its own (cross_tokens + its token
                           count): asr_serve_config and later asr_submit calls reject
                           one that cannot (EINVAL), since it could never finish */
  int32_t cross_tokens; /* positions charged for a request's cross cache (1500) */
  int32_t max_admit;    /* admissions per step, 1 .. max_prefill */
  int32_t tok_num;      /* output tokens per audio-second = tok_num / tok_den (27/10) */
  int32_t tok_den;
  int32_t start_token;  /* decoder input at position 0 */
  /* Dynamic policy switching (the future-work paragraph of Section 5: watch
   * the queue and switch among FCFS, SJF and HRRN).  0: the policy of
   * asr_set_policy throughout.  1: at the start of every step, FCFS while at
   * most depth_low requests are eligible (they all get in anyway); otherwise
   * HRRN when some eligible request's response ratio (wait + job) / job
   * exceeds starve_num / starve_den (a starvation signal), else SJF.  The
   * chosen policy orders that step's admissions and picks its victims. */
  int32_t dynamic;
  int32_t depth_low;
  int64_t starve_num;
  int64_t starve_den;   /* > 0 when dynamic */
  /* >= 1: overlapped prefill (Section 4.1 runs the engine with chunked
   * prefill).  An admitted request then produces its first token in the step
   * after the one that prefills it, so a step's prefill runs on a second
   * stream while the running rows decode on the bound stream.  A value above
   * 1 is the number of CUs the prefill's persistent GEMMs leave free for the
   * decode rows.  Every request's tokens are the same as without overlap.
   * On a queue-only context only the schedule changes (first tokens one step
   * later). */
  int32_t overlap;
} asr_serve_cfg;

/* Arrays are the caller's, each with room for cap >= the slot count
 * (min(max_slots, max_decode) on a GPU context, max_slots queue-only). */
typedef struct {
  int32_t cap;
  int32_t policy;         /* policy the step ran under (asr_policy) */
  int64_t* preempted;     int32_t n_preempted;
  int64_t* admitted;      int32_t* admitted_slot;  int32_t n_admitted;
  int64_t* decoded;       int32_t* token;          int32_t n_decoded;  /* token -1: no model ran */
  int64_t* finished;      int32_t n_finished;
} asr_serve_out;

/* Switches the context to continuous batching (the manual asr_pop_batch /
 * asr_step / asr_release_slot then return ESTATE).  ESTATE when slots are
 * occupied or popped requests wait; EINVAL for an inconsistent config. */
asr_status asr_serve_config(asr_ctx* ctx, const asr_serve_cfg* cfg);
/* One engine step on the GPU: plan, prefill the admitted requests, decode
 * every running request, commit.  Synchronises on the bound stream. */
asr_status asr_serve_step(asr_ctx* ctx, int64_t now_us, asr_serve_out* out);
/* The same schedule without running the model (tokens -1), for queue-only
 * contexts (device = -1; ESTATE otherwise): simulations and CPU tests. */
asr_status asr_serve_plan(asr_ctx* ctx, int64_t now_us, asr_serve_out* out);
/* Steps run under each policy since asr_serve_config (steps[ASR_FCFS] ..). */
asr_status asr_serve_stats(const asr_ctx* ctx, int64_t steps[3]);
/* Tokens of a finished request, once (ENOTFOUND otherwise; EINVAL when cap is
 * smaller than the token count). */
asr_status asr_serve_tokens(asr_ctx* ctx, int64_t id, int32_t* tokens, int32_t cap, int32_t* n);

/* Serving simulation (the evaluation of Section 4.1 and the burst appendix on
 * a virtual clock).  A step that admits a requests and decodes r rows lasts
 * prefill_us * a + (r > 0 ? step_us + row_us * r : 0) microseconds. */
typedef struct {
  int64_t prefill_us;
  int64_t step_us;
  int64_t row_us;
} asr_sim_cost;
/* Runs the continuous-batching schedule (asr_serve_plan steps) from t0_us,
 * jumping over idle time to the next arrival, until every submitted request
 * has finished.  Queue-only, serve-configured contexts; ids lists every
 * submitted request (EINVAL otherwise).  Per request ids[i]: time of its first
 * and last token (first_us, finish_us), token count and preemptions; token_us
 * (may be NULL) receives the emission time of every token, request after
 * request in ids order (token_cap entries at least; a position that a
 * recomputed request produces again is not emitted again).  *t_end_us is the
 * clock after the last step.  Latencies follow: TTFT = first_us - arrival,
 * E2EL = finish_us - arrival. */
asr_status asr_serve_simulate(asr_ctx* ctx, const asr_sim_cost* cost, int64_t t0_us, int32_t n,
                              const int64_t* ids, int64_t* first_us, int64_t* finish_us,
                              int32_t* n_tokens, int32_t* n_preempt, int64_t* token_us,
                              int64_t token_cap, int64_t* t_end_us);

/* Prefill clips split into n groups (1..4, default 2) whose encoder layers
 * run on n streams (the context's stream and n-1 of its own, default
 * priority), so one group's memory-bound LayerNorms and the last partial
 * round of a GEMM overlap another group's kernels; n = 1 runs the encoder as
 * one chain, where every launch owns the GPU (what per-kernel timing needs).
 * Results do not depend on n. */
asr_status asr_set_encoder_streams(asr_ctx* ctx, int32_t n);

/* Decode steps replayed from HIP graphs (on = 1, the default) or launched
 * kernel by kernel (on = 0).  With graphs, the decode kernels of each shape
 * (row count, logits wanted) are captured once -- at that shape's second
 * step, on a stream the context owns -- and every later step of the shape
 * replays them on the bound stream after uploading its rows.  Results are
 * the same either way; steps with per-launch timing selected always launch
 * directly. */
asr_status asr_set_decode_graphs(asr_ctx* ctx, int32_t on);

/* classes is a bit mask over the asr_kernel_class values: bit k selects class
 * k, 0 turns timing off, ASR_TIME_ALL times every class.  An event pair is
 * recorded on the context's stream around every launch (and phase) of a
 * selected class.  Each pair costs a little queue time, so a step timed with
 * a mask that selects the many short decode launches runs somewhat slower
 * than an untimed one. */
#define ASR_TIME_ALL ((1 << ASR_K_COUNT) - 1)
asr_status asr_set_timing(asr_ctx* ctx, int32_t classes);
/* Synchronises, then reports for one class since the last reset: summed
 * kernel milliseconds, launches, algorithmic flops and algorithmic HBM bytes
 * (the minimum traffic the launches need: operands read once, results
 * written once). */
asr_status asr_get_timing(asr_ctx* ctx, int32_t kernel_class, double* ms, int64_t* launches,
                          double* flops, double* bytes);
asr_status asr_reset_timing(asr_ctx* ctx);

/* ---- parity / debug entry points (synchronous; results copied to the host) */

/* Normalised log-mel features [n][3000][n_mels] float32 of n clips (pcm of
 * each clip at pcm[i], n_samples[i] samples; device pointers when
 * on_device).  n <= max_prefill. */
asr_status asr_debug_logmel(asr_ctx* ctx, const float* const* pcm, const int64_t* n_samples,
                            int32_t n, int32_t on_device, float* out);
/* Encoder output (after ln_post) [n][1500][d] float32 of n clips. */
asr_status asr_debug_encode(asr_ctx* ctx, const float* const* pcm, const int64_t* n_samples,
                            int32_t n, int32_t on_device, float* out);
/* Encoder self-attention kernel alone on given operands (Section 2's
 * encoder: softmax(q k^T / sqrt(64)) v per head, heads = consecutive 64-wide
 * column groups, no mask over the 1500 positions of a clip).  q, k, v, out:
 * host float32 [n][1500][d], n <= max_prefill.  q is given in the form the
 * QKV product hands the kernel: the queries times 1/sqrt(64) log2(e), so the
 * result is out = softmax_2(q k^T) v with softmax_2(s)_j = 2^s_j / sum 2^s.
 * A bf16 context rounds q, k, v to bf16 on the way in. */
asr_status asr_debug_attention(asr_ctx* ctx, const float* q, const float* k, const float* v,
                               int32_t n, float* out);
/* Fills slots[i] from a given encoder output E [n][1500][d] (float32): the
 * cross K/V of every decoder layer are projected into the slot's cache, the
 * position is reset to 0, the slot holds request id ids[i] (which must have
 * been popped, or be -1 for an anonymous sequence) with steps_left[i] steps. */
asr_status asr_debug_set_encoder_out(asr_ctx* ctx, const int32_t* slots, const int64_t* ids,
                                     const int32_t* steps_left, int32_t n, const float* E,
                                     int32_t on_device);
/* Reads (which = 0: self cache [n_dec][2][H][448][64]; which = 1: cross cache
 * [n_dec][2][H][1500][64]) of one slot as float32. */
asr_status asr_debug_get_kv(asr_ctx* ctx, int32_t slot, int32_t which, float* out);
/* Writes the self cache of an occupied slot from float32 [n_dec][2][H][448][64]
 * (host, or device when on_device) and sets its position to `length`
 * (positions >= length are ignored by attention and overwritten by later
 * steps). */
asr_status asr_debug_set_self_kv(asr_ctx* ctx, int32_t slot, const float* src, int32_t length,
                                 int32_t on_device);

/* ---- allocation-free variant ------------------------------------------
 * For callers that cannot allocate device memory or bind a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the log-mel front-end of asr_debug_logmel with its scratch in
 * a file-scope device array of the library (64 KiB per GPU, held until the
 * process ends) instead of a bound block.  Needs no context.
 *   pcm[i]: device pointer to clip i's float32 samples (n_samples[i] in
 *   [0, 480000]; may be NULL when 0); pcm and n_samples are host arrays of n
 *   entries, n in [1, 64].  n_mels: 80 or 128.  out: device float32
 *   [n][3000][n_mels], the normalised features (the same values
 *   asr_debug_logmel returns).  Work is enqueued on `stream` (NULL = default
 *   stream) of the current device; the call does not synchronise.
 * No allocation and no per-call copy: the clip list travels in the kernel
 * arguments.  The first call on a device resolves the array's address and
 * uploads the constant tables with synchronous copies, so a caller that
 * captures graphs makes one call before capturing.  All calls on one GPU
 * share its array (every call writes all the per-group maxima it reads, so
 * nothing carries over from an earlier call): calls that overlap on one GPU
 * race.
 * Errors: EINVAL (NULL argument, n or n_mels out of range, n_samples out of
 * range), EDEVICE (HIP error). */
asr_status asr_logmel_noalloc(const float* const* pcm, const int64_t* n_samples, int32_t n,
                              int32_t n_mels, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ASR_H */
