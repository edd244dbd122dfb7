/*
 * sprout.h -- C ABI of the MI355X (gfx950) batched, ragged-length Llama-2
 * greedy decode library.
 *
 * The operation is the inference server's hot loop in Sprout (arXiv
 * 2403.12900): autoregressive generation with a KV cache, where every request
 * carries a generation-directive prefix placed before its prompt and stops at
 * its own generation limit.  Section II-A defines the loop (predict the next
 * token until EOS or a preset limit; cached keys/values of earlier tokens are
 * reused); Definition 1 and Section III-E fix the token order (directive
 * first, as a system prompt ahead of the user prompt); Section IV names the
 * served model (Llama 2).  The model is a random-init Llama-2 architecture
 * drawn on the device from a seed.
 *
 * Conventions for every entry point:
 *   - Return value: SPR_OK (0) or a negative spr_status.  No exception or
 *     longjmp crosses the ABI.  spr_last_error() gives a message for the last
 *     failure on the calling thread.
 *   - Arguments are validated against the model's state before anything is
 *     enqueued; a call that fails validation changes no state.
 *   - A HIP runtime failure (SPR_ERR_HIP) is sticky: every later call on that
 *     model returns SPR_ERR_HIP; the model must be released.
 *   - Device-side checks: a decode step fed a token id outside [0, vocab)
 *     (possible only through the caller-written device token buffer), or a
 *     logits row holding a NaN or no finite maximum, sets a flag in mapped
 *     host memory.  The first call that starts after the faulty work has
 *     completed on the device returns SPR_ERR_DEVICE_CHECK, and so does every
 *     later call: the model must be released.  (The step itself reads the
 *     clamped id, or emits token 0, so no access leaves its buffers.)
 *   - Pointers marked "host" are read (or written) during the call only.
 *     Pointers marked "device" must stay valid until the work enqueued on the
 *     model's stream has completed; device outputs are valid once the caller
 *     has synchronised that stream.
 *   - Calls on one model are not re-entrant and must come from one thread at
 *     a time.  Work is enqueued on the HIP stream given at init.
 */
#ifndef SPROUT_H_
#define SPROUT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPR_OK = 0,
  SPR_ERR_INVALID_ARG = -1, /* malformed argument or unsupported shape */
  SPR_ERR_WORKSPACE = -2,   /* workspace missing, misaligned or too small */
  SPR_ERR_KV_FULL = -3,     /* not enough free KV-cache blocks */
  SPR_ERR_STATE = -4,       /* call does not match the slot state */
  SPR_ERR_HIP = -5,         /* HIP runtime error (sticky) */
  SPR_ERR_DEVICE_CHECK = -6 /* a device-side check of an earlier call failed (sticky) */
} spr_status;

typedef enum { SPR_F32 = 0, SPR_BF16 = 1 } spr_dtype;

/*
 * Model shape and capacity.  Llama-2 architecture (Section IV): pre-norm
 * decoder layers of RMSNorm -> attention with rotary position embedding ->
 * residual, RMSNorm -> SwiGLU MLP -> residual; untied embedding and LM head;
 * no biases.  Weights are stored in `dtype` and the KV cache in `kv_dtype`
 * (keys and values are rounded to it, nearest-even, when cached); the
 * residual stream, norms, softmax, accumulation and logits are fp32.
 *
 * Constraints: n_layers 1..255; head_dim 64 or 128; n_heads a multiple of
 * n_kv_heads with n_heads / n_kv_heads <= 16; d_model a multiple of 16;
 * d_ff, vocab >= 1; kv_block must be 16; max_slots 1..64; max_ctx >= 1;
 * kv_blocks >= 1 (the shared pool of 16-position blocks).
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rope_base; /* 10000 for Llama 2 */
  float rms_eps;   /* 1e-5 for Llama 2 */
  int32_t dtype;   /* spr_dtype */
  int32_t kv_block;  /* positions per KV block: 16 */
  int32_t max_slots; /* concurrent requests */
  int32_t max_ctx;   /* positions per request: prompt + generated - 1 */
  int32_t kv_blocks; /* KV blocks in the pool */
  int32_t kv_dtype;  /* spr_dtype of the KV cache; fp32 models need SPR_F32 */
} spr_config;

typedef struct spr_model spr_model; /* opaque, library-owned host state */

/* Device bytes the caller must provide for `cfg` (0 if cfg is invalid). */
size_t spr_workspace_bytes(const spr_config* cfg);

/*
 * Creates a model in the caller's device workspace and draws its weights on
 * the device.  dev_ws: device pointer, 256-byte aligned, ws_bytes >=
 * spr_workspace_bytes(cfg); owned by the caller, who keeps it alive until
 * spr_release.  The library allocates no device memory of its own.
 * hip_stream: a hipStream_t (NULL = the null stream).  Weight element (r, c)
 * of each matrix is the counter-based N(0, 0.02) draw of its row-major index
 * (SplitMix64 outputs -> Irwin-Hall sum of eight 16-bit lanes -> one fp32
 * multiply -> round to `dtype`); all RMSNorm gains are 1.  Synchronous: the
 * weights are ready when it returns.  *out receives the model.
 */
spr_status spr_init(const spr_config* cfg, uint64_t seed, void* dev_ws, size_t ws_bytes, void* hip_stream,
                    spr_model** out);

/*
 * Prefill: fills the KV cache of n new requests with their prompts and emits
 * each one's first generated token (Section II-A: the prompt populates the
 * cache; generation follows).  A request's prompt is its directive prefix
 * followed by its user prompt (Section III-E), at positions 0..seq_len-1.
 *   slots      host [n]: distinct free slot ids in [0, max_slots)
 *   tokens     host [sum(seq_lens)]: the prompts, concatenated in order
 *   seq_lens   host [n]: >= 1
 *   stop_lens  host [n]: tokens to generate, >= 1, seq_len + stop_len - 1 <= max_ctx
 *   tok        device int32 [max_slots], indexed by slot: tok[slot] receives
 *              the first generated token
 *   logits     device fp32 [n, vocab] or NULL: logits of each last prompt position
 *   retired    host int32 [n] or NULL: 1 where stop_len == 1 (the request is done)
 * KV blocks for seq_len + stop_len - 1 positions are reserved per request;
 * the call fails with SPR_ERR_KV_FULL (and reserves nothing) if the pool
 * cannot hold them all.
 */
spr_status spr_prefill(spr_model* m, int32_t n, const int32_t* slots, const int32_t* tokens,
                       const int32_t* seq_lens, const int32_t* stop_lens, int32_t* tok, float* logits,
                       int32_t* retired);

/*
 * One decode step over the active requests (Section II-A's loop, one
 * iteration for each request in the batch).  Each listed slot feeds
 * tok[slot] at position lens[k], attends to its cached positions 0..lens[k],
 * and tok[slot] is overwritten with the greedy (lowest index on ties) next
 * token.  tok may therefore be the buffer the previous step wrote
 * (free-running greedy decode without a host round trip) or hold tokens the
 * caller forced.
 *   n_active   1..max_slots
 *   slots      host [n_active]: distinct active slots
 *   lens       host [n_active]: cached positions of each slot; must equal the
 *              library's count (SPR_ERR_STATE otherwise)
 *   tok        device int32 [max_slots], indexed by slot, read then written
 *   logits     device fp32 [n_active, vocab] or NULL: row k = logits of slots[k]
 *   retired    host int32 [n_active] or NULL: 1 where this step produced the
 *              slot's stop_len-th token; that slot then accepts no more steps
 *              until spr_rewind_slot, and keeps its KV blocks until
 *              spr_free_slot
 */
spr_status spr_decode_step(spr_model* m, int32_t n_active, const int32_t* slots, const int32_t* lens, int32_t* tok,
                           float* logits, int32_t* retired);

/*
 * spr_decode_step for callers that cannot allocate device memory or touch the
 * model's workspace scratch (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): identical arguments, semantics
 * and results, but the step's scratch -- split partials (of attention and of
 * the projections' split-K slices), arrival counters and the LM head's
 * greedy candidates -- lives in a fixed 24 MiB array in device memory that
 * the library holds on each device it runs on until the process ends.  The call allocates nothing and makes no
 * allocating runtime call; it clears the counters it uses with a kernel
 * before the step.  Every call on one device shares that device's array:
 * calls that overlap on one device (on different streams, or from different
 * threads) race and must not be issued.  SPR_ERR_INVALID_ARG when the model
 * or batch does not fit the array: more than 128 KV heads, a vocabulary
 * above 130048, n_heads * (head_dim + 4) * 4 bytes * n_active above 16 MiB,
 * or d_ff or (n_heads + 2 * n_kv_heads) * head_dim above 30840; other
 * errors as spr_decode_step.
 */
spr_status spr_decode_step_static_scratch(spr_model* m, int32_t n_active, const int32_t* slots, const int32_t* lens,
                                          int32_t* tok, float* logits, int32_t* retired);

/*
 * Rolls a prefilled slot back to `len` cached positions with `produced`
 * tokens generated.  The prompt stays: 1 <= produced <= the tokens produced
 * so far, and len == prompt length + produced - 1 (SPR_ERR_INVALID_ARG
 * otherwise; SPR_ERR_STATE for a free slot).  Positions >= len are dropped;
 * the slot is active again if produced < its stop length.  Used to
 * regenerate from a prompt.
 */
spr_status spr_rewind_slot(spr_model* m, int32_t slot, int32_t len, int32_t produced);

/* Returns a slot's KV blocks to the pool and frees the slot. */
spr_status spr_free_slot(spr_model* m, int32_t slot);

/* Cached positions of a slot (-1 if free) and tokens produced so far. */
spr_status spr_slot_info(const spr_model* m, int32_t slot, int32_t* len, int32_t* produced, int32_t* stop_len);

/* Free KV blocks in the pool. */
int32_t spr_free_blocks(const spr_model* m);

/*
 * Reads rows [row0, row0 + nrows) of one logical weight matrix back as fp32
 * (exact values), row-major, into device memory `out` [nrows, cols].
 * tensor: 0 embedding [vocab, d], 1 Wq [H*hd, d], 2 Wk [Hkv*hd, d],
 * 3 Wv [Hkv*hd, d], 4 Wo [d, H*hd], 5 W1 gate [d_ff, d], 6 W3 up [d_ff, d],
 * 7 W2 down [d, d_ff], 8 LM head [vocab, d].  For checking the device
 * generator against an independent one.
 */
spr_status spr_export_weight_rows(spr_model* m, int32_t tensor, int32_t layer, int32_t row0, int32_t nrows,
                                  float* out);

/*
 * Measurement aid: enqueues `reps` back-to-back launches of one projection
 * kernel exactly as a decode step over n_rows rows launches it (launch r uses
 * layer r mod n_layers, so every layer's weights are streamed in turn),
 * brackets them with HIP events on the model's stream, waits, and writes the
 * mean launch duration in microseconds to *avg_us.  projection: 1 = O
 * (x += o Wo^T), 2 = gate/up with SwiGLU, 3 = down (x += h W2^T), 4 = LM head
 * with the greedy candidates.  It reads and writes only the forward pass's
 * scratch buffers (activations, residual, greedy candidates), which every
 * decode step rewrites before reading, so cached state is untouched; the QKV
 * projection, which appends to the KV cache, is refused (SPR_ERR_INVALID_ARG).
 * n_rows 1..128, reps 1..100000.  Synchronous.
 */
spr_status spr_time_projection(spr_model* m, int32_t projection, int32_t n_rows, int32_t reps, float* avg_us);

/*
 * Test aid (for tests of the greedy tie rule and of the device checks; no
 * other caller needs it): overwrites row dst of the LM-head matrix, with row
 * src when src >= 0 (a planted exact tie: both rows then give bitwise equal
 * logits), else with `fill` rounded to the weight format (a NaN fill makes
 * every later logits row hold a NaN).  The model is changed for the rest of
 * its life.  dst in [0, vocab), src < vocab, else SPR_ERR_INVALID_ARG.
 * Synchronous.
 */
spr_status spr_test_write_lm_head_row(spr_model* m, int32_t dst, int32_t src, float fill);

/*
 * Measurement aid: the HBM read ceiling of the projections' load form.
 * Streams every weight matrix a decode step reads (all layers' projections
 * and the LM head, resident in the model's workspace) once per rep with
 * 16-byte nontemporal loads, 8 in flight per thread and no arithmetic, brackets
 * the reps with HIP events on the model's stream, waits, and writes the mean
 * read rate in GB/s (1e9 bytes/s) to *gbps and the bytes read per rep to
 * *bytes.  Reads only; model state is untouched.  reps 1..1000; null outputs
 * are SPR_ERR_INVALID_ARG.  Synchronous.
 */
spr_status spr_time_read_ceiling(spr_model* m, int32_t reps, double* gbps, uint64_t* bytes);

#define SPR_MAX_LEVELS 8 /* directive levels a serving run can profile */

/* One request of a serving run (host memory, read during the call). */
typedef struct {
  const int32_t* tokens; /* prompt: directive prefix followed by the user prompt */
  int32_t n_tokens;      /* >= 1 */
  int32_t stop_len;      /* generation limit, >= 1; n_tokens + stop_len - 1 <= max_ctx */
  int32_t arrival;       /* first scheduler iteration it may be admitted in (0 = at once) */
  int32_t level;         /* directive level (Definition 1), 0..SPR_MAX_LEVELS-1; profiling tag only */
} spr_request;

typedef struct {
  int64_t iterations;    /* scheduler iterations run */
  int64_t decode_steps;  /* decode steps launched */
  int64_t prefill_calls; /* batched prefills launched */
  int64_t decode_tokens; /* decode rows launched (tokens past an EOS included) */
  int32_t max_batch;     /* largest decode batch */
  double mean_batch;     /* mean decode batch */
  double device_seconds; /* device time from the call's first work to its last iteration */
  /* Per directive level, the profiles Eq. 2 consumes (p: processing time per
     request).  Each iteration's device time is shared equally by the
     requests it served; a request's time is the sum of its shares. */
  int32_t level_requests[SPR_MAX_LEVELS]; /* requests of the level */
  double level_tokens[SPR_MAX_LEVELS];    /* mean generated tokens (lengths) per request */
  double level_seconds[SPR_MAX_LEVELS];   /* p: mean device seconds per request */
} spr_serve_stats;

/*
 * Serves n requests with continuous (iteration-level) batching: the
 * scheduling of the inference servers the paper deploys on (Section IV:
 * vLLM's paged KV cache; related work: Orca's iteration-level batching),
 * here over the decode step above.  Every iteration
 *   1. admits waiting requests, first come first served, whose arrival
 *      iteration has come, into free slots while fewer than max_active
 *      requests are in flight and the KV pool can reserve their blocks (a
 *      request that does not fit yet holds back the ones behind it);
 *   2. prefills the admitted requests together (first tokens);
 *   3. runs one decode step over every request still generating;
 *   4. retires requests that reached their stop length, freeing their slots
 *      and KV blocks for the next iteration;
 *   5. retires requests whose previous-iteration token was eos_id (Section
 *      II-A: generation ends at EOS or at the preset limit).  The tokens are
 *      read back one iteration late, so the host never waits for the
 *      iteration it has just enqueued; such a request runs one more decode
 *      row (two if EOS was its prefill token), whose token is discarded.
 * Iterations with nothing in flight skip to the next arrival.  Outputs are
 * the greedy tokens each request would get served alone.
 *   max_active 1..max_slots
 *   eos_id     token id that ends a request, or negative for none
 *   tok        device int32 [max_slots]: scratch token buffer, indexed by slot
 *   out        device int32 [sum of stop_len]: request i's tokens at offset
 *              stop_len[0] + ... + stop_len[i-1]; entries past its length
 *              are unspecified
 *   lengths    host int32 [n] or NULL: tokens generated per request, up to
 *              and including the first EOS, else stop_len
 *   stats      host, or NULL
 * Needs every slot free on entry (SPR_ERR_STATE otherwise) and leaves them
 * free.  A malformed request, or one that max_ctx or the KV pool could never
 * hold, fails with SPR_ERR_INVALID_ARG before any work is enqueued.
 * Synchronous: out is complete when it returns.  Uses a few HIP events and,
 * with an EOS id, 16 * max_slots bytes of pinned host memory for the call.
 */
spr_status spr_serve(spr_model* m, int32_t n, const spr_request* reqs, int32_t max_active, int32_t eos_id,
                     int32_t* tok, int32_t* out, int32_t* lengths, spr_serve_stats* stats);

/* Releases the host state.  The workspace is the caller's to free afterwards. */
spr_status spr_release(spr_model* m);

/* Message for the last failure on the calling thread ("" if none). */
const char* spr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPROUT_H_ */
