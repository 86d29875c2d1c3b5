/*
 * bcmt.h - C ABI of the BCMT token-mixing layer on AMD Instinct MI355X (gfx950).
 *
 * The layer is the one of "BCMT: Blockwise Causal Memory Transformer"
 * (arXiv 2608.13578), Sec. 3.2-3.8.  For an input X of B sequences, T
 * tokens and D features it computes, per sequence:
 *
 *   blocks     : N_b = ceil(T / L) contiguous blocks of at most L tokens
 *                (Sec. 3.2; the last block may be shorter);
 *   local MHA  : Q = X Wq, K = X Wk, V = X Wv; per head (width dh = D / H)
 *                and per block, softmax(Q K^T / sqrt(dh) + causal mask) V, where a
 *                token sees itself and earlier tokens of its own block only
 *                (Sec. 3.3, 3.6); heads concatenated, H = concat * Wo;
 *   summaries  : s = H wp, a = softmax of s over each block's tokens,
 *                S_i = sum_t a_t H[t] (Sec. 3.4);
 *   memory     : M_i = sum_{j<=i} g^(i-j) S_j / sum_{j<=i} g^(i-j), with the
 *                decay g in [0, 1) (written alpha in Sec. 3.5, fixed to 0.8
 *                there); P_i = M_i Wm; shifted by one block, C_1 = 0 and
 *                C_i = P_{i-1} (Sec. 3.5);
 *   injection  : every token of block i receives C_i (Sec. 3.7);
 *                G = sigmoid(H Wg), Y = H + G * C (Sec. 3.8).
 * With BCMT_FLAG_RESIDUAL the output is X + Y instead (for stacking layers;
 * the paper's layer output is Y).  There are no biases.
 *
 * Conventions
 *   - All tensors are row-major and live in device memory owned by the
 *     caller.  The layer entry points allocate nothing and create no streams
 *     or events; they keep no state between calls.
 *   - Activations X, Y, dY, dX are [B, T, D]; weights Wq, Wk, Wv, Wo, Wm, Wg
 *     are [D, D] input-major (y = x W; a torch Linear weight is the
 *     transpose), wp is [D].  They all have the element type cfg->dtype.
 *   - Weight and decay gradients are float32, with the same shapes.
 *   - Every pointer must be 16-byte aligned.
 *   - Work is enqueued on `stream` (a hipStream_t of the calling thread's
 *     current device; NULL means the default stream); nothing synchronises
 *     the host.  The backward passes may also take a caller-owned second
 *     stream (bcmt_side, below) for their weight-gradient products.
 *   - The GPU path needs a head width D / H of 64, 32 or 16 (the paper's
 *     model uses 16), D a multiple of 64 and D <= 2048.
 *
 * Errors
 *   Negative return values are bcmt_status codes.  All checks on the
 *   arguments happen before anything is enqueued, so BCMT_ERR_INVALID,
 *   BCMT_ERR_UNSUPPORTED and BCMT_ERR_WORKSPACE mean that nothing ran.
 *   BCMT_ERR_HIP reports a failed kernel launch; kernels enqueued before it
 *   may have run.
 *   On long sequences with few sequence x column slices the decayed scans
 *   of Sec. 3.5 pass partial sums between workgroups of one launch, all of
 *   which are resident at once.  Each wait for an earlier workgroup is
 *   bounded: one that runs out (only possible while other work holds the
 *   GPU that long) writes NaN into the outputs that depend on it instead
 *   of hanging, so a NaN there is the error report.
 */
#ifndef BCMT_H_
#define BCMT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BCMT_OK = 0,
  BCMT_ERR_INVALID = -1,     /* null or misaligned pointer, bad sizes, decay outside [0,1) */
  BCMT_ERR_UNSUPPORTED = -2, /* valid layer the GPU path does not run (head width not 16/32/64, D % 64, D > 2048) */
  BCMT_ERR_WORKSPACE = -3,   /* workspace smaller than bcmt_workspace_bytes() */
  BCMT_ERR_HIP = -4          /* a HIP launch failed */
} bcmt_status;

typedef enum { BCMT_F32 = 0, BCMT_BF16 = 1 } bcmt_dtype;

enum {
  BCMT_FLAG_RESIDUAL = 1,     /* Y = X + layer(X) */
  BCMT_FLAG_ACCUM_WGRAD = 2,  /* backward adds into the weight/decay gradients instead of overwriting */
  BCMT_FLAG_CHANNEL_DECAY = 4 /* one decay per feature channel: params->gamma_ch (see below) */
};

/* Passes for bcmt_workspace_bytes(). */
enum {
  BCMT_PASS_FORWARD = 0,   /* forward writing `saved` for a later backward */
  BCMT_PASS_INFERENCE = 1, /* forward with saved == NULL */
  BCMT_PASS_BACKWARD = 2
};

typedef struct {
  int32_t B;     /* sequences */
  int32_t T;     /* tokens per sequence */
  int32_t D;     /* features; on the GPU path D = H * dh with dh in {16, 32, 64} */
  int32_t H;     /* attention heads */
  int32_t L;     /* block size (L >= T gives a single block: dense causal attention) */
  float gamma;   /* memory decay, 0 <= gamma < 1 (0**0 is taken as 1) */
  int32_t dtype; /* bcmt_dtype: float32, or bfloat16 storage with float32 accumulation */
  int32_t flags; /* BCMT_FLAG_* */
} bcmt_config;

/* Per-channel decay (BCMT_FLAG_CHANNEL_DECAY): channel d of the memory runs
 * the recurrence of Sec. 3.5 with its own decay gamma_ch[d] in [0, 1) (the
 * paper uses one decay for all channels; cfg->gamma is then unused), and has
 * its own normaliser Z.  The backward writes the per-channel gradient to
 * dgamma_ch [D] (dgamma is not written); chunk states and their gradients
 * carry Z as [B, D].  The last member of each struct is read only with the
 * flag, so callers that never set it may use structs without it. */
typedef struct {
  const void *Wq, *Wk, *Wv, *Wo, *Wm, *Wg; /* [D, D] input-major, dtype */
  const void* wp;                          /* [D], dtype */
  const float* gamma_ch;                   /* [D] float32, with BCMT_FLAG_CHANNEL_DECAY */
} bcmt_params;

/* Float32 gradients.  A NULL member is not computed. */
typedef struct {
  float *dWq, *dWk, *dWv, *dWo, *dWm, *dWg; /* [D, D] */
  float* dwp;                               /* [D] */
  float* dgamma;                            /* scalar */
  float* dgamma_ch;                         /* [D], with BCMT_FLAG_CHANNEL_DECAY */
} bcmt_grads;

/* Optional second stream of the backward passes.  The weight-gradient
 * products (dWg, dWm, dwp, dWo, dWq, dWk, dWv), which no later step of the
 * pass reads, then run on side->stream beside the critical path: each is
 * ordered after its inputs on `stream` by recording side->fork on `stream`
 * and making side->stream wait for it, and before returning the pass records
 * side->join on side->stream and makes `stream` wait for it.  Work enqueued on
 * `stream` after the call therefore sees every output, exactly as if all of
 * it had run on `stream`.  The caller creates and owns the stream (same
 * device as `stream`, default priority) and the two events (timing may be
 * disabled), and must not use one bcmt_side in two calls that enqueue at the
 * same time.  Passing NULL runs everything on `stream`.  While stage tracing
 * is on, the second stream is not used. */
typedef struct {
  void* stream; /* hipStream_t */
  void* fork;   /* hipEvent_t, recorded on `stream` before each branch */
  void* join;   /* hipEvent_t, recorded on side->stream at the end */
} bcmt_side;

/* Optional helper: creates side->fork and side->join (side->stream is not
 * touched) on the calling thread's current device, with no timing and no
 * system-scope fence on record.  The fork and join only order two streams
 * of one device and the host never waits on them; an event recorded with
 * the default system-scope release writes back and invalidates the GPU's
 * caches between the kernels around it, which costs the critical path
 * several microseconds per record.  The caller owns the events and frees
 * them with bcmt_side_events_destroy.  Returns BCMT_OK, BCMT_ERR_INVALID
 * (side NULL) or BCMT_ERR_HIP (then nothing stays allocated and both
 * members are NULL). */
int bcmt_side_events_create(bcmt_side* side);

/* Destroys side->fork and side->join (NULL members are skipped) and sets
 * them to NULL.  The events must no longer be in use by enqueued work. */
int bcmt_side_events_destroy(bcmt_side* side);

/* Host-only check of a configuration; returns BCMT_OK or a negative status.
 * Makes no HIP call. */
int bcmt_validate(const bcmt_config* cfg);

/* Bytes of the `saved` buffer that forward fills and backward reads
 * (activations kept for the backward pass); 0 for an invalid config. */
size_t bcmt_saved_bytes(const bcmt_config* cfg);

/* Bytes of scratch workspace a pass needs (BCMT_PASS_*); 0 for an invalid
 * config.  The inference pass includes room for the activations that
 * `saved` would otherwise hold. */
size_t bcmt_workspace_bytes(const bcmt_config* cfg, int pass);

/* Forward pass (Sec. 3.2-3.8).
 *   X      [B, T, D] input, read only.
 *   params the seven weights, read only.
 *   Y      [B, T, D] output; must not overlap X.
 *   saved  bcmt_saved_bytes() bytes written for bcmt_layer_backward, or NULL
 *          for inference (then the workspace must hold BCMT_PASS_INFERENCE
 *          bytes).
 *   ws     scratch of at least bcmt_workspace_bytes(cfg, pass) bytes; its
 *          contents on entry are ignored and on exit are undefined. */
int bcmt_layer_forward(const bcmt_config* cfg, const void* X, const bcmt_params* params, void* Y,
                       void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward pass: gradients of sum(dY * Y) given the forward's `saved`.
 *   X      the forward input (read).
 *   saved  as written by bcmt_layer_forward with the same cfg, X and params.
 *   dY     [B, T, D] upstream gradient (read).
 *   dX     [B, T, D] input gradient (written), or NULL to skip it.
 *   grads  float32 weight/decay gradients (overwritten, or accumulated
 *          with BCMT_FLAG_ACCUM_WGRAD); NULL, or NULL members, skip them.
 *   ws     at least bcmt_workspace_bytes(cfg, BCMT_PASS_BACKWARD) bytes.
 *   side   a second stream for the weight-gradient products, or NULL
 *          (BCMT_ERR_INVALID if given without both events).
 * Every gradient is reduced in a fixed order, so repeated calls give the
 * same bits (the decay gradient from per-workgroup partials). */
int bcmt_layer_backward(const bcmt_config* cfg, const void* X, const bcmt_params* params,
                        const void* saved, const void* dY, void* dX, const bcmt_grads* grads,
                        void* ws, size_t ws_bytes, void* stream, const bcmt_side* side);

/* ---- Forward pass without allocation -------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid it.  The same forward
 * pass as bcmt_layer_forward, with its workspace taken from a device array
 * inside the library (BCMT_NOALLOC_SCRATCH_BYTES on each GPU, held from when
 * the library is loaded until the process ends) instead of a caller buffer.
 *   saved  required (bcmt_saved_bytes() bytes, caller-owned), as for a
 *          forward that a backward pass follows; inference uses it too.
 * Returns BCMT_ERR_WORKSPACE when the pass needs more scratch than the array
 * holds (bcmt_workspace_bytes(cfg, BCMT_PASS_FORWARD) above
 * BCMT_NOALLOC_SCRATCH_BYTES; the forward of B = 2, T = 65536, D = 1024 at
 * L = 256 needs 26 MiB), and BCMT_ERR_HIP if the array's address cannot be
 * obtained; other errors as for bcmt_layer_forward.  The call allocates
 * nothing and creates nothing.  Every call on one GPU uses that GPU's one
 * array: calls whose work overlaps on the GPU (several streams, or several
 * host threads) race on it and must be ordered by the caller. */
#define BCMT_NOALLOC_SCRATCH_BYTES (32u << 20)
int bcmt_layer_forward_noalloc(const bcmt_config* cfg, const void* X, const bcmt_params* params,
                               void* Y, void* saved, void* stream);

/* ---- Chunked execution ---------------------------------------------------
 * Only the memory of Sec. 3.5 crosses block boundaries, through the decayed
 * recurrence over blocks; attention, pooling and the gate stay inside a
 * block.  A sequence cut at block boundaries into consecutive chunks can
 * therefore run chunk by chunk, each call continuing the recurrence from the
 * state left by the blocks before it:
 *   N = sum_j g^(k-j) S_j,   Z = sum_j g^(k-j)   (j <= k, k the last block),
 * float32 in device memory.  The chunk's first block receives the memory
 * N / Z of the earlier blocks, projected by Wm, exactly as if the previous
 * chunk's last block preceded it in one call.  Z = 0 stands for an empty
 * history (the start of the sequences): the first block then receives 0,
 * and N must be 0.  Chaining chunks gives the whole-sequence layer when
 * every chunk except the last holds a multiple of L tokens (otherwise a
 * block would be cut in two).  Sequences of the batch may be at different
 * positions: Z is per sequence. */
typedef struct {
  float* N; /* [B, D] */
  float* Z; /* [B], or [B, D] with BCMT_FLAG_CHANNEL_DECAY */
} bcmt_carry;

/* Forward pass of one chunk.
 *   carry_in   state after the earlier blocks (read), or NULL for an empty
 *              history.
 *   carry_out  receives the state after the chunk's last block, or NULL.
 *              It may use the same buffers as carry_in (the incoming state
 *              is copied into `saved` before anything is written).
 * A carry given must have both members, N 16-byte and Z 4-byte aligned.
 * The other arguments are those of bcmt_layer_forward, with the same
 * workspace and `saved` sizes; `saved` written here is for
 * bcmt_layer_backward_chunk (bcmt_layer_backward would drop the incoming
 * state's contribution). */
int bcmt_layer_forward_chunk(const bcmt_config* cfg, const void* X, const bcmt_params* params,
                             const bcmt_carry* carry_in, void* Y, const bcmt_carry* carry_out,
                             void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward pass of one chunk, given the `saved` of bcmt_layer_forward_chunk:
 * gradients of sum(dY * Y) + sum(dN * N_out) + sum(dZ * Z_out), where
 * (N_out, Z_out) is the chunk's outgoing state and (dN, dZ) = *dcarry_out.
 *   dcarry_out  gradient arriving for the outgoing state (read), or NULL
 *               for none (the last chunk).
 *   dcarry_in   receives the gradient of the incoming state, or NULL.  It
 *               may use the same buffers as dcarry_out.
 * grads->dgamma includes the decay's effect through the incoming state's
 * first block.  Running the chunks' backward passes from the last to the
 * first, each given the dcarry_in of the chunk after it, with
 * BCMT_FLAG_ACCUM_WGRAD from the second call on, yields the gradients of
 * the whole sequence. */
int bcmt_layer_backward_chunk(const bcmt_config* cfg, const void* X, const bcmt_params* params,
                              const void* saved, const void* dY, const bcmt_carry* dcarry_out,
                              void* dX, const bcmt_carry* dcarry_in, const bcmt_grads* grads,
                              void* ws, size_t ws_bytes, void* stream, const bcmt_side* side);

/* ---- Incremental decoding ------------------------------------------------
 * The layer is causal (Sec. 3.6): the output of token t of block i depends
 * on the tokens of block i up to t (Sec. 3.3) and on the context C_i, which
 * the earlier blocks fix (Sec. 3.5, 3.7).  The decoder produces the layer's
 * output one token at a time for B sequences in step, from a decode state
 * that holds, per sequence, the current block's keys, values and local
 * outputs H (compute type), their pooling scores, the memory state (N, Z)
 * and the current block's context C (float32).  When a block's last token
 * has been decoded, the block's summary enters the memory and the next
 * block's context is formed, as in the layer.  Token by token, the outputs
 * equal those of bcmt_layer_forward over the whole sequence.
 *
 * cfg gives B, D, H, L, gamma, dtype and the residual flag (T is not used);
 * the decoder also needs L <= 4096, B <= 64 and heads of 64 dimensions
 * (else BCMT_ERR_UNSUPPORTED).
 * The state and the workspace are caller-owned device buffers of the sizes
 * below (0 for an unsupported config); the workspace is scratch. */
size_t bcmt_decode_state_bytes(const bcmt_config* cfg);
size_t bcmt_decode_workspace_bytes(const bcmt_config* cfg);

/* Starts decoding at a block boundary.  carry_in: the memory state after the
 * blocks already processed (for example the carry_out of
 * bcmt_layer_forward_chunk over a prompt of whole blocks), or NULL to start
 * a sequence.  Reads params->Wm only (the context (N / Z) Wm of the first
 * block); the other params members may be NULL. */
int bcmt_decode_reset(const bcmt_config* cfg, const bcmt_params* params,
                      const bcmt_carry* carry_in, void* state, void* ws, size_t ws_bytes,
                      void* stream);

/* Decodes one token per sequence.
 *   t  index of the token counted from the last reset (0, 1, 2, ...); the
 *      caller passes consecutive values, each once.  Token t sits at
 *      position t mod L of its block; t mod L == L - 1 completes the block.
 *   x  [B, D] the new token's layer input (dtype), read.
 *   y  [B, D] its layer output (dtype), written; must not overlap x.
 * The enqueued work allocates nothing and has a fixed launch sequence for a
 * given t mod L (suitable for capture in a HIP graph per position). */
int bcmt_decode_step(const bcmt_config* cfg, const bcmt_params* params, int64_t t,
                     const void* x, void* y, void* state, void* ws, size_t ws_bytes,
                     void* stream);

/* Static description of a status code. */
const char* bcmt_strerror(int status);

/* Library version, major * 10000 + minor * 100 + patch (2.1.0: helpers
 * that create and destroy a bcmt_side's events). */
int bcmt_version(void);

/* ---------------------------------------------------------------- language model
 * A decoder-only language model built from BCMT layers: the architecture of
 * the paper's experiments (Sec. 4.1 fixes d_model, layers, heads and batch;
 * the other parts are read as a pre-LN decoder of the period):
 *   x = E[tok] + Pe[t];  per layer x += mix(LN1(x)); x += gelu(LN2(x) W1) W2
 *   (hidden 4d, GELU in tanh form, no biases); logits = LNf(x) E^T (head tied
 *   to the embedding); loss = mean cross-entropy over all B T positions.
 * mix is the BCMT layer above (bf16, no residual flag, decay fixed); with
 * L >= T it is plain causal attention, the paper's Dense baseline.
 * LayerNorm has gain and bias, eps 1e-5.  bf16 only.
 *
 * Parameters live in one flat vector (float32 master copy `params`, its
 * bf16 working copy `params_bf16`, float32 `grads`, AdamW moments), arrays
 * back to back in this order (every length is a multiple of 64 elements):
 *   0  E  [Vp, d]  (Vp = V rounded up to a multiple of 128; rows V..Vp-1 are
 *                   never read as tokens and their logits are masked)
 *   1  Pe [T, d]
 *   2 + 13 l + k, layer l:  k = 0 ln1_g, 1 ln1_b [d]; 2..7 Wq, Wk, Wv, Wo,
 *                   Wm, Wg [d, d]; 8 wp [d]; 9 ln2_g, 10 ln2_b [d];
 *                   11 W1 [d, 4d]; 12 W2 [4d, d]   (input-major: y = x W)
 *   2 + 13 n_layer, +1:  lnf_g, lnf_b [d]
 * Weights are input-major as in the layer.  Gradients of every array are
 * written (not accumulated); E's gradient adds the tied head's and the
 * lookups' parts, the latter with float32 atomics (rows sharing a token add
 * in any order, so E's gradient may differ between runs by rounding).
 * Values below the stated minimums give BCMT_ERR_INVALID; d, V or B T
 * beyond the GPU path's limits give BCMT_ERR_UNSUPPORTED. */
typedef struct {
  int32_t V;       /* vocabulary size, 2 ..= 65536 */
  int32_t d;       /* model width: a multiple of 64, at most 1024 */
  int32_t H;       /* heads of each BCMT layer (d / H in {16, 32, 64}) */
  int32_t n_layer; /* >= 1 */
  int32_t B, T;    /* sequences per step and tokens per sequence; B T >= 8 */
  int32_t L;       /* block size of the layers (L >= T: the Dense model) */
  float gamma;     /* memory decay of the layers (fixed, not trained) */
} bcmt_model_config;

/* AdamW: p *= 1 - lr wd; m = b1 m + (1 - b1) g; v = b2 v + (1 - b2) g^2;
 * p -= lr (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps). */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
  int32_t step; /* 1 for the first update */
} bcmt_adamw;

/* Floats in the flat parameter vector; 0 for an invalid config. */
size_t bcmt_model_param_count(const bcmt_model_config* cfg);
/* Offset and length (in elements) of array `index` of the flat vector. */
int bcmt_model_param_array(const bcmt_model_config* cfg, int index, size_t* offset,
                           size_t* count);
/* Bytes of scratch workspace bcmt_model_train_step needs; 0 if invalid. */
size_t bcmt_model_workspace_bytes(const bcmt_model_config* cfg);
/* params_bf16 = bf16(params), the whole vector (enqueued on `stream`). */
int bcmt_model_cast(const bcmt_model_config* cfg, const float* params, void* params_bf16,
                    void* stream);
/* One training step on `stream`: forward over tokens [B, T] (int32, ids in
 * [0, V); others are clamped) with next-token targets [B, T], the mean
 * cross-entropy into *loss (device float), the backward into grads, and
 * with `opt` an AdamW update of params, adam_m, adam_v (all float32,
 * param_count long) that also rewrites params_bf16.  Without `opt` only
 * the gradients are computed (adam_m, adam_v may be NULL).  The forward
 * reads params_bf16 (weights) and params (LayerNorm gains and biases).
 * All pointers are device memory, 16-byte aligned; ws holds at least
 * bcmt_model_workspace_bytes(cfg).  `side` is passed to each layer's
 * backward pass (NULL: everything on `stream`).  Errors as for the layer. */
int bcmt_model_train_step(const bcmt_model_config* cfg, const int32_t* tokens,
                          const int32_t* targets, float* params, void* params_bf16,
                          float* grads, float* adam_m, float* adam_v, const bcmt_adamw* opt,
                          float* loss, void* ws, size_t ws_bytes, void* stream,
                          const bcmt_side* side);

/* ---- Stage tracing (profiling aid) -------------------------------------
 * While tracing is on, every kernel launch of bcmt_layer_forward and
 * bcmt_layer_backward is bracketed by two HIP events recorded on the call's
 * stream, so each stage's GPU time is measured in place.  While tracing is
 * on, the backward pass also keeps its weight-gradient products on the
 * call's stream instead of a second stream, so that every stage is timed
 * alone.  The timing events (a fixed pool of 16384) are created by
 * bcmt_trace_enable on the current device and reused; a launch that finds
 * the pool exhausted (too many launches between two reads) is not timed.  Stage names are static strings such as "fwd.qkv_gemm" or
 * "bwd.attention_dkdv". */
typedef struct {
  const char* name; /* static string */
  int32_t calls;    /* launches recorded since the last read */
  double total_ms;  /* summed GPU time of those launches */
} bcmt_trace_entry;

/* Turns tracing on (nonzero) or off; returns the previous setting. */
int bcmt_trace_enable(int on);

/* Waits for every recorded launch to finish, writes up to max_entries
 * per-stage totals (stages with at least one launch, in pipeline order),
 * clears them, and returns how many stages had launches (which may exceed
 * max_entries), or a negative status. */
int bcmt_trace_read(bcmt_trace_entry* out, int max_entries);

#ifdef __cplusplus
}
#endif

#endif /* BCMT_H_ */
