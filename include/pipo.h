/*
 * pipo.h - C ABI of the MI355X (gfx950) PIPO pair-in/pair-out library.
 *
 * PIPO (Pair-In, Pair-Out) decodes a token *pair* per backbone step (Sec. 3.1):
 *   1. pair-in compressor   z = W_c [E[a]; E[b]] + b_c            (eq. 1, App. B.1 Linear)
 *   2. backbone over latents h_b = Backbone(z^{<=i})              (eq. 2)
 *   3. backbone token        b  ~ LMHead(RMSNorm(h_b))             (eq. 3, tied head)
 *   4. MTP head + draft      h_d = W_fc[RMSNorm(h_b); RMSNorm(E[b])], d ~ LMHead(RMSNorm(h_d))
 *                                                                  (eqs. 4-5, App. B.2, one linear)
 *   5. confidence gate       c = sigmoid(w_c . RMSNorm([h_b; h_d])); accept iff c >= tau
 *                            next input pair = accept ? (b, d) : (b, PAD)   (eq. 6, Sec. 3.2)
 * Every step consumes exactly one latent position and emits one or two
 * tokens; the prompt is compressed two tokens per latent (ceil(n/2) latents,
 * PAD at the odd slot of an odd-length prompt).
 *
 * Conventions for every call:
 *   - Pointers named d_* are device pointers (hipMalloc'd or torch CUDA
 *     tensors' data_ptr()); the caller owns them.  Other pointers are host.
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *     Every call is stream-ordered and asynchronous: outputs are valid once
 *     the caller synchronises that stream.  One context must not be used
 *     from two threads at once.
 *   - Return value: PIPO_OK (0) or a negative PIPO_E* code.  Host-side
 *     argument and capacity checks run before any device work, so a failed
 *     call leaves the context unchanged.  A device fault from earlier work
 *     surfaces as PIPO_EHIP.  Nothing aborts; no C++ exception crosses the ABI.
 *   - pipo_last_error() returns the message of the most recent failure.
 *   - Debugging: with PIPO_CHECK=1 in the environment when a context is
 *     created, that context launches every kernel eagerly (no HIP graph),
 *     waits for the stream after each one, and returns the first failure as
 *     PIPO_EHIP with its launch site in pipo_last_error().
 *   - Decode attention merges its key splits through the L2 of the XCD they
 *     ran on when a probe at context creation finds workgroups placed on the
 *     eight XCDs in turn; PIPO_NO_XCD_MERGE=1 at creation keeps the separate
 *     merge launch (same results up to rounding order).
 */
#ifndef PIPO_H
#define PIPO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PIPO_OK          0
#define PIPO_EINVAL     -1   /* bad argument or unsupported shape            */
#define PIPO_ENOMEM     -2   /* device allocation failed                     */
#define PIPO_EHIP       -3   /* HIP runtime error (incl. earlier faults)     */
#define PIPO_ECAPACITY  -4   /* batch or latent KV capacity exceeded         */
#define PIPO_ESTATE     -5   /* decode before prefill                        */

typedef struct pipo_ctx pipo_ctx;   /* opaque; owns weights, KV cache, workspaces */

/* Model shape and capacities.  Constraints (PIPO_EINVAL otherwise):
 * hidden % 32 == 0, ffn % 32 == 0, vocab % 16 == 0, head_dim in {64, 128},
 * n_q_heads % n_kv_heads == 0 and n_q_heads / n_kv_heads <= 16,
 * (n_q_heads*head_dim) % 32 == 0, 1 <= max_batch <= 64, max_latent >= 1,
 * prefill_chunk >= 1. */
typedef struct {
    int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
    float   rope_base;       /* RoPE frequencies base^(-2j/d) over latent positions */
    float   rms_eps;         /* RMSNorm epsilon                                     */
    int32_t pad_id;          /* PAD token id; -1 selects vocab-1                    */
    int32_t max_batch;       /* sequences per context                               */
    int32_t max_latent;      /* KV capacity per sequence, in latent positions       */
    int32_t prefill_chunk;   /* latent positions per prefill chunk (e.g. 4096)      */
    int32_t gain_mode;       /* 0: RMSNorm gains 1; 1: gains 1 + 10*w (testing)     */
    int32_t heads;           /* 0: one-linear compressor, MTP and confidence heads;
                                else PIPO_HEADS_* flags for the App. B forms         */
} pipo_config;

/* The App. B forms of the three heads (pipo_config.heads):
 * MLP compressor (Table 4): z = E[a] + E[b] + W2 SiLU(W1 [E[a]; E[b]]), W1 2H->H,
 *   W2 H->H (the printed W2 SiLU(W1 .) is the residual branch of an a + b path);
 * MTP layer (App. B.2): h_d = Layer(W_fc [RMSNorm(h_b); RMSNorm(E[b])]), Layer a
 *   decoder layer shaped like the backbone's with its own KV cache over latent
 *   positions; during prefill the prompt's latents other than the last take the
 *   prompt token after their pair;
 * MLP confidence (App. B.3): c = sigmoid(w2 . SiLU(W1 RMSNorm([h_b; h_d]))), W1 2H->H. */
#define PIPO_HEADS_MLP_COMPRESSOR  1
#define PIPO_HEADS_MTP_LAYER       2
#define PIPO_HEADS_MLP_CONFIDENCE  4

/* Token selection and the confidence gate (Sec. 3.2).  Read during the call,
 * not retained except by value. */
typedef struct {
    float tau;               /* accept the draft iff sigmoid(s) >= tau             */
    float temperature;       /* <= 0: greedy argmax, ties to the lowest id          */
    float top_p;             /* nucleus mass in (0, 1]; used when temperature > 0   */
    const uint64_t *seeds;   /* host [batch] per-sequence sampler seeds; may be NULL
                                when greedy                                          */
    int32_t top_k;           /* sampling only: keep the tokens whose logit is at
                                least the k-th largest (ties kept); 0 or >= vocab
                                = off; negative: PIPO_EINVAL                        */
    float rep_penalty;       /* sampling only, > 0: logits of penalised tokens are
                                divided by it when positive, multiplied otherwise
                                (1 = off)                                           */
} pipo_sampling;
/* With top_k > 0 or rep_penalty != 1, selection is the evaluation sampler of
 * Sec. 4: repetition penalty, temperature, top-k, then top-p over the kept
 * tokens, drawn as in the plain top-p sampler.  The penalised tokens of a
 * sequence are its prompt's tokens and every token a decode step took as
 * input (the first of the pair, and the second unless PAD); the draft of a
 * pair also penalises that pair's backbone token.  Under greedy decoding
 * (temperature <= 0) top_k must be 0 and rep_penalty 1 (else PIPO_EINVAL). */

/* One pair step's result for one sequence (16 bytes). */
typedef struct {
    int32_t tok_b;           /* backbone token x^{2i+2}                            */
    int32_t tok_d;           /* draft token x^{2i+3}                               */
    float   conf;            /* confidence c^i = sigmoid(s)                         */
    int32_t accept;          /* 1 iff conf >= tau: the draft is emitted             */
} pipo_pair;

/* The model of Sec. 3.1: the pair-in compressor (eq. 1; App. B.1 Table 4), the
 * backbone (eq. 2), the tied LM head (eq. 3), the MTP head (eqs. 4-5; App.
 * B.2) and the confidence head (eq. 6; App. B.3).
 * Create a context: allocate weights, KV cache and workspaces on the current
 * device and fill every weight tensor from the counter-based generator
 * (SplitMix64-derived, N(0, 0.02)-shaped, bf16 storage) for `seed`.
 * On success *out receives the context (released by pipo_free).  Returns
 * PIPO_EINVAL for a bad config, PIPO_ENOMEM if device memory runs out. */
int pipo_init_weights(const pipo_config *cfg, uint64_t seed, void *stream, pipo_ctx **out);

/* Compressed-prompt prefill (Sec. 4.3 TTFT path): start `batch` new
 * sequences from d_tokens (device int32 [batch][n], row-major, ids in
 * [0, vocab)), pair them (PAD appended to an odd n), run the backbone over
 * the ceil(n/2) latents in chunks of prefill_chunk, and emit the first pair:
 * d_out (device pipo_pair [batch]).  d_logits_b / d_logits_d (device float
 * [batch][vocab]) receive the backbone / draft logits when non-NULL.
 * Errors: PIPO_EINVAL (NULL pointers, n < 1, bad sampling values),
 * PIPO_ECAPACITY (batch > max_batch or ceil(n/2) + 1 > max_latent). */
int pipo_prefill(pipo_ctx *ctx, int32_t batch, const int32_t *d_tokens, int32_t n,
                 const pipo_sampling *smp, pipo_pair *d_out,
                 float *d_logits_b, float *d_logits_d, void *stream);

/* Ragged batch (the serving shape of Sec. 4: requests of different prompt
 * lengths decoded together): as pipo_prefill, but sequence i's prompt is the
 * first lens[i] tokens of row i of d_tokens (device int32 [batch][stride]),
 * lens a host int32 [batch] array read before the call returns, each in
 * [1, stride].  Sequence i gets ceil(lens[i]/2) latents; its pair steps then
 * run at its own positions.  Errors: as pipo_prefill, PIPO_EINVAL for a NULL
 * lens or a length outside [1, stride], PIPO_ECAPACITY when the longest
 * prompt's latents + 1 exceed max_latent. */
int pipo_prefill_ragged(pipo_ctx *ctx, int32_t batch, const int32_t *d_tokens, int32_t stride,
                        const int32_t *lens, const pipo_sampling *smp, pipo_pair *d_out,
                        float *d_logits_b, float *d_logits_d, void *stream);

/* The pair-in, pair-out step of Sec. 3.2 (eqs. 1-6: compress the input pair,
 * one backbone position, backbone token, MTP draft, confidence gate).
 * One pair-decode step for every sequence of the last prefill.  The input
 * pair is d_in_pairs (device int32 [batch][2]) when non-NULL (teacher
 * forcing), else the pair the previous call produced on the device:
 * (tok_b, accept ? tok_d : pad_id).  Appends one latent per sequence.
 * Outputs as for pipo_prefill.  Errors: PIPO_ESTATE (no prefill yet),
 * PIPO_ECAPACITY (KV full). */
int pipo_decode_step(pipo_ctx *ctx, const int32_t *d_in_pairs, pipo_pair *d_out,
                     float *d_logits_b, float *d_logits_d, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops): pipo_decode_step with the same arguments,
 * outputs and errors, launched eagerly on `stream` (no HIP graph is built or
 * instantiated) and with its scratch (the decode attention's split partials
 * and the larger-batch GEMVs' k-range partial sums) in a 16 MiB device array
 * of the library, one per GPU, held until the process ends.  It calls no
 * hipMalloc or hipFree.  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (two streams, or two contexts on two host
 * threads) race and must be serialised by the caller.  Nothing in the array
 * needs to start at zero (each call writes the partials it reads).  Errors
 * as pipo_decode_step, plus PIPO_ECAPACITY when the attention partials
 * (batch * n_q_heads * splits * (head_dim + 2) floats, splits <= 64) exceed
 * the array; k-range partials that do not fit its remainder make those
 * GEMVs run their whole-K form instead.  Profiling (pipo_profile_enable)
 * does not time this call. */
int pipo_decode_step_noalloc(pipo_ctx *ctx, const int32_t *d_in_pairs, pipo_pair *d_out,
                             float *d_logits_b, float *d_logits_d, void *stream);

/* Regular one-token-per-step decoding on the same weights: the baseline the
 * pair decoder is compared against (Sec. 4.3, Fig. 4: the backbone itself,
 * one position per token, no compressor, MTP or confidence head).
 * pipo_regular_prefill starts `batch` sequences from d_tokens (device int32
 * [batch][n], row-major, ids in [0, vocab)) with the n embeddings as the
 * backbone's positions and writes the first generated token to d_tok
 * (device int32 [batch]); d_logits (device float [batch][vocab]) receives
 * its logits when non-NULL.  Selection as in pipo_sampling (tau unused;
 * top-p draws use slot 0 of each step).  A later pipo_decode_step needs a
 * new pipo_prefill.  Errors: PIPO_EINVAL (NULL pointers, n < 1, bad
 * sampling values), PIPO_ECAPACITY (batch > max_batch or n + 1 > max_latent). */
int pipo_regular_prefill(pipo_ctx *ctx, int32_t batch, const int32_t *d_tokens, int32_t n,
                         const pipo_sampling *smp, int32_t *d_tok, float *d_logits,
                         void *stream);

/* Ragged regular prefill: as pipo_regular_prefill with sequence i's prompt
 * the first lens[i] tokens of row i of d_tokens ([batch][stride]); lens as in
 * pipo_prefill_ragged. */
int pipo_regular_prefill_ragged(pipo_ctx *ctx, int32_t batch, const int32_t *d_tokens, int32_t stride,
                                const int32_t *lens, const pipo_sampling *smp, int32_t *d_tok,
                                float *d_logits, void *stream);

/* One regular decoding step: feed one token per sequence, append one
 * position, emit the next token.  The input is d_in_tok (device int32
 * [batch]) when non-NULL (teacher forcing), else the token the previous
 * call produced on the device.  Outputs as for pipo_regular_prefill.
 * Errors: PIPO_ESTATE (no regular prefill yet), PIPO_ECAPACITY (KV full). */
int pipo_regular_step(pipo_ctx *ctx, const int32_t *d_in_tok, int32_t *d_tok, float *d_logits,
                      void *stream);

/* ---- OPD training targets (App. C; no context needed) ---------------------
 * pipo_opd_teacher_rows: PAD compaction of the teacher pass.  For a
 * trajectory d_tokens (device int32 [T]) whose PADs the teacher never saw,
 * d_rows[t] (device int32 [T]) = (number of non-PAD tokens in tokens[0..t])
 * - 1: the teacher row of the last non-PAD position at or before t (-1 where
 * there is none).  Errors: PIPO_EINVAL (NULL pointers, T < 0).
 *
 * pipo_opd_targets: for each position t < T with label y = d_labels[t] >= 0,
 *   d_kl[t]    = log p_s(y) - log p_t(y), the sampled reverse-KL term,
 *   d_alpha[t] = exp(-max(d_kl[t], 0)) = min(p_t(y) / p_s(y), 1), the
 *                confidence head's target,
 * with p_s = softmax(d_logits_s[t]) (device float [T][V]) and p_t =
 * softmax(d_logits_t[r]) (device float [Tt][V]), r = d_teacher_rows[t]
 * (device int32 [T]; NULL: r = t).  Positions with a negative label are not
 * scored (kl 0, alpha 1); a scored position whose row is outside [0, Tt) or
 * whose label is >= V gets NaN.  When d_sums (device double [4]) is
 * non-NULL it receives {sum of kl, count} over the scored even positions
 * (backbone head), then over the odd ones (MTP head), added in a fixed
 * order.  The paper calls this per chunk of up to 2048 positions; T = 0 is
 * allowed (the arrays may then be NULL).  Errors: PIPO_EINVAL (NULL pointers
 * with T > 0, T < 0, V or Tt < 1, V not a multiple of 4, logit arrays not
 * 16-byte aligned), PIPO_EHIP (launch failure). */
int pipo_opd_teacher_rows(const int32_t *d_tokens, int32_t T, int32_t pad_id, int32_t *d_rows, void *stream);
int pipo_opd_targets(int32_t T, int32_t V, const float *d_logits_s, const float *d_logits_t, int32_t Tt,
                     const int32_t *d_teacher_rows, const int32_t *d_labels, float *d_kl, float *d_alpha,
                     double *d_sums, void *stream);
/* As pipo_opd_targets, with bf16 logit rows (device uint16 bit patterns,
 * [T][V] and [Tt][V], 8-byte aligned); the arithmetic is the same fp32. */
int pipo_opd_targets_bf16(int32_t T, int32_t V, const uint16_t *d_logits_s, const uint16_t *d_logits_t, int32_t Tt,
                          const int32_t *d_teacher_rows, const int32_t *d_labels, float *d_kl, float *d_alpha,
                          double *d_sums, void *stream);

/* Release a context made by pipo_init_weights and all its device memory.
 * NULL is a no-op (returns 0). */
int pipo_free(pipo_ctx *ctx);

/* Error reporting of this ABI (no passage of the paper): message of the most
 * recent failure on ctx (or of pipo_init_weights when ctx is NULL).  Never NULL; valid until the next call on the same context. */
const char *pipo_last_error(const pipo_ctx *ctx);

/* Testing aid (no passage of the paper): read the weights of the Sec. 3.1
 * model back in logical layout.
 * Copy `count` elements, starting at logical element `start` of the
 * row-major [out][in] tensor `name` (e.g. "embed", "w_comp", "l3.wq",
 * "l0.g_attn"), to host memory as bf16 bit patterns, undoing the device
 * packing.  Synchronous.  For verifying the device weight generator.
 * Errors: PIPO_EINVAL (unknown name or range). */
int pipo_read_weight(pipo_ctx *ctx, const char *name, int64_t start, int64_t count,
                     uint16_t *host_out);

/* Kernel classes of the profiling counters. */
#define PIPO_K_GEMV_LAYER   0   /* decode weight-streaming GEMM: QKV, O, gate/up, down */
#define PIPO_K_GEMV_LMHEAD  1   /* decode LM-head GEMM (both passes), argmax fused     */
#define PIPO_K_GEMV_SMALL   2   /* decode compressor, MTP and confidence GEMMs        */
#define PIPO_K_ATTN_DECODE  3   /* split-K flash-decode (merge included)               */
#define PIPO_K_SAMPLE       4   /* top-p sampler                                       */
#define PIPO_K_GATE         5   /* gate + next pair or token; step-input embeddings    */
#define PIPO_K_PREFILL_GEMM 6   /* prefill MFMA GEMMs                                  */
#define PIPO_K_PREFILL_ATTN 7   /* prefill causal flash attention                      */
#define PIPO_K_PREFILL_MISC 8   /* prefill gather, RMSNorm, last-latent pick           */
#define PIPO_K_CLASSES      9

/* Measurement aid (no passage of the paper; it times the kernels of Sec. 3.2
 * and Sec. 4.3).
 * Profiling: while on (on != 0), the prefill and step calls of both decoders launch
 * eagerly (no graph) with a HIP event recorded on the call's stream before
 * and after every kernel; durations accumulate per kernel class.  Turning it
 * on clears the accumulators.  Errors: PIPO_EINVAL (NULL ctx). */
int pipo_profile_enable(pipo_ctx *ctx, int on);

/* Measurement aid, as pipo_profile_enable.
 * Synchronise the pending profiling events and return, for kernel class
 * `kclass` (PIPO_K_*), the summed duration in milliseconds and the number of
 * launches since profiling was turned on.  Errors: PIPO_EINVAL. */
int pipo_profile_read(pipo_ctx *ctx, int kclass, double *total_ms, int64_t *launches);

/* Measurement aids (no passage of the paper; they compute nothing of the
 * method).  They give the attainable ceilings that the kernels of Sec. 3.2
 * and Sec. 4.3 are compared with.  Both are synchronous: they launch one
 * untimed and then `reps` timed back-to-back launches on `stream` and wait.
 *
 * pipo_calibrate_stream: each launch reads `bytes` of the device buffer
 * d_buf (`buf_bytes` long) with the decode GEMV's weight-stream pattern (one
 * contiguous 1 KB tile per wave load, 16 bytes per lane, nontemporal; two
 * batches of five tiles in flight per wave; 256 workgroups of eight waves).
 * Launch r reads the window starting at 1 KB tile (r * bytes/1024) mod
 * ((buf_bytes - bytes)/1024 + 1), so with buf_bytes well above the caches
 * (256 MB memory-side cache, 4 MB L2 per XCD) every launch reads from HBM.
 * *us = mean microseconds per launch.  The buffer is only read; its contents
 * do not matter.  Errors: PIPO_EINVAL (NULL pointer, bytes < 1024 or not a
 * multiple of 1024, buf_bytes < bytes, reps < 1), PIPO_ENOMEM, PIPO_EHIP.
 *
 * pipo_calibrate_mfma: issue rate of v_mfma_f32_16x16x32_bf16 with register
 * operands, as the prefill GEMM issues them (a 4 x 4 block of independent
 * accumulators per wave).  `waves_per_simd` (1, 2 or 4) waves run on every
 * SIMD of every compute unit, each `iters` rounds of 16 MFMAs on eight
 * operand registers loaded once from d_operands (at least 8 KB, bf16 bit
 * patterns the caller chooses: random data draws more power than zeros).
 * *tflops = 16384 flops per MFMA over the mean launch time.
 * Errors: PIPO_EINVAL, PIPO_ENOMEM, PIPO_EHIP. */
int pipo_calibrate_stream(const void *d_buf, int64_t buf_bytes, int64_t bytes, int32_t reps, double *us,
                          void *stream);
int pipo_calibrate_mfma(const void *d_operands, int32_t waves_per_simd, int32_t iters, int32_t reps,
                        double *tflops, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* PIPO_H */
