/*
 * tppsd.h - C ABI of the TPP-SD sampling hot path on MI355X (gfx950).
 *
 * TPP-SD ("speculative decoding for Transformer temporal point processes")
 * samples event sequences from a CDF-based Transformer TPP (the target model,
 * paper §4.2) by letting a smaller draft model propose gamma events that the
 * target scores in one parallel pass, then accepting a prefix and replacing
 * the first rejected event from an adjusted distribution (paper §4.3,
 * Algorithm 1, Theorem 1). The output law is that of naive autoregressive
 * sampling from the target (§4.2, App. A.2).
 *
 * Model (both target and draft, §4.2 "Encoder"/"Decoder", App. D.4):
 *   x_i = z(t_i) + W_type[k_i]          z_j(t) = sin / cos(t * 10000^-(j - j mod 2)/D)
 *   L pre-LN blocks: x += Wo MHA(LN1 x) + bo ; x += W2 relu(W1 LN2 x + b1) + b2
 *   h = LNf(x);  e = E h;  w = softmax(Vw e1 + bw);  mu = Vmu e2 + bmu;
 *   s = log sigma = Vsig e3 + bsig;  f = softmax(Vk2 tanh(Vk1 h + bk1) + bk2)
 *   The decoder at event i gives the law of event i+1: interval
 *   tau ~ sum_m w_m LogNormal(mu_m, sigma_m), type k ~ f.
 *
 * Conventions
 *   - Every pointer argument named d_* is a device pointer owned by the
 *     caller; the library never allocates or frees device memory. All
 *     device work is enqueued on the given stream and is asynchronous;
 *     buffers must stay alive until the stream has drained.
 *   - Arrays are row-major and batch-major: [B, ...]. Times are float32
 *     absolute times, types are int32 in [0, K). Mixture parameters are
 *     stored per position as [3, M] = (log w, mu, log sigma).
 *   - Every function returns a status; TPPSD_OK (0) on success. Argument
 *     and ordering errors are detected on the host before anything is
 *     enqueued; tppsd_last_error() then describes the failure (per thread).
 *   - Conditions found on the device (KV capacity, non-finite density,
 *     acceptance-rejection cap) set sticky bits read by tppsd_state_status.
 *   - One host thread at a time may use a state; a model may be shared.
 */
#ifndef TPPSD_H
#define TPPSD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define TPPSD_OK          0
#define TPPSD_E_ARG       1   /* null pointer, size or gamma out of range      */
#define TPPSD_E_CONFIG    2   /* unsupported model configuration               */
#define TPPSD_E_WORKSPACE 3   /* workspace too small or misaligned             */
#define TPPSD_E_ORDER     4   /* call out of order (e.g. verify before prefill) */
#define TPPSD_E_HIP       5   /* HIP runtime error; message names it           */

/* ---- precisions ---------------------------------------------------------- */
#define TPPSD_PREC_FP32 0     /* fp32 weights and activations                  */
#define TPPSD_PREC_BF16 1     /* bf16 matrices and Linear inputs, fp32 accumulate,
                                 fp32 residual stream, statistics and decoder math */

/* ---- state flags ----------------------------------------------------------- */
#define TPPSD_FLAG_BONUS 1u   /* all gamma drafts accepted -> one extra event from
                                 the target's next distribution (the extra target
                                 distribution of §2.3). Off: the round yields the
                                 gamma drafts (Algorithm 1 as printed).          */

/* ---- sticky device status bits (tppsd_state_status) ----------------------- */
#define TPPSD_STATUS_CAPACITY  1u  /* an append would pass max_events           */
#define TPPSD_STATUS_NONFINITE 2u  /* a log-density or sampled interval was NaN/Inf */
#define TPPSD_STATUS_AR_CAP    4u  /* Theorem-1 loop hit TPPSD_AR_ITER_CAP        */

#define TPPSD_AR_ITER_CAP (1 << 20)

/* ---- limits ------------------------------------------------------------------ */
#define TPPSD_MAX_GAMMA  32   /* draft length per round                          */
#define TPPSD_MAX_MIX    64   /* mixture components M                            */
#define TPPSD_MAX_TYPES  64   /* event types K                                   */

/* ---- encoders ---------------------------------------------------------------- */
#define TPPSD_ENC_THP    0    /* the model described above                      */
#define TPPSD_ENC_ATTNHP 1    /* AttNHP encoder (App. D.4): h^(0) = W_type[k_i];
                                 per layer q, k, v = W [z(t_i); h_i] + b (W is
                                 3D x 2D, the bias the constant 1 of [1; z; h])
                                 and h_i += tanh(sum_{j<=i} f_ij v_j / (1 + sum_{j<=i} f_ij)),
                                 f_ij = exp(q_i . k_j / sqrt(d_head)) per head; no
                                 LayerNorm, FFN or output projection; the decoder
                                 reads h^(L). z_j(t) = sin / cos(t / (m (5M/m)^((j - j mod 2)/D))). */

/* Model configuration. d_model % n_heads == 0; d_head = d_model / n_heads must
 * be 16, 32 or 64; bf16 models need d_model and d_ffn to be multiples of 32
 * (16 for fp32 models). AttNHP models ignore d_ffn and need
 * 0 < time_m <= time_M (the encoding's wavelength scales m, M). */
typedef struct {
  int32_t n_layers, d_model, n_heads, d_ffn, n_mix, n_types, prec;
  int32_t encoder;          /* TPPSD_ENC_* */
  float time_m, time_M;     /* AttNHP time scales; unused by THP models */
} tppsd_model_cfg;

typedef struct tppsd_model tppsd_model;   /* opaque host handle, read-only after create */
typedef struct tppsd_state tppsd_state;   /* opaque host handle, one per batch          */

/* Draft record of one round (§4.3 "Drafting"): for every sequence b and draft
 * position l = 0..gamma-1 the proposed interval, absolute time and type, the
 * draft's log-densities at them, and the draft's full decoder output (the
 * residual draws of Eq. (3)-(4) and Theorem 1 need g_D and f_D everywhere,
 * not only at the proposals). Device pointers; row stride is max_gamma. */
typedef struct {
  float   *tau;      /* [B, max_gamma]           proposed interval tau_hat_l     */
  float   *t;        /* [B, max_gamma]           absolute time t_hat_l           */
  int32_t *k;        /* [B, max_gamma]           proposed type k_hat_l           */
  float   *logg;     /* [B, max_gamma]           log g_D(tau_hat_l)              */
  float   *logf;     /* [B, max_gamma]           log f_D(k_hat_l)                */
  float   *mix;      /* [B, max_gamma, 3, M]     draft (log w, mu, log sigma)    */
  float   *logtype;  /* [B, max_gamma, K]        draft log f_D                   */
  float   *rate;     /* [B] NULL for a Transformer draft. Non-NULL marks a
                        homogeneous-Poisson draft (tppsd_draft_poisson writes
                        its rate here; `mix` is then unused and may be NULL) */
} tppsd_draft_buf;

/* Verification output (§4.3 "Verification"): the target's decoder output for
 * the pending event and the gamma drafts (gamma + 1 rows; row l scores draft
 * l + 1 and row gamma is the distribution after the last draft), plus the
 * target's log-densities at the drafts. Row stride is max_gamma + 1. */
typedef struct {
  float *logg;       /* [B, max_gamma]           log g_T(tau_hat_l)              */
  float *logf;       /* [B, max_gamma]           log f_T(k_hat_l)                */
  float *mix;        /* [B, max_gamma + 1, 3, M] target (log w, mu, log sigma)   */
  float *logtype;    /* [B, max_gamma + 1, K]    target log f_T                  */
} tppsd_verify_buf;

/* Accept output of one round. */
typedef struct {
  int32_t *L;        /* [B] first rejected draft position (1-based), gamma+1 if none; 0 if inactive */
  int32_t *n_new;    /* [B] events committed this round (after truncation at n_gen)      */
  int32_t *k_new;    /* [B, max_gamma + 1] types of the events produced this round       */
  float   *t_new;    /* [B, max_gamma + 1] absolute times of those events                */
  float   *tau_new;  /* [B, max_gamma + 1] their intervals                               */
  int32_t *ar_iter;  /* [B] index of the accepted Theorem-1 candidate, -1 if none drawn  */
  uint8_t *flags;    /* [B] bit0 tau redrawn, bit1 type redrawn, bit2 bonus event,
                            bit3 sequence finished, bit4 sequence was already finished,
                            bit5 finished by its end time (tppsd_prefill_window) */
} tppsd_accept_buf;

/* ---- weights ----------------------------------------------------------------- */

/* Size in bytes of the packed device weight buffer of a model (see
 * tppsd_weights_entry for its layout). Errors: TPPSD_E_ARG, TPPSD_E_CONFIG. */
int tppsd_weights_bytes(const tppsd_model_cfg *cfg, size_t *bytes);

/* Describes entry `index` (0-based) of the packed weight layout: its name
 * (static string, e.g. "layers.0.qkv.w"), byte offset (256-byte aligned),
 * shape [rows, cols] (cols = 1 for vectors) and element type (is_bf16 = 1 for
 * bf16, 0 for fp32). Linear matrices are [out, in] row-major; matrices are
 * bf16 for bf16 models, vectors are always fp32. Returns TPPSD_E_ARG past the
 * last entry, which is how a caller finds the count. */
int tppsd_weights_entry(const tppsd_model_cfg *cfg, int index, const char **name,
                        size_t *offset, int64_t *rows, int64_t *cols, int *is_bf16);

/* Creates a model handle over a packed device weight buffer that the caller
 * keeps alive for the handle's lifetime. Errors: TPPSD_E_ARG, TPPSD_E_CONFIG. */
int  tppsd_model_create(const tppsd_model_cfg *cfg, const void *d_weights, tppsd_model **out);
void tppsd_model_destroy(tppsd_model *m);

/* ---- sampler state ----------------------------------------------------------- */

/* Device workspace needed for a batch of B sequences with at most max_events
 * events each (history + generated + max_gamma + 1), draft length up to
 * max_gamma. It holds both KV caches ([layers][B][heads][max_events][d_head]
 * for keys and values), the committed events, per-sequence counters and
 * activation scratch. Errors: TPPSD_E_ARG. */
int tppsd_state_bytes(const tppsd_model *target, const tppsd_model *draft, int B,
                      int max_events, int max_gamma, size_t *bytes);

/* Creates a sampler state in the caller's workspace (256-byte aligned,
 * at least tppsd_state_bytes). `seed` keys the Philox4x64-10 streams of every
 * draw; `flags` is a combination of TPPSD_FLAG_*. The draft model may be NULL
 * for an AR-only state. Copies a small constant table into the workspace
 * (synchronously). Errors: TPPSD_E_ARG, TPPSD_E_WORKSPACE, TPPSD_E_CONFIG,
 * TPPSD_E_HIP. */
int  tppsd_state_create(const tppsd_model *target, const tppsd_model *draft, int B, int max_events,
                        int max_gamma, uint64_t seed, unsigned flags, void *d_workspace,
                        size_t ws_bytes, tppsd_state **out);
void tppsd_state_destroy(tppsd_state *s);

/* Starts a generation run: stores the seed histories d_t/d_k [B, n0]
 * (strictly increasing times, n0 >= 2), clears counters and status, and
 * encodes every history event except the last (the pending event whose
 * history embedding gives the next distribution) into the target's KV cache,
 * and all but the last two into the draft's. Each sequence will generate
 * exactly n_gen events. Errors: TPPSD_E_ARG (n0 < 2, n0 + n_gen + max_gamma + 1
 * > max_events), TPPSD_E_HIP. */
int tppsd_prefill(tppsd_state *s, const float *d_t, const int32_t *d_k, int n0, int n_gen,
                  hipStream_t stream);

/* tppsd_prefill with an end time per sequence (Algorithm 1's T): d_t_end [B]
 * (device, copied). Sequence b then ends at its n_gen-th new event or at its
 * first event past d_t_end[b], whichever comes first; that event is dropped
 * (an event exactly at the end time is kept and ends the sequence), and a
 * sequence whose pending event is already at or past its end time generates
 * nothing. d_t_end NULL: no end time (tppsd_prefill). Errors: as
 * tppsd_prefill. */
int tppsd_prefill_window(tppsd_state *s, const float *d_t, const int32_t *d_k, int n0, int n_gen,
                         const float *d_t_end, hipStream_t stream);

/* Drafting (§4.3 "Drafting", Algorithm 1's inner loop): gamma sequential draws
 * from the draft model for every unfinished sequence, using the Philox
 * counters (sequence, round, l, DRAFT). Fills `out` (all of it, for positions
 * 0..gamma-1). Errors: TPPSD_E_ARG (gamma outside 1..max_gamma, null buffer
 * pointer, out->rate not NULL), TPPSD_E_ORDER (no prefill, or no draft model),
 * TPPSD_E_HIP. */
int tppsd_draft(tppsd_state *s, int gamma, const tppsd_draft_buf *out, hipStream_t stream);

/* Verification (§4.3 "Verification"): one parallel target pass over the
 * pending event and the gamma drafts in `in` (tau, t, k are read; any source
 * may have filled them). Appends their keys/values to the target KV cache
 * (uncommitted until tppsd_accept) and fills `out`. Errors: TPPSD_E_ARG,
 * TPPSD_E_ORDER (no prefill), TPPSD_E_HIP. */
int tppsd_verify(tppsd_state *s, int gamma, const tppsd_draft_buf *in, const tppsd_verify_buf *out,
                 hipStream_t stream);

/* tppsd_verify for callers that cannot allocate device memory of their own
 * for the pass's temporaries (code under HIP graph capture, serving loops
 * that forbid allocation): the same kernels and results, with the pass's
 * activation scratch (residual stream, layer and decoder activations, logits,
 * attention key-split partials) in a static device array of the library
 * instead of the state's workspace. The array holds 64 MiB per GPU, kept
 * until the process ends; a pass that needs more (about B (gamma + 1) rows of
 * the widest model's activations plus the key-split partials) fails with
 * TPPSD_E_WORKSPACE. The array keeps the last call's contents and is shared by
 * every call on that GPU: calls that overlap on one GPU race. Arguments,
 * outputs and other errors as tppsd_verify; TPPSD_E_HIP if the array's device
 * address cannot be resolved. */
int tppsd_verify_noalloc(tppsd_state *s, int gamma, const tppsd_draft_buf *in, const tppsd_verify_buf *out,
                         hipStream_t stream);

/* Accept/reject and commit (§4.3, Eq. (3)-(4), Theorem 1, Algorithm 1).
 * Position l passes iff ln u_tau < log g_T - log g_D and ln u_k < log f_T -
 * log f_D; L is the first failing position. At L each failed component is
 * redrawn from its adjusted distribution (Theorem 1 acceptance-rejection for
 * the interval with the draft's g_D, the exponential density when draft->rate
 * is not NULL; Eq. (4) for the type) and each passed component is kept; if
 * none failed and TPPSD_FLAG_BONUS is set, one event is drawn from the
 * target's row gamma. Events are appended (truncated at n_gen per sequence)
 * and the KV cache lengths move to the committed prefix. d_uniforms, if not
 * NULL, gives (u_tau, u_k) per draft position [B, max_gamma, 2] in (0, 1);
 * otherwise they come from the Philox counters (sequence, round, l, ACCEPT).
 * Residual and bonus draws always use Philox. Every pointer in `out` must be
 * valid. Errors: TPPSD_E_ARG, TPPSD_E_ORDER, TPPSD_E_HIP. */
int tppsd_accept(tppsd_state *s, int gamma, const tppsd_draft_buf *draft,
                 const tppsd_verify_buf *verify, const float *d_uniforms,
                 const tppsd_accept_buf *out, hipStream_t stream);

/* Naive autoregressive sampling from the target (§4.2, App. A.1): n_events
 * sequential steps, each one target pass over the pending event followed by
 * a draw with the Philox counters (sequence, event index, 0, AR). Appends to
 * the state and, if d_t_out/d_k_out are not NULL, writes the generated events
 * [B, n_events]. Stops each sequence at its n_gen. Errors: TPPSD_E_ARG,
 * TPPSD_E_ORDER, TPPSD_E_HIP. */
int tppsd_sample_ar(tppsd_state *s, int n_events, float *d_t_out, int32_t *d_k_out,
                    hipStream_t stream);

/* Runs TPP-SD rounds (draft, verify, accept) with internal round buffers until
 * every sequence has its n_gen events or max_rounds rounds ran. Reads a done
 * counter back from the device once per round (one round behind). Returns the
 * number of rounds run in *rounds (may be NULL). Errors: as tppsd_draft. */
int tppsd_sample_sd(tppsd_state *s, int gamma, int max_rounds, int *rounds, hipStream_t stream);

/* ---- homogeneous-Poisson draft (App. D.3) ------------------------------------
 * A draft with no model: intervals Exp(rate), marks drawn from fixed
 * probabilities p, both maximum-likelihood estimates from observed sequences.
 * Parameters live on the device as d_params [1 + K] = (rate, log p_0 .. log
 * p_{K-1}), log 0 = -inf; K is the target's n_types. Such a state needs no
 * draft model (tppsd_state_create with draft NULL). */

/* Maximum-likelihood fit over B sequences of n0 events d_t/d_k [B, n0]
 * (device, strictly increasing times): rate = B (n0 - 1) / sum of the spans
 * t[n0-1] - t[0]; p_m = count of type m / count of types in [0, K) (types
 * outside it are ignored). Writes d_params [1 + K] (device). One workgroup,
 * enqueued on `stream`. Errors: TPPSD_E_ARG (null pointer, B < 1, n0 < 2,
 * K outside 1..TPPSD_MAX_TYPES, B * n0 >= 2^31), TPPSD_E_HIP. */
int tppsd_poisson_fit(const float *d_t, const int32_t *d_k, int B, int n0, int K, float *d_params,
                      hipStream_t stream);

/* Drafting from the Poisson draft: for every unfinished sequence, gamma
 * independent draws with the Philox counters (sequence, round, l, DRAFT):
 * tau_l = -ln(u_1) / rate, k_l the first m with u_3 * sum(p) < p_0 + .. + p_m.
 * Writes tau, t, k, logg = log rate - rate tau, logf = log p_k, logtype (log p
 * at every position) and rate[b]; out->rate must not be NULL. The buffer then
 * goes to tppsd_verify and tppsd_accept as usual; accept's Theorem-1 loop uses
 * the exponential density as g_D and Eq. (4) uses p as f_D. Errors:
 * TPPSD_E_ARG (gamma outside 1..max_gamma, null pointer), TPPSD_E_ORDER (no
 * prefill), TPPSD_E_HIP. */
int tppsd_draft_poisson(tppsd_state *s, int gamma, const float *d_params, const tppsd_draft_buf *out,
                        hipStream_t stream);

/* tppsd_sample_sd with the Poisson draft of d_params (device, kept alive and
 * unchanged while the call's work runs; graphs captured here embed the
 * pointer). Errors: as tppsd_draft_poisson. */
int tppsd_sample_sd_poisson(tppsd_state *s, int gamma, const float *d_params, int max_rounds, int *rounds,
                            hipStream_t stream);

/* Copies the committed events (history included) to d_t/d_k [B, max_events]
 * and the per-sequence event counts to d_n [B]. Any pointer may be NULL. */
int tppsd_read_events(tppsd_state *s, float *d_t, int32_t *d_k, int32_t *d_n, hipStream_t stream);

/* Model log-likelihood (Eq. (2)) of each sequence's generated events since
 * prefill, accumulated while sampling: the target's log g(tau_i) + log f(k_i)
 * at every committed event (tau_i the interval as drawn; event times are its
 * float32 running sum) in float64, plus, for a sequence ended by its end
 * time, log(1 - G(T - t_N)) under the target's distribution after its last
 * event. AR and TPP-SD runs accumulate the same quantity. Copies [B] doubles
 * to d_ll (device). Errors: TPPSD_E_ARG, TPPSD_E_HIP. */
int tppsd_read_loglik(tppsd_state *s, double *d_ll, hipStream_t stream);

/* Synchronises the stream and reads the sticky status bits and the number of
 * finished sequences. Accounting (may be NULL): accepted drafts, drafted
 * positions and Theorem-1 candidates drawn since prefill. */
int tppsd_state_status(tppsd_state *s, hipStream_t stream, uint32_t *bits, int32_t *n_done,
                       int64_t *accepted_drafts, int64_t *drafted, int64_t *ar_candidates);

/* Measurement of tppsd_sample_sd; the sampled events are unchanged.
 * TPPSD_TIME_KERNELS: rounds are launched directly instead of replaying a
 *   captured HIP graph (and tppsd_sample_ar launches its steps directly
 *   too, untimed), and every launch of the target's verify attention, of
 *   its verify GEMMs (QKV, attention output, FFN in, FFN out, decoder E), of
 *   the one-launch draft kernel and of each row-drafting launch (split
 *   attention, row kernel) is bracketed by HIP events stamped with the
 *   kernel's own start and stop.
 * TPPSD_TIME_PHASES: each round replays three captured graphs (draft, verify,
 *   accept) with HIP events recorded between them on the caller's stream.
 * The two modes are separate runs (both bits at once: TPPSD_E_ARG).
 * tppsd_timing_enable resets the sums; tppsd_timing_read copies them. Other
 * entry points are not timed. */
#define TPPSD_TIME_KERNELS 1
#define TPPSD_TIME_PHASES 2
typedef struct tppsd_timing {
  double attn_ms;          /* verify attention: summed kernel time */
  int64_t attn_launches;
  double gemm_ms;          /* verify GEMMs: summed kernel time */
  int64_t gemm_launches;
  double gemm_flop;        /* 2 * rows * N * K over the timed GEMM launches */
  double draft_ms, verify_ms, accept_ms;   /* phase times */
  int64_t rounds;          /* rounds timed */
  double draft_kernel_ms;  /* one-launch draft kernel: summed kernel time */
  int64_t draft_kernel_launches;
  double draft_attn_ms;    /* row drafting: split attention launches, summed kernel time */
  int64_t draft_attn_launches;
  double draft_rows_ms;    /* row drafting: per-sequence row launches, summed kernel time */
  int64_t draft_rows_launches;
} tppsd_timing;
int tppsd_timing_enable(tppsd_state *s, int modes);
int tppsd_timing_read(tppsd_state *s, tppsd_timing *out);

/* Thread-local description of the last error on this thread. */
const char *tppsd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TPPSD_H */
