// Internal interface between the C-ABI host library (tppsd.cpp) and the HIP
// kernels (tppsd_kernels.hip). Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tppsd_attention.h"

namespace tppsd {

typedef uint16_t bf16_t;   // raw bfloat16 bits

// Where the P tokens of a block forward come from: token p of sequence b is
// committed event (start[b] + start_off + p) for p < n_ev, otherwise draft
// slot (dr_off + p - n_ev).
struct TokSrc {
  const float *ev_t;
  const int32_t *ev_k;
  int ev_stride;            // max_events
  const int32_t *start;     // per-sequence base position
  int start_off;
  int n_ev;
  const float *dr_t;
  const int32_t *dr_k;
  int dr_stride;            // max_gamma
  int dr_off;
};

// GEMM epilogues: Y[r, n] = sum_k X[r, k] W[n, k]
enum EpiMode { EPI_STORE = 0, EPI_RESID = 1, EPI_RELU = 2, EPI_QKV = 3, EPI_HEAD = 4, EPI_F32 = 5 };

struct Epi {
  int mode;
  const float *bias;        // [N] (HEAD: [N - split])
  void *out;                // STORE/RELU/HEAD: act [T, ldo]; RESID, F32: float [T, ldo]
  int ldo;
  // EPI_QKV: n < d -> q[r, n]; n in [d, 2d) -> key cache; [2d, 3d) -> value cache
  void *q;
  void *kc, *vc;            // this layer's cache base, [B][H][cap][dh]
  const int32_t *start;
  int start_off;
  int P, H, dh, d, cap;
  uint32_t *status;
  int split;                // EPI_HEAD: columns < split stored raw, >= split tanh(acc + bias)
};

// Decoder epilogue modes
enum HeadMode { HEAD_VERIFY = 0, HEAD_DRAFT = 1, HEAD_AR = 2 };

struct HeadArgs {
  int mode;
  int P, p0;                // rows p0..P-1 of each sequence are decoded
  int B;
  // destination of (log w, mu, log sigma) [.., 3, M] and log f [.., K]
  float *mix, *logtype;
  int dst_stride;           // rows per sequence in mix/logtype (HEAD_AR: 1)
  int dst_row0;             // destination row of p0 (HEAD_DRAFT: slot)
  // HEAD_VERIFY: log-densities at the drafts
  int gamma;
  const float *dr_tau;
  const int32_t *dr_k;
  int dr_stride;
  float *v_logg, *v_logf;
  // HEAD_DRAFT: proposal record (slot dst_row0)
  float *d_tau, *d_t, *d_logg, *d_logf;
  int32_t *d_k;
  int slot, l_index;        // Philox slot counter word (1-based draft position)
  // state
  float *ev_t;
  int32_t *ev_k;
  int ev_stride;
  int32_t *n, *gen, *lenT, *done, *rnd, *n_done;
  int n_gen;
  const float *t_end;       // [B] end times (+inf: none)
  double *ll;               // [B] model log-likelihood of the generated events (Eq. (2))
  uint64_t seed;
  uint32_t *status;
  // HEAD_AR optional outputs [B, out_stride], written at column gen - gen0
  float *ar_t_out;
  int32_t *ar_k_out;
  int ar_out_stride;
  const int32_t *gen0;
};

struct AcceptArgs {
  int B, gamma, M, K, max_gamma, bonus;
  const float *d_tau, *d_t, *d_logg, *d_logf, *d_mix, *d_logtype;
  const int32_t *d_k;
  const float *v_logg, *v_logf, *v_mix, *v_logtype;
  const float *uniforms;    // nullable [B, max_gamma, 2]
  const float *d_rate;      // nullable [B]: homogeneous-Poisson draft rate (g_D exponential)
  int32_t *L, *n_new, *k_new, *ar_iter;
  float *t_new, *tau_new;
  uint8_t *flags;
  float *ev_t;
  int32_t *ev_k;
  int ev_stride;
  int32_t *n, *gen, *lenT, *lenD, *done, *rnd, *n_done;
  int n_gen;
  const float *t_end;       // [B] end times (+inf: none)
  double *ll;               // [B] model log-likelihood of the generated events (Eq. (2))
  uint64_t seed;
  uint32_t *status;
  unsigned long long *acc_stats;   // [B][3]: per sequence accepted drafts, drafted, A-R candidates
};

// Fused drafting: one workgroup per sequence runs all gamma draft steps.
#define FD_MAX_LAYERS 4
struct FusedLayerW {
  const void *qkv_w, *out_w, *ffn1_w, *ffn2_w;
  const float *ln1_g, *ln1_b, *qkv_b, *out_b, *ln2_g, *ln2_b, *ffn1_b, *ffn2_b;
};
struct DraftArgs {
  int B, gamma, d, H, F, M, K, L;
  FusedLayerW layer[FD_MAX_LAYERS];
  const void *type_emb, *Ek1_w, *mix_w, *k2_w;
  const float *lnf_g, *lnf_b, *k1_b, *mix_b, *k2_b;
  const float *freq;
  char *kc, *vc;            // draft cache bases; layer stride layer_bytes
  size_t layer_bytes;
  int cap;
  const float *ev_t;
  const int32_t *ev_k;
  int ev_stride;
  const int32_t *n, *lenD, *done, *rnd;
  uint64_t seed;
  uint32_t *status;
  float *d_tau, *d_t, *d_logg, *d_logf, *d_mix, *d_logtype;
  int32_t *d_k;
  int MG;                   // row stride of the draft record (max_gamma)
  int w_lds;                // stage the weight matrices in LDS (fused_draft_weight_elems more)
};
// whether the fused draft kernel supports a model of these sizes: the
// matrix-vector products need d / 8 and d_ffn / 8 to be powers of two <= 64,
// the attention a power-of-two head count and d_head = 16 (a thread holds a
// whole 8-position block of keys and values in registers)
inline bool fused_draft_ok(int L, int d, int H, int F) {
  auto pow2 = [](int v) { return v > 0 && (v & (v - 1)) == 0; };
  return L <= FD_MAX_LAYERS && d % 8 == 0 && F % 8 == 0 && pow2(d / 8) && pow2(F / 8) && d / 8 <= 64 &&
         F / 8 <= 64 && pow2(H) && d == 16 * H;
}
size_t fused_draft_lds_bytes(int L, int d, int F, int M, int K, int H);
// One wave per sequence (k_draft_wave): draft models of width 16 or 32
// (d_head 16), F = 2 d or 4 d, at most two layers, whose transposed matrices
// fit in LDS beside four waves' scratch
bool wave_draft_ok(int L, int d, int H, int F, int M, int K, int bf16);
size_t wave_draft_lds_bytes(int L, int D, int F, int M, int K, int elt);
void launch_draft_wave(const DraftArgs &a, int bf16, hipStream_t st, hipEvent_t ev0 = nullptr,
                       hipEvent_t ev1 = nullptr);
// raises the dynamic LDS limit of the wave-draft kernels; nonzero on failure
int allow_draft_wave_lds(size_t bytes);
// elements of the draft's weight matrices (per layer QKV, out, FFN; decoder), each
// row padded by pad elements (16 bytes) in LDS
size_t fused_draft_weight_elems(int L, int d, int F, int M, int K, int pad);
// LDS of one workgroup on gfx950
constexpr size_t LDS_PER_WG = 160 * 1024;

// Drafting for small batches over long contexts (k_rd_attn + k_rd_rows, per
// draft step and layer): the step's attention split over (key range, head,
// sequence) workgroups of RD_KEYS keys, then workgroups of RD_ROW_THREADS for
// the row-local rest (RD_FSPLIT per sequence for a non-last layer, one for the
// last). bf16 draft models with d = 128, four heads of 32, d_ffn = 512.
constexpr int RD_KEYS = 384;
constexpr int RD_ROW_THREADS = 512;
// event types whose embedding rows the row kernel stages in LDS (all of them)
constexpr int RD_MAX_TYPES = 32;
// floats of one sequence's split partials the row kernel stages in LDS
// (H S 2 (d_head + 2): 4 heads of 32 over 8192 positions take 4352; a
// multiple of RD_ROW_THREADS)
constexpr int RD_MAX_PART = 4608;
constexpr int RD_FSPLIT = 4;    // workgroups per sequence of a non-last layer's row launch (FFN hidden slices)
static_assert(RD_MAX_PART % RD_ROW_THREADS == 0, "partial staging: whole rounds of the row workgroup");
struct RowDraftArgs {
  DraftArgs d;              // model, cache, state and record pointers as for the one-launch draft
  float *x;                 // [B][2][d] residual stream of the step's rows
  bf16_t *xn;               // [B][2][d] the step's rows after the layer's LayerNorm (q, k, v input)
  float *part;              // [B][H][S][2][d_head + 2] split partials: maximum, sum, output sums
  float *fpart;             // [B][RD_FSPLIT][2][d] a non-last layer's FFN output, per slice of its hidden units
  float *rng;               // [B][MG][4] per draft step: u for the component, the normal deviate, u for the
                            // type (written by the step-0 launch)
  const bf16_t *pk;         // per layer Wo, W1, W2, Wqkv in MFMA fragment order (launch_pack_frags)
  const bf16_t *pk_e;       // [E; V_k1] in fragment order
  const bf16_t *pk_head;    // decoder head rows, zero-padded to 128, in fragment order (launch_pack_rd_head)
  int S;                    // key splits per (sequence, head): ceil(kv_cap / RD_KEYS)
  int step;                 // draft step (1-based); 0: embed the last two committed events
  int layer;
};
bool row_draft_ok(int bf16, int L, int d, int H, int F, int M, int K, int kv_cap);
inline int rd_splits(int kv_cap) { return (kv_cap + RD_KEYS - 1) / RD_KEYS; }
inline size_t rd_part_floats(int B, int H, int dh, int kv_cap) {
  return (size_t)B * H * rd_splits(kv_cap) * 2 * (dh + 2);
}
// elements of the row kernel's packed decoder: [E; V_k1] (4 d x d) and the heads (128 x d)
inline size_t rd_pack_dec_elems(int d) { return (size_t)4 * d * d + (size_t)128 * d; }
void launch_pack_rd_head(const void *mix_w, const void *k2_w, int M, int K, int D, void *out, hipStream_t st);
// all launches of one round's drafting: the step-0 row launch, then per step
// and layer the attention and the row launch (1 + 2 L gamma launches); ev
// (nullable) holds an event pair per launch, in that order
inline int rd_launches(int L, int gamma) { return 1 + 2 * L * gamma; }
void launch_draft_rows(RowDraftArgs a, hipStream_t st, const hipEvent_t *ev = nullptr);

// Fused row block of a THP forward pass (k_block): for a tile of 16 rows,
// everything between two attention launches. first: embed the tokens (else
// read the residual stream x); pre: output projection of o, residual, the
// feed-forward block of the layer whose attention just ran; then qkv: the
// next layer's LayerNorm and q, k, v (through the EPI_QKV epilogue), or head:
// the final LayerNorm, the decoder and its epilogue. store_x writes the
// stream back for the next launch.
struct BlockArgs {
  int T, P, d, F;
  int first, pre, qkv, head, store_x;
  TokSrc src;
  const void *type_emb;
  const float *freq;
  int n_types;
  float *x;
  const void *o;
  const void *out_w, *ffn1_w, *ffn2_w;
  const float *out_b, *ln2_g, *ln2_b, *ffn1_b, *ffn2_b;
  const void *qkv_w;
  const float *ln1_g, *ln1_b;
  Epi qe;                   // EPI_QKV epilogue of the next layer (bias = its qkv bias)
  const float *lnf_g, *lnf_b, *k1_b, *head_b;
  const void *Ek1_w, *head_w;
  int M, K;
  HeadArgs h;
};
// whether k_block serves a pass of T rows of a model of width d, FFN width F, M mixture components and K types
bool block_fusable(int bf16, int d, int F, int M, int K, long T);
// widths k_block / k_verify_seq have instances for; their weights are read
// in the packed order launch_pack_wbatch writes (wbatch_packed_elems each)
bool block_widths(int d, int F);
size_t wbatch_packed_elems(int N, int K);
void launch_pack_wbatch(const void *W, int N, int K, int bf16, void *out, hipStream_t s);
void launch_block(const BlockArgs &a, int bf16, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

// Per-sequence verify pass (k_verify_seq): one workgroup runs the whole target
// pass of one sequence's P = gamma + 1 positions (embedding, every layer with
// its attention, decoder, verify epilogue), the rows staying in LDS.
struct VerifySeqArgs {
  int P, d, F, H, L, M, K;
  FusedLayerW layer[FD_MAX_LAYERS];
  const void *type_emb, *Ek1_w, *head_w;
  const float *lnf_g, *lnf_b, *k1_b, *head_b, *freq;
  char *kc, *vc;            // target cache bases; layer stride layer_bytes
  size_t layer_bytes;
  int cap;
  const float *ev_t;
  const int32_t *ev_k;
  int ev_stride;
  const int32_t *lenT, *done;
  const float *dr_t;
  const int32_t *dr_k;
  int dr_stride;
  uint32_t *status;
  HeadArgs h;               // HEAD_VERIFY
};
// whether k_verify_seq serves a target of these sizes for P positions
bool verify_seq_ok(int bf16, int L, int d, int H, int F, int M, int K, int P);
void launch_verify_seq(const VerifySeqArgs &a, int B, int bf16, hipStream_t st, hipEvent_t ev0 = nullptr,
                       hipEvent_t ev1 = nullptr);

// Homogeneous-Poisson drafting (tppsd_poisson.hip)
struct PoissonDraftArgs {
  int B, gamma, K, MG;
  const float *params;      // [1 + K]: rate, log p
  const float *ev_t;
  int ev_stride;
  const int32_t *n, *done, *rnd;
  uint64_t seed;
  uint32_t *status;
  float *d_tau, *d_t, *d_logg, *d_logf, *d_logtype, *d_rate;
  int32_t *d_k;
};
void launch_poisson_fit(const float *t, const int32_t *k, int B, int n0, int K, float *params, hipStream_t st);
void launch_draft_poisson(const PoissonDraftArgs &a, hipStream_t st);

// ---- launchers (tppsd_kernels.hip) ----
void launch_draft_fused(const DraftArgs &a, int bf16, hipStream_t st, hipEvent_t ev0 = nullptr,
                        hipEvent_t ev1 = nullptr);
// raises the dynamic LDS limit of the fused draft kernels to `bytes`; nonzero on failure
int allow_draft_fused_lds(size_t bytes);
void launch_embed(float *x, int T, int d, int P, const TokSrc &src, const void *wtype, int bf16,
                  const float *freq, int K, hipStream_t st);
void launch_layernorm(const float *x, void *y, int bf16, const float *g, const float *b, int T, int d,
                      hipStream_t st);
// AttNHP: h^(0) = W_type[k] into x (fp32) and u = [z(t); h] (activation type, [T, 2d])
void launch_embed_attnhp(float *x, void *u, int T, int d, int P, const TokSrc &src, const void *wtype, int bf16,
                         const float *freq, int K, hipStream_t st);
// AttNHP: x += tanh(o) (o [T, d], activation type); u[:, d:] = a = x in the activation type
void launch_attnhp_update(float *x, const void *o, void *u, void *a, int bf16, int T, int d, hipStream_t st);
// A operand given as LayerNorm(x) of the fp32 stream x [T, K] with gain g and bias b
struct LnA {
  const float *x, *g, *b;
};
// Y = A W^T into the epilogue; A is X [T, K] of the operand type, or, when ln
// is not null, LayerNorm of ln->x computed inside the GEMM. ev0/ev1
// (optional): HIP events stamped with the kernel's own start and stop.
void launch_gemm(const void *X, const LnA *ln, const void *W, int bf16, int T, int N, int K, const Epi &epi,
                 hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// whether launch_gemm can take a LayerNorm operand of width K
bool gemm_ln_fusable(int bf16, int K);
// the layered pass runs LayerNorm as its own launch before a plain GEMM (see the definition)
bool gemm_ln_split(int bf16, int d, int T);
// Fused row-local part of a bf16 THP layer between two attention launches
// (output projection + residual, feed-forward block + residual, and with
// post the next layer's LayerNorm and q, k, v through qe), one launch over
// row tiles; layer_fused_ok: there is an instance; layer_fused_worth: it
// beats the layered kernels at T rows
struct LayerArgs {
  float *x;                                  // [T][D] residual stream (in / out)
  const bf16_t *o, *wo;                      // attention output [T][D], Wo [D][D] (weights: packed fragments)
  const float *bo;
  const float *ln2_g, *ln2_b, *b1, *b2;
  const bf16_t *w1, *w2;                     // [F][D], [D][F]
  const float *ln1_g, *ln1_b;                // post: the next layer's LayerNorm
  const bf16_t *wqkv;                        // post: [3D][D]
  Epi qe;                                    // post: EPI_QKV
  int T;
};
bool layer_fused_ok(int bf16, int d, int F);
// W [N][K] bf16 into the MFMA fragment order k_layer_fused reads (N % 16 == 0,
// K % 32 == 0; out holds N K elements)
void launch_pack_frags(const void *W, int N, int K, void *out, hipStream_t s);
bool layer_fused_worth(int d, long T);
void launch_layer_fused(const LayerArgs &a, int d, int F, bool post, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
// decoder epilogue over the rows' logits [.., ldl] (mixture w | mu | log sigma, then types)
void launch_head(const float *logits, int ldl, int M, int K, const HeadArgs &a, hipStream_t st);
// the decoder's block-diagonal (3M + K) x 4d matrix and its bias (3M + K)
void launch_build_head(const void *mix_w, const void *k2_w, const float *mix_b, const float *k2_b, int bf16, int d,
                       int M, int K, void *hw, float *hb, hipStream_t st);
// row stride of the decoder logits: 3M + K rounded up to 8
inline int head_ldl(int M, int K) { return (3 * M + K + 7) / 8 * 8; }
void launch_accept(const AcceptArgs &a, hipStream_t st);
void launch_prefill_init(const float *ht, const int32_t *hk, int B, int n0, int n_gen, const float *t_end_in,
                         float *ev_t, int32_t *ev_k, int ev_stride, int32_t *n, int32_t *gen, int32_t *lenT,
                         int32_t *lenD, int32_t *done, int32_t *rnd, int32_t *zeros, float *t_end, double *ll,
                         int32_t *n_done, uint32_t *status, unsigned long long *acc_stats, hipStream_t st);
void launch_snapshot(const int32_t *src, int32_t *dst, int B, hipStream_t st);
void launch_copy_events(const float *ev_t, const int32_t *ev_k, const int32_t *n, int B, int ev_stride,
                        float *t, int32_t *k, int32_t *nout, hipStream_t st);

}  // namespace tppsd
