// Host side of the TPP-SD C ABI: argument validation, packed weight layout,
// workspace layout, and the launch sequence of each entry point.
//
// Entry points follow Algorithm 1 of the paper: drafting (§4.3) is gamma
// sequential draft-model passes; verification is one target pass over the
// pending event plus the gamma drafts; accept runs the first-rejection test,
// the adjusted-distribution replacement (Eq. (3)-(4), Theorem 1) and the
// commit. Naive AR sampling (§4.2) is one target pass per event.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/tppsd.h"
#include "tppsd_internal.h"

using namespace tppsd;

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_check(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TPPSD_E_HIP, "%s: %s", what, hipGetErrorString(e));
  return TPPSD_OK;
}

int hip_check_rc(hipError_t e) {
  return e == hipSuccess ? TPPSD_OK : fail(TPPSD_E_HIP, "timing event: %s", hipGetErrorString(e));
}

void drop_graph(hipGraphExec_t *g) {
  if (*g) (void)hipGraphExecDestroy(*g);
  *g = nullptr;
}

constexpr size_t ALIGN = 256;
inline size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

constexpr int PREFILL_CHUNK = 16;

// ---- packed weight layout -------------------------------------------------
struct Entry {
  std::string name;
  size_t off;
  int64_t rows, cols;
  int bf16;
};

// Entries are 256-byte aligned, except that a few groups are packed back to
// back so that the kernels can read them as one matrix: [E; V_k1] (4d x d),
// [V_w; V_mu; V_sigma] (3M x d) and their biases (3M). AttNHP models have per
// layer only qkv.w (3d x 2d, over [z; h]) and qkv.b, and no final LayerNorm.
std::vector<Entry> layout(const tppsd_model_cfg &c) {
  std::vector<Entry> v;
  const int bf = c.prec == TPPSD_PREC_BF16;
  const size_t me = bf ? 2 : 4;
  size_t off = 0;
  auto add = [&](const std::string &n, int64_t r, int64_t cl, bool mat, bool aligned) {
    if (aligned) off = align_up(off);
    v.push_back({n, off, r, cl, mat ? bf : 0});
    off += (size_t)r * cl * (mat ? me : 4);
  };
  const int d = c.d_model, F = c.d_ffn, M = c.n_mix, K = c.n_types;
  const bool attnhp = c.encoder == TPPSD_ENC_ATTNHP;
  add("type_emb", K, d, true, true);
  for (int l = 0; l < c.n_layers && attnhp; ++l) {   // AttNHP: W [3d x 2d] over [z; h] and its bias
    const std::string p = "layers." + std::to_string(l) + ".";
    add(p + "qkv.w", 3 * d, 2 * d, true, true);
    add(p + "qkv.b", 3 * d, 1, false, true);
  }
  for (int l = 0; l < c.n_layers && !attnhp; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    add(p + "ln1.g", d, 1, false, true);
    add(p + "ln1.b", d, 1, false, true);
    add(p + "qkv.w", 3 * d, d, true, true);
    add(p + "qkv.b", 3 * d, 1, false, true);
    add(p + "out.w", d, d, true, true);
    add(p + "out.b", d, 1, false, true);
    add(p + "ln2.g", d, 1, false, true);
    add(p + "ln2.b", d, 1, false, true);
    add(p + "ffn1.w", F, d, true, true);
    add(p + "ffn1.b", F, 1, false, true);
    add(p + "ffn2.w", d, F, true, true);
    add(p + "ffn2.b", d, 1, false, true);
  }
  if (!attnhp) {
    add("lnf.g", d, 1, false, true);
    add("lnf.b", d, 1, false, true);
  }
  add("head.E", 3 * d, d, true, true);
  add("head.k1.w", d, d, true, false);
  add("head.k1.b", d, 1, false, true);
  add("head.w.w", M, d, true, true);
  add("head.mu.w", M, d, true, false);
  add("head.sigma.w", M, d, true, false);
  add("head.w.b", M, 1, false, true);
  add("head.mu.b", M, 1, false, false);
  add("head.sigma.b", M, 1, false, false);
  add("head.k2.w", K, d, true, true);
  add("head.k2.b", K, 1, false, true);
  v.push_back({"", align_up(off), 0, 0, 0});   // sentinel: total size
  return v;
}

int check_cfg(const tppsd_model_cfg *c) {
  if (!c) return fail(TPPSD_E_ARG, "null model configuration");
  if (c->encoder != TPPSD_ENC_THP && c->encoder != TPPSD_ENC_ATTNHP)
    return fail(TPPSD_E_CONFIG, "unknown encoder %d", c->encoder);
  const bool attnhp = c->encoder == TPPSD_ENC_ATTNHP;
  if (attnhp && !(c->time_m > 0.f && c->time_M >= c->time_m))
    return fail(TPPSD_E_CONFIG, "AttNHP needs 0 < time_m <= time_M");
  if (c->n_layers < 1 || c->d_model < 16 || c->n_heads < 1 || (!attnhp && c->d_ffn < 1) || c->n_mix < 1 ||
      c->n_types < 1)
    return fail(TPPSD_E_CONFIG, "model sizes must be positive (d_model >= 16)");
  if (c->prec != TPPSD_PREC_FP32 && c->prec != TPPSD_PREC_BF16)
    return fail(TPPSD_E_CONFIG, "unsupported precision %d", c->prec);
  if (c->d_model % c->n_heads) return fail(TPPSD_E_CONFIG, "d_model %% n_heads != 0");
  const int dh = c->d_model / c->n_heads;
  if (dh != 16 && dh != 32 && dh != 64) return fail(TPPSD_E_CONFIG, "d_head %d not in {16, 32, 64}", dh);
  if (c->d_model % 16) return fail(TPPSD_E_CONFIG, "d_model must be a multiple of 16");
  if (c->prec == TPPSD_PREC_BF16 && (c->d_model % 32 || (!attnhp && c->d_ffn % 32)))
    return fail(TPPSD_E_CONFIG, "bf16 models need d_model and d_ffn multiples of 32");
  if (!attnhp && c->d_ffn % 16) return fail(TPPSD_E_CONFIG, "d_ffn must be a multiple of 16");
  if (c->n_mix > TPPSD_MAX_MIX) return fail(TPPSD_E_CONFIG, "n_mix > %d", TPPSD_MAX_MIX);
  if (c->n_types > TPPSD_MAX_TYPES) return fail(TPPSD_E_CONFIG, "n_types > %d", TPPSD_MAX_TYPES);
  return TPPSD_OK;
}

}  // namespace

// ---- model handle -----------------------------------------------------------
struct LayerW {
  const void *qkv_w, *out_w, *ffn1_w, *ffn2_w;
  const float *ln1_g, *ln1_b, *qkv_b, *out_b, *ln2_g, *ln2_b, *ffn1_b, *ffn2_b;
};

struct tppsd_model {
  tppsd_model_cfg cfg;
  const char *w;
  std::vector<LayerW> layers;
  const void *type_emb, *Ek1_w, *mix_w, *k2_w;
  const float *lnf_g, *lnf_b, *k1_b, *mix_b, *k2_b;
  int bf16() const { return cfg.prec == TPPSD_PREC_BF16; }
  bool attnhp() const { return cfg.encoder == TPPSD_ENC_ATTNHP; }
  int d() const { return cfg.d_model; }
  int H() const { return cfg.n_heads; }
  int dh() const { return cfg.d_model / cfg.n_heads; }
  size_t act_bytes() const { return bf16() ? 2 : 4; }
};

// ---- state ------------------------------------------------------------------
struct ModelCache {
  void *head_w = nullptr;   // decoder block-diagonal matrix [(3M + K)][4d]
  float *head_b = nullptr;  // and bias [3M + K]
  // the matrices k_block and k_verify_seq read, in their packed order
  // (launch_pack_wbatch), for models of the widths they serve
  char *wb = nullptr;
  std::vector<const void *> wb_qkv, wb_out, wb_f1, wb_f2;
  const void *wb_ek1 = nullptr, *wb_head = nullptr;
  // per layer: keys [B][H][kv_cap][dh]; values the same for fp32, in
  // 8-position blocks [B][H][kv_cap / 8][dh][8] for bf16
  char *k = nullptr, *v = nullptr;
  size_t layer_bytes = 0;
  float *freq = nullptr;
};

struct tppsd_state {
  const tppsd_model *T = nullptr, *D = nullptr;
  int B = 0, cap = 0, max_gamma = 0, Pmax = 0;
  int kv_cap = 0;   // KV cache positions per (sequence, head): cap rounded up to 8
  uint64_t seed = 0;
  unsigned flags = 0;
  char *ws = nullptr;
  // device header + counters
  uint32_t *status = nullptr;
  int32_t *n_done = nullptr;
  unsigned long long *acc_stats = nullptr;
  int32_t *n = nullptr, *gen = nullptr, *lenT = nullptr, *lenD = nullptr, *done = nullptr, *rnd = nullptr,
          *zeros = nullptr;
  float *ev_t = nullptr;
  int32_t *ev_k = nullptr;
  float *t_end = nullptr;    // [B] end times (+inf: none)
  double *ll = nullptr;      // [B] model log-likelihood of the generated events
  ModelCache cT, cD;
  // activation scratch
  float *x = nullptr;
  void *a = nullptr, *q = nullptr, *o = nullptr, *hid = nullptr, *e = nullptr, *u = nullptr;
  float *logits = nullptr;
  bool heads_built = false;
  float *ar_mix = nullptr, *ar_logtype = nullptr;
  float *attn_part = nullptr;
  char *packT = nullptr;               // target weights in fragment order (nullptr: no fused layer kernel)
  size_t pack_layer = 0;
  char *packD = nullptr;               // draft weights in fragment order
  char *packDdec = nullptr;            // draft decoder in fragment order (row drafting)
  float *rd_rng = nullptr;             // [B][max_gamma][4] the draft draws' random numbers (row drafting)
  float *rd_fpart = nullptr;           // [B][RD_FSPLIT][2][d] FFN outputs per hidden slice (row drafting)
  size_t pack_layerD = 0;
  bool packs_built = false;
  bool wb_built = false;
  int32_t *gen0 = nullptr;
  // internal round buffers (tppsd_sample_sd)
  tppsd_draft_buf idr{};
  tppsd_draft_buf idr_p{};   // the same with the rate array (Poisson draft)
  tppsd_verify_buf ivf{};
  tppsd_accept_buf iac{};
  // host-side run state
  int n_gen = 0;
  bool prefilled = false, draft_ok = false, drafted_this_round = false;
  int32_t *host_ndone = nullptr;   // pinned, 2 slots
  hipEvent_t poll_ev[2] = {nullptr, nullptr};
  // measurement (tppsd_timing_enable): two event sets alternated per round
  // and read one round behind. Kernel mode: a pair of events around every
  // verify attention / GEMM launch (rounds launched directly); phase mode:
  // events between the draft, verify and accept graphs of each round.
  int timing = 0;
  std::vector<hipEvent_t> gev[2];
  std::vector<hipEvent_t> pev[2];
  hipEvent_t *cur_ev = nullptr;      // kernel events of the round being launched
  std::vector<char> ev_used;         // event pairs the verify pass records (per pair of cur_ev)
  tppsd_timing tm{};
  double round_flop = 0.0;           // verify GEMM flops of one round
  hipGraphExec_t phase_exec[3] = {nullptr, nullptr, nullptr};
  long long phase_key = -1;
  // HIP graphs of the sampling loops, captured on a private stream and
  // replayed on the caller's; keyed by what their kernel arguments embed
  hipStream_t cap_stream = nullptr;
  bool fused_draft = true;   // one-launch drafting when the draft model fits it
  bool wave_draft = false;   // ... with one wave per sequence (small draft models)
  bool fused_w_lds = false;  // ... with its weight matrices staged in LDS
  bool row_draft = false;    // split attention + row workgroups per sequence, per step and layer
  hipGraphExec_t sd_exec[2] = {nullptr, nullptr};
  long long sd_key = -1;
  const float *sd_params = nullptr, *phase_params = nullptr;   // Poisson draft parameters the graphs embed
  hipGraphExec_t ar_exec[2] = {nullptr, nullptr};   // 1 step, AR_CHUNK steps
  long long ar_key[2] = {-1, -1};
};

namespace {
constexpr int AR_CHUNK = 8;
}

namespace {

struct WsLayout {
  size_t total = 0;
  size_t status, n_done, acc, n, gen, lenT, lenD, done, rnd, zeros, ev_t, ev_k, t_end, ll;
  size_t freqT, freqD, kT, vT, kD, vD, layerT, layerD;
  size_t x, a, q, o, hid, e, u, ar_mix, ar_lt, attn_part, gen0;
  size_t logits, hwT, hbT, hwD, hbD;
  size_t packT = 0, pack_layer = 0;   // target weights in MFMA fragment order (fused layer kernel), per layer
  size_t packD = 0, pack_layerD = 0;  // the same for the draft model
  size_t packDdec = 0;                // the draft decoder's [E; V_k1] and heads in fragment order (row drafting)
  size_t rd_rng = 0;                  // the draft draws' random numbers per sequence and step (row drafting)
  size_t rd_fpart = 0;                // FFN outputs per hidden slice of a non-last layer (row drafting)
  size_t wbT = 0, wbD = 0, wb_nT = 0, wb_nD = 0;   // matrices in the k_block order (0 bytes: not served)
  size_t d_tau, d_t, d_k, d_logg, d_logf, d_mix, d_lt, d_rate;
  size_t v_logg, v_logf, v_mix, v_lt;
  size_t a_L, a_nnew, a_knew, a_tnew, a_taunew, a_ar, a_flags;
};

WsLayout ws_layout(const tppsd_model *T, const tppsd_model *D, int B, int cap, int MG) {
  WsLayout w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    off = align_up(off);
    size_t r = off;
    off += bytes;
    return r;
  };
  const size_t Bz = (size_t)B;
  w.status = take(4);
  w.n_done = take(4);
  w.acc = take((size_t)B * 3 * 8);   // per-sequence counters: accepted drafts, drafted, A-R candidates
  w.n = take(Bz * 4);
  w.gen = take(Bz * 4);
  w.lenT = take(Bz * 4);
  w.lenD = take(Bz * 4);
  w.done = take(Bz * 4);
  w.rnd = take(Bz * 4);
  w.zeros = take(Bz * 4);
  w.ev_t = take(Bz * cap * 4);
  w.ev_k = take(Bz * cap * 4);
  w.t_end = take(Bz * 4);
  w.ll = take(Bz * 8);
  w.freqT = take((size_t)T->d() * 4);
  w.freqD = take(D ? (size_t)D->d() * 4 : 0);
  const size_t kvc = kv_stride(cap);
  w.layerT = Bz * T->H() * kvc * T->dh() * T->act_bytes();
  w.kT = take(w.layerT * T->cfg.n_layers);
  w.vT = take(w.layerT * T->cfg.n_layers);
  w.layerD = D ? Bz * D->H() * kvc * D->dh() * D->act_bytes() : 0;
  w.kD = take(D ? w.layerD * D->cfg.n_layers : 0);
  w.vD = take(D ? w.layerD * D->cfg.n_layers : 0);
  const int Pmax = std::max(MG + 1, PREFILL_CHUNK);
  const size_t Tm = Bz * Pmax;
  const size_t dmax = std::max(T->d(), D ? D->d() : 0);
  const size_t fmax = std::max(T->cfg.d_ffn, D ? D->cfg.d_ffn : 0);
  const size_t mmax = std::max(T->cfg.n_mix, D ? D->cfg.n_mix : 0);
  const size_t kmax = std::max(T->cfg.n_types, D ? D->cfg.n_types : 0);
  w.x = take(Tm * dmax * 4);
  w.a = take(Tm * dmax * 4);
  w.q = take(Tm * dmax * 4);
  w.o = take(Tm * dmax * 4);
  w.hid = take(Tm * fmax * 4);
  w.e = take(Tm * 4 * dmax * 4);
  w.u = take(Tm * 2 * dmax * 4);   // AttNHP layer input [z; h]
  w.logits = take(Tm * head_ldl((int)mmax, (int)kmax) * 4);
  w.hwT = take((size_t)(3 * T->cfg.n_mix + T->cfg.n_types) * 4 * T->d() * T->act_bytes());
  w.hbT = take((size_t)(3 * T->cfg.n_mix + T->cfg.n_types) * 4);
  w.hwD = take(D ? (size_t)(3 * D->cfg.n_mix + D->cfg.n_types) * 4 * D->d() * D->act_bytes() : 0);
  w.hbD = take(D ? (size_t)(3 * D->cfg.n_mix + D->cfg.n_types) * 4 : 0);
  if (!T->attnhp() && layer_fused_ok(T->bf16(), T->d(), T->cfg.d_ffn)) {
    const size_t d = T->d(), F = T->cfg.d_ffn;
    w.pack_layer = (4 * d * d + 2 * d * F) * 2;   // Wo, W1, W2, Wqkv (bf16)
    w.packT = take(w.pack_layer * T->cfg.n_layers);
  }
  // per model: L x (qkv, out, ffn1, ffn2), [E; V_k1], decoder block matrix
  auto wb_bytes = [](const tppsd_model *m) -> size_t {
    if (!m || m->attnhp() || !block_widths(m->d(), m->cfg.d_ffn)) return 0;
    const int d = m->d(), F = m->cfg.d_ffn;
    const size_t layer = wbatch_packed_elems(3 * d, d) + wbatch_packed_elems(d, d) + wbatch_packed_elems(F, d) +
                         wbatch_packed_elems(d, F);
    return (m->cfg.n_layers * layer + wbatch_packed_elems(4 * d, d) +
            wbatch_packed_elems(3 * m->cfg.n_mix + m->cfg.n_types, 4 * d)) * m->act_bytes();
  };
  w.wbT = take(wb_bytes(T));
  w.wbD = take(wb_bytes(D));
  w.wb_nT = wb_bytes(T);
  w.wb_nD = wb_bytes(D);
  if (D && !D->attnhp() && layer_fused_ok(D->bf16(), D->d(), D->cfg.d_ffn)) {
    const size_t d = D->d(), F = D->cfg.d_ffn;
    w.pack_layerD = (4 * d * d + 2 * d * F) * 2;
    w.packD = take(w.pack_layerD * D->cfg.n_layers);
  }
  if (D && !D->attnhp() &&
      row_draft_ok(D->bf16(), D->cfg.n_layers, D->d(), D->H(), D->cfg.d_ffn, D->cfg.n_mix, D->cfg.n_types, (int)kvc)) {
    w.packDdec = take(rd_pack_dec_elems(D->d()) * 2);
    w.rd_rng = take(Bz * MG * 4 * 4);
    w.rd_fpart = take(Bz * RD_FSPLIT * 2 * D->d() * 4);
  }
  w.ar_mix = take(Bz * 3 * mmax * 4);
  w.ar_lt = take(Bz * kmax * 4);
  {
    const int qtm = (Pmax + 15) / 16;
    size_t pf = attn_part_floats(B, T->H(), T->dh(), qtm, (int)kvc);
    if (D) pf = std::max(pf, attn_part_floats(B, D->H(), D->dh(), qtm, (int)kvc));
    if (D && !D->attnhp() &&
        row_draft_ok(D->bf16(), D->cfg.n_layers, D->d(), D->H(), D->cfg.d_ffn, D->cfg.n_mix, D->cfg.n_types,
                     (int)kvc))
      pf = std::max(pf, rd_part_floats(B, D->H(), D->dh(), (int)kvc));
    w.attn_part = take(pf * 4);
  }
  w.gen0 = take(Bz * 4);
  const size_t M = T->cfg.n_mix, K = T->cfg.n_types;
  w.d_tau = take(Bz * MG * 4);
  w.d_t = take(Bz * MG * 4);
  w.d_k = take(Bz * MG * 4);
  w.d_logg = take(Bz * MG * 4);
  w.d_logf = take(Bz * MG * 4);
  w.d_mix = take(Bz * MG * 3 * M * 4);
  w.d_lt = take(Bz * MG * K * 4);
  w.d_rate = take(Bz * 4);
  w.v_logg = take(Bz * MG * 4);
  w.v_logf = take(Bz * MG * 4);
  w.v_mix = take(Bz * (MG + 1) * 3 * M * 4);
  w.v_lt = take(Bz * (MG + 1) * K * 4);
  w.a_L = take(Bz * 4);
  w.a_nnew = take(Bz * 4);
  w.a_knew = take(Bz * (MG + 1) * 4);
  w.a_tnew = take(Bz * (MG + 1) * 4);
  w.a_taunew = take(Bz * (MG + 1) * 4);
  w.a_ar = take(Bz * 4);
  w.a_flags = take(Bz);
  w.total = align_up(off);
  return w;
}

// Block forward of P new positions per sequence through model m (encoder of
// §4.2), keys/values appended at start[b] + start_off + p; optional decoder.
// verify: the target's verify pass (its attention launches carry their own
// kernel name; in kernel-timing mode its attention and GEMM launches are
// bracketed by the events of s->cur_ev: attention of layer l in pair l, GEMM j
// of the pass in pair n_layers + j).
int forward(tppsd_state *s, const tppsd_model *m, const ModelCache &c, const int32_t *start, int start_off,
            int P, const TokSrc &src, const HeadArgs *head, bool verify, hipStream_t st) {
  const int B = s->B, d = m->d(), H = m->H(), dh = m->dh(), F = m->cfg.d_ffn, bf = m->bf16();
  const int T = B * P, L = m->cfg.n_layers;
  const bool timed = verify && s->cur_ev != nullptr;
  auto ev = [&](int pair, int end) -> hipEvent_t {
    if (!timed) return nullptr;
    s->ev_used[pair] = 1;
    return s->cur_ev[2 * pair + end];
  };
  // LayerNorms run inside the GEMMs that consume them where the width allows
  const bool fuse_ln = gemm_ln_fusable(bf, d);
  if (m->attnhp()) {
    // AttNHP (App. D.4): per layer one GEMM over u = [z; h] for q, k, v (keys
    // and values into the cache), attention normalised by 1 + sum f, then
    // h += tanh(o) (refreshing u's h half and the decoder operand a = h)
    launch_embed_attnhp(s->x, s->u, T, d, P, src, m->type_emb, bf, c.freq, m->cfg.n_types, st);
    for (int l = 0; l < L; ++l) {
      const LayerW &w = m->layers[l];
      char *kc = c.k + c.layer_bytes * l, *vc = c.v + c.layer_bytes * l;
      Epi e{};
      e.mode = EPI_QKV;
      e.bias = w.qkv_b;
      e.q = s->q;
      e.kc = kc;
      e.vc = vc;
      e.start = start;
      e.start_off = start_off;
      e.P = P;
      e.H = H;
      e.dh = dh;
      e.d = d;
      e.cap = s->kv_cap;
      e.status = s->status;
      launch_gemm(s->u, nullptr, w.qkv_w, bf, T, 3 * d, 2 * d, e, st, ev(L + 4 * l, 0), ev(L + 4 * l, 1));
      launch_attention(s->q, kc, vc, s->o, bf, start, start_off, s->done, B, P, H, dh, s->kv_cap, s->attn_part,
                       1, verify ? 1 : 0, ev(l, 0), ev(l, 1), st);
      launch_attnhp_update(s->x, s->o, s->u, s->a, bf, T, d, st);
    }
  }
  if (!m->attnhp() && block_fusable(bf, d, F, m->cfg.n_mix, m->cfg.n_types, T)) {
    // small THP models: one k_block launch between consecutive attention
    // launches (embedding + LN1 + QKV; then output projection + FFN + the next
    // LN1 + QKV; the last one ends with LN_f and the decoder). Without a
    // decoder the last layer's output projection and FFN feed nothing and
    // are skipped.
    const int M = m->cfg.n_mix, K = m->cfg.n_types;
    BlockArgs ba{};
    ba.T = T;
    ba.P = P;
    ba.d = d;
    ba.F = F;
    ba.src = src;
    ba.type_emb = m->type_emb;
    ba.freq = c.freq;
    ba.n_types = K;
    ba.x = s->x;
    ba.o = s->o;
    ba.lnf_g = m->lnf_g;
    ba.lnf_b = m->lnf_b;
    ba.k1_b = m->k1_b;
    ba.Ek1_w = c.wb_ek1;   // (k_block reads its matrices in the packed order)
    ba.head_w = c.wb_head;
    ba.head_b = c.head_b;
    ba.M = M;
    ba.K = K;
    if (head) ba.h = *head;
    auto set_qkv = [&](int l) {
      const LayerW &w = m->layers[l];
      ba.qkv_w = c.wb_qkv[l];
      ba.ln1_g = w.ln1_g;
      ba.ln1_b = w.ln1_b;
      Epi &e = ba.qe;
      e = Epi{};
      e.mode = EPI_QKV;
      e.bias = w.qkv_b;
      e.q = s->q;
      e.kc = c.k + c.layer_bytes * l;
      e.vc = c.v + c.layer_bytes * l;
      e.start = start;
      e.start_off = start_off;
      e.P = P;
      e.H = H;
      e.dh = dh;
      e.d = d;
      e.cap = s->kv_cap;
      e.status = s->status;
    };
    ba.first = 1;
    ba.qkv = 1;
    ba.store_x = 1;
    set_qkv(0);
    launch_block(ba, bf, st, ev(L, 0), ev(L, 1));
    for (int l = 0; l < L; ++l) {
      char *kc = c.k + c.layer_bytes * l, *vc = c.v + c.layer_bytes * l;
      launch_attention(s->q, kc, vc, s->o, bf, start, start_off, s->done, B, P, H, dh, s->kv_cap, s->attn_part,
                       0, verify ? 1 : 0, ev(l, 0), ev(l, 1), st);
      const bool last = l + 1 == L;
      if (last && !head) break;
      const LayerW &w = m->layers[l];
      ba.first = 0;
      ba.pre = 1;
      ba.out_w = c.wb_out[l];
      ba.out_b = w.out_b;
      ba.ln2_g = w.ln2_g;
      ba.ln2_b = w.ln2_b;
      ba.ffn1_w = c.wb_f1[l];
      ba.ffn1_b = w.ffn1_b;
      ba.ffn2_w = c.wb_f2[l];
      ba.ffn2_b = w.ffn2_b;
      ba.qkv = !last;
      ba.store_x = !last;
      ba.head = last;
      if (!last) set_qkv(l + 1);
      launch_block(ba, bf, st, ev(L + l + 1, 0), ev(L + l + 1, 1));
    }
    return TPPSD_OK;
  }
  // the row-local part of each layer in one launch (output projection, FFN
  // with its hidden activations on chip, the next layer's q, k, v) where
  // there is an instance for the widths and enough rows to beat the layered kernels;
  // TPPSD_FFN_FUSED=0 / 1 forces the layered / fused form
  const char *ff = getenv("TPPSD_FFN_FUSED");
  char *const pack = m == s->T ? s->packT : s->packD;   // this model's weights in fragment order
  const size_t pack_layer = m == s->T ? s->pack_layer : s->pack_layerD;
  const bool use_layer_fused = fuse_ln && !m->attnhp() && pack && layer_fused_ok(bf, d, F) &&
                               (ff ? ff[0] == '1' : layer_fused_worth(d, T));
  auto qkv_epi = [&](int l) {
    Epi e{};
    e.mode = EPI_QKV;
    e.bias = m->layers[l].qkv_b;
    e.q = s->q;
    e.kc = c.k + c.layer_bytes * l;
    e.vc = c.v + c.layer_bytes * l;
    e.start = start;
    e.start_off = start_off;
    e.P = P;
    e.H = H;
    e.dh = dh;
    e.d = d;
    e.cap = s->kv_cap;
    e.status = s->status;
    return e;
  };
  if (!m->attnhp()) launch_embed(s->x, T, d, P, src, m->type_emb, bf, c.freq, m->cfg.n_types, st);
  // LayerNorm inside the consuming GEMM, or (wide rows, many rows) as its own launch
  const bool ln_gemm = fuse_ln && !gemm_ln_split(bf, d, T);
  for (int l = 0; l < m->cfg.n_layers && !m->attnhp(); ++l) {
    const LayerW &w = m->layers[l];
    char *kc = c.k + c.layer_bytes * l, *vc = c.v + c.layer_bytes * l;
    const LnA ln1{s->x, w.ln1_g, w.ln1_b}, ln2{s->x, w.ln2_g, w.ln2_b};
    if (!(use_layer_fused && l > 0)) {   // (else the previous fused launch wrote this layer's q, k, v)
      if (!ln_gemm) launch_layernorm(s->x, s->a, bf, w.ln1_g, w.ln1_b, T, d, st);
      const Epi e = qkv_epi(l);
      launch_gemm(s->a, ln_gemm ? &ln1 : nullptr, w.qkv_w, bf, T, 3 * d, d, e, st, ev(L + 4 * l, 0),
                  ev(L + 4 * l, 1));
    }
    launch_attention(s->q, kc, vc, s->o, bf, start, start_off, s->done, B, P, H, dh, s->kv_cap, s->attn_part,
                     0, verify ? 1 : 0, ev(l, 0), ev(l, 1), st);
    if (use_layer_fused) {
      LayerArgs la{};
      la.x = s->x;
      la.o = (const bf16_t *)s->o;
      const char *pk = pack + pack_layer * l;   // Wo, W1, W2 of this layer, fragment order
      la.wo = (const bf16_t *)pk;
      la.bo = w.out_b;
      la.ln2_g = w.ln2_g;
      la.ln2_b = w.ln2_b;
      la.w1 = (const bf16_t *)(pk + (size_t)d * d * 2);
      la.b1 = w.ffn1_b;
      la.w2 = (const bf16_t *)(pk + (size_t)(d * d + F * d) * 2);
      la.b2 = w.ffn2_b;
      const bool post = l + 1 < L;
      if (post) {
        const LayerW &wn = m->layers[l + 1];
        la.ln1_g = wn.ln1_g;
        la.ln1_b = wn.ln1_b;
        la.wqkv = (const bf16_t *)(pack + pack_layer * (l + 1) + (size_t)(d * d + 2 * F * d) * 2);
        la.qe = qkv_epi(l + 1);
      }
      la.T = T;
      launch_layer_fused(la, d, F, post, st, ev(L + 4 * l + 1, 0), ev(L + 4 * l + 1, 1));
      continue;
    }
    Epi eo{};
    eo.mode = EPI_RESID;
    eo.bias = w.out_b;
    eo.out = s->x;
    eo.ldo = d;
    launch_gemm(s->o, nullptr, w.out_w, bf, T, d, d, eo, st, ev(L + 4 * l + 1, 0), ev(L + 4 * l + 1, 1));
    if (!ln_gemm) launch_layernorm(s->x, s->a, bf, w.ln2_g, w.ln2_b, T, d, st);
    Epi e1{};
    e1.mode = EPI_RELU;
    e1.bias = w.ffn1_b;
    e1.out = s->hid;
    e1.ldo = F;
    launch_gemm(s->a, ln_gemm ? &ln2 : nullptr, w.ffn1_w, bf, T, F, d, e1, st, ev(L + 4 * l + 2, 0), ev(L + 4 * l + 2, 1));
    Epi e2{};
    e2.mode = EPI_RESID;
    e2.bias = w.ffn2_b;
    e2.out = s->x;
    e2.ldo = d;
    launch_gemm(s->hid, nullptr, w.ffn2_w, bf, T, d, F, e2, st, ev(L + 4 * l + 3, 0), ev(L + 4 * l + 3, 1));
  }
  if (head) {
    // THP: the decoder reads LN_f(x); AttNHP: h itself (a, written by the update)
    const LnA lnf{s->x, m->lnf_g, m->lnf_b};
    const bool ln_in_gemm = fuse_ln && !m->attnhp() && !gemm_ln_split(bf, d, T);
    if (!ln_in_gemm && !m->attnhp()) launch_layernorm(s->x, s->a, bf, m->lnf_g, m->lnf_b, T, d, st);
    Epi eh{};
    eh.mode = EPI_HEAD;
    eh.bias = m->k1_b;
    eh.out = s->e;
    eh.ldo = 4 * d;
    eh.split = 3 * d;
    launch_gemm(s->a, ln_in_gemm ? &lnf : nullptr, m->Ek1_w, bf, T, 4 * d, d, eh, st, ev(5 * L, 0), ev(5 * L, 1));
    const int M = m->cfg.n_mix, K = m->cfg.n_types, ldl = head_ldl(M, K);
    Epi el{};
    el.mode = EPI_F32;
    el.bias = c.head_b;
    el.out = s->logits;
    el.ldo = ldl;
    launch_gemm(s->e, nullptr, c.head_w, bf, T, 3 * M + K, 4 * d, el, st);
    launch_head(s->logits, ldl, M, K, *head, st);
  }
  return TPPSD_OK;
}

HeadArgs head_common(tppsd_state *s) {
  HeadArgs h{};
  h.B = s->B;
  h.ev_t = s->ev_t;
  h.ev_k = s->ev_k;
  h.ev_stride = s->cap;
  h.n = s->n;
  h.gen = s->gen;
  h.lenT = s->lenT;
  h.done = s->done;
  h.rnd = s->rnd;
  h.n_done = s->n_done;
  h.n_gen = s->n_gen;
  h.t_end = s->t_end;
  h.ll = s->ll;
  h.seed = s->seed;
  h.status = s->status;
  return h;
}

int check_draft_buf(const tppsd_draft_buf *b) {
  if (!b || !b->tau || !b->t || !b->k || !b->logg || !b->logf || (!b->mix && !b->rate) || !b->logtype)
    return fail(TPPSD_E_ARG, "draft buffer has a null pointer");
  return TPPSD_OK;
}
int check_verify_buf(const tppsd_verify_buf *b) {
  if (!b || !b->logg || !b->logf || !b->mix || !b->logtype)
    return fail(TPPSD_E_ARG, "verify buffer has a null pointer");
  return TPPSD_OK;
}
int check_accept_buf(const tppsd_accept_buf *b) {
  if (!b || !b->L || !b->n_new || !b->k_new || !b->t_new || !b->tau_new || !b->ar_iter || !b->flags)
    return fail(TPPSD_E_ARG, "accept buffer has a null pointer");
  return TPPSD_OK;
}

DraftArgs draft_args(tppsd_state *s, int gamma, const tppsd_draft_buf *out) {
  const tppsd_model *D = s->D;
  DraftArgs a{};
  a.B = s->B;
  a.gamma = gamma;
  a.d = D->d();
  a.H = D->H();
  a.F = D->cfg.d_ffn;
  a.M = D->cfg.n_mix;
  a.K = D->cfg.n_types;
  a.L = D->cfg.n_layers;
  for (int l = 0; l < a.L; ++l) {
    const LayerW &w = D->layers[l];
    a.layer[l] = {w.qkv_w, w.out_w, w.ffn1_w, w.ffn2_w, w.ln1_g, w.ln1_b, w.qkv_b,
                  w.out_b, w.ln2_g, w.ln2_b, w.ffn1_b, w.ffn2_b};
  }
  a.type_emb = D->type_emb;
  a.Ek1_w = D->Ek1_w;
  a.mix_w = D->mix_w;
  a.k2_w = D->k2_w;
  a.lnf_g = D->lnf_g;
  a.lnf_b = D->lnf_b;
  a.k1_b = D->k1_b;
  a.mix_b = D->mix_b;
  a.k2_b = D->k2_b;
  a.freq = s->cD.freq;
  a.kc = s->cD.k;
  a.vc = s->cD.v;
  a.layer_bytes = s->cD.layer_bytes;
  a.cap = s->kv_cap;
  a.ev_t = s->ev_t;
  a.ev_k = s->ev_k;
  a.ev_stride = s->cap;
  a.n = s->n;
  a.lenD = s->lenD;
  a.done = s->done;
  a.rnd = s->rnd;
  a.seed = s->seed;
  a.status = s->status;
  a.d_tau = out->tau;
  a.d_t = out->t;
  a.d_logg = out->logg;
  a.d_logf = out->logf;
  a.d_mix = out->mix;
  a.d_logtype = out->logtype;
  a.d_k = out->k;
  a.MG = s->max_gamma;
  a.w_lds = s->fused_w_lds ? 1 : 0;
  return a;
}

int do_draft_fused(tppsd_state *s, int gamma, const tppsd_draft_buf *out, hipStream_t st) {
  const tppsd_model *D = s->D;
  const DraftArgs a = draft_args(s, gamma, out);
  // kernel timing: the pair after the verify pass's attention and GEMM pairs
  const int dp = 5 * s->T->cfg.n_layers + 1;
  const bool timed = s->cur_ev != nullptr;
  if (timed) s->ev_used[dp] = 1;
  if (s->wave_draft)
    launch_draft_wave(a, D->bf16(), st, timed ? s->cur_ev[2 * dp] : nullptr, timed ? s->cur_ev[2 * dp + 1] : nullptr);
  else
    launch_draft_fused(a, D->bf16(), st, timed ? s->cur_ev[2 * dp] : nullptr,
                       timed ? s->cur_ev[2 * dp + 1] : nullptr);
  return hip_check("tppsd_draft");
}

int do_draft_rows(tppsd_state *s, int gamma, const tppsd_draft_buf *out, hipStream_t st) {
  RowDraftArgs a{};
  a.d = draft_args(s, gamma, out);
  a.x = s->x;
  a.xn = (bf16_t *)s->a;
  a.part = s->attn_part;
  a.rng = s->rd_rng;
  a.fpart = s->rd_fpart;
  a.pk = (const bf16_t *)s->packD;
  a.pk_e = (const bf16_t *)s->packDdec;
  a.pk_head = (const bf16_t *)(s->packDdec + (size_t)4 * s->D->d() * s->D->d() * 2);
  a.S = rd_splits(s->kv_cap);
  // kernel timing: a pair per launch, after the verify pass's and the one-launch draft's pairs
  const int p0 = 5 * s->T->cfg.n_layers + 2, nl = rd_launches(a.d.L, gamma);
  const bool timed = s->cur_ev != nullptr && (int)s->ev_used.size() >= p0 + nl;
  if (timed)
    for (int j = 0; j < nl; ++j) s->ev_used[p0 + j] = 1;
  launch_draft_rows(a, st, timed ? s->cur_ev + 2 * p0 : nullptr);
  return hip_check("tppsd_draft");
}

int do_draft(tppsd_state *s, int gamma, const tppsd_draft_buf *out, hipStream_t st) {
  const tppsd_model *D = s->D;
  if (s->wave_draft || s->fused_draft) return do_draft_fused(s, gamma, out, st);
  if (s->row_draft) return do_draft_rows(s, gamma, out, st);
  for (int l = 1; l <= gamma; ++l) {
    TokSrc src{};
    src.ev_t = s->ev_t;
    src.ev_k = s->ev_k;
    src.ev_stride = s->cap;
    src.start = s->lenD;
    src.dr_t = out->t;
    src.dr_k = out->k;
    src.dr_stride = s->max_gamma;
    HeadArgs h = head_common(s);
    h.mode = HEAD_DRAFT;
    h.mix = out->mix;
    h.logtype = out->logtype;
    h.dst_stride = s->max_gamma;
    h.dst_row0 = l - 1;
    h.dr_stride = s->max_gamma;
    h.d_tau = out->tau;
    h.d_t = out->t;
    h.d_k = out->k;
    h.d_logg = out->logg;
    h.d_logf = out->logf;
    h.slot = l - 1;
    h.l_index = l;
    int P, off;
    if (l == 1) {   // re-encode the last two committed events at lenD, lenD + 1
      P = 2;
      off = 0;
      src.start_off = 0;
      src.n_ev = 2;
      src.dr_off = 0;
    } else {        // draft l - 1 at lenD + l
      P = 1;
      off = l;
      src.start_off = l;
      src.n_ev = 0;
      src.dr_off = l - 2;
    }
    h.P = P;
    h.p0 = P - 1;
    int rc = forward(s, D, s->cD, s->lenD, off, P, src, &h, false, st);
    if (rc) return rc;
  }
  return hip_check("tppsd_draft");
}

int do_draft_poisson(tppsd_state *s, int gamma, const float *params, const tppsd_draft_buf *out, hipStream_t st) {
  PoissonDraftArgs a{};
  a.B = s->B;
  a.gamma = gamma;
  a.K = s->T->cfg.n_types;
  a.MG = s->max_gamma;
  a.params = params;
  a.ev_t = s->ev_t;
  a.ev_stride = s->cap;
  a.n = s->n;
  a.done = s->done;
  a.rnd = s->rnd;
  a.seed = s->seed;
  a.status = s->status;
  a.d_tau = out->tau;
  a.d_t = out->t;
  a.d_k = out->k;
  a.d_logg = out->logg;
  a.d_logf = out->logf;
  a.d_logtype = out->logtype;
  a.d_rate = out->rate;
  launch_draft_poisson(a, st);
  return hip_check("tppsd_draft_poisson");
}

int do_verify(tppsd_state *s, int gamma, const tppsd_draft_buf *in, const tppsd_verify_buf *out, hipStream_t st) {
  TokSrc src{};
  src.ev_t = s->ev_t;
  src.ev_k = s->ev_k;
  src.ev_stride = s->cap;
  src.start = s->lenT;
  src.start_off = 0;
  src.n_ev = 1;
  src.dr_t = in->t;
  src.dr_k = in->k;
  src.dr_stride = s->max_gamma;
  src.dr_off = 0;
  HeadArgs h = head_common(s);
  h.mode = HEAD_VERIFY;
  h.P = gamma + 1;
  h.p0 = 0;
  h.mix = out->mix;
  h.logtype = out->logtype;
  h.dst_stride = s->max_gamma + 1;
  h.dst_row0 = 0;
  h.gamma = gamma;
  h.dr_tau = in->tau;
  h.dr_k = in->k;
  h.dr_stride = s->max_gamma;
  h.v_logg = out->logg;
  h.v_logf = out->logf;
  const tppsd_model *m = s->T;
  if (!m->attnhp() &&
      verify_seq_ok(m->bf16(), m->cfg.n_layers, m->d(), m->H(), m->cfg.d_ffn, m->cfg.n_mix, m->cfg.n_types,
                    gamma + 1)) {
    // small targets: the whole pass of a sequence in one workgroup
    VerifySeqArgs a{};
    a.P = gamma + 1;
    a.d = m->d();
    a.F = m->cfg.d_ffn;
    a.H = m->H();
    a.L = m->cfg.n_layers;
    a.M = m->cfg.n_mix;
    a.K = m->cfg.n_types;
    for (int l = 0; l < a.L; ++l) {
      const LayerW &w = m->layers[l];
      // (k_verify_seq reads its matrices in the packed order)
      a.layer[l] = {s->cT.wb_qkv[l], s->cT.wb_out[l], s->cT.wb_f1[l], s->cT.wb_f2[l], w.ln1_g, w.ln1_b, w.qkv_b,
                    w.out_b, w.ln2_g, w.ln2_b, w.ffn1_b, w.ffn2_b};
    }
    a.type_emb = m->type_emb;
    a.Ek1_w = s->cT.wb_ek1;
    a.head_w = s->cT.wb_head;
    a.lnf_g = m->lnf_g;
    a.lnf_b = m->lnf_b;
    a.k1_b = m->k1_b;
    a.head_b = s->cT.head_b;
    a.freq = s->cT.freq;
    a.kc = s->cT.k;
    a.vc = s->cT.v;
    a.layer_bytes = s->cT.layer_bytes;
    a.cap = s->kv_cap;
    a.ev_t = s->ev_t;
    a.ev_k = s->ev_k;
    a.ev_stride = s->cap;
    a.lenT = s->lenT;
    a.done = s->done;
    a.dr_t = in->t;
    a.dr_k = in->k;
    a.dr_stride = s->max_gamma;
    a.status = s->status;
    a.h = h;
    const bool timed = s->cur_ev != nullptr;
    if (timed) s->ev_used[m->cfg.n_layers] = 1;
    launch_verify_seq(a, s->B, m->bf16(), st, timed ? s->cur_ev[2 * m->cfg.n_layers] : nullptr,
                      timed ? s->cur_ev[2 * m->cfg.n_layers + 1] : nullptr);
    return hip_check("tppsd_verify");
  }
  int rc = forward(s, s->T, s->cT, s->lenT, 0, gamma + 1, src, &h, true, st);
  if (rc) return rc;
  return hip_check("tppsd_verify");
}

int do_accept(tppsd_state *s, int gamma, const tppsd_draft_buf *dr, const tppsd_verify_buf *vf, const float *u,
              const tppsd_accept_buf *out, hipStream_t st) {
  AcceptArgs a{};
  a.B = s->B;
  a.gamma = gamma;
  a.M = s->T->cfg.n_mix;
  a.K = s->T->cfg.n_types;
  a.max_gamma = s->max_gamma;
  a.bonus = (s->flags & TPPSD_FLAG_BONUS) ? 1 : 0;
  a.d_tau = dr->tau;
  a.d_t = dr->t;
  a.d_k = dr->k;
  a.d_logg = dr->logg;
  a.d_logf = dr->logf;
  a.d_mix = dr->mix;
  a.d_logtype = dr->logtype;
  a.v_logg = vf->logg;
  a.v_logf = vf->logf;
  a.v_mix = vf->mix;
  a.v_logtype = vf->logtype;
  a.uniforms = u;
  a.d_rate = dr->rate;
  a.L = out->L;
  a.n_new = out->n_new;
  a.k_new = out->k_new;
  a.ar_iter = out->ar_iter;
  a.t_new = out->t_new;
  a.tau_new = out->tau_new;
  a.flags = out->flags;
  a.ev_t = s->ev_t;
  a.ev_k = s->ev_k;
  a.ev_stride = s->cap;
  a.n = s->n;
  a.gen = s->gen;
  a.lenT = s->lenT;
  a.lenD = s->lenD;
  a.done = s->done;
  a.rnd = s->rnd;
  a.n_done = s->n_done;
  a.n_gen = s->n_gen;
  a.t_end = s->t_end;
  a.ll = s->ll;
  a.seed = s->seed;
  a.status = s->status;
  a.acc_stats = s->acc_stats;
  launch_accept(a, st);
  return hip_check("tppsd_accept");
}

// ---- allocation-free verification -------------------------------------------
// tppsd_verify_noalloc runs the verify pass with its activation scratch (the
// residual stream, LayerNorm / attention / FFN / decoder activations, the
// decoder logits and the attention key-split partials) in a file-scope
// device array instead of the state's workspace, so that the call needs no
// memory of the caller's beyond the state, its inputs and its outputs. Each
// GPU that runs it holds the array until the process ends; every call on a
// GPU shares that GPU's copy (overlapping calls on one GPU race).
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) char scratch[NOALLOC_SCRATCH_BYTES];

constexpr int NOALLOC_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char *g_scratch[NOALLOC_MAX_DEVICES] = {};

// the device address of the current device's copy of `scratch`, resolved once
// per device (in host code the array's name only stands in for it)
int scratch_base(char **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return hip_check("tppsd_verify_noalloc: current device");
  if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return fail(TPPSD_E_HIP, "device %d outside the scratch table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(TPPSD_E_HIP, "tppsd_verify_noalloc: scratch address: %s", hipGetErrorString(e));
    g_scratch[dev] = (char *)p;
  }
  *out = g_scratch[dev];
  return TPPSD_OK;
}

// offsets of the verify pass's activation scratch for B sequences of P rows
// (the same per-buffer sizes as the state's workspace, for B * P rows)
struct ScratchLayout {
  size_t x, a, q, o, hid, e, u, logits, attn_part, total;
};
ScratchLayout scratch_layout(const tppsd_model *T, const tppsd_model *D, int B, int P, int kvc) {
  ScratchLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    off = align_up(off);
    const size_t r = off;
    off += bytes;
    return r;
  };
  const size_t Tm = (size_t)B * P;
  const size_t dmax = std::max(T->d(), D ? D->d() : 0);
  const size_t fmax = std::max(T->cfg.d_ffn, D ? D->cfg.d_ffn : 0);
  const size_t mmax = std::max(T->cfg.n_mix, D ? D->cfg.n_mix : 0);
  const size_t kmax = std::max(T->cfg.n_types, D ? D->cfg.n_types : 0);
  L.x = take(Tm * dmax * 4);
  L.a = take(Tm * dmax * 4);
  L.q = take(Tm * dmax * 4);
  L.o = take(Tm * dmax * 4);
  L.hid = take(Tm * fmax * 4);
  L.e = take(Tm * 4 * dmax * 4);
  L.u = take(Tm * 2 * dmax * 4);
  L.logits = take(Tm * head_ldl((int)mmax, (int)kmax) * 4);
  L.attn_part = take(attn_part_floats(B, T->H(), T->dh(), (P + 15) / 16, kvc) * 4);
  L.total = align_up(off);
  return L;
}

}  // namespace

extern "C" {

const char *tppsd_last_error(void) { return g_err.c_str(); }

int tppsd_weights_bytes(const tppsd_model_cfg *cfg, size_t *bytes) {
  if (int rc = check_cfg(cfg)) return rc;
  if (!bytes) return fail(TPPSD_E_ARG, "null output pointer");
  *bytes = layout(*cfg).back().off;
  return TPPSD_OK;
}

int tppsd_weights_entry(const tppsd_model_cfg *cfg, int index, const char **name, size_t *offset, int64_t *rows,
                        int64_t *cols, int *is_bf16) {
  if (int rc = check_cfg(cfg)) return rc;
  static thread_local std::vector<Entry> cache;
  cache = layout(*cfg);
  if (index < 0 || index >= (int)cache.size() - 1) return fail(TPPSD_E_ARG, "weight entry %d out of range", index);
  const Entry &e = cache[index];
  // names live in a static table so the pointer outlives this call
  static thread_local std::vector<std::string> names;
  if ((int)names.size() <= index) names.resize(index + 1);
  names[index] = e.name;
  if (name) *name = names[index].c_str();
  if (offset) *offset = e.off;
  if (rows) *rows = e.rows;
  if (cols) *cols = e.cols;
  if (is_bf16) *is_bf16 = e.bf16;
  return TPPSD_OK;
}

int tppsd_model_create(const tppsd_model_cfg *cfg, const void *d_weights, tppsd_model **out) {
  if (int rc = check_cfg(cfg)) return rc;
  if (!d_weights || !out) return fail(TPPSD_E_ARG, "null weights or output pointer");
  if ((uintptr_t)d_weights % ALIGN) return fail(TPPSD_E_ARG, "weights must be 256-byte aligned");
  std::vector<Entry> L = layout(*cfg);
  auto find = [&](const std::string &n) -> const char * {
    for (const Entry &e : L)
      if (e.name == n) return (const char *)d_weights + e.off;
    return nullptr;
  };
  tppsd_model *m = new tppsd_model();
  m->cfg = *cfg;
  m->w = (const char *)d_weights;
  m->type_emb = find("type_emb");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    LayerW w;
    w.ln1_g = (const float *)find(p + "ln1.g");
    w.ln1_b = (const float *)find(p + "ln1.b");
    w.qkv_w = find(p + "qkv.w");
    w.qkv_b = (const float *)find(p + "qkv.b");
    w.out_w = find(p + "out.w");
    w.out_b = (const float *)find(p + "out.b");
    w.ln2_g = (const float *)find(p + "ln2.g");
    w.ln2_b = (const float *)find(p + "ln2.b");
    w.ffn1_w = find(p + "ffn1.w");
    w.ffn1_b = (const float *)find(p + "ffn1.b");
    w.ffn2_w = find(p + "ffn2.w");
    w.ffn2_b = (const float *)find(p + "ffn2.b");
    m->layers.push_back(w);
  }
  m->lnf_g = (const float *)find("lnf.g");
  m->lnf_b = (const float *)find("lnf.b");
  m->Ek1_w = find("head.E");
  m->k1_b = (const float *)find("head.k1.b");
  m->mix_w = find("head.w.w");
  m->mix_b = (const float *)find("head.w.b");
  m->k2_w = find("head.k2.w");
  m->k2_b = (const float *)find("head.k2.b");
  *out = m;
  return TPPSD_OK;
}

void tppsd_model_destroy(tppsd_model *m) { delete m; }

int tppsd_state_bytes(const tppsd_model *T, const tppsd_model *D, int B, int max_events, int max_gamma,
                      size_t *bytes) {
  if (!T || !bytes) return fail(TPPSD_E_ARG, "null target model or output pointer");
  if (B < 1 || max_events < 3 || max_gamma < 1 || max_gamma > TPPSD_MAX_GAMMA)
    return fail(TPPSD_E_ARG, "need B >= 1, max_events >= 3, 1 <= max_gamma <= %d", TPPSD_MAX_GAMMA);
  if (D && (D->cfg.n_mix != T->cfg.n_mix || D->cfg.n_types != T->cfg.n_types))
    return fail(TPPSD_E_CONFIG, "draft and target must share n_mix and n_types");
  *bytes = ws_layout(T, D, B, max_events, max_gamma).total;
  return TPPSD_OK;
}

int tppsd_state_create(const tppsd_model *T, const tppsd_model *D, int B, int max_events, int max_gamma,
                       uint64_t seed, unsigned flags, void *d_ws, size_t ws_bytes, tppsd_state **out) {
  size_t need = 0;
  if (int rc = tppsd_state_bytes(T, D, B, max_events, max_gamma, &need)) return rc;
  if (!d_ws || !out) return fail(TPPSD_E_ARG, "null workspace or output pointer");
  if ((uintptr_t)d_ws % ALIGN) return fail(TPPSD_E_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need) return fail(TPPSD_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if (flags & ~TPPSD_FLAG_BONUS) return fail(TPPSD_E_ARG, "unknown flags 0x%x", flags);
  const WsLayout w = ws_layout(T, D, B, max_events, max_gamma);
  tppsd_state *s = new tppsd_state();
  s->T = T;
  s->D = D;
  s->B = B;
  s->cap = max_events;
  s->kv_cap = kv_stride(max_events);
  s->max_gamma = max_gamma;
  s->Pmax = std::max(max_gamma + 1, PREFILL_CHUNK);
  s->seed = seed;
  s->flags = flags;
  char *ws = (char *)d_ws;
  s->ws = ws;
  s->status = (uint32_t *)(ws + w.status);
  s->n_done = (int32_t *)(ws + w.n_done);
  s->acc_stats = (unsigned long long *)(ws + w.acc);
  s->n = (int32_t *)(ws + w.n);
  s->gen = (int32_t *)(ws + w.gen);
  s->lenT = (int32_t *)(ws + w.lenT);
  s->lenD = (int32_t *)(ws + w.lenD);
  s->done = (int32_t *)(ws + w.done);
  s->rnd = (int32_t *)(ws + w.rnd);
  s->zeros = (int32_t *)(ws + w.zeros);
  s->ev_t = (float *)(ws + w.ev_t);
  s->ev_k = (int32_t *)(ws + w.ev_k);
  s->t_end = (float *)(ws + w.t_end);
  s->ll = (double *)(ws + w.ll);
  s->cT.k = ws + w.kT;
  s->cT.v = ws + w.vT;
  s->cT.layer_bytes = w.layerT;
  s->cT.freq = (float *)(ws + w.freqT);
  if (D) {
    s->cD.k = ws + w.kD;
    s->cD.v = ws + w.vD;
    s->cD.layer_bytes = w.layerD;
    s->cD.freq = (float *)(ws + w.freqD);
  }
  s->x = (float *)(ws + w.x);
  s->a = ws + w.a;
  s->q = ws + w.q;
  s->o = ws + w.o;
  s->hid = ws + w.hid;
  s->e = ws + w.e;
  s->u = ws + w.u;
  s->logits = (float *)(ws + w.logits);
  s->packT = w.pack_layer ? ws + w.packT : nullptr;
  s->pack_layer = w.pack_layer;
  s->packD = w.pack_layerD ? ws + w.packD : nullptr;
  s->packDdec = w.packDdec ? ws + w.packDdec : nullptr;
  s->rd_rng = w.rd_rng ? (float *)(ws + w.rd_rng) : nullptr;
  s->rd_fpart = w.rd_fpart ? (float *)(ws + w.rd_fpart) : nullptr;
  s->pack_layerD = w.pack_layerD;
  s->cT.wb = w.wb_nT ? ws + w.wbT : nullptr;
  s->cD.wb = w.wb_nD ? ws + w.wbD : nullptr;
  s->cT.head_w = ws + w.hwT;
  s->cT.head_b = (float *)(ws + w.hbT);
  if (D) {
    s->cD.head_w = ws + w.hwD;
    s->cD.head_b = (float *)(ws + w.hbD);
  }
  s->ar_mix = (float *)(ws + w.ar_mix);
  s->ar_logtype = (float *)(ws + w.ar_lt);
  s->attn_part = (float *)(ws + w.attn_part);
  s->gen0 = (int32_t *)(ws + w.gen0);
  s->idr = {(float *)(ws + w.d_tau), (float *)(ws + w.d_t), (int32_t *)(ws + w.d_k), (float *)(ws + w.d_logg),
            (float *)(ws + w.d_logf), (float *)(ws + w.d_mix), (float *)(ws + w.d_lt), nullptr};
  s->idr_p = s->idr;
  s->idr_p.rate = (float *)(ws + w.d_rate);
  s->ivf = {(float *)(ws + w.v_logg), (float *)(ws + w.v_logf), (float *)(ws + w.v_mix), (float *)(ws + w.v_lt)};
  s->iac = {(int32_t *)(ws + w.a_L),      (int32_t *)(ws + w.a_nnew), (int32_t *)(ws + w.a_knew),
            (float *)(ws + w.a_tnew),     (float *)(ws + w.a_taunew), (int32_t *)(ws + w.a_ar),
            (uint8_t *)(ws + w.a_flags)};
  // frequency tables of the temporal encoding, float32: THP 10000^(-(j - j mod 2) / d),
  // AttNHP 1 / (m (5M/m)^((j - j mod 2) / d))
  for (int which = 0; which < (D ? 2 : 1); ++which) {
    const tppsd_model *m = which ? D : T;
    std::vector<float> f(m->d());
    for (int j = 0; j < m->d(); ++j) {
      const double e = (double)(j - j % 2) / (double)m->d();
      if (m->attnhp()) {
        const double tm = m->cfg.time_m, tM = m->cfg.time_M;
        f[j] = (float)(1.0 / (tm * pow(5.0 * tM / tm, e)));
      } else {
        f[j] = (float)pow(10000.0, -e);
      }
    }
    float *dst = which ? s->cD.freq : s->cT.freq;
    if (hipMemcpy(dst, f.data(), f.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
      delete s;
      return hip_check("tppsd_state_create: frequency table upload");
    }
  }
  {
    if (hipStreamCreateWithFlags(&s->cap_stream, hipStreamNonBlocking) != hipSuccess) {
      tppsd_state_destroy(s);
      return hip_check("tppsd_state_create: capture stream");
    }
    const char *nf = getenv("TPPSD_LAYERED_DRAFT");
    // one workgroup per sequence: worth it until the batch alone fills the chip
    // and the layered kernels amortise weights and latency over many rows
    // (and while contexts stay short: the whole sequence's draft cache
    // streams through one CU per step)
    s->fused_draft = D && !D->attnhp() && B <= 1024 && max_events <= 2048 &&
                     fused_draft_ok(D->cfg.n_layers, D->d(), D->H(), D->cfg.d_ffn) &&
                     fused_draft_lds_bytes(D->cfg.n_layers, D->d(), D->cfg.d_ffn, D->cfg.n_mix, D->cfg.n_types,
                                           D->H()) <= 64 * 1024 &&
                     !(nf && nf[0] == '1');
    // its weight matrices in LDS when they fit beside the rest and each
    // workgroup has a CU to itself anyway (one workgroup per sequence)
    const int wb = D && D->bf16() ? 2 : 4;
    s->fused_w_lds = s->fused_draft && B <= 256 &&
                     fused_draft_lds_bytes(D->cfg.n_layers, D->d(), D->cfg.d_ffn, D->cfg.n_mix, D->cfg.n_types,
                                           D->H()) +
                             fused_draft_weight_elems(D->cfg.n_layers, D->d(), D->cfg.d_ffn, D->cfg.n_mix,
                                                      D->cfg.n_types, 16 / wb) * wb <=
                         LDS_PER_WG - 4096;
    if (s->fused_w_lds && allow_draft_fused_lds(LDS_PER_WG - 4096)) {
      s->fused_w_lds = false;       // weights stay in global memory
      (void)hipGetLastError();      // the refused attribute is not an error of this call
    }
    // small draft models: one wave per sequence, the weights in LDS, where
    // the batch fills the chip with one wave per sequence or is tiny (a
    // workgroup's barriers then cost more than its extra lanes save).
    // Measured, draft us per round (wave / one workgroup per sequence /
    // per-step kernels): 4096 sequences 309 / - / 376, 64 sequences 222 /
    // 147 / 299, 1 sequence 47 / 61 / 128
    s->wave_draft = D && !D->attnhp() && !(nf && nf[0] == '1') && (B >= 1024 || B <= 8) &&
                    wave_draft_ok(D->cfg.n_layers, D->d(), D->H(), D->cfg.d_ffn, D->cfg.n_mix, D->cfg.n_types,
                                  D->bf16());
    if (s->wave_draft && allow_draft_wave_lds(LDS_PER_WG - 4096)) {
      s->wave_draft = false;
      (void)hipGetLastError();
    }
    // otherwise, for batches too small to fill the chip with per-step GEMM
    // tiles, the per-step split attention and the row workgroups per sequence
    s->row_draft = D && !D->attnhp() && !s->fused_draft && !s->wave_draft && !(nf && nf[0] == '1') &&
                   B <= 256 && s->packD && s->packDdec &&
                   row_draft_ok(D->bf16(), D->cfg.n_layers, D->d(), D->H(), D->cfg.d_ffn, D->cfg.n_mix,
                                D->cfg.n_types, s->kv_cap);
  }
  if (hipHostMalloc((void **)&s->host_ndone, 2 * sizeof(int32_t), hipHostMallocDefault) != hipSuccess ||
      hipEventCreateWithFlags(&s->poll_ev[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&s->poll_ev[1], hipEventDisableTiming) != hipSuccess) {
    tppsd_state_destroy(s);
    return hip_check("tppsd_state_create: host buffers");
  }
  *out = s;
  return TPPSD_OK;
}

void tppsd_state_destroy(tppsd_state *s) {
  if (!s) return;
  if (s->host_ndone) (void)hipHostFree(s->host_ndone);
  for (hipEvent_t e : s->poll_ev)
    if (e) (void)hipEventDestroy(e);
  drop_graph(&s->sd_exec[0]);
  drop_graph(&s->sd_exec[1]);
  for (hipGraphExec_t &g : s->phase_exec) drop_graph(&g);
  for (auto &v : s->gev)
    for (hipEvent_t e : v) (void)hipEventDestroy(e);
  for (auto &v : s->pev)
    for (hipEvent_t e : v) (void)hipEventDestroy(e);
  drop_graph(&s->ar_exec[0]);
  drop_graph(&s->ar_exec[1]);
  if (s->cap_stream) (void)hipStreamDestroy(s->cap_stream);
  delete s;
}

int tppsd_prefill(tppsd_state *s, const float *d_t, const int32_t *d_k, int n0, int n_gen, hipStream_t st) {
  return tppsd_prefill_window(s, d_t, d_k, n0, n_gen, nullptr, st);
}

int tppsd_prefill_window(tppsd_state *s, const float *d_t, const int32_t *d_k, int n0, int n_gen,
                         const float *d_t_end, hipStream_t st) {
  if (!s || !d_t || !d_k) return fail(TPPSD_E_ARG, "null argument");
  if (n0 < 2 || n_gen < 0) return fail(TPPSD_E_ARG, "need n0 >= 2 and n_gen >= 0");
  if ((long long)n0 + n_gen + s->max_gamma + 1 > s->cap)
    return fail(TPPSD_E_ARG, "n0 + n_gen + max_gamma + 1 = %lld exceeds max_events %d",
                (long long)n0 + n_gen + s->max_gamma + 1, s->cap);
  s->n_gen = n_gen;
  if (!s->heads_built) {
    for (int which = 0; which < (s->D ? 2 : 1); ++which) {
      const tppsd_model *m = which ? s->D : s->T;
      const ModelCache &c = which ? s->cD : s->cT;
      launch_build_head(m->mix_w, m->k2_w, m->mix_b, m->k2_b, m->bf16(), m->d(), m->cfg.n_mix, m->cfg.n_types,
                        c.head_w, c.head_b, st);
    }
    s->heads_built = true;
  }
  if (!s->wb_built) {
    for (int which = 0; which < 2; ++which) {
      const tppsd_model *m = which ? s->D : s->T;
      ModelCache &c = which ? s->cD : s->cT;
      if (!m || !c.wb) continue;
      const int d = m->d(), F = m->cfg.d_ffn, bf = m->bf16(), eb = m->act_bytes();
      char *p = c.wb;
      auto put = [&](const void *W, int N, int K) {
        launch_pack_wbatch(W, N, K, bf, p, st);
        const void *r = p;
        p += wbatch_packed_elems(N, K) * eb;
        return r;
      };
      c.wb_qkv.clear();
      c.wb_out.clear();
      c.wb_f1.clear();
      c.wb_f2.clear();
      for (int l = 0; l < m->cfg.n_layers; ++l) {
        const LayerW &w = m->layers[l];
        c.wb_qkv.push_back(put(w.qkv_w, 3 * d, d));
        c.wb_out.push_back(put(w.out_w, d, d));
        c.wb_f1.push_back(put(w.ffn1_w, F, d));
        c.wb_f2.push_back(put(w.ffn2_w, d, F));
      }
      c.wb_ek1 = put(m->Ek1_w, 4 * d, d);
      c.wb_head = put(c.head_w, 3 * m->cfg.n_mix + m->cfg.n_types, 4 * d);
    }
    s->wb_built = true;
  }
  if (!s->packs_built) {
    for (int which = 0; which < 2; ++which) {
      const tppsd_model *m = which ? s->D : s->T;
      char *base = which ? s->packD : s->packT;
      const size_t stride = which ? s->pack_layerD : s->pack_layer;
      if (!m || !base) continue;
      const int d = m->d(), F = m->cfg.d_ffn;
      for (int l = 0; l < m->cfg.n_layers; ++l) {
        const LayerW &w = m->layers[l];
        char *p = base + stride * l;
        launch_pack_frags(w.out_w, d, d, p, st);
        launch_pack_frags(w.ffn1_w, F, d, p + (size_t)d * d * 2, st);
        launch_pack_frags(w.ffn2_w, d, F, p + (size_t)(d * d + F * d) * 2, st);
        launch_pack_frags(w.qkv_w, 3 * d, d, p + (size_t)(d * d + 2 * F * d) * 2, st);
      }
      if (which && s->packDdec) {
        launch_pack_frags(m->Ek1_w, 4 * d, d, s->packDdec, st);
        launch_pack_rd_head(m->mix_w, m->k2_w, m->cfg.n_mix, m->cfg.n_types, d,
                            s->packDdec + (size_t)4 * d * d * 2, st);
      }
    }
    s->packs_built = true;
  }
  launch_prefill_init(d_t, d_k, s->B, n0, n_gen, d_t_end, s->ev_t, s->ev_k, s->cap, s->n, s->gen, s->lenT, s->lenD,
                      s->done, s->rnd, s->zeros, s->t_end, s->ll, s->n_done, s->status, s->acc_stats, st);
  // encode history events 0 .. n0 - 2 (target) and 0 .. n0 - 3 (draft) in position chunks
  for (int which = 0; which < (s->D ? 2 : 1); ++which) {
    const tppsd_model *m = which ? s->D : s->T;
    const ModelCache &c = which ? s->cD : s->cT;
    const int n_enc = n0 - 1 - which;
    for (int c0 = 0; c0 < n_enc; c0 += PREFILL_CHUNK) {
      const int P = std::min(PREFILL_CHUNK, n_enc - c0);
      TokSrc src{};
      src.ev_t = s->ev_t;
      src.ev_k = s->ev_k;
      src.ev_stride = s->cap;
      src.start = s->zeros;
      src.start_off = c0;
      src.n_ev = P;
      forward(s, m, c, s->zeros, c0, P, src, nullptr, false, st);
    }
  }
  s->prefilled = true;
  s->draft_ok = s->D != nullptr;
  s->drafted_this_round = false;
  return hip_check("tppsd_prefill");
}

static int check_round(tppsd_state *s, int gamma) {
  if (!s) return fail(TPPSD_E_ARG, "null state");
  if (gamma < 1 || gamma > s->max_gamma) return fail(TPPSD_E_ARG, "gamma %d outside 1..%d", gamma, s->max_gamma);
  if (!s->prefilled) return fail(TPPSD_E_ORDER, "call tppsd_prefill first");
  return TPPSD_OK;
}

int tppsd_draft(tppsd_state *s, int gamma, const tppsd_draft_buf *out, hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (int rc = check_draft_buf(out)) return rc;
  if (out->rate) return fail(TPPSD_E_ARG, "tppsd_draft needs out->rate == NULL (it marks a Poisson draft)");
  if (!out->mix) return fail(TPPSD_E_ARG, "draft buffer has a null pointer");
  if (!s->D) return fail(TPPSD_E_ORDER, "state has no draft model");
  if (!s->draft_ok)
    return fail(TPPSD_E_ORDER, "draft cache is stale (AR sampling or an external draft ran since prefill)");
  int rc = do_draft(s, gamma, out, st);
  if (rc == TPPSD_OK) s->drafted_this_round = true;
  return rc;
}

int tppsd_draft_poisson(tppsd_state *s, int gamma, const float *d_params, const tppsd_draft_buf *out,
                        hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (int rc = check_draft_buf(out)) return rc;
  if (!out->rate || !d_params) return fail(TPPSD_E_ARG, "Poisson draft needs out->rate and d_params");
  return do_draft_poisson(s, gamma, d_params, out, st);
}

int tppsd_poisson_fit(const float *d_t, const int32_t *d_k, int B, int n0, int K, float *d_params, hipStream_t st) {
  if (!d_t || !d_k || !d_params) return fail(TPPSD_E_ARG, "null argument");
  if (B < 1 || n0 < 2) return fail(TPPSD_E_ARG, "need B >= 1 and n0 >= 2");
  if (K < 1 || K > TPPSD_MAX_TYPES) return fail(TPPSD_E_ARG, "K %d outside 1..%d", K, TPPSD_MAX_TYPES);
  if ((long long)B * n0 >= (1LL << 31)) return fail(TPPSD_E_ARG, "B * n0 too large");
  launch_poisson_fit(d_t, d_k, B, n0, K, d_params, st);
  return hip_check("tppsd_poisson_fit");
}

int tppsd_verify(tppsd_state *s, int gamma, const tppsd_draft_buf *in, const tppsd_verify_buf *out, hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (int rc = check_draft_buf(in)) return rc;
  if (int rc = check_verify_buf(out)) return rc;
  return do_verify(s, gamma, in, out, st);
}

int tppsd_verify_noalloc(tppsd_state *s, int gamma, const tppsd_draft_buf *in, const tppsd_verify_buf *out,
                         hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (int rc = check_draft_buf(in)) return rc;
  if (int rc = check_verify_buf(out)) return rc;
  const ScratchLayout L = scratch_layout(s->T, s->D, s->B, gamma + 1, s->kv_cap);
  if (L.total > NOALLOC_SCRATCH_BYTES)
    return fail(TPPSD_E_WORKSPACE, "tppsd_verify_noalloc needs %zu bytes of scratch for B = %d, gamma = %d; its "
                "static array holds %zu", L.total, s->B, gamma, NOALLOC_SCRATCH_BYTES);
  char *base = nullptr;
  if (int rc = scratch_base(&base)) return rc;
  // the pass's kernels take the scratch pointers from the state at launch:
  // point them at the static array for this call, then back at the workspace
  float *const x = s->x, *const logits = s->logits, *const part = s->attn_part;
  void *const a = s->a, *const q = s->q, *const o = s->o, *const hid = s->hid, *const e = s->e, *const u = s->u;
  s->x = (float *)(base + L.x);
  s->a = base + L.a;
  s->q = base + L.q;
  s->o = base + L.o;
  s->hid = base + L.hid;
  s->e = base + L.e;
  s->u = base + L.u;
  s->logits = (float *)(base + L.logits);
  s->attn_part = (float *)(base + L.attn_part);
  const int rc = do_verify(s, gamma, in, out, st);
  s->x = x;
  s->a = a;
  s->q = q;
  s->o = o;
  s->hid = hid;
  s->e = e;
  s->u = u;
  s->logits = logits;
  s->attn_part = part;
  return rc;
}

int tppsd_accept(tppsd_state *s, int gamma, const tppsd_draft_buf *dr, const tppsd_verify_buf *vf,
                 const float *d_uniforms, const tppsd_accept_buf *out, hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (int rc = check_draft_buf(dr)) return rc;
  if (int rc = check_verify_buf(vf)) return rc;
  if (int rc = check_accept_buf(out)) return rc;
  int rc = do_accept(s, gamma, dr, vf, d_uniforms, out, st);
  if (!s->drafted_this_round) s->draft_ok = false;   // the draft cache missed this round's events
  s->drafted_this_round = false;
  return rc;
}

namespace {

// one AR step (§4.2 naive sampling): target pass over the pending event, then a draw
int ar_step(tppsd_state *s, int out_stride, float *d_t_out, int32_t *d_k_out, hipStream_t st) {
  TokSrc src{};
  src.ev_t = s->ev_t;
  src.ev_k = s->ev_k;
  src.ev_stride = s->cap;
  src.start = s->lenT;
  src.start_off = 0;
  src.n_ev = 1;
  HeadArgs h = head_common(s);
  h.mode = HEAD_AR;
  h.P = 1;
  h.p0 = 0;
  h.mix = s->ar_mix;
  h.logtype = s->ar_logtype;
  h.dst_stride = 1;
  h.dst_row0 = 0;
  h.ar_t_out = d_t_out;
  h.ar_k_out = d_k_out;
  h.ar_out_stride = out_stride;
  h.gen0 = s->gen0;
  return forward(s, s->T, s->cT, s->lenT, 0, 1, src, &h, false, st);
}

// Captures body() into an executable graph (on the private capture stream).
int capture(tppsd_state *s, const std::function<int(hipStream_t)> &body, hipGraphExec_t *out) {
  hipGraph_t g = nullptr;
  if (hipStreamBeginCapture(s->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
    return hip_check("graph capture begin");
  const int rc = body(s->cap_stream);
  const hipError_t e = hipStreamEndCapture(s->cap_stream, &g);
  if (rc != TPPSD_OK || e != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    return rc != TPPSD_OK ? rc : fail(TPPSD_E_HIP, "graph capture: %s", hipGetErrorString(e));
  }
  const hipError_t e2 = hipGraphInstantiate(out, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e2 != hipSuccess) return fail(TPPSD_E_HIP, "graph instantiate: %s", hipGetErrorString(e2));
  return TPPSD_OK;
}

}  // namespace

int tppsd_sample_ar(tppsd_state *s, int n_events, float *d_t_out, int32_t *d_k_out, hipStream_t st) {
  if (!s) return fail(TPPSD_E_ARG, "null state");
  if (!s->prefilled) return fail(TPPSD_E_ORDER, "call tppsd_prefill first");
  if (n_events < 0) return fail(TPPSD_E_ARG, "n_events < 0");
  if (n_events == 0) return TPPSD_OK;
  launch_snapshot(s->gen, s->gen0, s->B, st);   // output column = events generated in this call
  int i = 0;
  if (s->timing & TPPSD_TIME_KERNELS) {
    // kernel-timing runs launch each step directly (no graphs), so that
    // per-dispatch tools see the AR step's kernels one by one
    for (; i < n_events; ++i)
      if (int rc = ar_step(s, n_events, d_t_out, d_k_out, st)) return rc;
    s->draft_ok = false;
    return hip_check("tppsd_sample_ar");
  }
  {
    // graphs embed the output pointers, their stride and n_gen
    const long long key = ((long long)(uintptr_t)d_t_out * 31 + (long long)(uintptr_t)d_k_out) * 131 +
                          (long long)n_events * 1000003LL + s->n_gen;
    for (int w = 0; w < 2; ++w) {
      if (s->ar_exec[w] && s->ar_key[w] == key) continue;
      drop_graph(&s->ar_exec[w]);
      const int steps = w ? AR_CHUNK : 1;
      int rc = capture(s, [&](hipStream_t cs) {
        for (int k = 0; k < steps; ++k)
          if (int r = ar_step(s, n_events, d_t_out, d_k_out, cs)) return r;
        return hip_check("tppsd_sample_ar capture");
      }, &s->ar_exec[w]);
      if (rc) return rc;
      s->ar_key[w] = key;
    }
    for (; i + AR_CHUNK <= n_events; i += AR_CHUNK)
      if (hipGraphLaunch(s->ar_exec[1], st) != hipSuccess) return hip_check("tppsd_sample_ar: graph launch");
    for (; i < n_events; ++i)
      if (hipGraphLaunch(s->ar_exec[0], st) != hipSuccess) return hip_check("tppsd_sample_ar: graph launch");
  }
  s->draft_ok = false;
  return hip_check("tppsd_sample_ar");
}

namespace {
// adds the times recorded in event set w during its round (read one round behind)
void read_round_events(tppsd_state *s, int w) {
  const int L = s->T->cfg.n_layers;
  if (s->timing & TPPSD_TIME_KERNELS) {
    for (size_t i = 0; i + 1 < s->gev[w].size(); i += 2) {
      // pairs the pass does not use (AttNHP layers and k_block passes launch fewer kernels)
      const int pair = (int)(i / 2);
      if (pair >= (int)s->ev_used.size() || !s->ev_used[pair]) continue;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, s->gev[w][i], s->gev[w][i + 1]) != hipSuccess) {
        (void)hipGetLastError();   // a failed query must not reach the next launch check
        continue;
      }
      if (pair < L) {
        s->tm.attn_ms += ms;
        s->tm.attn_launches += 1;
      } else if (pair == 5 * L + 1) {
        s->tm.draft_kernel_ms += ms;
        s->tm.draft_kernel_launches += 1;
      } else if (pair >= 5 * L + 2) {
        // row drafting: launch 0 and every second one after it are row launches
        const int j = pair - (5 * L + 2);
        if (j > 0 && (j - 1) % 2 == 0) {
          s->tm.draft_attn_ms += ms;
          s->tm.draft_attn_launches += 1;
        } else {
          s->tm.draft_rows_ms += ms;
          s->tm.draft_rows_launches += 1;
        }
      } else {
        s->tm.gemm_ms += ms;
        s->tm.gemm_launches += 1;
      }
    }
    s->tm.gemm_flop += s->round_flop;
  }
  if (s->timing & TPPSD_TIME_PHASES) {
    float ms[3] = {0.f, 0.f, 0.f};
    for (int j = 0; j < 3; ++j)
      if (hipEventElapsedTime(&ms[j], s->pev[w][j], s->pev[w][j + 1]) != hipSuccess) {
        ms[j] = 0.f;
        (void)hipGetLastError();
      }
    s->tm.draft_ms += ms[0];
    s->tm.verify_ms += ms[1];
    s->tm.accept_ms += ms[2];
  }
  s->tm.rounds += 1;
}

int make_events(std::vector<hipEvent_t> *v, size_t n) {
  for (int w = 0; w < 2; ++w)
    if (v[w].size() != n) {
      for (hipEvent_t e : v[w]) (void)hipEventDestroy(e);
      v[w].assign(n, nullptr);
      for (hipEvent_t &e : v[w])
        if (hipEventCreate(&e) != hipSuccess) return hip_check("tppsd_sample_sd: timing events");
    }
  return TPPSD_OK;
}
}  // namespace

namespace {
// Rounds of draft, verify and accept on the internal buffers; params == NULL
// drafts from the draft model, otherwise from the Poisson draft of params.
int sd_loop(tppsd_state *s, int gamma, const float *params, int max_rounds, int *rounds, hipStream_t st) {
  const tppsd_draft_buf *dbuf = params ? &s->idr_p : &s->idr;
  auto draft = [&](hipStream_t cs) {
    return params ? do_draft_poisson(s, gamma, params, dbuf, cs) : do_draft(s, gamma, dbuf, cs);
  };
  // kernel timing launches the rounds directly so that host-recorded HIP
  // events can bracket single kernels; otherwise each round replays one
  // captured graph, or three (draft, verify, accept) when phases are timed
  const bool kern = (s->timing & TPPSD_TIME_KERNELS) != 0;
  const bool phases = (s->timing & TPPSD_TIME_PHASES) != 0;
  const bool graphs = !kern;
  const long long key = (long long)gamma * 100000007LL + s->n_gen;
  if (graphs && !phases && (!s->sd_exec[0] || s->sd_key != key || s->sd_params != params)) {
    drop_graph(&s->sd_exec[0]);
    s->sd_key = -1;
    int rc = capture(s, [&](hipStream_t cs) {
      int r = draft(cs);
      if (!r) r = do_verify(s, gamma, dbuf, &s->ivf, cs);
      if (!r) r = do_accept(s, gamma, dbuf, &s->ivf, nullptr, &s->iac, cs);
      return r;
    }, &s->sd_exec[0]);
    if (rc) return rc;
    s->sd_key = key;
    s->sd_params = params;
  }
  if (graphs && phases && (!s->phase_exec[0] || s->phase_key != key || s->phase_params != params)) {
    for (hipGraphExec_t &g : s->phase_exec) drop_graph(&g);
    s->phase_key = -1;
    int rc = capture(s, draft, &s->phase_exec[0]);
    if (!rc)
      rc = capture(s, [&](hipStream_t cs) { return do_verify(s, gamma, dbuf, &s->ivf, cs); }, &s->phase_exec[1]);
    if (!rc)
      rc = capture(s, [&](hipStream_t cs) { return do_accept(s, gamma, dbuf, &s->ivf, nullptr, &s->iac, cs); },
                   &s->phase_exec[2]);
    if (rc) return rc;
    s->phase_key = key;
    s->phase_params = params;
  }
  if (kern) {
    const tppsd_model *m = s->T;
    const int L = m->cfg.n_layers;
    const double d = m->d(), F = m->cfg.d_ffn, rows = (double)s->B * (gamma + 1);
    s->round_flop = m->attnhp() ? 2.0 * rows * (L * (3 * d * 2 * d) + 4 * d * d)
                                : 2.0 * rows * (L * (3 * d * d + d * d + 2 * d * F) + 4 * d * d);
    // pairs: attention of each layer, the pass's GEMMs, the one-launch draft,
    // then one per launch of row drafting
    const int nrd = (s->row_draft && !params) ? rd_launches(s->D->cfg.n_layers, gamma) : 0;
    if (int rc = make_events(s->gev, 2 * (5 * L + 2 + nrd))) return rc;
    s->ev_used.assign(5 * L + 2 + nrd, 0);
  }
  if (phases)
    if (int rc = make_events(s->pev, 4)) return rc;
  int r = 0;
  for (; r < max_rounds; ++r) {
    if (r >= 1) {
      // the done counter copied after round r - 1; waits for that round only
      if (hipEventSynchronize(s->poll_ev[(r - 1) & 1]) != hipSuccess) return hip_check("tppsd_sample_sd: poll");
      if (s->timing) read_round_events(s, (r - 1) & 1);
      if (s->host_ndone[(r - 1) & 1] >= s->B) break;
    }
    if (graphs && phases) {
      hipEvent_t *pe = s->pev[r & 1].data();
      for (int j = 0; j < 3; ++j)
        if (hipEventRecord(pe[j], st) != hipSuccess || hipGraphLaunch(s->phase_exec[j], st) != hipSuccess)
          return hip_check("tppsd_sample_sd: phase graph launch");
      if (hipEventRecord(pe[3], st) != hipSuccess) return hip_check("tppsd_sample_sd: phase event");
    } else if (graphs) {
      if (hipGraphLaunch(s->sd_exec[0], st) != hipSuccess) return hip_check("tppsd_sample_sd: graph launch");
    } else {
      hipEvent_t *pe = phases ? s->pev[r & 1].data() : nullptr;
      s->cur_ev = kern ? s->gev[r & 1].data() : nullptr;
      int rc = pe ? hip_check_rc(hipEventRecord(pe[0], st)) : 0;
      if (!rc) rc = draft(st);
      if (!rc && pe) rc = hip_check_rc(hipEventRecord(pe[1], st));
      if (!rc) rc = do_verify(s, gamma, dbuf, &s->ivf, st);
      if (!rc && pe) rc = hip_check_rc(hipEventRecord(pe[2], st));
      if (!rc) rc = do_accept(s, gamma, dbuf, &s->ivf, nullptr, &s->iac, st);
      if (!rc && pe) rc = hip_check_rc(hipEventRecord(pe[3], st));
      s->cur_ev = nullptr;
      if (rc) return rc;
    }
    if (hipMemcpyAsync(&s->host_ndone[r & 1], s->n_done, sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipEventRecord(s->poll_ev[r & 1], st) != hipSuccess)
      return hip_check("tppsd_sample_sd: poll");
  }
  if (s->timing && r == max_rounds && r >= 1) {
    if (hipEventSynchronize(s->poll_ev[(r - 1) & 1]) != hipSuccess) return hip_check("tppsd_sample_sd: poll");
    read_round_events(s, (r - 1) & 1);
  }
  if (rounds) *rounds = r;
  return hip_check("tppsd_sample_sd");
}
}  // namespace

int tppsd_sample_sd(tppsd_state *s, int gamma, int max_rounds, int *rounds, hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (!s->D) return fail(TPPSD_E_ORDER, "state has no draft model");
  if (!s->draft_ok) return fail(TPPSD_E_ORDER, "draft cache is stale; prefill again");
  return sd_loop(s, gamma, nullptr, max_rounds, rounds, st);
}

int tppsd_sample_sd_poisson(tppsd_state *s, int gamma, const float *d_params, int max_rounds, int *rounds,
                            hipStream_t st) {
  if (int rc = check_round(s, gamma)) return rc;
  if (!d_params) return fail(TPPSD_E_ARG, "null d_params");
  int r = 0;
  const int rc = sd_loop(s, gamma, d_params, max_rounds, &r, st);
  if (r > 0 || rc != TPPSD_OK) s->draft_ok = false;   // the draft model's cache missed these rounds
  if (rounds) *rounds = r;
  return rc;
}

int tppsd_read_events(tppsd_state *s, float *d_t, int32_t *d_k, int32_t *d_n, hipStream_t st) {
  if (!s) return fail(TPPSD_E_ARG, "null state");
  launch_copy_events(s->ev_t, s->ev_k, s->n, s->B, s->cap, d_t, d_k, d_n, st);
  return hip_check("tppsd_read_events");
}

int tppsd_read_loglik(tppsd_state *s, double *d_ll, hipStream_t st) {
  if (!s || !d_ll) return fail(TPPSD_E_ARG, "null argument");
  if (hipMemcpyAsync(d_ll, s->ll, (size_t)s->B * sizeof(double), hipMemcpyDeviceToDevice, st) != hipSuccess)
    return hip_check("tppsd_read_loglik");
  return TPPSD_OK;
}

int tppsd_state_status(tppsd_state *s, hipStream_t st, uint32_t *bits, int32_t *n_done, int64_t *accepted,
                       int64_t *drafted, int64_t *ar_candidates) {
  if (!s) return fail(TPPSD_E_ARG, "null state");
  uint32_t b = 0;
  int32_t nd = 0;
  // the counters are per sequence (each owned by one wave of the accept
  // kernel, so no atomics on shared addresses); summed here
  std::vector<unsigned long long> per((size_t)s->B * 3);
  if (hipMemcpyAsync(&b, s->status, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(&nd, s->n_done, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(per.data(), s->acc_stats, per.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost,
                     st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return hip_check("tppsd_state_status");
  unsigned long long acc[3] = {0, 0, 0};
  for (size_t i = 0; i < per.size(); ++i) acc[i % 3] += per[i];
  if (bits) *bits = b;
  if (n_done) *n_done = nd;
  if (accepted) *accepted = (int64_t)acc[0];
  if (drafted) *drafted = (int64_t)acc[1];
  if (ar_candidates) *ar_candidates = (int64_t)acc[2];
  return TPPSD_OK;
}

int tppsd_timing_enable(tppsd_state *s, int modes) {
  if (!s) return fail(TPPSD_E_ARG, "null state");
  if (modes & ~(TPPSD_TIME_KERNELS | TPPSD_TIME_PHASES))
    return fail(TPPSD_E_ARG, "unknown timing mode bits");
  if ((modes & TPPSD_TIME_KERNELS) && (modes & TPPSD_TIME_PHASES))
    return fail(TPPSD_E_ARG, "kernel and phase timing are separate runs");
  s->timing = modes;
  s->tm = tppsd_timing{};
  return TPPSD_OK;
}

int tppsd_timing_read(tppsd_state *s, tppsd_timing *out) {
  if (!s || !out) return fail(TPPSD_E_ARG, "null argument");
  *out = s->tm;
  return TPPSD_OK;
}

}  // extern "C"
