// Drafting for small batches over long contexts (§4.3 "Drafting", the inner
// loop of Algorithm 1), bf16 draft models.
//
// Each draft step runs two launches per layer:
//  - k_rd_attn: the step's queries (two in the first step, which re-encodes
//    the last two committed events, one after), formed in the launch from the
//    step's residual rows (the launch applies the layer's LayerNorm), against
//    the draft KV cache, split over (key
//    range, head, sequence) workgroups so that the cache streams through the
//    whole chip; the split holding the step's new position also forms and
//    appends its key and value; each split leaves its running maximum, sum
//    and unnormalised output;
//  - k_rd_rows: merges the splits and runs every row-local step up to the
//    next attention -- output projection and residual, the feed-forward
//    block; for a non-last layer four workgroups per sequence, each taking a
//    quarter of the FFN's hidden units (the next layer's launches add their
//    outputs to the rows); for the last layer one workgroup per sequence,
//    which also runs the decoder, the draft record, the draw, and the drawn
//    event's embedding (the next step's residual row).
// The matrix-vector products of a sequence's one or two rows run on MFMA
// 16-row tiles (rows past the token count are zero operands) with every weight
// fragment of a product in flight at once, and the next product's fragments
// loaded before the current one is multiplied out, so that a product costs
// about one memory latency. Rounding points are those of the layered kernels:
// LayerNorm outputs, q/k/v, the attention output, ReLU output and the
// decoder's e and tanh activations are bf16; the residual stream, softmax and
// decoder math are fp32.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tppsd_device.h"
#include "tppsd_philox.h"
#include "../../include/tppsd.h"

namespace tppsd {

namespace {

constexpr int RD_WAVES = RD_ROW_THREADS / 64;
constexpr int RD_VEC = 2048;   // floats of a row launch's staged vectors (RdVec)

// a load the compiler may issue as a scalar one wherever it can prove the
// address uniform: the word does not change while the kernel runs (the
// sequence's header words and draw numbers are written by other launches
// only)
template <class T>
__device__ __forceinline__ T load_const(const T *p) {
  return *(const __attribute__((address_space(4))) T *)p;
}

// ---------------------------------------------------------------------------
// split attention: workgroup (s, h, b) takes keys [s RD_KEYS, (s + 1) RD_KEYS)
// of head h of sequence b
// ---------------------------------------------------------------------------
template <int D, int DH>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void k_rd_attn(const int32_t *done_p,
                                                                                          const int32_t *len_p,
                                                                                          int step, int layer,
                                                                                          RowDraftArgs a) {
  constexpr int NG = 256 / DH;              // lane groups over the value blocks
  constexpr int BPL = RD_KEYS / 8 / NG;     // value blocks per lane
  static_assert(DH == 32 && D % 128 == 0, "q, k, v: 32 groups of 8 lanes, 16 elements per lane and pass of 128");
  __shared__ __attribute__((aligned(16))) float es[2][RD_KEYS];
  __shared__ float red[2][NG][DH];
  __shared__ float wred[2][4][2];
  __shared__ __attribute__((aligned(16))) bf16_t xl[2][D];        // LayerNorm'd rows of the step's tokens
  __shared__ float bs[3][DH];                                       // the head's q, k, v biases
  __shared__ float lnred[4][2];                                     // per wave: LayerNorm partial sums
  __shared__ float lngb[2 * D];                                     // LayerNorm gain, then bias
  __shared__ float qs[2][DH];                                       // queries (bf16-rounded)
  __shared__ __attribute__((aligned(16))) bf16_t kvn[2][2][DH];   // the new keys and values [k / v][row]
  const DraftArgs &d = a.d;
  const int s = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  constexpr int SEG = DH * 2 / 16;          // 16-byte segments of a key row
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, seg = tid % SEG;
  // q, k, v of the step's rows: group r = tid / 8 of eight lanes takes output
  // row r of the head, lane j = tid % 8 elements 16 j .. + 15 of every 128
  constexpr int NC = D / 128;               // 128-element chunks per row
  const int r = tid >> 3, j8 = tid & 7;
  // The leading arguments (the header words' arrays, step and layer) arrive
  // preloaded in registers; every other scalar the split needs (kernel
  // arguments, the layer's weight pointers, the sequence's header words) is
  // loaded up front in one batch and waited for once. (Left to itself the
  // compiler sinks each load to the branch that first needs it and pays a
  // round trip per branch.) The asm statement only takes values, which holds
  // each load ahead of it.
  const int cap = d.cap, nh = d.H;
  const char *kcb = d.kc, *vcb = d.vc;
  const size_t lbytes = d.layer_bytes;
  const FusedLayerW &lw = d.layer[layer];
  const bf16_t *wqkv = (const bf16_t *)lw.qkv_w;
  const float *qkvb = lw.qkv_b;
  const float *xres = a.x, *fpart = a.fpart, *l1g = lw.ln1_g, *l1b = lw.ln1_b;
  const int done = load_const(done_p + b), lenD = load_const(len_p + b);
  asm volatile("" ::"s"(cap), "s"(nh), "s"(kcb), "s"(vcb), "s"(lbytes), "s"(wqkv), "s"(qkvb), "s"(done),
               "s"(lenD), "s"(xres), "s"(fpart), "s"(l1g), "s"(l1b));
  auto wrow = [&](int which) { return wqkv + (size_t)(which * D + h * DH + r) * D + 16 * j8; };
  // the LayerNorm'd rows and this head's query rows of W_qkv
  const int P = step == 1 ? 2 : 1;
  // The launch applies the layer's LayerNorm itself to the residual rows
  // (stored by the launch before), thread t taking column t mod D of row
  // t / D; after a layer whose FFN ran in RD_FSPLIT slices (every layer but
  // the first) it first adds the slices' outputs. Every load is issued
  // unconditionally (layer 0 reads slices it then ignores) so that no branch
  // separates a load from its use; the gain (t < D) or bias (t >= D) of
  // column t mod D is staged in LDS.
  static_assert(2 * D == 256, "one column of the two rows per thread");
  const bool comb = layer > 0;
  float cx[1 + RD_FSPLIT], cgb;
  {
    const int rw = tid / D, cc = tid % D;
    cx[0] = xres[((size_t)b * 2 + rw) * D + cc];
#pragma unroll
    for (int j = 0; j < RD_FSPLIT; ++j) cx[1 + j] = fpart[(((size_t)b * RD_FSPLIT + j) * 2 + rw) * D + cc];
    cgb = rw ? l1b[cc] : l1g[cc];
  }
  // the head's biases, one per lane (staged in LDS with the rows)
  const int bi = min(tid, 3 * DH - 1);
  const float bias = qkvb[(bi / DH) * D + h * DH + bi % DH];
  uint4 wq[NC][2];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    wq[c][0] = *(const uint4 *)(wrow(0) + 128 * c);
    wq[c][1] = *(const uint4 *)(wrow(0) + 128 * c + 8);
  }
  const int pos0 = lenD + (step == 1 ? 0 : step);
  const int n_keys = min(pos0 + P, cap);
  const int k0 = s * RD_KEYS;
  if (done || k0 >= n_keys) return;   // whole workgroup; no barrier passed yet
  const size_t row0 = ((size_t)b * nh + h) * cap;
  bf16_t *kc = (bf16_t *)(kcb + lbytes * layer);
  bf16_t *vc = (bf16_t *)(vcb + lbytes * layer);
  // the step's new positions pos0 .. pos0 + P - 1 whose key and value this
  // split owns (it computes and appends them; they are in no other split)
  auto owned = [&](int p) { const int pn = pos0 + p; return p < P && pn >= k0 && pn < k0 + RD_KEYS && pn < cap; };
  const bool any_owned = owned(0) || owned(1);
  uint4 wk[NC][2], wv[NC][2];
  if (any_owned) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      wk[c][0] = *(const uint4 *)(wrow(1) + 128 * c);
      wk[c][1] = *(const uint4 *)(wrow(1) + 128 * c + 8);
      wv[c][0] = *(const uint4 *)(wrow(2) + 128 * c);
      wv[c][1] = *(const uint4 *)(wrow(2) + 128 * c + 8);
    }
  }
  // every load of the split in flight at once, each wave instruction reading
  // 1 KB of contiguous memory (non-temporal: the cache streams through once per
  // step and should not push the draft model's weights out of L2). Keys: lane
  // t of load i holds 16-byte segment t % SEG of key i KPI + t / SEG. Values:
  // lane (grp, col) holds the 8-position blocks of column col. The slots of
  // the step's new positions are replaced below. Slots past the key range
  // read the range's last key or value block (unconditional loads: a load
  // under a lane condition makes the compiler wait for every load before it),
  // and never count: their scores are masked, their blocks skipped.
  constexpr int KPI = 256 / SEG;            // keys per load
  constexpr int NKL = RD_KEYS / KPI;        // key loads per lane
  u32x4_t kr[NKL];
#pragma unroll
  for (int i = 0; i < NKL; ++i) {
    const int pos = min(k0 + i * KPI + tid / SEG, n_keys - 1);
    kr[i] = __builtin_nontemporal_load((const u32x4_t *)(kc + (row0 + pos) * DH) + seg);
  }
  const int col = tid % DH, grp = tid / DH;
  u32x4_t vr[BPL];
#pragma unroll
  for (int i = 0; i < BPL; ++i) {
    const int pb = min(k0 + 8 * (grp + i * NG), (n_keys - 1) & ~7);   // first position of the block
    vr[i] = __builtin_nontemporal_load((const u32x4_t *)(vc + v_at<bf16_t>(row0, pb, col, DH)));
  }
  // (keeps the rows' sums below the cache loads: formed ahead of them they
  // would wait for the rows' loads before the cache loads go out)
  __builtin_amdgcn_sched_barrier(0);
  {
    // LayerNorm (biased variance, eps 1e-5) of each row over its two waves
    const int rw = tid / D, cc = tid % D;
    float xs = cx[0];
#pragma unroll
    for (int j = 0; j < RD_FSPLIT; ++j) xs += cx[1 + j];
    const float x = comb ? xs : cx[0];   // (a select: stale slices never enter layer 0's rows)
    const float s1 = wave_sum(x);
    if (lane == 0) lnred[wave][0] = s1;
    lngb[tid] = cgb;
    __syncthreads();
    const float mean = (lnred[2 * rw][0] + lnred[2 * rw + 1][0]) / (float)D;
    const float dx = x - mean;
    const float s2 = wave_sum(dx * dx);
    if (lane == 0) lnred[wave][1] = s2;
    __syncthreads();
    const float rstd = 1.f / sqrtf((lnred[2 * rw][1] + lnred[2 * rw + 1][1]) / (float)D + 1e-5f);
    xl[rw][cc] = f2bf(dx * rstd * lngb[cc] + lngb[D + cc]);
  }
  if (tid < 3 * DH) (&bs[0][0])[tid] = bias;
  __syncthreads();
  // dot products of a weight row slice with a row's slice: v_dot2c over
  // the raw bf16 pairs (products exact in fp32)
  auto dot16 = [&](const uint4 (&w)[NC][2], int p) {
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int hlf = 0; hlf < 2; ++hlf) {
        const uint4 xx = *(const uint4 *)(&xl[p][0] + 128 * c + 16 * j8 + 8 * hlf);
        acc = dot2_bf(w[c][hlf].x, xx.x, acc);
        acc = dot2_bf(w[c][hlf].y, xx.y, acc);
        acc = dot2_bf(w[c][hlf].z, xx.z, acc);
        acc = dot2_bf(w[c][hlf].w, xx.w, acc);
      }
    return group_sum(acc, 8);
  };
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (p >= P) break;
    const float qa = dot16(wq, p);
    if (j8 == 0) qs[p][r] = bf2f(f2bf(qa + bs[0][r]));
    if (owned(p)) {   // workgroup-uniform
      const float ka = dot16(wk, p), va = dot16(wv, p);
      if (j8 == 0) {
        const bf16_t kb = f2bf(ka + bs[1][r]), vb = f2bf(va + bs[2][r]);
        kvn[0][p][r] = kb;
        kvn[1][p][r] = vb;
        const int pn = pos0 + p;
        kc[(row0 + pn) * DH + r] = kb;
        vc[v_at<bf16_t>(row0, pn, r, DH)] = vb;
      }
    }
  }
  __syncthreads();
  // the lane's 8 query elements (bf16 values) as pairs for v_dot2c
  uint32_t q[2][4];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int e = 0; e < 4; ++e) q[p][e] = pk2bf(qs[p][8 * seg + 2 * e], qs[p][8 * seg + 2 * e + 1]);
  // the owned new positions' keys and values replace what the loads read
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (!owned(p)) continue;
    const int pn = pos0 + p;
#pragma unroll
    for (int i = 0; i < NKL; ++i)
      if (k0 + i * KPI + tid / SEG == pn) kr[i] = *(const u32x4_t *)(&kvn[0][p][0] + 8 * seg);
    const uint32_t vb = kvn[1][p][col];
#pragma unroll
    for (int i = 0; i < BPL; ++i) {
      const int pb = k0 + 8 * (grp + i * NG);
      if (pn >= pb && pn < pb + 8) {
        const int e = pn - pb, wi = e >> 1;
        const uint32_t old = vr[i][wi];
        vr[i][wi] = (e & 1) ? ((old & 0x0000FFFFu) | (vb << 16)) : ((old & 0xFFFF0000u) | vb);
      }
    }
  }
  // scores, per query: q k / sqrt(d_head) (the SEG lanes of a key sum their
  // segments); keys past the query masked
  static_assert(SEG == 4 || SEG == 2, "key segments per quad");
  // scores in base-2 units (log2 e folded into 1 / sqrt(d_head)), so that
  // every exponential is one v_exp_f32; maxima leave in natural units
  const float scale2 = 1.4426950408889634f / sqrtf((float)DH);
  float sc[2][NKL];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (p >= P) break;
    const int last = pos0 + p;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NKL; ++i) {
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) dot = dot2_bf(kr[i][e], q[p][e], dot);
      dot += dpp_mov<0xB1>(dot);                 // lane ^ 1
      if (SEG == 4) dot += dpp_mov<0x4E>(dot);   // lane ^ 2
      const int pos = k0 + i * KPI + tid / SEG;
      sc[p][i] = (pos < n_keys && pos <= last) ? dot * scale2 : -INFINITY;
      mx = fmaxf(mx, sc[p][i]);
    }
    mx = wave_max(mx);
    if (lane == 0) wred[p][wave][0] = mx;
  }
  __syncthreads();
  float mq[2] = {-INFINITY, -INFINITY};
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (p >= P) break;
    mq[p] = fmaxf(fmaxf(wred[p][0][0], wred[p][1][0]), fmaxf(wred[p][2][0], wred[p][3][0]));
    float ls = 0.f;
#pragma unroll
    for (int i = 0; i < NKL; ++i) {
      const float e = sc[p][i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[p][i] - mq[p]);
      if (seg == 0) {
        es[p][i * KPI + tid / SEG] = e;
        ls += e;
      }
    }
    ls = wave_sum(ls);
    if (lane == 0) wred[p][wave][1] = ls;
  }
  __syncthreads();
  // output sums: lane (grp, col) over its value blocks; slots that are not
  // keys of the query carry weight 0 and possibly unwritten values, so they
  // are skipped rather than multiplied
  const int clean_end = min(n_keys, pos0 + 1);   // positions below are keys of every query
  float o[2] = {0.f, 0.f};
#pragma unroll
  for (int i = 0; i < BPL; ++i) {
    const int lb = 8 * (grp + i * NG), pb = k0 + lb;
    if (pb >= n_keys) continue;
    const uint32_t w[4] = {vr[i][0], vr[i][1], vr[i][2], vr[i][3]};
    float v[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(w[e] << 16);
      v[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
    const bool clean = pb + 8 <= clean_end;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      if (p >= P) break;
      const float4 e0 = *(const float4 *)&es[p][lb], e1 = *(const float4 *)&es[p][lb + 4];
      const float ee[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
      float acc = 0.f;
      if (clean) {
#pragma unroll
        for (int t = 0; t < 8; ++t) acc += ee[t] * v[t];
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) acc += ee[t] != 0.f ? ee[t] * v[t] : 0.f;
      }
      o[p] += acc;
    }
  }
  red[0][grp][col] = o[0];
  if (P > 1) red[1][grp][col] = o[1];
  __syncthreads();
  if (tid < P * DH) {
    const int p = tid / DH, c = tid - p * DH;
    float acc = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) acc += red[p][g][c];
    float *dst = a.part + ((((size_t)b * nh + h) * a.S + s) * 2 + p) * (DH + 2);
    dst[2 + c] = acc;
    if (c == 0) {
      dst[0] = (p ? mq[1] : mq[0]) * 0.69314718055994531f;   // natural units
      dst[1] = (wred[p][0][1] + wred[p][1][1]) + (wred[p][2][1] + wred[p][3][1]);
    }
  }
}

// ---------------------------------------------------------------------------
// row kernel
// ---------------------------------------------------------------------------

// a layer's matrices in fragment order: Wo, W1, W2, Wqkv (elements)
template <int D, int F> constexpr size_t rd_layer_elems() { return (size_t)4 * D * D + 2 * (size_t)D * F; }
template <int D, int F> constexpr size_t rd_off_qkv() { return (size_t)D * D + 2 * (size_t)D * F; }

// the decoder heads' rows -- mixture rows (w, mu, log sigma; 3 M) then type
// rows (K), zero up to 128 -- in fragment order (K = D)
__global__ void k_pack_rd_head(const bf16_t *__restrict__ mix_w, const bf16_t *__restrict__ k2_w, int M, int K,
                               int D, bf16_t *__restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;   // one 16-byte vector per thread
  const int KS = D / 32, total = 8 * KS * 64;
  if (i >= total) return;
  const int l = i & 63, f = i >> 6, nt = f / KS, ks = f - nt * KS;
  const int n = 16 * nt + (l & 15), k = 32 * ks + 8 * (l >> 4);
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (n < 3 * M) v = *(const uint4 *)(mix_w + (size_t)n * D + k);
  else if (n < 3 * M + K) v = *(const uint4 *)(k2_w + (size_t)(n - 3 * M) * D + k);
  *(uint4 *)(out + (size_t)i * 8) = v;
}

// One wave's weight fragments of Y = X W^T for W [N][KD] bf16: its 16-column
// tiles wave, wave + RD_WAVES, ... and every 32-wide k step of each (lane l:
// column l % 16 of the tile, k = 8 (l / 16) .. + 7 of the step).
template <int N, int KD> struct RdFrags {
  static constexpr int KS = KD / 32, TILES = (N + 15) / 16, TPW = (TILES + RD_WAVES - 1) / RD_WAVES;
  bf16x8_t f[TPW][KS];
  // W in fragment order (fragment (tile, ks) is 64 lanes x 8 elements at
  // (tile KS + ks) 512): one contiguous kilobyte per wave instruction
  // (tiles past the matrix read its last tile, unused by mul: a load under a
  // condition the compiler cannot prove wave-uniform would make it wait for
  // every load issued before)
  __device__ __forceinline__ void load_packed(const bf16_t *Wp) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = min(wave + t * RD_WAVES, TILES - 1);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        f[t][ks] = *(const bf16x8_t *)(Wp + ((size_t)(tile * KS + ks) * 64 + lane) * 8);
    }
  }
  // the same for the k steps ks0 .. ks0 + KS - 1 of a packed matrix of
  // ks_all k steps per tile (a slice of its inner dimension)
  __device__ __forceinline__ void load_packed_k(const bf16_t *Wp, int ks_all, int ks0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = min(wave + t * RD_WAVES, TILES - 1);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        f[t][ks] = *(const bf16x8_t *)(Wp + ((size_t)(tile * ks_all + ks0 + ks) * 64 + lane) * 8);
    }
  }
  // rows 0 .. NR - 1 of X (bf16 in LDS, row stride ldx elements; rows
  // r < nx read, the others zero); epi(r, n, acc) for r < NR on lanes 0..15
  template <int NR, typename EPI>
  __device__ __forceinline__ void mul(const bf16_t *X, int ldx, int nx, EPI epi) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15;
    auto xfrag = [&](int ks) {
      return r < nx ? *(const bf16x8_t *)(X + r * ldx + ks * 32 + 8 * (lane >> 4))
                    : __builtin_bit_cast(bf16x8_t, make_uint4(0u, 0u, 0u, 0u));
    };
    if constexpr (TPW == 1) {
      // one tile: each A fragment is used once, read as it is needed
      const int tile = wave;
      if (tile >= TILES) return;   // wave-uniform
      f32x4_t c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ks += 2) {
        c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xfrag(ks), f[0][ks], c0, 0, 0, 0);
        if (ks + 1 < KS) c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xfrag(ks + 1), f[0][ks + 1], c1, 0, 0, 0);
      }
      const int n = tile * 16 + r;
      if (lane < 16 && n < N) {
#pragma unroll
        for (int v = 0; v < NR; ++v) epi(v, n, c0[v] + c1[v]);
      }
      return;
    }
    bf16x8_t xa[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xa[ks] = xfrag(ks);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int tile = wave + t * RD_WAVES;
      if (tile >= TILES) continue;   // wave-uniform
      f32x4_t c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ks += 2) {
        c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[ks], f[t][ks], c0, 0, 0, 0);
        if (ks + 1 < KS) c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[ks + 1], f[t][ks + 1], c1, 0, 0, 0);
      }
      const int n = tile * 16 + r;
      if (lane < 16 && n < N) {
#pragma unroll
        for (int v = 0; v < NR; ++v) epi(v, n, c0[v] + c1[v]);
      }
    }
  }
};

__device__ __forceinline__ void rd_sync() { __syncthreads(); }


// LayerNorm (biased variance, eps 1e-5) of rows 0 .. np - 1 of xs [2][D]
// into bf16 rows of y (stride D); wave p takes row p
template <int D>
__device__ __forceinline__ void rd_layernorm(const float *xs, bf16_t *y, const float *g, const float *bt, int np) {
  constexpr int PER = D / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (wave >= np) return;
  float v[PER], sum = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    v[i] = xs[wave * D + lane + 64 * i];
    sum += v[i];
  }
  const float mean = wave_sum(sum) / (float)D;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    v[i] -= mean;
    sq += v[i] * v[i];
  }
  const float rstd = 1.f / sqrtf(wave_sum(sq) / (float)D + 1e-5f);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int j = lane + 64 * i;
    y[wave * D + j] = f2bf(v[i] * rstd * g[j] + bt[j]);
  }
}

template <int D, int F, int DH>
struct RdShared {
  float xs[2][D];                                      // residual stream rows
  __attribute__((aligned(16))) bf16_t ab[2][D];       // LayerNorm / attention output rows
  __attribute__((aligned(16))) bf16_t hb[2][F];       // FFN hidden rows
  __attribute__((aligned(16))) bf16_t eb[4][D];       // decoder e slices (w, mu, sigma) and tanh
  float hv[128];                                       // decoder outputs
  float part[RD_MAX_PART];                             // the sequence's split partials
  float vec[RD_VEC];                                   // the launch's biases and LayerNorm parameters (rd_vec_*)
  __attribute__((aligned(16))) bf16_t temb[RD_MAX_TYPES * D];   // last layer: every type's embedding row
  float tok_t;
  int tok_k;
};

// the next step's positions pos0 .. pos0 + np - 1: one past the cache
// capacity is flagged
__device__ __forceinline__ void rd_flag_capacity(int cap, uint32_t *status, int np, int pos0) {
  if (threadIdx.x == 0 && pos0 + np > cap) atomicOr(status, TPPSD_STATUS_CAPACITY);
}

// the THP embedding (sin / cos time encoding + type row) of event (t, k) into
// row p; the type rows [K][D] from temb (memory or an LDS copy)
template <int D>
__device__ __forceinline__ void rd_embed(int K, const float *freq, const bf16_t *temb, float *xrow, float t, int k) {
  const int tid = threadIdx.x;
  if (tid < D) {
    const float arg = t * freq[tid];
    const int kk = min(max(k, 0), K - 1);
    xrow[tid] = ((tid & 1) ? cosf(arg) : sinf(arg)) + bf2f(temb[(size_t)kk * D + tid]);
  }
}

// kernel arguments a row launch reads only late (the decoder, the draw and
// the next token), held in registers from the start
struct RdLate {
  const bf16_t *pk_e, *pk_head, *temb;
  uint32_t *status;
  float *tau, *t, *logg, *logf, *mix, *logtype;
  int32_t *k;
  int gamma;
};

// Offsets in RdShared::vec of the small vectors a row launch reads (the
// current layer's output / FFN biases and second LayerNorm; LN_f, the decoder
// biases and the next token's time frequencies). They are loaded before the matrices and
// read from LDS, so that no epilogue waits on a memory load issued behind the
// matrices.
template <int D, int F> struct RdVec {
  static constexpr int OUTB = 0, LN2G = D, LN2B = 2 * D, F1B = 3 * D, F2B = 3 * D + F, N1G = 4 * D + F,
                       N1B = 5 * D + F, K1B = 6 * D + F, MIXB = 7 * D + F, K2B = MIXB + 192, FREQ = K2B + 64,
                       END = FREQ + D;
  static_assert(END <= RD_VEC, "vector area");
};

// Launch modes: step 0 embeds the last two committed events and normalises
// them for layer 0; step l >= 1, layer ly finishes layer ly of the step's
// rows after its attention.
template <int D, int F, int DH, bool SPLIT>
__global__ __launch_bounds__(RD_ROW_THREADS) void k_rd_rows(const int32_t *done_p, const int32_t *len_p,
                                                            const float *part, float *xa, const bf16_t *pk, int l,
                                                            int ly, int part_cnt, RowDraftArgs a) {
  static_assert(D % 64 == 0 && F % 32 == 0 && D % 32 == 0, "row kernel widths");
  __shared__ RdShared<D, F, DH> sh;
  const DraftArgs &d = a.d;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // The leading arguments (the header words' arrays, the partials, the
  // residual rows, the packed matrices, step, layer and the partials per
  // sequence) arrive preloaded in registers, so the first loads and the
  // header words need no kernel-argument load. Every other scalar comes in
  // one batch, waited for once. (Left alone, the compiler loads each where it
  // is first needed and waits there: a dozen round trips before the first
  // barrier, more in the draw.) The asm statement only takes values, which
  // holds each load ahead of it.
  float *xg = xa + (size_t)b * 2 * D;
  const bf16_t *wl = pk + (size_t)ly * rd_layer_elems<D, F>();
  if (l == 0) {
    const int done = d.done[b], base = d.lenD[b], n = d.n[b];
    if (done) return;
    // every step's draw numbers for the round, which depend on no result of
    // the steps: thread j takes step j + 1 (u for the component, the
    // Box-Muller normal deviate, u for the type), and step 1's previous time,
    // the last committed event's (a later step's is written by the step
    // before it)
    const uint64_t rnd = (uint64_t)d.rnd[b];
    const float t_last = d.ev_t[(size_t)b * d.ev_stride + n - 1];
    for (int j = tid; j < d.gamma; j += RD_ROW_THREADS) {
      float u[4];
      philox_uniforms(d.seed, (uint64_t)b, rnd, (uint64_t)(j + 1), TAG_DRAFT, u);
      const float eps = sqrtf(-2.f * logf(u[1])) * cosf(6.28318530717958647692f * u[2]);
      *(float4 *)(a.rng + ((size_t)b * d.MG + j) * 4) = make_float4(u[0], eps, u[3], j == 0 ? t_last : 0.f);
    }
    for (int p = 0; p < 2; ++p) {
      const size_t i = (size_t)b * d.ev_stride + n - 2 + p;
      rd_embed<D>(d.K, d.freq, (const bf16_t *)d.type_emb, sh.xs[p], d.ev_t[i], d.ev_k[i]);
    }
    rd_sync();
    for (int i = tid; i < 2 * D; i += RD_ROW_THREADS) xg[i] = (&sh.xs[0][0])[i];
    rd_flag_capacity(d.cap, d.status, 2, base);
    return;
  }
  const int P = l == 1 ? 2 : 1;
  // every vector load of the launch in flight at once, in the order of use,
  // into registers: the split partials of the sequence (all splits of the
  // slab; those past the step's keys are ignored below), the residual rows,
  // the output projection, then (behind the scalar batch) the small vectors
  // and both FFN products (after the last layer the decoder's follow once the
  // first FFN product is done)
  constexpr int NPV = RD_MAX_PART / RD_ROW_THREADS;
  float pv[NPV];
  {
    const float *src = part + (size_t)b * part_cnt;
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      const int k = tid + i * RD_ROW_THREADS;
      pv[i] = k < part_cnt ? src[k] : 0.f;
    }
  }
  // the residual rows: after a layer whose FFN ran in slices, the rows plus
  // every slice's output
  const float *fp_in = a.fpart + (size_t)b * RD_FSPLIT * 2 * D;
  float xv = 0.f, xs_in[RD_FSPLIT];
  if (tid < P * D) {
    xv = xg[tid];
#pragma unroll
    for (int j = 0; j < RD_FSPLIT; ++j) xs_in[j] = ly > 0 ? fp_in[j * 2 * D + tid] : 0.f;
  }
  RdFrags<D, D> fo;
  fo.load_packed(wl);
  // the scalar batch
  const int L = d.L, M = d.M, K = d.K;
  const int nh = d.H, S = a.S, cap = d.cap, MG = d.MG;
  float *rngp = a.rng;
  const FusedLayerW &w = d.layer[ly];
  const float *outb = w.out_b, *ln2g = w.ln2_g, *ln2b = w.ln2_b, *f1b = w.ffn1_b, *f2b = w.ffn2_b;
  const float *n1g = d.lnf_g, *n1b = d.lnf_b;   // LN_f (the last layer's launch)
  const float *k1b = d.k1_b, *mixb = d.mix_b, *k2b = d.k2_b, *freq = d.freq;
  const int done = load_const(done_p + b), base = load_const(len_p + b);
  const RdLate late{a.pk_e, a.pk_head, (const bf16_t *)d.type_emb, d.status, d.d_tau, d.d_t, d.d_logg, d.d_logf,
                    d.d_mix, d.d_logtype, d.d_k, d.gamma};
  // (d.F only completes the four words from d.F to d.L, so that they come in
  // one load and no register of it is reused while in flight)
  asm volatile("" ::"s"(L), "s"(M), "s"(K), "s"(d.F), "s"(nh), "s"(S), "s"(cap), "s"(MG), "s"(rngp), "s"(outb),
               "s"(ln2g), "s"(ln2b), "s"(f1b), "s"(f2b), "s"(n1g), "s"(n1b), "s"(k1b), "s"(mixb), "s"(k2b),
               "s"(freq), "s"(done), "s"(base), "s"(late.pk_e), "s"(late.pk_head), "s"(late.temb),
               "s"(late.status), "s"(late.tau), "s"(late.t), "s"(late.logg), "s"(late.logf), "s"(late.mix),
               "s"(late.logtype), "s"(late.k), "s"(late.gamma));
  const bool last = ly == L - 1;
  // read late, waited for where used: the step's draw numbers (u for the
  // component, the normal deviate, u for the type) and the time the drawn
  // interval is added to (the last committed event's, or the previous
  // draft's)
  const float *rs = rngp + ((size_t)b * MG + (l - 1)) * 4;
  const float u_z = load_const(rs), eps = load_const(rs + 1), u_k = load_const(rs + 2), tprev = load_const(rs + 3);
  // the launch's small vectors, one unconditional load per element
  typedef RdVec<D, F> V;
  constexpr int NVL = RD_VEC / RD_ROW_THREADS;
  float vl[NVL];
  {
    struct Seg { const float *p; int off, n; };
    const Seg segs[] = {{outb, V::OUTB, D}, {ln2g, V::LN2G, D},       {ln2b, V::LN2B, D},   {f1b, V::F1B, F},
                        {f2b, V::F2B, D},   {n1g, V::N1G, D},         {n1b, V::N1B, D},     {k1b, V::K1B, D},
                        {mixb, V::MIXB, 3 * M}, {k2b, V::K2B, K},     {freq, V::FREQ, D}};
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int k = tid + i * RD_ROW_THREADS;
      const float *src = outb;   // (slots between segments read a valid element, unused)
#pragma unroll
      for (const Seg &g : segs)
        if (k >= g.off && k < g.off + g.n) src = g.p + (k - g.off);
      vl[i] = *src;
    }
  }
  // a non-last layer's launch (SPLIT) has RD_FSPLIT workgroups per sequence,
  // workgroup j taking hidden units j F / RD_FSPLIT .. of the FFN: its rows of
  // W1 and its columns of W2
  constexpr int FS = SPLIT ? F / RD_FSPLIT : F;
  const int js = SPLIT ? blockIdx.y : 0;
  RdFrags<FS, D> f1;
  f1.load_packed(wl + D * D + (size_t)js * FS * D);
  RdFrags<D, FS> f2;
  if (SPLIT) f2.load_packed_k(wl + D * D + F * D, F / 32, js * (FS / 32));
  else f2.load_packed(wl + D * D + F * D);
  RdFrags<4 * D, D> fe;
  RdFrags<128, D> fh;   // the heads' rows (mixture, then type; zero past 3 M + K), packed
  const int pos0 = base + (l == 1 ? 0 : l);
  // (keeps the stores below, which wait for the partials, behind every load)
  __builtin_amdgcn_sched_barrier(0);
  if (done) return;   // workgroup-uniform; the loads above are dropped
#pragma unroll
  for (int i = 0; i < NPV; ++i) sh.part[tid + i * RD_ROW_THREADS] = pv[i];
  if (tid < P * D) {
    float x = xv;
#pragma unroll
    for (int j = 0; j < RD_FSPLIT; ++j) x += xs_in[j];
    (&sh.xs[0][0])[tid] = x;
  }
  rd_sync();
  // merge the attention splits of each (row, head): output = sum_s e^{m_s - m} o_s / sum_s e^{m_s - m} l_s
  {
    const int n_keys = min(pos0 + P, cap);
    const int S_b = (n_keys + RD_KEYS - 1) / RD_KEYS;
    for (int i = tid; i < P * D; i += RD_ROW_THREADS) {
      const int p = i / D, hc = i - p * D, h = hc / DH, c = hc - h * DH;
      const float *pp = sh.part + h * S * 2 * (DH + 2) + p * (DH + 2);
      float mx = -INFINITY;
      for (int s = 0; s < S_b; ++s) mx = fmaxf(mx, pp[s * 2 * (DH + 2)]);
      float ls = 0.f, os = 0.f;
      for (int s = 0; s < S_b; ++s) {
        const float *ps = pp + s * 2 * (DH + 2);
        const float ms = ps[0];
        if (ms == -INFINITY) continue;
        const float f = expf(ms - mx);
        ls += f * ps[1];
        os += f * ps[2 + c];
      }
      sh.ab[p][hc] = f2bf(ls > 0.f ? os / ls : 0.f);
    }
  }
  // the small vectors (issued behind the output projection's fragments, so
  // this waits for those too, which the next product needs anyway)
#pragma unroll
  for (int i = 0; i < NVL; ++i) sh.vec[tid + i * RD_ROW_THREADS] = vl[i];
  rd_sync();
  // output projection + residual
  fo.template mul<2>(&sh.ab[0][0], D, P, [&](int p, int nn, float acc) {
    if (p < P) sh.xs[p][nn] += acc + sh.vec[V::OUTB + nn];
  });
  rd_sync();
  rd_layernorm<D>(&sh.xs[0][0], &sh.ab[0][0], sh.vec + V::LN2G, sh.vec + V::LN2B, P);
  rd_sync();
  f1.template mul<2>(&sh.ab[0][0], D, P, [&](int p, int nn, float acc) {
    if (p < P) sh.hb[p][nn] = f2bf(fmaxf(acc + sh.vec[V::F1B + js * FS + nn], 0.f));
  });
  // the first product's registers are free: after the last layer, the decoder's fragments
  const bool more = l < late.gamma;
  if (last) {
    fe.load_packed(late.pk_e);
    fh.load_packed(late.pk_head);
  }
  rd_sync();
  if constexpr (SPLIT) {
    // this slice's share of the FFN output, to memory; the next launches add
    // the slices to the rows, which workgroup 0 stores with the FFN's bias
    float *fp_out = a.fpart + ((size_t)b * RD_FSPLIT + js) * 2 * D;
    f2.template mul<2>(&sh.hb[0][0], F, P, [&](int p, int nn, float acc) {
      if (p < P) fp_out[p * D + nn] = acc;
    });
    if (js == 0)
      for (int i = tid; i < P * D; i += RD_ROW_THREADS) xg[i] = (&sh.xs[0][0])[i] + sh.vec[V::F2B + i % D];
    return;
  }
  f2.template mul<2>(&sh.hb[0][0], F, P, [&](int p, int nn, float acc) {
    if (p < P) sh.xs[p][nn] += acc + sh.vec[V::F2B + nn];
  });
  // ---- last layer (a launch without slices runs only for it and step 0):
  // decoder on the last row, the draw, the next token
  rd_sync();
  const int pl = P - 1;
  rd_layernorm<D>(&sh.xs[pl][0], &sh.ab[0][0], sh.vec + V::N1G, sh.vec + V::N1B, 1);
  // decoder heads as one product over the four e slices: column n < 3 M reads
  // mixture row n (slice n / M), the others type-head row n - 3 M (tanh slice)
  const int NH = 3 * M + K;
  rd_sync();
  fe.template mul<1>(&sh.ab[0][0], D, 1, [&](int, int nn, float acc) {
    const int slice = nn / D, c = nn - slice * D;
    sh.eb[slice][c] = f2bf(slice < 3 ? acc : tanhf(acc + sh.vec[V::K1B + c]));
  });
  // every type's embedding row for the drawn event, in the first decoder
  // product's freed registers (16-byte vectors, indices clamped into the
  // table's K D / 8), to LDS after the draw
  constexpr int NTE = RD_MAX_TYPES * D / 8 / RD_ROW_THREADS;
  static_assert(NTE * RD_ROW_THREADS * 8 == RD_MAX_TYPES * D, "type rows over the workgroup");
  uint4 te[NTE];
  {
    const int nvec = K * D / 8;
#pragma unroll
    for (int i = 0; i < NTE; ++i) te[i] = *((const uint4 *)late.temb + min(tid + i * RD_ROW_THREADS, nvec - 1));
  }
  rd_sync();
  fh.template mul<4>(&sh.eb[0][0], D, 4, [&](int r, int nn, float acc) {
    if (nn < NH && r == (nn < 3 * M ? nn / M : 3)) sh.hv[nn] = acc + sh.vec[nn < 3 * M ? V::MIXB + nn : V::K2B + nn - 3 * M];
  });
  rd_sync();
  // the log-softmaxes, the draft record and the draft event: wave 0 takes
  // the mixture (component, interval, log g), wave 1 the type (the two
  // chains are independent)
  const size_t di = (size_t)b * MG + (l - 1);
  // categorical over the lanes' log-probabilities: first index whose running
  // sum of exp exceeds u times the total
  auto draw = [&](float lp, int cnt, float uu) {
    float cs = lane < cnt ? expf(lp) : 0.f;
    cs = wave_cumsum(cs);
    const float tot = lane_val(cs, cnt - 1);
    const unsigned long long hit = __ballot(lane < cnt && uu * tot < cs);
    return hit ? (int)__builtin_ctzll(hit) : cnt - 1;
  };
  if (wave == 0) {
    const float lw = lane < M ? sh.hv[lane] : -INFINITY;
    const float mu = lane < M ? sh.hv[M + lane] : 0.f, sg = lane < M ? sh.hv[2 * M + lane] : 0.f;
    const float mw = wave_max(lw);
    const float logw = lw - mw - logf(wave_sum(lane < M ? expf(lw - mw) : 0.f));
    if (lane < M) {
      late.mix[di * 3 * M + lane] = logw;
      late.mix[di * 3 * M + M + lane] = mu;
      late.mix[di * 3 * M + 2 * M + lane] = sg;
    }
    const bool bad = lane < M && !(isfinite(logw) && isfinite(mu) && isfinite(sg));
    const int z = draw(logw, M, u_z);
    const float tau = expf(lane_val(mu, z) + expf(lane_val(sg, z)) * eps);
    const float lt = logf(tau);
    float cterm = -INFINITY;
    if (lane < M) {
      const float zz = lt - mu;
      cterm = logw - sg - 0.918938533204672742f - lt - 0.5f * zz * zz * expf(-2.f * sg);
    }
    const float cm = wave_max(cterm);
    const float lg = cm + logf(wave_sum(lane < M ? expf(cterm - cm) : 0.f));
    const bool bad_any = __ballot(bad) != 0ull;
    if (lane == 0) {
      const float tn = tprev + tau;
      late.tau[di] = tau;
      late.t[di] = tn;
      late.logg[di] = lg;
      if (bad_any || !isfinite(tau)) atomicOr(late.status, TPPSD_STATUS_NONFINITE);
      if (more) rngp[((size_t)b * MG + l) * 4 + 3] = tn;   // the next step's previous time
      sh.tok_t = tn;
    }
  } else if (wave == 1) {
    const float lk = lane < K ? sh.hv[3 * M + lane] : -INFINITY;
    const float mk = wave_max(lk);
    const float logk = lk - mk - logf(wave_sum(lane < K ? expf(lk - mk) : 0.f));
    if (lane < K) late.logtype[di * K + lane] = logk;
    const bool bad_any = __ballot(lane < K && !isfinite(logk)) != 0ull;
    const int kk = draw(logk, K, u_k);
    const float lf = lane_val(logk, kk);
    if (lane == 0) {
      late.k[di] = kk;
      late.logf[di] = lf;
      if (bad_any) atomicOr(late.status, TPPSD_STATUS_NONFINITE);
      sh.tok_k = kk;
    }
  }
  if (!more) return;   // workgroup-uniform
#pragma unroll
  for (int i = 0; i < NTE; ++i) *((uint4 *)sh.temb + tid + i * RD_ROW_THREADS) = te[i];
  rd_sync();
  // the drawn event is the next step's token, at position base + l + 1
  // (its row goes to memory as the residual; the next attention launch
  // applies layer 0's LayerNorm)
  rd_embed<D>(K, sh.vec + V::FREQ, sh.temb, sh.xs[0], sh.tok_t, sh.tok_k);
  if (tid < D) xg[tid] = sh.xs[0][tid];   // (the element this thread wrote)
  rd_flag_capacity(cap, late.status, 1, base + l + 1);
}

}  // namespace

bool row_draft_ok(int bf16, int L, int d, int H, int F, int M, int K, int kv_cap) {
  return bf16 && L >= 1 && L <= FD_MAX_LAYERS && d == 128 && H == 4 && F == 512 && M >= 1 && M <= 64 && K >= 1 &&
         K <= RD_MAX_TYPES && 3 * M + K <= 128 && (size_t)H * rd_splits(kv_cap) * 2 * (32 + 2) <= (size_t)RD_MAX_PART;
}

void launch_pack_rd_head(const void *mix_w, const void *k2_w, int M, int K, int D, void *out, hipStream_t st) {
  const int total = 8 * (D / 32) * 64;
  hipLaunchKernelGGL(k_pack_rd_head, dim3((total + 255) / 256), dim3(256), 0, st, (const bf16_t *)mix_w,
                     (const bf16_t *)k2_w, M, K, D, (bf16_t *)out);
}

void launch_draft_rows(RowDraftArgs a, hipStream_t st, const hipEvent_t *ev) {
  const int B = a.d.B, H = a.d.H;
  const int part_cnt = H * a.S * 2 * (32 + 2);   // split partials per sequence
  int j = 0;   // launch index: event pair j brackets launch j
  auto e0 = [&]() { return ev ? ev[2 * j] : nullptr; };
  auto e1 = [&]() { return ev ? ev[2 * j + 1] : nullptr; };
  // (the row kernel's leading arguments, preloaded into registers, repeat
  // fields of a that its first loads need; a non-last layer's launch has
  // RD_FSPLIT workgroups per sequence)
  auto rows = [&]() {
    if (a.step > 0 && a.layer < a.d.L - 1)
      hipExtLaunchKernelGGL(k_rd_rows<128, 512, 32, true>, dim3(B, RD_FSPLIT), dim3(RD_ROW_THREADS), 0, st, e0(),
                            e1(), 0, a.d.done, a.d.lenD, (const float *)a.part, a.x, a.pk, a.step, a.layer, part_cnt,
                            a);
    else
      hipExtLaunchKernelGGL(k_rd_rows<128, 512, 32, false>, dim3(B), dim3(RD_ROW_THREADS), 0, st, e0(), e1(), 0,
                            a.d.done, a.d.lenD, (const float *)a.part, a.x, a.pk, a.step, a.layer, part_cnt, a);
  };
  a.step = 0;
  a.layer = 0;
  rows();
  ++j;
  for (int l = 1; l <= a.d.gamma; ++l) {
    a.step = l;
    for (int ly = 0; ly < a.d.L; ++ly) {
      a.layer = ly;
      hipExtLaunchKernelGGL(k_rd_attn<128, 32>, dim3(a.S, H, B), dim3(256), 0, st, e0(), e1(), 0, a.d.done,
                            a.d.lenD, a.step, a.layer, a);
      ++j;
      rows();
      ++j;
    }
  }
}

}  // namespace tppsd
