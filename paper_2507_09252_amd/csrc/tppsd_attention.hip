// Causal attention of the verify, AR, prefill and layered draft passes over
// the KV caches (MFMA kernels for bf16 and fp32, and the merge of key
// splits), with their launchers.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <stdint.h>

#include "tppsd_device.h"

namespace tppsd {

// ---------------------------------------------------------------------------
// causal attention of P new queries per (sequence, head) over the KV cache
// (App. D.4: softmax-normalised exp(q.k / sqrt(d_head)) weights over the
// event and its predecessors). Query p of sequence b sees cached positions
// 0 .. start[b] + start_off + p. Online softmax over 64-key tiles.
// ---------------------------------------------------------------------------

// ROLE tags the instantiation only (1 = verify pass of the target, 0 = other
// passes), so that profiles report the verify launches under their own name.
// AttNHP attention (App. D.4) divides by 1 + sum f instead of sum f: the same
// as one more key of score 0 and value 0. Applied once, where the softmax
// state (max M, sum L, unnormalised output O) of all keys is complete.
__device__ __forceinline__ void sink_adjust(float &M, float &L, float &O) {
  const float ms = fmaxf(M, 0.f), f = (M == -INFINITY) ? 0.f : expf(M - ms);
  L = L * f + expf(-ms);
  O *= f;
}

// bf16 causal attention on MFMA with split keys (flash-decoding style).
// Grid (B * H, 1, splits), NW = 4 or 8 waves per workgroup; the workgroup
// serves all QT query tiles of 16 of its (sequence, head), so each key and
// value is read from memory once per split whatever the number of queries. A
// split owns a contiguous key range; its waves take 32-key steps round robin
// and keep their own online-softmax state per query tile, merged in LDS at
// the end (with eight waves, waves 4..7 first hand theirs to waves 0..3).
// With one split the merged result is the output, otherwise the split writes
// (max, sum, unnormalised output) and k_attn_combine merges. Eight waves and
// one split replace two splits of four waves: the same waves stream the keys,
// and the merge launch goes away.
//
// Per 32-key step and query tile, S^T = K Q^T is two 16x16 MFMA tiles whose
// rows are permuted so that lane l ends up holding the scores of query
// (l mod 16) for the 8 consecutive keys 8 (l / 16) .. + 7: exactly the B
// operand of O^T = V^T P^T. The A operand (8 consecutive keys of one value
// column) is one 16-byte load from the position-blocked value cache.

template <int DH, int ROLE, int QT, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_attn_mfma(int H, int P, const int32_t *__restrict__ start,
                                                   const int32_t *__restrict__ done, int start_off,
                                                   const bf16_t *__restrict__ q, const bf16_t *__restrict__ kc,
                                                   const bf16_t *__restrict__ vc, bf16_t *__restrict__ o, int cap,
                                                   int splits, float *__restrict__ part, int sink) {
  constexpr int KT = 32, NDT = DH / 16, NC = DH >= 32 ? DH / 32 : 1, NQ = 16 * QT;
  static_assert(NW == 4 || NW == 8, "four or eight waves");
  __shared__ float red_m[4][NQ], red_l[4][NQ];
  __shared__ float red_o[4][DH][NQ + 1];
  const int bh = blockIdx.x, b = bh / H, h = bh - b * H, split = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, rr = lane & 15, g = lane >> 4;
  const int d = H * DH;
  // the header words in one batch with the remaining arguments (the leading
  // ones arrive preloaded; the finished flag is read unconditionally, from
  // the start array when there is none)
  const int dv = done ? done[b] : start[b];
  const int sv = start[b];
  asm volatile("" ::"s"(dv), "s"(sv), "s"(cap), "s"(splits));
  const bool skip = done != nullptr && dv != 0;
  const int base = sv + start_off;
  const int n_keys = skip ? 0 : min(base + P, cap);   // never past the cache slab
  int chunk = (n_keys + splits - 1) / splits;
  chunk = (chunk + KT - 1) / KT * KT;
  const int k_begin = split * chunk, k_end = min(n_keys, k_begin + chunk);
  const size_t kvbase = ((size_t)b * H + h) * cap;
  // scores are kept in base-2 units (q.k / sqrt(d_head) times log2 e), so
  // that every exponential is one exp2 instruction; maxima leave the kernel
  // in natural units
  const float scale2 = 1.4426950408889634f / sqrtf((float)DH);
  constexpr float LN2 = 0.69314718055994531f;
  // all-ones A operand: O^T rows of ones give each query's sum of the
  // (bf16-rounded) probabilities the P V product takes
  const bf16x8_t ones = __builtin_bit_cast(bf16x8_t, make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));

  // query fragments (B operand of S^T): Q[16 t + rr][k slice of lane group g]
  bf16x8_t qf[QT][NC];
  short4_t qf16[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int my_q = 16 * t + rr;
    const bool q_ok = my_q < P;
    const bf16_t *qp = q + (size_t)(b * P + (q_ok ? my_q : 0)) * d + h * DH;
    if (DH >= 32) {
#pragma unroll
      for (int c = 0; c < NC; ++c) qf[t][c] = q_ok ? *(const bf16x8_t *)(qp + 32 * c + 8 * g) : (bf16x8_t){};
    } else {
      qf16[t] = q_ok ? *(const short4_t *)(qp + 4 * g) : (short4_t){0, 0, 0, 0};
    }
  }
  float m_run[QT];
  f32x4_t oacc[QT][NDT], lacc[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    lacc[t] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int td = 0; td < NDT; ++td) oacc[t][td] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }
  // permuted key rows of the two S^T halves loaded by this lane
  const int krow0 = 8 * (rr >> 2) + (rr & 3), krow1 = krow0 + 4;

  for (int kt = k_begin + wave * KT; kt < k_end; kt += NW * KT) {
    const bool interior = kt + KT <= k_end && kt + KT <= base + 1;   // every key visible to every query
    const size_t r0 = kvbase + min(kt + krow0, cap - 1), r1 = kvbase + min(kt + krow1, cap - 1);
    bf16x8_t a0[NC], a1[NC];
    short4_t b0 = {0, 0, 0, 0}, b1 = {0, 0, 0, 0};
    if (DH >= 32) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        a0[c] = *(const bf16x8_t *)(kc + r0 * DH + 32 * c + 8 * g);
        a1[c] = *(const bf16x8_t *)(kc + r1 * DH + 32 * c + 8 * g);
      }
    } else {
      b0 = *(const short4_t *)(kc + r0 * DH + 4 * g);
      b1 = *(const short4_t *)(kc + r1 * DH + 4 * g);
    }
    // values of keys kt + 8 g .. + 7, columns 16 td + rr; blocks past the key
    // range read the range's last block (unconditional loads: a load under a
    // lane condition makes the compiler wait for every load before it), and
    // positions past the range are zeroed (never-written cache slots may hold
    // NaN bits)
    const int k8 = kt + 8 * g, nv = k_end - k8;
    const int k8c = min(k8, (k_end - 1) & ~7);
    uint4 vw[NDT];
#pragma unroll
    for (int td = 0; td < NDT; ++td)
      vw[td] = *(const uint4 *)(vc + kvbase * DH + (size_t)(k8c >> 3) * (8 * DH) + (16 * td + rr) * 8);
    if (!interior && nv < 8) {
#pragma unroll
      for (int td = 0; td < NDT; ++td) {
        uint32_t w[4] = {vw[td].x, vw[td].y, vw[td].z, vw[td].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (2 * i >= nv) w[i] = 0u;
          else if (2 * i + 1 >= nv) w[i] &= 0xFFFFu;
        }
        vw[td] = (uint4){w[0], w[1], w[2], w[3]};
      }
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
      if (DH >= 32) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[c], qf[t][c], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[c], qf[t][c], s1, 0, 0, 0);
        }
      } else {
        s0 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(b0, qf16[t], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(b1, qf16[t], s1, 0, 0, 0);
      }
      // scores of keys kt + 8g + j, j = 0..7, for query 16 t + rr (steps
      // wholly inside every query's visible range skip the masks; padding
      // queries then carry finite scores of zero queries, never stored)
      const int my_q = 16 * t + rr, my_last = base + my_q;
      const bool q_ok = my_q < P;
      float sv[8];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int key = kt + 8 * g + j;
        const float raw = (j < 4) ? s0[j] : s1[j - 4];
        const bool ok = interior || (q_ok && key < k_end && key <= my_last);
        sv[j] = ok ? raw * scale2 : -INFINITY;
        mx = fmaxf(mx, sv[j]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run[t], mx);
      // (exp2 of -inf is 0: masked keys and an empty running state drop out)
      const float m_ref = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run[t] - m_ref);
      uint32_t pw[4];
#pragma unroll
      for (int j = 0; j < 8; j += 2)
        pw[j >> 1] = pk2bf(__builtin_amdgcn_exp2f(sv[j] - m_ref), __builtin_amdgcn_exp2f(sv[j + 1] - m_ref));
      // P V takes the probabilities in bf16; the normaliser (the ones rows)
      // sums the same rounded values, so the output stays a convex
      // combination of values
      const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, (uint4){pw[0], pw[1], pw[2], pw[3]});
      m_run[t] = m_new;
      // the accumulators are rescaled only when some query's maximum rose
      // (alpha is exactly 1 otherwise)
      if (__ballot(alpha != 1.f) != 0ull) {
        lacc[t] *= alpha;
#pragma unroll
        for (int td = 0; td < NDT; ++td) oacc[t][td] *= alpha;
      }
      lacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb, lacc[t], 0, 0, 0);
#pragma unroll
      for (int td = 0; td < NDT; ++td)
        oacc[t][td] =
            __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vw[td]), pb, oacc[t][td], 0, 0, 0);
    }
  }
  // lane (rr, g) holds O^T[16 td + 4 g + i][query 16 t + rr]
  if constexpr (NW == 8) {
    // waves 4..7 hand their state to waves 0..3 (same lane layout), which
    // fold it into theirs
    if (wave >= 4) {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        if (g == 0) {
          red_m[wave - 4][16 * t + rr] = m_run[t];
          red_l[wave - 4][16 * t + rr] = lacc[t][0];
        }
#pragma unroll
        for (int td = 0; td < NDT; ++td)
#pragma unroll
          for (int i = 0; i < 4; ++i) red_o[wave - 4][16 * td + 4 * g + i][16 * t + rr] = oacc[t][td][i];
      }
    }
    __syncthreads();
    if (wave < 4) {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const float mp = red_m[wave][16 * t + rr], lp = red_l[wave][16 * t + rr];
        const float mn = fmaxf(m_run[t], mp);
        const float fs = (m_run[t] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run[t] - mn);
        const float fp = (mp == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mp - mn);
        m_run[t] = mn;
        lacc[t][0] = lacc[t][0] * fs + lp * fp;
#pragma unroll
        for (int td = 0; td < NDT; ++td)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            oacc[t][td][i] = oacc[t][td][i] * fs + red_o[wave][16 * td + 4 * g + i][16 * t + rr] * fp;
      }
    }
    __syncthreads();
  }
  // merge the (first) four waves
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    if (wave < 4) {
      if (g == 0) {
        red_m[wave][16 * t + rr] = m_run[t];
        red_l[wave][16 * t + rr] = lacc[t][0];
      }
#pragma unroll
      for (int td = 0; td < NDT; ++td)
#pragma unroll
        for (int i = 0; i < 4; ++i) red_o[wave][16 * td + 4 * g + i][16 * t + rr] = oacc[t][td][i];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < NQ * DH; idx += 64 * NW) {
    const int qq = idx / DH, j = idx - qq * DH;
    if (qq >= P) continue;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, red_m[w][qq]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = (red_m[w][qq] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(red_m[w][qq] - M);
      L += red_l[w][qq] * f;
      O += red_o[w][j][qq] * f;
    }
    M *= LN2;   // natural units from here
    if (splits == 1) {
      if (sink) sink_adjust(M, L, O);
      o[(size_t)(b * P + qq) * d + h * DH + j] = f2bf(L > 0.f ? O / L : 0.f);
    } else {
      float *pp = part + (((size_t)bh * QT * 16 + qq) * splits + split) * (DH + 2);
      pp[2 + j] = O;
      if (j == 0) {
        pp[0] = M;
        pp[1] = L;
      }
    }
  }
}

// fp32 causal attention on MFMA (v_mfma_f32_16x16x4f32), same work split,
// query tiles per workgroup and permuted S^T rows as the bf16 kernel. One
// MFMA contracts four k values, one per lane group g: S^T takes d in float4
// slices (element e of lane group g is d = 4 g + e), and O^T = V^T P^T runs
// one MFMA per j = 0..7 over the keys 8 g + j, which are exactly the eight
// scores each lane holds. V is read straight from memory (16 consecutive
// columns of one key per lane group).
template <int DH, int ROLE, int QT>
__global__ __launch_bounds__(256) void k_attn_mfma_f32(int H, int P, const int32_t *__restrict__ start,
                                                       const int32_t *__restrict__ done, int start_off,
                                                       const float *__restrict__ q, const float *__restrict__ kc,
                                                       const float *__restrict__ vc, float *__restrict__ o, int cap,
                                                       int splits, float *__restrict__ part, int sink) {
  constexpr int KT = 32, NDT = DH / 16, NQ = 16 * QT;
  __shared__ float red_m[4][NQ], red_l[4][NQ];
  __shared__ float red_o[4][DH][NQ + 1];
  const int bh = blockIdx.x, b = bh / H, h = bh - b * H, split = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, rr = lane & 15, g = lane >> 4;
  const int d = H * DH;
  // the header words in one batch with the remaining arguments (the leading
  // ones arrive preloaded; the finished flag is read unconditionally, from
  // the start array when there is none)
  const int dv = done ? done[b] : start[b];
  const int sv = start[b];
  asm volatile("" ::"s"(dv), "s"(sv), "s"(cap), "s"(splits));
  const bool skip = done != nullptr && dv != 0;
  const int base = sv + start_off;
  const int n_keys = skip ? 0 : min(base + P, cap);   // never past the cache slab
  int chunk = (n_keys + splits - 1) / splits;
  chunk = (chunk + KT - 1) / KT * KT;
  const int k_begin = split * chunk, k_end = min(n_keys, k_begin + chunk);
  const size_t kvbase = ((size_t)b * H + h) * cap;
  const float scale = 1.f / sqrtf((float)DH);
  f32x4_t qf[QT][DH / 16];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int my_q = 16 * t + rr;
    const bool q_ok = my_q < P;
    const float *qp = q + (size_t)(b * P + (q_ok ? my_q : 0)) * d + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c)
      qf[t][c] = q_ok ? *(const f32x4_t *)(qp + 16 * c + 4 * g) : (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }
  float m_run[QT], l_run[QT];
  f32x4_t oacc[QT][NDT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int td = 0; td < NDT; ++td) oacc[t][td] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  }
  const int krow0 = 8 * (rr >> 2) + (rr & 3), krow1 = krow0 + 4;
  // a wave loads a batch of NB of its 32-key steps before computing any
  // (positions clamped into the range; steps past it are skipped), then takes
  // one online-softmax update per query tile for the whole batch
  constexpr int NB = (DH >= 32 || QT >= 2) ? 2 : 4;
  struct Step {
    f32x4_t a0[DH / 16], a1[DH / 16];
    float vv[NDT][8];
  };
  const int last_step = k_end > k_begin ? k_begin + (k_end - 1 - k_begin) / KT * KT : k_begin;
  for (int kb = k_begin + wave * KT; kb < k_end; kb += NB * 4 * KT) {
    Step f[NB];
#pragma unroll
    for (int sidx = 0; sidx < NB; ++sidx) {
      const int kt = min(kb + sidx * 4 * KT, last_step);
      const size_t r0 = kvbase + min(kt + krow0, cap - 1), r1 = kvbase + min(kt + krow1, cap - 1);
#pragma unroll
      for (int c = 0; c < DH / 16; ++c) {
        f[sidx].a0[c] = *(const f32x4_t *)(kc + r0 * DH + 16 * c + 4 * g);
        f[sidx].a1[c] = *(const f32x4_t *)(kc + r1 * DH + 16 * c + 4 * g);
      }
      // value column 16 td + rr of keys kt + 8 g + j (zero past the key range)
#pragma unroll
      for (int td = 0; td < NDT; ++td)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = kt + 8 * g + j;
          const float v = vc[(kvbase + min(key, k_end - 1)) * DH + 16 * td + rr];
          f[sidx].vv[td][j] = (key < k_end) ? v : 0.f;
        }
    }
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int my_q = 16 * t + rr, my_last = base + my_q;
      const bool q_ok = my_q < P;
      float sv[NB][8];
      float mx = -INFINITY;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx) {
        const int kt = kb + sidx * 4 * KT;
        if (kt >= k_end) {   // uniform across the wave
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[sidx][j] = -INFINITY;
          continue;
        }
        f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < DH / 16; ++c)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].a0[c][e], qf[t][c][e], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].a1[c][e], qf[t][c][e], s1, 0, 0, 0);
          }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = kt + 8 * g + j;
          const float raw = (j < 4) ? s0[j] : s1[j - 4];
          sv[sidx][j] = (q_ok && key < k_end && key <= my_last) ? raw * scale : -INFINITY;
          mx = fmaxf(mx, sv[sidx][j]);
        }
      }
      mx = fmaxf(mx, swz_xor<16>(mx));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run[t], mx);
      const float alpha = (m_new == -INFINITY) ? 1.f : expf(m_run[t] - m_new);
      float ps = 0.f;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          sv[sidx][j] = (sv[sidx][j] == -INFINITY) ? 0.f : expf(sv[sidx][j] - m_new);
          ps += sv[sidx][j];
        }
      ps += swz_xor<16>(ps);
      ps += __shfl_xor(ps, 32, 64);
      l_run[t] = l_run[t] * alpha + ps;
      m_run[t] = m_new;
#pragma unroll
      for (int td = 0; td < NDT; ++td) oacc[t][td] *= alpha;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx) {
        if (kb + sidx * 4 * KT >= k_end) break;
#pragma unroll
        for (int td = 0; td < NDT; ++td)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            oacc[t][td] = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].vv[td][j], sv[sidx][j], oacc[t][td], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    if (g == 0) {
      red_m[wave][16 * t + rr] = m_run[t];
      red_l[wave][16 * t + rr] = l_run[t];
    }
#pragma unroll
    for (int td = 0; td < NDT; ++td)
#pragma unroll
      for (int i = 0; i < 4; ++i) red_o[wave][16 * td + 4 * g + i][16 * t + rr] = oacc[t][td][i];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < NQ * DH; idx += 256) {
    const int qq = idx / DH, j = idx - qq * DH;
    if (qq >= P) continue;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, red_m[w][qq]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = (red_m[w][qq] == -INFINITY) ? 0.f : expf(red_m[w][qq] - M);
      L += red_l[w][qq] * f;
      O += red_o[w][j][qq] * f;
    }
    if (splits == 1) {
      if (sink) sink_adjust(M, L, O);
      o[(size_t)(b * P + qq) * d + h * DH + j] = L > 0.f ? O / L : 0.f;
    } else {
      float *pp = part + (((size_t)bh * QT * 16 + qq) * splits + split) * (DH + 2);
      pp[2 + j] = O;
      if (j == 0) {
        pp[0] = M;
        pp[1] = L;
      }
    }
  }
}

// merge of the split partials: one thread per output element
template <typename ACT, int DH>
__global__ void k_attn_combine(const float *__restrict__ part, ACT *__restrict__ o, int total, int P, int H,
                               int qtiles, int splits, int sink) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;   // over B * H * P * DH
  if (idx >= total) return;
  const int j = idx % DH;
  const int rest = idx / DH;
  const int p = rest % P, bh = rest / P;
  const int h = bh % H, b = bh / H;
  const float *pp = part + ((size_t)bh * qtiles * 16 + p) * splits * (DH + 2);
  float M = -INFINITY;
  for (int s = 0; s < splits; ++s) M = fmaxf(M, pp[s * (DH + 2)]);
  float L = 0.f, O = 0.f;
  for (int s = 0; s < splits; ++s) {
    const float m = pp[s * (DH + 2)];
    const float f = (m == -INFINITY) ? 0.f : expf(m - M);
    L += pp[s * (DH + 2) + 1] * f;
    O += pp[s * (DH + 2) + 2 + j] * f;
  }
  if (sink) sink_adjust(M, L, O);
  st(o, (size_t)(b * P + p) * (H * DH) + h * DH + j, L > 0.f ? O / L : 0.f);
}

// All query tiles of a (sequence, head) share one workgroup (QT = 1..3 for
// up to 48 new positions); the key range is split across workgroups when the
// (sequence, head) pairs alone do not fill the chip.
template <typename ACT, int DH, int ROLE>
static void attn_mfma(const ACT *Q, const ACT *Kc, const ACT *Vc, ACT *O, const int32_t *start, int start_off,
                      const int32_t *done, int B, int P, int H, int cap, float *part, int sink, hipEvent_t ev0,
                      hipEvent_t ev1, hipStream_t s) {
  const int qtiles = (P + 15) / 16;
  int splits = attn_splits(B, H, cap);
  // bf16: two splits of four waves become one workgroup of eight
  const bool eight = sizeof(ACT) == 2 && splits == 2;
  if (eight) splits = 1;
  dim3 grid(B * H, 1, splits);
  auto go = [&](auto kern, int nt) {
    hipExtLaunchKernelGGL(kern, grid, dim3(nt), 0, s, ev0, ev1, 0, H, P, start, done, start_off, Q, Kc, Vc, O, cap,
                          splits, part, sink);
  };
  if constexpr (sizeof(ACT) == 2) {
    if (eight) {
      if (qtiles == 1) go(k_attn_mfma<DH, ROLE, 1, 8>, 512);
      else if (qtiles == 2) go(k_attn_mfma<DH, ROLE, 2, 8>, 512);
      else go(k_attn_mfma<DH, ROLE, 3, 8>, 512);
    } else {
      if (qtiles == 1) go(k_attn_mfma<DH, ROLE, 1>, 256);
      else if (qtiles == 2) go(k_attn_mfma<DH, ROLE, 2>, 256);
      else go(k_attn_mfma<DH, ROLE, 3>, 256);
    }
  } else {
    if (qtiles == 1) go(k_attn_mfma_f32<DH, ROLE, 1>, 256);
    else if (qtiles == 2) go(k_attn_mfma_f32<DH, ROLE, 2>, 256);
    else go(k_attn_mfma_f32<DH, ROLE, 3>, 256);
  }
  if (splits > 1) {
    const int total = B * H * P * DH;
    k_attn_combine<ACT, DH><<<(total + 255) / 256, 256, 0, s>>>(part, O, total, P, H, qtiles, splits, sink);
  }
}

// ev0/ev1 (optional): HIP events stamped with the main kernel's own start and
// stop (hipExtLaunchKernelGGL), for the verify-attention timing
template <int ROLE>
static void attention_role(const void *q, const void *kc, const void *vc, void *o, int bf16, const int32_t *start,
                           int start_off, const int32_t *done, int B, int P, int H, int dh, int cap, float *part,
                           int sink, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (!bf16) {
    const float *Q = (const float *)q, *Kc = (const float *)kc, *Vc = (const float *)vc;
    float *O = (float *)o;
    switch (dh) {
      case 16: attn_mfma<float, 16, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
      case 32: attn_mfma<float, 32, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
      default: attn_mfma<float, 64, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
    }
    return;
  }
  const bf16_t *Q = (const bf16_t *)q, *Kc = (const bf16_t *)kc, *Vc = (const bf16_t *)vc;
  bf16_t *O = (bf16_t *)o;
  switch (dh) {
    case 16: attn_mfma<bf16_t, 16, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
    case 32: attn_mfma<bf16_t, 32, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
    default: attn_mfma<bf16_t, 64, ROLE>(Q, Kc, Vc, O, start, start_off, done, B, P, H, cap, part, sink, ev0, ev1, s); break;
  }
}

void launch_attention(const void *q, const void *kc, const void *vc, void *o, int bf16, const int32_t *start,
                      int start_off, const int32_t *done, int B, int P, int H, int dh, int cap, float *part,
                      int sink, int verify, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (verify)
    attention_role<1>(q, kc, vc, o, bf16, start, start_off, done, B, P, H, dh, cap, part, sink, ev0, ev1, s);
  else
    attention_role<0>(q, kc, vc, o, bf16, start, start_off, done, B, P, H, dh, cap, part, sink, ev0, ev1, s);
}

}  // namespace tppsd
