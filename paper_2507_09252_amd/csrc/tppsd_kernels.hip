// HIP kernels of the TPP-SD hot path for gfx950 (MI355X).
//
// Encoder and decoder of the CDF-based Transformer TPP (paper §4.2, App. D.4),
// block verification and the accept / adjusted-distribution step of TPP-SD
// (§4.3, Eq. (3)-(4), Theorem 1, Algorithm 1), and the sampling epilogues of
// drafting and naive AR sampling (§4.2, App. A.1).
//
// Precision: fp32 models run fp32 everywhere. bf16 models keep matrices and
// Linear inputs in bf16 (LN outputs, q/k/v, attention output, ReLU output, the
// decoder's e and tanh activations), accumulate in fp32 and keep the residual
// stream, LayerNorm statistics, softmax and all decoder math in fp32.
#include <algorithm>
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <math.h>
#include <stdlib.h>
#include <stdint.h>
#include <type_traits>

#include "tppsd_device.h"
#include "tppsd_philox.h"
#include "../../include/tppsd.h"

namespace tppsd {

// ---------------------------------------------------------------------------
// decoder math (log-normal mixture of §4.2; sampling as in App. A.1)
// ---------------------------------------------------------------------------

// log g(tau) = logsumexp_m [log w_m - s_m - log(2 pi)/2 - ln tau - (ln tau - mu_m)^2 / (2 e^{2 s_m})]
__device__ float mix_logpdf(const float *logw, const float *mu, const float *s, int M, float tau) {
  const float lt = logf(tau);
  float mx = -INFINITY;
  for (int m = 0; m < M; ++m) {
    float z = lt - mu[m];
    float c = logw[m] - s[m] - 0.918938533204672742f - lt - 0.5f * z * z * expf(-2.f * s[m]);
    mx = fmaxf(mx, c);
  }
  float acc = 0.f;
  for (int m = 0; m < M; ++m) {
    float z = lt - mu[m];
    float c = logw[m] - s[m] - 0.918938533204672742f - lt - 0.5f * z * z * expf(-2.f * s[m]);
    acc += expf(c - mx);
  }
  return mx + logf(acc);
}

// first index m with u * C_total < C_m, C the ascending running sum of exp(logp)
__device__ int sample_cat(const float *logp, int n, float u) {
  float tot = 0.f;
  for (int m = 0; m < n; ++m) tot += expf(logp[m]);
  const float x = u * tot;
  float c = 0.f;
  for (int m = 0; m < n; ++m) {
    c += expf(logp[m]);
    if (x < c) return m;
  }
  return n - 1;
}

// Wave-parallel form of the mixture log-density above for M <= 64 (lane m
// holds component m).
__device__ float wave_mix_logpdf(const float *logw, const float *mu, const float *s, int M, float tau) {
  const int lane = threadIdx.x & 63;
  const float lt = logf(tau);
  float c = -INFINITY;
  if (lane < M) {
    const float z = lt - mu[lane];
    c = logw[lane] - s[lane] - 0.918938533204672742f - lt - 0.5f * z * z * expf(-2.f * s[lane]);
  }
  const float mx = wave_max(c);
  return mx + logf(wave_sum(lane < M ? expf(c - mx) : 0.f));
}

// log(1 - G(x)) of the log-normal mixture whose component m sits in lane m
// (valid = false in the other lanes): log-sum-exp over m of log w_m +
// log Phi(-z_m), z_m = (ln x - mu_m) / sigma_m. With y = z / sqrt(2),
// Phi(-z) = erfc(y) / 2, taken as erfcx(y) e^(-y^2) / 2 for y > 0 so that the
// logarithm does not underflow. x <= 0 (wave-uniform) gives 0.
__device__ float wave_log_survival(float logw, float mu, float s, bool valid, float x) {
  if (!(x > 0.f)) return 0.f;
  float c = -INFINITY;
  if (valid) {
    const float y = (logf(x) - mu) * expf(-s) * 0.707106781186547524f;
    const float lphi = y > 0.f ? logf(0.5f * erfcxf(y)) - y * y : logf(0.5f * erfcf(y));
    c = logw + lphi;
  }
  const float mx = wave_max(c);
  return mx + logf(wave_sum(valid ? expf(c - mx) : 0.f));
}

// z ~ Categorical(w), eps = Box-Muller(u1, u2), tau = exp(mu_z + sigma_z eps)
__device__ float sample_tau(const float *logw, const float *mu, const float *s, int M, float uc, float u1,
                            float u2) {
  const int z = sample_cat(logw, M, uc);
  const float eps = sqrtf(-2.f * logf(u1)) * cosf(6.28318530717958647692f * u2);
  return expf(mu[z] + expf(s[z]) * eps);
}

// ---------------------------------------------------------------------------
// event embedding: x = z(t) + W_type[k]   (§4.2 Encoder, App. D.4 THP encoding)
// ---------------------------------------------------------------------------

template <typename W>
__global__ void k_embed(float *__restrict__ x, int d, int P, TokSrc src, const W *__restrict__ wtype,
                        const float *__restrict__ freq, int K) {
  const int tok = blockIdx.x;
  const int b = tok / P, p = tok % P;
  float t;
  int k;
  if (p < src.n_ev) {
    const size_t i = (size_t)b * src.ev_stride + src.start[b] + src.start_off + p;
    t = src.ev_t[i];
    k = src.ev_k[i];
  } else {
    const size_t i = (size_t)b * src.dr_stride + src.dr_off + (p - src.n_ev);
    t = src.dr_t[i];
    k = src.dr_k[i];
  }
  k = min(max(k, 0), K - 1);
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const float arg = t * freq[j];
    const float z = (j & 1) ? cosf(arg) : sinf(arg);
    x[(size_t)tok * d + j] = z + ld(wtype, (size_t)k * d + j);
  }
}

// AttNHP encoder pieces (App. D.4). The event's first-layer state is its
// type row; the time enters every layer through the layer input
// u = [z(t); h] (activation type, row stride 2d), z with the AttNHP
// wavelengths (the frequency table holds 1 / (m (5M/m)^((j - j mod 2)/d))).
template <typename W>
__global__ void k_embed_attnhp(float *__restrict__ x, W *__restrict__ u, int d, int P, TokSrc src,
                               const W *__restrict__ wtype, const float *__restrict__ freq, int K) {
  const int tok = blockIdx.x;
  const int b = tok / P, p = tok % P;
  float t;
  int k;
  if (p < src.n_ev) {
    const size_t i = (size_t)b * src.ev_stride + src.start[b] + src.start_off + p;
    t = src.ev_t[i];
    k = src.ev_k[i];
  } else {
    const size_t i = (size_t)b * src.dr_stride + src.dr_off + (p - src.n_ev);
    t = src.dr_t[i];
    k = src.dr_k[i];
  }
  k = min(max(k, 0), K - 1);
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const float arg = t * freq[j];
    const float h = ld(wtype, (size_t)k * d + j);
    x[(size_t)tok * d + j] = h;
    st(u, (size_t)tok * 2 * d + j, (j & 1) ? cosf(arg) : sinf(arg));
    st(u, (size_t)tok * 2 * d + d + j, h);
  }
}

// h += tanh(o) per element; the new h goes to the stream x, to u's h half and
// to a (the next decoder's operand)
template <typename ACT>
__global__ void k_attnhp_update(float *__restrict__ x, const ACT *__restrict__ o, ACT *__restrict__ u,
                                ACT *__restrict__ a, int T, int d) {
  const size_t n = (size_t)T * d;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t r = i / d, j = i - r * d;
    const float v = x[i] + tanhf(ld(o, i));
    x[i] = v;
    st(u, r * 2 * d + d + j, v);
    st(a, i, v);
  }
}

// ---------------------------------------------------------------------------
// LayerNorm (biased variance, eps 1e-5), one wave per row
// ---------------------------------------------------------------------------

constexpr int LN_REG_MAX = 16;   // row widths up to 1024 are held in registers
constexpr int LN_VEC_MAX = 4;    // as 16-byte vectors when the width is a multiple of 4
// four consecutive outputs (the index a multiple of 4)
__device__ __forceinline__ void st4(float *p, size_t i, float a, float b, float c, float d) {
  *(float4 *)(p + i) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void st4(bf16_t *p, size_t i, float a, float b, float c, float d) {
  *(uint2 *)(p + i) = make_uint2(pk2bf(a, b), pk2bf(c, d));
}
template <typename ACT>
__global__ __launch_bounds__(256) void k_layernorm(const float *__restrict__ x, ACT *__restrict__ y,
                                                   const float *__restrict__ g, const float *__restrict__ bt,
                                                   int T, int d) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T) return;
  const float *xr = x + (size_t)row * d;
  const bool vec = d % 4 == 0 && d <= 4 * 64 * LN_VEC_MAX &&
                   (((uintptr_t)x | (uintptr_t)g | (uintptr_t)bt) & 15) == 0 && ((uintptr_t)y & 7) == 0;
  if (vec) {
    // lane owns columns 4 (lane + 64 i) .. + 3: the row, gain and bias as
    // 16-byte loads, all issued before the reductions, and 4 columns per store
    float4 xv[LN_VEC_MAX], gv[LN_VEC_MAX], bv[LN_VEC_MAX];
#pragma unroll
    for (int i = 0; i < LN_VEC_MAX; ++i) {
      const int j = 4 * (lane + 64 * i), jc = min(j, d - 4);   // (columns past the row re-read its last four, unused)
      xv[i] = *(const float4 *)(xr + jc);
      gv[i] = *(const float4 *)(g + jc);
      bv[i] = *(const float4 *)(bt + jc);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < LN_VEC_MAX; ++i)
      if (4 * (lane + 64 * i) < d) s += (xv[i].x + xv[i].y) + (xv[i].z + xv[i].w);
    const float mean = wave_sum(s) / (float)d;
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < LN_VEC_MAX; ++i)
      if (4 * (lane + 64 * i) < d) {
        const float c0 = xv[i].x - mean, c1 = xv[i].y - mean, c2 = xv[i].z - mean, c3 = xv[i].w - mean;
        v += (c0 * c0 + c1 * c1) + (c2 * c2 + c3 * c3);
      }
    const float rstd = 1.f / sqrtf(wave_sum(v) / (float)d + 1e-5f);
#pragma unroll
    for (int i = 0; i < LN_VEC_MAX; ++i) {
      const int j = 4 * (lane + 64 * i);
      if (j >= d) continue;
      const float o0 = (xv[i].x - mean) * rstd * gv[i].x + bv[i].x, o1 = (xv[i].y - mean) * rstd * gv[i].y + bv[i].y;
      const float o2 = (xv[i].z - mean) * rstd * gv[i].z + bv[i].z, o3 = (xv[i].w - mean) * rstd * gv[i].w + bv[i].w;
      st4(y, (size_t)row * d + j, o0, o1, o2, o3);
    }
    return;
  }
  if (d <= 64 * LN_REG_MAX) {
    // the row in registers, read once (same summation order as below)
    float xv[LN_REG_MAX];
#pragma unroll
    for (int i = 0; i < LN_REG_MAX; ++i) xv[i] = lane + 64 * i < d ? xr[lane + 64 * i] : 0.f;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < LN_REG_MAX; ++i)
      if (lane + 64 * i < d) s += xv[i];
    const float mean = wave_sum(s) / (float)d;
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < LN_REG_MAX; ++i)
      if (lane + 64 * i < d) {
        const float c = xv[i] - mean;
        v += c * c;
      }
    const float rstd = 1.f / sqrtf(wave_sum(v) / (float)d + 1e-5f);
#pragma unroll
    for (int i = 0; i < LN_REG_MAX; ++i) {
      const int j = lane + 64 * i;
      if (j < d) st(y, (size_t)row * d + j, (xv[i] - mean) * rstd * g[j] + bt[j]);
    }
    return;
  }
  float s = 0.f;
  for (int j = lane; j < d; j += 64) s += xr[j];
  const float mean = wave_sum(s) / (float)d;
  float v = 0.f;
  for (int j = lane; j < d; j += 64) {
    const float c = xr[j] - mean;
    v += c * c;
  }
  const float var = wave_sum(v) / (float)d;
  const float rstd = 1.f / sqrtf(var + 1e-5f);
  for (int j = lane; j < d; j += 64) st(y, (size_t)row * d + j, (xr[j] - mean) * rstd * g[j] + bt[j]);
}

// ---------------------------------------------------------------------------
// GEMM epilogue
// ---------------------------------------------------------------------------

template <typename ACT>
__device__ __forceinline__ void epilogue(const Epi &e, int r, int n, float acc) {
  switch (e.mode) {
    case EPI_STORE:
      st((ACT *)e.out, (size_t)r * e.ldo + n, acc + (e.bias ? e.bias[n] : 0.f));
      break;
    case EPI_RESID:
      ((float *)e.out)[(size_t)r * e.ldo + n] += acc + e.bias[n];
      break;
    case EPI_RELU:
      st((ACT *)e.out, (size_t)r * e.ldo + n, fmaxf(acc + e.bias[n], 0.f));
      break;
    case EPI_QKV: {
      const float v = acc + e.bias[n];
      const int which = n / e.d, c = n - which * e.d;
      if (which == 0) {
        st((ACT *)e.q, (size_t)r * e.d + c, v);
      } else {
        const int b = r / e.P, p = r - b * e.P;
        const int h = c / e.dh, j = c - h * e.dh;
        const int pos = e.start[b] + e.start_off + p;
        if (pos < e.cap) {
          const size_t row0 = ((size_t)b * e.H + h) * e.cap;
          if (which == 1)
            st((ACT *)e.kc, (row0 + pos) * e.dh + j, v);
          else
            st((ACT *)e.vc, v_at<ACT>(row0, pos, j, e.dh), v);
        } else {
          atomicOr(e.status, TPPSD_STATUS_CAPACITY);
        }
      }
      break;
    }
    case EPI_HEAD:
      if (n < e.split)
        st((ACT *)e.out, (size_t)r * e.ldo + n, acc);
      else
        st((ACT *)e.out, (size_t)r * e.ldo + n, tanhf(acc + e.bias[n - e.split]));
      break;
    case EPI_F32:
      ((float *)e.out)[(size_t)r * e.ldo + n] = acc + (e.bias ? e.bias[n] : 0.f);
      break;
  }
}

// 8 consecutive columns n .. n + 7 of row r (n a multiple of 8, all < N;
// every destination row stride is a multiple of 8): the same arithmetic as
// epilogue(), with 16-byte loads and stores where the layout allows.
template <typename ACT> __device__ __forceinline__ void store8(ACT *p, const float v[8]);
template <> __device__ __forceinline__ void store8<float>(float *p, const float v[8]) {
  *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]);
  *(float4 *)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <> __device__ __forceinline__ void store8<bf16_t>(bf16_t *p, const float v[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = pk2bf(v[2 * i], v[2 * i + 1]);
  *(uint4 *)p = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void load8f(const float *p, float v[8]) {
  const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
// The operands of an 8-column epilogue that do not depend on the product
// (bias, the residual's row, the row's cache position), fetched apart so that
// a kernel can load them before its main loop.
struct Epi8In {
  float bv[8], xv[8];
  int pos;
};
__device__ __forceinline__ void epilogue8_fetch(const Epi &e, int r, int n, Epi8In &in) {
  switch (e.mode) {
    case EPI_STORE:
    case EPI_F32:
      if (e.bias) load8f(e.bias + n, in.bv);
      break;
    case EPI_RESID:
      load8f((const float *)e.out + (size_t)r * e.ldo + n, in.xv);
      load8f(e.bias + n, in.bv);
      break;
    case EPI_RELU:
      load8f(e.bias + n, in.bv);
      break;
    case EPI_QKV:
      load8f(e.bias + n, in.bv);
      if (n >= e.d) {
        const int b = r / e.P;
        in.pos = e.start[b] + e.start_off + (r - b * e.P);
      }
      break;
    case EPI_HEAD:
      if (n >= e.split) load8f(e.bias + (n - e.split), in.bv);
      break;
  }
}
template <typename ACT>
__device__ __forceinline__ void epilogue8(const Epi &e, int r, int n, const float acc[8], const Epi8In &in) {
  float v[8];
  switch (e.mode) {
    case EPI_STORE:
    case EPI_F32: {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = acc[i] + (e.bias ? in.bv[i] : 0.f);
      if (e.mode == EPI_F32) store8((float *)e.out + (size_t)r * e.ldo + n, v);
      else store8((ACT *)e.out + (size_t)r * e.ldo + n, v);
      break;
    }
    case EPI_RESID: {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = in.xv[i] + (acc[i] + in.bv[i]);
      store8((float *)e.out + (size_t)r * e.ldo + n, v);
      break;
    }
    case EPI_RELU: {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = fmaxf(acc[i] + in.bv[i], 0.f);
      store8((ACT *)e.out + (size_t)r * e.ldo + n, v);
      break;
    }
    case EPI_QKV: {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = acc[i] + in.bv[i];
      const int which = n / e.d, c = n - which * e.d;
      if (which == 0) {
        store8((ACT *)e.q + (size_t)r * e.d + c, v);
      } else {
        const int b = r / e.P;
        const int h = c / e.dh, j = c - h * e.dh;
        const int pos = in.pos;
        if (pos < e.cap) {
          const size_t row0 = ((size_t)b * e.H + h) * e.cap;
          if (which == 1) {
            store8((ACT *)e.kc + (row0 + pos) * e.dh + j, v);
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) st((ACT *)e.vc, v_at<ACT>(row0, pos, j + i, e.dh), v[i]);
          }
        } else {
          atomicOr(e.status, TPPSD_STATUS_CAPACITY);
        }
      }
      break;
    }
    case EPI_HEAD: {
      if (n < e.split) {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = acc[i];
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = tanhf(acc[i] + in.bv[i]);
      }
      store8((ACT *)e.out + (size_t)r * e.ldo + n, v);
      break;
    }
  }
}

// One k step of an MFMA tile product with fp32 accumulation: for every 16x16
// tile lane l holds row (l mod 16) of A and of W (W is stored [N, K], so its
// rows are B's columns) over one slice of the k range; the accumulator holds
// rows 4 (l / 16) + i, column l mod 16.
//   bf16: v_mfma_f32_16x16x32_bf16, lane slice = 8 consecutive k, 32 k per step.
//   fp32: v_mfma_f32_16x16x4f32, lane l loads 4 consecutive k (4 (l / 16) .. + 3)
//         and issues one MFMA per element; across the four MFMAs the 16 k of the
//         step are each used once, the same k for A and B (K must be a
//         multiple of 16).

template <typename ELT> struct MfmaStep;
template <> struct MfmaStep<bf16_t> {
  static constexpr int KSTEP = 32;
  typedef bf16x8_t frag;
  static __device__ __forceinline__ frag load(const bf16_t *p, int g) { return *(const bf16x8_t *)(p + 8 * g); }
  static __device__ __forceinline__ f32x4_t mma(frag a, frag b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct MfmaStep<float> {
  static constexpr int KSTEP = 16;
  typedef f32x4_t frag;
  static __device__ __forceinline__ frag load(const float *p, int g) { return *(const f32x4_t *)(p + 4 * g); }
  static __device__ __forceinline__ f32x4_t mma(frag a, frag b, f32x4_t c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
  }
};

// LDS-staged GEMM with fp32 accumulation: a workgroup of 4 waves (2 x 2)
// owns a BM x BN output tile and walks K in stages of BK = KSN MFMA k-steps
// (each stage costs a barrier and an LDS round trip, so tiles with few rows
// and a long K take long stages).
// The global loads of the next D stages are in flight in a register ring
// while the current stage is multiplied out of LDS (double-buffered, one
// barrier per stage). Rows of both LDS tiles are padded by one 16-byte vector
// so that the fragment reads (16 rows x 16 bytes per lane group) spread over
// the banks.
// LN: the A operand is LayerNorm(x) of the fp32 residual stream x [T, K]
// (biased variance, eps 1e-5), computed as it is staged so that the
// normalised activations never go to memory. All K of the tile's rows are in
// the register ring at once (K <= D * BK, checked by the launcher); each
// row's VPR vectors sit in VPR adjacent lanes, so its mean and then its
// variance (two passes over the registers) are lane-group reductions.
template <typename ELT> constexpr int gemm_bk() { return 2 * MfmaStep<ELT>::KSTEP; }
constexpr int GEMM_LN_MAX_DEPTH = 8;

template <typename ELT, int BM, int BN, bool LN, int D, int KSN>
__global__ __launch_bounds__(256) void k_gemm_lds(const ELT *__restrict__ X, const float *__restrict__ xf,
                                                  const float *__restrict__ lg, const float *__restrict__ lb,
                                                  const ELT *__restrict__ W, int T, int N, int K, Epi e) {
  typedef MfmaStep<ELT> S;
  constexpr int KS = S::KSTEP, BK = KSN * KS;
  constexpr int VE = 16 / sizeof(ELT);             // elements per 16-byte vector
  constexpr int LDR = BK + VE;                     // LDS row length (one vector of padding)
  constexpr int VPR = BK / VE;                     // vectors per tile row per stage
  constexpr int AV = BM * VPR / 256, BV = BN * VPR / 256;
  constexpr int XV = LN ? VE / 4 : 1;              // float4 of x per A vector
  constexpr int TM = BM / 32, TN = BN / 32;
  static_assert(AV >= 1 && BV >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) ELT As[2][BM][LDR];
  __shared__ __attribute__((aligned(16))) ELT Bs[2][BN][LDR];
  __shared__ __attribute__((aligned(16))) float gs[LN ? D * BK : 4], bs[LN ? D * BK : 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rr = lane & 15, g = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * (BN / 2);
  const int nst = (K + BK - 1) / BK;
  // register ring: stage s lives in slot s mod D
  uint4 ra[D][LN ? 1 : AV], rb[D][BV];
  float4 rx[D][LN ? AV * XV : 1];
  float mu[LN ? AV : 1], rs[LN ? AV : 1];
  // Loads are unconditional (rows and columns clamped into the matrices) so
  // that no branch separates them from their use: the compiler then waits
  // for each ring slot's own loads only, and the next stages stay in flight.
  // Columns past K are zeroed where the stage is stored to LDS.
  auto gload = [&](uint4 *pa, float4 *px, uint4 *pb, int k0) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + 256 * i, row = v / VPR, k = min(k0 + (v - row * VPR) * VE, K - VE);
      const size_t r = (size_t)min(m0 + row, T - 1);
      if (LN) {
#pragma unroll
        for (int c = 0; c < XV; ++c) px[i * XV + c] = *(const float4 *)(xf + r * K + k + 4 * c);
      } else {
        pa[i] = *(const uint4 *)(X + r * K + k);
      }
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int v = tid + 256 * i, row = v / VPR, k = min(k0 + (v - row * VPR) * VE, K - VE);
      const size_t r = (size_t)min(n0 + row, N - 1);
      pb[i] = *(const uint4 *)(W + r * K + k);
    }
  };
  auto lstore = [&](int buf, const uint4 *pa, const float4 *px, const uint4 *pb, int k0) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + 256 * i, row = v / VPR, kv = v - row * VPR;
      uint4 w;
      if (LN) {
        const int k = k0 + kv * VE;
        float y[VE];
#pragma unroll
        for (int c = 0; c < XV; ++c) {
          // K is a multiple of 4: a float4 of x is wholly inside or past K
          const int kk = k + 4 * c;
          const float4 xv = px[i * XV + c];
          if (kk < K) {
            const float4 gv = *(const float4 *)&gs[kk], bv = *(const float4 *)&bs[kk];
            y[4 * c + 0] = (xv.x - mu[i]) * rs[i] * gv.x + bv.x;
            y[4 * c + 1] = (xv.y - mu[i]) * rs[i] * gv.y + bv.y;
            y[4 * c + 2] = (xv.z - mu[i]) * rs[i] * gv.z + bv.z;
            y[4 * c + 3] = (xv.w - mu[i]) * rs[i] * gv.w + bv.w;
          } else {
            y[4 * c + 0] = y[4 * c + 1] = y[4 * c + 2] = y[4 * c + 3] = 0.f;
          }
        }
        if (sizeof(ELT) == 2) {
          uint32_t pk[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) pk[q] = pk2bf(y[2 * q], y[2 * q + 1]);
          w = make_uint4(pk[0], pk[1], pk[2], pk[3]);
        } else {
          w = make_uint4(__float_as_uint(y[0]), __float_as_uint(y[1]), __float_as_uint(y[2]), __float_as_uint(y[3]));
        }
      } else {
        w = (k0 + kv * VE < K) ? pa[i] : make_uint4(0u, 0u, 0u, 0u);
      }
      *(uint4 *)&As[buf][row][kv * VE] = w;
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int v = tid + 256 * i, row = v / VPR, kv = v - row * VPR;
      *(uint4 *)&Bs[buf][row][kv * VE] = (k0 + kv * VE < K) ? pb[i] : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  // the first D stages' loads go out before anything else
#pragma unroll
  for (int u = 0; u < D; ++u)
    if (u < nst) gload(ra[u], rx[u], rb[u], u * BK);
  // then, for tiles of one epilogue item per thread, the epilogue's operands
  // that do not depend on the product, so that the epilogue waits on no
  // memory (larger tiles fetch them in the epilogue: the registers would
  // cost occupancy)
  constexpr bool EPRE = BM * (BN / 8) <= 256;
  Epi8In ein;
  if (EPRE) {
    const int row = tid / (BN / 8), c8 = tid - row * (BN / 8);
    const int r = m0 + row, n = n0 + 8 * c8;
    if (tid < BM * (BN / 8) && r < T && n + 8 <= N) epilogue8_fetch(e, r, n, ein);
  }
  if (LN) {
    for (int k = tid; k < K; k += 256) {
      gs[k] = lg[k];
      bs[k] = lb[k];
    }
    // row statistics from the ring over the K real columns: mean, then the
    // sum of squared deviations
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int kv = (tid + 256 * i) % VPR;
      float sum = 0.f;
#pragma unroll
      for (int u = 0; u < D; ++u)
#pragma unroll
        for (int c = 0; c < XV; ++c) {
          const int k = u * BK + kv * VE + 4 * c;
          if (k < K) {
            const float4 xv = rx[u][i * XV + c];
            sum += (xv.x + xv.y) + (xv.z + xv.w);
          }
        }
#pragma unroll
      for (int off = 1; off < VPR; off <<= 1) sum += __shfl_xor(sum, off, 64);
      const float mean = sum / (float)K;
      float var = 0.f;
#pragma unroll
      for (int u = 0; u < D; ++u)
#pragma unroll
        for (int c = 0; c < XV; ++c) {
          const int k = u * BK + kv * VE + 4 * c;
          if (k < K) {
            const float4 xv = rx[u][i * XV + c];
            const float a = xv.x - mean, b = xv.y - mean, cc = xv.z - mean, dd = xv.w - mean;
            var += (a * a + b * b) + (cc * cc + dd * dd);
          }
        }
#pragma unroll
      for (int off = 1; off < VPR; off <<= 1) var += __shfl_xor(var, off, 64);
      mu[i] = mean;
      rs[i] = 1.f / sqrtf(var / (float)K + 1e-5f);
    }
    __syncthreads();
  }
  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nst; s0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      const int st_i = s0 + u;
      if (st_i < nst) {
        const int buf = st_i & 1;
        lstore(buf, ra[u], rx[u], rb[u], st_i * BK);
        __syncthreads();
        if (!LN && st_i + D < nst) gload(ra[u], rx[u], rb[u], (st_i + D) * BK);
#pragma unroll
        for (int ks = 0; ks < KSN; ++ks) {
          typename S::frag a[TM], b[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i)
            a[i] = *(const typename S::frag *)&As[buf][wm + 16 * i + rr][ks * KS + (KS / 4) * g];
#pragma unroll
          for (int j = 0; j < TN; ++j)
            b[j] = *(const typename S::frag *)&Bs[buf][wn + 16 * j + rr][ks * KS + (KS / 4) * g];
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = S::mma(a[i], b[j], acc[i][j]);
        }
      }
    }
  }
  // the tile goes through LDS (over the A stages, free after the last
  // barrier) so that each thread finishes 8 consecutive columns of a row with
  // 16-byte accesses
  constexpr int CLD = BN + 4;
  static_assert(sizeof(As) >= sizeof(float) * BM * CLD, "C tile must fit the A stages");
  float *Cs = (float *)&As[0][0][0];
  __syncthreads();   // every wave is done reading the last stage
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) Cs[(wm + 16 * i + 4 * g + v) * CLD + wn + 16 * j + rr] = acc[i][j][v];
  __syncthreads();
  for (int gi = tid; gi < BM * (BN / 8); gi += 256) {
    const int row = gi / (BN / 8), c8 = gi - row * (BN / 8);
    const int r = m0 + row, n = n0 + 8 * c8;
    if (r >= T || n >= N) continue;
    float cv[8];
    load8f(Cs + row * CLD + 8 * c8, cv);
    if (n + 8 <= N) {
      if (!EPRE) epilogue8_fetch(e, r, n, ein);
      epilogue8<ELT>(e, r, n, cv, ein);
    } else {
      for (int i = 0; i < N - n; ++i) epilogue<ELT>(e, r, n + i, cv[i]);
    }
  }
}

// ---------------------------------------------------------------------------
// Fused row-local part of a pre-LN THP layer (§4.2 encoder), bf16, over a
// tile of BM rows in one launch, between two attention launches:
//   PRE:  x += o Wo^T + bo                      (output projection, residual)
//         x += ReLU(LN2(x) W1^T + b1) W2^T + b2 (feed-forward block)
//   POST: q, k, v = LN1'(x) Wqkv'^T + b         (next layer, EPI_QKV epilogue)
// Nothing row-sized goes to HBM but o in, x out and q / k / v out: the FFN
// hidden activations are produced FC columns at a time into LDS and
// consumed at once by the second product, whose BM x D output accumulates
// in registers over the chunks; the fp32 x tile stays in LDS from the first
// residual to the last LayerNorm. Weights (small, L2-resident, read by every
// workgroup) go straight from global memory into MFMA operand registers.
// Rounding points are the layered kernels': LayerNorm outputs and hidden
// activations are bf16, products accumulate in fp32, residuals add
// x + (acc + bias). Waves split the columns (D / 4 or FC / 4 per wave) and
// each covers all BM rows; a row's LayerNorm statistics come from 16 lanes
// holding D / 16 consecutive values each. The barriers order LDS only, so
// weight loads stay in flight across them.
// ---------------------------------------------------------------------------
// Workgroup barrier that orders LDS only: global loads into registers and global
// stores stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// W [N][K] (bf16, N a multiple of 16, K of 32) into MFMA operand fragments:
// fragment (nt, ks) holds, for lane l = 16 g + r, W[16 nt + r][32 ks + 8 g ..
// + 7] at ((nt K/32 + ks) 64 + l) 8, so that a wave reads one fragment as 1 KB
// of contiguous memory
__global__ void k_pack_frags(const bf16_t *__restrict__ W, int N, int K, bf16_t *__restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;   // one 16-byte vector per thread
  const int KS = K / 32, total = (N / 16) * KS * 64;
  if (i >= total) return;
  const int l = i & 63, f = i >> 6, nt = f / KS, ks = f - nt * KS;
  *(uint4 *)(out + (size_t)i * 8) = *(const uint4 *)(W + (size_t)(16 * nt + (l & 15)) * K + 32 * ks + 8 * (l >> 4));
}

void launch_pack_frags(const void *W, int N, int K, void *out, hipStream_t s) {
  const int total = (N / 16) * (K / 32) * 64;
  k_pack_frags<<<(total + 255) / 256, 256, 0, s>>>((const bf16_t *)W, N, K, (bf16_t *)out);
}

template <int D, int F, int BM, int FC, bool PRE, bool POST>
__global__ __launch_bounds__(256) void k_layer_fused(LayerArgs a) {
  constexpr int XLD = D + 4, ALD = D + 8, HLD = FC + 8;   // row strides (pads spread LDS banks)
  constexpr int TM = BM / 16, TNA = FC / 64, TNB = D / 64;
  constexpr int KSD = D / 32, KSB = FC / 32, NCH = F / FC;
  constexpr int EPL = D / 16, NP = BM / 16;               // LayerNorm: values per lane, row passes
  static_assert(TNA >= 1 && TNB >= 1 && F % FC == 0 && BM % 16 == 0 && EPL % 4 == 0, "shape");
  static_assert(!POST || (3 * D) % 128 == 0, "q, k, v in chunks of 128 columns");
  __shared__ __attribute__((aligned(16))) float xs[BM * XLD];
  __shared__ __attribute__((aligned(16))) bf16_t as[BM * ALD];
  __shared__ __attribute__((aligned(16))) bf16_t hs[BM * HLD];
  __shared__ float b1s[F], b2s[D];   // (b1s holds the q, k, v bias once the FFN is done)
  __shared__ int rpos[POST ? BM : 1];    // POST: cache position of each row's event
  static_assert(!POST || F >= 3 * D, "q, k, v bias fits the FFN bias array");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rr = lane & 15, g = lane >> 4;
  const int T = a.T, m0 = blockIdx.x * BM;
  if (POST && tid < BM) {   // read now, used at the very end
    const int r = min(m0 + tid, T - 1), bq = r / a.qe.P;
    rpos[tid] = a.qe.start[bq] + a.qe.start_off + (r - bq * a.qe.P);
  }
  const bf16_t *W1 = a.w1, *W2 = a.w2;
  // weights are pre-packed in MFMA fragment order (k_pack_frags): fragment
  // (16-row tile nt, 32-column step ks) of a matrix with KS steps per row is
  // 64 lanes x 16 bytes, contiguous
  auto frag = [&](const bf16_t *Wp, int nt, int KS, int ks) {
    return *(const bf16x8_t *)(Wp + ((size_t)(nt * KS + ks) * 64 + lane) * 8);
  };
  // first FFN product's weights of chunk c: wave's hidden columns c FC + wave FC/4 + 16 j + rr
  bf16x8_t w1f[2][TNA][KSD];
  auto load_w1 = [&](int c, bf16x8_t (&dst)[TNA][KSD]) {
#pragma unroll
    for (int j = 0; j < TNA; ++j)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
        dst[j][ks] = frag(W1, c * (FC / 16) + wave * (FC / 64) + j, KSD, ks);
  };
  // LayerNorm of the xs rows into as (bf16): wave w normalises rows
  // w BM/4 + 4 p + g, 16 lanes per row; v holds the rows' values
  auto layernorm = [&](const float4 (&v)[NP][EPL / 4], const float *lg, const float *lb) {
    float4 gv[EPL / 4], bv[EPL / 4];
#pragma unroll
    for (int c = 0; c < EPL / 4; ++c) {
      gv[c] = *(const float4 *)(lg + rr * EPL + 4 * c);
      bv[c] = *(const float4 *)(lb + rr * EPL + 4 * c);
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int row = wave * (BM / 4) + 4 * p + g;
      float sum = 0.f;
#pragma unroll
      for (int c = 0; c < EPL / 4; ++c) sum += (v[p][c].x + v[p][c].y) + (v[p][c].z + v[p][c].w);
      const float mean = group_sum(sum, 16) / (float)D;
      float var = 0.f;
#pragma unroll
      for (int c = 0; c < EPL / 4; ++c) {
        const float a0 = v[p][c].x - mean, a1 = v[p][c].y - mean, a2 = v[p][c].z - mean, a3 = v[p][c].w - mean;
        var += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
      }
      const float rs = 1.f / sqrtf(group_sum(var, 16) / (float)D + 1e-5f);
#pragma unroll
      for (int c = 0; c < EPL / 4; ++c) {
        const float y0 = (v[p][c].x - mean) * rs * gv[c].x + bv[c].x;
        const float y1 = (v[p][c].y - mean) * rs * gv[c].y + bv[c].y;
        const float y2 = (v[p][c].z - mean) * rs * gv[c].z + bv[c].z;
        const float y3 = (v[p][c].w - mean) * rs * gv[c].w + bv[c].w;
        uint2 pk;
        pk.x = pk2bf(y0, y1);
        pk.y = pk2bf(y2, y3);
        *(uint2 *)&as[row * ALD + rr * EPL + 4 * c] = pk;
      }
    }
  };
  auto read_rows = [&](float4 (&v)[NP][EPL / 4]) {   // this lane's LayerNorm share of the xs rows
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int c = 0; c < EPL / 4; ++c)
        v[p][c] = *(const float4 *)&xs[(wave * (BM / 4) + 4 * p + g) * XLD + rr * EPL + 4 * c];
  };
  // D-wide product of the as rows with the D x D matrix W, computed
  // transposed (W rows as the MFMA's first operand) so that lane (rr, g)
  // holds row 16 i + rr, columns wave D/4 + 16 j + 4 g .. + 3 in acc[i][j]
  auto prod_dd = [&](const bf16_t *W, f32x4_t (&acc)[TM][TNB]) {
    bf16x8_t wf[TNB][KSD];
#pragma unroll
    for (int j = 0; j < TNB; ++j)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
        wf[j][ks] = frag(W, wave * (D / 64) + j, KSD, ks);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNB; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bf16x8_t af = *(const bf16x8_t *)&as[(16 * i + rr) * ALD + 32 * ks + 8 * g];
#pragma unroll
        for (int j = 0; j < TNB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j][ks], af, acc[i][j], 0, 0, 0);
      }
  };
  // xs[row][col .. col + 3] += acc + bias[col ..]: one float4 per lane
  auto resid4 = [&](int row, int col, const f32x4_t &acc, const float *bias) {
    float4 *xp = (float4 *)&xs[row * XLD + col];
    float4 xv4 = *xp;
    xv4.x = xv4.x + (acc[0] + bias[col]);
    xv4.y = xv4.y + (acc[1] + bias[col + 1]);
    xv4.z = xv4.z + (acc[2] + bias[col + 2]);
    xv4.w = xv4.w + (acc[3] + bias[col + 3]);
    *xp = xv4;
  };

  // x rows (and o rows) in
  float4 xv[NP][EPL / 4];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int row = wave * (BM / 4) + 4 * p + g;
    const size_t r = (size_t)min(m0 + row, T - 1);
#pragma unroll
    for (int c = 0; c < EPL / 4; ++c) xv[p][c] = *(const float4 *)(a.x + r * D + rr * EPL + 4 * c);
  }
  if (PRE) {
    constexpr int VR = D / 8;   // 16-byte vectors per o row
    for (int i = tid; i < BM * VR; i += 256) {
      const int row = i / VR, c = i - row * VR;
      *(uint4 *)&as[row * ALD + 8 * c] = *(const uint4 *)(a.o + (size_t)min(m0 + row, T - 1) * D + 8 * c);
    }
  }
  for (int i = tid; i < F; i += 256) b1s[i] = a.b1[i];
  for (int i = tid; i < D; i += 256) b2s[i] = a.b2[i];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int c = 0; c < EPL / 4; ++c) *(float4 *)&xs[(wave * (BM / 4) + 4 * p + g) * XLD + rr * EPL + 4 * c] = xv[p][c];
  load_w1(0, w1f[0]);
  lds_barrier();
  if (PRE) {
    // output projection and residual into the xs tile
    f32x4_t acc[TM][TNB];
    prod_dd(a.wo, acc);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNB; ++j) resid4(16 * i + rr, wave * (D / 4) + 16 * j + 4 * g, acc[i][j], a.bo);
    lds_barrier();   // xs complete, o operand reads done
    read_rows(xv);
  }
  layernorm(xv, a.ln2_g, a.ln2_b);
  lds_barrier();
  f32x4_t acc_o[TM][TNB];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TNB; ++j) acc_o[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (c + 1 < NCH) load_w1(c + 1, w1f[(c + 1) & 1]);
    // second product's weights of chunk c: wave's output columns wave D/4 + 16 j + rr
    bf16x8_t w2f[TNB][KSB];
#pragma unroll
    for (int j = 0; j < TNB; ++j)
#pragma unroll
      for (int ks = 0; ks < KSB; ++ks)
        w2f[j][ks] = frag(W2, wave * (D / 64) + j, F / 32, c * (FC / 32) + ks);
    // hidden chunk: ReLU(A W1_c^T + b1) -> bf16 -> LDS
    f32x4_t acc_h[TM][TNA];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNA; ++j) acc_h[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bf16x8_t af = *(const bf16x8_t *)&as[(16 * i + rr) * ALD + 32 * ks + 8 * g];
#pragma unroll
        for (int j = 0; j < TNA; ++j)
          acc_h[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1f[c & 1][j][ks], af, acc_h[i][j], 0, 0, 0);
      }
    // (transposed product: lane (rr, g) holds row 16 i + rr, hidden columns
    // wave FC/4 + 16 j + 4 g .. + 3, written as one 8-byte word)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNA; ++j) {
        const int col = wave * (FC / 4) + 16 * j + 4 * g;
        const float *bb = b1s + c * FC + col;
        uint2 pk;
        pk.x = pk2bf(fmaxf(acc_h[i][j][0] + bb[0], 0.f), fmaxf(acc_h[i][j][1] + bb[1], 0.f));
        pk.y = pk2bf(fmaxf(acc_h[i][j][2] + bb[2], 0.f), fmaxf(acc_h[i][j][3] + bb[3], 0.f));
        *(uint2 *)&hs[(16 * i + rr) * HLD + col] = pk;
      }
    lds_barrier();
#pragma unroll
    for (int ks = 0; ks < KSB; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bf16x8_t hf = *(const bf16x8_t *)&hs[(16 * i + rr) * HLD + 32 * ks + 8 * g];
#pragma unroll
        for (int j = 0; j < TNB; ++j)
          acc_o[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w2f[j][ks], hf, acc_o[i][j], 0, 0, 0);
      }
    lds_barrier();   // the chunk's hidden tile is read before the next overwrites it
  }
  constexpr int QC = 128, TNQ = QC / 64, SLD = QC + 4, NQC = POST ? 3 * D / QC : 1;
  bf16x8_t wq[2][TNQ][KSD];
  auto load_wq = [&](int c, bf16x8_t (&dst)[TNQ][KSD]) {
#pragma unroll
    for (int j = 0; j < TNQ; ++j)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
        dst[j][ks] = frag(a.wqkv, c * (QC / 16) + wave * (QC / 64) + j, KSD, ks);
  };
  if (POST) {
    load_wq(0, wq[0]);
    for (int i = tid; i < 3 * D; i += 256) b1s[i] = a.qe.bias[i];
  }
  // second residual in the LDS tile, then 16-byte stores of whole rows
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TNB; ++j) resid4(16 * i + rr, wave * (D / 4) + 16 * j + 4 * g, acc_o[i][j], b2s);
  lds_barrier();
  for (int idx = tid; idx < BM * (D / 4); idx += 256) {
    const int row = idx / (D / 4), c4 = idx - row * (D / 4);
    if (m0 + row < T) *(float4 *)(a.x + (size_t)(m0 + row) * D + 4 * c4) = *(const float4 *)&xs[row * XLD + 4 * c4];
  }
  if (!POST) return;
  // the next layer's LayerNorm and q, k, v, 128 columns at a time (the next
  // chunk's weights loading during the current one); each chunk's tile is
  // staged in xs (free once normalised) and stored with lanes running over
  // rows, so that the value cache's 2-byte stores of consecutive positions
  // (one 16-byte block holds 8 positions of a column) are adjacent
  read_rows(xv);
  layernorm(xv, a.ln1_g, a.ln1_b);
  lds_barrier();
  static_assert(SLD <= XLD, "q, k, v staging fits the x tile");
  const Epi &e = a.qe;
#pragma unroll
  for (int c = 0; c < NQC; ++c) {
    if (c + 1 < NQC) load_wq(c + 1, wq[(c + 1) & 1]);
    f32x4_t acc[TM][TNQ];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNQ; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const bf16x8_t af = *(const bf16x8_t *)&as[(16 * i + rr) * ALD + 32 * ks + 8 * g];
#pragma unroll
        for (int j = 0; j < TNQ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wq[c & 1][j][ks], af, acc[i][j], 0, 0, 0);
      }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TNQ; ++j)
        *(f32x4_t *)&xs[(16 * i + rr) * SLD + wave * (QC / 4) + 16 * j + 4 * g] = acc[i][j];
    lds_barrier();
    for (int gi = tid; gi < BM * (QC / 8); gi += 256) {
      const int row = gi % BM, c8 = gi / BM, r = m0 + row;
      if (r >= T) continue;
      const int n = c * QC + 8 * c8, which = n / D, cc = n - which * D;
      float v[8];
      load8f(xs + row * SLD + 8 * c8, v);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] += b1s[n + i];
      if (which == 0) {
        store8((bf16_t *)e.q + (size_t)r * D + cc, v);
      } else {
        const int bq = r / e.P, h = cc / e.dh, j = cc - h * e.dh, pos = rpos[row];
        if (pos < e.cap) {
          const size_t row0 = ((size_t)bq * e.H + h) * e.cap;
          if (which == 1) {
            store8((bf16_t *)e.kc + (row0 + pos) * e.dh + j, v);
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) st((bf16_t *)e.vc, v_at<bf16_t>(row0, pos, j + i, e.dh), v[i]);
          }
        } else {
          atomicOr(e.status, TPPSD_STATUS_CAPACITY);
        }
      }
    }
    lds_barrier();   // staging read before the next chunk writes it
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMM with operands moved straight from global memory into LDS
// (global_load_lds, 16 bytes per lane) through an S-stage ring. No register
// holds an operand in flight, so the loads of the next S - 1 stages overlap
// the MFMAs of the current one, and each wave waits for its own loads by
// count (s_waitcnt vmcnt). Tiles are stored unpadded with their 16-byte
// chunks XOR-swizzled by row (chunk c of row r at c ^ (r mod chunks per
// row)), so that the rows one MFMA fragment reads fall on different banks.
// Needs K to be a multiple of the stage depth BK = 32 KSN.
// ---------------------------------------------------------------------------

// waits until at most CNT vector-memory operations of this wave are outstanding
template <int CNT> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(CNT >= 0 && CNT < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((CNT & 15) | ((CNT >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef __attribute__((address_space(3))) void *lds_ptr_t;

// One LDS array per ring slot, addressed with compile-time slot numbers (the
// stage loop is unrolled by S) inside one inlined function that takes the
// slots as restrict pointers: the compiler then knows that reads of one slot
// never alias the loads still landing in the others and does not wait for
// them. The waits are explicit and per wave.
template <int BM, int BN, int KSN> struct DlTile {
  static constexpr int BK = 32 * KSN, CPR = BK / 8;     // 16-byte chunks per tile row
  static constexpr int ACH = BM * CPR, BCH = BN * CPR;  // chunks per stage
  static constexpr int NIA = ACH / 256, NIB = BCH / 256;
  static constexpr int NI = NIA + NIB;                   // DMA instructions per thread per stage
  static constexpr int STAGE = (ACH + BCH) * 16;         // bytes
  static_assert(NIA >= 1 && NIB >= 1 && ACH % 256 == 0 && BCH % 256 == 0, "tile too small for 256 threads");
};

template <int BM, int BN, int KSN, int S>
__device__ __forceinline__ void dl_mainloop(char *__restrict__ s0, char *__restrict__ s1, char *__restrict__ s2,
                                            char *__restrict__ s3, const bf16_t *const *srcA,
                                            const bf16_t *const *srcB, int nst, f32x4_t (*acc)[BN / 32]) {
  typedef DlTile<BM, BN, KSN> G;
  constexpr int CPR = G::CPR, ACH = G::ACH, NIA = G::NIA, NIB = G::NIB, NI = G::NI, BK = G::BK;
  constexpr int TM = BM / 32, TN = BN / 32;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rr = lane & 15, g = lane >> 4;
  const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * (BN / 2);
  char *const slots[4] = {s0, s1, s2, s3};
  auto issue = [&](char *base, int st) {
    const int k0 = st * BK;
#pragma unroll
    for (int i = 0; i < NIA; ++i)
      __builtin_amdgcn_global_load_lds((const void *)(srcA[i] + k0), (lds_ptr_t)(base + (4 * i + wave) * 1024), 16, 0,
                                       0);
#pragma unroll
    for (int i = 0; i < NIB; ++i)
      __builtin_amdgcn_global_load_lds((const void *)(srcB[i] + k0),
                                       (lds_ptr_t)(base + ACH * 16 + (4 * i + wave) * 1024), 16, 0, 0);
  };
#pragma unroll
  for (int u = 0; u < S - 1; ++u)
    if (u < nst) issue(slots[u], u);
  for (int s0i = 0; s0i < nst; s0i += S) {
#pragma unroll
    for (int u = 0; u < S; ++u) {
      const int st = s0i + u;
      if (st < nst) {
        // stage st has landed once only the stages issued after it are pending
        if (st + S - 2 < nst) wait_vmcnt<(S - 2) * NI>();
        else wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();   // all of stage st is in LDS; stage st - 1's slot is free
        if (st + S - 1 < nst) issue(slots[(u + S - 1) % S], st + S - 1);
        const char *As = slots[u], *Bs = As + ACH * 16;
#pragma unroll
        for (int ks = 0; ks < KSN; ++ks) {
          bf16x8_t a[TM], b[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int row = wm + 16 * i + rr;
            a[i] = *(const bf16x8_t *)(As + (row * CPR + ((4 * ks + g) ^ (row % CPR))) * 16);
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int row = wn + 16 * j + rr;
            b[j] = *(const bf16x8_t *)(Bs + (row * CPR + ((4 * ks + g) ^ (row % CPR))) * 16);
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
      }
    }
  }
}

template <int BM, int BN, int KSN, int S>
__global__ __launch_bounds__(256) void k_gemm_dl(const bf16_t *__restrict__ X, const bf16_t *__restrict__ W, int T,
                                                 int N, int K, Epi e) {
  typedef DlTile<BM, BN, KSN> G;
  constexpr int CPR = G::CPR, NIA = G::NIA, NIB = G::NIB, STAGE = G::STAGE, BK = G::BK;
  constexpr int TM = BM / 32, TN = BN / 32, CLD = BN + 4;
  static_assert(S >= 2 && S <= 4, "ring of 2 to 4 stages");
  __shared__ __attribute__((aligned(1024))) char st0[STAGE];
  __shared__ __attribute__((aligned(1024))) char st1[STAGE];
  __shared__ __attribute__((aligned(1024))) char st2[S > 2 ? STAGE : 1024];
  __shared__ __attribute__((aligned(1024))) char st3[S > 3 ? STAGE : 1024];
  __shared__ __attribute__((aligned(16))) float Cs[BM * CLD];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rr = lane & 15, g = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * (BN / 2);
  // DMA instruction i of this thread moves chunk p = (4 i + wave) 64 + lane of
  // the stage's A (then B) tile: row p / CPR, stored chunk p mod CPR, which
  // holds logical chunk (p mod CPR) ^ (row mod CPR). Rows past T or N are
  // clamped (their results are never stored).
  const bf16_t *srcA[NIA];
  const bf16_t *srcB[NIB];
#pragma unroll
  for (int i = 0; i < NIA; ++i) {
    const int p = (4 * i + wave) * 64 + lane, row = p / CPR, c = (p % CPR) ^ (row % CPR);
    srcA[i] = X + (size_t)min(m0 + row, T - 1) * K + 8 * c;
  }
#pragma unroll
  for (int i = 0; i < NIB; ++i) {
    const int p = (4 * i + wave) * 64 + lane, row = p / CPR, c = (p % CPR) ^ (row % CPR);
    srcB[i] = W + (size_t)min(n0 + row, N - 1) * K + 8 * c;
  }
  // the epilogue's operands that do not depend on the product, loaded
  // before the main loop (older than its loads, so its counted waits still
  // hold), so that the epilogue waits on no memory
  constexpr int NEP = (BM * (BN / 8) + 255) / 256;
  Epi8In ein[NEP];
#pragma unroll
  for (int k = 0; k < NEP; ++k) {
    const int gi = tid + 256 * k, row = gi / (BN / 8), c8 = gi - row * (BN / 8);
    const int r = m0 + row, n = n0 + 8 * c8;
    if (gi < BM * (BN / 8) && r < T && n + 8 <= N) epilogue8_fetch(e, r, n, ein[k]);
  }
  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  dl_mainloop<BM, BN, KSN, S>(st0, st1, st2, st3, srcA, srcB, K / BK, acc);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) Cs[(wm + 16 * i + 4 * g + v) * CLD + wn + 16 * j + rr] = acc[i][j][v];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < NEP; ++k) {
    const int gi = tid + 256 * k, row = gi / (BN / 8), c8 = gi - row * (BN / 8);
    const int r = m0 + row, n = n0 + 8 * c8;
    if (gi >= BM * (BN / 8) || r >= T || n >= N) continue;
    float cv[8];
    load8f(Cs + row * CLD + 8 * c8, cv);
    if (n + 8 <= N) {
      epilogue8<bf16_t>(e, r, n, cv, ein[k]);
    } else {
      for (int i = 0; i < N - n; ++i) epilogue<bf16_t>(e, r, n + i, cv[i]);
    }
  }
}

// ---------------------------------------------------------------------------
// decoder (§4.2): the mixture parameters (V_w e1, V_mu e2, V_sigma e3) and
// the type logits (V_k2 tanh(V_k1 h + b1)) of a row are one product of the
// concatenated [e1 e2 e3 tanh(.)] (4d wide) with a block-diagonal
// (3M + K) x 4d matrix built once per state from the model's heads; the
// kernel below then takes the log-softmaxes and runs the verify / draft / AR
// epilogue, one wave per row.
// ---------------------------------------------------------------------------

template <typename W>
__global__ void k_build_head(const W *__restrict__ mix_w, const W *__restrict__ k2_w,
                             const float *__restrict__ mix_b, const float *__restrict__ k2_b, int d, int M,
                             int K, W *__restrict__ hw, float *__restrict__ hb) {
  const int o = blockIdx.x;   // output row, < 3M + K
  const int grp = o < 3 * M ? o / M : 3;
  const W *src = o < 3 * M ? mix_w + (size_t)o * d : k2_w + (size_t)(o - 3 * M) * d;
  for (int c = threadIdx.x; c < 4 * d; c += blockDim.x) {
    const int k = c - grp * d;
    hw[(size_t)o * 4 * d + c] = (k >= 0 && k < d) ? src[k] : (W)0;
  }
  if (threadIdx.x == 0) hb[o] = o < 3 * M ? mix_b[o] : k2_b[o - 3 * M];
}

// The decoder epilogue of one row (sequence b, block position p) whose
// logits are lr[0 .. 3M + K), run by one whole wave.
__device__ void head_row(const float *lr, int M, int K, const HeadArgs &a, int b, int p) {
  const int lane = threadIdx.x & 63;
  // lane m: mixture logit, mean and log-scale of component m; type logit m
  const float lw = lane < M ? lr[lane] : -INFINITY;
  const float mu = lane < M ? lr[M + lane] : 0.f;
  const float sg = lane < M ? lr[2 * M + lane] : 0.f;
  const float lk = lane < K ? lr[3 * M + lane] : -INFINITY;
  const float mw = wave_max(lw);
  const float logw = lw - mw - logf(wave_sum(lane < M ? expf(lw - mw) : 0.f));
  const float mk = wave_max(lk);
  const float logk = lk - mk - logf(wave_sum(lane < K ? expf(lk - mk) : 0.f));
  const size_t drow = (size_t)b * a.dst_stride + a.dst_row0 + (p - a.p0);
  float *mixr = a.mix + drow * 3 * M;
  float *ltr = a.logtype + drow * K;
  if (lane < M) {
    mixr[lane] = logw;
    mixr[M + lane] = mu;
    mixr[2 * M + lane] = sg;
  }
  if (lane < K) ltr[lane] = logk;
  const bool active = a.done == nullptr || a.done[b] == 0;
  const bool bad = (lane < M && !(isfinite(logw) && isfinite(mu) && isfinite(sg))) || (lane < K && !isfinite(logk));
  if (__ballot(bad) != 0ull && active && lane == 0) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
  // component m's log-density term at tau, for the wave-parallel mixture sum
  auto logpdf = [&](float tau) {
    const float lt = logf(tau);
    float c = -INFINITY;
    if (lane < M) {
      const float z = lt - mu;
      c = logw - sg - 0.918938533204672742f - lt - 0.5f * z * z * expf(-2.f * sg);
    }
    const float mx = wave_max(c);
    return mx + logf(wave_sum(lane < M ? expf(c - mx) : 0.f));
  };
  // categorical over the lanes' log-probabilities (scan of exp, first index
  // whose running sum exceeds u times the total)
  auto sample = [&](float lp, int n, float u) {
    float c = lane < n ? expf(lp) : 0.f;
    c = wave_cumsum(c);
    const float tot = lane_val(c, n - 1);
    const unsigned long long hit = __ballot(lane < n && u * tot < c);
    return hit ? (int)__builtin_ctzll(hit) : n - 1;
  };
  auto draw_tau = [&](const float u[4]) {
    const int z = sample(logw, M, u[0]);
    const float eps = sqrtf(-2.f * logf(u[1])) * cosf(6.28318530717958647692f * u[2]);
    const float muz = lane_val(mu, z), sz = lane_val(sg, z);
    return expf(muz + expf(sz) * eps);
  };
  if (a.mode == HEAD_VERIFY) {
    if (p < a.gamma) {
      const size_t di = (size_t)b * a.dr_stride + p;
      const float lg = logpdf(a.dr_tau[di]);
      const int kk = min(max(a.dr_k[di], 0), K - 1);
      const float lf = lane_val(logk, kk);
      if (lane == 0) {
        a.v_logg[di] = lg;
        a.v_logf[di] = lf;
        if (!isfinite(lg) && active) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
      }
    }
  } else if (a.mode == HEAD_DRAFT) {
    float u[4];
    philox_uniforms(a.seed, (uint64_t)b, (uint64_t)a.rnd[b], (uint64_t)a.l_index, TAG_DRAFT, u);
    const float tau = draw_tau(u);
    const int kk = sample(logk, K, u[3]);
    const float lg = logpdf(tau);
    const float lf = lane_val(logk, kk);
    if (lane == 0) {
      const size_t di = (size_t)b * a.dr_stride + a.slot;
      const float tprev = (a.slot == 0) ? a.ev_t[(size_t)b * a.ev_stride + a.n[b] - 1] : a.d_t[di - 1];
      a.d_tau[di] = tau;
      a.d_t[di] = tprev + tau;
      a.d_k[di] = kk;
      a.d_logg[di] = lg;
      a.d_logf[di] = lf;
      if (!isfinite(tau) && active) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
    }
  } else {  // HEAD_AR
    if (!active) return;
    float u[4];
    const int g = a.gen[b];
    philox_uniforms(a.seed, (uint64_t)b, (uint64_t)g, 0ull, TAG_AR, u);
    const float tau = draw_tau(u);
    const int kk = sample(logk, K, u[3]);
    const int n = a.n[b];
    const float tlast = a.ev_t[(size_t)b * a.ev_stride + n - 1];
    const float tn = tlast + tau;
    const float T_end = a.t_end[b];
    // Eq. (2): log-density of the committed event, or, for an event past the
    // end time (dropped; the sequence ends), the survival log(1 - G(T - t_N))
    const bool past = tn > T_end;
    const float lterm = past ? wave_log_survival(logw, mu, sg, lane < M, T_end - tlast)
                             : logpdf(tau) + lane_val(logk, kk);
    if (lane != 0) return;
    a.ll[b] += (double)lterm;
    if (past) {
      a.done[b] = 1;
      atomicAdd(a.n_done, 1);
      return;
    }
    if (n >= a.ev_stride) {
      atomicOr(a.status, TPPSD_STATUS_CAPACITY);
      return;
    }
    a.ev_t[(size_t)b * a.ev_stride + n] = tn;
    a.ev_k[(size_t)b * a.ev_stride + n] = kk;
    const int col = g - a.gen0[b];
    if (col >= 0 && col < a.ar_out_stride) {
      if (a.ar_t_out) a.ar_t_out[(size_t)b * a.ar_out_stride + col] = tn;
      if (a.ar_k_out) a.ar_k_out[(size_t)b * a.ar_out_stride + col] = kk;
    }
    a.n[b] = n + 1;
    a.gen[b] = g + 1;
    a.lenT[b] = n;
    if (!isfinite(tau)) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
    if (g + 1 >= a.n_gen || tn >= T_end) {
      a.done[b] = 1;
      atomicAdd(a.n_done, 1);
    }
  }
}

__global__ __launch_bounds__(256) void k_head(const float *__restrict__ logits, int ldl, int M, int K,
                                              HeadArgs a) {
  const int w = threadIdx.x >> 6;
  const int rows_per_seq = a.P - a.p0;
  const int ridx = blockIdx.x * 4 + w;
  if (ridx >= a.B * rows_per_seq) return;   // whole waves; no barriers below
  const int b = ridx / rows_per_seq;
  const int p = a.p0 + (ridx - b * rows_per_seq);
  head_row(logits + ((size_t)b * a.P + p) * ldl, M, K, a, b, p);
}

// ---------------------------------------------------------------------------
// fused drafting (§4.3 "Drafting", Algorithm 1's inner loop): one workgroup
// per sequence runs all gamma sequential draft steps -- embedding, every
// layer, decoder and the draw -- in one launch. The draft model is small, so
// each step is a handful of matrix-vector products on at most two tokens
// (step 1 re-encodes the last two committed events). Activations live in
// LDS; keys/values go to the draft KV cache exactly as in the layered path,
// with the same bf16 rounding points.
// ---------------------------------------------------------------------------

template <typename ELT> __device__ __forceinline__ float rnd_act(float v);
template <> __device__ __forceinline__ float rnd_act<float>(float v) { return v; }
template <> __device__ __forceinline__ float rnd_act<bf16_t>(float v) { return bf2f(f2bf(v)); }

template <typename ELT> __device__ __forceinline__ void load8(const ELT *p, float w[8]);
template <> __device__ __forceinline__ void load8<float>(const float *p, float w[8]) {
  const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
  w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w; w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
}
template <> __device__ __forceinline__ void load8<bf16_t>(const bf16_t *p, float w[8]) {
  const uint4 u = *(const uint4 *)p;
  const uint32_t v[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    w[2 * i] = __uint_as_float(v[i] << 16);
    w[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
  }
}

// y[p][n] = sum_k W(n)[k] X(n, p)[k] for n < N, p < P (P <= 2), handed to
// epi(p, n, y) by one lane. bf16: the inputs X are bf16 rows too, and each
// 8-element chunk is four v_dot2c over the raw pairs. K is cut into 8-element chunks; a row's chunks
// are shared by LPR adjacent lanes (a power of two), CPL = K / (8 LPR) <= 8
// chunks each, loaded together before any is used, so a product costs about
// one memory latency plus a few lane-group additions. wrow(n) gives row n of
// W, xrow(n, p) the input that row n reads.
template <typename ELT, int CPL, typename WF, typename XF, typename EPI>
__device__ void wg_gemv_cpl(int N, int K, int P, WF wrow, XF xrow, EPI epi) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int lpr = (K >> 3) / CPL, rows = nt / lpr;
  const int sub = tid % lpr;
  for (int r0 = 0; r0 < N; r0 += rows) {
    const int n = r0 + tid / lpr, nn = min(n, N - 1);
    const ELT *wr = wrow(nn);
    float acc[2] = {0.f, 0.f};
    if constexpr (sizeof(ELT) == 2) {
      uint4 w[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) w[c] = *(const uint4 *)(wr + 8 * (sub + lpr * c));
      for (int p = 0; p < P; ++p) {
        const bf16_t *x = xrow(nn, p);
        float a = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const uint4 xv = *(const uint4 *)(x + 8 * (sub + lpr * c));
          a = dot2_bf(w[c].x, xv.x, a);
          a = dot2_bf(w[c].y, xv.y, a);
          a = dot2_bf(w[c].z, xv.z, a);
          a = dot2_bf(w[c].w, xv.w, a);
        }
        acc[p] = group_sum(a, lpr);
      }
    } else {
      float w[CPL][8];
#pragma unroll
      for (int c = 0; c < CPL; ++c) load8(wr + 8 * (sub + lpr * c), w[c]);
      for (int p = 0; p < P; ++p) {
        const float *x = xrow(nn, p);
        float a = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const float *xc = x + 8 * (sub + lpr * c);
#pragma unroll
          for (int e = 0; e < 8; ++e) a += w[c][e] * xc[e];
        }
        acc[p] = group_sum(a, lpr);
      }
    }
    if (n < N && sub == 0)
      for (int p = 0; p < P; ++p) epi(p, n, acc[p]);
  }
}
// chunks per lane for a K-wide product (K / 8 a power of two)
constexpr int gemv_cpl(int K) { return (K >> 3) < 8 ? (K >> 3) : 8; }

// LayerNorm of P <= 4 rows of x (stride d) into y (stride d), wave p per row
template <typename ELT, typename YT>
__device__ void wg_layernorm(const float *x, YT *y, const float *g, const float *bt, int P, int d) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (wave >= P) return;
  const float *xr = x + wave * d;
  float s = 0.f;
  for (int j = lane; j < d; j += 64) s += xr[j];
  const float mean = wave_sum(s) / (float)d;
  float v = 0.f;
  for (int j = lane; j < d; j += 64) {
    const float c = xr[j] - mean;
    v += c * c;
  }
  const float rstd = 1.f / sqrtf(wave_sum(v) / (float)d + 1e-5f);
  for (int j = lane; j < d; j += 64) st<YT>(y, wave * d + j, rnd_act<ELT>((xr[j] - mean) * rstd * g[j] + bt[j]));
}

// One 32-key step of the draft attention's MFMA formulation (d_head = 16),
// the fragments of lane (rr, g): the permuted key rows krow0 / krow1 of S^T
// and the values of keys kt + 8 g .. + 7 in value column rr. Loads are
// unconditional (positions clamped into the slab) and positions at or past
// n_keys are zeroed afterwards.
template <typename ELT> struct DraftStep;
template <> struct DraftStep<bf16_t> {
  short4_t k0, k1;
  uint4 v;
  __device__ void load(const bf16_t *kc, const bf16_t *vc, size_t row0, int kt, int n_keys, int krow0, int rr,
                       int g) {
    k0 = *(const short4_t *)(kc + (row0 + min(kt + krow0, n_keys - 1)) * 16 + 4 * g);
    k1 = *(const short4_t *)(kc + (row0 + min(kt + krow0 + 4, n_keys - 1)) * 16 + 4 * g);
    const int k8 = kt + 8 * g, nv = n_keys - k8;
    v = *(const uint4 *)(vc + v_at<bf16_t>(row0, min(k8, n_keys - 1) & ~7, rr, 16));
    uint32_t mk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) mk[i] = (2 * i >= nv) ? 0u : (2 * i + 1 >= nv) ? 0xFFFFu : 0xFFFFFFFFu;
    v = make_uint4(v.x & mk[0], v.y & mk[1], v.z & mk[2], v.w & mk[3]);
  }
};
template <> struct DraftStep<float> {
  f32x4_t k0, k1;
  float v[8];
  __device__ void load(const float *kc, const float *vc, size_t row0, int kt, int n_keys, int krow0, int rr,
                       int g) {
    k0 = *(const f32x4_t *)(kc + (row0 + min(kt + krow0, n_keys - 1)) * 16 + 4 * g);
    k1 = *(const f32x4_t *)(kc + (row0 + min(kt + krow0 + 4, n_keys - 1)) * 16 + 4 * g);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = vc[(row0 + min(kt + 8 * g + j, n_keys - 1)) * 16 + rr];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = (kt + 8 * g + j < n_keys) ? v[j] : 0.f;
  }
};

// Causal attention of P <= 2 new queries on the vector ALU, for draft
// models with at most 4 heads of width 16: the 256 threads split into H
// groups, one per head; thread `sub` of a group takes the key units sub,
// sub + 256 / H, ... (a unit is 4 keys for bf16 caches, half a block of the
// blocked value layout, 2 for fp32), loads the unit's key rows and values
// with 8- and 16-byte loads, scores them against both queries in fp32 and keeps its
// own online softmax (max, sum, 16 output columns per query). The threads of
// a head then merge: maximum, rescaled sums and outputs through wave
// reductions and LDS. With only one or two queries per head the MFMA form
// computes mostly padding; here every thread's loads go out together and
// the step costs about one memory latency per unit a thread holds.
// red: LDS scratch of at least 4 * 2 * 18 floats.
// one step of a recursive-halving wave reduction of 2N values per lane: the
// lane keeps its half (the upper one if hi), adds the partner's copy of it
template <int N, typename X>
__device__ __forceinline__ void halve_step(float (&v)[16], bool hi, X xchg) {
#pragma unroll
  for (int c = 0; c < N; ++c) {
    const float keep = hi ? v[c + N] : v[c], give = hi ? v[c] : v[c + N];
    v[c] = keep + xchg(give);
  }
}

template <typename ELT, int QN, typename OT>
__device__ void wg_attention_valu(const float *qs, OT *os, const ELT *kc, const ELT *vc, size_t seq_row0, int cap,
                                  int H, int P, int pos0, int d, float *red) {
  // QN = P queries; with one query a thread's 4-key unit (keys and values in
  // registers) fits beside the rest of the kernel in fp32 too
  constexpr int DH = 16, U = (sizeof(ELT) == 2 || QN == 1) ? 4 : 2;
  constexpr int NKV = U * DH * (int)sizeof(ELT) / 16;   // 16-byte vectors of a unit's keys (and of its fp32 values)
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int tph = blockDim.x / H, h = tid / tph, sub = tid - h * tph;
  const int n_keys = min(pos0 + P, cap);
  const size_t row0 = seq_row0 + (size_t)h * cap;
  float q[QN][DH];
#pragma unroll
  for (int p = 0; p < QN; ++p)
#pragma unroll
    for (int j = 0; j < DH; ++j) q[p][j] = qs[p * d + h * DH + j] * 0.25f;   // 1 / sqrt(16)
  // bf16: the scaled queries (bf16 values, scaled by a power of two) as
  // pairs for v_dot2c against the raw key words
  uint32_t qw[QN][sizeof(ELT) == 2 ? DH / 2 : 1];
  if constexpr (sizeof(ELT) == 2) {
#pragma unroll
    for (int p = 0; p < QN; ++p)
#pragma unroll
      for (int e = 0; e < DH / 2; ++e) qw[p][e] = pk2bf(q[p][2 * e], q[p][2 * e + 1]);
  }
  float m[QN], l[QN], o[QN][DH];
#pragma unroll
  for (int p = 0; p < QN; ++p) {
    m[p] = -INFINITY;
    l[p] = 0.f;
#pragma unroll
    for (int j = 0; j < DH; ++j) o[p][j] = 0.f;
  }
  const int nunits = (n_keys + U - 1) / U;
  for (int u = sub; u < nunits; u += tph) {
    const int k0 = u * U;
    // the unit lies inside the slab (k0 < cap, the slab holds cap rounded
    // up to 8 positions); keys at or past n_keys are masked below. Values
    // stay packed in registers and are widened where they are used.
    uint4 kr[NKV];
    uint2 vr2[16];
    uint4 vr4[sizeof(ELT) == 2 ? 1 : NKV];
    if constexpr (sizeof(ELT) == 2) {
      const uint4 *kp = (const uint4 *)(kc + (row0 + k0) * DH);   // 4 rows x 16
#pragma unroll
      for (int i = 0; i < NKV; ++i) kr[i] = kp[i];
      // value column j of the block holding k0: 8 positions, this unit's 4 at k0 & 4
      const bf16_t *vb = vc + v_at<bf16_t>(row0, k0 & ~7, 0, DH) + (k0 & 4);
#pragma unroll
      for (int j = 0; j < 16; ++j) vr2[j] = *(const uint2 *)(vb + 8 * j);
    } else {
      const uint4 *kp = (const uint4 *)(kc + (row0 + k0) * DH);   // U rows x 16
      const uint4 *vp = (const uint4 *)(vc + (row0 + k0) * DH);
#pragma unroll
      for (int i = 0; i < NKV; ++i) kr[i] = kp[i];
#pragma unroll
      for (int i = 0; i < NKV; ++i) vr4[i] = vp[i];
    }
    // element (key i, column j) of the unit's keys and values
    auto kval = [&](int i, int j) -> float {
      if constexpr (sizeof(ELT) == 2) {
        const uint4 w = kr[2 * i + (j >> 3)];
        const int e = (j & 7) >> 1;
        const uint32_t x = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
        return (j & 1) ? __uint_as_float(x & 0xFFFF0000u) : __uint_as_float(x << 16);
      } else {
        const uint4 w = kr[4 * i + (j >> 2)];
        const int e = j & 3;
        return __uint_as_float(e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w);
      }
    };
    auto vval = [&](int i, int j) -> float {
      if constexpr (sizeof(ELT) == 2) {
        const uint2 w = vr2[j];   // column j, the unit's 4 positions
        const uint32_t x = (i >> 1) ? w.y : w.x;
        return (i & 1) ? __uint_as_float(x & 0xFFFF0000u) : __uint_as_float(x << 16);
      } else {
        const uint4 w = vr4[4 * i + (j >> 2)];
        const int e = j & 3;
        return __uint_as_float(e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w);
      }
    };
    // every query in one pass over the unit (each key and value element is
    // widened once); query p sees keys up to position pos0 + p
    float sc[QN][U], mx[QN];
#pragma unroll
    for (int p = 0; p < QN; ++p) mx[p] = -INFINITY;
#pragma unroll
    for (int i = 0; i < U; ++i) {
      float a[QN];
#pragma unroll
      for (int p = 0; p < QN; ++p) a[p] = 0.f;
      if constexpr (sizeof(ELT) == 2) {
#pragma unroll
        for (int hv = 0; hv < 2; ++hv) {
          const uint4 w = kr[2 * i + hv];   // columns 8 hv .. 8 hv + 7 of key i
#pragma unroll
          for (int p = 0; p < QN; ++p) {
            a[p] = dot2_bf(w.x, qw[p][4 * hv], a[p]);
            a[p] = dot2_bf(w.y, qw[p][4 * hv + 1], a[p]);
            a[p] = dot2_bf(w.z, qw[p][4 * hv + 2], a[p]);
            a[p] = dot2_bf(w.w, qw[p][4 * hv + 3], a[p]);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < DH; ++j) {
          const float kv = kval(i, j);
#pragma unroll
          for (int p = 0; p < QN; ++p) a[p] += q[p][j] * kv;
        }
      }
      const int pos = k0 + i;
#pragma unroll
      for (int p = 0; p < QN; ++p) {
        sc[p][i] = (pos < n_keys && pos <= pos0 + p) ? a[p] : -INFINITY;
        mx[p] = fmaxf(mx[p], sc[p][i]);
      }
    }
    float al[QN], ex[QN][U];
#pragma unroll
    for (int p = 0; p < QN; ++p) {
      const float mn = fmaxf(m[p], mx[p]);
      // rescale factor (1 while a query has seen no key, its state being zero)
      al[p] = (mn == -INFINITY) ? 1.f : expf(m[p] - mn);
      l[p] *= al[p];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        ex[p][i] = (sc[p][i] == -INFINITY) ? 0.f : expf(sc[p][i] - mn);
        l[p] += ex[p][i];
      }
      m[p] = mn;
    }
    // slots at or past n_keys hold stale or unwritten values: a zero weight
    // times a non-finite value would still poison the sum, so they are skipped
#pragma unroll
    for (int j = 0; j < DH; ++j) {
      float sp[QN];
#pragma unroll
      for (int p = 0; p < QN; ++p) sp[p] = o[p][j] * al[p];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const float vv = (k0 + i < n_keys) ? vval(i, j) : 0.f;
#pragma unroll
        for (int p = 0; p < QN; ++p) sp[p] += ex[p][i] * vv;
      }
#pragma unroll
      for (int p = 0; p < QN; ++p) o[p][j] = sp[p];
    }
  }
  // merge the threads of each head: per wave first, then across the head's waves
  const int wph = tph >> 6;   // waves per head (1, 2 or 4)
#pragma unroll
  for (int p = 0; p < QN; ++p) {
    const float mw = wave_max(m[p]);
    if (lane == 0) red[wave * 36 + p * 18] = mw;
  }
  lds_barrier();
#pragma unroll
  for (int p = 0; p < QN; ++p) {
    float M = -INFINITY;
    for (int w = h * wph; w < (h + 1) * wph; ++w) M = fmaxf(M, red[w * 36 + p * 18]);
    const float f = (m[p] == -INFINITY) ? 0.f : expf(m[p] - M);
    const float lw = wave_sum(l[p] * f);
    float ow[DH];
#pragma unroll
    for (int j = 0; j < DH; ++j) ow[j] = o[p][j] * f;
    // the 16 column sums over the wave by recursive halving: each exchange
    // keeps half of the columns (the half named by the lane's bit) and adds
    // the partner's copy of that half; lane holds column (lane >> 2) & 15 at
    // the end, summed over the 4 lanes of its quad by two more exchanges
    halve_step<8>(ow, (lane & 32) != 0, [](float v) { return __shfl_xor(v, 32, 64); });
    halve_step<4>(ow, (lane & 16) != 0, [](float v) { return swz_xor<16>(v); });
    halve_step<2>(ow, (lane & 8) != 0, [](float v) { return swz_xor<8>(v); });
    halve_step<1>(ow, (lane & 4) != 0, [](float v) { return swz_xor<4>(v); });
    float oc = ow[0];
    oc += dpp_mov<0x4E>(oc);   // lane ^ 2
    oc += dpp_mov<0xB1>(oc);   // lane ^ 1
    if (lane == 0) red[wave * 36 + p * 18 + 1] = lw;
    if ((lane & 3) == 0) red[wave * 36 + p * 18 + 2 + (lane >> 2)] = oc;
  }
  lds_barrier();
  for (int idx = tid; idx < QN * H * DH; idx += blockDim.x) {
    const int p = idx / (H * DH), rest = idx - p * H * DH, hh = rest / DH, j = rest - hh * DH;
    float L = 0.f, O = 0.f;
    for (int w = hh * wph; w < (hh + 1) * wph; ++w) {
      L += red[w * 36 + p * 18 + 1];
      O += red[w * 36 + p * 18 + 2 + j];
    }
    st<OT>(os, p * d + hh * DH + j, rnd_act<ELT>(L > 0.f ? O / L : 0.f));
  }
}

// causal attention of P <= 2 new queries (positions pos0 .. pos0 + P - 1,
// already in the cache) over one sequence's cache, d_head = 16, on MFMA in
// the layout of k_attn_mfma: S^T = K Q^T with permuted key rows leaves lane
// (rr, g) the scores of query rr for keys 8 g .. + 7, the B operand of
// O^T = V^T P^T (queries P .. 15 of the tile are zero). Each head is served
// by 4 / H waves (one wave per head from H = 4; more heads loop), which take
// 32-key steps round robin; a wave loads a batch of steps (8 bf16, 4 fp32)
// before computing any.
// The waves of a head merge through LDS. red: LDS scratch of
// max(4, H) * 2 * 18 floats.
template <typename ELT, int DH, int QMAX = 2, int NB = 4, typename OT = float>   // NB: steps per load batch
__device__ void wg_attention(const float *qs, OT *os, const ELT *kc, const ELT *vc, size_t seq_row0, int cap,
                             int H, int P, int pos0, int ld, float *red) {
  static_assert(DH == 16, "the fused draft attention serves d_head = 16");
  constexpr int KT = 32;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rr = lane & 15, g = lane >> 4;
  const int nw = blockDim.x >> 6, wph = H >= nw ? 1 : nw / H, wsub = wave % wph;
  const int n_keys = min(pos0 + P, cap);
  const float scale = 0.25f;   // 1 / sqrt(16)
  const int krow0 = 8 * (rr >> 2) + (rr & 3);
  for (int h = wave / wph; h < H; h += nw / wph) {
    const size_t row0 = seq_row0 + (size_t)h * cap;
    // query fragment: dims 4 g .. + 3 of query rr (zero for rr >= P)
    const float *qp = qs + min(rr, P - 1) * ld + h * DH + 4 * g;
    const float q0 = rr < P ? qp[0] : 0.f, q1 = rr < P ? qp[1] : 0.f, q2 = rr < P ? qp[2] : 0.f,
                q3 = rr < P ? qp[3] : 0.f;
    float m_run = -INFINITY, l_run = 0.f;
    f32x4_t oacc = {0.f, 0.f, 0.f, 0.f};
    for (int kb = wsub * KT; kb < n_keys; kb += NB * wph * KT) {
      DraftStep<ELT> f[NB];
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx)
        f[sidx].load(kc, vc, row0, min(kb + sidx * wph * KT, n_keys - 1) & ~(KT - 1), n_keys, krow0, rr, g);
      // scores of the whole batch first, then one online-softmax update
      // (steps past the key range score -inf; their values were zeroed)
      float sv[NB][8];
      float mx = -INFINITY;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx) {
        const int kt = kb + sidx * wph * KT;
        if (kt >= n_keys) {   // uniform across the wave
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[sidx][j] = -INFINITY;
          continue;
        }
        f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
        if constexpr (sizeof(ELT) == 2) {
          const uint32_t w0 = pk2bf(q0, q1);
          const uint32_t w1 = pk2bf(q2, q3);
          const short4_t qf = __builtin_bit_cast(short4_t, make_uint2(w0, w1));
          s0 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(f[sidx].k0, qf, s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(f[sidx].k1, qf, s1, 0, 0, 0);
        } else {
          const float qv[4] = {q0, q1, q2, q3};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].k0[e], qv[e], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].k1[e], qv[e], s1, 0, 0, 0);
          }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = kt + 8 * g + j;
          const float raw = (j < 4) ? s0[j] : s1[j - 4];
          sv[sidx][j] = (rr < P && key < n_keys && key <= pos0 + rr) ? raw * scale : -INFINITY;
          mx = fmaxf(mx, sv[sidx][j]);
        }
      }
      mx = fmaxf(mx, swz_xor<16>(mx));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = (m_new == -INFINITY) ? 1.f : expf(m_run - m_new);
      float ps = 0.f;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          // bf16: P V takes the probabilities in bf16, and the normaliser sums
          // the same rounded values
          sv[sidx][j] = (sv[sidx][j] == -INFINITY) ? 0.f : rnd_act<ELT>(expf(sv[sidx][j] - m_new));
          ps += sv[sidx][j];
        }
      ps += swz_xor<16>(ps);
      ps += __shfl_xor(ps, 32, 64);
      l_run = l_run * alpha + ps;
      m_run = m_new;
      oacc *= alpha;
#pragma unroll
      for (int sidx = 0; sidx < NB; ++sidx) {
        if (kb + sidx * wph * KT >= n_keys) break;   // uniform across the wave
        if constexpr (sizeof(ELT) == 2) {
          uint32_t pw[4];
#pragma unroll
          for (int j = 0; j < 8; j += 2)
            pw[j >> 1] = pk2bf(sv[sidx][j], sv[sidx][j + 1]);
          const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
          oacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, f[sidx].v), pb, oacc, 0, 0, 0);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            oacc = __builtin_amdgcn_mfma_f32_16x16x4f32(f[sidx].v[j], sv[sidx][j], oacc, 0, 0, 0);
        }
      }
    }
    // lane (rr, g) holds O^T[4 g + i][query rr]
    if (rr < P) {
      float *r = red + ((h * wph + wsub) * QMAX + rr) * (DH + 2);
      if (g == 0) {
        r[0] = m_run;
        r[1] = l_run;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) r[2 + 4 * g + i] = oacc[i];
    }
  }
  lds_barrier();
  for (int idx = tid; idx < P * H * DH; idx += blockDim.x) {
    const int p = idx / (H * DH), rest = idx - p * H * DH, hh = rest / DH, j = rest - hh * DH;
    float M = -INFINITY;
    for (int w = 0; w < wph; ++w) M = fmaxf(M, red[((hh * wph + w) * QMAX + p) * (DH + 2)]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < wph; ++w) {
      const float *r = red + ((hh * wph + w) * QMAX + p) * (DH + 2);
      const float f = (r[0] == -INFINITY) ? 0.f : expf(r[0] - M);
      L += r[1] * f;
      O += r[2 + j] * f;
    }
    st<OT>(os, p * ld + hh * DH + j, rnd_act<ELT>(L > 0.f ? O / L : 0.f));
  }
}

// floats of the model's small fp32 vectors (LayerNorm gains and biases,
// linear biases, time-encoding frequencies) staged in LDS by the fused draft
inline __host__ __device__ int fused_draft_vec_floats(int L, int d, int F, int M, int K) {
  return L * (9 * d + F) + 4 * d + 3 * M + K;
}

// floats before the staged weights (activations, merge scratch, vectors),
// rounded up to a 16-byte boundary
// attention merge scratch: one (max, sum, output) slot per wave and query
inline __host__ __device__ int fused_draft_red_floats(int H, int dh) { return 4 * H * 2 * (dh + 2); }

inline __host__ __device__ int fused_draft_head_floats(int L, int d, int F, int M, int K, int H) {
  const int Fm = d > F ? d : F, dh = d / H;
  const int n = 2 * d + 2 * Fm + 2 * d + 2 * d + 2 * F + 4 * d + 3 * M + K + 8 + fused_draft_red_floats(H, dh) +
                fused_draft_vec_floats(L, d, F, M, K);
  return (n + 3) & ~3;
}

size_t fused_draft_weight_elems(int L, int d, int F, int M, int K, int pad) {
  return (size_t)L * ((size_t)(4 * d + F) * (d + pad) + (size_t)d * (F + pad)) + (size_t)(4 * d + 3 * M + K) * (d + pad);
}

size_t fused_draft_lds_bytes(int L, int d, int F, int M, int K, int H) {
  return (size_t)fused_draft_head_floats(L, d, F, M, K, H) * sizeof(float);
}

// CD / CF: chunks per lane of the matrix-vector products over d and over
// d_ffn (gemv_cpl), fixed per model so that each product has one code path
template <typename ELT, int DH, int CD, int CF, int NT>
__global__ __launch_bounds__(NT) void k_draft_fused(DraftArgs a) {
  extern __shared__ __attribute__((aligned(16))) float sm[];
  __shared__ float tok_t[2], t_last;
  __shared__ int tok_k[2];
  __shared__ float pu[TPPSD_MAX_GAMMA][4];   // the draws' uniforms, one Philox block per step
  const int d = a.d, F = a.F, M = a.M, K = a.K, H = a.H;
  const int Fm = d > F ? d : F;
  // the rows the matrix-vector products read are in the weights' element
  // type (bf16 halves of their float slots)
  using XT = typename std::conditional<sizeof(ELT) == 2, bf16_t, float>::type;
  float *xs = sm;                            // [2][d] residual stream
  XT *as = (XT *)(sm + 2 * d);               // [2][Fm] LayerNorm outputs
  float *qs = sm + 2 * d + 2 * Fm;           // [2][d] queries
  XT *os = (XT *)(qs + 2 * d);               // [2][d] attention outputs
  XT *hs = (XT *)(qs + 4 * d);               // [2][F] FFN hidden
  XT *es = (XT *)(qs + 4 * d + 2 * F);       // [4d] decoder e | tanh activations
  float *hv = qs + 8 * d + 2 * F;            // [3M + K] decoder outputs
  float *red = hv + 3 * M + K + 8;   // attention merge scratch
  float *vec = red + fused_draft_red_floats(H, DH);   // staged small vectors
  const int b = blockIdx.x, tid = threadIdx.x;
  if (a.done[b]) return;
  // every LayerNorm and bias vector of the model goes to LDS once, so that
  // the per-step phases read no small vectors from memory
  {
    auto cp = [&](float *dst, const float *src, int cnt) {
      for (int i = tid; i < cnt; i += blockDim.x) dst[i] = src[i];
    };
    for (int ly = 0; ly < a.L; ++ly) {
      const FusedLayerW &w = a.layer[ly];
      float *v = vec + ly * (9 * d + F);
      cp(v, w.ln1_g, d);
      cp(v + d, w.ln1_b, d);
      cp(v + 2 * d, w.qkv_b, 3 * d);
      cp(v + 5 * d, w.out_b, d);
      cp(v + 6 * d, w.ln2_g, d);
      cp(v + 7 * d, w.ln2_b, d);
      cp(v + 8 * d, w.ffn1_b, F);
      cp(v + 8 * d + F, w.ffn2_b, d);
    }
    float *v = vec + a.L * (9 * d + F);
    cp(v, a.lnf_g, d);
    cp(v + d, a.lnf_b, d);
    cp(v + 2 * d, a.k1_b, d);
    cp(v + 3 * d, a.mix_b, 3 * M);
    cp(v + 3 * d + 3 * M, a.k2_b, K);
    cp(v + 3 * d + 3 * M + K, a.freq, d);
  }
  // the weight matrices too, when the host found room for them: the
  // per-step matrix-vector products then read only LDS. LDS layout: per
  // layer QKV (3d x d), out (d x d), FFN in (F x d), FFN out (d x F); then
  // [E; V_k1] (4d x d), the mixture heads (3M x d), the type head (K x d).
  // Each row is padded by 16 bytes: the products read one row per lane, and
  // unpadded rows of 128 or 512 bytes would put every lane on the same banks.
  constexpr int PD = 16 / sizeof(ELT);
  ELT *const wl = (ELT *)(sm + fused_draft_head_floats(a.L, d, F, M, K, H));
  const int ldd = a.w_lds ? d + PD : d, ldf = a.w_lds ? F + PD : F;   // row strides of the matrices read
  const size_t LS = (size_t)(4 * d + F) * (d + PD) + (size_t)d * (F + PD);
  const size_t o_out = (size_t)3 * d * (d + PD), o_f1 = (size_t)4 * d * (d + PD),
               o_f2 = o_f1 + (size_t)F * (d + PD), o_mix = (size_t)4 * d * (d + PD),
               o_k2 = o_mix + (size_t)3 * M * (d + PD);
  if (a.w_lds) {
    // rows x cols (cols a multiple of 16 bytes) into rows of cols + PD
    auto cpw = [&](size_t off, const void *src, int rows, int cols) {
      const int vr = cols / PD;   // 16-byte vectors per row
      const uint4 *sp = (const uint4 *)src;
      uint4 *dp = (uint4 *)(wl + off);
      for (int i = tid; i < rows * vr; i += blockDim.x) {
        const int r = i / vr, c = i - r * vr;
        dp[r * (vr + 1) + c] = sp[i];
      }
    };
    for (int ly = 0; ly < a.L; ++ly) {
      cpw(ly * LS, a.layer[ly].qkv_w, 3 * d, d);
      cpw(ly * LS + o_out, a.layer[ly].out_w, d, d);
      cpw(ly * LS + o_f1, a.layer[ly].ffn1_w, F, d);
      cpw(ly * LS + o_f2, a.layer[ly].ffn2_w, d, F);
    }
    cpw(a.L * LS, a.Ek1_w, 4 * d, d);
    cpw(a.L * LS + o_mix, a.mix_w, 3 * M, d);
    cpw(a.L * LS + o_k2, a.k2_w, K, d);
  }
  auto wmat = [&](const void *glob, size_t off) -> const ELT * {
    return a.w_lds ? (const ELT *)(wl + off) : (const ELT *)glob;
  };
  const float *hvec = vec + a.L * (9 * d + F);
  const float *lnf_g = hvec, *lnf_b = hvec + d, *k1_b = hvec + 2 * d, *mix_b = hvec + 3 * d,
              *k2_b = hvec + 3 * d + 3 * M, *freq = hvec + 3 * d + 3 * M + K;
  const int n = a.n[b], base = a.lenD[b];
  const uint64_t r = (uint64_t)a.rnd[b];
  const size_t seq_row0 = (size_t)b * H * a.cap;
  const ELT *wtype = (const ELT *)a.type_emb;
  if (tid == 0) t_last = a.ev_t[(size_t)b * a.ev_stride + n - 1];
  if (tid < a.gamma) {   // the uniforms depend only on the counters: drawn up front, off the step chain
    float u[4];
    philox_uniforms(a.seed, (uint64_t)b, r, (uint64_t)(tid + 1), TAG_DRAFT, u);
    pu[tid][0] = u[0];
    pu[tid][1] = sqrtf(-2.f * logf(u[1])) * cosf(6.28318530717958647692f * u[2]);   // Box-Muller epsilon
    pu[tid][3] = u[3];
  }
  for (int l = 1; l <= a.gamma; ++l) {
    const int P = (l == 1) ? 2 : 1;
    const int pos0 = (l == 1) ? base : base + l;
    if (l == 1 && tid < 2) {
      const size_t i = (size_t)b * a.ev_stride + n - 2 + tid;
      tok_t[tid] = a.ev_t[i];
      tok_k[tid] = a.ev_k[i];
    }
    lds_barrier();
    for (int i = tid; i < P * d; i += blockDim.x) {
      const int p = i / d, j = i - p * d;
      const float arg = tok_t[p] * freq[j];
      const int kk = min(max(tok_k[p], 0), K - 1);
      xs[i] = ((j & 1) ? cosf(arg) : sinf(arg)) + ld(wtype, (size_t)kk * d + j);
    }
    lds_barrier();
    for (int ly = 0; ly < a.L; ++ly) {
      const FusedLayerW &w = a.layer[ly];
      ELT *kc = (ELT *)(a.kc + a.layer_bytes * ly);
      ELT *vc = (ELT *)(a.vc + a.layer_bytes * ly);
      const float *lv = vec + ly * (9 * d + F);
      const float *ln1_g = lv, *ln1_b = lv + d, *qkv_b = lv + 2 * d, *out_b = lv + 5 * d, *ln2_g = lv + 6 * d,
                  *ln2_b = lv + 7 * d, *ffn1_b = lv + 8 * d, *ffn2_b = lv + 8 * d + F;
      wg_layernorm<ELT>(xs, as, ln1_g, ln1_b, P, d);
      lds_barrier();
      const ELT *wq = wmat(w.qkv_w, ly * LS);
      wg_gemv_cpl<ELT, CD>(
          3 * d, d, P, [&](int nn) { return wq + (size_t)nn * ldd; }, [&](int, int p) { return (const XT *)(as + p * d); },
          [&](int p, int nn, float acc) {
            const float v = rnd_act<ELT>(acc + qkv_b[nn]);
            const int which = nn / d, c = nn - which * d;
            if (which == 0) {
              qs[p * d + c] = v;
            } else {
              const int h = c / DH, j = c - h * DH, pos = pos0 + p;
              const size_t row0 = seq_row0 + (size_t)h * a.cap;
              if (pos < a.cap)
                st(which == 1 ? kc : vc, which == 1 ? (row0 + pos) * DH + j : v_at<ELT>(row0, pos, j, DH), v);
              else
                atomicOr(a.status, TPPSD_STATUS_CAPACITY);
            }
          });
      __syncthreads();   // keys and values in the cache before the attention reads them
      if (H <= 4)
        P == 2 ? wg_attention_valu<ELT, 2, XT>(qs, os, kc, vc, seq_row0, a.cap, H, P, pos0, d, red)
               : wg_attention_valu<ELT, 1, XT>(qs, os, kc, vc, seq_row0, a.cap, H, P, pos0, d, red);
      else
        wg_attention<ELT, DH, 2, 4, XT>(qs, os, kc, vc, seq_row0, a.cap, H, P, pos0, d, red);
      lds_barrier();
      const ELT *wo = wmat(w.out_w, ly * LS + o_out);
      wg_gemv_cpl<ELT, CD>(
          d, d, P, [&](int nn) { return wo + (size_t)nn * ldd; }, [&](int, int p) { return (const XT *)(os + p * d); },
          [&](int p, int nn, float acc) { xs[p * d + nn] += acc + out_b[nn]; });
      lds_barrier();
      wg_layernorm<ELT>(xs, as, ln2_g, ln2_b, P, d);
      lds_barrier();
      const ELT *w1 = wmat(w.ffn1_w, ly * LS + o_f1);
      const ELT *w2 = wmat(w.ffn2_w, ly * LS + o_f2);
      wg_gemv_cpl<ELT, CD>(
          F, d, P, [&](int nn) { return w1 + (size_t)nn * ldd; }, [&](int, int p) { return (const XT *)(as + p * d); },
          [&](int p, int nn, float acc) { st<XT>(hs, p * F + nn, rnd_act<ELT>(fmaxf(acc + ffn1_b[nn], 0.f))); });
      lds_barrier();
      wg_gemv_cpl<ELT, CF>(
          d, F, P, [&](int nn) { return w2 + (size_t)nn * ldf; }, [&](int, int p) { return (const XT *)(hs + p * F); },
          [&](int p, int nn, float acc) { xs[p * d + nn] += acc + ffn2_b[nn]; });
      lds_barrier();
    }
    // decoder on the last token: e = E h and tanh(V_k1 h + b1) in one pass,
    // then the mixture (w, mu, log sigma from the slices of e) and type
    // logits in one pass
    wg_layernorm<ELT>(xs + (P - 1) * d, as, lnf_g, lnf_b, 1, d);
    lds_barrier();
    const ELT *we = wmat(a.Ek1_w, a.L * LS);
    wg_gemv_cpl<ELT, CD>(
        4 * d, d, 1, [&](int nn) { return we + (size_t)nn * ldd; }, [&](int, int) { return (const XT *)as; },
        [&](int, int nn, float acc) {
          st<XT>(es, nn, (nn < 3 * d) ? rnd_act<ELT>(acc) : rnd_act<ELT>(tanhf(acc + k1_b[nn - 3 * d])));
        });
    lds_barrier();
    const ELT *mw = wmat(a.mix_w, a.L * LS + o_mix);
    const ELT *kw = wmat(a.k2_w, a.L * LS + o_k2);
    wg_gemv_cpl<ELT, CD>(
        3 * M + K, d, 1,
        [&](int nn) { return nn < 3 * M ? mw + (size_t)nn * ldd : kw + (size_t)(nn - 3 * M) * ldd; },
        [&](int nn, int) { return (const XT *)(es + (nn < 3 * M ? nn / M : 3) * d); },
        [&](int, int nn, float acc) { hv[nn] = acc + (nn < 3 * M ? mix_b[nn] : k2_b[nn - 3 * M]); });
    lds_barrier();
    if (tid < 64) {
      // wave 0, from registers: the log-softmaxes of the mixture weights and
      // the types, the draft record, and the draft event (component,
      // Box-Muller interval, type)
      const int lane = tid;
      const float lw = lane < M ? hv[lane] : -INFINITY;
      const float mu_l = lane < M ? hv[M + lane] : 0.f, s_l = lane < M ? hv[2 * M + lane] : 0.f;
      const float lk = lane < K ? hv[3 * M + lane] : -INFINITY;
      const float mw2 = wave_max(lw);
      const float sw = wave_sum(lane < M ? expf(lw - mw2) : 0.f);
      const float mk = wave_max(lk);
      const float sk = wave_sum(lane < K ? expf(lk - mk) : 0.f);
      const float nlw = lw - mw2 - logf(sw), nlk = lk - mk - logf(sk);
      const size_t di = (size_t)b * a.MG + (l - 1);
      if (lane < M) {
        a.d_mix[di * 3 * M + lane] = nlw;
        a.d_mix[di * 3 * M + M + lane] = mu_l;
        a.d_mix[di * 3 * M + 2 * M + lane] = s_l;
      }
      if (lane < K) a.d_logtype[di * K + lane] = nlk;
      // first index whose running sum of exp(log p) exceeds u times the total
      auto draw = [&](float lp, int n, float u) {
        float c = lane < n ? expf(lp) : 0.f;
        c = wave_cumsum(c);
        const float tot = lane_val(c, n - 1);
        const unsigned long long hit = __ballot(lane < n && u * tot < c);
        return hit ? (int)__builtin_ctzll(hit) : n - 1;
      };
      auto at = [](float v, int i) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i)); };
      const float *u = pu[l - 1];
      const int z = draw(nlw, M, u[0]);
      const float tau = expf(at(mu_l, z) + expf(at(s_l, z)) * u[1]);
      const int kk = draw(nlk, K, u[3]);
      // log g of the drawn interval under the draft mixture
      const float lt = logf(tau);
      float c = -INFINITY;
      if (lane < M) {
        const float zz = lt - mu_l;
        c = nlw - s_l - 0.918938533204672742f - lt - 0.5f * zz * zz * expf(-2.f * s_l);
      }
      const float cm = wave_max(c);
      const float lg = cm + logf(wave_sum(lane < M ? expf(c - cm) : 0.f));
      const float lf = at(nlk, kk);
      if (tid == 0) {
        const float tn = t_last + tau;
        a.d_tau[di] = tau;
        a.d_t[di] = tn;
        a.d_k[di] = kk;
        a.d_logg[di] = lg;
        a.d_logf[di] = lf;
        if (!isfinite(tau)) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
        tok_t[0] = tn;
        tok_k[0] = kk;
        t_last = tn;
      }
    }
    lds_barrier();
  }
}

void launch_draft_fused(const DraftArgs &a, int bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const size_t lds = fused_draft_lds_bytes(a.L, a.d, a.F, a.M, a.K, a.H) +
                     (a.w_lds ? fused_draft_weight_elems(a.L, a.d, a.F, a.M, a.K, bf16 ? 8 : 4) * (bf16 ? 2 : 4) : 0);
  // chunks per lane of the d-wide and F-wide products: d / 16 (two lanes
  // per row at d = 32, four at d = 64), and F d / 2048 (the d rows of the
  // second FFN product over all 256 lanes), each within 2..8 -- measured
  // against one chunk set per lane of K / 8 <= 8: 180 -> 154 us per draft
  // round at d = 32 / F = 128, 480 -> 462 us at d = 64 / F = 256.
  int cd = std::min(8, std::max(2, a.d / 16)), cf = std::min(8, std::max(2, a.F * a.d / 2048));
  cd = std::min(cd, gemv_cpl(a.d));
  cf = std::min(cf, gemv_cpl(a.F));
  auto go = [&](auto kern, int nt) { hipExtLaunchKernelGGL(kern, dim3(a.B), dim3(nt), lds, s, ev0, ev1, 0, a); };
  // chunk counts 2, 4 or 8; four waves
#define TPPSD_FD(ELT, DH, NT)                                                       \
  if (cd == 2 && cf == 2) go(k_draft_fused<ELT, DH, 2, 2, NT>, NT);                 \
  else if (cd == 2 && cf == 4) go(k_draft_fused<ELT, DH, 2, 4, NT>, NT);            \
  else if (cd == 2) go(k_draft_fused<ELT, DH, 2, 8, NT>, NT);                       \
  else if (cd == 4 && cf == 2) go(k_draft_fused<ELT, DH, 4, 2, NT>, NT);            \
  else if (cd == 4 && cf == 4) go(k_draft_fused<ELT, DH, 4, 4, NT>, NT);            \
  else if (cd == 4) go(k_draft_fused<ELT, DH, 4, 8, NT>, NT);                       \
  else if (cf == 2) go(k_draft_fused<ELT, DH, 8, 2, NT>, NT);                       \
  else if (cf == 4) go(k_draft_fused<ELT, DH, 8, 4, NT>, NT);                       \
  else go(k_draft_fused<ELT, DH, 8, 8, NT>, NT);
  if (bf16) {
    TPPSD_FD(bf16_t, 16, 256)
  } else {
    TPPSD_FD(float, 16, 256)
  }
#undef TPPSD_FD
}

int allow_draft_fused_lds(size_t bytes) {
  int bad = 0;
  auto set = [&](auto kern) {
    bad |= hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) !=
           hipSuccess;
  };
#define TPPSD_FD(ELT)                                                                          \
  set(k_draft_fused<ELT, 16, 2, 2, 256>), set(k_draft_fused<ELT, 16, 2, 4, 256>), set(k_draft_fused<ELT, 16, 2, 8, 256>); \
  set(k_draft_fused<ELT, 16, 4, 2, 256>), set(k_draft_fused<ELT, 16, 4, 4, 256>), set(k_draft_fused<ELT, 16, 4, 8, 256>); \
  set(k_draft_fused<ELT, 16, 8, 2, 256>), set(k_draft_fused<ELT, 16, 8, 4, 256>), set(k_draft_fused<ELT, 16, 8, 8, 256>);
  TPPSD_FD(bf16_t)
  TPPSD_FD(float)
#undef TPPSD_FD
  return bad;
}

// ---------------------------------------------------------------------------
// Drafting for small draft models (§4.3 "Drafting"), one wave per sequence:
// all gamma draft steps of a sequence run in one wave with no workgroup
// barrier after the weights are staged. A model of width D <= 32 puts one
// token's activations on D lanes (the two tokens of the first step on lanes
// 0..D-1 and 32..32+D-1); every matrix-vector product reads its matrix
// transposed from LDS ([in][out], so that lanes take consecutive outputs and
// one input broadcast per step of the dot product), staged once per
// workgroup of four sequences. The attention gives each lane one 8-position
// block of a head's cache at a time (eight key rows and the value block, 16
// bytes per load) and merges the lanes of a head by cross-lane reductions.
// Rounding points are those of the layered kernels.
// ---------------------------------------------------------------------------
// LDS floats of one wave's scratch for a model of width D, FFN width F, M
// mixture components and K types (a multiple of 4: each wave's rows start on
// a 16-byte boundary)
inline __host__ __device__ int wave_draft_scratch_floats(int D, int F, int M, int K) {
  return (2 * 32 + 2 * 32 + 2 * 32 + 2 * 32 + 2 * F + 4 * D + 3 * M + K + 4 + 3) & ~3;
}
// elements of the transposed weight matrices staged in LDS, and the floats of
// the small vectors
inline __host__ __device__ int wave_draft_weight_elems(int L, int D, int F, int M, int K) {
  return L * (3 * D * D + D * D + D * F + F * D) + D * 4 * D + D * (3 * M + K);
}
inline __host__ __device__ int wave_draft_vec_floats(int L, int D, int F, int M, int K) {
  return (L * (9 * D + F) + 4 * D + 3 * M + K + 3) & ~3;
}
size_t wave_draft_lds_bytes(int L, int D, int F, int M, int K, int elt) {
  const size_t w = ((size_t)wave_draft_weight_elems(L, D, F, M, K) * elt + 15) / 16 * 16;
  return w + 4 * ((size_t)wave_draft_vec_floats(L, D, F, M, K) + 4 * (size_t)wave_draft_scratch_floats(D, F, M, K));
}

// y[p][n] = sum_k WT[k][n] x[p][k] for n < N, p < P, handed to epi(p, n, y);
// fp32 weights as WT [KD][N]; lane takes n = lane, lane + 64, ...
template <int P, typename XF, typename EPI>
__device__ __forceinline__ void wave_gemv(const float *WT, int N, int KD, XF xin, EPI epi) {
  const int lane = threadIdx.x & 63;
  for (int n = lane; n < N; n += 64) {
    float acc0 = 0.f, acc1 = 0.f;
    const float *x0 = xin(n, 0), *x1 = xin(n, P - 1);
    // a few dot-product steps' loads in flight, not all of them (registers)
#pragma unroll 8
    for (int k = 0; k < KD; ++k) {
      const float w = WT[(size_t)k * N + n];
      acc0 += w * x0[k];
      if constexpr (P == 2) acc1 += w * x1[k];
    }
    epi(0, n, acc0);
    if constexpr (P == 2) epi(1, n, acc1);
  }
}

// The same product in bf16: weights as [KD / 8][N] 16-byte octets (octet
// (kq, n) holds W[n][8 kq .. 8 kq + 7]) and bf16 inputs, two products per
// v_dot2c_f32_bf16 (each exact in fp32). Columns go 64 to a pass; a pass of at
// most 32 columns splits the k range over the two halves of the wave and adds
// the halves' sums. KD is a multiple of 16.
template <int P, typename XF, typename EPI>
__device__ __forceinline__ void wave_gemv(const bf16_t *WT, int N, int KD, XF xin, EPI epi) {
  const int lane = threadIdx.x & 63;
  const uint4 *W = (const uint4 *)WT;
  const int KQ = KD >> 3;
  for (int n0 = 0; n0 < N; n0 += 64) {
    const int rem = N - n0;
    const bool split = rem <= 32;
    const int c = split ? (lane & 31) : lane;
    const int n = n0 + min(c, rem - 1);
    const int q0 = split ? (lane >> 5) * (KQ >> 1) : 0, q1 = split ? q0 + (KQ >> 1) : KQ;
    const uint4 *x0 = (const uint4 *)xin(n, 0), *x1 = (const uint4 *)xin(n, P - 1);
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll 4
    for (int kq = q0; kq < q1; ++kq) {
      const uint4 w = W[(size_t)kq * N + n];
      const uint4 xa = x0[kq];
      acc0 = dot2_bf(w.x, xa.x, acc0);
      acc0 = dot2_bf(w.y, xa.y, acc0);
      acc0 = dot2_bf(w.z, xa.z, acc0);
      acc0 = dot2_bf(w.w, xa.w, acc0);
      if constexpr (P == 2) {
        const uint4 xb = x1[kq];
        acc1 = dot2_bf(w.x, xb.x, acc1);
        acc1 = dot2_bf(w.y, xb.y, acc1);
        acc1 = dot2_bf(w.z, xb.z, acc1);
        acc1 = dot2_bf(w.w, xb.w, acc1);
      }
    }
    if (split) {
      acc0 += __shfl_xor(acc0, 32, 64);
      if constexpr (P == 2) acc1 += __shfl_xor(acc1, 32, 64);
    }
    if (c < rem && (!split || lane < 32)) {
      epi(0, n, acc0);
      if constexpr (P == 2) epi(1, n, acc1);
    }
  }
}

// LDS written by some lanes of the wave, then read by others
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// resident workgroups of four waves per CU the register allocation aims at
// (4: 128 VGPRs with spills, c5 draft 472 us per round; 3: 168 VGPRs, 356 us;
// 2: ~180 VGPRs, 309 us)
#ifndef TPPSD_WAVE_DRAFT_WG_PER_CU
#define TPPSD_WAVE_DRAFT_WG_PER_CU 2
#endif
template <typename ELT, int D, int F, int H>
__global__ __launch_bounds__(256, TPPSD_WAVE_DRAFT_WG_PER_CU) void k_draft_wave(DraftArgs a) {
  constexpr int DH = D / H;
  static_assert(DH == 16 && D <= 32 && F <= 128, "one wave per sequence: d <= 32, d_head 16");
  extern __shared__ __attribute__((aligned(16))) float smw[];
  const int M = a.M, K = a.K, L = a.L;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // ---- weights (transposed) and vectors, staged once per workgroup
  ELT *wl = (ELT *)smw;
  const int LW = 3 * D * D + D * D + D * F + F * D;   // elements per layer
  const int NH = 3 * M + K;
  float *vec = smw + ((size_t)wave_draft_weight_elems(L, D, F, M, K) * sizeof(ELT) + 15) / 16 * 4;
  float *scr = vec + wave_draft_vec_floats(L, D, F, M, K) + wave * wave_draft_scratch_floats(D, F, M, K);
  {
    // W [N][Kd] (global) -> LDS in the layout wave_gemv reads: fp32 as WT
    // [Kd][N], bf16 as [Kd / 8][N] octets of 8 consecutive k
    auto wt = [](int k, int n, int N) -> size_t {
      if constexpr (sizeof(ELT) == 2)
        return ((size_t)(k >> 3) * N + n) * 8 + (k & 7);
      else
        return (size_t)k * N + n;
    };
    auto cpt = [&](ELT *dst, const void *src, int N, int Kd) {
      const ELT *sp = (const ELT *)src;
      for (int i = tid; i < N * Kd; i += blockDim.x) {
        const int n = i / Kd, k = i - n * Kd;
        dst[wt(k, n, N)] = sp[i];
      }
    };
    for (int ly = 0; ly < L; ++ly) {
      const FusedLayerW &w = a.layer[ly];
      ELT *b0 = wl + (size_t)ly * LW;
      cpt(b0, w.qkv_w, 3 * D, D);
      cpt(b0 + 3 * D * D, w.out_w, D, D);
      cpt(b0 + 4 * D * D, w.ffn1_w, F, D);
      cpt(b0 + 4 * D * D + D * F, w.ffn2_w, D, F);
    }
    ELT *hb = wl + (size_t)L * LW;
    cpt(hb, a.Ek1_w, 4 * D, D);
    // the decoder heads as one [D][3M + K] matrix: columns < 3M the mixture
    // heads (w, mu, log sigma, read from the e slices), then the type head
    const ELT *mw = (const ELT *)a.mix_w, *kw = (const ELT *)a.k2_w;
    for (int i = tid; i < NH * D; i += blockDim.x) {
      const int n = i / D, k = i - n * D;
      hb[4 * D * D + wt(k, n, NH)] = n < 3 * M ? mw[(size_t)n * D + k] : kw[(size_t)(n - 3 * M) * D + k];
    }
    auto cp = [&](float *dst, const float *src, int cnt) {
      for (int i = tid; i < cnt; i += blockDim.x) dst[i] = src[i];
    };
    for (int ly = 0; ly < L; ++ly) {
      const FusedLayerW &w = a.layer[ly];
      float *v = vec + ly * (9 * D + F);
      cp(v, w.ln1_g, D);
      cp(v + D, w.ln1_b, D);
      cp(v + 2 * D, w.qkv_b, 3 * D);
      cp(v + 5 * D, w.out_b, D);
      cp(v + 6 * D, w.ln2_g, D);
      cp(v + 7 * D, w.ln2_b, D);
      cp(v + 8 * D, w.ffn1_b, F);
      cp(v + 8 * D + F, w.ffn2_b, D);
    }
    float *v = vec + L * (9 * D + F);
    cp(v, a.lnf_g, D);
    cp(v + D, a.lnf_b, D);
    cp(v + 2 * D, a.k1_b, D);
    cp(v + 3 * D, a.mix_b, 3 * M);
    cp(v + 3 * D + 3 * M, a.k2_b, K);
    cp(v + 3 * D + 3 * M + K, a.freq, D);
  }
  __syncthreads();   // the only workgroup barrier: waves are independent from here
  const int b = blockIdx.x * 4 + wave;
  if (b >= a.B || a.done[b]) return;
  const float *hvec = vec + L * (9 * D + F);
  const float *lnf_g = hvec, *lnf_b = hvec + D, *k1_b = hvec + 2 * D, *mix_b = hvec + 3 * D,
              *k2_b = hvec + 3 * D + 3 * M, *freq = hvec + 3 * D + 3 * M + K;
  // per-wave scratch: token rows of 32 elements in slots of 32 floats; the
  // rows the products read are in the weights' element type
  using XT = typename std::conditional<sizeof(ELT) == 2, bf16_t, float>::type;
  float *xs = scr;                         // [2][32] residual stream
  XT *as = (XT *)(scr + 64);               // [2][32] LayerNorm output
  float *qs = scr + 128;                   // [2][32] queries
  XT *os = (XT *)(scr + 192);              // [2][32] attention output
  XT *hs = (XT *)(scr + 256);              // [2][F] FFN hidden
  XT *es = (XT *)(scr + 256 + 2 * F);      // [4D] decoder e | tanh
  float *hv = scr + 256 + 2 * F + 4 * D;   // [3M + K] decoder outputs
  auto gemv = [&](const ELT *W, int N, int KD, int P, auto xin, auto epi) {
    if (P == 2)
      wave_gemv<2>(W, N, KD, xin, epi);
    else
      wave_gemv<1>(W, N, KD, xin, epi);
  };
  const int n = a.n[b], base = a.lenD[b];
  const uint64_t r = (uint64_t)a.rnd[b];
  const size_t seq_row0 = (size_t)b * H * a.cap;
  const ELT *wtype = (const ELT *)a.type_emb;
  // the draws' uniforms: lane l - 1 holds step l's (Box-Muller epsilon in u[1])
  float u0 = 0.f, eps = 0.f, u3 = 0.f;
  if (lane < a.gamma) {
    float u[4];
    philox_uniforms(a.seed, (uint64_t)b, r, (uint64_t)(lane + 1), TAG_DRAFT, u);
    u0 = u[0];
    eps = sqrtf(-2.f * logf(u[1])) * cosf(6.28318530717958647692f * u[2]);
    u3 = u[3];
  }
  auto at = [](float v, int i) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i)); };
  float t_last = a.ev_t[(size_t)b * a.ev_stride + n - 1];
  float tok_t = 0.f;
  int tok_k = 0;
  // lane's token (p = lane / 32) and dimension (j = lane % 32) in the D-lane layout
  const int lp = lane >> 5, lj = lane & 31;
  for (int l = 1; l <= a.gamma; ++l) {
    const int P = (l == 1) ? 2 : 1;
    const int pos0 = (l == 1) ? base : base + l;
    // ---- embedding
    {
      float t;
      int k;
      if (l == 1) {
        const size_t i = (size_t)b * a.ev_stride + n - 2 + lp;
        t = a.ev_t[i];
        k = a.ev_k[i];
      } else {
        t = tok_t;
        k = tok_k;
      }
      if (lj < D && lp < P) {
        const float arg = t * freq[lj];
        const int kk = min(max(k, 0), K - 1);
        xs[lp * 32 + lj] = ((lj & 1) ? cosf(arg) : sinf(arg)) + ld(wtype, (size_t)kk * D + lj);
      }
    }
    wave_lds_sync();
    for (int ly = 0; ly < L; ++ly) {
      const ELT *wq = wl + (size_t)ly * LW, *wo = wq + 3 * D * D, *w1 = wq + 4 * D * D, *w2 = w1 + D * F;
      const float *lv = vec + ly * (9 * D + F);
      ELT *kc = (ELT *)(a.kc + a.layer_bytes * ly);
      ELT *vc = (ELT *)(a.vc + a.layer_bytes * ly);
      // LayerNorm of each token over its D lanes
      auto layernorm = [&](const float *g, const float *bt, XT *dst, int np) {
        const float xv = (lj < D && lp < np) ? xs[lp * 32 + lj] : 0.f;
        const float mean = group_sum(xv, 32) / (float)D;
        const float c = (lj < D) ? xv - mean : 0.f;
        const float rstd = 1.f / sqrtf(group_sum(c * c, 32) / (float)D + 1e-5f);
        if (lj < D && lp < np) st<XT>(dst, lp * 32 + lj, rnd_act<ELT>(c * rstd * g[lj] + bt[lj]));
        wave_lds_sync();
      };
      layernorm(lv, lv + D, as, P);
      // q, k, v; keys and values of positions pos0 .. pos0 + P - 1 into the cache
      gemv(wq, 3 * D, D, P, [&](int, int p) { return (const XT *)(as + p * 32); },
                     [&](int p, int nn, float acc) {
                       const float v = rnd_act<ELT>(acc + lv[2 * D + nn]);
                       const int which = nn / D, c = nn - which * D;
                       if (which == 0) {
                         qs[p * 32 + c] = v;
                       } else {
                         const int hh = c / DH, j = c - hh * DH, pos = pos0 + p;
                         const size_t row0 = seq_row0 + (size_t)hh * a.cap;
                         if (pos < a.cap)
                           st(which == 1 ? kc : vc, which == 1 ? (row0 + pos) * DH + j : v_at<ELT>(row0, pos, j, DH), v);
                         else
                           atomicOr(a.status, TPPSD_STATUS_CAPACITY);
                       }
                     });
      __threadfence_block();   // this wave's cache stores before its reads below
      wave_lds_sync();
      // ---- attention: head hh on lanes [hh * 64 / H, (hh + 1) * 64 / H); a lane
      // takes units of 2 positions (the unit's key rows, and for bf16 its two
      // positions of the position-blocked value block, for fp32 its value rows); one
      // query at a time (two only in the first step), so that a unit, the
      // query and its running output fit beside each other in registers
      for (int p = 0; p < P; ++p) {
        constexpr int LPH = 64 / H, U = 2;
        constexpr int NKV = U * DH * (int)sizeof(ELT) / 16;   // 16-byte vectors of a unit's keys
        const int hh = lane / LPH, sub = lane - hh * LPH;
        const int n_keys = min(pos0 + P, a.cap), last = pos0 + p;
        const size_t row0 = seq_row0 + (size_t)hh * a.cap;
        float q[DH];
#pragma unroll
        for (int j = 0; j < DH; ++j) q[j] = qs[p * 32 + hh * DH + j] * 0.25f;   // 1 / sqrt(16)
        // bf16: the scaled query (bf16 values times a power of two) as pairs
        // for v_dot2c against the raw key words
        uint32_t qw[sizeof(ELT) == 2 ? DH / 2 : 1];
        if constexpr (sizeof(ELT) == 2) {
#pragma unroll
          for (int e = 0; e < DH / 2; ++e) qw[e] = pk2bf(q[2 * e], q[2 * e + 1]);
        }
        float m = -INFINITY, lsum = 0.f, o[DH];
#pragma unroll
        for (int j = 0; j < DH; ++j) o[j] = 0.f;
        for (int u = sub; u * U < n_keys; u += LPH) {
          const int k0 = u * U;   // inside the slab (rounded up to 8 positions); slots past n_keys masked
          uint4 kr[NKV];
          uint32_t vr1[sizeof(ELT) == 2 ? 16 : 1];
          uint4 vr4[sizeof(ELT) == 2 ? 1 : NKV];
          const uint4 *kp = (const uint4 *)(kc + (row0 + k0) * DH);
#pragma unroll
          for (int i = 0; i < NKV; ++i) kr[i] = kp[i];
          if constexpr (sizeof(ELT) == 2) {
            // the unit's two positions of each value column's 8-position block
            const bf16_t *vb = (const bf16_t *)vc + v_at<bf16_t>(row0, k0 & ~7, 0, DH) + (k0 & 6);
#pragma unroll
            for (int j = 0; j < 16; ++j) vr1[j] = *(const uint32_t *)(vb + 8 * j);
          } else {
            const uint4 *vp = (const uint4 *)(vc + (row0 + k0) * DH);
#pragma unroll
            for (int i = 0; i < NKV; ++i) vr4[i] = vp[i];
          }
          // element (key i, column j) of the unit's keys and values
          auto kval = [&](int i, int j) -> float {
            if constexpr (sizeof(ELT) == 2) {
              const uint4 w = kr[2 * i + (j >> 3)];
              const int e = (j & 7) >> 1;
              const uint32_t x = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
              return (j & 1) ? __uint_as_float(x & 0xFFFF0000u) : __uint_as_float(x << 16);
            } else {
              const uint4 w = kr[4 * i + (j >> 2)];
              const int e = j & 3;
              return __uint_as_float(e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w);
            }
          };
          auto vval = [&](int i, int j) -> float {
            if constexpr (sizeof(ELT) == 2) {
              const uint32_t x = vr1[j];
              return (i & 1) ? __uint_as_float(x & 0xFFFF0000u) : __uint_as_float(x << 16);
            } else {
              const uint4 w = vr4[4 * i + (j >> 2)];
              const int e = j & 3;
              return __uint_as_float(e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w);
            }
          };
          float sc[U], mx = -INFINITY;
#pragma unroll
          for (int i = 0; i < U; ++i) {
            float dot = 0.f;
            if constexpr (sizeof(ELT) == 2) {
#pragma unroll
              for (int hv = 0; hv < 2; ++hv) {
                const uint4 w = kr[2 * i + hv];   // columns 8 hv .. 8 hv + 7 of key i
                dot = dot2_bf(w.x, qw[4 * hv], dot);
                dot = dot2_bf(w.y, qw[4 * hv + 1], dot);
                dot = dot2_bf(w.z, qw[4 * hv + 2], dot);
                dot = dot2_bf(w.w, qw[4 * hv + 3], dot);
              }
            } else {
#pragma unroll
              for (int j = 0; j < DH; ++j) dot += q[j] * kval(i, j);
            }
            sc[i] = (k0 + i < n_keys && k0 + i <= last) ? dot : -INFINITY;
            mx = fmaxf(mx, sc[i]);
          }
          const float mn = fmaxf(m, mx);
          const float al = (mn == -INFINITY) ? 1.f : expf(m - mn);
          lsum *= al;
#pragma unroll
          for (int j = 0; j < DH; ++j) o[j] *= al;
#pragma unroll
          for (int i = 0; i < U; ++i) {
            // masked slots hold unwritten or stale values: skipped, not weighted by 0
            if (sc[i] == -INFINITY) continue;
            const float e = expf(sc[i] - mn);
            lsum += e;
#pragma unroll
            for (int j = 0; j < DH; ++j) o[j] += e * vval(i, j);
          }
          m = mn;
        }
        // merge the head's lanes: maximum, rescaled sums, and the 16 column
        // sums by recursive halving (lane ends with column c of its group)
        float M_ = m;
        M_ = fmaxf(M_, dpp_mov<0xB1>(M_));
        M_ = fmaxf(M_, dpp_mov<0x4E>(M_));
        M_ = fmaxf(M_, swz_xor<4>(M_));
        M_ = fmaxf(M_, swz_xor<8>(M_));
        M_ = fmaxf(M_, swz_xor<16>(M_));
        if (LPH == 64) M_ = fmaxf(M_, __shfl_xor(M_, 32, 64));
        const float f = (m == -INFINITY) ? 0.f : expf(m - M_);
        const float lw = group_sum(lsum * f, LPH);
        float ow[16];
#pragma unroll
        for (int j = 0; j < DH; ++j) ow[j] = o[j] * f;
        if (LPH == 64) {
#pragma unroll
          for (int j = 0; j < DH; ++j) ow[j] += __shfl_xor(ow[j], 32, 64);
        }
        halve_step<8>(ow, (lane & 16) != 0, [](float v) { return swz_xor<16>(v); });
        halve_step<4>(ow, (lane & 8) != 0, [](float v) { return swz_xor<8>(v); });
        halve_step<2>(ow, (lane & 4) != 0, [](float v) { return swz_xor<4>(v); });
        halve_step<1>(ow, (lane & 2) != 0, [](float v) { return dpp_mov<0x4E>(v); });
        const float oc = ow[0] + dpp_mov<0xB1>(ow[0]);
        const int c = 8 * ((lane >> 4) & 1) + 4 * ((lane >> 3) & 1) + 2 * ((lane >> 2) & 1) + ((lane >> 1) & 1);
        if ((lane & 1) == 0 && (LPH == 32 || lane < 32)) st<XT>(os, p * 32 + hh * DH + c, rnd_act<ELT>(lw > 0.f ? oc / lw : 0.f));
      }
      wave_lds_sync();
      // output projection + residual
      gemv(wo, D, D, P, [&](int, int p) { return (const XT *)(os + p * 32); },
                     [&](int p, int nn, float acc) { xs[p * 32 + nn] += acc + lv[5 * D + nn]; });
      wave_lds_sync();
      layernorm(lv + 6 * D, lv + 7 * D, as, P);
      gemv(w1, F, D, P, [&](int, int p) { return (const XT *)(as + p * 32); },
                     [&](int p, int nn, float acc) { st<XT>(hs, p * F + nn, rnd_act<ELT>(fmaxf(acc + lv[8 * D + nn], 0.f))); });
      wave_lds_sync();
      gemv(w2, D, F, P, [&](int, int p) { return (const XT *)(hs + p * F); },
                     [&](int p, int nn, float acc) { xs[p * 32 + nn] += acc + lv[8 * D + F + nn]; });
      wave_lds_sync();
    }
    // ---- decoder on the last token
    {
      const int pl = P - 1;
      const float xv = (lj < D && lp == 0) ? xs[pl * 32 + lj] : 0.f;
      const float mean = group_sum(xv, 32) / (float)D;
      const float c = (lj < D) ? xv - mean : 0.f;
      const float rstd = 1.f / sqrtf(group_sum(c * c, 32) / (float)D + 1e-5f);
      if (lj < D && lp == 0) st<XT>(as, lj, rnd_act<ELT>(c * rstd * lnf_g[lj] + lnf_b[lj]));
      wave_lds_sync();
    }
    const ELT *we = wl + (size_t)L * LW, *wh = we + 4 * D * D;
    gemv(we, 4 * D, D, 1, [&](int, int) { return (const XT *)as; },
                   [&](int, int nn, float acc) {
                     st<XT>(es, nn, (nn < 3 * D) ? rnd_act<ELT>(acc) : rnd_act<ELT>(tanhf(acc + k1_b[nn - 3 * D])));
                   });
    wave_lds_sync();
    gemv(wh, NH, D, 1, [&](int nn, int) { return (const XT *)(es + (nn < 3 * M ? nn / M : 3) * D); },
                   [&](int, int nn, float acc) { hv[nn] = acc + (nn < 3 * M ? mix_b[nn] : k2_b[nn - 3 * M]); });
    wave_lds_sync();
    {
      // the log-softmaxes, the draft record, and the draft event
      const float lw = lane < M ? hv[lane] : -INFINITY;
      const float mu_l = lane < M ? hv[M + lane] : 0.f, s_l = lane < M ? hv[2 * M + lane] : 0.f;
      const float lk = lane < K ? hv[3 * M + lane] : -INFINITY;
      const float mw2 = wave_max(lw);
      const float sw = wave_sum(lane < M ? expf(lw - mw2) : 0.f);
      const float mk = wave_max(lk);
      const float sk = wave_sum(lane < K ? expf(lk - mk) : 0.f);
      const float nlw = lw - mw2 - logf(sw), nlk = lk - mk - logf(sk);
      const size_t di = (size_t)b * a.MG + (l - 1);
      if (lane < M) {
        a.d_mix[di * 3 * M + lane] = nlw;
        a.d_mix[di * 3 * M + M + lane] = mu_l;
        a.d_mix[di * 3 * M + 2 * M + lane] = s_l;
      }
      if (lane < K) a.d_logtype[di * K + lane] = nlk;
      auto draw = [&](float lp_, int cnt, float u) {
        float cs = lane < cnt ? expf(lp_) : 0.f;
        cs = wave_cumsum(cs);
        const float tot = lane_val(cs, cnt - 1);
        const unsigned long long hit = __ballot(lane < cnt && u * tot < cs);
        return hit ? (int)__builtin_ctzll(hit) : cnt - 1;
      };
      const int z = draw(nlw, M, at(u0, l - 1));
      const float tau = expf(at(mu_l, z) + expf(at(s_l, z)) * at(eps, l - 1));
      const int kk = draw(nlk, K, at(u3, l - 1));
      const float lt = logf(tau);
      float cterm = -INFINITY;
      if (lane < M) {
        const float zz = lt - mu_l;
        cterm = nlw - s_l - 0.918938533204672742f - lt - 0.5f * zz * zz * expf(-2.f * s_l);
      }
      const float cm = wave_max(cterm);
      const float lg = cm + logf(wave_sum(lane < M ? expf(cterm - cm) : 0.f));
      const float lf = at(nlk, kk);
      const float tn = t_last + tau;
      if (lane == 0) {
        a.d_tau[di] = tau;
        a.d_t[di] = tn;
        a.d_k[di] = kk;
        a.d_logg[di] = lg;
        a.d_logf[di] = lf;
        if (!isfinite(tau)) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
      }
      tok_t = tn;
      tok_k = kk;
      t_last = tn;
    }
    wave_lds_sync();
  }
}

bool wave_draft_ok(int L, int d, int H, int F, int M, int K, int bf16) {
  const bool shape = L <= 2 && H >= 1 && d == 16 * H && (d == 16 || d == 32) && (F == 2 * d || F == 4 * d) &&
                     3 * M + K <= 128 && M <= 64 && K <= 64;
  return shape && wave_draft_lds_bytes(L, d, F, M, K, bf16 ? 2 : 4) <= 128 * 1024;
}

void launch_draft_wave(const DraftArgs &a, int bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const size_t lds = wave_draft_lds_bytes(a.L, a.d, a.F, a.M, a.K, bf16 ? 2 : 4);
  auto go = [&](auto kern) {
    hipExtLaunchKernelGGL(kern, dim3((a.B + 3) / 4), dim3(256), lds, s, ev0, ev1, 0, a);
  };
#define TPPSD_DW(ELT)                                                  \
  if (a.d == 16) {                                                     \
    if (a.F == 32) go(k_draft_wave<ELT, 16, 32, 1>);                   \
    else go(k_draft_wave<ELT, 16, 64, 1>);                             \
  } else {                                                             \
    if (a.F == 64) go(k_draft_wave<ELT, 32, 64, 2>);                   \
    else go(k_draft_wave<ELT, 32, 128, 2>);                            \
  }
  if (bf16) {
    TPPSD_DW(bf16_t)
  } else {
    TPPSD_DW(float)
  }
#undef TPPSD_DW
}

int allow_draft_wave_lds(size_t bytes) {
  int bad = 0;
  auto set = [&](auto kern) {
    bad |= hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) !=
           hipSuccess;
  };
  set(k_draft_wave<bf16_t, 16, 32, 1>), set(k_draft_wave<bf16_t, 16, 64, 1>);
  set(k_draft_wave<bf16_t, 32, 64, 2>), set(k_draft_wave<bf16_t, 32, 128, 2>);
  set(k_draft_wave<float, 16, 32, 1>), set(k_draft_wave<float, 16, 64, 1>);
  set(k_draft_wave<float, 32, 64, 2>), set(k_draft_wave<float, 32, 128, 2>);
  return bad;
}

// ---------------------------------------------------------------------------
// Fused row block for small THP models (§4.2 Encoder and Decoder): between
// two attention launches of a forward pass every step is row-local (output
// projection, residual, feed-forward block, LayerNorm, next q, k, v; or the
// decoder), so one launch runs them all over tiles of 16 rows, the rows
// staying in LDS. Each product is a 16-row MFMA tile product with the weights
// read from global memory (a few hundred KB: L2-resident). The rounding points
// are those of the layered kernels.
// ---------------------------------------------------------------------------

// The weights one wave needs for a 16-row product Y = X W^T (W [N][K]
// row-major): its 16-column tiles wave, wave + nw, ..., at most TPW of them
// (the callers only take shapes where this covers every tile), and of each tile
// lane group kq = lane / 16's k range [kq K/4, (kq + 1) K/4) -- a
// permutation of the MFMA's k slots under which a lane's share of a weight
// row is contiguous. Loaded one step ahead of the product that uses it, so
// that the load latency overlaps the step before.
template <typename ELT, int K, int TPW> struct WBatch {
  static constexpr int SEG = K / 4;                           // k per lane group
  static constexpr int TPB = TPW;                             // column tiles per wave
  static constexpr int NV = SEG * (int)sizeof(ELT) / 16;      // 16-byte vectors per tile
  static_assert(NV >= 1 && SEG * sizeof(ELT) % 16 == 0, "K too small for the lane-group split");
  uint4 w[TPB][NV];
  // W in the packed order of k_pack_wbatch: tile t's vector i for lane l at
  // ((t NV + i) 64 + l) 16 bytes, so each load instruction of a wave reads 1 KB
  // of contiguous memory (tiles past the matrix clamped; results unused)
  __device__ __forceinline__ void load(const ELT *__restrict__ W, int N) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int last = (N + 15) / 16 - 1;
#pragma unroll
    for (int j = 0; j < TPB; ++j) {
      const int t = min(wave + j * nw, last);
      const uint4 *wr = (const uint4 *)W + (size_t)t * NV * 64 + lane;
#pragma unroll
      for (int i = 0; i < NV; ++i) w[j][i] = wr[i * 64];
    }
  }
};

// W [N][K] into the WBatch order: 16-row tile t, lane l = 16 kq + r holds
// row 16 t + r (clamped to N - 1), k segment kq K/4 .. + K/4, as K/4 * elt / 16
// consecutive 16-byte vectors i stored at ((t NV + i) 64 + l) 16 bytes
template <typename ELT>
__global__ void k_pack_wbatch(const ELT *__restrict__ W, int N, int K, ELT *__restrict__ out) {
  const int NV = (K / 4) * (int)sizeof(ELT) / 16, VE = 16 / (int)sizeof(ELT);
  const int tiles = (N + 15) / 16, total = tiles * NV * 64;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int l = idx & 63, ti = idx >> 6, t = ti / NV, i = ti - t * NV;
  const int n = min(16 * t + (l & 15), N - 1), kq = l >> 4;
  *(uint4 *)(out + (size_t)idx * VE) = *(const uint4 *)(W + (size_t)n * K + kq * (K / 4) + i * VE);
}

size_t wbatch_packed_elems(int N, int K) { return (size_t)(N + 15) / 16 * 16 * K; }

void launch_pack_wbatch(const void *W, int N, int K, int bf16, void *out, hipStream_t s) {
  const int NV = (K / 4) * (bf16 ? 2 : 4) / 16, total = (N + 15) / 16 * NV * 64;
  if (bf16)
    k_pack_wbatch<bf16_t><<<(total + 255) / 256, 256, 0, s>>>((const bf16_t *)W, N, K, (bf16_t *)out);
  else
    k_pack_wbatch<float><<<(total + 255) / 256, 256, 0, s>>>((const float *)W, N, K, (float *)out);
}

// Y[16 x N] = X[16 x K] W^T with X in LDS (fp32 values, row stride ldx) and
// the wave's weights in wb; epi(r, n, y) for r < 16, n < N, each element by
// one lane. Independent accumulators are interleaved (the tiles, or for a
// single tile four partial sums over k) so that consecutive MFMAs never wait
// for each other's results.
template <typename ELT, int K, int TPW, typename EPI>
__device__ __forceinline__ void tile_mm16(const WBatch<ELT, K, TPW> &wb, int N, const float *X, int ldx, EPI epi) {
  typedef WBatch<ELT, K, TPW> WB;
  constexpr int SEG = WB::SEG, TPB = WB::TPB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int rr = lane & 15, kq = lane >> 4;
  const int ntiles = (N + 15) >> 4;
  const float *xr = X + rr * ldx + kq * SEG;
  constexpr int NA = TPB > 1 ? TPB : 4;
  f32x4_t acc[NA];
#pragma unroll
  for (int j = 0; j < NA; ++j) acc[j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  if constexpr (sizeof(ELT) == 4) {
    float xa[SEG];
#pragma unroll
    for (int i = 0; i < SEG; i += 4) {
      const float4 v = *(const float4 *)(xr + i);
      xa[i] = v.x; xa[i + 1] = v.y; xa[i + 2] = v.z; xa[i + 3] = v.w;
    }
    auto wv = [&](int j, int i) -> float {
      const uint4 u = wb.w[j][i >> 2];
      const uint32_t e = (i & 3) == 0 ? u.x : (i & 3) == 1 ? u.y : (i & 3) == 2 ? u.z : u.w;
      return __uint_as_float(e);
    };
    if constexpr (TPB > 1) {
#pragma unroll
      for (int i = 0; i < SEG; ++i)
#pragma unroll
        for (int j = 0; j < TPB; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[i], wv(j, i), acc[j], 0, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < SEG; ++i) acc[i & 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[i], wv(0, i), acc[i & 3], 0, 0, 0);
      acc[0] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
  } else {
    constexpr int NV = WB::NV;
    bf16x8_t xa[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)   // LDS values are already rounded to bf16
        w[e] = pk2bf(xr[8 * i + 2 * e], xr[8 * i + 2 * e + 1]);
      xa[i] = __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
    }
    if constexpr (TPB > 1) {
#pragma unroll
      for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int j = 0; j < TPB; ++j)
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[i], __builtin_bit_cast(bf16x8_t, wb.w[j][i]), acc[j], 0, 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < NV; ++i)
        acc[i & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[i], __builtin_bit_cast(bf16x8_t, wb.w[0][i]), acc[i & 3], 0, 0, 0);
      acc[0] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
  }
#pragma unroll
  for (int j = 0; j < TPB; ++j) {
    const int t = wave + j * nw;
    const int nc = t * 16 + rr;
    if (t < ntiles && nc < N)
#pragma unroll
      for (int v = 0; v < 4; ++v) epi(4 * kq + v, nc, acc[j][v]);
  }
}

// LayerNorm (biased variance, eps 1e-5) of the tile's rows, one wave per row;
// rows at or past nr are zero (they only feed discarded MFMA rows)
template <typename ELT>
__device__ __forceinline__ void tile_layernorm(const float *x, int ldx, float *y, int ldy, const float *g,
                                               const float *bt, int nr, int d) {
  // 16 lanes per row: a wave normalises 4 rows at once
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int sub = lane & 15;
  for (int r = 4 * wave + (lane >> 4); r < 16; r += 4 * nw) {
    float *yr = y + r * ldy;
    const float *xr = x + r * ldx;
    float s = 0.f;
    for (int j = sub; j < d; j += 16) s += xr[j];
    s += dpp_mov<0xB1>(s);    // lane ^ 1
    s += dpp_mov<0x4E>(s);    // lane ^ 2
    s += dpp_mov<0x124>(s);   // row_ror:4
    s += dpp_mov<0x128>(s);   // row_ror:8: every lane of the row holds the sum
    const float mean = s / (float)d;
    float v = 0.f;
    for (int j = sub; j < d; j += 16) {
      const float c = xr[j] - mean;
      v += c * c;
    }
    v += dpp_mov<0xB1>(v);    // lane ^ 1
    v += dpp_mov<0x4E>(v);    // lane ^ 2
    v += dpp_mov<0x124>(v);   // row_ror:4
    v += dpp_mov<0x128>(v);   // row_ror:8: every lane of the row holds the sum
    const float rstd = 1.f / sqrtf(v / (float)d + 1e-5f);
    for (int j = sub; j < d; j += 16) yr[j] = r < nr ? rnd_act<ELT>((xr[j] - mean) * rstd * g[j] + bt[j]) : 0.f;
  }
}

// floats of the small vectors k_block stages in LDS: out_b, LN2 (g, b),
// ffn1_b, ffn2_b, LN1 (g, b), qkv_b, LN_f (g, b), k1_b, decoder bias
inline __host__ __device__ int block_vec_floats(int d, int F, int M, int K) { return 13 * d + F + 3 * M + K; }

template <typename ELT, int D, int F, int NT>
__global__ __launch_bounds__(NT) void k_block(BlockArgs a) {
  constexpr int LX = D + 4, LH = (F > 4 * D ? F : 4 * D) + 4;
  // column tiles per wave (NT / 64 waves) of each product; the decoder's
  // 3M + K logits are at most 64 (64 / d) wide (block_fusable)
  constexpr int NW = NT / 64;
  constexpr int TO = (D / 16 + NW - 1) / NW, T1 = (F / 16 + NW - 1) / NW, TE = (4 * D / 16 + NW - 1) / NW,
                TH = ((D >= 64 ? 1 : 64 / D) * 4 + NW - 1) / NW;
  extern __shared__ __attribute__((aligned(16))) float sm[];
  __shared__ int row_b[16], row_pos[16];
  float *xs = sm;              // [16][LX] residual stream
  float *as = xs + 16 * LX;    // [16][LX] LayerNorm outputs / attention outputs
  float *hs = as + 16 * LX;    // [16][LH] FFN hidden / decoder e | tanh
  float *hv = hs + 16 * LH;    // [16][LV] decoder logits
  const int LV = 3 * a.M + a.K + 1;
  float *vec = hv + 16 * LV;   // staged small vectors
  float *out_b = vec, *ln2_g = out_b + D, *ln2_b = ln2_g + D, *ffn1_b = ln2_b + D, *ffn2_b = ffn1_b + F,
        *ln1_g = ffn2_b + D, *ln1_b = ln1_g + D, *qkv_b = ln1_b + D, *lnf_g = qkv_b + 3 * D, *lnf_b = lnf_g + D,
        *k1_b = lnf_b + D, *head_b = k1_b + D;
  const int tid = threadIdx.x, r0 = blockIdx.x * 16, nr = min(16, a.T - r0);
  // Phase 0: every global load of the launch's inputs is issued before any
  // LDS store (the compiler keeps a load after an earlier store it cannot
  // prove disjoint): the small vectors of the steps this launch runs, the
  // rows of x (or the tokens) and of the attention output; then each row's
  // sequence and cache position.
  constexpr int VMAX = (13 * D + F + 3 * 64 + 64 + NT - 1) / NT;   // vector floats per thread
  float vv[VMAX];
  {
    const float *seg_src[12] = {a.out_b, a.ln2_g, a.ln2_b, a.ffn1_b, a.ffn2_b, a.ln1_g,
                                a.ln1_b, a.qe.bias, a.lnf_g, a.lnf_b, a.k1_b, a.head_b};
    const int pre = a.pre, qk = a.qkv, hd = a.head;
    const int seg_len[12] = {pre * D, pre * D, pre * D, pre * F, pre * D, qk * D,
                             qk * D,  qk * 3 * D, hd * D, hd * D, hd * D, hd * (3 * a.M + a.K)};
    const int seg_off[12] = {0, D, 2 * D, 3 * D, 3 * D + F, 4 * D + F, 5 * D + F, 6 * D + F, 9 * D + F,
                             10 * D + F, 11 * D + F, 12 * D + F};
#pragma unroll
    for (int i = 0; i < VMAX; ++i) {
      const int idx = tid + NT * i;
      vv[i] = 0.f;
      for (int sgi = 0; sgi < 12; ++sgi) {
        const int o = idx - seg_off[sgi];
        if (o >= 0 && o < seg_len[sgi]) vv[i] = seg_src[sgi][o];
      }
    }
  }
  float4 xv = make_float4(0.f, 0.f, 0.f, 0.f);
  const int xr_ = tid / (D / 4), xc_ = tid - xr_ * (D / 4);   // one float4 of x per thread (16 D / 4 <= NT)
  if (!a.first && xr_ < nr) xv = *(const float4 *)(a.x + (size_t)(r0 + xr_) * D + 4 * xc_);
  constexpr int OV = 16 / sizeof(ELT);                          // o elements per 16-byte load
  uint4 ov = make_uint4(0u, 0u, 0u, 0u);
  const int or_ = tid / (D / OV), oc_ = tid - or_ * (D / OV);
  if (a.pre && or_ < 16 && or_ < nr) ov = *(const uint4 *)((const ELT *)a.o + (size_t)(r0 + or_) * D + OV * oc_);
  // the first product's weights (output projection, else the next q, k, v or
  // the decoder's [E; V_k1]) and the feed-forward block's first matrix, issued
  // after the row loads so that waiting for those does not wait for these
  WBatch<ELT, D, TE> w_a;
  WBatch<ELT, D, T1> w_f1;
  if (a.pre)
    w_a.load((const ELT *)a.out_w, D);
  else if (a.qkv)
    w_a.load((const ELT *)a.qkv_w, 3 * D);
  else
    w_a.load((const ELT *)a.Ek1_w, 4 * D);
  if (a.pre) w_f1.load((const ELT *)a.ffn1_w, F);
#pragma unroll
  for (int i = 0; i < VMAX; ++i)
    if (tid + NT * i < 12 * D + F + 3 * a.M + a.K + D) vec[tid + NT * i] = vv[i];
  if (a.qkv && tid < 16) {
    const int R = min(r0 + tid, a.T - 1), b = R / a.P;
    row_b[tid] = b;
    row_pos[tid] = a.qe.start[b] + a.qe.start_off + (R - b * a.P);
  }
  if (a.first) {
    for (int idx = tid; idx < 16 * D; idx += blockDim.x) {
      const int r = idx / D, j = idx - r * D;
      float v = 0.f;
      if (r < nr) {
        const int R = r0 + r, b = R / a.P, p = R - b * a.P;
        const TokSrc &src = a.src;
        float t;
        int k;
        if (p < src.n_ev) {
          const size_t i = (size_t)b * src.ev_stride + src.start[b] + src.start_off + p;
          t = src.ev_t[i];
          k = src.ev_k[i];
        } else {
          const size_t i = (size_t)b * src.dr_stride + src.dr_off + (p - src.n_ev);
          t = src.dr_t[i];
          k = src.dr_k[i];
        }
        k = min(max(k, 0), a.n_types - 1);
        const float arg = t * a.freq[j];
        v = ((j & 1) ? cosf(arg) : sinf(arg)) + ld((const ELT *)a.type_emb, (size_t)k * D + j);
      }
      xs[r * LX + j] = v;
    }
  } else if (xr_ < 16) {
    *(float4 *)(xs + xr_ * LX + 4 * xc_) = xv;
  }
  if (a.pre && or_ < 16) {
    float ovf[OV];
    if constexpr (sizeof(ELT) == 4) {
      ovf[0] = __uint_as_float(ov.x); ovf[1] = __uint_as_float(ov.y);
      ovf[2] = __uint_as_float(ov.z); ovf[3] = __uint_as_float(ov.w);
    } else {
      const uint32_t w[4] = {ov.x, ov.y, ov.z, ov.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ovf[2 * e] = __uint_as_float(w[e] << 16);
        ovf[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
      }
    }
#pragma unroll
    for (int e = 0; e < OV; ++e) as[or_ * LX + OV * oc_ + e] = ovf[e];
  }
  WBatch<ELT, D, TE> w_n;   // after the feed-forward block: the next q, k, v or [E; V_k1]
  if (a.pre) {
    lds_barrier();
    tile_mm16(w_a, D, as, LX, [&](int r, int n, float y) { xs[r * LX + n] += y + out_b[n]; });
    lds_barrier();
    WBatch<ELT, F, TO> w_f2;
    w_f2.load((const ELT *)a.ffn2_w, D);
    tile_layernorm<ELT>(xs, LX, as, LX, ln2_g, ln2_b, nr, D);
    lds_barrier();
    tile_mm16(w_f1, F, as, LX,
              [&](int r, int n, float y) { hs[r * LH + n] = rnd_act<ELT>(fmaxf(y + ffn1_b[n], 0.f)); });
    lds_barrier();
    if (a.qkv)
      w_n.load((const ELT *)a.qkv_w, 3 * D);
    else
      w_n.load((const ELT *)a.Ek1_w, 4 * D);
    tile_mm16(w_f2, D, hs, LH, [&](int r, int n, float y) { xs[r * LX + n] += y + ffn2_b[n]; });
  } else {
    w_n = w_a;
  }
  lds_barrier();
  if (a.store_x)
    for (int idx = tid; idx < nr * (D / 4); idx += blockDim.x) {
      const int r = idx / (D / 4), c = idx - r * (D / 4);
      *(float4 *)(a.x + (size_t)(r0 + r) * D + 4 * c) = *(const float4 *)(xs + r * LX + 4 * c);
    }
  if (a.qkv) {
    tile_layernorm<ELT>(xs, LX, as, LX, ln1_g, ln1_b, nr, D);
    lds_barrier();
    // q to its rows, keys and values appended to the cache (the EPI_QKV
    // arithmetic with the row's sequence and position from LDS)
    const Epi &e = a.qe;
    const int dh = e.dh, lg = dh == 16 ? 4 : (dh == 32 ? 5 : 6);
    tile_mm16(w_n, 3 * D, as, LX, [&](int r, int n, float y) {
      if (r >= nr) return;
      const float v = y + qkv_b[n];
      const int which = n / D, c = n - which * D;
      if (which == 0) {
        st((ELT *)e.q, (size_t)(r0 + r) * D + c, v);
      } else {
        const int pos = row_pos[r], h = c >> lg, j = c & (dh - 1);
        if (pos < e.cap) {
          const size_t row0 = ((size_t)row_b[r] * e.H + h) * e.cap;
          if (which == 1)
            st((ELT *)e.kc, (row0 + pos) * dh + j, v);
          else
            st((ELT *)e.vc, v_at<ELT>(row0, pos, j, dh), v);
        } else {
          atomicOr(e.status, TPPSD_STATUS_CAPACITY);
        }
      }
    });
  }
  if (a.head) {
    WBatch<ELT, 4 * D, TH> w_h;
    w_h.load((const ELT *)a.head_w, 3 * a.M + a.K);
    tile_layernorm<ELT>(xs, LX, as, LX, lnf_g, lnf_b, nr, D);
    lds_barrier();
    tile_mm16(w_n, 4 * D, as, LX, [&](int r, int n, float y) {
      hs[r * LH + n] = n < 3 * D ? rnd_act<ELT>(y) : rnd_act<ELT>(tanhf(y + k1_b[n - 3 * D]));
    });
    lds_barrier();
    tile_mm16(w_h, 3 * a.M + a.K, hs, LH, [&](int r, int n, float y) { hv[r * LV + n] = y + head_b[n]; });
    lds_barrier();
    const int wave = tid >> 6, nw = blockDim.x >> 6;
    for (int r = wave; r < nr; r += nw) {
      const int R = r0 + r, b = R / a.P, p = R - b * a.P;
      if (p >= a.h.p0) head_row(hv + r * LV, a.M, a.K, a.h, b, p);
    }
  }
}

bool block_widths(int d, int F) { return (d == 32 && (F == 64 || F == 128)) || (d == 64 && (F == 128 || F == 256)); }

bool block_fusable(int bf16, int d, int F, int M, int K, long T) {
  // instantiated widths; every product's column tiles fit one weight batch of
  // the four waves (16 (64 / (k / 4)) columns per wave, at least 16): the
  // decoder's 3M + K logits over k = 4d need 3M + K <= 4 * 16 * max(1, 64 / d)
  const bool widths = block_widths(d, F);
  // a launch streams a layer's matrices through each workgroup: worth it while
  // they are small, or, for larger ones (fp32 d = 64 / F = 256, 192 KB), over
  // many rows. Measured with the matrices in the packed order: the 704-row
  // verify pass of that model 122.9 -> 118.4 us, its 64-row AR step slower
  // than the layered kernels (586K -> 564K events/s)
  const size_t layer_bytes = (size_t)(4 * d * d + 2 * d * F) * (bf16 ? 2 : 4);
  return widths && 3 * M + K <= 64 * (d >= 64 ? 1 : 64 / d) && (layer_bytes <= 64 * 1024 || T >= 512);
}



void launch_block(const BlockArgs &a, int bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int LX = a.d + 4, LH = (a.F > 4 * a.d ? a.F : 4 * a.d) + 4, LV = 3 * a.M + a.K + 1;
  const size_t lds = ((size_t)16 * (2 * LX + LH + LV) + block_vec_floats(a.d, a.F, a.M, a.K)) * sizeof(float);
  const dim3 grid((a.T + 15) / 16);
  auto go = [&](auto kern, int nt) { hipExtLaunchKernelGGL(kern, grid, dim3(nt), lds, s, ev0, ev1, 0, a); };
  // eight waves, each holding half the column tiles that four would: the
  // products' serial MFMA chains per wave halve. Measured against four: the
  // 704-row fp32 verify pass at d = 64 / F = 256 106.6 vs 118.6 us per round,
  // the bf16 d = 32 / F = 128 draft step over 4096 sequences 369 vs 422 us per
  // round; sixteen waves slower again (112 us). TPPSD_BLOCK_NT=256 keeps four
  // (A/B measurement).
  const char *nte = getenv("TPPSD_BLOCK_NT");
  const int nt = nte && atoi(nte) == 256 ? 256 : 512;
#define TPPSD_BLK(ELT, D_, F_)                 \
  if (nt == 512)                               \
    go(k_block<ELT, D_, F_, 512>, 512);        \
  else                                         \
    go(k_block<ELT, D_, F_, 256>, 256);
#define TPPSD_BLKS(ELT)                                         \
  if (a.d == 32 && a.F == 64) { TPPSD_BLK(ELT, 32, 64) }         \
  else if (a.d == 32) { TPPSD_BLK(ELT, 32, 128) }                \
  else if (a.F == 128) { TPPSD_BLK(ELT, 64, 128) }               \
  else { TPPSD_BLK(ELT, 64, 256) }
  if (bf16) {
    TPPSD_BLKS(bf16_t)
  } else {
    TPPSD_BLKS(float)
  }
#undef TPPSD_BLKS
#undef TPPSD_BLK
}

// ---------------------------------------------------------------------------
// Per-sequence verify pass for small THP targets (§4.3 "Verification"): one
// 512-thread workgroup runs the target over one sequence's P = gamma + 1 new
// positions -- the pending event and the drafts -- through every layer and
// the decoder, with the verify epilogue per row. The P rows are one 16-row
// MFMA tile; q, the attention output and the stream stay in LDS, keys and
// values go to the cache and the attention reads them back from it (as the
// layered pass). Each product's weights are loaded one step ahead.
// ---------------------------------------------------------------------------
inline __host__ __device__ int verify_seq_vec_floats(int L, int d, int F, int M, int K) {
  return L * (9 * d + F) + 3 * d + 3 * M + K;
}

template <typename ELT, int D, int F>
__global__ __launch_bounds__(512) void k_verify_seq(VerifySeqArgs a) {
  constexpr int LX = D + 4, LH = (F > 4 * D ? F : 4 * D) + 4, DH = 16;
  // column tiles per wave (8 waves) of each product; the decoder's 3M + K
  // logits are at most 128 (64 / d) wide (verify_seq_ok)
  constexpr int TQ = (4 * D + 127) / 128, TO = (D + 127) / 128, T1 = (F + 127) / 128, TH = D >= 64 ? 1 : 64 / D;
  extern __shared__ __attribute__((aligned(16))) float sm[];
  __shared__ float tok_t[16];
  __shared__ int tok_k[16];
  const int LV = 3 * a.M + a.K + 1;
  float *xs = sm, *as = xs + 16 * LX, *qs = as + 16 * LX, *os = qs + 16 * LX;
  float *hs = os + 16 * LX;          // [16][LH] FFN hidden / decoder e | tanh
  float *hv = hs + 16 * LH;          // [16][LV] decoder logits
  float *red = hv + 16 * LV;         // attention merge: [8 waves][16 queries][DH + 2]
  float *vec = red + 8 * 16 * (DH + 2);
  const int tid = threadIdx.x, b = blockIdx.x, P = a.P, H = a.H;
  if (a.done[b]) return;
  const int pos0 = a.lenT[b];
  const size_t seq_row0 = (size_t)b * H * a.cap;
  // phase 0: the small vectors (per layer LN1 g, b, qkv_b, out_b, LN2 g, b,
  // ffn1_b, ffn2_b; then LN_f g, b, k1_b, decoder bias), the tokens, and the
  // first layer's q, k, v weights, all loads issued before any LDS store
  const int nvec = verify_seq_vec_floats(a.L, D, F, a.M, a.K);
  constexpr int VMAX = (FD_MAX_LAYERS * (9 * D + F) + 3 * D + 3 * 64 + 64 + 511) / 512;
  float vv[VMAX];
#pragma unroll
  for (int i = 0; i < VMAX; ++i) {
    int o = tid + 512 * i;
    vv[i] = 0.f;
    if (o < nvec) {
      const int per = 9 * D + F;
      if (o < a.L * per) {
        const int ly = o / per;
        o -= ly * per;
        const FusedLayerW &w = a.layer[ly];
        vv[i] = o < D ? w.ln1_g[o] : o < 2 * D ? w.ln1_b[o - D] : o < 5 * D ? w.qkv_b[o - 2 * D]
              : o < 6 * D ? w.out_b[o - 5 * D] : o < 7 * D ? w.ln2_g[o - 6 * D] : o < 8 * D ? w.ln2_b[o - 7 * D]
              : o < 8 * D + F ? w.ffn1_b[o - 8 * D] : w.ffn2_b[o - 8 * D - F];
      } else {
        o -= a.L * per;
        vv[i] = o < D ? a.lnf_g[o] : o < 2 * D ? a.lnf_b[o - D] : o < 3 * D ? a.k1_b[o - 2 * D] : a.head_b[o - 3 * D];
      }
    }
  }
  float tt = 0.f;
  int tk = 0;
  if (tid < P) {
    if (tid == 0) {   // the pending committed event
      const size_t i = (size_t)b * a.ev_stride + pos0;
      tt = a.ev_t[i];
      tk = a.ev_k[i];
    } else {          // draft tid - 1
      const size_t i = (size_t)b * a.dr_stride + tid - 1;
      tt = a.dr_t[i];
      tk = a.dr_k[i];
    }
  }
  WBatch<ELT, D, TQ> w_q;   // q, k, v (3D columns) or [E; V_k1] (4D)
  w_q.load((const ELT *)a.layer[0].qkv_w, 3 * D);
#pragma unroll
  for (int i = 0; i < VMAX; ++i)
    if (tid + 512 * i < nvec) vec[tid + 512 * i] = vv[i];
  if (tid < 16) {
    tok_t[tid] = tt;
    tok_k[tid] = min(max(tk, 0), a.K - 1);
  }
  lds_barrier();
  for (int idx = tid; idx < 16 * D; idx += blockDim.x) {
    const int r = idx / D, j = idx - r * D;
    float v = 0.f;
    qs[r * LX + j] = 0.f;   // rows past P stay zero
    os[r * LX + j] = 0.f;
    if (r < P) {
      const float arg = tok_t[r] * a.freq[j];
      v = ((j & 1) ? cosf(arg) : sinf(arg)) + ld((const ELT *)a.type_emb, (size_t)tok_k[r] * D + j);
    }
    xs[r * LX + j] = v;
  }
  lds_barrier();
  const float *hvec = vec + a.L * (9 * D + F);
  for (int ly = 0; ly < a.L; ++ly) {
    const FusedLayerW &w = a.layer[ly];
    const float *lv = vec + ly * (9 * D + F);
    const float *ln1_g = lv, *ln1_b = lv + D, *qkv_b = lv + 2 * D, *out_b = lv + 5 * D, *ln2_g = lv + 6 * D,
                *ln2_b = lv + 7 * D, *ffn1_b = lv + 8 * D, *ffn2_b = lv + 8 * D + F;
    ELT *kc = (ELT *)(a.kc + a.layer_bytes * ly), *vc = (ELT *)(a.vc + a.layer_bytes * ly);
    tile_layernorm<ELT>(xs, LX, as, LX, ln1_g, ln1_b, P, D);
    lds_barrier();
    tile_mm16(w_q, 3 * D, as, LX, [&](int r, int n, float y) {
      if (r >= P) return;
      const float v = rnd_act<ELT>(y + qkv_b[n]);
      const int which = n / D, c = n - which * D;
      if (which == 0) {
        qs[r * LX + c] = v;
      } else {
        const int pos = pos0 + r, h = c >> 4, j = c & 15;
        if (pos < a.cap)
          st(which == 1 ? kc : vc, which == 1 ? (seq_row0 + (size_t)h * a.cap + pos) * DH + j
                                                : v_at<ELT>(seq_row0 + (size_t)h * a.cap, pos, j, DH), v);
        else
          atomicOr(a.status, TPPSD_STATUS_CAPACITY);
      }
    });
    __syncthreads();   // the new keys and values are in the cache
    // (fp32 steps take twice the registers: two per load batch)
    wg_attention<ELT, DH, 16, sizeof(ELT) == 4 ? 2 : 4>(qs, os, kc, vc, seq_row0, a.cap, H, P, pos0, LX, red);
    // at most two weight batches live at a time (512 threads: 256 registers)
    WBatch<ELT, D, TO> w_o;
    w_o.load((const ELT *)w.out_w, D);
    lds_barrier();
    WBatch<ELT, D, T1> w_f1;
    w_f1.load((const ELT *)w.ffn1_w, F);
    tile_mm16(w_o, D, os, LX, [&](int r, int n, float y) { xs[r * LX + n] += y + out_b[n]; });
    lds_barrier();
    tile_layernorm<ELT>(xs, LX, as, LX, ln2_g, ln2_b, P, D);
    lds_barrier();
    WBatch<ELT, F, TO> w_f2;
    w_f2.load((const ELT *)w.ffn2_w, D);
    tile_mm16(w_f1, F, as, LX,
              [&](int r, int n, float y) { hs[r * LH + n] = rnd_act<ELT>(fmaxf(y + ffn1_b[n], 0.f)); });
    lds_barrier();
    tile_mm16(w_f2, D, hs, LH, [&](int r, int n, float y) { xs[r * LX + n] += y + ffn2_b[n]; });
    if (ly + 1 < a.L)
      w_q.load((const ELT *)a.layer[ly + 1].qkv_w, 3 * D);
    else
      w_q.load((const ELT *)a.Ek1_w, 4 * D);
    lds_barrier();
  }
  // decoder on every row: LN_f, [E; V_k1] with tanh, the block-diagonal heads
  tile_layernorm<ELT>(xs, LX, as, LX, hvec, hvec + D, P, D);
  lds_barrier();
  const float *k1_b = hvec + 2 * D, *head_b = hvec + 3 * D;
  WBatch<ELT, 4 * D, TH> w_h;
  w_h.load((const ELT *)a.head_w, 3 * a.M + a.K);
  tile_mm16(w_q, 4 * D, as, LX, [&](int r, int n, float y) {
    hs[r * LH + n] = n < 3 * D ? rnd_act<ELT>(y) : rnd_act<ELT>(tanhf(y + k1_b[n - 3 * D]));
  });
  lds_barrier();
  tile_mm16(w_h, 3 * a.M + a.K, hs, LH, [&](int r, int n, float y) { hv[r * LV + n] = y + head_b[n]; });
  lds_barrier();
  for (int r = tid >> 6; r < P; r += blockDim.x >> 6) head_row(hv + r * LV, a.M, a.K, a.h, b, r);
}

static size_t verify_seq_lds_bytes(int L, int d, int F, int M, int K) {
  const int LX = d + 4, LH = (F > 4 * d ? F : 4 * d) + 4, LV = 3 * M + K + 1;
  return ((size_t)16 * (4 * LX + LH + LV) + 8 * 16 * (16 + 2) + verify_seq_vec_floats(L, d, F, M, K)) * sizeof(float);
}

bool verify_seq_ok(int bf16, int L, int d, int H, int F, int M, int K, int P) {
  // instantiated widths, d_head 16, one 16-row tile, every product's column
  // tiles inside one weight batch of the eight waves, default LDS limit.
  // Taken for d = 32 (measured: the verify pass of the small fp32 workload
  // 59 -> 36 us per round). At d = 64 the gain measured 8 % of the pass, and
  // the layered pass keeps the verify attention a kernel of its own, whose
  // KV bandwidth is reported; d = 64 stays layered.
  const bool widths = d == 32 && (F == 64 || F == 128);
  (void)bf16;
  return widths && d == 16 * H && L <= FD_MAX_LAYERS && P <= 16 && 3 * M + K <= 128 * (d >= 64 ? 1 : 64 / d) &&
         verify_seq_lds_bytes(L, d, F, M, K) <= 64 * 1024;
}

void launch_verify_seq(const VerifySeqArgs &a, int B, int bf16, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const size_t lds = verify_seq_lds_bytes(a.L, a.d, a.F, a.M, a.K);
  auto go = [&](auto kern) { hipExtLaunchKernelGGL(kern, dim3(B), dim3(512), lds, s, ev0, ev1, 0, a); };
#define TPPSD_VS(ELT)                                               \
  if (a.d == 32 && a.F == 64) go(k_verify_seq<ELT, 32, 64>);        \
  else if (a.d == 32) go(k_verify_seq<ELT, 32, 128>);               \
  else if (a.F == 128) go(k_verify_seq<ELT, 64, 128>);              \
  else go(k_verify_seq<ELT, 64, 256>);
  if (bf16) {
    TPPSD_VS(bf16_t)
  } else {
    TPPSD_VS(float)
  }
#undef TPPSD_VS
}

// ---------------------------------------------------------------------------
// accept / reject, adjusted-distribution replacement and commit (§4.3,
// Eq. (3)-(4), Theorem 1, Algorithm 1). One workgroup per sequence: its four
// waves run the same per-sequence steps (their results agree lane for lane;
// wave 0 writes them), and share Theorem 1's candidates, 256 per step, so a
// long acceptance-rejection loop takes a quarter of the steps.
// ---------------------------------------------------------------------------

// value of v in lane i (i uniform across the wave)
__device__ __forceinline__ float lane_f(float v, int i) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}

__global__ __launch_bounds__(256) void k_accept(AcceptArgs a) {
  __shared__ float acc_pre[4][8 * 64];   // per wave: staged mixture terms (Theorem-1 loop)
  __shared__ int ar_win[4];              // per wave: its lowest accepted candidate (INT_MAX: none)
  __shared__ float ar_tau[4], ar_lg[4];  // ... and that candidate's tau and target log g
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool writer = threadIdx.x == 0;
  const int b = blockIdx.x;
  if (b >= a.B) return;
  const int G = a.gamma, MG = a.max_gamma, M = a.M, K = a.K;
  // every per-sequence scalar the kernel needs is loaded at once, and so is
  // the draft record of position lane (lane < G): the commit below reads it
  // from registers, so no load waits on another after this point except the
  // last committed time, which needs n
  const int is_done = a.done[b], rnd_b = a.rnd[b], n = a.n[b], gen = a.gen[b];
  const float T_end = a.t_end[b];
  float my_tau = 0.f, my_lg = 0.f, my_lf = 0.f, my_dg = 0.f, my_df = 0.f;
  int my_k = 0;
  if (lane < G) {
    const size_t i = (size_t)b * MG + lane;
    my_tau = a.d_tau[i];
    my_k = a.d_k[i];
    my_lg = a.v_logg[i];
    my_lf = a.v_logf[i];
    my_dg = a.d_logg[i];
    my_df = a.d_logf[i];
  }
  if (is_done) {
    if (writer) {
      a.L[b] = 0;
      a.n_new[b] = 0;
      a.flags[b] = 16;
      a.ar_iter[b] = -1;
    }
    return;
  }
  const float t_last = a.ev_t[(size_t)b * a.ev_stride + n - 1];
  const uint64_t r = (uint64_t)rnd_b;
  // verification tests: ln u < log p_T - log p_D for the interval and the
  // type, by wave 0; L and the two outcomes at L go to the other waves
  __shared__ int s_res[3];
  int pass_t = 1, pass_k = 1;
  if (wave == 0 && lane < G) {
    float ut, uk;
    if (a.uniforms) {
      ut = a.uniforms[((size_t)b * MG + lane) * 2];
      uk = a.uniforms[((size_t)b * MG + lane) * 2 + 1];
    } else {
      float u[4];
      philox_uniforms(a.seed, (uint64_t)b, r, (uint64_t)(lane + 1), TAG_ACCEPT, u);
      ut = u[0];
      uk = u[1];
    }
    pass_t = logf(ut) < my_lg - my_dg;
    pass_k = logf(uk) < my_lf - my_df;
  }
  if (wave == 0) {
    const uint64_t fail = __ballot(lane < G && !(pass_t && pass_k));
    const int L0 = fail ? __ffsll((unsigned long long)fail) : G + 1;
    // (the lane reads run on the whole wave, before the lane-0 branch)
    const int at0 = L0 <= G ? __builtin_amdgcn_readlane(pass_t, L0 - 1) : 1;
    const int ak0 = L0 <= G ? __builtin_amdgcn_readlane(pass_k, L0 - 1) : 1;
    if (lane == 0) {
      s_res[0] = L0;
      s_res[1] = at0;
      s_res[2] = ak0;
    }
  }
  __syncthreads();
  const int L = s_res[0], at = s_res[1], ak = s_res[2];
  // waves 1-3 only draw Theorem 1's candidates
  if (wave != 0 && !(L <= G && !at)) return;
  float tauL = 0.f;
  float lgL = 0.f, lfL = 0.f;   // target log g, log f of the event drawn at L (or the bonus event)
  int kL = 0, ar_j = -1, flags = 0;
  if (L <= G) {
    const int li = L - 1;
    const float *Tr = a.v_mix + ((size_t)b * (MG + 1) + li) * 3 * M;
    // g_D: the draft's mixture, or the exponential density of a
    // homogeneous-Poisson draft (App. D.3), log g_D = log rate - rate tau
    const bool pois = a.d_rate != nullptr;
    const float rate = pois ? a.d_rate[b] : 0.f;
    const float lrate = pois ? logf(rate) : 0.f;
    const float *Dr = pois ? nullptr : a.d_mix + ((size_t)b * MG + li) * 3 * M;
    if (!at) {
      // Theorem 1: candidates tau ~ g_T, accept iff u_a < 1 - exp(-(log g_T - log g_D));
      // candidate j = base + 64 wave + lane, the lowest accepted index wins.
      // Per component m each wave first stages, in LDS, the terms that do not
      // depend on tau: log w_m - log sigma_m - log sqrt(2 pi), exp(-2 log
      // sigma_m), mu_m, sigma_m for both mixtures and the running sum of w_m
      // of the target; each lane then evaluates its candidate from LDS.
      float *pre = acc_pre[threadIdx.x >> 6];
      float *Ta = pre, *Te = pre + 64, *Tm = pre + 128, *Ts = pre + 192, *Tc = pre + 256;
      float *Da = pre + 320, *De = pre + 384, *Dm = pre + 448;
      if (lane < M) {
        Ta[lane] = Tr[lane] - Tr[2 * M + lane] - 0.918938533204672742f;
        Te[lane] = expf(-2.f * Tr[2 * M + lane]);
        Tm[lane] = Tr[M + lane];
        Ts[lane] = expf(Tr[2 * M + lane]);
        if (!pois) {
          Da[lane] = Dr[lane] - Dr[2 * M + lane] - 0.918938533204672742f;
          De[lane] = expf(-2.f * Dr[2 * M + lane]);
          Dm[lane] = Dr[M + lane];
        }
      }
      float c = lane < M ? expf(Tr[lane]) : 0.f;
      c = wave_cumsum(c);
      if (lane < M) Tc[lane] = c;
      const float tot = lane_val(c, M - 1);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      auto logpdf = [&](const float *A, const float *E, const float *Mu, float lt) {
        float mx = -INFINITY;
        for (int m = 0; m < M; ++m) {
          const float z = lt - Mu[m];
          mx = fmaxf(mx, A[m] - lt - 0.5f * z * z * E[m]);
        }
        float acc = 0.f;
        for (int m = 0; m < M; ++m) {
          const float z = lt - Mu[m];
          acc += expf(A[m] - lt - 0.5f * z * z * E[m] - mx);
        }
        return mx + logf(acc);
      };
      for (int base = 0;; base += 256) {
        if (base >= TPPSD_AR_ITER_CAP) {
          if (writer) atomicOr(a.status, TPPSD_STATUS_AR_CAP);
          ar_j = TPPSD_AR_ITER_CAP;
          break;
        }
        float u[4];
        const int jw = 64 * wave + lane;   // this lane's candidate: base + jw
        philox_uniforms(a.seed, (uint64_t)b, r, (uint64_t)(base + jw), TAG_RES_T, u);
        const float x = u[0] * tot;
        int z = M - 1;
        for (int m = 0; m < M; ++m)
          if (x < Tc[m]) {
            z = m;
            break;
          }
        const float eps = sqrtf(-2.f * logf(u[1])) * cosf(6.28318530717958647692f * u[2]);
        const float tau = expf(Tm[z] + Ts[z] * eps);
        const float lt = logf(tau);
        const float lgd = pois ? lrate - rate * tau : logpdf(Da, De, Dm, lt);
        const float lgt = logpdf(Ta, Te, Tm, lt);
        const float delta = lgt - lgd;
        const bool acc = delta > 0.f && u[3] < -expm1f(-delta);
        // the lowest accepted index of the step wins: each wave posts its
        // first, then every wave reads the four (uniform across the group)
        const uint64_t m = __ballot(acc);
        const int jl = m ? __ffsll((unsigned long long)m) - 1 : 0;
        if (lane == 0) ar_win[wave] = m ? 64 * wave + jl : INT_MAX;
        if (m && lane == jl) {
          ar_tau[wave] = tau;
          ar_lg[wave] = lgt;
        }
        if (!m && wave == 3 && lane == 63) {   // the step's last candidate, kept if the cap ends the loop
          ar_tau[3] = tau;
          ar_lg[3] = lgt;
        }
        __syncthreads();
        const int best = min(min(ar_win[0], ar_win[1]), min(ar_win[2], ar_win[3]));
        const int bw = best == INT_MAX ? 3 : best >> 6;
        tauL = ar_tau[bw];
        lgL = ar_lg[bw];
        __syncthreads();   // read before the next step posts
        if (best != INT_MAX) {
          ar_j = base + best;
          break;
        }
      }
      flags |= 1;
    } else {
      tauL = lane_f(my_tau, li);
      lgL = lane_f(my_lg, li);
    }
    if (wave != 0) return;   // the rest is wave 0's
    if (!ak) {
      // Eq. (4): k ~ norm(max(0, f_T - f_D)), lane kk holding type kk
      float u[4];
      philox_uniforms(a.seed, (uint64_t)b, r, 0ull, TAG_RES_K, u);
      const float *lT = a.v_logtype + ((size_t)b * (MG + 1) + li) * K;
      const float *lD = a.d_logtype + ((size_t)b * MG + li) * K;
      const float lt_k = lane < K ? lT[lane] : 0.f;
      float c = lane < K ? fmaxf(0.f, expf(lt_k) - expf(lD[lane])) : 0.f;
      c = wave_cumsum(c);
      const float tot = lane_val(c, K - 1);
      const unsigned long long hit = __ballot(lane < K && u[0] * tot < c);
      kL = hit ? (int)__builtin_ctzll(hit) : K - 1;
      lfL = lane_f(lt_k, kL);
      flags |= 2;
    } else {
      // the draft's type, kept: its target log f is the verify pass's
      kL = __builtin_amdgcn_readlane(my_k, li);
      lfL = lane_f(my_lf, li);
    }
  } else if (a.bonus) {
    const float *Tr = a.v_mix + ((size_t)b * (MG + 1) + G) * 3 * M;
    float u[4];
    philox_uniforms(a.seed, (uint64_t)b, r, 0ull, TAG_BONUS, u);
    tauL = sample_tau(Tr, Tr + M, Tr + 2 * M, M, u[0], u[1], u[2]);
    kL = sample_cat(a.v_logtype + ((size_t)b * (MG + 1) + G) * K, K, u[3]);
    lgL = wave_mix_logpdf(Tr, Tr + M, Tr + 2 * M, M, tauL);
    lfL = a.v_logtype[((size_t)b * (MG + 1) + G) * K + kL];
    flags |= 4;
  }
  // commit in order: at most n_gen - gen events, and none past the end time
  // (Algorithm 1 samples while t < T and drops events with t > T; an event
  // exactly at T is kept and ends the sequence). Every lane runs the loop so
  // that the survival term below can use the whole wave; thread 0 writes.
  const int count = (L <= G) ? L : (a.bonus ? G + 1 : G);
  const int room = a.n_gen - gen;
  const bool last_is_new = (L <= G) || a.bonus;
  float tp = t_last;
  int nn = 0, stop_row = -1;
  bool stopped = false;
  float x_surv = 0.f;
  double ll = 0.0;
  for (int i = 0; i < count; ++i) {
    const bool is_new = i == count - 1 && last_is_new;
    const float ti = is_new ? tauL : lane_f(my_tau, i);
    const int ki = is_new ? kL : __builtin_amdgcn_readlane(my_k, i);
    const float tprev = tp;
    tp = tp + ti;
    const size_t oi = (size_t)b * (MG + 1) + i;
    if (writer) {
      a.t_new[oi] = tp;
      a.tau_new[oi] = ti;
      a.k_new[oi] = ki;
    }
    if (stopped || i >= room) continue;
    if (tp > T_end) {           // first event past the end time: dropped
      stopped = true;
      stop_row = i;
      x_surv = T_end - tprev;
      continue;
    }
    if (writer) {
      if (n + nn < a.ev_stride) {
        a.ev_t[(size_t)b * a.ev_stride + n + nn] = tp;
        a.ev_k[(size_t)b * a.ev_stride + n + nn] = ki;
      } else {
        atomicOr(a.status, TPPSD_STATUS_CAPACITY);
      }
    }
    // Eq. (2): the target's log-density of the committed event (verify row i)
    ll += is_new ? (double)lgL + (double)lfL : (double)lane_f(my_lg, i) + (double)lane_f(my_lf, i);
    ++nn;
    if (tp >= T_end) stopped = true;   // exactly at T: survival of a zero interval adds log 1
  }
  if (stop_row >= 0) {
    // survival log(1 - G(T - t_N)) under the distribution of the dropped event
    const float *Sr = a.v_mix + ((size_t)b * (MG + 1) + stop_row) * 3 * M;
    const bool v = lane < M;
    ll += (double)wave_log_survival(v ? Sr[lane] : 0.f, v ? Sr[M + lane] : 0.f, v ? Sr[2 * M + lane] : 0.f, v,
                                    x_surv);
  }
  if (!writer) return;
  if (last_is_new && !isfinite(tauL)) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
  const int n2 = n + nn, g2 = gen + nn;
  a.n[b] = n2;
  a.gen[b] = g2;
  a.lenT[b] = n2 - 1;
  a.lenD[b] = n2 - 2;
  a.rnd[b] = (int)r + 1;
  a.ll[b] += ll;
  if (g2 >= a.n_gen || stopped) {
    a.done[b] = 1;
    atomicAdd(a.n_done, 1);
    flags |= 8;
    if (stopped) flags |= 32;
  }
  a.L[b] = L;
  a.n_new[b] = nn;
  a.flags[b] = (uint8_t)flags;
  a.ar_iter[b] = ar_j;
  // per-sequence counters: this workgroup owns sequence b (a shared counter
  // updated by every wave serialises thousands of atomics on one address)
  unsigned long long *cs = a.acc_stats + 3 * (size_t)b;
  cs[0] += (unsigned long long)(L - 1);
  cs[1] += (unsigned long long)G;
  cs[2] += (unsigned long long)(ar_j >= 0 ? ar_j + 1 : 0);
}

// ---------------------------------------------------------------------------
// run setup and event copies
// ---------------------------------------------------------------------------

__global__ void k_prefill_init(const float *ht, const int32_t *hk, int B, int n0, int n_gen, const float *t_end_in,
                               float *ev_t, int32_t *ev_k, int ev_stride, int32_t *n, int32_t *gen, int32_t *lenT,
                               int32_t *lenD, int32_t *done, int32_t *rnd, int32_t *zeros, float *t_end,
                               double *ll, uint32_t *status, unsigned long long *acc_stats) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < B * n0) {
    const int b = idx / n0, i = idx - b * n0;
    ev_t[(size_t)b * ev_stride + i] = ht[idx];
    ev_k[(size_t)b * ev_stride + i] = hk[idx];
  }
  if (idx < B) {
    n[idx] = n0;
    gen[idx] = 0;
    lenT[idx] = n0 - 1;
    lenD[idx] = n0 - 2;
    // no end time: +inf. A pending event at or past the end time generates nothing
    const float te = t_end_in ? t_end_in[idx] : INFINITY;
    t_end[idx] = te;
    done[idx] = (n_gen <= 0 || ht[(size_t)idx * n0 + n0 - 1] >= te) ? 1 : 0;
    rnd[idx] = 0;
    zeros[idx] = 0;
    ll[idx] = 0.0;
    acc_stats[3 * idx] = acc_stats[3 * idx + 1] = acc_stats[3 * idx + 2] = 0ull;
  }
  if (idx == 0) *status = 0u;
}

// n_done = number of sequences done at the start (one workgroup)
__global__ __launch_bounds__(256) void k_count_done(const int32_t *done, int B, int32_t *n_done) {
  __shared__ int part[256];
  int c = 0;
  for (int i = threadIdx.x; i < B; i += 256) c += done[i] != 0;
  part[threadIdx.x] = c;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) part[threadIdx.x] += part[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *n_done = part[0];
}

__global__ void k_snapshot(const int32_t *src, int32_t *dst, int B) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < B) dst[i] = src[i];
}

__global__ void k_copy_events(const float *ev_t, const int32_t *ev_k, const int32_t *n, int B, int ev_stride,
                              float *t, int32_t *k, int32_t *nout) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < (size_t)B * ev_stride) {
    if (t) t[idx] = ev_t[idx];
    if (k) k[idx] = ev_k[idx];
  }
  if (nout && idx < (size_t)B) nout[idx] = n[idx];
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

void launch_embed(float *x, int T, int d, int P, const TokSrc &src, const void *wtype, int bf16,
                  const float *freq, int K, hipStream_t s) {
  const int threads = d >= 256 ? 256 : (d >= 128 ? 128 : 64);
  if (bf16)
    k_embed<bf16_t><<<T, threads, 0, s>>>(x, d, P, src, (const bf16_t *)wtype, freq, K);
  else
    k_embed<float><<<T, threads, 0, s>>>(x, d, P, src, (const float *)wtype, freq, K);
}

void launch_embed_attnhp(float *x, void *u, int T, int d, int P, const TokSrc &src, const void *wtype, int bf16,
                         const float *freq, int K, hipStream_t s) {
  const int threads = d >= 256 ? 256 : (d >= 128 ? 128 : 64);
  if (bf16)
    k_embed_attnhp<bf16_t><<<T, threads, 0, s>>>(x, (bf16_t *)u, d, P, src, (const bf16_t *)wtype, freq, K);
  else
    k_embed_attnhp<float><<<T, threads, 0, s>>>(x, (float *)u, d, P, src, (const float *)wtype, freq, K);
}

void launch_attnhp_update(float *x, const void *o, void *u, void *a, int bf16, int T, int d, hipStream_t s) {
  const size_t n = (size_t)T * d;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  if (bf16)
    k_attnhp_update<bf16_t><<<blocks, 256, 0, s>>>(x, (const bf16_t *)o, (bf16_t *)u, (bf16_t *)a, T, d);
  else
    k_attnhp_update<float><<<blocks, 256, 0, s>>>(x, (const float *)o, (float *)u, (float *)a, T, d);
}

void launch_layernorm(const float *x, void *y, int bf16, const float *g, const float *b, int T, int d,
                      hipStream_t s) {
  const int blocks = (T + 3) / 4;
  if (bf16)
    k_layernorm<bf16_t><<<blocks, 256, 0, s>>>(x, (bf16_t *)y, g, b, T, d);
  else
    k_layernorm<float><<<blocks, 256, 0, s>>>(x, (float *)y, g, b, T, d);
}

bool gemm_ln_fusable(int bf16, int K) {
  return K <= GEMM_LN_MAX_DEPTH * (bf16 ? gemm_bk<bf16_t>() : gemm_bk<float>());
}

// LayerNorm as a launch of its own ahead of a plain bf16 GEMM: for wide rows
// over many rows, where every 32 x 32 tile of the fused form reads and
// normalises all K fp32 columns of its rows again and the plain operand takes
// the direct-to-LDS GEMM. Measured on a verify pass of 544 rows of width 512
// (32 sequences x 17 positions, 8 layers): the fused q, k, v and FFN-in GEMMs
// took 15.5 and 16.3 us; LayerNorm (5.3 us) + plain GEMM brought the pass's
// GEMMs and LayerNorms from 438 to 399 us.
bool gemm_ln_split(int bf16, int d, int T) { return bf16 && d >= 512 && d % 128 == 0 && T >= 512; }

template <typename ELT>
static void gemm_dispatch(const void *X, const LnA *ln, const void *W, int T, int N, int K, const Epi &epi,
                          hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const ELT *x = (const ELT *)X, *w = (const ELT *)W;
  const float *xf = ln ? ln->x : nullptr, *lg = ln ? ln->g : nullptr, *lb = ln ? ln->b : nullptr;
  // 64 x 64 tiles when they give the chip a few hundred workgroups, 32 x 32
  // otherwise (the B rows of draft and AR steps)
  const bool big = (long)((N + 63) / 64) * ((T + 63) / 64) >= 256;
  auto go = [&](auto kern, int bm, int bn) {
    dim3 grid((N + bn - 1) / bn, (T + bm - 1) / bm);
    hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, ev0, ev1, 0, x, xf, lg, lb, w, T, N, K, epi);
  };
  if (!ln) {
    // bf16, a few hundred 64 x 64 tiles or fewer over at least 512 rows, K a
    // multiple of 128: direct-to-LDS ring of 32 x 32 x 128 stages (measured
    // faster there; the register ring keeps the very tall GEMMs)
    if (sizeof(ELT) == 2 && T >= 512 && K % 128 == 0 && (long)((N + 63) / 64) * ((T + 63) / 64) < 1024) {
      dim3 grid((N + 31) / 32, (T + 31) / 32);
      hipExtLaunchKernelGGL(k_gemm_dl<32, 32, 4, 3>, grid, dim3(256), 0, s, ev0, ev1, 0, (const bf16_t *)X,
                            (const bf16_t *)W, T, N, K, epi);
      return;
    }
    if (big) {
      go(k_gemm_lds<ELT, 64, 64, false, 2, 2>, 64, 64);
    } else {
      // 32 x 32 tiles: 8 k-steps per stage for a long K over few workgroups,
      // else 4 (more resident workgroups per CU)
      const long tiles = (long)((N + 31) / 32) * ((T + 31) / 32);
      if (K >= 512 && tiles < 512) go(k_gemm_lds<ELT, 32, 32, false, 2, 8>, 32, 32);
      else go(k_gemm_lds<ELT, 32, 32, false, 2, 4>, 32, 32);
    }
    return;
  }
  // LayerNorm operand: the ring holds all of K. 64 x 64 tiles with stages of
  // 2 k-steps (ring depth 2 or 4) when they fill the chip, else 32 x 32 tiles
  // with stages of 4 k-steps
  constexpr int KS = MfmaStep<ELT>::KSTEP;
  const int nst2 = (K + 2 * KS - 1) / (2 * KS), nst4 = (K + 4 * KS - 1) / (4 * KS);
  if (big && nst2 <= 4) {
    if (nst2 <= 2) go(k_gemm_lds<ELT, 64, 64, true, 2, 2>, 64, 64);
    else go(k_gemm_lds<ELT, 64, 64, true, 4, 2>, 64, 64);
  } else {
    if (nst4 <= 2) go(k_gemm_lds<ELT, 32, 32, true, 2, 4>, 32, 32);
    else go(k_gemm_lds<ELT, 32, 32, true, 4, 4>, 32, 32);
  }
}

bool layer_fused_ok(int bf16, int d, int F) { return bf16 && ((d == 128 && F == 512) || (d == 256 && F == 1024)); }

// Where the fused layer kernel is used by default: at d = 128 from 8192 rows
// (32-row tiles; measured at 36864 rows: verify pass 1121 -> 810 us) and up
// to 64 rows (one or two tiles replacing four launches: the 32-sequence
// draft, 1364 -> 1346 us per round), at d = 256 from 2048 rows (16-row
// tiles; at 2816 rows 501 -> 461 us; with 32-row tiles it only matched the
// layered GEMMs)
bool layer_fused_worth(int d, long T) { return d == 128 ? (T >= 8192 || T <= 64) : T >= 2048; }

void launch_layer_fused(const LayerArgs &a, int d, int F, bool post, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  auto go = [&](auto kern, int bm) {
    hipExtLaunchKernelGGL(kern, dim3((a.T + bm - 1) / bm), dim3(256), 0, s, ev0, ev1, 0, a);
  };
  // 32-row tiles: with the weights in fragment order, twice the workgroups
  // beat the halved weight traffic of 64-row tiles (36864 rows at d = 128:
  // 46 vs 58 us per layer; 64-row tiles on eight waves, each wave keeping the
  // four-wave kernel's share, 43.7 vs 40.3 us)
  if (d == 128 && F == 512) {
    if (post) go(k_layer_fused<128, 512, 32, 128, true, true>, 32);
    else go(k_layer_fused<128, 512, 32, 128, true, false>, 32);
  } else {
    if (post) go(k_layer_fused<256, 1024, 16, 64, true, true>, 16);
    else go(k_layer_fused<256, 1024, 16, 64, true, false>, 16);
  }
}

void launch_gemm(const void *X, const LnA *ln, const void *W, int bf16, int T, int N, int K, const Epi &epi,
                 hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (bf16)
    gemm_dispatch<bf16_t>(X, ln, W, T, N, K, epi, s, ev0, ev1);
  else
    gemm_dispatch<float>(X, ln, W, T, N, K, epi, s, ev0, ev1);
}

void launch_head(const float *logits, int ldl, int M, int K, const HeadArgs &a, hipStream_t s) {
  const int rows = a.B * (a.P - a.p0);
  k_head<<<(rows + 3) / 4, 256, 0, s>>>(logits, ldl, M, K, a);
}

void launch_build_head(const void *mix_w, const void *k2_w, const float *mix_b, const float *k2_b, int bf16, int d,
                       int M, int K, void *hw, float *hb, hipStream_t s) {
  if (bf16)
    k_build_head<bf16_t><<<3 * M + K, 256, 0, s>>>((const bf16_t *)mix_w, (const bf16_t *)k2_w, mix_b, k2_b, d, M,
                                                   K, (bf16_t *)hw, hb);
  else
    k_build_head<float><<<3 * M + K, 256, 0, s>>>((const float *)mix_w, (const float *)k2_w, mix_b, k2_b, d, M, K,
                                                  (float *)hw, hb);
}

void launch_accept(const AcceptArgs &a, hipStream_t s) { k_accept<<<a.B, 256, 0, s>>>(a); }

void launch_prefill_init(const float *ht, const int32_t *hk, int B, int n0, int n_gen, const float *t_end_in,
                         float *ev_t, int32_t *ev_k, int ev_stride, int32_t *n, int32_t *gen, int32_t *lenT,
                         int32_t *lenD, int32_t *done, int32_t *rnd, int32_t *zeros, float *t_end, double *ll,
                         int32_t *n_done, uint32_t *status, unsigned long long *acc_stats, hipStream_t s) {
  const int total = B * n0 > B ? B * n0 : B;
  k_prefill_init<<<(total + 255) / 256, 256, 0, s>>>(ht, hk, B, n0, n_gen, t_end_in, ev_t, ev_k, ev_stride, n, gen,
                                                     lenT, lenD, done, rnd, zeros, t_end, ll, status, acc_stats);
  k_count_done<<<1, 256, 0, s>>>(done, B, n_done);
}

void launch_snapshot(const int32_t *src, int32_t *dst, int B, hipStream_t s) {
  k_snapshot<<<(B + 255) / 256, 256, 0, s>>>(src, dst, B);
}

void launch_copy_events(const float *ev_t, const int32_t *ev_k, const int32_t *n, int B, int ev_stride, float *t,
                        int32_t *k, int32_t *nout, hipStream_t s) {
  const size_t total = (size_t)B * ev_stride;
  k_copy_events<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(ev_t, ev_k, n, B, ev_stride, t, k, nout);
}

}  // namespace tppsd
