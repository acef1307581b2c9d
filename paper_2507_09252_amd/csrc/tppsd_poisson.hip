// Homogeneous-Poisson draft model of TPP-SD (App. D.3): intervals are
// Exp(rate) and marks are drawn from fixed probabilities p, both maximum-
// likelihood estimates from observed sequences (rate = intervals / time
// span, p_m = share of events of type m). Unlike a Transformer draft, the
// gamma draws of a round are independent of each other, so the whole block
// is drawn at once: one wave per sequence, lane l holding draft position l.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tppsd_device.h"
#include "tppsd_philox.h"
#include "../../include/tppsd.h"

namespace tppsd {

// Fit over B sequences of n0 events (one workgroup): the span sum runs in
// float64 over per-thread partial sums, the type counts in LDS.
__global__ __launch_bounds__(256) void k_poisson_fit(const float *__restrict__ t, const int32_t *__restrict__ k,
                                                     int B, int n0, int K, float *__restrict__ params) {
  __shared__ double part[256];
  __shared__ unsigned int cnt[TPPSD_MAX_TYPES];
  const int tid = threadIdx.x;
  if (tid < TPPSD_MAX_TYPES) cnt[tid] = 0u;
  __syncthreads();
  double sp = 0.0;
  for (int b = tid; b < B; b += 256)
    sp += (double)t[(size_t)b * n0 + n0 - 1] - (double)t[(size_t)b * n0];
  const size_t total = (size_t)B * n0;
  for (size_t i = tid; i < total; i += 256) {
    const int kk = k[i];
    if (kk >= 0 && kk < K) atomicAdd(&cnt[kk], 1u);
  }
  part[tid] = sp;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) part[tid] += part[tid + h];
    __syncthreads();
  }
  if (tid < K) {
    unsigned long long all = 0ull;
    for (int m = 0; m < K; ++m) all += cnt[m];
    params[1 + tid] = cnt[tid] ? (float)log((double)cnt[tid] / (double)all) : -INFINITY;
  }
  if (tid == 0) params[0] = (float)((double)B * (double)(n0 - 1) / part[0]);
}

// Draft position l of sequence b uses the Philox counter (b, round, l + 1,
// DRAFT): tau = -ln(u_1) / rate (inverse of the exponential CDF) and k the
// first m with u_3 * C_K < C_m, C the running sum of p. Times accumulate in
// float32 in draft order from the pending event's time.
__global__ __launch_bounds__(256) void k_draft_poisson(PoissonDraftArgs a) {
  __shared__ float cdf[4][64];
  __shared__ float taus[4][TPPSD_MAX_GAMMA];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + w;
  if (b >= a.B || a.done[b]) return;
  const int G = a.gamma, K = a.K, MG = a.MG;
  const float rate = a.params[0];
  const float lp = lane < K ? a.params[1 + lane] : -INFINITY;
  float c = lane < K ? expf(lp) : 0.f;
  c = wave_cumsum(c);
  cdf[w][lane] = c;
  const float tot = lane_val(c, K - 1);
  // if rounding puts u_3 C_K at C_K, the last type of positive probability
  const unsigned long long pos = __ballot(lane < K && lp > -INFINITY);
  const int k_last = pos ? 63 - __builtin_clzll(pos) : K - 1;
  const uint64_t r = (uint64_t)a.rnd[b];
  float tau = 0.f;
  int k = 0;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < G) {
    float u[4];
    philox_uniforms(a.seed, (uint64_t)b, r, (uint64_t)(lane + 1), TAG_DRAFT, u);
    tau = -logf(u[1]) / rate;
    const float x = u[3] * tot;
    k = k_last;
    for (int m = 0; m < K; ++m)
      if (x < cdf[w][m]) {
        k = m;
        break;
      }
    taus[w][lane] = tau;
  }
  const float lf = __shfl(lp, k, 64);   // every lane takes part; lanes >= G read lane 0
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < G) {
    float tt = a.ev_t[(size_t)b * a.ev_stride + a.n[b] - 1];
    for (int i = 0; i <= lane; ++i) tt = tt + taus[w][i];
    const size_t o = (size_t)b * MG + lane;
    a.d_tau[o] = tau;
    a.d_t[o] = tt;
    a.d_k[o] = k;
    a.d_logg[o] = logf(rate) - rate * tau;
    a.d_logf[o] = lf;
    if (!isfinite(tau) || !isfinite(tt)) atomicOr(a.status, TPPSD_STATUS_NONFINITE);
  }
  if (lane < K)
    for (int l = 0; l < G; ++l) a.d_logtype[((size_t)b * MG + l) * K + lane] = lp;
  if (lane == 0) a.d_rate[b] = rate;
}

void launch_poisson_fit(const float *t, const int32_t *k, int B, int n0, int K, float *params, hipStream_t s) {
  k_poisson_fit<<<1, 256, 0, s>>>(t, k, B, n0, K, params);
}

void launch_draft_poisson(const PoissonDraftArgs &a, hipStream_t s) {
  k_draft_poisson<<<(a.B + 3) / 4, 256, 0, s>>>(a);
}

}  // namespace tppsd
