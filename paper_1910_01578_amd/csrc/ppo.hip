// Section 3 (Eq. 1, optimised with PPO): the clipped surrogate over the K
// sampled placements of every graph and its gradient with respect to the
// device logits, the first step of the update path's backward pass.
//
//   r[g,k]  = exp(logp[g,k] - logp_old[g,k])
//   L_g     = -(1/K) sum_k min(r A, clip(r, 1 - eps, 1 + eps) A)
//   c[g,k]  = dL/dlogp[g,k] for L = (1/G) sum_g L_g: -(r A) / (K G) where the
//             unclipped branch attains the min, 0 where the clipped constant does
//   dL/dlogits[v, j] = sum_k c[g(v),k] 1[p_kv = j] - softmax(logits_v)_j sum_k c[g(v),k]
//
// Two kernels: one work-group per graph forms c and L_g (a fixed-order sum);
// four lanes per node then walk its K placements.  Deterministic.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

__global__ __launch_bounds__(256) void k_ppo_coef(const float* __restrict__ logp, const float* __restrict__ logp_old,
                                                  const float* __restrict__ adv, int G, int K, float eps,
                                                  float* __restrict__ coef, float* __restrict__ loss) {
  __shared__ float red[256 / kWave];
  const int g = blockIdx.x;
  float part = 0.f;
  for (int k = threadIdx.x; k < K; k += 256) {
    const size_t i = (size_t)g * K + k;
    const float r = expf(logp[i] - logp_old[i]);
    const float a = adv[i];
    const float un = r * a;
    const float cl = fminf(fmaxf(r, 1.0f - eps), 1.0f + eps) * a;
    part += fminf(un, cl);
    coef[i] = un <= cl ? -un / ((float)K * (float)G) : 0.0f;
  }
  // work-group sum in a fixed order: each wave's butterfly, then the waves in index order
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) part += xor_shfl(part, off);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int w = 0; w < 256 / kWave; ++w) s += red[w];
    loss[g] = -s / (float)K;
  }
}

// Four lanes per node: lane q of node v walks samples q, q + 4, ... (loads
// coalesced over v for each k), eight at a time, and sums the chosen devices'
// coefficients for devices [jb, jb + 8); the four partial sums combine by a
// fixed butterfly.
constexpr int kPpoLanes = 4;
__global__ __launch_bounds__(256) void k_ppo_dlogits(const float* __restrict__ logits, const float* __restrict__ lse,
                                                     const int* __restrict__ placements, const float* __restrict__ coef,
                                                     GraphTable gt, int n, int D, int K, float* __restrict__ dlogits) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int v = t / kPpoLanes, q = t % kPpoLanes;
  const bool live = v < n;                      // whole 4-lane groups; every lane takes part in the shuffles
  const int vv = live ? v : n - 1;
  const int g = graph_of_node(gt, vv);
  const float* c = coef + (size_t)g * K;
  const float* row = logits + (size_t)vv * D;
  float lz;
  if (lse) {
    lz = lse[vv];
  } else {
    float m = -INFINITY;
    for (int j = 0; j < D; ++j) m = fmaxf(m, row[j]);
    float s = 0.f;
    for (int j = 0; j < D; ++j) s += expf(row[j] - m);
    lz = m + logf(s);
  }
  float csum = 0.f;
  for (int k = 0; k < K; ++k) csum += c[k];
  for (int jb = 0; jb < D; jb += 8) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k0 = q; k0 < K; k0 += 8 * kPpoLanes) {
      int p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + u * kPpoLanes;
        p[u] = k < K ? placements[(size_t)k * n + vv] - jb : -1;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + u * kPpoLanes;
        const float ck = k < K ? c[k] : 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += p[u] == e ? ck : 0.0f;
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] += xor_shfl(acc[e], 1);
      acc[e] += xor_shfl(acc[e], 2);
    }
    if (live && q == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = jb + e;
        if (j < D) dlogits[(size_t)v * D + j] = acc[e] - expf(row[j] - lz) * csum;
      }
    }
  }
}

hipError_t launch_ppo(const float* logits, const float* lse, const int* placements, const float* logp,
                      const float* logp_old, const float* adv, float eps, const GraphTable& gt, int n, int D, int K,
                      float* coef, float* loss, float* dlogits, hipStream_t s) {
  hipLaunchKernelGGL(k_ppo_coef, dim3(gt.n), dim3(256), 0, s, logp, logp_old, adv, gt.n, K, eps, coef, loss);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t threads = (int64_t)n * kPpoLanes;
  hipLaunchKernelGGL(k_ppo_dlogits, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, logits, lse, placements,
                     coef, gt, n, D, K, dlogits);
  return hipGetLastError();
}

}  // namespace gdp
