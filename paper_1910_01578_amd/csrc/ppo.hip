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
// Two kernels: one work-group per graph forms c, L_g and sum_k c[g,k] (fixed-
// order sums); four lanes per node then walk its K placements.  Deterministic.
#include "device_common.h"
#include "host_plan.h"
#include "kernels.h"

namespace gdp {

__global__ __launch_bounds__(256) void k_ppo_coef(const float* __restrict__ logp, const float* __restrict__ logp_old,
                                                  const float* __restrict__ adv, int G, int K, float eps,
                                                  float* __restrict__ coef, float* __restrict__ loss) {
  __shared__ float red[256 / kWave], redc[256 / kWave];
  const int g = blockIdx.x;
  float part = 0.f, cpart = 0.f;
  for (int k = threadIdx.x; k < K; k += 256) {
    const size_t i = (size_t)g * K + k;
    const float r = expf(logp[i] - logp_old[i]);
    const float a = adv[i];
    const float un = r * a;
    const float cl = fminf(fmaxf(r, 1.0f - eps), 1.0f + eps) * a;
    part += fminf(un, cl);
    const float ck = un <= cl ? -un / ((float)K * (float)G) : 0.0f;
    coef[i] = ck;
    cpart += ck;
  }
  // work-group sum in a fixed order: each wave's butterfly, then the waves in index order
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    part += xor_shfl(part, off);
    cpart += xor_shfl(cpart, off);
  }
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[threadIdx.x / kWave] = part;
    redc[threadIdx.x / kWave] = cpart;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f, sc = 0.f;
    for (int w = 0; w < 256 / kWave; ++w) {
      s += red[w];
      sc += redc[w];
    }
    loss[g] = -s / (float)K;
    coef[(size_t)G * K + g] = sc;   // the graph's sum of coefficients
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
  const float csum = coef[(size_t)gt.n * K + g];   // sum_k c[g,k], formed with the coefficients
  // Loads past the end read the last element and are masked afterwards, so no
  // load sits behind a branch and each group of eight issues back to back.
  for (int jb = 0; jb < D; jb += 8) {
    float rv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) rv[e] = row[min(jb + e, D - 1)];
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k0 = q; k0 < K; k0 += 8 * kPpoLanes) {
      int p[8];
      float ck[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int kc = min(k0 + u * kPpoLanes, K - 1);
        p[u] = placements[(size_t)kc * n + vv];
        ck[u] = c[kc];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool in = k0 + u * kPpoLanes < K;
        const int pj = in ? p[u] - jb : -1;
        const float cu = in ? ck[u] : 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += pj == e ? cu : 0.0f;
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
        if (j < D) dlogits[(size_t)v * D + j] = acc[e] - expf(rv[e] - lz) * csum;
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

namespace gdp {

// ---- the head's backward pass (Fig. 1: logits = X W_out^T + b_out) ------------
// Chunk c of kHeadBwdRows rows: dx rows (dx[v] = dlogits[v] W_out) and the
// chunk's partial sums of dW_out = dlogits^T X and db_out = sum_v dlogits[v].
// Thread (rg, col), RG = 256 / d row groups: rows r0 + rg, r0 + rg + RG, ... of
// the chunk, column col of d, with column col of W_out in registers.  The row
// groups' dW_out partials meet in LDS in row-group order, kHeadBwdJ devices at
// a time; db_out's partial is a serial sum over the chunk's rows per device.
constexpr int kHeadBwdJ = 8;
template <typename T, int DMAX>
__global__ __launch_bounds__(256) void k_head_bwd_rows(const float* __restrict__ x, const T* __restrict__ w_out,
                                                       const float* __restrict__ dlogits, int n, int d, int D,
                                                       float* __restrict__ dx, float* __restrict__ partial) {
  __shared__ float red[256 * kHeadBwdJ];
  const int RG = 256 / d;                       // d divides 256
  const int rg = threadIdx.x / d, col = threadIdx.x % d;
  const int c = blockIdx.x;
  const int r0 = c * kHeadBwdRows, r1 = min(r0 + kHeadBwdRows, n);
  float wc[DMAX], aw[DMAX];
#pragma unroll
  for (int j = 0; j < DMAX; ++j) {
    wc[j] = j < D ? to_f32(w_out[(size_t)j * d + col]) : 0.f;
    aw[j] = 0.f;
  }
  for (int v = r0 + rg; v < r1; v += RG) {
    const float xv = x[(size_t)v * d + col];
    const float* dl = dlogits + (size_t)v * D;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < DMAX; ++j) {
      if (j < D) {
        const float g = dl[j];
        acc += g * wc[j];
        aw[j] += g * xv;
      }
    }
    dx[(size_t)v * d + col] = acc;
  }
  float* out = partial + (size_t)c * D * (d + 1);   // [D][d + 1]: dW_out row j, then db_out[j]
#pragma unroll
  for (int j0 = 0; j0 < DMAX; j0 += kHeadBwdJ) {
    if (j0 >= D) break;
#pragma unroll
    for (int e = 0; e < kHeadBwdJ; ++e) red[(e * RG + rg) * d + col] = aw[j0 + e];
    __syncthreads();
    for (int i = threadIdx.x; i < kHeadBwdJ * d; i += 256) {
      const int e = i / d, cc = i % d;
      float s = 0.f;
      for (int q = 0; q < RG; ++q) s += red[(e * RG + q) * d + cc];
      if (j0 + e < D) out[(size_t)(j0 + e) * (d + 1) + cc] = s;
    }
    __syncthreads();
  }
  if (threadIdx.x < D) {
    float s = 0.f;
    for (int v = r0; v < r1; ++v) s += dlogits[(size_t)v * D + threadIdx.x];
    out[(size_t)threadIdx.x * (d + 1) + d] = s;
  }
}

// The same for D <= kHeadBwdJ with four columns per thread: TPR = d / 4 threads
// per row, RG = 256 / TPR row groups, U rows of a row group in flight.  The
// chunk's dlogits rows sit in LDS (padded to kHeadBwdJ columns), so the row
// loop's only global loads are the X rows; the bias partial rides along on
// the dlogits values each thread reads back.
template <typename T>
__global__ __launch_bounds__(256) void k_head_bwd_rows4(const float* __restrict__ x, const T* __restrict__ w_out,
                                                        const float* __restrict__ dlogits, int n, int d, int D,
                                                        float* __restrict__ dx, float* __restrict__ partial) {
  constexpr int J = kHeadBwdJ, U = 8;
  static_assert(J == 8, "two float4 reads per dlogits row");
  __shared__ float4 red[256 * J];               // [RG][J][TPR]
  __shared__ float redb[64 * J];                // [RG][J]
  __shared__ float4 sdl[kHeadBwdRows * J / 4];  // [row][J]
  const int TPR = d >> 2, RG = 256 / TPR;
  const int rg = threadIdx.x / TPR, tc = threadIdx.x % TPR;
  const int r0 = blockIdx.x * kHeadBwdRows, r1 = min(r0 + kHeadBwdRows, n);
  float* sdlf = reinterpret_cast<float*>(sdl);
  for (int i = threadIdx.x; i < kHeadBwdRows * J; i += 256) {
    const int row = i / J, j = i % J;
    sdlf[i] = r0 + row < r1 && j < D ? dlogits[(size_t)(r0 + row) * D + j] : 0.f;
  }
  float4 wc[J], aw[J];
  float ab[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const T* w = w_out + (size_t)j * d + 4 * tc;
    wc[j] = j < D ? make_float4(to_f32(w[0]), to_f32(w[1]), to_f32(w[2]), to_f32(w[3])) : make_float4(0.f, 0.f, 0.f, 0.f);
    aw[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    ab[j] = 0.f;
  }
  __syncthreads();
  for (int v0 = r0 + rg; v0 < r1; v0 += U * RG) {
    float4 xv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * RG;
      xv[u] = v < r1 ? *reinterpret_cast<const float4*>(x + (size_t)v * d + 4 * tc) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + u * RG;
      const int lr = min(v, r1 - 1) - r0;       // a row past the chunk's end reads the last row, weighted 0
      const float4 ga = sdl[lr * 2], gb = sdl[lr * 2 + 1];
      const float gv[J] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
      const float keep = v < r1 ? 1.f : 0.f;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const float gj = keep * gv[j];
        acc.x += gj * wc[j].x; acc.y += gj * wc[j].y; acc.z += gj * wc[j].z; acc.w += gj * wc[j].w;
        aw[j].x += gj * xv[u].x; aw[j].y += gj * xv[u].y; aw[j].z += gj * xv[u].z; aw[j].w += gj * xv[u].w;
        ab[j] += gj;
      }
      if (v < r1) *reinterpret_cast<float4*>(dx + (size_t)v * d + 4 * tc) = acc;
    }
  }
#pragma unroll
  for (int j = 0; j < J; ++j) red[(rg * J + j) * TPR + tc] = aw[j];
  if (tc == 0) {
#pragma unroll
    for (int j = 0; j < J; ++j) redb[rg * J + j] = ab[j];
  }
  __syncthreads();
  float* out = partial + (size_t)blockIdx.x * D * (d + 1);   // [D][d + 1]: dW_out row j, then db_out[j]
  for (int i = threadIdx.x; i < J * TPR; i += 256) {
    const int j = i / TPR, c4 = i % TPR;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q = 0; q < RG; ++q) {
      const float4 t = red[(q * J + j) * TPR + c4];
      s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
    }
    if (j < D) {
      float* o = out + (size_t)j * (d + 1) + 4 * c4;
      o[0] = s.x; o[1] = s.y; o[2] = s.z; o[3] = s.w;
    }
  }
  if (threadIdx.x < D) {
    float s = 0.f;
    for (int q = 0; q < RG; ++q) s += redb[q * J + threadIdx.x];
    out[(size_t)threadIdx.x * (d + 1) + d] = s;
  }
}

// out[i] = sum over chunks of partial[c][i]: wave w of the block sums chunks
// w, w + 16, ... in order (four running sums), then the 16 waves' sums meet in
// LDS in wave order.  A block covers 64 consecutive outputs.
constexpr int kHeadReduceWaves = 16;
__global__ __launch_bounds__(64 * kHeadReduceWaves) void k_head_bwd_reduce(const float* __restrict__ partial, int chunks,
                                                                          int width, int d, float* __restrict__ dw_out,
                                                                          float* __restrict__ db_out) {
  __shared__ float sw[kHeadReduceWaves][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + lane;
  const int ic = min(i, width - 1);
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  constexpr int S = kHeadReduceWaves;
  for (int c = w; c < chunks; c += 4 * S) {
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = partial[(size_t)min(c + e * S, chunks - 1) * width + ic];
#pragma unroll
    for (int e = 0; e < 4; ++e) a[e] += c + e * S < chunks ? v[e] : 0.f;
  }
  sw[w][lane] = (a[0] + a[1]) + (a[2] + a[3]);
  __syncthreads();
  if (w == 0 && i < width) {
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < S; ++q) s += sw[q][lane];
    const int j = i / (d + 1), col = i % (d + 1);
    if (col < d) dw_out[(size_t)j * d + col] = s;
    else db_out[j] = s;
  }
}

template <typename T>
hipError_t launch_head_backward(const float* x, const T* w_out, const float* dlogits, int n, int d, int D, float* dx,
                                float* dw_out, float* db_out, float* partial, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (d < 1 || d > 256 || 256 % d != 0 || D < 1 || D > 64) return hipErrorInvalidValue;
  const int chunks = (n + kHeadBwdRows - 1) / kHeadBwdRows;
  if (D <= kHeadBwdJ && d % 4 == 0 && 1024 % d == 0 && d >= 16)
    hipLaunchKernelGGL((k_head_bwd_rows4<T>), dim3(chunks), dim3(256), 0, s, x, w_out, dlogits, n, d, D, dx, partial);
  else
    hipLaunchKernelGGL((k_head_bwd_rows<T, 64>), dim3(chunks), dim3(256), 0, s, x, w_out, dlogits, n, d, D, dx, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int width = D * (d + 1);
  hipLaunchKernelGGL(k_head_bwd_reduce, dim3((width + 63) / 64), dim3(64 * kHeadReduceWaves), 0, s, partial, chunks,
                     width, d, dw_out, db_out);
  return hipGetLastError();
}
template hipError_t launch_head_backward<float>(const float*, const float*, const float*, int, int, int, float*, float*,
                                                float*, float*, hipStream_t);
template hipError_t launch_head_backward<bf16>(const float*, const bf16*, const float*, int, int, int, float*, float*,
                                               float*, float*, hipStream_t);

}  // namespace gdp

namespace gdp {

// ---- Section 4: reward and advantage of measured run times ---------------------
// One work-group per graph: r = -sqrt(t) (or -10 for an invalid placement);
// the bias is the graph's running mean of all previous rewards (its batch
// mean when there is none), and the batch then joins the running state.
// The batch sum is taken in a fixed order (lanes, then waves in index order).
__global__ __launch_bounds__(256) void k_advantages(const float* __restrict__ run_time,
                                                    const uint8_t* __restrict__ valid, int K,
                                                    double* __restrict__ reward_sum,
                                                    int64_t* __restrict__ trial_count,
                                                    float* __restrict__ reward, float* __restrict__ adv) {
  __shared__ float red[256 / kWave];
  __shared__ float s_base;
  const int g = blockIdx.x;
  auto reward_at = [&](size_t i) { return !valid || valid[i] ? -sqrtf(run_time[i]) : -10.0f; };
  float part = 0.f;
  for (int k = threadIdx.x; k < K; k += 256) part += reward_at((size_t)g * K + k);
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) part += xor_shfl(part, off);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int w = 0; w < 256 / kWave; ++w) s += red[w];
    const int64_t n = trial_count[g];
    const double prev = reward_sum[g];
    s_base = n > 0 ? (float)(prev / (double)n) : s / (float)K;
    reward_sum[g] = prev + (double)s;
    trial_count[g] = n + K;
  }
  __syncthreads();
  const float base = s_base;
  for (int k = threadIdx.x; k < K; k += 256) {
    const size_t i = (size_t)g * K + k;
    const float r = reward_at(i);
    if (reward) reward[i] = r;
    adv[i] = r - base;
  }
}

hipError_t launch_advantages(const float* run_time, const uint8_t* valid, int G, int K, double* reward_sum,
                             int64_t* trial_count, float* reward, float* adv, hipStream_t s) {
  hipLaunchKernelGGL(k_advantages, dim3(G), dim3(256), 0, s, run_time, valid, K, reward_sum, trial_count, reward,
                     adv);
  return hipGetLastError();
}

}  // namespace gdp
