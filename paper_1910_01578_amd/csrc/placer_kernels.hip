// Section 3.3 (Eq. 4) conditioning and the output layer of the placer.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

// gamma[g][c] = 1 + W_g[c] . x0_g + b_g[c];  beta[g][c] = W_b[c] . x0_g + b_b[c].
// One wavefront per output element, lanes over the H inputs.
template <typename T>
__global__ __launch_bounds__(256) void k_film_gemv(const T* __restrict__ wg, const T* __restrict__ bg,
                                                   const T* __restrict__ wb, const T* __restrict__ bb,
                                                   const float* __restrict__ x0, int G, int d, int H,
                                                   float* __restrict__ gamma, float* __restrict__ beta) {
  const int lane = threadIdx.x & 63;
  const int idx = blockIdx.x * 4 + (threadIdx.x >> 6);   // over G * 2 * d
  if (idx >= G * 2 * d) return;
  const int g = idx / (2 * d);
  const int which = (idx / d) & 1;
  const int c = idx % d;
  const T* w = (which ? wb : wg) + (size_t)c * H;
  float acc = 0.f;
  for (int k = lane; k < H; k += 64) acc += to_f32(w[k]) * x0[(size_t)g * H + k];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += xor_shfl(acc, off);
  if (lane == 0) {
    if (which) beta[(size_t)g * d + c] = acc + to_f32(bb[c]);
    else gamma[(size_t)g * d + c] = 1.0f + acc + to_f32(bg[c]);
  }
}

template <typename T>
hipError_t launch_film_gemv(const T* wg, const T* bg, const T* wb, const T* bb, const float* x0, int G,
                            int d, int H, float* gamma, float* beta, hipStream_t s) {
  const int n = G * 2 * d;
  hipLaunchKernelGGL((k_film_gemv<T>), dim3((n + 3) / 4), dim3(256), 0, s, wg, bg, wb, bb, x0, G, d, H,
                     gamma, beta);
  return hipGetLastError();
}
template hipError_t launch_film_gemv<float>(const float*, const float*, const float*, const float*,
                                            const float*, int, int, int, float*, float*, hipStream_t);
template hipError_t launch_film_gemv<bf16>(const bf16*, const bf16*, const bf16*, const bf16*,
                                           const float*, int, int, int, float*, float*, hipStream_t);

// y[v] = gamma[g(v)] * x[v] + beta[g(v)] into the fp32 residual stream; with
// gamma == null the rows are only widened.  Each thread handles 4 columns.
template <typename T>
__global__ __launch_bounds__(256) void k_film_apply(const T* __restrict__ x, const float* __restrict__ gamma,
                                                    const float* __restrict__ beta, int n, int d,
                                                    GraphTable gt, float* __restrict__ y) {
  const int per_row = d / 4;
  const int64_t total = (int64_t)n * per_row;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / per_row);
    const int c = (int)(i % per_row) * 4;
    float4 o;
    float* of = reinterpret_cast<float*>(&o);
#pragma unroll
    for (int e = 0; e < 4; ++e) of[e] = to_f32(x[(size_t)v * d + c + e]);
    if (gamma) {
      const int g = graph_of_node(gt, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) of[e] = gamma[(size_t)g * d + c + e] * of[e] + beta[(size_t)g * d + c + e];
    }
    *reinterpret_cast<float4*>(y + (size_t)v * d + c) = o;
  }
}

template <typename T>
hipError_t launch_film_apply(const T* x, const float* gamma, const float* beta, int n, int d,
                             const GraphTable& gt, float* y, hipStream_t s) {
  const int64_t total = (int64_t)n * (d / 4);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL((k_film_apply<T>), dim3((unsigned)blocks), dim3(256), 0, s, x, gamma, beta, n, d, gt, y);
  return hipGetLastError();
}
template hipError_t launch_film_apply<float>(const float*, const float*, const float*, int, int,
                                             const GraphTable&, float*, hipStream_t);
template hipError_t launch_film_apply<bf16>(const bf16*, const float*, const float*, int, int,
                                            const GraphTable&, float*, hipStream_t);

// logits[v][j] = x[v] . W_out[j] + b_out[j] in fp32, lse[v] = log sum_j exp(logits[v][j]).
// DL lanes (the power of two >= D) serve one node, lane j computing logit j
// over the whole row (16-byte row reads, shared by the group); W_out sits in
// LDS as fp32 rows padded by 4 so the group's rows fall in different banks.
template <typename T, int DL>
__global__ __launch_bounds__(256) void k_head(const float* __restrict__ x, const T* __restrict__ w_out,
                                              const T* __restrict__ b_out, int n, int d, int D,
                                              float* __restrict__ logits, float* __restrict__ lse) {
  extern __shared__ float sw[];   // [D][d + 4] fp32
  constexpr int EPV = 4;
  const int ds = d + 4;
  for (int i = threadIdx.x; i < D * d; i += blockDim.x) sw[(i / d) * ds + (i % d)] = to_f32(w_out[i]);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int j = lane % DL;
  const int per_block = 256 / DL;
  const int v = blockIdx.x * per_block + threadIdx.x / DL;
  if (v >= n) return;
  const bool active = j < D;
  const float* wr = sw + (active ? j : 0) * ds;
  const float* xr = x + (size_t)v * d;
  float acc = 0.f;
  for (int k = 0; k < d; k += EPV) {
    const float4 xv = *reinterpret_cast<const float4*>(xr + k);
    acc = fmaf(xv.x, wr[k], acc);
    acc = fmaf(xv.y, wr[k + 1], acc);
    acc = fmaf(xv.z, wr[k + 2], acc);
    acc = fmaf(xv.w, wr[k + 3], acc);
  }
  const float logit = active ? acc + to_f32(b_out[j]) : -INFINITY;
  if (active) logits[(size_t)v * D + j] = logit;
  if (lse) {
    float m = logit;
#pragma unroll
    for (int off = DL / 2; off >= 1; off >>= 1) m = fmaxf(m, xor_shfl(m, off));
    float e = active ? expf(logit - m) : 0.f;
#pragma unroll
    for (int off = DL / 2; off >= 1; off >>= 1) e += xor_shfl(e, off);
    if (j == 0) lse[v] = m + logf(e);
  }
}

template <typename T, int DL>
static hipError_t launch_head_dl(const float* x, const T* w_out, const T* b_out, int n, int d, int D, float* logits,
                                 float* lse, hipStream_t s) {
  const int per_block = 256 / DL;
  const size_t lds = (size_t)D * (d + 4) * sizeof(float);
  if (lds > 48 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_head<T, DL>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_head<T, DL>), dim3((n + per_block - 1) / per_block), dim3(256), lds, s, x, w_out, b_out, n, d, D, logits, lse);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_head(const float* x, const T* w_out, const T* b_out, int n, int d, int D, float* logits,
                       float* lse, hipStream_t s) {
  if (D <= 2) return launch_head_dl<T, 2>(x, w_out, b_out, n, d, D, logits, lse, s);
  if (D <= 4) return launch_head_dl<T, 4>(x, w_out, b_out, n, d, D, logits, lse, s);
  if (D <= 8) return launch_head_dl<T, 8>(x, w_out, b_out, n, d, D, logits, lse, s);
  if (D <= 16) return launch_head_dl<T, 16>(x, w_out, b_out, n, d, D, logits, lse, s);
  if (D <= 32) return launch_head_dl<T, 32>(x, w_out, b_out, n, d, D, logits, lse, s);
  return launch_head_dl<T, 64>(x, w_out, b_out, n, d, D, logits, lse, s);
}
template hipError_t launch_head<float>(const float*, const float*, const float*, int, int, int, float*, float*,
                                       hipStream_t);
template hipError_t launch_head<bf16>(const float*, const bf16*, const bf16*, int, int, int, float*, float*,
                                      hipStream_t);

}  // namespace gdp
