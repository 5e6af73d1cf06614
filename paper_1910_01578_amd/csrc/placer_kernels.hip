// Section 3.3 (Eq. 4) conditioning and the output layer of the placer.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

// For every placer layer l of a group:
//   gamma_l[g][c] = 1 + W_g,l[c] . x0_g + b_g,l[c];  beta_l[g][c] = W_b,l[c] . x0_g + b_b,l[c].
// One launch covers up to kFilmLayersPerLaunch layers; one wavefront per output
// element, lanes over the H inputs.  Output of layer l at out + l * 2 * G * d
// (gamma, then beta).
template <typename T>
__global__ __launch_bounds__(256) void k_film_gemv(FilmLayers<T> w, int n_layers, const float* __restrict__ x0,
                                                   int G, int d, int H, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int idx = blockIdx.x * 4 + (threadIdx.x >> 6);   // over n_layers * G * 2 * d
  if (idx >= n_layers * G * 2 * d) return;
  const int l = idx / (G * 2 * d);
  const int rem = idx % (G * 2 * d);
  const int g = rem / (2 * d);
  const int which = (rem / d) & 1;
  const int c = rem % d;
  const T* wr = (which ? w.wb[l] : w.wg[l]) + (size_t)c * H;
  // four weight / input pairs per lane requested before any is used (indices
  // past H reload the last element and add nothing), summed in k order
  const float* xg = x0 + (size_t)g * H;
  float acc = 0.f;
  for (int k0 = lane; k0 < H; k0 += 4 * 64) {
    float wv[4], xv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = min(k0 + 64 * u, H - 1);
      wv[u] = to_f32(wr[k]);
      xv[u] = xg[k];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k0 + 64 * u < H) acc += wv[u] * xv[u];
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += xor_shfl(acc, off);
  if (lane == 0) {
    float* o = out + (size_t)l * 2 * G * d + (size_t)which * G * d + (size_t)g * d + c;
    *o = which ? acc + to_f32(w.bb[l][c]) : 1.0f + acc + to_f32(w.bg[l][c]);
  }
}

template <typename T>
hipError_t launch_film_gemv(const FilmLayers<T>& w, int n_layers, const float* x0, int G, int d, int H,
                            float* out, hipStream_t s) {
  if (n_layers < 1 || n_layers > kFilmLayersPerLaunch) return hipErrorInvalidValue;
  const int n = n_layers * G * 2 * d;
  hipLaunchKernelGGL((k_film_gemv<T>), dim3((n + 3) / 4), dim3(256), 0, s, w, n_layers, x0, G, d, H, out);
  return hipGetLastError();
}
template hipError_t launch_film_gemv<float>(const FilmLayers<float>&, int, const float*, int, int, int, float*,
                                            hipStream_t);
template hipError_t launch_film_gemv<bf16>(const FilmLayers<bf16>&, int, const float*, int, int, int, float*,
                                           hipStream_t);

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
