// Kernels of the policy's update step (Section 3: Eq. 1 optimised with PPO;
// Section 3.1: the graph embedding network trains jointly with the placement
// network; Section 3.2: the cached segment memory passes no gradient): the
// training forward pass that keeps every intermediate, the backward pass and
// the Adam update.  Everything here computes in fp32 (weights and inputs of
// bf16 problems are widened on load), with fixed summation orders, so results
// are deterministic.
#include <algorithm>

#include "device_common.h"
#include "kernels.h"
#include "train_kernels.h"

namespace gdp {
namespace tr {

__device__ __forceinline__ float ld(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ld(const bf16* p, size_t i) { return (float)p[i]; }

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// Strided GEMM: C(m, n) = epi(alpha * sum_k A(m, k) B(k, n)), tiles of 64 x 64
// with k steps of 16, 256 threads of 4 x 4 outputs.  With splits > 1, grid.z
// splits k and each split writes its raw sums to partial[z]; gemm_reduce adds
// them in split order and applies the epilogue.
// ---------------------------------------------------------------------------
constexpr int GBM = 64, GBN = 64, GBK = 16;

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void k_gemm_strided(GemmStrided<TA, TB> g, int k_per_split, float* partial) {
  __shared__ float As[GBK][GBM + 4];
  __shared__ float Bs[GBK][GBN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * GBM, n0 = blockIdx.x * GBN;
  const int kb = blockIdx.z * k_per_split, ke = min(g.K, kb + k_per_split);
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  const bool a_kfast = g.sak == 1, b_nfast = g.sbn == 1;
  for (int k0 = kb; k0 < ke; k0 += GBK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int l = tid + 256 * e;
      int mm, kk;
      if (a_kfast) { kk = l & 15; mm = l >> 4; } else { mm = l & 63; kk = l >> 6; }
      const int m = m0 + mm, k = k0 + kk;
      As[kk][mm] = (m < g.M && k < ke) ? ld(g.a, (size_t)m * g.sam + (size_t)k * g.sak) : 0.f;
      int nn;
      if (b_nfast) { nn = l & 63; kk = l >> 6; } else { kk = l & 15; nn = l >> 4; }
      const int n = n0 + nn, k2 = k0 + kk;
      Bs[kk][nn] = (n < g.N && k2 < ke) ? ld(g.b, (size_t)k2 * g.sbk + (size_t)n * g.sbn) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m >= g.M || n >= g.N) continue;
      if (partial) {
        partial[((size_t)blockIdx.z * g.M + m) * g.N + n] = acc[i][j];
      } else {
        float v = g.alpha * acc[i][j];
        if (g.bias_f) v += g.bias_f[n];
        if (g.bias_h) v += (float)g.bias_h[n];
        if (g.act == ACT_RELU) v = fmaxf(v, 0.f);
        else if (g.act == ACT_SIGMOID) v = sigmoidf_(v);
        if (g.mask && !(g.mask[(size_t)m * g.ldm + n] > 0.f)) v = 0.f;
        float* c = g.c + (size_t)m * g.ldc + n;
        *c = g.accumulate ? *c + v : v;
      }
    }
}

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void k_gemm_reduce(GemmStrided<TA, TB> g, int splits, const float* partial) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i >= (size_t)g.M * g.N) return;
  const int m = (int)(i / g.N), n = (int)(i % g.N);
  double s = 0.0;   // the splits' sums added in double: long reductions (k = rows) keep fp32 accuracy
  for (int z = 0; z < splits; ++z) s += (double)partial[(size_t)z * g.M * g.N + i];
  float v = g.alpha * (float)s;
  if (g.bias_f) v += g.bias_f[n];
  if (g.bias_h) v += (float)g.bias_h[n];
  if (g.act == ACT_RELU) v = fmaxf(v, 0.f);
  else if (g.act == ACT_SIGMOID) v = sigmoidf_(v);
  if (g.mask && !(g.mask[(size_t)m * g.ldm + n] > 0.f)) v = 0.f;
  float* c = g.c + (size_t)m * g.ldc + n;
  *c = g.accumulate ? *c + v : v;
}

template <typename TA, typename TB>
hipError_t launch_gemm_strided(const GemmStrided<TA, TB>& g, float* partial, size_t partial_floats, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const int tiles = ((g.M + GBM - 1) / GBM) * ((g.N + GBN - 1) / GBN);
  int splits = 1;
  // a long reduction (the weight gradients, k = rows) is split into pieces of
  // at most kSplitRows, each summed in fp32, the pieces added in double
  constexpr int kSplitRows = 1024;
  (void)tiles;
  if (partial && g.K > kSplitRows) {
    splits = (g.K + kSplitRows - 1) / kSplitRows;
    while (splits > 1 && (size_t)splits * g.M * g.N > partial_floats) --splits;
  }
  const int kps = splits > 1 ? (((g.K + splits - 1) / splits + GBK - 1) / GBK) * GBK : std::max(g.K, 1);
  splits = splits > 1 ? (g.K + kps - 1) / kps : 1;
  dim3 grid((g.N + GBN - 1) / GBN, (g.M + GBM - 1) / GBM, splits);
  hipLaunchKernelGGL((k_gemm_strided<TA, TB>), grid, dim3(256), 0, s, g, kps, splits > 1 ? partial : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const size_t n = (size_t)g.M * g.N;
  hipLaunchKernelGGL((k_gemm_reduce<TA, TB>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, g, splits,
                     (const float*)partial);
  return hipGetLastError();
}

#define GDP_GEMM_INST(TA, TB) \
  template hipError_t launch_gemm_strided<TA, TB>(const GemmStrided<TA, TB>&, float*, size_t, hipStream_t);
GDP_GEMM_INST(float, float)
GDP_GEMM_INST(float, bf16)
GDP_GEMM_INST(bf16, float)
GDP_GEMM_INST(bf16, bf16)
#undef GDP_GEMM_INST

// ---------------------------------------------------------------------------
// Column sums per graph: out[g][c] (+)= sum over rows v of graph g of
// A[v][c] (* B[v][c] when B is given), in a fixed order: 256-row chunks of
// each graph into partials, then each graph's chunks in order.
// ---------------------------------------------------------------------------
constexpr int kColRows = 256;

template <typename TA>
__global__ __launch_bounds__(256) void k_colsum_partial(const TA* a, int lda, const float* b, int ldb, int C,
                                                        GraphTable ct, float* partial) {
  const int chunk = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const int g = graph_of_block(ct, chunk);
  const int r0 = ct.ptr[g] + (chunk - ct.blk[g]) * kColRows;
  const int r1 = min(r0 + kColRows, ct.ptr[g + 1]);
  float s = 0.f;
  for (int r = r0; r < r1; ++r) {
    float v = ld(a, (size_t)r * lda + c);
    if (b) v *= b[(size_t)r * ldb + c];
    s += v;
  }
  partial[(size_t)chunk * C + c] = s;
}

__global__ __launch_bounds__(256) void k_colsum_final(const float* partial, int C, GraphTable ct, float* out, int ldo,
                                                      int accumulate) {
  const int g = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  double s = 0.0;   // chunk sums added in double
  for (int k = ct.blk[g]; k < ct.blk[g + 1]; ++k) s += (double)partial[(size_t)k * C + c];
  float* o = out + (size_t)g * ldo + c;
  *o = accumulate ? *o + (float)s : (float)s;
}

template <typename TA>
hipError_t launch_colsum(const TA* a, int lda, const float* b, int ldb, int C, const GraphTable& ct, int chunks,
                         float* partial, float* out, int ldo, bool accumulate, hipStream_t s) {
  if (C <= 0 || chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_colsum_partial<TA>), dim3((C + 255) / 256, chunks), dim3(256), 0, s, a, lda, b, ldb, C, ct,
                     partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_colsum_final, dim3((C + 255) / 256, ct.n), dim3(256), 0, s, (const float*)partial, C, ct, out,
                     ldo, accumulate ? 1 : 0);
  return hipGetLastError();
}
template hipError_t launch_colsum<float>(const float*, int, const float*, int, int, const GraphTable&, int, float*,
                                         float*, int, bool, hipStream_t);
template hipError_t launch_colsum<bf16>(const bf16*, int, const float*, int, int, const GraphTable&, int, float*,
                                        float*, int, bool, hipStream_t);

// ---------------------------------------------------------------------------
// Row-wise kernels: one wavefront per row of width d <= 1024.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// out = LN(r) * g + b  (eps 1e-5, biased variance)
template <typename T>
__global__ __launch_bounds__(256) void k_ln_fwd(const float* r, int n, int d, const T* g, const T* b, float* out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const float* x = r + (size_t)row * d;
  float s = 0.f;
  for (int c = lane; c < d; c += kWave) s += x[c];
  const float mu = wave_sum(s) / d;
  float q = 0.f;
  for (int c = lane; c < d; c += kWave) {
    const float t = x[c] - mu;
    q += t * t;
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / d + 1e-5f);
  for (int c = lane; c < d; c += kWave) out[(size_t)row * d + c] = (x[c] - mu) * rstd * ld(g, c) + ld(b, c);
}

// LayerNorm backward for out = LN(r) g + b and upstream dout: dr, and the
// per-row terms of the gain gradient (dout * xhat) in xg.
template <typename T>
__global__ __launch_bounds__(256) void k_ln_bwd(const float* r, const float* dout, int n, int d, const T* g,
                                                float* dr, float* xg) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const float* x = r + (size_t)row * d;
  const float* dy = dout + (size_t)row * d;
  float s = 0.f;
  for (int c = lane; c < d; c += kWave) s += x[c];
  const float mu = wave_sum(s) / d;
  float q = 0.f;
  for (int c = lane; c < d; c += kWave) {
    const float t = x[c] - mu;
    q += t * t;
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / d + 1e-5f);
  float s1 = 0.f, s2 = 0.f;
  for (int c = lane; c < d; c += kWave) {
    const float xh = (x[c] - mu) * rstd;
    const float gd = dy[c] * ld(g, c);
    s1 += gd;
    s2 += gd * xh;
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
  for (int c = lane; c < d; c += kWave) {
    const float xh = (x[c] - mu) * rstd;
    const float gd = dy[c] * ld(g, c);
    dr[(size_t)row * d + c] = rstd * (gd - s1 - xh * s2);
    xg[(size_t)row * d + c] = dy[c] * xh;
  }
}

template <typename T>
hipError_t launch_ln_fwd(const float* r, int n, int d, const T* g, const T* b, float* out, hipStream_t s) {
  hipLaunchKernelGGL((k_ln_fwd<T>), dim3((n + 3) / 4), dim3(256), 0, s, r, n, d, g, b, out);
  return hipGetLastError();
}
template <typename T>
hipError_t launch_ln_bwd(const float* r, const float* dout, int n, int d, const T* g, float* dr, float* xg,
                         hipStream_t s) {
  hipLaunchKernelGGL((k_ln_bwd<T>), dim3((n + 3) / 4), dim3(256), 0, s, r, dout, n, d, g, dr, xg);
  return hipGetLastError();
}
template hipError_t launch_ln_fwd<float>(const float*, int, int, const float*, const float*, float*, hipStream_t);
template hipError_t launch_ln_fwd<bf16>(const float*, int, int, const bf16*, const bf16*, float*, hipStream_t);
template hipError_t launch_ln_bwd<float>(const float*, const float*, int, int, const float*, float*, float*,
                                         hipStream_t);
template hipError_t launch_ln_bwd<bf16>(const float*, const float*, int, int, const bf16*, float*, float*,
                                        hipStream_t);

// ---------------------------------------------------------------------------
// Elementwise kernels.
// ---------------------------------------------------------------------------
// y[v][c] = gamma[g(v)][c] * x[v][c] + beta[g(v)][c]  (gamma, beta [G][d]; null: identity)
template <typename TX>
__global__ void k_film_apply(const TX* x, int n, int d, const float* gamma, const float* beta, GraphTable gt,
                             float* y) {
  const size_t total = (size_t)n * d;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / d), c = (int)(i % d);
    float val = ld(x, i);
    if (gamma) {
      const int g = graph_of_node(gt, v);
      val = gamma[(size_t)g * d + c] * val + beta[(size_t)g * d + c];
    }
    y[i] = val;
  }
}
template <typename TX>
hipError_t launch_film_apply(const TX* x, int n, int d, const float* gamma, const float* beta, const GraphTable& gt,
                             float* y, hipStream_t s) {
  const size_t total = (size_t)n * d;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL((k_film_apply<TX>), dim3(blocks), dim3(256), 0, s, x, n, d, gamma, beta, gt, y);
  return hipGetLastError();
}
template hipError_t launch_film_apply<float>(const float*, int, int, const float*, const float*, const GraphTable&,
                                             float*, hipStream_t);
template hipError_t launch_film_apply<bf16>(const bf16*, int, int, const float*, const float*, const GraphTable&,
                                            float*, hipStream_t);

// Elementwise ops on n values: out = op(a, b, c).
__global__ void k_ew(int op, const float* a, const float* b, const float* c, size_t n, float* out) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    float r;
    switch (op) {
      case EW_ADD: r = a[i] + b[i]; break;                                 // a + b
      case EW_MASK_POS: r = b[i] > 0.f ? a[i] : 0.f; break;                // a where b > 0 (ReLU')
      case EW_SIGMOID_GRAD: r = a[i] * b[i] * (1.0f - b[i]); break;        // a * s (1 - s)
      case EW_SCALE_BY: r = a[i] * b[i]; break;                             // a * b
      default: r = 0.f;
    }
    out[i] = r;
  }
}
hipError_t launch_ew(int op, const float* a, const float* b, const float* c, size_t n, float* out, hipStream_t s) {
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(k_ew, dim3(std::max(1u, blocks)), dim3(256), 0, s, op, a, b, c, n, out);
  return hipGetLastError();
}

// dX[v][c] = gamma[g(v)][c] * dY[v][c]  (the input side of FiLM's backward)
__global__ void k_film_dx(const float* dy, int n, int d, const float* gamma, GraphTable gt, float* dx) {
  const size_t total = (size_t)n * d;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / d), c = (int)(i % d);
    const float gm = gamma ? gamma[(size_t)graph_of_node(gt, v) * d + c] : 1.0f;
    dx[i] = gm * dy[i];
  }
}
hipError_t launch_film_dx(const float* dy, int n, int d, const float* gamma, const GraphTable& gt, float* dx,
                          hipStream_t s) {
  const size_t total = (size_t)n * d;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_film_dx, dim3(blocks), dim3(256), 0, s, dy, n, d, gamma, gt, dx);
  return hipGetLastError();
}

// dh[v][c] += dx0[g(v)][c] / n_g  (the mean pool's backward)
__global__ void k_meanpool_bwd(const float* dx0, int n, int H, GraphTable gt, float* dh) {
  const size_t total = (size_t)n * H;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / H), c = (int)(i % H);
    const int g = graph_of_node(gt, v);
    dh[i] += dx0[(size_t)g * H + c] / (float)(gt.ptr[g + 1] - gt.ptr[g]);
  }
}
hipError_t launch_meanpool_bwd(const float* dx0, int n, int H, const GraphTable& gt, float* dh, hipStream_t s) {
  const size_t total = (size_t)n * H;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_meanpool_bwd, dim3(blocks), dim3(256), 0, s, dx0, n, H, gt, dh);
  return hipGetLastError();
}

// x0[g][c] = mean over the rows of graph g: the graph's column sums (256-row
// chunks, then the chunks in order), divided by its node count.
__global__ void k_scale_rows_by_graph_size(float* x0, int H, GraphTable gt) {
  const int g = blockIdx.y, c = blockIdx.x * 256 + threadIdx.x;
  if (c < H) x0[(size_t)g * H + c] /= (float)(gt.ptr[g + 1] - gt.ptr[g]);
}
hipError_t launch_meanpool_f32(const float* h, int H, const GraphTable& chunks, int n_chunks, float* partial,
                               float* x0, hipStream_t s) {
  hipError_t e = launch_colsum<float>(h, H, nullptr, 0, H, chunks, n_chunks, partial, x0, H, false, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_scale_rows_by_graph_size, dim3((H + 255) / 256, chunks.n), dim3(256), 0, s, x0, H, chunks);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Eq. 2's max-pool with the winning neighbour of every element (ties: the
// lowest node id), and its backward: dP[u][c] = sum over the neighbours v of u
// (out-edges in CSR order, then in-edges in ascending order) whose element c
// was won by u of dA[v][c].  u in S(v) implies v in N(u), so every v that
// selected u is visited.
// ---------------------------------------------------------------------------
__global__ void k_gather_max_arg(const float* P, const int* s_ptr, const int* s_idx, int n, int H, float* A,
                                 int* arg) {
  const size_t total = (size_t)n * H;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / H), c = (int)(i % H);
    float best = 0.f;
    int who = -1;
    for (int e = s_ptr[v]; e < s_ptr[v + 1]; ++e) {
      const int u = s_idx[e];
      const float p = P[(size_t)u * H + c];
      if (who < 0 || p > best || (p == best && u < who)) {
        best = p;
        who = u;
      }
    }
    A[i] = who < 0 ? 0.f : best;
    arg[i] = who;
  }
}
hipError_t launch_gather_max_arg(const float* P, const int* s_ptr, const int* s_idx, int n, int H, float* A, int* arg,
                                 hipStream_t s) {
  const size_t total = (size_t)n * H;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_gather_max_arg, dim3(blocks), dim3(256), 0, s, P, s_ptr, s_idx, n, H, A, arg);
  return hipGetLastError();
}

__global__ void k_gather_max_bwd(const float* dA, const int* arg, const int* row_ptr, const int* col_idx,
                                 const int* in_ptr, const int* in_idx, int n, int H, float* dP) {
  const size_t total = (size_t)n * H;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int u = (int)(i / H), c = (int)(i % H);
    float s = 0.f;
    for (int e = row_ptr[u]; e < row_ptr[u + 1]; ++e) {
      const int v = col_idx[e];
      if (arg[(size_t)v * H + c] == u) s += dA[(size_t)v * H + c];
    }
    for (int e = in_ptr[u]; e < in_ptr[u + 1]; ++e) {
      const int v = in_idx[e];
      if (arg[(size_t)v * H + c] == u) s += dA[(size_t)v * H + c];
    }
    dP[i] = s;
  }
}
hipError_t launch_gather_max_bwd(const float* dA, const int* arg, const int* row_ptr, const int* col_idx,
                                 const int* in_ptr, const int* in_idx, int n, int H, float* dP, hipStream_t s) {
  const size_t total = (size_t)n * H;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_gather_max_bwd, dim3(blocks), dim3(256), 0, s, dA, arg, row_ptr, col_idx, in_ptr, in_idx, n, H,
                     dP);
  return hipGetLastError();
}

// Sorts each in-edge row ascending (rows filled by atomics come in any order),
// so the backward's sums run in a fixed order.  Insertion sort per row.
__global__ void k_sort_rows(const int* ptr, int n, int* idx) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n) return;
  const int a = ptr[v], b = ptr[v + 1];
  for (int i = a + 1; i < b; ++i) {
    const int x = idx[i];
    int j = i - 1;
    while (j >= a && idx[j] > x) {
      idx[j + 1] = idx[j];
      --j;
    }
    idx[j + 1] = x;
  }
}
hipError_t launch_sort_rows(const int* ptr, int n, int* idx, hipStream_t s) {
  hipLaunchKernelGGL(k_sort_rows, dim3((n + 255) / 256), dim3(256), 0, s, ptr, n, idx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Segment attention in fp32 for training (band form: the queries of a segment
// [q0, q1) of graph g attend to keys [max(g_start, q0 - mem_len), q1)).  One
// thread per (query, head); the softmax's log-sum-exp per (query, head) is
// kept for the backward.  qkv: [n, 3d] (Q | K | V, heads contiguous).
// ---------------------------------------------------------------------------
struct BandInfo {
  int k0, q0, q1;   // key start, segment [q0, q1)
};
__device__ __forceinline__ BandInfo band_of(const GraphTable& gt, int v, int seg, int mem) {
  const int g = graph_of_node(gt, v);
  const int gs = gt.ptr[g], ge = gt.ptr[g + 1];
  const int q0 = gs + ((v - gs) / seg) * seg;
  BandInfo b;
  b.q0 = q0;
  b.q1 = min(q0 + seg, ge);
  b.k0 = max(gs, q0 - mem);
  return b;
}

template <int DH>
__global__ __launch_bounds__(64) void k_attn_fwd(const float* qkv, int n, int d, int heads, int seg, int mem,
                                                 GraphTable gt, float scale, float* o, float* lse) {
  const int v = blockIdx.x * 64 + threadIdx.x;
  const int h = blockIdx.y;
  if (v >= n) return;
  const BandInfo b = band_of(gt, v, seg, mem);
  const int ld = 3 * d;
  float q[DH], acc[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    q[t] = qkv[(size_t)v * ld + h * DH + t] * scale;
    acc[t] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int j = b.k0; j < b.q1; ++j) {
    const float* kr = qkv + (size_t)j * ld + d + h * DH;
    float sc = 0.f;
#pragma unroll
    for (int t = 0; t < DH; ++t) sc = fmaf(q[t], kr[t], sc);
    const float mn = fmaxf(m, sc);
    const float corr = expf(m - mn), p = expf(sc - mn);
    l = l * corr + p;
    const float* vr = qkv + (size_t)j * ld + 2 * d + h * DH;
#pragma unroll
    for (int t = 0; t < DH; ++t) acc[t] = fmaf(p, vr[t], acc[t] * corr);
    m = mn;
  }
  const float inv = 1.0f / l;
#pragma unroll
  for (int t = 0; t < DH; ++t) o[(size_t)v * d + h * DH + t] = acc[t] * inv;
  lse[(size_t)v * heads + h] = m + logf(l);
}

// dq for every query: p = exp(s - lse), ds = p (dO . v_j - Dq), dq = scale * sum ds k_j
template <int DH>
__global__ __launch_bounds__(64) void k_attn_bwd_q(const float* qkv, const float* dO, const float* Dq,
                                                   const float* lse, int n, int d, int heads, int seg, int mem,
                                                   GraphTable gt, float scale, float* dqkv, int lddq) {
  const int v = blockIdx.x * 64 + threadIdx.x;
  const int h = blockIdx.y;
  if (v >= n) return;
  const BandInfo b = band_of(gt, v, seg, mem);
  const int ld = 3 * d;
  float q[DH], dov[DH], dq[DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    q[t] = qkv[(size_t)v * ld + h * DH + t] * scale;
    dov[t] = dO[(size_t)v * d + h * DH + t];
    dq[t] = 0.f;
  }
  const float L = lse[(size_t)v * heads + h], D = Dq[(size_t)v * heads + h];
  for (int j = b.k0; j < b.q1; ++j) {
    const float* kr = qkv + (size_t)j * ld + d + h * DH;
    const float* vr = qkv + (size_t)j * ld + 2 * d + h * DH;
    float sc = 0.f, dp = 0.f;
#pragma unroll
    for (int t = 0; t < DH; ++t) {
      sc = fmaf(q[t], kr[t], sc);
      dp = fmaf(dov[t], vr[t], dp);
    }
    const float ds = expf(sc - L) * (dp - D);
#pragma unroll
    for (int t = 0; t < DH; ++t) dq[t] = fmaf(ds, kr[t], dq[t]);
  }
#pragma unroll
  for (int t = 0; t < DH; ++t) dqkv[(size_t)v * lddq + h * DH + t] = dq[t] * scale;
}

// dk, dv for every key j, from the queries of its own segment (live: the key's
// row receives the gradient) and separately from the later segments whose
// memory holds it (the memory passes no gradient to its rows, only to the
// projection weights).
template <int DH>
__global__ __launch_bounds__(64) void k_attn_bwd_kv(const float* qkv, const float* dO, const float* Dq,
                                                    const float* lse, int n, int d, int heads, int seg, int mem,
                                                    GraphTable gt, float scale, float* dqkv_live, int ldl,
                                                    float* dkv_mem, int ldm) {
  const int j = blockIdx.x * 64 + threadIdx.x;
  const int h = blockIdx.y;
  if (j >= n) return;
  const int g = graph_of_node(gt, j);
  const int gs = gt.ptr[g], ge = gt.ptr[g + 1];
  const int ld = 3 * d;
  float kr[DH], vr[DH], dk[2][DH], dv[2][DH];
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    kr[t] = qkv[(size_t)j * ld + d + h * DH + t];
    vr[t] = qkv[(size_t)j * ld + 2 * d + h * DH + t];
    dk[0][t] = dk[1][t] = dv[0][t] = dv[1][t] = 0.f;
  }
  const int s_own = (j - gs) / seg;
  // segments that see key j: its own, and later ones with q0 - mem <= j
  for (int s = s_own;; ++s) {
    const int q0 = gs + s * seg;
    if (q0 >= ge || (s > s_own && q0 - mem > j)) break;
    const int q1 = min(q0 + seg, ge);
    const int w = s == s_own ? 0 : 1;
    for (int i = q0; i < q1; ++i) {
      const float* qr = qkv + (size_t)i * ld + h * DH;
      const float* dor = dO + (size_t)i * d + h * DH;
      float sc = 0.f, dp = 0.f;
#pragma unroll
      for (int t = 0; t < DH; ++t) {
        sc = fmaf(qr[t] * scale, kr[t], sc);
        dp = fmaf(dor[t], vr[t], dp);
      }
      const float p = expf(sc - lse[(size_t)i * heads + h]);
      const float ds = p * (dp - Dq[(size_t)i * heads + h]);
      if (w == 0) {
#pragma unroll
        for (int t = 0; t < DH; ++t) {
          dv[0][t] = fmaf(p, dor[t], dv[0][t]);
          dk[0][t] = fmaf(ds, qr[t], dk[0][t]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < DH; ++t) {
          dv[1][t] = fmaf(p, dor[t], dv[1][t]);
          dk[1][t] = fmaf(ds, qr[t], dk[1][t]);
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < DH; ++t) {
    dqkv_live[(size_t)j * ldl + d + h * DH + t] = dk[0][t] * scale;
    dqkv_live[(size_t)j * ldl + 2 * d + h * DH + t] = dv[0][t];
    dkv_mem[(size_t)j * ldm + h * DH + t] = dk[1][t] * scale;
    dkv_mem[(size_t)j * ldm + d + h * DH + t] = dv[1][t];
  }
}

// Dq[v][h] = dO[v] . O[v] over the head's columns
__global__ void k_attn_dq_rowdot(const float* dO, const float* O, int n, int d, int heads, float* Dq) {
  const size_t total = (size_t)n * heads;
  const int dh = d / heads;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int v = (int)(i / heads), h = (int)(i % heads);
    float s = 0.f;
    for (int t = 0; t < dh; ++t) s = fmaf(dO[(size_t)v * d + h * dh + t], O[(size_t)v * d + h * dh + t], s);
    Dq[i] = s;
  }
}

hipError_t launch_attn_fwd(const float* qkv, int n, int d, int heads, int seg, int mem, const GraphTable& gt,
                           float* o, float* lse, hipStream_t s) {
  const int dh = d / heads;
  const float scale = 1.0f / sqrtf((float)dh);
  dim3 grid((n + 63) / 64, heads);
  switch (dh) {
    case 16: hipLaunchKernelGGL((k_attn_fwd<16>), grid, dim3(64), 0, s, qkv, n, d, heads, seg, mem, gt, scale, o, lse); break;
    case 32: hipLaunchKernelGGL((k_attn_fwd<32>), grid, dim3(64), 0, s, qkv, n, d, heads, seg, mem, gt, scale, o, lse); break;
    case 64: hipLaunchKernelGGL((k_attn_fwd<64>), grid, dim3(64), 0, s, qkv, n, d, heads, seg, mem, gt, scale, o, lse); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const float* qkv, const float* O, const float* dO, const float* lse, int n, int d,
                           int heads, int seg, int mem, const GraphTable& gt, float* Dq, float* dqkv_live,
                           float* dkv_mem, hipStream_t s) {
  const int dh = d / heads;
  const float scale = 1.0f / sqrtf((float)dh);
  {
    const size_t total = (size_t)n * heads;
    const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(k_attn_dq_rowdot, dim3(blocks), dim3(256), 0, s, dO, O, n, d, heads, Dq);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  dim3 grid((n + 63) / 64, heads);
#define GDP_ATTN_BWD(DH)                                                                                         \
  hipLaunchKernelGGL((k_attn_bwd_q<DH>), grid, dim3(64), 0, s, qkv, dO, (const float*)Dq, lse, n, d, heads, seg, \
                     mem, gt, scale, dqkv_live, 3 * d);                                                         \
  hipLaunchKernelGGL((k_attn_bwd_kv<DH>), grid, dim3(64), 0, s, qkv, dO, (const float*)Dq, lse, n, d, heads, seg, \
                     mem, gt, scale, dqkv_live, 3 * d, dkv_mem, 2 * d);
  switch (dh) {
    case 16: GDP_ATTN_BWD(16) break;
    case 32: GDP_ATTN_BWD(32) break;
    case 64: GDP_ATTN_BWD(64) break;
    default: return hipErrorInvalidValue;
  }
#undef GDP_ATTN_BWD
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Adam (Kingma and Ba, 2015) on one parameter tensor: fp32 master weights and
// moments; the dtype copy the kernels read is rewritten from the master.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_adam(float* master, T* param, const float* grad, float* m, float* v, int64_t n, float lr, float b1,
                       float b2, float eps, float c1, float c2) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float g = grad[i];
    const float mi = b1 * m[i] + (1.0f - b1) * g;
    const float vi = b2 * v[i] + (1.0f - b2) * g * g;
    m[i] = mi;
    v[i] = vi;
    const float w = master[i] - lr * (mi / c1) / (sqrtf(vi / c2) + eps);
    master[i] = w;
    param[i] = from_f32<T>(w);
  }
}
template <typename T>
hipError_t launch_adam(float* master, T* param, const float* grad, float* m, float* v, int64_t n, float lr, float b1,
                       float b2, float eps, float c1, float c2, hipStream_t s) {
  const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL((k_adam<T>), dim3(std::max(1u, blocks)), dim3(256), 0, s, master, param, grad, m, v, n, lr, b1,
                     b2, eps, c1, c2);
  return hipGetLastError();
}
template hipError_t launch_adam<float>(float*, float*, const float*, float*, float*, int64_t, float, float, float,
                                       float, float, float, hipStream_t);
template hipError_t launch_adam<bf16>(float*, bf16*, const float*, float*, float*, int64_t, float, float, float,
                                      float, float, float, hipStream_t);

}  // namespace tr
}  // namespace gdp
