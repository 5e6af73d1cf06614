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
#include "host_plan.h"
#include "train_kernels.h"

namespace gdp {
namespace tr {

__device__ __forceinline__ float ld(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ld(const bf16* p, size_t i) { return (float)p[i]; }

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// Strided GEMM on the fp32 matrix cores (16x16x4 MFMA): C(m, n) = epi(alpha *
// sum_k A(m, k) B(k, n)).  A work-group (4 waves, 2 x 2) owns a BM x BM tile
// of C, each wave a (BM/2)^2 block of 16 x 16 MFMA tiles; k advances in steps
// of 16 through LDS tiles stored k-major (As[k][m], Bs[k][n], rows padded by
// 16 floats so the 4 lane groups of a fragment read fall in distinct banks),
// the next step's operands loaded into registers during this step's MFMAs.
// With splits > 1, grid.z splits k and each split writes its raw sums to
// partial[z]; gemm_reduce adds them in split order and applies the epilogue.
// ---------------------------------------------------------------------------
constexpr int GBK = 16;

// Operand tile loader: R x GBK (A: R = rows m) or GBK x R (B: R = columns n)
// elements, 4 consecutive elements of the fast dimension per vector.
template <typename T, int R>
struct TileLoad {
  static constexpr int NV = R * GBK / 4 / 256;      // vectors per thread
  float v[NV][4];
  // element (r, k) = p[r * sr + k * sk]; kfast: sk == 1 (vectors along k),
  // else sr == 1 (vectors along r); vec: every vector aligned and in one piece.
  __device__ __forceinline__ void load(const T* p, long sr, long sk, bool kfast, bool vec, int r0, int rmax, int k0,
                                       int kmax) {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int r = kfast ? e / (GBK / 4) : (e % (R / 4)) * 4;
      const int k = kfast ? (e % (GBK / 4)) * 4 : e / (R / 4);
#pragma unroll
      for (int t = 0; t < 4; ++t) v[q][t] = 0.f;
      const int rr = r0 + r, kk = k0 + k;
      if (vec && (kfast ? (rr < rmax && kk + 3 < kmax) : (rr + 3 < rmax && kk < kmax))) {
        load4(p + (size_t)rr * sr + (size_t)kk * sk, v[q]);
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int r2 = kfast ? rr : rr + t, k2 = kfast ? kk + t : kk;
          if (r2 < rmax && k2 < kmax) v[q][t] = ld(p, (size_t)r2 * sr + (size_t)k2 * sk);
        }
      }
    }
  }
  __device__ __forceinline__ void store(float* s, bool kfast) const {
    constexpr int LS = R + 16;
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int e = threadIdx.x + 256 * q;
      if (kfast) {
        const int r = e / (GBK / 4), k = (e % (GBK / 4)) * 4;
#pragma unroll
        for (int t = 0; t < 4; ++t) s[(k + t) * LS + r] = v[q][t];
      } else {
        const int r = (e % (R / 4)) * 4, k = e / (R / 4);
        *reinterpret_cast<float4*>(&s[k * LS + r]) = make_float4(v[q][0], v[q][1], v[q][2], v[q][3]);
      }
    }
  }
  static __device__ __forceinline__ void load4(const float* p, float (&o)[4]) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    o[0] = t.x; o[1] = t.y; o[2] = t.z; o[3] = t.w;
  }
  static __device__ __forceinline__ void load4(const bf16* p, float (&o)[4]) {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    o[0] = __uint_as_float(t.x << 16); o[1] = __uint_as_float(t.x & 0xffff0000u);
    o[2] = __uint_as_float(t.y << 16); o[3] = __uint_as_float(t.y & 0xffff0000u);
  }
};

template <typename TA, typename TB>
__device__ __forceinline__ void gemm_epilogue(const GemmStrided<TA, TB>& g, int m, int n, float acc) {
  float v = g.alpha * acc;
  if (g.bias_f) v += g.bias_f[n];
  if (g.bias_h) v += (float)g.bias_h[n];
  if (g.act == ACT_RELU) v = fmaxf(v, 0.f);
  else if (g.act == ACT_SIGMOID) v = sigmoidf_(v);
  if (g.mask && !(g.mask[(size_t)m * g.ldm + n] > 0.f)) v = 0.f;
  float* c = g.c + (size_t)m * g.ldc + n;
  *c = g.accumulate ? *c + v : v;
}

// vec_a / vec_b: the operand's vectors are aligned (host-checked).
template <typename TA, typename TB, int BM>
__global__ __launch_bounds__(256) void k_gemm_strided(GemmStrided<TA, TB> g, int k_per_split, float* partial,
                                                      int vec_a, int vec_b) {
  constexpr int WT = BM / 2, NB = WT / 16, LS = BM + 16;
  __shared__ __attribute__((aligned(16))) float As[GBK * LS];
  __shared__ __attribute__((aligned(16))) float Bs[GBK * LS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, g4 = lane >> 4;
  const int mw = (wave >> 1) * WT, nw = (wave & 1) * WT;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BM;
  const int kb = blockIdx.z * k_per_split, ke = min(g.K, kb + k_per_split);
  const bool a_kfast = g.sak == 1, b_kfast = g.sbk == 1;
  f32x4 acc[NB][NB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = zero4();
  TileLoad<TA, BM> la;
  TileLoad<TB, BM> lb;
  la.load(g.a, g.sam, g.sak, a_kfast, vec_a, m0, g.M, kb, ke);
  lb.load(g.b, g.sbn, g.sbk, b_kfast, vec_b, n0, g.N, kb, ke);
  for (int k0 = kb; k0 < ke; k0 += GBK) {
    __syncthreads();                 // the previous step's fragment reads are done
    la.store(As, a_kfast);
    lb.store(Bs, b_kfast);
    __syncthreads();
    if (k0 + GBK < ke) {
      la.load(g.a, g.sam, g.sak, a_kfast, vec_a, m0, g.M, k0 + GBK, ke);
      lb.load(g.b, g.sbn, g.sbk, b_kfast, vec_b, n0, g.N, k0 + GBK, ke);
    }
#pragma unroll
    for (int ks = 0; ks < GBK / 4; ++ks) {
      float a[NB], b[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) a[i] = As[(ks * 4 + g4) * LS + mw + 16 * i + col];
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = Bs[(ks * 4 + g4) * LS + nw + 16 * j + col];
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  // lane: C rows mw + 16 i + 4 g4 + r, column nw + 16 j + col
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + mw + 16 * i + 4 * g4 + r, n = n0 + nw + 16 * j + col;
        if (m >= g.M || n >= g.N) continue;
        if (partial) partial[((size_t)blockIdx.z * g.M + m) * g.N + n] = acc[i][j][r];
        else gemm_epilogue(g, m, n, acc[i][j][r]);
      }
}

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void k_gemm_reduce(GemmStrided<TA, TB> g, int splits, const float* partial) {
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i >= (size_t)g.M * g.N) return;
  const int m = (int)(i / g.N), n = (int)(i % g.N);
  double s = 0.0;   // the splits' sums added in double: long reductions (k = rows) keep fp32 accuracy
  for (int z = 0; z < splits; ++z) s += (double)partial[(size_t)z * g.M * g.N + i];
  gemm_epilogue(g, m, n, (float)s);
}

// Vectors of 4 elements of T along the fast dimension are aligned when the
// base and the other dimension's stride are multiples of 4 elements.
template <typename T>
static bool vec_aligned(const T* p, long stride) {
  return ((uintptr_t)p % (4 * sizeof(T))) == 0 && stride % 4 == 0;
}

template <typename TA, typename TB>
hipError_t launch_gemm_strided(const GemmStrided<TA, TB>& g, float* partial, size_t partial_floats, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if ((g.sak != 1 && g.sam != 1) || (g.sbk != 1 && g.sbn != 1)) return hipErrorInvalidValue;
  int splits = 1;
  // a long reduction (the weight gradients, k = rows) is split into pieces of
  // at most kSplitRows, each summed in fp32, the pieces added in double
  constexpr int kSplitRows = 1024;
  if (partial && g.K > kSplitRows) {
    splits = (g.K + kSplitRows - 1) / kSplitRows;
    while (splits > 1 && (size_t)splits * g.M * g.N > partial_floats) --splits;
  }
  const int kps = splits > 1 ? (((g.K + splits - 1) / splits + GBK - 1) / GBK) * GBK : std::max(g.K, 1);
  splits = splits > 1 ? (g.K + kps - 1) / kps : 1;
  const int va = vec_aligned(g.a, g.sak == 1 ? g.sam : g.sak) ? 1 : 0;
  const int vb = vec_aligned(g.b, g.sbk == 1 ? g.sbn : g.sbk) ? 1 : 0;
  float* part = splits > 1 ? partial : nullptr;
  // 128 x 128 tiles when they give at least two work-groups per CU, else 64 x 64
  const long tiles128 = (long)((g.M + 127) / 128) * ((g.N + 127) / 128) * splits;
  if (tiles128 >= 512) {
    dim3 grid((g.N + 127) / 128, (g.M + 127) / 128, splits);
    hipLaunchKernelGGL((k_gemm_strided<TA, TB, 128>), grid, dim3(256), 0, s, g, kps, part, va, vb);
  } else {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, splits);
    hipLaunchKernelGGL((k_gemm_strided<TA, TB, 64>), grid, dim3(256), 0, s, g, kps, part, va, vb);
  }
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
  // eight interleaved partial sums (rows r0 + 8 i + u go to sum u), combined in order
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  int r = r0;
  for (; r + 8 <= r1; r += 8) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float v = ld(a, (size_t)(r + u) * lda + c);
      if (b) v *= b[(size_t)(r + u) * ldb + c];
      s[u] += v;
    }
  }
  for (; r < r1; ++r) {             // the last (at most 7) rows into sum 0
    float v = ld(a, (size_t)r * lda + c);
    if (b) v *= b[(size_t)r * ldb + c];
    s[0] += v;
  }
  partial[(size_t)chunk * C + c] = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

// out[g][c] (+)= the graph's chunk sums added in double; 64 columns x 4 chunk
// quarters per work-group, the quarters combined in order.
__global__ __launch_bounds__(256) void k_colsum_final(const float* partial, int C, GraphTable ct, float* out, int ldo,
                                                      int accumulate) {
  __shared__ double q4[4][64];
  const int g = blockIdx.y;
  const int cl = threadIdx.x & 63, part = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + cl;
  const int k0 = ct.blk[g], k1 = ct.blk[g + 1];
  const int per = (k1 - k0 + 3) / 4;
  const int ka = k0 + part * per, kz = min(k1, ka + per);
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  if (c < C) {
    int k = ka;
    for (; k + 4 <= kz; k += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) s[u] += (double)partial[(size_t)(k + u) * C + c];
    }
    for (; k < kz; ++k) s[0] += (double)partial[(size_t)k * C + c];
  }
  q4[part][cl] = (s[0] + s[1]) + (s[2] + s[3]);
  __syncthreads();
  if (part == 0 && c < C) {
    const double t = (q4[0][cl] + q4[1][cl]) + (q4[2][cl] + q4[3][cl]);
    float* o = out + (size_t)g * ldo + c;
    *o = accumulate ? *o + (float)t : (float)t;
  }
}

template <typename TA>
hipError_t launch_colsum(const TA* a, int lda, const float* b, int ldb, int C, const GraphTable& ct, int chunks,
                         float* partial, float* out, int ldo, bool accumulate, hipStream_t s) {
  if (C <= 0 || chunks <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_colsum_partial<TA>), dim3((C + 255) / 256, chunks), dim3(256), 0, s, a, lda, b, ldb, C, ct,
                     partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_colsum_final, dim3((C + 63) / 64, ct.n), dim3(256), 0, s, (const float*)partial, C, ct, out,
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
// Segment attention in fp32 for training, on the fp32 matrix cores
// (16x16x4 MFMA).  Band form: the queries of a segment [seg0, seg1) of graph
// g attend to keys [max(g_start, seg0 - mem_len), seg1).  qkv: [n, 3d]
// (Q | K | V, heads contiguous).
//
// A work-group is 4 waves and one head; it owns 64 queries (forward, dQ) or
// 64 keys (dK, dV) of one segment, 16 a wave, one per lane column.  Scores are
// formed transposed, S^T = K Q^T (or S = Q K^T for the key-side kernel), so
// that a lane's accumulator holds 4 keys (queries) of its own column, rows
// 4 (lane / 16) + r.  The next product contracts over those keys (queries);
// ordering its k steps as {16 b + 4 g + r : g = 0..3} for r = 0..3 lets each
// lane pass its own accumulator values as the B operand, with the A operand
// read transposed from LDS.  Products over the head dimension order it as
// dim = (lane / 16) * DH / 4 + kk at k step kk, so that a lane's operand
// values are DH / 4 consecutive floats.  Scores are kept in log2 units (Q
// pre-multiplied by log2(e) / sqrt(d_h)).
// ---------------------------------------------------------------------------
constexpr int kAttnRows = 64;    // queries (keys) per work-group, 16 per wave
constexpr int kAttnTile = 64;    // keys (queries) staged per tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// The segment rows [r0, r1) of work block b (segments split into blocks of
// kAttnRows rows; gt.blk the per-graph prefix of blocks).
struct SegRows {
  int gs, ge, seg0, seg1, r0, r1;
};
__device__ __forceinline__ SegRows seg_rows(const GraphTable& gt, int b, int seg) {
  const int g = graph_of_block(gt, b);
  const int per = (seg + kAttnRows - 1) / kAttnRows;
  const int local = b - gt.blk[g];
  SegRows s;
  s.gs = gt.ptr[g];
  s.ge = gt.ptr[g + 1];
  s.seg0 = s.gs + (local / per) * seg;
  s.seg1 = min(s.seg0 + seg, s.ge);
  s.r0 = s.seg0 + (local % per) * kAttnRows;
  s.r1 = min(s.r0 + kAttnRows, s.seg1);
  return s;
}

// Rows [t0, t0 + kAttnTile) of columns [c0, c0 + DH) of src (row stride ld) into
// LDS, row-major with row stride DH + 4 (rows at or past t1 as zeros), times mul.
template <int DH>
__device__ __forceinline__ void stage_rows(float* dst, const float* src, int ld, int c0, int t0, int t1, float mul) {
  constexpr int C4 = DH / 4;
  for (int e = threadIdx.x; e < kAttnTile * C4; e += 256) {
    const int r = e / C4, c = (e % C4) * 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t0 + r < t1) v = *reinterpret_cast<const float4*>(src + (size_t)(t0 + r) * ld + c0 + c);
    v.x *= mul; v.y *= mul; v.z *= mul; v.w *= mul;
    *reinterpret_cast<float4*>(dst + r * (DH + 4) + c) = v;
  }
}
// The same rows transposed: dst[c][r], row stride kAttnTile + 4.
template <int DH>
__device__ __forceinline__ void stage_cols(float* dst, const float* src, int ld, int c0, int t0, int t1) {
  constexpr int C4 = DH / 4, TS = kAttnTile + 4;
  for (int e = threadIdx.x; e < kAttnTile * C4; e += 256) {
    const int r = e % kAttnTile, c = (e / kAttnTile) * 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t0 + r < t1) v = *reinterpret_cast<const float4*>(src + (size_t)(t0 + r) * ld + c0 + c);
    dst[(c + 0) * TS + r] = v.x;
    dst[(c + 1) * TS + r] = v.y;
    dst[(c + 2) * TS + r] = v.z;
    dst[(c + 3) * TS + r] = v.w;
  }
}

// acc[b] (b = 0..3, 16 rows each) += X[b*16 + col][dims] . y[dims] over the head
// dimension: X a row-major LDS tile (stride DH + 4), y the lane's B operand.
template <int DH>
__device__ __forceinline__ void dot_tile(f32x4 (&acc)[4], const float* X, const float (&y)[DH / 4], int col, int g4) {
  constexpr int KT = DH / 4;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    acc[b] = zero4();
    const float* xr = X + (b * 16 + col) * (DH + 4) + g4 * KT;
    float x[KT];
#pragma unroll
    for (int k = 0; k < KT; k += 4) *reinterpret_cast<float4*>(&x[k]) = *reinterpret_cast<const float4*>(xr + k);
#pragma unroll
    for (int k = 0; k < KT; ++k) acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(x[k], y[k], acc[b], 0, 0, 0);
  }
}

// out[db] (head-dim rows db*16 + .., the lane's column) += Y^T . w over the 64
// tile rows: Y^T a transposed LDS tile (stride kAttnTile + 4), w[b][r] the
// lane's accumulator values for tile rows b*16 + 4 g4 + r.
template <int DH>
__device__ __forceinline__ void acc_tile(f32x4 (&out)[DH / 16], const float* Yt, const f32x4 (&w)[4], int col, int g4) {
#pragma unroll
  for (int db = 0; db < DH / 16; ++db)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const float4 y = *reinterpret_cast<const float4*>(Yt + (db * 16 + col) * (kAttnTile + 4) + b * 16 + 4 * g4);
      out[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(y.x, w[b][0], out[db], 0, 0, 0);
      out[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(y.y, w[b][1], out[db], 0, 0, 0);
      out[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(y.z, w[b][2], out[db], 0, 0, 0);
      out[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(y.w, w[b][3], out[db], 0, 0, 0);
    }
}

// The lane's DH / 4 operand values of row v: src[v][c0 + g4 * DH/4 + k] * mul.
template <int DH>
__device__ __forceinline__ void lane_operand(float (&y)[DH / 4], const float* src, size_t ld, int v, bool ok, int c0,
                                             int g4, float mul) {
  constexpr int KT = DH / 4;
#pragma unroll
  for (int k = 0; k < KT; k += 4) {
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    if (ok) t = *reinterpret_cast<const float4*>(src + (size_t)v * ld + c0 + g4 * KT + k);
    y[k] = t.x * mul; y[k + 1] = t.y * mul; y[k + 2] = t.z * mul; y[k + 3] = t.w * mul;
  }
}

template <int DH>
__global__ __launch_bounds__(256) void k_attn_fwd(const float* __restrict__ qkv, int d, int heads, int seg, int mem,
                                                  GraphTable gt, float scale, float* __restrict__ o,
                                                  float* __restrict__ lse) {
  constexpr int DB = DH / 16;
  __shared__ __attribute__((aligned(16))) float sK[kAttnTile * (DH + 4)];
  __shared__ __attribute__((aligned(16))) float sVt[DH * (kAttnTile + 4)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, g4 = lane >> 4;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int head = logical % heads;
  const SegRows b = seg_rows(gt, logical / heads, seg);
  const int ld = 3 * d;
  const int k0 = max(b.gs, b.seg0 - mem), k1 = b.seg1;
  const int q = b.r0 + wave * 16 + col;
  const bool qok = q < b.r1;
  float qf[DH / 4];
  lane_operand<DH>(qf, qkv, ld, q, qok, head * DH, g4, scale * kLog2e);
  f32x4 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = zero4();
  float m = -INFINITY, lsum = 0.f;
  for (int t0 = k0; t0 < k1; t0 += kAttnTile) {
    __syncthreads();
    stage_rows<DH>(sK, qkv, ld, d + head * DH, t0, k1, 1.0f);
    stage_cols<DH>(sVt, qkv, ld, 2 * d + head * DH, t0, k1);
    __syncthreads();
    f32x4 s[4];
    dot_tile<DH>(s, sK, qf, col, g4);
    float tmax = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (t0 + kb * 16 + 4 * g4 + r >= k1) s[kb][r] = -INFINITY;
        tmax = fmaxf(tmax, s[kb][r]);
      }
    tmax = fmaxf(tmax, xor_shfl(tmax, 16));
    tmax = fmaxf(tmax, xor_shfl(tmax, 32));
    const float mn = fmaxf(m, tmax);
    const float corr = exp2f(m - mn);
    m = mn;
    lsum *= corr;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 4; ++r) oacc[db][r] *= corr;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        s[kb][r] = exp2f(s[kb][r] - mn);
        lsum += s[kb][r];
      }
    acc_tile<DH>(oacc, sVt, s, col, g4);
  }
  lsum += xor_shfl(lsum, 16);
  lsum += xor_shfl(lsum, 32);
  if (qok) {
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<float4*>(o + (size_t)q * d + head * DH + db * 16 + 4 * g4) =
          make_float4(oacc[db][0] * inv, oacc[db][1] * inv, oacc[db][2] * inv, oacc[db][3] * inv);
    if (g4 == 0) lse[(size_t)q * heads + head] = (m + log2f(lsum)) * kLn2;
  }
}

// dQ for the work-group's queries: p = exp(s - lse), ds = p (dO . v - Dq),
// dq = scale * sum_j ds_j k_j (into the Q columns of dqkv, row stride lddq).
template <int DH>
__global__ __launch_bounds__(256) void k_attn_bwd_q(const float* __restrict__ qkv, const float* __restrict__ dO,
                                                    const float* __restrict__ Dq, const float* __restrict__ lse,
                                                    int d, int heads, int seg, int mem, GraphTable gt, float scale,
                                                    float* __restrict__ dqkv, int lddq) {
  constexpr int DB = DH / 16;
  __shared__ __attribute__((aligned(16))) float sK[kAttnTile * (DH + 4)];
  __shared__ __attribute__((aligned(16))) float sV[kAttnTile * (DH + 4)];
  __shared__ __attribute__((aligned(16))) float sKt[DH * (kAttnTile + 4)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, g4 = lane >> 4;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int head = logical % heads;
  const SegRows b = seg_rows(gt, logical / heads, seg);
  const int ld = 3 * d;
  const int k0 = max(b.gs, b.seg0 - mem), k1 = b.seg1;
  const int q = b.r0 + wave * 16 + col;
  const bool qok = q < b.r1;
  float qf[DH / 4], df[DH / 4];
  lane_operand<DH>(qf, qkv, ld, q, qok, head * DH, g4, scale * kLog2e);
  lane_operand<DH>(df, dO, d, q, qok, head * DH, g4, 1.0f);
  const float L2 = qok ? lse[(size_t)q * heads + head] * kLog2e : 0.f;
  const float Dv = qok ? Dq[(size_t)q * heads + head] : 0.f;
  f32x4 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dq[db] = zero4();
  for (int t0 = k0; t0 < k1; t0 += kAttnTile) {
    __syncthreads();
    stage_rows<DH>(sK, qkv, ld, d + head * DH, t0, k1, 1.0f);
    stage_rows<DH>(sV, qkv, ld, 2 * d + head * DH, t0, k1, 1.0f);
    stage_cols<DH>(sKt, qkv, ld, d + head * DH, t0, k1);
    __syncthreads();
    f32x4 s[4], dp[4];
    dot_tile<DH>(s, sK, qf, col, g4);
    dot_tile<DH>(dp, sV, df, col, g4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = t0 + kb * 16 + 4 * g4 + r < k1;
        s[kb][r] = ok ? exp2f(s[kb][r] - L2) * (dp[kb][r] - Dv) : 0.f;
      }
    acc_tile<DH>(dq, sKt, s, col, g4);
  }
  if (qok) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<float4*>(dqkv + (size_t)q * lddq + head * DH + db * 16 + 4 * g4) =
          make_float4(dq[db][0] * scale, dq[db][1] * scale, dq[db][2] * scale, dq[db][3] * scale);
  }
}

// dK, dV for the work-group's keys, from the queries of their own segment
// (live: the key's row receives the gradient) and separately from the later
// segments whose memory holds them (that part stops at the projection
// weights: the memory passes no gradient to its rows).
template <int DH>
__global__ __launch_bounds__(256) void k_attn_bwd_kv(const float* __restrict__ qkv, const float* __restrict__ dO,
                                                     const float* __restrict__ Dq, const float* __restrict__ lse,
                                                     int d, int heads, int seg, int mem, GraphTable gt, float scale,
                                                     float* __restrict__ dqkv_live, int ldl,
                                                     float* __restrict__ dkv_mem, int ldm) {
  constexpr int DB = DH / 16;
  __shared__ __attribute__((aligned(16))) float sQ[kAttnTile * (DH + 4)];
  __shared__ __attribute__((aligned(16))) float sD[kAttnTile * (DH + 4)];
  __shared__ __attribute__((aligned(16))) float sQt[DH * (kAttnTile + 4)];
  __shared__ __attribute__((aligned(16))) float sDt[DH * (kAttnTile + 4)];
  __shared__ float sL[kAttnTile], sDq[kAttnTile];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, col = lane & 15, g4 = lane >> 4;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int head = logical % heads;
  const SegRows b = seg_rows(gt, logical / heads, seg);
  const int ld = 3 * d;
  const int key = b.r0 + wave * 16 + col;
  const bool kok = key < b.r1;
  float kf[DH / 4], vf[DH / 4];
  lane_operand<DH>(kf, qkv, ld, key, kok, d + head * DH, g4, 1.0f);
  lane_operand<DH>(vf, qkv, ld, key, kok, 2 * d + head * DH, g4, 1.0f);
  f32x4 dk[2][DB], dv[2][DB];
#pragma unroll
  for (int w = 0; w < 2; ++w)
#pragma unroll
    for (int db = 0; db < DB; ++db) dk[w][db] = dv[w][db] = zero4();
  // the key's own segment, then later segments whose band starts before r1
  for (int sg0 = b.seg0; sg0 < b.ge && (sg0 == b.seg0 || sg0 - mem < b.r1); sg0 += seg) {
    const int sg1 = min(sg0 + seg, b.ge);
    const int w = sg0 == b.seg0 ? 0 : 1;
    const bool seen = w == 0 || key >= sg0 - mem;        // the band of segment sg0 holds the key
    for (int t0 = sg0; t0 < sg1; t0 += kAttnTile) {
      __syncthreads();
      stage_rows<DH>(sQ, qkv, ld, head * DH, t0, sg1, scale * kLog2e);
      stage_rows<DH>(sD, dO, d, head * DH, t0, sg1, 1.0f);
      stage_cols<DH>(sQt, qkv, ld, head * DH, t0, sg1);
      stage_cols<DH>(sDt, dO, d, head * DH, t0, sg1);
      if (threadIdx.x < kAttnTile) {
        const int qi = t0 + threadIdx.x;
        sL[threadIdx.x] = qi < sg1 ? lse[(size_t)qi * heads + head] * kLog2e : 0.f;
        sDq[threadIdx.x] = qi < sg1 ? Dq[(size_t)qi * heads + head] : 0.f;
      }
      __syncthreads();
      f32x4 s[4], dp[4];
      dot_tile<DH>(s, sQ, kf, col, g4);
      dot_tile<DH>(dp, sD, vf, col, g4);
#pragma unroll
      for (int qb = 0; qb < 4; ++qb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int qi = qb * 16 + 4 * g4 + r;
          const float p = seen && t0 + qi < sg1 ? exp2f(s[qb][r] - sL[qi]) : 0.f;
          s[qb][r] = p;
          dp[qb][r] = p * (dp[qb][r] - sDq[qi]);
        }
      if (w == 0) {
        acc_tile<DH>(dv[0], sDt, s, col, g4);
        acc_tile<DH>(dk[0], sQt, dp, col, g4);
      } else {
        acc_tile<DH>(dv[1], sDt, s, col, g4);
        acc_tile<DH>(dk[1], sQt, dp, col, g4);
      }
    }
  }
  if (kok) {
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int c = head * DH + db * 16 + 4 * g4;
      *reinterpret_cast<float4*>(dqkv_live + (size_t)key * ldl + d + c) =
          make_float4(dk[0][db][0] * scale, dk[0][db][1] * scale, dk[0][db][2] * scale, dk[0][db][3] * scale);
      *reinterpret_cast<float4*>(dqkv_live + (size_t)key * ldl + 2 * d + c) =
          make_float4(dv[0][db][0], dv[0][db][1], dv[0][db][2], dv[0][db][3]);
      *reinterpret_cast<float4*>(dkv_mem + (size_t)key * ldm + c) =
          make_float4(dk[1][db][0] * scale, dk[1][db][1] * scale, dk[1][db][2] * scale, dk[1][db][3] * scale);
      *reinterpret_cast<float4*>(dkv_mem + (size_t)key * ldm + d + c) =
          make_float4(dv[1][db][0], dv[1][db][1], dv[1][db][2], dv[1][db][3]);
    }
  }
}

// Dq[v][h] = dO[v] . O[v] over the head's columns, one thread per (v, h).
template <int DH>
__global__ void k_attn_dq_rowdot(const float* __restrict__ dO, const float* __restrict__ O, int n, int d, int heads,
                                 float* __restrict__ Dq) {
  const size_t total = (size_t)n * heads;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const size_t base = (i / heads) * d + (i % heads) * DH;
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < DH; t += 4) {
      const float4 a = *reinterpret_cast<const float4*>(dO + base + t);
      const float4 c = *reinterpret_cast<const float4*>(O + base + t);
      s = fmaf(a.x, c.x, s);
      s = fmaf(a.y, c.y, s);
      s = fmaf(a.z, c.z, s);
      s = fmaf(a.w, c.w, s);
    }
    Dq[i] = s;
  }
}

// The attention blocks of every graph: segments in blocks of kAttnRows rows.
static int attn_table(const GraphTable& gt, int seg, GraphTable* t) {
  *t = gt;
  return prefix_blocks_attention(t->ptr, t->n, seg, kAttnRows, t->blk);
}

hipError_t launch_attn_fwd(const float* qkv, int n, int d, int heads, int seg, int mem, const GraphTable& gt,
                           float* o, float* lse, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int dh = d / heads;
  const float scale = 1.0f / sqrtf((float)dh);
  GraphTable t;
  const int blocks = attn_table(gt, seg, &t);
  dim3 grid(blocks * heads), block(256);
  switch (dh) {
    case 16: hipLaunchKernelGGL((k_attn_fwd<16>), grid, block, 0, s, qkv, d, heads, seg, mem, t, scale, o, lse); break;
    case 32: hipLaunchKernelGGL((k_attn_fwd<32>), grid, block, 0, s, qkv, d, heads, seg, mem, t, scale, o, lse); break;
    case 64: hipLaunchKernelGGL((k_attn_fwd<64>), grid, block, 0, s, qkv, d, heads, seg, mem, t, scale, o, lse); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const float* qkv, const float* O, const float* dO, const float* lse, int n, int d,
                           int heads, int seg, int mem, const GraphTable& gt, float* Dq, float* dqkv_live,
                           float* dkv_mem, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int dh = d / heads;
  const float scale = 1.0f / sqrtf((float)dh);
  GraphTable t;
  const int blocks = attn_table(gt, seg, &t);
  const unsigned rd_blocks = (unsigned)std::min<size_t>(((size_t)n * heads + 255) / 256, 8192);
  dim3 grid(blocks * heads), block(256);
#define GDP_ATTN_BWD(DH)                                                                                          \
  hipLaunchKernelGGL((k_attn_dq_rowdot<DH>), dim3(rd_blocks), dim3(256), 0, s, dO, O, n, d, heads, Dq);           \
  hipLaunchKernelGGL((k_attn_bwd_q<DH>), grid, block, 0, s, qkv, dO, (const float*)Dq, lse, d, heads, seg, mem, t, \
                     scale, dqkv_live, 3 * d);                                                                     \
  hipLaunchKernelGGL((k_attn_bwd_kv<DH>), grid, block, 0, s, qkv, dO, (const float*)Dq, lse, d, heads, seg, mem,   \
                     t, scale, dqkv_live, 3 * d, dkv_mem, 2 * d);
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
