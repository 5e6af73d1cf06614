// Launch interface of the update-step kernels (train.hip): the training
// forward that keeps every intermediate, the backward pass and Adam, all in
// fp32 arithmetic.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace gdp {
namespace tr {

enum Act { ACT_NONE = 0, ACT_RELU = 1, ACT_SIGMOID = 2 };

// C(m, n) = epi(alpha * sum_k A(m, k) B(k, n)) with A(m, k) = a[m sam + k sak]
// and B(k, n) = b[k sbk + n sbn]; epi adds a bias over n (fp32 or bf16),
// applies act, zeroes where mask[m ldm + n] <= 0, and writes or adds to c.
template <typename TA, typename TB>
struct GemmStrided {
  const TA* a;
  long sam, sak;
  const TB* b;
  long sbk, sbn;
  int M, N, K;
  float* c;
  long ldc;
  float alpha = 1.0f;
  const float* bias_f = nullptr;
  const bf16* bias_h = nullptr;
  int act = ACT_NONE;
  const float* mask = nullptr;
  long ldm = 0;
  bool accumulate = false;
};
// partial: scratch for split-k sums (partial_floats floats; null: no split).
template <typename TA, typename TB>
hipError_t launch_gemm_strided(const GemmStrided<TA, TB>& g, float* partial, size_t partial_floats, hipStream_t s);

// out[g][c] (+)= sum over graph g's rows of a[r][c] (* b[r][c]); ct holds the
// graphs and their 256-row chunks (chunks of them); partial: chunks * C floats.
constexpr int kColChunkRows = 256;
template <typename TA>
hipError_t launch_colsum(const TA* a, int lda, const float* b, int ldb, int C, const GraphTable& ct, int chunks,
                         float* partial, float* out, int ldo, bool accumulate, hipStream_t s);

template <typename T>
hipError_t launch_ln_fwd(const float* r, int n, int d, const T* g, const T* b, float* out, hipStream_t s);
// dr = LayerNorm backward; xg[r][c] = dout * xhat (the gain gradient's terms).
template <typename T>
hipError_t launch_ln_bwd(const float* r, const float* dout, int n, int d, const T* g, float* dr, float* xg,
                         hipStream_t s);

template <typename TX>
hipError_t launch_film_apply(const TX* x, int n, int d, const float* gamma, const float* beta, const GraphTable& gt,
                             float* y, hipStream_t s);
hipError_t launch_film_dx(const float* dy, int n, int d, const float* gamma, const GraphTable& gt, float* dx,
                          hipStream_t s);

enum Ew { EW_ADD = 0, EW_MASK_POS = 1, EW_SIGMOID_GRAD = 2, EW_SCALE_BY = 3 };
hipError_t launch_ew(int op, const float* a, const float* b, const float* c, size_t n, float* out, hipStream_t s);

// x0[g] = mean of graph g's rows of h; chunks: the graphs with their 256-row chunks (n_chunks of them),
// partial: n_chunks * H floats.
hipError_t launch_meanpool_f32(const float* h, int H, const GraphTable& chunks, int n_chunks, float* partial,
                               float* x0, hipStream_t s);
hipError_t launch_meanpool_bwd(const float* dx0, int n, int H, const GraphTable& gt, float* dh, hipStream_t s);

hipError_t launch_gather_max_arg(const float* P, const int* s_ptr, const int* s_idx, int n, int H, float* A, int* arg,
                                 hipStream_t s);
hipError_t launch_gather_max_bwd(const float* dA, const int* arg, const int* row_ptr, const int* col_idx,
                                 const int* in_ptr, const int* in_idx, int n, int H, float* dP, hipStream_t s);
hipError_t launch_sort_rows(const int* ptr, int n, int* idx, hipStream_t s);

// qkv [n, 3d] fp32; o [n, d]; lse [n, heads].
hipError_t launch_attn_fwd(const float* qkv, int n, int d, int heads, int seg, int mem, const GraphTable& gt,
                           float* o, float* lse, hipStream_t s);
// dqkv_live [n, 3d]: dQ and the own-segment dK, dV; dkv_mem [n, 2d]: the dK,
// dV that later segments' queries send to the row as memory; Dq [n, heads] scratch.
hipError_t launch_attn_bwd(const float* qkv, const float* O, const float* dO, const float* lse, int n, int d,
                           int heads, int seg, int mem, const GraphTable& gt, float* Dq, float* dqkv_live,
                           float* dkv_mem, hipStream_t s);

template <typename T>
hipError_t launch_adam(float* master, T* param, const float* grad, float* m, float* v, int64_t n, float lr, float b1,
                       float b2, float eps, float c1, float c2, hipStream_t s);

}  // namespace tr
}  // namespace gdp
