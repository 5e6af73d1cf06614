// Internal launch interface between the host API (gdp_api.hip) and the
// kernels.  Every launcher enqueues on `s` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdp.h"

namespace gdp {

struct GraphTable;

// ---- graph preparation and Section 3.1 -------------------------------------
hipError_t launch_fill_i32(int* p, int64_t n, int value, hipStream_t s);
hipError_t launch_in_degree(const int* col_idx, int64_t n_edges, int* in_deg, hipStream_t s);
// block_tmp: 2 * ceil(n / kScanBlock) ints of scratch.
constexpr int kScanBlock = 1024;
hipError_t launch_scan_degrees(const int* row_ptr, const int* in_deg, int n, int fanout,
                               int* in_ptr, int* s_ptr, int* block_tmp, hipStream_t s);
hipError_t launch_fill_reverse(const int* row_ptr, const int* col_idx, const int* in_ptr, int n,
                               int64_t n_edges, int* cursor, int* in_idx, hipStream_t s);
// heavy: n ints of scratch; heavy_count: one int, zero on entry.
hipError_t launch_nbr_sample(const int* row_ptr, const int* col_idx, const int* in_ptr,
                             const int* in_idx, const int* s_ptr, int n, int fanout,
                             uint64_t seed, const GraphTable& gt, int* s_idx, int* heavy,
                             int* heavy_count, hipStream_t s);
// A[v] = max over S(v) of P rows (0 if empty); P, A: [n, H] of type T.
template <typename T>
hipError_t launch_gather_max(const T* P, const int* s_ptr, const int* s_idx, int n, int H, T* A,
                             hipStream_t s);
// graph_emb[g] = mean of h rows of graph g (fixed-order two-pass reduction).
template <typename T>
hipError_t launch_meanpool(const T* h, int H, const GraphTable& chunks, int total_chunks,
                           float* partial, float* graph_emb, hipStream_t s);
constexpr int kMeanpoolRows = 64;

// ---- dense layers -------------------------------------------------------------
enum Epilogue { EPI_BIAS = 0, EPI_RELU = 1, EPI_SIGMOID = 2 };

// out[M, N] = act([a1 | a2] [w1 | w2]^T + bias): two K-segments, each with its
// own activation source and weight array (a2/w2 may be null with k2 = 0).
// TA: storage type of segment 1 of A (fp32 for the residual stream and the
// GNN's hidden layers); segment 2 of A, the weights and the MFMA use T; TO is
// the output type.
template <typename TA, typename T, typename TO>
struct GemmArgs {
  const TA* a1; int lda1; const T* w1; int k1;   // a1 [M, lda1], w1 [N, k1]
  const T* a2; int lda2; const T* w2; int k2;    // a2 [M, lda2], w2 [N, k2]
  const T* bias;    // [N]
  TO* out; int ldo;
  int M, N;
  // EPI_BIAS only: output columns [0, scale_cols) are multiplied by col_scale
  // (the pre-scaled Q of the attention's QKV projection).
  int scale_cols = 0;
  float col_scale = 1.0f;
};
template <typename TA, typename T, typename TO>
hipError_t launch_gemm(const GemmArgs<TA, T, TO>& a, int epi, hipStream_t s);
// The same product for N = 64, 128 or 256 and K segments that are multiples of
// the layer kernel's chunk (64 bf16 / 32 fp32 elements), with the whole output
// row held on chip; row_gemm_supported says whether a call qualifies.
template <typename T>
bool row_gemm_supported(const GemmArgs<T, T, T>& a);
template <typename T>
hipError_t launch_row_gemm(const GemmArgs<T, T, T>& a, int epi, hipStream_t s);
// Eq. 3's update (EPI_RELU, a.out = h') fused with the next layer's Eq. 2
// transform of the same rows: p_out = sigmoid(h' w_pool^T + b_pool), w_pool
// [N, N].  Needs row_gemm_supported(a) and N / chunk <= the A ring (bf16: N =
// 64, 128, 256; fp32: N = 64); row_gemm_pool_supported says whether it applies.
template <typename T>
struct RowPoolArgs {
  const T* w_pool;
  const T* b_pool;
  T* p_out;
  int ldp;
};
template <typename T>
bool row_gemm_pool_supported(const GemmArgs<T, T, T>& a, const RowPoolArgs<T>& q);
template <typename T>
hipError_t launch_row_gemm_pool(const GemmArgs<T, T, T>& a, const RowPoolArgs<T>& q, hipStream_t s);

// Everything of a placer layer after its attention, and the start of the next:
//   Z    = LN1(y + o W_o^T + b_o)
//   y'   = FiLM(LN2(Z + W_2 ReLU(W_1 Z + b_1) + b_2))   (FiLM of the next layer, optional)
//   qkv' = y' W_qkv^T + b_qkv                           (next layer's projection, optional)
// y and y' are the fp32 residual stream; d is 64, 128 or 256.
template <typename T>
struct PostAttnArgs {
  const T* o; int ldo;              // attention output [M, d]
  const float* y; int ldy;          // layer input [M, d]
  const T* w_o; const T* b_o;       // [d, d], [d]
  const T* ln1_g; const T* ln1_b;   // [d]
  const T* w1; const T* b1;         // [d_ff, d], [d_ff]
  const T* w2; const T* b2;         // [d, d_ff], [d]
  const T* ln2_g; const T* ln2_b;   // [d]
  const float* film_gamma;          // [G, film_stride] or null
  const float* film_beta;
  int film_stride;
  float* y_out; int ldyo;           // [M, d]
  const T* w_qkv; const T* b_qkv;   // [3d, d], [3d] or null
  T* qkv_out; int ldq;              // [M, ldq >= 3d]
  int M, d, d_ff;
  float q_scale = 1.0f;             // multiplies the q columns of qkv_out
  // Last layer only (then w_qkv is null and y_out may be null): the head,
  // logits [M, n_dev] = y' W_out^T + b_out and lse [M], for n_dev <= kFusedHeadDevices.
  const T* w_out = nullptr; const T* b_out = nullptr; int n_dev = 0;
  float* logits = nullptr; float* lse = nullptr;
  int row0 = 0;                     // the launch covers rows row0 .. M - 1
};
constexpr int kFusedHeadDevices = 8;
template <typename T>
hipError_t launch_post_attention(const PostAttnArgs<T>& a, const GraphTable& gt, hipStream_t s);

// The first layer's input and projection: y = FiLM_0(x) (identity when
// film_gamma is null) into the fp32 residual stream, qkv = y W_qkv^T + b_qkv
// with the q columns multiplied by q_scale.
template <typename T>
struct PreLayerArgs {
  const T* x; int ldx;              // node embeddings [M, d]
  const float* film_gamma;          // [G, film_stride] or null
  const float* film_beta;
  int film_stride;
  float* y_out; int ldyo;           // [M, d]
  const T* w_qkv; const T* b_qkv;   // [3d, d], [3d]
  T* qkv_out; int ldq;              // [M, ldq >= 3d]
  int M, d;
  float q_scale;
  int row0 = 0;                     // the launch covers rows row0 .. M - 1
};
template <typename T>
hipError_t launch_pre_layer(const PreLayerArgs<T>& a, const GraphTable& gt, hipStream_t s);

// The ablation's placer without attention (Section 4.4), all layers and the
// head in one kernel: X_0 = x; per layer Y = FiLM_l(X) (film: [L][2][G][d],
// gamma then beta, or null), X <- LN2_l(Y + W_2 ReLU(W_1 Y + b_1) + b_2); then
// logits = X W_out^T + b_out and lse when w_out is set (n_dev <= kFusedHeadDevices),
// and the final X (fp32) into y_out when that is set.
constexpr int kMlpMaxLayers = 16;
template <typename T>
struct MlpPlacerArgs {
  const T* x; int ldx;              // node embeddings [M, d]
  const float* film;
  int n_graphs;
  int n_layers;                     // 1 .. kMlpMaxLayers
  const T* w1[kMlpMaxLayers];       // [d_ff, d]
  const T* b1[kMlpMaxLayers];       // [d_ff]
  const T* w2[kMlpMaxLayers];       // [d, d_ff]
  const T* b2[kMlpMaxLayers];       // [d]
  const T* ln_g[kMlpMaxLayers];     // [d]
  const T* ln_b[kMlpMaxLayers];     // [d]
  int M, d, d_ff;
  const T* w_out; const T* b_out; int n_dev;
  float* logits; float* lse;
  float* y_out; int ldyo;
};
template <typename T>
hipError_t launch_mlp_placer(const MlpPlacerArgs<T>& a, const GraphTable& gt, hipStream_t s);

// ---- Section 3.2 / 3.3 --------------------------------------------------------
// Segment attention.  qkv: [N, 3d] with the q columns pre-scaled by
// attn_q_scale(d / heads); out: [N, d].  gt.blk = per-graph prefix of 128-query
// blocks.
template <typename T>
struct AttnArgs {
  const T* qkv; int ldq;
  T* out; int ldo;
  int d, heads, seg_len, mem_len;
  int total_qblocks;                // query blocks of this launch: qblock0 .. qblock0 + total_qblocks - 1
  int qblock0 = 0;
};
constexpr int kAttnBlockQ = 128;
// log2(e) / sqrt(d_head): the softmax runs in the log2 domain on 2^x.
inline float attn_q_scale(int d_head) { return 1.4426950408889634f / sqrtf((float)d_head); }
template <typename T>
hipError_t launch_attention(const AttnArgs<T>& a, const GraphTable& gt, hipStream_t s);

// gamma_l[g][c] = 1 + W_g,l x0_g + b_g,l and beta_l[g][c] = W_b,l x0_g + b_b,l for
// up to kFilmLayersPerLaunch placer layers l per launch; layer l at out + l * 2 * G * d.
constexpr int kFilmLayersPerLaunch = 16;
template <typename T>
struct FilmLayers {
  const T* wg[kFilmLayersPerLaunch];
  const T* bg[kFilmLayersPerLaunch];
  const T* wb[kFilmLayersPerLaunch];
  const T* bb[kFilmLayersPerLaunch];
};
template <typename T>
hipError_t launch_film_gemv(const FilmLayers<T>& w, int n_layers, const float* x0, int G, int d, int H,
                            float* out, hipStream_t s);
// logits[v] = x[v] W_out^T + b_out (fp32), lse[v] (nullable); x is the fp32 residual stream.
template <typename T>
hipError_t launch_head(const float* x, const T* w_out, const T* b_out, int n, int d, int D,
                       float* logits, float* lse, hipStream_t s);

// ---- sampling ---------------------------------------------------------------
constexpr int kSampleChunk = 256;
// Chunks [chunk0, chunk1) of the total_chunks (chunk1 < 0: to the end); each
// chunk's placements and partial sums are the same whichever launch forms them.
hipError_t launch_sample(const float* logits, const float* lse, int n, int D, int K, uint64_t seed,
                         const float* uniforms, const GraphTable& chunks, int total_chunks,
                         int* placements, float* partial, hipStream_t s, int chunk0 = 0, int chunk1 = -1);
hipError_t launch_logp_reduce(const float* partial, const GraphTable& chunks, int total_chunks, int K,
                              float* logp, hipStream_t s);
hipError_t launch_debug_uniforms(uint64_t seed, int n, int K, int D, float* out, hipStream_t s);
// Per-chunk partial log-probs of given placements (then launch_logp_reduce).
hipError_t launch_logp_given(const float* logits, const float* lse, int n, int D, int K, const int* placements,
                             const GraphTable& chunks, int total_chunks, float* partial, hipStream_t s);

// ---- the update path's first step ---------------------------------------------
// PPO's clipped surrogate per graph (loss [G]) and the gradient of the batch
// loss with respect to the logits (dlogits [n, D]); coef: G * (K + 1) floats of
// scratch (the coefficients, then each graph's sum of them).
hipError_t launch_ppo(const float* logits, const float* lse, const int* placements, const float* logp,
                      const float* logp_old, const float* adv, float eps, const GraphTable& gt, int n, int D, int K,
                      float* coef, float* loss, float* dlogits, hipStream_t s);
// The head's backward pass: dx [n, d] = dlogits W_out, dw_out [D, d] = dlogits^T x,
// db_out [D] = column sums of dlogits; partial: ceil(n / kHeadBwdRows) * D * (d + 1)
// floats of scratch.  d divides 256, D <= 64.
// Section 4's reward and advantage per graph (one work-group each); the running
// state reward_sum / trial_count [G] is read and updated.
hipError_t launch_advantages(const float* run_time, const uint8_t* valid, int G, int K, double* reward_sum,
                             int64_t* trial_count, float* reward, float* adv, hipStream_t s);
template <typename T>
hipError_t launch_head_backward(const float* x, const T* w_out, const float* dlogits, int n, int d, int D, float* dx,
                                float* dw_out, float* db_out, float* partial, hipStream_t s);

// ---- the simulated run time of sampled placements ----------------------------
// In-order list scheduling of every graph under each of K placements, with the
// per-device memory check; in_ptr / in_idx is the reverse CSR (predecessors).
struct EvalLaunch {
  const int* placements;       // [K, n]
  const int* op_cost;          // [n]
  const int* out_xfer;         // [n]
  const int* op_mem;           // [n]
  const int64_t* mem_cap;      // host [G]
  const int* in_ptr;           // [n + 1]
  const int* in_idx;           // [n_edges]
  int64_t n_edges;
  const GraphTable* gt;        // graphs (ptr)
  const GraphTable* chunk_table;   // graphs and their 256-node chunks (blk)
  int chunks;
  int n, D, K;
  double time_unit;
  void* rec;                   // scratch: n_edges int2
  void* memsum;                // scratch: G * K * D uint64
  unsigned* far;               // scratch: ceil(K / 64) * n * 64 uint32
  int64_t* makespan;           // [G, K]
  unsigned char* valid;        // [G, K]
  float* run_time;             // [G, K] or null
};
constexpr int kEvalChunk = 256;
hipError_t launch_evaluate(const EvalLaunch& L, hipStream_t s);

}  // namespace gdp
