// Host-only argument checks and workspace planning (no HIP dependency, so the
// same file also builds with a plain C++ compiler for sanitizer runs).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "gdp.h"

namespace gdp {

// Thread-local error reporting; returns `code` for convenient `return fail(...)`.
int fail(int code, const char* fmt, ...);
void clear_error();

// Field checks of the structs (no device memory is read).
int check_graph(const gdp_graph* g);
int check_gnn(const gdp_graph* g, const gdp_gnn* gnn);
int check_placer(const gdp_graph* g, const gdp_placer* p);
int check_sample(const gdp_graph* g, int32_t n_devices, int32_t k_samples);

size_t elem_size(int32_t dtype);

// Sub-allocations of one call, each 256-byte aligned.
struct Carve {
  size_t off[24];
  size_t total;
  int n;
};
void carve_init(Carve* c);
size_t carve_add(Carve* c, size_t bytes);   // returns the offset of the new region

// Per-graph block counts -> prefix (blk[0] = 0 .. blk[G] = total).
int prefix_blocks_rows(const int32_t* graph_ptr, int G, int rows_per_block, int32_t* blk);
int prefix_blocks_attention(const int32_t* graph_ptr, int G, int seg_len, int block_q, int32_t* blk);
// Of the blocks prefix_blocks_rows counts, the number (a prefix of them) whose
// rows all lie below row R; *started (if not null) receives the number whose
// first row lies below R, which exceeds the first by one when a block holds
// rows on both sides of R.
int blocks_below(const int32_t* graph_ptr, int G, int rows_per_block, int R, int* started = nullptr);
// The segment start (of any graph of the batch) nearest `target` rows and
// strictly inside (0, N), or 0 when there is none; *qblocks_below receives
// the number of attention query blocks (prefix_blocks_attention's order)
// whose queries lie below it.
int segment_split(const int32_t* graph_ptr, int G, int seg_len, int block_q, int target, int* qblocks_below);

struct EmbedPlan {
  Carve c;
  size_t counters;   // [in_deg: N | cursor: N | heavy_count: 1], zeroed by one fill
  size_t scan_tmp, heavy;
  size_t in_ptr, in_idx, s_ptr, s_idx, P, A, h0, h1, pool;
  int64_t s_cap;
  int pool_chunks;
};
struct PlacePlan {
  Carve c;
  size_t film, y0, y1, qkv, o;
  size_t qkv2;           // the second QKV buffer of the two-part layer schedule (split > 0)
  size_t head_partial;   // gdp_head_backward: per row chunk, D x d weight and D bias partial sums
  int qblocks;
  int split;             // rows 0 .. split - 1 form part A of the two-part layer schedule; 0: one part
  int split_qblocks;     // attention query blocks of part A
};
constexpr int kHeadBwdRows = 128;   // rows per head-backward chunk
struct SamplePlan {
  Carve c;
  size_t partial;
  size_t coef;        // gdp_ppo_grad: G * K coefficients, then their G per-graph sums
  int chunks;
};
struct EvalPlan {
  Carve c;
  size_t counters;    // [in_deg: N | cursor: N | spare: 1]
  size_t scan_tmp, in_ptr, s_ptr, in_idx, rec, memsum, far;
  int chunks;
};
void plan_evaluate(const gdp_graph* g, int32_t n_devices, int32_t k_samples, EvalPlan* p);

// The update step: what the training forward keeps (store) and the backward's
// temporaries (workspace).  Offsets into the two buffers, 256-byte aligned.
constexpr int kMaxTrainGnnLayers = 8;
constexpr int kMaxTrainPlacerLayers = 16;
struct TrainPlan {
  size_t store_total, ws_total;
  // store
  size_t s_ptr, s_idx, in_ptr, in_idx, x0, film;
  size_t P[kMaxTrainGnnLayers], A[kMaxTrainGnnLayers], arg[kMaxTrainGnnLayers], h[kMaxTrainGnnLayers + 1];
  size_t X[kMaxTrainPlacerLayers + 1], Y[kMaxTrainPlacerLayers], QKV[kMaxTrainPlacerLayers], O[kMaxTrainPlacerLayers],
      lse_att[kMaxTrainPlacerLayers], R1[kMaxTrainPlacerLayers], Z[kMaxTrainPlacerLayers], H1[kMaxTrainPlacerLayers],
      R2[kMaxTrainPlacerLayers];
  // workspace
  size_t counters, scan_tmp, heavy, dX, dY, dR, dZ, xg, dH, dqkv, dkvm, Dq, head_partial, dfilm, dx0, dh, dA, dP, dU,
      colpart, gemm_partial;
  size_t gemm_partial_floats;
  int chunks;      // 256-row chunks over the graphs (column sums)
  int64_t s_cap;
};
int check_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* p);
void plan_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* p, TrainPlan* t);
void plan_embed(const gdp_graph* g, const gdp_gnn* gnn, EmbedPlan* p);
void plan_place(const gdp_graph* g, const gdp_placer* pl, PlacePlan* p);
void plan_sample(const gdp_graph* g, int32_t k_samples, SamplePlan* p);

constexpr int kPoolRows = 64;       // rows per mean-pool chunk
constexpr int kAttnQ = 128;         // queries per attention work-group
// Rows of part A of the two-part layer schedule: 256 blocks of 128 rows, one
// post-attention work-group per compute unit.
constexpr int kSplitRows = 256 * 128;
constexpr int kSampleRows = 256;    // nodes per sampling work-group
constexpr int kEvalRows = 256;      // nodes per device-memory work-group of the evaluator

}  // namespace gdp
