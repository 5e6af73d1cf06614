/*
 * gdp.h -- C ABI of libgdp: the forward pass of the GDP device-placement
 * policy (Zhou et al., "GDP: Generalized Device Placement for Dataflow
 * Graphs") and whole-graph sampling of placements, on one AMD Instinct
 * MI355X (gfx950).
 *
 * The problem statement (Section 3): given a dataflow graph G(V, E) whose
 * vertices are ops and whose edges are data dependencies, a policy assigns a
 * device to every op of the graph.  The policy is a graph embedding network
 * (Section 3.1, Eq. 2-3) followed by a segment-recurrent attention placement
 * network (Section 3.2) whose layers are conditioned on the pooled graph
 * representation (Section 3.3, Eq. 4); its output is an N x d matrix of
 * per-op device logits (Fig. 1).
 *
 * Three calls make up one forward pass:
 *   gdp_embed   graph + features + GNN weights  -> node and graph embeddings
 *   gdp_place   embeddings + placer weights      -> device logits (+ lse)
 *   gdp_sample  logits + K + seed                -> K placements + log-probs
 * and the first steps of the update path (Section 3, PPO) follow them:
 *   gdp_ppo_grad       samples + old log-probs + advantages -> loss, dL/dlogits
 *   gdp_place_train    gdp_place that also keeps the head's input X
 *   gdp_head_backward  X + dL/dlogits -> dL/dX, dL/dW_out, dL/db_out
 *
 * Conventions shared by every call
 *  - Memory.  Every pointer documented "device" is HIP device memory owned by
 *    the caller; "host" pointers are ordinary host memory read during the
 *    call only.  The library never allocates or frees device memory.  Scratch
 *    memory comes from the caller's workspace (gdp_workspace_bytes).
 *  - Layout.  Matrices are row-major.  Weight matrices are [out, in] (each
 *    output unit's weights contiguous), so y = x W^T + b.
 *  - Element type.  A call works either entirely in fp32 (GDP_F32) or with
 *    bf16 storage and fp32 arithmetic (GDP_BF16): features, weights, biases,
 *    LayerNorm parameters and node embeddings then use bf16; graph
 *    embeddings, logits, lse and log-probs are always fp32.
 *  - Streams.  `stream` is a hipStream_t (NULL = the default stream).  Calls
 *    only enqueue work and return without synchronising.  A workspace may be
 *    shared by several calls only if they are ordered on one stream.
 *    gdp_place, gdp_place_train and gdp_place_sample may run part of their
 *    work on a second stream of the library's (see gdp_set_place_streams); it starts after
 *    the work enqueued on `stream` before the call, and work enqueued on
 *    `stream` after the call waits for it, so the ordering seen on `stream`
 *    is that of a single-stream call, HIP graph capture included.
 *  - Errors.  Calls return GDP_OK (0) or a negative gdp_status.  On a
 *    validation error nothing is enqueued and no output is touched;
 *    gdp_last_error() then describes the failure (thread-local string).
 *    Errors of already-enqueued work surface as GDP_E_HIP from a later call
 *    or from the caller's own synchronisation.  No C++ exception crosses
 *    this interface.
 *  - Preconditions on device data.  The device calls do not inspect the CSR
 *    arrays on the host; callers check them once with
 *    gdp_validate_graph_host (out-of-range ids in device arrays are
 *    undefined behaviour).
 */
#ifndef GDP_H_
#define GDP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GDP_ABI_VERSION 2

/* Limits of this implementation (violations return GDP_E_UNSUPPORTED). */
#define GDP_MAX_GRAPHS 128   /* graphs per ragged batch                      */
#define GDP_MAX_FANOUT 32    /* sampled neighbours per node                  */
#define GDP_MAX_DEVICES 64   /* devices d of the placement                   */

typedef enum gdp_status {
  GDP_OK = 0,
  GDP_E_INVALID_ARG = -1,  /* null pointer, bad size or flag               */
  GDP_E_BAD_GRAPH = -2,    /* graph structure violates the contract        */
  GDP_E_UNSUPPORTED = -3,  /* valid but outside this build's limits        */
  GDP_E_WORKSPACE = -4,    /* workspace smaller than gdp_workspace_bytes   */
  GDP_E_HIP = -5           /* a HIP runtime call failed                     */
} gdp_status;

typedef enum gdp_dtype { GDP_F32 = 0, GDP_BF16 = 1 } gdp_dtype;

/* gdp_graph.flags */
#define GDP_TOPO_IDS 1u  /* every edge u -> v has u < v (checked by the host validator) */

/*
 * A ragged batch of G dataflow graphs (Section 3: G(V, E); Section 3.3: a
 * batch of heterogeneous graphs).  Graph g owns the node ids
 * [graph_ptr_h[g], graph_ptr_h[g+1]); edges never cross graphs.  The CSR
 * holds out-edges (data dependencies u -> v); the neighbourhood N(v) of
 * Eq. 2 is taken over in- and out-edges.  Node order is also the order of the
 * placer's sequence (Section 3.2).
 */
typedef struct gdp_graph {
  int32_t n_graphs;            /* G, 1 .. GDP_MAX_GRAPHS                      */
  const int32_t* graph_ptr_h;  /* host [G+1]; 0 = ptr[0] < ptr[1] < ... = N   */
  int32_t n_nodes;             /* N >= 1                                      */
  const int32_t* row_ptr;      /* device [N+1], row_ptr[0] = 0, row_ptr[N] = E */
  const int32_t* col_idx;      /* device [E], global ids, no self-loops or
                                  duplicates, same graph as the row          */
  int64_t n_edges;             /* E, 0 .. INT32_MAX                           */
  const void* x;               /* device [N, F] node meta-features (dtype)    */
  int32_t feat_dim;            /* F, a multiple of 32                          */
  int32_t dtype;               /* gdp_dtype of x, weights and node_emb        */
  uint32_t flags;              /* GDP_TOPO_IDS or 0                           */
} gdp_graph;

/*
 * One iteration of the graph embedding network (Section 3.1).
 *   Eq. 2:  h_N(v) = max_{u in S(v)} sigmoid(w_pool h_u + b_pool)   (0 if S(v) is empty)
 *   Eq. 3:  h_v'   = ReLU(w_self h_v + w_neigh h_N(v) + b_upd),
 * i.e. f(concat(h_v, h_N(v))) with f's weight [w_self | w_neigh].
 * All device pointers in the graph's dtype.
 */
typedef struct gdp_gnn_layer {
  const void* w_pool;   /* [H, H_in]  */
  const void* b_pool;   /* [H]        */
  const void* w_self;   /* [H, H_in]  */
  const void* w_neigh;  /* [H, H]     */
  const void* b_upd;    /* [H]        */
} gdp_gnn_layer;

/*
 * The graph embedding network.  H_in is feat_dim for layer 0 and hidden
 * afterwards.  S(v) is N(v) when |N(v)| <= fanout; otherwise the fanout
 * members u with the smallest (key(v, u), u), where key is word 0 of
 * Philox4x64-10(counter = (v - g0, u - g0, 1, 0), key = (nbr_seed, 0)) and g0
 * is the first node of v's graph.  One sample serves all layers.
 */
typedef struct gdp_gnn {
  int32_t n_layers;               /* >= 1                                   */
  int32_t in_dim;                 /* F (must equal gdp_graph.feat_dim)      */
  int32_t hidden;                 /* H: 64, 128 or 256                      */
  int32_t fanout;                 /* 1 .. GDP_MAX_FANOUT                    */
  uint64_t nbr_seed;
  const gdp_gnn_layer* layers;    /* host array [n_layers]                  */
} gdp_gnn;

/*
 * One placer layer (Section 3.2 and Eq. 4).  With Y = gamma (.) X + beta the
 * conditioned layer input (gamma = 1 + film_wg x0 + film_bg,
 * beta = film_wb x0 + film_bb for the layer's graph), the layer computes
 *   Z  = LN1(Y + MHA(Y; memory) W_o^T + b_o)
 *   X' = LN2(Z + W_2 ReLU(W_1 Z + b_1) + b_2)
 * where MHA has no positional terms and no mask: the queries of a segment
 * [q0, q1) of graph g attend to the keys [max(g_start, q0 - mem_len), q1).
 * w_qkv stacks the Q, K and V projections; heads are contiguous column groups.
 * w_qkv, b_qkv, w_o, w_1, b_1 and w_2 must be 16-byte aligned (checked before
 * any launch: GDP_E_INVALID_ARG); the other vectors have no alignment rule.
 */
typedef struct gdp_placer_layer {
  const void *film_wg, *film_bg;  /* [d, H], [d]  (ignored when film = 0)   */
  const void *film_wb, *film_bb;  /* [d, H], [d]                            */
  const void *w_qkv, *b_qkv;      /* [3d, d], [3d]                          */
  const void *w_o, *b_o;          /* [d, d], [d]                            */
  const void *ln1_g, *ln1_b;      /* [d], [d]                               */
  const void *w_1, *b_1;          /* [d_ff, d], [d_ff]                      */
  const void *w_2, *b_2;          /* [d, d_ff], [d]                         */
  const void *ln2_g, *ln2_b;      /* [d], [d]                               */
} gdp_placer_layer;

/*
 * attention = 0 selects the placement network of the paper's ablation
 * (Section 4.4) that has no attention: each layer is then
 *   Y = FiLM_l(X),  X <- LN(Y + W_2 ReLU(W_1 Y + b_1) + b_2)   (LayerNorm ln2)
 * and w_qkv, b_qkv, w_o, b_o, ln1_g, ln1_b (may be NULL), n_heads, seg_len and
 * mem_len are not used; at most 16 layers.
 */
typedef struct gdp_placer {
  int32_t n_layers;               /* >= 1                                   */
  int32_t d_model;                /* d = gdp_gnn.hidden                     */
  int32_t n_heads;                /* d / n_heads in {16, 32, 64}            */
  int32_t d_ff;                   /* a multiple of 128                      */
  int32_t seg_len;                /* segment length S >= 1                  */
  int32_t mem_len;                /* memory length M >= 0                   */
  int32_t n_devices;              /* D, 2 .. GDP_MAX_DEVICES                */
  int32_t film;                   /* 1: condition on x0 (Eq. 4), 0: off     */
  int32_t attention;              /* 1: Section 3.2's placer, 0: the ablation's placer without attention */
  const gdp_placer_layer* layers; /* host array [n_layers]                  */
  const void* w_out;              /* [D, d] device, dtype                    */
  const void* b_out;              /* [D]                                    */
} gdp_placer;

/* Bytes of workspace needed by gdp_embed, gdp_place and gdp_sample for this
 * problem (the maximum of the three), and with a placer and k_samples > 0 also
 * by gdp_place_sample (whose sample regions follow the placer's).  Returns 0
 * on invalid arguments. */
size_t gdp_workspace_bytes(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer,
                           int32_t k_samples);

/*
 * Graph embedding network (Section 3.1, Eq. 2-3), then the per-graph mean of
 * the final node embeddings as the graph representation x0 (Eq. 4's x^(0)).
 *   node_emb   device [N, H], dtype         (output)
 *   graph_emb  device [G, H], fp32          (output)
 */
int gdp_embed(const gdp_graph* g, const gdp_gnn* gnn, void* node_emb, float* graph_emb,
              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Placement network (Section 3.2) with feature conditioning (Section 3.3,
 * Eq. 4) and the output layer producing per-node device logits (Fig. 1).
 *   node_emb   device [N, d], dtype         (input, from gdp_embed)
 *   graph_emb  device [G, d], fp32          (input; unused when film = 0)
 *   logits     device [N, D], fp32          (output)
 *   lse        device [N],    fp32          (output, may be NULL): log-sum-exp of each row
 */
int gdp_place(const gdp_graph* g, const void* node_emb, const float* graph_emb,
              const gdp_placer* placer, float* logits, float* lse,
              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Stream schedule of gdp_place and gdp_place_train for the calling thread
 * (a scheduling choice only: the results are the same bit for bit).
 *   n = 2 (the default): with attention and at least 40,960 nodes, the rows
 *     are split at a segment start near row 32,768 into parts A and B;
 *     every kernel of a layer runs once per part, A's on a second stream
 *     (one per device and calling thread, default priority, created at the
 *     first such call and kept until the process ends) and B's on `stream`,
 *     so that the parts of consecutive layers overlap.  The workspace holds
 *     a second copy of the QKV buffer for it.  A call made while `stream`
 *     is being captured into a HIP graph, before that thread has made an
 *     uncaptured one on the device, keeps every launch on `stream` (no
 *     stream is created during a capture).
 *   n = 1: every launch on `stream`, one launch per kernel and layer.
 * Returns GDP_E_INVALID_ARG for any other n.
 */
int gdp_set_place_streams(int32_t n);

/*
 * Whole-graph sampling: K placements of every op at once (Section 3), by
 * Gumbel-max over the device logits, with the log-probability of each
 * sampled placement (the quantity a PPO update needs, Section 3).
 *   placements[k, v] = argmax_j (logits[v, j] - ln(-ln u[k, v, j])), ties to the lowest j
 *   logp[g, k]       = sum over v in graph g of (logits[v, p] - lse[v])
 * u[k, v, j] = (2 * (h >> 9) + 1) * 2^-24 where h is the 32-bit half (j & 1,
 * 0 = low) of word (j & 7) >> 1 of Philox4x64-10(counter = (v, k, 2, j >> 3),
 * key = (seed, 0)), v the global node id.
 *   logits      device [N, D] fp32 (input)
 *   lse         device [N] fp32 (input, may be NULL: then recomputed)
 *   uniforms    device [K, N, D] fp32 or NULL: replaces the generator (testing)
 *   placements  device [K, N] int32 (output)
 *   logp        device [G, K] fp32 (output)
 */
int gdp_sample(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
               int32_t k_samples, uint64_t seed, const float* uniforms, int32_t* placements,
               float* logp, void* workspace, size_t workspace_bytes, void* stream);

/*
 * gdp_place followed by gdp_sample with n_devices = placer->n_devices, as one
 * call (Section 3: the policy's logits, then whole-graph sampling from them):
 * logits, lse, placements and logp are those of the two calls bit for bit.
 * In the two-part schedule with the head inside the last layer's kernel
 * (n_devices <= 8), the sampling of the 256-node chunks that lie wholly below
 * the split row starts on the second stream as soon as their logits are
 * final, beside the other part's last layer; a chunk with nodes on both sides
 * is sampled after the two streams join.  The workspace of gdp_workspace_bytes with this placer
 * and k_samples suffices (the placer's regions, then the sample's); the same
 * errors as either call, checked before anything is enqueued.
 */
int gdp_place_sample(const gdp_graph* g, const void* node_emb, const float* graph_emb,
                     const gdp_placer* placer, float* logits, float* lse, int32_t k_samples,
                     uint64_t seed, const float* uniforms, int32_t* placements, float* logp,
                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * gdp_place that also writes the placement network's output X (the head's
 * input, the last layer's LN2 output), which the backward pass needs.
 *   x_out  device [N, d] fp32 (output, 16-byte aligned)
 */
int gdp_place_train(const gdp_graph* g, const void* node_emb, const float* graph_emb,
                    const gdp_placer* placer, float* logits, float* lse, float* x_out,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * The head's backward pass (Fig. 1's output layer, logits = X W_out^T + b_out),
 * the second step of the update path: for a given dL/dlogits,
 *   dx      = dlogits W_out        device [N, d] fp32 (output, 16-byte aligned)
 *   dw_out  = dlogits^T X          device [D, d] fp32 (output)
 *   db_out  = sum_v dlogits[v]     device [D] fp32 (output)
 *   x       device [N, d] fp32 (input, from gdp_place_train, 16-byte aligned)
 *   dlogits device [N, D] fp32 (input, e.g. from gdp_ppo_grad)
 * W_out is read from placer (its dtype is the graph's).  The workspace of
 * gdp_workspace_bytes for this placer suffices.  Deterministic.
 */
int gdp_head_backward(const gdp_graph* g, const gdp_placer* placer, const float* x, const float* dlogits,
                      float* dx, float* dw_out, float* db_out, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * Reward and advantage (Section 4) of the K placements of each of G graphs
 * from their measured run times, the input of gdp_ppo_grad's advantages:
 *   reward[g, k]    = -sqrt(run_time[g, k]), or -10 where valid[g, k] == 0
 *                     (an invalid placement: out of memory, a broken constraint)
 *   advantage[g, k] = reward[g, k] - b[g],  b[g] = the average reward of all
 *                     previous trials of graph g (reward_sum[g] / trial_count[g]),
 *                     or this batch's mean for g when trial_count[g] == 0
 * and then reward_sum[g] += sum_k reward[g, k], trial_count[g] += K.  The K
 * trials of one call are not previous to each other.
 *   run_time     device [G, K] fp32 (input, >= 0 where valid)
 *   valid        device [G, K] uint8 (input, may be NULL: all valid)
 *   reward_sum   device [G] fp64 (in/out: the running state, zero to start)
 *   trial_count  device [G] int64 (in/out)
 *   reward       device [G, K] fp32 (output, may be NULL)
 *   advantage    device [G, K] fp32 (output)
 * 1 <= n_graphs <= GDP_MAX_GRAPHS, k_samples >= 1.  No workspace.  Calls on one
 * state must be ordered (same stream); deterministic.
 */
int gdp_advantages(int32_t n_graphs, int32_t k_samples, const float* run_time, const uint8_t* valid,
                   double* reward_sum, int64_t* trial_count, float* reward, float* advantage, void* stream);

/*
 * gdp_sample without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, kernels and results as gdp_sample (bit
 * for bit); the per-(sample, 256-node chunk) partial log-prob sums live in a
 * library-owned device array of GDP_NOALLOC_SCRATCH_BYTES per GPU, held until
 * the process ends.  K * (sum over graphs of ceil(nodes / 256)) * 4 bytes must
 * fit in it, else GDP_E_UNSUPPORTED and nothing is enqueued.  The call
 * allocates nothing.  Calls on one GPU share its array: calls that overlap in
 * time on that GPU (different streams, or different threads without ordering)
 * race and give undefined log-probs; calls ordered on one stream are safe.
 */
#define GDP_NOALLOC_SCRATCH_BYTES (4u << 20)
int gdp_sample_noalloc(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                       int32_t k_samples, uint64_t seed, const float* uniforms, int32_t* placements,
                       float* logp, void* stream);

/*
 * The first step of the policy update (Section 3: Eq. 1's objective, optimised
 * with PPO, Schulman et al. 2017): the clipped surrogate over the K sampled
 * placements of every graph and its gradient with respect to the logits.
 *   r[g, k]  = exp(logp[g, k] - logp_old[g, k])
 *   loss[g]  = -(1/K) sum_k min(r A[g, k], clip(r, 1 - clip_eps, 1 + clip_eps) A[g, k])
 *   dlogits  = d/d logits of (1/G) sum_g loss[g], through
 *              logp[g, k] = sum over v in g of (logits[v, p_kv] - lse[v])
 * The min takes the unclipped branch's slope where that branch attains it and
 * 0 where the clipped constant does.
 *   logits      device [N, D] fp32 (input, the ones the placements were drawn from)
 *   lse         device [N] fp32 (input, may be NULL: then recomputed)
 *   placements  device [K, N] int32 (input, from gdp_sample)
 *   logp        device [G, K] fp32 (input, from gdp_sample)
 *   logp_old    device [G, K] fp32 (input: the sampling policy's log-probs)
 *   advantages  device [G, K] fp32 (input)
 *   clip_eps    0 < clip_eps < 1
 *   loss        device [G] fp32 (output)
 *   dlogits     device [N, D] fp32 (output)
 * The workspace of gdp_workspace_bytes with the same k_samples suffices.
 * Deterministic (fixed summation orders).
 */
/*
 * Simulated run time and validity of every sampled placement (Section 4.1:
 * a placement is scored by the training step time it yields, and a placement
 * that runs out of memory is invalid; Section 2: placement with and without
 * simulation).  The paper measures on hardware; this call is an in-order list
 * scheduler: every device runs its ops one at a time in node-id order, and op v
 * on device p starts once p has finished its previous op and every input has
 * arrived, where the output of a predecessor u reaches another device
 * out_xfer[u] after u finishes (transfers overlap with compute and with each
 * other):
 *   finish(v)        = max(free[p], max_u finish(u) + [p_u != p] out_xfer[u]) + op_cost[v]
 *   makespan[g, k]   = the largest finish time of graph g under placement k
 *   valid[g, k]      = 1 if every device holds at most mem_cap_h[g] of op_mem
 *   run_time[g, k]   = (float)(makespan[g, k] * time_unit), the input of gdp_advantages
 * Integer arithmetic throughout, so results are exact and deterministic.
 *   placements  device [K, N] int32 in [0, n_devices) (input, from gdp_sample)
 *   op_cost     device [N] int32 >= 0 (compute time of each op)
 *   out_xfer    device [N] int32 >= 0 (time to move the op's output to another device)
 *   op_mem      device [N] int32 >= 0 (memory the op holds on its device)
 *   mem_cap_h   host [G] int64 >= 0 (per-device capacity of each graph)
 *   time_unit   >= 0, seconds per time unit (scales run_time only)
 *   makespan    device [G, K] int64 (output, 8-byte aligned); -1 where a
 *               finish time of the graph reaches 2^26 time units (a finish
 *               time shares a 32-bit word with its device); a sum of op_cost
 *               and out_xfer over the graph below 2^26 rules this out
 *   valid       device [G, K] uint8 (output)
 *   run_time    device [G, K] fp32 (output, may be NULL)
 * The CSR must be valid (gdp_validate_graph_host); its device arrays are not
 * read on the host.  Workspace: gdp_evaluate_workspace_bytes(g, n_devices, K).
 */
size_t gdp_evaluate_workspace_bytes(const gdp_graph* g, int32_t n_devices, int32_t k_samples);
int gdp_evaluate(const gdp_graph* g, int32_t n_devices, int32_t k_samples, const int32_t* placements,
                 const int32_t* op_cost, const int32_t* out_xfer, const int32_t* op_mem, const int64_t* mem_cap_h,
                 double time_unit, int64_t* makespan, uint8_t* valid, float* run_time, void* workspace,
                 size_t workspace_bytes, void* stream);

int gdp_ppo_grad(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                 int32_t k_samples, const int32_t* placements, const float* logp, const float* logp_old,
                 const float* advantages, float clip_eps, float* loss, float* dlogits, void* workspace,
                 size_t workspace_bytes, void* stream);

/* ---- the update step (Section 3: Eq. 1 with PPO) --------------------------
 *
 * The policy is trained end to end: the graph embedding network jointly with
 * the placement network (Section 3.1), the cached segment memory passing no
 * gradient (Section 3.2: hidden states of earlier segments are cached with
 * gradient flow disabled, as in Transformer-XL: a query still reaches the
 * memory's keys and values, so W_qkv receives their gradient, but the earlier
 * segments' activations do not).  One update:
 *   gdp_forward_train  the policy forward in fp32 arithmetic, keeping every
 *                      intermediate in a caller-owned store, and the logits
 *   gdp_log_prob       log pi(placement | graph) of given placements
 *   gdp_ppo_grad       dL/dlogits of PPO's clipped surrogate
 *   gdp_backward       dL/dtheta for every weight, from dL/dlogits and the store
 *   gdp_adam_step      Adam on every weight (fp32 master copies and moments)
 */

/* Gradients of one layer: fp32 device arrays shaped like the weights. */
typedef struct gdp_gnn_layer_grad {
  float *w_pool, *b_pool, *w_self, *w_neigh, *b_upd;
} gdp_gnn_layer_grad;
typedef struct gdp_placer_layer_grad {
  float *film_wg, *film_bg, *film_wb, *film_bb;  /* used when film = 1 (else may be NULL) */
  float *w_qkv, *b_qkv, *w_o, *b_o, *ln1_g, *ln1_b;  /* used when attention = 1 (else may be NULL) */
  float *w_1, *b_1, *w_2, *b_2, *ln2_g, *ln2_b;
} gdp_placer_layer_grad;
typedef struct gdp_grads {
  const gdp_gnn_layer_grad* gnn;       /* host array [gnn.n_layers]    */
  const gdp_placer_layer_grad* placer; /* host array [placer.n_layers] */
  float* w_out;                        /* [D, d]                       */
  float* b_out;                        /* [D]                          */
} gdp_grads;

/*
 * Sizes of the training forward's store and of the workspace of
 * gdp_forward_train / gdp_backward (bytes).  At most 8 GNN layers and 16
 * placer layers; d_model must equal the GNN's hidden width.  Returns
 * GDP_OK or an error (then the sizes are 0).
 */
int gdp_train_sizes(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, size_t* store_bytes,
                    size_t* workspace_bytes);

/*
 * The policy forward (Eq. 2-3, the mean pool, Eq. 4's FiLM, the placer of
 * Section 3.2 and the head) in fp32 arithmetic -- bf16 weights and features
 * are widened on load -- keeping every intermediate the backward pass needs
 * in store (256-byte aligned, gdp_train_sizes bytes; opaque layout, valid
 * for the weights and graph of this call).
 *   logits  device [N, D] fp32 (output)     lse  device [N] fp32 (output, may be NULL)
 */
int gdp_forward_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, void* store,
                      size_t store_bytes, float* logits, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * Gradient of L with respect to every weight, given dlogits = dL/dlogits
 * [N, D] fp32 (e.g. from gdp_ppo_grad) and the store of gdp_forward_train with
 * the same weights.  Writes (does not accumulate) every gradient array of
 * grads that the configuration uses.  Deterministic (fixed summation orders).
 */
int gdp_backward(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, const void* store,
                 size_t store_bytes, const float* dlogits, const gdp_grads* grads, void* workspace,
                 size_t workspace_bytes, void* stream);

/*
 * logp[g, k] = sum over v in graph g of (logits[v, placements[k, v]] - lse[v])
 * for given placements (the numerator of PPO's ratio after an update).
 *   logits device [N, D]; lse device [N] (may be NULL: recomputed);
 *   placements device [K, N] int32 in [0, D); logp device [G, K] (output).
 * The workspace of gdp_workspace_bytes with the same K suffices.
 */
int gdp_log_prob(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices, int32_t k_samples,
                 const int32_t* placements, float* logp, void* workspace, size_t workspace_bytes, void* stream);

/* One tensor of gdp_adam_step: the weights the kernels read (dtype), their
 * fp32 master copy, the gradient and Adam's two moments, n elements each. */
typedef struct gdp_adam_tensor {
  void* param;
  float* master;
  const float* grad;
  float* m;
  float* v;
  int64_t n;
} gdp_adam_tensor;

/*
 * Adam (Kingma and Ba, 2015), step t >= 1: m = b1 m + (1 - b1) g,
 * v = b2 v + (1 - b2) g^2, master -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps),
 * param = master rounded to dtype (GDP_F32 or GDP_BF16, round to nearest even).
 * tensors is a host array.  No workspace.
 */
int gdp_adam_step(int32_t n_tensors, const gdp_adam_tensor* tensors, int32_t dtype, float lr, float beta1,
                  float beta2, float eps, int64_t step, void* stream);

/*
 * Host-side check of a graph batch (all pointers host memory): graph_ptr
 * strictly increasing from 0, row_ptr monotone from 0 to E, col_idx in range,
 * no self-loops, no duplicate edges, no edge across graphs, acyclic (Kahn's
 * algorithm), and u < v on every edge when flags has GDP_TOPO_IDS.
 * Returns GDP_OK, GDP_E_INVALID_ARG or GDP_E_BAD_GRAPH (with gdp_last_error).
 */
int gdp_validate_graph_host(const int32_t* graph_ptr, int32_t n_graphs, const int32_t* row_ptr,
                            int32_t n_nodes, const int32_t* col_idx, int64_t n_edges,
                            uint32_t flags);

/* Description of the last failure on the calling thread ("" if none). */
const char* gdp_last_error(void);

/* GDP_ABI_VERSION of the loaded library. */
int gdp_abi_version(void);

/* ---- diagnostics (tests and benchmarks) --------------------------------- */

/*
 * The uniforms u[k, v, j] that gdp_sample draws for (seed, N, K, D), written
 * to out (device [K, N, D] fp32), for bit-exact checks of the generator.
 */
int gdp_debug_uniforms(uint64_t seed, int32_t n_nodes, int32_t k_samples, int32_t n_devices,
                       float* out, void* stream);

/*
 * The sampled neighbourhoods S(v) that gdp_embed uses: s_ptr device [N+1]
 * and s_idx device [capacity] (capacity >= min(2E, N * fanout)).  The order
 * of ids inside one row is unspecified.
 */
int gdp_debug_neighbors(const gdp_graph* g, const gdp_gnn* gnn, int32_t* s_ptr, int32_t* s_idx,
                        int64_t capacity, void* workspace, size_t workspace_bytes, void* stream);

/*
 * One intermediate of gdp_forward_train's store, copied to out (device): the
 * forward's discrete decisions, for comparisons that must take them the same
 * way.  which = 0: the feed-forward hidden layer of placer layer `layer`
 * ([N, d_ff] fp32, after ReLU); 1: the output of GNN layer `layer` ([N, H]
 * fp32, after ReLU); 2: the winning neighbour of every element of GNN layer
 * `layer`'s max-pool ([N, H] int32, -1 where S(v) is empty).
 */
int gdp_debug_train_tensor(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, const void* store,
                           size_t store_bytes, int32_t which, int32_t layer, void* out, size_t out_bytes, void* stream);

/* Kernel kinds for the event timer below. */
typedef enum gdp_kernel_kind {
  GDP_K_GRAPH_PREP = 0,  /* degree count, scans, reverse-edge fill          */
  GDP_K_NBR_SAMPLE,      /* neighbour sampling S(v)                          */
  GDP_K_GEMM_POOL,       /* sigmoid(h W_pool^T + b)                           */
  GDP_K_GATHER_MAX,      /* Eq. 2 max over S(v)                               */
  GDP_K_GEMM_UPDATE,     /* Eq. 3 ReLU(h W_self^T + A W_neigh^T + b)          */
  GDP_K_MEANPOOL,        /* x0 = per-graph mean                              */
  GDP_K_FILM,            /* gamma/beta GEMVs of all placer layers             */
  GDP_K_PRE_LAYER,       /* the first layer's Y = FiLM(X) and Y W_qkv^T + b   */
  GDP_K_ATTENTION,       /* segment attention                                */
  GDP_K_POST_ATTN,       /* fused rest of a layer: LN1(Y + O W_o^T + b),
                            LN2(Z + FFN(Z)), the next layer's FiLM and QKV,
                            and in the last layer the head (D <= 8)          */
  GDP_K_HEAD,            /* logits and lse when not fused (D > 8)            */
  GDP_K_SAMPLE,          /* Gumbel-max sampling                              */
  GDP_K_LOGP_REDUCE,     /* per-graph log-prob sums                          */
  GDP_K_MLP_PLACER,      /* the ablation's placer without attention, all layers */
  GDP_K_PPO,             /* PPO clipped surrogate and its logit gradient     */
  GDP_K_HEAD_BWD,        /* the head's backward pass                        */
  GDP_K_ADVANTAGE,       /* reward and advantage of measured run times      */
  GDP_K_EVALUATE,        /* simulated run time and validity of placements   */
  GDP_K_TRAIN_FWD,       /* the training forward (all intermediates kept)   */
  GDP_K_BACKWARD,        /* the backward pass                               */
  GDP_K_ADAM,            /* the Adam update                                 */
  GDP_K_LOGPROB,         /* log-probabilities of given placements           */
  GDP_K_GEMM_UPDATE_POOL, /* Eq. 3's update fused with the next layer's
                             Eq. 2 transform of the same rows               */
  GDP_K_COUNT
} gdp_kernel_kind;

/*
 * Event timer.  gdp_timer_begin(mask) makes every later launch of a kernel
 * kind whose bit (1u << kind) is set in mask record a HIP event pair on the
 * stream it is launched on.  gdp_timer_end synchronises those events and
 * writes, per kind, the summed elapsed milliseconds and the launch count
 * (arrays of GDP_K_COUNT entries; either may be NULL), then stops timing.
 * The timer's state is per calling thread: only launches made by the thread
 * that called gdp_timer_begin are timed, and that thread calls gdp_timer_end.
 */
int gdp_timer_begin(uint32_t kind_mask);
int gdp_timer_end(double* total_ms, int64_t* launches);
const char* gdp_kernel_kind_name(int32_t kind);

#ifdef __cplusplus
}
#endif
#endif /* GDP_H_ */
