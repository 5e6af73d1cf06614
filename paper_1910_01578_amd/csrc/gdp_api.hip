// C ABI entry points: argument checks, workspace carving and the launch
// sequence of each call (everything is enqueued on the caller's stream).
#include <hip/hip_runtime.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "device_common.h"
#include "gdp.h"
#include "host_plan.h"
#include "kernels.h"
#include "train_kernels.h"

namespace gdp {

static_assert(kPoolRows == kMeanpoolRows, "mean-pool chunk size");
static_assert(kAttnQ == kAttnBlockQ, "attention query block");
static_assert(kSampleRows == kSampleChunk, "sampling chunk");
static_assert(kEvalRows == kEvalChunk, "evaluator memory chunk");

// ---------------------------------------------------------------------------
// Event timer (diagnostics): an event pair around every launch of a selected
// kernel kind, on the stream of that launch.
// ---------------------------------------------------------------------------
namespace {
struct TimerRec {
  int kind;
  hipEvent_t a, b;
  bool recorded;    // false when the closing record failed: the launch is not counted
};
struct TimerState {
  uint32_t mask = 0;
  std::vector<TimerRec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t take() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    // Timing only: without the system-scope fence a record costs no cache
    // write-back (which would idle the GPU between the launches it brackets).
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
  }
};
// Per thread: launches of other threads are neither timed nor disturbed.
thread_local TimerState g_timer;

// A launch whose opening or closing record fails is left out of the totals
// (the failure itself surfaces through the launch or the next call).
struct Timed {
  hipStream_t s;
  hipEvent_t b = nullptr;
  size_t idx = 0;
  bool on;
  Timed(int kind, hipStream_t st) : s(st), on(((g_timer.mask >> kind) & 1u) != 0) {
    if (!on) return;
    hipEvent_t a = g_timer.take();
    b = g_timer.take();
    if (!a || !b || hipEventRecord(a, s) != hipSuccess) {
      if (a) g_timer.pool.push_back(a);
      if (b) g_timer.pool.push_back(b);
      on = false;
      return;
    }
    idx = g_timer.recs.size();
    g_timer.recs.push_back({kind, a, b, true});
  }
  ~Timed() {
    if (on && hipEventRecord(b, s) != hipSuccess) g_timer.recs[idx].recorded = false;
  }
};
}  // namespace

static int hip_fail(hipError_t e, const char* what) {
  return fail(GDP_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// A launch on stream `stream` (timed there when its kind is selected).
#define GDP_LAUNCH_ON(kind, stream, ...)                         \
  do {                                                           \
    hipError_t _e;                                               \
    {                                                            \
      Timed _t((kind), (stream));                                \
      _e = (__VA_ARGS__);                                        \
    }                                                            \
    if (_e != hipSuccess) return hip_fail(_e, #__VA_ARGS__);     \
  } while (0)
// A launch on the call's stream st.
#define GDP_LAUNCH(kind, ...) GDP_LAUNCH_ON(kind, st, __VA_ARGS__)

#define GDP_HIP(...)                                             \
  do {                                                           \
    const hipError_t _e = (__VA_ARGS__);                         \
    if (_e != hipSuccess) return hip_fail(_e, #__VA_ARGS__);     \
  } while (0)

namespace {
// A second stream of the calling thread on one device, for the two-part
// layer schedule of gdp_place, with the events that order it against the
// call's stream: fork and join, and two alternating pairs for the
// cross-part dependencies.  Created at a thread's first such call on the
// device (default priority, non-blocking) and held until the process ends.
struct SideStream {
  int device = -1;
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  hipEvent_t a[2] = {nullptr, nullptr}, b[2] = {nullptr, nullptr};
};
thread_local std::vector<SideStream> g_side;
// gdp_set_place_streams: 2 = two-part schedule where it applies, 1 = one stream
thread_local int g_place_streams = 2;

// *out = nullptr (and GDP_OK) when the stream does not exist yet and st is
// being captured into a graph: no stream is created during a capture, and
// the caller then keeps every launch on st.
int side_stream(hipStream_t st, SideStream** out) {
  *out = nullptr;
  int dev = -1;
  hipError_t e = hipStreamGetDevice(st, &dev);
  if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
  for (SideStream& x : g_side)
    if (x.device == dev) {
      *out = &x;
      return GDP_OK;
    }
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if ((e = hipStreamIsCapturing(st, &cap)) != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  if (cap != hipStreamCaptureStatusNone) return GDP_OK;
  int cur = -1;
  if ((e = hipGetDevice(&cur)) != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "hipSetDevice");
  SideStream x;
  x.device = dev;
  e = hipStreamCreateWithFlags(&x.s, hipStreamNonBlocking);
  hipEvent_t* evs[6] = {&x.fork, &x.join, &x.a[0], &x.a[1], &x.b[0], &x.b[1]};
  // Ordering between streams of one device needs no system-scope fence.
  for (int i = 0; i < 6 && e == hipSuccess; ++i)
    e = hipEventCreateWithFlags(evs[i], hipEventDisableTiming | hipEventDisableSystemFence);
  if (cur != dev) {
    const hipError_t e2 = hipSetDevice(cur);
    if (e == hipSuccess) e = e2;
  }
  if (e != hipSuccess) {   // release what was created
    for (int i = 0; i < 6; ++i)
      if (*evs[i]) (void)hipEventDestroy(*evs[i]);
    if (x.s) (void)hipStreamDestroy(x.s);
    return hip_fail(e, "side stream");
  }
  g_side.push_back(x);
  *out = &g_side.back();
  return GDP_OK;
}
}  // namespace

static GraphTable make_table(const gdp_graph* g) {
  GraphTable t;
  memset(&t, 0, sizeof(t));
  t.n = g->n_graphs;
  for (int i = 0; i <= g->n_graphs; ++i) t.ptr[i] = g->graph_ptr_h[i];
  return t;
}

template <typename T>
static inline T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

static int pending_hip_error() {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "earlier HIP work");
  return GDP_OK;
}

static int check_ws(void* ws, size_t have, size_t need) {
  if (need > have) return fail(GDP_E_WORKSPACE, "workspace %zu bytes < %zu required", have, need);
  if (need > 0 && !ws) return fail(GDP_E_INVALID_ARG, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(GDP_E_INVALID_ARG, "workspace must be 256-byte aligned");
  return GDP_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ---------------------------------------------------------------------------
// Neighbourhoods N(v) (in- and out-edges) and the sample S(v) (Section 3.1).
// ---------------------------------------------------------------------------
static int prep_neighbors(const gdp_graph* g, const gdp_gnn* gnn, const EmbedPlan& pl, void* ws, int* s_ptr,
                          int* s_idx, hipStream_t st) {
  const int N = g->n_nodes;
  const GraphTable gt = make_table(g);
  int* counters = at<int>(ws, pl.counters);
  int* in_deg = counters;
  int* cursor = counters + N;
  int* heavy_count = counters + 2 * N;
  int* in_ptr = at<int>(ws, pl.in_ptr);
  int* in_idx = at<int>(ws, pl.in_idx);
  GDP_LAUNCH(GDP_K_GRAPH_PREP, launch_fill_i32(counters, 2 * (int64_t)N + 1, 0, st));
  GDP_LAUNCH(GDP_K_GRAPH_PREP, launch_in_degree(g->col_idx, g->n_edges, in_deg, st));
  GDP_LAUNCH(GDP_K_GRAPH_PREP, launch_scan_degrees(g->row_ptr, in_deg, N, gnn->fanout, in_ptr, s_ptr,
                                                   at<int>(ws, pl.scan_tmp), st));
  GDP_LAUNCH(GDP_K_GRAPH_PREP, launch_fill_reverse(g->row_ptr, g->col_idx, in_ptr, N, g->n_edges, cursor, in_idx,
                                                   st));
  GDP_LAUNCH(GDP_K_NBR_SAMPLE, launch_nbr_sample(g->row_ptr, g->col_idx, in_ptr, in_idx, s_ptr, N, gnn->fanout,
                                                 gnn->nbr_seed, gt, s_idx, at<int>(ws, pl.heavy), heavy_count, st));
  return GDP_OK;
}

// ---------------------------------------------------------------------------
// gdp_embed: Eq. 2 and Eq. 3 for every layer, then the mean pool.
// ---------------------------------------------------------------------------
template <typename T>
static int embed_impl(const gdp_graph* g, const gdp_gnn* gnn, T* node_emb, float* graph_emb, const EmbedPlan& pl,
                      void* ws, hipStream_t st) {
  const int N = g->n_nodes, H = gnn->hidden;
  int* s_ptr = at<int>(ws, pl.s_ptr);
  int* s_idx = at<int>(ws, pl.s_idx);
  int r = prep_neighbors(g, gnn, pl, ws, s_ptr, s_idx, st);
  if (r != GDP_OK) return r;
  // Every GNN activation is a GEMM operand (rounded to T for the matrix
  // cores either way), so the hidden layers are stored in T.
  T* P = at<T>(ws, pl.P);
  T* A = at<T>(ws, pl.A);
  T* hb[2] = {at<T>(ws, pl.h0), at<T>(ws, pl.h1)};
  const T* h = static_cast<const T*>(g->x);
  const int L = gnn->n_layers;
  bool p_ready = false;                       // P of layer l already formed by layer l - 1's update
  for (int l = 0; l < L; ++l) {
    const gdp_gnn_layer& Lw = gnn->layers[l];
    const int hin = l == 0 ? g->feat_dim : H;
    T* hout = (l == L - 1) ? node_emb : hb[l & 1];
    if (!p_ready) {
      const GemmArgs<T, T, T> pool = {h, hin, static_cast<const T*>(Lw.w_pool), hin, nullptr, 0, nullptr, 0,
                                      static_cast<const T*>(Lw.b_pool), P, H, N, H};
      if (row_gemm_supported(pool)) GDP_LAUNCH(GDP_K_GEMM_POOL, (launch_row_gemm<T>(pool, EPI_SIGMOID, st)));
      else GDP_LAUNCH(GDP_K_GEMM_POOL, (launch_gemm<T, T, T>(pool, EPI_SIGMOID, st)));
    }
    GDP_LAUNCH(GDP_K_GATHER_MAX, launch_gather_max<T>(P, s_ptr, s_idx, N, H, A, st));
    const GemmArgs<T, T, T> upd = {h, hin, static_cast<const T*>(Lw.w_self), hin, A, H,
                                   static_cast<const T*>(Lw.w_neigh), H, static_cast<const T*>(Lw.b_upd), hout, H,
                                   N, H};
    // the next layer's transform of these rows in the same kernel (P is free:
    // this layer's gather has read it)
    p_ready = false;
    if (l + 1 < L) {
      const gdp_gnn_layer& Ln = gnn->layers[l + 1];
      const RowPoolArgs<T> nxt = {static_cast<const T*>(Ln.w_pool), static_cast<const T*>(Ln.b_pool), P, H};
      if (row_gemm_pool_supported(upd, nxt)) {
        GDP_LAUNCH(GDP_K_GEMM_UPDATE_POOL, launch_row_gemm_pool<T>(upd, nxt, st));
        p_ready = true;
      }
    }
    if (!p_ready) {
      if (row_gemm_supported(upd)) GDP_LAUNCH(GDP_K_GEMM_UPDATE, (launch_row_gemm<T>(upd, EPI_RELU, st)));
      else GDP_LAUNCH(GDP_K_GEMM_UPDATE, (launch_gemm<T, T, T>(upd, EPI_RELU, st)));
    }
    h = hout;
  }
  GraphTable ct = make_table(g);
  const int chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kPoolRows, ct.blk);
  GDP_LAUNCH(GDP_K_MEANPOOL, launch_meanpool<T>(node_emb, H, ct, chunks, at<float>(ws, pl.pool), graph_emb, st));
  return GDP_OK;
}

// ---------------------------------------------------------------------------
// gdp_place: FiLM (Eq. 4) + segment-recurrent Transformer layers + head.
// ---------------------------------------------------------------------------
// The policy sample that gdp_place_sample draws from the logits it has just
// formed (gdp_sample's kernels and their per-chunk partial sums).  Chunks
// [first, last) on stream s; launch_sample's chunks are the same whichever
// launch forms them, so splitting them over launches and streams changes no
// result.
struct SampleTail {
  int n_devices, k_samples;
  uint64_t seed;
  const float* uniforms;
  int32_t* placements;
  float* logp;
  float* partial;                 // [k_samples][chunks], outside the placer's workspace
  GraphTable ct;                  // the sampling chunks (kSampleRows rows, none across graphs)
  int chunks;
};

static int sample_chunks(const SampleTail& t, const gdp_graph* g, const float* logits, const float* lse, int first,
                         int last, hipStream_t s) {
  GDP_LAUNCH_ON(GDP_K_SAMPLE, s, launch_sample(logits, lse, g->n_nodes, t.n_devices, t.k_samples, t.seed, t.uniforms,
                                               t.ct, t.chunks, t.placements, t.partial, s, first, last));
  return GDP_OK;
}

static int sample_reduce(const SampleTail& t, hipStream_t st) {
  GDP_LAUNCH(GDP_K_LOGP_REDUCE, launch_logp_reduce(t.partial, t.ct, t.chunks, t.k_samples, t.logp, st));
  return GDP_OK;
}

template <typename T>
static int place_impl(const gdp_graph* g, const T* node_emb, const float* graph_emb, const gdp_placer* p,
                      float* logits, float* lse, float* x_out, const PlacePlan& pl, void* ws, hipStream_t st,
                      const SampleTail* tail = nullptr) {
  const int N = g->n_nodes, G = g->n_graphs, d = p->d_model, L = p->n_layers;
  const GraphTable gt = make_table(g);
  float* film = at<float>(ws, pl.film);       // [L][2][G][d]: gamma then beta
  auto gamma_of = [&](int l) { return film + (size_t)l * 2 * G * d; };
  auto beta_of = [&](int l) { return film + (size_t)l * 2 * G * d + (size_t)G * d; };
  // Residual stream (layer inputs Y) in fp32; attention inputs and outputs in T.
  float* ybuf[2] = {at<float>(ws, pl.y0), at<float>(ws, pl.y1)};
  T* o = at<T>(ws, pl.o);

  if (p->film) {
    for (int l0 = 0; l0 < L; l0 += kFilmLayersPerLaunch) {
      const int nl = std::min(kFilmLayersPerLaunch, L - l0);
      FilmLayers<T> fw;
      for (int i = 0; i < nl; ++i) {
        const gdp_placer_layer& Ly = p->layers[l0 + i];
        fw.wg[i] = static_cast<const T*>(Ly.film_wg);
        fw.bg[i] = static_cast<const T*>(Ly.film_bg);
        fw.wb[i] = static_cast<const T*>(Ly.film_wb);
        fw.bb[i] = static_cast<const T*>(Ly.film_bb);
      }
      GDP_LAUNCH(GDP_K_FILM, launch_film_gemv<T>(fw, nl, graph_emb, G, d, d, gamma_of(l0), st));
    }
  }

  if (!p->attention) {
    // the ablation's placer: every layer and the head in one row-local kernel
    MlpPlacerArgs<T> a = {};
    a.x = node_emb;
    a.ldx = d;
    a.film = p->film ? film : nullptr;
    a.n_graphs = G;
    a.n_layers = L;
    for (int l = 0; l < L; ++l) {
      const gdp_placer_layer& Ly = p->layers[l];
      a.w1[l] = static_cast<const T*>(Ly.w_1);
      a.b1[l] = static_cast<const T*>(Ly.b_1);
      a.w2[l] = static_cast<const T*>(Ly.w_2);
      a.b2[l] = static_cast<const T*>(Ly.b_2);
      a.ln_g[l] = static_cast<const T*>(Ly.ln2_g);
      a.ln_b[l] = static_cast<const T*>(Ly.ln2_b);
    }
    a.M = N;
    a.d = d;
    a.d_ff = p->d_ff;
    const bool fused = p->n_devices <= kFusedHeadDevices;
    float* xfinal = x_out ? x_out : ybuf[0];
    if (fused) {
      a.w_out = static_cast<const T*>(p->w_out);
      a.b_out = static_cast<const T*>(p->b_out);
      a.n_dev = p->n_devices;
      a.logits = logits;
      a.lse = lse;
    }
    if (!fused || x_out) {
      a.y_out = xfinal;
      a.ldyo = d;
    }
    GDP_LAUNCH(GDP_K_MLP_PLACER, launch_mlp_placer<T>(a, gt, st));
    if (!fused)
      GDP_LAUNCH(GDP_K_HEAD, launch_head<T>(xfinal, static_cast<const T*>(p->w_out),
                                            static_cast<const T*>(p->b_out), N, d, p->n_devices, logits, lse, st));
    if (!tail) return GDP_OK;
    int r = sample_chunks(*tail, g, logits, lse, 0, tail->chunks, st);
    return r != GDP_OK ? r : sample_reduce(*tail, st);
  }

  GraphTable qt = make_table(g);
  const int qblocks = prefix_blocks_attention(g->graph_ptr_h, G, p->seg_len, kAttnQ, qt.blk);
  const float q_scale = attn_q_scale(d / p->n_heads);
  // The head runs inside the last layer's kernel when D is small enough.
  const bool fused_head = p->n_devices <= kFusedHeadDevices;
  // Layer 0's FiLM and projection run in their own kernel; every later
  // projection is fused into the previous layer's post-attention kernel.
  auto pre_args = [&](T* qkv_out, int row0) {
    const gdp_placer_layer& L0 = p->layers[0];
    PreLayerArgs<T> a = {node_emb, d, p->film ? gamma_of(0) : nullptr, p->film ? beta_of(0) : nullptr, d,
                         ybuf[0], d, static_cast<const T*>(L0.w_qkv), static_cast<const T*>(L0.b_qkv),
                         qkv_out, 3 * d, N, d, q_scale};
    a.row0 = row0;
    return a;
  };
  auto attn_args = [&](const T* qkv_in, int qb0, int nqb) {
    AttnArgs<T> a = {qkv_in, 3 * d, o, d, d, p->n_heads, p->seg_len, p->mem_len, nqb};
    a.qblock0 = qb0;
    return a;
  };
  // Layer l's post-attention kernel on rows row0 .. N - 1, reading layer l's
  // input y and writing ynext and the next layer's QKV into qkv_out.
  auto post_args = [&](int l, const float* yin, float* ynext, T* qkv_out, int row0) {
    const gdp_placer_layer& Ly = p->layers[l];
    const bool last = l + 1 == L;
    const bool next_film = p->film && !last;
    const gdp_placer_layer* Ln = last ? nullptr : &p->layers[l + 1];
    PostAttnArgs<T> a = {o, d, yin, d,
                         static_cast<const T*>(Ly.w_o), static_cast<const T*>(Ly.b_o),
                         static_cast<const T*>(Ly.ln1_g), static_cast<const T*>(Ly.ln1_b),
                         static_cast<const T*>(Ly.w_1), static_cast<const T*>(Ly.b_1),
                         static_cast<const T*>(Ly.w_2), static_cast<const T*>(Ly.b_2),
                         static_cast<const T*>(Ly.ln2_g), static_cast<const T*>(Ly.ln2_b),
                         next_film ? gamma_of(l + 1) : nullptr, next_film ? beta_of(l + 1) : nullptr, d,
                         ynext, d,
                         Ln ? static_cast<const T*>(Ln->w_qkv) : nullptr,
                         Ln ? static_cast<const T*>(Ln->b_qkv) : nullptr,
                         Ln ? qkv_out : nullptr, 3 * d, N, d, p->d_ff, q_scale};
    if (last && fused_head) {
      a.y_out = x_out;                  // only the head reads the last layer's output, unless asked for
      a.w_out = static_cast<const T*>(p->w_out);
      a.b_out = static_cast<const T*>(p->b_out);
      a.n_dev = p->n_devices;
      a.logits = logits;
      a.lse = lse;
    }
    a.row0 = row0;
    return a;
  };
  auto ynext_of = [&](int l) { return l + 1 == L && x_out ? x_out : ybuf[(l + 1) & 1]; };

  SideStream* sd = nullptr;
  int tail_straddle[2] = {0, 0};   // sampling chunks with rows on both sides of the split
  if (pl.split > 0 && g_place_streams == 2) {
    const int r = side_stream(st, &sd);
    if (r != GDP_OK) return r;
  }
  if (!sd) {
    // one stream: projection, then per layer attention and post-attention
    T* qkv = at<T>(ws, pl.qkv);
    GDP_LAUNCH(GDP_K_PRE_LAYER, launch_pre_layer<T>(pre_args(qkv, 0), gt, st));
    for (int l = 0; l < L; ++l) {
      GDP_LAUNCH(GDP_K_ATTENTION, launch_attention<T>(attn_args(qkv, 0, qblocks), qt, st));
      GDP_LAUNCH(GDP_K_POST_ATTN, launch_post_attention<T>(post_args(l, ybuf[l & 1], ynext_of(l), qkv, 0), gt, st));
    }
  } else {
    // Two parts, rows A = [0, R) and B = [R, N) with R a segment start, so
    // that A's queries attend to keys of A only, while B's reach back into A
    // by up to mem_len rows.  A's launches go to a second stream s2, B's to
    // st; the two parts of consecutive layers overlap, which fills the
    // compute units that one part's last round of work-groups leaves idle.
    // Layer l reads QKV(l) from qkv[l & 1] and writes QKV(l + 1) to the
    // other buffer.  Orderings across the streams:
    //   A(l)  after A's QKV(l) rows are written (the projection or post-
    //         attention of part A): before B's attention of layer l, which
    //         reads those rows as memory;
    //   B(l)  after B's attention of layer l: before A's post-attention of
    //         layer l + 1, which overwrites the buffer that attention read.
    // Events a[l & 1] and b[l & 1] hold A(l) and B(l); each is waited on
    // (in host order) before it is recorded again.
    hipStream_t s2 = sd->s;
    const int R = pl.split, QA = pl.split_qblocks;
    // sampling chunks [0, tail_a) lie below R, [tail_b, chunks) at or above it
    int tail_b = 0;
    const int tail_a = tail ? blocks_below(g->graph_ptr_h, G, kSampleRows, R, &tail_b) : 0;
    tail_straddle[0] = tail_a;
    tail_straddle[1] = tail_b;
    T* qkv[2] = {at<T>(ws, pl.qkv), at<T>(ws, pl.qkv2)};
    GDP_HIP(hipEventRecord(sd->fork, st));
    GDP_HIP(hipStreamWaitEvent(s2, sd->fork, 0));
    // the launches, then the join, which st gets even when a launch fails
    auto parts = [&]() -> int {
      {
        PreLayerArgs<T> a = pre_args(qkv[0], 0);
        a.M = R;
        GDP_LAUNCH_ON(GDP_K_PRE_LAYER, s2, launch_pre_layer<T>(a, gt, s2));
        GDP_HIP(hipEventRecord(sd->a[0], s2));
        GDP_LAUNCH(GDP_K_PRE_LAYER, launch_pre_layer<T>(pre_args(qkv[0], R), gt, st));
      }
      for (int l = 0; l < L; ++l) {
        T* qin = qkv[l & 1];
        T* qout = qkv[(l + 1) & 1];
        // part B's attention
        GDP_HIP(hipStreamWaitEvent(st, sd->a[l & 1], 0));
        GDP_LAUNCH(GDP_K_ATTENTION, launch_attention<T>(attn_args(qin, QA, qblocks - QA), qt, st));
        GDP_HIP(hipEventRecord(sd->b[l & 1], st));
        // part A's attention and post-attention
        GDP_LAUNCH_ON(GDP_K_ATTENTION, s2, launch_attention<T>(attn_args(qin, 0, QA), qt, s2));
        if (l > 0) GDP_HIP(hipStreamWaitEvent(s2, sd->b[(l - 1) & 1], 0));
        {
          PostAttnArgs<T> a = post_args(l, ybuf[l & 1], ynext_of(l), qout, 0);
          a.M = R;
          GDP_LAUNCH_ON(GDP_K_POST_ATTN, s2, launch_post_attention<T>(a, gt, s2));
        }
        if (l + 1 < L) GDP_HIP(hipEventRecord(sd->a[(l + 1) & 1], s2));
        // part B's post-attention
        GDP_LAUNCH(GDP_K_POST_ATTN, launch_post_attention<T>(post_args(l, ybuf[l & 1], ynext_of(l), qout, R), gt, st));
      }
      // With the head fused, part A's logits are final once its last
      // post-attention has run: the sampling chunks wholly below R go on s2
      // beside part B's last layer, those wholly at or above R on st after
      // it; a chunk with rows on both sides waits for the join.
      if (tail && fused_head) {
        int r = sample_chunks(*tail, g, logits, lse, 0, tail_a, s2);
        if (r == GDP_OK) r = sample_chunks(*tail, g, logits, lse, tail_b, tail->chunks, st);
        if (r != GDP_OK) return r;
      }
      return GDP_OK;
    };
    const int r = parts();
    const hipError_t ej = hipEventRecord(sd->join, s2);
    const hipError_t ew = ej == hipSuccess ? hipStreamWaitEvent(st, sd->join, 0) : ej;
    if (r != GDP_OK) return r;
    if (ew != hipSuccess) return hip_fail(ew, "join of the second stream");
  }
  if (!fused_head)
    GDP_LAUNCH(GDP_K_HEAD, launch_head<T>(ynext_of(L - 1), static_cast<const T*>(p->w_out),
                                          static_cast<const T*>(p->b_out), N, d, p->n_devices, logits, lse, st));
  if (!tail) return GDP_OK;
  if (!(sd && fused_head)) {
    const int r = sample_chunks(*tail, g, logits, lse, 0, tail->chunks, st);
    if (r != GDP_OK) return r;
  } else if (tail_straddle[1] > tail_straddle[0]) {
    const int r = sample_chunks(*tail, g, logits, lse, tail_straddle[0], tail_straddle[1], st);
    if (r != GDP_OK) return r;
  }
  return sample_reduce(*tail, st);
}

}  // namespace gdp

using namespace gdp;

// ===========================================================================
extern "C" size_t gdp_workspace_bytes(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer,
                                      int32_t k_samples) {
  clear_error();
  if (check_graph(g) != GDP_OK) return 0;
  size_t need = 0;
  if (gnn) {
    if (check_gnn(g, gnn) != GDP_OK) return 0;
    EmbedPlan e;
    plan_embed(g, gnn, &e);
    need = e.c.total;
  }
  if (placer) {
    if (check_placer(g, placer) != GDP_OK) return 0;
    PlacePlan p;
    plan_place(g, placer, &p);
    if (p.c.total > need) need = p.c.total;
    if (k_samples > 0) {
      // gdp_place_sample: the sample's regions after the placer's
      SamplePlan s;
      plan_sample(g, k_samples, &s);
      if (p.c.total + s.c.total > need) need = p.c.total + s.c.total;
    }
  }
  if (k_samples > 0) {
    SamplePlan s;
    plan_sample(g, k_samples, &s);
    if (s.c.total > need) need = s.c.total;
  }
  return need;
}

extern "C" int gdp_embed(const gdp_graph* g, const gdp_gnn* gnn, void* node_emb, float* graph_emb, void* ws,
                         size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_gnn(g, gnn)) != GDP_OK) return r;
  if (!node_emb || !graph_emb) return fail(GDP_E_INVALID_ARG, "node_emb or graph_emb is NULL");
  if (!aligned16(node_emb) || !aligned16(g->x)) return fail(GDP_E_INVALID_ARG, "x and node_emb must be 16-byte aligned");
  EmbedPlan pl;
  plan_embed(g, gnn, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (g->dtype == GDP_BF16) return embed_impl<bf16>(g, gnn, static_cast<bf16*>(node_emb), graph_emb, pl, ws, st);
  return embed_impl<float>(g, gnn, static_cast<float*>(node_emb), graph_emb, pl, ws, st);
}

// The sample, when given, must already have passed check_sample and the
// pointer checks of gdp_sample; its partial sums go after the placer's regions.
struct SampleRequest {
  int32_t k_samples;
  uint64_t seed;
  const float* uniforms;
  int32_t* placements;
  float* logp;
};

static int place_entry(const gdp_graph* g, const void* node_emb, const float* graph_emb, const gdp_placer* placer,
                       float* logits, float* lse, float* x_out, void* ws, size_t ws_bytes, void* stream,
                       const SampleRequest* sample = nullptr) {
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_placer(g, placer)) != GDP_OK) return r;
  if (!node_emb || !logits) return fail(GDP_E_INVALID_ARG, "node_emb or logits is NULL");
  if (placer->film && !graph_emb) return fail(GDP_E_INVALID_ARG, "graph_emb is NULL with film = 1");
  if (!aligned16(node_emb)) return fail(GDP_E_INVALID_ARG, "node_emb must be 16-byte aligned");
  PlacePlan pl;
  plan_place(g, placer, &pl);
  SamplePlan sp;
  SampleTail tail;
  size_t need = pl.c.total;
  if (sample) {
    plan_sample(g, sample->k_samples, &sp);
    need += sp.c.total;
  }
  if ((r = check_ws(ws, ws_bytes, need)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  if (sample) {
    tail.n_devices = placer->n_devices;
    tail.k_samples = sample->k_samples;
    tail.seed = sample->seed;
    tail.uniforms = sample->uniforms;
    tail.placements = sample->placements;
    tail.logp = sample->logp;
    tail.partial = at<float>(ws, pl.c.total + sp.partial);
    tail.ct = make_table(g);
    tail.chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kSampleRows, tail.ct.blk);
  }
  const SampleTail* t = sample ? &tail : nullptr;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (g->dtype == GDP_BF16)
    return place_impl<bf16>(g, static_cast<const bf16*>(node_emb), graph_emb, placer, logits, lse, x_out, pl, ws, st, t);
  return place_impl<float>(g, static_cast<const float*>(node_emb), graph_emb, placer, logits, lse, x_out, pl, ws, st, t);
}

extern "C" int gdp_place(const gdp_graph* g, const void* node_emb, const float* graph_emb, const gdp_placer* placer,
                         float* logits, float* lse, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  return place_entry(g, node_emb, graph_emb, placer, logits, lse, nullptr, ws, ws_bytes, stream);
}

extern "C" int gdp_place_sample(const gdp_graph* g, const void* node_emb, const float* graph_emb,
                                const gdp_placer* placer, float* logits, float* lse, int32_t k_samples, uint64_t seed,
                                const float* uniforms, int32_t* placements, float* logp, void* ws, size_t ws_bytes,
                                void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_placer(g, placer)) != GDP_OK) return r;
  if ((r = check_sample(g, placer->n_devices, k_samples)) != GDP_OK) return r;
  if (!placements || !logp) return fail(GDP_E_INVALID_ARG, "placements or logp is NULL");
  const SampleRequest req = {k_samples, seed, uniforms, placements, logp};
  return place_entry(g, node_emb, graph_emb, placer, logits, lse, nullptr, ws, ws_bytes, stream, &req);
}

extern "C" int gdp_place_train(const gdp_graph* g, const void* node_emb, const float* graph_emb,
                               const gdp_placer* placer, float* logits, float* lse, float* x_out, void* ws,
                               size_t ws_bytes, void* stream) {
  clear_error();
  if (!x_out || !aligned16(x_out)) return fail(GDP_E_INVALID_ARG, "x_out is NULL or not 16-byte aligned");
  return place_entry(g, node_emb, graph_emb, placer, logits, lse, x_out, ws, ws_bytes, stream);
}

extern "C" int gdp_head_backward(const gdp_graph* g, const gdp_placer* placer, const float* x, const float* dlogits,
                                 float* dx, float* dw_out, float* db_out, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_placer(g, placer)) != GDP_OK) return r;
  if (!x || !dlogits || !dx || !dw_out || !db_out) return fail(GDP_E_INVALID_ARG, "a head-backward input or output is NULL");
  if (!aligned16(x) || !aligned16(dx)) return fail(GDP_E_INVALID_ARG, "x or dx is not 16-byte aligned");
  PlacePlan pl;
  plan_place(g, placer, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  float* partial = at<float>(ws, pl.head_partial);
  const int N = g->n_nodes, d = placer->d_model, D = placer->n_devices;
  if (g->dtype == GDP_BF16)
    GDP_LAUNCH(GDP_K_HEAD_BWD, launch_head_backward<bf16>(x, static_cast<const bf16*>(placer->w_out), dlogits, N, d, D,
                                                          dx, dw_out, db_out, partial, st));
  else
    GDP_LAUNCH(GDP_K_HEAD_BWD, launch_head_backward<float>(x, static_cast<const float*>(placer->w_out), dlogits, N, d,
                                                           D, dx, dw_out, db_out, partial, st));
  return GDP_OK;
}

extern "C" int gdp_advantages(int32_t n_graphs, int32_t k_samples, const float* run_time, const uint8_t* valid,
                              double* reward_sum, int64_t* trial_count, float* reward, float* advantage,
                              void* stream) {
  clear_error();
  if (n_graphs < 1 || n_graphs > GDP_MAX_GRAPHS)
    return fail(GDP_E_UNSUPPORTED, "n_graphs = %d outside 1..%d", n_graphs, GDP_MAX_GRAPHS);
  if (k_samples < 1) return fail(GDP_E_INVALID_ARG, "k_samples = %d < 1", k_samples);
  if (!run_time || !reward_sum || !trial_count || !advantage)
    return fail(GDP_E_INVALID_ARG, "run_time, reward_sum, trial_count or advantage is NULL");
  int r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  GDP_LAUNCH(GDP_K_ADVANTAGE, launch_advantages(run_time, valid, n_graphs, k_samples, reward_sum, trial_count, reward,
                                                advantage, st));
  return GDP_OK;
}

extern "C" int gdp_sample(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                          int32_t k_samples, uint64_t seed, const float* uniforms, int32_t* placements, float* logp,
                          void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_sample(g, n_devices, k_samples)) != GDP_OK) return r;
  if (!logits || !placements || !logp) return fail(GDP_E_INVALID_ARG, "logits, placements or logp is NULL");
  SamplePlan pl;
  plan_sample(g, k_samples, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  GraphTable ct = make_table(g);
  const int chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kSampleRows, ct.blk);
  float* partial = at<float>(ws, pl.partial);
  GDP_LAUNCH(GDP_K_SAMPLE, launch_sample(logits, lse, g->n_nodes, n_devices, k_samples, seed, uniforms, ct, chunks,
                                         placements, partial, st));
  GDP_LAUNCH(GDP_K_LOGP_REDUCE, launch_logp_reduce(partial, ct, chunks, k_samples, logp, st));
  return GDP_OK;
}

// ---------------------------------------------------------------------------
// gdp_sample_noalloc: gdp_sample's kernels with their per-(k, chunk) partial
// sums in a library-owned device array instead of the caller's workspace.
// The array is a file-scope __device__ symbol: each GPU holds its own copy,
// whose device address is looked up once per device (the first call made
// with that device current) and used from then on.  The symbol's name in host
// code is not a device address and is never passed to a kernel or copy.
// ---------------------------------------------------------------------------
static __device__ __align__(256) float scratch[GDP_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxScratchDevices] = {};
}  // namespace

static int scratch_for_current_device(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(GDP_E_UNSUPPORTED, "device %d beyond the %d devices the scratch table holds", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(GDP_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return GDP_OK;
}

extern "C" int gdp_sample_noalloc(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                                  int32_t k_samples, uint64_t seed, const float* uniforms, int32_t* placements,
                                  float* logp, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_sample(g, n_devices, k_samples)) != GDP_OK) return r;
  if (!logits || !placements || !logp) return fail(GDP_E_INVALID_ARG, "logits, placements or logp is NULL");
  GraphTable ct = make_table(g);
  const int chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kSampleRows, ct.blk);
  const size_t need = (size_t)k_samples * (size_t)chunks * sizeof(float);
  if (need > GDP_NOALLOC_SCRATCH_BYTES)
    return fail(GDP_E_UNSUPPORTED, "K * ceil(nodes / 256) partial sums need %zu bytes > GDP_NOALLOC_SCRATCH_BYTES = %zu",
                need, (size_t)GDP_NOALLOC_SCRATCH_BYTES);
  float* partial = nullptr;
  if ((r = scratch_for_current_device(&partial)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  GDP_LAUNCH(GDP_K_SAMPLE, launch_sample(logits, lse, g->n_nodes, n_devices, k_samples, seed, uniforms, ct, chunks,
                                         placements, partial, st));
  GDP_LAUNCH(GDP_K_LOGP_REDUCE, launch_logp_reduce(partial, ct, chunks, k_samples, logp, st));
  return GDP_OK;
}

extern "C" int gdp_ppo_grad(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                            int32_t k_samples, const int32_t* placements, const float* logp, const float* logp_old,
                            const float* advantages, float clip_eps, float* loss, float* dlogits, void* ws,
                            size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_sample(g, n_devices, k_samples)) != GDP_OK) return r;
  if (!logits || !placements || !logp || !logp_old || !advantages || !loss || !dlogits)
    return fail(GDP_E_INVALID_ARG, "a PPO input or output is NULL");
  if (!(clip_eps > 0.0f && clip_eps < 1.0f)) return fail(GDP_E_INVALID_ARG, "clip_eps = %g must lie in (0, 1)", clip_eps);
  SamplePlan pl;
  plan_sample(g, k_samples, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const GraphTable gt = make_table(g);
  GDP_LAUNCH(GDP_K_PPO, launch_ppo(logits, lse, placements, logp, logp_old, advantages, clip_eps, gt, g->n_nodes,
                                   n_devices, k_samples, at<float>(ws, pl.coef), loss, dlogits, st));
  return GDP_OK;
}

// ---------------------------------------------------------------------------
// gdp_evaluate: the simulated run time and validity of every sampled placement.
// ---------------------------------------------------------------------------
extern "C" size_t gdp_evaluate_workspace_bytes(const gdp_graph* g, int32_t n_devices, int32_t k_samples) {
  clear_error();
  if (check_graph(g) != GDP_OK) return 0;
  if (check_sample(g, n_devices, k_samples) != GDP_OK) return 0;
  EvalPlan pl;
  plan_evaluate(g, n_devices, k_samples, &pl);
  return pl.c.total;
}

extern "C" int gdp_evaluate(const gdp_graph* g, int32_t n_devices, int32_t k_samples, const int32_t* placements,
                            const int32_t* op_cost, const int32_t* out_xfer, const int32_t* op_mem,
                            const int64_t* mem_cap_h, double time_unit, int64_t* makespan, uint8_t* valid,
                            float* run_time, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_sample(g, n_devices, k_samples)) != GDP_OK) return r;
  if (!placements || !op_cost || !out_xfer || !op_mem || !makespan || !valid)
    return fail(GDP_E_INVALID_ARG, "an evaluator input or output is NULL");
  if (!mem_cap_h) return fail(GDP_E_INVALID_ARG, "mem_cap_h is NULL");
  for (int i = 0; i < g->n_graphs; ++i)
    if (mem_cap_h[i] < 0) return fail(GDP_E_INVALID_ARG, "mem_cap_h[%d] = %lld < 0", i, (long long)mem_cap_h[i]);
  if (!(time_unit >= 0.0) || time_unit > 1e30) return fail(GDP_E_INVALID_ARG, "time_unit = %g", time_unit);
  if (((uintptr_t)makespan & 7u) != 0) return fail(GDP_E_INVALID_ARG, "makespan must be 8-byte aligned");
  EvalPlan pl;
  plan_evaluate(g, n_devices, k_samples, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int N = g->n_nodes;
  int* counters = at<int>(ws, pl.counters);
  int* in_ptr = at<int>(ws, pl.in_ptr);
  int* in_idx = at<int>(ws, pl.in_idx);
  GDP_LAUNCH(GDP_K_EVALUATE, launch_fill_i32(counters, 2 * (int64_t)N + 1, 0, st));
  GDP_LAUNCH(GDP_K_EVALUATE, launch_in_degree(g->col_idx, g->n_edges, counters, st));
  GDP_LAUNCH(GDP_K_EVALUATE, launch_scan_degrees(g->row_ptr, counters, N, 1, in_ptr, at<int>(ws, pl.s_ptr),
                                                 at<int>(ws, pl.scan_tmp), st));
  GDP_LAUNCH(GDP_K_EVALUATE, launch_fill_reverse(g->row_ptr, g->col_idx, in_ptr, N, g->n_edges, counters + N, in_idx,
                                                 st));
  const GraphTable gt = make_table(g);
  GraphTable ct = make_table(g);
  const int chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kEvalRows, ct.blk);
  EvalLaunch L;
  L.placements = placements;
  L.op_cost = op_cost;
  L.out_xfer = out_xfer;
  L.op_mem = op_mem;
  L.mem_cap = mem_cap_h;
  L.in_ptr = in_ptr;
  L.in_idx = in_idx;
  L.n_edges = g->n_edges;
  L.gt = &gt;
  L.chunk_table = &ct;
  L.chunks = chunks;
  L.n = N;
  L.D = n_devices;
  L.K = k_samples;
  L.time_unit = time_unit;
  L.rec = at<void>(ws, pl.rec);
  L.memsum = at<void>(ws, pl.memsum);
  L.far = at<unsigned>(ws, pl.far);
  L.makespan = makespan;
  L.valid = valid;
  L.run_time = run_time;
  GDP_LAUNCH(GDP_K_EVALUATE, launch_evaluate(L, st));
  return GDP_OK;
}

// ===========================================================================
// The update step: training forward (all intermediates kept), backward, Adam.
// ===========================================================================
namespace gdp {
namespace {

inline void set_bias(tr::GemmStrided<float, float>& g, const float* b) { g.bias_f = b; }
inline void set_bias(tr::GemmStrided<bf16, bf16>& g, const bf16* b) { g.bias_h = b; }
inline void set_bias(tr::GemmStrided<float, bf16>& g, const bf16* b) { g.bias_h = b; }
inline void set_bias(tr::GemmStrided<bf16, float>& g, const float* b) { g.bias_f = b; }

struct TrainCtx {
  hipStream_t st;
  float* partial;          // split-k sums
  size_t partial_floats;
  float* colpart;          // column-sum partials
  GraphTable rows;         // all rows as one segment (256-row chunks in blk)
  int row_chunks;
  GraphTable graphs;       // the graphs, each in 256-row chunks
  int graph_chunks;
};

// C[M, N] (+)= act(A[M, K] W[N, K]^T + bias): a linear layer on row-major activations.
template <typename TA, typename TW>
hipError_t lin(const TA* A, int lda, const TW* W, int ldw, const TW* bias, int M, int N, int K, float* C, int ldc,
               int act, bool acc, const TrainCtx& cx) {
  tr::GemmStrided<TA, TW> g;
  g.a = A; g.sam = lda; g.sak = 1;
  g.b = W; g.sbk = 1; g.sbn = ldw;
  g.M = M; g.N = N; g.K = K;
  g.c = C; g.ldc = ldc;
  if (bias) set_bias(g, bias);
  g.act = act;
  g.accumulate = acc;
  return tr::launch_gemm_strided(g, nullptr, 0, cx.st);
}

// C[M, N] (+)= (dY[M, K] W[K, N]) masked where mask <= 0: a linear layer's input gradient.
template <typename TW>
hipError_t lin_dx(const float* dY, int ldy, const TW* W, int ldw, int M, int N, int K, float* C, int ldc,
                  const float* mask, int ldm, bool acc, const TrainCtx& cx) {
  tr::GemmStrided<float, TW> g;
  g.a = dY; g.sam = ldy; g.sak = 1;
  g.b = W; g.sbk = ldw; g.sbn = 1;
  g.M = M; g.N = N; g.K = K;
  g.c = C; g.ldc = ldc;
  g.mask = mask; g.ldm = ldm;
  g.accumulate = acc;
  return tr::launch_gemm_strided(g, nullptr, 0, cx.st);
}

// dW[M, N] (+)= sum over rows r of dY[r][m] X[r][n]: a linear layer's weight gradient.
template <typename TX>
hipError_t lin_dw(const float* dY, int ldy, const TX* X, int ldx, int M, int N, int rows, float* C, int ldc, bool acc,
                  const TrainCtx& cx) {
  tr::GemmStrided<float, TX> g;
  g.a = dY; g.sam = 1; g.sak = ldy;
  g.b = X; g.sbk = ldx; g.sbn = 1;
  g.M = M; g.N = N; g.K = rows;
  g.c = C; g.ldc = ldc;
  g.accumulate = acc;
  return tr::launch_gemm_strided(g, cx.partial, cx.partial_floats, cx.st);
}

// out[c] (+)= sum over all rows of a[r][c] (* b[r][c])
template <typename TA>
hipError_t colsum(const TA* a, int lda, const float* b, int ldb, int C, float* out, bool acc, const TrainCtx& cx) {
  return tr::launch_colsum(a, lda, b, ldb, C, cx.rows, cx.row_chunks, cx.colpart, out, 0, acc, cx.st);
}

GraphTable one_segment(int rows, int chunk_rows, int* chunks) {
  GraphTable t;
  memset(&t, 0, sizeof(t));
  t.n = 1;
  t.ptr[0] = 0;
  t.ptr[1] = rows;
  t.blk[0] = 0;
  t.blk[1] = (rows + chunk_rows - 1) / chunk_rows;
  *chunks = t.blk[1];
  return t;
}

template <typename T>
int train_forward_impl(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* p, const TrainPlan& tp, char* store,
                       char* ws, float* logits, float* lse, hipStream_t st) {
  const int N = g->n_nodes, G = g->n_graphs, H = gnn->hidden, d = p->d_model, dff = p->d_ff, F = g->feat_dim;
  const GraphTable gt = make_table(g);
  TrainCtx cx;
  cx.st = st;
  auto S = [&](size_t off) { return reinterpret_cast<float*>(store + off); };
  auto SI = [&](size_t off) { return reinterpret_cast<int*>(store + off); };
  // neighbourhoods and their sample (as gdp_embed), in-edge rows sorted
  {
    int* counters = reinterpret_cast<int*>(ws + tp.counters);
    int* in_ptr = SI(tp.in_ptr);
    int* in_idx = SI(tp.in_idx);
    GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_fill_i32(counters, 2 * (int64_t)N + 1, 0, st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_in_degree(g->col_idx, g->n_edges, counters, st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_scan_degrees(g->row_ptr, counters, N, gnn->fanout, in_ptr, SI(tp.s_ptr),
                                                    reinterpret_cast<int*>(ws + tp.scan_tmp), st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_fill_reverse(g->row_ptr, g->col_idx, in_ptr, N, g->n_edges, counters + N, in_idx,
                                                    st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_nbr_sample(g->row_ptr, g->col_idx, in_ptr, in_idx, SI(tp.s_ptr), N, gnn->fanout,
                                                  gnn->nbr_seed, gt, SI(tp.s_idx), reinterpret_cast<int*>(ws + tp.heavy),
                                                  counters + 2 * N, st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_sort_rows(in_ptr, N, in_idx, st));
  }
  // Eq. 2 and Eq. 3
  const T* x = static_cast<const T*>(g->x);
  for (int l = 0; l < gnn->n_layers; ++l) {
    const gdp_gnn_layer& Lw = gnn->layers[l];
    float* P = S(tp.P[l]);
    float* A = S(tp.A[l]);
    float* hout = S(tp.h[l + 1]);
    const T* wp = static_cast<const T*>(Lw.w_pool);
    const T* ws_ = static_cast<const T*>(Lw.w_self);
    if (l == 0) {
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<T, T>(x, F, wp, F, static_cast<const T*>(Lw.b_pool), N, H, F, P, H,
                                            tr::ACT_SIGMOID, false, cx));
    } else {
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(S(tp.h[l]), H, wp, H, static_cast<const T*>(Lw.b_pool), N, H, H, P, H,
                                                tr::ACT_SIGMOID, false, cx));
    }
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_gather_max_arg(P, SI(tp.s_ptr), SI(tp.s_idx), N, H, A, SI(tp.arg[l]), st));
    if (l == 0) {
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<T, T>(x, F, ws_, F, static_cast<const T*>(Lw.b_upd), N, H, F, hout, H,
                                            tr::ACT_NONE, false, cx));
    } else {
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(S(tp.h[l]), H, ws_, H, static_cast<const T*>(Lw.b_upd), N, H, H, hout,
                                                H, tr::ACT_NONE, false, cx));
    }
    GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(A, H, static_cast<const T*>(Lw.w_neigh), H, nullptr, N, H, H, hout, H,
                                              tr::ACT_NONE, true, cx));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_ew(tr::EW_MASK_POS, hout, hout, nullptr, (size_t)N * H, hout, st));
  }
  float* x0 = S(tp.x0);
  {
    GraphTable ct = make_table(g);
    const int nch = prefix_blocks_rows(g->graph_ptr_h, G, tr::kColChunkRows, ct.blk);
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_meanpool_f32(S(tp.h[gnn->n_layers]), H, ct, nch,
                                                        reinterpret_cast<float*>(ws + tp.colpart), x0, st));
  }
  // Eq. 4: gamma, beta of every layer
  float* film = S(tp.film);
  if (p->film) {
    for (int l0 = 0; l0 < p->n_layers; l0 += kFilmLayersPerLaunch) {
      const int nl = std::min(kFilmLayersPerLaunch, p->n_layers - l0);
      FilmLayers<T> fw;
      for (int i = 0; i < nl; ++i) {
        const gdp_placer_layer& Ly = p->layers[l0 + i];
        fw.wg[i] = static_cast<const T*>(Ly.film_wg);
        fw.bg[i] = static_cast<const T*>(Ly.film_bg);
        fw.wb[i] = static_cast<const T*>(Ly.film_wb);
        fw.bb[i] = static_cast<const T*>(Ly.film_bb);
      }
      GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_film_gemv<T>(fw, nl, x0, G, d, H, film + (size_t)l0 * 2 * G * d, st));
    }
  }
  // the placer
  for (int l = 0; l < p->n_layers; ++l) {
    const gdp_placer_layer& Ly = p->layers[l];
    const float* X = S(tp.X[l]);
    float* Y = S(tp.Y[l]);
    const float* gam = p->film ? film + (size_t)l * 2 * G * d : nullptr;
    const float* bet = p->film ? gam + (size_t)G * d : nullptr;
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_film_apply<float>(X, N, d, gam, bet, gt, Y, st));
    const float* ffn_in = Y;
    if (p->attention) {
      float* qkv = S(tp.QKV[l]);
      float* O = S(tp.O[l]);
      float* R1 = S(tp.R1[l]);
      float* Z = S(tp.Z[l]);
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(Y, d, static_cast<const T*>(Ly.w_qkv), d,
                                                static_cast<const T*>(Ly.b_qkv), N, 3 * d, d, qkv, 3 * d, tr::ACT_NONE,
                                                false, cx));
      GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_attn_fwd(qkv, N, d, p->n_heads, p->seg_len, p->mem_len, gt, O,
                                                      S(tp.lse_att[l]), st));
      GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(O, d, static_cast<const T*>(Ly.w_o), d, static_cast<const T*>(Ly.b_o),
                                                N, d, d, R1, d, tr::ACT_NONE, false, cx));
      GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_ew(tr::EW_ADD, R1, Y, nullptr, (size_t)N * d, R1, st));
      GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_ln_fwd<T>(R1, N, d, static_cast<const T*>(Ly.ln1_g),
                                                       static_cast<const T*>(Ly.ln1_b), Z, st));
      ffn_in = Z;
    }
    float* H1 = S(tp.H1[l]);
    float* R2 = S(tp.R2[l]);
    GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(ffn_in, d, static_cast<const T*>(Ly.w_1), d,
                                              static_cast<const T*>(Ly.b_1), N, dff, d, H1, dff, tr::ACT_RELU, false,
                                              cx));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, lin<float, T>(H1, dff, static_cast<const T*>(Ly.w_2), dff,
                                              static_cast<const T*>(Ly.b_2), N, d, dff, R2, d, tr::ACT_NONE, false,
                                              cx));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_ew(tr::EW_ADD, R2, ffn_in, nullptr, (size_t)N * d, R2, st));
    GDP_LAUNCH(GDP_K_TRAIN_FWD, tr::launch_ln_fwd<T>(R2, N, d, static_cast<const T*>(Ly.ln2_g),
                                                     static_cast<const T*>(Ly.ln2_b), S(tp.X[l + 1]), st));
  }
  GDP_LAUNCH(GDP_K_TRAIN_FWD, launch_head<T>(S(tp.X[p->n_layers]), static_cast<const T*>(p->w_out),
                                             static_cast<const T*>(p->b_out), N, d, p->n_devices, logits, lse, st));
  return GDP_OK;
}

template <typename T>
int backward_impl(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* p, const TrainPlan& tp,
                  const char* store, char* ws, const float* dlogits, const gdp_grads* gr, hipStream_t st) {
  const int N = g->n_nodes, G = g->n_graphs, H = gnn->hidden, d = p->d_model, dff = p->d_ff, F = g->feat_dim;
  const GraphTable gt = make_table(g);
  auto S = [&](size_t off) { return reinterpret_cast<const float*>(store + off); };
  auto SI = [&](size_t off) { return reinterpret_cast<const int*>(store + off); };
  auto W = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  TrainCtx cx;
  cx.st = st;
  cx.partial = W(tp.gemm_partial);
  cx.partial_floats = tp.gemm_partial_floats;
  cx.colpart = W(tp.colpart);
  cx.rows = one_segment(N, tr::kColChunkRows, &cx.row_chunks);
  cx.graphs = make_table(g);
  cx.graph_chunks = prefix_blocks_rows(g->graph_ptr_h, G, tr::kColChunkRows, cx.graphs.blk);
  float* dX = W(tp.dX);
  float* dY = W(tp.dY);
  float* dR = W(tp.dR);
  float* dZ = W(tp.dZ);
  float* xg = W(tp.xg);
  float* dH = W(tp.dH);
  // the head
  GDP_LAUNCH(GDP_K_BACKWARD, launch_head_backward<T>(S(tp.X[p->n_layers]), static_cast<const T*>(p->w_out), dlogits, N,
                                                     d, p->n_devices, dX, gr->w_out, gr->b_out, W(tp.head_partial), st));
  const float* film = S(tp.film);
  float* dfilm = W(tp.dfilm);
  for (int l = p->n_layers - 1; l >= 0; --l) {
    const gdp_placer_layer& Ly = p->layers[l];
    const gdp_placer_layer_grad& Gl = gr->placer[l];
    const float* Xin = S(tp.X[l]);
    const float* Y = S(tp.Y[l]);
    const float* ffn_in = p->attention ? S(tp.Z[l]) : Y;
    // LN2, the FFN and its residual: dZ = dR2 + dH W_1
    GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ln_bwd<T>(S(tp.R2[l]), dX, N, d, static_cast<const T*>(Ly.ln2_g), dR, xg, st));
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(xg, d, nullptr, 0, d, Gl.ln2_g, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dX, d, nullptr, 0, d, Gl.ln2_b, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dR, d, static_cast<const T*>(Ly.w_2), dff, N, dff, d, dH, dff, S(tp.H1[l]),
                                         dff, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dR, d, S(tp.H1[l]), dff, d, dff, N, Gl.w_2, dff, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dR, d, nullptr, 0, d, Gl.b_2, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dH, dff, static_cast<const T*>(Ly.w_1), d, N, d, dff, dZ, d, nullptr, 0, false,
                                         cx));
    GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ew(tr::EW_ADD, dZ, dR, nullptr, (size_t)N * d, dZ, st));
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dH, dff, ffn_in, d, dff, d, N, Gl.w_1, d, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dH, dff, nullptr, 0, dff, Gl.b_1, false, cx));
    const float* dYp = dZ;   // the gradient reaching Y
    if (p->attention) {
      const float* O = S(tp.O[l]);
      const float* qkv = S(tp.QKV[l]);
      float* dqkv = W(tp.dqkv);
      float* dkvm = W(tp.dkvm);
      // LN1 and the out-projection: dR = dR1, dO (in dX, free now)
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ln_bwd<T>(S(tp.R1[l]), dZ, N, d, static_cast<const T*>(Ly.ln1_g), dR, xg,
                                                      st));
      GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(xg, d, nullptr, 0, d, Gl.ln1_g, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dZ, d, nullptr, 0, d, Gl.ln1_b, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dR, d, static_cast<const T*>(Ly.w_o), d, N, d, d, dX, d, nullptr, 0, false,
                                           cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dR, d, O, d, d, d, N, Gl.w_o, d, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dR, d, nullptr, 0, d, Gl.b_o, false, cx));
      // attention: own-segment (live) and memory parts of dK, dV
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_attn_bwd(qkv, O, dX, S(tp.lse_att[l]), N, d, p->n_heads, p->seg_len,
                                                     p->mem_len, gt, W(tp.Dq), dqkv, dkvm, st));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dqkv, 3 * d, Y, d, 3 * d, d, N, Gl.w_qkv, d, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dkvm, 2 * d, Y, d, 2 * d, d, N, Gl.w_qkv + (size_t)d * d, d, true, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dqkv, 3 * d, nullptr, 0, 3 * d, Gl.b_qkv, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dkvm, 2 * d, nullptr, 0, 2 * d, Gl.b_qkv + d, true, cx));
      // dY = dR1 + [dQ | dK | dV]_live W_qkv (the memory's part stops at the weights)
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dqkv, 3 * d, static_cast<const T*>(Ly.w_qkv), d, N, d, 3 * d, dY, d, nullptr,
                                           0, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ew(tr::EW_ADD, dY, dR, nullptr, (size_t)N * d, dY, st));
      dYp = dY;
    }
    // FiLM: dX = gamma dY; dgamma[g] = sum_g dY X, dbeta[g] = sum_g dY
    if (p->film) {
      const float* gam = film + (size_t)l * 2 * G * d;
      float* dg = dfilm + (size_t)l * 2 * G * d;
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_film_dx(dYp, N, d, gam, gt, dX, st));
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_colsum<float>(dYp, d, Xin, d, d, cx.graphs, cx.graph_chunks, cx.colpart, dg,
                                                          d, false, st));
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_colsum<float>(dYp, d, nullptr, 0, d, cx.graphs, cx.graph_chunks, cx.colpart,
                                                          dg + (size_t)G * d, d, false, st));
    } else {
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_film_dx(dYp, N, d, nullptr, gt, dX, st));
    }
  }
  // FiLM weights and the graph embeddings' gradient dx0 [G, H]
  float* dx0 = W(tp.dx0);
  GDP_LAUNCH(GDP_K_BACKWARD, launch_fill_i32(reinterpret_cast<int*>(dx0), (int64_t)G * H, 0, st));
  if (p->film) {
    int gch = 0;
    const GraphTable grows = one_segment(G, tr::kColChunkRows, &gch);
    const float* x0 = S(tp.x0);
    for (int l = 0; l < p->n_layers; ++l) {
      const gdp_placer_layer& Ly = p->layers[l];
      const gdp_placer_layer_grad& Gl = gr->placer[l];
      const float* dg = dfilm + (size_t)l * 2 * G * d;
      const float* db = dg + (size_t)G * d;
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dg, d, x0, H, d, H, G, Gl.film_wg, H, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(db, d, x0, H, d, H, G, Gl.film_wb, H, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_colsum<float>(dg, d, nullptr, 0, d, grows, gch, cx.colpart, Gl.film_bg, 0,
                                                          false, st));
      GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_colsum<float>(db, d, nullptr, 0, d, grows, gch, cx.colpart, Gl.film_bb, 0,
                                                          false, st));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dg, d, static_cast<const T*>(Ly.film_wg), H, G, H, d, dx0, H, nullptr, 0,
                                           true, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(db, d, static_cast<const T*>(Ly.film_wb), H, G, H, d, dx0, H, nullptr, 0,
                                           true, cx));
    }
  }
  // the GNN: dh of the final embeddings = the placer's input gradient + the mean pool's share of dx0
  GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_meanpool_bwd(dx0, N, H, gt, dX, st));
  float* dh_cur = dX;
  float* dh_next = W(tp.dh);
  float* dU = W(tp.dU);
  float* dA = W(tp.dA);
  float* dP = W(tp.dP);
  const T* x = static_cast<const T*>(g->x);
  for (int l = gnn->n_layers - 1; l >= 0; --l) {
    const gdp_gnn_layer& Lw = gnn->layers[l];
    const gdp_gnn_layer_grad& Gl = gr->gnn[l];
    const int hin = l == 0 ? F : H;
    GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ew(tr::EW_MASK_POS, dh_cur, S(tp.h[l + 1]), nullptr, (size_t)N * H, dU, st));
    if (l == 0) {
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<T>(dU, H, x, F, H, F, N, Gl.w_self, F, false, cx));
    } else {
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dU, H, S(tp.h[l]), H, H, H, N, Gl.w_self, H, false, cx));
    }
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dU, H, S(tp.A[l]), H, H, H, N, Gl.w_neigh, H, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dU, H, nullptr, 0, H, Gl.b_upd, false, cx));
    GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dU, H, static_cast<const T*>(Lw.w_neigh), H, N, H, H, dA, H, nullptr, 0, false,
                                         cx));
    GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_gather_max_bwd(dA, SI(tp.arg[l]), g->row_ptr, g->col_idx, SI(tp.in_ptr),
                                                         SI(tp.in_idx), N, H, dP, st));
    GDP_LAUNCH(GDP_K_BACKWARD, tr::launch_ew(tr::EW_SIGMOID_GRAD, dP, S(tp.P[l]), nullptr, (size_t)N * H, dP, st));
    if (l == 0) {
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<T>(dP, H, x, F, H, F, N, Gl.w_pool, F, false, cx));
    } else {
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dw<float>(dP, H, S(tp.h[l]), H, H, H, N, Gl.w_pool, H, false, cx));
    }
    GDP_LAUNCH(GDP_K_BACKWARD, colsum<float>(dP, H, nullptr, 0, H, Gl.b_pool, false, cx));
    if (l > 0) {
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dU, H, static_cast<const T*>(Lw.w_self), hin, N, hin, H, dh_next, hin,
                                           nullptr, 0, false, cx));
      GDP_LAUNCH(GDP_K_BACKWARD, lin_dx<T>(dP, H, static_cast<const T*>(Lw.w_pool), hin, N, hin, H, dh_next, hin,
                                           nullptr, 0, true, cx));
      std::swap(dh_cur, dh_next);
    }
  }
  return GDP_OK;
}

int check_grads(const gdp_gnn* gnn, const gdp_placer* p, const gdp_grads* gr) {
  if (!gr || !gr->gnn || !gr->placer || !gr->w_out || !gr->b_out) return fail(GDP_E_INVALID_ARG, "grads has a NULL array");
  for (int l = 0; l < gnn->n_layers; ++l) {
    const gdp_gnn_layer_grad& G = gr->gnn[l];
    if (!G.w_pool || !G.b_pool || !G.w_self || !G.w_neigh || !G.b_upd)
      return fail(GDP_E_INVALID_ARG, "grads: GNN layer %d has a NULL array", l);
  }
  for (int l = 0; l < p->n_layers; ++l) {
    const gdp_placer_layer_grad& G = gr->placer[l];
    if (!G.w_1 || !G.b_1 || !G.w_2 || !G.b_2 || !G.ln2_g || !G.ln2_b)
      return fail(GDP_E_INVALID_ARG, "grads: placer layer %d has a NULL array", l);
    if (p->attention && (!G.w_qkv || !G.b_qkv || !G.w_o || !G.b_o || !G.ln1_g || !G.ln1_b))
      return fail(GDP_E_INVALID_ARG, "grads: placer layer %d has a NULL attention array", l);
    if (p->film && (!G.film_wg || !G.film_bg || !G.film_wb || !G.film_bb))
      return fail(GDP_E_INVALID_ARG, "grads: placer layer %d has a NULL FiLM array", l);
  }
  return GDP_OK;
}

}  // namespace
}  // namespace gdp

extern "C" int gdp_train_sizes(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, size_t* store_bytes,
                               size_t* workspace_bytes) {
  clear_error();
  if (store_bytes) *store_bytes = 0;
  if (workspace_bytes) *workspace_bytes = 0;
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_train(g, gnn, placer)) != GDP_OK) return r;
  if (!store_bytes || !workspace_bytes) return fail(GDP_E_INVALID_ARG, "store_bytes or workspace_bytes is NULL");
  TrainPlan tp;
  plan_train(g, gnn, placer, &tp);
  *store_bytes = tp.store_total;
  *workspace_bytes = tp.ws_total;
  return GDP_OK;
}

static int check_store(const void* store, size_t have, size_t need) {
  if (!store) return fail(GDP_E_INVALID_ARG, "store is NULL");
  if (have < need) return fail(GDP_E_WORKSPACE, "store %zu bytes < %zu required", have, need);
  if (((uintptr_t)store & 255u) != 0) return fail(GDP_E_INVALID_ARG, "store must be 256-byte aligned");
  return GDP_OK;
}

extern "C" int gdp_forward_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, void* store,
                                 size_t store_bytes, float* logits, float* lse, void* ws, size_t ws_bytes,
                                 void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_train(g, gnn, placer)) != GDP_OK) return r;
  if (!logits) return fail(GDP_E_INVALID_ARG, "logits is NULL");
  TrainPlan tp;
  plan_train(g, gnn, placer, &tp);
  if ((r = check_store(store, store_bytes, tp.store_total)) != GDP_OK) return r;
  if ((r = check_ws(ws, ws_bytes, tp.ws_total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (g->dtype == GDP_BF16)
    return train_forward_impl<bf16>(g, gnn, placer, tp, static_cast<char*>(store), static_cast<char*>(ws), logits, lse,
                                    st);
  return train_forward_impl<float>(g, gnn, placer, tp, static_cast<char*>(store), static_cast<char*>(ws), logits, lse,
                                   st);
}

extern "C" int gdp_backward(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer, const void* store,
                            size_t store_bytes, const float* dlogits, const gdp_grads* grads, void* ws, size_t ws_bytes,
                            void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_train(g, gnn, placer)) != GDP_OK) return r;
  if (!dlogits) return fail(GDP_E_INVALID_ARG, "dlogits is NULL");
  if ((r = check_grads(gnn, placer, grads)) != GDP_OK) return r;
  TrainPlan tp;
  plan_train(g, gnn, placer, &tp);
  if ((r = check_store(store, store_bytes, tp.store_total)) != GDP_OK) return r;
  if ((r = check_ws(ws, ws_bytes, tp.ws_total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (g->dtype == GDP_BF16)
    return backward_impl<bf16>(g, gnn, placer, tp, static_cast<const char*>(store), static_cast<char*>(ws), dlogits,
                               grads, st);
  return backward_impl<float>(g, gnn, placer, tp, static_cast<const char*>(store), static_cast<char*>(ws), dlogits,
                              grads, st);
}

extern "C" int gdp_log_prob(const gdp_graph* g, const float* logits, const float* lse, int32_t n_devices,
                            int32_t k_samples, const int32_t* placements, float* logp, void* ws, size_t ws_bytes,
                            void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_sample(g, n_devices, k_samples)) != GDP_OK) return r;
  if (!logits || !placements || !logp) return fail(GDP_E_INVALID_ARG, "logits, placements or logp is NULL");
  SamplePlan pl;
  plan_sample(g, k_samples, &pl);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  GraphTable ct = make_table(g);
  const int chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kSampleRows, ct.blk);
  float* partial = at<float>(ws, pl.partial);
  GDP_LAUNCH(GDP_K_LOGPROB, launch_logp_given(logits, lse, g->n_nodes, n_devices, k_samples, placements, ct, chunks,
                                              partial, st));
  GDP_LAUNCH(GDP_K_LOGPROB, launch_logp_reduce(partial, ct, chunks, k_samples, logp, st));
  return GDP_OK;
}

extern "C" int gdp_adam_step(int32_t n_tensors, const gdp_adam_tensor* tensors, int32_t dtype, float lr, float beta1,
                             float beta2, float eps, int64_t step, void* stream) {
  clear_error();
  if (n_tensors < 0 || (n_tensors > 0 && !tensors)) return fail(GDP_E_INVALID_ARG, "tensors is NULL");
  if (dtype != GDP_F32 && dtype != GDP_BF16) return fail(GDP_E_INVALID_ARG, "dtype = %d", dtype);
  if (step < 1) return fail(GDP_E_INVALID_ARG, "step = %lld < 1", (long long)step);
  if (!(lr >= 0.f) || !(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f))
    return fail(GDP_E_INVALID_ARG, "bad Adam hyper-parameters");
  for (int i = 0; i < n_tensors; ++i) {
    const gdp_adam_tensor& t = tensors[i];
    if (t.n < 0) return fail(GDP_E_INVALID_ARG, "tensor %d: n < 0", i);
    if (t.n > 0 && (!t.param || !t.master || !t.grad || !t.m || !t.v))
      return fail(GDP_E_INVALID_ARG, "tensor %d has a NULL array", i);
  }
  int r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const float c1 = (float)(1.0 - pow((double)beta1, (double)step));
  const float c2 = (float)(1.0 - pow((double)beta2, (double)step));
  for (int i = 0; i < n_tensors; ++i) {
    const gdp_adam_tensor& t = tensors[i];
    if (t.n == 0) continue;
    if (dtype == GDP_BF16)
      GDP_LAUNCH(GDP_K_ADAM, tr::launch_adam<bf16>(t.master, static_cast<bf16*>(t.param), t.grad, t.m, t.v, t.n, lr,
                                                   beta1, beta2, eps, c1, c2, st));
    else
      GDP_LAUNCH(GDP_K_ADAM, tr::launch_adam<float>(t.master, static_cast<float*>(t.param), t.grad, t.m, t.v, t.n, lr,
                                                    beta1, beta2, eps, c1, c2, st));
  }
  return GDP_OK;
}

extern "C" int gdp_debug_train_tensor(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* placer,
                                      const void* store, size_t store_bytes, int32_t which, int32_t layer, void* out,
                                      size_t out_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_train(g, gnn, placer)) != GDP_OK) return r;
  TrainPlan tp;
  plan_train(g, gnn, placer, &tp);
  if ((r = check_store(store, store_bytes, tp.store_total)) != GDP_OK) return r;
  const size_t N = (size_t)g->n_nodes;
  size_t off = 0, bytes = 0;
  if (which == 0 && layer >= 0 && layer < placer->n_layers) {
    off = tp.H1[layer];
    bytes = N * (size_t)placer->d_ff * 4;
  } else if (which == 1 && layer >= 0 && layer < gnn->n_layers) {
    off = tp.h[layer + 1];
    bytes = N * (size_t)gnn->hidden * 4;
  } else if (which == 2 && layer >= 0 && layer < gnn->n_layers) {
    off = tp.arg[layer];
    bytes = N * (size_t)gnn->hidden * 4;
  } else {
    return fail(GDP_E_INVALID_ARG, "which = %d, layer = %d", which, layer);
  }
  if (!out || out_bytes < bytes) return fail(GDP_E_INVALID_ARG, "out is NULL or smaller than %zu bytes", bytes);
  const hipError_t e = hipMemcpyAsync(out, static_cast<const char*>(store) + off, bytes, hipMemcpyDeviceToDevice,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  return GDP_OK;
}

extern "C" int gdp_debug_uniforms(uint64_t seed, int32_t n, int32_t k, int32_t d, float* out, void* stream) {
  clear_error();
  if (n < 1 || k < 1 || d < 1 || d > GDP_MAX_DEVICES || !out) return fail(GDP_E_INVALID_ARG, "bad arguments");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = launch_debug_uniforms(seed, n, k, d, out, st);
  if (e != hipSuccess) return hip_fail(e, "launch_debug_uniforms");
  return GDP_OK;
}

extern "C" int gdp_debug_neighbors(const gdp_graph* g, const gdp_gnn* gnn, int32_t* s_ptr, int32_t* s_idx,
                                   int64_t capacity, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  int r;
  if ((r = check_graph(g)) != GDP_OK) return r;
  if ((r = check_gnn(g, gnn)) != GDP_OK) return r;
  EmbedPlan pl;
  plan_embed(g, gnn, &pl);
  if (!s_ptr || !s_idx) return fail(GDP_E_INVALID_ARG, "s_ptr or s_idx is NULL");
  if (capacity < pl.s_cap) return fail(GDP_E_INVALID_ARG, "capacity %lld < %lld", (long long)capacity, (long long)pl.s_cap);
  if ((r = check_ws(ws, ws_bytes, pl.c.total)) != GDP_OK) return r;
  if ((r = pending_hip_error()) != GDP_OK) return r;
  return prep_neighbors(g, gnn, pl, ws, s_ptr, s_idx, static_cast<hipStream_t>(stream));
}

extern "C" int gdp_set_place_streams(int32_t n) {
  clear_error();
  if (n != 1 && n != 2) return fail(GDP_E_INVALID_ARG, "place streams must be 1 or 2, got %d", (int)n);
  g_place_streams = n;
  return GDP_OK;
}

extern "C" int gdp_timer_begin(uint32_t mask) {
  clear_error();
  if (g_timer.mask != 0 || !g_timer.recs.empty()) return fail(GDP_E_INVALID_ARG, "timer already running");
  g_timer.mask = mask & ((1u << GDP_K_COUNT) - 1u);
  return GDP_OK;
}

extern "C" int gdp_timer_end(double* total_ms, int64_t* launches) {
  clear_error();
  int r = GDP_OK;
  if (total_ms)
    for (int k = 0; k < GDP_K_COUNT; ++k) total_ms[k] = 0.0;
  if (launches)
    for (int k = 0; k < GDP_K_COUNT; ++k) launches[k] = 0;
  for (const TimerRec& rec : g_timer.recs) {
    if (!rec.recorded) {
      g_timer.pool.push_back(rec.a);
      g_timer.pool.push_back(rec.b);
      continue;
    }
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(rec.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, rec.a, rec.b);
    if (e != hipSuccess && r == GDP_OK) r = hip_fail(e, "timer event");
    if (total_ms) total_ms[rec.kind] += ms;
    if (launches) launches[rec.kind] += 1;
    g_timer.pool.push_back(rec.a);
    g_timer.pool.push_back(rec.b);
  }
  g_timer.recs.clear();
  g_timer.mask = 0;
  return r;
}

extern "C" const char* gdp_kernel_kind_name(int32_t kind) {
  static const char* names[GDP_K_COUNT] = {
      "graph_prep", "nbr_sample",    "gemm_pool_sigmoid", "gather_max", "gemm_update_relu",
      "meanpool",   "film",          "pre_layer",         "seg_attention", "post_attn",
      "head_lse",   "gumbel_sample", "logp_reduce",       "mlp_placer", "ppo_grad",  "head_backward", "advantages",
      "evaluate", "train_forward", "backward", "adam", "log_prob", "gemm_update_pool"};
  if (kind < 0 || kind >= GDP_K_COUNT) return "";
  return names[kind];
}
