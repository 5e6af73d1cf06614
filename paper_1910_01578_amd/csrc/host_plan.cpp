// Host-only argument checks, workspace planning and the graph validator.
#include "host_plan.h"

#include <limits.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

namespace gdp {

namespace {
thread_local char g_err[512] = "";
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_err[0] = '\0'; }

size_t elem_size(int32_t dtype) { return dtype == GDP_BF16 ? 2 : 4; }

static bool supported_width(int h) { return h == 64 || h == 128 || h == 256; }

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_graph(const gdp_graph* g) {
  if (!g) return fail(GDP_E_INVALID_ARG, "graph is NULL");
  if (g->n_graphs < 1) return fail(GDP_E_INVALID_ARG, "n_graphs = %d < 1", g->n_graphs);
  if (g->n_graphs > GDP_MAX_GRAPHS)
    return fail(GDP_E_UNSUPPORTED, "n_graphs = %d exceeds GDP_MAX_GRAPHS = %d", g->n_graphs, GDP_MAX_GRAPHS);
  if (!g->graph_ptr_h) return fail(GDP_E_INVALID_ARG, "graph_ptr_h is NULL");
  if (g->n_nodes < 1) return fail(GDP_E_INVALID_ARG, "n_nodes = %d < 1", g->n_nodes);
  if (g->graph_ptr_h[0] != 0) return fail(GDP_E_BAD_GRAPH, "graph_ptr_h[0] = %d, expected 0", g->graph_ptr_h[0]);
  for (int i = 0; i < g->n_graphs; ++i)
    if (g->graph_ptr_h[i + 1] <= g->graph_ptr_h[i])
      return fail(GDP_E_BAD_GRAPH, "graph %d is empty or graph_ptr_h decreases", i);
  if (g->graph_ptr_h[g->n_graphs] != g->n_nodes)
    return fail(GDP_E_BAD_GRAPH, "graph_ptr_h[G] = %d != n_nodes = %d", g->graph_ptr_h[g->n_graphs], g->n_nodes);
  if (g->n_edges < 0 || g->n_edges > INT32_MAX)
    return fail(GDP_E_INVALID_ARG, "n_edges = %lld out of range", (long long)g->n_edges);
  if (!g->row_ptr || !g->x) return fail(GDP_E_INVALID_ARG, "row_ptr or x is NULL");
  if (g->n_edges > 0 && !g->col_idx) return fail(GDP_E_INVALID_ARG, "col_idx is NULL");
  if (g->dtype != GDP_F32 && g->dtype != GDP_BF16) return fail(GDP_E_INVALID_ARG, "dtype = %d", g->dtype);
  if (g->feat_dim < 32 || g->feat_dim % 32 != 0)
    return fail(GDP_E_UNSUPPORTED, "feat_dim = %d must be a positive multiple of 32", g->feat_dim);
  if (g->flags & ~GDP_TOPO_IDS) return fail(GDP_E_INVALID_ARG, "unknown flags 0x%x", g->flags);
  return GDP_OK;
}

int check_gnn(const gdp_graph* g, const gdp_gnn* n) {
  if (!n) return fail(GDP_E_INVALID_ARG, "gnn is NULL");
  if (n->n_layers < 1) return fail(GDP_E_INVALID_ARG, "gnn.n_layers = %d < 1", n->n_layers);
  if (n->in_dim != g->feat_dim)
    return fail(GDP_E_INVALID_ARG, "gnn.in_dim = %d != feat_dim = %d", n->in_dim, g->feat_dim);
  if (!supported_width(n->hidden)) return fail(GDP_E_UNSUPPORTED, "gnn.hidden = %d not in {64,128,256}", n->hidden);
  if (n->fanout < 1 || n->fanout > GDP_MAX_FANOUT)
    return fail(GDP_E_UNSUPPORTED, "fanout = %d outside 1..%d", n->fanout, GDP_MAX_FANOUT);
  if (!n->layers) return fail(GDP_E_INVALID_ARG, "gnn.layers is NULL");
  for (int l = 0; l < n->n_layers; ++l) {
    const gdp_gnn_layer& L = n->layers[l];
    if (!L.w_pool || !L.b_pool || !L.w_self || !L.w_neigh || !L.b_upd)
      return fail(GDP_E_INVALID_ARG, "gnn layer %d has a NULL weight", l);
  }
  return GDP_OK;
}

int check_placer(const gdp_graph* g, const gdp_placer* p) {
  if (!p) return fail(GDP_E_INVALID_ARG, "placer is NULL");
  if (p->n_layers < 1) return fail(GDP_E_INVALID_ARG, "placer.n_layers = %d < 1", p->n_layers);
  if (!supported_width(p->d_model)) return fail(GDP_E_UNSUPPORTED, "d_model = %d not in {64,128,256}", p->d_model);
  if (p->attention != 0 && p->attention != 1)
    return fail(GDP_E_INVALID_ARG, "attention = %d must be 0 or 1", p->attention);
  if (p->attention) {
    if (p->n_heads < 1 || p->d_model % p->n_heads != 0)
      return fail(GDP_E_INVALID_ARG, "d_model = %d not divisible by n_heads = %d", p->d_model, p->n_heads);
    const int dh = p->d_model / p->n_heads;
    if (dh != 16 && dh != 32 && dh != 64) return fail(GDP_E_UNSUPPORTED, "head dim %d not in {16,32,64}", dh);
    if (p->seg_len < 1) return fail(GDP_E_INVALID_ARG, "seg_len = %d < 1", p->seg_len);
    if (p->mem_len < 0) return fail(GDP_E_INVALID_ARG, "mem_len = %d < 0", p->mem_len);
  } else if (p->n_layers > 16) {
    return fail(GDP_E_UNSUPPORTED, "n_layers = %d > 16 without attention", p->n_layers);
  }
  if (p->d_ff < 128 || p->d_ff % 128 != 0)
    return fail(GDP_E_UNSUPPORTED, "d_ff = %d must be a positive multiple of 128", p->d_ff);
  if (p->n_devices < 2 || p->n_devices > GDP_MAX_DEVICES)
    return fail(GDP_E_UNSUPPORTED, "n_devices = %d outside 2..%d", p->n_devices, GDP_MAX_DEVICES);
  if (p->film != 0 && p->film != 1) return fail(GDP_E_INVALID_ARG, "film = %d must be 0 or 1", p->film);
  if (!p->layers || !p->w_out || !p->b_out) return fail(GDP_E_INVALID_ARG, "placer weights are NULL");
  for (int l = 0; l < p->n_layers; ++l) {
    const gdp_placer_layer& L = p->layers[l];
    if (!L.w_1 || !L.b_1 || !L.w_2 || !L.b_2 || !L.ln2_g || !L.ln2_b ||
        (p->attention && (!L.w_qkv || !L.b_qkv || !L.w_o || !L.b_o || !L.ln1_g || !L.ln1_b)))
      return fail(GDP_E_INVALID_ARG, "placer layer %d has a NULL weight", l);
    if (p->film && (!L.film_wg || !L.film_bg || !L.film_wb || !L.film_bb))
      return fail(GDP_E_INVALID_ARG, "placer layer %d has a NULL FiLM weight", l);
    // The layer kernels stage these matrices and vectors by 16-byte loads.
    if (!aligned16(L.w_1) || !aligned16(L.b_1) || !aligned16(L.w_2) ||
        (p->attention && (!aligned16(L.w_qkv) || !aligned16(L.b_qkv) || !aligned16(L.w_o))))
      return fail(GDP_E_INVALID_ARG, "placer layer %d: w_qkv, b_qkv, w_o, w_1, b_1 and w_2 must be 16-byte aligned", l);
  }
  (void)g;
  return GDP_OK;
}

int check_sample(const gdp_graph* g, int32_t n_devices, int32_t k_samples) {
  (void)g;
  if (n_devices < 2 || n_devices > GDP_MAX_DEVICES)
    return fail(GDP_E_UNSUPPORTED, "n_devices = %d outside 2..%d", n_devices, GDP_MAX_DEVICES);
  if (k_samples < 1) return fail(GDP_E_INVALID_ARG, "k_samples = %d < 1", k_samples);
  if (k_samples > 65535) return fail(GDP_E_UNSUPPORTED, "k_samples = %d > 65535", k_samples);
  return GDP_OK;
}

void carve_init(Carve* c) {
  c->total = 0;
  c->n = 0;
}

size_t carve_add(Carve* c, size_t bytes) {
  const size_t off = c->total;
  c->total += (bytes + 255) & ~size_t(255);
  if (c->n < 24) c->off[c->n++] = off;
  return off;
}

int prefix_blocks_rows(const int32_t* gp, int G, int rows, int32_t* blk) {
  blk[0] = 0;
  for (int g = 0; g < G; ++g) blk[g + 1] = blk[g] + (gp[g + 1] - gp[g] + rows - 1) / rows;
  return blk[G];
}

int blocks_below(const int32_t* gp, int G, int rows, int R, int* started) {
  int n = 0, s = 0;
  for (int g = 0; g < G; ++g) {
    if (gp[g + 1] <= R) {
      n += (gp[g + 1] - gp[g] + rows - 1) / rows;
      s = n;
    } else {
      if (gp[g] < R) {
        n += (R - gp[g]) / rows;                // block b ends at gp[g] + (b + 1) rows <= R
        s = n + ((R - gp[g]) % rows != 0);      // a block starts below R and ends above it
      } else {
        s = n;
      }
      break;
    }
  }
  if (started) *started = s;
  return n;
}

int prefix_blocks_attention(const int32_t* gp, int G, int seg_len, int bq, int32_t* blk) {
  const int qbs = (seg_len + bq - 1) / bq;
  blk[0] = 0;
  for (int g = 0; g < G; ++g) {
    const int n = gp[g + 1] - gp[g];
    const int nseg = (n + seg_len - 1) / seg_len;
    const int last = n - (nseg - 1) * seg_len;
    blk[g + 1] = blk[g] + (nseg - 1) * qbs + (last + bq - 1) / bq;
  }
  return blk[G];
}

int segment_split(const int32_t* gp, int G, int seg_len, int bq, int target, int* qblocks_below) {
  const int qbs = (seg_len + bq - 1) / bq;
  const int N = gp[G];
  int best = 0, best_q = 0;
  long best_dist = -1;
  int qb = 0;   // query blocks of the graphs before g
  for (int g = 0; g < G; ++g) {
    const int n = gp[g + 1] - gp[g];
    const int nseg = (n + seg_len - 1) / seg_len;
    for (int k = 0; k < nseg; ++k) {
      const int b = gp[g] + k * seg_len;
      if (b <= 0 || b >= N) continue;
      const long dist = b > target ? (long)b - target : (long)target - b;
      if (best_dist < 0 || dist < best_dist) {
        best = b;
        best_q = qb + k * qbs;
        best_dist = dist;
      }
    }
    if (nseg > 0) qb += (nseg - 1) * qbs + (n - (nseg - 1) * seg_len + bq - 1) / bq;
  }
  *qblocks_below = best_q;
  return best;
}

void plan_embed(const gdp_graph* g, const gdp_gnn* gnn, EmbedPlan* p) {
  const size_t N = (size_t)g->n_nodes, E = (size_t)g->n_edges, H = (size_t)gnn->hidden;
  const size_t es = elem_size(g->dtype);
  int32_t blk[GDP_MAX_GRAPHS + 1];
  p->pool_chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kPoolRows, blk);
  const size_t cap_a = 2 * E, cap_b = N * (size_t)gnn->fanout;
  p->s_cap = (int64_t)(cap_a < cap_b ? cap_a : cap_b);
  carve_init(&p->c);
  p->counters = carve_add(&p->c, (2 * N + 1) * 4);
  p->scan_tmp = carve_add(&p->c, 2 * ((N + 1023) / 1024) * 4);
  p->heavy = carve_add(&p->c, N * 4);
  p->in_ptr = carve_add(&p->c, (N + 1) * 4);
  p->in_idx = carve_add(&p->c, (E > 0 ? E : 1) * 4);
  p->s_ptr = carve_add(&p->c, (N + 1) * 4);
  p->s_idx = carve_add(&p->c, (p->s_cap > 0 ? (size_t)p->s_cap : 1) * 4);
  p->P = carve_add(&p->c, N * H * es);
  p->A = carve_add(&p->c, N * H * es);
  p->h0 = carve_add(&p->c, gnn->n_layers > 1 ? N * H * es : 0);
  p->h1 = carve_add(&p->c, gnn->n_layers > 2 ? N * H * es : 0);
  p->pool = carve_add(&p->c, (size_t)p->pool_chunks * H * 4);
}

void plan_place(const gdp_graph* g, const gdp_placer* pl, PlacePlan* p) {
  const size_t N = (size_t)g->n_nodes, d = (size_t)pl->d_model, es = elem_size(g->dtype);
  int32_t blk[GDP_MAX_GRAPHS + 1];
  carve_init(&p->c);
  p->film = carve_add(&p->c, (size_t)pl->n_layers * g->n_graphs * d * 2 * 4);
  p->y0 = carve_add(&p->c, N * d * 4);      // residual stream: fp32
  p->head_partial = carve_add(&p->c, ((N + kHeadBwdRows - 1) / kHeadBwdRows) * (size_t)pl->n_devices * (d + 1) * 4);
  p->split = p->split_qblocks = 0;
  if (!pl->attention) {                     // only the head's input, when the head runs on its own
    p->qblocks = 0;
    p->y1 = p->qkv = p->qkv2 = p->o = p->y0;
    return;
  }
  p->qblocks = prefix_blocks_attention(g->graph_ptr_h, g->n_graphs, pl->seg_len, kAttnQ, blk);
  p->y1 = carve_add(&p->c, N * d * 4);
  p->qkv = carve_add(&p->c, N * 3 * d * es);
  p->o = carve_add(&p->c, N * d * es);
  // Two parts only where part B still fills a round of its own (and a
  // layer is long enough that the overlap outweighs the extra launches).
  if (N >= (size_t)kSplitRows + kSplitRows / 4)
    p->split = segment_split(g->graph_ptr_h, g->n_graphs, pl->seg_len, kAttnQ, kSplitRows, &p->split_qblocks);
  p->qkv2 = p->split > 0 ? carve_add(&p->c, N * 3 * d * es) : p->qkv;
}

void plan_evaluate(const gdp_graph* g, int32_t n_devices, int32_t k, EvalPlan* p) {
  const size_t N = (size_t)g->n_nodes, E = (size_t)g->n_edges;
  const size_t kb = ((size_t)k + 63) / 64;
  int32_t blk[GDP_MAX_GRAPHS + 1];
  p->chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kEvalRows, blk);
  carve_init(&p->c);
  p->counters = carve_add(&p->c, (2 * N + 1) * 4);
  p->scan_tmp = carve_add(&p->c, 2 * ((N + 1023) / 1024) * 4);
  p->in_ptr = carve_add(&p->c, (N + 1) * 4);
  p->s_ptr = carve_add(&p->c, (N + 1) * 4);
  p->in_idx = carve_add(&p->c, (E > 0 ? E : 1) * 4);
  p->rec = carve_add(&p->c, (E > 0 ? E : 1) * 8);
  p->memsum = carve_add(&p->c, (size_t)g->n_graphs * (size_t)k * (size_t)n_devices * 8);
  p->far = carve_add(&p->c, kb * N * 64 * 4);
}

int check_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* p) {
  int r;
  if ((r = check_gnn(g, gnn)) != GDP_OK) return r;
  if ((r = check_placer(g, p)) != GDP_OK) return r;
  if (gnn->n_layers > kMaxTrainGnnLayers)
    return fail(GDP_E_UNSUPPORTED, "training supports at most %d GNN layers (got %d)", kMaxTrainGnnLayers, gnn->n_layers);
  if (p->n_layers > kMaxTrainPlacerLayers)
    return fail(GDP_E_UNSUPPORTED, "training supports at most %d placer layers (got %d)", kMaxTrainPlacerLayers,
                p->n_layers);
  if (p->d_model != gnn->hidden)
    return fail(GDP_E_INVALID_ARG, "d_model = %d != gnn.hidden = %d", p->d_model, gnn->hidden);
  return GDP_OK;
}

void plan_train(const gdp_graph* g, const gdp_gnn* gnn, const gdp_placer* pl, TrainPlan* t) {
  const size_t N = (size_t)g->n_nodes, E = (size_t)g->n_edges, H = (size_t)gnn->hidden, d = (size_t)pl->d_model;
  const size_t G = (size_t)g->n_graphs, dff = (size_t)pl->d_ff, F = (size_t)g->feat_dim;
  const size_t heads = pl->attention ? (size_t)pl->n_heads : 1;
  int32_t blk[GDP_MAX_GRAPHS + 1];
  t->chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, 256, blk);
  const size_t cap_a = 2 * E, cap_b = N * (size_t)gnn->fanout;
  t->s_cap = (int64_t)(cap_a < cap_b ? cap_a : cap_b);
  Carve c;
  carve_init(&c);
  t->s_ptr = carve_add(&c, (N + 1) * 4);
  t->s_idx = carve_add(&c, (t->s_cap > 0 ? (size_t)t->s_cap : 1) * 4);
  t->in_ptr = carve_add(&c, (N + 1) * 4);
  t->in_idx = carve_add(&c, (E > 0 ? E : 1) * 4);
  t->x0 = carve_add(&c, G * H * 4);
  t->film = carve_add(&c, (size_t)pl->n_layers * 2 * G * d * 4);
  for (int l = 0; l < gnn->n_layers; ++l) {
    t->P[l] = carve_add(&c, N * H * 4);
    t->A[l] = carve_add(&c, N * H * 4);
    t->arg[l] = carve_add(&c, N * H * 4);
    t->h[l + 1] = carve_add(&c, N * H * 4);
  }
  t->h[0] = 0;
  t->X[0] = t->h[gnn->n_layers];
  for (int l = 0; l < pl->n_layers; ++l) {
    t->Y[l] = carve_add(&c, N * d * 4);
    t->QKV[l] = pl->attention ? carve_add(&c, N * 3 * d * 4) : 0;
    t->O[l] = pl->attention ? carve_add(&c, N * d * 4) : 0;
    t->lse_att[l] = pl->attention ? carve_add(&c, N * heads * 4) : 0;
    t->R1[l] = pl->attention ? carve_add(&c, N * d * 4) : 0;
    t->Z[l] = pl->attention ? carve_add(&c, N * d * 4) : 0;
    t->H1[l] = carve_add(&c, N * dff * 4);
    t->R2[l] = carve_add(&c, N * d * 4);
    t->X[l + 1] = carve_add(&c, N * d * 4);
  }
  t->store_total = c.total;

  const size_t wide = d > H ? d : H;
  const size_t fin = F > wide ? F : wide;
  carve_init(&c);
  t->counters = carve_add(&c, (2 * N + 1) * 4);
  t->scan_tmp = carve_add(&c, 2 * ((N + 1023) / 1024) * 4);
  t->heavy = carve_add(&c, N * 4);
  t->dX = carve_add(&c, N * d * 4);
  t->dY = carve_add(&c, N * d * 4);
  t->dR = carve_add(&c, N * d * 4);
  t->dZ = carve_add(&c, N * d * 4);
  t->xg = carve_add(&c, N * wide * 4);
  t->dH = carve_add(&c, N * dff * 4);
  t->dqkv = carve_add(&c, N * 3 * d * 4);
  t->dkvm = carve_add(&c, N * 2 * d * 4);
  t->Dq = carve_add(&c, N * heads * 4);
  t->head_partial = carve_add(&c, ((N + kHeadBwdRows - 1) / kHeadBwdRows) * (size_t)pl->n_devices * (d + 1) * 4);
  t->dfilm = carve_add(&c, (size_t)pl->n_layers * 2 * G * d * 4);
  t->dx0 = carve_add(&c, G * H * 4);
  t->dh = carve_add(&c, N * fin * 4);
  t->dA = carve_add(&c, N * H * 4);
  t->dP = carve_add(&c, N * H * 4);
  t->dU = carve_add(&c, N * H * 4);
  const size_t colw = 3 * d > dff ? 3 * d : dff;
  t->colpart = carve_add(&c, ((size_t)t->chunks + G) * (colw > fin ? colw : fin) * 4);
  const size_t big = (dff * d > 3 * d * d ? dff * d : 3 * d * d);
  const size_t splits = (N + 1023) / 1024;   // weight gradients: k = N split into pieces of 1,024 rows
  t->gemm_partial_floats = (splits > 1 ? splits : 1) * (big > H * fin ? big : H * fin);
  t->gemm_partial = carve_add(&c, t->gemm_partial_floats * 4);
  t->ws_total = c.total;
}

void plan_sample(const gdp_graph* g, int32_t k, SamplePlan* p) {
  int32_t blk[GDP_MAX_GRAPHS + 1];
  p->chunks = prefix_blocks_rows(g->graph_ptr_h, g->n_graphs, kSampleRows, blk);
  carve_init(&p->c);
  p->partial = carve_add(&p->c, (size_t)k * p->chunks * 4);
  p->coef = carve_add(&p->c, (size_t)g->n_graphs * (k + 1) * 4);
}

}  // namespace gdp

using namespace gdp;

extern "C" const char* gdp_last_error(void) { return g_err; }

extern "C" int gdp_abi_version(void) { return GDP_ABI_VERSION; }

extern "C" int gdp_validate_graph_host(const int32_t* graph_ptr, int32_t G, const int32_t* row_ptr,
                                       int32_t N, const int32_t* col_idx, int64_t E, uint32_t flags) {
  clear_error();
  if (!graph_ptr || !row_ptr || (E > 0 && !col_idx)) return fail(GDP_E_INVALID_ARG, "NULL array");
  if (G < 1 || N < 1 || E < 0 || E > INT32_MAX) return fail(GDP_E_INVALID_ARG, "bad sizes G=%d N=%d E=%lld", G, N, (long long)E);
  if (flags & ~GDP_TOPO_IDS) return fail(GDP_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (graph_ptr[0] != 0 || graph_ptr[G] != N) return fail(GDP_E_BAD_GRAPH, "graph_ptr must run from 0 to N");
  for (int g = 0; g < G; ++g)
    if (graph_ptr[g + 1] <= graph_ptr[g]) return fail(GDP_E_BAD_GRAPH, "graph %d is empty or graph_ptr decreases", g);
  if (row_ptr[0] != 0 || row_ptr[N] != E) return fail(GDP_E_BAD_GRAPH, "row_ptr must run from 0 to E");
  for (int v = 0; v < N; ++v)
    if (row_ptr[v + 1] < row_ptr[v]) return fail(GDP_E_BAD_GRAPH, "row_ptr decreases at node %d", v);
  std::vector<int32_t> indeg((size_t)N, 0);
  std::vector<int32_t> mark((size_t)N, -1);
  int g = 0;
  for (int u = 0; u < N; ++u) {
    while (u >= graph_ptr[g + 1]) ++g;
    for (int32_t e = row_ptr[u]; e < row_ptr[u + 1]; ++e) {
      const int32_t v = col_idx[e];
      if (v < 0 || v >= N) return fail(GDP_E_BAD_GRAPH, "edge %d: col_idx %d out of range", e, v);
      if (v == u) return fail(GDP_E_BAD_GRAPH, "self-loop at node %d", u);
      if (v < graph_ptr[g] || v >= graph_ptr[g + 1]) return fail(GDP_E_BAD_GRAPH, "edge %d -> %d crosses graphs", u, v);
      if ((flags & GDP_TOPO_IDS) && v < u) return fail(GDP_E_BAD_GRAPH, "edge %d -> %d breaks topological ids", u, v);
      if (mark[(size_t)v] == u) return fail(GDP_E_BAD_GRAPH, "duplicate edge %d -> %d", u, v);
      mark[(size_t)v] = u;
      ++indeg[(size_t)v];
    }
  }
  // Kahn's algorithm: every node must be removable.
  std::vector<int32_t> queue;
  queue.reserve((size_t)N);
  for (int v = 0; v < N; ++v)
    if (indeg[(size_t)v] == 0) queue.push_back(v);
  size_t head = 0;
  while (head < queue.size()) {
    const int32_t u = queue[head++];
    for (int32_t e = row_ptr[u]; e < row_ptr[u + 1]; ++e)
      if (--indeg[(size_t)col_idx[e]] == 0) queue.push_back(col_idx[e]);
  }
  if (queue.size() != (size_t)N) return fail(GDP_E_BAD_GRAPH, "graph has a cycle");
  return GDP_OK;
}
