// Drives every host-side validation path of libgdp's argument checks and
// graph validator (csrc/host_plan.cpp) with the expected status codes.  Built
// with a plain C++ compiler and AddressSanitizer / UndefinedBehaviorSanitizer
// by tests/test_host_sanitize_cpu.py: no HIP, no device memory.  Device
// pointers in the descriptors are never dereferenced on the host, so fixed
// non-null addresses stand in for them.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "gdp.h"
#include "host_plan.h"

using namespace gdp;

static int g_failures = 0;
static int g_checks = 0;

#define EXPECT(expr, code)                                                                            \
  do {                                                                                                \
    const int _r = (expr);                                                                            \
    ++g_checks;                                                                                       \
    if (_r != (code)) {                                                                               \
      ++g_failures;                                                                                   \
      printf("FAIL %s:%d %s = %d, expected %d (%s)\n", __FILE__, __LINE__, #expr, _r, (int)(code),    \
             gdp_last_error());                                                                       \
    } else if ((code) != GDP_OK && gdp_last_error()[0] == '\0') {                                     \
      ++g_failures;                                                                                   \
      printf("FAIL %s:%d %s: no error text\n", __FILE__, __LINE__, #expr);                            \
    }                                                                                                 \
  } while (0)

static const void* fake(uintptr_t a) { return reinterpret_cast<const void*>(a); }

// ---- gdp_validate_graph_host --------------------------------------------------
struct Csr {
  std::vector<int32_t> gp, rp, ci;
};

static int validate(const Csr& c, uint32_t flags = GDP_TOPO_IDS) {
  return gdp_validate_graph_host(c.gp.data(), (int32_t)c.gp.size() - 1, c.rp.data(), (int32_t)c.rp.size() - 1,
                                 c.ci.empty() ? nullptr : c.ci.data(), (int64_t)c.ci.size(), flags);
}

static Csr chain4() {  // 0 -> 1 -> 2, 0 -> 2 | 3 (second graph, one node)
  Csr c;
  c.gp = {0, 3, 4};
  c.rp = {0, 2, 3, 3, 3};
  c.ci = {1, 2, 2};
  return c;
}

static void validator_paths() {
  Csr ok = chain4();
  EXPECT(validate(ok), GDP_OK);
  EXPECT(validate(ok, 0), GDP_OK);
  EXPECT(gdp_validate_graph_host(nullptr, 2, ok.rp.data(), 4, ok.ci.data(), 3, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 2, nullptr, 4, ok.ci.data(), 3, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 2, ok.rp.data(), 4, nullptr, 3, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 0, ok.rp.data(), 4, ok.ci.data(), 3, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 2, ok.rp.data(), 0, ok.ci.data(), 3, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 2, ok.rp.data(), 4, ok.ci.data(), -1, 0), GDP_E_INVALID_ARG);
  EXPECT(gdp_validate_graph_host(ok.gp.data(), 2, ok.rp.data(), 4, ok.ci.data(), (int64_t)INT32_MAX + 1, 0),
         GDP_E_INVALID_ARG);
  EXPECT(validate(ok, 0x80u), GDP_E_INVALID_ARG);
  {  // graph_ptr not from 0 to N
    Csr c = ok;
    c.gp[0] = 1;
    EXPECT(validate(c), GDP_E_BAD_GRAPH);
    c = ok;
    c.gp[2] = 3;
    EXPECT(gdp_validate_graph_host(c.gp.data(), 2, c.rp.data(), 4, c.ci.data(), 3, GDP_TOPO_IDS), GDP_E_BAD_GRAPH);
  }
  {  // empty graph in the batch
    Csr c = ok;
    c.gp = {0, 3, 3, 4};
    EXPECT(validate(c), GDP_E_BAD_GRAPH);
  }
  {  // row_ptr not 0..E, decreasing
    Csr c = ok;
    c.rp[0] = 1;
    EXPECT(validate(c), GDP_E_BAD_GRAPH);
    c = ok;
    c.rp[4] = 2;
    EXPECT(validate(c), GDP_E_BAD_GRAPH);
    c = ok;
    c.rp = {0, 2, 1, 3, 3};
    EXPECT(validate(c), GDP_E_BAD_GRAPH);
  }
  {  // column out of range (negative and >= N)
    Csr c = ok;
    c.ci[0] = -1;
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
    c.ci[0] = 4;
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
    c.ci[0] = 1 << 30;
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
  }
  {  // self-loop
    Csr c = ok;
    c.ci[0] = 0;
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
  }
  {  // edge across graphs
    Csr c = ok;
    c.ci[2] = 3;
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
  }
  {  // duplicate edge
    Csr c = ok;
    c.ci = {1, 1, 2};
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
  }
  {  // non-topological ids: 1 -> 0 is fine without the flag, rejected with it
    Csr c;
    c.gp = {0, 3};
    c.rp = {0, 0, 2, 2};
    c.ci = {0, 2};
    EXPECT(validate(c, 0), GDP_OK);
    EXPECT(validate(c, GDP_TOPO_IDS), GDP_E_BAD_GRAPH);
  }
  {  // a cycle (only reachable without the topological-id flag)
    Csr c;
    c.gp = {0, 3};
    c.rp = {0, 1, 2, 3};
    c.ci = {1, 2, 0};
    EXPECT(validate(c, 0), GDP_E_BAD_GRAPH);
    EXPECT(validate(c, GDP_TOPO_IDS), GDP_E_BAD_GRAPH);
  }
  {  // no edges at all
    Csr c;
    c.gp = {0, 5};
    c.rp = {0, 0, 0, 0, 0, 0};
    EXPECT(validate(c), GDP_OK);
  }
}

// ---- check_graph / check_gnn / check_placer / check_sample ---------------------
static int32_t g_gp[3] = {0, 10, 16};

static gdp_graph good_graph() {
  gdp_graph g;
  memset(&g, 0, sizeof(g));
  g.n_graphs = 2;
  g.graph_ptr_h = g_gp;
  g.n_nodes = 16;
  g.row_ptr = static_cast<const int32_t*>(fake(0x10000));
  g.col_idx = static_cast<const int32_t*>(fake(0x20000));
  g.n_edges = 20;
  g.x = fake(0x30000);
  g.feat_dim = 64;
  g.dtype = GDP_BF16;
  g.flags = GDP_TOPO_IDS;
  return g;
}

static void graph_paths() {
  gdp_graph g = good_graph();
  EXPECT(check_graph(&g), GDP_OK);
  EXPECT(check_graph(nullptr), GDP_E_INVALID_ARG);
  g = good_graph(); g.n_graphs = 0; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.n_graphs = GDP_MAX_GRAPHS + 1; EXPECT(check_graph(&g), GDP_E_UNSUPPORTED);
  g = good_graph(); g.graph_ptr_h = nullptr; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.n_nodes = 0; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  {
    int32_t gp[3] = {1, 10, 16};
    g = good_graph(); g.graph_ptr_h = gp; EXPECT(check_graph(&g), GDP_E_BAD_GRAPH);
    int32_t gp2[3] = {0, 10, 10};
    g = good_graph(); g.graph_ptr_h = gp2; EXPECT(check_graph(&g), GDP_E_BAD_GRAPH);
    int32_t gp3[3] = {0, 10, 15};
    g = good_graph(); g.graph_ptr_h = gp3; EXPECT(check_graph(&g), GDP_E_BAD_GRAPH);
  }
  g = good_graph(); g.n_edges = -1; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.n_edges = (int64_t)INT32_MAX + 1; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.row_ptr = nullptr; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.x = nullptr; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.col_idx = nullptr; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.col_idx = nullptr; g.n_edges = 0; EXPECT(check_graph(&g), GDP_OK);
  g = good_graph(); g.dtype = 7; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
  g = good_graph(); g.feat_dim = 48; EXPECT(check_graph(&g), GDP_E_UNSUPPORTED);
  g = good_graph(); g.feat_dim = 0; EXPECT(check_graph(&g), GDP_E_UNSUPPORTED);
  g = good_graph(); g.flags = 6; EXPECT(check_graph(&g), GDP_E_INVALID_ARG);
}

static gdp_gnn_layer g_gnn_layers[3];

static gdp_gnn good_gnn() {
  for (auto& L : g_gnn_layers) {
    L.w_pool = fake(0x40000);
    L.b_pool = fake(0x41000);
    L.w_self = fake(0x42000);
    L.w_neigh = fake(0x43000);
    L.b_upd = fake(0x44000);
  }
  gdp_gnn n;
  memset(&n, 0, sizeof(n));
  n.n_layers = 3;
  n.in_dim = 64;
  n.hidden = 128;
  n.fanout = 10;
  n.nbr_seed = 7;
  n.layers = g_gnn_layers;
  return n;
}

static void gnn_paths() {
  const gdp_graph g = good_graph();
  gdp_gnn n = good_gnn();
  EXPECT(check_gnn(&g, &n), GDP_OK);
  EXPECT(check_gnn(&g, nullptr), GDP_E_INVALID_ARG);
  n = good_gnn(); n.n_layers = 0; EXPECT(check_gnn(&g, &n), GDP_E_INVALID_ARG);
  n = good_gnn(); n.in_dim = 32; EXPECT(check_gnn(&g, &n), GDP_E_INVALID_ARG);
  for (int h : {0, 32, 96, 192, 512}) {
    n = good_gnn(); n.hidden = h; EXPECT(check_gnn(&g, &n), GDP_E_UNSUPPORTED);
  }
  for (int h : {64, 128, 256}) {
    n = good_gnn(); n.hidden = h; EXPECT(check_gnn(&g, &n), GDP_OK);
  }
  n = good_gnn(); n.fanout = 0; EXPECT(check_gnn(&g, &n), GDP_E_UNSUPPORTED);
  n = good_gnn(); n.fanout = GDP_MAX_FANOUT + 1; EXPECT(check_gnn(&g, &n), GDP_E_UNSUPPORTED);
  n = good_gnn(); n.layers = nullptr; EXPECT(check_gnn(&g, &n), GDP_E_INVALID_ARG);
  n = good_gnn(); g_gnn_layers[2].w_neigh = nullptr; EXPECT(check_gnn(&g, &n), GDP_E_INVALID_ARG);
  n = good_gnn(); g_gnn_layers[0].b_upd = nullptr; EXPECT(check_gnn(&g, &n), GDP_E_INVALID_ARG);
}

static gdp_placer_layer g_pl_layers[4];

static gdp_placer good_placer() {
  uintptr_t a = 0x100000;
  for (auto& L : g_pl_layers) {
    const void** f = reinterpret_cast<const void**>(&L);
    for (size_t i = 0; i < sizeof(L) / sizeof(void*); ++i) f[i] = fake(a += 0x1000);
  }
  gdp_placer p;
  memset(&p, 0, sizeof(p));
  p.n_layers = 4;
  p.d_model = 128;
  p.n_heads = 8;
  p.d_ff = 512;
  p.seg_len = 128;
  p.mem_len = 128;
  p.n_devices = 8;
  p.film = 1;
  p.attention = 1;
  p.layers = g_pl_layers;
  p.w_out = fake(0x200000);
  p.b_out = fake(0x201000);
  return p;
}

static void placer_paths() {
  const gdp_graph g = good_graph();
  gdp_placer p = good_placer();
  EXPECT(check_placer(&g, &p), GDP_OK);
  EXPECT(check_placer(&g, nullptr), GDP_E_INVALID_ARG);
  p = good_placer(); p.n_layers = 0; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.d_model = 96; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  p = good_placer(); p.attention = 2; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.n_heads = 0; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.n_heads = 3; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.n_heads = 16; p.d_model = 128; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);  // d_h 8
  p = good_placer(); p.n_heads = 1; p.d_model = 128; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);   // d_h 128
  for (int h : {2, 4, 8}) {
    p = good_placer(); p.n_heads = h; EXPECT(check_placer(&g, &p), GDP_OK);
  }
  p = good_placer(); p.seg_len = 0; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.mem_len = -1; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.mem_len = 0; EXPECT(check_placer(&g, &p), GDP_OK);
  p = good_placer(); p.attention = 0; p.n_layers = 4; EXPECT(check_placer(&g, &p), GDP_OK);
  {
    static gdp_placer_layer many[17];
    for (auto& L : many) L = g_pl_layers[0];
    p = good_placer(); p.attention = 0; p.n_layers = 17; p.layers = many;
    EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  }
  p = good_placer(); p.d_ff = 0; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  p = good_placer(); p.d_ff = 200; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  p = good_placer(); p.n_devices = 1; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  p = good_placer(); p.n_devices = GDP_MAX_DEVICES + 1; EXPECT(check_placer(&g, &p), GDP_E_UNSUPPORTED);
  p = good_placer(); p.film = 3; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.layers = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.w_out = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.b_out = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[1].w_2 = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[3].ln1_g = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.attention = 0; g_pl_layers[3].ln1_g = nullptr; g_pl_layers[3].w_qkv = nullptr;
  EXPECT(check_placer(&g, &p), GDP_OK);          // the ablation's placer does not use them
  p = good_placer(); g_pl_layers[0].film_wb = nullptr; EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); p.film = 0; g_pl_layers[0].film_wb = nullptr; EXPECT(check_placer(&g, &p), GDP_OK);
  // 16-byte alignment of the matrices and vectors the layer kernels stage by 16-byte loads
  p = good_placer(); g_pl_layers[2].w_1 = fake(0x300004); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[2].b_1 = fake(0x300008); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[2].w_2 = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[0].w_qkv = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[0].b_qkv = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[0].w_o = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_E_INVALID_ARG);
  p = good_placer(); g_pl_layers[0].b_o = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_OK);
  p = good_placer(); p.attention = 0; g_pl_layers[0].w_qkv = fake(0x300002); EXPECT(check_placer(&g, &p), GDP_OK);
}

static void sample_paths() {
  const gdp_graph g = good_graph();
  EXPECT(check_sample(&g, 8, 64), GDP_OK);
  EXPECT(check_sample(&g, 1, 64), GDP_E_UNSUPPORTED);
  EXPECT(check_sample(&g, GDP_MAX_DEVICES + 1, 64), GDP_E_UNSUPPORTED);
  EXPECT(check_sample(&g, 8, 0), GDP_E_INVALID_ARG);
  EXPECT(check_sample(&g, 8, 65536), GDP_E_UNSUPPORTED);
}

// ---- workspace plans: offsets aligned, regions disjoint and inside the total ---
static bool carve_ok(const Carve& c) {
  for (int i = 0; i < c.n; ++i) {
    if (c.off[i] % 256 != 0 || c.off[i] > c.total) return false;
    if (i > 0 && c.off[i] < c.off[i - 1]) return false;
  }
  return c.total % 256 == 0;
}

static void plan_paths() {
  gdp_graph g = good_graph();
  const gdp_gnn n = good_gnn();
  gdp_placer p = good_placer();
  EmbedPlan e;
  plan_embed(&g, &n, &e);
  ++g_checks;
  if (!carve_ok(e.c) || e.s_cap != 40) {
    ++g_failures;
    printf("FAIL embed plan (s_cap %lld)\n", (long long)e.s_cap);
  }
  PlacePlan pp;
  plan_place(&g, &p, &pp);
  ++g_checks;
  if (!carve_ok(pp.c) || pp.qblocks != 2) {
    ++g_failures;
    printf("FAIL place plan (qblocks %d)\n", pp.qblocks);
  }
  p.attention = 0;
  plan_place(&g, &p, &pp);
  ++g_checks;
  if (!carve_ok(pp.c) || pp.qkv != pp.y0) {
    ++g_failures;
    printf("FAIL place plan without attention\n");
  }
  SamplePlan sp;
  plan_sample(&g, 65535, &sp);
  ++g_checks;
  if (!carve_ok(sp.c) || sp.chunks != 2) {
    ++g_failures;
    printf("FAIL sample plan\n");
  }
  // the largest batch: 128 graphs, one block count per graph
  static int32_t gp[GDP_MAX_GRAPHS + 1];
  for (int i = 0; i <= GDP_MAX_GRAPHS; ++i) gp[i] = i * 1000;
  g.n_graphs = GDP_MAX_GRAPHS;
  g.graph_ptr_h = gp;
  g.n_nodes = GDP_MAX_GRAPHS * 1000;
  EXPECT(check_graph(&g), GDP_OK);
  int32_t blk[GDP_MAX_GRAPHS + 1];
  ++g_checks;
  if (prefix_blocks_rows(gp, GDP_MAX_GRAPHS, 256, blk) != GDP_MAX_GRAPHS * 4) {
    ++g_failures;
    printf("FAIL prefix_blocks_rows\n");
  }
  ++g_checks;
  if (prefix_blocks_attention(gp, GDP_MAX_GRAPHS, 300, 128, blk) != GDP_MAX_GRAPHS * (3 * 3 + 1)) {
    ++g_failures;
    printf("FAIL prefix_blocks_attention %d\n", blk[GDP_MAX_GRAPHS]);
  }
}

// segment_split: the segment start nearest the target, strictly inside
// (0, N), ties to the lower one, and the query blocks below it.
static void split_paths() {
  struct Case {
    std::vector<int32_t> gp;
    int seg, target, want, want_q;
  };
  const Case cases[] = {
      {{0, 52000}, 512, 32768, 32768, 256},
      {{0, 36000, 72000}, 512, 32768, 32768, 256},
      {{0, 32768, 65536}, 512, 32768, 32768, 256},
      // graph 0: 3 full segments of 3 query blocks and one of 100 rows; then 63 segments of graph 1
      {{0, 1000, 40000}, 300, 20000, 19900, 10 + 63 * 3},
      {{0, 1000, 40000}, 300, 450, 300, 3},          // 300 and 600 are equally near
      {{0, 400}, 512, 200, 0, 0},                    // one segment: no inner start
      {{0, 5, 10}, 512, 0, 5, 1},                    // a graph start is a segment start
  };
  for (const Case& c : cases) {
    int q = -1;
    const int b = segment_split(c.gp.data(), (int)c.gp.size() - 1, c.seg, 128, c.target, &q);
    ++g_checks;
    if (b != c.want || q != c.want_q) {
      ++g_failures;
      printf("FAIL segment_split target %d: %d (%d blocks), expected %d (%d)\n", c.target, b, q, c.want, c.want_q);
    }
  }
  // the place plan: a second QKV buffer only with two parts
  gdp_graph g = good_graph();
  gdp_placer p = good_placer();
  PlacePlan pp;
  plan_place(&g, &p, &pp);
  ++g_checks;
  if (pp.split != 0 || pp.qkv2 != pp.qkv) {
    ++g_failures;
    printf("FAIL place plan of a small graph: split %d\n", pp.split);
  }
  static int32_t big[2] = {0, 52000};
  g.graph_ptr_h = big;
  g.n_graphs = 1;
  g.n_nodes = 52000;
  g.n_edges = 0;
  p.seg_len = 512;
  p.mem_len = 512;
  plan_place(&g, &p, &pp);
  ++g_checks;
  if (!carve_ok(pp.c) || pp.split != 32768 || pp.split_qblocks != 256 || pp.qkv2 == pp.qkv) {
    ++g_failures;
    printf("FAIL place plan of 52000 rows: split %d, %d blocks\n", pp.split, pp.split_qblocks);
  }
}

// blocks_below: the per-graph row blocks of prefix_blocks_rows whose rows all
// lie below R, and those whose first row does, against counts over the blocks
// one by one; at most one block holds rows on both sides of R.
static void blocks_below_paths() {
  const std::vector<std::vector<int32_t>> graphs = {
      {0, 52000}, {0, 45000}, {0, 1000, 40000}, {0, 300, 301, 5000, 5001}, {0, 1}, {0, 256, 512}};
  for (const auto& gp : graphs) {
    const int G = (int)gp.size() - 1;
    for (int R : {0, 1, 255, 256, 257, 300, 1000, 1255, 1256, 19900, 32700, 32768, gp[G] - 1, gp[G]}) {
      if (R < 0 || R > gp[G]) continue;
      int want = 0;
      for (int g = 0; g < G; ++g)
        for (int lo = gp[g]; lo < gp[g + 1]; lo += 256)
          if (std::min(lo + 256, (int)gp[g + 1]) <= R) ++want;
      // the counted blocks are a prefix of prefix_blocks_rows's order
      int prefix = 0;
      bool in_prefix = true;
      for (int g = 0; g < G && in_prefix; ++g)
        for (int lo = gp[g]; lo < gp[g + 1]; lo += 256) {
          if (std::min(lo + 256, (int)gp[g + 1]) <= R) ++prefix;
          else { in_prefix = false; break; }
        }
      int started_want = 0;
      for (int g = 0; g < G; ++g)
        for (int lo = gp[g]; lo < gp[g + 1]; lo += 256)
          if (lo < R) ++started_want;
      int started = -1;
      const int got = blocks_below(gp.data(), G, 256, R, &started);
      ++g_checks;
      if (got != want || got != prefix || started != started_want || started - got > 1) {
        ++g_failures;
        printf("FAIL blocks_below R %d over %d graphs: %d (started %d), expected %d (prefix %d, started %d)\n", R, G,
               got, started, want, prefix, started_want);
      }
    }
  }
}

static void train_paths() {
  const gdp_graph g = good_graph();
  gdp_gnn n = good_gnn();
  gdp_placer p = good_placer();
  EXPECT(check_train(&g, &n, &p), GDP_OK);
  p = good_placer(); p.d_model = 256; EXPECT(check_train(&g, &n, &p), GDP_E_INVALID_ARG);   // != gnn.hidden
  {
    static gdp_gnn_layer many[kMaxTrainGnnLayers + 1];
    for (auto& L : many) L = g_gnn_layers[0];
    n = good_gnn(); n.n_layers = kMaxTrainGnnLayers + 1; n.layers = many;
    p = good_placer();
    EXPECT(check_train(&g, &n, &p), GDP_E_UNSUPPORTED);
  }
  {
    static gdp_placer_layer many[kMaxTrainPlacerLayers + 1];
    for (auto& L : many) L = g_pl_layers[0];
    n = good_gnn(); p = good_placer(); p.n_layers = kMaxTrainPlacerLayers + 1; p.layers = many;
    EXPECT(check_train(&g, &n, &p), GDP_E_UNSUPPORTED);
  }
  n = good_gnn();
  p = good_placer();
  TrainPlan tp;
  plan_train(&g, &n, &p, &tp);
  ++g_checks;
  if (tp.store_total == 0 || tp.ws_total == 0 || tp.store_total % 256 || tp.ws_total % 256 ||
      tp.X[0] != tp.h[n.n_layers] || tp.X[p.n_layers] + 16ull * 128 * 4 > tp.store_total || tp.gemm_partial_floats == 0) {
    ++g_failures;
    printf("FAIL train plan\n");
  }
  p.attention = 0;
  plan_train(&g, &n, &p, &tp);
  ++g_checks;
  if (tp.QKV[0] != 0 || tp.Z[0] != 0 || tp.store_total % 256) {
    ++g_failures;
    printf("FAIL train plan without attention\n");
  }
}

static void error_text() {
  clear_error();
  ++g_checks;
  if (gdp_last_error()[0] != '\0') ++g_failures;
  // a message longer than the buffer is truncated, never overflows
  std::vector<char> big(4000, 'x');
  big.back() = '\0';
  fail(GDP_E_INVALID_ARG, "%s", big.data());
  ++g_checks;
  if (strlen(gdp_last_error()) >= 4000) ++g_failures;
  ++g_checks;
  if (gdp_abi_version() != GDP_ABI_VERSION) ++g_failures;
}

int main() {
  validator_paths();
  graph_paths();
  gnn_paths();
  placer_paths();
  sample_paths();
  plan_paths();
  split_paths();
  blocks_below_paths();
  train_paths();
  error_text();
  printf("%d checks, %d failures\n", g_checks, g_failures);
  return g_failures == 0 ? 0 : 1;
}
