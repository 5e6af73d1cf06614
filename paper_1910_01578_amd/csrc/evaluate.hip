// Simulated run time of sampled placements: in-order list scheduling of each
// graph on D devices with transfer costs, and the per-device memory check that
// makes a placement invalid (Section 4.1's run time and invalid placements;
// Section 2's placement "with and without simulation").
//
// Every device runs its ops one at a time in node-id order.  For op v placed
// on device p:  ready = max over predecessors u of finish(u) + [p_u != p] *
// out_xfer[u];  start = max(ready, free[p]);  finish(v) = start + op_cost[v];
// free[p] = finish(v).  A graph's run time is its largest finish time.
//
// The recurrence is sequential in v for one placement, so the K placements of
// a graph run side by side: one wavefront per graph and block of 64 samples,
// lane = sample, every lane at the same node (uniform control flow, the graph
// structure in scalar registers).  Per-lane state lives in LDS: the last kRing
// finish times and devices (a ring indexed by node), and each device's free
// time.  Finish times of older nodes are read back from a global copy written
// as the wave goes.  Integer arithmetic only, so the result is exact; 32-bit
// times, with a wrap check that marks the graph's result -1.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

namespace {

constexpr int kRing = 256;        // nodes whose finish times stay in LDS
constexpr int kTile = 64;         // nodes per placement tile

// Per-graph, per-device memory sums: one work-group per (256-node chunk, sample).
__global__ __launch_bounds__(256) void k_device_mem(const int* __restrict__ placements, const int* __restrict__ op_mem,
                                                    int n, int D, int K, GraphTable ct,
                                                    unsigned long long* __restrict__ memsum) {
  __shared__ unsigned long long hist[GDP_MAX_DEVICES];
  const int c = blockIdx.x, k = blockIdx.y;
  const int g = graph_of_block(ct, c);
  const int v = ct.ptr[g] + (c - ct.blk[g]) * 256 + threadIdx.x;
  if (threadIdx.x < GDP_MAX_DEVICES) hist[threadIdx.x] = 0ull;
  __syncthreads();
  if (v < ct.ptr[g + 1]) {
    const int p = placements[(size_t)k * n + v];
    if (p >= 0 && p < D) atomicAdd(&hist[p], (unsigned long long)(uint32_t)op_mem[v]);
  }
  __syncthreads();
  if (threadIdx.x < D && hist[threadIdx.x] != 0ull)
    atomicAdd(&memsum[((size_t)g * K + k) * D + threadIdx.x], hist[threadIdx.x]);
}

// rec[e] = (u, out_xfer[u]) for the reverse edge e (u -> v, v's e-th predecessor).
__global__ void k_pred_records(const int* __restrict__ in_idx, const int* __restrict__ out_xfer, int64_t n_edges,
                               int2* __restrict__ rec) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n_edges; e += (int64_t)gridDim.x * blockDim.x) {
    const int u = in_idx[e];
    rec[e] = make_int2(u, out_xfer[u]);
  }
}

struct EvalArgs {
  const int* placements;   // [K, N]
  const int* op_cost;      // [N]
  const int* in_ptr;       // [N + 1] reverse CSR
  const int2* rec;         // [E] (u, out_xfer[u])
  const unsigned long long* memsum;   // [G, K, D]
  unsigned* far_fin;       // [KB, N, 64] finish times of every node, per sample lane
  unsigned char* far_dev;  // [KB, N, 64]
  int n, D, K, KB;
  double time_unit;
  int64_t* makespan;       // [G, K]
  unsigned char* valid;    // [G, K]
  float* run_time;         // [G, K] or null
};

struct CapTable {
  long long cap[GDP_MAX_GRAPHS];
};

__global__ __launch_bounds__(64) void k_list_schedule(EvalArgs a, GraphTable gt, CapTable caps) {
  __shared__ unsigned ring_fin[kRing][kWave];
  __shared__ unsigned char ring_dev[kRing][kWave];
  __shared__ unsigned dev_free[GDP_MAX_DEVICES][kWave];
  __shared__ unsigned char tile[kTile][kWave];
  const int lane = threadIdx.x;
  const int g = blockIdx.x / a.KB, kb = blockIdx.x % a.KB;
  const int k = kb * kWave + lane;
  const bool active = k < a.K;
  const int g0 = gt.ptr[g], g1 = gt.ptr[g + 1];
  for (int d = 0; d < a.D; ++d) dev_free[d][lane] = 0u;
  unsigned* far_fin = a.far_fin + (size_t)kb * a.n * kWave;
  unsigned char* far_dev = a.far_dev + (size_t)kb * a.n * kWave;
  const int* prow = a.placements + (size_t)(active ? k : 0) * a.n;
  unsigned mk = 0u;
  bool wrapped = false;
  for (int v0 = g0; v0 < g1; v0 += kTile) {
    // this lane's devices for the next kTile nodes (its own column of the tile)
    const int cnt = min(kTile, g1 - v0);
    for (int t = 0; t < cnt; ++t) {
      const int p = active ? prow[v0 + t] : 0;
      tile[t][lane] = (unsigned char)((p >= 0 && p < a.D) ? p : 0);
    }
    for (int t = 0; t < cnt; ++t) {
      const int v = v0 + t;
      const int p = tile[t][lane];
      unsigned ready = 0u;
      const int e0 = a.in_ptr[v], e1 = a.in_ptr[v + 1];
      for (int e = e0; e < e1; ++e) {
        const int2 r = a.rec[e];
        const int u = r.x;
        if (u < g0 || u >= v) continue;   // not a predecessor in this graph (invalid input)
        unsigned fu;
        int du;
        if (v - u <= kRing) {
          fu = ring_fin[u & (kRing - 1)][lane];
          du = ring_dev[u & (kRing - 1)][lane];
        } else {
          fu = far_fin[(size_t)u * kWave + lane];
          du = far_dev[(size_t)u * kWave + lane];
        }
        const unsigned arrive = fu + (du != p ? (unsigned)r.y : 0u);
        wrapped |= arrive < fu;
        ready = max(ready, arrive);
      }
      const unsigned start = max(ready, dev_free[p][lane]);
      const unsigned fin = start + (unsigned)a.op_cost[v];
      wrapped |= fin < start;
      dev_free[p][lane] = fin;
      ring_fin[v & (kRing - 1)][lane] = fin;
      ring_dev[v & (kRing - 1)][lane] = (unsigned char)p;
      far_fin[(size_t)v * kWave + lane] = fin;
      far_dev[(size_t)v * kWave + lane] = (unsigned char)p;
      mk = max(mk, fin);
    }
  }
  if (!active) return;
  bool ok = true;
  const unsigned long long* ms = a.memsum + ((size_t)g * a.K + k) * a.D;
  for (int d = 0; d < a.D; ++d) ok &= ms[d] <= (unsigned long long)caps.cap[g];
  const size_t o = (size_t)g * a.K + k;
  const int64_t m = wrapped ? (int64_t)-1 : (int64_t)mk;
  a.makespan[o] = m;
  a.valid[o] = ok ? 1 : 0;
  if (a.run_time) a.run_time[o] = (float)((double)m * a.time_unit);
}

}  // namespace

hipError_t launch_evaluate(const EvalLaunch& L, hipStream_t s) {
  const int KB = (L.K + kWave - 1) / kWave;
  // memory sums
  hipError_t e = launch_fill_i32(reinterpret_cast<int*>(L.memsum), 2 * (int64_t)L.gt->n * L.K * L.D, 0, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_device_mem, dim3(L.chunks, L.K), dim3(256), 0, s, L.placements, L.op_mem, L.n, L.D, L.K,
                     *L.chunk_table, reinterpret_cast<unsigned long long*>(L.memsum));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (L.n_edges > 0) {
    const int64_t blocks = std::min<int64_t>((L.n_edges + 255) / 256, 4096);
    hipLaunchKernelGGL(k_pred_records, dim3((unsigned)blocks), dim3(256), 0, s, L.in_idx, L.out_xfer, L.n_edges,
                       reinterpret_cast<int2*>(L.rec));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  EvalArgs a;
  a.placements = L.placements;
  a.op_cost = L.op_cost;
  a.in_ptr = L.in_ptr;
  a.rec = reinterpret_cast<const int2*>(L.rec);
  a.memsum = reinterpret_cast<const unsigned long long*>(L.memsum);
  a.far_fin = L.far_fin;
  a.far_dev = L.far_dev;
  a.n = L.n;
  a.D = L.D;
  a.K = L.K;
  a.KB = KB;
  a.time_unit = L.time_unit;
  a.makespan = L.makespan;
  a.valid = L.valid;
  a.run_time = L.run_time;
  CapTable caps;
  for (int i = 0; i < GDP_MAX_GRAPHS; ++i) caps.cap[i] = i < L.gt->n ? L.mem_cap[i] : 0;
  hipLaunchKernelGGL(k_list_schedule, dim3(L.gt->n * KB), dim3(kWave), 0, s, a, *L.gt, caps);
  return hipGetLastError();
}

}  // namespace gdp
