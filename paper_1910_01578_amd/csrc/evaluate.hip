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
// as the wave goes.  Integer arithmetic only, so the result is exact; times
// below 2^26 units (they share a word with the device), with a check that
// marks the graph's result -1 once a finish time reaches 2^26 or wraps.
#include "device_common.h"
#include "kernels.h"
#include "lds_dma.h"

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
  unsigned* far;           // [KB, N, 64] packed (finish, device) of every node, per sample lane
  int n, D, K, KB;
  double time_unit;
  int64_t* makespan;       // [G, K]
  unsigned char* valid;    // [G, K]
  float* run_time;         // [G, K] or null
};

struct CapTable {
  long long cap[GDP_MAX_GRAPHS];
};

// A finish time and the device it ran on share one word: time << 6 | device.
constexpr unsigned kTimeLimit = 1u << 26;
__device__ __forceinline__ unsigned pack(unsigned t, int dev) { return (t << 6) | (unsigned)dev; }

// One direct global -> LDS load of a dword per lane: lane l reads base + voff
// and writes it to LDS at lds + 4 l.  The compiler keeps no count of these
// loads; the tile boundary waits for all of them (s_waitcnt vmcnt(0)).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma4(dma::gptr_t base, uint32_t voff, const void* lds) {
  const uint32_t la = (uint32_t)(uintptr_t)lds;
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(base), "s"(__builtin_amdgcn_readfirstlane(la)) : "memory", "m0");
}
__device__ __forceinline__ void wait_all_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// A global load that waits for itself (and everything before it): the slow
// path of a far predecessor that found no prefetch slot.  Written as inline
// assembly so that the compiler cannot merge it with the LDS reads of the
// common path into one generic (flat) load.
__device__ __forceinline__ unsigned load_wait(const unsigned* p) {
  unsigned w;
  asm volatile("global_load_dword %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=v"(w) : "v"(p) : "memory");
  return w;
}
#pragma clang diagnostic pop

constexpr int kRecSets = 4;                   // records per lane and tile: 4 * 64 per tile
constexpr int kFarCap = 128;                  // far predecessors prefetched per tile

// Lane i's view of node v0 + i of a tile: its predecessor range and cost.
struct Hdr {
  int ip0, ip1, cost;
};
// Lane i, set j: record rb + i + 64 j of a tile (rb its first record) and,
// for a far predecessor, its prefetch slot (-1: none or beyond kFarCap).
struct Recs {
  int u[kRecSets], x[kRecSets], slot[kRecSets];
};

__device__ __forceinline__ Hdr load_hdr(const EvalArgs& a, int v0, int g1) {
  const int v = v0 + (int)threadIdx.x;
  Hdr h = {0, 0, 0};
  if (v < g1) {
    h.ip0 = a.in_ptr[v];
    h.ip1 = a.in_ptr[v + 1];
    h.cost = a.op_cost[v];
  }
  return h;
}

__device__ __forceinline__ Recs load_recs(const EvalArgs& a, const Hdr& h, int v0, int g1) {
  Recs r;
  const int cnt_nodes = min(kTile, g1 - v0);
  const int rb = __builtin_amdgcn_readlane(h.ip0, 0);
  const int re = cnt_nodes > 0 ? __builtin_amdgcn_readlane(h.ip1, cnt_nodes - 1) : rb;
#pragma unroll
  for (int j = 0; j < kRecSets; ++j) {
    const int e = rb + (int)threadIdx.x + kWave * j;
    r.u[j] = -1;
    r.x[j] = 0;
    r.slot[j] = -1;
    if (e < re) {
      const int2 q = a.rec[e];
      r.u[j] = q.x;
      r.x[j] = q.y;
    }
  }
  return r;
}

__global__ __launch_bounds__(64) void k_list_schedule(EvalArgs a, GraphTable gt, CapTable caps) {
  // One LDS array holds the ring of packed (finish, device) words of nodes
  // v - kRing .. v - 1 ([kRing][64]) and the two prefetch buffers of far
  // predecessors ([2][kFarCap][64]), so a predecessor read is one LDS load from
  // a computed offset.
  __shared__ unsigned words[(kRing + 2 * kFarCap) * kWave];
  unsigned (*ring)[kWave] = reinterpret_cast<unsigned (*)[kWave]>(&words[0]);
  unsigned (*farbuf)[kFarCap][kWave] = reinterpret_cast<unsigned (*)[kFarCap][kWave]>(&words[kRing * kWave]);
  __shared__ unsigned ptile[kTile / 4][kWave];            // devices of the tile's nodes, 4 per word
  __shared__ unsigned dev_free[GDP_MAX_DEVICES][kWave];
  const int lane = threadIdx.x;
  const int g = blockIdx.x / a.KB, kb = blockIdx.x % a.KB;
  const int k = kb * kWave + lane;
  const bool active = k < a.K;
  const int g0 = gt.ptr[g], g1 = gt.ptr[g + 1];
  for (int d = 0; d < a.D; ++d) dev_free[d][lane] = 0u;
  unsigned* far = a.far + (size_t)kb * a.n * kWave;
  const dma::gptr_t far_base = dma::uniform_base(far);
  const int* prow = a.placements + (size_t)(active ? k : 0) * a.n;
  unsigned mk = 0u;
  bool wrapped = false;

  // pipeline: headers three tiles ahead, records two, far predecessors and
  // devices one
  Hdr h0 = load_hdr(a, g0, g1), h1 = load_hdr(a, g0 + kTile, g1), h2 = load_hdr(a, g0 + 2 * kTile, g1);
  Recs r0 = load_recs(a, h0, g0, g1), r1 = load_recs(a, h1, g0 + kTile, g1);
  int pl[kTile];
#pragma unroll
  for (int i = 0; i < kTile; ++i) pl[i] = (g0 + i < g1) ? prow[g0 + i] : 0;

  for (int v0 = g0, tl = 0; v0 < g1; v0 += kTile, ++tl) {
    wait_all_memory();
    // this tile's devices into LDS, 4 per word
#pragma unroll
    for (int q = 0; q < kTile / 4; ++q) {
      unsigned w = 0u;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int p = active ? pl[4 * q + b] : 0;
        w |= (unsigned)((p >= 0 && p < a.D) ? p : 0) << (8 * b);
      }
      ptile[q][lane] = w;
    }
    // far predecessors of the next tile (final since several tiles): slots and loads
    const int v1 = v0 + kTile;
    if (v1 < g1) {
      const int limit = v1 + kTile - kRing;      // u below this is read from the prefetch
      int base = 0;
#pragma unroll
      for (int j = 0; j < kRecSets; ++j) {
        const bool f = r1.u[j] >= g0 && r1.u[j] < limit;
        const uint64_t m = __ballot(f);
        const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
        const int s = base + rank;
        r1.slot[j] = f && s < kFarCap ? s : -1;
        base += __popcll(m);
        uint64_t mm = m;
        while (mm) {
          const int ln = __builtin_ctzll(mm);
          mm &= mm - 1;
          const int sl = __builtin_amdgcn_readlane(r1.slot[j], ln);
          if (sl < 0) break;
          const int u = __builtin_amdgcn_readlane(r1.u[j], ln);
          dma4(far_base, (uint32_t)(((size_t)u * kWave + lane) * 4u), &farbuf[(tl + 1) & 1][sl][0]);
        }
      }
    }
    // records two tiles ahead, headers three tiles ahead, devices of the next tile
    const Recs r2 = load_recs(a, h2, v0 + 2 * kTile, g1);
    const Hdr h3 = load_hdr(a, v0 + 3 * kTile, g1);
#pragma unroll
    for (int i = 0; i < kTile; ++i) pl[i] = (v1 + i < g1) ? prow[v1 + i] : 0;

    const int cnt = min(kTile, g1 - v0);
    const int rb = __builtin_amdgcn_readlane(h0.ip0, 0);
    const int limit = v0 + kTile - kRing;
    const int fb_off = (kRing + (tl & 1) * kFarCap) * kWave;
    for (int t = 0; t < cnt; ++t) {
      const int v = v0 + t;
      const int p = (ptile[t >> 2][lane] >> (8 * (t & 3))) & 0xff;
      const int e0 = __builtin_amdgcn_readlane(h0.ip0, t), e1 = __builtin_amdgcn_readlane(h0.ip1, t);
      const int c = __builtin_amdgcn_readlane(h0.cost, t);
      unsigned ready = 0u;
      for (int e = e0; e < e1; ++e) {
        const int r = e - rb;
        int u, x, slot;
        if (r < kRecSets * kWave) {
          const int j = r >> 6, ln = r & 63;
          const int uu = j == 0 ? r0.u[0] : j == 1 ? r0.u[1] : j == 2 ? r0.u[2] : r0.u[3];
          const int xx = j == 0 ? r0.x[0] : j == 1 ? r0.x[1] : j == 2 ? r0.x[2] : r0.x[3];
          const int ss = j == 0 ? r0.slot[0] : j == 1 ? r0.slot[1] : j == 2 ? r0.slot[2] : r0.slot[3];
          u = __builtin_amdgcn_readlane(uu, ln);
          x = __builtin_amdgcn_readlane(xx, ln);
          slot = __builtin_amdgcn_readlane(ss, ln);
        } else {
          const int2 q = a.rec[e];
          u = q.x;
          x = q.y;
          slot = -1;
        }
        if (u < g0 || u >= v) continue;   // not a predecessor in this graph (invalid input)
        // Ring and prefetch buffer: one LDS read at a computed offset (a
        // generic load here would wait for every outstanding memory operation
        // of the wave, the prefetches and stores included).
        unsigned w;
        if (u >= limit || slot >= 0) {
          const int off = u >= limit ? (u & (kRing - 1)) * kWave : fb_off + slot * kWave;
          w = words[off + lane];
        } else {
          w = load_wait(&far[(size_t)u * kWave + lane]);
        }
        const unsigned fu = w >> 6;
        const int du = (int)(w & 63u);
        const unsigned arrive = fu + (du != p ? (unsigned)x : 0u);
        ready = max(ready, arrive);
      }
      const unsigned start = max(ready, dev_free[p][lane]);
      const unsigned fin = start + (unsigned)c;
      wrapped |= fin >= kTimeLimit || fin < start;
      const unsigned pw = pack(fin & (kTimeLimit - 1), p);
      dev_free[p][lane] = fin;
      ring[v & (kRing - 1)][lane] = pw;
      far[(size_t)v * kWave + lane] = pw;
      mk = max(mk, fin);
    }
    h0 = h1;
    h1 = h2;
    h2 = h3;
    r0 = r1;
    r1 = r2;
  }
  wait_all_memory();
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
  a.far = L.far;
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
