// Section 3.1 kernels: neighbourhood construction, neighbour sampling, the
// Eq. 2 max-pool gather and the per-graph mean pool.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

// ---------------------------------------------------------------------------
__global__ void k_fill_i32(int* p, int64_t n, int value) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = value;
}

hipError_t launch_fill_i32(int* p, int64_t n, int value, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, value);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// in_deg[v] += 1 for every edge u -> v (integer atomics: order-independent).
__global__ void k_in_degree(const int* __restrict__ col_idx, int64_t n_edges, int* in_deg) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n_edges;
       e += (int64_t)gridDim.x * blockDim.x)
    atomicAdd(&in_deg[col_idx[e]], 1);
}

hipError_t launch_in_degree(const int* col_idx, int64_t n_edges, int* in_deg, hipStream_t s) {
  if (n_edges <= 0) return hipSuccess;
  int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_in_degree, dim3((unsigned)blocks), dim3(256), 0, s, col_idx, n_edges, in_deg);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Exclusive scans of the two degree arrays, in three launches (two for up
// to kScanDirectBlocks blocks, below):
//   in_ptr[i] = sum_{j<i} in_deg[j]
//   s_ptr[i]  = sum_{j<i} min(out_deg[j] + in_deg[j], fanout)
// (1) per-block totals of kScanBlock entries, (2) one work-group scans the
// block totals, (3) every block scans its entries and adds its offset.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int t = __shfl_up(v, off, kWave);
    if (lane >= off) v += t;
  }
  return v;
}

__device__ __forceinline__ void degree_pair(const int* __restrict__ row_ptr, const int* __restrict__ in_deg,
                                            int i, int n, int fanout, int& da, int& db) {
  da = 0;
  db = 0;
  if (i < n) {
    da = in_deg[i];
    const int tot = da + (row_ptr[i + 1] - row_ptr[i]);
    db = tot < fanout ? tot : fanout;
  }
}

// Block-wide exclusive scan of (a, b) pairs held one per thread (256 threads);
// returns the exclusive prefixes and writes the block totals to *ta / *tb.
__device__ __forceinline__ void block_scan2(int a, int b, int& ea, int& eb, int* ta, int* tb) {
  __shared__ int wa[4], wb[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ia = wave_incl_scan(a, lane), ib = wave_incl_scan(b, lane);
  if (lane == 63) { wa[wave] = ia; wb[wave] = ib; }
  __syncthreads();
  int oa = 0, ob = 0;
  for (int w = 0; w < wave; ++w) { oa += wa[w]; ob += wb[w]; }
  ea = oa + ia - a;
  eb = ob + ib - b;
  if (ta) *ta = wa[0] + wa[1] + wa[2] + wa[3];
  if (tb) *tb = wb[0] + wb[1] + wb[2] + wb[3];
  __syncthreads();
}

__global__ __launch_bounds__(256) void k_scan_block_sums(const int* __restrict__ row_ptr,
                                                         const int* __restrict__ in_deg, int n, int fanout,
                                                         int* __restrict__ bsum) {
  const int base = blockIdx.x * kScanBlock + threadIdx.x * 4;
  int sa = 0, sb = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int da, db;
    degree_pair(row_ptr, in_deg, base + j, n, fanout, da, db);
    sa += da;
    sb += db;
  }
  int ea, eb, ta, tb;
  block_scan2(sa, sb, ea, eb, &ta, &tb);
  if (threadIdx.x == 0) {
    bsum[2 * blockIdx.x] = ta;
    bsum[2 * blockIdx.x + 1] = tb;
  }
}

__global__ __launch_bounds__(256) void k_scan_block_offsets(int* __restrict__ bsum, int nblocks, int n,
                                                            int* __restrict__ in_ptr, int* __restrict__ s_ptr) {
  int carry_a = 0, carry_b = 0;
  for (int base = 0; base < nblocks; base += 256) {
    const int i = base + threadIdx.x;
    const int a = i < nblocks ? bsum[2 * i] : 0, b = i < nblocks ? bsum[2 * i + 1] : 0;
    int ea, eb, ta, tb;
    block_scan2(a, b, ea, eb, &ta, &tb);
    if (i < nblocks) {
      bsum[2 * i] = carry_a + ea;
      bsum[2 * i + 1] = carry_b + eb;
    }
    carry_a += ta;
    carry_b += tb;
  }
  if (threadIdx.x == 0) {
    in_ptr[n] = carry_a;
    s_ptr[n] = carry_b;
  }
}

__global__ __launch_bounds__(256) void k_scan_apply(const int* __restrict__ row_ptr, const int* __restrict__ in_deg,
                                                    int n, int fanout, const int* __restrict__ boff,
                                                    int* __restrict__ in_ptr, int* __restrict__ s_ptr) {
  const int base = blockIdx.x * kScanBlock + threadIdx.x * 4;
  int da[4], db[4], sa = 0, sb = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    degree_pair(row_ptr, in_deg, base + j, n, fanout, da[j], db[j]);
    sa += da[j];
    sb += db[j];
  }
  int ea, eb;
  block_scan2(sa, sb, ea, eb, nullptr, nullptr);
  ea += boff[2 * blockIdx.x];
  eb += boff[2 * blockIdx.x + 1];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = base + j;
    if (i < n) { in_ptr[i] = ea; s_ptr[i] = eb; }
    ea += da[j];
    eb += db[j];
  }
}

// (3) without (2), for up to kScanDirectBlocks blocks: each block adds up the
// totals of the blocks before it itself (at most a few KB from L2), and the
// last block writes the grand totals.  One launch fewer.
constexpr int kScanDirectBlocks = 1024;

__global__ __launch_bounds__(256) void k_scan_apply_direct(const int* __restrict__ row_ptr,
                                                           const int* __restrict__ in_deg, int n, int fanout,
                                                           const int* __restrict__ bsum, int nblocks,
                                                           int* __restrict__ in_ptr, int* __restrict__ s_ptr) {
  int pa = 0, pb = 0;
  for (int i = threadIdx.x; i < (int)blockIdx.x; i += 256) {
    pa += bsum[2 * i];
    pb += bsum[2 * i + 1];
  }
  int xa, xb, off_a, off_b;
  block_scan2(pa, pb, xa, xb, &off_a, &off_b);
  const int base = blockIdx.x * kScanBlock + threadIdx.x * 4;
  int da[4], db[4], sa = 0, sb = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    degree_pair(row_ptr, in_deg, base + j, n, fanout, da[j], db[j]);
    sa += da[j];
    sb += db[j];
  }
  int ea, eb, ta, tb;
  block_scan2(sa, sb, ea, eb, &ta, &tb);
  ea += off_a;
  eb += off_b;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = base + j;
    if (i < n) { in_ptr[i] = ea; s_ptr[i] = eb; }
    ea += da[j];
    eb += db[j];
  }
  if (blockIdx.x == nblocks - 1 && threadIdx.x == 0) {
    in_ptr[n] = off_a + ta;
    s_ptr[n] = off_b + tb;
  }
}

hipError_t launch_scan_degrees(const int* row_ptr, const int* in_deg, int n, int fanout, int* in_ptr,
                               int* s_ptr, int* block_tmp, hipStream_t s) {
  const int nb = (n + kScanBlock - 1) / kScanBlock;
  hipLaunchKernelGGL(k_scan_block_sums, dim3(nb), dim3(256), 0, s, row_ptr, in_deg, n, fanout, block_tmp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (nb <= kScanDirectBlocks) {
    hipLaunchKernelGGL(k_scan_apply_direct, dim3(nb), dim3(256), 0, s, row_ptr, in_deg, n, fanout, block_tmp, nb,
                       in_ptr, s_ptr);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_scan_block_offsets, dim3(1), dim3(256), 0, s, block_tmp, nb, n, in_ptr, s_ptr);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_scan_apply, dim3(nb), dim3(256), 0, s, row_ptr, in_deg, n, fanout, block_tmp, in_ptr, s_ptr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Reverse edges: in_idx[in_ptr[v] + slot] = u for every u -> v.  Slot order is
// whatever the atomics give; every consumer is order-invariant.
// One thread per edge e = (u -> v): u is the row whose [row_ptr[u], row_ptr[u+1])
// holds e (binary search), so high out-degree nodes spread over many threads.
__global__ void k_fill_reverse(const int* __restrict__ row_ptr, const int* __restrict__ col_idx,
                               const int* __restrict__ in_ptr, int n, int64_t n_edges, int* cursor,
                               int* __restrict__ in_idx) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n_edges;
       e += (int64_t)gridDim.x * blockDim.x) {
    int lo = 0, hi = n - 1;                  // largest u with row_ptr[u] <= e
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (row_ptr[mid] <= e) lo = mid; else hi = mid - 1;
    }
    const int v = col_idx[e];
    const int slot = atomicAdd(&cursor[v], 1);
    in_idx[in_ptr[v] + slot] = lo;
  }
}

hipError_t launch_fill_reverse(const int* row_ptr, const int* col_idx, const int* in_ptr, int n,
                               int64_t n_edges, int* cursor, int* in_idx, hipStream_t s) {
  if (n_edges <= 0) return hipSuccess;
  int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_fill_reverse, dim3((unsigned)blocks), dim3(256), 0, s, row_ptr, col_idx, in_ptr, n,
                     n_edges, cursor, in_idx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// S(v): all neighbours when |N(v)| <= fanout, else the fanout smallest
// (key, u) with key = word 0 of Philox4x64-10((v-g0, u-g0, 1, 0), (seed, 0)).
//
// Pass 1 (one thread per node) copies N(v) for the light nodes and queues the
// heavy ones (|N(v)| > fanout).  Pass 2 gives every heavy node a wavefront:
// lanes draw the keys of up to 64 * kHeavyPerLane neighbours at once, a
// radix select over the 64-bit keys finds the fanout-th smallest key T, and
// every neighbour with key < T is taken plus the smallest ids among the ones
// with key == T.  Nodes with more neighbours than that use a sorted register
// list on one lane.
__device__ __forceinline__ int nbr_at(const int* __restrict__ col_idx, const int* __restrict__ in_idx, int o0,
                                      int n_out, int i0, int e) {
  return e < n_out ? col_idx[o0 + e] : in_idx[i0 + e - n_out];
}

__global__ __launch_bounds__(256) void k_nbr_light(const int* __restrict__ row_ptr, const int* __restrict__ col_idx,
                                                   const int* __restrict__ in_ptr, const int* __restrict__ in_idx,
                                                   const int* __restrict__ s_ptr, int n, int fanout,
                                                   int* __restrict__ s_idx, int* heavy, int* heavy_count) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n) return;
  const int o0 = row_ptr[v], o1 = row_ptr[v + 1];
  const int i0 = in_ptr[v], i1 = in_ptr[v + 1];
  const int sp = s_ptr[v];                      // read with the others: one round of loads
  const int deg = (o1 - o0) + (i1 - i0);
  if (deg > fanout) {
    heavy[atomicAdd(heavy_count, 1)] = v;
    return;
  }
  // groups of four loads issued before their stores (a list may be empty, and
  // an empty edge array may not be read at all, so every load is guarded)
  int* out = s_idx + sp;
  int w = 0;
  for (int e = o0; e < o1; e += 4) {
    int u[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (e + k < o1) u[k] = col_idx[e + k];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (e + k < o1) out[w + k] = u[k];
    w += min(4, o1 - e);
  }
  for (int e = i0; e < i1; e += 4) {
    int u[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (e + k < i1) u[k] = in_idx[e + k];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (e + k < i1) out[w + k] = u[k];
    w += min(4, i1 - e);
  }
}

__device__ __forceinline__ bool pair_less(uint64_t ka, int ua, uint64_t kb, int ub) {
  return ka < kb || (ka == kb && ua < ub);
}

// One lane, any degree: keep the MAXF smallest pairs in a sorted register list.
template <int MAXF>
__device__ void select_serial(const int* __restrict__ col_idx, const int* __restrict__ in_idx, int o0, int n_out,
                              int i0, int deg, int v_loc, int g0, int fanout, uint64_t seed, int* out) {
  uint64_t key[MAXF];
  int id[MAXF];
#pragma unroll
  for (int i = 0; i < MAXF; ++i) { key[i] = ~0ull; id[i] = 0x7fffffff; }
  for (int e = 0; e < deg; ++e) {
    const int u = nbr_at(col_idx, in_idx, o0, n_out, i0, e);
    const uint64_t k = philox4x64_10((uint64_t)v_loc, (uint64_t)(u - g0), 1ull, 0ull, seed, 0ull).w[0];
#pragma unroll
    for (int i = MAXF - 1; i >= 0; --i) {
      const int ip = i > 0 ? i - 1 : 0;
      const bool shift = (i > 0) && pair_less(k, u, key[ip], id[ip]);
      if (shift) { key[i] = key[ip]; id[i] = id[ip]; }
      else if (pair_less(k, u, key[i], id[i])) { key[i] = k; id[i] = u; }
    }
  }
#pragma unroll
  for (int i = 0; i < MAXF; ++i)
    if (i < fanout) out[i] = id[i];
}

constexpr int kHeavyPerLane = 8;

__global__ __launch_bounds__(256) void k_nbr_heavy(const int* __restrict__ row_ptr, const int* __restrict__ col_idx,
                                                   const int* __restrict__ in_ptr, const int* __restrict__ in_idx,
                                                   const int* __restrict__ s_ptr, int fanout, uint64_t seed,
                                                   GraphTable gt, const int* __restrict__ heavy,
                                                   const int* __restrict__ heavy_count, int* __restrict__ s_idx) {
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nwaves = gridDim.x * 4;
  const int count = *heavy_count;
  for (int h = wave; h < count; h += nwaves) {
    const int v = heavy[h];
    const int o0 = row_ptr[v], n_out = row_ptr[v + 1] - o0;
    const int i0 = in_ptr[v], deg = n_out + (in_ptr[v + 1] - i0);
    const int g0 = gt.ptr[graph_of_node(gt, v)];
    int* out = s_idx + s_ptr[v];
    if (deg > 64 * kHeavyPerLane) {
      if (lane == 0) select_serial<GDP_MAX_FANOUT>(col_idx, in_idx, o0, n_out, i0, deg, v - g0, g0, fanout, seed, out);
      continue;
    }
    // R = key registers in use (wave-uniform): every loop below skips the rest.
    const int R = (deg + 63) >> 6;
    uint64_t key[kHeavyPerLane];
    int id[kHeavyPerLane];
#pragma unroll
    for (int r = 0; r < kHeavyPerLane; ++r) {
      const int e = lane + 64 * r;
      key[r] = ~0ull;
      id[r] = 0x7fffffff;
      if (r < R && e < deg) {
        id[r] = nbr_at(col_idx, in_idx, o0, n_out, i0, e);
        key[r] = philox4x64_10((uint64_t)(v - g0), (uint64_t)(id[r] - g0), 1ull, 0ull, seed, 0ull).w[0];
      }
    }
    // Radix select from the top bit.  The class is the keys whose bits above
    // `bit` equal prefix's; it holds `cand` keys, and `need` of them are still
    // to be taken (every key of a smaller class is taken).  Once cand == need
    // the whole class is taken and the rest of the bits decide nothing.
    uint64_t prefix = 0;
    int need = fanout, cand = deg;
    int bit = 63;
    for (; bit >= 0 && cand > need; --bit) {
      const uint64_t hi_mask = (bit == 63) ? 0ull : (~0ull << (bit + 1));
      int c0 = 0;
#pragma unroll
      for (int r = 0; r < kHeavyPerLane; ++r) {
        if (r >= R) break;
        const int e = lane + 64 * r;
        const bool m = e < deg && ((key[r] & hi_mask) == prefix) && !((key[r] >> bit) & 1ull);
        c0 += __popcll(__ballot(m));
      }
      if (need > c0) {
        prefix |= (1ull << bit);
        need -= c0;
        cand -= c0;
      } else {
        cand = c0;
      }
    }
    const uint64_t cmask = (bit == 63) ? 0ull : (~0ull << (bit + 1));
    const bool whole = cand == need;   // else: all 64 bits tie, decided by the smallest ids
    // take every key of a smaller class (and, when whole, of the class itself)
    int base = 0;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int r = 0; r < kHeavyPerLane; ++r) {
      if (r >= R) break;
      const int e = lane + 64 * r;
      const uint64_t kc = key[r] & cmask;
      const bool sel = e < deg && (kc < prefix || (whole && kc == prefix));
      const uint64_t bal = __ballot(sel);
      if (sel) out[base + __popcll(bal & lt_mask)] = id[r];
      base += __popcll(bal);
    }
    const uint64_t T = prefix;
    int last = -1;   // ids strictly above `last` are still eligible
    for (int t = 0; t < (whole ? 0 : need); ++t) {
      int best = 0x7fffffff;
#pragma unroll
      for (int r = 0; r < kHeavyPerLane; ++r) {
        if (r >= R) break;
        const int e = lane + 64 * r;
        if (e < deg && key[r] == T && id[r] > last && id[r] < best) best = id[r];
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) best = min(best, xor_shfl(best, off));
      if (lane == 0) out[base] = best;
      ++base;
      last = best;
    }
  }
}

hipError_t launch_nbr_sample(const int* row_ptr, const int* col_idx, const int* in_ptr, const int* in_idx,
                             const int* s_ptr, int n, int fanout, uint64_t seed, const GraphTable& gt, int* s_idx,
                             int* heavy, int* heavy_count, hipStream_t s) {
  hipLaunchKernelGGL(k_nbr_light, dim3((n + 255) / 256), dim3(256), 0, s, row_ptr, col_idx, in_ptr, in_idx, s_ptr, n,
                     fanout, s_idx, heavy, heavy_count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_nbr_heavy, dim3(256), dim3(256), 0, s, row_ptr, col_idx, in_ptr, in_idx, s_ptr, fanout, seed,
                     gt, heavy, heavy_count, s_idx);
  return hipGetLastError();
}

// Eq. 2's max over sampled neighbours.  A group of LPR lanes owns one node,
// each lane a 16-byte slice of the row: the group loads its node's sampled
// neighbour ids with one load (an id per lane, LPR at a time), then fetches
// the neighbours' rows four at a time, each lane taking the ids from the
// group's lanes by a shuffle.  So a node costs three dependent memory
// latencies (its range, its ids, its rows) whatever its degree, and a wave
// carries 64 / LPR nodes.  The max does not depend on the order of the
// rows, so the result is the same for any grouping.  Nodes without sampled
// neighbours get 0 (the rows are sigmoid outputs, all positive).
template <typename T, int H>
struct GatherGeo {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int LPR = H / VEC;          // lanes per row
  static constexpr int NPW = 64 / LPR;         // nodes per wave
  static constexpr int RB = 4;                 // rows in flight per lane
  static_assert(LPR >= RB && LPR <= 64 && 64 % LPR == 0 && LPR % RB == 0, "row width");
};

template <typename T, int H>
__global__ __launch_bounds__(256) void k_gather_max(const T* __restrict__ P,
                                                    const int* __restrict__ s_ptr,
                                                    const int* __restrict__ s_idx, int n,
                                                    T* __restrict__ A) {
  using G = GatherGeo<T, H>;
  constexpr int VEC = G::VEC, LPR = G::LPR, NPW = G::NPW, RB = G::RB;
  const int lane = threadIdx.x & 63;
  const int v0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * NPW;   // the wave's first node
  if (v0 >= n) return;                                          // whole waves
  const int grp = lane / LPR, sub = lane % LPR;
  const int v = v0 + grp;
  const bool live = v < n;
  // Every load below is unconditional, so none waits behind a branch: groups
  // past the last node read node n - 1's range, and masked slots read index
  // 0 and row 0 (s_idx is non-empty whenever some node of the wave has a
  // sampled neighbour, the only case in which the loop runs).
  const int vc = live ? v : n - 1;
  const int b = s_ptr[vc];
  const int e = s_ptr[vc + 1];
  const int cnt = live ? e - b : 0;
  // the largest count among the wave's nodes bounds every group's loop, so
  // all lanes take part in each shuffle
  int cmax = cnt;
#pragma unroll
  for (int off = LPR; off < 64; off <<= 1) cmax = max(cmax, xor_shfl(cmax, off));
  cmax = __builtin_amdgcn_readfirstlane(cmax);
  const int col = sub * VEC;
  float m[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) m[j] = 0.f;
  for (int k0 = 0; k0 < cmax; k0 += LPR) {
    const bool have = k0 + sub < cnt;
    int ids = s_idx[have ? b + k0 + sub : 0];
    ids = have ? ids : 0;
    const int nb = min(cmax - k0, LPR);
    for (int j0 = 0; j0 < nb; j0 += RB) {
      // j0 + q < LPR: the source lanes stay inside the group
      int u[RB];
#pragma unroll
      for (int q = 0; q < RB; ++q) u[q] = __shfl(ids, grp * LPR + j0 + q, 64);
      uint4 r[RB];
#pragma unroll
      for (int q = 0; q < RB; ++q) r[q] = *reinterpret_cast<const uint4*>(P + (size_t)u[q] * H + col);
#pragma unroll
      for (int q = 0; q < RB; ++q) {
        // a slot past the node's count becomes +0, which leaves the max of
        // positive rows as it is (an AND, not a branch around the load)
        const uint32_t keep = k0 + j0 + q < cnt ? 0xffffffffu : 0u;
        const uint4 w = make_uint4(r[q].x & keep, r[q].y & keep, r[q].z & keep, r[q].w & keep);
        const Vec16<T> x = __builtin_bit_cast(Vec16<T>, w);
#pragma unroll
        for (int j = 0; j < VEC; ++j) m[j] = fmaxf(m[j], to_f32(x.v[j]));
      }
    }
  }
  if (live) {
    Vec16<T> o;
#pragma unroll
    for (int j = 0; j < VEC; ++j) o.v[j] = from_f32<T>(m[j]);
    store16(A + (size_t)v * H + col, o);
  }
}

template <typename T, int H>
static void launch_gather_max_h(const T* P, const int* s_ptr, const int* s_idx, int n, T* A, hipStream_t s) {
  constexpr int NODES = 4 * GatherGeo<T, H>::NPW;   // per 256-thread work-group
  hipLaunchKernelGGL((k_gather_max<T, H>), dim3((n + NODES - 1) / NODES), dim3(256), 0, s, P, s_ptr, s_idx, n, A);
}

template <typename T>
hipError_t launch_gather_max(const T* P, const int* s_ptr, const int* s_idx, int n, int H, T* A,
                             hipStream_t s) {
  if (n <= 0) return hipSuccess;
  switch (H) {
    case 64: launch_gather_max_h<T, 64>(P, s_ptr, s_idx, n, A, s); break;
    case 128: launch_gather_max_h<T, 128>(P, s_ptr, s_idx, n, A, s); break;
    case 256: launch_gather_max_h<T, 256>(P, s_ptr, s_idx, n, A, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_gather_max<float>(const float*, const int*, const int*, int, int, float*, hipStream_t);
template hipError_t launch_gather_max<bf16>(const bf16*, const int*, const int*, int, int, bf16*, hipStream_t);

// ---------------------------------------------------------------------------
// Mean pool: chunks of kMeanpoolRows rows never cross a graph.  Each chunk sum
// adds its rows in a fixed order (16-byte row slices, then the row groups in
// LDS); each graph then adds its chunk sums in 16 interleaved fixed-order
// slices combined in a fixed tree.  Deterministic.
template <typename T, int H>
__global__ __launch_bounds__(256) void k_meanpool_partial(const T* __restrict__ h, GraphTable ct,
                                                          float* __restrict__ partial) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int TPR = H / EPV;
  constexpr int RG = 256 / TPR;
  __shared__ float red[RG][H];
  const int c = blockIdx.x;
  const int g = graph_of_block(ct, c);
  const int r0 = ct.ptr[g] + (c - ct.blk[g]) * kMeanpoolRows;
  const int r1 = min(r0 + kMeanpoolRows, ct.ptr[g + 1]);
  static_assert(kMeanpoolRows % RG == 0, "chunk rows split evenly over the row groups");
  const int rg = threadIdx.x / TPR, col = (threadIdx.x % TPR) * EPV;
  float acc[EPV];
#pragma unroll
  for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
  // every row of the chunk in one unrolled pass, so that all of a thread's
  // loads are in flight at once; rows past the chunk's end (a graph's last
  // chunk) read its last row and add nothing
#pragma unroll
  for (int i = 0; i < kMeanpoolRows / RG; ++i) {
    const int r = r0 + rg + i * RG;
    const Vec16<T> x = load16(h + (size_t)min(r, r1 - 1) * H + col);
    const float keep = r < r1 ? 1.0f : 0.0f;
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] += keep * to_f32(x.v[e]);
  }
#pragma unroll
  for (int e = 0; e < EPV; ++e) red[rg][col + e] = acc[e];
  __syncthreads();
  for (int i = threadIdx.x; i < H; i += 256) {
    float sum = 0.f;
    for (int q = 0; q < RG; ++q) sum += red[q][i];
    partial[(size_t)c * H + i] = sum;
  }
}

// graph_emb[g][col] = (sum over graph g's chunks of partial[c][col]) / |V_g|.
// A block covers 64 columns of one graph; wave w adds chunks w, w + 16, ... into
// eight running sums (chunk c0 + w + 16 (8 q + e) into sum e, so eight loads are
// in flight), and the 16 waves' sums meet in LDS in a fixed pairwise order.
constexpr int kPoolFinalWaves = 16;
__global__ __launch_bounds__(64 * kPoolFinalWaves) void k_meanpool_final(const float* __restrict__ partial, int H,
                                                                        GraphTable ct, float* __restrict__ out) {
  constexpr int W = kPoolFinalWaves, E = 8;
  __shared__ float red[W][64];
  const int g = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = blockIdx.y * 64 + lane;
  const int c0 = ct.blk[g], c1 = ct.blk[g + 1];
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  // past-the-end chunks load the last one and add nothing: no branch, so the
  // eight loads issue back to back
  if (col < H)
    for (int c = c0 + w; c < c1; c += W * E) {
      float v[E];
#pragma unroll
      for (int e = 0; e < E; ++e) v[e] = partial[(size_t)min(c + W * e, c1 - 1) * H + col];
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += c + W * e < c1 ? v[e] : 0.f;
    }
  red[w][lane] = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
  __syncthreads();
  if (w == 0 && col < H) {
    float t[W / 2];
#pragma unroll
    for (int i = 0; i < W / 2; ++i) t[i] = red[2 * i][lane] + red[2 * i + 1][lane];
#pragma unroll
    for (int i = 0; i < W / 4; ++i) t[i] = t[2 * i] + t[2 * i + 1];
#pragma unroll
    for (int i = 0; i < W / 8; ++i) t[i] = t[2 * i] + t[2 * i + 1];
    const float sum = t[0] + t[1];
    out[(size_t)g * H + col] = sum / (float)(ct.ptr[g + 1] - ct.ptr[g]);
  }
}

template <typename T>
hipError_t launch_meanpool(const T* h, int H, const GraphTable& ct, int total_chunks, float* partial,
                           float* graph_emb, hipStream_t s) {
  switch (H) {
    case 64: hipLaunchKernelGGL((k_meanpool_partial<T, 64>), dim3(total_chunks), dim3(256), 0, s, h, ct, partial); break;
    case 128: hipLaunchKernelGGL((k_meanpool_partial<T, 128>), dim3(total_chunks), dim3(256), 0, s, h, ct, partial); break;
    case 256: hipLaunchKernelGGL((k_meanpool_partial<T, 256>), dim3(total_chunks), dim3(256), 0, s, h, ct, partial); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_meanpool_final, dim3(ct.n, (H + 63) / 64), dim3(64 * kPoolFinalWaves), 0, s, partial, H, ct,
                     graph_emb);
  return hipGetLastError();
}
template hipError_t launch_meanpool<float>(const float*, int, const GraphTable&, int, float*, float*, hipStream_t);
template hipError_t launch_meanpool<bf16>(const bf16*, int, const GraphTable&, int, float*, float*, hipStream_t);

}  // namespace gdp
