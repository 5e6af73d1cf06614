// Whole-graph placement sampling: one fused Gumbel-max pass over (k, v).
//
// Thread (k, v): D uniforms from Philox4x64-10 with counter (v, k, 2, j >> 3)
// and key (seed, 0) (one call yields 8 devices), Gumbel noise -ln(-ln u),
// argmax of logits + noise (first maximum wins), and the chosen device's
// log-softmax term.  The log-prob terms are summed per work-group in a fixed
// tree order; a second kernel adds the work-group partials of each graph in
// chunk order, so results are bit-reproducible.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

__device__ __forceinline__ float uniform_at(const U64x4& r, int j) {
  const uint64_t w = r.w[(j & 7) >> 1];
  const uint32_t h = (j & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
  return half_to_uniform(h);
}

__global__ __launch_bounds__(kSampleChunk) void k_sample(const float* __restrict__ logits,
                                                         const float* __restrict__ lse, int n, int D,
                                                         uint64_t seed, const float* __restrict__ uniforms,
                                                         GraphTable ct, int total_chunks,
                                                         int* __restrict__ placements,
                                                         float* __restrict__ partial) {
  __shared__ float red[kSampleChunk];
  const int c = blockIdx.x, k = blockIdx.y;
  const int g = graph_of_block(ct, c);
  const int v = ct.ptr[g] + (c - ct.blk[g]) * kSampleChunk + threadIdx.x;
  float term = 0.f;
  if (v < ct.ptr[g + 1]) {
    const float* row = logits + (size_t)v * D;
    float lz;
    if (lse) {
      lz = lse[v];
    } else {
      float m = -INFINITY;
      for (int j = 0; j < D; ++j) m = fmaxf(m, row[j]);
      float s = 0.f;
      for (int j = 0; j < D; ++j) s += expf(row[j] - m);
      lz = m + logf(s);
    }
    float best = -INFINITY;
    int arg = 0;
    float best_logit = row[0];
    for (int jb = 0; jb < D; jb += 8) {
      U64x4 r;
      if (!uniforms) r = philox4x64_10((uint64_t)v, (uint64_t)k, 2ull, (uint64_t)(jb >> 3), seed, 0ull);
      const int jend = min(jb + 8, D);
      for (int j = jb; j < jend; ++j) {
        const float u = uniforms ? uniforms[((size_t)k * n + v) * D + j] : uniform_at(r, j);
        const float lg = row[j];
        const float sc = lg - logf(-logf(u));
        if (sc > best) { best = sc; arg = j; best_logit = lg; }
      }
    }
    placements[(size_t)k * n + v] = arg;
    term = best_logit - lz;
  }
  red[threadIdx.x] = term;
  __syncthreads();
#pragma unroll
  for (int w = kSampleChunk / 2; w >= 1; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[(size_t)k * total_chunks + c] = red[0];
}

hipError_t launch_sample(const float* logits, const float* lse, int n, int D, int K, uint64_t seed,
                         const float* uniforms, const GraphTable& ct, int total_chunks, int* placements,
                         float* partial, hipStream_t s) {
  dim3 grid(total_chunks, K), block(kSampleChunk);
  hipLaunchKernelGGL(k_sample, grid, block, 0, s, logits, lse, n, D, seed, uniforms, ct, total_chunks,
                     placements, partial);
  return hipGetLastError();
}

// logp[g][k]: one wavefront per (g, k); lane l adds chunks l, l + 64, ... of
// graph g in order, then a fixed butterfly combines the lanes.
__global__ __launch_bounds__(256) void k_logp_reduce(const float* __restrict__ partial, GraphTable ct,
                                                     int total_chunks, int K, float* __restrict__ logp) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);   // over G * K
  if (i >= ct.n * K) return;
  const int g = i / K, k = i % K;
  const float* p = partial + (size_t)k * total_chunks;
  float acc = 0.f;
  for (int c = ct.blk[g] + lane; c < ct.blk[g + 1]; c += 64) acc += p[c];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += xor_shfl(acc, off);
  if (lane == 0) logp[i] = acc;
}

hipError_t launch_logp_reduce(const float* partial, const GraphTable& ct, int total_chunks, int K,
                              float* logp, hipStream_t s) {
  const int n = ct.n * K;
  hipLaunchKernelGGL(k_logp_reduce, dim3((n + 3) / 4), dim3(256), 0, s, partial, ct, total_chunks, K, logp);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_debug_uniforms(uint64_t seed, int n, int K, int D,
                                                        float* __restrict__ out) {
  const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;   // over K * n
  if (i >= (int64_t)K * n) return;
  const int k = (int)(i / n), v = (int)(i % n);
  for (int jb = 0; jb < D; jb += 8) {
    const U64x4 r = philox4x64_10((uint64_t)v, (uint64_t)k, 2ull, (uint64_t)(jb >> 3), seed, 0ull);
    for (int j = jb; j < min(jb + 8, D); ++j) out[i * D + j] = uniform_at(r, j);
  }
}

hipError_t launch_debug_uniforms(uint64_t seed, int n, int K, int D, float* out, hipStream_t s) {
  const int64_t total = (int64_t)K * n;
  hipLaunchKernelGGL(k_debug_uniforms, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, seed, n, K, D, out);
  return hipGetLastError();
}

}  // namespace gdp
