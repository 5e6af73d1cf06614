// Whole-graph placement sampling: one fused Gumbel-max pass over (k, v).
//
// Thread (k, v), for a few consecutive k: D uniforms from Philox4x64-10 with
// counter (v, k, 2, j >> 3)
// and key (seed, 0) (one call yields 8 devices), Gumbel noise -ln(-ln u),
// argmax of logits + noise (first maximum wins), and the chosen device's
// log-softmax term.  The log-prob terms are summed per work-group in a fixed
// order; a second kernel adds the work-group partials of each graph in chunk
// order, so results are bit-reproducible.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

__device__ __forceinline__ float uniform_at(const U64x4& r, int j) {
  const uint64_t w = r.w[(j & 7) >> 1];
  const uint32_t h = (j & 1) ? (uint32_t)(w >> 32) : (uint32_t)w;
  return half_to_uniform(h);
}

// 2^x and log2 on the transcendental unit.
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// The Gumbel-max decision argmax_j (l_j - ln(-ln u_j)) in base 2: dividing
// every score by ln 2 and dropping the common constant log2(ln 2) leaves
// argmax_j (l_j / ln 2 - log2(-log2 u_j)).  -log2 u lies in [2^-23.5, 24]
// for the uniforms used here, so both logarithms see normal inputs.
__device__ __forceinline__ float gumbel_score(float logit, float u) {
  return fmaf(logit, 1.4426950408889634f, -fast_log2(-fast_log2(u)));
}

// Thread (k, v) for kSamplesPerThread consecutive k: their Philox calls are
// independent, so interleaving them hides each call's chain of dependent
// 64-bit products behind the other's.
constexpr int kSamplesPerThread = 4;

__global__ __launch_bounds__(kSampleChunk) void k_sample(const float* __restrict__ logits,
                                                         const float* __restrict__ lse, int n, int D, int K,
                                                         uint64_t seed, const float* __restrict__ uniforms,
                                                         GraphTable ct, int total_chunks, int chunk0,
                                                         int* __restrict__ placements,
                                                         float* __restrict__ partial) {
  constexpr int S = kSamplesPerThread;
  __shared__ float red[S][kSampleChunk / kWave];
  const int c = chunk0 + blockIdx.x, k0 = blockIdx.y * S;
  const int g = graph_of_block(ct, c);
  const int v = ct.ptr[g] + (c - ct.blk[g]) * kSampleChunk + threadIdx.x;
  float term[S];
#pragma unroll
  for (int q = 0; q < S; ++q) term[q] = 0.f;
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
    float best[S];
    int arg[S];
#pragma unroll
    for (int q = 0; q < S; ++q) {
      best[q] = -INFINITY;
      arg[q] = 0;
    }
    // one Philox call covers 8 devices; the 8 are unrolled so that every
    // uniform is taken from a fixed word of the result
    for (int jb = 0; jb < D; jb += 8) {
      U64x4 r[S];
      if (!uniforms) {
#pragma unroll
        for (int q = 0; q < S; ++q)   // (k beyond K: computed, never used)
          r[q] = philox4x64_10((uint64_t)v, (uint64_t)(k0 + q), 2ull, (uint64_t)(jb >> 3), seed, 0ull);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = jb + e;
        if (j < D) {
          const float lj = row[j];
#pragma unroll
          for (int q = 0; q < S; ++q) {
            if (k0 + q < K) {
              const float u = uniforms ? uniforms[((size_t)(k0 + q) * n + v) * D + j] : uniform_at(r[q], e);
              const float sc = gumbel_score(lj, u);
              if (sc > best[q]) { best[q] = sc; arg[q] = j; }   // first maximum wins
            }
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < S; ++q)
      if (k0 + q < K) {
        placements[(size_t)(k0 + q) * n + v] = arg[q];
        term[q] = row[arg[q]] - lz;
      }
  }
  // work-group sums in a fixed order: each wave's butterfly, then the waves in index order
#pragma unroll
  for (int q = 0; q < S; ++q) {
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) term[q] += xor_shfl(term[q], off);
    if ((threadIdx.x & (kWave - 1)) == 0) red[q][threadIdx.x / kWave] = term[q];
  }
  __syncthreads();
  if (threadIdx.x < S && k0 + (int)threadIdx.x < K) {
    const int q = threadIdx.x;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kSampleChunk / kWave; ++w) sum += red[q][w];
    partial[(size_t)(k0 + q) * total_chunks + c] = sum;
  }
}

hipError_t launch_sample(const float* logits, const float* lse, int n, int D, int K, uint64_t seed,
                         const float* uniforms, const GraphTable& ct, int total_chunks, int* placements,
                         float* partial, hipStream_t s, int chunk0, int chunk1) {
  if (chunk1 < 0) chunk1 = total_chunks;
  if (chunk0 < 0 || chunk0 > chunk1 || chunk1 > total_chunks) return hipErrorInvalidValue;
  if (chunk0 == chunk1) return hipSuccess;
  dim3 grid(chunk1 - chunk0, (K + kSamplesPerThread - 1) / kSamplesPerThread), block(kSampleChunk);
  hipLaunchKernelGGL(k_sample, grid, block, 0, s, logits, lse, n, D, K, seed, uniforms, ct, total_chunks, chunk0,
                     placements, partial);
  return hipGetLastError();
}

// The log-softmax term of given placements, summed per work-group in the same
// fixed order as k_sample's (the numerator of PPO's ratio after an update).
__global__ __launch_bounds__(kSampleChunk) void k_logp_given(const float* __restrict__ logits,
                                                             const float* __restrict__ lse, int n, int D,
                                                             const int* __restrict__ placements, GraphTable ct,
                                                             int total_chunks, float* __restrict__ partial) {
  __shared__ float red[kSampleChunk / kWave];
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
    int p = placements[(size_t)k * n + v];
    p = p < 0 ? 0 : (p >= D ? D - 1 : p);
    term = row[p] - lz;
  }
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) term += xor_shfl(term, off);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = term;
  __syncthreads();
  if (threadIdx.x == 0) {
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kSampleChunk / kWave; ++w) sum += red[w];
    partial[(size_t)k * total_chunks + c] = sum;
  }
}

hipError_t launch_logp_given(const float* logits, const float* lse, int n, int D, int K, const int* placements,
                             const GraphTable& ct, int total_chunks, float* partial, hipStream_t s) {
  hipLaunchKernelGGL(k_logp_given, dim3(total_chunks, K), dim3(kSampleChunk), 0, s, logits, lse, n, D, placements, ct,
                     total_chunks, partial);
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
  // lane l adds chunks c0 + l, c0 + l + 64, ... into four running sums; past
  // the end a lane reloads the last chunk and adds nothing, so four loads are
  // in flight with no branch between them
  const int c0 = ct.blk[g], c1 = ct.blk[g + 1];
  float a4[4] = {0.f, 0.f, 0.f, 0.f};
  for (int c = c0 + lane; c < c1; c += 4 * 64) {
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = p[min(c + 64 * e, c1 - 1)];
#pragma unroll
    for (int e = 0; e < 4; ++e) a4[e] += c + 64 * e < c1 ? v[e] : 0.f;
  }
  float acc = (a4[0] + a4[1]) + (a4[2] + a4[3]);
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
