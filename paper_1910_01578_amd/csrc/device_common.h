// Shared device-side definitions for the gfx950 kernels of libgdp.
//
// Element types: `float` (fp32 path) and `__bf16` (bf16 storage, fp32
// arithmetic).  Matrix-core work uses the 16x16 MFMA family; the lane layout
// of a 16 x 16 x K instruction with KV = K / 4 operand values per lane is
//   A (16 x K):  lane l holds row l % 16, k = KV * (l / 16) + [0, KV)
//   B (K x 16):  lane l holds column l % 16, k = KV * (l / 16) + [0, KV)
//   C/D (16x16): lane l holds column l % 16, rows 4 * (l / 16) + [0, 4)
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdp.h"

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace gdp {

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// 16 bytes of elements, moved as one vector access.
template <typename T>
struct alignas(16) Vec16 {
  static constexpr int N = 16 / sizeof(T);
  T v[N];
};

template <typename T>
__device__ __forceinline__ Vec16<T> load16(const T* p) {
  Vec16<T> r;
  *reinterpret_cast<uint4*>(&r) = *reinterpret_cast<const uint4*>(p);
  return r;
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const Vec16<T>& r) {
  *reinterpret_cast<uint4*>(p) = *reinterpret_cast<const uint4*>(&r);
}

// ---------------------------------------------------------------------------
// MFMA 16x16 traits.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int K = 32;
  static constexpr int KV = 8;
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const bf16* p) {
    return *reinterpret_cast<const frag*>(p);
  }
};

template <> struct Mfma<float> {
  static constexpr int K = 4;
  static constexpr int KV = 1;
  typedef float frag;
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
};

// bf16 16x16x16 (4 values per lane), used where the contraction is 16 long.
__device__ __forceinline__ f32x4 mfma_16x16x16_bf16(i16x4 a, i16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// ---------------------------------------------------------------------------
// Cross-lane helpers (wave64).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float xor_shfl(float v, int mask) { return __shfl_xor(v, mask, kWave); }
__device__ __forceinline__ int xor_shfl(int v, int mask) { return __shfl_xor(v, mask, kWave); }

// ---------------------------------------------------------------------------
// Work-groups of a launch are dealt to the 8 XCDs of the chip round-robin by
// id, and each XCD has its own L2.  This maps a work-group id to a logical
// tile id such that every XCD receives a contiguous run of logical tiles, so
// neighbouring tiles (which share operand rows) share an L2.  Bijective on
// [0, total).
// ---------------------------------------------------------------------------
constexpr int kNumXcd = 8;
__device__ __forceinline__ int xcd_remap(int p, int total) {
  const int per = total / kNumXcd, rem = total % kNumXcd;
  const int xcd = p % kNumXcd, idx = p / kNumXcd;
  return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

// ---------------------------------------------------------------------------
// Graph table passed by value: node starts of every graph of the batch plus a
// per-graph prefix of work blocks whose meaning depends on the kernel.
// ---------------------------------------------------------------------------
struct GraphTable {
  int n;
  int ptr[GDP_MAX_GRAPHS + 1];
  int blk[GDP_MAX_GRAPHS + 1];
};

// Largest g in [0, n) with t.blk[g] <= b.
__device__ __forceinline__ int graph_of_block(const GraphTable& t, int b) {
  int lo = 0, hi = t.n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (t.blk[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Largest g in [0, n) with t.ptr[g] <= v.
__device__ __forceinline__ int graph_of_node(const GraphTable& t, int v) {
  int lo = 0, hi = t.n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (t.ptr[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon et al., SC'11): 10 rounds of the 4x64 bijection; the
// key advances by the two Weyl constants between rounds.
// ---------------------------------------------------------------------------
struct U64x4 { uint64_t w[4]; };

// hi:lo = a * b (64 x 64 -> 128 bits) from four 32 x 32 -> 64 partial
// products, each carry folded into the next multiply-add, so that the low
// and high halves share their partial products.
__device__ __forceinline__ void mul64wide(uint64_t a, uint64_t b, uint64_t& lo, uint64_t& hi) {
  const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32), b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
  const uint64_t p00 = (uint64_t)a0 * b0;
  const uint64_t p01 = (uint64_t)a0 * b1 + (p00 >> 32);   // < 2^64
  const uint64_t t = (uint64_t)a1 * b0 + (uint32_t)p01;   // < 2^64
  lo = (t << 32) | (uint32_t)p00;
  hi = (uint64_t)a1 * b1 + ((p01 >> 32) + (t >> 32));
}

__device__ __forceinline__ U64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                               uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += W0; k1 += W1; }
    uint64_t lo0, hi0, lo1, hi1;
    mul64wide(M0, c0, lo0, hi0);
    mul64wide(M1, c2, lo1, hi1);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
  U64x4 r;
  r.w[0] = c0; r.w[1] = c1; r.w[2] = c2; r.w[3] = c3;
  return r;
}

// Uniform in (0, 1) from a 32-bit half: (2 * (h >> 9) + 1) * 2^-24, exact in fp32.
__device__ __forceinline__ float half_to_uniform(uint32_t h) {
  return (float)(2u * (h >> 9) + 1u) * 5.9604644775390625e-08f;
}

}  // namespace gdp
