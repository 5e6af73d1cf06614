// Dense layers on the matrix cores: out = epilogue(A W^T).
//
// A is [M, K] and W is [N, K] (each output unit's weights contiguous), so both
// MFMA operands are K-contiguous.  K may consist of two segments, each with
// its own activation source and weight array: that is how Eq. 3's
// f(concat(h_v, h_N(v))) runs without materialising either concatenation.
//
// A 256-thread work-group computes a BM x BN tile with four waves; each wave
// owns a WM x WN sub-tile of 16 x 16 MFMA blocks.  K advances in BK steps
// through double-buffered LDS tiles (global -> registers for step k+1 while
// step k is multiplied).  A may be stored in fp32 (the residual stream) and is
// rounded to the MFMA type on its way into LDS.  The product is accumulated
// transposed so that each lane ends with 4 consecutive outputs of one row,
// which the epilogue writes as one vector store.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

namespace {

template <typename T> struct KStep { static constexpr int BK = 64; };
template <> struct KStep<float> { static constexpr int BK = 32; };

template <typename T>
struct TileCfg {
  static constexpr int BK = KStep<T>::BK;
  static constexpr int EPV = 16 / sizeof(T);   // MFMA-type elements per 16 bytes
  static constexpr int STRIDE = BK + EPV;       // padded LDS row (conflict-free fragment reads)
};

template <typename TA, typename T> struct Cvt;
template <typename T> struct Cvt<T, T> {
  static __device__ __forceinline__ void store(T* lds, const uint4& r) { *reinterpret_cast<uint4*>(lds) = r; }
};
template <> struct Cvt<float, bf16> {
  // 4 floats -> 4 bf16 (8 bytes)
  static __device__ __forceinline__ void store(bf16* lds, const uint4& r) {
    const float* f = reinterpret_cast<const float*>(&r);
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    bf16x4_t o;
    o[0] = (bf16)f[0]; o[1] = (bf16)f[1]; o[2] = (bf16)f[2]; o[3] = (bf16)f[3];
    *reinterpret_cast<bf16x4_t*>(lds) = o;
  }
};

// Global -> register staging of a ROWS x BK tile of TA, stored to LDS as T.
// Chunk c is row c / CPR, columns (c % CPR) * EPA.  Rows >= rows_valid and
// columns >= cols_valid (the end of the K segment, a multiple of EPA) are
// never read and stage zeros.
template <typename TA, typename T, int ROWS>
struct TileLoader {
  static constexpr int BK = TileCfg<T>::BK;
  static constexpr int EPA = 16 / sizeof(TA);
  static constexpr int CPR = BK / EPA;
  static constexpr int CHUNKS = ROWS * CPR;
  static_assert(CHUNKS % 256 == 0, "tile must split evenly over 256 threads");
  static constexpr int PER = CHUNKS / 256;
  uint4 r[PER];

  __device__ __forceinline__ void load(const TA* base, int ld, int rows_valid, int k0, int cols_valid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * 256;
      const int row = c / CPR;
      const int col = (c % CPR) * EPA;
      if (row < rows_valid && k0 + col < cols_valid)
        r[i] = *reinterpret_cast<const uint4*>(base + (size_t)row * ld + k0 + col);
      else
        r[i] = make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __device__ __forceinline__ void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * 256;
      const int row = c / CPR;
      const int col = (c % CPR) * EPA;
      Cvt<TA, T>::store(lds + row * TileCfg<T>::STRIDE + col, r[i]);
    }
  }
};

// One BK step of a wave's WM x WN sub-tile from LDS.  The product is formed
// transposed (W-block x A-block^T), so in acc[i][j] lane l holds output row
// i * 16 + (l & 15) and the 4 consecutive output columns j * 16 + 4 * (l >> 4) + r:
// every lane owns 4 contiguous elements of one output row.
template <typename T, int WM, int WN>
__device__ __forceinline__ void mma_tile(const T* sA, const T* sB, int lane, f32x4 (&acc)[WM / 16][WN / 16]) {
  using MF = Mfma<T>;
  constexpr int S = TileCfg<T>::STRIDE;
  constexpr int BK = TileCfg<T>::BK;
  const int r = lane & 15, kq = MF::KV * (lane >> 4);
#pragma unroll
  for (int ks = 0; ks < BK / MF::K; ++ks) {
    typename MF::frag a[WM / 16], b[WN / 16];
#pragma unroll
    for (int i = 0; i < WM / 16; ++i) a[i] = MF::load(sA + (i * 16 + r) * S + ks * MF::K + kq);
#pragma unroll
    for (int j = 0; j < WN / 16; ++j) b[j] = MF::load(sB + (j * 16 + r) * S + ks * MF::K + kq);
#pragma unroll
    for (int i = 0; i < WM / 16; ++i)
#pragma unroll
      for (int j = 0; j < WN / 16; ++j) acc[i][j] = MF::mma(b[j], a[i], acc[i][j]);
  }
}

// Shared main loop: accumulates the block's BM x BN tile of [a1|a2] [w1|w2]^T.
// Segment 1 of A is stored as TA (fp32 for the residual stream), segment 2 as T.
template <typename TA, typename T, int BM, int BN, int WM, int WN>
__device__ __forceinline__ void gemm_mainloop(const TA* a1, int lda1, const T* w1, int k1, const T* a2, int lda2,
                                              const T* w2, int k2, int M, int m0, int n0, T* sA, T* sB,
                                              f32x4 (&acc)[WM / 16][WN / 16]) {
  constexpr int S = TileCfg<T>::STRIDE;
  constexpr int BK = TileCfg<T>::BK;
  constexpr int WAVES_N = BN / WN;
  constexpr bool kSameA = sizeof(TA) == sizeof(T);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  // Each K segment is tiled on its own (a segment's last tile may be partial).
  const int KT1 = (k1 + BK - 1) / BK;
  const int KT = KT1 + (k2 + BK - 1) / BK;
  const int rows_a = M - m0;

#pragma unroll
  for (int i = 0; i < WM / 16; ++i)
#pragma unroll
    for (int j = 0; j < WN / 16; ++j) acc[i][j] = zero4();

  TileLoader<TA, T, BM> la1;
  TileLoader<T, T, BM> la2;
  TileLoader<T, T, BN> lb;
  auto load_k = [&](int kt) {
    if (kt < KT1) {
      const int k = kt * BK;
      la1.load(a1 + (size_t)m0 * lda1, lda1, rows_a, k, k1);
      lb.load(w1 + (size_t)n0 * k1, k1, BN, k, k1);
    } else {
      const int k = (kt - KT1) * BK;
      if constexpr (kSameA)
        la1.load(reinterpret_cast<const TA*>(a2) + (size_t)m0 * lda2, lda2, rows_a, k, k2);
      else
        la2.load(a2 + (size_t)m0 * lda2, lda2, rows_a, k, k2);
      lb.load(w2 + (size_t)n0 * k2, k2, BN, k, k2);
    }
  };
  auto store_a = [&](int kt, T* dst) {
    if (kSameA || kt < KT1) la1.store(dst);
    else la2.store(dst);
  };

  load_k(0);
  store_a(0, sA);
  lb.store(sB);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) load_k(kt + 1);
    mma_tile<T, WM, WN>(sA + cur * BM * S + wm * WM * S, sB + cur * BN * S + wn * WN * S, lane, acc);
    if (kt + 1 < KT) {
      store_a(kt + 1, sA + (cur ^ 1) * BM * S);
      lb.store(sB + (cur ^ 1) * BN * S);
    }
    __syncthreads();
  }
}

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + __expf(-z)); }

// 4 consecutive outputs as one 16-byte (fp32) or 8-byte (bf16) store.
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(bf16* p, const float (&v)[4]) {
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  bf16x4_t o;
  o[0] = (bf16)v[0]; o[1] = (bf16)v[1]; o[2] = (bf16)v[2]; o[3] = (bf16)v[3];
  *reinterpret_cast<bf16x4_t*>(p) = o;
}

}  // namespace

// ---------------------------------------------------------------------------
template <typename TA, typename T, typename TO, int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs<TA, T, TO> p) {
  constexpr int S = TileCfg<T>::STRIDE;
  __shared__ __attribute__((aligned(16))) T smem[2 * (BM + BN) * S];
  T* sA = smem;
  T* sB = smem + 2 * BM * S;
  // 1-D grid over (row tile, column tile), column tiles fastest, remapped so
  // that the column tiles of one row tile (which share its A rows) share an XCD.
  const int nt = p.N / BN;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / nt) * BM, n0 = (tile % nt) * BN;
  f32x4 acc[WM / 16][WN / 16];
  gemm_mainloop<TA, T, BM, BN, WM, WN>(p.a1, p.lda1, p.w1, p.k1, p.a2, p.lda2, p.w2, p.k2, p.M, m0, n0, sA, sB, acc);

  // bias + activation; each lane stores 4 contiguous outputs of one row
  constexpr int WAVES_N = BN / WN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
#pragma unroll
  for (int j = 0; j < WN / 16; ++j) {
    const int n = n0 + wn * WN + j * 16 + 4 * (lane >> 4);
    float b[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) b[r] = to_f32(p.bias[n + r]);
#pragma unroll
    for (int i = 0; i < WM / 16; ++i) {
      const int m = m0 + wm * WM + i * 16 + (lane & 15);
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        v[r] = acc[i][j][r] + b[r];
        if (EPI == EPI_BIAS && n < p.scale_cols) v[r] *= p.col_scale;
        if (EPI == EPI_RELU) v[r] = fmaxf(v[r], 0.f);
        if (EPI == EPI_SIGMOID) v[r] = sigmoidf_(v[r]);
      }
      if (m < p.M) store4(p.out + (size_t)m * p.ldo + n, v);
    }
  }
}

template <typename TA, typename T, typename TO, int BM, int BN, int WM, int WN>
static hipError_t launch_gemm_cfg(const GemmArgs<TA, T, TO>& a, int epi, hipStream_t s) {
  dim3 grid((a.N / BN) * ((a.M + BM - 1) / BM)), block(256);
  switch (epi) {
    case EPI_BIAS: hipLaunchKernelGGL((k_gemm<TA, T, TO, BM, BN, WM, WN, EPI_BIAS>), grid, block, 0, s, a); break;
    case EPI_RELU: hipLaunchKernelGGL((k_gemm<TA, T, TO, BM, BN, WM, WN, EPI_RELU>), grid, block, 0, s, a); break;
    case EPI_SIGMOID:
      hipLaunchKernelGGL((k_gemm<TA, T, TO, BM, BN, WM, WN, EPI_SIGMOID>), grid, block, 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename TA, typename T, typename TO>
hipError_t launch_gemm(const GemmArgs<TA, T, TO>& a, int epi, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  // K segments must be whole 16-byte chunks of both A and W (callers pass multiples of 32).
  if (a.k1 <= 0 || a.k1 % 8 || a.k2 < 0 || a.k2 % 8 || (a.k2 > 0 && (!a.a2 || !a.w2))) return hipErrorInvalidValue;
  if (a.N % 128 == 0) return launch_gemm_cfg<TA, T, TO, 128, 128, 64, 64>(a, epi, s);
  if (a.N % 64 == 0) return launch_gemm_cfg<TA, T, TO, 128, 64, 64, 32>(a, epi, s);
  return hipErrorInvalidValue;
}
template hipError_t launch_gemm<float, float, float>(const GemmArgs<float, float, float>&, int, hipStream_t);
template hipError_t launch_gemm<bf16, bf16, bf16>(const GemmArgs<bf16, bf16, bf16>&, int, hipStream_t);
template hipError_t launch_gemm<float, bf16, bf16>(const GemmArgs<float, bf16, bf16>&, int, hipStream_t);
template hipError_t launch_gemm<bf16, bf16, float>(const GemmArgs<bf16, bf16, float>&, int, hipStream_t);
template hipError_t launch_gemm<float, bf16, float>(const GemmArgs<float, bf16, float>&, int, hipStream_t);

}  // namespace gdp
