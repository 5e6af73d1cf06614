// Section 3.2: the position-wise feed-forward half of a placer layer, fused:
//
//   Y' = FiLM_{l+1}( LN2( Z + W_2 ReLU(W_1 Z + b_1) + b_2 ) )
//
// One 512-thread work-group (8 waves) owns BM = 128 rows and the whole d-wide
// output row.  The d_ff hidden layer never leaves the chip: it is produced
// and consumed in chunks of FC = 64 hidden units (32 in fp32).
//   phase 1  H_c = ReLU(Z W1_c^T + b1_c)   [128 x FC], K = d
//            wave = 32 rows (16 in fp32) x its share of the chunk's units;
//            its rows of Z stay in registers as operand fragments for every
//            chunk, so each W1 fragment read from LDS feeds 2 (1) MFMAs.
//   phase 2  Out += H_c W2_c^T             [128 x d], K = FC
//            2 x 4 waves of 64 rows x d/4 columns: each fragment read feeds 4
//            MFMAs.
// Both products are formed transposed (weights x activations^T), so every
// lane ends up with 4 consecutive columns of one row: H is written to LDS and
// the output to memory as whole vectors, and LayerNorm's row sums are mostly
// in-lane.  W1_c, W2_c and b1_c sit in double-buffered LDS; chunk c+1
// travels global -> registers during phase 1 of chunk c.  Z (fp32, the residual
// stream) is read twice: as the operand and as the residual.
#include "device_common.h"
#include "kernels.h"

namespace gdp {

namespace {
constexpr int FBM = 128;       // rows per work-group
constexpr int kFfnWaves = 8;
constexpr int FNT = 64 * kFfnWaves;
// Hidden units per chunk and phase-1 row blocks per wave: 64 and 2 for bf16;
// 32 and 1 for fp32, so that the weight buffers of a d = 256 layer still fit
// in LDS and the fp32 Z fragments in registers.
template <typename T> struct FfnCfg { static constexpr int FC = 64, RB1 = 2; };
template <> struct FfnCfg<float> { static constexpr int FC = 32, RB1 = 1; };

// Register staging of a ROWS x COLS weight block, read from a row-major
// matrix with leading dimension ld and written to LDS with row stride S.
template <typename T, int ROWS, int COLS, int S>
struct WStage {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int CPR = COLS / EPV;
  static constexpr int CHUNKS = ROWS * CPR;
  static_assert(CHUNKS % FNT == 0, "weight block must split evenly over the work-group");
  static constexpr int PER = CHUNKS / FNT;
  // Held as 32-bit words: an array of 16-byte vectors that stays live across
  // the chunk loop's barriers is kept in scratch memory by the compiler.
  uint32_t r[4 * PER];
  __device__ __forceinline__ void load(const T* base, size_t ld) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = threadIdx.x + i * FNT;
      const uint4 v = *reinterpret_cast<const uint4*>(base + (size_t)(q / CPR) * ld + (q % CPR) * EPV);
      r[4 * i] = v.x;
      r[4 * i + 1] = v.y;
      r[4 * i + 2] = v.z;
      r[4 * i + 3] = v.w;
    }
  }
  __device__ __forceinline__ void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = threadIdx.x + i * FNT;
      *reinterpret_cast<uint4*>(lds + (q / CPR) * S + (q % CPR) * EPV) =
          make_uint4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
    }
  }
};

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v = {(bf16)lo, (bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// The MFMA A-operand fragment of row `zr` at k (KV consecutive fp32 values, rounded to T).
template <typename T> struct ZFrag;
template <> struct ZFrag<bf16> {
  static __device__ __forceinline__ bf16x8 load(const float* zr, int k) {
    const float4 a = *reinterpret_cast<const float4*>(zr + k);
    const float4 b = *reinterpret_cast<const float4*>(zr + k + 4);
    const uint4 u = make_uint4(pack2_bf16(a.x, a.y), pack2_bf16(a.z, a.w), pack2_bf16(b.x, b.y),
                               pack2_bf16(b.z, b.w));
    return __builtin_bit_cast(bf16x8, u);
  }
};
template <> struct ZFrag<float> {
  static __device__ __forceinline__ float load(const float* zr, int k) { return zr[k]; }
};

// 4 consecutive hidden units as one LDS store (8 bytes in bf16, 16 in fp32).
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(bf16* p, const float (&v)[4]) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]));
}
}  // namespace

template <typename T, int D>
__global__ __launch_bounds__(FNT) void k_ffn_fused(FfnArgs<T> p, GraphTable gt) {
  using MF = Mfma<T>;
  constexpr int FC = FfnCfg<T>::FC;
  constexpr int RB1 = FfnCfg<T>::RB1;       // phase-1 row blocks per wave
  constexpr int P1M = FBM / (16 * RB1);     // phase-1 wave grid: P1M row groups x P1N unit groups
  constexpr int P1N = kFfnWaves / P1M;
  constexpr int HPW = FC / P1N;             // hidden units per wave in phase 1
  constexpr int JB1 = HPW / 16;
  constexpr int EPV = 16 / sizeof(T);
  constexpr int S1 = D + EPV;               // sW1 row stride: W1_c rows (hidden units), K = d
  constexpr int S2 = FC + EPV;              // sW2 row stride: W2 rows (outputs), K = the chunk's units
  constexpr int SH = FC + EPV;              // sH row stride
  constexpr int KS1 = D / MF::K;
  constexpr int KS2 = FC / MF::K;
  constexpr int WM2 = 2, WN2 = 4;           // phase-2 wave grid
  constexpr int MB2 = FBM / WM2 / 16;       // row blocks per wave
  constexpr int NB2 = D / WN2 / 16;         // column blocks per wave
  static_assert(P1M * P1N == kFfnWaves && JB1 >= 1 && NB2 >= 1, "wave grids");
  __shared__ __attribute__((aligned(16))) T sW1[2][FC * S1];
  __shared__ __attribute__((aligned(16))) T sW2[2][D * S2];
  __shared__ __attribute__((aligned(16))) T sH[FBM * SH];
  __shared__ __attribute__((aligned(16))) T sB1[2][FC];
  __shared__ float red[FBM][WN2];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, g4 = lane >> 4;
  const int m0 = blockIdx.x * FBM;
  const int NC = p.d_ff / FC;

  // ---- this wave's phase-1 rows of Z as operand fragments -------------------
  const int p1m = wave / P1N, p1n = wave % P1N;
  typename MF::frag zf[RB1][KS1];
#pragma unroll
  for (int i = 0; i < RB1; ++i) {
    const int row = m0 + (p1m * RB1 + i) * 16 + col;
    const float* zr = p.z + (size_t)(row < p.M ? row : p.M - 1) * p.ldz;
#pragma unroll
    for (int s = 0; s < KS1; ++s) zf[i][s] = ZFrag<T>::load(zr, s * MF::K + MF::KV * g4);
  }
  const int w2m = wave / WN2, w2n = wave % WN2;

  // ---- weight staging: W1_c = W1 rows [c*FC, c*FC+FC) x d; W2_c = W2 rows 0..d x
  // columns [c*FC, c*FC+FC).  The chunk's FC biases travel with its weights
  // (16-byte pieces held by the first BCH threads) and are read from LDS, so
  // that no wait in phase 1 is a wait on global memory (which would include
  // the next chunk's prefetch).
  WStage<T, FC, D, S1> st1;
  WStage<T, D, FC, S2> st2;
  constexpr int BCH = FC / EPV;
  uint4 bst = make_uint4(0u, 0u, 0u, 0u);

  f32x4 oacc[MB2][NB2];
#pragma unroll
  for (int i = 0; i < MB2; ++i)
#pragma unroll
    for (int j = 0; j < NB2; ++j) oacc[i][j] = zero4();

  if (threadIdx.x < BCH) bst = *reinterpret_cast<const uint4*>(p.b1 + threadIdx.x * EPV);
  st1.load(p.w1, D);
  st2.load(p.w2, p.d_ff);
  st1.store(sW1[0]);
  st2.store(sW2[0]);
  if (threadIdx.x < BCH) *reinterpret_cast<uint4*>(&sB1[0][threadIdx.x * EPV]) = bst;
  __syncthreads();

  for (int c = 0; c < NC; ++c) {
    const int cur = c & 1;
    if (c + 1 < NC) {
      st1.load(p.w1 + (size_t)(c + 1) * FC * D, D);
      st2.load(p.w2 + (size_t)(c + 1) * FC, p.d_ff);
      if (threadIdx.x < BCH) bst = *reinterpret_cast<const uint4*>(p.b1 + (c + 1) * FC + threadIdx.x * EPV);
    }
    // phase 1: H_c on this wave's RB1 x 16 rows x HPW units
    f32x4 hacc[RB1][JB1];
#pragma unroll
    for (int i = 0; i < RB1; ++i)
#pragma unroll
      for (int j = 0; j < JB1; ++j) hacc[i][j] = zero4();
#pragma unroll
    for (int s = 0; s < KS1; ++s) {
#pragma unroll
      for (int j = 0; j < JB1; ++j) {
        const typename MF::frag bw = MF::load(&sW1[cur][(p1n * HPW + j * 16 + col) * S1 + s * MF::K + MF::KV * g4]);
#pragma unroll
        for (int i = 0; i < RB1; ++i) hacc[i][j] = MF::mma(bw, zf[i][s], hacc[i][j]);
      }
    }
    // Chunk c + 1 lands in the other buffers now: they were last read in
    // chunk c - 1, before its final barrier, and phase 2 needs no staging
    // registers this way.
    if (c + 1 < NC) {
      st1.store(sW1[cur ^ 1]);
      st2.store(sW2[cur ^ 1]);
      if (threadIdx.x < BCH) *reinterpret_cast<uint4*>(&sB1[cur ^ 1][threadIdx.x * EPV]) = bst;
    }
    // lane holds row (p1m * RB1 + i) * 16 + col and the 4 consecutive units hc + [0, 4)
#pragma unroll
    for (int j = 0; j < JB1; ++j) {
      const int hc = p1n * HPW + j * 16 + 4 * g4;
      float b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = to_f32(sB1[cur][hc + r]);
#pragma unroll
      for (int i = 0; i < RB1; ++i) {
        float h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) h[r] = fmaxf(hacc[i][j][r] + b[r], 0.f);
        store4(&sH[((p1m * RB1 + i) * 16 + col) * SH + hc], h);
      }
    }
    __syncthreads();                 // sH and chunk c + 1 complete

    // phase 2: Out += H_c W2_c^T on this wave's 64 rows x d/4 columns
#pragma unroll
    for (int s = 0; s < KS2; ++s) {
      typename MF::frag af[MB2], bf[NB2];
#pragma unroll
      for (int i = 0; i < MB2; ++i)
        af[i] = MF::load(&sH[(w2m * MB2 * 16 + i * 16 + col) * SH + s * MF::K + MF::KV * g4]);
#pragma unroll
      for (int j = 0; j < NB2; ++j)
        bf[j] = MF::load(&sW2[cur][(w2n * NB2 * 16 + j * 16 + col) * S2 + s * MF::K + MF::KV * g4]);
#pragma unroll
      for (int i = 0; i < MB2; ++i)
#pragma unroll
        for (int j = 0; j < NB2; ++j) oacc[i][j] = MF::mma(bf[j], af[i], oacc[i][j]);
    }
    __syncthreads();                 // sH and this chunk's buffers free
  }

  // ---- epilogue: + b2 + residual Z, LayerNorm over the d columns, FiLM ------
  // Lane holds row lrow(i) and the 4 consecutive columns ccol(j) + [0, 4).
  const int rbase = w2m * MB2 * 16 + col;
  const int cbase = w2n * NB2 * 16 + 4 * g4;
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    const int row = m0 + rbase + i * 16;
#pragma unroll
    for (int j = 0; j < NB2; ++j) {
      const int cn = cbase + j * 16;
      float4 res = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < p.M) res = *reinterpret_cast<const float4*>(p.z + (size_t)row * p.ldz + cn);
      oacc[i][j][0] += to_f32(p.b2[cn + 0]) + res.x;
      oacc[i][j][1] += to_f32(p.b2[cn + 1]) + res.y;
      oacc[i][j][2] += to_f32(p.b2[cn + 2]) + res.z;
      oacc[i][j][3] += to_f32(p.b2[cn + 3]) + res.w;
    }
  }
  // Row statistics: in-lane, across the 4 lane groups of a row, then the WN2 column waves.
  float mean[MB2], rstd[MB2];
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < NB2; ++j) sum += (oacc[i][j][0] + oacc[i][j][1]) + (oacc[i][j][2] + oacc[i][j][3]);
    sum += xor_shfl(sum, 16);
    sum += xor_shfl(sum, 32);
    if (g4 == 0) red[rbase + i * 16][w2n] = sum;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < WN2; ++q) sum += red[rbase + i * 16][q];
    mean[i] = sum * (1.0f / D);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < NB2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float dl = oacc[i][j][r] - mean[i];
        sum += dl * dl;
      }
    sum += xor_shfl(sum, 16);
    sum += xor_shfl(sum, 32);
    if (g4 == 0) red[rbase + i * 16][w2n] = sum;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < WN2; ++q) sum += red[rbase + i * 16][q];
    rstd[i] = rsqrtf(sum * (1.0f / D) + 1e-5f);
  }
#pragma unroll
  for (int i = 0; i < MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    const float* fg = nullptr;
    const float* fb = nullptr;
    if (p.film_gamma) {
      const size_t g = (size_t)graph_of_node(gt, row < p.M ? row : p.M - 1) * p.film_stride;
      fg = p.film_gamma + g;
      fb = p.film_beta + g;
    }
#pragma unroll
    for (int j = 0; j < NB2; ++j) {
      const int cn = cbase + j * 16;
      float y[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        y[r] = (oacc[i][j][r] - mean[i]) * rstd[i] * to_f32(p.ln_g[cn + r]) + to_f32(p.ln_b[cn + r]);
        if (fg) y[r] = fg[cn + r] * y[r] + fb[cn + r];
      }
      if (row < p.M) *reinterpret_cast<float4*>(p.out + (size_t)row * p.ldo + cn) = make_float4(y[0], y[1], y[2], y[3]);
    }
  }
}

template <typename T>
hipError_t launch_ffn_fused(const FfnArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.d_ff <= 0 || a.d_ff % FfnCfg<T>::FC) return hipErrorInvalidValue;
  dim3 grid((a.M + FBM - 1) / FBM), block(FNT);
  switch (a.d) {
    case 64: hipLaunchKernelGGL((k_ffn_fused<T, 64>), grid, block, 0, s, a, gt); break;
    case 128: hipLaunchKernelGGL((k_ffn_fused<T, 128>), grid, block, 0, s, a, gt); break;
    case 256: hipLaunchKernelGGL((k_ffn_fused<T, 256>), grid, block, 0, s, a, gt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_ffn_fused<float>(const FfnArgs<float>&, const GraphTable&, hipStream_t);
template hipError_t launch_ffn_fused<bf16>(const FfnArgs<bf16>&, const GraphTable&, hipStream_t);

}  // namespace gdp
