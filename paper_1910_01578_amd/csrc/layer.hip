// Section 3.2: everything of a placer layer that follows its attention, and
// the start of the next layer, fused over blocks of 128 rows (nodes):
//
//   Z    = LN1( Y + O W_o^T + b_o )                           phase 0
//   Y'   = FiLM_{l+1}( LN2( Z + W_2 ReLU(W_1 Z + b_1) + b_2 ) )  FFN
//   QKV' = Y' W_qkv'^T + b_qkv'           (when a next layer exists)
//
// Every step is row-local, so a work-group (8 waves) owns 128 rows and the
// whole d-wide row.  Z and the d_ff hidden layer never leave the chip; Y is
// read once (as the residual) and Y' written once.  Two register tilings are
// used, both with the product formed transposed (weights x activations^T) so
// that a lane holds 4 consecutive columns of one row:
//   "unit" tiling   wave = 32 rows (16 in fp32) x a share of FC output units,
//                   its rows of the activation held in registers as MFMA
//                   fragments; each weight fragment read from LDS feeds 2 (1)
//                   MFMAs.  Used for W_1 and W_qkv.
//   "row" tiling    2 x 4 waves of 64 rows x d/4 columns accumulating the
//                   d-wide output; both operands from LDS, each fragment read
//                   feeds 4 MFMAs.  Used for W_o and W_2; the accumulator
//                   holds Y + b_o, then Z, then Z + FFN(Z), so both
//                   residuals come for free.
// Weights stream through double-buffered LDS in chunks of FC units (K steps
// of FC for W_o and W_2), chunk c+1 travelling global -> registers while
// chunk c is multiplied.  Switching from the row tiling to the unit tiling
// passes the activation through LDS once (as the MFMA element type).
#include "device_common.h"
#include "kernels.h"

namespace gdp {

namespace {

constexpr int LBM = 128;       // rows per work-group
constexpr int kLayerWaves = 8;
constexpr int LNT = 64 * kLayerWaves;

// Units per chunk and unit-tiling row blocks per wave: 64 and 2 for bf16; 32
// and 1 for fp32, so that the weight buffers of a d = 256 layer fit in LDS
// and the fp32 activation fragments in registers.
template <typename T> struct LayerCfg { static constexpr int FC = 64, RB1 = 2; };
template <> struct LayerCfg<float> { static constexpr int FC = 32, RB1 = 1; };

// Register staging of a ROWS x COLS block of a row-major matrix (leading
// dimension ld), written to LDS with row stride S.  Rows >= rows_valid are
// not read and stage zeros.  Held as 32-bit words: an array of 16-byte vectors
// that stays live across barriers is kept in scratch memory by the compiler.
template <typename T, int ROWS, int COLS, int S>
struct Stage {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int CPR = COLS / EPV;
  static constexpr int CHUNKS = ROWS * CPR;
  static_assert(CHUNKS % LNT == 0, "block must split evenly over the work-group");
  static constexpr int PER = CHUNKS / LNT;
  uint32_t r[4 * PER];
  __device__ __forceinline__ void load(const T* base, size_t ld, int rows_valid = ROWS) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = threadIdx.x + i * LNT;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (q / CPR < rows_valid) v = *reinterpret_cast<const uint4*>(base + (size_t)(q / CPR) * ld + (q % CPR) * EPV);
      r[4 * i] = v.x;
      r[4 * i + 1] = v.y;
      r[4 * i + 2] = v.z;
      r[4 * i + 3] = v.w;
    }
  }
  __device__ __forceinline__ void store_piece(T* lds, int i) const {
    const int q = threadIdx.x + i * LNT;
    *reinterpret_cast<uint4*>(lds + (q / CPR) * S + (q % CPR) * EPV) =
        make_uint4(r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]);
  }
  __device__ __forceinline__ void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) store_piece(lds, i);
  }
};

// FC biases of a chunk: 16-byte pieces held by the first FC / EPV threads,
// staged to LDS with the chunk's weights (so that reading them never waits
// on global memory, which would include the next chunk's prefetch).
template <typename T, int FC>
struct BiasStage {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int THREADS = FC / EPV;
  uint4 r = make_uint4(0u, 0u, 0u, 0u);
  __device__ __forceinline__ void load(const T* b) {
    if (threadIdx.x < THREADS) r = *reinterpret_cast<const uint4*>(b + threadIdx.x * EPV);
  }
  __device__ __forceinline__ void store(T* lds) const {
    if (threadIdx.x < THREADS) *reinterpret_cast<uint4*>(lds + threadIdx.x * EPV) = r;
  }
};

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v = {(bf16)lo, (bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// 4 consecutive elements of T read as one vector and widened.
__device__ __forceinline__ void load4f(const float* p, float (&v)[4]) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
__device__ __forceinline__ void load4f(const bf16* p, float (&v)[4]) {
  const uint2 x = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(x.x << 16); v[1] = __uint_as_float(x.x & 0xffff0000u);
  v[2] = __uint_as_float(x.y << 16); v[3] = __uint_as_float(x.y & 0xffff0000u);
}

// 4 consecutive values as one store (8 bytes in bf16, 16 in fp32).
__device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(bf16* p, const float (&v)[4]) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2_bf16(v[0], v[1]), pack2_bf16(v[2], v[3]));
}

// Tile geometry and the LDS carve shared by all phases.  The phases use the
// memory one after another, so their regions overlap:
//   phase 0   O chunks [2][LBM x SH], W_o chunks [2][d x S2]
//   FFN       W_1 chunks [2][FC x S1], W_2 chunks [2][d x S2], H [LBM x SH], b_1 [2][FC]
//   switch    activation [LBM x SZ] (MFMA type)
//   QKV       W_qkv chunks [2][FC x S1], b_qkv [2][FC]
// plus the LayerNorm partial sums red[LBM][WN2] behind all of them.
template <typename T, int D>
struct Geo {
  using MF = Mfma<T>;
  static constexpr int FC = LayerCfg<T>::FC;
  static constexpr int RB1 = LayerCfg<T>::RB1;
  static constexpr int P1M = LBM / (16 * RB1);    // unit tiling: P1M row groups x P1N unit groups
  static constexpr int P1N = kLayerWaves / P1M;
  static constexpr int HPW = FC / P1N;            // units per wave and chunk
  static constexpr int JB1 = HPW / 16;
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int S1 = D + EPV;              // unit-tiling weight rows: K = d
  static constexpr int S2 = FC + EPV;             // row-tiling weight rows: K = FC
  static constexpr int SH = FC + EPV;             // row-tiling activation chunk rows
  static constexpr int SZ = D + EPV;              // activation rows at the switch
  static constexpr int KS1 = D / MF::K;
  static constexpr int KS2 = FC / MF::K;
  static constexpr int WM2 = 2, WN2 = 4;          // row tiling
  static constexpr int MB2 = LBM / WM2 / 16;
  static constexpr int NB2 = D / WN2 / 16;
  static_assert(P1M * P1N == kLayerWaves && JB1 >= 1 && NB2 >= 1, "wave grids");
  static_assert(D % FC == 0, "d must be a multiple of the chunk");
  typedef f32x4 UnitAcc[RB1][JB1];                       // unit-tiling accumulators
  typedef f32x4 RowAcc[MB2][NB2];                        // row-tiling accumulators
  typedef typename MF::frag ActFrags[RB1][KS1];          // unit-tiling activation fragments
  typedef float Red[WN2];

  static constexpr int W1B = FC * S1 * sizeof(T);
  static constexpr int W2B = D * S2 * sizeof(T);
  static constexpr int HB = LBM * SH * sizeof(T);
  static constexpr int BB = FC * sizeof(T);
  // FFN carve
  static constexpr int OFF_W1 = 0, OFF_W2 = 2 * W1B, OFF_H = OFF_W2 + 2 * W2B, OFF_B1 = OFF_H + HB;
  static constexpr int FFN_END = OFF_B1 + 2 * BB;
  // phase-0 carve: O chunks first, then the W_o chunks
  static constexpr int OFF_O = 0, OFF_WO = 2 * HB;
  static constexpr int P0_END = OFF_WO + 2 * W2B;
  // switch
  static constexpr int SW_END = LBM * SZ * (int)sizeof(T);
  static constexpr int mx(int a, int b) { return a > b ? a : b; }
  static constexpr int OFF_RED = (mx(mx(FFN_END, P0_END), SW_END) + 15) / 16 * 16;
  static constexpr int TOTAL = OFF_RED + LBM * WN2 * (int)sizeof(float);
  static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

// Per-lane position in the two tilings.
struct Lanes {
  int lane, wave, col, g4;
  int p1m, p1n;        // unit tiling
  int w2m, w2n;        // row tiling
};

// unit tiling: hacc[i][j] = W_c(rows p1n*HPW + j*16 + ..) x act(rows (p1m*RB1 + i)*16 + ..)^T.
// after_step(s) runs after the MFMAs of k step s have been issued: other
// work placed there executes while they are in the matrix pipe.
template <typename T, int D, typename Hook>
__device__ __forceinline__ void unit_mma(typename Geo<T, D>::UnitAcc& hacc, const typename Geo<T, D>::ActFrags& af,
                                         const T* sW, const Lanes& ln, Hook&& after_step) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
#pragma unroll
  for (int i = 0; i < G::RB1; ++i)
#pragma unroll
    for (int j = 0; j < G::JB1; ++j) hacc[i][j] = zero4();
#pragma unroll
  for (int s = 0; s < G::KS1; ++s) {
#pragma unroll
    for (int j = 0; j < G::JB1; ++j) {
      const typename MF::frag bw = MF::load(&sW[(ln.p1n * G::HPW + j * 16 + ln.col) * G::S1 + s * MF::K + MF::KV * ln.g4]);
#pragma unroll
      for (int i = 0; i < G::RB1; ++i) hacc[i][j] = MF::mma(bw, af[i][s], hacc[i][j]);
    }
    after_step(s);
  }
}
template <typename T, int D>
__device__ __forceinline__ void unit_mma(typename Geo<T, D>::UnitAcc& hacc, const typename Geo<T, D>::ActFrags& af,
                                         const T* sW, const Lanes& ln) {
  unit_mma<T, D>(hacc, af, sW, ln, [](int) {});
}

// row tiling: acc += A_c W_c^T with A_c = sA rows [LBM x FC] (stride SH), W_c = sW rows [d x FC] (stride S2)
template <typename T, int D>
__device__ __forceinline__ void row_mma(typename Geo<T, D>::RowAcc& acc, const T* sA, const T* sW, const Lanes& ln) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
#pragma unroll
  for (int s = 0; s < G::KS2; ++s) {
    typename MF::frag af[G::MB2], bf[G::NB2];
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
      af[i] = MF::load(&sA[(ln.w2m * G::MB2 * 16 + i * 16 + ln.col) * G::SH + s * MF::K + MF::KV * ln.g4]);
#pragma unroll
    for (int j = 0; j < G::NB2; ++j)
      bf[j] = MF::load(&sW[(ln.w2n * G::NB2 * 16 + j * 16 + ln.col) * G::S2 + s * MF::K + MF::KV * ln.g4]);
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) acc[i][j] = MF::mma(bf[j], af[i], acc[i][j]);
  }
}

// LayerNorm (eps 1e-5, biased variance) of every row held in the row tiling,
// in place: in-lane partial sums, the 4 lane groups of a row (xor 16, 32),
// then the WN2 column waves through LDS; two passes (mean, centred second moment).
template <typename T, int D>
__device__ __forceinline__ void ln_rows(typename Geo<T, D>::RowAcc& acc, const T* gamma, const T* beta,
                                        typename Geo<T, D>::Red* red, const Lanes& ln) {
  using G = Geo<T, D>;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  float mean[G::MB2], rstd[G::MB2];
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) sum += (acc[i][j][0] + acc[i][j][1]) + (acc[i][j][2] + acc[i][j][3]);
    sum += xor_shfl(sum, 16);
    sum += xor_shfl(sum, 32);
    if (ln.g4 == 0) red[rbase + i * 16][ln.w2n] = sum;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < G::WN2; ++q) sum += red[rbase + i * 16][q];
    mean[i] = sum * (1.0f / D);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float dl = acc[i][j][r] - mean[i];
        sum += dl * dl;
      }
    sum += xor_shfl(sum, 16);
    sum += xor_shfl(sum, 32);
    if (ln.g4 == 0) red[rbase + i * 16][ln.w2n] = sum;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < G::WN2; ++q) sum += red[rbase + i * 16][q];
    rstd[i] = rsqrtf(sum * (1.0f / D) + 1e-5f);
  }
#pragma unroll
  for (int j = 0; j < G::NB2; ++j) {
    float gm[4], bt[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      gm[r] = to_f32(gamma[cbase + j * 16 + r]);
      bt[r] = to_f32(beta[cbase + j * 16 + r]);
    }
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = (acc[i][j][r] - mean[i]) * rstd[i] * gm[r] + bt[r];
  }
}

// Row tiling -> unit tiling: the activation in acc goes to LDS as T, and each
// wave reads back its unit-tiling rows as MFMA fragments.  Ends with a
// barrier after which the LDS is free again.
template <typename T, int D>
__device__ __forceinline__ void to_unit_tiling(const typename Geo<T, D>::RowAcc& acc, T* sZ,
                                               typename Geo<T, D>::ActFrags& af, const Lanes& ln) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i)
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      store4(&sZ[(rbase + i * 16) * G::SZ + cbase + j * 16], v);
    }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < G::RB1; ++i)
#pragma unroll
    for (int s = 0; s < G::KS1; ++s)
      af[i][s] = MF::load(&sZ[((ln.p1m * G::RB1 + i) * 16 + ln.col) * G::SZ + s * MF::K + MF::KV * ln.g4]);
  __syncthreads();
}

// QKV = act W_qkv^T + b_qkv for the work-group's rows, chunks of FC output
// units, with the activation in the row tiling in acc (it passes to the unit
// tiling through LDS; every LDS region must be free on entry).  The q columns
// are multiplied by q_scale.  Two register sets alternate so that chunk q + 2
// is requested while chunk q is multiplied.
template <typename T, int D>
__device__ __forceinline__ void qkv_phase(const typename Geo<T, D>::RowAcc& acc, char* smem,
                                          typename Geo<T, D>::ActFrags& af, const Lanes& ln, int m0, int M,
                                          const T* w_qkv, const T* b_qkv, T* qkv_out, int ldq, float q_scale) {
  using G = Geo<T, D>;
  constexpr int FC = G::FC;
  T* sW1 = reinterpret_cast<T*>(smem + G::OFF_W1);
  T* sB = reinterpret_cast<T*>(smem + G::OFF_B1);
  {
    Stage<T, FC, D, G::S1> stA, stB;
    BiasStage<T, FC> sbA, sbB;
    constexpr int NQ = 3 * D / FC;
    stA.load(w_qkv, D);
    sbA.load(b_qkv);
    if (NQ > 1) {
      stB.load(w_qkv + (size_t)FC * D, D);
      sbB.load(b_qkv + FC);
    }
    to_unit_tiling<T, D>(acc, reinterpret_cast<T*>(smem), af, ln);
    stA.store(sW1);
    sbA.store(sB);
    __syncthreads();
    // chunk q: weights in buffer q & 1; `next` holds chunk q + 1, `mine` is free
    auto step = [&](int q, Stage<T, FC, D, G::S1>& mine, BiasStage<T, FC>& mine_b, Stage<T, FC, D, G::S1>& next,
                    BiasStage<T, FC>& next_b) {
      const int cur = q & 1;
      typename G::UnitAcc hacc;
      unit_mma<T, D>(hacc, af, sW1 + cur * FC * G::S1, ln);
      if (q + 1 < NQ) {
        next.store(sW1 + (cur ^ 1) * FC * G::S1);   // last read in chunk q - 1
        next_b.store(sB + (cur ^ 1) * FC);
      }
      if (q + 2 < NQ) {
        mine.load(w_qkv + (size_t)(q + 2) * FC * D, D);
        mine_b.load(b_qkv + (q + 2) * FC);
      }
      const float scale = q * FC < D ? q_scale : 1.0f;   // a chunk lies wholly in q, k or v
#pragma unroll
      for (int j = 0; j < G::JB1; ++j) {
        const int hc = ln.p1n * G::HPW + j * 16 + 4 * ln.g4;
        float b[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) b[r] = to_f32(sB[cur * FC + hc + r]);
#pragma unroll
        for (int i = 0; i < G::RB1; ++i) {
          const int row = m0 + (ln.p1m * G::RB1 + i) * 16 + ln.col;
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = (hacc[i][j][r] + b[r]) * scale;
          if (row < M) store4(qkv_out + (size_t)row * ldq + q * FC + hc, v);
        }
      }
      __syncthreads();                 // this chunk's buffers free
    };
    for (int q = 0; q < NQ; q += 2) {
      step(q, stA, sbA, stB, sbB);
      if (q + 1 < NQ) step(q + 1, stB, sbB, stA, sbA);
    }
  }
}


// The placement head on the rows held in the row tiling (Fig. 1's N x d
// output): logits[row][e] = act[row] . W_out[e] + b_out[e] for e < n_dev <=
// kFusedHeadDevices, and their logsumexp.  W_out goes to LDS as fp32; each
// lane forms the partial sums of its rows over its columns, the 4 lane groups
// of a row combine by butterfly and the WN2 column waves through LDS.  Every
// LDS region must be free on entry.
template <typename T, int D>
__device__ __forceinline__ void head_epilogue(const typename Geo<T, D>::RowAcc& acc, char* smem, const Lanes& ln,
                                              int m0, int M, const T* w_out, const T* b_out, int n_dev,
                                              float* logits, float* lse) {
  using G = Geo<T, D>;
  constexpr int E = kFusedHeadDevices;
  float* sW = reinterpret_cast<float*>(smem);                                  // [E][D]
  float (*hred)[G::WN2][E] = reinterpret_cast<float (*)[G::WN2][E]>(smem + E * D * sizeof(float));
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  for (int i = threadIdx.x; i < E * D; i += LNT) sW[i] = i < n_dev * D ? to_f32(w_out[i]) : 0.f;
  __syncthreads();
  float part[G::MB2][E];
#pragma unroll
  for (int i = 0; i < G::MB2; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) part[i][e] = 0.f;
#pragma unroll
  for (int j = 0; j < G::NB2; ++j)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float4 w = *reinterpret_cast<const float4*>(&sW[e * D + cbase + j * 16]);
#pragma unroll
      for (int i = 0; i < G::MB2; ++i)
        part[i][e] += acc[i][j][0] * w.x + acc[i][j][1] * w.y + acc[i][j][2] * w.z + acc[i][j][3] * w.w;
    }
#pragma unroll
  for (int i = 0; i < G::MB2; ++i)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float v = part[i][e];
      v += xor_shfl(v, 16);
      v += xor_shfl(v, 32);
      if (ln.g4 == 0) hred[rbase + i * 16][ln.w2n][e] = v;
    }
  __syncthreads();
  if (threadIdx.x < LBM) {
    const int row = m0 + threadIdx.x;
    if (row < M) {
      float l[E], mx = -INFINITY;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        float v = 0.f;
#pragma unroll
        for (int q = 0; q < G::WN2; ++q) v += hred[threadIdx.x][q][e];
        l[e] = e < n_dev ? v + to_f32(b_out[e < n_dev ? e : 0]) : -INFINITY;
        mx = fmaxf(mx, l[e]);
      }
      float sum = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (e < n_dev) {
          sum += expf(l[e] - mx);
          logits[(size_t)row * n_dev + e] = l[e];
        }
      lse[row] = mx + logf(sum);
    }
  }
}

}  // namespace

// HEAD: the last layer's variant, with the placement head instead of a QKV projection.
template <typename T, int D, bool HEAD>
__global__ __launch_bounds__(LNT) void k_post_attention(PostAttnArgs<T> p, GraphTable gt) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
  constexpr int FC = G::FC;
  __shared__ __attribute__((aligned(16))) char smem[G::TOTAL];
  typename G::Red* red = reinterpret_cast<typename G::Red*>(smem + G::OFF_RED);

  Lanes ln;
  ln.lane = threadIdx.x & 63;
  ln.wave = threadIdx.x >> 6;
  ln.col = ln.lane & 15;
  ln.g4 = ln.lane >> 4;
  ln.p1m = ln.wave / G::P1N;
  ln.p1n = ln.wave % G::P1N;
  ln.w2m = ln.wave / G::WN2;
  ln.w2n = ln.wave % G::WN2;
  const int m0 = blockIdx.x * LBM;
  const int rows_valid = p.M - m0;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;      // row tiling: rows rbase + 16 i
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;   //             columns cbase + 16 j + [0, 4)

  // ---- phase 0: acc = Y + b_o + O W_o^T, then LN1 --------------------------
  typename G::RowAcc acc;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      const int cn = cbase + j * 16;
      float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < p.M) y = *reinterpret_cast<const float4*>(p.y + (size_t)row * p.ldy + cn);
      acc[i][j][0] = y.x + to_f32(p.b_o[cn + 0]);
      acc[i][j][1] = y.y + to_f32(p.b_o[cn + 1]);
      acc[i][j][2] = y.z + to_f32(p.b_o[cn + 2]);
      acc[i][j][3] = y.w + to_f32(p.b_o[cn + 3]);
    }
  }
  {
    T* sO = reinterpret_cast<T*>(smem + G::OFF_O);       // [2][LBM * SH]
    T* sWo = reinterpret_cast<T*>(smem + G::OFF_WO);     // [2][D * S2]
    Stage<T, LBM, FC, G::SH> so;
    Stage<T, D, FC, G::S2> sw;
    constexpr int NK = D / FC;
    so.load(p.o + (size_t)m0 * p.ldo, p.ldo, rows_valid);
    sw.load(p.w_o, D);
    so.store(sO);
    sw.store(sWo);
    __syncthreads();
    for (int kc = 0; kc < NK; ++kc) {
      const int cur = kc & 1;
      if (kc + 1 < NK) {
        so.load(p.o + (size_t)m0 * p.ldo + (kc + 1) * FC, p.ldo, rows_valid);
        sw.load(p.w_o + (kc + 1) * FC, D);
      }
      row_mma<T, D>(acc, sO + cur * LBM * G::SH, sWo + cur * D * G::S2, ln);
      if (kc + 1 < NK) {
        // the other buffers were last read in step kc - 1, before its barrier
        so.store(sO + (cur ^ 1) * LBM * G::SH);
        sw.store(sWo + (cur ^ 1) * D * G::S2);
      }
      __syncthreads();
    }
  }
  ln_rows<T, D>(acc, p.ln1_g, p.ln1_b, red, ln);       // acc = Z

  // ---- FFN: acc += W_2 ReLU(W_1 Z + b_1), chunks of FC hidden units ----------
  T* sW1 = reinterpret_cast<T*>(smem + G::OFF_W1);       // [2][FC * S1]
  T* sW2 = reinterpret_cast<T*>(smem + G::OFF_W2);       // [2][D * S2]
  T* sH = reinterpret_cast<T*>(smem + G::OFF_H);         // [LBM * SH]
  T* sB = reinterpret_cast<T*>(smem + G::OFF_B1);        // [2][FC]
  typename G::ActFrags af;
  {
    Stage<T, FC, D, G::S1> st1;
    Stage<T, D, FC, G::S2> st2;
    BiasStage<T, FC> sb;
    const int NC = p.d_ff / FC;
    st1.load(p.w1, D);
    st2.load(p.w2, p.d_ff);
    sb.load(p.b1);
    auto load_chunk = [&](int c) {
      st1.load(p.w1 + (size_t)c * FC * D, D);
      st2.load(p.w2 + (size_t)c * FC, p.d_ff);
      sb.load(p.b1 + c * FC);
    };
    to_unit_tiling<T, D>(acc, reinterpret_cast<T*>(smem), af, ln);
    st1.store(sW1);
    st2.store(sW2);
    sb.store(sB);
    if (NC > 1) load_chunk(1);
    __syncthreads();
    // Chunk c + 1 sits in registers from the start of the second product of
    // chunk c - 1 until after the first product of chunk c, so its global
    // latency hides under both.
    for (int c = 0; c < NC; ++c) {
      const int cur = c & 1;
      typename G::UnitAcc hacc;
      // Chunk c + 1 lands in the other buffers during the first product, one
      // 16-byte piece per thread after each k step: those buffers were last
      // read in chunk c - 1, before its final barrier.
      constexpr int P1 = decltype(st1)::PER, P2 = decltype(st2)::PER;
      const bool more = c + 1 < NC;
      T* n1 = sW1 + (cur ^ 1) * FC * G::S1;
      T* n2 = sW2 + (cur ^ 1) * D * G::S2;
      unit_mma<T, D>(hacc, af, sW1 + cur * FC * G::S1, ln, [&](int s) {
        if (!more) return;
#pragma unroll
        for (int k = (s * (P1 + P2)) / G::KS1; k < ((s + 1) * (P1 + P2)) / G::KS1; ++k) {
          if (k < P1) st1.store_piece(n1, k);
          else st2.store_piece(n2, k - P1);
        }
      });
      if (more) sb.store(sB + (cur ^ 1) * FC);
      // lane holds hidden row (p1m * RB1 + i) * 16 + col, units hc + [0, 4)
#pragma unroll
      for (int j = 0; j < G::JB1; ++j) {
        const int hc = ln.p1n * G::HPW + j * 16 + 4 * ln.g4;
        float b[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) b[r] = to_f32(sB[cur * FC + hc + r]);
#pragma unroll
        for (int i = 0; i < G::RB1; ++i) {
          float h[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) h[r] = fmaxf(hacc[i][j][r] + b[r], 0.f);
          store4(&sH[((ln.p1m * G::RB1 + i) * 16 + ln.col) * G::SH + hc], h);
        }
      }
      __syncthreads();                 // H and chunk c + 1 complete
      if (c + 2 < NC) load_chunk(c + 2);
      row_mma<T, D>(acc, sH, sW2 + cur * D * G::S2, ln);
      __syncthreads();                 // H and this chunk's buffers free
    }
  }

  // ---- + b_2, LN2, FiLM of the next layer; store Y' ---------------------------
#pragma unroll
  for (int j = 0; j < G::NB2; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float b = to_f32(p.b2[cbase + j * 16 + r]);
#pragma unroll
      for (int i = 0; i < G::MB2; ++i) acc[i][j][r] += b;
    }
  ln_rows<T, D>(acc, p.ln2_g, p.ln2_b, red, ln);
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    if (p.film_gamma) {
      const size_t g = (size_t)graph_of_node(gt, row < p.M ? row : p.M - 1) * p.film_stride;
#pragma unroll
      for (int j = 0; j < G::NB2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int cn = cbase + j * 16 + r;
          acc[i][j][r] = p.film_gamma[g + cn] * acc[i][j][r] + p.film_beta[g + cn];
        }
    }
    if (p.y_out && row < p.M) {
#pragma unroll
      for (int j = 0; j < G::NB2; ++j)
        *reinterpret_cast<float4*>(p.y_out + (size_t)row * p.ldyo + cbase + j * 16) =
            make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
  if constexpr (HEAD) {
    head_epilogue<T, D>(acc, smem, ln, m0, p.M, p.w_out, p.b_out, p.n_dev, p.logits, p.lse);
  } else {
    if (!p.w_qkv) return;
    qkv_phase<T, D>(acc, smem, af, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
  }
}

template <typename T>
hipError_t launch_post_attention(const PostAttnArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.d_ff <= 0 || a.d_ff % LayerCfg<T>::FC) return hipErrorInvalidValue;
  if (a.w_qkv && (!a.b_qkv || !a.qkv_out || a.ldq < 3 * a.d)) return hipErrorInvalidValue;
  if (a.w_out && (!a.b_out || !a.logits || !a.lse || a.n_dev < 1 || a.n_dev > kFusedHeadDevices || a.w_qkv))
    return hipErrorInvalidValue;
  dim3 grid((a.M + LBM - 1) / LBM), block(LNT);
  const bool head = a.w_out != nullptr;
  switch (a.d) {
    case 64:
      if (head) hipLaunchKernelGGL((k_post_attention<T, 64, true>), grid, block, 0, s, a, gt);
      else hipLaunchKernelGGL((k_post_attention<T, 64, false>), grid, block, 0, s, a, gt);
      break;
    case 128:
      if (head) hipLaunchKernelGGL((k_post_attention<T, 128, true>), grid, block, 0, s, a, gt);
      else hipLaunchKernelGGL((k_post_attention<T, 128, false>), grid, block, 0, s, a, gt);
      break;
    case 256:
      if (head) hipLaunchKernelGGL((k_post_attention<T, 256, true>), grid, block, 0, s, a, gt);
      else hipLaunchKernelGGL((k_post_attention<T, 256, false>), grid, block, 0, s, a, gt);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_post_attention<float>(const PostAttnArgs<float>&, const GraphTable&, hipStream_t);
template hipError_t launch_post_attention<bf16>(const PostAttnArgs<bf16>&, const GraphTable&, hipStream_t);


// The first placer layer's input and projection (Eq. 4, Section 3.2):
//   Y = FiLM_0(X) (X = the node embeddings; identity without conditioning) into
//   the fp32 residual stream, and QKV = Y W_qkv^T + b_qkv,
// with the same tiles as the post-attention kernel's QKV phase.
template <typename T, int D>
__global__ __launch_bounds__(LNT) void k_pre_layer(PreLayerArgs<T> p, GraphTable gt) {
  using G = Geo<T, D>;
  __shared__ __attribute__((aligned(16))) char smem[G::TOTAL];
  Lanes ln;
  ln.lane = threadIdx.x & 63;
  ln.wave = threadIdx.x >> 6;
  ln.col = ln.lane & 15;
  ln.g4 = ln.lane >> 4;
  ln.p1m = ln.wave / G::P1N;
  ln.p1n = ln.wave % G::P1N;
  ln.w2m = ln.wave / G::WN2;
  ln.w2n = ln.wave % G::WN2;
  const int m0 = blockIdx.x * LBM;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  typename G::RowAcc acc;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    const int rr = row < p.M ? row : p.M - 1;
    const float* fg = nullptr;
    const float* fb = nullptr;
    if (p.film_gamma) {
      const size_t g = (size_t)graph_of_node(gt, rr) * p.film_stride;
      fg = p.film_gamma + g;
      fb = p.film_beta + g;
    }
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      const int cn = cbase + j * 16;
      float x[4];
      load4f(p.x + (size_t)rr * p.ldx + cn, x);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = fg ? fg[cn + r] * x[r] + fb[cn + r] : x[r];
      if (row < p.M)
        *reinterpret_cast<float4*>(p.y_out + (size_t)row * p.ldyo + cn) =
            make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
    }
  }
  typename G::ActFrags af;
  qkv_phase<T, D>(acc, smem, af, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
}

template <typename T>
hipError_t launch_pre_layer(const PreLayerArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (!a.x || !a.y_out || !a.w_qkv || !a.b_qkv || !a.qkv_out || a.ldq < 3 * a.d) return hipErrorInvalidValue;
  dim3 grid((a.M + LBM - 1) / LBM), block(LNT);
  switch (a.d) {
    case 64: hipLaunchKernelGGL((k_pre_layer<T, 64>), grid, block, 0, s, a, gt); break;
    case 128: hipLaunchKernelGGL((k_pre_layer<T, 128>), grid, block, 0, s, a, gt); break;
    case 256: hipLaunchKernelGGL((k_pre_layer<T, 256>), grid, block, 0, s, a, gt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_pre_layer<float>(const PreLayerArgs<float>&, const GraphTable&, hipStream_t);
template hipError_t launch_pre_layer<bf16>(const PreLayerArgs<bf16>&, const GraphTable&, hipStream_t);

}  // namespace gdp
