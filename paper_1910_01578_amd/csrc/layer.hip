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
//
// Operand staging.  Weights (and the attention output O) stream through LDS
// in chunks of FC units by direct global -> LDS loads (global_load_lds, 16
// bytes a lane): no registers hold a chunk in transit, which leaves them to
// prefetch the next k step's MFMA fragments from LDS.  Such a load writes the
// 64 lanes' 16-byte granules contiguously, so LDS tiles are unpadded and keep
// their rows' granules in XOR-permuted order (swz_key) so that the 16 rows
// read by one fragment load fall in distinct banks.  Chunk c + 1 is loaded
// during chunk c into the other buffer of a pair; each staging buffer is a
// __shared__ array of its own and the buffer parity of every step is a
// compile-time constant, so the compiler can tell which LDS reads depend on
// which load and waits for none that is still in flight.
#include "device_common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace gdp {

namespace {

using dma::gptr_t;
using dma::swz_key;
using dma::swz;
using dma::uniform_base;
using dma::dma16;
template <typename T, int ROWS, int COLS, int NW = 8>
using DmaTile = dma::DmaTile<T, ROWS, COLS, NW>;

constexpr int LBM = 128;       // rows per work-group
constexpr int kLayerWaves = 8;
constexpr int LNT = 64 * kLayerWaves;

// Units per chunk and unit-tiling row blocks per wave: 64 and 2 for bf16; 32
// and 1 for fp32, so that the staging buffers of a d = 256 layer fit in LDS
// and the fp32 activation fragments in registers.
template <typename T> struct LayerCfg { static constexpr int FC = 64, RB1 = 2; };
template <> struct LayerCfg<float> { static constexpr int FC = 32, RB1 = 1; };

template <int P> struct Par { static constexpr int v = P; };

// f(Par<I>) for I = B .. E - 1, unrolled.
template <int I, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < E) {
    f(Par<I>{});
    static_for<I + 1, E>(f);
  }
}

// Chunks c = 0 .. n - 1 two at a time, chunk c with buffer parity (P0 + c) & 1
// as a compile-time argument.  n must be even when EVEN.
template <int P0, bool EVEN, typename F>
__device__ __forceinline__ void chunk_pairs(int n, F&& f) {
  int c = 0;
  for (; c + 1 < n; c += 2) {
    f(c, Par<P0>{});
    f(c + 1, Par<P0 ^ 1>{});
  }
  if constexpr (!EVEN) {
    if (c < n) f(c, Par<P0>{});
  }
}

// Rows beyond row_max are read as row row_max (a ragged block of O); weight
// tiles are whole.
template <typename T, int ROWS, int COLS>
__device__ __forceinline__ void dma_tile(T* tile, const T* src, int ld, int row_max) {
  if (row_max < ROWS - 1) DmaTile<T, ROWS, COLS>(tile, src, ld, row_max).template all<true>();
  else DmaTile<T, ROWS, COLS>(tile, src, ld, row_max).template all<false>();
}

// UNITS biases of a chunk (a multiple of 16 bytes, at most 1 KB) by the first lanes of wave 0.
template <typename T, int UNITS>
__device__ __forceinline__ void dma_bias(T* lds, const T* b) {
  constexpr int EPV = 16 / sizeof(T);
  static_assert(UNITS % EPV == 0 && UNITS / EPV <= 64, "bias chunk");
  if (threadIdx.x < UNITS / EPV) dma16(uniform_base(b), threadIdx.x * 16, lds);
}

// Barrier after which every direct load issued before it is in LDS.
__device__ __forceinline__ void publish() { dma::wait_loads_then_barrier(); }

// Barrier for data written to LDS by ds_write only: direct loads in flight
// stay in flight.
__device__ __forceinline__ void bar_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

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

// Tile geometry.
template <typename T, int D>
struct Geo {
  using MF = Mfma<T>;
  static constexpr int FC = LayerCfg<T>::FC;
  static constexpr int RB1 = LayerCfg<T>::RB1;
  static constexpr int P1M = LBM / (16 * RB1);    // unit tiling: P1M row groups x P1N unit groups
  static constexpr int P1N = kLayerWaves / P1M;
  static constexpr int HPW = FC / P1N;            // units per wave and chunk
  static constexpr int JB1 = HPW / 16;
  static constexpr int KS1 = D / MF::K;
  static constexpr int KS2 = FC / MF::K;
  static constexpr int WM2 = 2, WN2 = 4;          // row tiling
  static constexpr int MB2 = LBM / WM2 / 16;
  static constexpr int NB2 = D / WN2 / 16;
  static constexpr int NK0 = D / FC;              // phase-0 chunks
  // QKV chunks of FCQ = QH * FC units, half h of a chunk in the u (h = 0) or
  // r (h = 1) buffer of its parity; a unit-tiling wave covers one half.
  static constexpr int QH = P1N == 2 && (3 * D) % (2 * FC) == 0 ? 2 : 1;
  static constexpr int FCQ = QH * FC;
  static constexpr int NQ = 3 * D / FCQ;
  static constexpr int HPWQ = FCQ / P1N;
  static constexpr int JBQ = HPWQ / 16;
  // elements of a staging buffer: a weight chunk (FC x D or D x FC) or an O chunk (LBM x FC)
  static constexpr int BUF = FC * (D > LBM ? D : LBM);
  // At a switch from the row to the unit tiling the activation passes through
  // LDS as NZ column parts of ZC columns, one staging buffer each.
  static constexpr int NZ = LBM / FC;
  static constexpr int ZC = D / NZ;
  static_assert(P1M * P1N == kLayerWaves && JB1 >= 1 && NB2 >= 1, "wave grids");
  static_assert(D % FC == 0 && (NZ == 2 || NZ == 4) && ZC % MF::K == 0, "tile shapes");
  static_assert(ZC % (D / WN2) == 0, "a row-tiling wave writes within one part");
  static_assert(FC * D <= BUF && LBM * FC <= BUF && LBM * ZC <= BUF, "every staged tile fits a buffer");
  static_assert(QH == 1 || HPWQ == FC, "a wave's QKV units lie in one half");
  static_assert(D % FCQ == 0, "a QKV chunk lies wholly in q, k or v");
  typedef f32x4 UnitAcc[RB1][JB1];                       // unit-tiling accumulators (FFN)
  typedef f32x4 UnitAccQ[RB1][JBQ];                      // (QKV)
  typedef f32x4 RowAcc[MB2][NB2];                        // row-tiling accumulators
  typedef typename MF::frag ActFrags[RB1][KS1];          // unit-tiling activation fragments
  typedef float Red[WN2];
  static constexpr int LDS_BYTES = (4 * BUF + LBM * FC + 2 * FCQ) * (int)sizeof(T) + LBM * WN2 * (int)sizeof(float);
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
};

// The work-group's LDS: staging buffer pairs u (unit-tiling weights, O chunks)
// and r (row-tiling weights), the hidden chunk h, chunk biases b, and the
// LayerNorm partial sums.  Activation parts at a switch use u and r buffers.
template <typename T>
struct Lds {
  T *u0, *u1, *r0, *r1, *b0, *b1, *h;
  float* red;
  template <int P> __device__ __forceinline__ T* u() const { return P ? u1 : u0; }
  template <int P> __device__ __forceinline__ T* r() const { return P ? r1 : r0; }
  template <int P> __device__ __forceinline__ T* b() const { return P ? b1 : b0; }
};

#define GDP_LAYER_LDS(T, G)                                                  \
  __shared__ __attribute__((aligned(16))) T lds_u0_[G::BUF];               \
  __shared__ __attribute__((aligned(16))) T lds_u1_[G::BUF];               \
  __shared__ __attribute__((aligned(16))) T lds_r0_[G::BUF];               \
  __shared__ __attribute__((aligned(16))) T lds_r1_[G::BUF];               \
  __shared__ __attribute__((aligned(16))) T lds_b0_[G::FCQ];               \
  __shared__ __attribute__((aligned(16))) T lds_b1_[G::FCQ];               \
  __shared__ __attribute__((aligned(16))) T lds_h_[LBM * G::FC];           \
  __shared__ __attribute__((aligned(16))) float lds_red_[LBM * G::WN2];    \
  const Lds<T> L{lds_u0_, lds_u1_, lds_r0_, lds_r1_, lds_b0_, lds_b1_, lds_h_, lds_red_}

// Per-lane position in the two tilings.
struct Lanes {
  int lane, wave, col, g4;
  int p1m, p1n;        // unit tiling
  int w2m, w2n;        // row tiling
};

template <typename T, int D>
__device__ __forceinline__ Lanes make_lanes() {
  using G = Geo<T, D>;
  Lanes ln;
  ln.lane = threadIdx.x & 63;
  ln.wave = threadIdx.x >> 6;
  ln.col = ln.lane & 15;
  ln.g4 = ln.lane >> 4;
  ln.p1m = ln.wave / G::P1N;
  ln.p1n = ln.wave % G::P1N;
  ln.w2m = ln.wave / G::WN2;
  ln.w2n = ln.wave % G::WN2;
  return ln;
}

// unit tiling: hacc[i][j] = W_c(tile rows u0 + j*16 + ..) x act(rows (p1m*RB1 + i)*16 + ..)^T,
// W_c a swizzled FC x D tile.  The fragments of k step s + 1 are requested
// before the MFMAs of step s issue.
// after_step(s) runs once the MFMAs of k step s are issued, so that work
// placed there (issuing the next chunk's loads) executes in their shadow.
template <typename T, int D, int JB>
using UnitAccJ = f32x4[Geo<T, D>::RB1][JB];

template <typename T, int D, int JB, typename Hook>
__device__ __forceinline__ void unit_mma(UnitAccJ<T, D, JB>& hacc, const typename Geo<T, D>::ActFrags& af,
                                         const T* sW, int u0, const Lanes& ln, Hook&& after_step) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
  typename MF::frag bw[2][JB];
#pragma unroll
  for (int i = 0; i < G::RB1; ++i)
#pragma unroll
    for (int j = 0; j < JB; ++j) hacc[i][j] = zero4();
#pragma unroll
  for (int j = 0; j < JB; ++j)
    bw[0][j] = MF::load(&sW[swz<T, D>(u0 + j * 16 + ln.col, MF::KV * ln.g4)]);
#pragma unroll
  for (int s = 0; s < G::KS1; ++s) {
    if (s + 1 < G::KS1) {
#pragma unroll
      for (int j = 0; j < JB; ++j)
        bw[(s + 1) & 1][j] = MF::load(&sW[swz<T, D>(u0 + j * 16 + ln.col, (s + 1) * MF::K + MF::KV * ln.g4)]);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch ahead of this step's MFMAs
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int i = 0; i < G::RB1; ++i) hacc[i][j] = MF::mma(bw[s & 1][j], af[i][s], hacc[i][j]);
    __builtin_amdgcn_sched_barrier(0);
    after_step(s);
  }
}

// row tiling: acc += A_c W_c^T with A_c a swizzled LBM x FC tile and W_c a
// swizzled D x FC tile, step s + 1's fragments requested before step s's MFMAs.
template <typename T, int D>
__device__ __forceinline__ void row_mma(typename Geo<T, D>::RowAcc& acc, const T* sA, const T* sW, const Lanes& ln) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
  constexpr int FC = G::FC;
  typename MF::frag af[2][G::MB2], bf[2][G::NB2];
  auto load = [&](int s, typename MF::frag (&a)[G::MB2], typename MF::frag (&b)[G::NB2]) {
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
      a[i] = MF::load(&sA[swz<T, FC>(ln.w2m * G::MB2 * 16 + i * 16 + ln.col, s * MF::K + MF::KV * ln.g4)]);
#pragma unroll
    for (int j = 0; j < G::NB2; ++j)
      b[j] = MF::load(&sW[swz<T, FC>(ln.w2n * G::NB2 * 16 + j * 16 + ln.col, s * MF::K + MF::KV * ln.g4)]);
  };
  load(0, af[0], bf[0]);
#pragma unroll
  for (int s = 0; s < G::KS2; ++s) {
    if (s + 1 < G::KS2) load(s + 1, af[(s + 1) & 1], bf[(s + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch ahead of this step's MFMAs
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) acc[i][j] = MF::mma(bf[s & 1][j], af[s & 1][i], acc[i][j]);
    __builtin_amdgcn_sched_barrier(0);
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

// Row tiling -> unit tiling: the activation in acc goes to LDS as T in NZ
// column parts (the buffers of parity ZP when NZ = 2, all four when NZ = 4),
// and each wave reads back its unit-tiling rows as MFMA fragments.  On exit
// the parts may still be read by other waves, except for NZ = 4, where a
// barrier frees every buffer.
template <typename T, int D, int ZP>
__device__ __forceinline__ void to_unit_tiling(const typename Geo<T, D>::RowAcc& acc, const Lds<T>& L,
                                               typename Geo<T, D>::ActFrags& af, const Lanes& ln) {
  using G = Geo<T, D>;
  using MF = Mfma<T>;
  constexpr int ZC = G::ZC;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  const int zpart = ln.w2n * G::NB2 * 16 / ZC;          // wave-uniform
  auto write = [&](T* part) {
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) {
        const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4(&part[swz<T, ZC>(rbase + i * 16, cbase + j * 16 - zpart * ZC)], v);
      }
  };
  auto part_of = [&](auto zc) -> T* {
    constexpr int z = decltype(zc)::v;
    if constexpr (G::NZ == 2) return z == 0 ? L.template u<ZP>() : L.template r<ZP>();
    else return z == 0 ? L.u0 : z == 1 ? L.u1 : z == 2 ? L.r0 : L.r1;
  };
  if constexpr (G::NZ == 2) {
    if (zpart == 0) write(part_of(Par<0>{}));
    else write(part_of(Par<1>{}));
  } else {
    if (zpart == 0) write(part_of(Par<0>{}));
    else if (zpart == 1) write(part_of(Par<1>{}));
    else if (zpart == 2) write(part_of(Par<2>{}));
    else write(part_of(Par<3>{}));
  }
  bar_lds();
  static_for<0, G::KS1>([&](auto sc) {
    constexpr int s = decltype(sc)::v;
    constexpr int z = s * MF::K / ZC;
    const T* part = part_of(Par<z>{});
#pragma unroll
    for (int i = 0; i < G::RB1; ++i)
      af[i][s] = MF::load(&part[swz<T, ZC>((ln.p1m * G::RB1 + i) * 16 + ln.col, s * MF::K - z * ZC + MF::KV * ln.g4)]);
  });
  if constexpr (G::NZ == 4) bar_lds();
}

template <bool C, typename A, typename B> struct Pick { typedef A type; };
template <typename A, typename B> struct Pick<false, A, B> { typedef B type; };

// The loads of one chunk, all at once (all()) or spread over the k steps of a
// unit-tiling product (step()): tile A (FC x D), an optional tile B (D x FC
// when BT = 1, FC x D when BT = 2) and BU biases, issued by waves 0 .. NW - 1
// (the callers' branch).
template <typename T, int D, int BT, int BU, int NW = kLayerWaves>
struct ChunkDma {
  using G = Geo<T, D>;
  using TA = DmaTile<T, G::FC, D, NW>;
  using TB = typename Pick<BT == 1, DmaTile<T, D, G::FC, NW>, DmaTile<T, G::FC, D, NW>>::type;
  static constexpr int NA = TA::PER, NB = BT ? TB::PER : 0, N = NA + NB + 1;
  TA ta;
  TB tb;
  T* bias_lds;
  const T* bias;
  __device__ __forceinline__ ChunkDma(T* a, const T* wa, T* b, const T* wb, int ldb, T* b_lds, const T* bsrc)
      : ta(a, wa, D, G::FC - 1), tb(b, wb, ldb, BT == 1 ? D - 1 : G::FC - 1), bias_lds(b_lds), bias(bsrc) {}
  __device__ __forceinline__ void piece(int k) const {
    if (k < NA) ta.piece(k);
    else if (k < NA + NB) tb.piece(k - NA);
    else dma_bias<T, BU>(bias_lds, bias);
  }
  __device__ __forceinline__ void step(int s) const {
#pragma unroll
    for (int k = s * N / G::KS1; k < (s + 1) * N / G::KS1; ++k) piece(k);
  }
  __device__ __forceinline__ void all() const {
#pragma unroll
    for (int k = 0; k < N; ++k) piece(k);
  }
};

// The fp32 residual rows held in the row tiling, to y_out[M, ldyo].  With an
// even NB2 they leave in 16-row x 32-column pieces through the wave's own 2 KB
// of H (which must be free of other waves' use), read back as 16-byte parts
// of whole 128-byte row segments: a store then writes 8 full lines instead
// of 16 half lines.
template <typename T, int D>
__device__ __forceinline__ void store_residual(const typename Geo<T, D>::RowAcc& acc, const Lds<T>& L,
                                               const Lanes& ln, int m0, int M, float* y_out, int ldyo) {
  using G = Geo<T, D>;
  if constexpr (G::NB2 % 2 != 0) {
    const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
#pragma unroll
    for (int i = 0; i < G::MB2; ++i) {
      const int row = m0 + ln.w2m * G::MB2 * 16 + ln.col + i * 16;
      if (row < M) {
#pragma unroll
        for (int j = 0; j < G::NB2; ++j)
          *reinterpret_cast<float4*>(y_out + (size_t)row * ldyo + cbase + j * 16) =
              make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      }
    }
  } else {
    static_assert(kLayerWaves * 16 * 32 * sizeof(float) <= LBM * G::FC * sizeof(T), "per-wave staging in H");
    float* reg = reinterpret_cast<float*>(L.h) + ln.wave * (16 * 32);
#pragma unroll
    for (int i = 0; i < G::MB2; ++i) {
      const int rblk = m0 + ln.w2m * G::MB2 * 16 + i * 16;
#pragma unroll
      for (int jh = 0; jh < G::NB2 / 2; ++jh) {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const f32x4 a4 = acc[i][2 * jh + jj];
          const float v[4] = {a4[0], a4[1], a4[2], a4[3]};
          store4(&reg[swz<float, 32>(ln.col, jj * 16 + 4 * ln.g4)], v);
        }
        const int c0 = ln.w2n * G::NB2 * 16 + jh * 32;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int rr = (ln.lane >> 3) + 8 * hf, gg = ln.lane & 7;
          const float4 v = *reinterpret_cast<const float4*>(&reg[swz<float, 32>(rr, gg * 4)]);
          if (rblk + rr < M) *reinterpret_cast<float4*>(y_out + (size_t)(rblk + rr) * ldyo + c0 + gg * 4) = v;
        }
      }
    }
  }
}

// Loads of QKV chunk q (units q*FCQ .. + FCQ of W_qkv and b_qkv) into the
// buffers of parity P, by waves 0 .. NW - 1.
template <typename T, int D, int P, int NW = kLayerWaves>
__device__ __forceinline__ ChunkDma<T, D, Geo<T, D>::QH == 2 ? 2 : 0, Geo<T, D>::FCQ, NW> qkv_chunk(
    const Lds<T>& L, const T* w_qkv, const T* b_qkv, int q) {
  using G = Geo<T, D>;
  const T* w = w_qkv + (size_t)q * G::FCQ * D;
  return ChunkDma<T, D, G::QH == 2 ? 2 : 0, G::FCQ, NW>(L.template u<P>(), w, L.template r<P>(), w + (size_t)G::FC * D,
                                                         D, L.template b<P>(), b_qkv + q * G::FCQ);
}

// Waves issuing the loads spread over a product.  (Leaving them to waves 0-3,
// so that each SIMD keeps one wave free of load stalls, measured slower.)
constexpr int kDmaWaves = kLayerWaves;

// bf16 layers whose QKV chunks span both buffers of a pair (d = 128, 256) use
// qkv_phase_wide (below) for their QKV projection.
template <typename T, int D> constexpr bool kWideQkv = sizeof(T) == 2 && Geo<T, D>::QH == 2;

// wave index as a scalar (uniform) value
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// QKV = act W_qkv^T + b_qkv for the work-group's rows, the activation in the
// row tiling in acc; the q columns are multiplied by q_scale.  Chunk q uses
// buffer parity (q + QP) & 1; the activation passes to the unit tiling through
// the parity QP ^ 1 buffers.  With NZ = 2 chunk 0 must already be in flight
// (or in place) in the parity QP buffers; every other buffer must be free.
template <typename T, int D, int QP>
__device__ __forceinline__ void qkv_phase(const typename Geo<T, D>::RowAcc& acc, const Lds<T>& L,
                                          typename Geo<T, D>::ActFrags& af, const Lanes& ln, int m0, int M,
                                          const T* w_qkv, const T* b_qkv, T* qkv_out, int ldq, float q_scale) {
  using G = Geo<T, D>;
  to_unit_tiling<T, D, QP ^ 1>(acc, L, af, ln);
  if constexpr (G::NZ == 4) qkv_chunk<T, D, QP>(L, w_qkv, b_qkv, 0).all();
  constexpr int FCQ = G::FCQ, JB = G::JBQ;
  // Chunk q's outputs stay in registers until after the barrier that opens
  // chunk q + 1: that barrier waits for all of a wave's outstanding memory
  // operations, stores included, and a store issued a chunk earlier has
  // completed by then.
  float out[G::RB1][JB][4];
  int out_q = -1;
  auto store_out = [&]() {
    if (out_q < 0) return;
    if constexpr (G::QH == 2) {
      // The MFMA layout gives a lane 4 units of one row; a store instruction
      // would write 16 rows x 32 bytes.  Each wave passes its 16-row blocks
      // (64 units = 128 bytes a row) through its own 2 KB of H, read back as
      // 16-byte pieces of 8 whole rows, and writes full 128-byte lines.  The
      // region is the wave's own, so LDS program order is the only ordering.
      constexpr int WU = G::HPWQ;                                  // 64 units a row
      static_assert(kLayerWaves * 16 * WU <= LBM * G::FC && WU * sizeof(T) == 128, "per-wave staging in H");
      T* reg = L.h + ln.wave * (16 * WU);
      const int col0 = out_q * FCQ + ln.p1n * WU;
#pragma unroll
      for (int i = 0; i < G::RB1; ++i) {
#pragma unroll
        for (int j = 0; j < JB; ++j) store4(&reg[swz<T, WU>(ln.col, j * 16 + 4 * ln.g4)], out[i][j]);
        const int rblk = m0 + (ln.p1m * G::RB1 + i) * 16;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int rr = (ln.lane >> 3) + 8 * hf, gg = ln.lane & 7;
          const uint4 v = *reinterpret_cast<const uint4*>(&reg[swz<T, WU>(rr, gg * 8)]);
          if (rblk + rr < M) *reinterpret_cast<uint4*>(qkv_out + (size_t)(rblk + rr) * ldq + col0 + gg * 8) = v;
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < JB; ++j) {
        const int hc = ln.p1n * G::HPWQ + j * 16 + 4 * ln.g4;
#pragma unroll
        for (int i = 0; i < G::RB1; ++i) {
          const int row = m0 + (ln.p1m * G::RB1 + i) * 16 + ln.col;
          if (row < M) store4(qkv_out + (size_t)row * ldq + out_q * FCQ + hc, out[i][j]);
        }
      }
    }
  };
  chunk_pairs<QP, (G::NQ % 2) == 0>(G::NQ, [&](int q, auto pc) {
    constexpr int P = decltype(pc)::v;
    publish();                       // chunk q in place; chunk q - 1's buffers (and the parts) free
    store_out();
    const bool more = q + 1 < G::NQ;
    const auto next = qkv_chunk<T, D, P ^ 1, kDmaWaves>(L, w_qkv, b_qkv, more ? q + 1 : q);
    const bool loader = wave_id() < kDmaWaves;
    f32x4 hacc[G::RB1][JB];
    // the wave's units: half p1n of the chunk (or a share of a one-buffer chunk)
    const T* sW = G::QH == 2 && ln.p1n ? L.template r<P>() : L.template u<P>();
    unit_mma<T, D, JB>(hacc, af, sW, G::QH == 2 ? 0 : ln.p1n * G::HPWQ, ln, [&](int s) {
      if (more && loader) next.step(s);
    });
    const float scale = q * FCQ < D ? q_scale : 1.0f;   // a chunk lies wholly in q, k or v
    const T* sB = L.template b<P>();
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int hc = ln.p1n * G::HPWQ + j * 16 + 4 * ln.g4;
      float b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = to_f32(sB[hc + r]);
#pragma unroll
      for (int i = 0; i < G::RB1; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) out[i][j][r] = (hacc[i][j][r] + b[r]) * scale;
    }
    out_q = q;
  });
  store_out();
}

// The QKV phase for bf16 with 64-row unit-tiling waves: the residual
// accumulator is dead here, so a wave can hold 64 rows of the activation (4
// row blocks) instead of 32 and each W_qkv fragment read from LDS feeds 4
// MFMAs, read by 2 waves instead of 4.  Waves form 2 row groups x 4 unit
// groups of 32 units; otherwise as qkv_phase.
template <typename T, int D>
struct GeoQW {
  using G = Geo<T, D>;
  static constexpr int RB = 4;                       // 16-row blocks per wave
  static constexpr int PM = LBM / (16 * RB);         // 2 row groups
  static constexpr int PN = kLayerWaves / PM;        // 4 unit groups
  static constexpr int HPW = G::FCQ / PN;            // 32 units a wave and chunk
  static constexpr int JB = HPW / 16;
  static_assert(G::QH == 2 && G::FC % HPW == 0 && PM * PN == kLayerWaves, "wide QKV tiling");
};

template <typename T, int D, int QP>
__device__ __forceinline__ void qkv_phase_wide(const typename Geo<T, D>::RowAcc& acc, const Lds<T>& L, const Lanes& ln,
                                               int m0, int M, const T* w_qkv, const T* b_qkv, T* qkv_out, int ldq,
                                               float q_scale) {
  using G = Geo<T, D>;
  using Q = GeoQW<T, D>;
  using MF = Mfma<T>;
  constexpr int ZC = G::ZC, RB = Q::RB, JB = Q::JB, FCQ = G::FCQ, WU = Q::HPW;
  static_assert(G::NZ == 2, "the activation passes through one buffer pair");
  const int pm = ln.wave / Q::PN, pn = ln.wave % Q::PN;
  // row tiling -> this wave's 64 rows of the activation, through the parity QP ^ 1 pair
  typename MF::frag af[RB][G::KS1];
  {
    const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
    const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
    const int zpart = ln.w2n * G::NB2 * 16 / ZC;     // wave-uniform
    T* part = zpart == 0 ? L.template u<QP ^ 1>() : L.template r<QP ^ 1>();
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) {
        const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4(&part[swz<T, ZC>(rbase + i * 16, cbase + j * 16 - zpart * ZC)], v);
      }
    bar_lds();
#pragma unroll
    for (int s = 0; s < G::KS1; ++s) {
      const int z = s * MF::K / ZC;
      const T* src = z == 0 ? L.template u<QP ^ 1>() : L.template r<QP ^ 1>();
#pragma unroll
      for (int i = 0; i < RB; ++i)
        af[i][s] = MF::load(&src[swz<T, ZC>((pm * RB + i) * 16 + ln.col, s * MF::K - z * ZC + MF::KV * ln.g4)]);
    }
  }
  // Chunk q's outputs stay in registers until after the barrier that opens
  // chunk q + 1 (see qkv_phase).  They leave through the wave's own 1 KB of
  // H, 16 rows x 32 units at a time, read back as 16-byte pieces of whole
  // 64-byte row segments.
  float out[RB][JB][4];
  int out_q = -1;
  auto store_out = [&]() {
    if (out_q < 0) return;
    static_assert(kLayerWaves * 16 * WU <= LBM * G::FC && WU * sizeof(T) == 64, "per-wave staging in H");
    T* reg = L.h + ln.wave * (16 * WU);
    const int col0 = out_q * FCQ + pn * WU;
#pragma unroll
    for (int i = 0; i < RB; ++i) {
#pragma unroll
      for (int j = 0; j < JB; ++j) store4(&reg[swz<T, WU>(ln.col, j * 16 + 4 * ln.g4)], out[i][j]);
      const int rblk = m0 + (pm * RB + i) * 16;
      const int rr = ln.lane >> 2, gg = ln.lane & 3;
      const uint4 v = *reinterpret_cast<const uint4*>(&reg[swz<T, WU>(rr, gg * 8)]);
      if (rblk + rr < M) *reinterpret_cast<uint4*>(qkv_out + (size_t)(rblk + rr) * ldq + col0 + gg * 8) = v;
    }
  };
  chunk_pairs<QP, (G::NQ % 2) == 0>(G::NQ, [&](int q, auto pc) {
    constexpr int P = decltype(pc)::v;
    publish();                       // chunk q in place; chunk q - 1's buffers (and the parts) free
    store_out();
    const bool more = q + 1 < G::NQ;
    const auto next = qkv_chunk<T, D, P ^ 1, kDmaWaves>(L, w_qkv, b_qkv, more ? q + 1 : q);
    const bool loader = wave_id() < kDmaWaves;
    // the wave's units: pn * 32 .. + 32 of the chunk, in the u (first half) or r buffer
    const T* sW = pn * WU < G::FC ? L.template u<P>() : L.template r<P>();
    const int u0 = (pn * WU) % G::FC;
    f32x4 hacc[RB][JB];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < JB; ++j) hacc[i][j] = zero4();
    typename MF::frag bw[2][JB];
#pragma unroll
    for (int j = 0; j < JB; ++j) bw[0][j] = MF::load(&sW[swz<T, D>(u0 + j * 16 + ln.col, MF::KV * ln.g4)]);
#pragma unroll
    for (int s = 0; s < G::KS1; ++s) {
      if (s + 1 < G::KS1) {
#pragma unroll
        for (int j = 0; j < JB; ++j)
          bw[(s + 1) & 1][j] = MF::load(&sW[swz<T, D>(u0 + j * 16 + ln.col, (s + 1) * MF::K + MF::KV * ln.g4)]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < JB; ++j)
#pragma unroll
        for (int i = 0; i < RB; ++i) hacc[i][j] = MF::mma(bw[s & 1][j], af[i][s], hacc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
      if (more && loader) next.step(s);
    }
    const float scale = q * FCQ < D ? q_scale : 1.0f;   // a chunk lies wholly in q, k or v
    const T* sB = L.template b<P>();
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int hc = pn * WU + j * 16 + 4 * ln.g4;
      float b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = to_f32(sB[hc + r]);
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) out[i][j][r] = (hacc[i][j][r] + b[r]) * scale;
    }
    out_q = q;
  });
  store_out();
}

// The placement head on the rows held in the row tiling (Fig. 1's N x d
// output): logits[row][e] = act[row] . W_out[e] + b_out[e] for e < n_dev <=
// kFusedHeadDevices, and their logsumexp.  W_out goes to LDS as fp32 (in u0);
// each lane forms the partial sums of its rows over its columns, the 4 lane
// groups of a row combine by butterfly and the WN2 column waves through LDS
// (in h).  u0 and h must be free on entry.
template <typename T, int D>
__device__ __forceinline__ void head_epilogue(const typename Geo<T, D>::RowAcc& acc, const Lds<T>& L,
                                              const Lanes& ln, int m0, int M, const T* w_out, const T* b_out,
                                              int n_dev, float* logits, float* lse) {
  using G = Geo<T, D>;
  constexpr int E = kFusedHeadDevices;
  static_assert(E * D * sizeof(float) <= G::BUF * sizeof(T), "W_out fits a staging buffer");
  static_assert(LBM * G::WN2 * E * sizeof(float) <= LBM * G::FC * sizeof(T), "head sums fit h");
  float* sW = reinterpret_cast<float*>(L.u0);                      // [E][D]
  float (*hred)[G::WN2][E] = reinterpret_cast<float (*)[G::WN2][E]>(L.h);
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
      if (lse) lse[row] = mx + logf(sum);
    }
  }
}

template <typename T>
bool aligned_16(const T* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

// HEAD: the last layer's variant, with the placement head instead of a QKV projection.
// acc += W_2 ReLU(W_1 act + b_1) (the position-wise FFN of a placer layer),
// over d_ff / FC chunks of hidden units that never leave the chip; af holds
// the activation in the unit tiling.  Chunk c uses the buffers of parity
// (P0 + c) & 1; chunk 0 must be in flight (or in place) in the parity P0
// buffers and every other buffer free.  Chunk c + 1 loads during chunk c;
// during the last chunk tail(s) runs after k step s on the loading waves,
// to start the next phase's loads into the parity P0 buffers.
template <typename T, int D, int P0, typename Tail>
__device__ __forceinline__ void ffn_chunks(typename Geo<T, D>::RowAcc& acc, const typename Geo<T, D>::ActFrags& af,
                                           const Lds<T>& L, const Lanes& ln, const T* w1, const T* b1, const T* w2,
                                           int d_ff, Tail&& tail) {
  using G = Geo<T, D>;
  constexpr int FC = G::FC;
  const int NC = d_ff / FC;                           // even
  chunk_pairs<P0, true>(NC, [&](int c, auto pc) {
    constexpr int P = decltype(pc)::v;
    publish();                       // chunk c in place; chunk c - 1's buffers, H and the parts free
    const bool more = c + 1 < NC;
    const int cn = more ? c + 1 : 0;
    const ChunkDma<T, D, 1, FC, kDmaWaves> next_ffn(L.template u<P ^ 1>(), w1 + (size_t)cn * FC * D,
                                                    L.template r<P ^ 1>(), w2 + (size_t)cn * FC, d_ff,
                                                    L.template b<P ^ 1>(), b1 + cn * FC);
    const bool loader = wave_id() < kDmaWaves;
    typename G::UnitAcc hacc;
    unit_mma<T, D, G::JB1>(hacc, af, L.template u<P>(), ln.p1n * G::HPW, ln, [&](int s) {
      if (loader) {
        if (more) next_ffn.step(s);
        else tail(s);
      }
    });
    const T* sB = L.template b<P>();
    // lane holds hidden row (p1m * RB1 + i) * 16 + col, units hc + [0, 4)
#pragma unroll
    for (int j = 0; j < G::JB1; ++j) {
      const int hc = ln.p1n * G::HPW + j * 16 + 4 * ln.g4;
      float b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = to_f32(sB[hc + r]);
#pragma unroll
      for (int i = 0; i < G::RB1; ++i) {
        float h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) h[r] = fmaxf(hacc[i][j][r] + b[r], 0.f);
        store4(&L.h[swz<T, FC>((ln.p1m * G::RB1 + i) * 16 + ln.col, hc)], h);
      }
    }
    bar_lds();                       // H complete
    row_mma<T, D>(acc, L.h, L.template r<P>(), ln);
  });
}

// acc[i][j][r] = gamma[c] * acc + beta[c] for the FiLM vectors of each row's
// graph (gamma / beta: [G, stride]); the lane's column vectors are loaded
// again only when a row belongs to another graph than the previous one.
template <typename T, int D>
__device__ __forceinline__ void film_rows(typename Geo<T, D>::RowAcc& acc, const float* gamma, const float* beta,
                                          int stride, const GraphTable& gt, const Lanes& ln, int m0, int M) {
  using G = Geo<T, D>;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  float4 fgm[G::NB2], fbt[G::NB2];
  int gprev = -1;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    const int gi = graph_of_node(gt, row < M ? row : M - 1);
    if (gi != gprev) {
      const size_t g = (size_t)gi * stride;
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) {
        fgm[j] = *reinterpret_cast<const float4*>(gamma + g + cbase + j * 16);
        fbt[j] = *reinterpret_cast<const float4*>(beta + g + cbase + j * 16);
      }
      gprev = gi;
    }
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      acc[i][j][0] = fgm[j].x * acc[i][j][0] + fbt[j].x;
      acc[i][j][1] = fgm[j].y * acc[i][j][1] + fbt[j].y;
      acc[i][j][2] = fgm[j].z * acc[i][j][2] + fbt[j].z;
      acc[i][j][3] = fgm[j].w * acc[i][j][3] + fbt[j].w;
    }
  }
}

// acc[i][j][r] += b[c] (the second FFN bias) for the lane's columns.
template <typename T, int D>
__device__ __forceinline__ void add_col_bias(typename Geo<T, D>::RowAcc& acc, const T* b, const Lanes& ln) {
  using G = Geo<T, D>;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
#pragma unroll
  for (int j = 0; j < G::NB2; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float bv = to_f32(b[cbase + j * 16 + r]);
#pragma unroll
      for (int i = 0; i < G::MB2; ++i) acc[i][j][r] += bv;
    }
}

template <typename T, int D, bool HEAD>
__global__ __launch_bounds__(LNT) void k_post_attention(PostAttnArgs<T> p, GraphTable gt) {
  using G = Geo<T, D>;
  constexpr int FC = G::FC;
  constexpr int NK0 = G::NK0;
  GDP_LAYER_LDS(T, G);
  typename G::Red* red = reinterpret_cast<typename G::Red*>(L.red);

  const Lanes ln = make_lanes<T, D>();
  const int m0 = p.row0 + blockIdx.x * LBM;
  const int rows_valid = p.M - m0;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;      // row tiling: rows rbase + 16 i
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;   //             columns cbase + 16 j + [0, 4)
  const bool qkv_next = !HEAD && p.w_qkv != nullptr;

  // Chunk c of the FFN: W_1 rows, W_2 columns and b_1 entries c*FC .. + FC.
  auto dma_ffn = [&](int c, auto pc) {
    constexpr int P = decltype(pc)::v;
    dma_tile<T, FC, D>(L.template u<P>(), p.w1 + (size_t)c * FC * D, D, FC - 1);
    dma_tile<T, D, FC>(L.template r<P>(), p.w2 + (size_t)c * FC, p.d_ff, D - 1);
    dma_bias<T, FC>(L.template b<P>(), p.b1 + c * FC);
  };
  // Chunk kc of phase 0: O columns and W_o columns kc*FC .. + FC, parity kc & 1.
  auto dma_p0 = [&](auto kcc) {
    constexpr int kc = decltype(kcc)::v;
    dma_tile<T, LBM, FC>(L.template u<kc & 1>(), p.o + (size_t)m0 * p.ldo + kc * FC, p.ldo, rows_valid - 1);
    dma_tile<T, D, FC>(L.template r<kc & 1>(), p.w_o + kc * FC, D, D - 1);
  };

  // ---- phase 0: acc = Y + b_o + O W_o^T, then LN1 --------------------------
  dma_p0(Par<0>{});
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
  static_for<0, NK0>([&](auto kcc) {
    constexpr int kc = decltype(kcc)::v;
    publish();                       // chunk kc in place; chunk kc - 1's buffers free
    if constexpr (kc + 1 < NK0) dma_p0(Par<kc + 1>{});
    else if constexpr (G::NZ == 2) dma_ffn(0, Par<NK0 & 1>{});   // FFN chunk 0 into the other pair
    row_mma<T, D>(acc, L.template u<kc & 1>(), L.template r<kc & 1>(), ln);
  });
  ln_rows<T, D>(acc, p.ln1_g, p.ln1_b, red, ln);       // acc = Z

  // ---- FFN: acc += W_2 ReLU(W_1 Z + b_1), chunks of FC hidden units ----------
  typename G::ActFrags af;
  to_unit_tiling<T, D, (NK0 + 1) & 1>(acc, L, af, ln);
  if constexpr (G::NZ == 4) dma_ffn(0, Par<NK0 & 1>{});
  // after the last chunk the first QKV chunk (whose W_qkv tile has the W_1
  // tile's shape) loads during it
  const auto first_qkv = qkv_chunk<T, D, NK0 & 1, kDmaWaves>(L, p.w_qkv, p.b_qkv, 0);
  ffn_chunks<T, D, NK0 & 1>(acc, af, L, ln, p.w1, p.b1, p.w2, p.d_ff, [&](int s) {
    if (G::NZ == 2 && qkv_next) first_qkv.step(s);
  });

  // ---- + b_2, LN2, FiLM of the next layer; store Y' ---------------------------
  add_col_bias<T, D>(acc, p.b2, ln);
  ln_rows<T, D>(acc, p.ln2_g, p.ln2_b, red, ln);
  if (p.film_gamma) film_rows<T, D>(acc, p.film_gamma, p.film_beta, p.film_stride, gt, ln, m0, p.M);
  // (issuing these stores after the first QKV barrier instead, to overlap
  // their HBM writes with its products, keeps acc live there and measured
  // 12 % slower)
  if (p.y_out) store_residual<T, D>(acc, L, ln, m0, p.M, p.y_out, p.ldyo);
  if constexpr (HEAD) {
    head_epilogue<T, D>(acc, L, ln, m0, p.M, p.w_out, p.b_out, p.n_dev, p.logits, p.lse);
  } else {
    if (!qkv_next) return;
    // the FFN's last chunk used parity (NK0 + 1) & 1 (an even number of chunks)
    if constexpr (kWideQkv<T, D>)
      qkv_phase_wide<T, D, NK0 & 1>(acc, L, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
    else
      qkv_phase<T, D, NK0 & 1>(acc, L, af, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
  }
}

template <typename T>
hipError_t launch_post_attention(const PostAttnArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  constexpr int EPV = 16 / sizeof(T);
  if (a.d_ff <= 0 || a.d_ff % (2 * LayerCfg<T>::FC)) return hipErrorInvalidValue;
  if (a.ldo % EPV || !aligned_16(a.o) || !aligned_16(a.w_o) || !aligned_16(a.w1) || !aligned_16(a.w2) ||
      !aligned_16(a.b1))
    return hipErrorInvalidValue;
  if (a.w_qkv && (!a.b_qkv || !a.qkv_out || a.ldq < 3 * a.d || a.ldq % EPV || !aligned_16(a.w_qkv) ||
                  !aligned_16(a.b_qkv) || !aligned_16(a.qkv_out)))
    return hipErrorInvalidValue;
  if (a.w_out && (!a.b_out || !a.logits || a.n_dev < 1 || a.n_dev > kFusedHeadDevices || a.w_qkv))
    return hipErrorInvalidValue;
  if (a.film_gamma && (!a.film_beta || a.film_stride % 4 || !aligned_16(a.film_gamma) || !aligned_16(a.film_beta)))
    return hipErrorInvalidValue;
  if (a.y_out && (a.ldyo % 4 || !aligned_16(a.y_out))) return hipErrorInvalidValue;
  if (a.row0 < 0) return hipErrorInvalidValue;
  if (a.row0 >= a.M) return hipSuccess;
  dim3 grid((a.M - a.row0 + LBM - 1) / LBM), block(LNT);
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


// The ablation's placement network without attention (Section 4.4): every
// layer is row-local, Y = FiLM_l(X), X <- LN2_l(Y + W_2 ReLU(W_1 Y + b_1) + b_2),
// so one work-group runs all layers of its 128 rows with the activation in
// its accumulators, and ends with the head.  Layer l's FFN chunk c uses the
// buffers of parity c & 1 (an even number of chunks), so every layer starts
// at parity 0, its first chunk loading during the previous layer's last one.
template <typename T, int D>
__global__ __launch_bounds__(LNT) void k_mlp_placer(MlpPlacerArgs<T> p, GraphTable gt) {
  using G = Geo<T, D>;
  constexpr int FC = G::FC;
  GDP_LAYER_LDS(T, G);
  typename G::Red* red = reinterpret_cast<typename G::Red*>(L.red);
  const Lanes ln = make_lanes<T, D>();
  const int m0 = blockIdx.x * LBM;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  auto first_chunk = [&](int l) {
    return ChunkDma<T, D, 1, FC, kDmaWaves>(L.template u<0>(), p.w1[l], L.template r<0>(), p.w2[l], p.d_ff,
                                             L.template b<0>(), p.b1[l]);
  };
  if constexpr (G::NZ == 2) first_chunk(0).all();
  typename G::RowAcc acc;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    const int rr = row < p.M ? row : p.M - 1;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      float x[4];
      load4f(p.x + (size_t)rr * p.ldx + cbase + j * 16, x);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = x[r];
    }
  }
  typename G::ActFrags af;
  const size_t gd = (size_t)p.n_graphs * D;
  for (int l = 0; l < p.n_layers; ++l) {
    if (p.film) film_rows<T, D>(acc, p.film + 2 * l * gd, p.film + (2 * l + 1) * gd, D, gt, ln, m0, p.M);
    to_unit_tiling<T, D, 1>(acc, L, af, ln);
    if constexpr (G::NZ == 4) first_chunk(l).all();
    const bool more = l + 1 < p.n_layers;
    const auto next = first_chunk(more ? l + 1 : l);
    ffn_chunks<T, D, 0>(acc, af, L, ln, p.w1[l], p.b1[l], p.w2[l], p.d_ff, [&](int s) {
      if (G::NZ == 2 && more) next.step(s);
    });
    add_col_bias<T, D>(acc, p.b2[l], ln);
    ln_rows<T, D>(acc, p.ln_g[l], p.ln_b[l], red, ln);   // its barriers free every buffer
  }
  if (p.y_out) store_residual<T, D>(acc, L, ln, m0, p.M, p.y_out, p.ldyo);
  if (p.w_out) head_epilogue<T, D>(acc, L, ln, m0, p.M, p.w_out, p.b_out, p.n_dev, p.logits, p.lse);
}

template <typename T>
hipError_t launch_mlp_placer(const MlpPlacerArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.n_layers < 1 || a.n_layers > kMlpMaxLayers || !a.x || a.ldx % (16 / (int)sizeof(T)) || !aligned_16(a.x))
    return hipErrorInvalidValue;
  if (a.d_ff <= 0 || a.d_ff % (2 * LayerCfg<T>::FC)) return hipErrorInvalidValue;
  for (int l = 0; l < a.n_layers; ++l)
    if (!a.w1[l] || !a.b1[l] || !a.w2[l] || !a.b2[l] || !a.ln_g[l] || !a.ln_b[l] || !aligned_16(a.w1[l]) ||
        !aligned_16(a.w2[l]) || !aligned_16(a.b1[l]))
      return hipErrorInvalidValue;
  if (a.film && (a.n_graphs < 1 || !aligned_16(a.film))) return hipErrorInvalidValue;
  if (a.w_out && (!a.b_out || !a.logits || a.n_dev < 1 || a.n_dev > kFusedHeadDevices))
    return hipErrorInvalidValue;
  if (a.y_out && (a.ldyo % 4 || !aligned_16(a.y_out))) return hipErrorInvalidValue;
  if (!a.w_out && !a.y_out) return hipErrorInvalidValue;
  dim3 grid((a.M + LBM - 1) / LBM), block(LNT);
  switch (a.d) {
    case 64: hipLaunchKernelGGL((k_mlp_placer<T, 64>), grid, block, 0, s, a, gt); break;
    case 128: hipLaunchKernelGGL((k_mlp_placer<T, 128>), grid, block, 0, s, a, gt); break;
    case 256: hipLaunchKernelGGL((k_mlp_placer<T, 256>), grid, block, 0, s, a, gt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_mlp_placer<float>(const MlpPlacerArgs<float>&, const GraphTable&, hipStream_t);
template hipError_t launch_mlp_placer<bf16>(const MlpPlacerArgs<bf16>&, const GraphTable&, hipStream_t);

// The first placer layer's input and projection (Eq. 4, Section 3.2):
//   Y = FiLM_0(X) (X = the node embeddings; identity without conditioning) into
//   the fp32 residual stream, and QKV = Y W_qkv^T + b_qkv,
// with the same tiles as the post-attention kernel's QKV phase.
template <typename T, int D>
__global__ __launch_bounds__(LNT) void k_pre_layer(PreLayerArgs<T> p, GraphTable gt) {
  using G = Geo<T, D>;
  GDP_LAYER_LDS(T, G);
  const Lanes ln = make_lanes<T, D>();
  const int m0 = p.row0 + blockIdx.x * LBM;
  const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  if constexpr (G::NZ == 2) qkv_chunk<T, D, 0>(L, p.w_qkv, p.b_qkv, 0).all();
  typename G::RowAcc acc;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i) {
    const int row = m0 + rbase + i * 16;
    const int rr = row < p.M ? row : p.M - 1;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      float x[4];
      load4f(p.x + (size_t)rr * p.ldx + cbase + j * 16, x);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = x[r];
    }
  }
  // gamma / beta as 16-byte vectors, loaded again only where a row block starts another graph
  if (p.film_gamma) film_rows<T, D>(acc, p.film_gamma, p.film_beta, p.film_stride, gt, ln, m0, p.M);
  store_residual<T, D>(acc, L, ln, m0, p.M, p.y_out, p.ldyo);
  if constexpr (kWideQkv<T, D>) {
    qkv_phase_wide<T, D, 0>(acc, L, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
  } else {
    typename G::ActFrags af;
    qkv_phase<T, D, 0>(acc, L, af, ln, m0, p.M, p.w_qkv, p.b_qkv, p.qkv_out, p.ldq, p.q_scale);
  }
}

template <typename T>
hipError_t launch_pre_layer(const PreLayerArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (!a.x || !a.y_out || !a.w_qkv || !a.b_qkv || !a.qkv_out || a.ldq < 3 * a.d) return hipErrorInvalidValue;
  if (!aligned_16(a.w_qkv) || !aligned_16(a.b_qkv) || !aligned_16(a.qkv_out) || a.ldq % (16 / (int)sizeof(T)))
    return hipErrorInvalidValue;
  if (a.ldyo % 4 || !aligned_16(a.y_out)) return hipErrorInvalidValue;
  if (a.film_gamma && (!a.film_beta || a.film_stride % 4 || !aligned_16(a.film_gamma) || !aligned_16(a.film_beta)))
    return hipErrorInvalidValue;
  if (a.row0 < 0) return hipErrorInvalidValue;
  if (a.row0 >= a.M) return hipSuccess;
  dim3 grid((a.M - a.row0 + LBM - 1) / LBM), block(LNT);
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


// Section 3.1, Eq. 2 and Eq. 3: the GNN's dense layers,
//   out = act([A1 | A2] [W1 | W2]^T + b)      (act = sigmoid or ReLU),
// over blocks of 128 rows with the row tiling of the kernel above: the
// accumulator holds the block's whole d-wide output, A and W stream through
// LDS in K chunks of FC by direct loads, and the result leaves through each
// wave's slice of H as whole row segments.  K1 and K2 are multiples of FC;
// d = N is 64, 128 or 256.
//
// A comes from HBM, W from L2: the A chunks run through a ring of R slots,
// R - 1 chunks ahead, and W chunks through two buffers.  Chunk c - 1's top
// issues W(c) and then A(c + R - 2); in this loop the loads are a wave's only
// memory operations and complete in order, so chunk c waits for all but the
// A(c + R - 2) loads (vmcnt) before its barrier.
using dma::wait_vm_barrier;

template <typename T, int D, int EPI, bool POOL>
__global__ __launch_bounds__(LNT) void k_row_gemm(GemmArgs<T, T, T> p, RowPoolArgs<T> q) {
  using G = Geo<T, D>;
  constexpr int FC = G::FC;
  constexpr int R = D >= 256 ? 4 : 2;                     // A ring slots
  static_assert(!POOL || (EPI == EPI_RELU && D / FC <= R), "the update's output fits the A ring");
  constexpr int AS = LBM * FC, WS = D * FC;               // elements of an A / W chunk
  constexpr int WC = G::NB2 * 16;                         // a row-tiling wave's columns
  using TA = DmaTile<T, LBM, FC>;
  __shared__ __attribute__((aligned(16))) T sA[R * AS];
  __shared__ __attribute__((aligned(16))) T sW0[WS];
  __shared__ __attribute__((aligned(16))) T sW1[WS];
  __shared__ __attribute__((aligned(16))) T sH[kLayerWaves * 16 * WC];
  const Lanes ln = make_lanes<T, D>();
  const int m0 = blockIdx.x * LBM;
  const int rows_valid = p.M - m0;
  const int nk1 = p.k1 / FC, nk = nk1 + p.k2 / FC;
  typename G::RowAcc acc;
#pragma unroll
  for (int i = 0; i < G::MB2; ++i)
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) acc[i][j] = zero4();
  // chunk c: columns c*FC .. + FC of [A1 | A2] (rows m0 .. + 128) and of [W1 | W2]
  auto issue_a = [&](int c) {
    const bool s1 = c < nk1;
    const int cc = (s1 ? c : c - nk1) * FC;
    const T* a = s1 ? p.a1 + (size_t)m0 * p.lda1 + cc : p.a2 + (size_t)m0 * p.lda2 + cc;
    dma_tile<T, LBM, FC>(sA + (c % R) * AS, a, s1 ? p.lda1 : p.lda2, rows_valid - 1);
  };
  auto issue_w = [&](int c, T* buf) {
    const bool s1 = c < nk1;
    const int cc = (s1 ? c : c - nk1) * FC;
    dma_tile<T, D, FC>(buf, (s1 ? p.w1 : p.w2) + cc, s1 ? p.k1 : p.k2, D - 1);
  };
  // pool transform weights, chunk c: columns c*FC .. + FC of W_pool [D, D]
  auto issue_wp = [&](int c, T* buf) { dma_tile<T, D, FC>(buf, q.w_pool + c * FC, D, D - 1); };
  for (int c = 0; c < R - 1 && c < nk; ++c) issue_a(c);
  issue_w(0, sW0);
  chunk_pairs<0, false>(nk, [&](int c, auto pc) {
    constexpr int P = decltype(pc)::v;
    // A(c) and W(c) in place (each wave waits for its own loads, then the barrier)
    if (R > 2 && c >= 1 && c + R - 2 < nk) wait_vm_barrier<TA::PER>();
    else wait_vm_barrier<0>();
    if (c + 1 < nk) issue_w(c + 1, P ? sW0 : sW1);      // buffer of chunk c - 1
    else if (POOL) issue_wp(0, P ? sW0 : sW1);          // the transform's first chunk
    if (c + R - 1 < nk) issue_a(c + R - 1);             // slot of chunk c - 1
    row_mma<T, D>(acc, sA + (c % R) * AS, P ? sW1 : sW0, ln);
  });

  // bias + activation
  const int cbase = ln.w2n * G::NB2 * 16 + 4 * ln.g4;
  auto bias_act = [&](const T* bias, auto epi) {
    constexpr int E = decltype(epi)::v;
#pragma unroll
    for (int j = 0; j < G::NB2; ++j) {
      float b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = to_f32(bias[cbase + j * 16 + r]);
#pragma unroll
      for (int i = 0; i < G::MB2; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = acc[i][j][r] + b[r];
          if (E == EPI_RELU) v = fmaxf(v, 0.f);
          // the reciprocal instruction (about 1 ulp) instead of an IEEE division
          if (E == EPI_SIGMOID) v = __builtin_amdgcn_rcpf(1.0f + __expf(-v));
          acc[i][j][r] = v;
        }
    }
  };
  bias_act(p.bias, Par<EPI>{});
  T* out = p.out;
  int ldo = p.ldo;
  if constexpr (POOL) {
    // Eq. 2 of the next layer on the same rows: h' (rounded to T, as the
    // separate transform would read it) becomes the A operand in the ring
    // slots; W_pool streams through the two W buffers, chunk c in the buffer
    // of parity PL ^ 1 ^ (c & 1) (PL: the update's last chunk).
    constexpr int NC2 = D / FC;
    using TW = DmaTile<T, D, FC>;
    const int pl = (nk - 1) & 1;
    bar_lds();                                          // every wave is done with the update's tiles
    if (NC2 > 1) issue_wp(1, pl ? sW1 : sW0);           // into the update's last W buffer
    const int rbase = ln.w2m * G::MB2 * 16 + ln.col;
#pragma unroll
    for (int i = 0; i < G::MB2; ++i)
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) {
        const int c = cbase + j * 16;
        const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4(&sA[(c / FC) * AS + swz<T, FC>(rbase + i * 16, c % FC)], v);
        acc[i][j] = zero4();
      }
    // Chunk c: W_pool(c) and h' in place (chunk 0 leaves W_pool(1), the
    // wave's only later load, in flight); W_pool(c + 1), c >= 1, goes into the
    // buffer of chunk c - 1.  Once the last chunk's barrier has passed, no
    // wait for loads follows, so h' leaves then, from the ring slots as whole
    // 16-byte granules of its rows, beside that chunk's products.
    for (int c = 0; c < NC2; ++c) {
      if (c == 0 && NC2 > 1) wait_vm_barrier<TW::PER>();
      else wait_vm_barrier<0>();
      T* cur = ((pl ^ 1 ^ c) & 1) ? sW1 : sW0;
      if (c >= 1 && c + 1 < NC2) issue_wp(c + 1, cur == sW0 ? sW1 : sW0);
      if (c == NC2 - 1) {
        constexpr int EPV = 16 / (int)sizeof(T), GR = D / EPV, GC = FC / EPV;
        for (int e = threadIdx.x; e < LBM * GR; e += LNT) {
          const int row = e / GR, gc = e % GR;
          if (m0 + row < p.M)
            *reinterpret_cast<uint4*>(p.out + (size_t)(m0 + row) * p.ldo + gc * EPV) =
                *reinterpret_cast<const uint4*>(&sA[(gc / GC) * AS + swz<T, FC>(row, (gc % GC) * EPV)]);
        }
      }
      row_mma<T, D>(acc, sA + c * AS, cur, ln);
    }
    bias_act(q.b_pool, Par<EPI_SIGMOID>{});
    out = q.p_out;
    ldo = q.ldp;
  }
  constexpr int RB = WC * (int)sizeof(T);                 // bytes of a row of the wave's columns
  if constexpr (sizeof(T) == 2 && RB >= 64) {
    // 16-row blocks through the wave's own slice of sH, read back as 16-byte
    // parts of whole row segments
    constexpr int LPR = RB / 16, RPI = 64 / LPR, EPV = 16 / (int)sizeof(T);
    T* reg = sH + ln.wave * (16 * WC);
#pragma unroll
    for (int i = 0; i < G::MB2; ++i) {
#pragma unroll
      for (int j = 0; j < G::NB2; ++j) {
        const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        store4(&reg[swz<T, WC>(ln.col, j * 16 + 4 * ln.g4)], v);
      }
      const int rblk = m0 + ln.w2m * G::MB2 * 16 + i * 16;
#pragma unroll
      for (int hf = 0; hf < 16 / RPI; ++hf) {
        const int rr = ln.lane / LPR + RPI * hf, gg = ln.lane % LPR;
        const uint4 v = *reinterpret_cast<const uint4*>(&reg[swz<T, WC>(rr, gg * EPV)]);
        if (rblk + rr < p.M)
          *reinterpret_cast<uint4*>(out + (size_t)(rblk + rr) * ldo + ln.w2n * WC + gg * EPV) = v;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < G::MB2; ++i) {
      const int row = m0 + ln.w2m * G::MB2 * 16 + ln.col + i * 16;
      if (row < p.M) {
#pragma unroll
        for (int j = 0; j < G::NB2; ++j) {
          const float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
          store4(out + (size_t)row * ldo + cbase + j * 16, v);
        }
      }
    }
  }
}

template <typename T>
bool row_gemm_supported(const GemmArgs<T, T, T>& a) {
  constexpr int FC = LayerCfg<T>::FC, EPV = 16 / sizeof(T);
  return (a.N == 64 || a.N == 128 || a.N == 256) && a.k1 > 0 && a.k1 % FC == 0 && a.k2 >= 0 && a.k2 % FC == 0 &&
         (a.k2 == 0 || (a.a2 && a.w2 && a.lda2 % EPV == 0 && aligned_16(a.a2) && aligned_16(a.w2))) &&
         a.lda1 % EPV == 0 && a.ldo % EPV == 0 && aligned_16(a.a1) && aligned_16(a.w1) && aligned_16(a.out) &&
         a.scale_cols == 0;
}
template bool row_gemm_supported<float>(const GemmArgs<float, float, float>&);
template bool row_gemm_supported<bf16>(const GemmArgs<bf16, bf16, bf16>&);

template <typename T>
hipError_t launch_row_gemm(const GemmArgs<T, T, T>& a, int epi, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (!row_gemm_supported(a)) return hipErrorInvalidValue;
  dim3 grid((a.M + LBM - 1) / LBM), block(LNT);
  const RowPoolArgs<T> none = {};
#define GDP_ROW_GEMM(DV)                                                                                          \
  switch (epi) {                                                                                                  \
    case EPI_BIAS: hipLaunchKernelGGL((k_row_gemm<T, DV, EPI_BIAS, false>), grid, block, 0, s, a, none); break;   \
    case EPI_RELU: hipLaunchKernelGGL((k_row_gemm<T, DV, EPI_RELU, false>), grid, block, 0, s, a, none); break;   \
    case EPI_SIGMOID:                                                                                             \
      hipLaunchKernelGGL((k_row_gemm<T, DV, EPI_SIGMOID, false>), grid, block, 0, s, a, none);                    \
      break;                                                                                                      \
    default: return hipErrorInvalidValue;                                                                         \
  }
  switch (a.N) {
    case 64: GDP_ROW_GEMM(64) break;
    case 128: GDP_ROW_GEMM(128) break;
    case 256: GDP_ROW_GEMM(256) break;
    default: return hipErrorInvalidValue;
  }
#undef GDP_ROW_GEMM
  return hipGetLastError();
}
template hipError_t launch_row_gemm<float>(const GemmArgs<float, float, float>&, int, hipStream_t);
template hipError_t launch_row_gemm<bf16>(const GemmArgs<bf16, bf16, bf16>&, int, hipStream_t);

template <typename T>
bool row_gemm_pool_supported(const GemmArgs<T, T, T>& a, const RowPoolArgs<T>& q) {
  return row_gemm_supported(a) && a.N / LayerCfg<T>::FC <= (a.N >= 256 ? 4 : 2) && q.w_pool && q.b_pool &&
         q.p_out && aligned_16(q.w_pool) && aligned_16(q.p_out) && q.ldp % (16 / (int)sizeof(T)) == 0;
}
template bool row_gemm_pool_supported<float>(const GemmArgs<float, float, float>&, const RowPoolArgs<float>&);
template bool row_gemm_pool_supported<bf16>(const GemmArgs<bf16, bf16, bf16>&, const RowPoolArgs<bf16>&);

template <typename T>
hipError_t launch_row_gemm_pool(const GemmArgs<T, T, T>& a, const RowPoolArgs<T>& q, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (!row_gemm_pool_supported(a, q)) return hipErrorInvalidValue;
  dim3 grid((a.M + LBM - 1) / LBM), block(LNT);
  switch (a.N) {
    case 64: hipLaunchKernelGGL((k_row_gemm<T, 64, EPI_RELU, true>), grid, block, 0, s, a, q); break;
    case 128:
      if constexpr (LayerCfg<T>::FC == 64) hipLaunchKernelGGL((k_row_gemm<T, 128, EPI_RELU, true>), grid, block, 0, s, a, q);
      else return hipErrorInvalidValue;
      break;
    case 256:
      if constexpr (LayerCfg<T>::FC == 64) hipLaunchKernelGGL((k_row_gemm<T, 256, EPI_RELU, true>), grid, block, 0, s, a, q);
      else return hipErrorInvalidValue;
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_row_gemm_pool<float>(const GemmArgs<float, float, float>&, const RowPoolArgs<float>&,
                                                hipStream_t);
template hipError_t launch_row_gemm_pool<bf16>(const GemmArgs<bf16, bf16, bf16>&, const RowPoolArgs<bf16>&,
                                               hipStream_t);

}  // namespace gdp
