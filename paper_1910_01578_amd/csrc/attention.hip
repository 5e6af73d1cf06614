// Section 3.2: segment-recurrent attention without positional terms.
//
// Transformer-XL caches each layer's inputs of the previous positions and
// lets the next segment attend over [memory ; segment].  In a forward pass
// that is the same as running each layer over all nodes at once with a band:
// the queries of segment [q0, q1) of graph g attend to the keys
// [max(g_start, q0 - mem_len), q1) of the same layer's input.  There is no
// causal mask (the placement of all ops is emitted at once) and no positional
// term, so every work-group is independent.
//
// Work-group = (128 queries of one segment, one head); wave w owns queries
// [32w, 32w + 32) as two 16-column MFMA blocks.  Scores are formed transposed,
// S^T = K Q^T, so that a lane owns one query column: the row max is an
// in-lane max plus a 4-way exchange, and the probabilities feed the P V
// product (O^T = V^T P^T) straight from the score registers.  K and V move
// through LDS in 64-key tiles: by direct loads into a ring of three buffers
// (bf16, d_h >= 32), otherwise through registers into two.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace gdp {

namespace {

constexpr int BQ = kAttnBlockQ;  // queries per work-group
constexpr int BKV = 64;          // keys per tile
constexpr float kLazyRescale = 8.0f;

// 2^x on the transcendental unit; results below the normal range flush to 0,
// which only drops probabilities that are negligible against the row's maximum.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Contraction over the head dimension: instruction shape per element type.
template <typename T, int DH> struct QkShape;
template <int DH> struct QkShape<bf16, DH> {   // DH = 32, 64: 16x16x32
  static constexpr int K = 32, KV = 8, STEPS = DH / 32;
};
template <> struct QkShape<bf16, 16> { static constexpr int K = 16, KV = 4, STEPS = 1; };
template <int DH> struct QkShape<float, DH> { static constexpr int K = 4, KV = 1, STEPS = DH / 4; };

template <typename T, int DH>
struct QkFrag;
template <int DH> struct QkFrag<bf16, DH> {
  typedef bf16x8 t;
  static __device__ __forceinline__ t load(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
  static __device__ __forceinline__ t zero() { t z; for (int i = 0; i < 8; ++i) z[i] = (bf16)0.f; return z; }
  static __device__ __forceinline__ f32x4 mma(t a, t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct QkFrag<bf16, 16> {
  typedef i16x4 t;
  static __device__ __forceinline__ t load(const bf16* p) { return *reinterpret_cast<const i16x4*>(p); }
  static __device__ __forceinline__ t zero() { return i16x4{0, 0, 0, 0}; }
  static __device__ __forceinline__ f32x4 mma(t a, t b, f32x4 c) { return mfma_16x16x16_bf16(a, b, c); }
};
template <int DH> struct QkFrag<float, DH> {
  typedef float t;
  static __device__ __forceinline__ t load(const float* p) { return *p; }
  static __device__ __forceinline__ t zero() { return 0.f; }
  static __device__ __forceinline__ f32x4 mma(t a, t b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Four consecutive elements held as one raw vector (8 bytes of bf16, 16 of fp32),
// and the 4 x 4 transpose used to stage V^T: column(rows, e) gathers element e
// of four row blocks.
template <typename T> struct VBlock;
template <> struct VBlock<bf16> {
  typedef uint2 raw;
  static __device__ __forceinline__ raw zero() { return make_uint2(0u, 0u); }
  static __device__ __forceinline__ uint32_t half(const raw& r, int e) {
    const uint32_t w = (e < 2) ? r.x : r.y;
    return (e & 1) ? (w >> 16) : (w & 0xffffu);
  }
  // element e of rows 0, 1 (and 2, 3) packed into one word: a byte permute of
  // the two source words (bytes 0-1 from the first, 2-3 from the second)
  static __device__ __forceinline__ raw column(const raw (&r)[4], int e) {
    const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
    const uint32_t w0 = e < 2 ? r[0].x : r[0].y, w1 = e < 2 ? r[1].x : r[1].y;
    const uint32_t w2 = e < 2 ? r[2].x : r[2].y, w3 = e < 2 ? r[3].x : r[3].y;
    return make_uint2(__builtin_amdgcn_perm(w1, w0, sel), __builtin_amdgcn_perm(w3, w2, sel));
  }
};
template <> struct VBlock<float> {
  typedef uint4 raw;
  static __device__ __forceinline__ raw zero() { return make_uint4(0u, 0u, 0u, 0u); }
  static __device__ __forceinline__ uint32_t word(const raw& r, int e) {
    return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w;
  }
  static __device__ __forceinline__ raw column(const raw (&r)[4], int e) {
    return make_uint4(word(r[0], e), word(r[1], e), word(r[2], e), word(r[3], e));
  }
};

// stands in for dma::RowStream where tiles go through registers
struct NoStream {
  __device__ __forceinline__ NoStream(const void*, int) {}
};

}  // namespace

// Bounds of the max-free pass (see the kernel): a query column's sum of 2^s
// inside [2^-50, 2^100] puts its largest term inside [2^-60, 2^100], where no
// term overflows and the terms flushed to zero are below 2^-66 of it.
constexpr float kFastSumLo = 0x1p-50f;
constexpr float kFastSumHi = 0x1p100f;

// Direct loads for both K and V (bf16, d_h >= 32): V stays row-major in LDS
// and its MFMA fragments come from transposing reads.
template <typename T, int DH>
struct AttnCfg {
  static constexpr bool KDMA = sizeof(T) == 2 && DH >= 32;
  static constexpr bool VDMA = KDMA;
  // tile buffers: with direct loads a ring of three, loads two tiles ahead
  static constexpr int NS = VDMA ? 3 : 2;
  static constexpr int WPE = DH >= 64 || (sizeof(T) == 4 && DH >= 32) ? 2 : 4;   // waves per SIMD the registers allow
};

// ds_read_b64_tr_b16: within each group of 16 lanes, destination lane 4q + p
// receives in slot e element p of the 8-byte word addressed by source lane
// 4e + q.
__device__ __forceinline__ uint2 lds_read_tr16(const bf16* p) {
  typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
  const bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4_t*)((__attribute__((address_space(3))) bf16*)p));
  return __builtin_bit_cast(uint2, v);
}

// Four waves per SIMD (at most 128 VGPRs) where d_h <= 32: the exponentials
// of one wave overlap the matrix-core products of another.
//
// Softmax.  Scores arrive in the log2 domain (Q pre-scaled by log2(e)/sqrt(d_h)).
// A first pass forms 2^s with no offset at all: fp32 and bf16 share an 8-bit
// exponent, so unless a query's scores leave roughly [-60, 100] nothing
// overflows or vanishes, and the normalised result is the same as with a
// running maximum.  The sum of each query column, which the pass produces
// anyway, tells whether that held; if it fails for any column, the whole
// work-group repeats the segment with the running-offset softmax (the
// offset is raised only when a tile exceeds it by 2^8).
template <typename T, int DH>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(AttnCfg<T, DH>::WPE)))
void k_seg_attention(AttnArgs<T> p, GraphTable gt) {
  constexpr int EPV = 16 / sizeof(T);
  // bf16 with d_h >= 32: K and V tiles arrive by direct global -> LDS loads
  // into unpadded, XOR-swizzled row-major tiles; otherwise through registers,
  // K into rows padded to KS and V transposed.
  constexpr bool KDMA = AttnCfg<T, DH>::KDMA;
  constexpr bool VDMA = AttnCfg<T, DH>::VDMA;
  constexpr int KS = KDMA ? DH : DH + EPV;  // sK row stride
  // sV^T row stride on the register path: 68 elements puts the 16 rows of an
  // 8-byte bf16 fragment read on distinct bank pairs (an odd number of 8-byte words).
  constexpr int VS = BKV + 4;
  constexpr int DB = DH / 16;           // 16-row blocks of the head dim
  using QS = QkShape<T, DH>;
  using QF = QkFrag<T, DH>;
  constexpr int NS = AttnCfg<T, DH>::NS;
  __shared__ __attribute__((aligned(16))) T sK[NS][BKV * KS];
  __shared__ __attribute__((aligned(16))) T sV[NS][VDMA ? BKV * DH : DH * VS];
  __shared__ int s_redo;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, g4 = lane >> 4;
  // heads fastest, remapped so that the heads of one query block (whose K/V
  // slices share cache lines) run on one XCD
  const int logical = p.qblock0 * p.heads + xcd_remap(blockIdx.x, gridDim.x);
  const int head = logical % p.heads;
  const int qblk = logical / p.heads;

  // ---- which graph / segment / query block -----------------------------------
  const int g = graph_of_block(gt, qblk);
  const int qbs = (p.seg_len + BQ - 1) / BQ;
  const int local = qblk - gt.blk[g];
  const int seg = local / qbs, qb = local % qbs;
  const int gs = gt.ptr[g], ge = gt.ptr[g + 1];
  const int seg0 = gs + seg * p.seg_len;
  const int seg1 = min(seg0 + p.seg_len, ge);
  const int q0 = seg0 + qb * BQ;
  const int qend = min(q0 + BQ, seg1);
  const int k0 = max(gs, seg0 - p.mem_len);
  const int k1 = seg1;
  const int ntiles = (k1 - k0 + BKV - 1) / BKV;

  const T* Qp = p.qkv + head * DH;
  const T* Kp = p.qkv + p.d + head * DH;
  const T* Vp = p.qkv + 2 * p.d + head * DH;

  // ---- Q fragments (B operand of S^T = K Q^T), kept in registers -------------
  typename QF::t qf[2][QS::STEPS];
  auto load_q = [&]() {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int q = q0 + wave * 32 + c * 16 + col;
#pragma unroll
      for (int s = 0; s < QS::STEPS; ++s)
        qf[c][s] = q < qend ? QF::load(Qp + (size_t)q * p.ldq + s * QS::K + QS::KV * g4) : QF::zero();
    }
  };

  // ---- K / V tile staging -------------------------------------------------------
  // Register path: K in 16-byte chunks of key rows; V transposed, each thread
  // moving a 4-key x 4-dim block (lanes consecutive along keys) so that every
  // LDS store writes 4 consecutive keys of one dim.
  constexpr int CPR = DH / EPV;                 // 16-byte chunks per key row
  constexpr int CHUNKS = BKV * CPR;
  constexpr int VTHREADS = (BKV / 4) * (DH / 4);
  static_assert(VTHREADS <= 256, "V block split");
  using V4 = typename VBlock<T>::raw;           // 4 consecutive elements
  constexpr int RK = KDMA ? 1 : (CHUNKS + 255) / 256;
  constexpr int RV = VDMA ? 1 : 4;
  uint4 rk[RK] = {};
  V4 rv[RV] = {};
  const int vkg = threadIdx.x % (BKV / 4), vdg = threadIdx.x / (BKV / 4);
  // direct loads per wave and tile (K and V)
  constexpr int VMT = VDMA ? 2 * (BKV * DH / EPV) / (64 * 4) : 0;
  // direct loads: the key rows of the band, one 64-row block per tile
  using Stream = typename std::conditional<KDMA, dma::RowStream<T, BKV, DH, 4>, NoStream>::type;
  const Stream kstream(Kp + (size_t)k0 * p.ldq, p.ldq);
  const Stream vstream(Vp + (size_t)k0 * p.ldq, p.ldq);
  auto load_tile = [&](int t, int buf) {
    const int kb = k0 + t * BKV;
    // keys past the band end read the last valid row: their scores are masked
    // to -inf, so they carry P = 0 against finite values
    const int row_max = k1 - 1 - kb;
    if constexpr (KDMA) {
      static_assert(VDMA, "K and V move the same way");
      if (row_max < BKV - 1) {
        kstream.template load<true>(&sK[buf][0], t * BKV, row_max);
        vstream.template load<true>(&sV[buf][0], t * BKV, row_max);
      } else {
        kstream.template load<false>(&sK[buf][0], t * BKV, row_max);
        vstream.template load<false>(&sV[buf][0], t * BKV, row_max);
      }
    } else {
#pragma unroll
      for (int i = 0; i < RK; ++i) {
        const int c = threadIdx.x + i * 256;
        const int row = c / CPR, cc = (c % CPR) * EPV;
        const int key = min(kb + row, k1 - 1);
        if (CHUNKS % 256 == 0 || c < CHUNKS) rk[i] = *reinterpret_cast<const uint4*>(Kp + (size_t)key * p.ldq + cc);
      }
    }
    if constexpr (!VDMA) {
      if (threadIdx.x < VTHREADS) {               // whole waves
#pragma unroll
        for (int j = 0; j < RV; ++j) {
          const int key = min(kb + 4 * vkg + j, k1 - 1);
          rv[j] = *reinterpret_cast<const V4*>(Vp + (size_t)key * p.ldq + 4 * vdg);
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
    if constexpr (!KDMA) {
#pragma unroll
      for (int i = 0; i < RK; ++i) {
        const int c = threadIdx.x + i * 256;
        if (c < CHUNKS) {
          const int row = c / CPR, cc = (c % CPR) * EPV;
          *reinterpret_cast<uint4*>(&sK[buf][row * KS + cc]) = rk[i];
        }
      }
    }
    if constexpr (!VDMA) {
      if (threadIdx.x < VTHREADS) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          *reinterpret_cast<V4*>(&sV[buf][(4 * vdg + e) * VS + 4 * vkg]) = VBlock<T>::column(rv, e);
      }
    }
  };

  // O^T accumulators, and the softmax denominators: every row of osum[c]
  // holds sum_k P[k][q] for the lane's query column (a matrix-core product
  // with a block of ones, from the same rounded P as the numerator).
  f32x4 oacc[DB][2];
  f32x4 osum[2];
  // With direct loads and one K fragment per key block (d_h = 32), a tile's
  // K fragments are read right after the barrier that publishes the tile,
  // which sits after the previous tile's score products: their LDS latency
  // then hides under that tile's exponentials and P V product instead of
  // opening the next one.
  constexpr bool KP = VDMA && QS::STEPS == 1;
  typename QF::t kfn[4];
  auto read_k = [&](int buf) {
    if constexpr (KP) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kfn[kb] = QF::load(&sK[buf][dma::swz<T, DH>(kb * 16 + col, QS::KV * g4)]);
    }
  };

  // One pass over the segment's key tiles.  EXACT: scores relative to a
  // running offset m per query column (log2 domain).
  auto run = [&](auto exact_tag) {
    constexpr bool EXACT = decltype(exact_tag)::value;
    osum[0] = zero4();
    osum[1] = zero4();
#pragma unroll
    for (int b = 0; b < DB; ++b) { oacc[b][0] = zero4(); oacc[b][1] = zero4(); }
    float mrun[2] = {0.f, 0.f};

    // Tile t sits in buffer t % NS.  Direct loads: tiles t + 1 and t + 2 are
    // in flight while tile t is consumed, and the barrier that publishes
    // tile t + 1 waits for the older of the two only; it comes after tile
    // t's score products (KP) or at tile t's end.  Tile t + 2 goes into tile
    // t - 1's buffer, whose reads every wave finished before the barrier
    // that published tile t.  Register path: tile t + 1 travels through
    // registers during tile t and is stored at its end.
    // Q is requested in the first pass after the first tiles, and the wait
    // for all of them is one the compiler sees: inside the loop it then
    // tracks no outstanding loads of its own, and the only waits there are
    // the explicit ones for the tiles.
    load_tile(0, 0);
    if (VDMA && ntiles > 1) load_tile(1, 1);
    if constexpr (!EXACT) load_q();
    store_tile(0);
    dma::wait_loads_then_barrier();
    read_k(0);
    int cur = 0;
    for (int t = 0; t < ntiles; ++t) {
      const int nxt = cur + 1 == NS ? 0 : cur + 1;
      const int kvalid = k1 - (k0 + t * BKV);     // keys of this tile that exist (>= 1)

      // S^T blocks: 4 key blocks x 2 query blocks; in the exact pass every
      // block starts from -m, so the MFMA leaves the offset score s - m.
      f32x4 sacc[4][2];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if constexpr (EXACT) {
          sacc[kb][0] = f32x4{-mrun[0], -mrun[0], -mrun[0], -mrun[0]};
          sacc[kb][1] = f32x4{-mrun[1], -mrun[1], -mrun[1], -mrun[1]};
        } else {
          sacc[kb][0] = zero4();
          sacc[kb][1] = zero4();
        }
#pragma unroll
        for (int s = 0; s < QS::STEPS; ++s) {
          const int krow = kb * 16 + col, kcol = s * QS::K + QS::KV * g4;
          int kidx;
          if constexpr (KDMA) kidx = dma::swz<T, DH>(krow, kcol);
          else kidx = krow * KS + kcol;
          const typename QF::t kf = KP ? kfn[kb] : QF::load(&sK[cur][kidx]);
          sacc[kb][0] = QF::mma(kf, qf[0][s], sacc[kb][0]);
          sacc[kb][1] = QF::mma(kf, qf[1][s], sacc[kb][1]);
        }
      }
      // bf16: this tile's V^T fragments for the P V product, read now so that
      // their LDS latency hides under the softmax.  16x16x32 k slot 8*g4 + i holds
      // key 32c + 4*g4 + i (i < 4) or 32c + 16 + 4*g4 + (i - 4).
      bf16x8 vfr[2][DB];
      if constexpr (VDMA) {
        // transposing reads of the row-major tile: source lane (g4, s) addresses
        // key 32c + 16h + 4*g4 + s/4, dims 16b + 4(s%4) .. + 3, so that lane
        // (g4, d) receives dim 16b + d of keys 32c + 16h + 4*g4 + e in slot e
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
          for (int b = 0; b < DB; ++b) {
            const int key = 32 * c2 + 4 * g4 + (col >> 2), dim = 16 * b + 4 * (col & 3);
            const uint2 lo = lds_read_tr16(&sV[cur][dma::swz<T, DH>(key, dim)]);
            const uint2 hi = lds_read_tr16(&sV[cur][dma::swz<T, DH>(key + 16, dim)]);
            vfr[c2][b] = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
          }
      } else if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
          for (int b = 0; b < DB; ++b) {
            const T* vrow = &sV[cur][(b * 16 + col) * VS + 32 * c2 + 4 * g4];
            const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
            const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
            vfr[c2][b] = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
          }
      }
      if constexpr (VDMA) {
        if (t + 2 < ntiles) load_tile(t + 2, nxt + 1 == NS ? 0 : nxt + 1);
      } else {
        if (t + 1 < ntiles) load_tile(t + 1, nxt);
      }

      if constexpr (KP) {
        // tile t + 1 in place (tile t + 2 may stay in flight)
        if (t + 1 < ntiles) {
          if (t + 2 < ntiles) dma::wait_vm_barrier<VMT>();
          else dma::wait_vm_barrier<0>();
          read_k(nxt);
        }
      }
      // mask keys past the band end (only the last tile has them)
      if (kvalid < BKV) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kb * 16 + 4 * g4 + r >= kvalid) { sacc[kb][0][r] = -INFINITY; sacc[kb][1][r] = -INFINITY; }
      }

      if constexpr (EXACT) {
        // The offset m is the first tile's maximum and is only raised when a
        // later tile exceeds it by more than kLazyRescale (a factor 2^8):
        // below that the exponentials stay in range, and the normalised
        // result does not depend on the offset.  The common case needs only
        // each lane's own maximum and a wave vote; the exchange between the 4
        // lanes of a query column and the O and denominator rescale run on
        // the few tiles where some offset moves.
        float mx[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          float m = -INFINITY;
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) m = fmaxf(m, sacc[kb][c][r]);
          mx[c] = m;                              // this lane's keys, relative to the offset
        }
        const bool first = t == 0;
        if (__ballot(first || mx[0] > kLazyRescale || mx[1] > kLazyRescale)) {
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            float m = fmaxf(mx[c], xor_shfl(mx[c], 16));
            m = fmaxf(m, xor_shfl(m, 32));        // the column's maximum
            const float delta = first ? m : fmaxf(m, 0.f);
            const float alpha = first ? 0.f : fast_exp2(-delta);   // nothing accumulated before the first tile
            mrun[c] += delta;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sacc[kb][c] -= delta;
            osum[c] *= alpha;
#pragma unroll
            for (int b = 0; b < DB; ++b) oacc[b][c] *= alpha;
          }
        }
      }
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) sacc[kb][c][r] = fast_exp2(sacc[kb][c][r]);

      // O^T += V^T P^T
      if constexpr (sizeof(T) == 2) {
        bf16x8 ones;
#pragma unroll
        for (int i = 0; i < 8; ++i) ones[i] = (bf16)1.0f;
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          bf16x8 pf[2];
#pragma unroll
          for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              pf[c][i] = (bf16)sacc[2 * c2][c][i];
              pf[c][4 + i] = (bf16)sacc[2 * c2 + 1][c][i];
            }
#pragma unroll
          for (int b = 0; b < DB; ++b) {
            oacc[b][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vfr[c2][b], pf[0], oacc[b][0], 0, 0, 0);
            oacc[b][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vfr[c2][b], pf[1], oacc[b][1], 0, 0, 0);
          }
          osum[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[0], osum[0], 0, 0, 0);
          osum[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[1], osum[1], 0, 0, 0);
        }
      } else {
        // 16x16x4 fp32: chunk (kb, i) puts key 16kb + 4*g4 + i in slot g4
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int b = 0; b < DB; ++b) {
              const float vf = to_f32(sV[cur][(b * 16 + col) * VS + kb * 16 + 4 * g4 + i]);
              oacc[b][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf, sacc[kb][0][i], oacc[b][0], 0, 0, 0);
              oacc[b][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf, sacc[kb][1][i], oacc[b][1], 0, 0, 0);
            }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            osum[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(1.0f, sacc[kb][0][i], osum[0], 0, 0, 0);
            osum[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(1.0f, sacc[kb][1][i], osum[1], 0, 0, 0);
          }
      }

      if constexpr (KP) {
        // published after the score products above
      } else if constexpr (VDMA) {
        // tile t + 1 in place; buffer cur free for tile t + 3
        if (t + 2 < ntiles) dma::wait_vm_barrier<VMT>();
        else dma::wait_vm_barrier<0>();
      } else {
        if (t + 1 < ntiles) store_tile(nxt);
        dma::wait_loads_then_barrier();
      }
      cur = nxt;
    }
  };

  if (threadIdx.x == 0) s_redo = 0;   // published by the first tile's barrier
  run(std::false_type{});
  // every query column's sum inside the bounds (NaN fails the test too)?
  const bool ok = osum[0][0] >= kFastSumLo && osum[0][0] <= kFastSumHi && osum[1][0] >= kFastSumLo &&
                  osum[1][0] <= kFastSumHi;
  if (__ballot(!ok) && lane == 0) s_redo = 1;
  __syncthreads();
  if (s_redo) run(std::true_type{});   // work-group-uniform

  // ---- normalise and store ---------------------------------------------------------
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const float inv = 1.0f / osum[c][0];
    const int q = q0 + wave * 32 + c * 16 + col;
    if (q < qend) {
#pragma unroll
      for (int b = 0; b < DB; ++b) {
        T* o = p.out + (size_t)q * p.ldo + head * DH + b * 16 + 4 * g4;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = from_f32<T>(oacc[b][c][r] * inv);
      }
    }
  }
}

template <typename T>
hipError_t launch_attention(const AttnArgs<T>& a, const GraphTable& gt, hipStream_t s) {
  if (a.total_qblocks <= 0) return hipSuccess;
  if (a.qblock0 < 0) return hipErrorInvalidValue;
  const int dh = a.d / a.heads;
  dim3 grid(a.total_qblocks * a.heads), block(256);
  switch (dh) {
    case 16: hipLaunchKernelGGL((k_seg_attention<T, 16>), grid, block, 0, s, a, gt); break;
    case 32: hipLaunchKernelGGL((k_seg_attention<T, 32>), grid, block, 0, s, a, gt); break;
    case 64: hipLaunchKernelGGL((k_seg_attention<T, 64>), grid, block, 0, s, a, gt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template hipError_t launch_attention<float>(const AttnArgs<float>&, const GraphTable&, hipStream_t);
template hipError_t launch_attention<bf16>(const AttnArgs<bf16>&, const GraphTable&, hipStream_t);

}  // namespace gdp
