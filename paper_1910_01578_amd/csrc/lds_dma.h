// Direct global -> LDS staging for the matrix-core kernels (gfx950).
//
// global_load_lds_dwordx4 moves 16 bytes a lane from global memory into LDS
// without passing through registers; the 64 lanes' granules land
// contiguously at the (wave-uniform) LDS base.  Tiles staged this way are
// therefore unpadded, and each row's 16-byte granules are XOR-permuted
// (swz_key) so that a fragment read of 16 consecutive rows hits distinct
// banks.  The loads are issued as inline assembly: the compiler keeps no
// bookkeeping for them, and whoever reads their data waits for them
// explicitly (wait_loads_then_barrier()).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdp {
namespace dma {

// XOR key of row r in a tile whose rows hold GPR 16-byte granules: granule g
// of row r is stored at granule g ^ swz_key(r), a permutation of each row.
// Any 8 aligned rows place a given granule in distinct 16-byte bank groups.
// The keys were chosen by measuring LDS bank conflicts on gfx950 for the MFMA
// fragment reads (16 rows x 4 granules per instruction) that these tiles
// serve: with them those reads take the minimum four LDS cycles per
// instruction.  (For 128-byte rows, folding bit 3 of the row into the key,
// as (r & 7) ^ ((r >> 3) & 1) does, measured twice that.)
template <int GPR>
__device__ __forceinline__ int swz_key(int r) {
  if constexpr (GPR >= 16) return r & 15;
  else if constexpr (GPR == 8) return r & 7;
  else {
    static_assert(GPR == 4, "tile rows of at least 64 bytes");
    return ((r >> 2) ^ (r >> 1)) & 3;
  }
}

// Element offset of (r, c) in a swizzled LDS tile of COLS columns of T.
template <typename T, int COLS>
__device__ __forceinline__ int swz(int r, int c) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int GPR = COLS / EPV;
  return r * COLS + (((c / EPV) ^ swz_key<GPR>(r)) * EPV) + (c % EPV);
}

typedef const __attribute__((address_space(1))) char* gptr_t;

// p as a global pointer in scalar registers (p must be wave-uniform).
__device__ __forceinline__ gptr_t uniform_base(const void* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (gptr_t)(((uint64_t)hi << 32) | lo);
}

// One direct global -> LDS load: lane l reads the 16 bytes at base + voff
// and writes them to LDS at lds + 16 l (lds wave-uniform).  Issued as inline
// assembly so that the compiler keeps no bookkeeping of its own for these
// loads (it would otherwise make later LDS accesses wait for all of them);
// publish() is the only point that waits for them.  M0 holds the LDS base;
// nothing else in these kernels keeps a value in M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(gptr_t base, uint32_t voff, const void* lds) {
  const uint32_t la = (uint32_t)(uintptr_t)lds;   // a generic LDS address's low word is the LDS offset
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(__builtin_amdgcn_readfirstlane(la)) : "memory", "m0");
}
#pragma clang diagnostic pop

// ROWS x COLS block of a row-major matrix (leading dimension ld; rows beyond
// row_max read row row_max) into a swizzled LDS tile, by waves 0 .. NW - 1
// with DmaTile::PER loads each.  Load i of wave w fills tile granules
// [(w * PER + i) * 64, + 64), lane l the granule at offset l.
template <typename T, int ROWS, int COLS, int NW>
struct DmaTile {
  static constexpr int EPV = 16 / sizeof(T);
  static constexpr int GPR = COLS / EPV;
  static constexpr int GRANULES = ROWS * GPR;
  static_assert(GRANULES % (64 * NW) == 0, "tile must split evenly over the loading waves");
  static_assert(GPR >= 4 && GPR <= 64, "a load covers whole rows or one row");
  static constexpr int PER = GRANULES / (64 * NW);
  T* tile;
  gptr_t base;
  int ld, row_max;
  __device__ __forceinline__ DmaTile(T* tile_, const T* src, int ld_, int row_max_)
      : tile(tile_), base(uniform_base(src)), ld(ld_), row_max(row_max_) {}
  // A load covers 64 / GPR whole rows from rb = q / GPR on (rb aligned to
  // that count), so lane l handles row rb + l / GPR, granule l % GPR, and
  // swz_key(rb + l / GPR) = swz_key(rb) ^ swz_key(l / GPR): the row base and
  // its key are wave-uniform, the rest a per-lane constant.
  template <bool CLAMP>
  __device__ __forceinline__ void piece(int i) const {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int q = (wave * PER + i) * 64;
    const int rb = q / GPR;
    const int lr = lane / GPR;
    const int g = (lane % GPR) ^ swz_key<GPR>(lr) ^ swz_key<GPR>(rb);
    int r0 = rb, rel = lr;
    if (CLAMP) {
      r0 = rb < row_max ? rb : row_max;
      rel = (rb + lr < row_max ? rb + lr : row_max) - r0;
    }
    const uint32_t off = ((uint32_t)rel * (uint32_t)ld + (uint32_t)(g * EPV)) * (uint32_t)sizeof(T);
    dma16(base + (size_t)r0 * ld * sizeof(T), off, tile + q * EPV);
  }
  __device__ __forceinline__ void piece(int i) const { piece<false>(i); }
  template <bool CLAMP = false>
  __device__ __forceinline__ void all() const {
#pragma unroll
    for (int i = 0; i < PER; ++i) piece<CLAMP>(i);
  }
};

// The tile of DmaTile taken again and again from ROWS-row blocks of one
// matrix: the per-lane offsets are formed once, and a block's loads add only
// the block's row offset to the scalar base.
template <typename T, int ROWS, int COLS, int NW>
struct RowStream {
  using Tile = DmaTile<T, ROWS, COLS, NW>;
  static constexpr int PER = Tile::PER, EPV = Tile::EPV, GPR = Tile::GPR;
  gptr_t base;          // row 0 of block 0
  int ld;
  uint32_t off[PER];    // per lane and piece: row * ld + swizzled column, in bytes
  __device__ __forceinline__ RowStream(const T* src, int ld_) : base(uniform_base(src)), ld(ld_) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = (wave * PER + i) * 64, rb = q / GPR, lr = lane / GPR;
      const int g = (lane % GPR) ^ swz_key<GPR>(lr) ^ swz_key<GPR>(rb);
      off[i] = ((uint32_t)(rb + lr) * (uint32_t)ld + (uint32_t)(g * EPV)) * (uint32_t)sizeof(T);
    }
  }
  // The block whose first row is r0 into tile; with CLAMP, rows past row_max
  // (counted from r0) read row row_max instead.
  template <bool CLAMP>
  __device__ __forceinline__ void load(T* tile, int r0, int row_max) const {
    const gptr_t b = base + (size_t)r0 * ld * sizeof(T);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = (wave * PER + i) * 64;
      uint32_t o = off[i];
      if (CLAMP) {
        const int lane = threadIdx.x & 63, rb = q / GPR, lr = lane / GPR;
        const int g = (lane % GPR) ^ swz_key<GPR>(lr) ^ swz_key<GPR>(rb);
        const int row = rb + lr < row_max ? rb + lr : row_max;
        o = ((uint32_t)row * (uint32_t)ld + (uint32_t)(g * EPV)) * (uint32_t)sizeof(T);
      }
      dma16(b, o, tile + q * EPV);
    }
  }
};

// Barrier after which the data of every direct load issued before it by any
// wave is in LDS.  (The work-group fence of a plain barrier does not cover
// those loads, so each wave first waits for all of its own memory operations.)
__device__ __forceinline__ void wait_loads_then_barrier() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Barrier after which all but the N most recent vector memory operations of
// every wave are done.  Valid where a wave's outstanding vector memory
// operations are all loads, which complete in issue order; LDS operations
// are drained too.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"i"(N) : "memory");
}

}  // namespace dma
}  // namespace gdp
