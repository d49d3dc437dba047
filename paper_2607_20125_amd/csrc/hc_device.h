// Device-side helpers shared by the gfx950 kernels of the HeadCast library
// (bf16 vector types, global loads, MFMA wrapper, LDS staging by DMA, wait
// counters, XCD-aware work mapping).  Included by the .hip sources only.
//
// Matrix-core mapping used by both attention kernels.  They compute S^T = K Q^T
// with v_mfma_f32_32x32x16_bf16 (A = 32 keys x 16 dims, B = 16 dims x 32
// queries), so a lane owns one query column and 16 key rows of every 32x32
// score block: the row max / row sum of the online softmax stay inside a lane
// plus one exchange between the two 32-lane halves.  The output is accumulated
// transposed, O^T = V^T P^T, so the per-query rescale is a per-lane multiply.
// For the P^T operand to come straight out of the score registers, the K rows
// of each 16-key half are fed to the MFMA with bits 2 and 3 of the row index
// swapped; then lane half g holds keys 8g..8g+7 of every 16-key step in
// register order, and the matching V^T operand is 8 consecutive keys of one
// head dimension, which the 8-key-grouped V layout ([keys/8][d][8]) stores as
// 16 contiguous bytes.
//
// All arithmetic: bf16 inputs, fp32 accumulation, exp2 on log2-scaled logits.
#pragma once

#include "hc_internal.h"

#include <cmath>
#include <type_traits>

namespace hc {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kMInit = -1.0e30f;   // finite start of the running max

typedef const u32x4 __attribute__((address_space(1))) *gptr16;

// 16-byte load through the global address space (keeps the load off the LDS counter)
__device__ __forceinline__ u32x4 gld16(const uint16_t *p) {
  return *(gptr16)(p);
}

__device__ __forceinline__ bf16x8 ld_g16(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, gld16(p));
}

// Lazy rescaling: the running max only moves when a tile's max exceeds it by
// more than 2^kRescale in probability units, so exp2(x - m) stays <= 2^kRescale.
constexpr float kRescale = 8.0f;


__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// swap bits 2 and 3 of a row index inside a 32-row block
__device__ __forceinline__ int kperm(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// Position of 16-byte chunk c of K row r in LDS.  The LDS serves a 128-bit read
// 16 lanes at a time over 64 banks (256 bytes); an MFMA A-operand read has 16
// consecutive lanes on 16 consecutive rows at the same chunk, so the chunk is
// XOR-ed with 4 bits of the row: 16 different 16-byte bank groups.  With 64-dim
// heads (8 chunks, two rows per 256 bytes) bit 0 of the row already separates
// row pairs and bits 1-3 are used.
template <int D>
__device__ __forceinline__ int kswz(int r, int c) {
  if constexpr (D >= 128) return c ^ (r & 15);
  else return c ^ ((r >> 1) & 7);
}

// Combine a value with the one held 32 lanes away (the other half of a query's
// key rows).  v_permlane32_swap exchanges the halves of two registers in the
// vector unit, so each lane ends up with both values: no LDS round trip.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// The acceptance test of a fixed-offset pass: row sum in [2^-60, 2^96] and
// every |accumulator| below 2^121.  It compares bit patterns as unsigned
// integers, in which non-negative floats keep their order while infinities,
// NaNs and negative values sort above every finite bound, so a NaN (an
// overflowed probability times a 0 of the row-sum selector, or +inf - inf in
// an accumulator) fails it whatever the compiler assumes about NaN in
// floating-point comparisons.
__device__ __forceinline__ uint32_t abs_bits(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }
__device__ __forceinline__ bool fixed_offset_ok(float row_sum, uint32_t acc_abs_bits_max) {
  const uint32_t lb = __float_as_uint(row_sum);
  return lb >= __builtin_bit_cast(uint32_t, 0x1p-60f) && lb <= __builtin_bit_cast(uint32_t, 0x1p96f) &&
         acc_abs_bits_max < __builtin_bit_cast(uint32_t, 0x1p121f);
}

// ---------------------------------------------------------------------------
// LDS staging.  K and V tiles go global -> LDS with the gfx950
// global_load_lds_dwordx4 instruction (no VGPR staging): one wave instruction
// moves 1 KB, lane i writing bytes [16 i, 16 i + 16) of the destination.
//  * K tile: row r of LDS holds key (r & ~31) | kperm(r & 31) (the MFMA row
//    order), and 16-byte chunk c of a row is stored at position kswz(r, c), so
//    the lanes of an A-operand read (consecutive rows, one chunk) hit different
//    bank groups.
//  * V tile: copied as is from the 8-key-grouped layout [groups][d][8 keys].
//
// The DMA is issued from inline assembly.  The compiler's wait-count pass
// treats a DMA it can see as a pending write to its whole LDS array and drains
// every outstanding DMA (vmcnt(0)) before the next read of that array, which
// would serialise the ring: the tile issued for two steps ahead would have to
// land before the current one is used.  The kernels order DMA and LDS reads
// themselves (vmcnt waits for their own tiles, then a barrier), and the
// "memory" clobber keeps the compiler from moving LDS accesses across a DMA.
// M0 (the LDS base of the instruction) is saved and restored around each run
// of instructions.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void *lvoid;

// Wave-uniform LDS byte address of a location in a __shared__ array.  Taken
// once outside the key loops: the cast from a generic pointer carries a null test.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lvoid)p);
}

// N DMA instructions into consecutive 1 KB of LDS: instruction j moves 16
// bytes per lane from base + a[j] (bytes) + 1024 j to LDS lds + 1024 j + 16 lane.
// The immediate offset of global_load_lds applies to the global and the LDS
// address alike, so M0 is written once for the run (and restored after it).
// N <= 4 keeps the offsets inside the instruction's 13-bit signed field.
template <int N>
__device__ __forceinline__ void lds_dma16_run(const uint16_t *base, const uint32_t *a, uint32_t lds) {
  static_assert(N >= 1 && N <= 4, "run length");
  uint32_t saved;
  if constexpr (N == 1) {
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(a[0]), "s"(base), "s"(lds)
        : "memory");
  } else if constexpr (N == 2) {
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %4\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %3\n\t"
        "global_load_lds_dwordx4 %2, %3 offset:1024\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(a[0]), "v"(a[1]), "s"(base), "s"(lds)
        : "memory");
  } else if constexpr (N == 3) {
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %5\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %4\n\t"
        "global_load_lds_dwordx4 %2, %4 offset:1024\n\t"
        "global_load_lds_dwordx4 %3, %4 offset:2048\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "s"(base), "s"(lds)
        : "memory");
  } else {
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %6\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %5\n\t"
        "global_load_lds_dwordx4 %2, %5 offset:1024\n\t"
        "global_load_lds_dwordx4 %3, %5 offset:2048\n\t"
        "global_load_lds_dwordx4 %4, %5 offset:3072\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "s"(base), "s"(lds)
        : "memory");
  }
}

// M DMA instructions into consecutive 1 KB of LDS, in runs of at most four:
// instruction j moves 16 bytes per lane from base + a[j] + 1024 j to LDS
// lds + 1024 j + 16 lane (a[j]: the byte offset of its source less 1024 j).
template <int M>
__device__ __forceinline__ void lds_dma16_runs(const uint16_t *base, const uint32_t *a, uint32_t lds) {
  if constexpr (M > 0) {
    constexpr int N = M < 4 ? M : 4;
    lds_dma16_run<N>(base, a, lds);
    lds_dma16_runs<M - N>(base + 2048, a + N, lds + 4096);
  }
}

// s_waitcnt vmcnt(N), other counters untouched (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Map the launch index to a work unit so that each XCD (work groups are dealt
// round-robin to the 8 XCDs) runs a contiguous run of units: units are ordered
// so that neighbours share K/V, which then stays in that XCD's L2.
__device__ __forceinline__ int xcd_unit(int bid, int n) {
  const int per = n / 8, rem = n % 8;
  const int x = bid % 8, i = bid / 8;
  return x * per + min(x, rem) + i;
}


}  // namespace dev
}  // namespace hc
