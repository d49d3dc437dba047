// gfx950 (CDNA4) kernels of the HeadCast routed-attention path.
//
// attn_dense   -- softmax attention of 128-query tiles over a contiguous key range
//                 (Global path: the whole window; Sink/Dummy paths: one block;
//                 classification proxies O_ref, O_sink, O_dummy).  Sec. 4.4, Eq. 2.
// attn_spatial -- softmax attention of each query over the (2r+1)^2 positions around
//                 it in every window frame, addressed by index arithmetic (Sec. 4.2
//                 Spatial proxy; the deployed Spatial path of this library).
// kv_scatter   -- cache split and block append into the per-archetype buffers (Sec. 4.3).
// cls_stats    -- per-token cosines and squared errors for Eq. 3 and Eq. 4.
//
// Matrix-core mapping.  Both attention kernels compute S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (A = 32 keys x 16 dims, B = 16 dims x 32 queries), so a
// lane owns one query column and 16 key rows of every 32x32 score block: the
// row max / row sum of the online softmax stay inside a lane plus one exchange
// between the two 32-lane halves.  The output is accumulated transposed,
// O^T = V^T P^T, so the per-query rescale is a per-lane multiply.  For the
// P^T operand to come straight out of the score registers, the K rows of each
// 16-key half are fed to the MFMA with bits 2 and 3 of the row index swapped;
// then lane half g holds keys 8g..8g+7 of every 16-key step in register order,
// and the matching V^T operand is 8 consecutive keys of one head dimension,
// which the 8-key-grouped V layout ([keys/8][d][8]) stores as 16 contiguous bytes.
//
// All arithmetic: bf16 inputs, fp32 accumulation, exp2 on log2-scaled logits.
#include "hc_internal.h"

#include <cmath>
#include <type_traits>

namespace hc {
namespace {

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

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32, 64); }

// ---------------------------------------------------------------------------
// LDS staging.  K and V tiles (64 keys) go global -> LDS with the gfx950
// global_load_lds_dwordx4 instruction (no VGPR staging): one wave instruction
// moves 1 KB, lane i writing bytes [16 i, 16 i + 16) of the destination.
//  * K tile: row r of LDS holds key (r & ~31) | kperm(r & 31) (the MFMA row
//    order), and 16-byte chunk c of a row is stored at position c ^ (r & 7), so
//    the 32 lanes of an A-operand read (rows r..r+31, one chunk) hit 32
//    different bank groups.
//  * V tile: copied as is from the 8-key-grouped layout [8 groups][d][8 keys].
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(1))) const void *gvoid;
typedef __attribute__((address_space(3))) void *lvoid;

__device__ __forceinline__ void lds_dma16(const uint16_t *src, uint16_t *lds_dst) {
  __builtin_amdgcn_global_load_lds((gvoid)src, (lvoid)lds_dst, 16, 0, 0);
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

// ---------------------------------------------------------------------------
// Dense kernel: one work group = 128 queries of one unit on 4 waves of 32
// queries; two work groups share a CU (two waves per SIMD, 2 x 80 KB of LDS),
// so one group's barrier waits and softmax overlap the other's matrix work.  The key loop is software-pipelined inside each
// wave: while the matrix cores compute S(t+1) = K(t+1) Q^T, the vector units
// turn S(t) into probabilities; while they accumulate O += V(t) P(t), the vector
// units take the row max of S(t+1).  K tiles are read one tile ahead of V
// tiles, so K has a 2-buffer and V a 3-buffer LDS ring; one barrier per tile.
// ---------------------------------------------------------------------------
// kRole only separates the symbols of the three callers in profiles:
// 0 routed step, 1 full-window step (all heads Global), 2 classification.
template <int D, int kRole>
__global__ __launch_bounds__(256, 2) void attn_dense_kernel(DenseArgs a) {
  constexpr int NW = 4;                      // waves per work group
  constexpr int KT = kKTile;
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int CPR = D / 8;                 // 16-byte chunks per K row
  constexpr int RPI = 64 / CPR;              // K rows per 1 KB wave instruction
  constexpr int TILE = KT * D;               // elements per tile
  constexpr int LPW = TILE / 512 / NW;       // 1 KB instructions per wave per tensor
  static_assert(LPW >= 1, "tile too small for the wave count");
  __shared__ __attribute__((aligned(1024))) uint16_t sK[2][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[3][TILE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, g = lane >> 5;
  const DenseUnit u = a.units[xcd_unit(blockIdx.x, a.n_units)];
  const int L = a.L;

  bf16x8 qf[NKK];
  {
    const int row = u.q0 + wave * 32 + n;
    const uint16_t *qp = a.q + ((size_t)u.head * L + (row < L ? row : L - 1)) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = ld_g16(qp + 16 * kk + 8 * g);
  }

  const int nkeys = u.kv1 - u.kv0;
  const int nt = (nkeys + KT - 1) / KT;
  const int rem_last = nkeys - (nt - 1) * KT;      // keys in the last tile
  const uint16_t *kbase = u.k + (size_t)u.kv0 * D;
  const uint16_t *vbase = u.v + (size_t)u.kv0 * D;

  int koff[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int ins = wave * LPW + j;
    const int r = ins * RPI + lane / CPR;
    const int key = (r & ~31) | kperm(r & 31);
    const int c = kswz<D>(r, lane % CPR);
    koff[j] = key * D + c * 8;
  }
  // DMA of tile t: K first, then V (the waits below rely on this order)
  auto issue = [&](int t) {
    const uint16_t *kt = kbase + (size_t)t * TILE;
    const uint16_t *vt = vbase + (size_t)t * TILE;
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      lds_dma16(kt + koff[j], &sK[t & 1][(wave * LPW + j) * 512]);
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      lds_dma16(vt + (wave * LPW + j) * 512 + lane * 8, &sV[t % 3][(wave * LPW + j) * 512]);
  };

  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
  float m_run = kMInit, l_run = 0.f;
  const float sl2 = a.scale_log2;

  // two independent accumulation chains (kb = 0, 1) interleaved
  auto qk = [&](int t, f32x16 (&s)[2]) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(
            &sK[t & 1][(32 * kb + n) * D + kswz<D>(32 * kb + n, 2 * kk + g) * 8]);
        s[kb] = mfma32(kf, qf[kk], s[kb]);
      }
  };
  // keys at or past `rem` of this tile get no weight
  auto mask = [&](f32x16 (&s)[2], int rem) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (32 * kb + kperm(8 * (r >> 2) + 4 * g + (r & 3)) >= rem) s[kb][r] = -INFINITY;
  };
  auto rowmax = [&](const f32x16 (&s)[2]) -> float {
    float m0 = fmaxf(s[0][0], fmaxf(s[0][1], s[0][2]));
    float m1 = fmaxf(s[1][0], fmaxf(s[1][1], s[1][2]));
#pragma unroll
    for (int r = 3; r < 15; r += 2) {
      m0 = fmaxf(m0, fmaxf(s[0][r], s[0][r + 1]));
      m1 = fmaxf(m1, fmaxf(s[1][r], s[1][r + 1]));
    }
    float m = fmaxf(fmaxf(m0, s[0][15]), fmaxf(m1, s[1][15]));
    m = fmaxf(m, xor32(m));
    return m * sl2;
  };
  auto rescale = [&](float mx) {
    if (__any(mx > m_run + kRescale)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db] *= alpha;
    }
  };
  // probabilities in bf16 (the PV operand); the row sum adds the same rounded
  // values, two per v_dot2 against (1, 1)
  auto softmax = [&](const f32x16 (&s)[2], bf16x8 (&pf)[2][2]) {
    const float nm = -m_run;
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[kb][h][e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[kb][8 * h + e], sl2, nm));
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2 pr = {pf[kb][h][e], pf[kb][h][e + 1]};
          if (e & 2) ps1 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps1, false);
          else ps0 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps0, false);
        }
      }
    l_run += ps0 + ps1;
  };
  // consecutive MFMAs go to different output blocks (independent chains)
  auto pv = [&](int t, const bf16x8 (&pf)[2][2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const int grp = 4 * kb + 2 * h + g;
          const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(
              &sV[t % 3][(grp * D + 32 * db + n) * 8]);
          acc[db] = mfma32(vf, pf[kb][h], acc[db]);
        }
  };

  // prologue: K(0), V(0), K(1), V(1) in flight; S(0) and its max
  issue(0);
  if (nt > 1) issue(1);
  if (nt > 1) wait_vmcnt<3 * LPW>(); else wait_vmcnt<LPW>();   // K(0) landed
  __syncthreads();
  f32x16 sa[2], sb[2];
  qk(0, sa);
  if (nt == 1 && rem_last < KT) mask(sa, rem_last);
  float mxa = rowmax(sa);

  // steady state: iteration t computes S(t+1) and PV(t); t+1 is not the last tile
  int t = 0;
  for (; t + 2 < nt; ++t) {
    wait_vmcnt<LPW>();          // everything but V(t+1) of the previous issue: K(t+1), V(t)
    __syncthreads();            // ... landed for every wave, and iteration t-1 is over
    if (t + 2 < nt) issue(t + 2);
    rescale(mxa);
    bf16x8 pf[2][2];
    qk(t + 1, sb);
    softmax(sa, pf);
    pv(t, pf);
    const float mxb = rowmax(sb);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) sa[kb] = sb[kb];
    mxa = mxb;
  }
  // t + 1 == nt - 1: S of the last (possibly ragged) tile, PV(t)
  if (t + 1 < nt) {
    wait_vmcnt<0>();
    __syncthreads();
    rescale(mxa);
    bf16x8 pf[2][2];
    qk(t + 1, sb);
    softmax(sa, pf);
    pv(t, pf);
    if (rem_last < KT) mask(sb, rem_last);
    const float mxb = rowmax(sb);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) sa[kb] = sb[kb];
    mxa = mxb;
    ++t;
  }
  // last tile: PV(nt - 1)
  if (nt > 0) {
    wait_vmcnt<0>();
    __syncthreads();
    rescale(mxa);
    bf16x8 pf[2][2];
    softmax(sa, pf);
    pv(t, pf);
  }

  const int lrow = wave * 32 + n;
  const int row = u.q0 + lrow;
  const float l_tot = l_run + xor32(l_run);
  if (u.slot < 0) {
    if (row < L) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      float *obase = u.out_sel == 0 ? a.o[0] : (u.out_sel == 1 ? a.o[1] : a.o[2]);
      float *op = obase + ((size_t)u.head * L + row) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          f32x4 v4 = {acc[db][4 * rq + 0] * inv, acc[db][4 * rq + 1] * inv,
                      acc[db][4 * rq + 2] * inv, acc[db][4 * rq + 3] * inv};
          *reinterpret_cast<f32x4 *>(op + 32 * db + 8 * rq + 4 * g) = v4;
        }
    }
  } else {
    float *pp = a.part + (size_t)u.slot * partial_floats(D);
    float *op = pp + (size_t)lrow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        f32x4 v4 = {acc[db][4 * rq + 0], acc[db][4 * rq + 1], acc[db][4 * rq + 2],
                    acc[db][4 * rq + 3]};
        *reinterpret_cast<f32x4 *>(op + 32 * db + 8 * rq + 4 * g) = v4;
      }
    if (g == 0) {
      pp[(size_t)kQTile * D + lrow] = m_run;
      pp[(size_t)kQTile * D + kQTile + lrow] = l_tot;
    }
  }
}

// ---------------------------------------------------------------------------
// Combine: O = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i over the partial
// slots of one (head, 256-query tile).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  __shared__ float w_s[kMaxSrcBlocks][kQTile];
  __shared__ float inv_s[kQTile];
  const CombineItem it = a.items[blockIdx.x];
  const int D = a.D;
  const int64_t pf = (int64_t)kQTile * (D + 2);
  for (int r = threadIdx.x; r < kQTile; r += 256) {
    float M = kMInit;
    for (int i = 0; i < it.n_slots; ++i)
      M = fmaxf(M, a.part[(it.slot0 + i) * pf + (int64_t)kQTile * D + r]);
    float den = 0.f;
    for (int i = 0; i < it.n_slots; ++i) {
      const float *pp = a.part + (it.slot0 + i) * pf + (int64_t)kQTile * D;
      const float wgt = __builtin_amdgcn_exp2f(pp[r] - M);
      w_s[i][r] = wgt;
      den += wgt * pp[kQTile + r];
    }
    inv_s[r] = den > 0.f ? 1.f / den : 0.f;
  }
  __syncthreads();
  float *obase = it.out_sel == 0 ? a.o[0] : (it.out_sel == 1 ? a.o[1] : a.o[2]);
  const int nq = D / 4;
  for (int e = threadIdx.x; e < kQTile * nq; e += 256) {
    const int row = e / nq, c4 = e % nq;
    if (it.q0 + row >= a.L) continue;
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < it.n_slots; ++i) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(
          a.part + (it.slot0 + i) * pf + (int64_t)row * D + 4 * c4);
      sum += v * w_s[i][row];
    }
    *reinterpret_cast<f32x4 *>(obase + ((size_t)it.head * a.L + it.q0 + row) * D + 4 * c4) =
        sum * inv_s[row];
  }
}

// s_waitcnt vmcnt(n) for a wave-uniform n in [0, 32]
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  switch (n) {
#define HC_W(N) case N: wait_vmcnt<N>(); break;
    HC_W(0) HC_W(1) HC_W(2) HC_W(3) HC_W(4) HC_W(5) HC_W(6) HC_W(7) HC_W(8) HC_W(9) HC_W(10)
    HC_W(11) HC_W(12) HC_W(13) HC_W(14) HC_W(15) HC_W(16) HC_W(17) HC_W(18) HC_W(19) HC_W(20)
    HC_W(21) HC_W(22) HC_W(23) HC_W(24) HC_W(25) HC_W(26) HC_W(27) HC_W(28) HC_W(29) HC_W(30)
    HC_W(31)
#undef HC_W
    default: wait_vmcnt<32>(); break;
  }
}

// ---------------------------------------------------------------------------
// Spatial kernel.  One work group = F waves; wave f owns the 32 queries of
// query frame f, rows y0..y0+3, columns x0..x0+7 (lane n: row y0 + n/8,
// column x0 + n%8).  A query (f, y, x) attends to key rows y-r..y+r and columns
// x-r..x+r of every window frame, so the F waves share one key set: the halo
// rows y0-r..y0+3+r, columns [8 gs, 8 gs + RW) (G aligned 8-key groups covering
// x0-r..x0+7+r).  The halo is streamed per key frame in 64-key tiles of
// 64/RW halo rows by DMA (K ring of 2, V ring of 3, one barrier per tile) and
// the loop is software-pipelined like the dense kernel.  Keys outside a
// query's window, outside the frame or in clipped rows get no weight; the
// masks come from index arithmetic only.
// ---------------------------------------------------------------------------
template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_spatial_kernel(SpatialArgs a) {
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int RW = 8 * G;              // keys per halo row
  constexpr int RPT = 64 / RW;           // halo rows per 64-key tile
  constexpr int CPR = D / 8;             // 16-byte chunks per K row
  constexpr int KRPI = 64 / CPR;         // K rows per 1 KB DMA instruction
  constexpr int TILE = 64 * D;           // elements of K (or V) per tile
  constexpr int NINS = TILE / 512;       // 1 KB DMA instructions per tensor per tile
  __shared__ __attribute__((aligned(1024))) uint16_t sK[2][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[3][TILE];

  const int tid = threadIdx.x;
  // wave-uniform values live in scalar registers, so conditions on them branch uniformly
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int NW = blockDim.x >> 6;        // = frames per block
  const int n = lane & 31, g = lane >> 5;
  // this wave's DMA instructions per tensor per tile
  const int my_ins = NINS / NW + (wave < NINS % NW ? 1 : 0);

  const int bid = xcd_unit(blockIdx.x, gridDim.x);
  const int ct = bid % a.n_ct;
  const int rg = (bid / a.n_ct) % a.n_rowgroups;
  const int hs = bid / a.n_ct / a.n_rowgroups;

  const int Hg = a.Hg, Wg = a.Wg, Wgp = a.Wgp, F = a.F, r = a.r;
  const int P = Hg * Wg;
  const int c = a.c_lo + ct;
  const int x0 = 8 * c - 8 + (r & 7);
  const int gs = c - 1 - (r >> 3);        // first halo group (may be < 0)
  const int ngrp = Wgp / 8;
  const int head = a.heads[hs];
  const int y0 = 4 * rg;

  // query slot of this lane
  const int qy = y0 + (n >> 3), qx = x0 + (n & 7);
  const bool qvalid = qy < Hg && qx >= 0 && qx < Wg;
  const int tq = qvalid ? wave * P + qy * Wg + qx : 0;
  bf16x8 qf[NKK];
  {
    const uint16_t *qp = a.q + ((size_t)head * a.L + tq) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = qvalid ? ld_g16(qp + 16 * kk + 8 * g) : bf16x8{};
  }

  const uint16_t *kb = a.k + (size_t)hs * a.head_stride;
  const uint16_t *vb = a.v + (size_t)hs * a.head_stride;
  const int hrows = 4 + 2 * r;                       // halo rows per key frame
  const int tpf = (hrows + RPT - 1) / RPT;           // tiles per key frame
  const int nt = a.n_slots * F * tpf;

  auto key_pos = [&](int phi, int hr, int cg) -> size_t {
    int yy = y0 - r + hr;
    yy = min(max(yy, 0), Hg - 1);
    cg = min(max(cg, 0), ngrp - 1);
    return ((size_t)phi * Hg + yy) * Wgp + 8 * cg;
  };
  auto issue = [&](int t) {
    const int phi = t / tpf, tj = t % tpf;
    uint16_t *dk = sK[t & 1], *dv = sV[t % 3];
    for (int ins = wave; ins < NINS; ins += NW) {
      const int lr = ins * KRPI + lane / CPR;              // LDS row of K
      const int kap = (lr & ~31) | kperm(lr & 31);         // key slot held there
      const int hr = tj * RPT + kap / RW, col = kap % RW;
      const int cpos = kswz<D>(lr, lane % CPR);
      const size_t pos = key_pos(phi, hr, gs + col / 8) + col % 8;
      lds_dma16(kb + pos * D + cpos * 8, dk + ins * 512);
    }
    for (int ins = wave; ins < NINS; ins += NW) {
      const int e0 = ins * 512 + lane * 8;
      const int grp = e0 / (8 * D);
      const int hr = tj * RPT + (8 * grp) / RW, cg = gs + (8 * grp % RW) / 8;
      const size_t gpos = key_pos(phi, hr, cg) / 8;
      lds_dma16(vb + gpos * 8 * D + (e0 % (8 * D)), dv + ins * 512);
    }
  };

  // per score register (two 32-key chains): halo row inside the tile and
  // column validity for this lane's query
  uint32_t colmask = 0;                  // bit kb*16 + rr
  uint32_t rowbits[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) rowbits[i] = 0;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int kap = 32 * kb + kperm(8 * (rr >> 2) + 4 * g + (rr & 3));
      const int xk = 8 * gs + kap % RW;
      const bool ok = xk >= 0 && xk < Wg && xk - qx <= r && qx - xk <= r;
      colmask |= (ok ? 1u : 0u) << (16 * kb + rr);
      rowbits[kap / RW] |= 1u << (16 * kb + rr);
    }
  const int hr_lo = n >> 3;              // this lane's window in halo rows: [hr_lo, hr_lo + 2r]

  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
  float m_run = kMInit, l_run = 0.f;
  const float sl2 = a.scale_log2;
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};

  auto qk = [&](int t, f32x16 (&s)[2]) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(
            &sK[t & 1][(32 * kb + n) * D + kswz<D>(32 * kb + n, 2 * kk + g) * 8]);
        s[kb] = mfma32(kf, qf[kk], s[kb]);
      }
    // mask: halo rows outside this lane's window or the frame, invalid columns
    const int tj = t % tpf;
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int hr = tj * RPT + i;
      const int yy = y0 - r + hr;
      const bool live = hr >= hr_lo && hr <= hr_lo + 2 * r && yy >= 0 && yy < Hg;
      m |= live ? rowbits[i] : 0u;
    }
    m &= colmask;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr)
        s[kb][rr] = ((m >> (16 * kb + rr)) & 1u) ? s[kb][rr] : -INFINITY;
  };
  auto rowmax = [&](const f32x16 (&s)[2]) -> float {
    float m0 = fmaxf(s[0][0], fmaxf(s[0][1], s[0][2]));
    float m1 = fmaxf(s[1][0], fmaxf(s[1][1], s[1][2]));
#pragma unroll
    for (int q = 3; q < 15; q += 2) {
      m0 = fmaxf(m0, fmaxf(s[0][q], s[0][q + 1]));
      m1 = fmaxf(m1, fmaxf(s[1][q], s[1][q + 1]));
    }
    float m = fmaxf(fmaxf(m0, s[0][15]), fmaxf(m1, s[1][15]));
    m = fmaxf(m, xor32(m));
    return m * sl2;
  };
  auto rescale = [&](float mx) {
    if (__any(mx > m_run + kRescale)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db] *= alpha;
    }
  };
  auto softmax = [&](const f32x16 (&s)[2], bf16x8 (&pf)[2][2]) {
    const float nm = -m_run;
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[kb][h][e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[kb][8 * h + e], sl2, nm));
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2 pr = {pf[kb][h][e], pf[kb][h][e + 1]};
          if (e & 2) ps1 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps1, false);
          else ps0 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps0, false);
        }
      }
    l_run += ps0 + ps1;
  };
  auto pv = [&](int t, const bf16x8 (&pf)[2][2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const int grp = 4 * kb + 2 * h + g;
          const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(
              &sV[t % 3][(grp * D + 32 * db + n) * 8]);
          acc[db] = mfma32(vf, pf[kb][h], acc[db]);
        }
  };

  // DMA order per tile: K then V; `my_ins` instructions each
  issue(0);
  if (nt > 1) issue(1);
  wait_vmcnt_dyn(nt > 1 ? 3 * my_ins : my_ins);          // K(0) landed
  __syncthreads();
  f32x16 sa[2], sb[2];
  qk(0, sa);
  float mxa = rowmax(sa);
  int t = 0;
  for (; t + 1 < nt; ++t) {
    wait_vmcnt_dyn(my_ins);     // all but V(t+1): K(t+1) and V(t) landed
    __syncthreads();
    if (t + 2 < nt) issue(t + 2);
    rescale(mxa);
    bf16x8 pf[2][2];
    qk(t + 1, sb);
    softmax(sa, pf);
    pv(t, pf);
    const float mxb = rowmax(sb);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) sa[kb] = sb[kb];
    mxa = mxb;
  }
  if (nt > 0) {
    wait_vmcnt_dyn(0);
    __syncthreads();
    rescale(mxa);
    bf16x8 pf[2][2];
    softmax(sa, pf);
    pv(t, pf);
  }

  const float l_tot = l_run + xor32(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    float *op = a.o + ((size_t)head * a.L + tq) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        f32x4 v4 = {acc[db][4 * rq + 0] * inv, acc[db][4 * rq + 1] * inv,
                    acc[db][4 * rq + 2] * inv, acc[db][4 * rq + 3] * inv};
        *reinterpret_cast<f32x4 *>(op + 32 * db + 8 * rq + 4 * g) = v4;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Scatter: one work group = 64 tokens of one (head, source block).
// K rows are copied as 16-byte chunks; V goes through LDS and is written in the
// 8-key-grouped layout, 16 bytes per (8 keys, dim) when the 8 keys are one
// aligned group, else element by element.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void kv_scatter_kernel(ScatterArgs a) {
  constexpr int TT = 64;
  constexpr int VS = D + 8;
  __shared__ __attribute__((aligned(16))) uint16_t sV[TT * VS];
  const int ntt = (a.L + TT - 1) / TT;
  int bid = blockIdx.x;
  const int tt = bid % ntt;
  bid /= ntt;
  const int i = bid % a.n_src;
  const int h = bid / a.n_src;

  const uint8_t kind = a.head_kind[h];
  uint16_t *kd, *vd;
  int64_t kph;      // keys per head of the destination buffer
  int mode;         // 0 dense rows, 1 spatial rows
  int64_t kbase = 0;
  if (kind == 0 /*sink*/ || kind == 1 /*dummy*/) {
    const bool take = (kind == 0) ? (a.src_is_block0[i] != 0) : (i == a.cur_src);
    if (!take) return;
    kd = a.k_sd; vd = a.v_sd; kph = a.sd_keys; mode = 0;
  } else if (kind == 3 /*global*/) {
    kd = a.k_g; vd = a.v_g; kph = a.g_keys; mode = 0;
    kbase = (int64_t)a.src_slot[i] * a.L;
  } else {
    kd = a.k_sp; vd = a.v_sp; kph = a.sp_keys; mode = 1;
  }
  const int64_t hoff = (int64_t)a.head_slot[h] * kph * D;
  kd += hoff;
  vd += hoff;
  const int slot = a.src_slot[i];
  const int P = a.Hg * a.Wg;
  auto key_of = [&](int tok) -> int64_t {
    if (mode == 0) return kbase + tok;
    const int fr = tok / P, p = tok % P;
    const int yy = p / a.Wg, xx = p % a.Wg;
    return (((int64_t)slot * a.F + fr) * a.Hg + yy) * a.Wgp + xx;
  };

  const int t0 = tt * TT;
  const uint16_t *sk = a.src_k + ((size_t)(h * a.n_src + i) * a.L) * D;
  const uint16_t *sv = a.src_v + ((size_t)(h * a.n_src + i) * a.L) * D;
  constexpr int CPR = D / 8;
  for (int c = threadIdx.x; c < TT * CPR; c += 256) {
    const int tok = t0 + c / CPR, col = c % CPR;
    if (tok < a.L) {
      const u32x4 kv = *reinterpret_cast<const u32x4 *>(sk + (size_t)tok * D + col * 8);
      *reinterpret_cast<u32x4 *>(kd + key_of(tok) * D + col * 8) = kv;
      *reinterpret_cast<u32x4 *>(&sV[(c / CPR) * VS + col * 8]) =
          *reinterpret_cast<const u32x4 *>(sv + (size_t)tok * D + col * 8);
    }
  }
  __syncthreads();
  for (int w = threadIdx.x; w < D * (TT / 8); w += 256) {
    const int d = w % D, j = w / D;
    const int tokA = t0 + 8 * j;
    if (tokA >= a.L) continue;
    const int64_t kA = key_of(tokA);
    const bool full = tokA + 7 < a.L && (kA & 7) == 0 && key_of(tokA + 7) == kA + 7;
    if (full) {
      uint16_t vals[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) vals[e] = sV[(8 * j + e) * VS + d];
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk[e] = (uint32_t)vals[2 * e] | ((uint32_t)vals[2 * e + 1] << 16);
      *reinterpret_cast<u32x4 *>(vd + ((kA >> 3) * D + d) * 8) = pk;
    } else {
      for (int e = 0; e < 8 && tokA + e < a.L; ++e) {
        const int64_t ke = key_of(tokA + e);
        vd[((ke >> 3) * D + d) * 8 + (ke & 7)] = sV[(8 * j + e) * VS + d];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Classification statistics: one wave per token row, fp64 accumulation.
// out[row] = {cos(sink, ref), cos(dummy, ref), cos(spatial, ref), sum (sp - ref)^2}
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__global__ __launch_bounds__(256) void cls_stats_kernel(StatsArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave_g = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nw = gridDim.x * 4;
  for (int row = wave_g; row < a.n_rows; row += nw) {
    const size_t base = (size_t)row * a.D;
    double rr = 0, ss = 0, dd = 0, pp = 0, sr = 0, dr = 0, pr = 0, e2 = 0;
    for (int d = lane; d < a.D; d += 64) {
      const double r = a.o_ref[base + d], s = a.o_sink[base + d];
      const double u = a.o_dummy[base + d], p = a.o_sp[base + d];
      rr += r * r; ss += s * s; dd += u * u; pp += p * p;
      sr += s * r; dr += u * r; pr += p * r;
      e2 += (p - r) * (p - r);
    }
    rr = wave_sum(rr); ss = wave_sum(ss); dd = wave_sum(dd); pp = wave_sum(pp);
    sr = wave_sum(sr); dr = wave_sum(dr); pr = wave_sum(pr); e2 = wave_sum(e2);
    if (lane == 0) {
      const double nr = sqrt(rr);
      double *o = a.out + (size_t)row * 4;
      o[0] = sr / fmax(sqrt(ss) * nr, 1e-30);
      o[1] = dr / fmax(sqrt(dd) * nr, 1e-30);
      o[2] = pr / fmax(sqrt(pp) * nr, 1e-30);
      o[3] = e2;
    }
  }
}

}  // namespace

hipError_t launch_dense(const DenseArgs &a, int head_dim, DenseRole role, hipStream_t s) {
  if (a.n_units <= 0) return hipSuccess;
  dim3 grid(a.n_units), block(256);
#define HC_DENSE(DD, RR) hipLaunchKernelGGL((attn_dense_kernel<DD, RR>), grid, block, 0, s, a)
  if (head_dim == 128) {
    if (role == DenseRole::kRouted) HC_DENSE(128, 0);
    else if (role == DenseRole::kFullWindow) HC_DENSE(128, 1);
    else HC_DENSE(128, 2);
  } else {
    if (role == DenseRole::kRouted) HC_DENSE(64, 0);
    else if (role == DenseRole::kFullWindow) HC_DENSE(64, 1);
    else HC_DENSE(64, 2);
  }
#undef HC_DENSE
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(a.n_items), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_spatial(const SpatialArgs &a, int head_dim, hipStream_t s) {
  const int64_t nblk = (int64_t)a.n_sp * a.n_rowgroups * a.n_ct;
  if (nblk <= 0) return hipSuccess;
  const int G = (8 + 2 * a.r + 7) / 8;
  dim3 grid((unsigned)nblk), block(64 * a.F);
#define HC_SP(DD, GG) hipLaunchKernelGGL((attn_spatial_kernel<DD, GG>), grid, block, 0, s, a)
  if (head_dim == 128) {
    if (G <= 1) HC_SP(128, 1); else if (G <= 2) HC_SP(128, 2); else HC_SP(128, 4);
  } else {
    if (G <= 1) HC_SP(64, 1); else if (G <= 2) HC_SP(64, 2); else HC_SP(64, 4);
  }
#undef HC_SP
  return hipGetLastError();
}

hipError_t launch_scatter(const ScatterArgs &a, int n_heads, hipStream_t s) {
  const int ntt = (a.L + 63) / 64;
  dim3 grid((unsigned)(n_heads * a.n_src * ntt)), block(256);
  if (a.D == 128)
    hipLaunchKernelGGL((kv_scatter_kernel<128>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((kv_scatter_kernel<64>), grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_stats(const StatsArgs &a, hipStream_t s) {
  int blocks = (a.n_rows + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(cls_stats_kernel, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace hc
