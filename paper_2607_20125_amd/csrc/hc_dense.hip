// Dense softmax attention of 128-query tiles over a contiguous key range, and
// the merge of per-block partial results.  Global path (the whole window),
// Sink/Dummy paths (one block) and the classification proxies O_ref, O_sink,
// O_dummy (Sec. 4.4, Eq. 2).
#include "hc_device.h"

namespace hc {
namespace {
using namespace dev;

// ---------------------------------------------------------------------------
// Dense kernel: one work group = kQTile (128) queries of one unit on 4 waves of
// 32 queries; two work groups share a CU (two waves per SIMD, 2 x 80 KB of LDS),
// so one group's barrier waits and softmax overlap the other's matrix work.
// K/V tiles of 64 keys are fetched kDist tiles ahead of use (K ring of kDist,
// V ring of kDist + 1 buffers); one barrier per tile.
// The key loop is software-pipelined inside each wave: while the matrix cores
// compute S(t+1) = K(t+1) Q^T, the vector units turn S(t) into probabilities;
// in the running-max pass they also take the row max of S(t+1) while the
// matrix cores accumulate O += V(t) P(t).  A unit first runs a fixed-offset
// pass with no row max at all and falls back to the running-max pass only when
// its row sums leave a safe range (see `run` below).
// ---------------------------------------------------------------------------
constexpr int kDenseWaves = kQTile / 32;
constexpr int kDist = 2;

// kRole only separates the symbols of the callers in profiles: 0 routed step,
// 1 full-window step (all heads Global), 2 classification, 3 routed step of a
// context with the cell or two-block variant, 4 a table of Sink and Dummy heads only.
template <int D, int kRole>
__global__ __launch_bounds__(64 * kDenseWaves, 2) void attn_dense_kernel(DenseArgs a) {
  constexpr int NW = kDenseWaves;            // waves per work group
  constexpr int KT = kKTile;
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int CPR = D / 8;                 // 16-byte chunks per K row
  constexpr int RPI = 64 / CPR;              // K rows per 1 KB wave instruction
  constexpr int TILE = KT * D;               // elements per tile
  constexpr int LPW = TILE / 512 / NW;       // 1 KB instructions per wave per tensor
  constexpr int RK = kDist, RV = kDist + 1;  // ring buffers
  static_assert(LPW >= 1, "tile too small for the wave count");
  static_assert(kDist >= 2 && kDist <= 4, "prefetch distance");
  static_assert((RK + RV) * TILE * 2 <= 80 * 1024, "LDS: two work groups per CU");
  __shared__ __attribute__((aligned(1024))) uint16_t sK[RK][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[RV][TILE];

  const int tid = threadIdx.x;
  // the wave index is uniform: in a scalar register, the LDS targets of the DMA are too
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, g = lane >> 5;
  const DenseUnit u = a.units[xcd_unit(blockIdx.x, a.n_units)];
  if (u.head < 0) return;                    // padding of the unit list: no work
  const int L = a.L;

  // this lane's query: row lrow of the unit, token `row` of the block
  const int lrow = wave * 32 + n;
  bool rvalid;
  int row;
  if (u.qn > 0) {
    rvalid = lrow < u.qn;
    row = a.qmap[u.q0 + (rvalid ? lrow : 0)];
  } else {
    row = u.q0 + lrow;
    rvalid = row < L;
  }
  bf16x8 qf[NKK];
  {
    const uint16_t *qp = a.q + ((size_t)u.head * L + (rvalid ? row : L - 1)) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = ld_g16(qp + 16 * kk + 8 * g);
  }
  const float sl2 = a.scale_log2;             // logits in log2 units: s * scale * log2(e)

  const int nkeys = u.kv1 - u.kv0;
  const int nt = (nkeys + KT - 1) / KT;
  const int rem_last = nkeys - (nt - 1) * KT;      // keys in the last tile
  const uint16_t *kbase = u.k + (size_t)u.kv0 * D;
  const uint16_t *vbase = u.v + (size_t)u.kv0 * D;

  // DMA sources of this wave's LPW instructions per tensor, in bytes: K rows
  // permuted and swizzled (kperm, kswz), the V tile in order.  Instruction j
  // also adds 1024 j through its immediate offset (which moves the LDS target
  // by the same amount), so it is taken off here; the K base is taken 4 KB
  // lower (and added back here) so that no offset goes below zero.
  static_assert(LPW == 1 || LPW == 2 || LPW == 4, "DMA run length");
  uint32_t ka[LPW], va[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int ins = wave * LPW + j;
    const int r = ins * RPI + lane / CPR;
    const int key = (r & ~31) | kperm(r & 31);
    const int c = kswz<D>(r, lane % CPR);
    ka[j] = (uint32_t)((key * D + c * 8) * 2 + 4096 - 1024 * j);
    va[j] = (uint32_t)(wave * LPW * 1024 + lane * 16);
  }
  // this wave's DMA targets in ring slot 0
  const uint32_t k_dst = lds_addr(&sK[0][wave * LPW * 512]);
  const uint32_t v_dst = lds_addr(&sV[0][wave * LPW * 512]);
  // DMA of tile t: K first, then V (the waits below rely on this order)
  auto issue = [&](int t) {
    const uint16_t *kt = kbase + (size_t)t * TILE - 2048;
    const uint16_t *vt = vbase + (size_t)t * TILE;
    const uint32_t kd = k_dst + (uint32_t)((t % RK) * TILE * 2);
    const uint32_t vd = v_dst + (uint32_t)((t % RV) * TILE * 2);
    lds_dma16_run<LPW>(kt, ka, kd);
    lds_dma16_run<LPW>(vt, va, vd);
  };
  f32x16 acc[NDB];
  float m_run, l_run;
  // Row sums of the fixed-offset pass on the matrix cores: a 16x16x32 product of
  // a 0/1 selector with the P operand.  Lane l of P holds query l % 32 and key
  // half l / 32, so B column n gathers queries n (k-groups 0, 2) and n + 16
  // (k-groups 1, 3); selector row 0 takes groups 0 and 2, row 1 groups 1 and 3.
  // Lane n < 16 then holds the sum of query n in lacc[0], of n + 16 in lacc[1].
  f32x4 lacc;
  bf16x8 sel;
  {
    const int i = lane & 15, kg = lane >> 4;
    const float v = (i == 0 && (kg & 1) == 0) || (i == 1 && (kg & 1) == 1) ? 1.f : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sel[e] = (__bf16)v;
  }

  // two independent accumulation chains (kb = 0, 1) interleaved
  auto qk = [&](int t, f32x16 (&s)[2]) {
    s[0] = f32x16{};
    s[1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(
            &sK[t % RK][(32 * kb + n) * D + kswz<D>(32 * kb + n, 2 * kk + g) * 8]);
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
    const float m = fmaxf(fmaxf(m0, s[0][15]), fmaxf(m1, s[1][15]));
    return max_xor32(m) * sl2;
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
  // values: on the matrix cores in the fixed-offset pass (FO, see lacc), two per
  // v_dot2 against (1, 1) in the running-max pass.  The FO pass takes
  // 2^(s * scale * log2 e) with no running max.
  auto softmax = [&](auto fo, const f32x16 (&s)[2], bf16x8 (&pf)[2][2]) {
    constexpr bool FO = decltype(fo)::value;
    const float nm = -m_run;
    const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[kb][h][e] = (__bf16)__builtin_amdgcn_exp2f(FO ? s[kb][8 * h + e] * sl2
                                                           : fmaf(s[kb][8 * h + e], sl2, nm));
        if constexpr (!FO) {
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const bf16x2 pr = {pf[kb][h][e], pf[kb][h][e + 1]};
            if (e & 2) ps1 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps1, false);
            else ps0 = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps0, false);
          }
        }
      }
    if constexpr (!FO) l_run += ps0 + ps1;
  };
  // V operand reads: the LDS byte address of this lane's row in ring slot 0; a
  // tile adds its slot once, and each read of the tile is that base plus a
  // constant carried in the read instruction's offset field
  const uint32_t v_lane = (uint32_t)(uintptr_t)(lvoid)&sV[0][(g * D + n) * 8];
  auto v_base = [&](int t) {
    uint32_t b = v_lane + (uint32_t)((t % RV) * TILE * 2);
    asm volatile("" : "+v"(b));   // opaque, so that the constants below stay offsets
    return b;
  };
  // consecutive MFMAs go to different output blocks (independent chains); in
  // the FO pass each 16-key chunk of P also goes through the row-sum product
  auto pv = [&](auto fo, uint32_t vb, const bf16x8 (&pf)[2][2]) {
    constexpr bool FO = decltype(fo)::value;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const uint32_t off = (uint32_t)(((4 * kb + 2 * h) * D + 32 * db) * 16);
          const bf16x8 vf = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8 *>(
              (uintptr_t)(vb + off));
          acc[db] = mfma32(vf, pf[kb][h], acc[db]);
        }
        if constexpr (FO) lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, pf[kb][h], lacc, 0, 0, 0);
      }
  };

  // One pass over the unit's keys.  The running-max pass (fo = false) is the
  // online softmax with lazy rescaling.  The fixed-offset pass (fo = true) keeps
  // the offset at 0: each probability is 2^x for the logit x in log2 units,
  // with no row max, no subtraction and no rescale.  That is exact softmax
  // arithmetic as long as nothing overflows or underflows, which is checked on
  // the row sums afterwards.
  auto run = [&](auto fo) {
    constexpr bool FO = decltype(fo)::value;
#pragma unroll
    for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
    m_run = FO ? 0.f : kMInit;
    l_run = 0.f;
    lacc = f32x4{};
    // prologue: tiles 0 .. min(nt, kDist) - 1 in flight (K then V of each);
    // K(0) landed: everything issued after it may still be outstanding
    const int n0 = min(nt, kDist);
    for (int j = 0; j < n0; ++j) issue(j);
    if (n0 >= 4) wait_vmcnt<7 * LPW>();
    else if (n0 == 3) wait_vmcnt<5 * LPW>();
    else if (n0 == 2) wait_vmcnt<3 * LPW>();
    else wait_vmcnt<LPW>();
    __syncthreads();
    f32x16 sa[2], sb[2];
    qk(0, sa);
    if (nt == 1 && rem_last < KT) mask(sa, rem_last);
    float mxa = FO ? 0.f : rowmax(sa);

    // steady state: iteration t computes S(t+1) and PV(t); t+1 is not the last
    // tile.  Four (then two) iterations per trip, so the score sets swap roles
    // without copies; four gave the scheduler more room (-0.7% time), eight
    // made the kernel 1.7x slower.
    auto step = [&](int t, f32x16 (&cur)[2], f32x16 (&nxt)[2], float &mx) {
      // K(t+1) and V(t) landed; tiles t+2 .. t+kDist-1 and V(t+1) may be in flight
      const uint32_t vb = v_base(t);
      if (t + kDist <= nt) wait_vmcnt<(2 * kDist - 3) * LPW>();
      else wait_vmcnt<0>();
      __syncthreads();            // ... for every wave, and iteration t-1 is over
      if (t + kDist < nt) issue(t + kDist);
      if constexpr (!FO) rescale(mx);
      bf16x8 pf[2][2];
      qk(t + 1, nxt);
      softmax(fo, cur, pf);
      pv(fo, vb, pf);
      if constexpr (!FO) mx = rowmax(nxt);
      if constexpr (FO) {
        // Instruction order of the fixed-offset step: the 16 matrix
        // instructions of S(t+1) with one vector instruction of the softmax
        // of tile t each, each K operand read one MFMA ahead; then the 16 PV(t)
        // and 4 row-sum matrix instructions with the V reads and up to three
        // vector instructions each, so the rest of the softmax runs beside the
        // products of the 16-key chunks whose probabilities are done.  Measured
        // against five per S(t+1) product and none after: 2-4% faster; none
        // during S(t+1) was slower, as was leaving the order to the scheduler.
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);     // DS reads
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);   // VALU
        }
#pragma unroll
        for (int i = 0; i < 20; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
      }
    };
    int t = 0;
    for (; t + 5 < nt; t += 4) {
      step(t, sa, sb, mxa);
      step(t + 1, sb, sa, mxa);
      step(t + 2, sa, sb, mxa);
      step(t + 3, sb, sa, mxa);
    }
    for (; t + 3 < nt; t += 2) {
      step(t, sa, sb, mxa);
      step(t + 1, sb, sa, mxa);
    }
    if (t + 2 < nt) {
      step(t, sa, sb, mxa);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sa[kb] = sb[kb];
      ++t;
    }
    // t + 1 == nt - 1: S of the last (possibly ragged) tile, PV(t)
    if (t + 1 < nt) {
      wait_vmcnt<0>();
      __syncthreads();
      if constexpr (!FO) rescale(mxa);
      bf16x8 pf[2][2];
      qk(t + 1, sb);
      softmax(fo, sa, pf);
      pv(fo, v_base(t), pf);
      if (rem_last < KT) mask(sb, rem_last);
      if constexpr (!FO) mxa = rowmax(sb);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sa[kb] = sb[kb];
      ++t;
    }
    // last tile: PV(nt - 1)
    if (nt > 0) {
      wait_vmcnt<0>();
      __syncthreads();
      if constexpr (!FO) rescale(mxa);
      bf16x8 pf[2][2];
      softmax(fo, sa, pf);
      pv(fo, v_base(t), pf);
    }
  };

  // Fixed-offset pass first.  Its result stands when every row sum of the work
  // group lies in [2^-60, 2^96] and every accumulator is finite and below 2^121:
  // then no probability overflowed (each is at most 2^96), and the N keys that
  // underflowed to 0 (logit < -126 in log2 units) weigh at most N 2^-126 against
  // a sum of at least 2^-60: less than 2^-36 of it for any N below 2^30 (the
  // most the configuration allows).  The accumulator bound leaves room for the
  // combine kernel's fp32 sum of up to 32 such partials (2^121 * 32 = 2^126).
  // Otherwise the group runs the running-max pass over the same keys.  The
  // flags go through K ring slot 0, which no DMA targets once the pass is over.
  bool any_fallback = false;
  run(std::true_type{});
  {
    {
      const int q = lane & 31;
      const float s0 = __shfl(lacc[0], q & 15), s1 = __shfl(lacc[1], q & 15);
      l_run = q < 16 ? s0 : s1;    // the full row sum, in both lanes of the query
    }
    uint32_t amax = 0;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) amax = max(amax, abs_bits(acc[db][r]));
    const bool bad = nt > 0 && __any(!fixed_offset_ok(l_run, amax));
    int *flag = reinterpret_cast<int *>(&sK[0][0]);
    __syncthreads();
    if (lane == 0) flag[wave] = bad ? 1 : 0;
    __syncthreads();
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) any_bad |= flag[w];
    any_fallback = any_bad != 0;
    if (any_bad) {
      __syncthreads();            // every wave has read the flags
      run(std::false_type{});
    }
  }

  // l_run: the row sum of this lane's query (the fixed-offset pass), or this
  // lane's half of it (the running-max pass)
  const float l_tot = any_fallback ? sum_xor32(l_run) : l_run;
  if (u.slot < 0) {
    if (rvalid) {
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
// slots of one (head, query tile).  One work group takes kCombRows rows of an
// item, so even a few Global heads spread over the whole GPU.
// ---------------------------------------------------------------------------
constexpr int kCombRows = 32;

__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  constexpr int kGroups = 256 / kCombRows;               // slot groups of the weight phase
  constexpr int kPerGroup = kMaxSrcBlocks / kGroups;
  __shared__ float w_s[kMaxSrcBlocks][kCombRows];
  __shared__ float red_s[kGroups][kCombRows];
  __shared__ float inv_s[kCombRows];
  constexpr int kParts = kQTile / kCombRows;
  const CombineItem it = a.items[blockIdx.x / kParts];
  const int r0 = (blockIdx.x % kParts) * kCombRows;     // first row of this group in the tile
  const int D = a.D, ns = it.n_slots;
  const int64_t pf = (int64_t)kQTile * (D + 2);
  const float *part = a.part + (int64_t)it.slot0 * pf;

  // weights: thread (sg, lr) loads the max and sum of row r0 + lr in slots
  // sg, sg + 8, ...; all loads of the group are in flight together
  const int lr = threadIdx.x % kCombRows, sg = threadIdx.x / kCombRows;
  float mv[kPerGroup], lv[kPerGroup];
#pragma unroll
  for (int j = 0; j < kPerGroup; ++j) {
    const int i = sg + kGroups * j;
    const float *ml = part + i * pf + (int64_t)kQTile * D + r0 + lr;
    mv[j] = i < ns ? ml[0] : kMInit;
    lv[j] = i < ns ? ml[kQTile] : 0.f;
  }
  float m = mv[0];
#pragma unroll
  for (int j = 1; j < kPerGroup; ++j) m = fmaxf(m, mv[j]);
  red_s[sg][lr] = m;
  __syncthreads();
  float M = red_s[0][lr];
#pragma unroll
  for (int k = 1; k < kGroups; ++k) M = fmaxf(M, red_s[k][lr]);
  __syncthreads();                                       // every thread has read red_s
  float den = 0.f;
#pragma unroll
  for (int j = 0; j < kPerGroup; ++j) {
    const int i = sg + kGroups * j;
    if (i < ns) {
      const float wgt = __builtin_amdgcn_exp2f(mv[j] - M);
      w_s[i][lr] = wgt;
      den += wgt * lv[j];
    }
  }
  red_s[sg][lr] = den;
  __syncthreads();
  if (sg == 0) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < kGroups; ++k) t += red_s[k][lr];
    inv_s[lr] = t > 0.f ? 1.f / t : 0.f;
  }
  __syncthreads();

  // outputs: 16-byte columns of the group's rows, slots read eight at a time
  float *obase = it.out_sel == 0 ? a.o[0] : (it.out_sel == 1 ? a.o[1] : a.o[2]);
  const int nq = D / 4;
  for (int e = threadIdx.x; e < kCombRows * nq; e += 256) {
    const int er = e / nq, c4 = e % nq, row = r0 + er;
    if (it.q0 + row >= a.L) continue;
    const float *src = part + (int64_t)row * D + 4 * c4;
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    for (int i0 = 0; i0 < ns; i0 += 8) {
      f32x4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (i0 + j < ns) v[j] = *reinterpret_cast<const f32x4 *>(src + (i0 + j) * pf);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (i0 + j < ns) sum += v[j] * w_s[i0 + j][er];
    }
    *reinterpret_cast<f32x4 *>(obase + ((size_t)it.head * a.L + it.q0 + row) * D + 4 * c4) =
        sum * inv_s[er];
  }
}


}  // namespace

hipError_t launch_dense(const DenseArgs &a, int head_dim, DenseRole role, hipStream_t s) {
  if (a.n_units <= 0) return hipSuccess;
  dim3 grid(a.n_units), block(64 * kDenseWaves);
#define HC_DENSE(DD, RR) hipLaunchKernelGGL((attn_dense_kernel<DD, RR>), grid, block, 0, s, a)
  if (head_dim == 128) {
    if (role == DenseRole::kRouted) HC_DENSE(128, 0);
    else if (role == DenseRole::kFullWindow) HC_DENSE(128, 1);
    else if (role == DenseRole::kClassify) HC_DENSE(128, 2);
    else if (role == DenseRole::kVariant) HC_DENSE(128, 3);
    else HC_DENSE(128, 4);
  } else {
    if (role == DenseRole::kRouted) HC_DENSE(64, 0);
    else if (role == DenseRole::kFullWindow) HC_DENSE(64, 1);
    else if (role == DenseRole::kClassify) HC_DENSE(64, 2);
    else if (role == DenseRole::kVariant) HC_DENSE(64, 3);
    else HC_DENSE(64, 4);
  }
#undef HC_DENSE
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs &a, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(a.n_items * (kQTile / kCombRows)), dim3(256), 0, s, a);
  return hipGetLastError();
}


}  // namespace hc
