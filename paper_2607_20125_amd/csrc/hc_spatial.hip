// Spatial softmax attention: each query against the (2r+1)^2 positions around
// it in every window frame, addressed by index arithmetic (Sec. 4.2 Spatial
// proxy; the deployed Spatial path of this library).
#include "hc_device.h"

#include <algorithm>

namespace hc {
namespace {
using namespace dev;

// ---------------------------------------------------------------------------
// Spatial kernel.  One work group = F waves; wave f owns the 32 queries of
// query frame f, rows y0..y0+3, columns x0..x0+7 (lane n: row y0 + n/8,
// column x0 + n%8).  A query (f, y, x) attends to key rows y-r..y+r and columns
// x-r..x+r of every window frame, so the F waves share one key set: the halo
// rows y0-r..y0+3+r, columns [8 gs, 8 gs + RW) (G aligned 8-key groups covering
// x0-r..x0+7+r).  The halo is streamed per key frame in tiles of 32·KB keys
// (32·KB/RW halo rows) by DMA into a K ring of 2 and a V ring of 3 buffers,
// issued two tiles ahead, one barrier per tile; as in the dense kernel, the
// matrix cores compute S(t+1) while the vector units turn S(t) into P(t).
// Small tiles keep the LDS of a work group at 40 KB and a wave under 168
// registers, so four work groups (twelve waves) share a CU and hide each
// other's DMA waits and softmax.  Keys outside a query's window, outside the
// frame or in clipped rows get no weight; the masks come from index
// arithmetic only.
// ---------------------------------------------------------------------------
// kRole only separates the symbols of the callers in profiles: 0 routed step,
// 1 classification proxy (radius r_p), 2 a table of Spatial heads only.
template <int D, int G, int F, int KB, int kRole>
__global__ __launch_bounds__(64 * F, (F >= 3 ? 3 : F)) void attn_spatial_kernel(SpatialArgs a) {
  constexpr int TK = 32 * KB;            // keys per tile
  constexpr int NKK = D / 16;
  constexpr int NDB = D / 32;
  constexpr int RW = 8 * G;              // keys per halo row
  constexpr int RPT = TK / RW;           // halo rows per tile
  static_assert(RPT >= 1 && RPT * RW == TK, "tile shape");
  constexpr int CPR = D / 8;             // 16-byte chunks per K row
  constexpr int KRPI = 64 / CPR;         // K rows per 1 KB DMA instruction
  constexpr int TILE = TK * D;           // elements of K (or V) per tile
  constexpr int NINS = TILE / 512;       // 1 KB DMA instructions per tensor per tile
  constexpr int RK = 2, RV = 3;          // K and V ring buffers
  constexpr int MAXI = (NINS + F - 1) / F;   // DMA instructions per wave per tensor, at most
  __shared__ __attribute__((aligned(1024))) uint16_t sK[RK][TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[RV][TILE];

  const int tid = threadIdx.x;
  // wave-uniform values live in scalar registers, so conditions on them branch uniformly
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, g = lane >> 5;
  const int my_ins = NINS / F + (wave < NINS % F ? 1 : 0);

  const int bid = xcd_unit(blockIdx.x, gridDim.x);
  const int ct = bid % a.n_ct;
  const int rg = (bid / a.n_ct) % a.n_rowgroups;
  const int hs = (bid / a.n_ct / a.n_rowgroups) % a.n_sp;
  const int split = bid / a.n_ct / a.n_rowgroups / a.n_sp;

  const int Hg = a.Hg, Wg = a.Wg, r = a.r;
  const int P = Hg * Wg;
  const int c = a.c_lo + ct;
  const int x0 = 8 * c - 8 + (r & 7);
  const int gs = c - 1 - (r >> 3);        // first halo group (may lie outside the frame)
  const int head = a.heads[hs];
  const int y0 = kSpRows * rg;

  // query slot of this lane
  const int qy = y0 + (n >> 3), qx = x0 + (n & 7);
  const bool qvalid = qy < Hg && qx >= 0 && qx < Wg;
  const int tq = qvalid ? wave * P + qy * Wg + qx : 0;
  bf16x8 qf[NKK];
  {
    const uint16_t *qp = a.q + ((size_t)head * a.L + tq) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qf[kk] = qvalid ? ld_g16(qp + 16 * kk + 8 * g) : bf16x8{};
    // Q in registers before any DMA is issued: the compiler then has no load of
    // its own pending inside the key loop (it cannot count the DMAs)
    wait_vmcnt<0>();
  }

  const uint16_t *kb = a.k + (size_t)hs * a.head_stride;
  const uint16_t *vb = a.v + (size_t)hs * a.head_stride;
  const int hrows = kSpRows + 2 * r;                 // halo rows per key frame
  // tiles of a key frame that hold at least one halo row inside the frame (at
  // the top and bottom borders the others are skipped): tj_lo .. tj_hi
  const int tj_lo = max(0, r - y0) / RPT;
  const int tj_hi = min(hrows - 1, Hg - 1 - y0 + r) / RPT;
  const int tpf = tj_hi - tj_lo + 1;                 // tiles per key frame
  // key frames [f_lo, f_hi) of this group's split of the window
  const int nf = a.n_slots * F;
  const int f_lo = split * nf / a.n_split, f_hi = (split + 1) * nf / a.n_split;
  const int nt = (f_hi - f_lo) * tpf;
  const int64_t row_elems = (int64_t)a.geo.pitch * D;
  const int64_t frame_elems = (int64_t)a.geo.rows * row_elems;
  const int ngrp = a.geo.pitch / 8;

  // DMA sources, fixed per lane: lane l of this wave's k-th instruction
  // (ins = wave + k F) moves 16 bytes of K row lr = ins KRPI + l / CPR (key slot
  // kperm(lr), chunk kswz(lr, .)) and 16 bytes of the 8-key-grouped V tile, at
  // koff / voff (elements) past the first element of the tile's first halo
  // row.  A halo column group outside the frame is read from the nearest group
  // of the same row; its keys are masked like any key outside the frame.
  auto col_elems = [&](int key) {          // offset of tile key `key` from its row's start
    const int xk = 8 * gs + key % RW;
    const int gq = min(max(xk >> 3, 0), ngrp - 1);
    return (int64_t)(key / RW) * row_elems + (int64_t)(8 * gq + (xk & 7)) * D;
  };
  // This wave moves the pieces ins0 .. ins0 + my_ins - 1 of each tile: 1 KB
  // of LDS each, contiguous, so a run of up to four sets M0 once
  // (lds_dma16_runs).  ka / va hold the source offsets in bytes less the
  // 1024 k that the k-th instruction's immediate offset adds, and 8 KB above a
  // tile base taken 8 KB low, so that none goes below zero.
  const int ins0 = wave * (NINS / F) + min(wave, NINS % F);
  uint32_t ka[MAXI], va[MAXI];
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int ins = min(ins0 + k, NINS - 1);
    const int lr = ins * KRPI + lane / CPR;
    const int kap = (lr & ~31) | kperm(lr & 31);
    ka[k] = (uint32_t)((col_elems(kap) + kswz<D>(lr, lane % CPR) * 8) * 2 + 8192 - 1024 * k);
    const int e0 = ins * 512 + lane * 8;                // element of the V tile
    const int grp = e0 / (8 * D);                       // its 8-key group
    va[k] = (uint32_t)((col_elems(8 * grp) + e0 % (8 * D)) * 2 + 8192 - 1024 * k);
  }
  static_assert(MAXI <= 8, "DMA offsets");
  // this wave's first DMA target in ring slot 0
  const uint32_t k_dst = lds_addr(&sK[0][ins0 * 512]);
  const uint32_t v_dst = lds_addr(&sV[0][ins0 * 512]);
  // tile tj of key frame phi: halo rows y0-r+tj RPT .. (rows above the frame,
  // at most RPT-1 of them, lie in the storage before it)
  auto issue = [&](int phi, int tj, int kbuf, int vbuf) {
    const int64_t tb = (int64_t)phi * frame_elems + (int64_t)(y0 - r + tj * RPT) * row_elems;
    const uint16_t *kt = kb + tb - 4096, *vt = vb + tb - 4096;
    const uint32_t kd = k_dst + (uint32_t)(kbuf * TILE * 2);
    const uint32_t vd = v_dst + (uint32_t)(vbuf * TILE * 2);
    // every wave moves MAXI - 1 pieces of each tensor, the first NINS % F
    // waves one more (K first, then V)
    constexpr int L = MAXI - 1;
    lds_dma16_runs<L>(kt, ka, kd);
    if (my_ins > L) lds_dma16_run<1>(kt + 512 * L, ka + L, kd + 1024 * L);
    lds_dma16_runs<L>(vt, va, vd);
    if (my_ins > L) lds_dma16_run<1>(vt + 512 * L, va + L, vd + 1024 * L);
  };

  // Masks are kept as wave-wide lane masks in scalar registers.  Score
  // register rr of chain kb holds, in lane half g, the key in tile slot
  // kslot(kb, rr, g); its column decides cm[] once, its halo row decides per
  // tile together with the lane's query row (rowlive).
  auto kslot = [](int kb, int rr, int gg) { return 32 * kb + kperm(8 * (rr >> 2) + 4 * gg + (rr & 3)); };
  uint64_t cm[16 * KB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int xk = 8 * gs + (g ? kslot(kb, rr, 1) : kslot(kb, rr, 0)) % RW;
      cm[16 * kb + rr] = __builtin_amdgcn_ballot_w64(xk >= 0 && xk < Wg && xk - qx <= r && qx - xk <= r);
    }
  // halo rows in this lane's window and inside the frame (hrows <= 28 < 32)
  uint32_t rowlive = 0;
  for (int hr = n >> 3; hr <= (n >> 3) + 2 * r; ++hr) {
    const int yy = y0 - r + hr;
    rowlive |= (yy >= 0 && yy < Hg) ? 1u << hr : 0u;
  }
  // LDS element offset of this lane's K operand row; chunk 2kk+g of it sits at
  // (kswz(n, g) * 8) ^ (16 kk) since the swizzle is an XOR of the chunk index
  const int krow = n * D + kswz<D>(n, g) * 8;

  f32x16 acc[NDB];
  float m_run, l_run;
  // Row sums of the fixed-offset pass on the matrix cores, as in the dense
  // kernel: each 16-key chunk of P (lane l: query l % 32, key half l / 32) is
  // the B operand of a 16x16x32 product with a 0/1 selector whose row 0 takes
  // k-groups 0 and 2 (query n of column n) and row 1 groups 1 and 3 (query
  // n + 16); lane n < 16 then holds the sums of queries n and n + 16.
  f32x4 lacc;
  bf16x8 sel;
  {
    const int i = lane & 15, kg = lane >> 4;
    const float v = (i == 0 && (kg & 1) == 0) || (i == 1 && (kg & 1) == 1) ? 1.f : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sel[e] = (__bf16)v;
  }
  const float sl2 = a.scale_log2;
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};

  // Scores start from the tile's mask (0 or -inf) as the matrix cores'
  // accumulator input: one select per score register before the products,
  // which can overlap the first K operand reads, and S = mask + K Q^T needs
  // no pass afterwards (-inf plus finite products stays -inf).
  auto init_mask = [&](int tjx, f32x16 (&sx)[KB]) {
    uint64_t rowok[RPT];
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      rowok[i] = __builtin_amdgcn_ballot_w64((rowlive >> (tjx * RPT + i)) & 1u);
    constexpr uint64_t kLo = 0x00000000FFFFFFFFull;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int i0 = kslot(kb, rr, 0) / RW, i1 = kslot(kb, rr, 1) / RW;
        const uint64_t live = i0 == i1 ? rowok[i0] : ((rowok[i0] & kLo) | (rowok[i1] & ~kLo));
        const bool keep = __builtin_amdgcn_inverse_ballot_w64(live & cm[16 * kb + rr]);
        sx[kb][rr] = keep ? 0.f : -INFINITY;
      }
  };
  // byte offset of this lane's K operand row; chunk 2kk+g sits at kbyte ^ (32 kk)
  const uint32_t kbyte = (uint32_t)krow * 2u;
  auto qk_acc = [&](const uint16_t *kt, f32x16 (&sx)[KB]) {
    uint32_t kr = kbyte;
    asm volatile("" : "+v"(kr));   // per-tile XORs instead of NKK held addresses
    const char *kc = reinterpret_cast<const char *>(kt);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(kc + 64 * kb * D + (kr ^ (32u * kk)));
        sx[kb] = mfma32(kf, qf[kk], sx[kb]);
      }
  };
  auto rowmax = [&](const f32x16 (&sx)[KB]) -> float {
    float mx = sx[0][0];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int rr = (kb == 0 ? 1 : 0); rr < 16; ++rr) mx = fmaxf(mx, sx[kb][rr]);
    return max_xor32(mx) * sl2;
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
  // fixed-offset pass (FO): 2^(s * scale * log2 e), no running max; its row
  // sums go through the matrix cores (lacc), the running-max pass adds the
  // rounded probabilities two per v_dot2 against (1, 1)
  auto softmax = [&](auto fo, const f32x16 (&sx)[KB], bf16x8 (&pf)[KB][2]) {
    constexpr bool FO = decltype(fo)::value;
    const float nm = -m_run;
    float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pf[kb][h][e] = (__bf16)__builtin_amdgcn_exp2f(FO ? sx[kb][8 * h + e] * sl2
                                                           : fmaf(sx[kb][8 * h + e], sl2, nm));
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
  // V operands: one lane base per tile, the (kb, h, db) parts as immediate offsets
  const int vlane = (g * D + n) * 8;
  auto pv = [&](auto fo, const uint16_t *vt, const bf16x8 (&pf)[KB][2]) {
    constexpr bool FO = decltype(fo)::value;
    const uint16_t *vl = vt + vlane;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(vl + ((4 * kb + 2 * h) * D + 32 * db) * 8);
          acc[db] = mfma32(vf, pf[kb][h], acc[db]);
        }
        if constexpr (FO) lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, pf[kb][h], lacc, 0, 0, 0);
      }
  };

  auto wait_but = [&](int tiles_k, int tiles_v) {   // my DMAs still allowed in flight
    // (the per-wave count is NINS/F or one more; both are compile-time branches)
    const int k = tiles_k + tiles_v;
    if (my_ins == MAXI) {
      if (k == 3) wait_vmcnt<3 * MAXI>(); else if (k == 2) wait_vmcnt<2 * MAXI>();
      else if (k == 1) wait_vmcnt<MAXI>(); else wait_vmcnt<0>();
    } else {
      constexpr int m = NINS / F;
      if (k == 3) wait_vmcnt<3 * m>(); else if (k == 2) wait_vmcnt<2 * m>();
      else if (k == 1) wait_vmcnt<m>(); else wait_vmcnt<0>();
    }
  };

  // One pass over the group's key tiles: the running-max pass (fo = false,
  // online softmax with lazy rescaling) or the fixed-offset pass (fo = true,
  // offset 0, no row max and no rescale; exact while nothing overflows or
  // underflows, checked on the row sums afterwards).
  auto run = [&](auto fo) {
    constexpr bool FO = decltype(fo)::value;
#pragma unroll
    for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
    m_run = FO ? 0.f : kMInit;
    l_run = 0.f;
    lacc = f32x4{};
    // issue stream
    int iphi = f_lo, itj = tj_lo, ikb = 0, ivb = 0;
    auto issue_next = [&]() {
      issue(iphi, itj, ikb, ivb);
      ikb = ikb == RK - 1 ? 0 : ikb + 1;
      ivb = ivb == RV - 1 ? 0 : ivb + 1;
      if (++itj > tj_hi) { itj = tj_lo; ++iphi; }
    };
    if (nt > 0) issue_next();
    if (nt > 1) issue_next();

    // K ring of two, V ring of three: iteration t computes S(t+1) while the
    // vector units turn S(t) into P(t), then PV(t) (as in the dense kernel)
    if (nt > 1) wait_but(1, 2); else wait_but(0, 1);   // K(0) landed
    __syncthreads();
    f32x16 sa[KB], sb[KB];
    // halo tile of key tile t is tj_lo + t mod tpf; tj tracks tile t+1 in the steps
    int tj = tj_lo;
    init_mask(tj, sa);
    qk_acc(sK[0], sa);
    if (++tj > tj_hi) tj = tj_lo;
    float mxa = FO ? 0.f : rowmax(sa);
    auto step = [&](int t, f32x16 (&cur)[KB], f32x16 (&nxt)[KB]) {
      // K(t+1) and V(t) landed, V(t+1) may be in flight
      wait_but(0, 1);
      __syncthreads();
      if (t + 2 < nt) issue_next();
      if constexpr (!FO) rescale(mxa);
      init_mask(tj, nxt);
      qk_acc(sK[(t + 1) & 1], nxt);
      if (++tj > tj_hi) tj = tj_lo;
      bf16x8 pf[KB][2];
      softmax(fo, cur, pf);
      pv(fo, sV[t % 3], pf);
      if constexpr (!FO) mxa = rowmax(nxt);
    };
    int t = 0;
    for (; t + 4 < nt; t += 4) {
      step(t, sa, sb);
      step(t + 1, sb, sa);
      step(t + 2, sa, sb);
      step(t + 3, sb, sa);
    }
    for (; t + 2 < nt; t += 2) {
      step(t, sa, sb);
      step(t + 1, sb, sa);
    }
    if (t + 1 < nt) {
      step(t, sa, sb);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) sa[kb] = sb[kb];
      ++t;
    }
    if (nt > 0) {
      wait_but(0, 0);
      __syncthreads();
      if constexpr (!FO) rescale(mxa);
      bf16x8 pf[KB][2];
      softmax(fo, sa, pf);
      pv(fo, sV[t % 3], pf);
    }
  };

  // Fixed-offset pass first; it stands when the row sum of every query of the
  // work group lies in [2^-60, 2^96] and every accumulator is below 2^121.
  // Then no probability overflowed, and the keys flushed to 0 (logit below
  // -126 in log2 units) weigh at most N 2^-126 against a sum of at least
  // 2^-60, with N <= W F (2r+1)^2 <= 32 * 4 * 625 < 2^17 keys per query: less
  // than 2^-49 of it.  The accumulator bound leaves room for the merge of up
  // to 8 split partials (and the dense kernel's 32 block partials) in fp32.
  // Lanes without a query (outside the frame) do not vote: at small radii
  // some have no key in the frame at all.  Otherwise the group reruns the
  // keys with the running max.  The flags go through K ring slot 0, which no
  // DMA targets once the pass is over.
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
      for (int rr = 0; rr < 16; ++rr) amax = max(amax, abs_bits(acc[db][rr]));
    const bool bad = nt > 0 && __any(qvalid && !fixed_offset_ok(l_run, amax));
    int *flag = reinterpret_cast<int *>(&sK[0][0]);
    __syncthreads();
    if (lane == 0) flag[wave] = bad ? 1 : 0;
    __syncthreads();
    int any_bad = 0;
#pragma unroll
    for (int w = 0; w < F; ++w) any_bad |= flag[w];
    any_fallback = any_bad != 0;
    if (any_bad) {
      __syncthreads();            // every wave has read the flags
      run(std::false_type{});
    }
  }

  // l_run: the row sum of this lane's query (the fixed-offset pass), or this
  // lane's half of it (the running-max pass)
  const float l_tot = any_fallback ? sum_xor32(l_run) : l_run;
  if (!qvalid) return;
  float inv = 1.f;
  float *op;
  if (a.n_split == 1) {
    inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    op = a.o + ((size_t)head * a.L + tq) * D;
  } else {
    const size_t row = ((size_t)split * a.n_sp + hs) * a.L + tq;
    op = a.part + row * D;
    if (g == 0) {
      a.part_ml[2 * row] = m_run;
      a.part_ml[2 * row + 1] = l_tot;
    }
  }
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

// ---------------------------------------------------------------------------
// Merge of the per-split partial results of the Spatial heads: for each
// (head, query) O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, M = max_s m_s.
// One thread per 4 output dims.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void spatial_merge_kernel(SpatialArgs a, int D) {
  const int nq = D / 4;
  const int64_t total = (int64_t)a.n_sp * a.L * nq;
  const int64_t plane = (int64_t)a.n_sp * a.L;        // rows per split
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t row = e / nq;                          // hs * L + token
    const int c4 = (int)(e % nq);
    float M = kMInit;
    for (int sp = 0; sp < a.n_split; ++sp) M = fmaxf(M, a.part_ml[2 * (sp * plane + row)]);
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int sp = 0; sp < a.n_split; ++sp) {
      const int64_t rs = sp * plane + row;
      const float w = __builtin_amdgcn_exp2f(a.part_ml[2 * rs] - M);
      den += w * a.part_ml[2 * rs + 1];
      sum += w * *reinterpret_cast<const f32x4 *>(a.part + rs * D + 4 * c4);
    }
    const int hs = (int)(row / a.L), tok = (int)(row % a.L);
    const float inv = den > 0.f ? 1.f / den : 0.f;
    *reinterpret_cast<f32x4 *>(a.o + ((size_t)a.heads[hs] * a.L + tok) * D + 4 * c4) = sum * inv;
  }
}

template <int D, int F, int R>
hipError_t launch_spatial_f(const SpatialArgs &a, dim3 grid, hipStream_t s) {
  const int G = spatial_groups(a.r);
  dim3 block(64 * F);
  if (G == 1) hipLaunchKernelGGL((attn_spatial_kernel<D, 1, F, 1, R>), grid, block, 0, s, a);
  else if (G == 2) hipLaunchKernelGGL((attn_spatial_kernel<D, 2, F, 1, R>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((attn_spatial_kernel<D, 4, F, 1, R>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <int D, int R>
hipError_t launch_spatial_d(const SpatialArgs &a, dim3 grid, hipStream_t s) {
  switch (a.F) {
    case 1: return launch_spatial_f<D, 1, R>(a, grid, s);
    case 2: return launch_spatial_f<D, 2, R>(a, grid, s);
    case 3: return launch_spatial_f<D, 3, R>(a, grid, s);
    default: return launch_spatial_f<D, 4, R>(a, grid, s);
  }
}

template <int D>
hipError_t launch_spatial_r(const SpatialArgs &a, dim3 grid, SpatialRole role, hipStream_t s) {
  if (role == SpatialRole::kRouted) return launch_spatial_d<D, 0>(a, grid, s);
  if (role == SpatialRole::kClassify) return launch_spatial_d<D, 1>(a, grid, s);
  return launch_spatial_d<D, 2>(a, grid, s);
}

}  // namespace

hipError_t launch_spatial(const SpatialArgs &a, int head_dim, SpatialRole role, hipStream_t s) {
  const int64_t nblk = (int64_t)a.n_sp * a.n_rowgroups * a.n_ct * a.n_split;
  if (nblk <= 0) return hipSuccess;
  if (a.F < 1 || a.F > 4 || a.n_split < 1 || (a.n_split > 1 && (!a.part || !a.part_ml)))
    return hipErrorInvalidValue;
  dim3 grid((unsigned)nblk);
  hipError_t e = head_dim == 128 ? launch_spatial_r<128>(a, grid, role, s)
                                 : launch_spatial_r<64>(a, grid, role, s);
  if (e != hipSuccess || a.n_split == 1) return e;
  const int64_t threads = (int64_t)a.n_sp * a.L * (head_dim / 4);
  const unsigned blocks = (unsigned)std::min<int64_t>((threads + 255) / 256, 8192);
  hipLaunchKernelGGL(spatial_merge_kernel, dim3(blocks), dim3(256), 0, s, a, head_dim);
  return hipGetLastError();
}

}  // namespace hc
