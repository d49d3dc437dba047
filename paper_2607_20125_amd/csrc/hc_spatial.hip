// Spatial softmax attention: each query against the (2r+1)^2 positions around
// it in every window frame, addressed by index arithmetic (Sec. 4.2 Spatial
// proxy; the deployed Spatial path of this library).
#include "hc_device.h"

namespace hc {
namespace {
using namespace dev;

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


}  // namespace

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


}  // namespace hc
