// Cache split and block append into the per-archetype buffers (Sec. 4.3), and
// the per-token statistics of the classification rule (Eq. 3 and Eq. 4).
#include "hc_device.h"

namespace hc {
namespace {
using namespace dev;

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
    const int sd = kind == 0 ? a.sink_slot[i] : a.dummy_slot[i];
    if (sd < 0) return;
    kd = a.k_sd; vd = a.v_sd; kph = a.sd_keys; mode = 0;
    kbase = (int64_t)sd * a.L;
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
    if (a.cell > 0) {
      const int cy = min(yy / a.cell, a.ncy - 1), cx = min(xx / a.cell, a.ncx - 1);
      const int ch = cy == a.ncy - 1 ? a.Hg - cy * a.cell : a.cell;
      const int cw = cx == a.ncx - 1 ? a.Wg - cx * a.cell : a.cell;
      return a.cell_off[cy * a.ncx + cx] + ((int64_t)slot * a.F + fr) * ch * cw +
             (yy - cy * a.cell) * cw + (xx - cx * a.cell);
    }
    return (((int64_t)slot * a.F + fr) * a.geo.rows + a.geo.y0 + yy) * a.geo.pitch + a.geo.x0 + xx;
  };

  const int t0 = tt * TT;
  const uint16_t *sk = a.src_k + ((size_t)(h * a.n_src + i) * a.L) * D;
  const uint16_t *sv = a.src_v + ((size_t)(h * a.n_src + i) * a.L) * D;
  // destination key of every token of the group, computed once (the Spatial
  // layouts need integer divisions)
  __shared__ int64_t skey[TT];
  if (threadIdx.x < TT) skey[threadIdx.x] = t0 + threadIdx.x < a.L ? key_of(t0 + threadIdx.x) : -1;
  __syncthreads();
  constexpr int CPR = D / 8;
  for (int c = threadIdx.x; c < TT * CPR; c += 256) {
    const int lt = c / CPR, col = c % CPR;
    const int tok = t0 + lt;
    if (tok < a.L) {
      const u32x4 kv = *reinterpret_cast<const u32x4 *>(sk + (size_t)tok * D + col * 8);
      *reinterpret_cast<u32x4 *>(kd + skey[lt] * D + col * 8) = kv;
      *reinterpret_cast<u32x4 *>(&sV[lt * VS + col * 8]) =
          *reinterpret_cast<const u32x4 *>(sv + (size_t)tok * D + col * 8);
    }
  }
  __syncthreads();
  for (int w = threadIdx.x; w < D * (TT / 8); w += 256) {
    const int d = w % D, j = w / D;
    const int tokA = t0 + 8 * j;
    if (tokA >= a.L) continue;
    const int64_t kA = skey[8 * j];
    const bool full = tokA + 7 < a.L && (kA & 7) == 0 && skey[8 * j + 7] == kA + 7;
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
        const int64_t ke = skey[8 * j + e];
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


// ---------------------------------------------------------------------------
// Per-head reduction of the token statistics: sums in float64 (a tree over the
// work group) and the 5th percentile of the Spatial cosines by radix selection
// of order statistics: the cosines become 64-bit keys in the same order, and
// eight passes of an 8-bit digit histogram narrow the key down to the k-th
// smallest, exactly (no sort, any L).
// ---------------------------------------------------------------------------
constexpr int kRedThreads = 256;

__device__ __forceinline__ uint64_t order_key(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
__device__ __forceinline__ double key_double(uint64_t k) {
  return __longlong_as_double((long long)((k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k));
}

// k-th smallest (0-based) of the Spatial cosines of one head
__device__ double select_kth(const double *tok, int L, int k, unsigned *hist, uint64_t *s_pre,
                             int *s_k) {
  const int tid = threadIdx.x;
  uint64_t prefix = 0, mask = 0;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kRedThreads) hist[i] = 0;
    __syncthreads();
    for (int t = tid; t < L; t += kRedThreads) {
      const uint64_t key = order_key(tok[4 * (size_t)t + 2]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int below = 0, b = 0;
      for (; b < 255; ++b) {
        if (below + (int)hist[b] > k) break;
        below += (int)hist[b];
      }
      *s_pre = prefix | ((uint64_t)b << shift);
      *s_k = k - below;
    }
    __syncthreads();
    prefix = *s_pre;
    k = *s_k;
    mask |= 255ull << shift;
    __syncthreads();
  }
  return key_double(prefix);
}

__global__ __launch_bounds__(kRedThreads) void cls_reduce_kernel(ClsReduceArgs a) {
  __shared__ double red[4][kRedThreads / 64];
  __shared__ unsigned hist[256];
  __shared__ uint64_t s_pre;
  __shared__ int s_k;
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int L = a.L;
  const double *tok = a.tok + (size_t)h * L * 4;
  double sum[4] = {0, 0, 0, 0};
  for (int t = tid; t < L; t += kRedThreads)
#pragma unroll
    for (int j = 0; j < 4; ++j) sum[j] += tok[4 * (size_t)t + j];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    double v = sum[j];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    if (lane == 0) red[j][w] = v;
  }
  __syncthreads();
  double tot[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    tot[j] = 0;
#pragma unroll
    for (int i = 0; i < kRedThreads / 64; ++i) tot[j] += red[j][i];
  }
  const double rank = 0.05 * (L - 1);
  const int lo = (int)floor(rank);
  const double v_lo = select_kth(tok, L, lo, hist, &s_pre, &s_k);
  const double v_hi = lo + 1 < L ? select_kth(tok, L, lo + 1, hist, &s_pre, &s_k) : v_lo;
  if (tid == 0) {
    const double p5 = v_lo + (rank - lo) * (v_hi - v_lo);
    const double mse = tot[3] / ((double)L * a.D);
    double *o = a.out + (size_t)h * 6;
    o[0] = tot[0] / L;
    o[1] = tot[1] / L;
    o[2] = tot[2] / L;
    o[3] = p5;
    o[4] = mse;
    o[5] = p5 - a.gamma * mse;
  }
}


}  // namespace

hipError_t launch_cls_reduce(const ClsReduceArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(cls_reduce_kernel, dim3(a.n_heads), dim3(kRedThreads), 0, s, a);
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
