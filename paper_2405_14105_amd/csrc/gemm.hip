// Window GEMM: Y[M, N] = X[M, K] . W[N, K]^T for the k+1 (or a few dozen)
// rows of a verification window, with fused epilogues.
//
// The k+1 window rows are one batch through the target (Section 2): every
// weight byte is read once per verification while each weight feeds only M
// (6..64) rows, so the kernel is bound by streaming W from HBM.  Design:
//  * W is pre-packed into 1 KB MFMA tiles (16 rows x 32 k, bf16), one
//    dwordx4 per lane, so every wavefront load is 1 KB contiguous and lands
//    in registers already in A-operand order (no LDS round trip for W);
//  * activations come as pre-split bf16 hi/lo packs (B operand, L2-resident)
//    and each tile costs two 16x16x32 MFMAs, giving ~fp32 accuracy;
//  * a workgroup owns NBW n-blocks (16 features each) and its NW waves split
//    K; partial tiles are reduced through LDS in a fixed order
//    (deterministic, no float atomics) and handed to the epilogue;
//  * weight loads for the next U k-blocks are issued before the MFMAs of the
//    current ones so every wave keeps U*NBW KB in flight.
#include <algorithm>

#include "device_util.h"

namespace dsi {

namespace {

// EPI_RESID inputs of the one epilogue item a thread owns (residual and gain
// values), loaded before the main loop so that their latency is hidden.
struct ResidIn {
  float4 x, g;
};
template <int MT, int NBW, int NW>
__device__ __forceinline__ ResidIn resid_prefetch(const GemmArgs& a, int nb0) {
  static_assert(NBW * MT <= NW, "finish() must give each thread at most one item");
  ResidIn r{};
  const int it = threadIdx.x;
  if (it < NBW * MT * 64) {
    const int l = it & 63, jm = it >> 6;
    const int nb = nb0 + jm / MT, m = (jm % MT) * 16 + (l & 15);
    if (nb < a.Nb && m < a.M) {
      const int n0 = nb * 16 + (l >> 4) * 4;
      r.x = *(const float4*)(a.epi.x + (size_t)m * a.epi.ld + n0);
      r.g = *(const float4*)(a.epi.gain + n0);
    }
  }
  return r;
}

// Returns the sum of the squared residual values it wrote (EPI_RESID), else 0.
template <int WT, int EPI>
__device__ __forceinline__ float epilogue(const EpiArgs& e, int nb, int r0, int m, int split, f32x4 s,
                                          const ResidIn& pre) {
  switch (EPI) {
    case EPI_STORE: {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = nb * 16 + r0 + j;
        if (n < e.n_valid) e.out[(size_t)m * e.ld + n] = s[j];
      }
      break;
    }
    case EPI_PARTRES: {
      // device-scope stores: written through to the point where the
      // group's last workgroup reads them (no L2 write-back needed)
      float* o = e.out + split * e.part_stride + (size_t)m * e.ld;
      const int n0 = nb * 16 + r0;
      if (n0 + 3 < e.n_valid) {
        store4_device(o + n0, s);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (n0 + j < e.n_valid) __hip_atomic_store(o + n0 + j, s[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      break;
    }
    case EPI_PART: {
      float* o = e.out + split * e.part_stride + (size_t)m * e.ld;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = nb * 16 + r0 + j;
        if (n < e.n_valid) o[n] = s[j];
      }
      break;
    }
    case EPI_SILU: {
      // rows 4g+0, 4g+1: gate of features f, f+1; rows 4g+2, 4g+3: up
      const int f = nb * 8 + (r0 >> 2) * 2;
      if (f < e.ff) pack_store(e.pack, WT, m, f, silu_f(s[0]) * s[2]);
      if (f + 1 < e.ff) pack_store(e.pack, WT, m, f + 1, silu_f(s[1]) * s[3]);
      break;
    }
    case EPI_QKV: {
      const int hd = e.hd;
      const int bph = hd >> 4;                       // 16-row blocks per head
      const int nq = e.n_heads * bph, nk = e.n_kv * bph;
      const int R = e.rows.rows_per_window;
      const int win = e.rows.window0 + m / R;
      const int pos = e.rows.lens[win] + (m % R);
      if (nb < nq + nk) {
        const int sb = nb < nq ? nb : nb - nq;
        const int h = sb / bph;
        const int ja = (sb % bph) * 8 + (r0 >> 2) * 2;   // pair indices ja, ja+1
        const int half = hd >> 1;
        const float2 ca = e.rope[(size_t)m * half + ja];
        const float2 cb = e.rope[(size_t)m * half + ja + 1];
        const float a1 = s[0] * ca.x - s[2] * ca.y, a2 = s[2] * ca.x + s[0] * ca.y;
        const float b1 = s[1] * cb.x - s[3] * cb.y, b2 = s[3] * cb.x + s[1] * cb.y;
        if (nb < nq) {
          float* qr = e.q_out + (size_t)m * (e.n_heads * hd) + h * hd;
          qr[ja] = a1;
          qr[ja + half] = a2;
          qr[ja + 1] = b1;
          qr[ja + 1 + half] = b2;
        } else {
          const size_t base = (((size_t)win * e.n_kv + h) * e.maxlen + pos) * hd;
          if (e.kv_bf16) {
            uint16_t* kc = (uint16_t*)e.kcache + base;
            kc[ja] = f2bf_bits(a1);
            kc[ja + half] = f2bf_bits(a2);
            kc[ja + 1] = f2bf_bits(b1);
            kc[ja + 1 + half] = f2bf_bits(b2);
          } else {
            float* kc = (float*)e.kcache + base;
            kc[ja] = a1;
            kc[ja + half] = a2;
            kc[ja + 1] = b1;
            kc[ja + 1 + half] = b2;
          }
        }
      } else {
        const int vb = nb - nq - nk;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = vb * 16 + r0 + j;
          const int h = n / hd, dd = n % hd;
          const size_t idx = ((((size_t)win * e.n_kv + h) * (e.maxlen >> 5) + (pos >> 5)) * hd + dd) * 32 +
                             (pos & 31);
          if (e.kv_bf16) ((uint16_t*)e.vcache)[idx] = f2bf_bits(s[j]);
          else ((float*)e.vcache)[idx] = s[j];
        }
      }
      break;
    }
    case EPI_RESID: {
      // four consecutive features n0..n0+3 of row m (x, gain prefetched)
      const int n0 = nb * 16 + r0;
      const float xn[4] = {pre.x.x + s[0], pre.x.y + s[1], pre.x.z + s[2], pre.x.w + s[3]};
      *(float4*)(e.x + (size_t)m * e.ld + n0) = float4{xn[0], xn[1], xn[2], xn[3]};
      const float y[4] = {xn[0] * pre.g.x, xn[1] * pre.g.y, xn[2] * pre.g.z, xn[3] * pre.g.w};
      pack_store4(e.pack, WT, m, n0, y);
      return xn[0] * xn[0] + xn[1] * xn[1] + xn[2] * xn[2] + xn[3] * xn[3];
    }
  }
  return 0.f;
}

// RMSNorm scale of each input row from the per-n-block sums of squares the
// producing GEMM wrote (EPI_RESID, layout [row][ssq_n]):
// rs[m] = 1/sqrt(sum_nb ssq[m][nb] / d + eps).  One wave per row: lane l sums
// entries l, l+64, ... and a butterfly finishes, a fixed order that does not
// depend on the number of rows.
template <int NW>
__device__ __forceinline__ void row_scales(const GemmArgs& a, float* rs) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int m = w; m < a.M; m += NW) {
    const float* p = a.ssq + (size_t)m * a.ssq_n;
    float sum = 0.f;
#pragma unroll 4
    for (int i = lane; i < a.ssq_n; i += 64) sum += p[i];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
    if (lane == 0) rs[m] = 1.0f / sqrtf(sum / (float)a.norm_d + a.eps);
  }
}

// EPI_PARTRES tail (see the Epi enum).  The partials are device-scope
// stores; every wave waits until its stores are complete before the
// workgroup counts its arrival (a device-scope atomic), and the last arrival
// reads the partials with device-scope loads, so partials written from
// another XCD are seen without a write-back or invalidation of any L2.
// Items are 4 consecutive features of one row, one item per thread (at most
// MT*16 rows x NBW n-blocks x 4 <= NW*64); the four lanes of one (row,
// n-block) are adjacent, so the n-block's sum of squares is a two-step
// butterfly.  The residual and gain values of the thread's item are loaded
// at the start of the kernel (fold_prefetch), off the critical path.
struct FoldIn {
  float4 x, g;
};
template <int MT, int NBW, int NW>
__device__ __forceinline__ FoldIn fold_prefetch(const GemmArgs& a, int nb0, int nbv) {
  static_assert(MT * NBW <= NW, "one fold item per thread");
  FoldIn f{};
  const int it = threadIdx.x;
  if (it < a.M * nbv * 4) {
    const int q = it & 3, jm = it >> 2;
    const int m = jm / nbv, n0 = (nb0 + jm % nbv) * 16 + q * 4;
    f.x = *(const float4*)(a.epi.x + (size_t)m * a.epi.ld + n0);
    f.g = *(const float4*)(a.epi.gain + n0);
  }
  return f;
}

template <int WT, int NW>
__device__ __forceinline__ void part_fold(const GemmArgs& a, int nb0, int nbv, const FoldIn& pre) {
  __shared__ int s_last;
  const EpiArgs& e = a.epi;
  const int g = blockIdx.x / a.S;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    s_last = __hip_atomic_fetch_add(e.cnt + g, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == a.S - 1;
  __syncthreads();
  if (!s_last) return;
  {
    const int it = threadIdx.x;
    const bool ok = it < a.M * nbv * 4;
    const int q = it & 3, jm = it >> 2;
    const int m = ok ? jm / nbv : 0, nb = nb0 + (ok ? jm % nbv : 0);
    const int n0 = nb * 16 + q * 4;
    float sq = 0.f;
    if (ok) {
      float4 xv = pre.x;
      for (int sp = 0; sp < a.S; ++sp) {
        const float* pp = e.out + sp * e.part_stride + (size_t)m * e.ld + n0;
        xv.x += __hip_atomic_load(pp + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        xv.y += __hip_atomic_load(pp + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        xv.z += __hip_atomic_load(pp + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        xv.w += __hip_atomic_load(pp + 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      *(float4*)(e.x + (size_t)m * e.ld + n0) = xv;
      if (e.copy) *(float4*)(e.copy + (size_t)m * e.ld + n0) = xv;
      const float4 gv = pre.g;
      const float y[4] = {xv.x * gv.x, xv.y * gv.y, xv.z * gv.z, xv.w * gv.w};
      pack_store4(e.pack, WT, m, n0, y);
      sq = xv.x * xv.x + xv.y * xv.y + xv.z * xv.z + xv.w * xv.w;
    }
    sq += __shfl_xor(sq, 1);
    sq += __shfl_xor(sq, 2);
    if (ok && q == 0) e.ssq[(size_t)m * a.Nb + nb] = sq;
  }
  if (threadIdx.x == 0) __hip_atomic_store(e.cnt + g, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// rs: per-row RMSNorm scales (row_scales) or nullptr.  The iteration count
// is uniform across a wave, so the EPI_RESID lane reduction is safe.
// NBW here is the number of n-blocks of one reduction round (red holds
// NW x NBW x MT tiles); n-blocks j >= nvalid of the round are skipped.
template <int WT, int EPI, int MT, int NBW, int NW>
__device__ __forceinline__ void finish(const GemmArgs& a, const f32x4* red, const float* rs, int nb0,
                                       int nvalid, int split, const ResidIn& pre) {
  constexpr int ACC = NBW * MT;
  for (int it = threadIdx.x; it < ACC * 64; it += NW * 64) {
    const int l = it & 63, jm = it >> 6;
    const int j = jm / MT, t = jm % MT;
    f32x4 v = red[jm * 64 + l];
    for (int ww = 1; ww < NW; ++ww) v += red[(ww * ACC + jm) * 64 + l];
    const int nb = nb0 + j, m = t * 16 + (l & 15);
    const bool ok = j < nvalid && nb < a.Nb && m < a.M;
    if (ok && rs) v *= rs[m];
    float sq = 0.f;
    if (ok) sq = epilogue<WT, EPI>(a.epi, nb, (l >> 4) * 4, m, split, v, pre);
    if constexpr (EPI == EPI_RESID) {
      // lanes l, l+16, l+32, l+48 hold the 16 features of row m
      sq += __shfl_xor(sq, 16);
      sq += __shfl_xor(sq, 32);
      if (ok && l < 16) a.epi.ssq[(size_t)m * a.Nb + nb] = sq;
    }
  }
}

// workgroup -> (n-block group, K split); wave -> contiguous k-blocks of it
struct Work {
  int nb0, nbv, split, kb_beg, kb_end;
};
template <int NBW, int NW>
__device__ __forceinline__ Work work_of(const GemmArgs& a) {
  Work w;
  const int g = blockIdx.x / a.S;
  w.split = blockIdx.x % a.S;
  w.nb0 = g * NBW;
  w.nbv = min(NBW, a.Nb - w.nb0);
  const int k0 = (w.split * a.Kb) / a.S;
  const int k1 = ((w.split + 1) * a.Kb) / a.S;
  const int per = (k1 - k0 + NW - 1) / NW;
  const int wave = threadIdx.x >> 6;
  w.kb_beg = min(k1, k0 + wave * per);
  w.kb_end = min(k1, w.kb_beg + per);
  return w;
}

// n-blocks per LDS reduction round: all of them when NW x NBW x MT tiles
// (1 KB each) fit in kRedTiles KB, else as many as fit (several rounds)
constexpr int kRedTiles = 128;
template <int MT, int NBW, int NW>
constexpr int red_nb() {
  return NW * NBW * MT <= kRedTiles ? NBW : (kRedTiles / (NW * MT) > 0 ? kRedTiles / (NW * MT) : 1);
}

template <int MT, int NBW, int NW, int U, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemm_bf16(GemmArgs a) {
  constexpr int NBR = red_nb<MT, NBW, NW>();
  static_assert(EPI != EPI_RESID || NBR == NBW, "EPI_RESID reduces in one round");
  __shared__ f32x4 red[NW * NBR * MT * 64];
  __shared__ float rs[kMaxRows];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const Work wk = work_of<NBW, NW>(a);
  const int nb0 = wk.nb0, nbv = wk.nbv, kb_beg = wk.kb_beg, kb_end = wk.kb_end;
  const u32x4* __restrict__ W = (const u32x4*)a.W;
  const u32x4* __restrict__ Xh = (const u32x4*)a.Xhi;
  const u32x4* __restrict__ Xl = (const u32x4*)a.Xlo;

  f32x4 acc[NBW][MT];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 cur[U][NBW];
  auto load_w = [&](u32x4 (&dst)[U][NBW], int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        if (kb + u < kb_end && j < nbv)
          dst[u][j] = __builtin_nontemporal_load(&W[((size_t)(nb0 + j) * a.Kb + kb + u) * 64 + lane]);
        else
          dst[u][j] = u32x4{0u, 0u, 0u, 0u};
      }
  };
  if (kb_beg < kb_end) load_w(cur, kb_beg);
  ResidIn pre{};
  if constexpr (EPI == EPI_RESID) pre = resid_prefetch<MT, NBW, NW>(a, nb0);
  FoldIn fpre{};
  if constexpr (EPI == EPI_PARTRES) fpre = fold_prefetch<MT, NBW, NW>(a, nb0, nbv);
  if (a.ssq) row_scales<NW>(a, rs);   // overlaps the first weight loads
  for (int kb = kb_beg; kb < kb_end; kb += U) {
    u32x4 nxt[U][NBW];
    if (kb + U < kb_end) load_w(nxt, kb + U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kb + u < kb_end) {
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const size_t xi = ((size_t)t * a.Kb + kb + u) * 64 + lane;
          const bf16x8 xh = as_bf16x8(Xh[xi]);
          const bf16x8 xl = as_bf16x8(Xl[xi]);
#pragma unroll
          for (int j = 0; j < NBW; ++j) {
            const bf16x8 wv = as_bf16x8(cur[u][j]);
            acc[j][t] = mfma_bf16(wv, xh, acc[j][t]);
            acc[j][t] = mfma_bf16(wv, xl, acc[j][t]);
          }
        }
      }
    }
    if (kb + U < kb_end) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < NBW; ++j) cur[u][j] = nxt[u][j];
    }
  }

#pragma unroll
  for (int j0 = 0; j0 < NBW; j0 += NBR) {
    if (j0 > 0) __syncthreads();   // the previous round's tiles have been read
#pragma unroll
    for (int jj = 0; jj < NBR; ++jj)
#pragma unroll
      for (int t = 0; t < MT; ++t)
        if (j0 + jj < NBW) red[((w * NBR + jj) * MT + t) * 64 + lane] = acc[j0 + jj][t];
    __syncthreads();
    finish<W_BF16, EPI, MT, NBR, NW>(a, red, a.ssq ? rs : nullptr, nb0 + j0, min(NBR, NBW - j0),
                                     wk.split, pre);
  }
  if constexpr (EPI == EPI_PARTRES) part_fold<W_BF16, NW>(a, nb0, nbv, fpre);
}

template <int MT, int NBW, int NW, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemm_f32(GemmArgs a) {
  constexpr int ACC = NBW * MT;
  __shared__ f32x4 red[NW * ACC * 64];
  __shared__ float rs[kMaxRows];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const Work wk = work_of<NBW, NW>(a);
  const int nb0 = wk.nb0, nbv = wk.nbv, kb_beg = wk.kb_beg, kb_end = wk.kb_end;
  const float4* __restrict__ W = (const float4*)a.W;
  const float4* __restrict__ X = (const float4*)a.Xhi;
  ResidIn pre{};
  if constexpr (EPI == EPI_RESID) pre = resid_prefetch<MT, NBW, NW>(a, nb0);
  FoldIn fpre{};
  if constexpr (EPI == EPI_PARTRES) fpre = fold_prefetch<MT, NBW, NW>(a, nb0, nbv);
  if (a.ssq) row_scales<NW>(a, rs);

  f32x4 acc[NBW][MT];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb = kb_beg; kb < kb_end; ++kb) {
    F8 wf[NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      if (j < nbv) {
        const size_t wi = (((size_t)(nb0 + j) * a.Kb + kb) * 64 + lane) * 2;
        wf[j].a = W[wi];
        wf[j].b = W[wi + 1];
      } else {
        wf[j].a = wf[j].b = float4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const size_t xi = (((size_t)t * a.Kb + kb) * 64 + lane) * 2;
      F8 xf;
      xf.a = X[xi];
      xf.b = X[xi + 1];
#pragma unroll
      for (int e8 = 0; e8 < 8; ++e8)
#pragma unroll
        for (int j = 0; j < NBW; ++j) acc[j][t] = mfma_f32(f8_get(wf[j], e8), f8_get(xf, e8), acc[j][t]);
    }
  }

#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) red[((w * NBW + j) * MT + t) * 64 + lane] = acc[j][t];
  __syncthreads();
  finish<W_F32, EPI, MT, NBW, NW>(a, red, a.ssq ? rs : nullptr, nb0, NBW, wk.split, pre);
  if constexpr (EPI == EPI_PARTRES) part_fold<W_F32, NW>(a, nb0, nbv, fpre);
}

// Grid shaping.  Each wave reuses every activation fragment it loads across
// the NBW n-blocks of its workgroup (activation reads from L2, not the
// weight stream, are what limit a one-n-block-per-wave GEMM); waves split K
// inside the workgroup and reduce through LDS.  Narrow EPI_PART GEMMs (O and
// down projections) also split K across S workgroups, each writing its own
// partial buffer, so the grid still covers every CU without any
// cross-workgroup synchronisation.
template <int MT, int EPI, int NBW, int NW, int U>
hipError_t launch_bf16_cfg(GemmArgs a, hipStream_t s) {
  const int grid = ((a.Nb + NBW - 1) / NBW) * a.S;
  hipLaunchKernelGGL((k_gemm_bf16<MT, NBW, NW, U, EPI>), dim3(grid), dim3(NW * 64), 0, s, a);
  return hipGetLastError();
}

// Launch configurations per GEMM role (n-blocks per workgroup x waves x
// k-blocks per batch), from a sweep over the 8B shapes.  The K partition --
// the wave count and the K-split count -- depends only on the role and the
// GEMM shape, never on the number of row tiles, so every output element is
// summed in the same order whether a window is verified alone or in a batch
// (bit-identical results).  Only the n-blocks per workgroup and the k-blocks
// per load batch (neither changes any summation order) change with the
// row-tile count and with the output width: the gate/up
// projection takes 7 n-blocks per workgroup when that makes exactly one
// workgroup per CU (e.g. 1792 n-blocks on 256 CUs); the LM head takes 12
// (wide output, one k-block per batch).  Measured with 32 layers' weights
// rotated so that no launch finds its weights in a cache.
template <int EPI>
struct Role;
template <>
struct Role<EPI_QKV> {
  static constexpr int NW = 16, U = 4;
};
template <>
struct Role<EPI_PART> {
  static constexpr int NW = 16, U = 2;
};
template <>
struct Role<EPI_PARTRES> : Role<EPI_PART> {};
template <>
struct Role<EPI_SILU> {
  static constexpr int NW = 12, U = 1;
};
template <>
struct Role<EPI_STORE> {
  static constexpr int NW = 8, U = 1;
};
template <>
struct Role<EPI_RESID> {
  static constexpr int NW = 16, U = 4;
};

inline int part_nbw(int mt) { return mt >= 2 ? 2 : 4; }

// CU rounds x n-blocks per workgroup: the time a CU spends streaming
inline long cost_of(int Nb, int nbw) {
  const long wgs = (Nb + nbw - 1) / nbw;
  return ((wgs + 255) / 256) * nbw;
}

template <int MT, int EPI>
hipError_t launch_bf16(const GemmArgs& a, hipStream_t s) {
  constexpr int NW = Role<EPI>::NW, U = Role<EPI>::U;
  if constexpr (MT >= 2) {
    // several row tiles (measured on whole steps of a 42-row batch of 7
    // windows): one n-block per workgroup for the O projection (256
    // workgroups), 4 for gate/up with two k-blocks per batch and for the
    // down projection, 2 for QKV, 8 for the LM head
    if constexpr (EPI == EPI_SILU) return launch_bf16_cfg<MT, EPI, 4, NW, 2>(a, s);
    else if constexpr (EPI == EPI_STORE) return launch_bf16_cfg<MT, EPI, 8, NW, 1>(a, s);
    else if constexpr (EPI == EPI_RESID) return launch_bf16_cfg<MT, EPI, 1, NW, U>(a, s);
    else if constexpr (EPI == EPI_PART || EPI == EPI_PARTRES) return launch_bf16_cfg<MT, EPI, 4, NW, 1>(a, s);
    else return launch_bf16_cfg<MT, EPI, 2, NW, (U < 2 ? U : 2)>(a, s);
  } else if constexpr (EPI == EPI_QKV) {
    // one n-block per workgroup (e.g. 384 workgroups at the 8B shape): slower
    // alone than two, faster inside the step (measured over whole steps)
    return launch_bf16_cfg<MT, EPI, 1, NW, U>(a, s);
  } else if constexpr (EPI == EPI_PART || EPI == EPI_PARTRES) {
    return launch_bf16_cfg<MT, EPI, 4, NW, 1>(a, s);
  } else if constexpr (EPI == EPI_RESID) {
    return launch_bf16_cfg<MT, EPI, 1, NW, U>(a, s);
  } else if constexpr (EPI == EPI_SILU) {
    if (cost_of(a.Nb, 7) < cost_of(a.Nb, 4)) return launch_bf16_cfg<MT, EPI, 7, NW, U>(a, s);
    return launch_bf16_cfg<MT, EPI, 4, NW, U>(a, s);
  } else {
    return launch_bf16_cfg<MT, EPI, 12, NW, U>(a, s);
  }
}

template <int MT, int EPI>
hipError_t launch_f32(const GemmArgs& a, hipStream_t s) {
  constexpr int NBW = 1, NW = 4;
  const int grid = ((a.Nb + NBW - 1) / NBW) * a.S;
  hipLaunchKernelGGL((k_gemm_f32<MT, NBW, NW, EPI>), dim3(grid), dim3(NW * 64), 0, s, a);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(int wtype, int mt, const GemmArgs& a, hipStream_t s) {
  if (wtype == W_BF16) {
    switch (mt) {
      case 1: return launch_bf16<1, EPI>(a, s);
      case 2: return launch_bf16<2, EPI>(a, s);
      case 3: return launch_bf16<3, EPI>(a, s);
      case 4: return launch_bf16<4, EPI>(a, s);
    }
  } else {
    switch (mt) {
      case 1: return launch_f32<1, EPI>(a, s);
      case 2: return launch_f32<2, EPI>(a, s);
      case 3: return launch_f32<3, EPI>(a, s);
      case 4: return launch_f32<4, EPI>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace

int gemm_part_splits(int wtype, int Nb, int Kb, int mt) {
  (void)mt;   // the split must not depend on the row count (batch invariance)
  if (wtype != W_BF16) return 1;
  const int groups = (Nb + 3) / 4;
  int S = std::max(1, std::min(kMaxSplits, 256 / std::max(1, groups)));
  while (S > 1 && Kb / S < Role<EPI_PART>::NW) --S;   // keep >= 1 k-block per wave
  return S;
}

hipError_t launch_gemm(int wtype, int mt, const GemmArgs& a, hipStream_t s) {
  if (a.Nb <= 0 || a.M <= 0) return hipSuccess;
  if (a.S < 1 || (a.S > 1 && a.epi.kind != EPI_PART && a.epi.kind != EPI_PARTRES)) return hipErrorInvalidValue;
  switch (a.epi.kind) {
    case EPI_STORE: return launch_epi<EPI_STORE>(wtype, mt, a, s);
    case EPI_PART: return launch_epi<EPI_PART>(wtype, mt, a, s);
    case EPI_QKV: return launch_epi<EPI_QKV>(wtype, mt, a, s);
    case EPI_SILU: return launch_epi<EPI_SILU>(wtype, mt, a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(wtype, mt, a, s);
    case EPI_PARTRES: return launch_epi<EPI_PARTRES>(wtype, mt, a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dsi
