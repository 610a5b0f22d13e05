// Window GEMM: Y[M, N] = X[M, K] . W[N, K]^T for the k+1 (or a few dozen)
// rows of a verification window, with fused epilogues.
//
// The k+1 window rows are one batch through the target (Section 2): every
// weight byte is read once per verification while each weight feeds only M
// (6..64) rows, so the kernel is bound by streaming W from HBM.  Design:
//  * W is pre-packed into 1 KB MFMA tiles (16 rows x 32 k, bf16), one
//    dwordx4 per lane, so every wavefront load is 1 KB contiguous and lands
//    in registers already in A-operand order (no LDS round trip for W); the
//    wide projections group their tiles so that a workgroup's loads at each
//    step are adjacent (wtile_index);
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

// Per-role K partition: waves per workgroup (NW), k-blocks per load batch
// (U), and whether a wave's k-blocks are dealt round-robin (RR: wave w takes
// k-blocks w, w + NW, ..., so the workgroup's waves read adjacent tiles of
// the grouped layout at every step) or as one contiguous range.  NW and RR
// fix the summation order and never change with the row-tile count.
template <int EPI>
struct Role;
template <>
struct Role<EPI_QKV> {
  static constexpr int NW = 16, U = 4;
  static constexpr bool RR = false;
};
template <>
struct Role<EPI_PART> {
  static constexpr int NW = 16, U = 2;
  static constexpr bool RR = false;
};
template <>
struct Role<EPI_PARTRES> : Role<EPI_PART> {};
template <>
struct Role<EPI_SILU> {
  static constexpr int NW = 12, U = 1;
  static constexpr bool RR = true;
};
template <>
struct Role<EPI_STORE> {
  static constexpr int NW = 8, U = 1;
  static constexpr bool RR = true;
};
template <>
struct Role<EPI_RESID> {
  static constexpr int NW = 16, U = 4;
  static constexpr bool RR = false;
};

// Inputs of the one epilogue item a thread owns, loaded before the main loop
// so that their latency is hidden: EPI_RESID the residual and gain values,
// EPI_QKV the rotary (cos, sin) pairs of the item's two feature pairs and the
// cache slot of its row.
struct EpiIn {
  float4 x, g;
  float4 rope;
  int pos;
};
template <int MT, int NBW, int NW, int EPI>
__device__ __forceinline__ EpiIn epi_prefetch(const GemmArgs& a, int nb0) {
  EpiIn r{};
  if constexpr (EPI == EPI_RESID || EPI == EPI_QKV) {
    static_assert(NBW * MT <= NW, "finish() must give each thread at most one item");
    const int it = threadIdx.x;
    if (it < NBW * MT * 64) {
      const int l = it & 63, jm = it >> 6;
      const int nb = nb0 + jm / MT, m = (jm % MT) * 16 + (l & 15);
      if (nb < a.Nb && m < a.M) {
        const EpiArgs& e = a.epi;
        if constexpr (EPI == EPI_RESID) {
          const int n0 = nb * 16 + (l >> 4) * 4;
          r.x = *(const float4*)(e.x + (size_t)m * e.ld + n0);
          r.g = *(const float4*)(e.gain + n0);
        } else {
          const int bph = e.hd >> 4, nq = e.n_heads * bph, nk = e.n_kv * bph;
          const int R = e.rows.rows_per_window;
          r.pos = e.rows.lens[e.rows.window0 + m / R];   // + m % R in the epilogue
          if (nb < nq + nk) {
            const int sb = nb < nq ? nb : nb - nq;
            const int ja = (sb % bph) * 8 + (l >> 4) * 2;
            const float2 ca = e.rope[(size_t)m * (e.hd >> 1) + ja];
            const float2 cb = e.rope[(size_t)m * (e.hd >> 1) + ja + 1];
            r.rope = float4{ca.x, ca.y, cb.x, cb.y};
          }
        }
      }
    }
  }
  return r;
}

// Returns the sum of the squared residual values it wrote (EPI_RESID), else 0.
template <int WT, int EPI>
__device__ __forceinline__ float epilogue(const EpiArgs& e, int nb, int r0, int m, int split, f32x4 s,
                                          const EpiIn& pre) {
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
      const int pos = pre.pos + (m % R);
      if (nb < nq + nk) {
        const int sb = nb < nq ? nb : nb - nq;
        const int h = sb / bph;
        const int ja = (sb % bph) * 8 + (r0 >> 2) * 2;   // pair indices ja, ja+1
        const int half = hd >> 1;
        const float2 ca{pre.rope.x, pre.rope.y};   // rope[m][ja], rope[m][ja + 1]
        const float2 cb{pre.rope.z, pre.rope.w};
        const float a1 = s[0] * ca.x - s[2] * ca.y, a2 = s[2] * ca.x + s[0] * ca.y;
        const float b1 = s[1] * cb.x - s[3] * cb.y, b2 = s[3] * cb.x + s[1] * cb.y;
        if (nb < nq) {
          float* qr = e.q_out + (size_t)m * (e.n_heads * hd) + h * hd;
          qr[ja] = a1;
          qr[ja + half] = a2;
          qr[ja + 1] = b1;
          qr[ja + 1 + half] = b2;
        } else {
          const size_t base = ((size_t)win * e.n_kv + h) * e.maxlen * hd;
          const size_t i0 = base + kc_off(pos, ja, hd), i1 = base + kc_off(pos, ja + half, hd);
          const size_t i2 = base + kc_off(pos, ja + 1, hd), i3 = base + kc_off(pos, ja + 1 + half, hd);
          if (e.kv_bf16) {
            uint16_t* kc = (uint16_t*)e.kcache;
            kc[i0] = f2bf_bits(a1);
            kc[i1] = f2bf_bits(a2);
            kc[i2] = f2bf_bits(b1);
            kc[i3] = f2bf_bits(b2);
          } else {
            float* kc = (float*)e.kcache;
            kc[i0] = a1;
            kc[i1] = a2;
            kc[i2] = b1;
            kc[i3] = b2;
          }
        }
      } else {
        const int vb = nb - nq - nk;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = vb * 16 + r0 + j;
          const int h = n / hd, dd = n % hd;
          const size_t idx = ((size_t)win * e.n_kv + h) * e.maxlen * hd + vc_off(pos, dd, hd);
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
// depend on the number of rows.  The entries of the wave's first row are
// loaded before the weights (ssq_prefetch): loads retire in order, so
// waiting for them then does not wait for any weight batch.
constexpr int kSsqPer = 8;   // prefetched entries per lane: ssq_n <= 512
struct SsqIn {
  float v[kSsqPer];
  bool ok;   // v holds row w's entries
};
template <int EPI>
__device__ __forceinline__ SsqIn ssq_prefetch(const GemmArgs& a) {
  SsqIn r;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int c = 0; c < kSsqPer; ++c) r.v[c] = 0.f;
  r.ok = false;
  // only the normed-input roles (QKV, gate/up) take row scales
  if constexpr (EPI == EPI_QKV || EPI == EPI_SILU) {
    if (a.ssq && w < a.M && a.ssq_n <= 64 * kSsqPer) {
      const float* p = a.ssq + (size_t)w * a.ssq_n;
#pragma unroll
      for (int c = 0; c < kSsqPer; ++c)
        if (lane + 64 * c < a.ssq_n) r.v[c] = p[lane + 64 * c];
      r.ok = true;
    }
  }
  return r;
}

template <int NW>
__device__ __forceinline__ void row_scales(const GemmArgs& a, const SsqIn& pre, float* rs) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int m = w; m < a.M; m += NW) {
    float sum = 0.f;
    if (m == w && pre.ok) {
#pragma unroll
      for (int c = 0; c < kSsqPer; ++c)
        if (lane + 64 * c < a.ssq_n) sum += pre.v[c];
    } else {
      const float* p = a.ssq + (size_t)m * a.ssq_n;
#pragma unroll 4
      for (int i = lane; i < a.ssq_n; i += 64) sum += p[i];
    }
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
// Items are 4 consecutive features of one row (rows x n-blocks x 4 of
// them), taken by the threads in rounds of the workgroup size; the four
// lanes of one (row, n-block) are adjacent, so the n-block's sum of squares
// is a two-step butterfly.  The residual and gain values of each thread's
// first item are loaded at the start of the kernel (fold_prefetch), off the
// critical path.
struct FoldIn {
  float4 x, g;
};
__device__ __forceinline__ FoldIn fold_prefetch(const GemmArgs& a, int nb0, int nbv) {
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
  const int total = a.M * nbv * 4;
  for (int base = 0; base < total; base += NW * 64) {   // uniform trip count
    const int it = base + threadIdx.x;
    const bool ok = it < total;
    const int q = it & 3, jm = it >> 2;
    const int m = ok ? jm / nbv : 0, nb = nb0 + (ok ? jm % nbv : 0);
    const int n0 = nb * 16 + q * 4;
    float sq = 0.f;
    if (ok) {
      // every split's values are requested before the first add (split
      // index clamped; the extra loads are never added), then added in
      // split order
      float pv[kMaxSplits][4];
#pragma unroll
      for (int sp = 0; sp < kMaxSplits; ++sp) {
        const float* pp = e.out + min(sp, a.S - 1) * e.part_stride + (size_t)m * e.ld + n0;
#pragma unroll
        for (int c = 0; c < 4; ++c) pv[sp][c] = __hip_atomic_load(pp + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      float4 xv = pre.x, gv = pre.g;
      if (base > 0) {
        xv = *(const float4*)(e.x + (size_t)m * e.ld + n0);
        gv = *(const float4*)(e.gain + n0);
      }
#pragma unroll
      for (int sp = 0; sp < kMaxSplits; ++sp) {
        if (sp < a.S) {
          xv.x += pv[sp][0];
          xv.y += pv[sp][1];
          xv.z += pv[sp][2];
          xv.w += pv[sp][3];
        }
      }
      *(float4*)(e.x + (size_t)m * e.ld + n0) = xv;
      if (e.copy) *(float4*)(e.copy + (size_t)m * e.ld + n0) = xv;
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
                                       int nvalid, int split, const EpiIn& pre) {
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

// workgroup -> (n-block group, K split); wave -> its k-blocks of the split:
// nk of them, kb_beg + i * kstep for i < nk
struct Work {
  int nb0, nbv, split, kb_beg, nk, kstep;
};
template <int NBW, int NW, bool RR>
__device__ __forceinline__ Work work_of(const GemmArgs& a) {
  Work w;
  const int g = blockIdx.x / a.S;
  w.split = blockIdx.x % a.S;
  w.nb0 = g * NBW;
  w.nbv = min(NBW, a.Nb - w.nb0);
  const int k0 = (w.split * a.Kb) / a.S;
  const int k1 = ((w.split + 1) * a.Kb) / a.S;
  // uniform across the wave: the k-block loop runs on scalar branches
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (RR) {
    w.kb_beg = k0 + wave;
    w.nk = w.kb_beg < k1 ? (k1 - w.kb_beg + NW - 1) / NW : 0;
    w.kstep = NW;
  } else {
    const int per = (k1 - k0 + NW - 1) / NW;
    w.kb_beg = min(k1, k0 + wave * per);
    w.nk = min(k1, w.kb_beg + per) - w.kb_beg;
    w.kstep = 1;
  }
  return w;
}

// n-blocks per LDS reduction round: all of them when NW x NBW x MT tiles
// (1 KB each) fit in kRedTiles KB, else as many as fit (several rounds)
constexpr int kRedTiles = 128;
template <int MT, int NBW, int NW>
constexpr int red_nb() {
  return NW * NBW * MT <= kRedTiles ? NBW : (kRedTiles / (NW * MT) > 0 ? kRedTiles / (NW * MT) : 1);
}

// Main loop of a launch: the two-set weight pipeline (one row tile, and up
// to three row tiles for the QKV, O and gate/up roles, whose shapes leave
// registers for a second weight set), else the loop that requests the first
// two weight batches before any MFMA (the down projection and the LM head
// with several row tiles: their accumulators leave no room; measured on a
// 42-row batch, pipelining them was slower).
template <int MT, int EPI>
constexpr bool kPipelined =
    MT == 1 || (MT <= 3 && (EPI == EPI_QKV || EPI == EPI_RESID || EPI == EPI_SILU));

template <int MT, int NBW, int NW, int U, int EPI>
__global__ __launch_bounds__(NW * 64) void k_gemm_bf16(GemmArgs a) {
  constexpr int NBR = red_nb<MT, NBW, NW>();
  static_assert((EPI != EPI_RESID && EPI != EPI_QKV) || NBR == NBW, "prefetched epilogues reduce in one round");
  __shared__ f32x4 red[NW * NBR * MT * 64];
  __shared__ float rs[kMaxRows];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  constexpr int KS = Role<EPI>::RR ? NW : 1;
  const Work wk = work_of<NBW, NW, Role<EPI>::RR>(a);
  const int nb0 = wk.nb0, nbv = wk.nbv, kb_beg = wk.kb_beg, nk = wk.nk;
  const u32x4* __restrict__ W = (const u32x4*)a.W;
  const u32x4* __restrict__ Xh = (const u32x4*)a.Xhi;
  const u32x4* __restrict__ Xl = (const u32x4*)a.Xlo;

  f32x4 acc[NBW][MT];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // tile (nb0 + j, kb) of the grouped layout is tb[j] + kb * ts[j]
  size_t tb[NBW];
  int ts[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    const int nb = min(nb0 + j, a.Nb - 1), gi = nb / a.G;
    tb[j] = (size_t)gi * a.G * a.Kb + (nb - gi * a.G);
    ts[j] = min(a.G, a.Nb - gi * a.G);
  }
  // Every load inside the pipeline is issued unconditionally (indices are
  // clamped into the matrix; tiles past the wave's k-blocks are never fed to
  // an MFMA and n-blocks past the matrix only reach accumulators that are
  // never stored), so the compiler knows how many loads are younger than the
  // one it waits for: loads retire in order, and a wait behind a conditional
  // load would also wait for every weight load issued after it.
  auto load_w = [&](u32x4 (&dst)[U][NBW], int i) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int kb = kb_beg + min(i + u, nk - 1) * KS;
        dst[u][j] = __builtin_nontemporal_load(&W[(tb[j] + (size_t)kb * ts[j]) * 64 + lane]);
      }
  };
  // activation fragments of batch i, loaded as one group
  auto load_x = [&](bf16x8 (&xh)[U][MT], bf16x8 (&xl)[U][MT], int i) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int kb = kb_beg + min(i + u, nk - 1) * KS;
        const size_t xi = ((size_t)t * a.Kb + kb) * 64 + lane;
        xh[u][t] = as_bf16x8(Xh[xi]);
        xl[u][t] = as_bf16x8(Xl[xi]);
      }
  };
  auto mma = [&](const u32x4 (&w)[U][NBW], const bf16x8 (&xh)[U][MT], const bf16x8 (&xl)[U][MT], int nu) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nu) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int j = 0; j < NBW; ++j) {
            const bf16x8 wv = as_bf16x8(w[u][j]);
            acc[j][t] = mfma_bf16(wv, xh[u][t], acc[j][t]);
            acc[j][t] = mfma_bf16(wv, xl[u][t], acc[j][t]);
          }
      }
    }
  };
  // epilogue inputs and the RMSNorm sums go first: waiting for them then
  // waits for no weight load
  const SsqIn spre = ssq_prefetch<EPI>(a);
  const EpiIn pre = epi_prefetch<MT, NBW, NW, EPI>(a, nb0);
  FoldIn fpre{};
  if constexpr (EPI == EPI_PARTRES) fpre = fold_prefetch(a, nb0, nbv);
  if constexpr (kPipelined<MT, EPI>) {
    if (nk > 0) {
      // two weight register sets used in turn (a copy from one to the other
      // would make the compiler wait for a batch before issuing the next)
      u32x4 wa[U][NBW], wz[U][NBW];
      load_w(wa, 0);
      if (a.ssq) row_scales<NW>(a, spre, rs);   // overlaps the first weight loads
      // a batch with a successor: its activations, then the next batch's
      // weights, then its MFMAs, so the MFMAs wait for the activations and
      // never for the next weights
      auto full = [&](const u32x4 (&wc)[U][NBW], u32x4 (&wn)[U][NBW], int i) {
        bf16x8 xh[U][MT], xl[U][MT];
        load_x(xh, xl, i);
        __builtin_amdgcn_sched_barrier(0);
        load_w(wn, i + U);
        __builtin_amdgcn_sched_barrier(0);
        mma(wc, xh, xl, U);
      };
      auto last = [&](const u32x4 (&wc)[U][NBW], int i) {
        bf16x8 xh[U][MT], xl[U][MT];
        load_x(xh, xl, i);
        mma(wc, xh, xl, nk - i);
      };
      const int nfull = (nk - 1) / U;   // batches followed by another
      int i = 0;
      for (int p = 0; p < nfull / 2; ++p, i += 2 * U) {   // branch-free body
        full(wa, wz, i);
        full(wz, wa, i + U);
      }
      if (nfull & 1) {
        full(wa, wz, i);
        last(wz, i + U);
      } else {
        last(wa, i);
      }
    } else if (a.ssq) {
      row_scales<NW>(a, spre, rs);
    }
  } else {
    // The first two weight batches are requested before the first MFMA and
    // the activations are loaded next to their MFMAs (each of those waits
    // also waits for the weights issued before it).
    u32x4 cur[U][NBW];
    auto load_w_guarded = [&](u32x4 (&dst)[U][NBW], int i) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
          const int kb = kb_beg + (i + u) * KS;
          if (i + u < nk && j < nbv)
            dst[u][j] = __builtin_nontemporal_load(&W[(tb[j] + (size_t)kb * ts[j]) * 64 + lane]);
          else
            dst[u][j] = u32x4{0u, 0u, 0u, 0u};
        }
    };
    if (nk > 0) load_w_guarded(cur, 0);
    if (a.ssq) row_scales<NW>(a, spre, rs);
    for (int i = 0; i < nk; i += U) {
      u32x4 nxt[U][NBW];
      if (i + U < nk) load_w_guarded(nxt, i + U);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (i + u < nk) {
          const int kb = kb_beg + (i + u) * KS;
#pragma unroll
          for (int t = 0; t < MT; ++t) {
            const size_t xi = ((size_t)t * a.Kb + kb) * 64 + lane;
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
      if (i + U < nk) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int j = 0; j < NBW; ++j) cur[u][j] = nxt[u][j];
      }
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
  const Work wk = work_of<NBW, NW, false>(a);
  const int nb0 = wk.nb0, nbv = wk.nbv, kb_beg = wk.kb_beg, kb_end = wk.kb_beg + wk.nk;
  const float4* __restrict__ W = (const float4*)a.W;
  const float4* __restrict__ X = (const float4*)a.Xhi;
  const EpiIn pre = epi_prefetch<MT, NBW, NW, EPI>(a, nb0);
  FoldIn fpre{};
  if constexpr (EPI == EPI_PARTRES) fpre = fold_prefetch(a, nb0, nbv);
  if (a.ssq) row_scales<NW>(a, ssq_prefetch<EPI>(a), rs);

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

// ------------------------------------------------------------------ ring GEMM
//
// One-row-tile launches (M <= 16) over weights in the ring layout (RingCfg):
// each of the 8 waves of a workgroup streams its own contiguous run of
// nk * nbw tiles through a register ring of kRingDepth tiles.  The whole run
// is unrolled at compile time, so the position of every load in the wave's
// load order is static: consuming tile u waits for exactly the loads issued
// before it while the next kRingDepth - 1 tiles stay in flight, and the ring
// never drains until the wave's last tiles.  The activation fragments of a
// k-block (hi and lo halves, token rows past M skipped by out-of-range buffer
// loads) are requested just before its first weight tile, so they arrive
// with it and their bytes are spread over the stream; the epilogue inputs
// and RMSNorm sums are requested before everything else.  Partial tiles are
// reduced across the waves through LDS in wave order and handed to the same
// epilogues as the packed kernel.
constexpr int kRingDepth = 8;

// Weight tiles in flight per wave for MT row tiles: 8, or 4 where the
// registers would not hold 8 -- the narrow roles (one or two n-blocks per
// workgroup) with several row tiles, whose activation slots (hi and lo of MT
// tiles per k-block in flight) grow with MT, and gate/up's 7 x 4 accumulator
// tiles at four row tiles.  The depth does not change any sum.
constexpr int ring_depth(int nbw, int mt) { return ((mt > 1 && nbw <= 2) || (mt >= 4 && nbw >= 7)) ? 4 : kRingDepth; }
// n-blocks per LDS reduction round: kRingWaves x NBR x MT tiles of 1 KB
// within 128 KB
constexpr int ring_red_nb(int nbw, int mt) { return 16 / mt < nbw ? 16 / mt : nbw; }

// RMSNorm sums of rows w and w + kRingWaves (the first 16 rows), requested
// before the weights and reduced after the main loop; rows beyond 16 (wave
// w: rows w + 8h) are loaded after it, all at once (42-row batch: step 4.65
// -> 4.62 ms against one conditional load after another)
struct RingSsq {
  float v[2][kSsqPer];
};
template <int EPI>
__device__ __forceinline__ RingSsq ring_ssq_prefetch(const GemmArgs& a) {
  RingSsq r;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int c = 0; c < kSsqPer; ++c) r.v[h][c] = 0.f;
  if constexpr (EPI == EPI_QKV || EPI == EPI_SILU) {
    if (a.ssq) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int m = w + h * kRingWaves;
        if (m < a.M) {
          const float* p = a.ssq + (size_t)m * a.ssq_n;
#pragma unroll
          for (int c = 0; c < kSsqPer; ++c)
            if (lane + 64 * c < a.ssq_n) r.v[h][c] = p[lane + 64 * c];
        }
      }
    }
  }
  return r;
}

// rs[m] = 1/sqrt(sum / d + eps) for the MT*16 rows; row m is reduced by wave
// m % 8 in the same order for every MT (lane entries, then a butterfly)
template <int MT>
__device__ __forceinline__ void ring_row_scales(const GemmArgs& a, const RingSsq& pre, float* rs) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // rows past the first 16: every load issued at once (indices clamped into
  // the buffer, invalid entries zeroed after), one wait for all of them
  constexpr int HL = 2 * MT - 2 > 0 ? 2 * MT - 2 : 1;
  float late[HL][kSsqPer];
#pragma unroll
  for (int h = 2; h < 2 * MT; ++h) {
    const int m = min(w + h * kRingWaves, a.M - 1);
#pragma unroll
    for (int c = 0; c < kSsqPer; ++c) late[h - 2][c] = a.ssq[(size_t)m * a.ssq_n + min(lane + 64 * c, a.ssq_n - 1)];
  }
#pragma unroll
  for (int h = 0; h < 2 * MT; ++h) {
    const int m = w + h * kRingWaves;
    float v[kSsqPer];
#pragma unroll
    for (int c = 0; c < kSsqPer; ++c) {
      if (h < 2) {
        v[c] = pre.v[h < 2 ? h : 0][c];
      } else {
        v[c] = (m < a.M && lane + 64 * c < a.ssq_n) ? late[h < 2 ? 0 : h - 2][c] : 0.f;
      }
    }
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < kSsqPer; ++c) sum += v[c];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
    if (lane == 0 && m < a.M) rs[m] = 1.0f / sqrtf(sum / (float)a.norm_d + a.eps);
  }
}

// MT row tiles (1..4) of the activation pack; every row's sums are formed
// in the same order for every MT -- each wave's k-blocks in order, hi then
// lo, the waves reduced in order -- so a row's results do not depend on
// how many rows share the launch.
template <int NK, int NBW, int EPI, int MT>
__global__ __launch_bounds__(kRingWaves * 64) void k_gemm_ring(GemmArgs a) {
  constexpr int NW = kRingWaves, D = ring_depth(NBW, MT), N = NK * NBW;
  // activation slots: k-block i's fragments are requested together with its
  // first weight tile (D tiles ahead of use) and live until its last tile;
  // when one is requested, tile u has just been consumed and tiles
  // u+1 .. u+D-1 still need ceil((D-1)/NBW) k-blocks
  constexpr int A = (D - 1 + NBW - 1) / NBW + 1;
  constexpr int NBR = ring_red_nb(NBW, MT);
  static_assert(N >= D, "a wave's run must fill the ring");
  __shared__ f32x4 red[NW * NBR * MT * 64];
  __shared__ float rs[MT * 16];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = blockIdx.x / a.S, split = blockIdx.x - g * a.S;
  const int nb0 = g * NBW;
  const int nbv = min(NBW, a.Nb - nb0);
  const int kb0 = split * (NW * NK) + w * NK;
  const u32x4* __restrict__ Ws = (const u32x4*)a.Ws + ((size_t)(blockIdx.x * NW + w) * N) * 64 + lane;
  // activation packs as buffers: a lane whose token row is padding (>= M)
  // or whose k-block lies past the matrix reads out of range, which returns
  // zeros without a memory access
  const int nrec = MT * a.Kb * 1024;
  const __amdgpu_buffer_rsrc_t Rh = __builtin_amdgcn_make_buffer_rsrc((void*)a.Xhi, (short)0, nrec, 0x00020000);
  const __amdgpu_buffer_rsrc_t Rl = __builtin_amdgcn_make_buffer_rsrc((void*)a.Xlo, (short)0, nrec, 0x00020000);
  auto xoff = [&](int i, int t) -> int {
    return ((lane & 15) + 16 * t < a.M && kb0 + i < a.Kb) ? ((t * a.Kb + kb0 + i) * 64 + lane) * 16 : 0x7ffffff0;
  };

  const EpiIn pre = epi_prefetch<MT, NBW, NW, EPI>(a, nb0);
  FoldIn fpre{};
  if constexpr (EPI == EPI_PARTRES) fpre = fold_prefetch(a, nb0, nbv);
  const RingSsq spre = ring_ssq_prefetch<EPI>(a);
  __builtin_amdgcn_sched_barrier(0);
  u32x4 ring[D];
  u32x4 xh[A][MT], xl[A][MT];
  // issue position u: the fragments of k-block u / NBW when u starts one,
  // then weight tile u
  auto issue = [&](int u) {
    if (u % NBW == 0) {
      const int i = u / NBW;
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        xh[i % A][t] = __builtin_amdgcn_raw_buffer_load_b128(Rh, xoff(i, t), 0, 0);
        xl[i % A][t] = __builtin_amdgcn_raw_buffer_load_b128(Rl, xoff(i, t), 0, 0);
      }
    }
    ring[u % D] = __builtin_nontemporal_load(Ws + (size_t)u * 64);
  };
#pragma unroll
  for (int r = 0; r < D; ++r) {
    issue(r);
    __builtin_amdgcn_sched_barrier(0);   // issue order = ring order
  }
  f32x4 acc[NBW][MT];
#pragma unroll
  for (int j = 0; j < NBW; ++j)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[j][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const bf16x8 wv = as_bf16x8(ring[u % D]);
    const int i = u / NBW;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      acc[u % NBW][t] = mfma_bf16(wv, as_bf16x8(xh[i % A][t]), acc[u % NBW][t]);
      acc[u % NBW][t] = mfma_bf16(wv, as_bf16x8(xl[i % A][t]), acc[u % NBW][t]);
    }
    if (u + D < N) issue(u + D);
    __builtin_amdgcn_sched_barrier(0);   // consume tile u, then refill its slot
  }
  if (a.ssq) ring_row_scales<MT>(a, spre, rs);
#pragma unroll
  for (int j0 = 0; j0 < NBW; j0 += NBR) {
    if (j0 > 0) __syncthreads();   // the previous round's tiles have been read
#pragma unroll
    for (int jj = 0; jj < NBR; ++jj)
#pragma unroll
      for (int t = 0; t < MT; ++t)
        if (j0 + jj < NBW) red[((w * NBR + jj) * MT + t) * 64 + lane] = acc[j0 + jj][t];
    __syncthreads();
    finish<W_BF16, EPI, MT, NBR, NW>(a, red, a.ssq ? rs : nullptr, nb0 + j0, min(NBR, NBW - j0), split, pre);
  }
  if constexpr (EPI == EPI_PARTRES) part_fold<W_BF16, NW>(a, nb0, nbv, fpre);
}

// n-blocks per workgroup of each role's ring layout: the O projection one
// (256 workgroups at d = 4096), QKV two (192 at the 8B shape; one when one
// round of single-n-block workgroups covers every n-block, e.g. 192 at the
// 1B shape: 0.826 -> 0.811 ms per step, where two would leave 96
// workgroups; at the 8B shape one is far slower, 18.4 vs 13.7 us, as every
// CU then takes in twice the activation bytes), gate/up seven (one
// workgroup per CU for 1792 n-blocks), the down projection four with its K
// split (as the packed launch), the LM head eight
template <int EPI>
struct RingRole;
template <>
struct RingRole<EPI_QKV> {
  static constexpr int NBW = 2;
  static int nbw(int Nb) { return Nb <= 256 ? 1 : 2; }
};
template <>
struct RingRole<EPI_RESID> {
  static constexpr int NBW = 1;
  static int nbw(int) { return NBW; }
};
template <>
struct RingRole<EPI_SILU> {
  static constexpr int NBW = 7;
  static int nbw(int) { return NBW; }
};
template <>
struct RingRole<EPI_PART> {
  static constexpr int NBW = 4;
  static int nbw(int) { return NBW; }
};
template <>
struct RingRole<EPI_PARTRES> : RingRole<EPI_PART> {};
template <>
struct RingRole<EPI_STORE> {   // the LM head: many rounds of workgroups
  static constexpr int NBW = 8;
  static int nbw(int) { return NBW; }
};

// k-blocks per wave the ring kernel is built for (a shape's k-range per wave
// is rounded up to one of them; the extra tiles are zero)
constexpr int kRingNk[] = {1, 2, 4, 8, 14, 16};

template <int EPI, int NBW, int NK, int MT>
hipError_t launch_ring_nk(const GemmArgs& a, hipStream_t s) {
  if constexpr (NK * NBW < kRingDepth) {
    return hipErrorInvalidValue;
  } else {
    const int grid = ((a.Nb + NBW - 1) / NBW) * a.S;
    hipLaunchKernelGGL((k_gemm_ring<NK, NBW, EPI, MT>), dim3(grid), dim3(kRingWaves * 64), 0, s, a);
    return hipGetLastError();
  }
}

template <int EPI, int NBW, int MT>
hipError_t launch_ring_mt(const GemmArgs& a, hipStream_t s) {
  switch (a.ring_nk) {
    case 1: return launch_ring_nk<EPI, NBW, 1, MT>(a, s);
    case 2: return launch_ring_nk<EPI, NBW, 2, MT>(a, s);
    case 4: return launch_ring_nk<EPI, NBW, 4, MT>(a, s);
    case 8: return launch_ring_nk<EPI, NBW, 8, MT>(a, s);
    case 14: return launch_ring_nk<EPI, NBW, 14, MT>(a, s);
    case 16: return launch_ring_nk<EPI, NBW, 16, MT>(a, s);
  }
  return hipErrorInvalidValue;
}

template <int EPI, int NBW>
hipError_t launch_ring_nbw(const GemmArgs& a, int mt, hipStream_t s) {
  switch (mt) {
    case 1: return launch_ring_mt<EPI, NBW, 1>(a, s);
    case 2: return launch_ring_mt<EPI, NBW, 2>(a, s);
    case 3: return launch_ring_mt<EPI, NBW, 3>(a, s);
    case 4: return launch_ring_mt<EPI, NBW, 4>(a, s);
  }
  return hipErrorInvalidValue;
}

// the layout's n-blocks per workgroup (a.ring_nbw) picks the kernel
template <int EPI>
hipError_t launch_ring(const GemmArgs& a, int mt, hipStream_t s) {
  if constexpr (EPI == EPI_QKV) {
    if (a.ring_nbw == 1) return launch_ring_nbw<EPI, 1>(a, mt, s);
  }
  if (a.ring_nbw != RingRole<EPI>::NBW) return hipErrorInvalidValue;
  return launch_ring_nbw<EPI, RingRole<EPI>::NBW>(a, mt, s);
}

// ring layout from the packed layout: one thread per 16 bytes of a tile
__global__ void k_restream(const u32x4* __restrict__ src, int Nb, int Kb, int G, RingCfg c,
                           u32x4* __restrict__ dst) {
  const size_t total = c.tiles() * 64;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const size_t t = i >> 6;
    const int run = c.nk * c.nbw;                       // tiles per wave
    const size_t wave = t / run;                        // blockIdx * waves + w
    const int u = (int)(t - wave * run);
    const int wg = (int)(wave / kRingWaves), w = (int)(wave % kRingWaves);
    const int ii = u / c.nbw, j = u % c.nbw;
    const int nb = (wg / c.S) * c.nbw + j;
    const int kb = (wg % c.S) * (kRingWaves * c.nk) + w * c.nk + ii;
    u32x4 v{0u, 0u, 0u, 0u};
    if (nb < Nb && kb < Kb) v = src[wtile_index(nb, kb, Nb, Kb, G) * 64 + lane];
    dst[i] = v;
  }
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
// (wide output, one k-block per batch).  Both are packed in groups of that
// many n-blocks with their k-blocks dealt round-robin to the waves, so a
// workgroup streams one contiguous region (gate/up 37.8 -> 36.3 us and LM
// head 174 -> 162 us as pure weight streams).  Measured with 32 layers'
// weights rotated so that no launch finds its weights in a cache.

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
    // workgroups), 4 for gate/up and for the down projection, 2 for QKV, 8
    // for the LM head; the k-blocks per batch of the pipelined roles keep
    // both weight register sets and a batch of activations within the
    // register budget (three row tiles: gate/up and QKV one, O two)
    constexpr bool P = kPipelined<MT, EPI>;
    if constexpr (EPI == EPI_SILU) return launch_bf16_cfg<MT, EPI, 4, NW, (P ? 1 : 2)>(a, s);
    else if constexpr (EPI == EPI_STORE) return launch_bf16_cfg<MT, EPI, 8, NW, 1>(a, s);
    else if constexpr (EPI == EPI_RESID) return launch_bf16_cfg<MT, EPI, 1, NW, (P ? 2 : U)>(a, s);
    else if constexpr (EPI == EPI_PART || EPI == EPI_PARTRES) return launch_bf16_cfg<MT, EPI, 4, NW, 1>(a, s);
    else return launch_bf16_cfg<MT, EPI, 2, NW, (MT == 3 ? 1 : 2)>(a, s);
  } else if constexpr (EPI == EPI_QKV) {
    // two n-blocks per workgroup (192 workgroups at the 8B shape, one per CU
    // with room for both weight register sets): each activation fragment
    // feeds two weight tiles (measured over whole steps: 8B 3.449 -> 3.425
    // ms, 13B/32k 10.33 -> 10.25 ms against one n-block on the short-wave
    // loop); four (two k-blocks per batch for the registers) when two would
    // still need a second round of workgroups (13B/32k 10.08 -> 9.81 ms), one
    // when one round of single-n-block workgroups covers them all (1B
    // 0.886 -> 0.868 ms)
    if (a.Nb > 512) return launch_bf16_cfg<MT, EPI, 4, NW, 2>(a, s);
    if (a.Nb <= 256) return launch_bf16_cfg<MT, EPI, 1, NW, U>(a, s);
    return launch_bf16_cfg<MT, EPI, 2, NW, U>(a, s);
  } else if constexpr (EPI == EPI_PART || EPI == EPI_PARTRES) {
    return launch_bf16_cfg<MT, EPI, 4, NW, 1>(a, s);
  } else if constexpr (EPI == EPI_RESID) {
    // more n-blocks than CUs (e.g. 320 at the 13B shape): two per workgroup,
    // one round of workgroups instead of two (13B/32k 10.27 -> 10.03 ms)
    if (a.Nb > 256) return launch_bf16_cfg<MT, EPI, 2, NW, U>(a, s);
    return launch_bf16_cfg<MT, EPI, 1, NW, U>(a, s);
  } else if constexpr (EPI == EPI_SILU) {
    // the weights were packed in groups of the n-blocks per workgroup
    if (a.G == 7) return launch_bf16_cfg<MT, EPI, 7, NW, U>(a, s);
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

int gemm_wgroup(int wtype, int epi_kind, int Nb) {
  if (wtype != W_BF16) return 1;
  if (epi_kind == EPI_SILU) return cost_of(Nb, 7) < cost_of(Nb, 4) ? 7 : 4;
  if (epi_kind == EPI_STORE) return 12;
  return 1;
}

bool ring_config(int wtype, int epi_kind, int Nb, int Kb, int S, RingCfg* out) {
  *out = RingCfg{};
  if (wtype != W_BF16 || Nb < 1 || Kb < 1 || S < 1) return false;
  int nbw = 0;
  switch (epi_kind) {
    case EPI_QKV: nbw = RingRole<EPI_QKV>::nbw(Nb); break;
    case EPI_RESID: nbw = RingRole<EPI_RESID>::nbw(Nb); break;
    case EPI_SILU: nbw = RingRole<EPI_SILU>::nbw(Nb); break;
    case EPI_PART:
    case EPI_PARTRES: nbw = RingRole<EPI_PART>::nbw(Nb); break;
    case EPI_STORE: nbw = RingRole<EPI_STORE>::nbw(Nb); break;
    default: return false;
  }
  if (S > 1 && epi_kind != EPI_PART && epi_kind != EPI_PARTRES) return false;
  const int need = (Kb + S * kRingWaves - 1) / (S * kRingWaves);   // k-blocks per wave
  int nk = 0;
  for (int v : kRingNk)
    if (v >= need && v * nbw >= kRingDepth) {
      nk = v;
      break;
    }
  if (!nk) return false;
  out->nbw = nbw;
  out->nk = nk;
  out->S = S;
  out->wgs = ((Nb + nbw - 1) / nbw) * S;
  return true;
}

hipError_t launch_restream(const void* src, int Nb, int Kb, int G, const RingCfg& c, void* dst,
                           hipStream_t s) {
  if (c.nbw < 1 || c.nk < 1 || c.S < 1 || G < 1) return hipErrorInvalidValue;
  const size_t total = c.tiles() * 64;
  const int grid = (int)std::min<size_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_restream, dim3(grid), dim3(256), 0, s, (const u32x4*)src, Nb, Kb, G, c, (u32x4*)dst);
  return hipGetLastError();
}

hipError_t launch_gemm(int wtype, int mt, const GemmArgs& a, hipStream_t s) {
  if (a.Nb <= 0 || a.M <= 0) return hipSuccess;
  if (a.Ws && wtype == W_BF16 && mt >= 1 && mt <= kMaxMt && a.M <= 16 * mt) {
    switch (a.epi.kind) {
      case EPI_QKV: return launch_ring<EPI_QKV>(a, mt, s);
      case EPI_RESID: return launch_ring<EPI_RESID>(a, mt, s);
      case EPI_SILU: return launch_ring<EPI_SILU>(a, mt, s);
      case EPI_PART: return launch_ring<EPI_PART>(a, mt, s);
      case EPI_PARTRES: return launch_ring<EPI_PARTRES>(a, mt, s);
      case EPI_STORE: return launch_ring<EPI_STORE>(a, mt, s);
    }
    return hipErrorInvalidValue;
  }
  if (a.G < 1 || (wtype != W_BF16 && a.G != 1)) return hipErrorInvalidValue;
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
