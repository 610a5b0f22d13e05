// Causal window-over-prefix attention with grouped KV heads, split over key
// chunks (one workgroup of eight, or four, waves per chunk), plus the log-sum-exp
// combine of the chunk partials (a second launch; when the plan has a single
// chunk the attention kernel normalises its own output instead).
//
// Row i of window b (position L_b + i) attends to keys [0, L_b + i]: the
// cached prefix and the window rows before it (the k+1 prompts of one
// verification, Section 2).  For one (window, KV head) the G = n_heads /
// n_kv query heads times R window rows form the query side; they are cut
// into tiles of 16 queries.  Per 32-key step a wavefront computes
//   S^T[key][query] = K . Q^T     (A = 16 K rows, B = Q^T hi/lo)
//   O^T[d][query]  += V^T . P^T   (A = V^T rows)
// with 16x16x32 bf16 MFMAs (two per product for the hi/lo query or
// probability split), so every operand is a 16-byte lane load and the
// query owned by a lane (l % 16) is the same in S^T, P^T and O^T: the
// online-softmax rescale is lane-local.  The K rows of the two S^T tiles are
// permuted so that lane l ends up holding keys p0 + 8*(l/16) + 0..7, which is
// exactly its P^T B-operand fragment.  fp32 caches use 16x16x4 fp32 MFMAs
// on the same data arrangement.  The cache is stored in 32-position blocks
// (kc_off / vc_off): the keys and the values of one step are each one
// contiguous block (8 KB at hd = 128) and every fragment load reads whole
// 128-byte lines.
#include <math.h>

#include "device_util.h"

namespace dsi {

namespace {

// PIPE: each wave handles several 32-key steps (long prefixes); the loads
// of its next step are issued as soon as the current step's K (after S) and
// V (after O) fragments have been consumed, so they overlap the math.
// NTL: keys and values read by this workgroup only (one query tile) are
// loaded nontemporally, streaming them past the caches: a long prefix then
// reads at ~6.7-7.0 instead of ~5.6-5.9 TB/s.
// TREE: token-tree rows -- a window key L + j is visible to query row i only
// if node j is an ancestor of node i (or i itself), per AttnArgs::anc.
// NWV: waves per workgroup, 8, or 4 (many windows in flight: more, smaller
// workgroups), for bf16 caches with registers capped so that three
// workgroups share a CU.
template <int KVB, int HD, int PIPE, int TREE, int NWV, int NTL>
__global__ __launch_bounds__(NWV * 64, (NWV == 4 && KVB) ? 3 : 1) void k_attn(AttnArgs a) {
  constexpr int DS = HD / 32;
  constexpr int DT = HD / 16;
  __shared__ float sm[NWV][16];
  __shared__ float sl[NWV][16];
  __shared__ f32x4 so[NWV][DT][64];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform: scalar branches
  // XCD-aware order: workgroups are dispatched to the 8 XCDs round-robin by
  // linear id, so ids 8 r + x land on XCD x.  Every (chunk, query tile) of
  // one (window, KV head) z gets an id congruent to z mod 8 -- the same XCD
  // and L2 -- so the query tiles of a chunk read its keys and values from
  // HBM once (8B at 2048 keys: 7.55 -> 7.28 us per launch against one XCD
  // per chunk).  The order affects speed only: a kernel boundary makes
  // every write visible to every XCD.
  const int xcd = blockIdx.x & 7, rr = blockIdx.x >> 3;
  const int y = rr % a.n_qtiles;
  const int c = (rr / a.n_qtiles) % a.n_chunks;
  const int z = (rr / (a.n_qtiles * a.n_chunks)) * 8 + xcd;
  if (z >= a.n_windows * a.n_kv) return;
  const int win = z / a.n_kv, kvh = z % a.n_kv;
  const int G = a.n_heads / a.n_kv;
  const int R = a.rows.rows_per_window;
  const int wabs = a.rows.window0 + win;
  const int len = a.rows.lens[wabs];
  const int klen = len + R;
  const int c0 = c * a.chunk;
  const int c1 = min(klen, c0 + a.chunk);

  const int qi = y * 16 + (lane & 15);
  const bool qvalid = qi < G * R;
  const int gh = qvalid ? qi / R : 0;
  const int ri = qvalid ? qi % R : 0;
  const int qpos = qvalid ? len + ri : -1;
  const int mtok = win * R + ri;
  const int head = kvh * G + gh;
  unsigned long long anc = ~0ull;
  if constexpr (TREE) anc = qvalid ? a.anc[mtok] : 0ull;

  const size_t kbase = ((size_t)wabs * a.n_kv + kvh) * (size_t)a.maxlen * HD;
  const size_t vbase = ((size_t)wabs * a.n_kv + kvh) * (size_t)HD * a.maxlen;
  const int r16 = lane & 15;
  const int kgrp = (lane >> 4) * 8;
  const float scale2 = a.scale * 1.44269504088896340736f;   // log2 e

  // K and V of one 32-key step
  struct KV16 {
    u32x4 k[2][DS], v[DT];
  };
  struct KV32 {
    F8 k[2][DS], v[DT];
  };
  KV16 b16;
  KV32 b32;
  auto load_k_into = [&](KV16& d16, KV32& d32, int p0) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int key = p0 + (r16 >> 2) * 8 + t * 4 + (r16 & 3);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const size_t kidx = kbase + kc_off(key, ds * 32 + kgrp, HD);
        if (KVB) {
          const u32x4* src = (const u32x4*)((const uint16_t*)a.kc + kidx);
          d16.k[t][ds] = NTL ? __builtin_nontemporal_load(src) : *src;
        } else {
          d32.k[t][ds].a = *(const float4*)((const float*)a.kc + kidx);
          d32.k[t][ds].b = *(const float4*)((const float*)a.kc + kidx + 4);
        }
      }
    }
  };
  auto load_v_into = [&](KV16& d16, KV32& d32, int p0) {
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      // dims t*16 + r16 of the step's block, keys kgrp .. kgrp + 7
      const size_t vidx = vbase + vc_off(p0 + kgrp, t * 16 + r16, HD);
      if (KVB) {
        const u32x4* src = (const u32x4*)((const uint16_t*)a.vc + vidx);
        d16.v[t] = NTL ? __builtin_nontemporal_load(src) : *src;
      } else {
        d32.v[t].a = *(const float4*)((const float*)a.vc + vidx);
        d32.v[t].b = *(const float4*)((const float*)a.vc + vidx + 4);
      }
    }
  };
  // query (B operand of S^T): Q[q][ds*32 + 8*(l/16) + e].  Its loads are
  // issued first, then the first step's K and V loads, and the query is
  // split into hi/lo while those are in flight.
  const float* qrow = a.q + (size_t)mtok * (a.n_heads * HD) + head * HD;
  F8 qf[DS];
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) {
    // unconditional (an invalid lane reads row 0 of its window and zeroes
    // it), so that later waits count the loads exactly
    const int d0 = ds * 32 + (lane >> 4) * 8;
    const float4 qa = *(const float4*)(qrow + d0);
    const float4 qb = *(const float4*)(qrow + d0 + 4);
    const float mk = qvalid ? 1.f : 0.f;   // rows are finite: x * 0 = 0
    qf[ds].a = float4{qa.x * mk, qa.y * mk, qa.z * mk, qa.w * mk};
    qf[ds].b = float4{qb.x * mk, qb.y * mk, qb.z * mk, qb.w * mk};
  }
  // The first step's loads do not wait for the window length: they are
  // issued for every step inside the chunk and the allocation (keys beyond
  // the window are masked).  A wave whose first step lies past the chunk or
  // the allocation loads the chunk's last 32 keys instead and discards
  // them: the loads are unconditional, so the compiler's waits count them
  // exactly (loads retire in order).  Chunk starts, chunk sizes and the
  // allocation are multiples of 32, so pfirst < plim implies
  // pfirst + 32 <= plim.
  const int stride = 32 * NWV;
  const int pfirst = c0 + 32 * w;
  const int plim = min(c0 + a.chunk, a.maxlen);
  load_k_into(b16, b32, max(0, min(pfirst, plim - 32)));
  load_v_into(b16, b32, max(0, min(pfirst, plim - 32)));
  __builtin_amdgcn_sched_barrier(0);   // issue them here, not next to their use
  bf16x8 qh[DS], ql[DS];
  if (KVB) {
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint16_t h, l2;
        split_bf16(f8_get(qf[ds], e), h, l2);
        qh[ds][e] = __builtin_bit_cast(__bf16, h);
        ql[ds][e] = __builtin_bit_cast(__bf16, l2);
      }
  }

  float mrun = -INFINITY, lrun = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // one 32-key step on the K/V held in (d16, d32); with pnext >= 0 the
  // loads of step pnext go into the same registers as soon as the step's K
  // (after S) and V (after O) have been consumed
  auto step = [&](int p0, KV16& d16, KV32& d32, int pnext) {
    f32x4 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        if (KVB) {
          const bf16x8 kb = as_bf16x8(d16.k[t][ds]);
          st[t] = mfma_bf16(kb, qh[ds], st[t]);
          st[t] = mfma_bf16(kb, ql[ds], st[t]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) st[t] = mfma_f32(f8_get(d32.k[t][ds], e), f8_get(qf[ds], e), st[t]);
        }
      }
    }
    if (pnext >= 0 && pnext < c1) load_k_into(d16, d32, pnext);
    // Lane holds keys p0 + kgrp + (t*4 + j) for query (lane & 15).  Scores
    // are kept in base-2 units (scale times log2 e), so that each
    // exponential is one v_exp_f32.  A step whose keys are all live keys of
    // the chunk that every query row sees -- prefix keys (rows sit at
    // positions len and later; a tree row sees the keys before len only) --
    // needs no mask, a test that is the same for the whole wave.
    const bool full = p0 + 32 <= c1 && p0 + 32 <= (TREE ? len : len + 1);
    float sv[8];
    float mloc = -INFINITY;
    if (full) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sv[e] = st[e >> 2][e & 3] * scale2;
        mloc = fmaxf(mloc, sv[e]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int key = p0 + kgrp + e;
        bool vis = key <= qpos && key < c1;
        if constexpr (TREE) vis = vis && (key < len || ((anc >> ((key - len) & 63)) & 1ull));
        sv[e] = vis ? st[e >> 2][e & 3] * scale2 : -INFINITY;
        mloc = fmaxf(mloc, sv[e]);
      }
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float mnew = fmaxf(mrun, mloc);
    const float base = (mnew == -INFINITY) ? 0.f : mnew;
    float pv[8];
    float lsum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv[e] = __builtin_amdgcn_exp2f(sv[e] - base);
      lsum += pv[e];
    }
    // rescale only when some row's running maximum moved (else alpha is 1)
    if (__ballot(mnew != mrun)) {
      const float alpha = __builtin_amdgcn_exp2f(mrun - base);
      lrun *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t) o[t] *= alpha;
    }
    lrun += lsum;
    mrun = mnew;

    // keys at or past c1 (past the window's rows: dead cache rows or beyond
    // the allocation) have probability 0, but 0 * NaN is not 0: their V
    // elements are zeroed, so that whatever a dead row holds never reaches
    // the output (dsi_kv_poison)
    const int nv = c1 - (p0 + kgrp);   // valid keys among the lane's 8
    if (!full && nv < 8) {
      if (KVB) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t keep = (2 * i < nv ? 0x0000FFFFu : 0u) | (2 * i + 1 < nv ? 0xFFFF0000u : 0u);
#pragma unroll
          for (int t = 0; t < DT; ++t) d16.v[t][i] &= keep;
        }
      } else {
        auto zero4 = [&](float4& x, int e0) {
          x.x = e0 < nv ? x.x : 0.f;
          x.y = e0 + 1 < nv ? x.y : 0.f;
          x.z = e0 + 2 < nv ? x.z : 0.f;
          x.w = e0 + 3 < nv ? x.w : 0.f;
        };
#pragma unroll
        for (int t = 0; t < DT; ++t) {
          zero4(d32.v[t].a, 0);
          zero4(d32.v[t].b, 4);
        }
      }
    }
    if (KVB) {
      bf16x8 ph, pl;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint16_t h, l2;
        split_bf16(pv[e], h, l2);
        ph[e] = __builtin_bit_cast(__bf16, h);
        pl[e] = __builtin_bit_cast(__bf16, l2);
      }
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const bf16x8 vv = as_bf16x8(d16.v[t]);
        o[t] = mfma_bf16(vv, ph, o[t]);
        o[t] = mfma_bf16(vv, pl, o[t]);
      }
    } else {
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[t] = mfma_f32(f8_get(d32.v[t], e), pv[e], o[t]);
    }
    if (pnext >= 0 && pnext < c1) load_v_into(d16, d32, pnext);
  };

  if constexpr (PIPE == 1) {
    for (int p0 = pfirst; p0 < c1; p0 += stride) step(p0, b16, b32, p0 + stride);
  } else if (pfirst < c1) {
    // unpipelined plans have chunk == 32 * NWV (launch_main takes PIPE 0
    // only then): a single step per wave, on the loads issued above
    step(pfirst, b16, b32, -1);
  }

  // combine the waves of this workgroup into one partial (m, l, O)
  lrun += __shfl_xor(lrun, 16);
  lrun += __shfl_xor(lrun, 32);
  if (lane < 16) {
    sm[w][lane] = mrun;
    sl[w][lane] = lrun;
  }
#pragma unroll
  for (int t = 0; t < DT; ++t) so[w][t][lane] = o[t];
  __syncthreads();
  if (a.n_chunks == 1) {
    // one key chunk: normalise here, no partials and no combine launch
    for (int it = threadIdx.x; it < DT * 64; it += NWV * 64) {
      const int t = it >> 6, l = it & 63, q = l & 15;
      const int qc = y * 16 + q;
      if (qc >= G * R) continue;
      float M = sm[0][q];
#pragma unroll
      for (int ww = 1; ww < NWV; ++ww) M = fmaxf(M, sm[ww][q]);
      const float b = (M == -INFINITY) ? 0.f : M;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      float L = 0.f;
#pragma unroll
      for (int ww = 0; ww < NWV; ++ww) {
        const float f = __builtin_amdgcn_exp2f(sm[ww][q] - b);
        acc += so[ww][t][l] * f;
        L += sl[ww][q] * f;
      }
      const float inv = 1.0f / L;
      const float y4[4] = {acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
      pack_store4(a.out, a.wtype, win * R + qc % R, (kvh * G + qc / R) * HD + t * 16 + (l >> 4) * 4, y4);
    }
    return;
  }
  const size_t zy = (size_t)z * a.n_qtiles + y;
  const size_t zyc = zy * a.n_chunks + c;
  for (int it = threadIdx.x; it < DT * 64; it += NWV * 64) {
    const int t = it >> 6, l = it & 63, q = l & 15;
    float M = sm[0][q];
#pragma unroll
    for (int ww = 1; ww < NWV; ++ww) M = fmaxf(M, sm[ww][q]);
    const float b = (M == -INFINITY) ? 0.f : M;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ww = 0; ww < NWV; ++ww) acc += so[ww][t][l] * __builtin_amdgcn_exp2f(sm[ww][q] - b);
    float* dst = a.part_o + (zyc * 16 + q) * HD + t * 16 + (l >> 4) * 4;
    *(float4*)dst = float4{acc[0], acc[1], acc[2], acc[3]};
  }
  if (threadIdx.x < 16) {
    const int q = threadIdx.x;
    float M = sm[0][q];
#pragma unroll
    for (int ww = 1; ww < NWV; ++ww) M = fmaxf(M, sm[ww][q]);
    const float b = (M == -INFINITY) ? 0.f : M;
    float L = 0.f;
#pragma unroll
    for (int ww = 0; ww < NWV; ++ww) L += sl[ww][q] * __builtin_amdgcn_exp2f(sm[ww][q] - b);
    a.part_ml[zyc * 16 + q] = make_float2(M * 0.69314718055994530942f, L);   // back to natural units
  }

}

// Log-sum-exp combine of the chunk partials of one (window, KV head, query
// tile): out = sum_c e^(m_c - M) O_c / sum_c e^(m_c - M) l_c, chunks in
// order.  One workgroup per (HD/32 column slice, query tile, window x KV
// head), in the attention launch's XCD order; one thread per (query, 4
// columns).  Each thread loads the (m, l) pairs and
// partial columns of up to CB chunks at once, so the loads of a batch are in
// flight together; across batches the running sums are rescaled to the new
// maximum (with at most CB chunks there is one batch: plain two-pass form).
template <int HD>
__global__ __launch_bounds__(128) void k_attn_combine(AttnArgs a) {
  constexpr int CB = 16;
  // ids 8 r + x run on XCD x: (window, KV head) z on XCD z mod 8, as in the
  // attention launch
  const int xcd = blockIdx.x & 7, rc = blockIdx.x >> 3;
  const int xs = rc % (HD / 32), y = (rc / (HD / 32)) % a.n_qtiles;
  const int z = (rc / ((HD / 32) * a.n_qtiles)) * 8 + xcd;
  if (z >= a.n_windows * a.n_kv) return;
  const int win = z / a.n_kv, kvh = z % a.n_kv;
  const int G = a.n_heads / a.n_kv;
  const int R = a.rows.rows_per_window;
  const size_t zy = (size_t)z * a.n_qtiles + y;
  // 128 threads: 16 queries x 8 float4 columns = 32 columns of this slice
  const int q = threadIdx.x >> 3;
  const int d = xs * 32 + (threadIdx.x & 7) * 4;
  const int qi = y * 16 + q;
  if (qi >= G * R) return;
  const float2* ml = a.part_ml + zy * a.n_chunks * 16 + q;
  const float* po = a.part_o + (zy * a.n_chunks * 16 + q) * HD + d;
  float M = -INFINITY, base = 0.f, L = 0.f;
  float4 acc = float4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < a.n_chunks; c0 += CB) {
    float2 mv[CB];
    float4 ov[CB];
#pragma unroll
    for (int i = 0; i < CB; ++i)
      if (c0 + i < a.n_chunks) {
        mv[i] = ml[(size_t)(c0 + i) * 16];
        ov[i] = *(const float4*)(po + (size_t)(c0 + i) * 16 * HD);
      }
#pragma unroll
    for (int i = 0; i < CB; ++i)
      if (c0 + i < a.n_chunks) M = fmaxf(M, mv[i].x);
    const float b = (M == -INFINITY) ? 0.f : M;
    if (c0 > 0) {
      const float r = expf(base - b);
      L *= r;
      acc.x *= r;
      acc.y *= r;
      acc.z *= r;
      acc.w *= r;
    }
    base = b;
#pragma unroll
    for (int i = 0; i < CB; ++i)
      if (c0 + i < a.n_chunks) {
        const float f = expf(mv[i].x - b);
        L += mv[i].y * f;
        acc.x += ov[i].x * f;
        acc.y += ov[i].y * f;
        acc.z += ov[i].z * f;
        acc.w += ov[i].w * f;
      }
  }
  const float inv = 1.0f / L;
  const float y4[4] = {acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv};
  pack_store4(a.out, a.wtype, win * R + qi % R, (kvh * G + qi / R) * HD + d, y4);
}

template <int KVB, int HD, int NWV>
void launch_main(const AttnArgs& a, dim3 grid, hipStream_t s) {
  const dim3 blk(NWV * 64);
  const bool pipe = a.chunk > NWV * 32;
  if constexpr (KVB && NWV == kAttnWaves) {
    // several steps per wave and one query tile: no other workgroup reads
    // these keys and values
    if (pipe && a.n_qtiles == 1 && !a.anc) {
      hipLaunchKernelGGL((k_attn<KVB, HD, 1, 0, NWV, 1>), grid, blk, 0, s, a);
      return;
    }
  }
  if (a.anc) {
    if (pipe)
      hipLaunchKernelGGL((k_attn<KVB, HD, 1, 1, NWV, 0>), grid, blk, 0, s, a);
    else
      hipLaunchKernelGGL((k_attn<KVB, HD, 0, 1, NWV, 0>), grid, blk, 0, s, a);
  } else {
    if (pipe)
      hipLaunchKernelGGL((k_attn<KVB, HD, 1, 0, NWV, 0>), grid, blk, 0, s, a);
    else
      hipLaunchKernelGGL((k_attn<KVB, HD, 0, 0, NWV, 0>), grid, blk, 0, s, a);
  }
}

template <int KVB, int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  const int z8 = (a.n_windows * a.n_kv + 7) / 8 * 8;   // (window, KV head) groups, padded to the XCDs
  dim3 g1(z8 * a.n_chunks * a.n_qtiles);
  if (a.waves == 4)
    launch_main<KVB, HD, 4>(a, g1, s);
  else
    launch_main<KVB, HD, kAttnWaves>(a, g1, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_chunks == 1) return e;
  dim3 g2(z8 * (HD / 32) * a.n_qtiles);
  hipLaunchKernelGGL((k_attn_combine<HD>), g2, dim3(128), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int kv_bf16, int hd, const AttnArgs& a, hipStream_t s) {
  if (a.waves != 4 && a.waves != kAttnWaves) return hipErrorInvalidValue;
  if (a.chunk % (a.waves * 32)) return hipErrorInvalidValue;
  if (kv_bf16) {
    switch (hd) {
      case 32: return launch_hd<1, 32>(a, s);
      case 64: return launch_hd<1, 64>(a, s);
      case 96: return launch_hd<1, 96>(a, s);
      case 128: return launch_hd<1, 128>(a, s);
    }
  } else {
    switch (hd) {
      case 32: return launch_hd<0, 32>(a, s);
      case 64: return launch_hd<0, 64>(a, s);
      case 96: return launch_hd<0, 96>(a, s);
      case 128: return launch_hd<0, 128>(a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace dsi
