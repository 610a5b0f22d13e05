// Token-tree verification: the drafts of several drafters, each continuing
// the same committed prefix, verified in one target forward (Algorithm 1
// runs one thread per drafter on every prefix; with lookahead their drafts
// form a tree rooted at the last committed token w0).
//
// Node i of a window's tree (node 0 = w0, parent[i] < i for i > 0) is one
// row of the forward: its K/V go to cache slot L + i, its RoPE position is
// L + depth(i), and it attends to the prefix and to the slots of its own
// ancestors (an ancestor bit mask per row, 64 nodes at most).  From the
// rows' logits the exact-match walk of Algorithm 1 picks the accepted path:
// from the root, repeatedly take the target's greedy token t at the current
// node and move to the child of smallest index (the j* rule: children are
// numbered in drafter order) whose token is t; stop when there is none.
//
// Three launches besides the forward and the row statistics:
//   prep    -- one wave per window: validates the parent array and forms
//              depth and ancestor masks;
//   decide  -- one workgroup per window: row argmax from the chunk
//              statistics, then the walk by wave 0 (one lane per node);
//   compact -- one workgroup per (layer, window, KV head): moves the K/V of
//              the accepted path's nodes 1..n to slots L+1..L+n so the
//              committed cache is the ordinary causal one.
#include <limits.h>
#include <math.h>

#include "internal.h"

namespace dsi {

namespace {

__global__ __launch_bounds__(64) void k_tprep(TreeArgs a) {
  __shared__ int sp[kMaxRows];
  const int b = blockIdx.x, i = threadIdx.x;
  const int R = a.R;
  int p = -1;
  bool ok = true;
  if (i < R) {
    p = a.parent[b * R + i];
    ok = i == 0 ? p == -1 : (p >= 0 && p < i);
    sp[i] = p;
  }
  __syncthreads();
  const bool invalid = __any(!ok);
  if (i < R) {
    int dep = 0;
    unsigned long long m = 1ull << i;
    if (!invalid) {
      // parents strictly decrease, so the walk ends at the root
      for (int c = p; c >= 0; c = sp[c]) {
        m |= 1ull << c;
        ++dep;
      }
    }
    a.depth[b * R + i] = dep;
    a.anc[b * R + i] = m;
  }
  if (i == 0) {
    a.bad[b] = invalid ? 1 : 0;
    if (invalid) atomicOr(a.err, 8);
  }
}

__global__ __launch_bounds__(256) void k_tdecide(TreeArgs a) {
  __shared__ int sArg[kMaxRows];
  const int b = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int R = a.R;
  // each wave: the argmax of a row from its chunk (max, argmax) pairs;
  // larger value wins, ties to the smaller token id
  for (int i = w; i < R; i += 4) {
    const size_t r = (size_t)b * R + i;
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int c = lane; c < a.C; c += 64) {
      const float2 pa = a.part_arg[r * a.C + c];
      const int ia = __float_as_int(pa.y);
      if (pa.x > bv || (pa.x == bv && ia < bi)) {
        bv = pa.x;
        bi = ia;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (lane == 0) sArg[i] = bi;
  }
  __syncthreads();
  if (w != 0) return;
  int tok = -1, par = -1;
  bool badtok = false;
  if (lane < R) {
    tok = a.tokens[b * R + lane];
    par = a.parent[b * R + lane];
    badtok = tok < 0 || tok >= a.V;
  }
  const bool anybadtok = __any(badtok);
  const bool invalid = anybadtok || a.bad[b] != 0;
  int v = 0, n = 0, mine = lane == 0 ? 0 : -1;
  if (!invalid) {
    // children have larger indices than their parent: at most R - 1 moves
    for (;;) {
      const int t = sArg[v];
      const unsigned long long hit = __ballot(lane > 0 && lane < R && par == v && tok == t);
      if (!hit) break;
      v = __ffsll((long long)hit) - 1;
      ++n;
      if (lane == n) mine = v;
    }
  }
  if (lane < R) a.path[b * R + lane] = invalid ? -1 : mine;
  if (lane == 0) {
    const int wi = a.window0 + b;
    const int L = a.lens ? a.lens[wi] : 0;
    if (invalid) {
      a.n_out[b] = -1;
      a.tok_out[b] = -1;
      if (anybadtok) atomicOr(a.err, 2);
      a.decision[b] = make_int4(0, L, 1, 0);
    } else {
      a.n_out[b] = n;
      a.tok_out[b] = sArg[v];
      a.decision[b] = make_int4(n, L, 0, 0);
      if (a.commit && a.lens) a.lens[wi] = L + n + 1;
    }
  }
}

// Path rows 1..n of one (layer, window, KV head): every source is read
// into LDS before any destination is written (a destination slot L + i can
// be the source of a later path entry).  n <= kMaxRows - 1 and hd <= 128.
template <typename T>
__global__ __launch_bounds__(256) void k_tcompact(TreeArgs a, T* kc, T* vc, size_t layer_elems,
                                                   size_t win_elems, int n_kv, int hd, int maxlen) {
  __shared__ T st[(kMaxRows - 1) * 128];
  int id = blockIdx.x;
  const int h = id % n_kv;
  id /= n_kv;
  const int b = id % a.B;
  const int l = id / a.B;
  const int4 dec = a.decision[b];
  if (dec.z) return;
  const int n = dec.x, L = dec.y;
  if (n == 0) return;
  const int* path = a.path + (size_t)b * a.R;
  const size_t base = (size_t)l * layer_elems + (size_t)(a.window0 + b) * win_elems;
  T* K = kc + base + (size_t)h * maxlen * hd;
  T* Vt = vc + base + (size_t)h * hd * maxlen;
  const int cnt = n * hd;
  for (int e = threadIdx.x; e < cnt; e += 256) {
    const int i = e / hd + 1, d = e - (i - 1) * hd;
    st[e] = K[kc_off(L + path[i], d, hd)];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < cnt; e += 256) {
    const int i = e / hd + 1, d = e - (i - 1) * hd;
    K[kc_off(L + i, d, hd)] = st[e];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < cnt; e += 256) {
    const int i = e / hd + 1, d = e - (i - 1) * hd;
    st[e] = Vt[vc_off(L + path[i], d, hd)];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < cnt; e += 256) {
    const int i = e / hd + 1, d = e - (i - 1) * hd;
    Vt[vc_off(L + i, d, hd)] = st[e];
  }
}

}  // namespace

hipError_t launch_tree_prep(const TreeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_tprep, dim3(a.B), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tree_decide(const TreeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_tdecide, dim3(a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tree_compact(const TreeArgs& a, int kv_bf16, void* kc, void* vc, int n_layers,
                               size_t layer_elems, size_t win_elems, int n_kv, int hd, int maxlen,
                               hipStream_t s) {
  if (a.R > kMaxRows || hd > 128) return hipErrorInvalidValue;
  const dim3 g((unsigned)(n_layers * a.B * n_kv));
  if (kv_bf16)
    hipLaunchKernelGGL(k_tcompact<uint16_t>, g, dim3(256), 0, s, a, (uint16_t*)kc, (uint16_t*)vc,
                       layer_elems, win_elems, n_kv, hd, maxlen);
  else
    hipLaunchKernelGGL(k_tcompact<float>, g, dim3(256), 0, s, a, (float*)kc, (float*)vc, layer_elems,
                       win_elems, n_kv, hd, maxlen);
  return hipGetLastError();
}

}  // namespace dsi
