// Elementwise passes: weight pre-packing, embedding gather + RMSNorm into a
// GEMM activation pack (plus the rotary cos/sin table of the window
// positions), RMSNorm into a pack, and KV length / content operations.
#include <limits>

#include "device_util.h"

namespace dsi {

namespace {

// deterministic block sum of one float per thread (blockDim.x = 256)
__device__ float block_sum_256(float v, float* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  const float t = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  __syncthreads();
  return t;
}

template <typename T>
__global__ void k_prepack(const T* __restrict__ src, int N, int K, T* __restrict__ dst, int Kb,
                          int dst_nb0, int n_blocks, int rowmap, int hd, int which, int dst_Nb, int G) {
  const size_t total = (size_t)n_blocks * Kb * 512;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int e = (int)(i & 7);
    const int lane = (int)((i >> 3) & 63);
    const size_t tile = i >> 9;
    const int kb = (int)(tile % Kb);
    const int nbl = (int)(tile / Kb);       // section-local n-block
    const int r = lane & 15, g = r >> 2, jj = r & 3;
    const int k = kb * 32 + (lane >> 4) * 8 + e;
    int row;
    bool mine = true;
    if (rowmap == 0) {
      row = nbl * 16 + r;
    } else if (rowmap == 1) {
      const int bph = hd >> 4;
      const int h = nbl / bph, j0 = (nbl % bph) * 8;
      row = h * hd + j0 + 2 * g + (jj & 1) + (jj >> 1) * (hd >> 1);
    } else {
      mine = (jj >> 1) == which;
      row = nbl * 8 + 2 * g + (jj & 1);
    }
    if (!mine) continue;
    const T v = (row < N && k < K) ? src[(size_t)row * K + k] : T(0);
    dst[(wtile_index(dst_nb0 + nbl, kb, dst_Nb, Kb, G) * 64 + lane) * 8 + e] = v;
  }
}

// Row-wise RMSNorm into a GEMM pack.  One workgroup per token row; each
// thread owns groups of 8 consecutive features (two 16-byte loads, one
// 16-byte store per pack half), kept in registers between the two passes.
constexpr int kNormGroups = 4;   // d_model <= 256 threads * 8 * 4 = 8192

__device__ __forceinline__ void load8(const void* p, int wtype, size_t i, float* v) {
  if (wtype == W_BF16) {
    const u32x4 r = *(const u32x4*)((const uint16_t*)p + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(r[e] << 16);
      v[2 * e + 1] = __uint_as_float(r[e] & 0xFFFF0000u);
    }
  } else {
    const float4 a = *(const float4*)((const float*)p + i);
    const float4 b = *(const float4*)((const float*)p + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

__device__ __forceinline__ void norm_row(float (&v)[kNormGroups][8], int d, int m, const float* gain,
                                         float eps, int wtype, const PackRef& pack, float* sh) {
  const int ng = d >> 3;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kNormGroups; ++i) {
    const int g = threadIdx.x + 256 * i;
    if (g < ng) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += v[i][e] * v[i][e];
    }
  }
  const float tot = block_sum_256(ss, sh);
  const float rs = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int i = 0; i < kNormGroups; ++i) {
    const int g = threadIdx.x + 256 * i;
    if (g < ng) {
      const float4 g0 = *(const float4*)(gain + 8 * g);
      const float4 g1 = *(const float4*)(gain + 8 * g + 4);
      const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = v[i][e] * rs * gg[e];
      pack_store8(pack, wtype, m, 8 * g, y);
    }
  }
}

__global__ __launch_bounds__(256) void k_embed_norm(EmbedArgs a) {
  __shared__ float sh[4];
  const int m = blockIdx.x;
  int tok = a.tokens[m];
  if (tok < 0 || tok >= a.V) {
    if (threadIdx.x == 0) atomicOr(a.err, 1);
    tok = 0;
  }
  float v[kNormGroups][8];
  const int ng = a.d >> 3;
#pragma unroll
  for (int i = 0; i < kNormGroups; ++i) {
    const int g = threadIdx.x + 256 * i;
    if (g < ng) {
      load8(a.E, a.wtype, (size_t)tok * a.d + 8 * g, v[i]);
      float* xr = a.x + (size_t)m * a.d + 8 * g;
      *(float4*)xr = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
      *(float4*)(xr + 4) = float4{v[i][4], v[i][5], v[i][6], v[i][7]};
      if (a.hidden0) {
        float* hr = a.hidden0 + (size_t)m * a.d + 8 * g;
        *(float4*)hr = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
        *(float4*)(hr + 4) = float4{v[i][4], v[i][5], v[i][6], v[i][7]};
      }
    }
  }
  norm_row(v, a.d, m, a.gain, a.eps, a.wtype, a.pack, sh);
  // rotary table of this row's position: angle = pos * base^(-2j/hd), fp64
  const int R = a.rows.rows_per_window;
  const int pos = a.rows.lens[a.rows.window0 + m / R] + (a.rows.depth ? a.rows.depth[m] : m % R);
  const int half = a.hd >> 1;
  for (int j = threadIdx.x; j < half; j += 256) {
    const double inv = exp2(-2.0 * (double)j / (double)a.hd * a.log2_base);
    double sn, cs;
    sincos((double)pos * inv, &sn, &cs);
    a.rope[(size_t)m * half + j] = make_float2((float)cs, (float)sn);
  }
}

// S (compile time) partials are folded in split order; every load of a row
// group is issued before the sums so they are in flight together.
template <int S>
__global__ __launch_bounds__(256) void k_rmsnorm_pack(float* __restrict__ x, const float* __restrict__ delta,
                                                       size_t dstride, int d,
                                                       const float* __restrict__ gain, float eps,
                                                       int wtype, PackRef pack, float* copy_out) {
  __shared__ float sh[4];
  const int m = blockIdx.x;
  float v[kNormGroups][8];
  const int ng = d >> 3;
#pragma unroll
  for (int i = 0; i < kNormGroups; ++i) {
    const int g = threadIdx.x + 256 * i;
    if (g < ng) {
      const size_t off = (size_t)m * d + 8 * g;
      load8(x, W_F32, off, v[i]);
      if constexpr (S > 0) {
        float p[S][8];
#pragma unroll
        for (int sp = 0; sp < S; ++sp) load8(delta + sp * dstride, W_F32, off, p[sp]);
#pragma unroll
        for (int sp = 0; sp < S; ++sp)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[i][e] += p[sp][e];
        float* xr = x + off;
        *(float4*)xr = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
        *(float4*)(xr + 4) = float4{v[i][4], v[i][5], v[i][6], v[i][7]};
      }
      if (copy_out) {
        float* hr = copy_out + off;
        *(float4*)hr = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
        *(float4*)(hr + 4) = float4{v[i][4], v[i][5], v[i][6], v[i][7]};
      }
    }
  }
  norm_row(v, d, m, gain, eps, wtype, pack, sh);
}

__global__ void k_kv_rollback(int* lens, int window, int new_len, int* err) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    if (new_len < 0 || new_len > lens[window]) atomicOr(err, 4);
    else lens[window] = new_len;
  }
}
__global__ void k_kv_set(int* lens, int window, int v) {
  if (threadIdx.x == 0 && blockIdx.x == 0) lens[window] = v;
}
// advance a window by n prompt tokens if every id is valid
__global__ void k_kv_add_checked(int* lens, int window, const int* tokens, int n, int V, int* err) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x)
    if (tokens[i] < 0 || tokens[i] >= V) bad = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    if (bad) atomicOr(err, 1);
    else lens[window] += n;
  }
}

// copy [n_kv][len][hd] <-> cache (n_kv regions of maxlen * hd, kc_off / vc_off)
template <typename T>
__global__ void k_kv_copy(int to_cache, T* kc, T* vc, int n_kv, int hd, int maxlen, int len,
                          T* dk, T* dv) {
  const size_t total = (size_t)n_kv * len * hd;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int dd = (int)(i % hd);
    const int p = (int)((i / hd) % len);
    const int h = (int)(i / ((size_t)hd * len));
    const size_t ki = (size_t)h * maxlen * hd + kc_off(p, dd, hd);
    const size_t vi = (size_t)h * maxlen * hd + vc_off(p, dd, hd);
    if (to_cache) {
      kc[ki] = dk[i];
      vc[vi] = dv[i];
    } else {
      dk[i] = kc[ki];
      dv[i] = vc[vi];
    }
  }
}

// NaN into the dead rows [lens[window], maxlen) of one window: one block per
// (layer, KV head); kc / vc: the window's layer-0 K and V, layer_stride
// elements apart (kc_off / vc_off inside a head's region)
template <typename T>
__global__ void k_kv_poison(T* kc, T* vc, size_t layer_stride, int n_kv, int hd, int maxlen, const int* lens,
                            int window, T nan) {
  const int layer = blockIdx.x / n_kv, h = blockIdx.x % n_kv;
  const int len = lens[window];
  T* k = kc + layer * layer_stride + (size_t)h * maxlen * hd;
  T* v = vc + layer * layer_stride + (size_t)h * maxlen * hd;
  const size_t n = (size_t)(maxlen - len) * hd;
  for (size_t i = threadIdx.x; i < n; i += blockDim.x) {
    const int p = len + (int)(i / hd), dd = (int)(i % hd);
    k[kc_off(p, dd, hd)] = nan;
    v[vc_off(p, dd, hd)] = nan;
  }
}

// Streaming read rate (diagnostics): each wave reads a contiguous run of
// per_wave_vec 16-byte vectors, 8 loads of 1 KB in flight (a ring, as the
// GEMM weight streams), nontemporal when NT.  The XOR of the data is stored
// only if it equals a fixed pattern, which keeps every load.
template <int NT>
__global__ __launch_bounds__(512) void k_stream_read(const u32x4* __restrict__ buf, size_t per_wave_vec,
                                                     u32x4* sink) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const u32x4* p = buf + ((size_t)blockIdx.x * 8 + w) * per_wave_vec + lane;
  const size_t iters = per_wave_vec / (8 * 64);
  u32x4 acc = {0u, 0u, 0u, 0u};
  u32x4 ring[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) ring[i] = NT ? __builtin_nontemporal_load(p + i * 64) : p[i * 64];
  for (size_t it = 1; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      acc ^= ring[i];
      const u32x4* q = p + (it * 8 + i) * 64;
      ring[i] = NT ? __builtin_nontemporal_load(q) : *q;
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) acc ^= ring[i];
  if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0x85EBCA6Bu && acc.w == 0xC2B2AE35u) *sink = acc;
}

__global__ void k_fill_zero(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

__global__ void k_copy(const float* __restrict__ s, float* __restrict__ d, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    d[i] = s[i];
}

int grid_for(size_t n, int block) {
  size_t g = (n + block - 1) / block;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (int)g;
}

}  // namespace

hipError_t launch_prepack(int wtype, const void* src, int N, int K, void* dst, int Kb, int dst_nb0,
                          int rowmap, int hd, int which, int dst_Nb, int G, hipStream_t s) {
  int n_blocks;
  if (rowmap == 2) n_blocks = (N + 7) / 8;
  else n_blocks = (N + 15) / 16;
  if (G < 1 || dst_nb0 + n_blocks > dst_Nb) return hipErrorInvalidValue;
  const size_t total = (size_t)n_blocks * Kb * 512;
  const int g = grid_for(total, 256);
  if (wtype == W_BF16)
    hipLaunchKernelGGL(k_prepack<uint16_t>, dim3(g), dim3(256), 0, s, (const uint16_t*)src, N, K,
                       (uint16_t*)dst, Kb, dst_nb0, n_blocks, rowmap, hd, which, dst_Nb, G);
  else
    hipLaunchKernelGGL(k_prepack<float>, dim3(g), dim3(256), 0, s, (const float*)src, N, K,
                       (float*)dst, Kb, dst_nb0, n_blocks, rowmap, hd, which, dst_Nb, G);
  return hipGetLastError();
}

hipError_t launch_embed_norm(const EmbedArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_embed_norm, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_pack(float* x, const float* delta, int S, size_t delta_stride, int M, int d,
                               const float* gain, float eps, int wtype, PackRef pack, float* copy_out,
                               hipStream_t s) {
#define DSI_NORM_LAUNCH(SS)                                                                       \
  hipLaunchKernelGGL(k_rmsnorm_pack<SS>, dim3(M), dim3(256), 0, s, x, delta, delta_stride, d, gain, eps, \
                     wtype, pack, copy_out)
  switch (S) {
    case 0: DSI_NORM_LAUNCH(0); break;
    case 1: DSI_NORM_LAUNCH(1); break;
    case 2: DSI_NORM_LAUNCH(2); break;
    case 3: DSI_NORM_LAUNCH(3); break;
    case 4: DSI_NORM_LAUNCH(4); break;
    default: return hipErrorInvalidValue;
  }
#undef DSI_NORM_LAUNCH
  return hipGetLastError();
}

hipError_t launch_kv_rollback(int* lens, int window, int new_len, int* err, hipStream_t s) {
  hipLaunchKernelGGL(k_kv_rollback, dim3(1), dim3(64), 0, s, lens, window, new_len, err);
  return hipGetLastError();
}
hipError_t launch_kv_set(int* lens, int window, int new_len, hipStream_t s) {
  hipLaunchKernelGGL(k_kv_set, dim3(1), dim3(64), 0, s, lens, window, new_len);
  return hipGetLastError();
}
hipError_t launch_kv_add_checked(int* lens, int window, const int* tokens, int n, int V, int* err,
                                 hipStream_t s) {
  hipLaunchKernelGGL(k_kv_add_checked, dim3(1), dim3(256), 0, s, lens, window, tokens, n, V, err);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int to_cache, int kv_bf16, void* kc, void* vc, int n_kv, int hd, int maxlen,
                          int len, void* dk, void* dv, hipStream_t s) {
  const size_t total = (size_t)n_kv * len * hd;
  if (total == 0) return hipSuccess;
  const int g = grid_for(total, 256);
  if (kv_bf16)
    hipLaunchKernelGGL(k_kv_copy<uint16_t>, dim3(g), dim3(256), 0, s, to_cache, (uint16_t*)kc,
                       (uint16_t*)vc, n_kv, hd, maxlen, len, (uint16_t*)dk, (uint16_t*)dv);
  else
    hipLaunchKernelGGL(k_kv_copy<float>, dim3(g), dim3(256), 0, s, to_cache, (float*)kc, (float*)vc,
                       n_kv, hd, maxlen, len, (float*)dk, (float*)dv);
  return hipGetLastError();
}

hipError_t launch_kv_poison(int kv_bf16, void* kc, void* vc, size_t layer_stride, int n_layers, int n_kv, int hd,
                            int maxlen, const int* lens, int window, hipStream_t s) {
  const dim3 grid(n_layers * n_kv), blk(256);
  if (kv_bf16)
    hipLaunchKernelGGL(k_kv_poison<uint16_t>, grid, blk, 0, s, (uint16_t*)kc, (uint16_t*)vc, layer_stride, n_kv,
                       hd, maxlen, lens, window, (uint16_t)0x7FC0u);
  else
    hipLaunchKernelGGL(k_kv_poison<float>, grid, blk, 0, s, (float*)kc, (float*)vc, layer_stride, n_kv, hd,
                       maxlen, lens, window, std::numeric_limits<float>::quiet_NaN());
  return hipGetLastError();
}

hipError_t launch_stream_read(const void* buf, size_t per_wave_vec, int workgroups, int nontemporal, void* sink,
                              hipStream_t s) {
  if (workgroups < 1 || workgroups > kStreamMaxWorkgroups) return hipErrorInvalidValue;
  if (nontemporal)
    hipLaunchKernelGGL(k_stream_read<1>, dim3(workgroups), dim3(512), 0, s, (const u32x4*)buf, per_wave_vec,
                       (u32x4*)sink);
  else
    hipLaunchKernelGGL(k_stream_read<0>, dim3(workgroups), dim3(512), 0, s, (const u32x4*)buf, per_wave_vec,
                       (u32x4*)sink);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(n, 256)), dim3(256), 0, s, (uint32_t*)p, n);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const float* src, float* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy, dim3(grid_for(n, 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

}  // namespace dsi
