// Drafter sampling: from the drafter's logits of the row that ends the
// current context, the stored distribution q = softmax(z / T) (fp64, stored
// fp32) and the next draft, drawn from that stored row by inverse CDF
// (Section 2: the drafter proposes each lookahead token by sampling its own
// next-token distribution given the tokens before it).
//
// The draw: the smallest token t with sum_{v <= t} q_v > u * sum_v q_v, the
// sums taken in fp64 over the fp32 values in ascending token order; if
// rounding leaves no such t, the last t with q_t > 0.  Three launches, all
// with fixed reduction orders (run-to-run identical):
//   1. per 4096-entry chunk: max of z / T and sum of exp(z / T - max) (fp64);
//   2. per chunk: combine all chunk statistics (same order in every block),
//      write the chunk's q = (float) exp(z / T - M) / S, and the fp64 sum of
//      those fp32 values (per-thread runs of 16, then a workgroup scan);
//   3. one workgroup: a wave prefix over the chunk sums locates the chunk
//      holding u * total, the chunk is rescanned in the same order, and the
//      token is written to its slot of the verification window.
#include <limits.h>
#include <math.h>

#include "scan.h"

namespace dsi {

namespace {

constexpr int ST = 256;                  // threads per workgroup
constexpr int SPER = kVerifyChunk / ST;  // 16 entries per thread

__global__ __launch_bounds__(ST) void k_dstat(DraftArgs a) {
  __shared__ double shd[4];
  __shared__ float shv[4];
  const int c = blockIdx.x;
  const int v0 = c * kVerifyChunk;
  const int v1 = min(a.V, v0 + kVerifyChunk);
  float vals[SPER];
  float zmax = -INFINITY;
#pragma unroll
  for (int i = 0; i < SPER; ++i) vals[i] = a.logits[min(v0 + (int)threadIdx.x + ST * i, v1 - 1)];
#pragma unroll
  for (int i = 0; i < SPER; ++i) {
    if (v0 + (int)threadIdx.x + ST * i >= v1) vals[i] = -INFINITY;
    zmax = fmaxf(zmax, vals[i]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) zmax = fmaxf(zmax, __shfl_xor(zmax, o));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) shv[w] = zmax;
  __syncthreads();
  zmax = fmaxf(fmaxf(shv[0], shv[1]), fmaxf(shv[2], shv[3]));
  const double m = (double)zmax / a.temperature;
  double sum = 0.0;
#pragma unroll
  for (int i = 0; i < SPER; ++i) {
    const int v = v0 + threadIdx.x + ST * i;
    if (v < v1) sum += exp((double)vals[i] / a.temperature - m);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  if ((threadIdx.x & 63) == 0) shd[w] = sum;
  __syncthreads();
  if (threadIdx.x == 0) a.part[c] = make_double2(m, (shd[0] + shd[1]) + (shd[2] + shd[3]));
}

// the row's max and normaliser from the chunk statistics: wave 0, chunks
// lane, lane + 64, ... then a butterfly (every block computes the same)
__device__ __forceinline__ void row_stats(const DraftArgs& a, double* sM, double* sS) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    double m = -INFINITY;
    for (int c = lane; c < a.C; c += 64) m = fmax(m, a.part[c].x);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
    double s = 0.0;
    for (int c = lane; c < a.C; c += 64) s += a.part[c].y * exp(a.part[c].x - m);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) {
      *sM = m;
      *sS = s;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(ST) void k_dq(DraftArgs a) {
  __shared__ double sM, sS;
  __shared__ double sh[ST / 64];
  row_stats(a, &sM, &sS);
  const int c = blockIdx.x;
  const double M = sM, S = sS;
  // thread t: entries c*4096 + 16 t .. +15 in order (the rescan's order)
  const int v0 = c * kVerifyChunk + threadIdx.x * SPER;
  double own = 0.0;
  float zv[SPER];
#pragma unroll
  for (int i = 0; i < SPER; ++i) zv[i] = a.logits[min(v0 + i, a.V - 1)];
#pragma unroll
  for (int i = 0; i < SPER; ++i) {
    const int v = v0 + i;
    if (v < a.V) {
      const float q = (float)(exp((double)zv[i] / a.temperature - M) / S);
      a.q_out[v] = q;
      own += (double)q;
    }
  }
  const double incl = block_scan_incl<ST / 64>(own, sh);
  if (threadIdx.x == ST - 1) a.csum[c] = incl;
}

__global__ __launch_bounds__(ST) void k_ddraw(DraftArgs a) {
  __shared__ double sh[ST / 64];
  __shared__ double sincl[ST];
  __shared__ double s_base, s_target;
  __shared__ int s_chunk, s_first, s_last;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    // inclusive prefix over the chunk sums, 64 chunks at a time
    auto prefix = [&](int g, double carry) {
      const int c = g * 64 + lane;
      double x = c < a.C ? a.csum[c] : 0.0;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double t = __shfl_up(x, o);
        if (lane >= o) x += t;
      }
      return carry + x;
    };
    double carry = 0.0;
    const int groups = (a.C + 63) / 64;
    for (int g = 0; g < groups; ++g) carry = __shfl(prefix(g, carry), 63);
    const double target = (double)a.u[0] * carry;
    int chunk = -1;
    double base = 0.0;
    carry = 0.0;
    for (int g = 0; g < groups; ++g) {
      const double incl = prefix(g, carry);
      const double prev = __shfl_up(incl, 1);
      const double excl = lane ? prev : carry;   // exact prefix before chunk g*64+lane
      const unsigned long long hit = __ballot(g * 64 + lane < a.C && incl > target);
      if (hit) {   // uniform across the wave
        const int l = __ffsll((long long)hit) - 1;
        chunk = g * 64 + l;
        base = __shfl(excl, l);
        break;
      }
      carry = __shfl(incl, 63);
    }
    if (chunk < 0) {
      // rounding left no crossing: the last chunk with mass (drawn from its
      // last nonzero entry below)
      for (int c = a.C - 1; c >= 0; --c)
        if (a.csum[c] > 0.0) {
          chunk = c;
          break;
        }
      if (chunk < 0) chunk = a.C - 1;
      base = INFINITY;   // no entry crosses
    }
    if (lane == 0) {
      s_chunk = chunk;
      s_base = base;
      s_target = target;
      s_first = INT_MAX;
      s_last = -1;
    }
  }
  __syncthreads();
  const int v0 = s_chunk * kVerifyChunk + threadIdx.x * SPER;
  double vals[SPER];
  double own = 0.0;
  int lastpos = -1;
  // all loads first (clamped index, masked after): a wait behind a
  // conditional load is a wait for every load issued before it
  float qv[SPER];
#pragma unroll
  for (int i = 0; i < SPER; ++i) qv[i] = a.q_out[min(v0 + i, a.V - 1)];
#pragma unroll
  for (int i = 0; i < SPER; ++i) {
    const int v = v0 + i;
    vals[i] = v < a.V ? (double)qv[i] : 0.0;
    own += vals[i];
    if (vals[i] > 0.0) lastpos = v;
  }
  const double incl = block_scan_incl<ST / 64>(own, sh);
  sincl[threadIdx.x] = incl;
  __syncthreads();
  int first = INT_MAX;
  if (s_base != INFINITY) {
    double cw = threadIdx.x > 0 ? sincl[threadIdx.x - 1] : 0.0;
    for (int i = 0; i < SPER; ++i) {
      cw += vals[i];
      if (s_base + cw > s_target && vals[i] > 0.0) {
        first = v0 + i;
        break;
      }
    }
  }
  if (first != INT_MAX) atomicMin(&s_first, first);
  if (lastpos >= 0) atomicMax(&s_last, lastpos);
  __syncthreads();
  if (threadIdx.x == 0) {
    int tok = s_first != INT_MAX ? s_first : s_last;
    if (tok < 0) tok = 0;
    *a.tok_out = tok;
  }
}

}  // namespace

size_t draft_workspace_bytes(int V) {
  const int C = (V + kVerifyChunk - 1) / kVerifyChunk;
  return (size_t)C * (sizeof(double2) + sizeof(double)) + 256;
}

hipError_t launch_draft_sample(DraftArgs a, void* ws, hipStream_t s) {
  a.C = (a.V + kVerifyChunk - 1) / kVerifyChunk;
  a.part = (double2*)ws;
  a.csum = (double*)((char*)ws + (((size_t)a.C * sizeof(double2) + 15) & ~(size_t)15));
  hipLaunchKernelGGL(k_dstat, dim3(a.C), dim3(ST), 0, s, a);
  hipLaunchKernelGGL(k_dq, dim3(a.C), dim3(ST), 0, s, a);
  hipLaunchKernelGGL(k_ddraw, dim3(1), dim3(ST), 0, s, a);
  return hipGetLastError();
}

}  // namespace dsi
