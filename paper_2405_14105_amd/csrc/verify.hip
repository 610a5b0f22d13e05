// Accept/reject of B verification windows from their target logits.
//
// Sampling mode (the lossless rule the paper adopts from its cited works,
// Sections 2 and 3.1), per window with rows z_0..z_k:
//   p_i = softmax(z_{i-1} / T); a_i = p_i(d_i) / q_i(d_i); A_i = [u_i < a_i];
//   n = min{i : A_i = 0} - 1 (else k), the accepted count of Theorem 2's
//   proof; token drawn by inverse CDF with u_{k+1} from max(0, p_{n+1} -
//   q_{n+1}) (n < k; p_{n+1} if that has no mass) or from p_{k+1} (n = k).
// Greedy mode (Algorithm 1's exact match): A_i = [d_i = argmax z_{i-1}],
//   token = argmax z_n, ties to the lowest id.
// All softmax statistics, ratios and CDF sums are fp64 (an fp32 CDF over
// 128k entries picks visibly different tokens); every reduction has a fixed
// order, so results are run-to-run identical.
//
// Four launches:
//   1. row statistics: per (row, 4096-entry chunk) max, sum exp, argmax;
//   2. decide: one wavefront per window combines chunk statistics, tests the
//      k drafts in parallel and finds the first rejection with a ballot;
//      greedy windows finish here;
//   3. per (window, chunk): fp64 sums of the residual (and of p) over the
//      chunk, via the same block scan used in step 4;
//   4. sample: one workgroup per window locates the chunk that holds
//      u_{k+1} R, rescans it and emits the token; commits the KV length.
#include <limits.h>
#include <math.h>

#include "scan.h"

namespace dsi {

namespace {

constexpr int VT = 256;                  // threads per workgroup
constexpr int PER = kVerifyChunk / VT;   // 16 entries per thread

__global__ __launch_bounds__(VT) void k_vrow(VerifyArgs a) {
  __shared__ double shd[4];
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const float* z = a.logits + (size_t)r * a.V;
  const int v0 = c * kVerifyChunk;
  const int v1 = min(a.V, v0 + kVerifyChunk);
  float vals[PER];
  float zmax = -INFINITY;
  int zarg = INT_MAX;
  // all loads first and unconditional (clamped index, masked after), so
  // they are in flight together: a wait behind a conditional load is a
  // wait for every load (loads retire in order)
#pragma unroll
  for (int i = 0; i < PER; ++i) vals[i] = z[min(v0 + (int)threadIdx.x + VT * i, v1 - 1)];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int v = v0 + threadIdx.x + VT * i;
    if (v >= v1) vals[i] = -INFINITY;
    if (v < v1 && (vals[i] > zmax || (vals[i] == zmax && v < zarg))) {
      zmax = vals[i];
      zarg = v;
    }
  }
  // argmax: larger value wins, ties to the smaller index
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(zmax, o);
    const int oi = __shfl_xor(zarg, o);
    if (ov > zmax || (ov == zmax && oi < zarg)) {
      zmax = ov;
      zarg = oi;
    }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    shv[w] = zmax;
    shi[w] = zarg;
  }
  __syncthreads();
  zmax = shv[0];
  zarg = shi[0];
  for (int i = 1; i < 4; ++i)
    if (shv[i] > zmax || (shv[i] == zmax && shi[i] < zarg)) {
      zmax = shv[i];
      zarg = shi[i];
    }
  const double m = (double)zmax / a.temperature;
  double sum = 0.0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int v = v0 + threadIdx.x + VT * i;
    if (v < v1) sum += exp((double)vals[i] / a.temperature - m);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  if ((threadIdx.x & 63) == 0) shd[w] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double tot = (shd[0] + shd[1]) + (shd[2] + shd[3]);
    a.part[(size_t)r * a.C + c] = make_double2(m, tot);
    a.part_arg[(size_t)r * a.C + c] = make_float2(zmax, __int_as_float(zarg));
  }
}

// one workgroup per window: each wave combines the chunk statistics of a
// row (lanes over chunks, butterfly in fixed order), then wave 0 decides
__global__ __launch_bounds__(VT) void k_vdecide(VerifyArgs a) {
  __shared__ double sM[kMaxRows], sS[kMaxRows];
  __shared__ int sArg[kMaxRows];
  const int b = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = a.k, R = k + 1;
  for (int i = w; i < R; i += VT / 64) {
    const int r = b * R + i;
    double m = -INFINITY;
    for (int c = lane; c < a.C; c += 64) m = fmax(m, a.part[(size_t)r * a.C + c].x);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
    double sum = 0.0;
    float bv = -INFINITY;
    int bi = INT_MAX;
    for (int c = lane; c < a.C; c += 64) {
      const double2 pc = a.part[(size_t)r * a.C + c];
      sum += pc.y * exp(pc.x - m);
      const float2 pa = a.part_arg[(size_t)r * a.C + c];
      const int ia = __float_as_int(pa.y);
      if (pa.x > bv || (pa.x == bv && ia < bi)) {
        bv = pa.x;
        bi = ia;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      sum += __shfl_xor(sum, o);
      const float ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (lane == 0) {
      sM[i] = m;
      sS[i] = sum;
      sArg[i] = bi;
      a.rowstat[r] = make_double2(m, sum);
      a.rowarg[r] = bi;
    }
  }
  __syncthreads();
  if (w != 0) return;
  const double M = lane < R ? sM[lane] : 0.0;
  const double S = lane < R ? sS[lane] : 1.0;
  const int arg = lane < R ? sArg[lane] : 0;
  int bad = 0;
  bool acc = true;
  if (lane < R) {
    const int t = a.tokens[b * R + lane];
    if (t < 0 || t >= a.V) bad = 1;
  }
  if (lane < k && !bad) {
    const int d = a.tokens[b * R + lane + 1];
    const int r = b * R + lane;
    if (a.greedy) {
      acc = (d == arg);
    } else {
      const float qd = a.q[((size_t)b * k + lane) * a.V + d];
      if (!(qd > 0.f) || !isfinite(qd)) {
        bad = 1;
      } else {
        const double p = exp((double)a.logits[(size_t)r * a.V + d] / a.temperature - M) / S;
        const double ratio = p / (double)qd;
        acc = (double)a.u[b * R + lane] < ratio;
      }
    }
  }
  const bool anybad = __any(bad);
  const unsigned long long rej = __ballot(lane < k && !acc);
  const int n = rej ? (__ffsll((long long)rej) - 1) : k;
  const int tokn = __shfl(arg, n);
  if (lane == 0) {
    if (anybad) {
      a.n_out[b] = -1;
      a.tok_out[b] = -1;
      atomicOr(a.err, 2);
      a.decision[b] = make_int4(n, b * R + n, 0, 1);
    } else if (a.greedy) {
      a.n_out[b] = n;
      a.tok_out[b] = tokn;
      if (a.commit && a.lens) a.lens[a.window0 + b] += n + 1;
      a.decision[b] = make_int4(n, b * R + n, 0, 1);
    } else {
      a.decision[b] = make_int4(n, b * R + n, n < k ? 1 : 0, 0);
    }
  }
}

// r_v of an entry with logit z and drafter probability q for the window's
// drawing distribution
__device__ __forceinline__ double entry_mass(const VerifyArgs& a, float z, float q, double M, double S,
                                             bool residual) {
  const double p = exp((double)z / a.temperature - M) / S;
  if (!residual) return p;
  const double d = p - (double)q;
  return d > 0.0 ? d : 0.0;
}

// The PER logits (and drafter probabilities, when qrow is given) from entry
// v0 on, all loads issued before any is used (indices clamped into the row,
// entries past it are never used): a wait behind a conditional load would
// be a wait for every load (loads retire in order).
__device__ __forceinline__ void load_entries(const VerifyArgs& a, const float* zrow, const float* qrow, int v0,
                                             float (&zv)[PER], float (&qv)[PER]) {
#pragma unroll
  for (int i = 0; i < PER; ++i) zv[i] = zrow[min(v0 + i, a.V - 1)];
  if (qrow) {
#pragma unroll
    for (int i = 0; i < PER; ++i) qv[i] = qrow[min(v0 + i, a.V - 1)];
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) qv[i] = 0.f;
  }
}

__global__ __launch_bounds__(VT) void k_vresid(VerifyArgs a) {
  __shared__ double sh[4];
  const int c = blockIdx.x, b = blockIdx.y;
  const int4 dec = a.decision[b];
  if (dec.w) return;
  const int n = dec.x, r = dec.y;
  const bool residual = dec.z != 0;
  const double2 st = a.rowstat[r];
  const float* zrow = a.logits + (size_t)r * a.V;
  const float* qrow = residual ? a.q + ((size_t)b * a.k + n) * a.V : nullptr;
  const int v0 = c * kVerifyChunk + threadIdx.x * PER;
  float zv[PER], qv[PER];
  load_entries(a, zrow, qrow, v0, zv, qv);
  double sr = 0.0, sp = 0.0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (v0 + i < a.V) {
      sr += entry_mass(a, zv[i], qv[i], st.x, st.y, residual);
      sp += entry_mass(a, zv[i], qv[i], st.x, st.y, false);
    }
  }
  const double ir = block_scan_incl<VT / 64>(sr, sh);
  const double ip = block_scan_incl<VT / 64>(sp, sh);
  if (threadIdx.x == VT - 1) a.csum[(size_t)b * a.C + c] = make_double2(ir, ip);
}

__global__ __launch_bounds__(VT) void k_vsample(VerifyArgs a) {
  __shared__ double sh[4];
  __shared__ double s_base, s_target;
  __shared__ int s_chunk, s_usep, s_found;
  __shared__ int s_first, s_last;
  const int b = blockIdx.x;
  const int4 dec = a.decision[b];
  if (dec.w) return;
  const int n = dec.x, r = dec.y;
  const bool residual0 = dec.z != 0;
  const double2 st = a.rowstat[r];
  if (threadIdx.x < 64) {
    // wave 0: prefix sums over the chunk sums, 64 chunks at a time, in one
    // fixed order for the total and for locating the chunk
    const int lane = threadIdx.x;
    const int groups = (a.C + 63) / 64;
    auto prefix = [&](int g, double carry, int usep) {
      const int c = g * 64 + lane;
      double x = 0.0;
      if (c < a.C) {
        const double2 cs = a.csum[(size_t)b * a.C + c];
        x = usep ? cs.y : cs.x;
      }
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double t = __shfl_up(x, o);
        if (lane >= o) x += t;
      }
      return carry + x;
    };
    int usep = 0;
    double R = 0.0;
    for (int g = 0; g < groups; ++g) R = __shfl(prefix(g, R, 0), 63);
    if (residual0 && !(R > 0.0)) {   // no residual mass: draw from p
      usep = 1;
      R = 0.0;
      for (int g = 0; g < groups; ++g) R = __shfl(prefix(g, R, 1), 63);
    }
    const double target = (double)a.u[b * (a.k + 1) + a.k] * R;
    int chunk = -1;
    double base = 0.0, carry = 0.0;
    for (int g = 0; g < groups; ++g) {
      const double incl = prefix(g, carry, usep);
      const double prev = __shfl_up(incl, 1);
      const double excl = lane ? prev : carry;
      const unsigned long long hit = __ballot(g * 64 + lane < a.C && incl > target);
      if (hit) {   // uniform across the wave
        const int l = __ffsll((long long)hit) - 1;
        chunk = g * 64 + l;
        base = __shfl(excl, l);
        break;
      }
      carry = __shfl(incl, 63);
    }
    int found = 1;
    if (chunk < 0) {               // rounding left no crossing: last chunk with mass
      found = 0;
      for (int c = a.C - 1; c >= 0; --c) {
        const double2 cs = a.csum[(size_t)b * a.C + c];
        if ((usep ? cs.y : cs.x) > 0.0) {
          chunk = c;
          break;
        }
      }
      if (chunk < 0) chunk = a.C - 1;
    }
    if (lane == 0) {
      s_chunk = chunk;
      s_base = base;
      s_target = target;
      s_usep = usep;
      s_found = found;
      s_first = INT_MAX;
      s_last = -1;
    }
  }
  __syncthreads();
  const bool residual = residual0 && !s_usep;
  const float* zrow = a.logits + (size_t)r * a.V;
  const float* qrow = residual ? a.q + ((size_t)b * a.k + n) * a.V : nullptr;
  const int v0 = s_chunk * kVerifyChunk + threadIdx.x * PER;
  float zv[PER], qv[PER];
  load_entries(a, zrow, qrow, v0, zv, qv);
  double vals[PER];
  double own = 0.0;
  int lastpos = -1;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int v = v0 + i;
    vals[i] = v < a.V ? entry_mass(a, zv[i], qv[i], st.x, st.y, residual) : 0.0;
    own += vals[i];
    if (vals[i] > 0.0) lastpos = v;
  }
  const double incl = block_scan_incl<VT / 64>(own, sh);
  // exclusive prefix of this thread = inclusive prefix of the previous one
  __shared__ double sincl[VT];
  sincl[threadIdx.x] = incl;
  __syncthreads();
  double run = s_base + (threadIdx.x > 0 ? sincl[threadIdx.x - 1] : 0.0);
  int first = INT_MAX;
  if (s_found) {
    double cw = threadIdx.x > 0 ? sincl[threadIdx.x - 1] : 0.0;
    for (int i = 0; i < PER; ++i) {
      cw += vals[i];
      run = s_base + cw;
      if (run > s_target && vals[i] > 0.0) {
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
    a.n_out[b] = n;
    a.tok_out[b] = tok;
    if (a.commit && a.lens) a.lens[a.window0 + b] += n + 1;
  }
}

}  // namespace

size_t verify_workspace_bytes(int rows, int B, int V) {
  const int C = (V + kVerifyChunk - 1) / kVerifyChunk;
  size_t s = 0;
  s += (size_t)rows * C * sizeof(double2);   // part
  s += (size_t)rows * C * sizeof(float2);    // part_arg
  s += (size_t)rows * sizeof(double2);       // rowstat
  s += (size_t)rows * sizeof(int) + 16;      // rowarg
  s += (size_t)B * sizeof(int4);             // decision
  s += (size_t)B * C * sizeof(double2);      // csum
  return s + 256;
}

void verify_bind_workspace(VerifyArgs& a, void* ws, int rows, int B, int V) {
  const int C = (V + kVerifyChunk - 1) / kVerifyChunk;
  char* p = (char*)ws;
  auto take = [&](size_t bytes) {
    char* q = p;
    p += (bytes + 15) & ~(size_t)15;
    return q;
  };
  a.C = C;
  a.part = (double2*)take((size_t)rows * C * sizeof(double2));
  a.part_arg = (float2*)take((size_t)rows * C * sizeof(float2));
  a.rowstat = (double2*)take((size_t)rows * sizeof(double2));
  a.rowarg = (int*)take((size_t)rows * sizeof(int));
  a.decision = (int4*)take((size_t)B * sizeof(int4));
  a.csum = (double2*)take((size_t)B * C * sizeof(double2));
}

hipError_t launch_verify_rowstats(const VerifyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_vrow, dim3(a.C, a.B * (a.k + 1)), dim3(VT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_verify(const VerifyArgs& a, hipStream_t s) {
  const int rows = a.B * (a.k + 1);
  hipLaunchKernelGGL(k_vrow, dim3(a.C, rows), dim3(VT), 0, s, a);
  hipLaunchKernelGGL(k_vdecide, dim3(a.B), dim3(VT), 0, s, a);
  if (!a.greedy) {
    hipLaunchKernelGGL(k_vresid, dim3(a.C, a.B), dim3(VT), 0, s, a);
    hipLaunchKernelGGL(k_vsample, dim3(a.B), dim3(VT), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace dsi
