// Stage 3: pruning bounds (Sec. 3.2.2).
//
// For every frame t the locally optimal start p_t maximises Eq. (8),
//   score(t,p) = -gx(t,p-1) + gy(t,p) + gy(t,p+1) + ... + gy(t,p+S-1),
// over p in [0, P], P = max(0, U-S+1) ("green arcs minus red arc"; Eq. (7)
// is the S = 4, p = 2 instance). The sum is evaluated in fp32 in exactly that
// order (no contraction: additions only), y'(t,-1) counts as 0 and slots above
// U add 0, so equal inputs give bit-identical bounds on any IEEE fp32 machine.
// Ties go to the smallest p and NaN never wins.
//
// The raw bounds are clamped to the envelope [P - (S-1)(T-1-t), min(P, (S-1)t)]
// (the band must hold the start node at t = 0 and the final node at t = T-1,
// and consecutive starts may differ by at most S-1), then made consistent with
// Eq. (9) (monotone) and Eq. (10) (no skip) by the procedure the paper's
// LaTeX source gives in a commented-out block of Sec. 3.2.2: suffix minimum,
// reflect by (S-1)t, suffix minimum, reflect back, max with 0. All of that is
// integer arithmetic.
//
// Two kernels: the scores, one wave per frame of the whole batch with the
// lanes spread over p (coalesced loads of the occupation row) and a (score, p)
// reduction to the first maximum; then one workgroup per utterance for the
// clamp and the two suffix minima, Hillis-Steele scans over LDS (min is exact
// and associative, so the order does not matter).
#include "kernels.h"
#include "prof.h"

namespace {

constexpr int kPruneThreads = 1024;

// Lexicographic (largest score, then smallest p); NaN compares as -inf.
DEV void better(float& bs, int& bp, float s, int p) {
  if (s > bs || (s == bs && p < bp)) {
    bs = s;
    bp = p;
  }
}

DEV void suffix_min(int* a, int* tmp, int Tn) {
  int* src = a;
  int* dst = tmp;
  for (int off = 1; off < Tn; off <<= 1) {
    for (int t = threadIdx.x; t < Tn; t += kPruneThreads)
      dst[t] = (t + off < Tn) ? min(src[t], src[t + off]) : src[t];
    __syncthreads();
    int* x = src;
    src = dst;
    dst = x;
  }
  if (src != a) {
    for (int t = threadIdx.x; t < Tn; t += kPruneThreads) a[t] = src[t];
    __syncthreads();
  }
}

// Scores of Eq. (8) and the raw argmax, one wave per frame over the whole
// batch; the raw start is parked in ranges[n][t][0] for the scan kernel.
__global__ __launch_bounds__(256) void prune_score_kernel(BatchDev b, int S, const float* __restrict__ gx,
                                                          const float* __restrict__ gy, int* __restrict__ ranges) {
#pragma clang fp contract(off)
  const int T = b.T, U1 = b.U + 1;
  const int lane = threadIdx.x & 63;
  const int f = blockIdx.x * 4 + (threadIdx.x >> 6);  // frame index over N*T
  if (f >= b.N * T) return;
  const int n = f / T, t = f - n * T;
  int Tn, Un;
  utt_dims(b, n, Tn, Un);
  if (t >= Tn) return;
  const int P = max(0, Un - S + 1);
  const float* gxr = gx + (size_t)f * U1;
  const float* gyr = gy + (size_t)f * U1;
  float bs = kNegInfF;
  int bp = 0;
  for (int p0 = 0; p0 <= P; p0 += 64) {
    const int q = p0 + lane;
    if (q <= P) {
      float acc = (q == 0) ? 0.0f : -gxr[q - 1];
      for (int k = 0; k < S; ++k) {
        const int u = q + k;
        acc = acc + ((u <= Un) ? gyr[u] : 0.0f);
      }
      better(bs, bp, (acc != acc) ? kNegInfF : acc, q);
    }
  }
  // the best (score, p) of the wave: within each 16-lane row by DPP
  // rotations, then across the rows (a total order: any order of the
  // comparisons selects the same pair)
  better(bs, bp, dpp_row_ror<8>(bs), __float_as_int(dpp_row_ror<8>(__int_as_float(bp))));
  better(bs, bp, dpp_row_ror<4>(bs), __float_as_int(dpp_row_ror<4>(__int_as_float(bp))));
  better(bs, bp, dpp_row_ror<2>(bs), __float_as_int(dpp_row_ror<2>(__int_as_float(bp))));
  better(bs, bp, dpp_row_ror<1>(bs), __float_as_int(dpp_row_ror<1>(__int_as_float(bp))));
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    const float os = __shfl_xor(bs, off, 64);
    const int op = __shfl_xor(bp, off, 64);
    better(bs, bp, os, op);
  }
  if (lane == 0) ranges[(size_t)f * S] = bp;
}

// Envelope clamp and the suffix-minimum / reflection adjustment, one
// workgroup per utterance (integer arithmetic only).
__global__ __launch_bounds__(kPruneThreads) void prune_scan_kernel(BatchDev b, int S, int* __restrict__ ranges) {
  extern __shared__ int sp[];  // [2 * T]
  int* p = sp;
  int* tmp = sp + b.T;
  const int n = blockIdx.x;
  const int T = b.T;
  int Tn, Un;
  utt_dims(b, n, Tn, Un);
  const int P = max(0, Un - S + 1);
  int* out = ranges + (size_t)n * T * S;
  for (int t = threadIdx.x; t < Tn; t += kPruneThreads) {
    const int lo = P - (S - 1) * (Tn - 1 - t);
    const int hi = min(P, (S - 1) * t);
    p[t] = min(max(out[(size_t)t * S], lo), hi);
  }
  __syncthreads();
  suffix_min(p, tmp, Tn);
  for (int t = threadIdx.x; t < Tn; t += kPruneThreads) p[t] = (S - 1) * t - p[t];
  __syncthreads();
  suffix_min(p, tmp, Tn);
  for (int i = threadIdx.x; i < T * S; i += kPruneThreads) {
    const int t = i / S, s = i - t * S;
    out[i] = (t < Tn) ? max(0, (S - 1) * t - p[t]) + s : s;
  }
}

}  // namespace

size_t prune_smem_bytes(int T) { return (size_t)2 * T * sizeof(int); }

hipError_t launch_prune(const BatchDev& b, int S, const float* gx, const float* gy, int* ranges,
                        hipStream_t s) {
  {
    RNNT_PROF(s, "prune_score");
    hipLaunchKernelGGL(prune_score_kernel, dim3((b.N * b.T + 3) / 4), dim3(256), 0, s, b, S, gx, gy, ranges);
  }
  {
    RNNT_PROF(s, "prune_scan");
    hipLaunchKernelGGL(prune_scan_kernel, dim3(b.N), dim3(kPruneThreads), prune_smem_bytes(b.T), s, b, S, ranges);
  }
  return hipGetLastError();
}
