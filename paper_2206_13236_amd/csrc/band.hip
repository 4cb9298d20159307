// Stage 4b: the recursion of Eq. (3) on the pruned lattice (Sec. 3.2,
// Fig. 1(b)): only nodes p_t <= u < p_t + S (and u <= U) exist; every
// transition into any other node is -inf. Loss and band occupations.
//
// Anti-diagonal schedule. Band node (t, s) (u = p_t + s) lies on diagonal
// d = t + u = e_t + s with e_t = t + p_t strictly increasing in t. Its
// vertical predecessor (t, s-1) is on diagonal d-1 of the same frame and its
// horizontal predecessor (t-1, u) is on diagonal d-1 of frame t-1. So a wave
// can advance the whole band one diagonal per step: lane l handles the frames
// t = l, l+64, l+128, ... in turn (a frame is active for at most S <= 32
// consecutive diagonals, so a lane is always free when its next frame
// starts), keeps its own vertical carry in a register and receives the
// horizontal value from lane l-1 by one rotate. The sequential depth is
// T + U diagonals instead of T * S slot updates.
//
// Wave 0 runs the forward (alpha) pass and wave 1 the backward (beta) pass
// concurrently; then all waves form the occupations. Band log-probs and the
// bounds are staged in LDS first. Same precision scheme as the full lattice:
// log2 domain, fp64 accumulators, fp32 exp2/log2 only for LogAdd's bounded
// correction term.
#include "kernels.h"
#include "prof.h"

namespace {

constexpr int kBandThreads = 256;

struct BandView {
  const float* X;  // px [T*S] of the utterance (LDS or global)
  const float* Y;  // py
  const int* P;    // p_t [T]
  int Tn, Un, S;
};

DEV void band_frame(const BandView& v, int t, int& e, int& ns) {
  if (t >= 0 && t < v.Tn) {
    const int p = v.P[t];
    e = t + p;
    ns = min(v.S, v.Un - p + 1);
  } else {
    e = 1 << 30;
    ns = 0;
  }
}

DEV void band_alpha(const BandView& v, double* __restrict__ alpha, int lane) {
  const int D = v.Tn + v.Un;
  int t = lane, e, ns;
  band_frame(v, t, e, ns);
  double hout = kNegInfD, vout = kNegInfD;
  const int src = (lane + 63) & 63;
  for (int d = 0; d < D; ++d) {
    double hin = __shfl(hout, src, 64);
    int s = d - e;
    if (s >= ns && t < v.Tn) {
      t += 64;
      band_frame(v, t, e, ns);
      s = d - e;
    }
    double nh = kNegInfD, nv = kNegInfD;
    if (s >= 0 && s < ns) {
      const int k = t * v.S + s;
      const double x2 = (double)v.X[k] * kLog2e;
      const double y2 = (double)v.Y[k] * kLog2e;
      if (t == 0) hin = kNegInfD;
      const double vin = (s == 0) ? kNegInfD : vout;
      const double al = (d == 0) ? 0.0 : log2add(hin, vin);
      alpha[k] = al;
      nh = al + y2;
      nv = al + x2;
    }
    hout = nh;
    vout = nv;
  }
}

DEV void band_beta(const BandView& v, double* __restrict__ beta, int lane) {
  const int D = v.Tn + v.Un;
  // this lane's frames in descending order: the largest t = lane (mod 64) below Tn
  int t = (lane < v.Tn) ? lane + 64 * ((v.Tn - 1 - lane) / 64) : -1;
  int e, ns;
  band_frame(v, t, e, ns);
  double bout = kNegInfD;
  const int src = (lane + 1) & 63;
  for (int d = D - 1; d >= 0; --d) {
    double hin = __shfl(bout, src, 64);
    int s = d - e;
    if (s < 0 && t >= 0) {
      t -= 64;
      band_frame(v, t, e, ns);
      s = d - e;
    }
    double nb = kNegInfD;
    if (t >= 0 && s >= 0 && s < ns) {
      const int k = t * v.S + s;
      const double x2 = (double)v.X[k] * kLog2e;
      const double y2 = (double)v.Y[k] * kLog2e;
      if (t == v.Tn - 1) hin = (v.P[t] + s == v.Un) ? 0.0 : kNegInfD;
      const double vin = (s + 1 < ns) ? bout : kNegInfD;
      nb = log2add(y2 + hin, x2 + vin);
      beta[k] = nb;
    }
    bout = nb;
  }
}

__global__ __launch_bounds__(kBandThreads) void band_kernel(BandArgs a) {
  extern __shared__ __align__(16) float sm[];
  __shared__ double sL;
  const int n = blockIdx.x;
  const int T = a.b.T, S = a.S;
  int Tn, Un;
  const bool ok = utt_dims(a.b, n, Tn, Un);
  const size_t base = (size_t)n * T * S;
  const int* rng = a.ranges + base;
  float* X = sm;
  float* Y = sm + (size_t)T * S;
  int* P = reinterpret_cast<int*>(sm + (size_t)2 * T * S);
  for (int i = threadIdx.x; i < Tn * S; i += kBandThreads) {
    X[i] = a.px[base + i];
    Y[i] = a.py[base + i];
  }
  // p_t, clamped so that every index derived from it stays in the band arrays
  for (int t = threadIdx.x; t < Tn; t += kBandThreads) P[t] = min(max(rng[(size_t)t * S], 0), Un);
  __syncthreads();
  BandView v;
  v.X = X;
  v.Y = Y;
  v.P = P;
  v.Tn = Tn;
  v.Un = Un;
  v.S = S;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  double* alpha = a.alpha + base;
  double* beta = a.beta + base;
  if (wave == 0) band_alpha(v, alpha, lane);
  else if (wave == 1) band_beta(v, beta, lane);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int pl = v.P[Tn - 1];
    const int se = Un - pl;
    double L = kNegInfD;
    if (se >= 0 && se < S) L = alpha[(size_t)(Tn - 1) * S + se] + (double)v.Y[(Tn - 1) * S + se] * kLog2e;
    sL = ok ? L : __builtin_nan("");
  }
  __syncthreads();
  const double L2 = sL;
  if (threadIdx.x == 0) a.loss[n] = (L2 == L2) ? (float)(-L2 * kLn2) : __builtin_nanf("");
  if (!a.gx && !a.gy) return;
  const bool live = (L2 == L2) && (L2 != kNegInfD);
  // Per-anti-diagonal normalisers (every complete path crosses diagonal
  // d = t + u at exactly one band node): the occupations of the edges leaving
  // diagonal d are normalised by that diagonal's own total, which cancels the
  // common part of the rounding accumulated by alpha and beta.
  double* Ld = reinterpret_cast<double*>(sm + (size_t)2 * T * S + T + (T & 1));
  const int D = Tn + Un;
  if (live) {
    for (int d = threadIdx.x; d < D; d += kBandThreads) {
      // last frame whose band starts at or before d (e_t = t + p_t is increasing)
      int lo = 0, hi = Tn - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (mid + P[mid] <= d) lo = mid;
        else hi = mid - 1;
      }
      double mx = kNegInfD;
      for (int t = lo; t >= 0 && d - (t + P[t]) < S; --t) {
        const int s = d - (t + P[t]);
        if (s >= 0 && P[t] + s <= Un) {
          const double x = alpha[(size_t)t * S + s] + beta[(size_t)t * S + s];
          mx = x > mx ? x : mx;
        }
      }
      double sum = 0.0;
      for (int t = lo; t >= 0 && d - (t + P[t]) < S; --t) {
        const int s = d - (t + P[t]);
        if (s >= 0 && P[t] + s <= Un) {
          const double x = alpha[(size_t)t * S + s] + beta[(size_t)t * S + s];
          if (x != kNegInfD) sum += (double)exp2f((float)(x - mx));
        }
      }
      Ld[d] = mx + log2(sum);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < T * S; i += kBandThreads) {
    const int t = i / S, s = i - t * S;
    float gxv = 0.f, gyv = 0.f;
    if (live && t < Tn) {
      const int p = v.P[t];
      const int u = p + s;
      if (u <= Un) {
        const double al = alpha[i];
        const double Lt = Ld[t + u];
        if (s + 1 < S && u + 1 <= Un)
          gxv = exp2_occ(al + (double)v.X[i] * kLog2e + beta[i + 1] - Lt);
        double nb;
        if (t + 1 < Tn) {
          const int s2 = u - v.P[t + 1];
          nb = (s2 >= 0 && s2 < S) ? beta[(size_t)(t + 1) * S + s2] : kNegInfD;
        } else {
          nb = (u == Un) ? 0.0 : kNegInfD;
        }
        gyv = exp2_occ(al + (double)v.Y[i] * kLog2e + nb - Lt);
      }
    }
    if (a.gx) a.gx[base + i] = gxv;
    if (a.gy) a.gy[base + i] = gyv;
  }
}

}  // namespace

// px, py [T*S] floats, p_t [T] ints (padded to 8 bytes), per-diagonal totals [T+U+1] doubles
size_t band_smem_bytes(int T, int U, int S) {
  return (size_t)T * S * 2 * sizeof(float) + (size_t)(T + (T & 1)) * sizeof(int) + (size_t)(T + U + 1) * sizeof(double);
}

hipError_t launch_band(const BandArgs& a, hipStream_t s) {
  const size_t sm = band_smem_bytes(a.b.T, a.b.U, a.S);
  if (sm > 150 * 1024) return hipErrorInvalidValue;
  if (sm > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(band_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
  }
  {
    RNNT_PROF(s, "band");
    hipLaunchKernelGGL(band_kernel, dim3(a.b.N), dim3(kBandThreads), sm, s, a);
  }
  return hipGetLastError();
}
