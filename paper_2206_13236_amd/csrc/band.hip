// Stage 4b: the recursion of Eq. (3) on the pruned lattice (Sec. 3.2,
// Fig. 1(b)): only nodes p_t <= u < p_t + S (and u <= U) exist; every
// transition into any other node is -inf. Loss and band occupations.
//
// band_fb_kernel, anti-diagonal schedule. Band node (t, s) (u = p_t + s) lies
// on diagonal d = t + u = e_t + s with e_t = t + p_t strictly increasing in t.
// Its vertical predecessor (t, s-1) is on diagonal d-1 of the same frame and
// its horizontal predecessor (t-1, u) is on diagonal d-1 of frame t-1. So a
// wave advances the whole band one diagonal per step: lane l handles the
// frames t = l, l+64, l+128, ... in turn (a frame is active for at most
// S <= 32 consecutive diagonals, so a lane is always free when its next frame
// starts), keeps its vertical carry in a register and receives the horizontal
// value from lane l-1 by one DPP wave rotate. The sequential depth is T + U
// diagonals instead of T * S slot updates. Wave 0 runs alpha and wave 1 beta
// concurrently; band log-probs and bounds are staged in LDS and each lane
// prefetches its next node's values one step ahead.
//
// band_occ_kernel: one wave per frame of the batch, lanes over the S slots.
// Every complete path leaves frame t through exactly one blank edge, so the
// frame's own log-sum of alpha + blank + beta(next) equals the total; the
// occupations of frame t are normalised by it (cancelling the rounding the
// alpha and beta chains accumulate in common).
//
// Same precision scheme as the full lattice: log2 domain, fp64 accumulators,
// fp32 exp2/log2 only for LogAdd's bounded correction term.
#include "kernels.h"
#include "prof.h"

namespace {

constexpr int kBandThreads = 128;

struct BandView {
  const float* X;  // px [T*S] of the utterance (LDS)
  const float* Y;  // py
  const int* P;    // p_t [T]
  int Tn, Un, S;
};

// Start diagonal e = t + p_t and number of present slots of frame t (e huge
// and no slots outside [0, Tn)); the LDS read is unconditional.
DEV void band_frame(const BandView& v, int t, int& e, int& ns) {
  const bool in = (t >= 0) && (t < v.Tn);
  const int p = v.P[in ? t : 0];
  e = in ? t + p : (1 << 30);
  ns = in ? min(v.S, v.Un - p + 1) : 0;
}

// The step loops below are branch-free: frame switches are selects, the
// geometry of the lane's following frame is re-read from LDS every step (and
// only used at the next switch), the values of the next node are prefetched
// every step, and lanes without a node store to kOob (a dropped buffer
// store). Divergent branches with LDS reads would make every step wait for
// them.
DEV void band_alpha(const BandView& v, Rsrc alpha, int lane) {
  const int D = v.Tn + v.Un, S = v.S;
  int t = lane, e, ns;
  band_frame(v, t, e, ns);
  int tn = t + 64, en, nsn;
  band_frame(v, tn, en, nsn);
  double hout = kNegInfD, vout = kNegInfD;
  int kn = (t < v.Tn) ? t * S : 0;  // the next node this lane will process
  float xn = v.X[kn], yn = v.Y[kn];
  for (int d = 0; d < D; ++d) {
    const double hin0 = dpp_move_d<kDppWaveRor1>(hout, kNegInfD);
    const bool adv = (d - e >= ns) && (t < v.Tn);
    t = adv ? tn : t;
    e = adv ? en : e;
    ns = adv ? nsn : ns;
    tn = t + 64;
    band_frame(v, tn, en, nsn);
    const int s = d - e;
    const bool act = (s >= 0) && (s < ns);
    const int k = act ? t * S + s : 0;
    const double x2 = (double)xn * kLog2e;
    const double y2 = (double)yn * kLog2e;
    const double hin = (t == 0) ? kNegInfD : hin0;
    const double vin = (s == 0) ? kNegInfD : vout;
    const double al = (d == 0) ? 0.0 : log2add(hin, vin);
    buf_store_f64(alpha, act ? (uint32_t)k * 8u : kOob, al);
    hout = act ? al + y2 : kNegInfD;
    vout = act ? al + x2 : kNegInfD;
    // next node: (t, s+1) while the frame lasts, else the first node of frame t+64
    kn = act ? ((s + 1 < ns) ? k + 1 : (tn < v.Tn ? tn * S : 0)) : kn;
    xn = v.X[kn];
    yn = v.Y[kn];
  }
}

DEV void band_beta(const BandView& v, Rsrc beta, int lane) {
  const int D = v.Tn + v.Un, S = v.S;
  // this lane's frames in descending order: the largest t = lane (mod 64) below Tn
  int t = (lane < v.Tn) ? lane + 64 * ((v.Tn - 1 - lane) / 64) : -1;
  int e, ns;
  band_frame(v, t, e, ns);
  int tn = t - 64, en, nsn;
  band_frame(v, tn, en, nsn);
  double bout = kNegInfD;
  int kn = (t >= 0) ? t * S + ns - 1 : 0;  // the next node this lane will process
  float xn = v.X[kn], yn = v.Y[kn];
  for (int d = D - 1; d >= 0; --d) {
    const double hin0 = dpp_move_d<kDppWaveRol1>(bout, kNegInfD);
    const bool adv = (d - e < 0) && (t >= 0);
    t = adv ? tn : t;
    e = adv ? en : e;
    ns = adv ? nsn : ns;
    tn = t - 64;
    band_frame(v, tn, en, nsn);
    const int s = d - e;
    const bool act = (t >= 0) && (s >= 0) && (s < ns);
    const int k = act ? t * S + s : 0;
    const double x2 = (double)xn * kLog2e;
    const double y2 = (double)yn * kLog2e;
    // the successor of the last frame's final node is the end (beta = 0)
    const double hin = (t == v.Tn - 1) ? ((e - t + s == v.Un) ? 0.0 : kNegInfD) : hin0;
    const double vin = (s + 1 < ns) ? bout : kNegInfD;
    const double be = log2add(y2 + hin, x2 + vin);
    buf_store_f64(beta, act ? (uint32_t)k * 8u : kOob, be);
    bout = act ? be : kNegInfD;
    // next node: (t, s-1) while the frame lasts, else the top node of frame t-64
    kn = act ? ((s > 0) ? k - 1 : (tn >= 0 ? tn * S + nsn - 1 : 0)) : kn;
    xn = v.X[kn];
    yn = v.Y[kn];
  }
}

__global__ __launch_bounds__(kBandThreads) void band_fb_kernel(BandArgs a) {
  extern __shared__ __align__(16) float sm[];
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
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: the resources stay scalar
  double* alpha = a.alpha + base;
  if (wave == 0) band_alpha(v, make_rsrc(alpha, (size_t)T * S * sizeof(double)), lane);
  else band_beta(v, make_rsrc(a.beta + base, (size_t)T * S * sizeof(double)), lane);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int se = Un - P[Tn - 1];
    double L = kNegInfD;
    if (se >= 0 && se < S) L = alpha[(size_t)(Tn - 1) * S + se] + (double)Y[(Tn - 1) * S + se] * kLog2e;
    const double L2 = ok ? L : __builtin_nan("");
    a.Lutt[n] = L2;
    a.loss[n] = (L2 == L2) ? (float)(-L2 * kLn2) : __builtin_nanf("");
  }
}

__global__ __launch_bounds__(256) void band_occ_kernel(BandArgs a) {
  const int T = a.b.T, S = a.S;
  const int lane = threadIdx.x & 63;
  const int f = blockIdx.x * 4 + (threadIdx.x >> 6);  // frame over N*T
  if (f >= a.b.N * T) return;
  const int n = f / T, t = f - n * T;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const double Lu = a.Lutt[n];
  const bool live = (Lu == Lu) && (Lu != kNegInfD) && t < Tn;
  const int s = lane;
  double ey = kNegInfD, ex = kNegInfD;
  if (live && s < S) {
    const int p = min(max(a.ranges[(size_t)f * S], 0), Un);
    const int u = p + s;
    if (u <= Un) {
      const size_t k = (size_t)f * S + s;
      const double al = a.alpha[k];
      double nb;
      if (t + 1 < Tn) {
        const int pn = min(max(a.ranges[(size_t)(f + 1) * S], 0), Un);
        const int s2 = u - pn;
        nb = (s2 >= 0 && s2 < S) ? a.beta[(size_t)(f + 1) * S + s2] : kNegInfD;
      } else {
        nb = (u == Un) ? 0.0 : kNegInfD;
      }
      ey = al + (double)a.py[k] * kLog2e + nb;
      if (s + 1 < S && u + 1 <= Un) ex = al + (double)a.px[k] * kLog2e + a.beta[k + 1];
    }
  }
  const double mx = wave_max_d(ey);
  const double sum = wave_sum_d((ey != kNegInfD) ? (double)exp2f((float)(ey - mx)) : 0.0);
  const double Lt = mx + log2(sum);
  if (s < S) {
    float gxv = 0.f, gyv = 0.f;
    if (live && ey != kNegInfD) gyv = exp2_occ(ey - Lt);
    if (live && ex != kNegInfD) gxv = exp2_occ(ex - Lt);
    if (a.gx) a.gx[(size_t)f * S + s] = gxv;
    if (a.gy) a.gy[(size_t)f * S + s] = gyv;
  }
}

}  // namespace

// px, py [T*S] floats, p_t [T] ints
size_t band_smem_bytes(int T, int U, int S) {
  (void)U;
  return (size_t)T * S * 2 * sizeof(float) + (size_t)T * sizeof(int);
}

hipError_t launch_band(const BandArgs& a, hipStream_t s) {
  const size_t sm = band_smem_bytes(a.b.T, a.b.U, a.S);
  if (sm > 150 * 1024) return hipErrorInvalidValue;
  if (sm > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(band_fb_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
  }
  {
    RNNT_PROF(s, "band_fb");
    hipLaunchKernelGGL(band_fb_kernel, dim3(a.b.N), dim3(kBandThreads), sm, s, a);
  }
  if (a.gx || a.gy) {
    RNNT_PROF(s, "band_occ");
    hipLaunchKernelGGL(band_occ_kernel, dim3((a.b.N * a.b.T + 3) / 4), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}
