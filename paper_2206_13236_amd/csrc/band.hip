// Stage 4b: the recursion of Eq. (3) on the pruned lattice (Sec. 3.2,
// Fig. 1(b)): only nodes p_t <= u < p_t + S (and u <= U) exist; every
// transition into any other node is -inf. Loss and band occupations.
//
// Band node (t, s) (u = p_t + s) lies on anti-diagonal d = t + u = e_t + s,
// e_t = t + p_t strictly increasing in t, so a diagonal holds at most one
// node per slot s. Its predecessors lie on diagonal d-1: the vertical one
// (t, s-1) in slot s-1, the horizontal one (t-1, s + delta_t) in slot
// s + delta_t, delta_t = p_t - p_{t-1}. The successors of beta lie on d+1:
// (t, s+1) and (t+1, s - delta_{t+1}).
//
// Short label sequences (U + 1 <= 64) take the full lattice's recursion:
// band_mask_kernel writes the lattice's diagonal-major layout with one row per
// lane, band nodes holding their log-probs and all other nodes -inf, which
// removes every transition into a node outside the band. One DPP shift per
// step and no per-node lane lookup make this the shorter chain.
//
// Longer ones take the slot layout [D, S] (D = T + U diagonals):
// band_prep_kernel scatters the band log-probs into it with, per slot, the
// two shifts and a validity bit; band_fb_kernel runs one workgroup per
// utterance, wave 0 alpha and wave 1 beta, lane s owning slot s, so a step
// advances one diagonal with one DPP shift (the vertical neighbour) and one
// ds_bpermute (the horizontal neighbour, from a per-node lane), with loads
// issued P diagonals ahead and contiguous stores. The depth is T_n + U_n
// steps on either path.
//
// band_occ_kernel (both layouts): one wave per frame of the batch, lanes over
// the S band offsets.
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
constexpr int kBandPrefetch = 8;

// Per-slot meta word: bit 16 valid; bits 0-7 delta_t (kNoShift: no
// horizontal predecessor, t = 0); bits 8-15 delta_{t+1} (kNoShift: last frame
// and not the final node; kEndNode: the final node (T_n-1, U_n), whose
// successor is the end of the lattice).
constexpr int kNoShift = 255;
constexpr int kEndNode = 254;
constexpr uint32_t kValid = 1u << 16;

DEV int band_p(const BandArgs& a, int n, int t, int Un) {
  return min(max(a.ranges[((size_t)n * a.b.T + t) * a.S], 0), Un);
}

// One thread per (n, t): writes every slot of the diagonals whose start
// e = d - s lies in (e_{t-1}, e_t] (e_{-1} = -1): the frame's own nodes, and
// invalid markers for its slots s >= ns_t and for the start diagonals that
// no frame takes (when p jumps). The last frame also covers the starts after
// e_{T_n-1}, so every slot a recursion reads is written exactly once.
__global__ __launch_bounds__(256) void band_prep_kernel(BandArgs a) {
  const int T = a.b.T, S = a.S, D = a.D;  // W == S on this path
  const int f = blockIdx.x * blockDim.x + threadIdx.x;
  if (f >= a.b.N * T) return;
  const int n = f / T, t = f - n * T;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (t >= Tn) return;
  const int p = band_p(a, n, t, Un);
  const int ns = min(S, Un - p + 1);
  const int pp = (t == 0) ? 0 : band_p(a, n, t - 1, Un);
  const int e = t + p, e_prev = (t == 0) ? -1 : t - 1 + pp;
  const int da = (t == 0) ? kNoShift : p - pp;
  const int db_next = (t + 1 < Tn) ? band_p(a, n, t + 1, Un) - p : kNoShift;
  const size_t src = (size_t)f * S;
  const size_t row0 = (size_t)n * D * S;
  const int Dn = Tn + Un;
  const int e_end = (t + 1 < Tn) ? e : Dn - 1;  // the last frame also covers the starts after its own
  for (int ee = max(e_prev + 1, 0); ee <= e_end; ++ee) {
    for (int s = 0; s < S; ++s) {
      const int d = ee + s;
      if (d >= Dn) break;  // beyond the last diagonal the recursion reads
      const size_t o = row0 + (size_t)d * S + s;
      if (ee == e && s < ns) {
        const int db = (t + 1 < Tn) ? db_next : ((p + s == Un) ? kEndNode : kNoShift);
        a.pxd[o] = (DiagT)((double)a.px[src + s] * kLog2e);
        a.pyd[o] = (DiagT)((double)a.py[src + s] * kLog2e);
        a.meta[o] = kValid | (uint32_t)da | ((uint32_t)db << 8);
      } else {
        a.meta[o] = 0u;
      }
    }
  }
}

// Masked-lattice path: one thread per cell (d, u) of the [D, 64] layout of
// every utterance, in log2 units; -inf off the band and at every cell that is
// no node of the utterance's lattice, as the lattice recursion requires.
__global__ __launch_bounds__(256) void band_mask_kernel(BandArgs a) {
  const int T = a.b.T, S = a.S, D = a.D;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)a.b.N * D * 64) return;
  const int u = (int)(i & 63);
  const int nd = (int)(i >> 6);
  const int n = nd / D, d = nd - n * D;
  const int t = d - u;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  double x = kNegInfD, y = kNegInfD;
  if (t >= 0 && t < Tn && u <= Un) {
    const int s = u - band_p(a, n, t, Un);
    if (s >= 0 && s < S) {
      const size_t k = ((size_t)n * T + t) * S + s;
      x = (double)a.px[k] * kLog2e;
      y = (double)a.py[k] * kLog2e;
    }
  }
  a.pxd[i] = (DiagT)x;
  a.pyd[i] = (DiagT)y;
}

DEV double bpermute_d(double v, int src_lane) {
  const int lo = __builtin_amdgcn_ds_bpermute(src_lane * 4, __double2loint(v));
  const int hi = __builtin_amdgcn_ds_bpermute(src_lane * 4, __double2hiint(v));
  return __hiloint2double(hi, lo);
}

struct BandDiag {
  Rsrc px, py, meta, out;  // [D, S] of the utterance
  int S, Dn;               // Dn = T_n + U_n diagonals
};

// Slot s of diagonal d (start diagonal e = d - s >= 0; slots with e < 0 are
// never written and read as invalid).
DEV void band_load(const BandDiag& v, int d, int lane, bool live, DiagT& x, DiagT& y, uint32_t& m) {
  const bool in = live && d >= lane && d < v.Dn;
  const uint32_t cell = (uint32_t)(d * v.S + lane);
  x = diag_load(v.px, in ? cell * (uint32_t)sizeof(DiagT) : kOob);
  y = diag_load(v.py, in ? cell * (uint32_t)sizeof(DiagT) : kOob);
  m = __builtin_amdgcn_raw_buffer_load_b32(v.meta, (int)(in ? cell * 4u : kOob), 0, 0);  // 0 (invalid) out of range
}

DEV void band_alpha(const BandDiag& v, int lane) {
  const bool live = lane < v.S;
  double hout = kNegInfD, vout = kNegInfD;
  DiagT xr[kBandPrefetch], yr[kBandPrefetch];
  uint32_t mr[kBandPrefetch];
#pragma unroll
  for (int k = 0; k < kBandPrefetch; ++k) band_load(v, k, lane, live, xr[k], yr[k], mr[k]);
  // drained once, so that the loop's wait counts cover only its own loads,
  // a whole ring old
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  for (int d0 = 0; d0 < v.Dn; d0 += kBandPrefetch) {
#pragma unroll
    for (int k = 0; k < kBandPrefetch; ++k) {
      const int d = d0 + k;
      const uint32_t m = mr[k];
      const bool act = (m & kValid) != 0;
      const int da = (int)(m & 0xffu);
      // horizontal: slot s + delta_t of the previous diagonal; vertical: slot s-1
      const int src = (da == kNoShift) ? lane : min(lane + da, 63);
      const double hin0 = bpermute_d(hout, src);
      const double vin = dpp_move_d<kDppWaveShr1>(vout, kNegInfD);
      const double hin = (da == kNoShift) ? kNegInfD : hin0;
      const double al = (d == 0) ? 0.0 : log2add(hin, vin);
      buf_store_f64(v.out, act ? (uint32_t)(d * v.S + lane) * 8u : kOob, al);
      hout = act ? al + (double)yr[k] : kNegInfD;
      vout = act ? al + (double)xr[k] : kNegInfD;
      band_load(v, d + kBandPrefetch, lane, live, xr[k], yr[k], mr[k]);
    }
  }
}

DEV void band_beta(const BandDiag& v, int lane) {
  const bool live = lane < v.S;
  double bout = kNegInfD;
  DiagT xr[kBandPrefetch], yr[kBandPrefetch];
  uint32_t mr[kBandPrefetch];
#pragma unroll
  for (int k = 0; k < kBandPrefetch; ++k) band_load(v, v.Dn - 1 - k, lane, live, xr[k], yr[k], mr[k]);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  for (int d0 = v.Dn - 1; d0 >= 0; d0 -= kBandPrefetch) {
#pragma unroll
    for (int k = 0; k < kBandPrefetch; ++k) {
      const int d = d0 - k;
      const uint32_t m = mr[k];
      const bool act = (m & kValid) != 0;
      const int db = (int)((m >> 8) & 0xffu);
      // horizontal successor: slot s - delta_{t+1} of the next diagonal; vertical: slot s+1
      const int src = (db >= kEndNode) ? lane : max(lane - db, 0);
      const double h0 = bpermute_d(bout, src);
      const double vn = dpp_move_d<kDppWaveShl1>(bout, kNegInfD);
      const double hin = (db == kEndNode) ? 0.0 : ((db == kNoShift || lane - db < 0) ? kNegInfD : h0);
      const double be = log2add((double)yr[k] + hin, (double)xr[k] + vn);
      buf_store_f64(v.out, act ? (uint32_t)(d * v.S + lane) * 8u : kOob, be);
      bout = act ? be : kNegInfD;
      band_load(v, d - kBandPrefetch, lane, live, xr[k], yr[k], mr[k]);
    }
  }
}

__global__ __launch_bounds__(kBandThreads) void band_fb_kernel(BandArgs a) {
  const int n = blockIdx.x;
  const int S = a.S, D = a.D;  // W == S on this path
  int Tn, Un;
  const bool ok = utt_dims(a.b, n, Tn, Un);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: the resources stay scalar
  const size_t base = (size_t)n * D * S;
  const size_t cells = (size_t)D * S;
  BandDiag v;
  v.px = make_rsrc(a.pxd + base, cells * sizeof(DiagT));
  v.py = make_rsrc(a.pyd + base, cells * sizeof(DiagT));
  v.meta = make_rsrc(a.meta + base, cells * sizeof(uint32_t));
  v.S = S;
  v.Dn = Tn + Un;
  if (wave == 0) {
    v.out = make_rsrc(a.alpha + base, cells * sizeof(double));
    band_alpha(v, lane);
  } else {
    v.out = make_rsrc(a.beta + base, cells * sizeof(double));
    band_beta(v, lane);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int pl = band_p(a, n, Tn - 1, Un);
    const int se = Un - pl;  // slot of the final node (T_n-1, U_n), if the band holds it
    double L = kNegInfD;
    if (se >= 0 && se < S) {
      const size_t o = base + (size_t)(Tn - 1 + Un) * S + se;
      L = a.alpha[o] + (double)a.pyd[o];
    }
    const double L2 = ok ? L : __builtin_nan("");
    a.Lutt[n] = L2;
    a.loss[n] = (L2 == L2) ? (float)(-L2 * kLn2) : __builtin_nanf("");
  }
}

// Slot of node (t, u = p + s) on its diagonal.
DEV int band_slot(const BandArgs& a, int u, int s) { return a.masked ? u : s; }

__global__ __launch_bounds__(256) void band_occ_kernel(BandArgs a) {
  const int T = a.b.T, S = a.S, D = a.D, W = a.W;
  const int lane = threadIdx.x & 63;
  const int f = blockIdx.x * 4 + (threadIdx.x >> 6);  // frame over N*T
  if (f >= a.b.N * T) return;
  const int n = f / T, t = f - n * T;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const double Lu = a.Lutt[n];
  const bool live = (Lu == Lu) && (Lu != kNegInfD) && t < Tn;
  const int s = lane;
  const size_t base = (size_t)n * D * W;
  double ey = kNegInfD, ex = kNegInfD;
  if (live && s < S) {
    const int p = band_p(a, n, t, Un);
    const int u = p + s;
    if (u <= Un) {
      const size_t k = (size_t)f * S + s;
      const int d = t + p + s;
      const double al = a.alpha[base + (size_t)d * W + band_slot(a, u, s)];
      double nb;
      if (t + 1 < Tn) {
        const int s2 = u - band_p(a, n, t + 1, Un);  // slot of (t+1, u), on diagonal d+1
        nb = (s2 >= 0 && s2 < S) ? a.beta[base + (size_t)(d + 1) * W + band_slot(a, u, s2)] : kNegInfD;
      } else {
        nb = (u == Un) ? 0.0 : kNegInfD;
      }
      ey = al + (double)a.py[k] * kLog2e + nb;
      if (s + 1 < S && u + 1 <= Un)
        ex = al + (double)a.px[k] * kLog2e + a.beta[base + (size_t)(d + 1) * W + band_slot(a, u + 1, s + 1)];
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

bool band_masked(int U, int S) {
  (void)S;
  return U + 1 <= 64;
}

int band_slots(int U, int S) { return band_masked(U, S) ? 64 : S; }

int band_diagonals(int T, int U, int S) {
  // every node (t, u) with t < T, u <= U lies on a diagonal below T + U,
  // whatever the bounds (they are clamped to [0, U_n] but not trusted beyond)
  (void)S;
  return T + U;
}

hipError_t launch_band(const BandArgs& a, hipStream_t s) {
  if (a.masked) {
    {
      RNNT_PROF(s, "band_prep");
      const size_t cells = (size_t)a.b.N * a.D * 64;
      hipLaunchKernelGGL(band_mask_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s, a);
    }
    SimpleArgs l{};
    l.b = a.b;
    l.V = 0;  // the symbols were checked by the joiner
    l.pxd = a.pxd;
    l.pyd = a.pyd;
    l.alpha = a.alpha;
    l.beta = a.beta;
    l.Lutt = a.Lutt;
    l.loss = a.loss;
    const hipError_t e = launch_lattice_recursion(l, s);
    if (e != hipSuccess) return e;
  } else {
    {
      RNNT_PROF(s, "band_prep");
      hipLaunchKernelGGL(band_prep_kernel, dim3((a.b.N * a.b.T + 255) / 256), dim3(256), 0, s, a);
    }
    RNNT_PROF(s, "band_fb");
    hipLaunchKernelGGL(band_fb_kernel, dim3(a.b.N), dim3(kBandThreads), 0, s, a);
  }
  if (a.gx || a.gy) {
    RNNT_PROF(s, "band_occ");
    hipLaunchKernelGGL(band_occ_kernel, dim3((a.b.N * a.b.T + 3) / 4), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}
