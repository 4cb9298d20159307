// Stage 2: forward-backward over the full T x (U+1) lattice of the trivial
// joiner (Sec. 2, Eq. (3)), and the occupation counts of Sec. 3.2.2
// (derivatives of the total log-prob w.r.t. px = y(t,u) and py = blank(t,u)).
//
// One workgroup per utterance. Wave 0 runs the forward recursion (alpha) and
// wave 1 the backward recursion (beta) at the same time, both along
// anti-diagonals d = t + u: every node of diagonal d depends only on nodes of
// diagonal d-1 (d+1 for beta), so a wave updates a whole diagonal per step.
// Lane l owns the rows u in [l*R, l*R + R); the only cross-lane value per step
// is the neighbouring row's output (one shuffle). The px/py loads of each
// row's node are issued P diagonals ahead. After both waves finish, all 16
// waves compute the occupations, the loss, and the helper arrays of the
// simple-loss gradient.
//
// Precision: the recursions run in the log2 domain with fp64 accumulators;
// only the bounded correction term of LogAdd goes through fp32 exp2/log2
// (see log2add). alpha and beta are stored in fp64.
#include "kernels.h"
#include "prof.h"

namespace {

constexpr int kLatThreads = 1024;

template <int R, int P>
DEV void lattice_load(const float* __restrict__ px, const float* __restrict__ py, int d, int lane, int Tn,
                      int Un, int U1, float (&x)[R], float (&y)[R]) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int u = lane * R + r, t = d - u;
    const bool act = (t >= 0) && (t < Tn) && (u <= Un);
    const size_t idx = act ? (size_t)t * U1 + u : 0;
    x[r] = act ? px[idx] : 0.f;
    y[r] = act ? py[idx] : 0.f;
  }
}

template <int R, int P>
DEV void alpha_pass(const float* __restrict__ px, const float* __restrict__ py, double* __restrict__ alpha,
                    int Tn, int Un, int U1, int lane) {
  const int D = Tn + Un;  // diagonals 0 .. Tn-1+Un
  double hout[R], vout[R];
#pragma unroll
  for (int r = 0; r < R; ++r) hout[r] = vout[r] = kNegInfD;
  float xr[P][R], yr[P][R];
#pragma unroll
  for (int k = 0; k < P; ++k) lattice_load<R, P>(px, py, k, lane, Tn, Un, U1, xr[k], yr[k]);
  for (int d0 = 0; d0 < D; d0 += P) {
#pragma unroll
    for (int k = 0; k < P; ++k) {
      const int d = d0 + k;
      if (d < D) {
        double vfirst = shfl_up_d(vout[R - 1], 1);
        if (lane == 0) vfirst = kNegInfD;
        double nh[R], nv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int u = lane * R + r, t = d - u;
          const bool act = (t >= 0) && (t < Tn) && (u <= Un);
          const double vin = (r == 0) ? vfirst : vout[r - 1];
          double al = (d == 0) ? 0.0 : log2add(hout[r], vin);
          if (act) {
            nh[r] = al + (double)yr[k][r] * kLog2e;
            nv[r] = al + (double)xr[k][r] * kLog2e;
            alpha[(size_t)t * U1 + u] = al;
          } else {
            nh[r] = kNegInfD;
            nv[r] = kNegInfD;
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          hout[r] = nh[r];
          vout[r] = nv[r];
        }
        lattice_load<R, P>(px, py, d + P, lane, Tn, Un, U1, xr[k], yr[k]);
      }
    }
  }
}

template <int R, int P>
DEV void beta_pass(const float* __restrict__ px, const float* __restrict__ py, double* __restrict__ beta,
                   int Tn, int Un, int U1, int lane) {
  const int D = Tn + Un;
  // beta of my rows on the previous (higher) diagonal; the virtual node
  // (Tn, Un) after the final blank has beta = 0.
  double bprev[R];
#pragma unroll
  for (int r = 0; r < R; ++r) bprev[r] = (lane * R + r == Un) ? 0.0 : kNegInfD;
  float xr[P][R], yr[P][R];
#pragma unroll
  for (int k = 0; k < P; ++k) lattice_load<R, P>(px, py, D - 1 - k, lane, Tn, Un, U1, xr[k], yr[k]);
  for (int d0 = D - 1; d0 >= 0; d0 -= P) {
#pragma unroll
    for (int k = 0; k < P; ++k) {
      const int d = d0 - k;
      if (d >= 0) {
        double vlast = shfl_down_d(bprev[0], 1);
        if (lane == 63) vlast = kNegInfD;
        double nb[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const int u = lane * R + r, t = d - u;
          const bool act = (t >= 0) && (t < Tn) && (u <= Un);
          const double vin = (r == R - 1) ? vlast : bprev[r + 1];
          if (act) {
            const double be = log2add((double)yr[k][r] * kLog2e + bprev[r], (double)xr[k][r] * kLog2e + vin);
            nb[r] = be;
            beta[(size_t)t * U1 + u] = be;
          } else {
            nb[r] = kNegInfD;
          }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) bprev[r] = nb[r];
        lattice_load<R, P>(px, py, d - P, lane, Tn, Un, U1, xr[k], yr[k]);
      }
    }
  }
}

template <int R, int P>
__global__ __launch_bounds__(kLatThreads) void lattice_kernel(SimpleArgs a) {
  __shared__ double red[2 * kLatThreads];
  __shared__ double sL;
  const int n = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.b.T, U1 = a.b.U + 1;
  int Tn, Un;
  bool ok = utt_dims(a.b, n, Tn, Un);
  const size_t base = (size_t)n * T * U1;
  const float* px = a.px + base;
  const float* py = a.py + base;
  double* alpha = a.alpha + base;
  double* beta = a.beta + base;

  if (wave == 0) alpha_pass<R, P>(px, py, alpha, Tn, Un, U1, lane);
  else if (wave == 1) beta_pass<R, P>(px, py, beta, Tn, Un, U1, lane);
  __syncthreads();
  if (tid == 0) {
    // symbols outside [0, V) make the utterance invalid
    bool sok = true;
    for (int u = 0; u < Un; ++u) symbol_at(a.b, n, u, a.V, sok);
    const double L = alpha[(size_t)(Tn - 1) * U1 + Un] + (double)py[(size_t)(Tn - 1) * U1 + Un] * kLog2e;
    sL = (ok && sok) ? L : __builtin_nan("");
  }
  __syncthreads();
  const double L2 = sL;
  const bool live = (L2 == L2) && (L2 != kNegInfD);
  if (tid == 0) a.loss[n] = (L2 == L2) ? (float)(-L2 * kLn2) : __builtin_nanf("");

  // Every complete path crosses each anti-diagonal d = t + u at exactly one
  // node, so L = log2 sum_{t+u=d} 2^(alpha + beta) for every d. Normalising
  // the occupations of the edges leaving diagonal d by that diagonal's own
  // sum cancels the rounding that alpha and beta accumulate along their
  // chains (their common part), which otherwise scales all occupations alike.
  double* Ld = a.Ldiag + (size_t)n * (T + U1);
  const int D = Tn + Un;
  if (live) {
    for (int d = wave; d < D; d += kLatThreads / 64) {
      double v[R];
      double mx = kNegInfD;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int u = lane * R + r, t = d - u;
        const bool on = (t >= 0) && (t < Tn) && (u <= Un);
        const size_t i = on ? (size_t)t * U1 + u : 0;
        v[r] = on ? alpha[i] + beta[i] : kNegInfD;
        mx = v[r] > mx ? v[r] : mx;
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const double o = __shfl_xor(mx, off, 64);
        mx = o > mx ? o : mx;
      }
      double s = 0.0;
#pragma unroll
      for (int r = 0; r < R; ++r) s += (v[r] != kNegInfD) ? (double)exp2f((float)(v[r] - mx)) : 0.0;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
      if (lane == 0) Ld[d] = mx + log2(s);
    }
  }
  __syncthreads();

  const float* ma = a.m_a + (size_t)n * T;
  const float* ml = a.m_l + (size_t)n * U1;
  float* gx = a.gx + base;
  float* gy = a.gy + base;
  float* Wt = a.want_bwd ? a.Wt + (size_t)n * T * a.ldw : nullptr;
  // Occupations, one frame per wave and lanes across u (coalesced). The row
  // sums of gy (blank column of d am) are wave reductions; the column sums of
  // gx and gy (target and blank columns of d lm) stay in fp64 registers per
  // lane and are added across waves in a fixed order.
  constexpr int NW = kLatThreads / 64;
  double cxa[R], cya[R];
#pragma unroll
  for (int c = 0; c < R; ++c) cxa[c] = cya[c] = 0.0;
  for (int t = wave; t < T; t += NW) {
    double rs = 0.0;
    const bool trow = live && t < Tn;
    const float mat = trow ? ma[t] : 0.f;
#pragma unroll
    for (int c = 0; c < R; ++c) {
      const int u = c * 64 + lane;
      if (u >= U1) continue;
      const size_t idx = (size_t)t * U1 + u;
      float gxv = 0.f, gyv = 0.f;
      const bool on = trow && u <= Un;
      if (on) {
        const double al = alpha[idx];
        const double Lt = Ld[t + u];
        if (u < Un) gxv = exp2_occ(al + (double)px[idx] * kLog2e + beta[idx + 1] - Lt);
        const double nb = (t + 1 < Tn) ? beta[idx + U1] : (u == Un ? 0.0 : kNegInfD);
        gyv = exp2_occ(al + (double)py[idx] * kLog2e + nb - Lt);
      }
      gx[idx] = gxv;
      gy[idx] = gyv;
      if (Wt) {
        Wt[(size_t)t * a.ldw + u] = on ? (gxv + gyv) * expf(mat + ml[u] - a.Z[base + idx]) : 0.f;
        rs += (double)gyv;
        cxa[c] += (double)gxv;
        cya[c] += (double)gyv;
      }
    }
    if (Wt) {
      if (lane < a.ldw - U1) Wt[(size_t)t * a.ldw + U1 + lane] = 0.f;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) rs += __shfl_xor(rs, off, 64);
      if (lane == 0) a.ry[(size_t)n * T + t] = rs;
    }
  }
  if (!a.want_bwd) return;
  for (int c = 0; c < R; ++c) {
    red[wave * 64 + lane] = cxa[c];
    red[kLatThreads + wave * 64 + lane] = cya[c];
    __syncthreads();
    const int u = c * 64 + tid;
    if (tid < 64 && u < U1) {
      double sx = 0.0, sy = 0.0;
      for (int w = 0; w < NW; ++w) {
        sx += red[w * 64 + tid];
        sy += red[kLatThreads + w * 64 + tid];
      }
      a.cx[(size_t)n * U1 + u] = sx;
      a.cy[(size_t)n * U1 + u] = sy;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_lattice(const SimpleArgs& a, hipStream_t s) {
  const int U1 = a.b.U + 1;
  const int need = (U1 + 63) / 64;
  dim3 grid(a.b.N), block(kLatThreads);
  RNNT_PROF(s, "lattice");
  if (need <= 1) hipLaunchKernelGGL((lattice_kernel<1, 8>), grid, block, 0, s, a);
  else if (need <= 2) hipLaunchKernelGGL((lattice_kernel<2, 8>), grid, block, 0, s, a);
  else if (need <= 4) hipLaunchKernelGGL((lattice_kernel<4, 4>), grid, block, 0, s, a);
  else if (need <= 8) hipLaunchKernelGGL((lattice_kernel<8, 2>), grid, block, 0, s, a);
  else if (need <= 16) hipLaunchKernelGGL((lattice_kernel<16, 2>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}
