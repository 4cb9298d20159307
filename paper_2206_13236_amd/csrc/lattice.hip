// Stage 2: forward-backward over the full T x (U+1) lattice of the trivial
// joiner (Sec. 2, Eq. (3)), and the occupation counts of Sec. 3.2.2
// (derivatives of the total log-prob w.r.t. px = y(t,u) and py = blank(t,u)).
//
// lattice_fb_kernel: one workgroup per utterance. Wave 0 runs the forward
// recursion (alpha) and wave 1 the backward recursion (beta) at the same time,
// both along anti-diagonals d = t + u: every node of diagonal d depends only
// on nodes of diagonal d-1 (d+1 for beta), so a wave updates a whole diagonal
// per step. Lane l owns the rows u in [l*R, l*R + R); the only cross-lane
// value per step is the neighbouring row's output, moved by one DPP wave
// shift. The px/py loads of each row's node are issued P diagonals ahead.
// The recursion reads copies of px, py and writes alpha, beta in the
// diagonal-major layout described in kernels.h, so that every load and
// store of a step is contiguous across the wave.
//
// lattice_occ_kernel: one wave per frame over the whole batch. Every complete
// path leaves frame t through exactly one blank edge (t,u) -> (t+1,u) (the
// final blank at t = T-1), so
//   L = log2 sum_u 2^(alpha(t,u) + blank(t,u) + beta(t+1,u))   for every t.
// The occupations of frame t are normalised by that frame's own sum, which
// cancels the rounding the alpha and beta chains accumulate in common. The
// kernel also writes W(t,u) = (gx + gy) e^{m_a + m_l - Z} for the gradient,
// the row sums of gx and gy and per-16-frame partial column sums of gx and gy.
//
// Precision: log2 domain with fp64 accumulators; only the bounded correction
// term of LogAdd goes through fp32 exp2/log2 (see lse2). alpha and beta are
// stored in fp64.
// A NaN px or py at a node of the lattice is flagged on the side and makes
// the utterance's loss NaN, like an out-of-range length or symbol.
#include "kernels.h"
#include "prof.h"

namespace {

constexpr int kOccFrames = 16;  // frames (waves) per workgroup of the occupation kernel

// The recursion loops are kept free of branches, selects and 64-bit address
// arithmetic. px, py (fp64, log2 units) and alpha/beta of the utterance are
// buffer resources over the diagonal-major layout [D, W], so the lane's row r
// of diagonal d sits at d*W + r*64 + lane and every load and store of a step
// is contiguous across the wave. Every cell that is no node of the utterance
// holds -inf in px and py, so a node outside the lattice needs no test:
//   alpha: a node at t < 0 has only such nodes before it and stays -inf; a
//          node at t >= T_n or u > U_n may take a finite value, but both of
//          its outgoing sums add its own -inf inputs, so nothing reaches a
//          node of the lattice from it;
//   beta:  every such node gets -inf (both of its terms add its own -inf
//          inputs), except the virtual node (T_n, U_n) after the final
//          blank, which is the initial value 0.
// Their stored values land in cells that no reader takes. Diagonals beyond
// the layout (the idle steps at the end of a loop) have byte offsets at or
// past the resource's size, negative ones included after the unsigned
// conversion: their loads read 0 and their stores are dropped.
struct LatView {
  Rsrc px, py, out;  // pxd, pyd (DiagT) and alpha or beta (f64) of the utterance, [D, W]
  int Tn, Un, W;
};

template <int R>
DEV void lattice_load(const LatView& v, int d, int lane, DiagT (&x)[R], DiagT (&y)[R]) {
  const int dW = d * v.W + lane;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t off = (uint32_t)(dW + r * 64) * (uint32_t)sizeof(DiagT);
    x[r] = diag_load(v.px, off);
    y[r] = diag_load(v.py, off);
  }
}

// A NaN among the inputs of a step is flagged in `bad` rather than carried
// through the recursion.
template <int R>
DEV void lattice_check(const DiagT (&x)[R], const DiagT (&y)[R], bool& bad) {
#pragma unroll
  for (int r = 0; r < R; ++r) bad |= __builtin_isunordered(x[r], y[r]);
}

// log2(2^a + 2^b) for the recursions: the bounded correction
// log2(1 + 2^-|a-b|) through the fp32 hardware exp2/log2. The difference is
// formed directly, so that only the sum's own max waits for both inputs
// beside it; a NaN difference (two -inf inputs, or a NaN input, which is
// flagged on the side) is clamped to 0, so that two -inf give -inf + 1.
DEV double lse2(double a, double b) {
  const double mx = __builtin_fmax(a, b);
  const float d = __builtin_fminf((float)(-__builtin_fabs(a - b)), 0.0f);
  return mx + (double)__builtin_amdgcn_logf(1.0f + __builtin_amdgcn_exp2f(d));
}

// Returns whether this lane saw a NaN input.
template <int R, int P>
DEV bool alpha_pass(const LatView& v, int lane) {
  const int D = v.Tn + v.Un;  // diagonals 0 .. Tn-1+Un (the loop may run up to P-1 idle steps past them)
  // alpha(0, 0) = 0 comes out of the first step as LogAdd(0, -inf)
  double hout[R], vout[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    hout[r] = (lane * R + r == 0) ? 0.0 : kNegInfD;
    vout[r] = kNegInfD;
  }
  // The symbol term into row 0 comes from the lane below by one DPP wave
  // shift whose destination is carried from step to step: lane 0 receives
  // nothing and keeps the -inf it starts with, so that no step resets it.
  double vsh = kNegInfD;
  bool bad = false;
  DiagT xr[P][R], yr[P][R];  // converted at use, not at load
#pragma unroll
  for (int k = 0; k < P; ++k) lattice_load<R>(v, k, lane, xr[k], yr[k]);
  // The loop's wait counts then cover only the loads of its own steps, a
  // whole ring old, rather than the order the loads above were issued in.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  for (int d0 = 0; d0 < D; d0 += P) {
#pragma unroll
    for (int k = 0; k < P; ++k) {
      const int d = d0 + k;
      const int dW = d * v.W + lane;
      vsh = dpp_move_d<kDppWaveShr1>(vout[R - 1], vsh);
      double nh[R], nv[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const double vin = (r == 0) ? vsh : vout[r - 1];
        const double al = lse2(hout[r], vin);
        nh[r] = al + (double)yr[k][r];
        nv[r] = al + (double)xr[k][r];
        buf_store_f64(v.out, (uint32_t)(dW + r * 64) * 8u, al);
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        hout[r] = nh[r];
        vout[r] = nv[r];
      }
      lattice_check<R>(xr[k], yr[k], bad);
      lattice_load<R>(v, d + P, lane, xr[k], yr[k]);
      // no later step's work is hoisted into this one, where it would wait
      // for loads issued a step ago
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  return bad;
}

template <int R, int P>
DEV bool beta_pass(const LatView& v, int lane) {
  const int D = v.Tn + v.Un;
  // beta of my rows on the previous (higher) diagonal; the virtual node
  // (Tn, Un) after the final blank has beta = 0.
  double bprev[R];
#pragma unroll
  for (int r = 0; r < R; ++r) bprev[r] = (lane * R + r == v.Un) ? 0.0 : kNegInfD;
  double vsh = kNegInfD;  // lane 63 receives nothing from the shift and keeps -inf
  bool bad = false;
  DiagT xr[P][R], yr[P][R];  // converted at use, not at load
#pragma unroll
  for (int k = 0; k < P; ++k) lattice_load<R>(v, D - 1 - k, lane, xr[k], yr[k]);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), as in the forward pass
  for (int d0 = D - 1; d0 >= 0; d0 -= P) {
#pragma unroll
    for (int k = 0; k < P; ++k) {
      const int d = d0 - k;
      const int dW = d * v.W + lane;
      vsh = dpp_move_d<kDppWaveShl1>(bprev[0], vsh);
      double nb[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const double vin = (r == R - 1) ? vsh : bprev[r + 1];
        nb[r] = lse2((double)yr[k][r] + bprev[r], (double)xr[k][r] + vin);
        buf_store_f64(v.out, (uint32_t)(dW + r * 64) * 8u, nb[r]);
      }
#pragma unroll
      for (int r = 0; r < R; ++r) bprev[r] = nb[r];
      lattice_check<R>(xr[k], yr[k], bad);
      lattice_load<R>(v, d - P, lane, xr[k], yr[k]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  return bad;
}

template <int R, int P>
__global__ __launch_bounds__(128) void lattice_fb_kernel(SimpleArgs a) {
  const int n = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the resources stay scalar
  const int T = a.b.T, U1 = a.b.U + 1;
  int Tn, Un;
  const bool ok = utt_dims(a.b, n, Tn, Un);
  const int W = 64 * R;
  const size_t cells = (size_t)(T + U1 - 1) * W;
  const size_t base = (size_t)n * cells;
  LatView v;
  v.px = make_rsrc(a.pxd + base, cells * sizeof(DiagT));
  v.py = make_rsrc(a.pyd + base, cells * sizeof(DiagT));
  v.Tn = Tn;
  v.Un = Un;
  v.W = W;
  bool bad;
  if (wave == 0) {
    v.out = make_rsrc(a.alpha + base, cells * sizeof(double));
    bad = alpha_pass<R, P>(v, lane);
  } else {
    v.out = make_rsrc(a.beta + base, cells * sizeof(double));
    bad = beta_pass<R, P>(v, lane);
  }
  // symbols outside [0, V) make the utterance invalid (V = 0: not checked here);
  // each thread checks a strided share of them
  bool sok = true;
  if (a.V > 0)
    for (int u = tid; u < Un; u += blockDim.x) symbol_at(a.b, n, u, a.V, sok);
  const bool sbad = __syncthreads_or(!sok || bad) != 0;  // or a NaN input
  if (tid == 0) {
    const size_t last = base + (size_t)(Tn - 1 + Un) * W + lattice_slot(Un, R);
    const double L = a.alpha[last] + (double)a.pyd[last];
    const double L2 = (ok && !sbad) ? L : __builtin_nan("");
    a.Lutt[n] = L2;
    a.loss[n] = (L2 == L2) ? (float)(-L2 * kLn2) : __builtin_nanf("");
  }
}

// px, py [N, T, U+1] -> the diagonal-major copies in log2 units (for
// producers that do not write them directly): one thread per node of the
// rectangle, then one per cell of the copies, which take -inf where no node
// of the utterance lies.
__global__ __launch_bounds__(256) void lattice_diag_copy_kernel(SimpleArgs a, int R) {
  const int T = a.b.T, U1 = a.b.U + 1;
  const size_t L = (size_t)a.b.N * T * U1;
  const int rect_blocks = (int)((L + 255) / 256);  // blocks of 256 threads
  if ((int)blockIdx.x >= rect_blocks) {
    lattice_fill_outside(a.pxd, a.pyd, (int)blockIdx.x - rect_blocks, threadIdx.x, 256, T, U1, R);
    return;
  }
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= L) return;
  const int n = (int)(i / ((size_t)T * U1));
  const int rem = (int)(i - (size_t)n * T * U1);
  const int t = rem / U1, u = rem - t * U1;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const bool node = t < Tn && u <= Un;
  const size_t o = (size_t)n * (T + U1 - 1) * 64 * R + (size_t)(t + u) * 64 * R + lattice_slot(u, R);
  a.pxd[o] = (DiagT)((node && u < Un) ? (double)a.px[i] * kLog2e : kNegInfD);
  a.pyd[o] = (DiagT)(node ? (double)a.py[i] * kLog2e : kNegInfD);
}

template <int R>
__global__ __launch_bounds__(64 * kOccFrames) void lattice_occ_kernel(SimpleArgs a) {
  __shared__ double sx[kOccFrames][64], sy[kOccFrames][64];
  const int n = blockIdx.y, blk = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int T = a.b.T, U1 = a.b.U + 1;
  const int t = blk * kOccFrames + wave;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const double Lu = a.Lutt[n];
  const bool frow = (Lu == Lu) && (Lu != kNegInfD) && t < Tn;
  const size_t base = (size_t)n * T * U1;
  const int W = 64 * R;
  const double* alpha = a.alpha + (size_t)n * (T + U1 - 1) * W;
  const double* beta = a.beta + (size_t)n * (T + U1 - 1) * W;
  const float* px = a.px + base;
  const float* py = a.py + base;
  // log2-domain weights of the frame's blank edges (ey) and vertical edges (ex)
  double ey[R], ex[R];
  double mx = kNegInfD;
#pragma unroll
  for (int c = 0; c < R; ++c) {
    const int u = c * 64 + lane;
    const bool on = frow && u <= Un;
    const size_t idx = on ? (size_t)t * U1 + u : 0;
    ey[c] = ex[c] = kNegInfD;
    if (on) {
      const size_t dg = (size_t)(t + u) * W;  // diagonal of (t, u); (t+1, u) and (t, u+1) lie on the next
      const double al = alpha[dg + lattice_slot(u, R)];
      const double nb = (t + 1 < Tn) ? beta[dg + W + lattice_slot(u, R)] : (u == Un ? 0.0 : kNegInfD);
      ey[c] = al + (double)py[idx] * kLog2e + nb;
      if (u < Un) ex[c] = al + (double)px[idx] * kLog2e + beta[dg + W + lattice_slot(u + 1, R)];
    }
    mx = ey[c] > mx ? ey[c] : mx;
  }
  mx = wave_max_d(mx);
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < R; ++c) s += (ey[c] != kNegInfD) ? (double)exp2f((float)(ey[c] - mx)) : 0.0;
  s = wave_sum_d(s);
  const double Lt = mx + log2(s);
  const bool trow = t < T;
  const float mat = (frow && a.Wt) ? a.m_a[(size_t)n * T + t] : 0.f;
  double ry = 0.0, rx = 0.0;
#pragma unroll
  for (int c = 0; c < R; ++c) {
    const int u = c * 64 + lane;
    float gxv = 0.f, gyv = 0.f;
    if (frow && u <= Un) {
      gxv = exp2_occ(ex[c] - Lt);
      gyv = exp2_occ(ey[c] - Lt);
    }
    if (trow && u < U1) {
      const size_t idx = base + (size_t)t * U1 + u;
      a.gx[idx] = gxv;
      a.gy[idx] = gyv;
      if (a.Wt)
        a.Wt[((size_t)n * T + t) * a.ldw + u] =
            (frow && u <= Un) ? (gxv + gyv) * expf(mat + a.m_l[(size_t)n * U1 + u] - a.Z[idx]) : 0.f;
    }
    ry += (double)gyv;
    rx += (double)gxv;
    {
      sx[wave][lane] = (double)gxv;
      sy[wave][lane] = (double)gyv;
      __syncthreads();
      if (wave == 0 && u < U1) {
        double cx = 0.0, cy = 0.0;
        for (int w = 0; w < kOccFrames; ++w) {
          cx += sx[w][lane];
          cy += sy[w][lane];
        }
        const size_t pi = ((size_t)n * a.ncolblk + blk) * U1 + u;
        a.cpx[pi] = cx;
        a.cpy[pi] = cy;
      }
      __syncthreads();
    }
  }
  if (trow) {
    if (a.Wt && lane < a.ldw - U1) a.Wt[((size_t)n * T + t) * a.ldw + U1 + lane] = 0.f;
    ry = wave_sum_d(ry);
    rx = wave_sum_d(rx);
    if (lane == 0) {
      a.ry[(size_t)n * T + t] = ry;
      a.rx[(size_t)n * T + t] = rx;
    }
  }
}

template <int R, int P>
void launch_lattice_r(const SimpleArgs& a, hipStream_t s) {
  {
    RNNT_PROF(s, "lattice_fb");
    hipLaunchKernelGGL((lattice_fb_kernel<R, P>), dim3(a.b.N), dim3(128), 0, s, a);
  }
  {
    RNNT_PROF(s, "lattice_occ");
    hipLaunchKernelGGL((lattice_occ_kernel<R>), dim3(a.ncolblk, a.b.N), dim3(64 * kOccFrames), 0, s, a);
  }
}

}  // namespace

int lattice_colblocks(int T) { return (T + kOccFrames - 1) / kOccFrames; }

int lattice_rows_per_lane(int U1) {
  const int need = (U1 + 63) / 64;
  return need <= 6 ? (need < 1 ? 1 : need) : need <= 8 ? 8 : need <= 12 ? 12 : 16;
}

hipError_t launch_lattice_diag_copy(const SimpleArgs& a, hipStream_t s) {
  const size_t blocks =
      ((size_t)a.b.N * a.b.T * (a.b.U + 1) + 255) / 256 + (size_t)a.b.N * lattice_fill_blocks(a.b.T, a.b.U, 256);
  {
    RNNT_PROF(s, "lattice_diag_copy");
    hipLaunchKernelGGL(lattice_diag_copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a,
                       lattice_rows_per_lane(a.b.U + 1));
  }
  return hipGetLastError();
}

hipError_t launch_lattice_recursion(const SimpleArgs& a, hipStream_t s) {
  if (a.b.U + 1 > 64 * 16) return hipErrorInvalidValue;
  RNNT_PROF(s, "band_fb");
  switch (lattice_rows_per_lane(a.b.U + 1)) {
    case 1: hipLaunchKernelGGL((lattice_fb_kernel<1, 8>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 2: hipLaunchKernelGGL((lattice_fb_kernel<2, 8>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 3: hipLaunchKernelGGL((lattice_fb_kernel<3, 8>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 4: hipLaunchKernelGGL((lattice_fb_kernel<4, 8>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 5: hipLaunchKernelGGL((lattice_fb_kernel<5, 6>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 6: hipLaunchKernelGGL((lattice_fb_kernel<6, 5>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 8: hipLaunchKernelGGL((lattice_fb_kernel<8, 4>), dim3(a.b.N), dim3(128), 0, s, a); break;
    case 12: hipLaunchKernelGGL((lattice_fb_kernel<12, 3>), dim3(a.b.N), dim3(128), 0, s, a); break;
    default: hipLaunchKernelGGL((lattice_fb_kernel<16, 2>), dim3(a.b.N), dim3(128), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_lattice(const SimpleArgs& a, hipStream_t s) {
  const int U1 = a.b.U + 1;
  if (U1 > 64 * 16) return hipErrorInvalidValue;
  switch (lattice_rows_per_lane(U1)) {
    case 1: launch_lattice_r<1, 8>(a, s); break;
    case 2: launch_lattice_r<2, 8>(a, s); break;
    case 3: launch_lattice_r<3, 8>(a, s); break;
    case 4: launch_lattice_r<4, 8>(a, s); break;
    case 5: launch_lattice_r<5, 6>(a, s); break;
    case 6: launch_lattice_r<6, 5>(a, s); break;
    case 8: launch_lattice_r<8, 4>(a, s); break;
    case 12: launch_lattice_r<12, 3>(a, s); break;
    default: launch_lattice_r<16, 2>(a, s); break;
  }
  return hipGetLastError();
}
