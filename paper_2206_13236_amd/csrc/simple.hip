// Stage 1 of the pruned RNN-T loss: the trivial joiner of Sec. 3.1.
//
//   L_trivial(t,u,v) = am[t,v] + lm[u,v] - Z(t,u)               (Eq. (5))
//   Z(t,u) = log sum_v exp(am[t,v] + lm[u,v])                    (Eq. (6))
//
// Z is evaluated as the paper suggests, as an ordinary matrix product after
// applying offsets: with m_a[t] = max_v am[t,v] and m_l[u] = max_v lm[u,v],
//   Z(t,u) = m_a[t] + m_l[u] + log( sum_v e^{am[t,v]-m_a[t]} e^{lm[u,v]-m_l[u]} ),
// every factor is <= 1 so the product cannot overflow. The contraction over v
// runs on fp32 MFMA; the exponentials are formed while staging tiles to LDS
// and the px/py lookups (Eqs. (1)-(2)) are fused into the epilogue.
//
// The gradient w.r.t. am and lm (the simple loss is trained, Sec. 3.3) is two
// more contractions of the same shape:
//   d am[t,v] = sc (e^{am-m_a}[t,v] * sum_u W(t,u) e^{lm-m_l}[u,v]
//                   - sum_u gx(t,u) [v = y_{u+1}] - sum_u gy(t,u) [v = blank])
//   d lm[u,v] = sc (e^{lm-m_l}[u,v] * sum_t W(t,u) e^{am-m_a}[t,v]
//                   - sum_t gx(t,u) [v = y_{u+1}] - sum_t gy(t,u) [v = blank])
// with W(t,u) = (gx + gy)(t,u) e^{m_a + m_l - Z}: the log-softmax backward
// (gradient of the target/blank entries minus softmax times their sum).
//
// Smoothed joiner (Sec. 3.3.1), with weights a = a_lm, b = a_ac, c = 1-a-b:
//   L = c L_trivial + a L_lm + b L_acoustic,   L_lm(u,v) = lm[u,v] - Zlm[u],
//   L_acoustic(t,v) = am[t,v] + lavg[v] - Zac[t],
//   lavg[v] = log (1/(U+1)) sum_u e^{lm[u,v] - Zlm[u]},  Zlm, Zac row log-sum-exps.
// With Gx(u), Gy(u) the column sums and R(t) the row sums of gx + gy, and
// P_ac, P_lm the softmaxes of those joiners, the gradients gain
//   d am += b (R(t) P_ac[t,v] - sparse)       (sparse: the target/blank terms)
//   d lm += a ((Gx+Gy)(u) P_lm[u,v] - sparse) + b P_lm[u,v] (q[v] - s_u)
// where q[v] = g[v] / ((U+1) e^{lavg[v]}), g[v] = sum_t R(t) P_ac[t,v] - Sy(v)
// is the gradient w.r.t. lavg / b (Sy: target/blank column sums) and
// s_u = sum_v q[v] P_lm[u,v] (the chain rule through the average of softmaxes).
#include <float.h>

#include "gemm.h"
#include "kernels.h"
#include "prof.h"

namespace {

DEV float keep_nan_max(float m, float x) { return (x > m || x != x) ? x : m; }

// A workgroup barrier after this thread's LDS writes have completed. Unlike
// __syncthreads() it does not wait for outstanding global loads, so that the
// next step's loads stay in flight across it.
DEV void sg_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

DEV float4 buf_load_f4(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}


// Length of each of `splits` contiguous K ranges over [0, K), a multiple of bk.
DEV int split_chunk(int K, int splits, int bk) { return ((K + splits - 1) / splits + bk - 1) / bk * bk; }

// ---------------------------------------------------------------------------
// Row maxima of am (rows t < T_n) and lm (rows u <= U_n): one wave per row.
// ---------------------------------------------------------------------------
// One wave per row: rows [0, N*T) of am, then rows [0, N*(U+1)) of lm.
__global__ __launch_bounds__(256) void rowmax_kernel(const float* __restrict__ am, const float* __restrict__ lm,
                                                     int N, int T, int U1, int V, BatchDev b,
                                                     float* __restrict__ m_a, float* __restrict__ m_l) {
  const int gr = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (gr >= N * (T + U1)) return;
  const int is_lm = gr >= N * T;
  const int row = is_lm ? gr - N * T : gr;
  const int R = is_lm ? U1 : T;
  const float* x = is_lm ? lm : am;
  float* out = is_lm ? m_l : m_a;
  const int n = row / R, i = row % R;
  int Tn, Un;
  utt_dims(b, n, Tn, Un);
  const int lim = is_lm ? Un + 1 : Tn;
  if (i >= lim) {
    if (lane == 0) out[row] = 0.f;
    return;
  }
  const float* r = x + (size_t)row * V;
  float m = kNegInfF;
  if ((V & 3) == 0) {
    const float4* r4 = reinterpret_cast<const float4*>(r);
#pragma unroll 4
    for (int v = lane; v < V / 4; v += 64) {
      float4 q = r4[v];
      m = keep_nan_max(m, q.x);
      m = keep_nan_max(m, q.y);
      m = keep_nan_max(m, q.z);
      m = keep_nan_max(m, q.w);
    }
  } else {
#pragma unroll 4
    for (int v = lane; v < V; v += 64) m = keep_nan_max(m, r[v]);
  }
  // within each 16-lane row by DPP rotations, then across the rows
  m = keep_nan_max(m, dpp_row_ror<8>(m));
  m = keep_nan_max(m, dpp_row_ror<4>(m));
  m = keep_nan_max(m, dpp_row_ror<2>(m));
  m = keep_nan_max(m, dpp_row_ror<1>(m));
  m = keep_nan_max(m, __shfl_xor(m, 16, 64));
  m = keep_nan_max(m, __shfl_xor(m, 32, 64));
  if (lane == 0) out[row] = m;
}

// ---------------------------------------------------------------------------
// Smoothing statistics (Sec. 3.3.1), one utterance's rows at a time.
// ---------------------------------------------------------------------------
// Zlm[n,u] = m_l + log sum_v e^{lm[u,v] - m_l}: one wave per row u <= U_n.
__global__ __launch_bounds__(256) void lm_lse_kernel(SimpleArgs a) {
  const int U1 = a.b.U + 1, V = a.V;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= a.b.N * U1) return;
  const int n = row / U1, u = row - n * U1;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (u > Un) {
    if (lane == 0) a.Zlm[row] = 0.f;
    return;
  }
  const float* x = a.lm + (size_t)row * V;
  const float m = a.m_l[row];
  float sum = 0.f;
  for (int v = lane; v < V; v += 64) sum += expf(x[v] - m);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
  if (lane == 0) a.Zlm[row] = m + logf(sum);
}

// lavg[n,v] = log (1/(U_n+1)) sum_{u <= U_n} e^{lm[u,v] - Zlm[u]}: threads over v.
__global__ __launch_bounds__(256) void lm_avg_kernel(SimpleArgs a) {
  const int n = blockIdx.y, V = a.V, U1 = a.b.U + 1;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= V) return;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const float* lmn = a.lm + (size_t)n * U1 * V;
  const float* z = a.Zlm + (size_t)n * U1;
  float s = 0.f;
  for (int u = 0; u <= Un; ++u) s += expf(lmn[(size_t)u * V + v] - z[u]);
  a.lavg[(size_t)n * V + v] = logf(s / (float)(Un + 1));
}

// Zac[n,t] = log sum_v e^{am[t,v] + lavg[v]}: one wave per frame t < T_n.
__global__ __launch_bounds__(256) void ac_lse_kernel(SimpleArgs a) {
  const int T = a.b.T, V = a.V;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= a.b.N * T) return;
  const int n = row / T, t = row - n * T;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (t >= Tn) {
    if (lane == 0) a.Zac[row] = 0.f;
    return;
  }
  const float* x = a.am + (size_t)row * V;
  const float* la = a.lavg + (size_t)n * V;
  float m = kNegInfF;
  for (int v = lane; v < V; v += 64) m = fmaxf(m, x[v] + la[v]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  float sum = 0.f;
  for (int v = lane; v < V; v += 64) sum += expf(x[v] + la[v] - m);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
  if (lane == 0) a.Zac[row] = m + logf(sum);
}

// Gx[n,u], Gy[n,u]: column sums of the occupations over frames, from the
// per-16-frame partials in fixed order (fp64).
__global__ __launch_bounds__(256) void colsum_kernel(SimpleArgs a) {
  const int U1 = a.b.U + 1;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.b.N * U1) return;
  const int n = i / U1, u = i - n * U1;
  const double* px_ = a.cpx + (size_t)n * a.ncolblk * U1 + u;
  const double* py_ = a.cpy + (size_t)n * a.ncolblk * U1 + u;
  double cx = 0.0, cy = 0.0;
  // unrolled so that eight blocks' loads are in flight before the first add
  // (the adds keep their order)
#pragma unroll 8
  for (int q = 0; q < a.ncolblk; ++q) {
    cx += px_[(size_t)q * U1];
    cy += py_[(size_t)q * U1];
  }
  a.Gx[i] = cx;
  a.Gy[i] = cy;
}

// q[n,v] = (sum_t R(t) P_ac[t,v] - Sy(v)) / ((U_n+1) e^{lavg[v]}): threads over v.
__global__ __launch_bounds__(256) void ac_colsum_kernel(SimpleArgs a) {
  const int n = blockIdx.y, V = a.V, T = a.b.T, U1 = a.b.U + 1;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= V) return;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const float* amn = a.am + (size_t)n * T * V;
  const float la = a.lavg[(size_t)n * V + v];
  double g = 0.0;
  for (int t = 0; t < Tn; ++t) {
    const double R = a.rx[(size_t)n * T + t] + a.ry[(size_t)n * T + t];
    g += R * (double)expf(amn[(size_t)t * V + v] + la - a.Zac[(size_t)n * T + t]);
  }
  for (int u = 0; u < Un; ++u) {
    bool ok = true;
    if (symbol_at(a.b, n, u, V, ok) == v) g -= a.Gx[(size_t)n * U1 + u];
  }
  if (v == a.b.blank)
    for (int u = 0; u <= Un; ++u) g -= a.Gy[(size_t)n * U1 + u];
  a.q[(size_t)n * V + v] = (float)(g / ((double)(Un + 1) * (double)expf(la)));
}

// su[n,u] = sum_v q[v] e^{lm[u,v] - Zlm[u]}: one wave per row u <= U_n.
__global__ __launch_bounds__(256) void lm_s_kernel(SimpleArgs a) {
  const int U1 = a.b.U + 1, V = a.V;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= a.b.N * U1) return;
  const int n = row / U1, u = row - n * U1;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (u > Un) return;
  const float* x = a.lm + (size_t)row * V;
  const float* qn = a.q + (size_t)n * V;
  const float z = a.Zlm[row];
  float sum = 0.f;
  for (int v = lane; v < V; v += 64) sum += qn[v] * expf(x[v] - z);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
  if (lane == 0) a.su[row] = sum;
}

// Loads x[row][k..k+3] and the row max for exp(x - max); positions beyond the
// row end or of an invalid row load -inf, whose exponential is 0.
DEV void load_exp4(const float* x, const float* mx, int row, int k, int V, bool valid, RawExp<4>& r) {
  r.m = valid ? mx[row] : 0.f;
  const float* rowp = x + (size_t)(valid ? row : 0) * V;
  if (valid && ((V & 3) == 0) && (k + 4 <= V)) {
    float4 q = *reinterpret_cast<const float4*>(rowp + k);
    r.x[0] = q.x;
    r.x[1] = q.y;
    r.x[2] = q.z;
    r.x[3] = q.w;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) r.x[i] = (valid && k + i < V) ? rowp[k + i] : kNegInfF;
  }
}
// exp(x - max) of a staged operand (x <= max: the value lies in [0, 1]) with
// the hardware exp2: a few ulp, far below the contractions' fp32 rounding,
// and a fraction of the full-precision expf's instructions on the staging
// path that runs between the MFMAs.
DEV void finish_exp4(const RawExp<4>& r, float (&v)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = __expf(r.x[i] - r.m);
}
DEV void load_plain4(const float* p, bool valid, RawF<4>& r) {
  if (valid) {
    float4 q = *reinterpret_cast<const float4*>(p);
    r.v[0] = q.x;
    r.v[1] = q.y;
    r.v[2] = q.z;
    r.v[3] = q.w;
  } else {
    r.v[0] = r.v[1] = r.v[2] = r.v[3] = 0.f;
  }
}
DEV void finish_plain4(const RawF<4>& r, float (&v)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = r.v[i];
}

// ---------------------------------------------------------------------------
// Normaliser contraction, per utterance: C[t][u] = sum_v Ea[t][v] El[u][v].
// ---------------------------------------------------------------------------
using NormCfg = GemmCfg<64, 64, 32, false>;
// From this vocabulary on, the three contractions of the simple loss (K or N
// = V) take the joiner's 128 x 128 tiles of 8 waves: enough tiles remain to
// fill the chip, and a 32 x 32 or 16 x 32 wave tile spends most of its time
// staging operands.
constexpr int kSimpleBigV = 2048;
using BigCfg = GemmCfg<128, 128, 32, false, 4, 2>;

struct ExpRowsKC {  // rows r0 + row of x[.][V], value exp(x - max[row]); rows < lim
  using Raw = RawExp<4>;
  const float* x;
  const float* mx;
  int r0, lim, V;
  DEV void kc_load(int row, int k, Raw& r) const { load_exp4(x, mx, r0 + row, k, V, r0 + row < lim, r); }
  DEV void kc_finish(const Raw& r, float (&v)[4]) const { finish_exp4(r, v); }
};

// Split over v into nsplit K ranges (the contraction alone has too few tiles
// per batch to fill the chip); each writes its partial sums, and the
// epilogue kernel adds them in split order.
template <class Cfg>
__global__ __launch_bounds__(Cfg::NT) void normalizer_kernel(SimpleArgs a) {
  __shared__ __align__(16) float smem[Cfg::SMEM_BYTES / sizeof(float)];
  const int n = blockIdx.z / a.nsplit, sk = blockIdx.z - n * a.nsplit;
  const int t0 = blockIdx.x * Cfg::BM, u0 = blockIdx.y * Cfg::BN;
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (t0 >= Tn || u0 > Un) return;
  const int kc = split_chunk(V, a.nsplit, Cfg::BK);
  const int k0 = min(V, sk * kc), k1 = min(V, k0 + kc);
  floatx4 acc[Cfg::FM][Cfg::FN];
  ExpRowsKC sa{a.am + (size_t)n * T * V, a.m_a + (size_t)n * T, t0, Tn, V};
  ExpRowsKC sb{a.lm + (size_t)n * U1 * V, a.m_l + (size_t)n * U1, u0, Un + 1, V};
  KCLoader<Cfg, Cfg::BM, ExpRowsKC> la(sa);
  KCLoader<Cfg, Cfg::BN, ExpRowsKC> lb(sb);
  gemm_mainloop<Cfg>(la, lb, k0, k1, smem, acc);
  float* part = a.npart + ((size_t)sk * a.b.N + n) * T * U1;
#pragma unroll
  for (int j = 0; j < Cfg::FN; ++j) {
    const int u = u0 + tile_col<Cfg>(j);
    if (u > Un) continue;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + tile_row<Cfg>(i, r);
        if (t < Tn) part[(size_t)t * U1 + u] = acc[i][j][r];
      }
  }
}

// Z = m_a + m_l + log(sum of the partials), px and py (Eqs. (1)-(2), (5)).
// A block takes a tile of kEpiTileCells cells: FT = kEpiTileCells / (64 R)
// frames of one utterance times the 64 R slots of a row of the lattice
// layout, kEpiNodes per thread with all their loads issued together (the
// kernel is a chain of two dependent load rounds: partial sums, offsets and
// symbols, then the am / lm values at the symbols). The nodes are formed in
// row-major order (coalesced reads of the partials and writes of Z, px,
// py), their diagonal-major copies go to LDS, and are then written diagonal
// by diagonal, so that the cells of one diagonal in the tile (consecutive
// slots) are written together. The blocks after the tiles fill the cells of
// the copies that no node of the rectangle maps to, kEpiNodes cells per
// thread. Small lattices take one node per thread (enough blocks to fill the
// chip), those of more than kEpiWideNodes nodes four.
constexpr int kEpiThreads = 512;
constexpr long long kEpiWideNodes = 1 << 20;
__host__ __device__ inline int epi_tile_frames(int R, int nodes) {
  const int f = kEpiThreads * nodes / (64 * R);
  return f > 1 ? f : 1;
}
static int epi_nodes(int N, int T, int U1) { return (long long)N * T * U1 > kEpiWideNodes ? 4 : 1; }

template <int kEpiNodes>
__global__ __launch_bounds__(kEpiThreads) void normalizer_epi_kernel(SimpleArgs a) {
  constexpr int kEpiTileCells = kEpiThreads * kEpiNodes < 64 * 16 ? 64 * 16 : kEpiThreads * kEpiNodes;
  __shared__ double tx[kEpiTileCells], ty[kEpiTileCells];  // [frame of the tile][slot]
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V;
  const int R = lattice_rows_per_lane_dev(U1), W = 64 * R, FT = epi_tile_frames(R, kEpiNodes);
  const int tiles_per_utt = (T + FT - 1) / FT;
  const int tile_blocks = a.b.N * tiles_per_utt;
  if ((int)blockIdx.x >= tile_blocks) {
#pragma unroll
    for (int k = 0; k < kEpiNodes; ++k)
      lattice_fill_outside(a.pxd, a.pyd, (int)blockIdx.x - tile_blocks, threadIdx.x + k * kEpiThreads,
                           kEpiThreads * kEpiNodes, T, U1, R);
    return;
  }
  const int n = blockIdx.x / tiles_per_utt, t0 = (blockIdx.x - n * tiles_per_utt) * FT;
  const size_t L = (size_t)a.b.N * T * U1;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const int blank = a.b.blank;
  const bool smooth = a.lm_only != 0.f || a.am_only != 0.f;
  // round 1: partial sums, row offsets and symbols of the thread's nodes
  static_assert(kEpiNodes == 1 || kEpiThreads * kEpiNodes >= 64 * 16, "a tile holds at least one frame");
  for (int c0 = 0; c0 < FT * W; c0 += kEpiThreads * kEpiNodes) {
  int tl[kEpiNodes], uu[kEpiNodes], yy[kEpiNodes];
  bool cell[kEpiNodes], node[kEpiNodes];
  size_t idx[kEpiNodes];
  float sm[kEpiNodes], ma[kEpiNodes], ml[kEpiNodes];
#pragma unroll
  for (int k = 0; k < kEpiNodes; ++k) {
    const int c = c0 + threadIdx.x + k * kEpiThreads;
    tl[k] = c / W;
    uu[k] = c - tl[k] * W;
    const int t = t0 + tl[k], u = uu[k];
    cell[k] = tl[k] < FT && u < U1 && t < T;  // FT * W may fall short of the tile's cells
    node[k] = cell[k] && t < Tn && u <= Un;
    idx[k] = cell[k] ? ((size_t)n * T + t) * U1 + u : 0;
    sm[k] = 0.f;
    ma[k] = node[k] ? a.m_a[(size_t)n * T + t] : 0.f;
    ml[k] = node[k] ? a.m_l[(size_t)n * U1 + u] : 0.f;
    bool ok = true;
    yy[k] = (node[k] && u < Un) ? symbol_at(a.b, n, u, V, ok) : 0;
  }
  for (int q0 = 0; q0 < a.nsplit; q0 += 4) {  // the split partials in order, loads of 4 per node issued together
    float pv[kEpiNodes][4];
#pragma unroll
    for (int k = 0; k < kEpiNodes; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) pv[k][j] = (node[k] && q0 + j < a.nsplit) ? a.npart[(size_t)(q0 + j) * L + idx[k]] : 0.f;
#pragma unroll
    for (int k = 0; k < kEpiNodes; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) sm[k] += pv[k][j];
  }
  // round 2: the am and lm values at blank and at the symbol
  float ab[kEpiNodes], lb[kEpiNodes], ay[kEpiNodes], ly[kEpiNodes];
#pragma unroll
  for (int k = 0; k < kEpiNodes; ++k) {
    const float* amt = a.am + ((size_t)n * T + (node[k] ? t0 + tl[k] : 0)) * V;
    const float* lmu = a.lm + ((size_t)n * U1 + (node[k] ? uu[k] : 0)) * V;
    ab[k] = node[k] ? amt[blank] : 0.f;
    lb[k] = node[k] ? lmu[blank] : 0.f;
    ay[k] = node[k] ? amt[yy[k]] : 0.f;
    ly[k] = node[k] ? lmu[yy[k]] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < kEpiNodes; ++k) {
    const int t = t0 + tl[k], u = uu[k];
    double dx = kNegInfD, dy = kNegInfD;
    if (cell[k]) {
      if (!node[k]) {
        a.Z[idx[k]] = 0.f;
        a.px[idx[k]] = kNegInfF;
        a.py[idx[k]] = kNegInfF;
      } else {
        const float s1 = (sm[k] > FLT_MIN || sm[k] != sm[k]) ? sm[k] : FLT_MIN;
        const float z = ma[k] + ml[k] + logf(s1);
        a.Z[idx[k]] = z;
        float py = ab[k] + lb[k] - z;
        float px = ay[k] + ly[k] - z;
        if (smooth) {
          // smoothed joiner: c L_trivial + a L_lm + b L_acoustic (Sec. 3.3.1)
          const float cw = 1.f - a.lm_only - a.am_only;
          const float zl = a.Zlm[(size_t)n * U1 + u], za = a.Zac[(size_t)n * T + t];
          const float* la = a.lavg + (size_t)n * V;
          py = cw * py + a.lm_only * (lb[k] - zl) + a.am_only * (ab[k] + la[blank] - za);
          px = cw * px + a.lm_only * (ly[k] - zl) + a.am_only * (ay[k] + la[yy[k]] - za);
        }
        a.py[idx[k]] = py;
        a.px[idx[k]] = (u < Un) ? px : kNegInfF;
        dy = (double)py * kLog2e;
        dx = (u < Un) ? (double)px * kLog2e : kNegInfD;
      }
    }
    if (tl[k] < FT) {
      tx[tl[k] * W + lattice_slot(u, R)] = dx;
      ty[tl[k] * W + lattice_slot(u, R)] = dy;
    }
  }
  }
  __syncthreads();
  // diagonal d = t0 + k holds the tile's nodes (t0 + FT-1-j', u = d - t) for
  // the FT frames; item (k, j): u = k - (FT-1) + j, so that consecutive j are
  // consecutive u on one diagonal
  const int ft = min(FT, T - t0), nd = FT - 1 + U1;
  const size_t base = (size_t)n * (T + U1 - 1) * W;
  for (int it = threadIdx.x; it < nd * FT; it += blockDim.x) {
    const int k = it / FT, j = it - k * FT;
    const int u = k - (FT - 1) + j, tl = k - u;
    if (u < 0 || u >= U1 || tl < 0 || tl >= ft) continue;
    const int sl = lattice_slot(u, R);
    const size_t o = base + (size_t)(t0 + k) * W + sl;
    a.pxd[o] = (DiagT)tx[tl * W + sl];
    a.pyd[o] = (DiagT)ty[tl * W + sl];
  }
}

// ---------------------------------------------------------------------------
// Normaliser and its epilogue in one kernel (U + 1 <= 320). One workgroup
// of 8 waves per (utterance, 32 frames) holds C[t][u] for every u of its
// frames: C = sum over chunks of v of e^{am - m_a} [32 x CV] .
// e^{lm - m_l}^T [CV x U+1], both exponentials staged through two LDS
// stages: the MFMAs of chunk c read one stage, then the exponentials of
// chunk c+1 (loaded two chunks before) go to the other and chunk c+3's loads
// are issued; one barrier per chunk. Then Z, px and py of its nodes (Eqs.
// (1)-(2), (5)) go to the rectangle, and through LDS (the stages reused) to
// the diagonal-major copies, diagonal by diagonal. No split over v: no
// partial sums and no second launch. Wave w holds the C blocks of rows
// 16 (w & 1) .. +15 whose u block is (w >> 1) + 4 i. The blocks after the
// tiles fill the cells of the copies that no node of the rectangle maps to.
// ---------------------------------------------------------------------------
constexpr int kNfT = 32;         // frames per workgroup
constexpr int kNfV = 64;         // v per chunk at U + 1 <= 64 (32 above: two stages of 64 would halve the workgroups per CU)
constexpr int kNfThreads = 512;
constexpr int kNfMaxU1 = 320;
constexpr int kNfFill = 4;       // cells per thread of a fill block
constexpr float kLog2eF = 1.44269504f;

template <int KP>
struct alignas(16) NfSmem {
  static constexpr int CV = KP > 64 ? 32 : kNfV;  // v per chunk
  static constexpr int S = CV + 4;                // row stride of a stage (conflict-free fragment reads)
  union {
    struct {
      float ea[2][kNfT * S];  // e^{am - m_a}, [stage][t][v]
      float el[2][KP * S];    // e^{lm - m_l}, [stage][u][v]
    } g;
    struct {
      float px[kNfT * KP];    // px, py of the tile's cells, [frame][slot of the lattice row]
      float py[kNfT * KP];
    } d;
  };
  float ma[kNfT], ab[kNfT], za[kNfT];  // per frame: m_a, am[t, blank], Zac
  float ml[KP], lb[KP], lyv[KP], zl[KP], lay[KP];  // per u: m_l, lm[u, blank], lm[u, y], Zlm, lavg[y]
  int yy[KP];                          // y_{u+1}
};

// One chunk's loads in registers: a thread takes float4 number tid of the
// am rows (if any) and tid + 512 i of the lm rows, the same rows in every
// chunk (their maxima stay in registers).
template <int KP>
struct NfPrefetch {
  static constexpr int Q = NfSmem<KP>::CV / 4;   // float4 per staged row
  static constexpr int AQ = kNfT * Q;            // float4 of the am rows
  static constexpr int NL = KP * Q / kNfThreads; // float4 of the lm rows per thread
  static_assert(AQ <= kNfThreads && NL * kNfThreads == KP * Q, "staging split");
  float4 x;
  float4 l[NL];
};

template <int KP, bool V4>
DEV void nf_load(Rsrc am, Rsrc lm, int t0, int v0, int Tn, int Un, int V, NfPrefetch<KP>& f) {
  using P = NfPrefetch<KP>;
  const int tid = threadIdx.x;
  {
    const int t = t0 + tid / P::Q, v = v0 + 4 * (tid % P::Q);
    const bool in = tid < P::AQ && t < Tn && v < V;
    const uint32_t o = (uint32_t)(t * V + v) * 4u;
    if (V4) {
      f.x = buf_load_f4(am, in ? o : kOob);
    } else {
      f.x.x = buf_load_f32(am, in ? o : kOob);
      f.x.y = buf_load_f32(am, in && v + 1 < V ? o + 4u : kOob);
      f.x.z = buf_load_f32(am, in && v + 2 < V ? o + 8u : kOob);
      f.x.w = buf_load_f32(am, in && v + 3 < V ? o + 12u : kOob);
    }
  }
#pragma unroll
  for (int i = 0; i < P::NL; ++i) {
    const int q = tid + i * kNfThreads, u = q / P::Q, v = v0 + 4 * (q % P::Q);
    const bool in = u <= Un && v < V;
    const uint32_t o = (uint32_t)(u * V + v) * 4u;
    if (V4) {
      f.l[i] = buf_load_f4(lm, in ? o : kOob);
    } else {
      f.l[i].x = buf_load_f32(lm, in ? o : kOob);
      f.l[i].y = buf_load_f32(lm, in && v + 1 < V ? o + 4u : kOob);
      f.l[i].z = buf_load_f32(lm, in && v + 2 < V ? o + 8u : kOob);
      f.l[i].w = buf_load_f32(lm, in && v + 3 < V ? o + 12u : kOob);
    }
  }
}

// e^{x - m} = 2^{(x - m) log2(e)} of one chunk into stage st (m per staged
// row; x - m first, so that a row's maximum gives exactly 1 and no rounding
// of m log2(e) biases a whole row). Rows past the utterance (loaded as
// zeros) only feed C entries of absent nodes, which nothing reads; the
// columns past V (the last chunk only, TAIL) are zeroed.
template <int KP, bool TAIL>
DEV void nf_store(NfSmem<KP>& sm, int st, const NfPrefetch<KP>& f, float mA, const float (&mL)[NfPrefetch<KP>::NL],
                  int v0, int V) {
  using P = NfPrefetch<KP>;
  constexpr int S = NfSmem<KP>::S;
  const int tid = threadIdx.x;
  auto ex = [&](float4 x, float m, int c) {
    const float xv[4] = {x.x, x.y, x.z, x.w};
    float e[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      e[j] = __builtin_amdgcn_exp2f((xv[j] - m) * kLog2eF);
      if (TAIL && v0 + c + j >= V) e[j] = 0.f;
    }
    return make_float4(e[0], e[1], e[2], e[3]);
  };
  if (tid < P::AQ) {
    const int t = tid / P::Q, c = 4 * (tid % P::Q);
    *reinterpret_cast<float4*>(&sm.g.ea[st][t * S + c]) = ex(f.x, mA, c);
  }
#pragma unroll
  for (int i = 0; i < P::NL; ++i) {
    const int q = tid + i * kNfThreads, u = q / P::Q, c = 4 * (q % P::Q);
    *reinterpret_cast<float4*>(&sm.g.el[st][u * S + c]) = ex(f.l[i], mL[i], c);
  }
}

template <int KP>
DEV void nf_store_chunk(NfSmem<KP>& sm, int st, const NfPrefetch<KP>& f, float mA,
                        const float (&mL)[NfPrefetch<KP>::NL], int v0, int V) {
  if (v0 + NfSmem<KP>::CV <= V) nf_store<KP, false>(sm, st, f, mA, mL, v0, V);
  else nf_store<KP, true>(sm, st, f, mA, mL, v0, V);
}

template <int KP, bool V4>
__global__ __launch_bounds__(kNfThreads) void normalizer_fused_kernel(SimpleArgs a) {
  __shared__ NfSmem<KP> sm;
  using P = NfPrefetch<KP>;
  constexpr int CV = NfSmem<KP>::CV, S = NfSmem<KP>::S;
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V, blank = a.b.blank;
  const int ntt = (T + kNfT - 1) / kNfT, tiles = a.b.N * ntt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int R = lattice_rows_per_lane_dev(U1), W = 64 * R;  // W <= KP
  if ((int)blockIdx.x >= tiles) {
#pragma unroll
    for (int k = 0; k < kNfFill; ++k)
      lattice_fill_outside(a.pxd, a.pyd, (int)blockIdx.x - tiles, tid + k * kNfThreads, kNfFill * kNfThreads, T,
                           U1, R);
    return;
  }
  const int n = blockIdx.x / ntt, t0 = (blockIdx.x - n * ntt) * kNfT;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const bool smooth = a.lm_only != 0.f || a.am_only != 0.f;
  const float* amn = a.am + (size_t)n * T * V;
  const float* lmn = a.lm + (size_t)n * U1 * V;
  // per-frame and per-u values of the epilogue (and the maxima of the staging)
  if (tid < kNfT) {
    const int t = t0 + tid;
    const bool node = t < Tn;
    sm.ma[tid] = node ? a.m_a[(size_t)n * T + t] : 0.f;
    sm.ab[tid] = node ? amn[(size_t)t * V + blank] : 0.f;
    sm.za[tid] = (node && smooth) ? a.Zac[(size_t)n * T + t] : 0.f;
  }
  for (int u = tid; u < KP; u += kNfThreads) {
    const bool row = u <= Un;
    bool ok = true;
    const int y = (u < Un) ? symbol_at(a.b, n, u, V, ok) : 0;
    sm.yy[u] = y;
    sm.ml[u] = row ? a.m_l[(size_t)n * U1 + u] : 0.f;
    sm.lb[u] = row ? lmn[(size_t)u * V + blank] : 0.f;
    sm.lyv[u] = row ? lmn[(size_t)u * V + y] : 0.f;
    sm.zl[u] = (row && smooth) ? a.Zlm[(size_t)n * U1 + u] : 0.f;
    sm.lay[u] = (row && smooth) ? a.lavg[(size_t)n * V + y] : 0.f;
  }
  __syncthreads();
  const int kn = (Un + 1 + 15) / 16 * 16;
  const int tb = wave & 1, ubw = __builtin_amdgcn_readfirstlane(wave >> 1);
  constexpr int NB = KP / 64;  // C blocks per wave: u block (w >> 1) + 4 i
  floatx4 acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (t0 < Tn) {
    const Rsrc amr = make_rsrc(amn, (size_t)T * V * 4), lmr = make_rsrc(lmn, (size_t)U1 * V * 4);
    const float mA = tid < P::AQ ? sm.ma[tid / P::Q] : 0.f;
    float mL[P::NL];
#pragma unroll
    for (int i = 0; i < P::NL; ++i) mL[i] = sm.ml[(tid + i * kNfThreads) / P::Q];
    const int nc = (V + CV - 1) / CV;
    // chunk c (> 0) in f[c % 2]; chunks past V load zeros (kOob): the loads
    // stay unconditional, so that each store waits only for its own chunk
    P f[2];
    nf_load<KP, V4>(amr, lmr, t0, 0, Tn, Un, V, f[0]);
    nf_store_chunk<KP>(sm, 0, f[0], mA, mL, 0, V);
    nf_load<KP, V4>(amr, lmr, t0, CV, Tn, Un, V, f[1]);
    nf_load<KP, V4>(amr, lmr, t0, 2 * CV, Tn, Un, V, f[0]);
    sg_barrier();
    auto step = [&](int c, P& fn) {
      const int st = c & 1;
      // chunk c: every fragment of the stage first, then the MFMAs of the
      // wave's u blocks that hold rows of the utterance
      floatx4 fa[CV / 16], fb[CV / 16][NB];
#pragma unroll
      for (int k = 0; k < CV / 16; ++k) {
        fa[k] = *reinterpret_cast<const floatx4*>(&sm.g.ea[st][(16 * tb + l16) * S + 16 * k + 4 * g4]);
#pragma unroll
        for (int i = 0; i < NB; ++i)
          fb[k][i] = *reinterpret_cast<const floatx4*>(&sm.g.el[st][(16 * (ubw + 4 * i) + l16) * S + 16 * k + 4 * g4]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int k = 0; k < CV / 16; ++k)
#pragma unroll
        for (int i = 0; i < NB; ++i)
          if (16 * (ubw + 4 * i) < kn) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
              acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[k][q], fb[k][i][q], acc[i], 0, 0, 0);
          }
      // chunk c+1 into the other stage (last read by chunk c-1, before the
      // previous barrier), then chunk c+3's loads
      if (c + 1 < nc) nf_store_chunk<KP>(sm, st ^ 1, fn, mA, mL, (c + 1) * CV, V);
      nf_load<KP, V4>(amr, lmr, t0, (c + 3) * CV, Tn, Un, V, fn);
      sg_barrier();
    };
    for (int c = 0; c < nc; c += 2) {
      step(c, f[1]);
      if (c + 1 < nc) step(c + 1, f[0]);
    }
  }
  // epilogue: the target logits am[t, y_u] of the lane's nodes first (one gather round)
  const Rsrc amr = make_rsrc(amn, (size_t)T * V * 4);
  float ay[NB][4];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int u = 16 * (ubw + 4 * i) + l16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + 16 * tb + 4 * g4 + r;
      const bool node = t < Tn && u < Un;
      ay[i][r] = buf_load_f32(amr, node ? (uint32_t)(t * V + sm.yy[u]) * 4u : kOob);
    }
  }
  sg_barrier();  // every wave's MFMAs are done with the stages
  const float cw = 1.f - a.lm_only - a.am_only;
  const float* la = a.lavg + (size_t)n * V;
  const float lab = smooth ? la[blank] : 0.f;
  const size_t L0 = ((size_t)n * T) * U1;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int u = 16 * (ubw + 4 * i) + l16;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int tl = 16 * tb + 4 * g4 + r, t = t0 + tl;
      const bool cell = t < T && u < U1, node = t < Tn && u <= Un;
      float z = 0.f, px = kNegInfF, py = kNegInfF;
      if (node) {
        const float sv = acc[i][r];
        const float s1 = (sv > FLT_MIN || sv != sv) ? sv : FLT_MIN;
        z = sm.ma[tl] + sm.ml[u] + logf(s1);
        py = sm.ab[tl] + sm.lb[u] - z;
        float pxv = ay[i][r] + sm.lyv[u] - z;
        if (smooth) {
          // smoothed joiner: c L_trivial + a L_lm + b L_acoustic (Sec. 3.3.1)
          py = cw * py + a.lm_only * (sm.lb[u] - sm.zl[u]) + a.am_only * (sm.ab[tl] + lab - sm.za[tl]);
          pxv = cw * pxv + a.lm_only * (sm.lyv[u] - sm.zl[u]) + a.am_only * (ay[i][r] + sm.lay[u] - sm.za[tl]);
        }
        px = (u < Un) ? pxv : kNegInfF;
      }
      if (cell) {
        const size_t idx = L0 + (size_t)t * U1 + u;
        a.Z[idx] = z;
        a.px[idx] = px;
        a.py[idx] = py;
      }
      if (u < U1) {
        sm.d.px[tl * KP + lattice_slot(u, R)] = px;
        sm.d.py[tl * KP + lattice_slot(u, R)] = py;
      }
    }
  }
  __syncthreads();
  // diagonal d = t0 + k holds the tile's nodes (t0 + tl, u = k - tl); item
  // (k, j): u = k - (kNfT - 1) + j, so that consecutive j are consecutive u
  // on one diagonal
  const int ft = min(kNfT, T - t0), nd = kNfT - 1 + U1;
  const size_t base = (size_t)n * (T + U1 - 1) * W;
  for (int it = tid; it < nd * kNfT; it += kNfThreads) {
    const int k = it / kNfT, j = it - k * kNfT;
    const int u = k - (kNfT - 1) + j, tl = k - u;
    if (u < 0 || u >= U1 || tl < 0 || tl >= ft) continue;
    const int sl = lattice_slot(u, R);
    const size_t o = base + (size_t)(t0 + k) * W + sl;
    a.pxd[o] = (DiagT)((double)sm.d.px[tl * KP + sl] * kLog2e);
    a.pyd[o] = (DiagT)((double)sm.d.py[tl * KP + sl] * kLog2e);
  }
}

// ---------------------------------------------------------------------------
// d am: per utterance C[t][v] = sum_u Wt[t][u] El[u][v]  (K = U_n + 1)
// ---------------------------------------------------------------------------
using DamCfg = GemmCfg<32, 64, 32, false>;
constexpr int kDamSymChunk = 128;  // symbols per pass of the d am kernel's target columns

struct WtSrcKC {  // A(t, u) = Wt[t][u], rows padded to ldw (multiple of 4, zero-filled)
  using Raw = RawF<4>;
  const float* Wt;
  int t0, Tn, ldw;
  DEV void kc_load(int row, int k, Raw& r) const {
    const int t = t0 + row;
    const bool ok = t < Tn && k < ldw;
    load_plain4(Wt + (ok ? (size_t)t * ldw + k : 0), ok, r);
  }
  DEV void kc_finish(const Raw& r, float (&v)[4]) const { finish_plain4(r, v); }
};
struct ExpSrcMNC {  // B(k, col) = exp(x[k][c0+col] - mx[k]) for rows k < klim, cols < V
  using Raw = RawExp<4>;
  const float* x;  // [rows][V]
  const float* mx;
  int c0, klim, V;
  DEV void mnc_load(int k, int col, Raw& r) const { load_exp4(x, mx, k, c0 + col, V, k < klim, r); }
  DEV void mnc_finish(const Raw& r, float (&v)[4]) const { finish_exp4(r, v); }
};

template <class Cfg>
__global__ __launch_bounds__(Cfg::NT) void dam_kernel(SimpleArgs a) {
  __shared__ __align__(16) float smem[Cfg::SMEM_BYTES / sizeof(float)];
  const int n = blockIdx.z;
  const int t0 = blockIdx.x * Cfg::BM, v0 = blockIdx.y * Cfg::BN;
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const bool active = t0 < Tn;
  floatx4 acc[Cfg::FM][Cfg::FN];
  if (active) {
    WtSrcKC sa{a.Wt + (size_t)n * T * a.ldw, t0, Tn, a.ldw};
    ExpSrcMNC sb{a.lm + (size_t)n * U1 * V, a.m_l + (size_t)n * U1, v0, Un + 1, V};
    KCLoader<Cfg, Cfg::BM, WtSrcKC> la(sa);
    MNCLoader<Cfg, Cfg::BN, ExpSrcMNC> lb(sb);
    gemm_mainloop<Cfg>(la, lb, 0, Un + 1, smem, acc);
  }
  const float* amn = a.am + (size_t)n * T * V;
  const float* ma = a.m_a + (size_t)n * T;
  const float* gxn = a.gx + (size_t)n * T * U1;
  float* out = a.am_grad + (size_t)n * T * V;
  const bool smooth = a.lm_only != 0.f || a.am_only != 0.f;
  const float c = 1.f - a.lm_only - a.am_only;  // weight of the trivial joiner
  const float ks = 1.f - a.lm_only;             // weight of the target/blank terms
  // dense part: c e^{am - m_a} * acc (+ b R(t) P_ac[t,v] when smoothed)
  float res[Cfg::FM][Cfg::FN][4];
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + tile_row<Cfg>(i, r);
      const bool tv = active && t < Tn;
      const float mx = tv ? ma[t] : 0.f;
      const float bR = (tv && smooth) ? a.am_only * (float)(a.rx[(size_t)n * T + t] + a.ry[(size_t)n * T + t]) : 0.f;
      const float za = (tv && smooth) ? a.Zac[(size_t)n * T + t] : 0.f;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int v = v0 + tile_col<Cfg>(j);
        float d = 0.f;
        if (tv && v < V) {
          const float x = amn[(size_t)t * V + v];
          d = c * expf(x - mx) * acc[i][j][r];
          if (smooth) d += bR * expf(x + a.lavg[(size_t)n * V + v] - za);
        }
        res[i][j][r] = d;
      }
    }
  if (active) {
    // sparse part: the target columns. Per chunk of kDamSymChunk symbols the
    // u whose symbol falls in the tile's columns are listed in ascending
    // order (ballot compaction), their gx values for the tile's frames are
    // gathered by all threads at once, and each lane subtracts them in the
    // list's order (ascending u: deterministic).
    constexpr int kChunk = kDamSymChunk;
    int* mu = reinterpret_cast<int*>(smem);  // [kChunk] listed u
    int* my = mu + kChunk;                   // [kChunk] their symbols
    constexpr int kWaves = Cfg::NT / 64;
    int* wcnt = my + kChunk;                 // [kWaves] per-wave counts
    float* g = reinterpret_cast<float*>(wcnt + kWaves);  // [kChunk][BM] gathered gx
    static_assert((2 * kChunk + kWaves) * 4 + kChunk * Cfg::BM * 4 <= Cfg::SMEM_BYTES, "sparse chunk fits");
    static_assert(Cfg::NT >= kChunk, "one thread per symbol of a chunk");
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    for (int c0 = 0; c0 < Un; c0 += kChunk) {
      __syncthreads();  // the previous user of smem is done
      const int u = c0 + threadIdx.x;
      int y = -1;
      if (threadIdx.x < kChunk && u < Un) {
        bool ok = true;
        y = symbol_at(a.b, n, u, V, ok);
      }
      const bool hit = y >= v0 && y < v0 + Cfg::BN;
      const uint64_t bal = __ballot(hit);
      if (lane == 0) wcnt[wv] = __popcll(bal);
      __syncthreads();
      int base = 0, nm = 0;
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
        base += (w < wv) ? wcnt[w] : 0;
        nm += wcnt[w];
      }
      if (hit) {
        const int k = base + __popcll(bal & ((1ull << lane) - 1));
        mu[k] = u;
        my[k] = y;
      }
      __syncthreads();
      for (int it = threadIdx.x; it < nm * Cfg::BM; it += blockDim.x) {
        const int k = it / Cfg::BM, tr = it - k * Cfg::BM, t = t0 + tr;
        g[it] = (t < Tn) ? gxn[(size_t)t * U1 + mu[k]] : 0.f;
      }
      __syncthreads();
      for (int k = 0; k < nm; ++k) {
        const int yk = my[k];
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j) {
          if (v0 + tile_col<Cfg>(j) != yk) continue;
#pragma unroll
          for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) res[i][j][r] -= ks * g[k * Cfg::BM + tile_row<Cfg>(i, r)];
        }
      }
    }
    const int blank = a.b.blank;
    if (blank >= v0 && blank < v0 + Cfg::BN) {
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        if (v0 + tile_col<Cfg>(j) != blank) continue;
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = t0 + tile_row<Cfg>(i, r);
            if (t < Tn) res[i][j][r] = (float)((double)res[i][j][r] - (double)ks * a.ry[(size_t)n * T + t]);
          }
      }
    }
  }
  const float sc = a.scale ? a.scale[n] : 1.f;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + tile_row<Cfg>(i, r);
      if (t >= T) continue;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int v = v0 + tile_col<Cfg>(j);
        if (v < V) out[(size_t)t * V + v] = (active && t < Tn) ? sc * res[i][j][r] : 0.f;
      }
    }
}

// ---------------------------------------------------------------------------
// d lm: per utterance C[u][v] = sum_t Wt[t][u] Ea[t][v]  (K = T_n)
// ---------------------------------------------------------------------------
using DlmCfg = GemmCfg<32, 64, 32, false>;

struct WtSrcMNC {  // A(u, t) = Wt[t][u]: global is [t][u], u-contiguous
  using Raw = RawF<4>;
  const float* Wt;
  int u0, Tn, ldw;
  DEV void mnc_load(int k, int col, Raw& r) const {
    const int u = u0 + col;
    const bool ok = k < Tn && u < ldw;
    load_plain4(Wt + (ok ? (size_t)k * ldw + u : 0), ok, r);
  }
  DEV void mnc_finish(const Raw& r, float (&v)[4]) const { finish_plain4(r, v); }
};

// Split over frames into lsplit K ranges; partial sums C[u][v] per split,
// finished by dlm_epi_kernel.
template <class Cfg>
__global__ __launch_bounds__(Cfg::NT) void dlm_kernel(SimpleArgs a) {
  __shared__ __align__(16) float smem[Cfg::SMEM_BYTES / sizeof(float)];
  const int n = blockIdx.z / a.lsplit, sk = blockIdx.z - n * a.lsplit;
  const int u0 = blockIdx.x * Cfg::BM, v0 = blockIdx.y * Cfg::BN;
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (u0 > Un) return;
  const int kc = split_chunk(Tn, a.lsplit, Cfg::BK);
  const int k0 = min(Tn, sk * kc), k1 = min(Tn, k0 + kc);
  floatx4 acc[Cfg::FM][Cfg::FN];
  WtSrcMNC sa{a.Wt + (size_t)n * T * a.ldw, u0, Tn, a.ldw};
  ExpSrcMNC sb{a.am + (size_t)n * T * V, a.m_a + (size_t)n * T, v0, Tn, V};
  MNCLoader<Cfg, Cfg::BM, WtSrcMNC> la(sa);
  MNCLoader<Cfg, Cfg::BN, ExpSrcMNC, decltype(la)::NBLK> lb(sb);  // threads after A's blocks
  gemm_mainloop<Cfg>(la, lb, k0, k1, smem, acc);
  float* part = a.lpart + ((size_t)sk * a.b.N + n) * U1 * V;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int u = u0 + tile_row<Cfg>(i, r);
      if (u > Un) continue;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int v = v0 + tile_col<Cfg>(j);
        if (v < V) part[(size_t)u * V + v] = acc[i][j][r];
      }
    }
}

// d lm[u,v] = sc (e^{lm - m_l} sum_splits C - [v = y_{u+1}] sum_t gx - [v = blank] sum_t gy);
// one thread per 4 consecutive v of a row.
__global__ __launch_bounds__(256) void dlm_epi_kernel(SimpleArgs a) {
  const int U1 = a.b.U + 1, V = a.V;
  const int nvg = (V + 3) / 4;
  const size_t g = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= (size_t)a.b.N * U1 * nvg) return;
  const int row = (int)(g / nvg);  // n * U1 + u
  const int v0 = (int)(g - (size_t)row * nvg) * 4;
  const int n = row / U1, u = row - n * U1;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  float* out = a.lm_grad + (size_t)row * V;
  if (u > Un) {
    for (int v = v0; v < min(V, v0 + 4); ++v) out[v] = 0.f;
    return;
  }
  const float sc = a.scale ? a.scale[n] : 1.f;
  const int blank = a.b.blank;
  bool ok = true;
  const int y = (u < Un) ? symbol_at(a.b, n, u, V, ok) : -1;
  const float ml = a.m_l[row];
  const float* lmr = a.lm + (size_t)row * V;
  const size_t stride = (size_t)a.b.N * U1 * V;
  const size_t base = (size_t)row * V;
  const bool smooth = a.lm_only != 0.f || a.am_only != 0.f;
  const float cw = 1.f - a.lm_only - a.am_only;  // weight of the trivial joiner
  const double ks = 1.0 - (double)a.am_only;      // weight of the target/blank terms
  // the target and blank columns collect Gx(u) = sum_t gx(t,u) and Gy(u) (fp64)
  const double gx = a.Gx[row], gy = a.Gy[row];
  const float zl = smooth ? a.Zlm[row] : 0.f;
  const float aG = smooth ? a.lm_only * (float)(gx + gy) : 0.f;
  const float su = smooth ? a.su[row] : 0.f;
  for (int v = v0; v < min(V, v0 + 4); ++v) {
    float c = 0.f;
    for (int q = 0; q < a.lsplit; ++q) c += a.lpart[(size_t)q * stride + base + v];
    float d = cw * expf(lmr[v] - ml) * c;
    if (smooth) {
      const float p = expf(lmr[v] - zl);
      d += aG * p + a.am_only * p * (a.q[(size_t)n * V + v] - su);
    }
    double gd = (double)d;
    if (v == y) gd -= ks * gx;
    if (v == blank) gd -= ks * gy;
    out[v] = (float)(sc * gd);
  }
}

// ---------------------------------------------------------------------------
// d am and d lm in one pass (U + 1 <= 320, plain trivial joiner).
//
// One workgroup per (utterance, 64 columns of v, range of frames). The
// columns' e^{lm - m_l} (every u) is formed once into LDS; per step of 32
// frames the workgroup stages W(t, u) and e^{am - m_a} through LDS and runs
// both contractions on them:
//   d am [32 x 64] = W [32 x U+1] . e^{lm - m_l} [U+1 x 64], finished at once
//     (times e^{am - m_a}, minus the target and blank terms) and stored;
//   d lm [U+1 x 64] += W^T [U+1 x 32] . e^{am - m_a} [32 x 64], kept in
//     registers over the range's frames and finished at the end (a single
//     range) or stored as the range's partial sums for dlm_epi_kernel.
// am is read once for both, every exponential is formed once, and the next
// step's global loads are in flight during the current step's MFMAs. Eight
// waves (two per SIMD, so that one's LDS waits overlap the other's MFMAs):
// wave w computes the d am block of rows 16 (w & 1) .. +15, columns
// 16 (w >> 1) .. +15 of a step, and the d lm blocks of columns 16 (w & 3) ..
// +15 whose u block has the parity w >> 2.
// ---------------------------------------------------------------------------
constexpr int kSgT = 32;        // frames per step
constexpr int kSgV = 64;        // columns per workgroup
constexpr int kSgMaxU1 = 320;   // the fused kernel takes U + 1 up to this
constexpr int kSgThreads = 512;
constexpr int kSgWaves = kSgThreads / 64;
constexpr int kSgDam = 8 / kSgWaves;  // d am blocks of a step per wave (along v)
constexpr int kSgUg = kSgWaves / 4;   // wave groups sharing the d lm u blocks of a column block
constexpr int kSgList = 32;     // listed targets whose gx one gather round stages
constexpr int kSgTS = kSgT + 4; // row stride of eaT (16-byte rows, conflict-free fragment reads)

template <int KP>  // u extent staged: U + 1 <= KP (a multiple of 16)
struct alignas(16) SgSmem {
  static constexpr int K = KP + 4;  // row stride of wt and elT
  float wt[kSgT * K];               // W(t, u) of the step's frames, [t][u] (zero past ldw)
  float eaT[kSgV * kSgTS];          // e^{am - m_a}, [v][t] (zero past T_n or V)
  float elT[kSgV * K];              // e^{lm - m_l}, [v][u] (zero past U_n or V)
  float g[kSgList * kSgT];          // gx(t, u_k) of listed targets, [k][t]
  double ry[kSgT];                  // row sums of gy
  int lu[KP], ly[KP];               // targets in the columns (ascending u) and their symbols
  int sym[KP];                      // y_{u+1}
  int cnt[kSgWaves];
};

struct SgPrefetch {  // one step's global loads, held until the step's LDS writes
  float4 w[kSgMaxU1 * 8 / kSgThreads];  // W: 32 ldw floats
  float4 x[512 / kSgThreads];           // am: 32 x 64 values
  float ma[512 / kSgThreads];
  float gx[kSgT * kSgList / kSgThreads];
  double ry;
};

// The utterance's arrays as buffer resources: every step load is issued
// unconditionally (kOob where there is nothing to load), so that the step's
// code is straight-line and the wait counts stay exact.
struct SgSrc {
  Rsrc wt, am, ma, gx, ry;
  int ldw, V, U1, Tn;
};

template <int KP, bool V4>  // V4: V is a multiple of 4 (16-byte loads of am)
DEV void sg_load(const SgSrc& c, int t0, int v0, int nml, const int* lu, SgPrefetch& f) {
  const int tid = threadIdx.x, q4 = c.ldw / 4;
#pragma unroll
  for (int i = 0; i < KP * 8 / kSgThreads; ++i) {  // the step's rows of W are one contiguous block; rows past T fall outside
    const int q = tid + i * kSgThreads;
    f.w[i] = buf_load_f4(c.wt, q < kSgT * q4 ? (uint32_t)(t0 * c.ldw + 4 * q) * 4u : kOob);
  }
#pragma unroll
  for (int i = 0; i < 512 / kSgThreads; ++i) {
    const int q = tid + i * kSgThreads, t = t0 + q / 16, v = v0 + 4 * (q % 16);
    const bool in = t < c.Tn && v < c.V;
    const uint32_t o = (uint32_t)(t * c.V + v) * 4u;
    f.ma[i] = buf_load_f32(c.ma, t < c.Tn ? (uint32_t)t * 4u : kOob);
    if (V4) {
      f.x[i] = buf_load_f4(c.am, in ? o : kOob);
    } else {
      f.x[i].x = buf_load_f32(c.am, in ? o : kOob);
      f.x[i].y = buf_load_f32(c.am, in && v + 1 < c.V ? o + 4u : kOob);
      f.x[i].z = buf_load_f32(c.am, in && v + 2 < c.V ? o + 8u : kOob);
      f.x[i].w = buf_load_f32(c.am, in && v + 3 < c.V ? o + 12u : kOob);
    }
  }
#pragma unroll
  for (int i = 0; i < kSgT * kSgList / kSgThreads; ++i) {
    const int q = tid + i * kSgThreads, k = q / kSgT, t = t0 + q % kSgT;
    f.gx[i] = buf_load_f32(c.gx, (k < nml && t < c.Tn) ? (uint32_t)(t * c.U1 + lu[k]) * 4u : kOob);
  }
  f.ry = buf_load_f64(c.ry, (tid < kSgT && t0 + tid < c.Tn) ? (uint32_t)(t0 + tid) * 8u : kOob);
}

template <int KP>
DEV void sg_store(SgSmem<KP>& sm, const SgPrefetch& f, int t0, int v0, int Tn, int V, int ldw) {
  constexpr int K = SgSmem<KP>::K;
  const int tid = threadIdx.x, q4 = ldw / 4;
#pragma unroll
  for (int i = 0; i < KP * 8 / kSgThreads; ++i) {
    const int q = tid + i * kSgThreads;
    if (q < kSgT * q4) *reinterpret_cast<float4*>(&sm.wt[(q / q4) * K + 4 * (q % q4)]) = f.w[i];
  }
#pragma unroll
  for (int i = 0; i < 512 / kSgThreads; ++i) {
    const int q = tid + i * kSgThreads, t = q / 16, c = 4 * (q % 16);
    const bool row = t0 + t < Tn;
    const float xv[4] = {f.x[i].x, f.x[i].y, f.x[i].z, f.x[i].w};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      sm.eaT[(c + j) * kSgTS + t] = (row && v0 + c + j < V) ? __expf(xv[j] - f.ma[i]) : 0.f;
  }
#pragma unroll
  for (int i = 0; i < kSgT * kSgList / kSgThreads; ++i) sm.g[tid + i * kSgThreads] = f.gx[i];
  if (tid < kSgT) sm.ry[tid] = f.ry;
}

// One work item: utterance n, the 64 columns from v0, frame range sk.
template <int KP, bool V4>
DEV void sg_item(const SimpleArgs& a, int splits, SgSmem<KP>& sm, int v0, int sk, int n) {
  constexpr int K = SgSmem<KP>::K;
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V, blank = a.b.blank;
  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, g4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // (uniform: the block guards below are scalar)
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  const int kn = (Un + 1 + 15) / 16 * 16;  // contraction length of d am; u blocks of d lm = kn / 16
  const float sc = a.scale ? a.scale[n] : 1.f;
  // setup: zeroed W tile (columns past ldw stay zero), symbols, e^{lm - m_l}
  for (int i = tid; i < kSgT * K; i += kSgThreads) sm.wt[i] = 0.f;
  for (int u = tid; u < KP; u += kSgThreads) {
    bool ok = true;
    sm.sym[u] = (u < Un) ? symbol_at(a.b, n, u, V, ok) : -1;
  }
  for (int q = tid; q < KP * 16; q += kSgThreads) {
    const int u = q / 16, c = 4 * (q % 16), v = v0 + c;
    const bool row = u <= Un;
    const float* lr = a.lm + ((size_t)n * U1 + (row ? u : 0)) * V;
    const float ml = row ? a.m_l[(size_t)n * U1 + u] : 0.f;
    float x[4];
    if (row && (V & 3) == 0 && v + 4 <= V) {
      const float4 q4 = *reinterpret_cast<const float4*>(lr + v);
      x[0] = q4.x; x[1] = q4.y; x[2] = q4.z; x[3] = q4.w;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = (row && v + j < V) ? lr[v + j] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) sm.elT[(c + j) * K + u] = (row && v + j < V) ? __expf(x[j] - ml) : 0.f;
  }
  __syncthreads();
  // the targets that fall in the columns, ascending u (ballot compaction)
  {
    const int y = (tid < Un) ? sm.sym[tid] : -1;  // U_n < KP <= kSgThreads
    const bool hit = y >= v0 && y < v0 + kSgV;
    const uint64_t bal = __ballot(hit);
    if (lane == 0) sm.cnt[wave] = __popcll(bal);
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += sm.cnt[w];
    if (hit) {
      const int k = base + __popcll(bal & ((1ull << lane) - 1));
      sm.lu[k] = tid;
      sm.ly[k] = y;
    }
    __syncthreads();
  }
  int nm = 0;
#pragma unroll
  for (int w = 0; w < kSgWaves; ++w) nm += sm.cnt[w];
  const int nml = min(nm, kSgList);
  const int tb = wave & 1, vb0 = (wave >> 1) * kSgDam;  // d am blocks
  const int lvb = wave & 3, ug = wave >> 2;              // d lm column block and u-block group
  // the list entries whose symbol is the lane's d am column j (bit k of KP)
  constexpr int MW = (KP + 63) / 64;
  uint64_t mk[kSgDam][MW];
#pragma unroll
  for (int j = 0; j < kSgDam; ++j)
#pragma unroll
    for (int w = 0; w < MW; ++w) mk[j][w] = 0;
  for (int k = 0; k < nm; ++k) {  // (words picked by compares: no indexing of the register array)
    const int y = sm.ly[k];
#pragma unroll
    for (int j = 0; j < kSgDam; ++j)
#pragma unroll
      for (int w = 0; w < MW; ++w)
        if (y == v0 + 16 * (vb0 + j) + l16 && (k >> 6) == w) mk[j][w] |= 1ull << (k & 63);
  }
  // frame steps of this range (rows up to T: those past T_n get zeros)
  SgSrc src;
  src.wt = make_rsrc(a.Wt + (size_t)n * T * a.ldw, (size_t)T * a.ldw * 4);
  src.am = make_rsrc(a.am + (size_t)n * T * V, (size_t)T * V * 4);
  src.ma = make_rsrc(a.m_a + (size_t)n * T, (size_t)T * 4);
  src.gx = make_rsrc(a.gx + (size_t)n * T * U1, (size_t)T * U1 * 4);
  src.ry = make_rsrc(a.ry + (size_t)n * T, (size_t)T * 8);
  src.ldw = a.ldw;
  src.V = V;
  src.U1 = U1;
  src.Tn = Tn;
  const Rsrc gout = make_rsrc(a.am_grad + (size_t)n * T * V, (size_t)T * V * 4);
  const int nsteps = (T + kSgT - 1) / kSgT, per = (nsteps + splits - 1) / splits;
  const int s0 = sk * per, s1 = min(nsteps, s0 + per);
  constexpr int NUB = KP / 16 / kSgUg;  // d lm u blocks per wave (u block ug + kSgUg i)
  static_assert(KP % 64 == 0, "d am reads its fragments in batches of 64 rows");
  floatx4 accl[NUB];
#pragma unroll
  for (int i = 0; i < NUB; ++i) accl[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  SgPrefetch f;
  if (s0 < s1) sg_load<KP, V4>(src, s0 * kSgT, v0, nml, sm.lu, f);
  for (int st = s0; st < s1; ++st) {
    const int t0 = st * kSgT;
    sg_barrier();  // the previous step's LDS reads are done
    sg_store<KP>(sm, f, t0, v0, Tn, V, a.ldw);
    sg_barrier();
    // the next step's loads, in flight during this step's MFMAs and stores
    if (st + 1 < s1) sg_load<KP, V4>(src, t0 + kSgT, v0, nml, sm.lu, f);
    const bool live = t0 < Tn;
    floatx4 accd[kSgDam];
#pragma unroll
    for (int j = 0; j < kSgDam; ++j) accd[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (live) {
      // d am: W rows of the wave's 16 frames against e^{lm - m_l} columns,
      // over the utterance's kn rows in batches of 64 (the batch's fragments
      // read first; KP is a multiple of 64, so they are inside the rows)
#pragma unroll
      for (int kb = 0; kb < KP; kb += 64) {
        if (kb < kn) {
          floatx4 fa[4], fb[4][kSgDam];
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4) {
            const int kk = kb + 16 * s4;
            fa[s4] = *reinterpret_cast<const floatx4*>(&sm.wt[(16 * tb + l16) * K + kk + 4 * g4]);
#pragma unroll
            for (int j = 0; j < kSgDam; ++j)
              fb[s4][j] = *reinterpret_cast<const floatx4*>(&sm.elT[(16 * (vb0 + j) + l16) * K + kk + 4 * g4]);
          }
#pragma unroll
          for (int s4 = 0; s4 < 4; ++s4)
            if (kb + 16 * s4 < kn) {
#pragma unroll
              for (int j = 0; j < kSgDam; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                  accd[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[s4][q], fb[s4][j][q], accd[j], 0, 0, 0);
            }
        }
      }
      // d lm: W^T (u rows) against e^{am - m_a} of the wave's 16 columns; the
      // A fragment's 4 frames are one per row of wt (k-permuted like B). All
      // fragments of a 16-frame half are read first (rows past kn too: they
      // are inside wt), then the MFMAs of the u blocks that hold rows.
#pragma unroll
      for (int kk = 0; kk < kSgT; kk += 16) {
        const floatx4 fb = *reinterpret_cast<const floatx4*>(&sm.eaT[(16 * lvb + l16) * kSgTS + kk + 4 * g4]);
        float fa[NUB][4];
#pragma unroll
        for (int i = 0; i < NUB; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) fa[i][q] = sm.wt[(kk + 4 * g4 + q) * K + 16 * (ug + kSgUg * i) + l16];
#pragma unroll
        for (int i = 0; i < NUB; ++i)
          if (16 * (ug + kSgUg * i) < kn) {  // (a guard, not an exit: the loop stays fully unrolled)
#pragma unroll
            for (int q = 0; q < 4; ++q) accl[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][q], fb[q], accl[i], 0, 0, 0);
          }
      }
    }
    // d am epilogue: e^{am - m_a} * acc, minus gx at the targets (ascending
    // u) and the blank column's row sum of gy
    float res[kSgDam][4];
#pragma unroll
    for (int j = 0; j < kSgDam; ++j) {
      const floatx4 ea = *reinterpret_cast<const floatx4*>(&sm.eaT[(16 * (vb0 + j) + l16) * kSgTS + 16 * tb + 4 * g4]);
#pragma unroll
      for (int r = 0; r < 4; ++r) res[j][r] = ea[r] * accd[j][r];
    }
    if (live) {
      for (int k0 = 0; k0 < nm; k0 += kSgList) {
        if (k0 > 0) {  // more targets than one gather round holds: the next ones, synchronously
          sg_barrier();
          for (int q = tid; q < kSgT * kSgList; q += kSgThreads) {
            const int k = k0 + q / kSgT, t = t0 + q % kSgT;
            sm.g[q] = (k < nm && t < Tn) ? a.gx[((size_t)n * T + t) * U1 + sm.lu[k]] : 0.f;
          }
          sg_barrier();
        }
#pragma unroll
        for (int j = 0; j < kSgDam; ++j) {
          uint64_t word = 0;
#pragma unroll
          for (int w = 0; w < MW; ++w) word = (w == (k0 >> 6)) ? mk[j][w] : word;
          uint32_t bits = (uint32_t)(word >> (k0 & 63));
          while (bits) {  // the lane's targets in ascending u
            const int k = __builtin_ctz(bits);
            bits &= bits - 1;
#pragma unroll
            for (int r = 0; r < 4; ++r) res[j][r] -= sm.g[k * kSgT + 16 * tb + 4 * g4 + r];
          }
        }
      }
#pragma unroll
      for (int j = 0; j < kSgDam; ++j)
        if (v0 + 16 * (vb0 + j) + l16 == blank)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int tl = 16 * tb + 4 * g4 + r;
            if (t0 + tl < Tn) res[j][r] = (float)((double)res[j][r] - sm.ry[tl]);
          }
    }
#pragma unroll
    for (int j = 0; j < kSgDam; ++j) {
      const int v = v0 + 16 * (vb0 + j) + l16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {  // rows past T fall outside the resource
        const int t = t0 + 16 * tb + 4 * g4 + r;
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint((t < Tn) ? sc * res[j][r] : 0.f), gout,
                                              (int)(v < V ? (uint32_t)(t * V + v) * 4u : kOob), 0, 0);
      }
    }
  }
  // d lm: the range's partial sums, or (one range) the finished gradient
  const int v = v0 + 16 * lvb + l16;
  if (v >= V) return;
#pragma unroll
  for (int i = 0; i < NUB; ++i) {
    const int ub = ug + kSgUg * i;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int u = 16 * ub + 4 * g4 + r;
      if (u >= U1) continue;
      if (splits > 1) {
        if (u <= Un) a.lpart[(((size_t)sk * a.b.N + n) * U1 + u) * V + v] = accl[i][r];
        continue;
      }
      float out = 0.f;
      if (u <= Un) {
        const float d = sm.elT[(16 * lvb + l16) * K + u] * accl[i][r];
        double gd = (double)d;
        if (v == sm.sym[u]) gd -= a.Gx[(size_t)n * U1 + u];
        if (v == blank) gd -= a.Gy[(size_t)n * U1 + u];
        out = (float)(sc * gd);
      }
      a.lm_grad[((size_t)n * U1 + u) * V + v] = out;
    }
  }
}

// Work items in order (column tiles of an utterance's frame range next to
// each other); a grid smaller than the item count loops over them.
template <int KP, bool V4>
__global__ __launch_bounds__(kSgThreads) void simple_grad_kernel(SimpleArgs a, int splits, int items) {
  __shared__ SgSmem<KP> sm;
  const int nvt = (a.V + kSgV - 1) / kSgV;
  for (int it = blockIdx.x; it < items; it += gridDim.x) {
    const int vt = it % nvt, rest = it / nvt;
    sg_item<KP, V4>(a, splits, sm, vt * kSgV, rest % splits, rest / splits);
    __syncthreads();  // the next item rewrites the LDS
  }
}

__global__ void fill_f32_kernel(float* p, size_t n, float v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

}  // namespace

hipError_t launch_rowmax(const SimpleArgs& a, hipStream_t s) {
  const int N = a.b.N, T = a.b.T, U1 = a.b.U + 1;
  {
    RNNT_PROF(s, "rowmax");
    hipLaunchKernelGGL(rowmax_kernel, dim3((N * (T + U1) + 3) / 4), dim3(256), 0, s, a.am, a.lm, N, T, U1, a.V, a.b,
                       a.m_a, a.m_l);
  }
  return hipGetLastError();
}

// Split counts: enough K ranges for about 1024 workgroups, each range at
// least two K-steps long.
static int split_count(long long tiles, int K, int bk) {
  long long sk = (1024 + tiles - 1) / tiles;
  const long long most = (K + 2 * bk - 1) / (2 * bk);
  if (sk > most) sk = most;
  if (sk > 16) sk = 16;
  return sk < 1 ? 1 : (int)sk;
}

template <class Cfg>
static int normalizer_splits_cfg(int N, int T, int U, int V) {
  const long long tiles = (long long)N * ((T + Cfg::BM - 1) / Cfg::BM) * ((U + 1 + Cfg::BN - 1) / Cfg::BN);
  return split_count(tiles, V, Cfg::BK);
}
int normalizer_splits(int N, int T, int U, int V) {
  return V >= kSimpleBigV ? normalizer_splits_cfg<BigCfg>(N, T, U, V) : normalizer_splits_cfg<NormCfg>(N, T, U, V);
}

template <class Cfg>
static int dlm_splits_cfg(int N, int T, int U, int V) {
  const long long tiles = (long long)N * ((U + 1 + Cfg::BM - 1) / Cfg::BM) * ((V + Cfg::BN - 1) / Cfg::BN);
  return split_count(tiles, T, Cfg::BK);
}
int dlm_splits(int N, int T, int U, int V) {
  return V >= kSimpleBigV ? dlm_splits_cfg<BigCfg>(N, T, U, V) : dlm_splits_cfg<DlmCfg>(N, T, U, V);
}

// Frame ranges of the fused d am / d lm kernel: enough for about
// kSgBlocks workgroups (one per CU: the kernel runs beside the pruned stage
// on a second stream, and more workgroups measured no faster per step);
// 0 where the kernel does not apply.
constexpr int kSgBlocks = 256;
int simple_grad_splits(int N, int T, int U, int V) {
  // one utterance's am must stay below 2^31 bytes (32-bit buffer offsets)
  if (U + 1 > kSgMaxU1 || (long long)T * V * 4 >= (1ll << 31)) return 0;
  const long long base = (long long)N * ((V + kSgV - 1) / kSgV);
  const int steps = (T + kSgT - 1) / kSgT;
  long long s = (kSgBlocks + base - 1) / base;
  if (s > steps) s = steps;
  return s < 1 ? 1 : (int)s;
}

template <int KP>
static void launch_normalizer_fused(const SimpleArgs& a, bool v4, unsigned blocks, hipStream_t s) {
  if (v4) hipLaunchKernelGGL((normalizer_fused_kernel<KP, true>), dim3(blocks), dim3(kNfThreads), 0, s, a);
  else hipLaunchKernelGGL((normalizer_fused_kernel<KP, false>), dim3(blocks), dim3(kNfThreads), 0, s, a);
}

hipError_t launch_normalizer(const SimpleArgs& a, hipStream_t s) {
  const int T = a.b.T, U1 = a.b.U + 1;
  const long long tiles = (long long)a.b.N * ((T + kNfT - 1) / kNfT);
  const int chunks = (a.V + kNfV - 1) / kNfV;
  if (U1 <= kNfMaxU1 && (long long)T * a.V * 4 < (1ll << 31) && (long long)U1 * a.V * 4 < (1ll << 31) &&
      (tiles >= 192 || chunks <= 16)) {
    // every u of 32 frames per workgroup, the epilogue in the same kernel;
    // u extent as in the fused gradient kernel. Its workgroups run the whole
    // of V in sequence: with far fewer tiles than CUs and a long V (160
    // tiles, 79 chunks of 64 at V = 5000: 112 against 108 us) the split
    // kernels below are faster; with 248 tiles and 125 chunks (V = 8000,
    // U + 1 <= 301) this one is (550 against 756 us).
    const size_t blocks = (size_t)a.b.N * ((T + kNfT - 1) / kNfT) +
                          (size_t)a.b.N * lattice_fill_blocks(T, a.b.U, kNfFill * kNfThreads);
    const bool v4 = (a.V & 3) == 0;
    RNNT_PROF(s, "normalizer");
    if (U1 <= 64) launch_normalizer_fused<64>(a, v4, (unsigned)blocks, s);
    else if (U1 <= 128) launch_normalizer_fused<128>(a, v4, (unsigned)blocks, s);
    else if (U1 <= 192) launch_normalizer_fused<192>(a, v4, (unsigned)blocks, s);
    else launch_normalizer_fused<kNfMaxU1>(a, v4, (unsigned)blocks, s);
    return hipGetLastError();
  }
  {
    RNNT_PROF(s, "normalizer");
    if (a.V >= kSimpleBigV) {
      const dim3 grid((T + BigCfg::BM - 1) / BigCfg::BM, (U1 + BigCfg::BN - 1) / BigCfg::BN, a.b.N * a.nsplit);
      hipLaunchKernelGGL(normalizer_kernel<BigCfg>, grid, dim3(BigCfg::NT), 0, s, a);
    } else {
      const dim3 grid((T + NormCfg::BM - 1) / NormCfg::BM, (U1 + NormCfg::BN - 1) / NormCfg::BN, a.b.N * a.nsplit);
      hipLaunchKernelGGL(normalizer_kernel<NormCfg>, grid, dim3(NormCfg::NT), 0, s, a);
    }
  }
  // tiles of the rectangle's nodes, then the cells of the diagonal-major copies
  const int nodes = epi_nodes(a.b.N, T, U1);
  const int FT = epi_tile_frames(lattice_rows_per_lane(U1), nodes);
  const size_t blocks =
      (size_t)a.b.N * ((T + FT - 1) / FT) + (size_t)a.b.N * lattice_fill_blocks(T, a.b.U, kEpiThreads * nodes);
  {
    RNNT_PROF(s, "normalizer_epi");
    if (nodes == 4) hipLaunchKernelGGL(normalizer_epi_kernel<4>, dim3((unsigned)blocks), dim3(kEpiThreads), 0, s, a);
    else hipLaunchKernelGGL(normalizer_epi_kernel<1>, dim3((unsigned)blocks), dim3(kEpiThreads), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_smoothing_stats(const SimpleArgs& a, hipStream_t s) {
  if (a.lm_only == 0.f && a.am_only == 0.f) return hipSuccess;
  const int N = a.b.N, T = a.b.T, U1 = a.b.U + 1;
  {
    RNNT_PROF(s, "smooth_stats");
    hipLaunchKernelGGL(lm_lse_kernel, dim3((N * U1 + 3) / 4), dim3(256), 0, s, a);
    hipLaunchKernelGGL(lm_avg_kernel, dim3((a.V + 255) / 256, N), dim3(256), 0, s, a);
    hipLaunchKernelGGL(ac_lse_kernel, dim3((N * T + 3) / 4), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// u extent KP: the smallest of 64, 128, 192, 320 that holds U + 1 (LDS and
// the d lm accumulators scale with it)
template <int KP>
static void launch_simple_grad(const SimpleArgs& a, int gs, bool v4, hipStream_t s) {
  // one workgroup per item (grids capped at 128-256 workgroups, leaving CUs
  // to the pruned stage, measured no faster at the stress and long shapes)
  const int items = a.b.N * gs * ((a.V + kSgV - 1) / kSgV);
  const dim3 grid(items);
  if (v4) hipLaunchKernelGGL((simple_grad_kernel<KP, true>), grid, dim3(kSgThreads), 0, s, a, gs, items);
  else hipLaunchKernelGGL((simple_grad_kernel<KP, false>), grid, dim3(kSgThreads), 0, s, a, gs, items);
}

hipError_t launch_simple_grads(const SimpleArgs& a, hipStream_t s) {
  const int T = a.b.T, U1 = a.b.U + 1, V = a.V;
  {
    RNNT_PROF(s, "simple_colsum");
    hipLaunchKernelGGL(colsum_kernel, dim3((a.b.N * U1 + 255) / 256), dim3(256), 0, s, a);
  }
  if (a.lm_only != 0.f || a.am_only != 0.f) {
    RNNT_PROF(s, "smooth_grad_stats");
    hipLaunchKernelGGL(ac_colsum_kernel, dim3((V + 255) / 256, a.b.N), dim3(256), 0, s, a);
    hipLaunchKernelGGL(lm_s_kernel, dim3((a.b.N * U1 + 3) / 4), dim3(256), 0, s, a);
  }
  const bool big = V >= kSimpleBigV;
  const int gs = simple_grad_splits(a.b.N, T, a.b.U, V);
  if (gs > 0 && a.am_grad && a.lm_grad && a.lm_only == 0.f && a.am_only == 0.f) {
    {
      RNNT_PROF(s, "simple_grad");
      const bool v4 = (V & 3) == 0;
      if (U1 <= 64) launch_simple_grad<64>(a, gs, v4, s);
      else if (U1 <= 128) launch_simple_grad<128>(a, gs, v4, s);
      else if (U1 <= 192) launch_simple_grad<192>(a, gs, v4, s);
      else launch_simple_grad<kSgMaxU1>(a, gs, v4, s);
    }
    if (gs > 1) {
      SimpleArgs e = a;
      e.lsplit = gs;  // the workspace holds max(dlm_splits, simple_grad_splits) partial sets
      const size_t groups = (size_t)a.b.N * U1 * ((V + 3) / 4);
      RNNT_PROF(s, "simple_dlm_epi");
      hipLaunchKernelGGL(dlm_epi_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, s, e);
    }
    return hipGetLastError();
  }
  if (a.am_grad) {
    RNNT_PROF(s, "simple_dam");
    if (big) {
      const dim3 grid((T + BigCfg::BM - 1) / BigCfg::BM, (V + BigCfg::BN - 1) / BigCfg::BN, a.b.N);
      hipLaunchKernelGGL(dam_kernel<BigCfg>, grid, dim3(BigCfg::NT), 0, s, a);
    } else {
      const dim3 grid((T + DamCfg::BM - 1) / DamCfg::BM, (V + DamCfg::BN - 1) / DamCfg::BN, a.b.N);
      hipLaunchKernelGGL(dam_kernel<DamCfg>, grid, dim3(DamCfg::NT), 0, s, a);
    }
  }
  if (a.lm_grad) {
    {
      RNNT_PROF(s, "simple_dlm");
      if (big) {
        const dim3 grid((U1 + BigCfg::BM - 1) / BigCfg::BM, (V + BigCfg::BN - 1) / BigCfg::BN, a.b.N * a.lsplit);
        hipLaunchKernelGGL(dlm_kernel<BigCfg>, grid, dim3(BigCfg::NT), 0, s, a);
      } else {
        const dim3 grid((U1 + DlmCfg::BM - 1) / DlmCfg::BM, (V + DlmCfg::BN - 1) / DlmCfg::BN, a.b.N * a.lsplit);
        hipLaunchKernelGGL(dlm_kernel<DlmCfg>, grid, dim3(DlmCfg::NT), 0, s, a);
      }
    }
    const size_t groups = (size_t)a.b.N * U1 * ((V + 3) / 4);
    {
      RNNT_PROF(s, "simple_dlm_epi");
      hipLaunchKernelGGL(dlm_epi_kernel, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, s, a);
    }
  }
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  {
    RNNT_PROF(s, "fill");
    hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  }
  return hipGetLastError();
}
