// Stage 4a/4c: the full joiner evaluated only on the pruned (t, u) pairs
// (Sec. 3.2, Fig. 1(b)) and its backward pass.
//
// Rows. Every valid frame of the batch contributes S consecutive rows
// m = (frame_off[n] + t) * S + s (padding frames take no rows), so the GEMMs
// see one dense M = S * sum_n T_n dimension. A prep kernel writes, per row,
// the offsets of enc[n,t] and dec[n,u] (u = ranges[n,t,s]), the target symbol
// y_{u+1} (-1 at u = U_n, -2 when it lies outside [0, V)) and the output index
// n*T*S + t*S + s (-1 when the slot is absent, u > U_n).
//
// Forward (per chunk of rows): h = tanh(enc + dec) once per element into a
// chunk buffer, then logits = h W + bias on MFMA (fp32 16x16x4 or bf16
// 16x16x32, fp32 accumulation), both operands staged without conversion.
// The epilogue reduces every (row, 64-column slice) to (max, sum exp) and
// captures the target and blank logits; a combine kernel turns them into
// lse, px = logit[y_{u+1}] - lse and py = logit[blank] - lse. The logits
// reach memory only when the caller asks for them ([N, T, S, V], the size
// the method's memory scales with).
//
// Backward (per chunk of at most a fixed number of rows, independent of the
// batch, so that d(logits), h and the d dec pieces are held for one chunk
// only and no [N, T, S, V] array exists):
//   1. dl = sc * ((gx+gy) softmax - gx [v=y] - gy [v=blank]) (log-softmax
//      backward) by recomputing h and the logits GEMM (or, when the caller
//      kept the forward's logits, by a streaming kernel over them); write the
//      chunk and column sums (db);
//   2. dh = dl W^T, dpre = dh (1 - h^2)  (tanh backward), kept in LDS: the
//      epilogue sums it into d enc[n,t] = sum_s dpre(row(t,s)) for the frames
//      inside the 128-row tile, and into per-tile pieces of the frames the
//      tile cuts and of d dec[n,u] = sum over the (t,s) with p_t + s = u;
//   3. dW += h^T dl with split-K partial sums;
//   4. the d dec pieces of the chunk are added to d dec in tile order;
// then a tail kernel adds the d enc pieces in tile order and sums dW and db
// over their partials, all in a fixed order.
#include "gemm.h"
#include "kernels.h"
#include "prof.h"

namespace {

// 8 waves in a 4 x 2 grid (32 x 64 wave tiles): about 100 registers per
// lane, so two workgroups (four waves per SIMD) share a CU.
constexpr int kGemmThreads = 512;
// fp32: operands staged through registers (the forward forms tanh(enc + dec)
// while staging; dW transposes both operands in registers)
using CfgF = GemmCfg<128, 128, 32, false, 4, 2>;
// bf16: every operand is read k-contiguous (h, d(logits) and their
// transposes, W and its transposed copy) straight into LDS
using CfgB = LdsCfg<128, 128, 64, 4, 2>;
using CfgBw = CfgB;
// bf16 forward at wide vocabularies: 256 x 256 tiles of 16 waves (64 x 64
// wave tiles, one workgroup per CU) read a third fewer operand bytes from
// LDS per MFMA than the 32 x 64 wave tiles; measured 1015 against 831
// TFLOP/s on the main loop at 6941 x 8000 x 768, slower where V gives few
// column tiles (608 against 832 at 16384 x 512 x 512)
using CfgBWide = LdsCfg<256, 256, 64, 4, 4>;
constexpr int kFwdWideV = 2048;
static_assert(CfgBWide::WN == 64, "the forward's partial log-sum-exp slices are 64 columns");
static_assert(CfgF::NT == kGemmThreads && CfgB::NT == kGemmThreads, "joiner GEMM block size");
static_assert(CfgF::WN == 64 && CfgB::WN == 64, "the forward's partial log-sum-exp slices are 64 columns");
static_assert(CfgF::BM == CfgB::BM && CfgF::WGM == CfgB::WGM, "db partial rows per row tile");

template <bool BF>
struct In;
template <>
struct In<false> {
  using T = float;
  using Cfg = CfgF;
};
template <>
struct In<true> {
  using T = uint16_t;
  using Cfg = CfgB;
};

// Whether the forward reads h from a buffer written by the h kernel (bf16:
// its operands go straight into LDS, with no register stage where tanh could
// be formed) or forms it while staging the A tile (fp32: measured ~5 us
// faster per step at the BPE size than a separate h pass).
template <bool BF>
constexpr bool kFwdHbuf = BF;

DEV float ld_in(const float* p, size_t i) { return p[i]; }
DEV float ld_in(const uint16_t* p, size_t i) { return bf2f(p[i]); }

// ---------------------------------------------------------------------------
// Operand loads through buffer resources (make_rsrc, kOob: see common.h). A
// masked-out lane (row past the end, absent slot, k beyond K) loads from kOob
// and reads zeros instead of taking a divergent branch, so the loads of a
// K-step issue back to back. Every operand array is below 2^31 bytes
// (checked by the entry points).
// ---------------------------------------------------------------------------
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int W>
DEV void buf_words(Rsrc r, uint32_t off, uint32_t* w) {
  if constexpr (W == 4) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  } else if constexpr (W == 2) {
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
    w[0] = v.x; w[1] = v.y;
  } else {
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)(off + 4 * i), 0, 0);
  }
}

// ---------------------------------------------------------------------------
// Raw operand registers: N elements of TIn kept as 32-bit words until the
// loader's finish step, so that no conversion waits on an in-flight load.
// ---------------------------------------------------------------------------
template <typename TIn, int N>
struct RawVec {
  static constexpr int W = (N * (int)sizeof(TIn) + 3) / 4;
  uint32_t w[W];
};

// How a row segment may be loaded (uniform over a launch):
//   kSegVector: rows are 16-byte aligned and every segment is entirely inside
//               or entirely outside its row: one vector load;
//   kSegWords:  32-bit words, each inside or outside (fp32, or bf16 rows of
//               even length);
//   kSegElems:  bf16 element by element (odd row length).
enum SegMode { kSegVector = 0, kSegWords = 1, kSegElems = 2 };

template <typename TIn>
DEV int seg_mode(int row_len, int seg) {
  if (row_len % seg == 0) return kSegVector;
  return (sizeof(TIn) == 4 || row_len % 2 == 0) ? kSegWords : kSegElems;
}

// Loads the N elements at byte offset `off`, of which the first `nvalid` are
// inside the row (nvalid <= 0: none; zeros beyond).
template <typename TIn, int N>
DEV void raw_load(Rsrc r, uint32_t off, int nvalid, int mode, RawVec<TIn, N>& out) {
  constexpr int W = RawVec<TIn, N>::W;
  if (mode == kSegVector) {
    buf_words<W>(r, nvalid > 0 ? off : kOob, out.w);
  } else if (sizeof(TIn) == 4 || mode == kSegWords) {
    constexpr int EPW = 4 / (int)sizeof(TIn);  // elements per word
#pragma unroll
    for (int i = 0; i < W; ++i)
      out.w[i] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)(EPW * i < nvalid ? off + 4 * i : kOob), 0, 0);
  } else {
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(r, (int)(2 * i < nvalid ? off + 4 * i : kOob), 0, 0);
      const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(r, (int)(2 * i + 1 < nvalid ? off + 4 * i + 2 : kOob), 0, 0);
      out.w[i] = lo | (hi << 16);
    }
  }
}

template <typename TIn, int N>
DEV void raw_to_float(const RawVec<TIn, N>& r, float (&v)[N]) {
  if constexpr (sizeof(TIn) == 4) {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = __uint_as_float(r.w[i]);
  } else {
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      v[2 * i] = __uint_as_float(r.w[i] << 16);
      v[2 * i + 1] = __uint_as_float(r.w[i] & 0xffff0000u);
    }
  }
}

DEV float4 f4add(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }

// ---------------------------------------------------------------------------
// Operand sources
// ---------------------------------------------------------------------------

// enc / dec resources of a launch (row offsets from rowinfo are element offsets).
template <typename TIn>
struct EncDec {
  Rsrc enc, dec;
  DEV EncDec(const JoinerArgs& a)
      : enc(make_rsrc(a.enc, (size_t)a.b.N * a.b.T * a.J * sizeof(TIn))),
        dec(make_rsrc(a.dec, (size_t)a.b.N * (a.b.U + 1) * a.J * sizeof(TIn))) {}
};

// A(m, j) = tanh(enc[row] + dec[row]) formed while staging (rowinfo of the
// tile's rows in LDS): the fp32 forward, where the tanh work hides under the
// MFMAs and a separate h pass would only add its HBM traffic.
template <class Cfg, typename TIn>
struct HSrcKC {
  struct Raw {
    RawVec<TIn, Cfg::KV> e, d;
  };
  EncDec<TIn> ed;
  const int4* ri;
  int J;
  DEV void kc_load(int row, int k, Raw& r) const {
    const int4 q = ri[row];
    const int n = (q.w >= 0 && k < J) ? Cfg::KV : 0;
    raw_load(ed.enc, (uint32_t)(q.x + k) * sizeof(TIn), n, kSegVector, r.e);
    raw_load(ed.dec, (uint32_t)(q.y + k) * sizeof(TIn), n, kSegVector, r.d);
  }
  DEV void kc_finish(const Raw& r, float (&v)[Cfg::KV]) const {
    float e[Cfg::KV], d[Cfg::KV];
    raw_to_float(r.e, e);
    raw_to_float(r.d, d);
#pragma unroll
    for (int i = 0; i < Cfg::KV; ++i) v[i] = fast_tanh(e[i] + d[i]);
  }
};

// A(m, j) = h[m - cm0][j] from a chunk buffer of h = tanh(enc + dec) (zero
// rows for absent slots).
template <class Cfg>
struct HbufSrcKC {
  static constexpr bool kDirect = true;
  using T = typename Cfg::T;
  using Raw = RawVec<T, Cfg::KV>;
  Rsrc h;
  int m0, cm0, mend, J;
  DEV void kc_load(int row, int k, Raw& r) const {
    const int m = m0 + row;
    const int n = (m < mend && k < J) ? Cfg::KV : 0;
    raw_load(h, (uint32_t)((m - cm0) * J + k) * sizeof(T), n, kSegVector, r);
  }
  DEV void kc_finish(const Raw& r, float (&v)[Cfg::KV]) const { raw_to_float(r, v); }
};

// B(j, v) = W[j][v]: global row-contiguous along v.
// MODE = seg_mode<TIn>(V, NV), fixed per launch so that the loads compile
// without branches.
template <class Cfg, typename TIn, int MODE>
struct WSrcMNC {
  static constexpr bool kDirect = true;
  static constexpr int NV = 16 / Cfg::KV;
  static constexpr int mode = MODE;
  using Raw = RawVec<TIn, NV>;
  Rsrc W;
  int v0, V, J;
  DEV WSrcMNC(const JoinerArgs& a, int v0_)
      : W(make_rsrc(a.W, (size_t)a.J * a.V * sizeof(TIn))), v0(v0_), V(a.V), J(a.J) {}
  DEV void mnc_load(int k, int col, Raw& r) const {
    const int c = v0 + col;
    const int n = (k < J) ? V - c : 0;
    raw_load(W, (uint32_t)(k * V + c) * sizeof(TIn), n, mode, r);
  }
  DEV void mnc_finish(const Raw& r, float (&v)[NV]) const { raw_to_float(r, v); }
};

// A(m, v) = dl[m][v] from the chunk buffer (rows padded to ldl with zeros).
template <class Cfg>
struct DlSrcKC {
  static constexpr bool kDirect = true;
  using T = typename Cfg::T;
  using Raw = RawVec<T, Cfg::KV>;
  Rsrc dl;  // row (m - cm0)
  int m0, cm0, mend, ldl;
  DEV void kc_load(int row, int k, Raw& r) const {
    const int m = m0 + row;
    const int n = (m < mend && k < ldl) ? Cfg::KV : 0;
    raw_load(dl, (uint32_t)((m - cm0) * ldl + k) * sizeof(T), n, kSegVector, r);
  }
  DEV void kc_finish(const Raw& r, float (&v)[Cfg::KV]) const { raw_to_float(r, v); }
};

// B(v, j) = W[j][v]: global k-contiguous along v for each j.
// MODE = seg_mode<TIn>(V, KV), fixed per launch.
template <class Cfg, typename TIn, int MODE>
struct WtSrcKC {
  static constexpr bool kDirect = true;
  static constexpr int mode = MODE;
  using Raw = RawVec<TIn, Cfg::KV>;
  Rsrc W;
  int j0, J, V, ld;  // ld: row stride of W, or of its zero-padded copy
  DEV WtSrcKC(const JoinerArgs& a, int j0_)
      : W(make_rsrc(a.wpad ? a.wpad : a.W, (size_t)a.J * (a.wpad ? a.ldl : a.V) * sizeof(TIn))),
        j0(j0_), J(a.J), V(a.V), ld(a.wpad ? a.ldl : a.V) {}
  DEV void kc_load(int row, int k, Raw& r) const {
    const int j = j0 + row;
    const int n = (j < J) ? V - k : 0;
    raw_load(W, (uint32_t)(j * ld + k) * sizeof(TIn), n, mode, r);
  }
  DEV void kc_finish(const Raw& r, float (&v)[Cfg::KV]) const { raw_to_float(r, v); }
};

// A(j, m) = h(m, j) from the chunk's hbuf [rows, J] (j-contiguous).
template <class Cfg>
struct HbufSrcMNC {
  static constexpr bool kDirect = true;
  using T = typename Cfg::T;
  static constexpr int NV = 16 / Cfg::KV;
  using Raw = RawVec<T, NV>;
  Rsrc h;
  int cm0, mend, j0, J;
  DEV void mnc_load(int k, int col, Raw& r) const {
    const int j = j0 + col;
    const int n = (k < mend && j < J) ? NV : 0;
    raw_load(h, (uint32_t)((k - cm0) * J + j) * sizeof(T), n, kSegVector, r);
  }
  DEV void mnc_finish(const Raw& r, float (&v)[NV]) const { raw_to_float(r, v); }
};

// B(m, v) = dl[m][v]: global row-contiguous along v.
template <class Cfg>
struct DlSrcMNC {
  static constexpr bool kDirect = true;
  using T = typename Cfg::T;
  static constexpr int NV = 16 / Cfg::KV;
  using Raw = RawVec<T, NV>;
  Rsrc dl;
  int cm0, mend, v0, ldl;
  DEV void mnc_load(int k, int col, Raw& r) const {
    const int c = v0 + col;
    const int n = (k < mend && c < ldl) ? NV : 0;
    raw_load(dl, (uint32_t)((k - cm0) * ldl + c) * sizeof(T), n, kSegVector, r);
  }
  DEV void mnc_finish(const Raw& r, float (&v)[NV]) const { raw_to_float(r, v); }
};

DEV float bias_at(const void* bias, int bf16, int v) {
  if (!bias) return 0.f;
  return bf16 ? bf2f(reinterpret_cast<const uint16_t*>(bias)[v]) : reinterpret_cast<const float*>(bias)[v];
}

// The bias of this lane's FN output columns v0 + tile_col(j) (0 past V or
// without a bias), with branch-free buffer loads: issued ahead of the main
// loop (bf16) or right after it (fp32, whose main loop has no registers to
// spare), and waited for once with wait_vmem() before the epilogue. A load
// inside a per-column branch would instead make the compiler wait again at
// every later branch, and with it for every store issued in between.
template <class Cfg, bool BF>
DEV void bias_cols(const JoinerArgs& a, int v0, float (&bj)[Cfg::FN]) {
  constexpr uint32_t esz = BF ? 2 : 4;
  const Rsrc rb = make_rsrc(a.bias, a.bias ? (size_t)a.V * esz : 0);
#pragma unroll
  for (int j = 0; j < Cfg::FN; ++j) {
    const int col = v0 + tile_col<Cfg>(j);
    const uint32_t off = col < a.V ? (uint32_t)col * esz : kOob;
    if constexpr (BF) bj[j] = bf2f(__builtin_amdgcn_raw_buffer_load_b16(rb, (int)off, 0, 0));
    else bj[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rb, (int)off, 0, 0));
  }
}

// ---------------------------------------------------------------------------
// Prep: per-utterance frame offsets and per-row info.
// ---------------------------------------------------------------------------
// W [J, V] bf16 copied into wpad [J, ldl] with zeros after column V: one
// 8-element group per thread.
DEV void prep_wpad(const JoinerArgs& a, int b) {
  const int gpr = a.ldl / 8;
  const int g = b * 256 + threadIdx.x;
  if (g >= a.J * gpr) return;
  const int j = g / gpr, c = (g - j * gpr) * 8;
  const uint16_t* src = reinterpret_cast<const uint16_t*>(a.W) + (size_t)j * a.V;
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = (c + 2 * q < a.V) ? src[c + 2 * q] : 0u;
    const uint32_t hi = (c + 2 * q + 1 < a.V) ? src[c + 2 * q + 1] : 0u;
    w[q] = lo | (hi << 16);
  }
  *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.wpad) + (size_t)j * a.ldl + c) = make_uint4(w[0], w[1], w[2], w[3]);
}

int prep_wpad_blocks(const JoinerArgs& a) { return a.wpad ? (a.J * (a.ldl / 8) + 255) / 256 : 0; }

// W [J, V] bf16 transposed into wt [V, J], one 64 x 64 tile per block through
// LDS: W read along v (consecutive threads, consecutive v), wt written in
// 16-byte groups of 8 consecutive j (J is a multiple of 8).
constexpr int kWtTile = 64;
DEV void prep_wt(const JoinerArgs& a, int b) {
  __shared__ uint16_t tile[kWtTile][kWtTile + 2];
  const int nvt = (a.V + kWtTile - 1) / kWtTile;
  const int j0 = (b / nvt) * kWtTile, v0 = (b % nvt) * kWtTile;
  const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);
  const int c = threadIdx.x % kWtTile;
  for (int r = threadIdx.x / kWtTile; r < kWtTile; r += 256 / kWtTile) {
    const int j = j0 + r, v = v0 + c;
    tile[r][c] = (j < a.J && v < a.V) ? W[(size_t)j * a.V + v] : (uint16_t)0;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < kWtTile * (kWtTile / 8); q += 256) {
    const int vr = q / (kWtTile / 8), jg = (q % (kWtTile / 8)) * 8;
    const int v = v0 + vr, j = j0 + jg;
    if (v >= a.V || j >= a.J) continue;
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) w[k] = (uint32_t)tile[jg + 2 * k][vr] | ((uint32_t)tile[jg + 2 * k + 1][vr] << 16);
    *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.wt) + (size_t)v * a.J + j) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

int prep_wt_blocks(const JoinerArgs& a) {
  return a.wt ? ((a.J + kWtTile - 1) / kWtTile) * ((a.V + kWtTile - 1) / kWtTile) : 0;
}

__global__ __launch_bounds__(256) void joiner_prep_kernel(JoinerArgs a, int wpad_blocks) {
  __shared__ int s_part[4];
  const int per = (a.b.T * a.S + 255) / 256;  // blocks per utterance: one (t, s) slot per thread
  if ((int)blockIdx.x >= a.b.N * per) {  // blocks after the utterances' copy W for dh, then transpose it
    const int b = blockIdx.x - a.b.N * per;
    if (b < wpad_blocks) prep_wpad(a, b);
    else prep_wt(a, b - wpad_blocks);
    return;
  }
  const int n = blockIdx.x / per, i = (blockIdx.x - n * per) * 256 + threadIdx.x;
  const int T = a.b.T, U1 = a.b.U + 1, S = a.S, J = a.J;
  // frame offset of utterance n: sum of T_q over q < n, the lengths loaded
  // in parallel and summed by a block reduction
  int part = 0;
  for (int q = threadIdx.x; q < n; q += blockDim.x) {
    int Tq, Uq;
    utt_dims(a.b, q, Tq, Uq);
    part += Tq;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) part += __shfl_xor(part, o, 64);
  if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = part;
  __syncthreads();
  const int off = s_part[0] + s_part[1] + s_part[2] + s_part[3];
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  if (i == 0) {
    a.frame_off[n] = off;
    if (n == a.b.N - 1) a.frame_off[a.b.N] = off + Tn;
  }
  if (i >= Tn * S) return;
  const int t = i / S, s = i - t * S;
  const size_t nts = ((size_t)n * T + t) * S + s;
  const int u = a.ranges[nts];
  if (s == 0 && a.frame_nt) {
    a.frame_nt[off + t] = n * T + t;
    a.frame_p[off + t] = u;
  }
  int4 r;
  if (u >= 0 && u <= Un) {
    bool ok = true;
    r.x = (int)(((size_t)n * T + t) * J);
    r.y = (int)(((size_t)n * U1 + u) * J);
    r.z = (u < Un) ? symbol_at(a.b, n, u, a.V, ok) : -1;
    if (!ok) r.z = -2;  // symbol outside [0, V): px is NaN, so the utterance's loss is NaN
    r.w = (int)nts;
  } else {
    r = make_int4(0, 0, -1, -1);
  }
  a.rowinfo[(size_t)(off + t) * S + s] = r;
}

// ---------------------------------------------------------------------------
// h = tanh(enc + dec) of the rows [cm0, min(cm1, M)) into the chunk buffer
// hbuf [rows, J] in the GEMM operand type (zero rows for absent slots):
// kHItems 16-byte groups of J per thread (consecutive threads, consecutive
// groups), whose row info, then enc and dec loads, are issued together; the
// batch's row count M is loaded beside the row info (rows past it hold no
// row info and are skipped).
// ---------------------------------------------------------------------------
constexpr int kHItems = 4;
// Block blk of NT threads of an h pass into hdst (the chunk's rows from cm0).
template <bool BF, int NT>
DEV void h_rows_block(const JoinerArgs& a, void* hdst, int cm0, int cm1, int blk) {
  using TIn = typename In<BF>::T;
  constexpr int KV = 16 / (int)sizeof(TIn);
  const int cpr = a.J / KV;
  const size_t base = (size_t)blk * (NT * kHItems) + threadIdx.x;
  int rr[kHItems], jj[kHItems];
  int4 info[kHItems];
#pragma unroll
  for (int k = 0; k < kHItems; ++k) {
    const size_t i = base + (size_t)k * NT;
    rr[k] = (int)(i / cpr);
    jj[k] = (int)(i - (size_t)rr[k] * cpr) * KV;
    // within the row info array (cm1 <= N*T*S); rows past M are masked below
    info[k] = cm0 + rr[k] < cm1 ? a.rowinfo[cm0 + rr[k]] : make_int4(0, 0, -1, -1);
  }
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  const EncDec<TIn> ed(a);
  RawVec<TIn, KV> e[kHItems], d[kHItems];
#pragma unroll
  for (int k = 0; k < kHItems; ++k) {
    const int n = (cm0 + rr[k] < mend && info[k].w >= 0) ? KV : 0;
    raw_load(ed.enc, (uint32_t)(info[k].x + jj[k]) * sizeof(TIn), n, kSegVector, e[k]);
    raw_load(ed.dec, (uint32_t)(info[k].y + jj[k]) * sizeof(TIn), n, kSegVector, d[k]);
  }
#pragma unroll
  for (int k = 0; k < kHItems; ++k) {
    if (cm0 + rr[k] >= mend) continue;
    float fe[KV], fd[KV], h[KV];
    raw_to_float(e[k], fe);
    raw_to_float(d[k], fd);
#pragma unroll
    for (int q = 0; q < KV; ++q) h[q] = info[k].w >= 0 ? fast_tanh(fe[q] + fd[q]) : 0.f;
    uint4 o;
    if constexpr (BF) {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) w[q] = (uint32_t)f2bf(h[2 * q]) | ((uint32_t)f2bf(h[2 * q + 1]) << 16);
      o = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
      o = make_uint4(__float_as_uint(h[0]), __float_as_uint(h[1]), __float_as_uint(h[2]), __float_as_uint(h[3]));
    }
    *reinterpret_cast<uint4*>(reinterpret_cast<TIn*>(hdst) + (size_t)rr[k] * a.J + jj[k]) = o;
  }
}

template <bool BF>
__global__ __launch_bounds__(256) void joiner_h_kernel(JoinerArgs a, int cm0, int cm1) {
  h_rows_block<BF, 256>(a, a.hbuf, cm0, cm1, blockIdx.x);
}

// The h pass of the next forward chunk, run by the trailing blocks of the
// current chunk's GEMM launch (bf16): rows [cm0, cm1) into h.
struct HNext {
  void* h;
  int cm0, cm1, blocks;
};

// ---------------------------------------------------------------------------
// Forward GEMM + partial log-sum-exp over the rows [cm0, cm1) (h in hbuf)
// ---------------------------------------------------------------------------
template <bool BF, int WM, bool WIDE = false>
__global__ __launch_bounds__(WIDE ? CfgBWide::NT : kGemmThreads, 4) void joiner_fwd_kernel(JoinerArgs a, int cm0, int cm1,
                                                                                            int ncol, int ngemm,
                                                                                            HNext hn) {
  using TIn = typename In<BF>::T;
  using Cfg = typename std::conditional<WIDE, CfgBWide, typename In<BF>::Cfg>::type;
  static_assert(!WIDE || BF, "wide tiles for bf16");
  __shared__ __align__(16) typename Cfg::T smem[Cfg::SMEM_BYTES / sizeof(typename Cfg::T)];
  __shared__ int4 ri[Cfg::BM];
  // blocks past the ngemm tile blocks: the next chunk's h pass (its own slot)
  if ((int)blockIdx.x >= ngemm) {
    if constexpr (BF) h_rows_block<BF, Cfg::NT>(a, hn.h, hn.cm0, hn.cm1, blockIdx.x - ngemm);
    return;
  }
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  // the column tiles of one row tile are consecutive tile ids (one XCD, shared A panel)
  const int tile = xcd_tile_id(mend > cm0 ? (mend - cm0 + Cfg::BM - 1) / Cfg::BM * ncol : 0);
  if (tile < 0) return;
  const int mt = tile / ncol, nt = tile - mt * ncol;
  const int m0 = cm0 + mt * Cfg::BM;
  const int v0 = nt * Cfg::BN;
  const int V = a.V, J = a.J;
  for (int r = threadIdx.x; r < Cfg::BM; r += Cfg::NT)
    ri[r] = (m0 + r < mend) ? a.rowinfo[m0 + r] : make_int4(0, 0, -1, -1);
  __syncthreads();
  float bj[Cfg::FN];
  if constexpr (BF) bias_cols<Cfg, BF>(a, v0, bj);
  floatx4 acc[Cfg::FM][Cfg::FN];
  if constexpr (BF) {
    static_assert(kFwdHbuf<BF>, "the bf16 forward reads h from the h pass");
    // h of the chunk and W^T (the prep kernel's copy), both k = j contiguous
    const LdsSrc<2> sa{make_rsrc(a.hbuf, (size_t)a.chunk_rows * J * 2), m0 - cm0, mend - m0, J, 0, J};
    const LdsSrc<2> sb{make_rsrc(a.wt, (size_t)V * J * 2), v0, V - v0, J, 0, J};
    gemm_mainloop_lds<Cfg>(sa, sb, 0, J, reinterpret_cast<unsigned char*>(smem), acc);
  } else {
    static_assert(!kFwdHbuf<BF>, "the fp32 forward forms h while staging");
    WSrcMNC<Cfg, TIn, WM> sb(a, v0);
    MNCLoader<Cfg, Cfg::BN, WSrcMNC<Cfg, TIn, WM>> lb(sb);
    HSrcKC<Cfg, TIn> sa{EncDec<TIn>(a), ri, J};
    KCLoader<Cfg, Cfg::BM, HSrcKC<Cfg, TIn>> la(sa);
    gemm_mainloop<Cfg>(la, lb, 0, J, smem, acc);
  }

  if constexpr (!BF) bias_cols<Cfg, BF>(a, v0, bj);
  wait_vmem();
  const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) % Cfg::WGN;
  const int slice = nt * Cfg::WGN + wn;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = tile_row<Cfg>(i, r);
      const int4 info = ri[row];
      float lg[Cfg::FN];
      float mx = kNegInfF;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int col = v0 + tile_col<Cfg>(j);
        lg[j] = (col < V) ? acc[i][j][r] + bj[j] : kNegInfF;
        mx = fmaxf(mx, lg[j]);
      }
      mx = row16_max(mx);
      float se = 0.f;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int col = v0 + tile_col<Cfg>(j);
        se += (col < V) ? __expf(lg[j] - mx) : 0.f;
      }
      se = row16_sum(se);
      if (info.w >= 0) {
        const int m = m0 + row;
        if ((lane & 15) == 0 && slice < a.nparts) a.part[(size_t)m * a.nparts + slice] = make_float2(mx, se);
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j) {
          const int col = v0 + tile_col<Cfg>(j);
          if (col < V) {
            if (col == info.z) a.tgt[m] = lg[j];
            if (col == a.b.blank) a.blk[m] = lg[j];
            if (a.logits) a.logits[(size_t)info.w * V + col] = lg[j];
            if (m < a.head_rows) a.head[(size_t)m * a.ldl + col] = lg[j];
          }
        }
      }
    }
}

__global__ __launch_bounds__(256) void joiner_combine_kernel(JoinerArgs a) {
  const int T = a.b.T, S = a.S;
  const size_t total = (size_t)a.b.N * T * S;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int n = (int)(i / ((size_t)T * S));
  const int rem = (int)(i - (size_t)n * T * S);
  const int t = rem / S, s = rem - t * S;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  float px = kNegInfF, py = kNegInfF, l = 0.f;
  if (t < Tn) {
    const int m = (a.frame_off[n] + t) * S + s;
    const int4 info = a.rowinfo[m];
    if (info.w >= 0) {
      const float2* pp = a.part + (size_t)m * a.nparts;
      float M = kNegInfF;
      for (int p = 0; p < a.nparts; ++p) M = fmaxf(M, pp[p].x);
      float sum = 0.f;
      for (int p = 0; p < a.nparts; ++p) sum += pp[p].y * __expf(pp[p].x - M);
      l = M + __logf(sum);
      py = a.blk[m] - l;
      px = (info.z >= 0) ? a.tgt[m] - l : (info.z == -2 ? __builtin_nanf("") : kNegInfF);
    }
  }
  a.px[i] = px;
  a.py[i] = py;
  a.lse[i] = l;
}

// The same for wide vocabularies (more than kCombineSerialParts slices of 64
// columns): one wave per output, lanes over the slices (coalesced reads), the
// max and the sum each by a lane-ordered pass and a fixed reduction across
// the lanes, so the result does not depend on scheduling.
constexpr int kCombineSerialParts = 16;
__global__ __launch_bounds__(256) void joiner_combine_wide_kernel(JoinerArgs a) {
  const int T = a.b.T, S = a.S, lane = threadIdx.x & 63;
  const size_t total = (size_t)a.b.N * T * S;
  const size_t i = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= total) return;
  const int n = (int)(i / ((size_t)T * S));
  const int rem = (int)(i - (size_t)n * T * S);
  const int t = rem / S, s = rem - t * S;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  float px = kNegInfF, py = kNegInfF, l = 0.f;
  if (t < Tn) {
    const int m = (a.frame_off[n] + t) * S + s;
    const int4 info = a.rowinfo[m];
    if (info.w >= 0) {
      const float2* pp = a.part + (size_t)m * a.nparts;
      float M = kNegInfF;
      for (int p = lane; p < a.nparts; p += 64) M = fmaxf(M, pp[p].x);
      M = row16_max(M);  // within each 16-lane row, then across the rows
      M = fmaxf(M, __shfl_xor(M, 16, 64));
      M = fmaxf(M, __shfl_xor(M, 32, 64));
      float sum = 0.f;
      for (int p = lane; p < a.nparts; p += 64) sum += pp[p].y * __expf(pp[p].x - M);
      sum = row16_sum(sum);
      sum += __shfl_xor(sum, 16, 64);
      sum += __shfl_xor(sum, 32, 64);
      l = M + __logf(sum);
      py = a.blk[m] - l;
      px = (info.z >= 0) ? a.tgt[m] - l : (info.z == -2 ? __builtin_nanf("") : kNegInfF);
    }
  }
  if (lane == 0) {
    a.px[i] = px;
    a.py[i] = py;
    a.lse[i] = l;
  }
}

// ---------------------------------------------------------------------------
// LDS of the backward's GEMM tiles: the operand stages (also the epilogue's
// C tile), then per-row info and per-row scalars of the row tile. One size
// for all of them, so that tiles of different kinds share one launch.
// ---------------------------------------------------------------------------
constexpr int kBwdStageBytes = CfgF::SMEM_BYTES > CfgB::SMEM_BYTES ? CfgF::SMEM_BYTES : CfgB::SMEM_BYTES;
static_assert(CfgBw::SMEM_BYTES <= kBwdStageBytes, "dW stages fit");
constexpr int kBwdLdsBytes = kBwdStageBytes + CfgF::BM * (int)sizeof(int4) + CfgF::BM * (int)sizeof(float4);

template <class Cfg>
DEV typename Cfg::T* lds_stages(unsigned char* lds) { return reinterpret_cast<typename Cfg::T*>(lds); }
DEV int4* lds_rowinfo(unsigned char* lds) { return reinterpret_cast<int4*>(lds + kBwdStageBytes); }
DEV float4* lds_rowx(unsigned char* lds) {
  return reinterpret_cast<float4*>(lds + kBwdStageBytes + CfgF::BM * sizeof(int4));
}

// Tile `tile` (row tile tile / ncol, column tile tile % ncol) of the rows
// [cm0, cm1) whose count of active tiles (rows present) is computed here: -1
// for blocks beyond it. The XCD-aware order of xcd_tile_id over a part of a
// launch: v is the block's index within its part of nblocks blocks.
DEV int part_tile(int v, int nblocks, int n_active) {
  const int n = min(n_active, nblocks);
  if (v >= n) return -1;
  const int per = n / kNumXcd, rem = n % kNumXcd;
  const int x = v % kNumXcd, loc = v / kNumXcd;
  return (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + loc;
}
DEV int chunk_row_tiles(const JoinerArgs& a, int cm0, int cm1, int bm) {
  const int mend = min(cm1, a.frame_off[a.b.N] * a.S);
  return mend > cm0 ? (mend - cm0 + bm - 1) / bm : 0;
}

// ---------------------------------------------------------------------------
// Backward 1: recompute logits from h (hbuf, rows of the chunk), d(logits)
// of one 128 x 128 tile into the chunk buffer dl (and, for bf16, its
// transpose dlT, the dW operand: the lane's 4 consecutive rows of one column
// as one 8-byte store; rows past the chunk's end up to the tile end get
// zeros), db partials (one row per wave row of each row tile of the chunk;
// the first chunk writes them, later chunks add to them).
// ---------------------------------------------------------------------------
template <bool BF, int WM>
DEV void dlogits_tile(const JoinerArgs& a, int cm0, int cm1, int v, int nblocks, int ncol, unsigned char* lds) {
  using TIn = typename In<BF>::T;
  using Cfg = typename In<BF>::Cfg;
  int4* ri = lds_rowinfo(lds);
  float4* rx = lds_rowx(lds);  // lse, gx, gy, scale
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  const int tile = part_tile(v, nblocks, chunk_row_tiles(a, cm0, cm1, Cfg::BM) * ncol);
  if (tile < 0) return;
  const int mtl = tile / ncol, nt = tile - mtl * ncol;
  const int m0 = cm0 + mtl * Cfg::BM;
  const int v0 = nt * Cfg::BN;
  const int V = a.V, J = a.J, TS = a.b.T * a.S;
  for (int r = threadIdx.x; r < Cfg::BM; r += Cfg::NT) {
    int4 info = (m0 + r < mend) ? a.rowinfo[m0 + r] : make_int4(0, 0, -1, -1);
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (info.w >= 0) {
      const int n = info.w / TS;
      x = make_float4(a.lse_in[info.w], a.gxo[info.w], a.gyo[info.w], a.scale ? a.scale[n] : 1.f);
    }
    ri[r] = info;
    rx[r] = x;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) / Cfg::WGN;
  // this lane's db_part entries (lanes < 16 of each wave row; a later chunk
  // adds to what the earlier ones left) and bias values, loaded before the
  // epilogue's stores: see bias_cols
  const int mt = (m0 - cm0) / Cfg::BM;
  float* dbq = a.db_part + ((size_t)mt * Cfg::WGM + wm) * V + v0;
  float bj[Cfg::FN], dbold[Cfg::FN];
  auto early_loads = [&]() {
    bias_cols<Cfg, BF>(a, v0, bj);
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
      const int c = tile_col<Cfg>(j);
      dbold[j] = (cm0 != 0 && lane < 16 && v0 + c < V) ? dbq[c] : 0.f;
    }
  };
  if constexpr (BF) early_loads();
  floatx4 acc[Cfg::FM][Cfg::FN];
  if constexpr (BF) {
    const LdsSrc<2> sa{make_rsrc(a.hbuf, (size_t)a.chunk_rows * J * 2), m0 - cm0, mend - m0, J, 0, J};
    const LdsSrc<2> sb{make_rsrc(a.wt, (size_t)V * J * 2), v0, V - v0, J, 0, J};
    gemm_mainloop_lds<Cfg>(sa, sb, 0, J, lds, acc);
  } else {
    HbufSrcKC<Cfg> sa{make_rsrc(a.hbuf, (size_t)a.chunk_rows * J * sizeof(typename Cfg::T)), m0, cm0, mend, J};
    WSrcMNC<Cfg, TIn, WM> sb(a, v0);
    KCLoader<Cfg, Cfg::BM, HbufSrcKC<Cfg>> la(sa);
    MNCLoader<Cfg, Cfg::BN, WSrcMNC<Cfg, TIn, WM>> lb(sb);
    gemm_mainloop<Cfg>(la, lb, 0, J, lds_stages<Cfg>(lds), acc);
    early_loads();
  }
  wait_vmem();

  typename Cfg::T* dl = reinterpret_cast<typename Cfg::T*>(a.dl);
  float colsum[Cfg::FN];
#pragma unroll
  for (int j = 0; j < Cfg::FN; ++j) colsum[j] = 0.f;
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = tile_row<Cfg>(i, r);
      const int m = m0 + row;
      const int4 info = ri[row];
      const float4 x = rx[row];
      const float g = x.y + x.z;
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int col = v0 + tile_col<Cfg>(j);
        float d = 0.f;
        if (info.w >= 0 && col < V) {
          const float p = __expf(acc[i][j][r] + bj[j] - x.x);
          float gd = g * p;
          if (col == info.z) gd -= x.y;
          if (col == a.b.blank) gd -= x.z;
          d = x.w * gd;
          if (a.logits_grad) a.logits_grad[(size_t)info.w * V + col] = d;
        }
        if (m < mend && col < a.ldl) {
          if constexpr (BF) dl[(size_t)(m - cm0) * a.ldl + col] = f2bf(d);
          else dl[(size_t)(m - cm0) * a.ldl + col] = d;
        }
        colsum[j] += d;
        acc[i][j][r] = d;
      }
    }
  if constexpr (BF) {
    uint16_t* dlT = reinterpret_cast<uint16_t*>(a.dlT);
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int col = v0 + tile_col<Cfg>(j);
        if (col >= a.ldl) continue;
        const int mr0 = m0 + tile_row<Cfg>(i, 0) - cm0;
        *reinterpret_cast<uint2*>(dlT + (size_t)col * a.chunk_rows + mr0) =
            make_uint2((uint32_t)f2bf(acc[i][j][0]) | ((uint32_t)f2bf(acc[i][j][1]) << 16),
                       (uint32_t)f2bf(acc[i][j][2]) | ((uint32_t)f2bf(acc[i][j][3]) << 16));
      }
  }
  // db partial: sum over this wave's WM rows, one row of db_part per (m-tile
  // of the chunk, wave row); the first chunk writes it, later ones add to it.
#pragma unroll
  for (int j = 0; j < Cfg::FN; ++j) {
    float s = colsum[j];
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    const int c = tile_col<Cfg>(j);
    if (lane < 16 && v0 + c < V) dbq[c] = dbold[j] + s;
  }
}

// ---------------------------------------------------------------------------
// Backward 1, stored logits: the same d(logits) streamed from the logits the
// forward kept, either all of them ([N, T, S, V], logits_in) or those of the
// first chunk (head, rows in joiner-row order, for chunk 0 only). One block
// per kDlRows rows of the chunk, threads over groups of 4 columns (padding
// columns up to ldl get zeros), several rows per thread with their loads
// issued together; the block's column sums are one db_part row.
// ---------------------------------------------------------------------------
constexpr int kDlRows = 32;
constexpr int kDlThreads = 256;
constexpr int kDlInFlight = 16;  // rows per thread whose loads are issued together

// Threads per row of a block (over the ng 4-column groups of a row); a block
// takes tpr groups of kDlRows rows, and grid.y the ceil(ng / tpr) column
// ranges, so that wide rows spread over many blocks.
__host__ __device__ inline int dl_threads_per_row(int ng) {
  return ng <= 64 ? 64 : (ng <= 128 ? 128 : (ng <= 256 ? 256 : kDlThreads));
}
static dim3 dl_grid(int rows, int ldl) {
  const int ng = ldl / 4;
  return dim3((unsigned)((rows + kDlRows - 1) / kDlRows), (unsigned)((ng + dl_threads_per_row(ng) - 1) / dl_threads_per_row(ng)));
}

struct DlSmem {
  int4 ri[kDlRows];
  float4 rx[kDlRows];  // lse, gx, gy, scale
  float4 red[kDlThreads];
};

// Block (bx, by) of the d(logits) stream: rows cm0 + 32 bx .., column groups of by.
template <bool BF>
DEV void dl_block(const JoinerArgs& a, int cm0, int cm1, int bx, int by, DlSmem& sm) {
  int4* ri = sm.ri;
  float4* rx = sm.rx;
  float4* red = sm.red;
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  const int m0 = cm0 + bx * kDlRows;
  if (m0 >= mend) return;
  const int V = a.V, TS = a.b.T * a.S, ldl = a.ldl, blank = a.b.blank;
  const int nrows = min(kDlRows, mend - m0);
  if (threadIdx.x < kDlRows) {
    const int r = threadIdx.x;
    int4 info = (r < nrows) ? a.rowinfo[m0 + r] : make_int4(0, 0, -1, -1);
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (info.w >= 0) {
      const int n = info.w / TS;
      x = make_float4(a.lse_in[info.w], a.gxo[info.w], a.gyo[info.w], a.scale ? a.scale[n] : 1.f);
    }
    ri[r] = info;
    rx[r] = x;
  }
  __syncthreads();
  const bool from_head = a.logits_in == nullptr;  // chunk 0 from the head rows
  const float* __restrict__ lg = from_head ? a.head : a.logits_in;
  typename In<BF>::Cfg::T* __restrict__ dl = reinterpret_cast<typename In<BF>::Cfg::T*>(a.dl);
  const int ng = ldl / 4;
  const int tpr = dl_threads_per_row(ng);
  const int nrg = kDlThreads / tpr, rg = threadIdx.x / tpr, ct = threadIdx.x - rg * tpr;
  // a thread's rows are contiguous (rpt of them from rb), so that bf16 can
  // also write d(logits) transposed for dW straight from registers: per
  // column, 8 or 16 consecutive rows in one or two 16-byte stores (rows past
  // the chunk's last row as zeros: dW's 16-byte loads may reach them)
  const int rpt = kDlRows / nrg, rb = rg * rpt;
  const bool vec = from_head || (V & 3) == 0;
  {
    const int g0 = by * tpr;  // this block's column groups
    const int c = 4 * (g0 + ct);
    const bool gok = g0 + ct < ng;
    float cs[4] = {0.f, 0.f, 0.f, 0.f};
    if (gok) {
      for (int p0 = 0; p0 < rpt; p0 += kDlInFlight) {
        const int r0 = rb + p0, nk = min(kDlInFlight, rpt - p0);
        float l[kDlInFlight][4];
        uint32_t tw[4][kDlInFlight / 2];  // bf16 pairs of d, rows r0 .. r0 + nk - 1, per column
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int k = 0; k < kDlInFlight / 2; ++k) tw[q][k] = 0u;
#pragma unroll
        for (int k = 0; k < kDlInFlight; ++k) {
          const int r = r0 + k;
          const int4 info = ri[min(r, kDlRows - 1)];
          const bool ok = k < nk && r < nrows && info.w >= 0 && c < V;
          const float* src = lg + (ok ? (from_head ? (size_t)(m0 + r) * ldl : (size_t)info.w * V) + c : 0);
          if (ok && vec) {
            const float4 q = *reinterpret_cast<const float4*>(src);
            l[k][0] = q.x; l[k][1] = q.y; l[k][2] = q.z; l[k][3] = q.w;
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) l[k][q] = (ok && c + q < V) ? src[q] : 0.f;
          }
        }
#pragma unroll
        for (int k = 0; k < kDlInFlight; ++k) {
          const int r = r0 + k;
          if (k >= nk || r >= nrows) break;
          const int4 info = ri[r];
          const float4 x = rx[r];
          const float g = x.y + x.z;
          float d[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = c + q;
            d[q] = 0.f;
            if (info.w >= 0 && col < V) {
              float gd = g * __expf(l[k][q] - x.x);
              if (col == info.z) gd -= x.y;
              if (col == blank) gd -= x.z;
              d[q] = x.w * gd;
              if (a.logits_grad) a.logits_grad[(size_t)info.w * V + col] = d[q];
            }
            cs[q] += d[q];
          }
          const size_t o = (size_t)(m0 + r - cm0) * ldl + c;
          if constexpr (BF) {
            *reinterpret_cast<uint2*>(dl + o) =
                make_uint2((uint32_t)f2bf(d[0]) | ((uint32_t)f2bf(d[1]) << 16),
                           (uint32_t)f2bf(d[2]) | ((uint32_t)f2bf(d[3]) << 16));
#pragma unroll
            for (int q = 0; q < 4; ++q) tw[q][k >> 1] |= (uint32_t)f2bf(d[q]) << (16 * (k & 1));
          } else {
            *reinterpret_cast<float4*>(dl + o) = make_float4(d[0], d[1], d[2], d[3]);
          }
        }
        if constexpr (BF) {
          uint16_t* dlT = reinterpret_cast<uint16_t*>(a.dlT) + (size_t)c * a.chunk_rows + (m0 - cm0 + r0);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint4* dst = reinterpret_cast<uint4*>(dlT + (size_t)q * a.chunk_rows);
            dst[0] = make_uint4(tw[q][0], tw[q][1], tw[q][2], tw[q][3]);
            if (nk > 8) dst[1] = make_uint4(tw[q][4], tw[q][5], tw[q][6], tw[q][7]);
          }
        }
      }
    }
    if (nrg > 1) {  // ng <= tpr here, so every thread runs this loop exactly once
      red[threadIdx.x] = make_float4(cs[0], cs[1], cs[2], cs[3]);
      __syncthreads();
      if (rg == 0) {
        for (int k = 1; k < nrg; ++k) {
          const float4 o = red[k * tpr + ct];
          cs[0] += o.x; cs[1] += o.y; cs[2] += o.z; cs[3] += o.w;
        }
      }
    }
    if (rg == 0 && gok) {
      float* db = a.db_part + (size_t)((m0 - cm0) / kDlRows) * V;  // the chunk's row; later chunks add
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (c + q < V) db[c + q] = cm0 == 0 ? cs[q] : db[c + q] + cs[q];
    }
  }
}

template <bool BF>
__global__ __launch_bounds__(kDlThreads) void joiner_dl_kernel(JoinerArgs a, int cm0, int cm1) {
  __shared__ DlSmem sm;
  dl_block<BF>(a, cm0, cm1, blockIdx.x, blockIdx.y, sm);
}

// ---------------------------------------------------------------------------
// d enc and d dec pieces of one row tile of dpre, formed from the tile in
// LDS so that dpre never goes to HBM. Rows are (frame, slot)
// pairs, S per frame, frames of the batch in order; slot s of frame (n, t)
// is node u = p_t + s.
//   d enc: a frame whose S rows all lie in the tile is summed (ascending s)
//          straight into enc_grad; a frame cut by the tile's first or last
//          row leaves its piece in enc_part[tile][0 (cut at the start) or
//          1], for the tail to add the pieces in tile order.
//   d dec: the rows of one u in the tile (one per frame, slot decreasing as
//          p_t grows) are summed in ascending t into the chunk's row of dpre
//          of the first of them; the chunk's d dec pass adds those pieces of
//          u to d dec in tile order.
// ---------------------------------------------------------------------------
constexpr int kTileFrames = 130;  // frames a 128-row tile can touch (S = 1: 128; plus cut ends)

// Frames [fa, fa + nf) touched by rows [m0, mt_end) of a tile.
DEV void tile_frames(int m0, int mt_end, int S, int& fa, int& nf) {
  fa = m0 / S;
  nf = (mt_end - 1) / S - fa + 1;
}

// Thread k < nf: frame_nt and frame_p of frame fa + k, loaded before the
// main loop so that their latency hides under it.
struct TileFrameRegs {
  int nt, p;
};
DEV TileFrameRegs tile_frames_fetch(const JoinerArgs& a, int m0, int mend, int bm) {
  int fa, nf;
  tile_frames(m0, min(m0 + bm, mend), a.S, fa, nf);
  TileFrameRegs r{0, 0};
  if ((int)threadIdx.x < nf) {
    r.nt = a.frame_nt[fa + threadIdx.x];
    r.p = a.frame_p[fa + threadIdx.x];
  }
  return r;
}

template <class Cfg>
DEV void tile_enc_dec(const JoinerArgs& a, const float* C, int LDC, int cm0, int m0, int mend, int j0,
                      const int4* ri, TileFrameRegs fr) {
  static_assert(Cfg::NT >= kTileFrames && Cfg::NT >= Cfg::BM, "one thread per frame and per row of the tile");
  __shared__ int fr_nt[kTileFrames], fr_n[kTileFrames], fr_p[kTileFrames];
  __shared__ int16_t next_row[Cfg::BM];  // tile row of the next frame's row of the same u, or -1
  __shared__ int16_t first_row[Cfg::BM];  // rows that start a d dec piece (any order)
  __shared__ int n_first;
  const int S = a.S, J = a.J, T = a.b.T;
  const int mt_end = min(m0 + Cfg::BM, mend);  // rows [m0, mt_end) of the tile
  const int rows = mt_end - m0;
  int fa, nf;
  tile_frames(m0, mt_end, S, fa, nf);
  if ((int)threadIdx.x < nf) {
    fr_nt[threadIdx.x] = fr.nt;
    fr_n[threadIdx.x] = fr.nt / T;
    fr_p[threadIdx.x] = fr.p;
  }
  if (threadIdx.x == 0) n_first = 0;
  __syncthreads();
  // one thread per row: is it the first row of its u in the tile (the
  // previous frame's row of u, slot u - p_{t-1}, is absent, of another
  // utterance or before the tile), and which row of the tile comes next
  if ((int)threadIdx.x < rows && ri[threadIdx.x].w >= 0) {
    const int r = threadIdx.x, m = m0 + r, f = m / S, s = m - f * S, k = f - fa;
    const int n = fr_n[k], u = fr_p[k] + s;
    bool first = true;
    if (k > 0 && fr_n[k - 1] == n) {
      const int sp = u - fr_p[k - 1];
      first = !(sp < S && r - s - S + sp >= 0);
    }
    int nx = -1;
    if (k + 1 < nf && fr_n[k + 1] == n) {
      const int s2 = u - fr_p[k + 1], r2 = r - s + S + s2;
      if (s2 >= 0 && r2 < rows) nx = r2;
    }
    next_row[r] = (int16_t)nx;
    if (first) first_row[atomicAdd(&n_first, 1)] = (int16_t)r;
  }
  __syncthreads();
  constexpr int CG = Cfg::BN / 4;  // 4-column groups
  const int tile = m0 / Cfg::BM;
  // d enc
  for (int it = threadIdx.x; it < nf * CG; it += Cfg::NT) {
    const int k = it / CG, cg = it - k * CG, jj = j0 + 4 * cg;
    if (jj >= J) continue;
    const int fs = (fa + k) * S, r0 = max(fs, m0), r1 = min(fs + S, mt_end);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int m = r0; m < r1; ++m) acc = f4add(acc, *reinterpret_cast<const float4*>(C + (m - m0) * LDC + 4 * cg));
    float* dst;
    if (fs >= m0 && fs + S <= mt_end) dst = a.enc_grad + (size_t)fr_nt[k] * J + jj;
    else dst = a.enc_part + ((size_t)tile * 2 + (fs <= m0 ? 0 : 1)) * J + jj;
    *reinterpret_cast<float4*>(dst) = acc;
  }
  // d dec: each piece's rows in ascending t, into the row of its first one
  const int nfirst = n_first;
  for (int it = threadIdx.x; it < nfirst * CG; it += Cfg::NT) {
    const int i = it / CG, cg = it - i * CG, jj = j0 + 4 * cg;
    if (jj >= J) continue;
    const int r = first_row[i];
    float4 acc = *reinterpret_cast<const float4*>(C + r * LDC + 4 * cg);
    for (int r2 = next_row[r]; r2 >= 0; r2 = next_row[r2])
      acc = f4add(acc, *reinterpret_cast<const float4*>(C + r2 * LDC + 4 * cg));
    *reinterpret_cast<float4*>(a.dpre + (size_t)(m0 - cm0 + r) * J + jj) = acc;  // the chunk's row
  }
}

// ---------------------------------------------------------------------------
// Backward 2: dh = dl W^T, dpre = dh (1 - h^2), summed into the d enc / d dec
// pieces in LDS. With `write_h` (the path that streams stored logits, where
// no h pass ran) it also leaves h of the chunk's rows as the dW
// contraction's operand (zero for absent slots): [rows, J] in hbuf for fp32,
// transposed [J, chunk_rows] in hT for bf16.
// ---------------------------------------------------------------------------
template <bool BF, int WM>
DEV void dh_tile(const JoinerArgs& a, int cm0, int cm1, int v, int nblocks, int ncol, unsigned char* lds,
                 bool write_h) {
  using TIn = typename In<BF>::T;
  using Cfg = typename In<BF>::Cfg;
  int4* ri = lds_rowinfo(lds);
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  const int tile = part_tile(v, nblocks, chunk_row_tiles(a, cm0, cm1, Cfg::BM) * ncol);
  if (tile < 0) return;
  const int mtl = tile / ncol, nt = tile - mtl * ncol;
  const int m0 = cm0 + mtl * Cfg::BM;
  const int j0 = nt * Cfg::BN;
  const int J = a.J;
  for (int r = threadIdx.x; r < Cfg::BM; r += Cfg::NT)
    ri[r] = (m0 + r < mend) ? a.rowinfo[m0 + r] : make_int4(0, 0, -1, -1);
  __syncthreads();
  const TileFrameRegs fr = tile_frames_fetch(a, m0, mend, Cfg::BM);
  // enc and dec of this thread's 4-column groups of the tile (the epilogue's
  // h = tanh(enc + dec)), all issued together: ahead of the main loop for
  // bf16, right after it for fp32 (whose main loop has no registers to
  // spare), then waited for once
  constexpr int NIT = Cfg::BM * Cfg::BN / 4 / Cfg::NT;  // 4-column groups per thread
  static_assert(Cfg::BM * Cfg::BN / 4 % Cfg::NT == 0, "whole groups per thread");
  const EncDec<TIn> ed(a);
  RawVec<TIn, 4> pe[NIT], pd[NIT];
  auto fetch_enc_dec = [&]() {
#pragma unroll
    for (int q8 = 0; q8 < NIT; ++q8) {
      const int it = threadIdx.x + q8 * Cfg::NT;
      const int row = it / (Cfg::BN / 4), jj = j0 + (it - row * (Cfg::BN / 4)) * 4;
      const int4 info = ri[row];  // absent (w < 0) for rows past mend
      const int n = (info.w >= 0 && jj < J) ? 4 : 0;  // J is a multiple of 8: a group is all in or out
      raw_load(ed.enc, (uint32_t)(info.x + jj) * sizeof(TIn), n, kSegVector, pe[q8]);
      raw_load(ed.dec, (uint32_t)(info.y + jj) * sizeof(TIn), n, kSegVector, pd[q8]);
    }
  };
  if constexpr (BF) fetch_enc_dec();
  floatx4 acc[Cfg::FM][Cfg::FN];
  if constexpr (BF) {
    // d(logits) of the chunk and W (or its zero-padded copy), both k = v contiguous
    const int ldw = a.wpad ? a.ldl : a.V;
    const LdsSrc<2> sa{make_rsrc(a.dl, (size_t)a.chunk_rows * a.ldl * 2), m0 - cm0, mend - m0, a.ldl, 0, a.ldl};
    const LdsSrc<2> sb{make_rsrc(a.wpad ? a.wpad : a.W, (size_t)J * ldw * 2), j0, J - j0, ldw, 0, ldw};
    gemm_mainloop_lds<Cfg>(sa, sb, 0, a.V, lds, acc);
  } else {
    DlSrcKC<Cfg> sa{make_rsrc(a.dl, (size_t)a.chunk_rows * a.ldl * sizeof(typename Cfg::T)), m0, cm0, mend, a.ldl};
    WtSrcKC<Cfg, TIn, WM> sb(a, j0);
    KCLoader<Cfg, Cfg::BM, DlSrcKC<Cfg>> la(sa);
    KCLoader<Cfg, Cfg::BN, WtSrcKC<Cfg, TIn, WM>> lb(sb);
    gemm_mainloop<Cfg>(la, lb, 0, a.V, lds_stages<Cfg>(lds), acc);
    fetch_enc_dec();
  }
  wait_vmem();

  // Epilogue through LDS (the operand stages are free after the main loop's
  // last barrier): the tile goes to LDS in the MFMA layout and comes back row
  // by row, so that enc, dec, dpre and h are read and written with 16-byte
  // accesses per thread along J.
  constexpr int LDC = Cfg::BN + 4;
  static_assert(Cfg::BM * LDC * 4 <= kBwdStageBytes, "epilogue tile fits the operand stages");
  float* C = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) C[tile_row<Cfg>(i, r) * LDC + tile_col<Cfg>(j)] = acc[i][j][r];
  __syncthreads();
  float4 hk[BF ? NIT : 1];  // bf16: h of this thread's groups, back to the tile after the d enc / d dec pieces
#pragma unroll
  for (int q8 = 0; q8 < NIT; ++q8) {
    const int it = threadIdx.x + q8 * Cfg::NT;
    const int row = it / (Cfg::BN / 4), cg = it - row * (Cfg::BN / 4);
    const int m = m0 + row, jj = j0 + cg * 4;
    if constexpr (BF) hk[q8] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (jj >= J) continue;  // J is a multiple of 8: the group is all in or all out
    float* cr = C + row * LDC + cg * 4;
    const bool on = ri[row].w >= 0;  // absent (w < 0) for rows past mend
    float fe[4], fd[4], h[4], dp[4];
    raw_to_float(pe[q8], fe);
    raw_to_float(pd[q8], fd);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[q] = on ? fast_tanh(fe[q] + fd[q]) : 0.f;
      dp[q] = on ? cr[q] * (1.f - h[q] * h[q]) : 0.f;
    }
    if constexpr (BF) {
      hk[q8] = make_float4(h[0], h[1], h[2], h[3]);
    } else {
      // h [rows, J] for the fp32 dW
      if (write_h && m < mend)
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.hbuf) + (size_t)(m - cm0) * J + jj) =
            make_float4(h[0], h[1], h[2], h[3]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) cr[q] = dp[q];  // dpre stays in the tile for the d enc / d dec pieces
  }
  __syncthreads();
  tile_enc_dec<Cfg>(a, C, LDC, cm0, m0, mend, j0, ri, fr);
  if constexpr (BF) {
    if (!write_h) return;
    // h back to the tile (0 past mend), then h^T [J, chunk_rows] for the
    // bf16 dW: the lane's 4 consecutive rows of the MFMA layout as one
    // 8-byte store
    __syncthreads();
#pragma unroll
    for (int q8 = 0; q8 < NIT; ++q8) {
      const int it = threadIdx.x + q8 * Cfg::NT;
      const int row = it / (Cfg::BN / 4), cg = it - row * (Cfg::BN / 4);
      *reinterpret_cast<float4*>(C + row * LDC + cg * 4) = hk[q8];
    }
    __syncthreads();
    uint16_t* hT = reinterpret_cast<uint16_t*>(a.hT);
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) {
        const int jj = j0 + tile_col<Cfg>(j);
        if (jj >= J) continue;
        float hv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) hv[r] = C[tile_row<Cfg>(i, r) * LDC + tile_col<Cfg>(j)];
        const int mr0 = m0 + tile_row<Cfg>(i, 0) - cm0;
        *reinterpret_cast<uint2*>(hT + (size_t)jj * a.chunk_rows + mr0) =
            make_uint2((uint32_t)f2bf(hv[0]) | ((uint32_t)f2bf(hv[1]) << 16),
                       (uint32_t)f2bf(hv[2]) | ((uint32_t)f2bf(hv[3]) << 16));
      }
  }
}

// ---------------------------------------------------------------------------
// Backward 3: dW partial += h^T dl over one split of the chunk's rows (the
// first chunk writes the partials, later chunks add to them). Tiles: the
// (j, v) tiles of one split are consecutive tile ids, so one XCD reads that
// split's rows.
// ---------------------------------------------------------------------------
template <bool BF>
DEV void dw_tile(const JoinerArgs& a, int cm0, int cm1, int first, int v, int nj, int nv, unsigned char* lds) {
  using Cfg = typename std::conditional<BF, CfgBw, CfgF>::type;
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(cm1, M);
  const int per_split = nj * nv;
  const int tile = part_tile(v, per_split * a.splits, per_split * a.splits);
  const int z = tile / per_split, jv = tile - z * per_split;
  const int jt = jv / nv, vt = jv - jt * nv;
  const int j0 = jt * Cfg::BM, v0 = vt * Cfg::BN;
  const int rows = cm1 - cm0;
  const int per = ((rows + a.splits - 1) / a.splits + Cfg::BK - 1) / Cfg::BK * Cfg::BK;
  const int kb = cm0 + z * per;
  const int ke = min(kb + per, mend);
  const int V = a.V, J = a.J;
  float* part = a.dw_part + (size_t)z * J * V;
  if (kb >= ke) {
    // no rows for this split: the first chunk still defines the partial
    if (first) {
      for (int e = threadIdx.x; e < Cfg::BM * Cfg::BN; e += Cfg::NT) {
        const int j = j0 + e / Cfg::BN, vv = v0 + e % Cfg::BN;
        if (j < J && vv < V) part[(size_t)j * V + vv] = 0.f;
      }
    }
    return;
  }
  // the partials the earlier chunks left for this thread's elements, loaded
  // together before any store (ahead of the main loop for bf16, after it for
  // fp32) rather than one load-add-store round trip per element
  float old[Cfg::FM][Cfg::FN][4];
  auto fetch_old = [&]() {
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = j0 + tile_row<Cfg>(i, r);
#pragma unroll
        for (int jj = 0; jj < Cfg::FN; ++jj) {
          const int vv = v0 + tile_col<Cfg>(jj);
          old[i][jj][r] = (!first && j < J && vv < V) ? part[(size_t)j * V + vv] : 0.f;
        }
      }
  };
  if constexpr (BF) fetch_old();
  floatx4 acc[Cfg::FM][Cfg::FN];
  if constexpr (BF) {
    // h^T and d(logits)^T of the chunk (k = m - cm0 contiguous). Rows past
    // mend hold zeros up to the 128-row tile end, so a chunk of 8 rows that
    // crosses ke reads zeros there; split boundaries inside a chunk are K-step
    // aligned.
    const size_t tb = (size_t)a.chunk_rows * 2;
    const LdsSrc<2> sa{make_rsrc(a.hT, tb * J), j0, J - j0, a.chunk_rows, cm0, ke};
    const LdsSrc<2> sb{make_rsrc(a.dlT, tb * a.ldl), v0, V - v0, a.chunk_rows, cm0, ke};
    gemm_mainloop_lds<Cfg>(sa, sb, kb, ke, lds, acc);
  } else {
    HbufSrcMNC<Cfg> sa{make_rsrc(a.hbuf, (size_t)a.chunk_rows * J * sizeof(typename Cfg::T)), cm0, ke, j0, J};
    DlSrcMNC<Cfg> sb{make_rsrc(a.dl, (size_t)a.chunk_rows * a.ldl * sizeof(typename Cfg::T)), cm0, ke, v0, a.ldl};
    MNCLoader<Cfg, Cfg::BM, HbufSrcMNC<Cfg>> la(sa);
    MNCLoader<Cfg, Cfg::BN, DlSrcMNC<Cfg>, decltype(la)::NBLK> lb(sb);  // threads after A's blocks
    gemm_mainloop<Cfg>(la, lb, kb, ke, lds_stages<Cfg>(lds), acc);
    fetch_old();
  }
  wait_vmem();
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = j0 + tile_row<Cfg>(i, r);
      if (j >= J) continue;
#pragma unroll
      for (int jj = 0; jj < Cfg::FN; ++jj) {
        const int vv = v0 + tile_col<Cfg>(jj);
        if (vv < V) part[(size_t)j * V + vv] = first ? acc[i][jj][r] : old[i][jj][r] + acc[i][jj][r];
      }
    }
}

// The tail of the backward: dW and db summed from their partials, d enc and
// d dec from their pieces. Four independent, latency-bound reductions, run as
// one launch whose block ranges take one part each (d dec, d enc, dW, db), so
// that their memory latencies overlap.
constexpr int kTailThreads = 256;

// dW = sum of the split partials, in split order: four consecutive elements
// per thread (16-byte loads, 16 partials in flight) where J*V and dW's
// address allow, else one.
constexpr int kWsumVec = 4;

DEV bool tail_wsum_vec(const JoinerArgs& a) {
  return (((size_t)a.J * a.V) % kWsumVec) == 0 && (reinterpret_cast<uintptr_t>(a.W_grad) & 15) == 0;
}

DEV void tail_wsum(const JoinerArgs& a, int b) {
  const size_t JV = (size_t)a.J * a.V;
  const size_t i = (size_t)b * kTailThreads + threadIdx.x;
  if (tail_wsum_vec(a)) {
    if (i * kWsumVec >= JV) return;
    const float4* src = reinterpret_cast<const float4*>(a.dw_part) + i;
    const size_t stride = JV / kWsumVec;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 16
    for (int z = 0; z < a.splits; ++z) {
      const float4 v = src[(size_t)z * stride];
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    reinterpret_cast<float4*>(a.W_grad)[i] = s;
    return;
  }
  if (i >= JV) return;
  float s = 0.f;
#pragma unroll 8
  for (int z = 0; z < a.splits; ++z) s += a.dw_part[(size_t)z * JV + i];
  a.W_grad[i] = s;
}

// db = sum of the column partials written by the d(logits) kernel (one per
// 32 rows of a chunk streamed, one per wave row of a GEMM tile recomputed,
// each summed over the chunks): a block takes 16 columns; each of its 16
// thread groups sums a contiguous sixteenth of the rows in ascending order,
// 8 loads in flight, then the sixteenths are added in order.
constexpr int kDbCols = 16;

DEV void tail_dbsum(const JoinerArgs& a, int b, float (*red)[kDbCols]) {
  const int c = threadIdx.x % kDbCols, part = threadIdx.x / kDbCols;  // 16 parts
  constexpr int kParts = kTailThreads / kDbCols;
  const int v = b * kDbCols + c;
  const int M = min(a.frame_off[a.b.N] * a.S, a.chunk_rows);  // rows of the first (largest) chunk
  // the rows the first chunk wrote: one per 32 rows streamed (stored logits
  // or the head), one per wave row of each recomputed tile (the same 32-row
  // groups, whole tiles); a later chunk only adds to a prefix of them
  const bool streamed = a.logits_in || (a.head && a.head_rows == a.chunk_rows);
  const int rows = streamed ? (M + kDlRows - 1) / kDlRows : CfgF::WGM * ((M + CfgF::BM - 1) / CfgF::BM);
  const int q = (rows + kParts - 1) / kParts, r0 = min(rows, part * q), r1 = min(rows, r0 + q);
  float s = 0.f;
  if (v < a.V) {
    const float* col = a.db_part + v;
    for (int r = r0; r < r1; r += 8) {
      float x[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) x[k] = (r + k < r1) ? col[(size_t)(r + k) * a.V] : 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) s += x[k];
    }
  }
  red[part][c] = s;
  __syncthreads();
  if (part == 0 && v < a.V) {
    float t = red[0][c];
    for (int k = 1; k < kParts; ++k) t += red[k][c];
    a.bias_grad[v] = t;
  }
}

// d enc rows per block: threads over float4 column groups of J.
DEV int encdec_rows_per_block(int J) {
  const int tpr = J / 4;
  return tpr >= kTailThreads ? 1 : kTailThreads / tpr;
}


// d enc and d dec from the pieces the dh kernel left (see tile_enc_dec).
// d enc: frames cut by a row tile add their pieces in tile order (the others
// are already written); zero rows past T_n.
constexpr int kTileRows = CfgF::BM;  // the dh row tile (both configurations)

DEV void tail_enc_pieces(const JoinerArgs& a, int b) {
  const int T = a.b.T, S = a.S, J = a.J, tpr = J / 4;
  const int R = encdec_rows_per_block(J);
  const int rr = threadIdx.x / tpr, c = threadIdx.x - rr * tpr;
  const int row = b * R + rr;  // n * T + t
  if (rr >= R || row >= a.b.N * T) return;
  const int n = row / T, t = row - n * T;
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  float4* out = reinterpret_cast<float4*>(a.enc_grad + (size_t)row * J);
  if (t >= Tn) {
    for (int g = c; g < tpr; g += kTailThreads) out[g] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const int fs = (a.frame_off[n] + t) * S, ia = fs / kTileRows, ib = (fs + S - 1) / kTileRows;
  if (ia == ib) return;  // the frame lies in one tile: written by the dh kernel
  for (int g = c; g < tpr; g += kTailThreads) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i = ia; i <= ib; ++i)
      acc = f4add(acc, reinterpret_cast<const float4*>(a.enc_part + ((size_t)i * 2 + (fs <= i * kTileRows ? 0 : 1)) * J)[g]);
    out[g] = acc;
  }
}

// d dec[n, u] from the pieces of u in one chunk of rows [cm0, cm1): one
// piece per row tile that holds rows of u, each in the chunk's row of dpre
// of its first row (ascending t). The row of u in frame t,
// m_t = (frame_off[n] + t) S + u - p_t, grows with t (p_{t+1} - p_t < S
// while u stays in the band), so the chunk's frames of u and the first frame
// of each tile are found by binary searches; the pieces are loaded 8 at a
// time and added in tile order, onto d dec as the earlier chunks left it
// (0 in the chunk that holds the first row of u), so that the sum's order is
// that of one pass over all tiles. The first chunk also writes the zero rows
// (u > U_n, or u in no frame's band).
// u rows of one utterance per d dec block: the block loads the utterance's
// band starts once and its row groups (J / 4 threads each) take the rows.
// Four rows are one pass of the GEMM launch's 512-thread blocks at J = 512;
// longer groups serialise the latency-bound searches of several passes in
// one block and measured slower (16 rows: +5% per step at BPE, +7% long).
constexpr int kDecGroup = 4;
__host__ __device__ inline int dec_blocks(int N, int U1) { return N * ((U1 + kDecGroup - 1) / kDecGroup); }

DEV void tail_dec_pieces(const JoinerArgs& a, int b, int* sp, int cm0, int cm1, const float* dpre) {
  const int nt = blockDim.x;
  const int T = a.b.T, U1 = a.b.U + 1, S = a.S, J = a.J, tpr = J / 4;
  const int ng = (U1 + kDecGroup - 1) / kDecGroup;
  const int n = b / ng, u0 = (b - n * ng) * kDecGroup, u1 = min(U1, u0 + kDecGroup);
  int Tn, Un;
  utt_dims(a.b, n, Tn, Un);
  // row groups: tpr threads per u row (all threads, looping, when a row is wider)
  const int rgw = tpr < nt ? tpr : nt, nrg = nt / rgw;
  const int rg = threadIdx.x / rgw, ct = threadIdx.x - rg * rgw;
  auto zero_row = [&](int u) {
    float4* out = reinterpret_cast<float4*>(a.dec_grad + ((size_t)n * U1 + u) * J);
    for (int g = ct; g < tpr; g += rgw) out[g] = make_float4(0.f, 0.f, 0.f, 0.f);
  };
  // No row of utterance n in the chunk (most blocks: an utterance spans one
  // or two chunks): the first chunk zeroes the rows, which the chunk holding
  // the first row of each u overwrites; later chunks have nothing to add.
  const int off = a.frame_off[n];
  if (u0 > Un || (size_t)a.frame_off[n + 1] * S <= (size_t)cm0 || (size_t)off * S >= (size_t)cm1) {
    if (cm0 == 0 && rg < nrg)
      for (int u = u0 + rg; u < u1; u += nrg) zero_row(u);
    return;
  }
  for (int t = threadIdx.x; t < Tn; t += nt) sp[t] = a.ranges[((size_t)n * T + t) * S];
  __syncthreads();
  if (rg >= nrg) return;
  const int mend = min(cm1, a.frame_off[a.b.N] * S);
  const int rows = __builtin_amdgcn_readfirstlane(a.chunk_rows);  // keeps the resource scalar
  const Rsrc dr = make_rsrc(dpre, (size_t)rows * J * sizeof(float));
  for (int u = u0 + rg; u < u1; u += nrg) {
    if (u > Un) {
      if (cm0 == 0) zero_row(u);
      continue;
    }
    // frames [t0, t1) whose band holds u
    int lo = 0, hi = Tn;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sp[mid] > u - S) hi = mid;
      else lo = mid + 1;
    }
    const int t0 = lo;
    hi = Tn;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sp[mid] > u) hi = mid;
      else lo = mid + 1;
    }
    const int t1 = lo;
    auto row_of = [&](int t) { return (off + t) * S + u - sp[t]; };
    // the first frame in [l, h] whose row of u is at least r (h + 1: none)
    auto first_at = [&](int l, int h, int r) {
      int e = h + 1;
      while (l < e) {
        const int mid = (l + e) >> 1;
        if (row_of(mid) >= r) e = mid;
        else l = mid + 1;
      }
      return l;
    };
    if (t1 <= t0) {
      if (cm0 == 0) zero_row(u);
      continue;
    }
    const int ta = first_at(t0, t1 - 1, cm0), tb = first_at(ta, t1 - 1, mend);  // frames of u in the chunk
    if (ta >= tb) continue;
    const bool starts = row_of(t0) >= cm0;  // the chunk holds the first row of u
    const int ia = row_of(ta) / kTileRows, ib = row_of(tb - 1) / kTileRows;
    float4* out = reinterpret_cast<float4*>(a.dec_grad + ((size_t)n * U1 + u) * J);
    for (int g = ct; g < tpr; g += rgw) {
      float4 acc = starts ? make_float4(0.f, 0.f, 0.f, 0.f) : out[g];
      for (int i0 = ia; i0 <= ib; i0 += 8) {
        float4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int i = i0 + k;
          const int t = (i > ia && i <= ib) ? first_at(ta, tb - 1, i * kTileRows) : ta;  // first frame of u in tile i
          const uint32_t o = (uint32_t)(((size_t)(row_of(t) - cm0) * J + 4 * g) * sizeof(float));
          const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(dr, (int)(i <= ib ? o : kOob), 0, 0);
          v[k] = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w));
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) acc = f4add(acc, v[k]);
      }
      out[g] = acc;
    }
  }
}

// h = tanh(enc + dec) of a chunk's rows [cm0, cm1) for the recomputed logits
// (rows [rows, J] in h) and, for bf16, for dW (transposed [J, chunk_rows] in
// hT), zero for absent slots and, in hT, for rows past the last row up to
// the 128-row tile end (the dW loads read 16-byte segments across it).
struct HPass {
  int blocks, cm0, cm1;
  void* h;
  void* hT;
};

// fp32: one 16-byte group of J per thread.
DEV void h_pass_f32(const JoinerArgs& a, const HPass& hp, int b) {
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(hp.cm1, M);
  const int cpr = a.J / 4;
  const size_t i = (size_t)b * blockDim.x + threadIdx.x;
  const int rr = (int)(i / cpr), c = (int)(i - (size_t)rr * cpr);
  const int m = hp.cm0 + rr;
  if (m >= mend) return;
  const int4 info = a.rowinfo[m];
  const int j = c * 4;
  const EncDec<float> ed(a);
  RawVec<float, 4> e, d;
  const int n = info.w >= 0 ? 4 : 0;
  raw_load(ed.enc, (uint32_t)(info.x + j) * 4, n, kSegVector, e);
  raw_load(ed.dec, (uint32_t)(info.y + j) * 4, n, kSegVector, d);
  float fe[4], fd[4], h[4];
  raw_to_float(e, fe);
  raw_to_float(d, fd);
#pragma unroll
  for (int q = 0; q < 4; ++q) h[q] = info.w >= 0 ? fast_tanh(fe[q] + fd[q]) : 0.f;
  *reinterpret_cast<float4*>(reinterpret_cast<float*>(hp.h) + (size_t)rr * a.J + j) = make_float4(h[0], h[1], h[2], h[3]);
}

// bf16: a 64-row x 64-column tile per 256 threads (tid: the thread among
// them; the two halves of a 512-thread block take two tiles) through LDS,
// both layouts written 16 bytes per thread. Every thread of the block reaches
// the barrier, with or without a tile (`active`).
constexpr int kHTile = 64;
constexpr int kHThreads = 256;
static int h_pass_bf16_blocks(int rows, int J) {
  const int rt = (rows + CfgF::BM - 1) / CfgF::BM * (CfgF::BM / kHTile);  // to the 128-row tile end
  return rt * ((J + kHTile - 1) / kHTile);
}
DEV void h_pass_bf16(const JoinerArgs& a, const HPass& hp, int b, int tid, bool active, uint16_t (*tile)[kHTile + 8]) {
  const int M = a.frame_off[a.b.N] * a.S;
  const int mend = min(hp.cm1, M);
  const int ncj = (a.J + kHTile - 1) / kHTile;
  const int rt = b / ncj, jt = b - rt * ncj;
  const int r0 = rt * kHTile, j0 = jt * kHTile;  // rows (m - cm0), columns j
  const int ty = tid >> 3, tx = tid & 7;
  const EncDec<uint16_t> ed(a);
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int r = ty + 32 * hh, m = hp.cm0 + r0 + r, j = j0 + tx * 8;
    uint4 o = make_uint4(0, 0, 0, 0);
    if (active && m < mend && j < a.J) {
      const int4 info = a.rowinfo[m];
      if (info.w >= 0) {
        RawVec<uint16_t, 8> e, d;
        raw_load(ed.enc, (uint32_t)(info.x + j) * 2, 8, kSegVector, e);
        raw_load(ed.dec, (uint32_t)(info.y + j) * 2, 8, kSegVector, d);
        float fe[8], fd[8];
        raw_to_float(e, fe);
        raw_to_float(d, fd);
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          w[q] = (uint32_t)f2bf(fast_tanh(fe[2 * q] + fd[2 * q])) |
                 ((uint32_t)f2bf(fast_tanh(fe[2 * q + 1] + fd[2 * q + 1])) << 16);
        o = make_uint4(w[0], w[1], w[2], w[3]);
      }
      *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(hp.h) + (size_t)(r0 + r) * a.J + j) = o;
    }
    *reinterpret_cast<uint4*>(&tile[r][tx * 8]) = o;
  }
  __syncthreads();
  if (!active) return;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int c = ty + 32 * hh;  // column within the tile: hT row
    if (j0 + c >= a.J) continue;
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      w[q] = (uint32_t)tile[tx * 8 + 2 * q][c] | ((uint32_t)tile[tx * 8 + 2 * q + 1][c] << 16);
    *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(hp.hT) + (size_t)(j0 + c) * a.chunk_rows + r0 + tx * 8) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

struct TailRanges {
  int dec, enc, wsum, dbsum;  // block counts, in launch order
  int cm0, cm1;               // the chunk whose d dec pieces the dec blocks add
  HPass h0, h1;               // h passes of later chunks (recomputed path), run after them
};

// One launch per chunk of rows: its d dec pieces and the h passes of later
// chunks; the last chunk's launch also runs the d enc, dW and db reductions.
template <bool BF>
__global__ __launch_bounds__(kTailThreads) void joiner_tail_kernel(JoinerArgs a, TailRanges r) {
  extern __shared__ int sp[];  // p_t of one utterance (d dec blocks)
  __shared__ float red[kTailThreads / kDbCols][kDbCols];  // db blocks
  __shared__ uint16_t htile[BF ? kHTile : 1][kHTile + 8];  // bf16 h pass
  int b = blockIdx.x;
  if (b < r.dec) { tail_dec_pieces(a, b, sp, r.cm0, r.cm1, a.dpre); return; }
  b -= r.dec;
  if (b < r.enc) { tail_enc_pieces(a, b); return; }
  b -= r.enc;
  if (b < r.wsum) { tail_wsum(a, b); return; }
  b -= r.wsum;
  if (b < r.dbsum) { tail_dbsum(a, b, red); return; }
  b -= r.dbsum;
  const HPass& hp = b < r.h0.blocks ? r.h0 : r.h1;
  if (b >= r.h0.blocks) b -= r.h0.blocks;
  if constexpr (BF) h_pass_bf16(a, hp, b, threadIdx.x, true, htile);
  else h_pass_f32(a, hp, b);
}

// The backward's first launch when chunk 0's logits come from the head: the
// d(logits) stream of chunk 0 (the first dlx * dly blocks) and the h passes
// of the first chunks (the rest) as block kinds of one launch. Both are
// memory-bound and independent, so that they run side by side instead of one
// after the other.
template <bool BF>
__global__ __launch_bounds__(kTailThreads) void joiner_head_kernel(JoinerArgs a, TailRanges r, int cm0, int cm1,
                                                                   int dlx, int dly) {
  __shared__ DlSmem dsm;
  __shared__ uint16_t htile[BF ? kHTile : 1][kHTile + 8];  // bf16 h pass
  static_assert(kTailThreads == kDlThreads, "one block size for both kinds");
  int b = blockIdx.x;
  if (b < dlx * dly) {
    dl_block<BF>(a, cm0, cm1, b % dlx, b / dlx, dsm);
    return;
  }
  b -= dlx * dly;
  const HPass& hp = b < r.h0.blocks ? r.h0 : r.h1;
  if (b >= r.h0.blocks) b -= r.h0.blocks;
  if constexpr (BF) h_pass_bf16(a, hp, b, threadIdx.x, true, htile);
  else h_pass_f32(a, hp, b);
}

// The backward's GEMM kernel. Every block kind runs in one kernel, each on
// its own range of blocks, so that the recomputed logits of the next chunk
// (L), dh of the current chunk (D) and its dW (W) share a launch (a chunk's
// dh alone puts only one workgroup on each CU), and so that the memory- and
// latency-bound passes of the pipeline run in the slots the GEMM tiles leave
// free at the end of the launch instead of as launches of their own: the h
// pass of a later chunk (H) and the d dec pass of the previous chunk (E).
struct BwdParts {
  int nL, nLcol;   // blocks and column tiles of L (chunk [lm0, lm1) of `nxt`)
  int nD, nDcol;   // blocks and column tiles of D (chunk [cm0, cm1) of `cur`)
  int nW, nWj, nWv;  // blocks and (j, v) tiles per split of W (same chunk)
  int lm0, lm1, cm0, cm1, first;
  int d_first;     // D's tiles (K = V) are longer than W's (K = a split's rows): dispatched before them
  int write_h;     // D also leaves h for a later W (no h pass ran)
  int nH;          // blocks of H (its HPass: chunk rows, target buffers; bf16: two 64 x 64 tiles a block)
  HPass h;
  int nE;          // blocks of E: one per (n, u) row of d dec, adding the pieces of chunk [ecm0, ecm1) in edpre
  int ecm0, ecm1;
  const float* edpre;
};

// Blocks in the order E, then W and D (the kind with the longer K loop
// first), L, H: the d dec blocks first (short and latency-bound; dispatched
// last they would run after the GEMM tiles and lengthen the launch's tail),
// then the longest GEMM tiles, so that the shorter ones fill in around them.
template <bool BF, int WMF, int WMH>
__global__ __launch_bounds__(kGemmThreads, 4) void joiner_bwd_gemm_kernel(JoinerArgs cur, JoinerArgs nxt, BwdParts p) {
  __shared__ __align__(16) unsigned char lds[kBwdLdsBytes];
  int b = blockIdx.x;
  if (b < p.nE) {
    static_assert(kBwdLdsBytes >= 16384 * (int)sizeof(int), "p_t of one utterance (T <= 16384) in LDS");
    tail_dec_pieces(cur, b, reinterpret_cast<int*>(lds), p.ecm0, p.ecm1, p.edpre);
    return;
  }
  b -= p.nE;
  if (b < p.nW + p.nD) {
    const int bd = p.d_first ? b : b - p.nW;  // index among the D blocks (negative: a W block)
    if (bd >= 0 && bd < p.nD) dh_tile<BF, WMH>(cur, p.cm0, p.cm1, bd, p.nD, p.nDcol, lds, p.write_h != 0);
    else dw_tile<BF>(cur, p.cm0, p.cm1, p.first, p.d_first ? b - p.nD : b, p.nWj, p.nWv, lds);
    return;
  }
  b -= p.nW + p.nD;
  if (b < p.nL) {
    dlogits_tile<BF, WMF>(nxt, p.lm0, p.lm1, b, p.nL, p.nLcol, lds);
    return;
  }
  b -= p.nL;
  if (b < p.nH) {
    if constexpr (BF) {
      static_assert(kGemmThreads == 2 * kHThreads, "two h tiles per block");
      const int half = threadIdx.x / kHThreads, hb = 2 * b + half;
      uint16_t (*tile)[kHTile + 8] = reinterpret_cast<uint16_t (*)[kHTile + 8]>(lds) + half * kHTile;
      h_pass_bf16(cur, p.h, hb, threadIdx.x - half * kHThreads, hb < p.h.blocks, tile);
    } else {
      h_pass_f32(cur, p.h, b);
    }
    return;
  }
}



// ranges[n,t,s] = s: every (t, u) of the lattice as a "band" of width U+1.
__global__ __launch_bounds__(256) void full_ranges_kernel(int* ranges, size_t total, int S) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < total) ranges[i] = (int)(i % (size_t)S);
}

}  // namespace

hipError_t launch_full_ranges(int* ranges, int N, int T, int S, hipStream_t s) {
  const size_t total = (size_t)N * T * S;
  {
    RNNT_PROF(s, "full_ranges");
    hipLaunchKernelGGL(full_ranges_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, ranges, total, S);
  }
  return hipGetLastError();
}

int joiner_nparts(int V) { return (V + 63) / 64; }
int joiner_ldl(int V) { return (V + 7) / 8 * 8; }

// Rows of a chunk buffer whose rows of `row_elems` fp32 words stay below
// 2^31 bytes (chunk buffers are read through 32-bit buffer offsets), as a
// multiple of the 128-row tile; 0 when not even one tile fits.
static long long joiner_rsrc_rows(long long row_elems) {
  return ((0x7fffffffll / (row_elems * 4)) / 128) * 128;
}

int joiner_bwd_chunk_max_rows(int J, int V) {
  const long long w = (long long)(J > joiner_ldl(V) ? J : joiner_ldl(V));
  const long long r = joiner_rsrc_rows(w);
  return (int)(r < (1ll << 30) ? r : (1ll << 30));
}

// The padded row count mmax in chunks of at most `cap` rows, split evenly
// (so that no chunk is left nearly empty), as a multiple of the 128-row tile.
static long long even_chunk(long long mmax, long long cap) {
  const long long n = (mmax + cap - 1) / cap;
  return ((mmax + n - 1) / n + 127) / 128 * 128;
}

// The backward's chunk: d(logits) of about 16 MiB, but 8,192 to 16,384 rows
// (64 to 128 row tiles, so that each launch of the pipelined backward puts
// one or two workgroups of every kind on each CU), within the 32-bit limit.
// The head the forward keeps is one chunk: the bound keeps it well below the
// whole [N, T, S, V] logits at the benchmark shapes (a 32 MiB bound would
// hold every row of the BPE batch in it).
// The bound depends on J, V and the dtype only, not on N or T. Chunks are
// taken whole from the start of the padded rows: rows past the last frame of
// the batch (padding frames take none) are absent, so a trailing chunk that
// holds only those costs a few empty launches, while splitting the present
// rows evenly would leave both chunks under-filled. `request` (a multiple of
// 128, or 0) overrides the size.
int joiner_bwd_chunk_rows(int N, int T, int S, int J, int V, int bf16, int request) {
  const long long mmax = (long long)N * T * S;
  const long long all = (mmax + 127) / 128 * 128;
  if (request > 0) return (int)(request < all ? request : all);
  const long long bytes_per_row = (long long)joiner_ldl(V) * (bf16 ? 2 : 4);
  long long cap = ((16ll << 20) / bytes_per_row) / 128 * 128;
  cap = cap < 8192 ? 8192 : cap > 16384 ? 16384 : cap;
  const long long lim = joiner_bwd_chunk_max_rows(J, V);
  if (cap > lim) cap = lim;
  return (int)(cap < all ? cap : all);
}

int joiner_fwd_chunk_rows(int N, int T, int S, int J, int bf16) {
  const long long mmax = (long long)N * T * S;
  if (!(bf16 ? kFwdHbuf<true> : kFwdHbuf<false>)) return (int)((mmax + 127) / 128 * 128);  // no h buffer
  long long cap = 32768;  // h of one chunk: at most 32,768 rows (48 MiB at J = 768, bf16)
  const long long lim = joiner_rsrc_rows(J);
  if (cap > lim) cap = lim;
  return (int)even_chunk(mmax, cap);
}

bool joiner_fwd_uses_hbuf(int bf16) { return bf16 ? kFwdHbuf<true> : kFwdHbuf<false>; }

// dW splits a chunk's rows into ranges of about max(J, V) rows (fp32), so
// that a dW tile does about the work of a dh or recomputed-logits tile of the
// same launch (their K is V or J): no block kind outlasts the others. bf16
// takes ranges four times as long: its dW tiles run at the rate of the
// others, start first (the longest tiles of a launch do), and a quarter as
// many partials are written and re-read per chunk (measured: long step
// 0.818 -> 0.807 ms against twice as long; no change at the stress size).
int joiner_bwd_splits(int J, int V, int chunk_rows, int bf16) {
  const int target = (J > V ? J : V) * (bf16 ? 4 : 1);
  int s = (chunk_rows + target / 2) / target;
  if (s < 1) s = 1;
  if (s > 32) s = 32;
  return s;
}

int joiner_db_rows(int chunk_rows) {
  const long long mmax = chunk_rows;
  const long long streamed = (mmax + kDlRows - 1) / kDlRows;
  const long long tiled = ((mmax + CfgF::BM - 1) / CfgF::BM) * CfgF::WGM;
  return (int)(streamed > tiled ? streamed : tiled);
}

hipError_t launch_joiner_prep(const JoinerArgs& a, hipStream_t s) {
  {
    RNNT_PROF(s, "joiner_prep");
    const int wpad_blocks = prep_wpad_blocks(a);
    hipLaunchKernelGGL(joiner_prep_kernel, dim3(a.b.N * ((a.b.T * a.S + 255) / 256) + wpad_blocks + prep_wt_blocks(a)),
                       dim3(256), 0, s, a, wpad_blocks);
  }
  return hipGetLastError();
}

// seg_mode on the host: how rows of length row_len split into segments of seg elements
static int host_seg_mode(int row_len, int seg, int bf16) {
  if (row_len % seg == 0) return kSegVector;
  return (!bf16 || row_len % 2 == 0) ? kSegWords : kSegElems;
}

hipError_t launch_joiner_h(const JoinerArgs& a, int cm0, int cm1, hipStream_t s) {
  const size_t groups = (size_t)(cm1 - cm0) * (a.J / (a.bf16 ? 8 : 4));
  const dim3 grid((unsigned)((groups + 256 * kHItems - 1) / (256 * kHItems)));
  RNNT_PROF(s, "joiner_h");
  if (a.bf16) hipLaunchKernelGGL(joiner_h_kernel<true>, grid, dim3(256), 0, s, a, cm0, cm1);
  else hipLaunchKernelGGL(joiner_h_kernel<false>, grid, dim3(256), 0, s, a, cm0, cm1);
  return hipGetLastError();
}

hipError_t launch_joiner_fwd(const JoinerArgs& a, hipStream_t s) {
  const int mmax = a.b.N * a.b.T * a.S;
  const int C = a.chunk_rows;
  const int nch = (mmax + C - 1) / C;
  auto lo = [&](int k) { return k * C; };
  auto hi = [&](int k) { return (k + 1) * C < mmax ? (k + 1) * C : mmax; };
  const bool hbuf = a.bf16 ? kFwdHbuf<true> : kFwdHbuf<false>;
  // bf16: h of chunk k in slot k % 2; chunk 0's h pass runs alone, that of
  // chunk k + 1 as the trailing blocks of chunk k's GEMM launch (they write
  // the slot chunk k - 1's launch read)
  auto slot = [&](int k) { return a.hring[k % 2]; };
  if (hbuf) {
    JoinerArgs c = a;
    c.hbuf = slot(0);
    const hipError_t e = launch_joiner_h(c, lo(0), hi(0), s);
    if (e != hipSuccess) return e;
  }
  for (int k = 0; k < nch; ++k) {
    const int cm0 = lo(k), cm1 = hi(k);
    JoinerArgs c = a;
    HNext hn{};
    if (hbuf) c.hbuf = slot(k);
    const bool wide = a.bf16 && a.V >= kFwdWideV;
    const int bm = wide ? CfgBWide::BM : 128, bn = wide ? CfgBWide::BN : 128;
    const int nt = wide ? CfgBWide::NT : kGemmThreads;
    if (hbuf && k + 1 < nch) {
      const size_t groups = (size_t)(hi(k + 1) - lo(k + 1)) * (a.J / (a.bf16 ? 8 : 4));
      hn = HNext{slot(k + 1), lo(k + 1), hi(k + 1), (int)((groups + nt * kHItems - 1) / (nt * kHItems))};
    }
    const int ncol = (a.V + bn - 1) / bn;
    const int ngemm = (cm1 - cm0 + bm - 1) / bm * ncol;
    const dim3 grid((unsigned)(ngemm + hn.blocks));
    RNNT_PROF(s, "joiner_fwd");
    // fp32 W rows (length V) are read in segments of 4 elements; bf16 reads
    // the transposed copy, whose rows (length J) are whole 16-byte chunks
    const int wm = host_seg_mode(a.V, 4, 0);
    if (wide) {
      hipLaunchKernelGGL((joiner_fwd_kernel<true, kSegVector, true>), grid, dim3(nt), 0, s, c, cm0, cm1, ncol, ngemm,
                         hn);
    } else if (a.bf16) {
      hipLaunchKernelGGL((joiner_fwd_kernel<true, kSegVector>), grid, dim3(nt), 0, s, c, cm0, cm1, ncol, ngemm, hn);
    } else {
      if (wm == kSegVector)
        hipLaunchKernelGGL((joiner_fwd_kernel<false, kSegVector>), grid, dim3(nt), 0, s, c, cm0, cm1, ncol, ngemm, hn);
      else
        hipLaunchKernelGGL((joiner_fwd_kernel<false, kSegWords>), grid, dim3(nt), 0, s, c, cm0, cm1, ncol, ngemm, hn);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t total = (size_t)a.b.N * a.b.T * a.S;
  {
    RNNT_PROF(s, "joiner_combine");
    if (a.nparts > kCombineSerialParts)
      hipLaunchKernelGGL(joiner_combine_wide_kernel, dim3((unsigned)((total + 3) / 4)), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(joiner_combine_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

// Joiner args of chunk k's buffers in the recomputed path's rings: h (and
// h^T) in slot k % 3, d(logits) (and its transpose) and the d dec pieces in
// slot k % 2.
static JoinerArgs ring_slot(const JoinerArgs& a, int k) {
  JoinerArgs c = a;
  c.hbuf = a.hring[k % 3];
  c.hT = a.hTring[k % 3];
  c.dl = a.dlring[k % 2];
  c.dlT = a.dlTring[k % 2];
  c.dpre = a.dpring[k % 2];
  return c;
}

static TailRanges tail_ranges(const JoinerArgs& a, int cm0, int cm1, bool last) {
  const size_t JV = (size_t)a.J * a.V;
  const int R = (a.J / 4 >= kTailThreads) ? 1 : kTailThreads / (a.J / 4);
  TailRanges tr{};
  tr.cm0 = cm0;
  tr.cm1 = cm1;
  tr.dec = (cm1 > cm0) ? dec_blocks(a.b.N, a.b.U + 1) : 0;
  tr.enc = last ? (a.b.N * a.b.T + R - 1) / R : 0;
  const bool wvec = JV % kWsumVec == 0 && (reinterpret_cast<uintptr_t>(a.W_grad) & 15) == 0;
  const size_t wthreads = wvec ? JV / kWsumVec : JV;
  tr.wsum = (last && a.W_grad) ? (int)((wthreads + kTailThreads - 1) / kTailThreads) : 0;
  tr.dbsum = (last && a.bias_grad) ? (a.V + kDbCols - 1) / kDbCols : 0;
  return tr;
}

static HPass h_pass(const JoinerArgs& slot, int cm0, int cm1) {
  HPass h{};
  h.cm0 = cm0;
  h.cm1 = cm1;
  h.h = slot.hbuf;
  h.hT = slot.hT;
  const int rows = cm1 - cm0;
  h.blocks = slot.bf16 ? h_pass_bf16_blocks(rows, slot.J)
                       : (int)(((size_t)rows * (slot.J / 4) + kTailThreads - 1) / kTailThreads);
  return h;
}

static hipError_t launch_tail(const JoinerArgs& a, const TailRanges& tr, hipStream_t s, const char* name) {
  const int blocks = tr.dec + tr.enc + tr.wsum + tr.dbsum + tr.h0.blocks + tr.h1.blocks;
  if (blocks == 0) return hipSuccess;
  RNNT_PROF(s, name);
  const size_t sh = (size_t)a.b.T * sizeof(int);
  if (a.bf16) hipLaunchKernelGGL(joiner_tail_kernel<true>, dim3(blocks), dim3(kTailThreads), sh, s, a, tr);
  else hipLaunchKernelGGL(joiner_tail_kernel<false>, dim3(blocks), dim3(kTailThreads), sh, s, a, tr);
  return hipGetLastError();
}

// A GEMM launch of the backward: L of chunk [lm0, lm1) (ring slot of
// `nxt`), D and/or W of chunk [cm0, cm1) (slot of `cur`); an empty range or
// a false flag skips its part.
// The other block kinds a pipeline launch may carry: the h pass of a later
// chunk (H) and the d dec pass of the previous one (E).
struct BwdExtras {
  const HPass* h = nullptr;
  const JoinerArgs* dec = nullptr;  // the previous chunk's args (its d dec pieces, in its dpre)
  int dcm0 = 0, dcm1 = 0;
};

static hipError_t launch_bwd_gemms(const JoinerArgs& cur, const JoinerArgs& nxt, int lm0, int lm1, int cm0,
                                   int cm1, bool do_D, bool do_W, bool write_h, hipStream_t s,
                                   const BwdExtras& x = BwdExtras()) {
  const int V = cur.V, J = cur.J;
  BwdParts p{};
  p.lm0 = lm0;
  p.lm1 = lm1;
  p.cm0 = cm0;
  p.cm1 = cm1;
  p.first = cm0 == 0;
  p.write_h = write_h;
  p.nLcol = (V + 127) / 128;
  p.nL = lm1 > lm0 ? (lm1 - lm0 + 127) / 128 * p.nLcol : 0;
  p.nDcol = (J + 127) / 128;
  p.nD = (do_D && cm1 > cm0) ? (cm1 - cm0 + 127) / 128 * p.nDcol : 0;
  p.nWj = (J + 127) / 128;
  p.nWv = (V + 127) / 128;
  p.nW = (do_W && cm1 > cm0) ? p.nWj * p.nWv * cur.splits : 0;
  {
    const int bk = cur.bf16 ? CfgBw::BK : CfgF::BK;
    const int per = ((cm1 - cm0 + cur.splits - 1) / cur.splits + bk - 1) / bk * bk;  // a split's rows (dw_tile)
    p.d_first = cur.ldl > per;
  }
  if (x.h && x.h->cm1 > x.h->cm0) {
    p.h = *x.h;
    p.nH = cur.bf16 ? (x.h->blocks + 1) / 2
                    : (int)(((size_t)(x.h->cm1 - x.h->cm0) * (J / 4) + kGemmThreads - 1) / kGemmThreads);
  }
  if (x.dec && x.dcm1 > x.dcm0) {
    p.nE = dec_blocks(cur.b.N, cur.b.U + 1);
    p.ecm0 = x.dcm0;
    p.ecm1 = x.dcm1;
    p.edpre = x.dec->dpre;
  }
  const int blocks = p.nL + p.nD + p.nW + p.nH + p.nE;
  if (blocks == 0) return hipSuccess;
  // profiling names: the stored-logits path's separate dh and dW launches,
  // and every launch of the recomputed path's pipeline as one kernel
  const char* name = (p.nD && !p.nL && !p.nW) ? "joiner_dh" : (p.nW && !p.nL && !p.nD) ? "joiner_dw" : "joiner_bwd";
  RNNT_PROF(s, name);
  const dim3 g(blocks), t(kGemmThreads);
  if (cur.bf16) {
    // every bf16 operand is read in 16-byte chunks (W through its transposed
    // or zero-padded copies)
    hipLaunchKernelGGL((joiner_bwd_gemm_kernel<true, kSegVector, kSegVector>), g, t, 0, s, cur, nxt, p);
  } else {
    // fp32 W rows are read in segments of 4 elements, by the recomputed
    // logits across rows and by dh along them
    const int wm_f = host_seg_mode(V, 4, 0);
    if (wm_f == kSegVector) hipLaunchKernelGGL((joiner_bwd_gemm_kernel<false, kSegVector, kSegVector>), g, t, 0, s, cur, nxt, p);
    else hipLaunchKernelGGL((joiner_bwd_gemm_kernel<false, kSegWords, kSegWords>), g, t, 0, s, cur, nxt, p);
  }
  return hipGetLastError();
}

// Stored logits: per chunk, d(logits) streamed from them (for bf16 also
// transposed for dW), then dh (which also leaves h for dW), dW, and the
// chunk's d dec pass (one ring slot).
static hipError_t launch_joiner_bwd_stored(const JoinerArgs& a, hipStream_t s) {
  const int mmax = a.b.N * a.b.T * a.S;
  hipError_t e = hipSuccess;
  for (int cm0 = 0; cm0 < mmax && e == hipSuccess; cm0 += a.chunk_rows) {
    const int cm1 = (cm0 + a.chunk_rows < mmax) ? cm0 + a.chunk_rows : mmax;
    const dim3 gdl = dl_grid(cm1 - cm0, a.ldl);
    {
      RNNT_PROF(s, "joiner_dl");
      if (a.bf16) hipLaunchKernelGGL(joiner_dl_kernel<true>, gdl, dim3(kDlThreads), 0, s, a, cm0, cm1);
      else hipLaunchKernelGGL(joiner_dl_kernel<false>, gdl, dim3(kDlThreads), 0, s, a, cm0, cm1);
    }
    e = hipGetLastError();
    if (e == hipSuccess) e = launch_bwd_gemms(a, a, 0, 0, cm0, cm1, true, false, true, s);  // dh, leaves h
    if (e == hipSuccess) e = launch_bwd_gemms(a, a, 0, 0, cm0, cm1, false, true, false, s);  // dW
    if (e == hipSuccess) e = launch_tail(a, tail_ranges(a, cm0, cm1, cm1 >= mmax), s, cm1 >= mmax ? "joiner_tail" : "joiner_dec");
  }
  return e;
}

hipError_t launch_joiner_bwd(const JoinerArgs& a, hipStream_t s) {
  const int mmax = a.b.N * a.b.T * a.S;
  const int C = a.chunk_rows;
  hipError_t e = hipSuccess;
  if (a.logits_grad) {
    e = launch_fill_f32(a.logits_grad, (size_t)mmax * a.V, 0.f, s);
    if (e != hipSuccess) return e;
  }
  if (a.logits_in) return launch_joiner_bwd_stored(a, s);
  // Recomputed logits, software-pipelined over the chunks with rings of
  // chunk buffers (h and h^T: 3 slots; d(logits), its transpose and the d dec
  // pieces: 2 slots):
  //   tail{H(0), H(1)}; gemm{L(0)} (or chunk 0 streamed from the head);
  //   for each chunk k: gemm{W(k), D(k), L(k+1), H(k+2), E(k-1)};
  //   tail{E(last), d enc, dW and db sums}
  // (H: h pass, L: recomputed logits and d(logits), D: dh and the d enc /
  // d dec pieces, W: dW, E: a chunk's d dec pass). Every launch's reads were
  // written by earlier launches on the stream; within a launch, H writes the
  // h slot of chunk k+2 while W and L read those of chunks k and k+1, L
  // writes the d(logits) slot of chunk k+1 while D and W read chunk k's, and
  // E reads chunk k-1's pieces while D writes chunk k's.
  const int nch = (mmax + C - 1) / C;
  auto lo = [&](int k) { return k * C; };
  auto hi = [&](int k) { return (k + 1) * C < mmax ? (k + 1) * C : mmax; };
  TailRanges tr{};
  tr.h0 = h_pass(ring_slot(a, 0), lo(0), hi(0));
  if (nch > 1) tr.h1 = h_pass(ring_slot(a, 1), lo(1), hi(1));
  if (a.head && a.head_rows == C) {
    // chunk 0's logits were kept by the forward: stream them (for bf16 the
    // stream also writes d(logits) transposed for dW) instead of the one
    // recomputation launch
    // the pipeline cannot fill; the stream shares its launch with the first
    // h passes
    const dim3 gdl = dl_grid(hi(0) - lo(0), a.ldl);
    {
      RNNT_PROF(s, "joiner_dl");
      const unsigned blocks = gdl.x * gdl.y + tr.h0.blocks + tr.h1.blocks;
      if (a.bf16)
        hipLaunchKernelGGL(joiner_head_kernel<true>, dim3(blocks), dim3(kTailThreads), 0, s, a, tr, lo(0), hi(0),
                           (int)gdl.x, (int)gdl.y);
      else
        hipLaunchKernelGGL(joiner_head_kernel<false>, dim3(blocks), dim3(kTailThreads), 0, s, a, tr, lo(0), hi(0),
                           (int)gdl.x, (int)gdl.y);
    }
    e = hipGetLastError();
  } else {
    e = launch_tail(a, tr, s, "joiner_h");
    if (e == hipSuccess) e = launch_bwd_gemms(ring_slot(a, 0), ring_slot(a, 0), lo(0), hi(0), 0, 0, false, false, false, s);
  }
  for (int k = 0; k < nch && e == hipSuccess; ++k) {
    const JoinerArgs cur = ring_slot(a, k), nxt = ring_slot(a, k + 1), prev = ring_slot(a, k > 0 ? k - 1 : 0);
    const bool more = k + 1 < nch;
    BwdExtras x;
    HPass hp{};
    if (k + 2 < nch) {
      hp = h_pass(ring_slot(a, k + 2), lo(k + 2), hi(k + 2));
      x.h = &hp;
    }
    if (k >= 1) {
      x.dec = &prev;
      x.dcm0 = lo(k - 1);
      x.dcm1 = hi(k - 1);
    }
    e = launch_bwd_gemms(cur, nxt, more ? lo(k + 1) : 0, more ? hi(k + 1) : 0, lo(k), hi(k), true, true, false, s, x);
  }
  if (e == hipSuccess) {
    const JoinerArgs last = ring_slot(a, nch - 1);
    e = launch_tail(last, tail_ranges(last, lo(nch - 1), hi(nch - 1), true), s, "joiner_tail");
  }
  return e;
}
