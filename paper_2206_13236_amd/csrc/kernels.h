// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

// Element type of the diagonal-major copies of px and py that the lattice
// recursions read (log2 units), and its load from a buffer resource. fp64:
// the wavefront step then adds them without a conversion.
using DiagT = double;
DEV DiagT diag_load(Rsrc r, uint32_t byte_off) { return buf_load_f64(r, byte_off); }

// ---- stage 1-2: trivial joiner, full lattice --------------------------------
struct SimpleArgs {
  BatchDev b;
  int V;
  const float* am;     // [N, T, V]
  const float* lm;     // [N, U+1, V]
  const float* scale;  // [N] or null
  float* m_a;          // ws [N*T]
  float* m_l;          // ws [N*(U+1)]
  float* Z;            // ws [N, T, U+1]
  float* npart;        // ws [nsplit, N, T, U+1]: normaliser partial sums per K range
  int nsplit;
  float* lpart;        // ws [lsplit, N, U+1, V]: d lm partial sums per frame range
  int lsplit;
  float* px;           // [N, T, U+1] (caller's or ws)
  float* py;
  DiagT* pxd;          // ws [N, D, W]: px, py in the diagonal-major lattice layout, log2 units
  DiagT* pyd;          //   (times log2 e), -inf at every cell that is no node of the utterance
  double* alpha;       // ws [N, D, W], log2 domain, diagonal-major
  double* beta;        // ws [N, D, W], log2 domain, diagonal-major
  double* Lutt;        // ws [N]: total log2-prob (NaN for an invalid utterance)
  float* loss;         // [N]
  float* gx;           // [N, T, U+1]
  float* gy;
  float* Wt;           // ws [N, T, ldw]: W(t,u) for the simple loss's gradient (null: not written)
  int ldw;
  double* ry;          // ws [N*T]      row sums of gy (fp64)
  double* cpx;         // ws [N, ncolblk, U+1]: column sums of gx over 16-frame blocks
  double* cpy;         //                       same for gy
  int ncolblk;
  double* rx;          // ws [N*T]      row sums of gx (fp64)
  double* Gx;          // ws [N*(U+1)]  column sums of gx over frames (fp64)
  double* Gy;          //               same for gy
  // smoothed trivial joiner (Sec. 3.3.1): weights and per-utterance statistics
  float lm_only;       // a_lm
  float am_only;       // a_ac
  float* Zlm;          // ws [N*(U+1)]  log sum_v exp(lm[u,v])
  float* lavg;         // ws [N, V]     L_dec^avg(v)
  float* Zac;          // ws [N*T]      log sum_v exp(am[t,v] + L_dec^avg(v))
  float* q;            // ws [N, V]     gradient of the loss w.r.t. L_dec^avg, over (U_n+1) avg(v)
  float* su;           // ws [N*(U+1)]  sum_v q(v) softmax(lm[u])(v)
  float* am_grad;      // [N, T, V] or null
  float* lm_grad;      // [N, U+1, V] or null
};

hipError_t launch_rowmax(const SimpleArgs& a, hipStream_t s);
hipError_t launch_normalizer(const SimpleArgs& a, hipStream_t s);
int normalizer_splits(int N, int T, int U, int V);
int dlm_splits(int N, int T, int U, int V);
// frame ranges of the fused d am / d lm kernel (0: it does not apply to these sizes)
int simple_grad_splits(int N, int T, int U, int V);
hipError_t launch_lattice(const SimpleArgs& a, hipStream_t s);
hipError_t launch_lattice_diag_copy(const SimpleArgs& a, hipStream_t s);
// the recursion alone (no occupations) on a.pxd / a.pyd; a.V = 0 skips the symbol check
hipError_t launch_lattice_recursion(const SimpleArgs& a, hipStream_t s);
int lattice_colblocks(int T);

// Diagonal-major lattice layout (internal): node (t, u) of an utterance sits
// on diagonal d = t + u at slot (u % R) * 64 + u / R of a row of W = 64 R
// slots, where R = lattice_rows_per_lane(U + 1) rows of the lattice belong
// to each lane of the recursion's wave. One anti-diagonal step of the
// recursion then reads and writes contiguous slots. D = T + U diagonals.
int lattice_rows_per_lane(int U1);
inline size_t lattice_diag_cells(int T, int U) {
  return (size_t)(T + U) * 64 * lattice_rows_per_lane(U + 1);
}
inline int lattice_fill_blocks(int T, int U, int bs) { return (int)((lattice_diag_cells(T, U) + bs - 1) / bs); }
DEV int lattice_slot(int u, int R) { return (u % R) * 64 + u / R; }
// Cells of the diagonal-major layout [T+U, 64R] of an utterance's lattice
// that no (t, u) of the [T, U+1] rectangle maps to are set to -inf in both
// copies by a fill of bs-cell blocks (bs threads) per utterance (32-bit index
// arithmetic; the rectangle's own cells are written by their producer).
DEV int lattice_fill_blocks_dev(int T, int U1, int R, int bs) { return ((T + U1 - 1) * 64 * R + bs - 1) / bs; }
DEV void lattice_fill_outside(DiagT* pxd, DiagT* pyd, int blk, int tid, int bs, int T, int U1, int R) {
  const int per = lattice_fill_blocks_dev(T, U1, R, bs);
  const int n = blk / per;
  const uint32_t W = 64u * (uint32_t)R, DW = (uint32_t)(T + U1 - 1) * W;
  const uint32_t c = (uint32_t)(blk - n * per) * (uint32_t)bs + (uint32_t)tid;
  if (c >= DW) return;
  const int d = (int)(c / W), slot = (int)(c % W);
  const int u = (slot & 63) * R + (slot >> 6), t = d - u;
  if (u >= U1 || t < 0 || t >= T) {
    const size_t j = (size_t)n * DW + c;
    pxd[j] = (DiagT)kNegInfD;
    pyd[j] = (DiagT)kNegInfD;
  }
}
// Rows of the lattice per lane: the fewest that hold U + 1 rows up to 6
// (every padding row costs a log-add per diagonal step), then 8, 12 or 16.
DEV int lattice_rows_per_lane_dev(int U1) {
  const int need = (U1 + 63) / 64;
  return need <= 6 ? (need < 1 ? 1 : need) : need <= 8 ? 8 : need <= 12 ? 12 : 16;
}
hipError_t launch_smoothing_stats(const SimpleArgs& a, hipStream_t s);
hipError_t launch_simple_grads(const SimpleArgs& a, hipStream_t s);

// ---- stage 3: pruning bounds -----------------------------------------------
hipError_t launch_prune(const BatchDev& b, int S, const float* gx, const float* gy, int* ranges,
                        hipStream_t s);
size_t prune_smem_bytes(int T);

// ---- stage 4: pruned joiner -----------------------------------------------
struct JoinerArgs {
  BatchDev b;
  int S, J, V;
  int bf16;
  const void* enc;     // [N, T, J]
  const void* dec;     // [N, U+1, J]
  const void* W;       // [J, V]
  const void* bias;    // [V] or null
  const int* ranges;   // [N, T, S]
  int* frame_off;      // ws [N+1]
  int* frame_nt;       // ws [N*T] (backward only, else null): n*T + t of the f-th frame of the batch
  int* frame_p;        //                                    and its band start p_t
  int4* rowinfo;       // ws [N*T*S]: enc_off, dec_off, sym (-1: none), out index (-1: absent)
  // forward
  float2* part;        // ws [N*T*S, nparts] (max, sum exp) per 64-column slice
  int nparts;
  float* tgt;          // ws [N*T*S]
  float* blk;          // ws [N*T*S]
  float* px;           // [N, T, S]
  float* py;
  float* lse;
  float* logits;       // [N, T, S, V] or null: the forward also stores the logits
  float* head;         // [head_rows, ldl] or null: the logits of the first head_rows rows (the backward's
  int head_rows;       //   first chunk), stored by the forward and streamed by the backward
  // backward
  const float* lse_in;
  const float* logits_in;  // [N, T, S, V] or null: stored logits (else recomputed)
  const float* gxo;    // band occupations [N, T, S]
  const float* gyo;
  const float* scale;  // [N] or null
  void* dl;            // ws chunk [chunk_rows, ldl] (f32 or bf16)
  int ldl;
  void* dlT;           // ws chunk [ldl, chunk_rows] (bf16 only): d(logits) transposed for dW
  void* wpad;          // ws [J, ldl] bf16 or null: W with its rows padded by zeros to ldl elements, so
                       // that dh reads W in 16-byte segments when V is not a multiple of 8
  void* wt;            // ws [V, J] bf16 or null: W transposed (k = j contiguous), the B operand of the
                       // bf16 forward and recomputed logits, written by the prep kernel
  int chunk_rows;
  float* dpre;         // ws chunk [chunk_rows, J]: the chunk's d dec pieces, each in the row of its first row
  float* enc_part;     // ws [ceil(N*T*S/128), 2, J]: d enc pieces of frames cut by a 128-row tile
  void* hbuf;          // ws chunk [chunk_rows, J] (f32 or bf16): h = tanh(enc + dec) of the chunk's rows
                       // (written by an h pass, or by dh when the logits were stored)
  void* hT;            // ws chunk [J, chunk_rows] (bf16 only): h transposed, the dW operand
  void* hring[3];      // the recomputed backward's rings of chunk buffers: hbuf and hT of 3 slots,
  void* hTring[3];     //   dl and dlT of 2, dpre of 2 (the fields above are those of slot 0)
  void* dlring[2];
  void* dlTring[2];
  float* dpring[2];
  float* dw_part;      // ws [splits, J, V]
  int splits;
  float* db_part;      // ws [n_db_rows, V]: column sums per row group of a chunk, summed over the chunks
  int n_db_rows;
  float* enc_grad;
  float* dec_grad;
  float* W_grad;
  float* bias_grad;
  float* logits_grad;
};

hipError_t launch_joiner_prep(const JoinerArgs& a, hipStream_t s);
hipError_t launch_full_ranges(int* ranges, int N, int T, int S, hipStream_t s);
hipError_t launch_joiner_fwd(const JoinerArgs& a, hipStream_t s);
hipError_t launch_joiner_bwd(const JoinerArgs& a, hipStream_t s);
// rows of the backward's chunk (request: a multiple of 128 overriding the
// library's choice, or 0), and the largest chunk the 32-bit offsets allow
int joiner_bwd_chunk_rows(int N, int T, int S, int J, int V, int bf16, int request);
int joiner_bwd_chunk_max_rows(int J, int V);
int joiner_fwd_chunk_rows(int N, int T, int S, int J, int bf16);
bool joiner_fwd_uses_hbuf(int bf16);
int joiner_bwd_splits(int J, int V, int chunk_rows, int bf16);
int joiner_db_rows(int chunk_rows);  // db partial rows of one chunk
int joiner_nparts(int V);
int joiner_ldl(int V);

// ---- stage 4: pruned recursion ---------------------------------------------
struct BandArgs {
  BatchDev b;
  int S;
  int D;               // diagonals of the layout: band_diagonals(T, U, S)
  int W;               // slots per diagonal: band_slots(U, S)
  bool masked;         // W == 64: the lattice layout with R = 1 (slot u), else slot s = u - p_t
  const float* px;     // [N, T, S]
  const float* py;
  const int* ranges;   // [N, T, S]
  DiagT* pxd;          // ws [N, D, W]: px, py in a diagonal-major layout, log2 units
  DiagT* pyd;
  uint32_t* meta;      // ws [N, D, W] per-slot shifts and validity (band path only)
  double* alpha;       // ws [N, D, W] log2 domain, diagonal-major
  double* beta;
  double* Lutt;        // ws [N]: total log2-prob (NaN for an invalid utterance)
  float* loss;
  float* gx;           // [N, T, S] or null
  float* gy;
  // chunked scan over frames (S <= 16)
  int C;               // frames per chunk
  int nchunk;          // chunks of the padded T: ceil(T / C)
  double* M;           // ws [N, nchunk, S, S]: arrivals at a chunk's first frame -> at the next chunk's
  double* E;           // ws [N, S]: arrivals at the last chunk's first frame -> end of the lattice
  double* V;           // ws [N, nchunk, S]: arrivals (forward messages) at each chunk's first frame
  double* Wb;          // ws [N, nchunk, S]: beta at each chunk's first frame
};
hipError_t launch_band(const BandArgs& a, hipStream_t s);
hipError_t launch_band_scan(const BandArgs& a, hipStream_t s);
constexpr int kScanMaxS = 16;   // band width the scan supports (one 16-lane row per chain)
constexpr int kScanMaxC = 32;   // frames per chunk at most
int band_scan_chunk(int T);     // default frames per chunk for a padded length T
int band_diagonals(int T, int U, int S);
// Two layouts for the band recursion. U + 1 <= 64: the full lattice's
// diagonal-major layout with one row per lane (W = 64, slot u), band nodes
// holding their log-probs and every other node -inf, so the full recursion
// computes the band's sums. Otherwise one slot per band offset (W = S, slot
// s = u - p_t), each slot carrying the shifts to its predecessors.
bool band_masked(int U, int S);
int band_slots(int U, int S);  // W

// ---- per-utterance validation and the training loss --------------------------
// flags[n] (cleared first) gets the RNNT_FLAG_* bits of utterance n
hipError_t launch_validate(const BatchDev& b, int V, int S, int J, int bf16, const float* am, const float* lm,
                           const void* enc, const void* dec, int* flags, hipStream_t s);
hipError_t launch_combine_losses(int N, const float* simple, const float* pruned, float ss, float ps, int mean,
                                 float* loss, float* total, hipStream_t s);

// ---- generic fills -----------------------------------------------------------
hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t s);
