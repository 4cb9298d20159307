/*
 * rnnt_pruned.h - C ABI of the MI355X (gfx950) pruned RNN-T loss library.
 *
 * Implements the computation of "Pruned RNN-T for fast, memory-efficient ASR
 * training" (Kuang et al., arXiv 2206.13236) as four stages:
 *
 *   1. rnnt_simple_loss        trivial joiner (Sec. 3.1, Eqs. (5)-(6)) and the
 *                              full-lattice recursion (Sec. 2, Eqs. (1)-(4));
 *                              yields the occupation counts of Sec. 3.2.2 and,
 *                              optionally, the gradients w.r.t. am and lm.
 *      rnnt_simple_loss_backward
 *                              those gradients later, from the state the
 *                              forward call left in its workspace (so that a
 *                              caller can run them on a second stream while
 *                              the pruned stages proceed).
 *   2. rnnt_prune_ranges       locally optimal pruning bounds, Eq. (8), made
 *                              consistent with Eqs. (9)-(10) (Sec. 3.2.2).
 *   3. rnnt_pruned_joiner      the full non-linear joiner evaluated only at the
 *                              pruned (t, u) pairs (Sec. 3.2, Fig. 1(b)),
 *                              reduced to target/blank log-probs.
 *      rnnt_pruned_loss        the same recursion on the pruned lattice, whose
 *                              entries outside p_t <= u < p_t + S are -inf.
 *      rnnt_pruned_joiner_backward
 *                              the pruned loss's gradients w.r.t. the joiner
 *                              inputs and parameters.
 *   4. rnnt_combine_losses     the training loss of Sec. 3.3: the scaled sum
 *                              of the simple and the pruned losses, per
 *                              utterance and summed or averaged.
 *   rnnt_validate_inputs       a synchronous check of a batch against the
 *                              problem statement of Sec. 2 (debugging aid).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every array pointer is a DEVICE pointer to a dense, row-major array. The
 *   caller owns all memory; the library never allocates or frees device
 *   memory and keeps no state between calls.
 * - Every call only enqueues kernels on `stream` (a hipStream_t; NULL = the
 *   null stream) and returns without synchronising (except the debugging
 *   aid rnnt_validate_inputs, which waits for its result).
 * - Scalars and pointers are checked on the host before any launch; a failed
 *   check returns a non-zero status and enqueues nothing. The message is
 *   available from rnnt_last_error() (thread-local).
 * - Data-dependent problems never fail the call. An utterance whose lengths
 *   are out of range (t_len[n] < 1 or > T, u_len[n] < 0 or > U) or whose
 *   symbols are outside [0, V) gets a NaN loss; indices are clamped so every
 *   memory access stays in bounds.
 * - Lattice layout: T frames x (U+1) token positions. symbols[n, u] is
 *   y_{u+1}; y_0 is the beginning-of-sentence blank (Sec. 2). `blank` may
 *   equal a symbol value (then that symbol's and the blank's log-probs
 *   coincide, which is well defined).
 * - Losses are per utterance: loss[n] = -log P(y | x) (minus the total
 *   log-probability of Sec. 2). Gradients are gradients of
 *   sum_n scale[n] * loss[n]; scale may be NULL (all ones).
 * - Entries outside t < t_len[n], u <= u_len[n] are written with defined
 *   fills: 0 for occupations and gradients, -inf for log-probs.
 */
#ifndef RNNT_PRUNED_H
#define RNNT_PRUNED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define RNNT_OK 0
#define RNNT_EINVAL 1        /* a scalar or pointer argument is invalid            */
#define RNNT_EWORKSPACE 2    /* workspace missing or smaller than the query result */
#define RNNT_EUNSUPPORTED 3  /* a size outside what the kernels support           */
#define RNNT_EHIP 4          /* a HIP runtime call failed                           */

/* Element types of the joiner inputs (enc, dec, W, bias). */
#define RNNT_F32 0
#define RNNT_BF16 1

/* Limits of this build. */
#define RNNT_MAX_U 1023      /* U + 1 <= 1024 lattice rows                          */
#define RNNT_MAX_S 32        /* pruning width                                       */

typedef struct rnnt_batch {
  int32_t N;                 /* utterances                                         */
  int32_t T;                 /* padded frame count (max t_len)                      */
  int32_t U;                 /* padded token count (max u_len); lattice has U+1 rows */
  const int32_t* t_len;      /* [N] device, 1 <= t_len[n] <= T                      */
  const int32_t* u_len;      /* [N] device, 0 <= u_len[n] <= U                      */
  const int32_t* symbols;    /* [N, U] device, symbols[n, u] = y_{u+1} in [0, V)    */
  int32_t blank;             /* blank id in [0, V) (0 in the paper, Sec. 2)         */
} rnnt_batch;

/* ABI version of this header (bumped on any signature change). */
int rnnt_abi_version(void);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* rnnt_last_error(void);

/* ------------------------------------------------------------------------ */
/* Stage 1-2: trivial joiner + full-lattice forward-backward                 */
/* ------------------------------------------------------------------------ */

/* Workspace bytes needed by rnnt_simple_loss for these sizes (pure function of
 * the arguments; 0 on invalid sizes). */
size_t rnnt_simple_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t V);

/* Simple (trivial-joiner) loss of Sec. 3.1 and its occupation counts.
 *
 * am [N, T, V] fp32   L_enc(t, v): un-normalised logits from the encoder side.
 * lm [N, U+1, V] fp32 L_dec(u, v): un-normalised logits from the decoder side.
 * The joiner is L(t,u,v) = am[t,v] + lm[u,v] - L_normalizer(t,u) (Eq. (5))
 * with L_normalizer = log sum_v exp(am[t,v] + lm[u,v]) (Eq. (6)), evaluated as
 * a max-shifted matrix product.
 *
 * Outputs:
 *   loss   [N]          fp32, required.
 *   px_occ [N, T, U+1]  fp32, required: dL_tot/dy(t,u), the occupation of the
 *                       vertical (symbol) transition leaving (t,u), in [0,1].
 *   py_occ [N, T, U+1]  fp32, required: dL_tot/dblank(t,u).
 *   px, py [N, T, U+1]  fp32, nullable: the log-probs y(t,u), blank(t,u)
 *                       (Eqs. (1)-(2)); px[.., U_n..] = -inf.
 *   am_grad [N, T, V], lm_grad [N, U+1, V]  fp32, nullable: gradients of
 *                       sum_n scale[n] * loss[n].
 *   scale  [N] fp32, nullable (all ones); only read when a gradient is asked.
 * lm_only_scale, am_only_scale: weights a_lm, a_ac >= 0 (a_lm + a_ac <= 1) of
 *   the smoothed trivial joiner of Sec. 3.3.1,
 *     L = (1 - a_lm - a_ac) L_trivial + a_lm L_lm + a_ac L_acoustic,
 *   L_lm(u,v) = LogSoftmax_v lm[u,v], L_acoustic(t,v) = LogSoftmax_v(am[t,v] +
 *   L_dec^avg(v)), L_dec^avg(v) = log of the mean over u <= U_n of
 *   Softmax_v lm[u,v]. (The printed combination repeats L_lm in its third
 *   term; the acoustic joiner the section defines is used.) 0, 0 gives the
 *   plain trivial joiner.
 * workspace: device buffer of at least rnnt_simple_loss_workspace_size() bytes,
 *   256-byte aligned. On return (in stream order) it holds what
 *   rnnt_simple_loss_backward needs.
 */
int rnnt_simple_loss(const rnnt_batch* batch, int32_t V,
                     const float* am, const float* lm, const float* scale,
                     float lm_only_scale, float am_only_scale,
                     float* loss, float* px_occ, float* py_occ,
                     float* px, float* py, float* am_grad, float* lm_grad,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Gradients of sum_n scale[n] * simple_loss[n] w.r.t. am and lm (the
 * log-softmax backward through Eq. (5), two contractions of the forward's
 * shape), computed from the state a preceding rnnt_simple_loss call left in
 * `workspace`: the same batch, V, am, lm, smoothing weights, its px_occ
 * output, and the same workspace, unmodified since, with that call ordered
 * before this one (same stream, or an event). Results equal those of the
 * forward call asked for the gradients directly.
 *
 * px_occ [N, T, U+1]: the forward's px_occ output (required).
 * am_grad [N, T, V], lm_grad [N, U+1, V] fp32: outputs (at least one).
 */
int rnnt_simple_loss_backward(const rnnt_batch* batch, int32_t V,
                              const float* am, const float* lm, const float* scale,
                              float lm_only_scale, float am_only_scale,
                              const float* px_occ, float* am_grad, float* lm_grad,
                              void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Stage 3: pruning bounds (Sec. 3.2.2)                                      */
/* ------------------------------------------------------------------------ */

/* ranges [N, T, S] int32 output: ranges[n,t,s] = p_t + s for t < t_len[n] and
 * ranges[n,t,s] = s for padding frames. p_t is the argmax over p in [0, P],
 * P = max(0, U_n - S + 1), of Eq. (8):
 *     -px_occ(t, p-1) + py_occ(t, p) + ... + py_occ(t, p+S-1),
 * evaluated in fp32 left to right (y'(t,-1) = 0; slots above U_n add 0; ties
 * to the smallest p; NaN never wins). The raw bounds are clamped to the
 * envelope [P - (S-1)(T_n-1-t), min(P, (S-1)t)] and then made monotone
 * (Eq. (9)) and skip-free (Eq. (10)) by the suffix-minimum / reflection
 * procedure of the commented-out part of Sec. 3.2.2 of the paper's source.
 * For identical occupation inputs the result is bit-identical to a CPU fp32
 * evaluation in that order. 1 <= S <= RNNT_MAX_S. No workspace.
 */
int rnnt_prune_ranges(const rnnt_batch* batch, int32_t S,
                      const float* px_occ, const float* py_occ,
                      int32_t* ranges, void* stream);

/* ------------------------------------------------------------------------ */
/* Stage 4: full joiner on the pruned pairs, pruned recursion, backward      */
/* ------------------------------------------------------------------------ */

/* Workspace bytes for rnnt_pruned_joiner. */
size_t rnnt_pruned_joiner_workspace_size(int32_t N, int32_t T, int32_t S, int32_t J,
                                         int32_t V, int32_t dtype);

/* Full joiner at u = ranges[n,t,s] only (Sec. 3.2): h = tanh(enc[n,t] + dec[n,u]),
 * logits = h W + bias, lse = log sum_v exp(logits). The log-softmax is reduced
 * in the GEMM epilogue: each (row, 64-column slice) keeps a partial
 * (max, sum exp) and the target and blank logits.
 *
 * enc [N, T, J], dec [N, U+1, J], W [J, V], bias [V] (nullable = 0): dtype
 *   RNNT_F32 (float) or RNNT_BF16 (bfloat16 bits); accumulation is fp32.
 * ranges [N, T, S] int32 from rnnt_prune_ranges (u values above u_len[n] mark
 *   absent slots).
 * Outputs, fp32 [N, T, S]: px = logits[y_{u+1}] - lse (u < U_n, else -inf),
 *   py = logits[blank] - lse, lse (0 for absent slots).
 * logits [N, T, S, V] fp32 (nullable, caller-owned, 16-byte aligned): when given, the logits
 *   are stored as well (entries of absent slots and padding frames are left
 *   untouched), so that rnnt_pruned_joiner_backward can stream them instead
 *   of recomputing the projection. This is the [N, T, S, V] memory the
 *   method's cost scales with (Sec. 3.2).
 */
int rnnt_pruned_joiner(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype,
                       const void* enc, const void* dec, const void* W, const void* bias,
                       const int32_t* ranges, float* px, float* py, float* lse, float* logits,
                       void* workspace, size_t workspace_bytes, void* stream);

/* rnnt_pruned_joiner that also keeps the logits of the backward's first
 * chunk of rows: head [head_rows, ldl] fp32 (ldl = V rounded up to a
 * multiple of 8; caller-owned, 16-byte aligned, nullable) receives the
 * logits of joiner rows 0 .. head_rows-1 in the library's own row order
 * (an opaque cache: pass it unmodified to rnnt_pruned_joiner_backward_ex
 * with the same head_rows). head_rows: a positive multiple of 128, normally
 * rnnt_pruned_joiner_backward_chunk_rows(); ignored when head is NULL. At
 * most 16,384 rows: a bounded buffer, not the [N, T, S, V] logits. */
int rnnt_pruned_joiner_ex(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype,
                          const void* enc, const void* dec, const void* W, const void* bias,
                          const int32_t* ranges, float* px, float* py, float* lse, float* logits,
                          float* head, int32_t head_rows, void* workspace, size_t workspace_bytes,
                          void* stream);

/* Workspace bytes for rnnt_pruned_loss (the algorithm it picks). */
size_t rnnt_pruned_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S);

/* The recursion of Eq. (3) on the pruned lattice (Sec. 3.2): entries outside
 * p_t <= u < p_t + S are -inf. px, py [N, T, S] fp32 are the band log-probs
 * (from rnnt_pruned_joiner). Outputs: loss [N] (+inf when no complete path
 * exists in the band, then occupations are 0); px_occ, py_occ [N, T, S]
 * (nullable) band occupations dL_tot/dpx, dL_tot/dpy in [0,1].
 */
int rnnt_pruned_loss(const rnnt_batch* batch, int32_t S,
                     const float* px, const float* py, const int32_t* ranges,
                     float* loss, float* px_occ, float* py_occ,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Algorithms of the pruned recursion (same results up to rounding order):
 *   RNNT_BAND_AUTO       the library's choice for the shapes;
 *   RNNT_BAND_WAVEFRONT  anti-diagonal wavefront, depth T_n + U_n steps;
 *   RNNT_BAND_SCAN       chunked scan over frames, depth about 2C + T_n / C
 *                        frame steps for chunks of C frames (S <= 16 only).
 */
#define RNNT_BAND_AUTO 0
#define RNNT_BAND_WAVEFRONT 1
#define RNNT_BAND_SCAN 2
#define RNNT_SCAN_MAX_S 16
#define RNNT_SCAN_MAX_CHUNK 32

/* Workspace bytes for rnnt_pruned_loss_ex with the given algorithm and chunk
 * (chunk 0 = the library's choice; 0 is returned for unsupported choices).
 */
size_t rnnt_pruned_loss_ex_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S,
                                          int32_t algorithm, int32_t chunk);

/* rnnt_pruned_loss with an explicit algorithm. The band recursion of
 * Eq. (3) composes frame by frame: inside a frame only symbol moves occur
 * (an affine recurrence over the band's slots in the log semiring) and the
 * blank moves map one frame's band onto the next, so RNNT_BAND_SCAN forms
 * the S x S transfer matrix of every chunk of `chunk` frames in parallel,
 * chains the matrices per utterance and replays each chunk from its
 * incoming messages. chunk in [1, RNNT_SCAN_MAX_CHUNK], or 0 for the
 * library's choice; ignored by the wavefront. Arguments, outputs and error
 * behaviour are those of rnnt_pruned_loss; RNNT_EUNSUPPORTED for the scan
 * with S > RNNT_SCAN_MAX_S.
 */
int rnnt_pruned_loss_ex(const rnnt_batch* batch, int32_t S, int32_t algorithm, int32_t chunk,
                        const float* px, const float* py, const int32_t* ranges,
                        float* loss, float* px_occ, float* py_occ,
                        void* workspace, size_t workspace_bytes, void* stream);

/* rnnt_pruned_loss for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same recursion (the library's choice of algorithm), with
 * its workspace in a static device array of the library, RNNT_SCRATCH_BYTES
 * per GPU, held from the first call on a GPU until the process ends. No
 * allocation of any kind happens in the call. Arguments, outputs and error
 * behaviour are those of rnnt_pruned_loss; a batch whose workspace would
 * exceed the scratch is refused with RNNT_EUNSUPPORTED before any device
 * call (rnnt_pruned_loss_workspace_size tells). The device that owns
 * `stream` must be current. Every call on a GPU uses that GPU's one scratch:
 * calls that overlap on one GPU (on different streams or host threads
 * without ordering) race and give undefined results. Nothing in the scratch
 * needs to start at zero: each call writes what it reads.
 */
#define RNNT_SCRATCH_BYTES (4u << 20)
int rnnt_pruned_loss_noalloc(const rnnt_batch* batch, int32_t S, const float* px, const float* py,
                             const int32_t* ranges, float* loss, float* px_occ, float* py_occ,
                             void* stream);

/* Workspace bytes for rnnt_pruned_joiner_backward. */
size_t rnnt_pruned_joiner_backward_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S,
                                                  int32_t J, int32_t V, int32_t dtype);

/* Gradients of sum_n scale[n] * pruned_loss[n] through the log-softmax, the
 * projection, tanh and the sum enc + dec, in chunks of rows (the S rows of
 * every valid frame, frames in batch order): d(logits), h and the d dec
 * pieces are held for one chunk at a time. The chunk's size depends on J, V
 * and the dtype only, never on N or T (8,192 to 16,384 rows: d(logits) of
 * about 16 MiB at V = 500), so without the forward's logits no [N, T, S, V]
 * array exists at any time.
 *
 * lse, px_occ, py_occ [N, T, S]: from rnnt_pruned_joiner / rnnt_pruned_loss.
 * logits [N, T, S, V] (nullable): the logits stored by rnnt_pruned_joiner
 *   for the same inputs; when null they are recomputed (one more GEMM).
 * Outputs (fp32): enc_grad [N, T, J], dec_grad [N, U+1, J] (required, 16-byte aligned);
 *   W_grad [J, V], bias_grad [V] (nullable);
 *   logits_grad [N, T, S, V] (nullable; debugging aid for small shapes).
 * Reductions run in a fixed order: results are bitwise reproducible.
 */
int rnnt_pruned_joiner_backward(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V,
                                int32_t dtype, const void* enc, const void* dec,
                                const void* W, const void* bias, const int32_t* ranges,
                                const float* lse, const float* logits,
                                const float* px_occ, const float* py_occ,
                                const float* scale, float* enc_grad, float* dec_grad,
                                float* W_grad, float* bias_grad, float* logits_grad,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes for rnnt_pruned_joiner_backward_ex with this chunk size
 * (0 = the library's choice; 0 is returned for an invalid chunk size). */
size_t rnnt_pruned_joiner_backward_ex_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S,
                                                     int32_t J, int32_t V, int32_t dtype,
                                                     int32_t chunk_rows);

/* Rows of the backward's chunk for these sizes and chunk request (0 = the
 * library's choice); 0 for an invalid request. */
int32_t rnnt_pruned_joiner_backward_chunk_rows(int32_t N, int32_t T, int32_t S, int32_t J, int32_t V,
                                               int32_t dtype, int32_t chunk_rows);

/* rnnt_pruned_joiner_backward with an explicit chunk size and, optionally,
 * the first chunk's logits kept by rnnt_pruned_joiner_ex.
 * chunk_rows: rows of a chunk (a positive multiple of 128, at most what
 *   keeps each chunk buffer below 2^31 bytes: RNNT_EUNSUPPORTED beyond), or 0
 *   for the library's choice. The results do not depend on the chunk size
 *   up to the summation order of dW and db; d enc and d dec are bitwise the
 *   same. A smaller chunk holds less memory and launches more kernels.
 * head, head_rows: the head written by rnnt_pruned_joiner_ex for the same
 *   inputs (nullable); head_rows must equal
 *   rnnt_pruned_joiner_backward_chunk_rows(..., chunk_rows) (RNNT_EINVAL
 *   otherwise). The first chunk's d(logits) is then streamed from it instead
 *   of recomputing its logits. Ignored when logits is given.
 * Everything else is as in rnnt_pruned_joiner_backward. */
int rnnt_pruned_joiner_backward_ex(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V,
                                   int32_t dtype, int32_t chunk_rows, const void* enc,
                                   const void* dec, const void* W, const void* bias,
                                   const int32_t* ranges, const float* lse, const float* logits,
                                   const float* head, int32_t head_rows,
                                   const float* px_occ, const float* py_occ, const float* scale,
                                   float* enc_grad, float* dec_grad, float* W_grad,
                                   float* bias_grad, float* logits_grad, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* The training loss (Sec. 3.3)                                              */
/* ------------------------------------------------------------------------ */

#define RNNT_REDUCE_SUM 0
#define RNNT_REDUCE_MEAN 1

/* The paper trains on a weighted sum of the simple loss (Sec. 3.1) and the
 * pruned loss (Sec. 3.2), Sec. 3.3 (0.5 and 1 in its experiments):
 *   loss[n] = simple_scale * simple_loss[n] + pruned_scale * pruned_loss[n]
 * and total[0] = sum_n loss[n] (RNNT_REDUCE_SUM) or that sum / N
 * (RNNT_REDUCE_MEAN), accumulated in fp64 in a fixed order. A term whose
 * scale is 0 contributes exactly 0, whatever its loss (the pruned part is
 * switched off during the warm-up of Sec. 4; pruned_loss may then be NULL).
 * simple_loss, pruned_loss [N] fp32 device (each required when its scale is
 * non-zero); scales >= 0; outputs loss [N] and total [1] fp32 device, at
 * least one given. Asynchronous on `stream`; no workspace. */
int rnnt_combine_losses(int32_t N, const float* simple_loss, const float* pruned_loss,
                        float simple_scale, float pruned_scale, int32_t reduction,
                        float* loss, float* total, void* stream);

/* ------------------------------------------------------------------------ */
/* Input validation (debugging aid; synchronous)                             */
/* ------------------------------------------------------------------------ */

/* Bits of the per-utterance flags written by rnnt_validate_inputs. */
#define RNNT_FLAG_T_LEN 1     /* t_len[n] outside [1, T]                                 */
#define RNNT_FLAG_U_LEN 2     /* u_len[n] outside [0, U]                                 */
#define RNNT_FLAG_SYMBOL 4    /* some y_{u+1}, u < U_n, outside [0, V)                   */
#define RNNT_FLAG_AM 8        /* am[n, t, v] not finite for some t < T_n                 */
#define RNNT_FLAG_LM 16       /* lm[n, u, v] not finite for some u <= U_n                */
#define RNNT_FLAG_ENC 32      /* enc[n, t, j] not finite for some t < T_n                */
#define RNNT_FLAG_DEC 64      /* dec[n, u, j] not finite for some u <= U_n               */
#define RNNT_FLAG_NO_BAND 128 /* U_n > (S-1) T_n: no complete path fits a band of width S
                                 (the pruned loss is then +inf)                         */

/* Checks every utterance of a batch against the problem statement of Sec. 2:
 * T_n frames with 1 <= T_n <= T, U_n tokens with 0 <= U_n <= U, each token
 * y_1..y_{U_n} in [0, V) (y_0 is the blank, Sec. 2), finite scores on the
 * utterance's own frames and tokens (padding is not inspected), and, for
 * S > 0, that a band of width S can hold a complete path (Sec. 3.2.2:
 * Eqs. (9)-(10) with p_0 = 0 allow at most U_n <= (S-1) T_n). The other
 * entry points never fail on such data (an utterance that breaks the
 * statement gets a NaN loss, an infeasible band +inf); this call says why.
 *
 * am [N, T, V], lm [N, U+1, V] fp32 and enc [N, T, J], dec [N, U+1, J]
 * (dtype RNNT_F32 or RNNT_BF16) are device pointers, each nullable (not
 * inspected). S = 0 skips the band check; J and dtype are read only with enc
 * or dec. flags [N] int32 device (required): the RNNT_FLAG_* bits of each
 * utterance, 0 when it is valid. n_bad (host, nullable): the number of
 * utterances with a non-zero flag. Enqueues on `stream` and waits for it
 * (synchronous), so it is not meant for a training loop's hot path.
 */
int rnnt_validate_inputs(const rnnt_batch* batch, int32_t V, int32_t S, int32_t J, int32_t dtype,
                         const float* am, const float* lm, const void* enc, const void* dec,
                         int32_t* flags, int32_t* n_bad, void* stream);

/* ------------------------------------------------------------------------ */
/* For comparison: the unpruned loss with the same joiner                    */
/* ------------------------------------------------------------------------ */

/* Workspace bytes for rnnt_full_loss. */
size_t rnnt_full_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t J, int32_t V, int32_t dtype);

/* The RNN-T loss of Sec. 2 with the full joiner evaluated at every (t, u) of
 * the lattice, the (N, T, U+1, V) computation that the pruned loss avoids
 * (Sec. 1, Sec. 3.2), and its gradients: the same joiner, recursion and
 * backward kernels as the pruned path, with every row of the lattice as the
 * "band" (S = U+1, all p_t = 0). It is the in-library comparison for the
 * method's memory and speed claims.
 *
 * enc, dec, W, bias, dtype: as in rnnt_pruned_joiner. scale [N] (nullable).
 * Outputs: loss [N] fp32 (required); enc_grad [N, T, J], dec_grad [N, U+1, J]
 *   (required, 16-byte aligned); W_grad [J, V], bias_grad [V] (nullable);
 *   logits [N, T, U+1, V] fp32 (nullable, 16-byte aligned): when given, the
 *   unpruned logits are stored and streamed by the backward, as a framework
 *   that materialises them would; when null they are recomputed in row
 *   chunks.
 */
int rnnt_full_loss(const rnnt_batch* batch, int32_t J, int32_t V, int32_t dtype,
                   const void* enc, const void* dec, const void* W, const void* bias,
                   const float* scale, float* loss, float* enc_grad, float* dec_grad,
                   float* W_grad, float* bias_grad, float* logits,
                   void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Kernel timing (opt-in; for benchmarks and profiling)                      */
/* ------------------------------------------------------------------------ */

/* Enable (on != 0) or disable recording of per-kernel HIP events. While
 * enabled, every kernel launch of the library is bracketed by two events
 * recorded on its stream, under a fixed kernel name ("joiner_fwd",
 * "joiner_dlogits", "joiner_dh", "joiner_dw", "lattice", "band", ...). */
int rnnt_profile_enable(int on);

/* Restrict recording to the kernels named in `names` (comma-separated, as in
 * rnnt_profile_names); NULL or "" records every kernel again. Each recorded
 * launch costs two event packets on its stream, so timing one kernel inside
 * a throughput measurement should select just that kernel. */
int rnnt_profile_select(const char* names);

/* Forget all records (waits for the recorded events to complete). */
int rnnt_profile_reset(void);

/* Number of recorded launches of kernel `name` and their summed duration in
 * milliseconds. Synchronises on the recorded events. */
int rnnt_profile_query(const char* name, int32_t* launches, double* total_ms);

/* Comma-separated names of the kernels recorded so far, into buf[cap]. */
int rnnt_profile_names(char* buf, size_t cap);

#ifdef __cplusplus
}
#endif

#endif /* RNNT_PRUNED_H */
