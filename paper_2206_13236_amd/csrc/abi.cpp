// C ABI of the pruned RNN-T library: argument checks, workspace layout and
// launch sequencing. Every check runs on the host before any HIP call, so a
// rejected call enqueues nothing. No entry point allocates, frees or
// synchronises.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "rnnt_pruned.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return RNNT_OK;
}

int hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return ok();
  return fail(RNNT_EHIP, "%s: %s", where, hipGetErrorString(e));
}

// Bump allocator over the caller's workspace. With base == nullptr it only
// measures, so the *_workspace_size queries and the entry points share one
// layout.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t n) {
    off = (off + 255) / 256 * 256;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

const long long kI32 = 0x7fffffffll;

int check_batch(const rnnt_batch* b, bool need_symbols_ptr) {
  if (!b) return fail(RNNT_EINVAL, "batch is NULL");
  if (b->N < 1) return fail(RNNT_EINVAL, "N must be >= 1 (got %d)", b->N);
  if (b->T < 1) return fail(RNNT_EINVAL, "T must be >= 1 (got %d)", b->T);
  if (b->U < 0) return fail(RNNT_EINVAL, "U must be >= 0 (got %d)", b->U);
  if (b->U > RNNT_MAX_U) return fail(RNNT_EUNSUPPORTED, "U = %d exceeds RNNT_MAX_U = %d", b->U, RNNT_MAX_U);
  if (!b->t_len || !b->u_len) return fail(RNNT_EINVAL, "t_len and u_len must be device pointers");
  if (need_symbols_ptr && b->U > 0 && !b->symbols) return fail(RNNT_EINVAL, "symbols is NULL with U > 0");
  if ((long long)b->N * b->T * (b->U + 1) > kI32) return fail(RNNT_EUNSUPPORTED, "N*T*(U+1) exceeds 2^31-1");
  return RNNT_OK;
}

BatchDev to_dev(const rnnt_batch* b) {
  BatchDev d;
  d.N = b->N;
  d.T = b->T;
  d.U = b->U;
  d.t_len = b->t_len;
  d.u_len = b->u_len;
  d.symbols = b->symbols;
  d.blank = b->blank;
  return d;
}

int ldw_of(int U) { return (U + 1 + 3) / 4 * 4; }

struct SimpleWs {
  float* m_a;
  float* m_l;
  float* Z;
  float* px;
  float* py;
  DiagT* pxd;
  DiagT* pyd;
  double* alpha;
  double* beta;
  double* Lutt;
  float* Wt;
  double* ry;
  double* cpx;
  double* cpy;
  float* npart;
  int nsplit;
  float* lpart;
  int lsplit;
  double* rx;
  double* Gx;
  double* Gy;
  float* Zlm;
  float* lavg;
  float* Zac;
  float* q;
  float* su;
  size_t bytes;
};

SimpleWs simple_layout(void* base, int N, int T, int U, int V) {
  Carve c(base);
  SimpleWs w;
  const size_t NT = (size_t)N * T, NU = (size_t)N * (U + 1), L = NT * (U + 1);
  w.m_a = c.take<float>(NT);
  w.m_l = c.take<float>(NU);
  w.Z = c.take<float>(L);
  w.px = c.take<float>(L);
  w.py = c.take<float>(L);
  const size_t LD = (size_t)N * lattice_diag_cells(T, U);
  w.pxd = c.take<DiagT>(LD);
  w.pyd = c.take<DiagT>(LD);
  w.alpha = c.take<double>(LD);
  w.beta = c.take<double>(LD);
  w.Lutt = c.take<double>((size_t)N);
  w.Wt = c.take<float>(NT * ldw_of(U));
  w.ry = c.take<double>(NT);
  w.cpx = c.take<double>((size_t)N * lattice_colblocks(T) * (U + 1));
  w.cpy = c.take<double>((size_t)N * lattice_colblocks(T) * (U + 1));
  w.nsplit = normalizer_splits(N, T, U, V);
  w.npart = c.take<float>((size_t)w.nsplit * L);
  w.lsplit = dlm_splits(N, T, U, V);
  const int gsplit = simple_grad_splits(N, T, U, V);
  w.lpart = c.take<float>((size_t)(gsplit > w.lsplit ? gsplit : w.lsplit) * NU * V);
  w.rx = c.take<double>(NT);
  w.Gx = c.take<double>(NU);
  w.Gy = c.take<double>(NU);
  w.Zlm = c.take<float>(NU);
  w.lavg = c.take<float>((size_t)N * V);
  w.Zac = c.take<float>(NT);
  w.q = c.take<float>((size_t)N * V);
  w.su = c.take<float>(NU);
  w.bytes = c.off;
  return w;
}

// Arguments shared by the simple loss's forward and backward entry points:
// everything but the caller's outputs. The occupation kernel always leaves
// the backward's state (W(t,u), row and column sums) in the workspace.
SimpleArgs simple_args(const rnnt_batch* batch, int V, const float* am, const float* lm, const float* scale,
                       float lm_only, float am_only, const SimpleWs& w) {
  SimpleArgs a{};
  a.b = to_dev(batch);
  a.V = V;
  a.lm_only = lm_only;
  a.am_only = am_only;
  a.am = am;
  a.lm = lm;
  a.scale = scale;
  a.m_a = w.m_a;
  a.m_l = w.m_l;
  a.Z = w.Z;
  a.npart = w.npart;
  a.nsplit = w.nsplit;
  a.lpart = w.lpart;
  a.lsplit = w.lsplit;
  a.px = w.px;
  a.py = w.py;
  a.pxd = w.pxd;
  a.pyd = w.pyd;
  a.alpha = w.alpha;
  a.beta = w.beta;
  a.Lutt = w.Lutt;
  a.Wt = w.Wt;
  a.ldw = ldw_of(batch->U);
  a.ry = w.ry;
  a.cpx = w.cpx;
  a.cpy = w.cpy;
  a.ncolblk = lattice_colblocks(batch->T);
  a.rx = w.rx;
  a.Gx = w.Gx;
  a.Gy = w.Gy;
  a.Zlm = w.Zlm;
  a.lavg = w.lavg;
  a.Zac = w.Zac;
  a.q = w.q;
  a.su = w.su;
  return a;
}

struct JoinerFwdWs {
  int* frame_off;
  int4* rowinfo;
  float2* part;
  float* tgt;
  float* blk;
  void* h[2];
  void* wt;
  int chunk_rows;
  size_t bytes;
};

JoinerFwdWs joiner_fwd_layout(void* base, int N, int T, int S, int J, int V, int bf16) {
  Carve c(base);
  JoinerFwdWs w;
  const size_t M = (size_t)N * T * S;
  w.chunk_rows = joiner_fwd_chunk_rows(N, T, S, J, bf16);
  w.frame_off = c.take<int>((size_t)N + 1);
  w.rowinfo = c.take<int4>(M);
  w.part = c.take<float2>(M * joiner_nparts(V));
  w.tgt = c.take<float>(M);
  w.blk = c.take<float>(M);
  // two h slots: a chunk's GEMM launch writes the next chunk's h beside it
  const size_t h_elems = joiner_fwd_uses_hbuf(bf16) ? (size_t)w.chunk_rows * J : 0;
  for (int k = 0; k < 2; ++k)
    w.h[k] = h_elems == 0 ? nullptr : bf16 ? (void*)c.take<uint16_t>(h_elems) : (void*)c.take<float>(h_elems);
  w.wt = bf16 ? (void*)c.take<uint16_t>((size_t)V * J) : nullptr;
  w.bytes = c.off;
  return w;
}

struct JoinerBwdWs {
  int* frame_off;
  int* frame_nt;
  int* frame_p;
  int4* rowinfo;
  void* dl[2];
  void* dlT[2];
  void* wpad;
  void* wt;
  float* dpre[2];
  float* enc_part;
  void* hbuf[3];
  void* hT[3];
  float* dw_part;
  float* db_part;
  int chunk_rows, splits, n_db_rows;
  size_t bytes;
};

// stored_only: the caller always passes the logits (the unpruned loss), so
// the backward streams them chunk by chunk through slot 0 and the rings of
// the recomputed path's pipeline shrink to that one slot.
JoinerBwdWs joiner_bwd_layout(void* base, int N, int T, int S, int J, int V, int bf16, int chunk_request = 0,
                              bool stored_only = false) {
  Carve c(base);
  JoinerBwdWs w;
  const size_t M = (size_t)N * T * S;
  w.chunk_rows = joiner_bwd_chunk_rows(N, T, S, J, V, bf16, chunk_request);
  w.splits = joiner_bwd_splits(J, V, w.chunk_rows, bf16);
  w.n_db_rows = joiner_db_rows(w.chunk_rows);
  w.frame_off = c.take<int>((size_t)N + 1);
  w.frame_nt = c.take<int>((size_t)N * T);
  w.frame_p = c.take<int>((size_t)N * T);
  w.rowinfo = c.take<int4>(M);
  // rings of chunk buffers: 2 slots of d(logits) and its bf16 transpose, 3
  // of h and its bf16 transpose (1 of each when stored_only)
  const size_t dl_elems = (size_t)w.chunk_rows * joiner_ldl(V);
  const size_t h_elems = (size_t)w.chunk_rows * J;
  for (int k = 0; k < 2; ++k) {
    if (stored_only && k > 0) {
      w.dl[k] = w.dl[0];
      w.dlT[k] = w.dlT[0];
      continue;
    }
    w.dl[k] = bf16 ? (void*)c.take<uint16_t>(dl_elems) : (void*)c.take<float>(dl_elems);
    w.dlT[k] = bf16 ? (void*)c.take<uint16_t>(dl_elems) : nullptr;
  }
  for (int k = 0; k < 3; ++k) {
    if (stored_only && k > 0) {
      w.hbuf[k] = w.hbuf[0];
      w.hT[k] = w.hT[0];
      continue;
    }
    w.hbuf[k] = bf16 ? (void*)c.take<uint16_t>(h_elems) : (void*)c.take<float>(h_elems);
    w.hT[k] = bf16 ? (void*)c.take<uint16_t>(h_elems) : nullptr;
  }
  w.wpad = (bf16 && V % 8 != 0) ? (void*)c.take<uint16_t>((size_t)J * joiner_ldl(V)) : nullptr;
  w.wt = bf16 ? (void*)c.take<uint16_t>((size_t)V * J) : nullptr;
  for (int k = 0; k < 2; ++k) w.dpre[k] = (stored_only && k > 0) ? w.dpre[0] : c.take<float>((size_t)w.chunk_rows * J);
  w.enc_part = c.take<float>((M + 127) / 128 * 2 * J);
  w.dw_part = c.take<float>((size_t)w.splits * J * V);
  w.db_part = c.take<float>((size_t)w.n_db_rows * V);
  w.bytes = c.off;
  return w;
}

int check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return RNNT_OK;
  if (!ws) return fail(RNNT_EWORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0) return fail(RNNT_EWORKSPACE, "workspace must be 256-byte aligned");
  if (have < need) return fail(RNNT_EWORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return RNNT_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

int check_joiner_sizes(const rnnt_batch* b, int S, int J, int V, int dtype) {
  if (S < 1 || S > RNNT_MAX_S) return fail(RNNT_EUNSUPPORTED, "S = %d outside [1, %d]", S, RNNT_MAX_S);
  if (V < 1) return fail(RNNT_EINVAL, "V must be >= 1 (got %d)", V);
  if (b->blank < 0 || b->blank >= V) return fail(RNNT_EINVAL, "blank = %d outside [0, V)", b->blank);
  if (J < 8 || J % 8 != 0) return fail(RNNT_EUNSUPPORTED, "J = %d must be a positive multiple of 8", J);
  if (dtype != RNNT_F32 && dtype != RNNT_BF16) return fail(RNNT_EINVAL, "dtype must be RNNT_F32 or RNNT_BF16");
  if ((long long)b->N * b->T * S > kI32) return fail(RNNT_EUNSUPPORTED, "N*T*S exceeds 2^31-1");
  // operands are read through 32-bit buffer offsets: each array stays below 2^31 bytes
  const long long esz = dtype == RNNT_BF16 ? 2 : 4;
  if ((long long)b->N * b->T * J * esz > kI32 || (long long)b->N * (b->U + 1) * J * esz > kI32 ||
      (long long)J * joiner_ldl(V) * esz > kI32)
    return fail(RNNT_EUNSUPPORTED, "enc, dec or W exceeds 2^31-1 bytes");
  // the row-chunk buffers (h, d(logits), the d dec pieces) must hold one
  // 128-row tile below 2^31 bytes
  if (joiner_bwd_chunk_max_rows(J, V) < 128)
    return fail(RNNT_EUNSUPPORTED, "J = %d or V = %d too large for one 128-row chunk", J, V);
  if ((size_t)b->T * sizeof(int) > 64 * 1024) return fail(RNNT_EUNSUPPORTED, "T = %d too large", b->T);
  return RNNT_OK;
}

int check_chunk_request(int J, int V, int chunk_rows) {
  if (chunk_rows == 0) return RNNT_OK;
  if (chunk_rows < 128 || chunk_rows % 128 != 0)
    return fail(RNNT_EINVAL, "chunk_rows = %d must be 0 or a positive multiple of 128", chunk_rows);
  if (chunk_rows > joiner_bwd_chunk_max_rows(J, V))
    return fail(RNNT_EUNSUPPORTED, "chunk_rows = %d exceeds %d (buffers below 2^31 bytes)", chunk_rows,
                joiner_bwd_chunk_max_rows(J, V));
  return RNNT_OK;
}

JoinerArgs joiner_args(const rnnt_batch* batch, int S, int J, int V, int dtype, const void* enc, const void* dec,
                       const void* W, const void* bias, const int32_t* ranges) {
  JoinerArgs a{};
  a.b = to_dev(batch);
  a.S = S;
  a.J = J;
  a.V = V;
  a.bf16 = dtype == RNNT_BF16;
  a.enc = enc;
  a.dec = dec;
  a.W = W;
  a.bias = bias;
  a.ranges = ranges;
  return a;
}

void set_joiner_fwd(JoinerArgs& a, const JoinerFwdWs& w, float* px, float* py, float* lse, float* logits) {
  a.ldl = joiner_ldl(a.V);
  a.frame_off = w.frame_off;
  a.rowinfo = w.rowinfo;
  a.part = w.part;
  a.nparts = joiner_nparts(a.V);
  a.tgt = w.tgt;
  a.blk = w.blk;
  a.hbuf = w.h[0];
  a.hring[0] = w.h[0];
  a.hring[1] = w.h[1];
  a.wt = w.wt;
  a.chunk_rows = w.chunk_rows;
  a.px = px;
  a.py = py;
  a.lse = lse;
  a.logits = logits;
}

void set_joiner_bwd(JoinerArgs& a, const JoinerBwdWs& w, const float* lse, const float* logits, const float* gx,
                    const float* gy, const float* scale, float* enc_grad, float* dec_grad, float* W_grad,
                    float* bias_grad, float* logits_grad) {
  a.frame_off = w.frame_off;
  a.frame_nt = w.frame_nt;
  a.frame_p = w.frame_p;
  a.rowinfo = w.rowinfo;
  a.lse_in = lse;
  a.logits_in = logits;
  a.gxo = gx;
  a.gyo = gy;
  a.scale = scale;
  a.dl = w.dl[0];
  a.dlT = w.dlT[0];
  a.hT = w.hT[0];
  for (int k = 0; k < 3; ++k) {
    a.hring[k] = w.hbuf[k];
    a.hTring[k] = w.hT[k];
  }
  for (int k = 0; k < 2; ++k) {
    a.dlring[k] = w.dl[k];
    a.dlTring[k] = w.dlT[k];
    a.dpring[k] = w.dpre[k];
  }
  a.wpad = w.wpad;
  a.wt = w.wt;
  a.ldl = joiner_ldl(a.V);
  a.chunk_rows = w.chunk_rows;
  a.dpre = w.dpre[0];
  a.enc_part = w.enc_part;
  a.hbuf = w.hbuf[0];
  a.dw_part = w.dw_part;
  a.splits = w.splits;
  a.db_part = w.db_part;
  a.n_db_rows = w.n_db_rows;
  a.enc_grad = enc_grad;
  a.dec_grad = dec_grad;
  a.W_grad = W_grad;
  a.bias_grad = bias_grad;
  a.logits_grad = logits_grad;
}

// The unpruned loss's backward chunk: about 256 MiB of d(logits) (within the
// 32-bit limit), a comparison path that holds the [N, T, U+1, V] scale of
// memory by design and runs fewest, fullest launches.
int full_chunk_rows(int J, int V, int bf16) {
  long long r = (256ll << 20) / ((long long)joiner_ldl(V) * (bf16 ? 2 : 4)) / 128 * 128;
  const long long lim = joiner_bwd_chunk_max_rows(J, V);
  if (r > lim) r = lim;
  return (int)(r < 128 ? 128 : r);
}

// Workspace of rnnt_full_loss: the lattice-sized arrays, then one region
// that the joiner's forward and backward use in turn.
struct FullWs {
  int* ranges;
  float *px, *py, *lse, *gx, *gy;
  DiagT *pxd, *pyd;
  double *alpha, *beta, *Lutt, *ry, *rx, *cpx, *cpy;
  void* joiner;
  size_t bytes;
};

FullWs full_layout(void* base, int N, int T, int U, int J, int V, int bf16) {
  Carve c(base);
  FullWs w;
  const int S = U + 1;
  const size_t L = (size_t)N * T * S;
  w.ranges = c.take<int>(L);
  w.px = c.take<float>(L);
  w.py = c.take<float>(L);
  w.lse = c.take<float>(L);
  w.gx = c.take<float>(L);
  w.gy = c.take<float>(L);
  const size_t LD = (size_t)N * lattice_diag_cells(T, U);
  w.pxd = c.take<DiagT>(LD);
  w.pyd = c.take<DiagT>(LD);
  w.alpha = c.take<double>(LD);
  w.beta = c.take<double>(LD);
  w.Lutt = c.take<double>((size_t)N);
  w.ry = c.take<double>((size_t)N * T);
  w.rx = c.take<double>((size_t)N * T);
  w.cpx = c.take<double>((size_t)N * lattice_colblocks(T) * S);
  w.cpy = c.take<double>((size_t)N * lattice_colblocks(T) * S);
  const size_t jf = joiner_fwd_layout(nullptr, N, T, S, J, V, bf16).bytes;
  const size_t jb = joiner_bwd_layout(nullptr, N, T, S, J, V, bf16, full_chunk_rows(J, V, bf16), true).bytes;
  w.joiner = c.take<unsigned char>(jf > jb ? jf : jb);
  w.bytes = c.off;
  return w;
}

// Workspace of rnnt_pruned_loss_noalloc: a file-scope device array, one copy
// per GPU for the life of the process. Host code never passes its name to a
// kernel (in host code it is a stand-in, not a device address): each
// device's address comes from hipGetSymbolAddress, taken once per device with
// that device current and kept in g_scratch_ptr.
constexpr size_t kScratchBytes = RNNT_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// The scratch's address on the device that owns `stream` (which must be the
// current device), resolved on the first call on that device.
int scratch_for(hipStream_t stream, void** out) {
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (stream) {
    hipDevice_t sd = -1;
    e = hipStreamGetDevice(stream, &sd);
    if (e != hipSuccess) return hip_status(e, "hipStreamGetDevice");
    if ((int)sd != cur) return fail(RNNT_EINVAL, "the stream's device (%d) must be the current device (%d)", (int)sd, cur);
  }
  if (cur < 0 || cur >= kMaxDevices) return fail(RNNT_EUNSUPPORTED, "device %d beyond %d devices", cur, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[cur]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(RNNT_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[cur] = p;
  }
  *out = g_scratch_ptr[cur];
  return RNNT_OK;
}

}  // namespace

extern "C" {

int rnnt_abi_version(void) { return 8; }

const char* rnnt_last_error(void) { return g_err.c_str(); }

size_t rnnt_simple_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t V) {
  if (N < 1 || T < 1 || U < 0 || V < 1) return 0;
  return simple_layout(nullptr, N, T, U, V).bytes;
}

int check_smoothing(float lm_only, float am_only) {
  if (!(lm_only >= 0.f && am_only >= 0.f && lm_only + am_only <= 1.f))
    return fail(RNNT_EINVAL, "smoothing weights must be >= 0 with sum <= 1 (got %g, %g)", lm_only, am_only);
  return RNNT_OK;
}

int rnnt_simple_loss(const rnnt_batch* batch, int32_t V, const float* am, const float* lm, const float* scale,
                     float lm_only_scale, float am_only_scale, float* loss, float* px_occ, float* py_occ,
                     float* px, float* py, float* am_grad, float* lm_grad, void* workspace,
                     size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  if (V < 1) return fail(RNNT_EINVAL, "V must be >= 1 (got %d)", V);
  if (batch->blank < 0 || batch->blank >= V) return fail(RNNT_EINVAL, "blank = %d outside [0, V)", batch->blank);
  if (!am || !lm) return fail(RNNT_EINVAL, "am and lm are required");
  if (!loss || !px_occ || !py_occ) return fail(RNNT_EINVAL, "loss, px_occ and py_occ are required");
  if ((px == nullptr) != (py == nullptr)) return fail(RNNT_EINVAL, "px and py must be given together");
  rc = check_smoothing(lm_only_scale, am_only_scale);
  if (rc) return rc;
  const SimpleWs need = simple_layout(nullptr, batch->N, batch->T, batch->U, V);
  rc = check_ws(workspace, workspace_bytes, need.bytes);
  if (rc) return rc;
  const SimpleWs w = simple_layout(workspace, batch->N, batch->T, batch->U, V);
  hipStream_t s = static_cast<hipStream_t>(stream);
  SimpleArgs a = simple_args(batch, V, am, lm, scale, lm_only_scale, am_only_scale, w);
  if (px) a.px = px;
  if (py) a.py = py;
  a.loss = loss;
  a.gx = px_occ;
  a.gy = py_occ;
  a.am_grad = am_grad;
  a.lm_grad = lm_grad;
  hipError_t e = launch_rowmax(a, s);
  if (e == hipSuccess) e = launch_smoothing_stats(a, s);
  if (e == hipSuccess) e = launch_normalizer(a, s);
  if (e == hipSuccess) e = launch_lattice(a, s);
  if (e == hipSuccess && (am_grad || lm_grad)) e = launch_simple_grads(a, s);
  return hip_status(e, "rnnt_simple_loss");
}

int rnnt_simple_loss_backward(const rnnt_batch* batch, int32_t V, const float* am, const float* lm,
                              const float* scale, float lm_only_scale, float am_only_scale,
                              const float* px_occ, float* am_grad, float* lm_grad,
                              void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  if (V < 1) return fail(RNNT_EINVAL, "V must be >= 1 (got %d)", V);
  if (batch->blank < 0 || batch->blank >= V) return fail(RNNT_EINVAL, "blank = %d outside [0, V)", batch->blank);
  if (!am || !lm || !px_occ) return fail(RNNT_EINVAL, "am, lm and px_occ are required");
  if (!am_grad && !lm_grad) return fail(RNNT_EINVAL, "at least one of am_grad and lm_grad is required");
  rc = check_smoothing(lm_only_scale, am_only_scale);
  if (rc) return rc;
  const SimpleWs need = simple_layout(nullptr, batch->N, batch->T, batch->U, V);
  rc = check_ws(workspace, workspace_bytes, need.bytes);
  if (rc) return rc;
  const SimpleWs w = simple_layout(workspace, batch->N, batch->T, batch->U, V);
  SimpleArgs a = simple_args(batch, V, am, lm, scale, lm_only_scale, am_only_scale, w);
  a.gx = const_cast<float*>(px_occ);  // read only by the gradient kernels
  a.am_grad = am_grad;
  a.lm_grad = lm_grad;
  return hip_status(launch_simple_grads(a, static_cast<hipStream_t>(stream)), "rnnt_simple_loss_backward");
}

int rnnt_prune_ranges(const rnnt_batch* batch, int32_t S, const float* px_occ, const float* py_occ,
                      int32_t* ranges, void* stream) {
  int rc = check_batch(batch, false);
  if (rc) return rc;
  if (S < 1 || S > RNNT_MAX_S) return fail(RNNT_EUNSUPPORTED, "S = %d outside [1, %d]", S, RNNT_MAX_S);
  if (!px_occ || !py_occ || !ranges) return fail(RNNT_EINVAL, "px_occ, py_occ and ranges are required");
  if (prune_smem_bytes(batch->T) > 64 * 1024) return fail(RNNT_EUNSUPPORTED, "T = %d too large", batch->T);
  if ((long long)batch->N * batch->T * S > kI32) return fail(RNNT_EUNSUPPORTED, "N*T*S exceeds 2^31-1");
  hipError_t e = launch_prune(to_dev(batch), S, px_occ, py_occ, ranges, static_cast<hipStream_t>(stream));
  return hip_status(e, "rnnt_prune_ranges");
}

size_t rnnt_pruned_joiner_workspace_size(int32_t N, int32_t T, int32_t S, int32_t J, int32_t V, int32_t dtype) {
  if (N < 1 || T < 1 || S < 1 || J < 1 || V < 1) return 0;
  return joiner_fwd_layout(nullptr, N, T, S, J, V, dtype == RNNT_BF16).bytes;
}

int rnnt_pruned_joiner_ex(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype, const void* enc,
                          const void* dec, const void* W, const void* bias, const int32_t* ranges, float* px,
                          float* py, float* lse, float* logits, float* head, int32_t head_rows, void* workspace,
                          size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  rc = check_joiner_sizes(batch, S, J, V, dtype);
  if (rc) return rc;
  if (!enc || !dec || !W || !ranges) return fail(RNNT_EINVAL, "enc, dec, W and ranges are required");
  if (!px || !py || !lse) return fail(RNNT_EINVAL, "px, py and lse are required");
  if (!aligned16(logits) || !aligned16(head)) return fail(RNNT_EINVAL, "logits and head must be 16-byte aligned");
  if (head && (head_rows < 128 || head_rows % 128 != 0 || head_rows > joiner_bwd_chunk_max_rows(J, V)))
    return fail(RNNT_EINVAL, "head_rows = %d must be a positive multiple of 128 within the chunk limit", head_rows);
  const int bf = dtype == RNNT_BF16;
  rc = check_ws(workspace, workspace_bytes, joiner_fwd_layout(nullptr, batch->N, batch->T, S, J, V, bf).bytes);
  if (rc) return rc;
  const JoinerFwdWs w = joiner_fwd_layout(workspace, batch->N, batch->T, S, J, V, bf);
  JoinerArgs a = joiner_args(batch, S, J, V, dtype, enc, dec, W, bias, ranges);
  set_joiner_fwd(a, w, px, py, lse, logits);
  a.head = head;
  a.head_rows = head ? head_rows : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_joiner_prep(a, s);
  if (e == hipSuccess) e = launch_joiner_fwd(a, s);
  return hip_status(e, "rnnt_pruned_joiner");
}

int rnnt_pruned_joiner(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype, const void* enc,
                       const void* dec, const void* W, const void* bias, const int32_t* ranges, float* px, float* py,
                       float* lse, float* logits, void* workspace, size_t workspace_bytes, void* stream) {
  return rnnt_pruned_joiner_ex(batch, S, J, V, dtype, enc, dec, W, bias, ranges, px, py, lse, logits, nullptr, 0,
                               workspace, workspace_bytes, stream);
}

// Workspace of rnnt_pruned_loss: the band in a diagonal-major layout of
// band_slots(U, S) slots per diagonal (the per-slot meta only on the slot layout).
struct BandWs {
  DiagT *pxd, *pyd;
  uint32_t* meta;
  double *alpha, *beta, *Lutt;
  size_t bytes;
};

BandWs band_layout(void* base, int N, int T, int U, int S) {
  Carve c(base);
  BandWs w;
  const size_t cells = (size_t)N * band_diagonals(T, U, S) * band_slots(U, S);
  w.pxd = c.take<DiagT>(cells);
  w.pyd = c.take<DiagT>(cells);
  w.meta = band_masked(U, S) ? nullptr : c.take<uint32_t>(cells);
  w.alpha = c.take<double>(cells);
  w.beta = c.take<double>(cells);
  w.Lutt = c.take<double>((size_t)N);
  w.bytes = c.off;
  return w;
}

// Workspace of the chunked scan.
struct ScanWs {
  double *M, *E, *V, *Wb, *Lutt;
  size_t bytes;
};

ScanWs scan_layout(void* base, int N, int T, int S, int C) {
  Carve c(base);
  ScanWs w;
  const size_t nc = (size_t)(T + C - 1) / C;
  w.M = c.take<double>((size_t)N * nc * S * S);
  w.E = c.take<double>((size_t)N * S);
  w.V = c.take<double>((size_t)N * nc * S);
  w.Wb = c.take<double>((size_t)N * nc * S);
  w.Lutt = c.take<double>((size_t)N);
  w.bytes = c.off;
  return w;
}

// The algorithm rnnt_pruned_loss uses: the scan wherever it applies.
int band_auto(int S) { return S <= kScanMaxS ? RNNT_BAND_SCAN : RNNT_BAND_WAVEFRONT; }

size_t pruned_ws_bytes(int N, int T, int U, int S, int algorithm, int chunk) {
  if (N < 1 || T < 1 || U < 0 || S < 1) return 0;
  if (algorithm == RNNT_BAND_AUTO) algorithm = band_auto(S);
  if (algorithm == RNNT_BAND_WAVEFRONT) return band_layout(nullptr, N, T, U, S).bytes;
  if (algorithm != RNNT_BAND_SCAN || S > kScanMaxS || chunk < 0 || chunk > kScanMaxC) return 0;
  return scan_layout(nullptr, N, T, S, chunk ? chunk : band_scan_chunk(T)).bytes;
}

size_t rnnt_pruned_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S) {
  return pruned_ws_bytes(N, T, U, S, RNNT_BAND_AUTO, 0);
}

size_t rnnt_pruned_loss_ex_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S, int32_t algorithm,
                                          int32_t chunk) {
  return pruned_ws_bytes(N, T, U, S, algorithm, chunk);
}

int rnnt_pruned_loss(const rnnt_batch* batch, int32_t S, const float* px, const float* py, const int32_t* ranges,
                     float* loss, float* px_occ, float* py_occ, void* workspace, size_t workspace_bytes,
                     void* stream) {
  return rnnt_pruned_loss_ex(batch, S, RNNT_BAND_AUTO, 0, px, py, ranges, loss, px_occ, py_occ, workspace,
                             workspace_bytes, stream);
}

int rnnt_pruned_loss_ex(const rnnt_batch* batch, int32_t S, int32_t algorithm, int32_t chunk, const float* px,
                        const float* py, const int32_t* ranges, float* loss, float* px_occ, float* py_occ,
                        void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, false);
  if (rc) return rc;
  if (S < 1 || S > RNNT_MAX_S) return fail(RNNT_EUNSUPPORTED, "S = %d outside [1, %d]", S, RNNT_MAX_S);
  if (!px || !py || !ranges || !loss) return fail(RNNT_EINVAL, "px, py, ranges and loss are required");
  if (algorithm < RNNT_BAND_AUTO || algorithm > RNNT_BAND_SCAN)
    return fail(RNNT_EINVAL, "unknown algorithm %d", algorithm);
  if (algorithm == RNNT_BAND_AUTO) algorithm = band_auto(S);
  if (algorithm == RNNT_BAND_SCAN) {
    if (S > kScanMaxS) return fail(RNNT_EUNSUPPORTED, "the scan needs S <= %d (S = %d)", kScanMaxS, S);
    if (chunk < 0 || chunk > kScanMaxC)
      return fail(RNNT_EINVAL, "chunk = %d outside [0, %d]", chunk, kScanMaxC);
    if ((long long)batch->N * batch->T * S > kI32)
      return fail(RNNT_EUNSUPPORTED, "N*T*S is too large");
    const int C = chunk ? chunk : band_scan_chunk(batch->T);
    const ScanWs need = scan_layout(nullptr, batch->N, batch->T, S, C);
    rc = check_ws(workspace, workspace_bytes, need.bytes);
    if (rc) return rc;
    const ScanWs w = scan_layout(workspace, batch->N, batch->T, S, C);
    BandArgs a{};
    a.b = to_dev(batch);
    a.S = S;
    a.px = px;
    a.py = py;
    a.ranges = ranges;
    a.Lutt = w.Lutt;
    a.loss = loss;
    a.gx = px_occ;
    a.gy = py_occ;
    a.C = C;
    a.nchunk = (batch->T + C - 1) / C;
    a.M = w.M;
    a.E = w.E;
    a.V = w.V;
    a.Wb = w.Wb;
    hipError_t e = launch_band_scan(a, static_cast<hipStream_t>(stream));
    return hip_status(e, "rnnt_pruned_loss");
  }
  const int D = band_diagonals(batch->T, batch->U, S);
  const int Wb = band_slots(batch->U, S);
  if ((long long)batch->N * batch->T * S > kI32 || (long long)D * Wb * 8 > kI32 ||
      (long long)batch->N * D * Wb > kI32)
    return fail(RNNT_EUNSUPPORTED, "N*T*S or the band of one utterance is too large");
  const BandWs need = band_layout(nullptr, batch->N, batch->T, batch->U, S);
  rc = check_ws(workspace, workspace_bytes, need.bytes);
  if (rc) return rc;
  const BandWs w = band_layout(workspace, batch->N, batch->T, batch->U, S);
  BandArgs a{};
  a.b = to_dev(batch);
  a.S = S;
  a.D = D;
  a.W = Wb;
  a.masked = band_masked(batch->U, S);
  a.px = px;
  a.py = py;
  a.ranges = ranges;
  a.pxd = w.pxd;
  a.pyd = w.pyd;
  a.meta = w.meta;
  a.alpha = w.alpha;
  a.beta = w.beta;
  a.Lutt = w.Lutt;
  a.loss = loss;
  a.gx = px_occ;
  a.gy = py_occ;
  hipError_t e = launch_band(a, static_cast<hipStream_t>(stream));
  return hip_status(e, "rnnt_pruned_loss");
}

int rnnt_pruned_loss_noalloc(const rnnt_batch* batch, int32_t S, const float* px, const float* py,
                             const int32_t* ranges, float* loss, float* px_occ, float* py_occ, void* stream) {
  // host-side checks first, so that a refused call touches no device
  int rc = check_batch(batch, false);
  if (rc) return rc;
  if (S < 1 || S > RNNT_MAX_S) return fail(RNNT_EUNSUPPORTED, "S = %d outside [1, %d]", S, RNNT_MAX_S);
  if (!px || !py || !ranges || !loss) return fail(RNNT_EINVAL, "px, py, ranges and loss are required");
  const size_t need = pruned_ws_bytes(batch->N, batch->T, batch->U, S, RNNT_BAND_AUTO, 0);
  if (need == 0) return fail(RNNT_EUNSUPPORTED, "sizes outside what the pruned recursion supports");
  if (need > kScratchBytes)
    return fail(RNNT_EUNSUPPORTED,
                "this batch needs %zu bytes of workspace, the static scratch holds %zu: call rnnt_pruned_loss "
                "with a workspace",
                need, kScratchBytes);
  void* ws = nullptr;
  rc = scratch_for(static_cast<hipStream_t>(stream), &ws);
  if (rc) return rc;
  // the kernels write every workspace element they read before reading it,
  // so nothing in the scratch needs clearing between calls
  return rnnt_pruned_loss_ex(batch, S, RNNT_BAND_AUTO, 0, px, py, ranges, loss, px_occ, py_occ, ws, kScratchBytes,
                             stream);
}

size_t rnnt_pruned_joiner_backward_ex_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S, int32_t J,
                                                     int32_t V, int32_t dtype, int32_t chunk_rows) {
  (void)U;
  if (N < 1 || T < 1 || S < 1 || J < 1 || V < 1 || chunk_rows < 0 || chunk_rows % 128 != 0) return 0;
  if (chunk_rows > joiner_bwd_chunk_max_rows(J, V)) return 0;
  return joiner_bwd_layout(nullptr, N, T, S, J, V, dtype == RNNT_BF16, chunk_rows).bytes;
}

size_t rnnt_pruned_joiner_backward_workspace_size(int32_t N, int32_t T, int32_t U, int32_t S, int32_t J, int32_t V,
                                                  int32_t dtype) {
  return rnnt_pruned_joiner_backward_ex_workspace_size(N, T, U, S, J, V, dtype, 0);
}

int32_t rnnt_pruned_joiner_backward_chunk_rows(int32_t N, int32_t T, int32_t S, int32_t J, int32_t V, int32_t dtype,
                                               int32_t chunk_rows) {
  if (N < 1 || T < 1 || S < 1 || J < 1 || V < 1 || chunk_rows < 0 || chunk_rows % 128 != 0) return 0;
  if (chunk_rows > joiner_bwd_chunk_max_rows(J, V) || joiner_bwd_chunk_max_rows(J, V) < 128) return 0;
  return joiner_bwd_chunk_rows(N, T, S, J, V, dtype == RNNT_BF16, chunk_rows);
}

int rnnt_pruned_joiner_backward_ex(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype,
                                   int32_t chunk_rows, const void* enc, const void* dec, const void* W,
                                   const void* bias, const int32_t* ranges, const float* lse, const float* logits,
                                   const float* head, int32_t head_rows, const float* px_occ,
                                   const float* py_occ, const float* scale, float* enc_grad, float* dec_grad,
                                   float* W_grad, float* bias_grad, float* logits_grad, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  rc = check_joiner_sizes(batch, S, J, V, dtype);
  if (rc) return rc;
  rc = check_chunk_request(J, V, chunk_rows);
  if (rc) return rc;
  if (!enc || !dec || !W || !ranges || !lse || !px_occ || !py_occ)
    return fail(RNNT_EINVAL, "enc, dec, W, ranges, lse, px_occ and py_occ are required");
  if (!enc_grad || !dec_grad) return fail(RNNT_EINVAL, "enc_grad and dec_grad are required");
  if (!aligned16(enc_grad) || !aligned16(dec_grad) || !aligned16(logits))
    return fail(RNNT_EINVAL, "enc_grad, dec_grad and logits must be 16-byte aligned");
  if (logits_grad && (long long)batch->N * batch->T * S * (long long)V > (1ll << 40))
    return fail(RNNT_EUNSUPPORTED, "logits_grad is a debugging aid for small shapes");
  const int bf = dtype == RNNT_BF16;
  if (head) {
    if (!aligned16(head)) return fail(RNNT_EINVAL, "head must be 16-byte aligned");
    const int C = joiner_bwd_chunk_rows(batch->N, batch->T, S, J, V, bf, chunk_rows);
    if (head_rows != C)
      return fail(RNNT_EINVAL, "head_rows = %d must equal the backward's chunk of %d rows", head_rows, C);
  }
  rc = check_ws(workspace, workspace_bytes,
                joiner_bwd_layout(nullptr, batch->N, batch->T, S, J, V, bf, chunk_rows).bytes);
  if (rc) return rc;
  const JoinerBwdWs w = joiner_bwd_layout(workspace, batch->N, batch->T, S, J, V, bf, chunk_rows);
  JoinerArgs a = joiner_args(batch, S, J, V, dtype, enc, dec, W, bias, ranges);
  set_joiner_bwd(a, w, lse, logits, px_occ, py_occ, scale, enc_grad, dec_grad, W_grad, bias_grad, logits_grad);
  a.head = logits ? nullptr : const_cast<float*>(head);  // with all logits stored the head is not needed
  a.head_rows = a.head ? head_rows : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_joiner_prep(a, s);
  if (e == hipSuccess) e = launch_joiner_bwd(a, s);
  return hip_status(e, "rnnt_pruned_joiner_backward");
}

int rnnt_pruned_joiner_backward(const rnnt_batch* batch, int32_t S, int32_t J, int32_t V, int32_t dtype,
                                const void* enc, const void* dec, const void* W, const void* bias,
                                const int32_t* ranges, const float* lse, const float* logits,
                                const float* px_occ, const float* py_occ,
                                const float* scale, float* enc_grad, float* dec_grad, float* W_grad, float* bias_grad,
                                float* logits_grad, void* workspace, size_t workspace_bytes, void* stream) {
  return rnnt_pruned_joiner_backward_ex(batch, S, J, V, dtype, 0, enc, dec, W, bias, ranges, lse, logits, nullptr, 0,
                                        px_occ, py_occ, scale, enc_grad, dec_grad, W_grad, bias_grad, logits_grad,
                                        workspace, workspace_bytes, stream);
}

int rnnt_validate_inputs(const rnnt_batch* batch, int32_t V, int32_t S, int32_t J, int32_t dtype, const float* am,
                         const float* lm, const void* enc, const void* dec, int32_t* flags, int32_t* n_bad,
                         void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  if (V < 1) return fail(RNNT_EINVAL, "V must be >= 1 (got %d)", V);
  if (batch->blank < 0 || batch->blank >= V) return fail(RNNT_EINVAL, "blank = %d outside [0, V)", batch->blank);
  if (S < 0 || S > RNNT_MAX_S) return fail(RNNT_EINVAL, "S = %d outside [0, %d]", S, RNNT_MAX_S);
  if ((enc || dec) && J < 1) return fail(RNNT_EINVAL, "J must be >= 1 with enc or dec (got %d)", J);
  if ((enc || dec) && dtype != RNNT_F32 && dtype != RNNT_BF16)
    return fail(RNNT_EINVAL, "dtype must be RNNT_F32 or RNNT_BF16");
  if (!flags) return fail(RNNT_EINVAL, "flags is required");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_validate(to_dev(batch), V, S, J, dtype == RNNT_BF16, am, lm, enc, dec, flags, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_status(e, "rnnt_validate_inputs");
  if (n_bad) {
    std::vector<int32_t> h((size_t)batch->N);
    e = hipMemcpy(h.data(), flags, h.size() * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_status(e, "rnnt_validate_inputs");
    int32_t c = 0;
    for (int32_t f : h) c += f != 0;
    *n_bad = c;
  }
  return ok();
}

int rnnt_combine_losses(int32_t N, const float* simple_loss, const float* pruned_loss, float simple_scale,
                        float pruned_scale, int32_t reduction, float* loss, float* total, void* stream) {
  if (N < 1) return fail(RNNT_EINVAL, "N must be >= 1 (got %d)", N);
  if (reduction != RNNT_REDUCE_SUM && reduction != RNNT_REDUCE_MEAN)
    return fail(RNNT_EINVAL, "reduction must be RNNT_REDUCE_SUM or RNNT_REDUCE_MEAN");
  if (!(simple_scale >= 0.f) || !(pruned_scale >= 0.f))
    return fail(RNNT_EINVAL, "the scales must be >= 0 (got %g, %g)", simple_scale, pruned_scale);
  if (simple_scale != 0.f && !simple_loss) return fail(RNNT_EINVAL, "simple_loss is required with simple_scale != 0");
  if (pruned_scale != 0.f && !pruned_loss) return fail(RNNT_EINVAL, "pruned_loss is required with pruned_scale != 0");
  if (!loss && !total) return fail(RNNT_EINVAL, "at least one of loss and total is required");
  hipError_t e = launch_combine_losses(N, simple_loss, pruned_loss, simple_scale, pruned_scale,
                                       reduction == RNNT_REDUCE_MEAN, loss, total, static_cast<hipStream_t>(stream));
  return hip_status(e, "rnnt_combine_losses");
}

size_t rnnt_full_loss_workspace_size(int32_t N, int32_t T, int32_t U, int32_t J, int32_t V, int32_t dtype) {
  if (N < 1 || T < 1 || U < 0 || J < 1 || V < 1) return 0;
  return full_layout(nullptr, N, T, U, J, V, dtype == RNNT_BF16).bytes;
}

int rnnt_full_loss(const rnnt_batch* batch, int32_t J, int32_t V, int32_t dtype, const void* enc, const void* dec,
                   const void* W, const void* bias, const float* scale, float* loss, float* enc_grad,
                   float* dec_grad, float* W_grad, float* bias_grad, float* logits, void* workspace,
                   size_t workspace_bytes, void* stream) {
  int rc = check_batch(batch, true);
  if (rc) return rc;
  const int S = batch->U + 1;
  if (V < 1) return fail(RNNT_EINVAL, "V must be >= 1 (got %d)", V);
  if (batch->blank < 0 || batch->blank >= V) return fail(RNNT_EINVAL, "blank = %d outside [0, V)", batch->blank);
  if (J < 8 || J % 8 != 0) return fail(RNNT_EUNSUPPORTED, "J = %d must be a positive multiple of 8", J);
  if (dtype != RNNT_F32 && dtype != RNNT_BF16) return fail(RNNT_EINVAL, "dtype must be RNNT_F32 or RNNT_BF16");
  const long long esz = dtype == RNNT_BF16 ? 2 : 4;
  if ((long long)batch->N * batch->T * S > kI32 || (long long)batch->N * batch->T * J * esz > kI32 ||
      (long long)batch->N * S * J * esz > kI32 || (long long)J * joiner_ldl(V) * esz > kI32 ||
      joiner_bwd_chunk_max_rows(J, V) < 128)
    return fail(RNNT_EUNSUPPORTED, "the unpruned joiner is too large for this build");
  if ((size_t)batch->T * sizeof(int) > 64 * 1024) return fail(RNNT_EUNSUPPORTED, "T = %d too large", batch->T);
  if (!enc || !dec || !W || !loss) return fail(RNNT_EINVAL, "enc, dec, W and loss are required");
  if (!enc_grad || !dec_grad) return fail(RNNT_EINVAL, "enc_grad and dec_grad are required");
  if (!aligned16(enc_grad) || !aligned16(dec_grad) || !aligned16(logits))
    return fail(RNNT_EINVAL, "enc_grad, dec_grad and logits must be 16-byte aligned");
  const int bf = dtype == RNNT_BF16;
  const FullWs need = full_layout(nullptr, batch->N, batch->T, batch->U, J, V, bf);
  rc = check_ws(workspace, workspace_bytes, need.bytes);
  if (rc) return rc;
  const FullWs w = full_layout(workspace, batch->N, batch->T, batch->U, J, V, bf);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the joiner on every (t, u): ranges[n,t,s] = s with S = U + 1
  hipError_t e = launch_full_ranges(w.ranges, batch->N, batch->T, S, s);
  JoinerArgs jf = joiner_args(batch, S, J, V, dtype, enc, dec, W, bias, w.ranges);
  set_joiner_fwd(jf, joiner_fwd_layout(w.joiner, batch->N, batch->T, S, J, V, bf), w.px, w.py, w.lse, logits);
  if (e == hipSuccess) e = launch_joiner_prep(jf, s);
  if (e == hipSuccess) e = launch_joiner_fwd(jf, s);
  // the recursion of Eq. (3) on the [T, U+1] lattice and its occupations
  SimpleArgs la{};
  la.b = to_dev(batch);
  la.V = V;
  la.px = w.px;
  la.py = w.py;
  la.pxd = w.pxd;
  la.pyd = w.pyd;
  la.alpha = w.alpha;
  la.beta = w.beta;
  la.Lutt = w.Lutt;
  la.loss = loss;
  la.gx = w.gx;
  la.gy = w.gy;
  la.Wt = nullptr;
  la.ry = w.ry;
  la.rx = w.rx;
  la.cpx = w.cpx;
  la.cpy = w.cpy;
  la.ncolblk = lattice_colblocks(batch->T);
  if (e == hipSuccess) e = launch_lattice_diag_copy(la, s);
  if (e == hipSuccess) e = launch_lattice(la, s);
  // the joiner's backward on every (t, u)
  JoinerArgs jb = joiner_args(batch, S, J, V, dtype, enc, dec, W, bias, w.ranges);
  set_joiner_bwd(jb, joiner_bwd_layout(w.joiner, batch->N, batch->T, S, J, V, bf, full_chunk_rows(J, V, bf), true), w.lse,
                 logits, w.gx, w.gy,
                 scale, enc_grad, dec_grad, W_grad, bias_grad, nullptr);
  if (e == hipSuccess) e = launch_joiner_prep(jb, s);
  if (e == hipSuccess) e = launch_joiner_bwd(jb, s);
  return hip_status(e, "rnnt_full_loss");
}

}  // extern "C"
