// Per-utterance kernels around the four stages:
//   * input validation against the problem statement of Sec. 2 (lengths,
//     tokens y_1..y_U in [0, V), finite scores on every node of the
//     utterance) and the band-feasibility condition of the pruned lattice
//     (Sec. 3.2.2: a complete path inside a band of width S exists only if
//     U_n <= (S-1) T_n);
//   * the training loss of Sec. 3.3, a weighted sum of the simple and the
//     pruned losses per utterance, and its sum or mean over the batch in a
//     fixed order.
#include "kernels.h"
#include "prof.h"
#include "rnnt_pruned.h"

namespace {

constexpr int kValThreads = 256;

DEV bool finite_f32(float x) { return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u; }
DEV bool finite_bf16(uint16_t h) { return (h & 0x7f80u) != 0x7f80u; }

// Whether rows [0, rows) of a [*, cols] slab hold a non-finite element; the
// slab's elements are split over `nblk` blocks (this one is `blk`).
DEV bool slab_bad_f32(const float* p, size_t rows, size_t cols, int blk, int nblk) {
  const size_t n = rows * cols;
  bool bad = false;
  for (size_t i = (size_t)blk * kValThreads + threadIdx.x; i < n; i += (size_t)nblk * kValThreads)
    bad |= !finite_f32(p[i]);
  return bad;
}
DEV bool slab_bad_bf16(const uint16_t* p, size_t rows, size_t cols, int blk, int nblk) {
  const size_t n = rows * cols;
  bool bad = false;
  for (size_t i = (size_t)blk * kValThreads + threadIdx.x; i < n; i += (size_t)nblk * kValThreads)
    bad |= !finite_bf16(p[i]);
  return bad;
}

__global__ __launch_bounds__(kValThreads) void validate_clear_kernel(int* flags, int N) {
  const int i = blockIdx.x * kValThreads + threadIdx.x;
  if (i < N) flags[i] = 0;
}

struct ValidateArgs {
  BatchDev b;
  int V, S, J, bf16;
  const float* am;  // [N, T, V] or null
  const float* lm;  // [N, U+1, V] or null
  const void* enc;  // [N, T, J] or null
  const void* dec;  // [N, U+1, J] or null
  int* flags;       // [N]
};

// Grid nblk * N (nblk blocks per utterance). Every block of utterance n
// scans its share of the utterance's nodes (t < T_n, u <= U_n, clamped into
// the padded shape) and ORs what it found into flags[n]; block 0 also checks
// the lengths, the tokens and the band condition.
__global__ __launch_bounds__(kValThreads) void validate_kernel(ValidateArgs a, int nblk) {
  const int n = blockIdx.x / nblk, blk = blockIdx.x - n * nblk;
  int Tn, Un;
  const bool dims_ok = utt_dims(a.b, n, Tn, Un);
  int f = 0;
  if (blk == 0) {
    if (threadIdx.x == 0 && !dims_ok) {
      const int t = a.b.t_len[n], u = a.b.u_len[n];
      if (t < 1 || t > a.b.T) f |= RNNT_FLAG_T_LEN;
      if (u < 0 || u > a.b.U) f |= RNNT_FLAG_U_LEN;
    }
    for (int u = threadIdx.x; u < Un; u += kValThreads) {
      const int y = a.b.symbols[(size_t)n * a.b.U + u];
      if (y < 0 || y >= a.V) f |= RNNT_FLAG_SYMBOL;
    }
    if (threadIdx.x == 0 && a.S > 0 && (long long)Un > (long long)(a.S - 1) * Tn) f |= RNNT_FLAG_NO_BAND;
  }
  const size_t T = a.b.T, U1 = (size_t)a.b.U + 1;
  if (a.am && slab_bad_f32(a.am + (size_t)n * T * a.V, Tn, a.V, blk, nblk)) f |= RNNT_FLAG_AM;
  if (a.lm && slab_bad_f32(a.lm + (size_t)n * U1 * a.V, Un + 1, a.V, blk, nblk)) f |= RNNT_FLAG_LM;
  if (a.bf16) {
    if (a.enc && slab_bad_bf16(reinterpret_cast<const uint16_t*>(a.enc) + (size_t)n * T * a.J, Tn, a.J, blk, nblk))
      f |= RNNT_FLAG_ENC;
    if (a.dec && slab_bad_bf16(reinterpret_cast<const uint16_t*>(a.dec) + (size_t)n * U1 * a.J, Un + 1, a.J, blk,
                               nblk))
      f |= RNNT_FLAG_DEC;
  } else {
    if (a.enc && slab_bad_f32(reinterpret_cast<const float*>(a.enc) + (size_t)n * T * a.J, Tn, a.J, blk, nblk))
      f |= RNNT_FLAG_ENC;
    if (a.dec && slab_bad_f32(reinterpret_cast<const float*>(a.dec) + (size_t)n * U1 * a.J, Un + 1, a.J, blk, nblk))
      f |= RNNT_FLAG_DEC;
  }
  // OR over the block, then one atomic per block with anything to report
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) f |= __shfl_xor(f, o, 64);
  __shared__ int s_f[kValThreads / 64];
  if ((threadIdx.x & 63) == 0) s_f[threadIdx.x >> 6] = f;
  __syncthreads();
  if (threadIdx.x == 0) {
    int g = 0;
    for (int w = 0; w < kValThreads / 64; ++w) g |= s_f[w];
    if (g) atomicOr(a.flags + n, g);
  }
}

// loss[n] = simple_scale * simple[n] + pruned_scale * pruned[n] (a term
// whose scale is 0 contributes 0, whatever its loss, as during the warm-up
// of Sec. 4 when the pruned loss is not evaluated), and its sum or mean in
// fp64: thread i adds n = i, i + 256, ... in order, then a fixed tree.
__global__ __launch_bounds__(kValThreads) void combine_kernel(int N, const float* simple, const float* pruned,
                                                              float ss, float ps, int mean, float* loss,
                                                              float* total) {
  __shared__ double red[kValThreads];
  double acc = 0.0;
  for (int n = threadIdx.x; n < N; n += kValThreads) {
    const float a = (ss != 0.f && simple) ? ss * simple[n] : 0.f;
    const float b = (ps != 0.f && pruned) ? ps * pruned[n] : 0.f;
    const float l = a + b;
    if (loss) loss[n] = l;
    acc += (double)l;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = kValThreads / 2; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0 && total) total[0] = (float)(mean ? red[0] / N : red[0]);
}

}  // namespace

hipError_t launch_validate(const BatchDev& b, int V, int S, int J, int bf16, const float* am, const float* lm,
                           const void* enc, const void* dec, int* flags, hipStream_t s) {
  {
    RNNT_PROF(s, "validate_clear");
    hipLaunchKernelGGL(validate_clear_kernel, dim3((b.N + kValThreads - 1) / kValThreads), dim3(kValThreads), 0, s,
                       flags, b.N);
  }
  ValidateArgs a{b, V, S, J, bf16, am, lm, enc, dec, flags};
  // enough blocks per utterance to spread the largest slab over the chip
  const size_t per_utt = (size_t)(b.T > b.U + 1 ? b.T : b.U + 1) * (size_t)(V > J ? V : J);
  size_t nb = (per_utt + 16 * kValThreads - 1) / (16 * kValThreads);
  const size_t cap = (2048 + b.N - 1) / b.N;
  nb = nb < 1 ? 1 : nb > cap ? cap : nb;
  {
    RNNT_PROF(s, "validate");
    hipLaunchKernelGGL(validate_kernel, dim3((unsigned)(nb * b.N)), dim3(kValThreads), 0, s, a, (int)nb);
  }
  return hipGetLastError();
}

hipError_t launch_combine_losses(int N, const float* simple, const float* pruned, float ss, float ps, int mean,
                                 float* loss, float* total, hipStream_t s) {
  RNNT_PROF(s, "combine_losses");
  hipLaunchKernelGGL(combine_kernel, dim3(1), dim3(kValThreads), 0, s, N, simple, pruned, ss, ps, mean, loss, total);
  return hipGetLastError();
}
