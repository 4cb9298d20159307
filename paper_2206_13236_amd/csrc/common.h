// Device helpers shared by the gfx950 kernels of the pruned RNN-T library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define DEV __device__ __forceinline__

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kNegInfF = -__builtin_inff();
constexpr double kNegInfD = -__builtin_inf();
constexpr double kLog2e = 1.4426950408889634074;
constexpr double kLn2 = 0.69314718055994530942;

// Plain-old-data view of rnnt_batch passed to kernels by value.
struct BatchDev {
  int N, T, U;
  const int* t_len;
  const int* u_len;
  const int* symbols;  // [N, U]
  int blank;
};

// Per-utterance sizes, clamped into range so that every index derived from
// them stays in bounds. Returns false when the caller's lengths were invalid
// (that utterance's loss is then reported as NaN).
DEV bool utt_dims(const BatchDev& b, int n, int& Tn, int& Un) {
  int t = b.t_len[n], u = b.u_len[n];
  bool ok = (t >= 1) && (t <= b.T) && (u >= 0) && (u <= b.U);
  Tn = min(max(t, 1), b.T);
  Un = min(max(u, 0), b.U);
  return ok;
}

// y_{u+1} of utterance n clamped to [0, V); `ok` is cleared when it was not.
DEV int symbol_at(const BatchDev& b, int n, int u, int V, bool& ok) {
  int y = b.symbols[(size_t)n * b.U + u];
  if (y < 0 || y >= V) {
    ok = false;
    y = min(max(y, 0), V - 1);
  }
  return y;
}

// Buffer resources. A buffer access whose byte offset lies at or past the
// resource's size reads zeros (loads) or is dropped (stores), so a lane with
// nothing to load or store passes kOob instead of branching. Offsets are
// 32-bit: every array accessed this way is below 2^31 bytes.
using Rsrc = __amdgpu_buffer_rsrc_t;
constexpr uint32_t kOob = 0x80000000u;

DEV Rsrc make_rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)(uint32_t)bytes, 0x00020000);
}
DEV float buf_load_f32(Rsrc r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
DEV double buf_load_f64(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}
DEV void buf_store_f64(Rsrc r, uint32_t off, double v) {
  typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), r, (int)off, 0, 0);
}

// log2(2^a + 2^b) for log2-domain values held in fp64. The large-magnitude
// additions stay in fp64; only the bounded correction log2(1 + 2^-|a-b|),
// which lies in [0, 1], goes through the fp32 hardware exp2/log2. NaN in either
// argument propagates.
DEV double log2add(double a, double b) {
  double mx = a > b ? a : b;
  double mn = a > b ? b : a;
  if (mn == kNegInfD) return mx;
  float d = (float)(mn - mx);
  float c = __builtin_amdgcn_logf(1.0f + __builtin_amdgcn_exp2f(d));
  return mx + (double)c;
}

// The same sum for recursions that detect NaN inputs on the side: no
// compare-and-select on the dependency chain. v_max/v_min pass over a NaN;
// the difference is clamped to <= 0, which also turns the NaN of
// (-inf) - (-inf) into 0, so that two -inf give -inf + 1 = -inf.
DEV double log2add_nonan(double a, double b) {
  const double mx = __builtin_fmax(a, b), mn = __builtin_fmin(a, b);
  const float d = __builtin_fminf((float)(mn - mx), 0.0f);
  return mx + (double)__builtin_amdgcn_logf(1.0f + __builtin_amdgcn_exp2f(d));
}

// 2^x for an fp64 log2-domain argument that is <= ~0 (an occupation).
DEV float exp2_occ(double x) {
  if (!(x > -200.0)) return (x != x) ? x : 0.0f;  // NaN stays NaN, tiny -> 0
  return exp2f((float)x);
}

// Round-to-nearest-even fp32 -> bf16 bits (NaN kept quiet).
DEV uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
DEV float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// tanh from one hardware exp2 and one reciprocal: tanh(x) = 1 - 2 / (e^{2x} + 1).
// Absolute error ~1e-7 over the whole range; saturates cleanly to +-1.
DEV float fast_tanh(float x) {
  float e = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);  // 2*log2(e)
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(e + 1.0f);
}

// Waits until every vector memory access this wave has issued is complete.
// The compiler's wait tracking sees it, so registers loaded before it need no
// wait of their own at their uses, in whatever branch those are.
DEV void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0), expcnt and lgkmcnt not waited

DEV double shfl_up_d(double v, int delta) { return __shfl_up(v, delta, 64); }
DEV double shfl_down_d(double v, int delta) { return __shfl_down(v, delta, 64); }

// Whole-wave DPP lane moves (GFX9 wave_shr/shl/ror/rol by one lane), for a
// double held in two VGPRs. Lanes without a source keep `old`.
constexpr int kDppWaveShl1 = 0x130;  // lane i <- lane i+1
constexpr int kDppWaveRol1 = 0x134;  // lane i <- lane (i+1) mod 64
constexpr int kDppWaveShr1 = 0x138;  // lane i <- lane i-1
constexpr int kDppWaveRor1 = 0x13C;  // lane i <- lane (i-1) mod 64

template <int CTRL>
DEV double dpp_move_d(double v, double old) {
  const int lo = __builtin_amdgcn_update_dpp(__double2loint(old), __double2loint(v), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(__double2hiint(old), __double2hiint(v), CTRL, 0xf, 0xf, false);
  return __hiloint2double(hi, lo);
}

// Max and sum over the 16 lanes of a DPP row (lanes 16 k .. 16 k + 15, the
// lanes that share an MFMA output row), the result in every lane of the row:
// the row rotated by 8, 4, 2 and 1 lanes (DPP row_ror) and folded in, one
// VALU instruction per step instead of a permute through LDS. Each pairing
// is commutative, so every lane of the row ends with the same bits.
template <int N>
DEV float dpp_row_ror(float v) {
  static_assert(N >= 1 && N <= 15, "row rotation");
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x120 + N, 0xf, 0xf, false));
}
DEV float row16_max(float v) {
  v = fmaxf(v, dpp_row_ror<8>(v));
  v = fmaxf(v, dpp_row_ror<4>(v));
  v = fmaxf(v, dpp_row_ror<2>(v));
  return fmaxf(v, dpp_row_ror<1>(v));
}
DEV float row16_sum(float v) {
  v += dpp_row_ror<8>(v);
  v += dpp_row_ror<4>(v);
  v += dpp_row_ror<2>(v);
  return v + dpp_row_ror<1>(v);
}

// The same for doubles (two VGPRs moved per step).
template <int N>
DEV double dpp_row_ror_d(double v) {
  static_assert(N >= 1 && N <= 15, "row rotation");
  return dpp_move_d<0x120 + N>(v, v);
}
DEV double row16_max_d(double v) {
  double o = dpp_row_ror_d<8>(v);
  v = o > v ? o : v;
  o = dpp_row_ror_d<4>(v);
  v = o > v ? o : v;
  o = dpp_row_ror_d<2>(v);
  v = o > v ? o : v;
  o = dpp_row_ror_d<1>(v);
  return o > v ? o : v;
}
DEV double row16_sum_d(double v) {
  v += dpp_row_ror_d<8>(v);
  v += dpp_row_ror_d<4>(v);
  v += dpp_row_ror_d<2>(v);
  return v + dpp_row_ror_d<1>(v);
}

// Wave-wide max and sum of doubles in a fixed order (deterministic): within
// each 16-lane row by DPP, then across the rows.
DEV double wave_max_d(double v) {
  v = row16_max_d(v);
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    const double o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}
DEV double wave_sum_d(double v) {
  v = row16_sum_d(v);
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) v += __shfl_xor(v, off, 64);
  return v;
}

DEV size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// This wave's instruction-issue priority raised to the highest level, for
// kernels on a step's critical path that share CUs with work on another
// stream. It orders issue between waves only and changes no result.
DEV void raise_wave_priority() { __builtin_amdgcn_s_setprio(3); }
