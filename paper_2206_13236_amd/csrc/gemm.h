// MFMA GEMM main loop for gfx950, shared by every contraction of the library.
//
// A workgroup of WGM x WGN wave64s (NT threads) computes a BM x BN
// tile of C = A * B with K-steps of BK. Operand tiles are staged through LDS
// in a k-contiguous layout ([row][k], rows padded by 16 bytes) so that every
// lane fetches one 16-byte fragment per 16x16 output block per k-slice:
//   fp32: v_mfma_f32_16x16x4_f32, a fragment holds 4 consecutive k and feeds
//         4 MFMAs (the k order inside a slice is permuted identically for A
//         and B, which leaves the sum unchanged);
//   bf16: v_mfma_f32_16x16x32_bf16, a fragment holds 8 consecutive k.
// Accumulation is fp32 in both cases. Global -> register fetches of the next
// K-step (or the one after, for DEEP configurations) are issued before the
// MFMAs of the current one; LDS is double buffered, so there is one barrier
// per K-step.
//
// Operand sources are supplied by each kernel, in two halves so that global
// loads for the next K-step stay in flight while the current one computes:
//   KC  source (global is k-contiguous):
//     kc_load(row, k, Raw&)            issue the loads only
//     kc_finish(const Raw&, v[KV])     turn them into KV fp32 values
//   MNC source (global is row-contiguous): mnc_load(k, row, Raw&) and
//     mnc_finish(const Raw&, v[16/KV]).
// Generated operands (exp(x - max), widened inputs) are formed in *_finish,
// which runs after the MFMAs of the current K-step; the loader packs them.
// A source whose raw registers already hold the LDS element type declares
// kDirect: its words go to LDS as loaded (KC), or regrouped by byte
// permutes (MNC transpose), with no conversion.
//
// Output element (i, j, r) of a lane: row = wm*WM + i*16 + 4*(lane>>4) + r,
// col = wn*WN + j*16 + (lane & 15).
#pragma once

#include <type_traits>

#include "common.h"

// DEEP_: global fetches run two K-steps ahead (two register sets; for
// configurations whose K-step is too short to cover a load's latency).
template <int BM_, int BN_, int BK_, bool BF16_, int WGM_ = 2, int WGN_ = 2, bool DEEP_ = false>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_;
  static constexpr bool BF16 = BF16_;
  static constexpr bool DEEP = DEEP_;
  using T = typename std::conditional<BF16_, uint16_t, float>::type;
  static constexpr int ESZ = (int)sizeof(T);
  static constexpr int KV = 16 / ESZ;         // k values per 16-byte fragment
  static constexpr int KSLICE = 4 * KV;       // k covered by one fragment across 4 lane groups
  static constexpr int LDK = BK + KV;         // padded LDS row stride (elements)
  static constexpr int WGM = WGM_, WGN = WGN_;       // wave grid
  static constexpr int NT = 64 * WGM * WGN;          // threads per workgroup
  static constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
  static constexpr int FM = WM / 16, FN = WN / 16;
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK;
  static constexpr int STAGE_ELEMS = A_ELEMS + B_ELEMS;
  static constexpr int SMEM_BYTES = 2 * STAGE_ELEMS * ESZ;
  static_assert(BK % KSLICE == 0, "BK must be a multiple of the fragment k-slice");
  static_assert(FM >= 1 && FN >= 1, "tile too small");
};

// Whether a source declares kDirect = true (absent: false).
template <class S, class = void>
struct src_direct : std::false_type {};
template <class S>
struct src_direct<S, std::void_t<decltype(S::kDirect)>> : std::bool_constant<S::kDirect> {};

// Raw operand registers of a source whose values need no transform.
template <int N>
struct RawF {
  float v[N];
};

// Raw registers of an exp(x - m) source: the loaded values and the row max.
template <int N>
struct RawExp {
  float x[N];
  float m;
};

template <class Cfg>
DEV void pack_store16(typename Cfg::T* dst, const float* v) {
  if constexpr (Cfg::BF16) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)f2bf(v[2 * i]) | ((uint32_t)f2bf(v[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

// Operand tile whose global source is k-contiguous.
template <class Cfg, int ROWS, class Src>
struct KCLoader {
  static constexpr int KV = Cfg::KV;
  static constexpr int CPR = Cfg::BK / KV;               // 16-byte chunks per row
  static constexpr int NCH = (ROWS * CPR + Cfg::NT - 1) / Cfg::NT;  // chunks per thread
  struct Reg { typename Src::Raw v[NCH]; };
  const Src& src;
  DEV explicit KCLoader(const Src& s) : src(s) {}
  DEV void fetch(int k0, Reg& r) const {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      int c = threadIdx.x + Cfg::NT * i;
      if (ROWS * CPR % Cfg::NT == 0 || c < ROWS * CPR) src.kc_load(c / CPR, k0 + (c % CPR) * KV, r.v[i]);
    }
  }
  DEV void put(const Reg& r, typename Cfg::T* lds) const {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      int c = threadIdx.x + Cfg::NT * i;
      if (ROWS * CPR % Cfg::NT == 0 || c < ROWS * CPR) {
        typename Cfg::T* dst = lds + (c / CPR) * Cfg::LDK + (c % CPR) * KV;
        if constexpr (src_direct<Src>::value) {
          const uint32_t* w = r.v[i].w;
          *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
          float v[KV];
          src.kc_finish(r.v[i], v);
          pack_store16<Cfg>(dst, v);
        }
      }
    }
  }
};

// Operand tile whose global source is row-contiguous ([k][row]); the loader
// transposes KV x (16/KV) blocks in registers so LDS stays k-contiguous.
// Blocks go to threads from TOFF on (modulo NT): when both operands of a
// contraction have fewer blocks than threads, giving them disjoint threads
// spreads the staging over all waves.
template <class Cfg, int ROWS, class Src, int TOFF = 0>
struct MNCLoader {
  static constexpr int KV = Cfg::KV;
  static constexpr int NV = 16 / KV;                       // rows per block (4 fp32, 2 bf16)
  static constexpr int NBR = ROWS / NV;                    // blocks along rows
  static constexpr int NKB = Cfg::BK / KV;                 // blocks along k
  static constexpr int NBLK = NKB * NBR;
  // Consecutive lanes take consecutive k-blocks of the same rows: a transposed
  // LDS store of NKB lanes then fills one padded row contiguously (fewer bank
  // conflicts than lanes 4 rows apart), and each global load still reads
  // NKB x 16 contiguous bytes per row.
  static constexpr int NPT = (NBLK + Cfg::NT - 1) / Cfg::NT;
  struct Reg { typename Src::Raw v[NPT][KV]; };
  const Src& src;
  DEV explicit MNCLoader(const Src& s) : src(s) {}
  DEV void fetch(int k0, Reg& r) const {
#pragma unroll
    for (int b = 0; b < NPT; ++b) {
      int blk = (threadIdx.x + TOFF) % Cfg::NT + Cfg::NT * b;
      if (NBLK % Cfg::NT == 0 || blk < NBLK) {
        const int kb = blk % NKB, nb = blk / NKB;
#pragma unroll
        for (int i = 0; i < KV; ++i) src.mnc_load(k0 + kb * KV + i, nb * NV, r.v[b][i]);
      }
    }
  }
  DEV void put(const Reg& r, typename Cfg::T* lds) const {
#pragma unroll
    for (int b = 0; b < NPT; ++b) {
      int blk = (threadIdx.x + TOFF) % Cfg::NT + Cfg::NT * b;
      if (NBLK % Cfg::NT == 0 || blk < NBLK) {
        const int kb = blk % NKB, nb = blk / NKB;
        if constexpr (src_direct<Src>::value) {
          // r.v[b][i] holds row elements nb*NV .. nb*NV+NV-1 at k = kb*KV + i
#pragma unroll
          for (int c = 0; c < NV; ++c) {
            uint32_t o[4];
            if constexpr (Cfg::BF16) {
              // two bf16 rows per word: row c's k pair (2q, 2q+1) is the low
              // (c = 0) or high (c = 1) halves of the words of k = 2q, 2q+1
#pragma unroll
              for (int q = 0; q < 4; ++q)
                o[q] = __builtin_amdgcn_perm(r.v[b][2 * q + 1].w[0], r.v[b][2 * q].w[0],
                                             c == 0 ? 0x05040100u : 0x07060302u);
            } else {
#pragma unroll
              for (int q = 0; q < 4; ++q) o[q] = r.v[b][q].w[c];
            }
            *reinterpret_cast<uint4*>(lds + (nb * NV + c) * Cfg::LDK + kb * KV) = make_uint4(o[0], o[1], o[2], o[3]);
          }
        } else {
          float m[KV][NV];
#pragma unroll
          for (int i = 0; i < KV; ++i) src.mnc_finish(r.v[b][i], m[i]);
#pragma unroll
          for (int c = 0; c < NV; ++c) {
            float col[KV];
#pragma unroll
            for (int i = 0; i < KV; ++i) col[i] = m[i][c];
            pack_store16<Cfg>(lds + (nb * NV + c) * Cfg::LDK + kb * KV, col);
          }
        }
      }
    }
  }
};

// MFMAs of the k-slices [K0, K1) of one LDS stage.
template <class Cfg, int K0 = 0, int K1 = Cfg::BK>
DEV void gemm_compute_stage(const typename Cfg::T* As, const typename Cfg::T* Bs,
                            floatx4 (&acc)[Cfg::FM][Cfg::FN]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;
  const typename Cfg::T* a_base = As + (wm * Cfg::WM + (lane & 15)) * Cfg::LDK + (lane >> 4) * Cfg::KV;
  const typename Cfg::T* b_base = Bs + (wn * Cfg::WN + (lane & 15)) * Cfg::LDK + (lane >> 4) * Cfg::KV;
#pragma unroll
  for (int kk = K0; kk < K1; kk += Cfg::KSLICE) {
    if constexpr (Cfg::BF16) {
      bf16x8 fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) fa[i] = *reinterpret_cast<const bf16x8*>(a_base + i * 16 * Cfg::LDK + kk);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) fb[j] = *reinterpret_cast<const bf16x8*>(b_base + j * 16 * Cfg::LDK + kk);
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    } else {
      floatx4 fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) fa[i] = *reinterpret_cast<const floatx4*>(a_base + i * 16 * Cfg::LDK + kk);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) fb[j] = *reinterpret_cast<const floatx4*>(b_base + j * 16 * Cfg::LDK + kk);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int j = 0; j < Cfg::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][s], fb[j][s], acc[i][j], 0, 0, 0);
    }
  }
}

// Runs the K loop over [k_begin, k_end) and leaves the tile in `acc`.
// Must be called by all NT threads of the workgroup (it contains barriers).
template <class Cfg, class LA, class LB>
DEV void gemm_mainloop(const LA& la, const LB& lb, int k_begin, int k_end,
                       typename Cfg::T* smem, floatx4 (&acc)[Cfg::FM][Cfg::FN]) {
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nk = (k_end - k_begin + Cfg::BK - 1) / Cfg::BK;
  if (nk <= 0) return;
  typename Cfg::T* As0 = smem;
  typename Cfg::T* Bs0 = smem + Cfg::A_ELEMS;
  typename Cfg::T* As1 = smem + Cfg::STAGE_ELEMS;
  typename Cfg::T* Bs1 = smem + Cfg::STAGE_ELEMS + Cfg::A_ELEMS;
  constexpr int KH = (Cfg::BK / Cfg::KSLICE) / 2 * Cfg::KSLICE;
  if constexpr (Cfg::DEEP) {
    // Register set p holds the fetch of K-step kt+1 while step kt computes;
    // step kt+2 is fetched into the other set, freed by the previous put.
    typename LA::Reg ra[2];
    typename LB::Reg rb[2];
    la.fetch(k_begin, ra[0]);
    lb.fetch(k_begin, rb[0]);
    if (nk > 1) {
      la.fetch(k_begin + Cfg::BK, ra[1]);
      lb.fetch(k_begin + Cfg::BK, rb[1]);
    }
    la.put(ra[0], As0);
    lb.put(rb[0], Bs0);
    __syncthreads();
    auto step = [&](int kt, auto par) {
      constexpr int P = decltype(par)::value;  // kt & 1
      if (kt + 2 < nk) {
        la.fetch(k_begin + (kt + 2) * Cfg::BK, ra[P]);
        lb.fetch(k_begin + (kt + 2) * Cfg::BK, rb[P]);
      }
      const typename Cfg::T* Ac = P ? As1 : As0;
      const typename Cfg::T* Bc = P ? Bs1 : Bs0;
      gemm_compute_stage<Cfg, 0, KH>(Ac, Bc, acc);
      if (kt + 1 < nk) {
        la.put(ra[1 - P], P ? As0 : As1);
        lb.put(rb[1 - P], P ? Bs0 : Bs1);
      }
      gemm_compute_stage<Cfg, KH, Cfg::BK>(Ac, Bc, acc);
      __syncthreads();
    };
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, std::integral_constant<int, 0>{});
      if (kt + 1 < nk) step(kt + 1, std::integral_constant<int, 1>{});
    }
    return;
  }
  typename LA::Reg ra;
  typename LB::Reg rb;
  la.fetch(k_begin, ra);
  lb.fetch(k_begin, rb);
  la.put(ra, As0);
  lb.put(rb, Bs0);
  __syncthreads();
  // The next stage is staged between the two halves of the current stage's
  // MFMAs: its global loads have the first half to land, and its transforms
  // and LDS stores can issue while the second half's MFMAs execute.
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      la.fetch(k_begin + (kt + 1) * Cfg::BK, ra);
      lb.fetch(k_begin + (kt + 1) * Cfg::BK, rb);
    }
    const bool odd = kt & 1;
    const typename Cfg::T* Ac = odd ? As1 : As0;
    const typename Cfg::T* Bc = odd ? Bs1 : Bs0;
    gemm_compute_stage<Cfg, 0, KH>(Ac, Bc, acc);
    if (more) {
      la.put(ra, odd ? As0 : As1);
      lb.put(rb, odd ? Bs0 : Bs1);
    }
    gemm_compute_stage<Cfg, KH, Cfg::BK>(Ac, Bc, acc);
    __syncthreads();
  }
}

// XCD-aware tile order. Workgroup w of a launch (x fastest, then y, then z)
// is dispatched to XCD w % 8, and every XCD has its own L2. Tile ids are
// renumbered so that each XCD receives one contiguous run of them: tiles
// that are neighbours in tile-id order (and share an operand panel) then run
// on the same XCD at about the same time and share its L2.
// Only the first n_active workgroups get a tile (-1 for the rest), so that a
// grid sized for the padded maximum spreads its real tiles over all XCDs.
constexpr int kNumXcd = 8;
DEV int xcd_tile_id(int n_active) {
  const int w = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int n = min(n_active, (int)(gridDim.x * gridDim.y * gridDim.z));
  if (w >= n) return -1;
  const int per = n / kNumXcd, rem = n % kNumXcd;
  const int x = w % kNumXcd, loc = w / kNumXcd;
  return (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + loc;
}

// Row/column of output element (i, j, r) of this lane within the tile.
template <class Cfg>
DEV int tile_row(int i, int r) {
  const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) / Cfg::WGN;
  return wm * Cfg::WM + i * 16 + 4 * (lane >> 4) + r;
}
template <class Cfg>
DEV int tile_col(int j) {
  const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) % Cfg::WGN;
  return wn * Cfg::WN + j * 16 + (lane & 15);
}

// ---------------------------------------------------------------------------
// Main loop with both operands loaded straight from global memory into LDS
// (buffer_load_dwordx4 ... lds: the 16 bytes of lane i land at the
// instruction's LDS base + 16 i). Nothing is staged through registers, so a
// K-step's loads stay in flight at no register cost while the previous
// K-step computes, and two workgroups share a CU (64 KiB of LDS each at
// 128 x 128 and 128-byte rows, two stages).
//
// Both operands must be k-contiguous in global memory, in 16-byte chunks
// (8 bf16 or 4 fp32) at 16-byte aligned offsets. An LDS row holds BK
// elements unpadded; the chunks of row r are stored XOR-swizzled (chunk c at
// position c ^ (r & 7)), so that the fragment reads of 8 consecutive rows fall
// in distinct banks. MFMAs and accumulator layout are those of GemmCfg
// (tile_row, tile_col).
// ---------------------------------------------------------------------------
template <int BM_, int BN_, int BK_, int WGM_, int WGN_, bool BF16_ = true>
struct LdsCfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_;
  static constexpr bool BF16 = BF16_;
  using T = typename std::conditional<BF16_, uint16_t, float>::type;
  static constexpr int ESZ = (int)sizeof(T);
  static constexpr int KV = 16 / ESZ;          // k values per 16-byte chunk
  static constexpr int WGM = WGM_, WGN = WGN_;
  static constexpr int NW = WGM * WGN, NT = 64 * NW;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 16, FN = WN / 16;
  static constexpr int CH = BK / KV;           // chunks per row
  static constexpr int ROWB = BK * ESZ;        // bytes per LDS row
  static constexpr int RPI = 64 / CH;          // rows filled by one wave-wide load
  static constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
  static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
  static constexpr int SMEM_BYTES = 2 * STAGE_BYTES;
  static constexpr int A_IPW = BM / RPI / NW, B_IPW = BN / RPI / NW;  // loads per wave per stage
  static_assert(CH >= 8 && CH % 4 == 0, "the swizzle needs at least 8 chunks per row");
  static_assert((BM / RPI) % NW == 0 && (BN / RPI) % NW == 0, "whole loads per wave");
  static_assert(FM >= 1 && FN >= 1, "tile too small");
};

// Operand rows [row0, row0 + nvalid) of a k-contiguous array of ESZ-byte
// elements with row stride ld (elements); element (r, k) of the tile is
// array[row0 + r][k - kofs] for k < kend, zero elsewhere (loads past the end
// read through kOob).
template <int ESZ>
struct LdsSrc {
  Rsrc rsrc;
  int row0, nvalid, ld, kofs, kend;
  DEV uint32_t off(int r, int k) const {
    return (r < nvalid && k < kend) ? (uint32_t)((row0 + r) * ld + (k - kofs)) * (uint32_t)ESZ : kOob;
  }
};

typedef __attribute__((address_space(3))) void* LdsPtr;

// One operand tile for K-step k0 into `lds`: wave w issues loads
// w*IPW .. w*IPW+IPW-1, load q filling tile rows [q*RPI, (q+1)*RPI).
template <class Cfg, int IPW>
DEV void lds_fetch(const LdsSrc<Cfg::ESZ>& s, int k0, unsigned char* lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int q = wave * IPW + i;
    const int r = q * Cfg::RPI + lane / Cfg::CH;
    const int c = (lane % Cfg::CH) ^ (r & 7);  // the chunk stored at this lane's position
    __builtin_amdgcn_raw_ptr_buffer_load_lds(s.rsrc, (LdsPtr)(lds + q * 1024), 16, s.off(r, k0 + c * Cfg::KV), 0, 0, 0);
  }
}

template <class Cfg>
DEV void lds_compute_stage(const unsigned char* As, const unsigned char* Bs, floatx4 (&acc)[Cfg::FM][Cfg::FN]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;
  const int lr = lane & 15, lq = lane >> 4;
  // fragment rows are 16-aligned plus lr, so their swizzle key is lr & 7
  const unsigned char* a_row = As + (wm * Cfg::WM + lr) * Cfg::ROWB;
  const unsigned char* b_row = Bs + (wn * Cfg::WN + lr) * Cfg::ROWB;
#pragma unroll
  for (int kc = 0; kc < Cfg::CH; kc += 4) {
    const int pos = ((kc + lq) ^ (lr & 7)) * 16;
    if constexpr (Cfg::BF16) {
      bf16x8 fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) fa[i] = *reinterpret_cast<const bf16x8*>(a_row + i * 16 * Cfg::ROWB + pos);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) fb[j] = *reinterpret_cast<const bf16x8*>(b_row + j * 16 * Cfg::ROWB + pos);
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    } else {
      // a chunk holds 4 consecutive k; MFMA s takes element s of every lane's
      // chunk (the same permutation of k for A and B)
      floatx4 fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
      for (int i = 0; i < Cfg::FM; ++i) fa[i] = *reinterpret_cast<const floatx4*>(a_row + i * 16 * Cfg::ROWB + pos);
#pragma unroll
      for (int j = 0; j < Cfg::FN; ++j) fb[j] = *reinterpret_cast<const floatx4*>(b_row + j * 16 * Cfg::ROWB + pos);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
          for (int j = 0; j < Cfg::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][q], fb[j][q], acc[i][j], 0, 0, 0);
    }
  }
}

// Waits for this wave's outstanding loads, then meets the other waves. An
// explicit s_waitcnt + s_barrier rather than __syncthreads(), whose release
// fence the compiler would also place after the next stage's loads.
DEV void lds_stage_barrier() { asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory"); }

// K loop over [k_begin, k_end) with two LDS stages: at step kt the loads of
// step kt+1 run while step kt computes; one barrier per step. Leaves the
// tile in `acc` and LDS free for the caller (it ends with a barrier). Must be
// called by all NT threads of the workgroup.
template <class Cfg>
DEV void gemm_mainloop_lds(const LdsSrc<Cfg::ESZ>& sa, const LdsSrc<Cfg::ESZ>& sb, int k_begin, int k_end,
                           unsigned char* smem, floatx4 (&acc)[Cfg::FM][Cfg::FN]) {
#pragma unroll
  for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nk = (k_end - k_begin + Cfg::BK - 1) / Cfg::BK;
  if (nk <= 0) return;
  lds_fetch<Cfg, Cfg::A_IPW>(sa, k_begin, smem);
  lds_fetch<Cfg, Cfg::B_IPW>(sb, k_begin, smem + Cfg::A_BYTES);
  for (int kt = 0; kt < nk; ++kt) {
    lds_stage_barrier();  // step kt landed everywhere; step kt-1's slot is free
    if (kt + 1 < nk) {
      unsigned char* st = smem + ((kt + 1) & 1) * Cfg::STAGE_BYTES;
      lds_fetch<Cfg, Cfg::A_IPW>(sa, k_begin + (kt + 1) * Cfg::BK, st);
      lds_fetch<Cfg, Cfg::B_IPW>(sb, k_begin + (kt + 1) * Cfg::BK, st + Cfg::A_BYTES);
    }
    const unsigned char* cs = smem + (kt & 1) * Cfg::STAGE_BYTES;
    lds_compute_stage<Cfg>(cs, cs + Cfg::A_BYTES, acc);
  }
  __syncthreads();
}
