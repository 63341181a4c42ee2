// Window-score passes of K-VEC on gfx950 (paper Sec. 4.1 Eq. eviction, the O'
// variant of Sec. 4.1, and the global importance I of Sec. 4.2).
//
// For one layer, every query row r of the extended window (positions
// T-O'..T-1) attends causally over the keys; the eviction score of key t is
// the window mean of the attention it receives, per KV head (the mean over
// the head's G query heads), and I is the window mean of its max over heads.
//
// The softmax needs each row's normaliser before any probability can be
// summed over rows, so the work is two passes over K:
//   pass 1  per (row, key tile): partial (max, sum of exp) of the logits;
//           a separate task folds the tiles into lse2 = log2 of the
//           normaliser.
//   pass 2  per key tile, all KV heads of one row tile in one work-group:
//           p = exp2(logit*log2e/sqrt(d) - lse2), summed over the tile's rows
//           per head (P and P over O'), and, for the rows of the last-O
//           window, max over heads through LDS then summed over rows (I).
//
// MFMA mapping (v_mfma_f32_16x16x32_bf16, or 16x16x4_f32 for fp32 inputs):
// A = 16 query rows x 32 head-dim elements, B = 32 elements x 16 keys.  Lane
// l supplies row/key (l % 16); with c = l / 16, its 16-byte piece c of each
// 64-byte span of the row feeds one k-step (for fp32 the four floats of a
// piece go to four k-steps, a permutation of the reduction index, which the
// dot product allows).  The output lane l holds rows 4c..4c+3 of the block
// for key (l % 16).
//
// Keys reach the MFMA through LDS: in that layout the lanes of one load
// would touch 16 different rows, which the vector memory pipeline serves one
// lane at a time.  Instead each wave copies its next 16 keys with direct
// global-to-LDS loads in which consecutive lanes read consecutive 16-byte
// pieces (whole rows, fully coalesced), into a private ring of LDS slots,
// and reads its fragments back with ds_read_b128.  Piece q of key n is
// stored at position q ^ (n mod 16), so the 16 keys a fragment read touches
// fall in distinct LDS banks.  A wave owns one KV head and
// NB = G*RB blocks: rows ordered (g, window row), so the G query heads of one
// window row land in the same lane and their mean is a register sum.
// Work-groups are 8 waves: 8/H row tiles of H heads each.
#pragma once

#include <math.h>

#include "kvec_internal.h"

namespace kvec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct BF16 {};
struct F32 {};

template <class TT, int D>
struct Frag;

template <int D>
struct Frag<BF16, D> {
  static constexpr int KS = D / 32;
  bf16x8 v[KS];
  __device__ __forceinline__ void load(const void* row, int c) {
    const uint4* p = static_cast<const uint4*>(row);
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = __builtin_bit_cast(bf16x8, p[4 * j + c]);
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  }
  // key n of a swizzled LDS slot (rows of D*2 bytes, 16-byte pieces)
  __device__ __forceinline__ void load_lds(const uint4* slot, int n, int c, int swz) {
    const uint4* row = slot + n * (D / 8);
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = __builtin_bit_cast(bf16x8, row[(4 * j + c) ^ (n & swz)]);
  }
};

template <int D>
struct Frag<F32, D> {
  static constexpr int KS = D / 4;
  float v[KS];
  __device__ __forceinline__ void load(const void* row, int c) {
    const uint4* p = static_cast<const uint4*>(row);
#pragma unroll
    for (int j = 0; j < KS / 4; ++j) {
      const uint4 u = p[4 * j + c];
      v[4 * j + 0] = __uint_as_float(u.x);
      v[4 * j + 1] = __uint_as_float(u.y);
      v[4 * j + 2] = __uint_as_float(u.z);
      v[4 * j + 3] = __uint_as_float(u.w);
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = 0.f;
  }
  // key n of a swizzled LDS slot (rows of D*4 bytes, 16-byte pieces)
  __device__ __forceinline__ void load_lds(const uint4* slot, int n, int c, int swz) {
    const uint4* row = slot + n * (D / 4);
#pragma unroll
    for (int j = 0; j < KS / 4; ++j) {
      const uint4 u = row[(4 * j + c) ^ (n & swz)];
      v[4 * j + 0] = __uint_as_float(u.x);
      v[4 * j + 1] = __uint_as_float(u.y);
      v[4 * j + 2] = __uint_as_float(u.z);
      v[4 * j + 3] = __uint_as_float(u.w);
    }
  }
};

template <int D>
__device__ __forceinline__ f32x4 mma(const Frag<BF16, D>& a, const Frag<BF16, D>& b, f32x4 acc) {
#pragma unroll
  for (int j = 0; j < Frag<BF16, D>::KS; ++j)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v[j], b.v[j], acc, 0, 0, 0);
  return acc;
}

template <int D>
__device__ __forceinline__ f32x4 mma(const Frag<F32, D>& a, const Frag<F32, D>& b, f32x4 acc) {
#pragma unroll
  for (int j = 0; j < Frag<F32, D>::KS; ++j)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
  return acc;
}

// One k-step (32 bf16 or 4 fp32 elements of the head dimension) of a block.
template <int D>
__device__ __forceinline__ f32x4 mma1(const Frag<BF16, D>& a, const Frag<BF16, D>& b, f32x4 acc, int j) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v[j], b.v[j], acc, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ f32x4 mma1(const Frag<F32, D>& a, const Frag<F32, D>& b, f32x4 acc, int j) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
}

template <class TT>
constexpr int elem_bytes() { return __is_same(TT, BF16) ? 2 : 4; }

// Cross-lane reductions on DPP and the gfx950 lane-swap instructions (VALU
// only, no LDS round trip).  A DPP row is 16 lanes: the lanes of one MFMA
// output column group.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppSwap1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppSwap2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppRor8 = 0x128;        // row_ror:8 (lane n <-> n ^ 8 within a row)
constexpr int kDppMirror = 0x140;      // row_mirror

// Transpose-reduce over the 16 lanes of each DPP row: v<k> holds a lane's
// term of quantity k (k < 16); afterwards lane n of the row returns the row
// total of quantity n.  Four exchange rounds pair lanes 8 apart, mirrored
// within 8, 2 apart and 1 apart; in each, a lane keeps the half of its
// quantities that its side of the pair owns and adds the partner's terms of
// that half (15 lane moves for 16 sums instead of 64).  Written on scalars:
// the selects must stay selects of values, not of array elements.
template <int CTRL>
__device__ __forceinline__ float xchg_keep(bool up, float lo, float hi) {
  return (up ? hi : lo) + dpp_f<CTRL>(up ? lo : hi);
}
__device__ __forceinline__ float row_transpose_sum16(
    int n, float v0, float v1, float v2, float v3, float v4, float v5, float v6, float v7,
    float v8, float v9, float v10, float v11, float v12, float v13, float v14, float v15) {
  const bool u8 = (n & 8) != 0, u4 = (n & 4) != 0, u2 = (n & 2) != 0, u1 = (n & 1) != 0;
  const float a0 = xchg_keep<kDppRor8>(u8, v0, v8), a1 = xchg_keep<kDppRor8>(u8, v1, v9);
  const float a2 = xchg_keep<kDppRor8>(u8, v2, v10), a3 = xchg_keep<kDppRor8>(u8, v3, v11);
  const float a4 = xchg_keep<kDppRor8>(u8, v4, v12), a5 = xchg_keep<kDppRor8>(u8, v5, v13);
  const float a6 = xchg_keep<kDppRor8>(u8, v6, v14), a7 = xchg_keep<kDppRor8>(u8, v7, v15);
  const float b0 = xchg_keep<kDppHalfMirror>(u4, a0, a4), b1 = xchg_keep<kDppHalfMirror>(u4, a1, a5);
  const float b2 = xchg_keep<kDppHalfMirror>(u4, a2, a6), b3 = xchg_keep<kDppHalfMirror>(u4, a3, a7);
  const float c0 = xchg_keep<kDppSwap2>(u2, b0, b2), c1 = xchg_keep<kDppSwap2>(u2, b1, b3);
  return xchg_keep<kDppSwap1>(u1, c0, c1);
}

__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp_f<kDppSwap1>(v));
  v = fmaxf(v, dpp_f<kDppSwap2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return v;
}
// v_permlane32_swap / v_permlane16_swap exchange the upper half-wave (odd
// rows) of a with the lower half-wave (even rows) of b.  Written out: the
// compiler's builtin returns the first register for both results.  The s_nop
// covers the wait states after the VALU writes of a and b.
__device__ __forceinline__ void lane_swap32(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void lane_swap16(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
// Sum of lanes l, l^16, l^32, l^48 (the four rows of a column), in every lane.
__device__ __forceinline__ float col_sum4(float v) {
  float a = v, b = v;
  lane_swap32(a, b);  // a = v[l mod 32], b = v[l mod 32 + 32]
  v = a + b;
  a = v;
  b = v;
  lane_swap16(a, b);  // a = even row of the pair, b = odd row
  return a + b;
}
__device__ __forceinline__ float col_max4(float v) {
  float a = v, b = v;
  lane_swap32(a, b);
  v = fmaxf(a, b);
  a = v;
  b = v;
  lane_swap16(a, b);
  return fmaxf(a, b);
}

// LDS atomic max without return.  Written out: for the builtin the compiler
// first drains every direct-to-LDS load in flight (it cannot tell the
// addresses apart), which would stall the key ring at every step.
__device__ __forceinline__ void lds_max_u32(unsigned* p, unsigned v) {
  const auto* lp = (__attribute__((address_space(3))) unsigned*)p;
  asm volatile("ds_max_u32 %0, %1" ::"v"(lp), "v"(v) : "memory");
}

// Wait until at most N vector memory operations of this wave are pending.
// Direct global-to-LDS loads are not tracked by the compiler's own waits, so
// the key ring waits explicitly; the asm statement also keeps LDS reads from
// being scheduled above it.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier that orders LDS only: this wave's LDS operations have
// completed (lgkmcnt) before it arrives.  Written out because the compiler's
// release fence would also drain the key ring's direct-to-LDS loads, which
// must stay in flight across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Combine two (max, sum of 2^(x - max)) pairs.
__device__ __forceinline__ void lse_merge(float& m, float& l, float m2, float l2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) {
    m = mm;
    l = 0.f;
    return;
  }
  l = l * __builtin_amdgcn_exp2f(m - mm) + l2 * __builtin_amdgcn_exp2f(m2 - mm);
  m = mm;
}

// Pointers of one layer for the score passes.
struct ScoreIO {
  const char* q;      // layer's q window, element strides qs_*
  const char* k;      // layer's keys
  int64_t qs_b, qs_h, qs_r;
  int64_t ks_b, ks_h, ks_t;
  float2* lse_part;   // [b][HQ][Wn][n_kt1]
  float* lse2;        // [b][HQ][Wn]
  const float* lse_in;  // nullable: caller's natural-log normalisers, rows contiguous
  int64_t lse_b, lse_h;
  float* psum_base;   // [b][n_rt][H][Tc]
  float* psum_all;    // [b][n_rt][H][Tc]
  float* ipart;       // [b][n_rt][Tc]
};

// Word 3 of a raw buffer resource on the gfx9 family (32-bit data format,
// no swizzle); loads outside num_records return zero.
constexpr int kBufferWord3 = 0x00020000;
// A vector offset past every buffer of the score passes (num_records < 2^31).
constexpr int kOutOfRange = (int)0x80000000u;

// Per-wave LDS ring of key steps (16 keys per step).
template <class TT, int D>
struct KeyRing {
  static constexpr int ES = elem_bytes<TT>();
  static constexpr int CPR = D * ES / 16;                // 16-byte pieces per key row
  static constexpr int SWZ = (CPR < 16 ? CPR : 16) - 1;  // piece swizzle mask
  static constexpr int SLOT = 16 * CPR * 16;             // bytes per step
  static constexpr int NI = CPR / 4;                     // 1 KiB loads per step
  static constexpr int KPI = 64 / CPR;                   // keys per load
  static constexpr int R = key_ring_slots(ES, D);        // slots (steps in flight)
  static_assert((size_t)(kThreads / 64) * R * SLOT == key_ring_bytes(ES, D), "ring size");
};

// One pass over one key tile for the row tiles of this work-group.
// Block: 512 threads; wave w -> head w % H, row tile rtg*(8/H) + w / H.
// The state lives in a struct whose methods are all force-inlined, so every
// array is indexed by compile-time constants and stays in registers.
//
// Pass 1 accumulates sum 2^(x - M) per row, with one reference M per 16-row
// block, uniform across the wave: the largest logit of the block's rows at
// the tile's first 16 keys.  A row whose logits later exceed M by more than
// the fp32 exponent range (sum overflows) or stay far below it (sum < 2^-64,
// so low bits could be lost) is flagged with an infinite sum and the row
// normaliser recomputes that (row, tile) partial exactly.

template <class TT, int D, int G, int PASS>
struct ScoreTile {
  using Tl = Tiling<G>;
  static constexpr int RB = Tl::RB, NB = Tl::NB, WR = Tl::WR;
  static constexpr int NBP = (NB + 3) & ~3;  // blocks padded to groups of four (pass-1 store)
  static constexpr int ES = elem_bytes<TT>();

  const Problem& P;
  const ScoreIO& io;
  int b, kt, rtg;
  int lane, c, n, tpw, h, hs, nh, slot, rt;
  bool active, idle, exch;
  int r_lo, base_lo, tend, ks, ke, lim_min, nsteps, rr0;
  const char* kbase;
  bool tile_base, tile_mixed, wg_base;
  float *mbuf, *obuf, *ibuf;

  using KR = KeyRing<TT, D>;
  Frag<TT, D> qf[NB];
  // key fragments of the current and the next step; with seven or eight row
  // blocks one register set (the next step's read waits for this step's
  // products to be issued), which keeps the queries and sums in registers
  static constexpr int NKF = NB >= 7 ? 1 : 2;
  Frag<TT, D> kf[NKF];
  uint4* ring;                    // this wave's LDS slots
  __amdgpu_buffer_rsrc_t krsrc;   // keys [0, tend) of (b, h)
  int kstride;                    // bytes between consecutive keys
  int voff[KR::NI];               // byte offset of this lane's piece in each load
  f32x4 acc[NB];
  float mref[NBP];  // pass 1: wave-uniform reference of each block
  float lsum[NBP][4], nlse[NB][4];
  int pos[RB][4];

  // part: which row tiles and heads.  ALL and BASE: wave w takes head
  // w % H of row tile rtg * (8 / H) + w / H (with H not dividing 8 the last
  // waves are idle).  EXT: every wave has a task of its own, given by the
  // caller (b, kt and rtg may differ between the waves): hmask holds its one
  // head (0: no task) and rtg its extended-window row tile.
  __device__ __forceinline__ ScoreTile(const Problem& P_, const ScoreIO& io_, int b_, int kt_,
                                       int rtg_, float* smem, Part part, uint32_t hmask)
      : P(P_), io(io_), b(b_), kt(kt_), rtg(rtg_) {
    // wave-uniform by construction; readfirstlane lets the compiler keep the
    // wave's head, tile and buffer resource in scalar registers
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    lane = threadIdx.x & 63;
    c = lane >> 4;
    n = lane & 15;
    const bool ext = part == PART_EXT;
    nh = ext ? 1 : P.H;
    tpw = 8 / nh;
    hs = w % nh;
    slot = w / nh;
    idle = ext ? hmask == 0u : slot >= tpw;
    h = ext ? (hmask ? (int)__builtin_ctz(hmask) : 0) : hs;
    const int rt0 = ext ? P.n_rt_base : 0;
    const int rt_end = part == PART_BASE ? P.n_rt_base : P.n_rt;
    rt = ext ? rt0 + rtg : rt0 + rtg * tpw + slot;
    active = !idle && rt < rt_end;
    r_lo = P.Wn - (rt + 1) * WR;  // lowest window row of this tile (may be < 0)
    base_lo = P.Wn - P.O;         // first row of the last-O window

#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) pos[rb][i] = P.T - P.Wn + (r_lo + rb * 16 + 4 * c + i);

    tend = PASS == 1 ? P.T : P.Tc;
    const int tile = PASS == 1 ? P.tile1 : P.tile2;
    ks = kt * tile;
    ke = min(ks + tile, tend);
    lim_min = P.T - P.Wn + max(r_lo, 0);
    kbase = io.k + ((int64_t)b * io.ks_b + (int64_t)h * io.ks_h) * ES;
    kstride = (int)(io.ks_t * ES);  // the host checks tend * kstride < 2^31
    krsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kbase), 0, tend * kstride, kBufferWord3);
#pragma unroll
    for (int i = 0; i < KR::NI; ++i) {
      const int kin = i * KR::KPI + lane / KR::CPR;             // key within the step
      const int piece = (lane % KR::CPR) ^ (kin & KR::SWZ);     // stored at lane % CPR
      voff[i] = kin * kstride + piece * 16;
    }
    ring = reinterpret_cast<uint4*>(smem) + w * (KR::R * KR::SLOT / 16);
    // Steps are padded to an even count (the loop alternates two fragment
    // registers) and, in pass 2, to the importance exchange; keys at or past
    // ke read as zero and are masked (pass 1) or never stored (pass 2).
    nsteps = (ke - ks + 15) / 16;
    const int pad = PASS == 2 ? max(2, P.SK / 16) : 2;
    nsteps = (nsteps + pad - 1) / pad * pad;

    tile_base = tile_mixed = wg_base = false;
    if constexpr (PASS == 1) {
#pragma unroll
      for (int bk = 0; bk < NBP; ++bk) {
#pragma unroll
        for (int i = 0; i < 4; ++i) lsum[bk][i] = 0.f;
        if (bk >= NB) mref[bk] = 0.f;  // padding blocks are never stored
      }
    } else {
      tile_base = active && r_lo + WR > base_lo;
      tile_mixed = tile_base && r_lo < base_lo;
      // A work-group exchanges importance rows when any of its tiles holds base
      // rows; the first tile of the group is the newest, so checking it
      // suffices.  EXT tiles hold no base rows.
      wg_base = part != PART_EXT && (P.Wn - (rt0 + rtg * tpw + 1) * WR) + WR > base_lo;
    }
    exch = PASS == 2 && wg_base && nh > 1;
    rr0 = max(0, base_lo - r_lo);
    // pass-2 LDS per tile slot (after the key rings): two buffers of the
    // running max over heads [WR][SK + 4] (passes that can exchange), the
    // staged per-key sums of each head, and the staged importance of the tile
    const bool layout_x = part != PART_EXT && P.H > 1;
    mbuf = smem + key_ring_bytes(ES, D) / 4 + slot * p2_slot_floats(nh, WR, P.SK, P.tile2, layout_x, P.nsum);
    obuf = mbuf + (layout_x ? exchange_buffers(P.SK, P.tile2) * WR * (P.SK + 4) : 0);
    ibuf = obuf + P.nsum * nh * P.tile2;
  }

  // Query fragments.  Padding rows (r < 0) load row 0 and inactive waves
  // load their clamped rows: neither is ever stored, pass 1 leaves padding
  // rows out of the block references and pass 2 gives them a zero weight.
  __device__ __forceinline__ void load_queries() {
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      const int g = bk / RB, rb = bk % RB;
      const int r = r_lo + rb * 16 + n;
      const int j = h * G + g;
      qf[bk].load(io.q + ((int64_t)b * io.qs_b + (int64_t)j * io.qs_h + (int64_t)max(r, 0) * io.qs_r) * ES,
                  c);
    }
  }

  // Copy the 16 keys of step st into ring slot u (lane l writes 16 bytes at
  // l * 16 of each 1 KiB load; its global piece is pre-swizzled in voff).
  // A step whose keys all lie in [ks, ke) passes the step offset in the
  // scalar offset.  Any other step (the tile's ragged end, padding steps and
  // the copies issued ahead past the last step) moves the whole offset into
  // the vector offset, which the buffer range check covers, and points keys
  // outside the tile past the end of the buffer: those read as zero without
  // touching memory, and the number of copies in flight stays the same.
  // Pass 2's copies carry the non-temporal hint (cache-policy bit nt): in the
  // layer pipeline they are the last reads of most of a layer's keys, and
  // streaming them past the caches leaves more of what pass 1 read for the
  // later stages of the pipeline (about 1.5% off the 32k step; pass 1 with
  // the hint is 7% slower).
  static constexpr int kCopyAux = PASS == 2 ? 2 : 0;
  __device__ __forceinline__ void dma(int u, int st) {
    auto* dst = (__attribute__((address_space(3))) char*)(reinterpret_cast<char*>(ring) + u * KR::SLOT);
    const int k0 = ks + 16 * st;
    if (k0 + 16 <= ke) {
      const int soff = k0 * kstride;
#pragma unroll
      for (int i = 0; i < KR::NI; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(krsrc, dst + i * 1024, 16, voff[i], soff, 0, kCopyAux);
    } else {
#pragma unroll
      for (int i = 0; i < KR::NI; ++i) {
        const int kk = k0 + i * KR::KPI + lane / KR::CPR;
        const int off = kk < ke ? voff[i] + k0 * kstride : kOutOfRange;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(krsrc, dst + i * 1024, 16, off, 0, 0, kCopyAux);
      }
    }
  }

  template <int F>
  __device__ __forceinline__ void read_frag(int u) {
    kf[F % NKF].load_lds(ring + u * (KR::SLOT / 16), n, c, KR::SWZ);
  }

  template <int F>
  __device__ __forceinline__ void mma_frag() {
    // k-step-major: consecutive MFMAs write different blocks, so each block's
    // accumulation chain has NB - 1 independent products between its links
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) acc[bk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < Frag<TT, D>::KS; ++j)
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) acc[bk] = mma1<D>(qf[bk], kf[F % NKF], acc[bk], j);
  }

  // Pass-2 epilogue shapes, fixed per wave before the key loop.  EP_GEN
  // decides per step from the tile's flags (any geometry).  With one per-key
  // sum per head (no row tile mixes last-O and earlier rows): EP_SUM for a
  // tile without last-O rows (the sums only), EP_IMP for a tile of last-O rows
  // only (the sums and the max over heads, no row masked out).
  enum { EP_GEN = 0, EP_SUM = 1, EP_IMP = 2 };

  // Running max over the heads of this slot: p >= 0, so the float order is
  // the order of the bit patterns (ds_max_u32).  Rows before rr0 (not in the
  // last-O window) fold in a zero when ROW_MASK.
  template <bool ROW_MASK>
  __device__ __forceinline__ void fold_max(int s, const float (&gs)[RB][4]) {
    const int kk = ((s * 16) & (P.SK - 1)) + n;
    const int buf = exchange_buffers(P.SK, P.tile2) == 2 ? (((s * 16) >> P.sk_shift) & 1) : 0;
    unsigned* mb = reinterpret_cast<unsigned*>(mbuf) + buf * WR * (P.SK + 4);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rr = rb * 16 + 4 * c + i;
        lds_max_u32(mb + rr * (P.SK + 4) + kk,
                    !ROW_MASK || rr >= rr0 ? __float_as_uint(gs[rb][i]) : 0u);
      }
  }

  template <bool MASKED, int EP>
  __device__ __forceinline__ void epilogue(int s) {
    const int t = ks + 16 * s + n;
    if constexpr (PASS == 1) {
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int rb = bk % RB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = fmaf(acc[bk][i], P.sc, -mref[bk]);
          if constexpr (MASKED) x = (t <= pos[rb][i] && t < ke) ? x : -INFINITY;
          lsum[bk][i] += __builtin_amdgcn_exp2f(x);
        }
      }
    } else {
      // gs: sum over the G query heads of each row (p >= 0, so starting from
      // the first term instead of 0 changes no bit)
      float gs[RB][4];
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int rb = bk % RB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float p = __builtin_amdgcn_exp2f(fmaf(acc[bk][i], P.sc, nlse[bk][i]));
          if constexpr (MASKED) p = t <= pos[rb][i] ? p : 0.f;
          gs[rb][i] = bk < RB ? p : gs[rb][i] + p;
        }
      }
      float s_all = gs[0][0];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = rb == 0 ? 1 : 0; i < 4; ++i) s_all += gs[rb][i];
      if constexpr (EP != EP_GEN) {
        s_all = col_sum4(s_all);
        if (c == 0) obuf[hs * P.tile2 + s * 16 + n] = s_all;
        if constexpr (EP == EP_IMP) {
          if (nh == 1) {
            if (c == 0) ibuf[s * 16 + n] = s_all;
          } else {
            fold_max<false>(s, gs);
          }
        }
        return;
      }
      float s_base = 0.f;
      if (tile_mixed) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            s_base += (r_lo + rb * 16 + 4 * c + i >= base_lo) ? gs[rb][i] : 0.f;
      }
      if (tile_base && !tile_mixed) s_base = s_all;
      s_all = col_sum4(s_all);
      s_base = col_sum4(s_base);
      // Stage the per-key sums in LDS; they are written out after the loop so
      // that the loop issues no global stores (exact load counting).
      if (c == 0) {
        // with one sum per head (no mixed tiles) the last-O sum of a base
        // tile equals its all-row sum and is never read for other tiles
        obuf[(hs * P.nsum) * P.tile2 + s * 16 + n] = s_all;
        if (P.nsum == 2) obuf[(hs * 2 + 1) * P.tile2 + s * 16 + n] = s_base;
      }
      if (tile_base) {
        if (nh == 1) {
          // one head: the max over heads is the head itself
          if (c == 0) ibuf[s * 16 + n] = s_base;
        } else {
          fold_max<true>(s, gs);
        }
      }
    }
  }

  // End of an exchange period of SK keys (step s is its last): once every
  // head of the slot has folded its rows in, the slot's waves share the keys
  // of the period: lane (kc, rg) of a wave sums rows rg, rg + 4, ... of key
  // kc, the four row groups are added across lanes, and the buffer is
  // cleared for its reuse two periods later (after the next barrier).
  __device__ __forceinline__ void exchange(int s) {
    lds_barrier();
    if (!tile_base) return;
    const int period = (s * 16) >> P.sk_shift;
    float* mb = mbuf + (exchange_buffers(P.SK, P.tile2) == 2 ? (period & 1) : 0) * WR * (P.SK + 4);
    const int kpw = (P.SK + nh - 1) / nh;
    const int kb0 = hs * kpw, kb1 = min(P.SK, kb0 + kpw);
    const int rg = lane >> 4;
    for (int k0 = kb0; k0 < kb1; k0 += 16) {
      const int kc = k0 + (lane & 15);
      const bool ok = kc < kb1;
      float v = 0.f;
      if (ok) {
#pragma unroll
        for (int rr = rg; rr < WR; rr += 4) {
          v += mb[rr * (P.SK + 4) + kc];
          mb[rr * (P.SK + 4) + kc] = 0.f;
        }
      }
      v = col_sum4(v);
      if (ok && rg == 0) ibuf[period * P.SK + kc] = v;
    }
  }

  // Key steps in flight ahead of the one being read: step s + kAhead is
  // issued at step s into slot (s + kAhead) mod R, whose previous step was
  // read at step s + kAhead - R - 1 < s.
  static constexpr int kAhead = KR::R > 1 ? KR::R - 1 : 1;

  // One step: the products of step s (fragment F, read during step s - 1),
  // then the copy of step s + kAhead, the read of step s + 1's fragment once
  // its copy has landed, and the exponentials of step s while that read is in
  // flight.  u is the slot of step s + 1.
  template <int F, bool TILE_MASKED, int EP>
  __device__ __forceinline__ void step(int s, int u) {
    mma_frag<F>();
    const int ua = KR::R > 1 ? (u + kAhead - 1) % KR::R : 0;
    dma(ua, s + kAhead);
    wait_vmem<(kAhead - 1) * KR::NI>();
    read_frag<F ^ 1>(u);
    __builtin_amdgcn_sched_barrier(0);  // issue the reads before the exponentials
    if constexpr (TILE_MASKED) {
      const int t0 = ks + 16 * s;
      if (t0 + 15 > lim_min || (PASS == 1 && t0 + 16 > ke))
        epilogue<true, EP>(s);
      else
        epilogue<false, EP>(s);
    } else {
      epilogue<false, EP>(s);
    }
    if constexpr (PASS == 2) {
      if (exch && (((s + 1) * 16) & (P.SK - 1)) == 0) exchange(s);
    }
    if constexpr (NB >= 7) {
      // The next step's products read this fragment only after this step's
      // exponentials: with seven or eight blocks two sets of products would
      // not fit in registers next to the queries.
#pragma unroll
      for (int j = 0; j < Frag<TT, D>::KS; ++j) asm volatile("" : "+v"(kf[(F ^ 1) % NKF].v[j]));
    }
    // Keep the steps in program order (the next step's waits stay after
    // this step's work).
    __builtin_amdgcn_sched_barrier(0);
  }

  template <bool TILE_MASKED, int EP>
  __device__ __forceinline__ void run() {
    int u = KR::R > 1 ? 1 : 0;  // slot of step s + 1
    for (int s = 0; s < nsteps; s += 2) {
      step<0, TILE_MASKED, EP>(s, u);
      u = u + 1 == KR::R ? 0 : u + 1;
      step<1, TILE_MASKED, EP>(s + 1, u);
      u = u + 1 == KR::R ? 0 : u + 1;
    }
  }

  template <int EP>
  __device__ __forceinline__ void run_ep(bool masked) {
    if (masked)
      run<true, EP>();
    else
      run<false, EP>();
  }

  // Pass 2: log2 of each row's normaliser, from pass 1 or the caller's
  // natural log times log2(e) (pass 2 works with base-2 exponentials).
  __device__ __forceinline__ void load_normalisers(float (&v)[NB][4]) {
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      const int g = bk / RB, rb = bk % RB;
      const int j = h * G + g;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = max(r_lo + rb * 16 + 4 * c + i, 0);
        v[bk][i] = io.lse_in ? io.lse_in[(int64_t)b * io.lse_b + (int64_t)j * io.lse_h + r] *
                                   1.4426950408889634f
                             : io.lse2[((int64_t)b * P.HQ + j) * P.Wn + r];
      }
    }
  }

  __device__ __forceinline__ void execute() {
    if (idle) {
      // no tile: only meet the work-group barrier of the write-out
      if constexpr (PASS == 2) lds_barrier();
      return;
    }
    // Steps 0..kAhead-1 are in flight before the loop, the queries loaded
    // right after step 0's keys (both long-latency), then pass 2's row
    // normalisers, so that the three share one memory round trip; step 0's
    // fragment is read as soon as all have landed.
    dma(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    load_queries();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 1; st < kAhead; ++st) dma(st % KR::R, st);
    if constexpr (PASS == 2) {
      float v[NB][4];
      load_normalisers(v);
      // clear the running-max buffers before any head folds rows in
      if (exch) {
        const int nf = exchange_buffers(P.SK, P.tile2) * WR * (P.SK + 4);
        for (int i = lane + hs * 64; i < nf; i += 64 * nh) mbuf[i] = 0.f;
        lds_barrier();
      }
#pragma unroll
      for (int bk = 0; bk < NB; ++bk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          nlse[bk][i] = active && r_lo + (bk % RB) * 16 + 4 * c + i >= 0 ? -v[bk][i] : -INFINITY;
    }
    wait_vmem<(kAhead - 1) * KR::NI>();
    read_frag<0>(0);
    if constexpr (PASS == 1) {
      // Block references from the first 16 keys (recomputed by step 0).  A
      // row with any valid key in this tile sees the tile's first key, so a
      // block is -inf only when none of its rows has a valid key here.
      mma_frag<0>();
      const int t = ks + n;
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool real = r_lo + (bk % RB) * 16 + 4 * c + i >= 0;  // not a padding row
          const bool valid = real && t <= pos[bk % RB][i] && t < ke;
          m = fmaxf(m, valid ? acc[bk][i] * P.sc : -INFINITY);
        }
        m = col_max4(row_max16(m));
        mref[bk] = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(m)));
      }
    }
    // Only tiles that reach the causal edge, T or their own end need masks;
    // every other tile runs a loop without any masking code.
    const int last_t0 = ks + 16 * (nsteps - 1);
    const bool masked = last_t0 + 15 > lim_min || (PASS == 1 && last_t0 + 16 > ke);
    if constexpr (PASS == 1) {
      run_ep<EP_GEN>(masked);
    } else if (P.nsum == 1 && !tile_base) {
      run_ep<EP_SUM>(masked);
    } else if (P.nsum == 1 && !tile_mixed) {
      run_ep<EP_IMP>(masked);
    } else {
      run_ep<EP_GEN>(masked);
    }
    finish();
  }

  // Pass 1: the (reference, sum) partials of blocks Q0 .. Q0 + 3 of this key
  // tile, one store for the wave (compile-time indices only, so the sums stay
  // in registers).
  template <int Q0>
  __device__ __forceinline__ void store_partials() {
    float l = row_transpose_sum16(
        n, lsum[Q0][0], lsum[Q0][1], lsum[Q0][2], lsum[Q0][3], lsum[Q0 + 1][0], lsum[Q0 + 1][1],
        lsum[Q0 + 1][2], lsum[Q0 + 1][3], lsum[Q0 + 2][0], lsum[Q0 + 2][1], lsum[Q0 + 2][2],
        lsum[Q0 + 2][3], lsum[Q0 + 3][0], lsum[Q0 + 3][1], lsum[Q0 + 3][2], lsum[Q0 + 3][3]);
    const int bq = n >> 2, i = n & 3;
    const int bk = Q0 + bq;
    const int g = bk / RB, rb = bk % RB;
    const int j = h * G + g;
    const int r = r_lo + rb * 16 + 4 * c + i;
    const float m0 = mref[Q0], m1 = mref[Q0 + 1], m2 = mref[Q0 + 2], m3 = mref[Q0 + 3];
    const float mb = bq == 0 ? m0 : bq == 1 ? m1 : bq == 2 ? m2 : m3;
    // rows past the tile's first key hold no valid key here: (-inf, 0)
    const bool has_keys = ks <= P.T - P.Wn + r;
    const float m = has_keys ? mb : -INFINITY;
    if (!has_keys) l = 0.f;
    else if (!(l >= 0x1p-64f && l < INFINITY)) l = INFINITY;  // exact recompute
    if (active && r >= 0 && bk < NB)
      io.lse_part[(((int64_t)b * P.HQ + j) * P.Wn + r) * P.n_kt1 + kt] = make_float2(m, l);
  }

  __device__ __forceinline__ void finish() {
    if constexpr (PASS == 2) {
      lds_barrier();
      if (active) {
        const int64_t o = (((int64_t)b * P.n_rt + rt) * P.H + h) * P.Tc;
        for (int i = lane; i < P.tile2; i += 64) {
          const int t = ks + i;
          if (t < P.Tc) {
            io.psum_all[o + t] = obuf[(hs * P.nsum) * P.tile2 + i];
            io.psum_base[o + t] = obuf[(hs * P.nsum + P.nsum - 1) * P.tile2 + i];
          }
        }
        if (tile_base && hs == 0) {
          for (int i = lane; i < P.tile2; i += 64) {
            const int t = ks + i;
            if (t < P.Tc) io.ipart[((int64_t)b * P.n_rt + rt) * P.Tc + t] = ibuf[i];
          }
        }
      }
    } else {
      // Row sums of 4 blocks (16 quantities: block, row of the lane group) at a
      // time; lane n of each row ends with quantity n and stores its partial.
      static_assert(NBP == 4 || NBP == 8, "blocks in groups of four");
      store_partials<0>();
      if constexpr (NBP == 8) store_partials<4>();
    }
  }
};

template <class TT, int D, int G, int PASS>
__device__ __forceinline__ void score_tile(const Problem& P, const ScoreIO& io, int b, int kt, int rtg,
                                           float* smem, Part part = PART_ALL, uint32_t hmask = 0) {
  ScoreTile<TT, D, G, PASS> st(P, io, b, kt, rtg, smem, part, hmask);
  st.execute();
}

// Exact (max, sum) of one row over one pass-1 key tile by the online
// recurrence m' = max(m, x), l' = l * 2^(m - m') + 2^(x - m'), dot products
// on the vector ALU.  Only used when the tile's fast partial overflowed.
template <class TT, int D>
__device__ __forceinline__ float2 lse_partial_exact(const Problem P, const char* q, const char* k,
                                                  int64_t qrow, int64_t kb, int64_t ks_t, int pos,
                                                  int kt) {
  constexpr int ES = elem_bytes<TT>();
  constexpr int EPP = 16 / ES;  // elements per 16-byte piece
  // 16-byte pieces of the query row and each key row, converted as they are
  // read (no private copy of the row)
  const uint4* qp = reinterpret_cast<const uint4*>(q + qrow * ES);
  float m = -INFINITY, l = 0.f;
  const int t1 = min((kt + 1) * P.tile1, min(P.T, pos + 1));
  for (int t = kt * P.tile1; t < t1; ++t) {
    const uint4* kp = reinterpret_cast<const uint4*>(k + (kb + (int64_t)t * ks_t) * ES);
    float dot = 0.f;
    for (int pc = 0; pc < D / EPP; ++pc) {
      const uint4 a = qp[pc], bv = kp[pc];
      const uint32_t qa[4] = {a.x, a.y, a.z, a.w}, ka[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (ES == 2) {
          dot = fmaf(__uint_as_float(qa[w] << 16), __uint_as_float(ka[w] << 16), dot);
          dot = fmaf(__uint_as_float(qa[w] & 0xffff0000u), __uint_as_float(ka[w] & 0xffff0000u), dot);
        } else {
          dot = fmaf(__uint_as_float(qa[w]), __uint_as_float(ka[w]), dot);
        }
      }
    }
    const float x = dot * P.sc;
    const float mm = fmaxf(m, x);
    l = l * __builtin_amdgcn_exp2f(m - mm) + __builtin_amdgcn_exp2f(x - mm);
    m = mm;
  }
  return make_float2(m, l);
}

// Row normalisers: lse2 = log2 of the softmax normaliser of each window row,
// folded from the pass-1 key-tile partials in tile order.  A task reduces
// kLseRows rows of the window rows [r0, r0 + nr) of the heads in hmask; 8
// threads share a row and merge their partials by shuffles.
constexpr int kLseRows = 64;

template <class TT, int D, int G>
__device__ __forceinline__ void task_lse(const Problem& P, const ScoreIO& io, int b, int task, int r0,
                                         int nr, uint32_t hmask) {
  if (nr <= 0) return;
  const int nrows = P.HQ * nr;
  // local row = j * nr + rr, window row r = r0 + rr
  const int lrow = task * kLseRows + (int)(threadIdx.x >> 3);
  const int sub = threadIdx.x & 7;
  const int rr = lrow % nr, j = lrow / nr;
  const int r = r0 + rr;
  const int64_t row = ((int64_t)b * P.HQ + j) * P.Wn + r;
  const bool live = lrow < nrows && ((hmask >> (j / G)) & 1u);
  float m = -INFINITY, l = 0.f;
  if (live) {
    const float2* pp = io.lse_part + row * P.n_kt1;
    for (int t = sub; t < P.n_kt1; t += 8) {
      float2 p = pp[t];
      if (!(p.y < INFINITY)) {
        const int64_t qrow = (int64_t)b * io.qs_b + (int64_t)j * io.qs_h + (int64_t)r * io.qs_r;
        const int64_t kb = (int64_t)b * io.ks_b + (int64_t)(j / G) * io.ks_h;
        p = lse_partial_exact<TT, D>(P, io.q, io.k, qrow, kb, io.ks_t, P.T - P.Wn + r, t);
      }
      lse_merge(m, l, p.x, p.y);
    }
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) {
    const float m2 = __shfl_xor(m, o), l2 = __shfl_xor(l, o);
    lse_merge(m, l, m2, l2);
  }
  if (live && sub == 0) io.lse2[row] = m + log2f(l);
}

}  // namespace kvec
