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
// l supplies row/key (l % 16) and the head-dim slice [c*D/4, (c+1)*D/4) with
// c = l / 16, split into k-steps; the dot product is order-free, so this
// permutation of the reduction index is legal and gives each lane one
// contiguous D/4-element load per row or key.  The output lane l holds rows
// 4c..4c+3 of the block for key (l % 16).  A wave owns one KV head and
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
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(row) + c * (D / 4));
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = __builtin_bit_cast(bf16x8, p[j]);
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int j = 0; j < KS; ++j) v[j] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  }
};

template <int D>
struct Frag<F32, D> {
  static constexpr int KS = D / 4;
  float v[KS];
  __device__ __forceinline__ void load(const void* row, int c) {
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const float*>(row) + c * (D / 4));
#pragma unroll
    for (int j = 0; j < KS / 4; ++j) {
      const uint4 u = p[j];
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

template <class TT>
constexpr int elem_bytes() { return __is_same(TT, BF16) ? 2 : 4; }

// Work-group barrier that orders LDS only: pending global loads (the K
// prefetch ring) stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
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
  float* psum_base;   // [b][n_rt][H][Tc]
  float* psum_all;    // [b][n_rt][H][Tc]
  float* ipart;       // [b][n_rt][Tc]
};

constexpr int kPrefetch = 4;  // K fragments in flight per wave (divides the steps of a tile)

// One pass over one key tile for the row tiles of this work-group.
// Block: 512 threads; wave w -> head w % H, row tile rtg*(8/H) + w / H.
// The state lives in a struct whose methods are all force-inlined, so every
// array is indexed by compile-time constants and stays in registers.
#ifndef KVEC_PIPELINE_MMA
#define KVEC_PIPELINE_MMA 1
#endif
// When set, the matrix products of step s+1 are issued before the exponentials
// of step s (two accumulator sets); otherwise each step multiplies, then
// exponentiates.
constexpr bool kPipelineMma = KVEC_PIPELINE_MMA != 0;

template <class TT, int D, int G, int PASS>
struct ScoreTile {
  using Tl = Tiling<G>;
  static constexpr int RB = Tl::RB, NB = Tl::NB, WR = Tl::WR;
  static constexpr int ES = elem_bytes<TT>();

  const Problem& P;
  const ScoreIO& io;
  int b, kt, rtg;
  int lane, c, n, tpw, h, slot, rt;
  bool active;
  int r_lo, base_lo, tend, ks, ke, lim_min, nsteps, rr0;
  const char* kbase;
  bool tile_base, tile_mixed, wg_base;
  float *xbuf, *ired, *obuf, *ibuf;

  Frag<TT, D> qf[NB];
  Frag<TT, D> kr[kPrefetch];
  f32x4 acc[2][NB];
  float mref[NB][4], lsum[NB][4], nlse[NB][4];
  int pos[RB][4];

  __device__ __forceinline__ ScoreTile(const Problem& P_, const ScoreIO& io_, int b_, int kt_,
                                       int rtg_, float* smem)
      : P(P_), io(io_), b(b_), kt(kt_), rtg(rtg_) {
    const int w = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    c = lane >> 4;
    n = lane & 15;
    tpw = 8 / P.H;  // row tiles per work-group
    h = w % P.H;
    slot = w / P.H;
    rt = rtg * tpw + slot;
    active = slot < tpw && rt < P.n_rt;
    r_lo = P.Wn - (rt + 1) * WR;  // lowest window row of this tile (may be < 0)
    base_lo = P.Wn - P.O;         // first row of the last-O window

    // Query fragments; loads are unconditional (clamped rows) so the compiler
    // can count outstanding loads exactly, then padding rows are zeroed.
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      const int g = bk / RB, rb = bk % RB;
      const int r = r_lo + rb * 16 + n;
      const int j = h * G + g;
      qf[bk].load(io.q + ((int64_t)b * io.qs_b + (int64_t)j * io.qs_h + (int64_t)max(r, 0) * io.qs_r) * ES,
                  c);
    }
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      const int r = r_lo + (bk % RB) * 16 + n;
      if (!(active && r >= 0)) qf[bk].zero();
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) pos[rb][i] = P.T - P.Wn + (r_lo + rb * 16 + 4 * c + i);

    tend = PASS == 1 ? P.T : P.Tc;
    const int tile = PASS == 1 ? kTile1 : kTile2;
    ks = kt * tile;
    ke = min(ks + tile, tend);
    lim_min = P.T - P.Wn + max(r_lo, 0);
    kbase = io.k + ((int64_t)b * io.ks_b + (int64_t)h * io.ks_h) * ES;
    // Steps are padded to a multiple of the prefetch depth (and, in pass 2, of
    // the importance exchange) so the unrolled loop has no step guard; keys at
    // or past ke are masked (pass 1) or never stored (pass 2).
    nsteps = (ke - ks + 15) / 16;
    const int sub = PASS == 2 ? max(kPrefetch, P.SK / 16) : kPrefetch;
    nsteps = (nsteps + sub - 1) / sub * sub;

    tile_base = tile_mixed = wg_base = false;
    if constexpr (PASS == 1) {
#pragma unroll
      for (int bk = 0; bk < NB; ++bk)
#pragma unroll
        for (int i = 0; i < 4; ++i) lsum[bk][i] = 0.f;
    } else {
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int g = bk / RB, rb = bk % RB;
        const int j = h * G + g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = r_lo + rb * 16 + 4 * c + i;
          const float v = io.lse2[((int64_t)b * P.HQ + j) * P.Wn + max(r, 0)];
          nlse[bk][i] = (active && r >= 0) ? -v : -INFINITY;
        }
      }
      tile_base = active && r_lo + WR > base_lo;
      tile_mixed = tile_base && r_lo < base_lo;
      // A work-group exchanges importance rows when any of its tiles holds base
      // rows; the first tile of the group is the newest, so checking it suffices.
      wg_base = (P.Wn - (rtg * tpw + 1) * WR) + WR > base_lo;
    }
    rr0 = max(0, base_lo - r_lo);
    // pass-2 LDS per tile slot: importance exchange, its reduction, the staged
    // per-key sums of each head, and the staged importance of the key tile
    xbuf = smem + slot * (P.H * WR * P.SK + 64 * P.H + 2 * P.H * kTile2 + kTile2);
    ired = xbuf + P.H * WR * P.SK;
    obuf = ired + 64 * P.H;
    ibuf = obuf + 2 * P.H * kTile2;
  }

  __device__ __forceinline__ void load_keys(int u, int step) {
    // unconditional: rows clamped to tend-1 (masked or never stored)
    const int t = min(ks + 16 * step + n, tend - 1);
    kr[u].load(kbase + (int64_t)t * io.ks_t * ES, c);
  }

  template <int SET, int RING>
  __device__ __forceinline__ void mma_step() {
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) acc[SET][bk] = mma<D>(qf[bk], kr[RING], f32x4{0.f, 0.f, 0.f, 0.f});
  }

  template <int SET, bool MASKED>
  __device__ __forceinline__ void epilogue(int s) {
    const int t = ks + 16 * s + n;
    if constexpr (PASS == 1) {
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int rb = bk % RB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = fmaf(acc[SET][bk][i], P.sc, -mref[bk][i]);
          if constexpr (MASKED) x = (t <= pos[rb][i] && t < ke) ? x : -INFINITY;
          lsum[bk][i] += __builtin_amdgcn_exp2f(x);
        }
      }
    } else {
      float gs[RB][4];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) gs[rb][i] = 0.f;
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int rb = bk % RB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float p = __builtin_amdgcn_exp2f(fmaf(acc[SET][bk][i], P.sc, nlse[bk][i]));
          if constexpr (MASKED) p = t <= pos[rb][i] ? p : 0.f;
          gs[rb][i] += p;
        }
      }
      float s_all = 0.f, s_base = 0.f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s_all += gs[rb][i];
          if (tile_mixed) s_base += (r_lo + rb * 16 + 4 * c + i >= base_lo) ? gs[rb][i] : 0.f;
        }
      if (tile_base && !tile_mixed) s_base = s_all;
      s_all += __shfl_xor(s_all, 16);
      s_all += __shfl_xor(s_all, 32);
      s_base += __shfl_xor(s_base, 16);
      s_base += __shfl_xor(s_base, 32);
      // Stage the per-key sums in LDS; they are written out after the loop so
      // that the loop issues no global stores (exact load counting).
      if (c == 0) {
        obuf[(h * 2 + 0) * kTile2 + s * 16 + n] = s_all;
        obuf[(h * 2 + 1) * kTile2 + s * 16 + n] = s_base;
      }
      if (wg_base && tile_base) {
        const int kk = (s * 16) % P.SK + n;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int rr = rb * 16 + 4 * c + i;
            if (rr >= rr0) xbuf[(h * WR + rr) * P.SK + kk] = gs[rb][i];
          }
      }
    }
  }

  // Importance of one exchange block: max over heads, then sum over base rows.
  __device__ __forceinline__ void exchange(int s) {
    lds_barrier();
    const int nthr = 64 * P.H;
    const int ts = threadIdx.x - slot * nthr;  // thread index within the slot
    if (tile_base && slot < tpw) {
      const int kcol = ts % P.SK, rg = ts / P.SK, nrg = nthr / P.SK;
      float acc_i = 0.f;
      for (int rr = rr0 + rg; rr < WR; rr += nrg) {
        float m = xbuf[rr * P.SK + kcol];
        for (int hh = 1; hh < P.H; ++hh) m = fmaxf(m, xbuf[(hh * WR + rr) * P.SK + kcol]);
        acc_i += m;
      }
      ired[rg * P.SK + kcol] = acc_i;
    }
    lds_barrier();
    if (tile_base && slot < tpw && ts < P.SK) {
      float v = 0.f;
      for (int g2 = 0; g2 < nthr / P.SK; ++g2) v += ired[g2 * P.SK + ts];
      ibuf[(s + 1) * 16 - P.SK + ts] = v;
    }
    lds_barrier();
  }

  // One step of the software pipeline: the MFMAs of step s+1 are issued into
  // the other accumulator set before the epilogue of step s, so matrix cores
  // and vector ALU work concurrently; then ring slot U (step s, already
  // consumed) is refilled with step s + kPrefetch.
  template <int U, bool TILE_MASKED>
  __device__ __forceinline__ void step(int s) {
    constexpr int CUR = kPipelineMma ? (U & 1) : 0, NXT = CUR ^ 1;
    if constexpr (kPipelineMma) {
      if (s + 1 < nsteps) mma_step<NXT, (U + 1) % kPrefetch>();
    } else {
      mma_step<0, U>();
    }
    load_keys(U, s + kPrefetch);
    if constexpr (TILE_MASKED) {
      const int t0 = ks + 16 * s;
      if (t0 + 15 > lim_min || (PASS == 1 && t0 + 16 > ke))
        epilogue<CUR, true>(s);
      else
        epilogue<CUR, false>(s);
    } else {
      epilogue<CUR, false>(s);
    }
    if constexpr (PASS == 2) {
      if (wg_base && ((s + 1) * 16) % P.SK == 0) exchange(s);
    }
  }

  template <bool TILE_MASKED>
  __device__ __forceinline__ void run() {
    for (int s0 = 0; s0 < nsteps; s0 += kPrefetch) {
      static_assert(kPrefetch == 4, "the step sequence below assumes four ring slots");
      step<0, TILE_MASKED>(s0);
      step<1, TILE_MASKED>(s0 + 1);
      step<2, TILE_MASKED>(s0 + 2);
      step<3, TILE_MASKED>(s0 + 3);
    }
  }

  __device__ __forceinline__ void execute() {
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) load_keys(u, u);
    if constexpr (PASS == 1) {
      mma_step<0, 0>();
      // Reference of each (lane, row): its logit at the first key it sees; an
      // invalid first key leaves -inf, and then every later key of that lane
      // and row is masked too (keys only grow).
      const int t = ks + n;
      const bool m0 = ks + 15 > lim_min || ks + 16 > ke;
#pragma unroll
      for (int bk = 0; bk < NB; ++bk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool valid = !m0 || (t <= pos[bk % RB][i] && t < ke);
          mref[bk][i] = valid ? acc[0][bk][i] * P.sc : -INFINITY;
        }
    } else if constexpr (kPipelineMma) {
      mma_step<0, 0>();
    }
    // Only tiles that reach the causal edge, T or their own end need masks;
    // every other tile runs a loop without any masking code.
    const int last_t0 = ks + 16 * (nsteps - 1);
    if (last_t0 + 15 > lim_min || (PASS == 1 && last_t0 + 16 > ke))
      run<true>();
    else
      run<false>();
    finish();
  }

  __device__ __forceinline__ void finish() {
    if constexpr (PASS == 2) {
      lds_barrier();
      if (active) {
        const int64_t o = (((int64_t)b * P.n_rt + rt) * P.H + h) * P.Tc;
        for (int i = lane; i < kTile2; i += 64) {
          const int t = ks + i;
          if (t < P.Tc) {
            io.psum_all[o + t] = obuf[(h * 2 + 0) * kTile2 + i];
            io.psum_base[o + t] = obuf[(h * 2 + 1) * kTile2 + i];
          }
        }
        if (tile_base && h == 0) {
          for (int i = lane; i < kTile2; i += 64) {
            const int t = ks + i;
            if (t < P.Tc) io.ipart[((int64_t)b * P.n_rt + rt) * P.Tc + t] = ibuf[i];
          }
        }
      }
    } else {
      // A lane whose later logits exceed its reference by more than the fp32
      // exponent range leaves a non-finite sum; the row-normaliser task then
      // recomputes that tile's partial with the exact online recurrence.
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int g = bk / RB, rb = bk % RB;
        const int j = h * G + g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float m = mref[bk][i], l = lsum[bk][i];
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) {
            const float m2 = __shfl_xor(m, o), l2 = __shfl_xor(l, o);
            lse_merge(m, l, m2, l2);
          }
          const int r = r_lo + rb * 16 + 4 * c + i;
          if (active && n == 0 && r >= 0)
            io.lse_part[(((int64_t)b * P.HQ + j) * P.Wn + r) * P.n_kt1 + kt] = make_float2(m, l);
        }
      }
    }
  }
};

template <class TT, int D, int G, int PASS>
__device__ __forceinline__ void score_tile(const Problem& P, const ScoreIO& io, int b, int kt, int rtg,
                                           float* smem) {
  ScoreTile<TT, D, G, PASS> st(P, io, b, kt, rtg, smem);
  st.execute();
}

// Exact (max, sum) of one row over one pass-1 key tile by the online
// recurrence m' = max(m, x), l' = l * 2^(m - m') + 2^(x - m'), dot products
// on the vector ALU.  Only used when the tile's fast partial overflowed.
template <class TT, int D>
__device__ __noinline__ float2 lse_partial_exact(const Problem P, const char* q, const char* k,
                                                  int64_t qrow, int64_t kb, int64_t ks_t, int pos,
                                                  int kt) {
  constexpr int ES = elem_bytes<TT>();
  float qv[D];
  for (int i = 0; i < D; ++i) {
    if constexpr (ES == 2) {
      const uint16_t u = reinterpret_cast<const uint16_t*>(q + qrow * ES)[i];
      qv[i] = __uint_as_float((uint32_t)u << 16);
    } else {
      qv[i] = reinterpret_cast<const float*>(q + qrow * ES)[i];
    }
  }
  float m = -INFINITY, l = 0.f;
  const int t1 = min((kt + 1) * kTile1, min(P.T, pos + 1));
  for (int t = kt * kTile1; t < t1; ++t) {
    const char* kr = k + (kb + (int64_t)t * ks_t) * ES;
    float dot = 0.f;
    for (int i = 0; i < D; ++i) {
      float kv;
      if constexpr (ES == 2)
        kv = __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(kr)[i] << 16);
      else
        kv = reinterpret_cast<const float*>(kr)[i];
      dot = fmaf(qv[i], kv, dot);
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
// kLseRows rows; 8 threads share a row and merge their partials by shuffles.
constexpr int kLseRows = 64;

template <class TT, int D, int G>
__device__ __forceinline__ void task_lse(const Problem& P, const ScoreIO& io, int part) {
  const int nrows = P.batch * P.HQ * P.Wn;
  const int row = part * kLseRows + (int)(threadIdx.x >> 3);
  const int sub = threadIdx.x & 7;
  float m = -INFINITY, l = 0.f;
  if (row < nrows) {
    const float2* pp = io.lse_part + (int64_t)row * P.n_kt1;
    for (int t = sub; t < P.n_kt1; t += 8) {
      float2 p = pp[t];
      if (!(p.y < INFINITY)) {
        // row = (b * HQ + j) * Wn + r
        const int r = row % P.Wn, bj = row / P.Wn;
        const int j = bj % P.HQ, b = bj / P.HQ;
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
  if (row < nrows && sub == 0) io.lse2[row] = m + log2f(l);
}

}  // namespace kvec
