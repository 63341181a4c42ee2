// Window scores of K-VEC on gfx950 (paper Sec. 4.1 Eq. eviction, the O'
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
//           a small kernel folds the tiles into lse2 = log2 of the normaliser.
//   pass 2  per key tile, all KV heads of one row tile in one work-group:
//           p = exp2(logit*log2e/sqrt(d) - lse2), summed over the tile's rows
//           per head (P and P over O'), and, for the rows of the last-O
//           window, max over heads through LDS then summed over rows (I).
// A final kernel adds the row-tile partial sums in a fixed order.
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
#include "kvec_internal.h"

#include <math.h>

namespace kvec {
namespace {

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

struct ScoreArgs {
  const char* q;
  const char* k;
  int64_t qs_b, qs_h, qs_r;  // element strides
  int64_t ks_b, ks_h, ks_t;
  int T, Wn, O, Tc, H, HQ;
  int n_rt, n_kt1;
  int tile;   // keys per work-group
  int SK;     // pass 2: keys per importance exchange
  float sc;   // log2(e) / sqrt(d)
  float2* lse_part;
  const float* lse2;
  float* psum_base;
  float* psum_all;
  float* ipart;
};

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

template <int G>
struct Tiling {
  static constexpr int RB = G >= 4 ? 1 : 4 / G;  // 16-row window blocks per row tile
  static constexpr int NB = G * RB;               // MFMA row blocks per wave
  static constexpr int WR = 16 * RB;              // window rows per row tile
};

// grid (key tiles, row tiles, batch), block 64*H: wave h = KV head h.
template <class TT, int D, int G, int PASS, bool ROBUST>
__device__ __forceinline__ void score_body(const ScoreArgs& a, float* smem) {
  using Tl = Tiling<G>;
  constexpr int RB = Tl::RB, NB = Tl::NB, WR = Tl::WR;
  constexpr int ES = elem_bytes<TT>();

  const int h = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int c = lane >> 4, n = lane & 15;
  const int kt = blockIdx.x, rt = blockIdx.y, b = blockIdx.z;
  const int r_lo = a.Wn - (rt + 1) * WR;  // lowest window row of this tile (may be < 0)
  const int base_lo = a.Wn - a.O;         // first row of the last-O window

  // Query fragments of this head's row tile (rows ordered (g, window row)).
  Frag<TT, D> qf[NB];
#pragma unroll
  for (int bk = 0; bk < NB; ++bk) {
    const int g = bk / RB, rb = bk % RB;
    const int r = r_lo + rb * 16 + n;
    const int j = h * G + g;
    if (r >= 0)
      qf[bk].load(a.q + ((int64_t)b * a.qs_b + (int64_t)j * a.qs_h + (int64_t)r * a.qs_r) * ES, c);
    else
      qf[bk].zero();
  }

  // Causal limit of each output row held by this lane: row r sees keys <= T-Wn+r.
  int pos[RB][4];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) pos[rb][i] = a.T - a.Wn + (r_lo + rb * 16 + 4 * c + i);

  const int tend = PASS == 1 ? a.T : a.Tc;
  const int ks = kt * a.tile;
  const int ke = min(ks + a.tile, tend);
  // Steps whose keys can exceed some row's causal limit need per-element masks.
  const int lim_min = a.T - a.Wn + max(r_lo, 0);
  const char* kbase = a.k + ((int64_t)b * a.ks_b + (int64_t)h * a.ks_h) * ES;

  int nsteps = (ke - ks + 15) / 16;
  if (PASS == 2) {
    const int sub = a.SK / 16;
    nsteps = (nsteps + sub - 1) / sub * sub;
  }

  // Pass-1 state: per (block, row) running reference and sum.
  float mref[NB][4], lsum[NB][4];
  // Pass-2 state: negated row normalisers (-inf for padding rows).
  float nlse[NB][4];
  bool tile_base = false, tile_mixed = false;
  if constexpr (PASS == 1) {
#pragma unroll
    for (int bk = 0; bk < NB; ++bk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        mref[bk][i] = -INFINITY;
        lsum[bk][i] = 0.f;
      }
  } else {
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      const int g = bk / RB, rb = bk % RB;
      const int j = h * G + g;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = r_lo + rb * 16 + 4 * c + i;
        nlse[bk][i] = r >= 0 ? -a.lse2[((int64_t)b * a.HQ + j) * a.Wn + r] : -INFINITY;
      }
    }
    tile_base = r_lo + WR > base_lo;                 // tile holds last-O window rows
    tile_mixed = tile_base && r_lo < base_lo;        // ... and extra rows
  }
  const int rr0 = max(0, base_lo - r_lo);            // first base row within the tile

  Frag<TT, D> kf, kn;
  {
    const int t = ks + n;
    if (t < tend) kf.load(kbase + (int64_t)t * a.ks_t * ES, c);
    else kf.zero();
  }

  for (int s = 0; s < nsteps; ++s) {
    const int t0 = ks + 16 * s;
    const int t = t0 + n;
    // Prefetch the next step's keys.
    if (s + 1 < nsteps) {
      const int tn = t + 16;
      if (tn < tend) kn.load(kbase + (int64_t)tn * a.ks_t * ES, c);
      else kn.zero();
    }
    f32x4 acc[NB];
#pragma unroll
    for (int bk = 0; bk < NB; ++bk) {
      acc[bk] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc[bk] = mma<D>(qf[bk], kf, acc[bk]);
    }
    const bool masked = t0 + 15 > lim_min;

    if constexpr (PASS == 1) {
#pragma unroll
      for (int bk = 0; bk < NB; ++bk) {
        const int rb = bk % RB;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool valid = !masked || t <= pos[rb][i];
          if constexpr (ROBUST) {
            if (valid) {
              const float cs = acc[bk][i] * a.sc;
              const float mm = fmaxf(mref[bk][i], cs);
              lsum[bk][i] = lsum[bk][i] * __builtin_amdgcn_exp2f(mref[bk][i] - mm) +
                            __builtin_amdgcn_exp2f(cs - mm);
              mref[bk][i] = mm;
            }
          } else if (s == 0) {
            mref[bk][i] = valid ? acc[bk][i] * a.sc : -INFINITY;
            lsum[bk][i] = valid ? 1.f : 0.f;
          } else {
            float x = fmaf(acc[bk][i], a.sc, -mref[bk][i]);
            if (masked) x = valid ? x : -INFINITY;
            lsum[bk][i] += __builtin_amdgcn_exp2f(x);
          }
        }
      }
    } else {
      // Probabilities, then the mean over the G query heads of each window row.
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
          float p = __builtin_amdgcn_exp2f(fmaf(acc[bk][i], a.sc, nlse[bk][i]));
          if (masked) p = t <= pos[rb][i] ? p : 0.f;
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
      if (tile_base) {
        s_base += __shfl_xor(s_base, 16);
        s_base += __shfl_xor(s_base, 32);
      }
      if (c == 0 && t < a.Tc) {
        const int64_t o = (((int64_t)b * a.n_rt + rt) * a.H + h) * a.Tc + t;
        a.psum_all[o] = s_all;
        if (tile_base) a.psum_base[o] = s_base;
      }
      if (tile_base) {
        // Importance: stage this head's row means; the work-group takes the
        // max over heads once every SK keys.
        const int kk = (s * 16) % a.SK + n;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int rr = rb * 16 + 4 * c + i;
            if (rr >= rr0) smem[(h * WR + rr) * a.SK + kk] = gs[rb][i];
          }
        if (((s + 1) * 16) % a.SK == 0) {
          __syncthreads();
          const int nthr = blockDim.x;
          float* ired = smem + a.H * WR * a.SK;
          const int kcol = threadIdx.x % a.SK, rg = threadIdx.x / a.SK, nrg = nthr / a.SK;
          float acc_i = 0.f;
          for (int rr = rr0 + rg; rr < WR; rr += nrg) {
            float m = smem[rr * a.SK + kcol];
            for (int hh = 1; hh < a.H; ++hh) m = fmaxf(m, smem[(hh * WR + rr) * a.SK + kcol]);
            acc_i += m;
          }
          ired[rg * a.SK + kcol] = acc_i;
          __syncthreads();
          if ((int)threadIdx.x < a.SK) {
            float v = 0.f;
            for (int g2 = 0; g2 < nrg; ++g2) v += ired[g2 * a.SK + threadIdx.x];
            const int tt = ks + (s + 1) * 16 - a.SK + threadIdx.x;
            if (tt < a.Tc) a.ipart[((int64_t)b * a.n_rt + rt) * a.Tc + tt] = v;
          }
          __syncthreads();
        }
      }
    }
    kf = kn;
  }

  if constexpr (PASS == 1) {
    // Fold the 16 key lanes of each row, then write (max, sum) per row.
    bool bad = false;
#pragma unroll
    for (int bk = 0; bk < NB; ++bk)
#pragma unroll
      for (int i = 0; i < 4; ++i) bad |= !(lsum[bk][i] < INFINITY);
    if constexpr (!ROBUST) {
      if (__any(bad)) {
        // A logit exceeded the lane's reference by more than the fp32 range:
        // recompute this tile with the exact online recurrence.
        score_body<TT, D, G, PASS, true>(a, smem);
        return;
      }
    }
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
        if (n == 0 && r >= 0)
          a.lse_part[(((int64_t)b * a.HQ + j) * a.Wn + r) * a.n_kt1 + kt] = make_float2(m, l);
      }
    }
  }
}

template <class TT, int D, int G, int PASS, int MAXT>
__global__ __launch_bounds__(MAXT) void score_kernel(ScoreArgs a) {
  extern __shared__ float smem[];
  score_body<TT, D, G, PASS, false>(a, smem);
}

// lse2[b][j][r] = log2 of the softmax normaliser of row (j, r), from the
// per-tile partials, folded in tile order.
__global__ void lse_reduce_kernel(const float2* part, float* lse2, int rows, int n_kt) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows) return;
  float m = -INFINITY, l = 0.f;
  for (int t = 0; t < n_kt; ++t) {
    const float2 p = part[(int64_t)i * n_kt + t];
    lse_merge(m, l, p.x, p.y);
  }
  lse2[i] = m + log2f(l);
}

// P, P over O', I from the row-tile partial sums (fixed order).
__global__ void finalize_kernel(const float* psum_base, const float* psum_all, const float* ipart,
                                float* p_raw, float* p_ext, float* imp, int H, int Tc, int n_rt,
                                int n_rt_base, float inv_go, float inv_gwn) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int y = blockIdx.y, b = blockIdx.z;
  if (t >= Tc) return;
  if (y < H) {
    float sb = 0.f, sa = 0.f;
    for (int rt = 0; rt < n_rt; ++rt) {
      const int64_t o = (((int64_t)b * n_rt + rt) * H + y) * Tc + t;
      if (rt < n_rt_base) sb += psum_base[o];
      sa += psum_all[o];
    }
    p_raw[((int64_t)b * H + y) * Tc + t] = sb * inv_go;
    p_ext[((int64_t)b * H + y) * Tc + t] = sa * inv_gwn;
  } else {
    float s = 0.f;
    for (int rt = 0; rt < n_rt_base; ++rt) s += ipart[((int64_t)b * n_rt + rt) * Tc + t];
    imp[(int64_t)b * Tc + t] = s * inv_go;
  }
}

// Work-groups of up to 8 waves (H <= 8) leave each wave 256 registers; larger
// head counts use the 16-wave variant.
template <class TT, int D, int G, int MAXT>
hipError_t launch_passes(const Geometry& g, ScoreArgs a, hipStream_t s, hipEvent_t* ev) {
  using Tl = Tiling<G>;
  const dim3 block(64 * g.H);
  hipError_t e;
  if (ev) hipEventRecord(ev[0], s);
  a.tile = kTilePass1;
  hipLaunchKernelGGL((score_kernel<TT, D, G, 1, MAXT>), dim3(g.n_kt1, g.n_rt, g.batch), block, 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev) hipEventRecord(ev[1], s);
  const int rows = g.batch * g.HQ * g.Wn;
  hipLaunchKernelGGL(lse_reduce_kernel, dim3((rows + 255) / 256), dim3(256), 0, s, a.lse_part,
                     const_cast<float*>(a.lse2), rows, g.n_kt1);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev) hipEventRecord(ev[2], s);
  a.tile = kTilePass2;
  const size_t lds = (size_t)(g.H * Tl::WR * g.SK + 64 * g.H) * sizeof(float);
  if (lds > 65536) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&score_kernel<TT, D, G, 2, MAXT>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((score_kernel<TT, D, G, 2, MAXT>), dim3(g.n_kt2, g.n_rt, g.batch), block, lds, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev) hipEventRecord(ev[3], s);
  return hipSuccess;
}

template <class TT, int D>
hipError_t dispatch_group(const Geometry& g, ScoreArgs a, hipStream_t s, hipEvent_t* ev) {
  const bool big = g.H > 8;
  switch (g.G) {
    case 1: return big ? launch_passes<TT, D, 1, 1024>(g, a, s, ev) : launch_passes<TT, D, 1, 512>(g, a, s, ev);
    case 2: return big ? launch_passes<TT, D, 2, 1024>(g, a, s, ev) : launch_passes<TT, D, 2, 512>(g, a, s, ev);
    case 4: return big ? launch_passes<TT, D, 4, 1024>(g, a, s, ev) : launch_passes<TT, D, 4, 512>(g, a, s, ev);
    case 8: return big ? launch_passes<TT, D, 8, 1024>(g, a, s, ev) : launch_passes<TT, D, 8, 512>(g, a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int row_blocks_per_tile(int G) {
  switch (G) {
    case 1: return Tiling<1>::RB;
    case 2: return Tiling<2>::RB;
    case 4: return Tiling<4>::RB;
    default: return Tiling<8>::RB;
  }
}

hipError_t launch_score(const Geometry& g, const void* q, const int64_t qs[3], const void* k,
                        const int64_t ks[3], float* p_raw, float* p_ext, float* imp, char* ws,
                        const Workspace& w, hipStream_t s, hipEvent_t* ev) {
  ScoreArgs a;
  a.q = static_cast<const char*>(q);
  a.k = static_cast<const char*>(k);
  a.qs_b = qs[0]; a.qs_h = qs[1]; a.qs_r = qs[2];
  a.ks_b = ks[0]; a.ks_h = ks[1]; a.ks_t = ks[2];
  a.T = g.T; a.Wn = g.Wn; a.O = g.O; a.Tc = g.Tc; a.H = g.H; a.HQ = g.HQ;
  a.n_rt = g.n_rt; a.n_kt1 = g.n_kt1;
  a.tile = 0;
  a.SK = g.SK;
  a.sc = (float)(1.4426950408889634 / sqrt((double)g.D));
  a.lse_part = reinterpret_cast<float2*>(ws + w.lse_part);
  a.lse2 = reinterpret_cast<const float*>(ws + w.lse2);
  a.psum_base = reinterpret_cast<float*>(ws + w.psum_base);
  a.psum_all = reinterpret_cast<float*>(ws + w.psum_all);
  a.ipart = reinterpret_cast<float*>(ws + w.ipart);
  hipError_t e;
  if (g.dtype == KVEC_BF16)
    e = g.D == 64 ? dispatch_group<BF16, 64>(g, a, s, ev) : dispatch_group<BF16, 128>(g, a, s, ev);
  else
    e = g.D == 64 ? dispatch_group<F32, 64>(g, a, s, ev) : dispatch_group<F32, 128>(g, a, s, ev);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(finalize_kernel, dim3((g.Tc + 255) / 256, g.H + 1, g.batch), dim3(256), 0, s,
                     a.psum_base, a.psum_all, a.ipart, p_raw, p_ext, imp, g.H, g.Tc, g.n_rt,
                     g.n_rt_base, (float)(1.0 / ((double)g.G * g.O)),
                     (float)(1.0 / ((double)g.G * g.Wn)));
  return hipGetLastError();
}

}  // namespace kvec
