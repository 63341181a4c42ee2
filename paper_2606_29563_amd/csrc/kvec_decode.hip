// Decode-step attention over the compacted cache.
//
// The eviction step stores the kept K/V of every KV head (Sec. 4.1); the
// decoding phase then attends from each new token's query heads to those
// rows.  For one decode token, query head j of sequence b computes
//   out[b][j] = sum_i softmax_i(q_j . k_i / sqrt(d)) v_i
// over the rows i of its KV head j / G, leaving out the padding rows that
// kvec_compact writes when T <= B (idx -1).
//
// The work is bound by reading the cache once.  Two launches:
//   partial  one work-group per (row chunk, KV head, sequence): the G query
//            heads of the KV head share every K/V row read.  A row is read by
//            a group of lanes, 16 bytes each (fully coalesced), the group's
//            partial dot products are summed with DPP lane moves, and each
//            lane keeps an online-softmax state (max, sum, weighted V
//            elements) per query head.  States merge across the row groups
//            of a wave by shuffles, across waves through LDS, and the
//            chunk's (max, sum, V[d]) go to the workspace.
//   combine  one work-group per (query head, sequence) merges the chunks.
// (A single launch in which the last partial work-group of each head
// combines, behind an arrival counter, measured slower: the combine then
// runs as a serial tail after the slowest chunk, and the release/acquire
// fences it needs across the XCDs' caches cost more than the launch saved.)
#include <math.h>

#include <mutex>

#include "kvec_internal.h"
#include "kvec_score_dev.h"  // DPP lane moves

namespace kvec {
namespace {

constexpr int kDecThreads = 256;        // 4 waves per partial work-group
constexpr int kDecWaves = kDecThreads / 64;
constexpr int kDecUnroll = 4;           // rows in flight per lane group

template <class T>
struct DecElem;
template <>
struct DecElem<__bf16> {
  static constexpr int N = 8;  // elements per 16-byte piece
  __device__ static void unpack(const uint4& u, float (&f)[N]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <>
struct DecElem<float> {
  static constexpr int N = 4;
  __device__ static void unpack(const uint4& u, float (&f)[N]) {
    f[0] = __uint_as_float(u.x);
    f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z);
    f[3] = __uint_as_float(u.w);
  }
};

struct DecArgs {
  const char* q;
  int64_t qs_b, qs_h;   // elements
  const char* k;
  const char* v;
  int64_t cs_b, cs_h;   // elements; rows contiguous (d elements apart)
  const int32_t* idx;   // nullable [b][H][B]
  float* part;          // [b][HQ][S][D + 2]
  float* out;           // [b][HQ][D]
  int H, HQ, B, n_ctx, chunk, S;
  float sc;             // log2(e) / sqrt(d)
};

// Merge (m2, l2, a2) into (m, l, a); m = -inf means an empty state.
// Branch-free, so the lane moves feeding a batch of merges stay in flight
// together.
__device__ __forceinline__ void dec_merge(float& m, float& l, float* a, float m2, float l2,
                                          const float* a2, int n) {
  const float mm = fmaxf(m, m2);
  const float f1 = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mm);
  const float f2 = m2 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m2 - mm);
  l = l * f1 + l2 * f2;
  for (int e = 0; e < n; ++e) a[e] = a[e] * f1 + a2[e] * f2;
  m = mm;
}

// Sum over each aligned group of LPR lanes, every lane of the group getting
// the total: quad swaps, the half-row mirror and the row rotation by 8 (DPP,
// no LDS round trip), lane shuffles only across 16-lane rows.
template <int LPR>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (LPR >= 2) v += dpp_f<kDppSwap1>(v);
  if constexpr (LPR >= 4) v += dpp_f<kDppSwap2>(v);
  if constexpr (LPR >= 8) v += dpp_f<kDppHalfMirror>(v);
  if constexpr (LPR >= 16) v += dpp_f<kDppRor8>(v);
  if constexpr (LPR >= 32) v += __shfl_xor(v, 16);
  if constexpr (LPR >= 64) v += __shfl_xor(v, 32);
  return v;
}

template <class T, int D, int G>
__global__ __launch_bounds__(kDecThreads) void decode_partial(DecArgs a) {
  using E = DecElem<T>;
  constexpr int EPL = E::N;            // elements of d per lane
  constexpr int LPR = D / EPL;         // lanes per row
  constexpr int RPW = 64 / LPR;        // rows per wave and round
  __shared__ float sm[kDecWaves][G][2];
  __shared__ float sa[kDecWaves][G][D];
  const int s = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int grp = lane / LPR, pc = lane % LPR;  // row group, piece of the row
  const int r0 = s * a.chunk, r1 = min(a.n_ctx, r0 + a.chunk);

  float qv[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 u = reinterpret_cast<const uint4*>(
        a.q + ((int64_t)b * a.qs_b + (int64_t)(h * G + g) * a.qs_h) * sizeof(T))[pc];
    E::unpack(u, qv[g]);
  }
  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }
  const char* kb = a.k + ((int64_t)b * a.cs_b + (int64_t)h * a.cs_h) * sizeof(T);
  const char* vb = a.v + ((int64_t)b * a.cs_b + (int64_t)h * a.cs_h) * sizeof(T);
  const int32_t* ib = a.idx ? a.idx + ((int64_t)b * a.H + h) * a.B : nullptr;
  // without idx every lane reads word 0 of its K rows instead (unused), so
  // the loads below need no branch
  const int32_t* ibp = ib ? ib : reinterpret_cast<const int32_t*>(kb);
  const int imax = ib ? a.B - 1 : 0;
  constexpr int kStep = kDecWaves * RPW;  // rows per round of the work-group
  for (int base = r0; base < r1; base += kStep * kDecUnroll) {
    uint4 ku[kDecUnroll], vu[kDecUnroll];
    int iv[kDecUnroll];
    bool live[kDecUnroll];
    // issue every load of the unrolled rounds first, with no wait in between:
    // the idx entries at clamped (in-bounds) positions, and the rows below
    // n_ctx (all in bounds) whether or not idx masks them
#pragma unroll
    for (int uu = 0; uu < kDecUnroll; ++uu) {
      const int r = base + uu * kStep + w * RPW + grp;
      // rows past the chunk load the chunk's last row (never used)
      const int rl = min(r, r1 - 1);
      iv[uu] = ibp[min(r, imax)];
      live[uu] = r < r1;
      ku[uu] = reinterpret_cast<const uint4*>(kb + (int64_t)rl * D * sizeof(T))[pc];
      vu[uu] = reinterpret_cast<const uint4*>(vb + (int64_t)rl * D * sizeof(T))[pc];
    }
#pragma unroll
    for (int uu = 0; uu < kDecUnroll; ++uu) {
      const int r = base + uu * kStep + w * RPW + grp;
      if (ib && r < a.B && iv[uu] < 0) live[uu] = false;
      float kf[EPL], vf[EPL];
      E::unpack(ku[uu], kf);
      E::unpack(vu[uu], vf);
      float x[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d = fmaf(qv[g][e], kf[e], d);
        x[g] = d;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        // every lane takes part in the lane moves, masked rows included
        const float dsum = group_sum<LPR>(x[g]);
        x[g] = live[uu] ? dsum * a.sc : -INFINITY;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        // online softmax; a masked row (x = -inf) leaves the state as it is
        const float mm = fmaxf(m[g], x[g]);
        const float f = m[g] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[g] - mm);
        const float p = x[g] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(x[g] - mm);
        l[g] = l[g] * f + p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e] * f);
        m[g] = mm;
      }
    }
  }
  // merge the RPW row groups of the wave (lanes with the same piece)
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a2[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) a2[e] = __shfl_xor(acc[g][e], o);
      const float m2 = __shfl_xor(m[g], o), l2 = __shfl_xor(l[g], o);
      dec_merge(m[g], l[g], acc[g], m2, l2, a2, EPL);
    }
  }
  if (grp == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (pc == 0) {
        sm[w][g][0] = m[g];
        sm[w][g][1] = l[g];
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) sa[w][g][pc * EPL + e] = acc[g][e];
    }
  }
  __syncthreads();
  // merge the waves: thread (g, e) for every element of every query head
  for (int t = threadIdx.x; t < G * D; t += kDecThreads) {
    const int g = t / D, e = t % D;
    float mm = -INFINITY, ll = 0.f, av = 0.f;
    for (int ww = 0; ww < kDecWaves; ++ww) dec_merge(mm, ll, &av, sm[ww][g][0], sm[ww][g][1], &sa[ww][g][e], 1);
    float* pp = a.part + (((int64_t)b * a.HQ + h * G + g) * a.S + s) * (D + 2);
    pp[2 + e] = av;
    if (e == 0) {
      pp[0] = mm;
      pp[1] = ll;
    }
  }
}

// Chunk states are read in batches of kDecBatch with every load of a batch in
// flight at once (the chunks were written by other work-groups, on other
// XCDs, so each read is a memory round trip): up to kDecBatch chunks in one
// round trip, more in two passes (the maximum, then the rescaled sums).  Both
// orders add the chunks in ascending order.
constexpr int kDecBatch = 16;

template <int D>
__device__ __forceinline__ float combine_elem(const DecArgs& a, int b, int j, int e) {
  const float* pp = a.part + ((int64_t)b * a.HQ + j) * a.S * (D + 2);
  float m = -INFINITY, l = 0.f, av = 0.f;
  if (a.S <= kDecBatch) {
    float ms[kDecBatch], ls[kDecBatch], as[kDecBatch];
#pragma unroll
    for (int i = 0; i < kDecBatch; ++i) {
      const bool ok = i < a.S;
      const float* q = pp + (int64_t)(ok ? i : 0) * (D + 2);
      ms[i] = ok ? q[0] : -INFINITY;
      ls[i] = q[1];
      as[i] = q[2 + e];
    }
#pragma unroll
    for (int i = 0; i < kDecBatch; ++i) m = fmaxf(m, ms[i]);
    if (m != -INFINITY) {
#pragma unroll
      for (int i = 0; i < kDecBatch; ++i) {
        // empty chunks (m = -inf) weigh exp2(-inf) = 0
        const float f = __builtin_amdgcn_exp2f(ms[i] - m);
        l = fmaf(ls[i], f, l);
        av = fmaf(as[i], f, av);
      }
    }
    return l > 0.f ? av / l : 0.f;
  }
  for (int s0 = 0; s0 < a.S; s0 += kDecBatch) {
    float ms[kDecBatch];
#pragma unroll
    for (int i = 0; i < kDecBatch; ++i) ms[i] = s0 + i < a.S ? pp[(s0 + i) * (D + 2)] : -INFINITY;
#pragma unroll
    for (int i = 0; i < kDecBatch; ++i) m = fmaxf(m, ms[i]);
  }
  if (m != -INFINITY) {
    for (int s0 = 0; s0 < a.S; s0 += kDecBatch) {
      float ms[kDecBatch], ls[kDecBatch], as[kDecBatch];
#pragma unroll
      for (int i = 0; i < kDecBatch; ++i) {
        const bool ok = s0 + i < a.S;
        const float* q = pp + (int64_t)(ok ? s0 + i : 0) * (D + 2);
        ms[i] = ok ? q[0] : -INFINITY;
        ls[i] = q[1];
        as[i] = q[2 + e];
      }
#pragma unroll
      for (int i = 0; i < kDecBatch; ++i) {
        const float f = __builtin_amdgcn_exp2f(ms[i] - m);
        l = fmaf(ls[i], f, l);
        av = fmaf(as[i], f, av);
      }
    }
  }
  return l > 0.f ? av / l : 0.f;
}

template <int D>
__global__ __launch_bounds__(D) void decode_combine(DecArgs a) {
  const int j = blockIdx.x, b = blockIdx.y, e = threadIdx.x;
  a.out[((int64_t)b * a.HQ + j) * D + e] = combine_elem<D>(a, b, j, e);
}

typedef void (*DecFn)(DecArgs);

template <class T, int D>
DecFn dec_pick(int G) {
  switch (G) {
    case 1: return decode_partial<T, D, 1>;
    case 2: return decode_partial<T, D, 2>;
    case 3: return decode_partial<T, D, 3>;
    case 4: return decode_partial<T, D, 4>;
    case 5: return decode_partial<T, D, 5>;
    case 6: return decode_partial<T, D, 6>;
    case 7: return decode_partial<T, D, 7>;
    default: return decode_partial<T, D, 8>;
  }
}

}  // namespace

// Partial states of the allocation-free entry point: a file-scope device
// array instead of a caller workspace.  Each device the library runs on holds
// its own copy until the process ends; its device address is taken once per
// device (with that device current) and kept, and only that address is
// passed to the kernels.  Every call on a device shares the array, so calls
// that overlap on one device race.  Nothing in it needs clearing: the
// partial kernel writes every chunk state the combine kernel reads.
static __device__ __align__(256) char scratch[kDecodeScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch`, per device
}  // namespace

hipError_t decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

// Row chunk per work-group: enough work-groups to cover the chip (about
// 512 over batch x heads), at least 64 rows each.
DecodePlan decode_plan(const Problem& P, int n_ctx) {
  DecodePlan d;
  const int per = 512 / (P.batch * P.H) > 1 ? 512 / (P.batch * P.H) : 1;
  int chunk = (n_ctx + per - 1) / per;
  chunk = chunk < 64 ? 64 : (chunk + 63) / 64 * 64;
  d.chunk = chunk;
  d.S = (n_ctx + chunk - 1) / chunk;
  d.ws_bytes = (size_t)P.batch * P.HQ * d.S * (P.D + 2) * 4;
  return d;
}

hipError_t run_decode(const Geometry& g, const void* q, const int64_t qs[2], const void* k,
                      const void* v, const int64_t cs[2], int n_ctx, const int32_t* idx, float* out,
                      void* ws, hipStream_t s) {
  const Problem& P = g.p;
  const DecodePlan pl = decode_plan(P, n_ctx);
  DecArgs a;
  a.q = static_cast<const char*>(q);
  a.qs_b = qs[0];
  a.qs_h = qs[1];
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.cs_b = cs[0];
  a.cs_h = cs[1];
  a.idx = idx;
  a.part = static_cast<float*>(ws);
  a.out = out;
  a.H = P.H;
  a.HQ = P.HQ;
  a.B = P.B;
  a.n_ctx = n_ctx;
  a.chunk = pl.chunk;
  a.S = pl.S;
  a.sc = P.sc;
  DecFn fn = P.esize == 2 ? (P.D == 64 ? dec_pick<__bf16, 64>(P.G) : dec_pick<__bf16, 128>(P.G))
                          : (P.D == 64 ? dec_pick<float, 64>(P.G) : dec_pick<float, 128>(P.G));
  hipLaunchKernelGGL(fn, dim3(pl.S, P.H, P.batch), dim3(kDecThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (P.D == 64)
    hipLaunchKernelGGL(decode_combine<64>, dim3(P.HQ, P.batch), dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL(decode_combine<128>, dim3(P.HQ, P.batch), dim3(128), 0, s, a);
  return hipGetLastError();
}

}  // namespace kvec
