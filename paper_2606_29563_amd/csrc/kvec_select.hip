// Selection of one layer (paper Algorithm 1, then the top-B of Sec. 4.1):
//
//   pool_stats    max-pool of P and of the extended-window P along t, and the
//                 per-block float64 sums of pooled P and its square (for sigma).
//   htop_keep     per (sequence, head): sigma of every head, H_top = the delta
//                 heads with the lowest sigma (Sec. 4.1), the head's selected
//                 score P_sel (extended-window score if in H_top), and the
//                 preserve set = its first K tokens by (P_sel desc, t asc)
//                 (Sec. 4.2).
//   final_select  per (sequence, head): n_t from the coverage bitmap of the
//                 earlier layers, P' = P_sel + lambda * I * (1 - n_t/(l+1))
//                 in fp32 (one rounding per operation), P' = 1 on the preserve
//                 set, the first B-O tokens by (P' desc, t asc) emitted in
//                 ascending order followed by the window, and the layer's
//                 bitmap row (atomic OR over heads).
//
// Top-k is an exact most-significant-digit radix select over order-preserving
// 32-bit keys of the fp32 scores (4 passes of 8 bits with an LDS histogram),
// which yields the k-th key; ties at that key are then taken in index order
// by a blocked prefix scan, so the result is the unique first-k set.
#include "kvec_internal.h"

namespace kvec {
namespace {

struct SelectShared {
  uint32_t hist[256];
  int misc[4];
  int scan[17];
};

// k-th largest key (1 <= k <= n) and how many keys equal to it are taken.
template <class KeyFn>
__device__ void radix_select(KeyFn key, int n, int k, uint32_t& thr, int& take, SelectShared& sh) {
  uint32_t prefix = 0, mask = 0;
  int rem = k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) sh.hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint32_t kk = key(i);
      if ((kk & mask) == prefix) atomicAdd(&sh.hist[(kk >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      int cnt[4], s = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cnt[e] = (int)sh.hist[255 - 4 * lane - e];
        s += cnt[e];
      }
      const int incl = wave_incl_scan(s);
      const int excl = incl - s;
      if (excl < rem && rem <= incl) {
        int run = excl;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (run + cnt[e] >= rem) {
            sh.misc[0] = 255 - 4 * lane - e;
            sh.misc[1] = rem - run;
            break;
          }
          run += cnt[e];
        }
      }
    }
    __syncthreads();
    const uint32_t digit = (uint32_t)sh.misc[0];
    rem = sh.misc[1];
    prefix |= digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  thr = prefix;
  take = rem;
}

// Enumerate the first k of n tokens by (key desc, index asc) in ascending token
// order: emit(t, rank_in_output).  Threads own contiguous, `align`-aligned
// ranges of tokens; emit_word(first_t) is called once per owned range chunk
// boundary through `flush` so callers can pack bits per word.
template <class KeyFn, class Emit>
__device__ void select_first_k(KeyFn key, int n, int k, int align, Emit emit, SelectShared& sh) {
  uint32_t thr = 0;
  int take = 0;
  const bool all = k >= n;
  if (k <= 0) return;
  if (!all) radix_select(key, n, k, thr, take, sh);
  const int per0 = (n + blockDim.x - 1) / blockDim.x;
  const int per = (per0 + align - 1) / align * align;
  const int lo = min(n, (int)threadIdx.x * per), hi = min(n, lo + per);
  int c_eq = 0;
  if (!all)
    for (int t = lo; t < hi; ++t) c_eq += key(t) == thr;
  int total;
  int eq_before = block_excl_scan(c_eq, sh.scan, total);
  int c_sel = 0;
  {
    int e = eq_before;
    for (int t = lo; t < hi; ++t) {
      bool sel = all;
      if (!all) {
        const uint32_t kk = key(t);
        sel = kk > thr || (kk == thr && e < take);
        e += kk == thr;
      }
      c_sel += sel;
    }
  }
  int o = block_excl_scan(c_sel, sh.scan, total);
  int e = eq_before;
  for (int t = lo; t < hi; ++t) {
    bool sel = all;
    if (!all) {
      const uint32_t kk = key(t);
      sel = kk > thr || (kk == thr && e < take);
      e += kk == thr;
    }
    if (sel) emit(t, o++);
  }
}

__global__ void pool_stats_kernel(const float* __restrict__ p_raw, const float* __restrict__ p_ext,
                                  float* __restrict__ pooled, float* __restrict__ pooled_ext,
                                  double2* __restrict__ stats, int H, int Tc, int pool, int n_blk) {
  __shared__ double red[2][8];
  const int b = blockIdx.z, h = blockIdx.y;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = ((int64_t)b * H + h) * Tc;
  double x = 0.0;
  if (t < Tc) {
    const int r = pool / 2;
    const int u0 = max(0, t - r), u1 = min(Tc - 1, t + r);
    float m = p_raw[row + u0], me = p_ext[row + u0];
    for (int u = u0 + 1; u <= u1; ++u) {
      m = fmaxf(m, p_raw[row + u]);
      me = fmaxf(me, p_ext[row + u]);
    }
    pooled[row + t] = m;
    pooled_ext[row + t] = me;
    x = (double)m;
  }
  double s1 = wave_sum(x), s2 = wave_sum(x * x);
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) {
    red[0][wid] = s1;
    red[1][wid] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double a1 = 0.0, a2 = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      a1 += red[0][w];
      a2 += red[1][w];
    }
    stats[((int64_t)b * H + h) * n_blk + blockIdx.x] = make_double2(a1, a2);
  }
}

struct HtopArgs {
  const float* pooled;
  const float* pooled_ext;
  const double2* stats;
  int32_t* use_ext;
  uint32_t* keep;
  uint32_t* htop_mask;
  int H, Tc, n_blk, delta, Kp, keep_words;
};

__global__ __launch_bounds__(kSelectThreads) void htop_keep_kernel(HtopArgs a) {
  __shared__ SelectShared sh;
  __shared__ double var[16];
  __shared__ int in_top[16];
  const int h = blockIdx.x, b = blockIdx.y;
  if ((int)threadIdx.x < a.H) {
    const int g = threadIdx.x;
    double s1 = 0.0, s2 = 0.0;
    for (int i = 0; i < a.n_blk; ++i) {
      const double2 v = a.stats[((int64_t)b * a.H + g) * a.n_blk + i];
      s1 += v.x;
      s2 += v.y;
    }
    const double mean = s1 / a.Tc;
    var[g] = s2 / a.Tc - mean * mean;
  }
  __syncthreads();
  if ((int)threadIdx.x < a.H) {
    const int g = threadIdx.x;
    int rank = 0;
    for (int o = 0; o < a.H; ++o) rank += (var[o] < var[g]) || (var[o] == var[g] && o < g);
    in_top[g] = rank < a.delta;
  }
  __syncthreads();
  if (h == 0 && threadIdx.x == 0 && a.htop_mask) {
    uint32_t m = 0;
    for (int g = 0; g < a.H; ++g) m |= (uint32_t)in_top[g] << g;
    a.htop_mask[b] = m;
  }
  const bool ext = in_top[h] != 0;
  if (threadIdx.x == 0) a.use_ext[b * a.H + h] = ext;
  const float* src = (ext ? a.pooled_ext : a.pooled) + ((int64_t)b * a.H + h) * a.Tc;
  uint32_t* keep = a.keep + ((int64_t)b * a.H + h) * a.keep_words;
  // Owned word range of this thread (32-token aligned ranges).
  const int per0 = (a.Tc + blockDim.x - 1) / blockDim.x;
  const int per = (per0 + 31) / 32 * 32;
  const int w_lo = min(a.keep_words, (int)threadIdx.x * per / 32);
  const int w_hi = min(a.keep_words, w_lo + per / 32);
  for (int w = w_lo; w < w_hi; ++w) keep[w] = 0u;
  __syncthreads();
  auto key = [&](int t) { return float_key(src[t]); };
  // Words are owned by exactly one thread, so plain read-modify-write is safe.
  select_first_k(key, a.Tc, a.Kp, 32, [&](int t, int) { keep[t >> 5] |= 1u << (t & 31); }, sh);
}

struct FinalArgs {
  const float* pooled;
  const float* pooled_ext;
  const float* imp;
  const int32_t* use_ext;
  const uint32_t* keep;
  uint32_t* keys;
  uint64_t* bits;
  int32_t* idx;
  int H, Tc, T, O, B, M, L, W, layer, keep_words;
  float lam;
};

__global__ __launch_bounds__(kSelectThreads) void final_select_kernel(FinalArgs a) {
  __shared__ SelectShared sh;
  const int h = blockIdx.x, b = blockIdx.y;
  const bool ext = a.use_ext[b * a.H + h] != 0;
  const float* src = (ext ? a.pooled_ext : a.pooled) + ((int64_t)b * a.H + h) * a.Tc;
  const float* imp = a.imp + (int64_t)b * a.Tc;
  const uint32_t* keep = a.keep + ((int64_t)b * a.H + h) * a.keep_words;
  uint32_t* keys = a.keys + ((int64_t)b * a.H + h) * a.Tc;
  const uint64_t* lbits = a.bits + (int64_t)b * a.L * a.W;
  const float denom = (float)(a.layer + 1);

  // P' keys, 64-token words per thread; n_t by bit-sliced counting over the
  // earlier layers' bitmap rows (8 bit-planes: counts up to 255 layers).
  const int per0 = (a.Tc + blockDim.x - 1) / blockDim.x;
  const int per = (per0 + 63) / 64 * 64;
  const int lo = min(a.Tc, (int)threadIdx.x * per), hi = min(a.Tc, lo + per);
  for (int w0 = lo; w0 < hi; w0 += 64) {
    const int wi = w0 >> 6;
    uint64_t plane[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int l = 0; l < a.layer; ++l) {
      uint64_t carry = lbits[(int64_t)l * a.W + wi];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const uint64_t tmp = plane[p] & carry;
        plane[p] ^= carry;
        carry = tmp;
      }
    }
    const int wend = min(hi, w0 + 64);
    for (int t = w0; t < wend; ++t) {
      const int bit = t & 63;
      int nt = 0;
#pragma unroll
      for (int p = 0; p < 8; ++p) nt |= (int)((plane[p] >> bit) & 1u) << p;
      float pp;
      if ((keep[t >> 5] >> (t & 31)) & 1u) {
        pp = 1.0f;
      } else {
        const float cov = __fdiv_rn((float)nt, denom);
        const float focus = __fmul_rn(imp[t], __fsub_rn(1.0f, cov));
        pp = __fadd_rn(src[t], __fmul_rn(a.lam, focus));
      }
      keys[t] = float_key(pp);
    }
  }
  __syncthreads();

  int32_t* out = a.idx + ((int64_t)b * a.H + h) * a.B;
  uint64_t* row = a.bits + ((int64_t)b * a.L + a.layer) * a.W;
  // Ranges are 64-token aligned, so each thread packs whole bitmap words.
  uint64_t word = 0;
  int cur = -1;
  auto key = [&](int t) { return keys[t]; };
  select_first_k(key, a.Tc, a.M, 64,
                 [&](int t, int o) {
                   out[o] = t;
                   const int wi = t >> 6;
                   if (wi != cur) {
                     if (cur >= 0 && word) atomicOr((unsigned long long*)&row[cur], (unsigned long long)word);
                     cur = wi;
                     word = 0;
                   }
                   word |= 1ull << (t & 63);
                 },
                 sh);
  if (cur >= 0 && word) atomicOr((unsigned long long*)&row[cur], (unsigned long long)word);
  // The observation window is always kept.
  for (int w = threadIdx.x; w < a.O; w += blockDim.x) out[a.M + w] = a.Tc + w;
  if (h == 0) {
    for (int t = a.Tc + threadIdx.x; t < a.T; t += blockDim.x)
      atomicOr((unsigned long long*)&row[t >> 6], 1ull << (t & 63));
  }
}

// T <= B: every token is kept.
__global__ void keep_all_kernel(int32_t* idx, uint64_t* bits, int H, int B, int T, int L, int W,
                                int layer) {
  const int b = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < H * B) idx[(int64_t)b * H * B + i] = (i % B) < T ? (i % B) : -1;
  if (i < W) {
    const int t0 = i * 64;
    const int nb = min(64, T - t0);
    bits[((int64_t)b * L + layer) * W + i] = nb >= 64 ? ~0ull : ((1ull << nb) - 1ull);
  }
}

__global__ void coverage_kernel(const uint64_t* bits, int64_t* count, int L, int W, int upto) {
  __shared__ int64_t red[16];
  const int b = blockIdx.x;
  int64_t c = 0;
  for (int w = threadIdx.x; w < W; w += blockDim.x) {
    uint64_t u = 0;
    for (int l = 0; l <= upto; ++l) u |= bits[((int64_t)b * L + l) * W + w];
    c += __popcll(u);
  }
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t s = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
    count[b] = s;
  }
}

__global__ void zero_words_kernel(uint64_t* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

}  // namespace

hipError_t launch_select(const Geometry& g, int layer, const float* p_raw, const float* p_ext,
                         const float* imp, uint64_t* bits, int32_t* idx, uint32_t* htop_mask,
                         char* ws, const Workspace& w, hipStream_t s) {
  float* pooled = reinterpret_cast<float*>(ws + w.pooled);
  float* pooled_ext = reinterpret_cast<float*>(ws + w.pooled_ext);
  double2* stats = reinterpret_cast<double2*>(ws + w.stats);
  hipLaunchKernelGGL(pool_stats_kernel, dim3(g.n_pool_blk, g.H, g.batch), dim3(kPoolBlock), 0, s,
                     p_raw, p_ext, pooled, pooled_ext, stats, g.H, g.Tc, g.pool, g.n_pool_blk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  HtopArgs ha;
  ha.pooled = pooled;
  ha.pooled_ext = pooled_ext;
  ha.stats = stats;
  ha.use_ext = reinterpret_cast<int32_t*>(ws + w.use_ext);
  ha.keep = reinterpret_cast<uint32_t*>(ws + w.keep);
  ha.htop_mask = htop_mask;
  ha.H = g.H;
  ha.Tc = g.Tc;
  ha.n_blk = g.n_pool_blk;
  ha.delta = (g.Wn > g.O) ? min(g.delta, g.H) : 0;
  ha.Kp = g.Kp;
  ha.keep_words = (g.Tc + 31) / 32;
  hipLaunchKernelGGL(htop_keep_kernel, dim3(g.H, g.batch), dim3(kSelectThreads), 0, s, ha);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  FinalArgs fa;
  fa.pooled = pooled;
  fa.pooled_ext = pooled_ext;
  fa.imp = imp;
  fa.use_ext = ha.use_ext;
  fa.keep = ha.keep;
  fa.keys = reinterpret_cast<uint32_t*>(ws + w.keys);
  fa.bits = bits;
  fa.idx = idx;
  fa.H = g.H;
  fa.Tc = g.Tc;
  fa.T = g.T;
  fa.O = g.O;
  fa.B = g.B;
  fa.M = g.M;
  fa.L = g.layers;
  fa.W = g.words;
  fa.layer = layer;
  fa.keep_words = ha.keep_words;
  fa.lam = g.lam;
  hipLaunchKernelGGL(final_select_kernel, dim3(g.H, g.batch), dim3(kSelectThreads), 0, s, fa);
  return hipGetLastError();
}

hipError_t launch_keep_all(const Geometry& g, int layer, uint64_t* bits, int32_t* idx, hipStream_t s) {
  const int n = max(g.H * g.B, g.words);
  hipLaunchKernelGGL(keep_all_kernel, dim3((n + 255) / 256, g.batch), dim3(256), 0, s, idx, bits,
                     g.H, g.B, g.T, g.layers, g.words, layer);
  return hipGetLastError();
}

hipError_t launch_coverage(const Geometry& g, const uint64_t* bits, int upto, int64_t* count,
                           hipStream_t s) {
  hipLaunchKernelGGL(coverage_kernel, dim3(g.batch), dim3(256), 0, s, bits, count, g.layers,
                     g.words, upto);
  return hipGetLastError();
}

hipError_t launch_zero_bits(const Geometry& g, uint64_t* bits, hipStream_t s) {
  const int64_t n = (int64_t)g.batch * g.layers * g.words;
  hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, bits, n);
  return hipGetLastError();
}

}  // namespace kvec
