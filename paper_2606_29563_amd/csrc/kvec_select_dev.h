// Selection stages of K-VEC (paper Algorithm 1, then the top-B of Sec. 4.1).
//
//   pool      max-pool of P and of the extended-window P along t, the
//             float64 sums of pooled P and its square per block (sigma), and
//             4096-bin histograms of both pooled scores per head.
//   prep      per (sequence, head, token block): sigma of every head and
//             H_top = the delta heads with the lowest sigma (Sec. 4.1); the
//             head's selected score P_sel; then, from the histogram, a
//             coverage-independent superset ("members") of every token that
//             can be preserved or finally kept, in ascending token order.
//   select A  per (layer, sequence, head): the members in ascending order and
//             the preserve set = first K tokens by (P_sel desc, t asc)
//             (Sec. 4.2); needs nothing of the earlier layers.
//   select B  per (layer, sequence, head), run in layer order, one launch
//             after select A: P' = P_sel + lambda * I * (1 - n_t/(l+1)) in
//             fp32 with one rounding per operation and P' = 1 on the preserve
//             set, the first B-O by (P' desc, t asc) emitted in ascending order
//             then the window, and the kept tokens OR-ed into the layer's
//             bitmap row.
//   count     the running coverage counts n_t of the pipeline.
//
// Why the superset is exact: for a non-preserved token, 0 <= bonus <=
// lambda*I, so P_sel <= P' <= U = fl(P_sel + fl(lambda*I)) (fp32 rounding is
// monotone).  The M = B-O tokens with the largest P_sel all have
// P' >= min(P_sel, 1), so the M-th largest P' is >= min(c, 1) where c is the
// M-th largest P_sel; a token with U < min(c, 1) can never be kept.  Every
// token that can be preserved has P_sel >= the K-th largest P_sel.  Both
// thresholds are replaced by the lower edge of the histogram bin holding
// that order statistic, which only enlarges the superset.
#pragma once

#include "kvec_internal.h"

namespace kvec {

__device__ __forceinline__ float key_float(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

// Pointers of one layer for the selection stages.
struct SelectIO {
  const float* psum_base;  // pipeline: score partials [b][n_rt][H][Tc]
  const float* psum_all;
  const float* ipart;      // [b][n_rt][Tc]
  const float* p_raw;      // standalone: raw scores [b][H][Tc] (used when psum_* null)
  const float* p_ext;
  const float* imp_in;     // standalone: [b][Tc]
  float* imp;              // [b][Tc] importance (written by pool in the pipeline)
  float* pooled;           // [b][H][Tc]
  float* pooled_ext;
  double2* stats;          // [b][H][n_pool]
  uint32_t* hist;          // [b][2][H][kHistBins]
  int32_t* mem_t;          // [b][H][Tc] members of each prep chunk at chunk offsets
  float* mem_ps;
  float* mem_i;
  int32_t* mem_n;          // [b][H][n_prep]
  uint32_t* htop_mask;     // nullable [b]
  float* out_p;            // nullable copies of this layer's scores before pooling: P
  float* out_pe;           // [b][H][Tc], P over O' (H_top heads) [b][H][Tc],
  float* out_imp;          // and I [b][Tc]
  uint32_t* spill_keys;    // [b][H][Tc] member arrays when members exceed the LDS capacity
  int32_t* spill_t;
  float* spill_ps;
  float* spill_i;
  const uint8_t* cnt_in;   // [b][T] counts of earlier layers (null: none)
  const uint64_t* bits_prev; // bitmap row of the previous layer, [b] stride L*W (null: none)
  uint64_t* bits;          // [b][L][W] coverage bitmap
  int32_t* idx;            // [b][H][B] of this layer
};

// ---------------------------------------------------------------------------
// pool: grid item (b, h, chunk); 512 threads.  want_p: pool P (with the sigma
// sums, the P histogram and, for head 0, I); want_e: pool P over O' (and its
// histogram).  In the layer pipeline the two run at different times: P first
// (H_top needs its sigma), P over O' once the extended rows of the H_top
// heads are scored.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void task_pool(const Problem& P, const SelectIO& io, int b, int h, int c0,
                                          int c1, char* smem, bool want_p = true,
                                          bool want_e = true) {
  // Wave w pools chunk c0 + w (kPoolChunk tokens, kPoolChunk / 64 per lane,
  // lane-strided so stores coalesce) out of one LDS window holding the whole
  // span with its halo.
  const int r = P.pool / 2;
  const int t0 = c0 * kPoolChunk;
  const int t1 = min(P.Tc, c1 * kPoolChunk);
  const int a0 = max(0, t0 - r), a1 = min(P.Tc, t1 + r);
  float* sp = reinterpret_cast<float*>(smem);        // raw P   [a0, a1)
  float* se = sp + (kPoolPer * kPoolChunk + 64);      // raw P'  [a0, a1)
  uint32_t* hp = reinterpret_cast<uint32_t*>(se + (kPoolPer * kPoolChunk + 64));
  uint32_t* he = hp + kHistBins;
  double2* wst = reinterpret_cast<double2*>(he + kHistBins);  // [kPoolPer] chunk sums
  for (int i = threadIdx.x; i < 2 * kHistBins; i += blockDim.x) hp[i] = 0u;
  const int64_t row = ((int64_t)b * P.H + h) * P.Tc;
  // The window is at most kPoolPer * kPoolChunk + 62 tokens: kSpan loads per
  // thread, unrolled so that every load of the thread is in flight at once.
  constexpr int kSpan = (kPoolPer * kPoolChunk + 64) / kThreads + 1;
  float vp[kSpan], ve[kSpan];
#pragma unroll
  for (int k = 0; k < kSpan; ++k) {
    vp[k] = 0.f;
    ve[k] = 0.f;
  }
  if (io.psum_all) {
    // rows summed in row-tile order, as in the stand-alone finaliser; four
    // row tiles' loads are issued before any of them is used
    const int nrt = want_e ? P.n_rt : P.n_rt_base;
    for (int rt0 = 0; rt0 < nrt; rt0 += 4) {
      float lp[4][kSpan], le[4][kSpan];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rt = rt0 + q;
        const bool add_p = want_p && rt < P.n_rt_base;
        const int64_t o = (((int64_t)b * P.n_rt + rt) * P.H + h) * P.Tc;
#pragma unroll
        for (int k = 0; k < kSpan; ++k) {
          const int t = a0 + (int)threadIdx.x + k * kThreads;
          lp[q][k] = add_p && t < a1 ? io.psum_base[o + t] : 0.f;
          le[q][k] = want_e && rt < nrt && t < a1 ? io.psum_all[o + t] : 0.f;
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < kSpan; ++k) {
          vp[k] += lp[q][k];
          ve[k] += le[q][k];
        }
    }
#pragma unroll
    for (int k = 0; k < kSpan; ++k) {
      vp[k] *= P.inv_go;
      ve[k] *= P.inv_gwn;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kSpan; ++k) {
      const int t = a0 + (int)threadIdx.x + k * kThreads;
      if (t < a1) {
        if (want_p) vp[k] = io.p_raw[row + t];
        if (want_e) ve[k] = io.p_ext[row + t];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kSpan; ++k) {
    const int t = a0 + (int)threadIdx.x + k * kThreads;
    if (t < a1) {
      sp[t - a0] = vp[k];
      se[t - a0] = ve[k];
      // the caller's copy of the scores this work-group owns (no halo)
      if (t >= t0 && t < t1) {
        if (want_p && io.out_p) io.out_p[row + t] = vp[k];
        if (want_e && io.out_pe) io.out_pe[row + t] = ve[k];
      }
    }
  }
  if (want_p && h == 0 && io.psum_all) {
    constexpr int kOwn = kPoolPer * kPoolChunk / kThreads;
    float si[kOwn];
#pragma unroll
    for (int k = 0; k < kOwn; ++k) si[k] = 0.f;
    for (int rt = 0; rt < P.n_rt_base; ++rt) {
#pragma unroll
      for (int k = 0; k < kOwn; ++k) {
        const int t = t0 + (int)threadIdx.x + k * kThreads;
        if (t < t1) si[k] += io.ipart[((int64_t)b * P.n_rt + rt) * P.Tc + t];
      }
    }
#pragma unroll
    for (int k = 0; k < kOwn; ++k) {
      const int t = t0 + (int)threadIdx.x + k * kThreads;
      if (t < t1) {
        io.imp[(int64_t)b * P.Tc + t] = si[k] * P.inv_go;
        if (io.out_imp) io.out_imp[(int64_t)b * P.Tc + t] = si[k] * P.inv_go;
      }
    }
  }
  __syncthreads();
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int chunk = c0 + w;
  if (chunk < c1) {
    const int ct0 = chunk * kPoolChunk, ct1 = min(P.Tc, ct0 + kPoolChunk);
    double s1 = 0.0, s2 = 0.0;
    for (int t = ct0 + lane; t < ct1; t += 64) {
      const int u0 = max(0, t - r), u1 = min(P.Tc - 1, t + r);
      float m = sp[u0 - a0], me = se[u0 - a0];
      for (int u = u0 + 1; u <= u1; ++u) {
        m = fmaxf(m, sp[u - a0]);
        me = fmaxf(me, se[u - a0]);
      }
      if (want_p) {
        io.pooled[row + t] = m;
        s1 += (double)m;
        // sigma: sum of squares; entropy: sum of x ln x (0 ln 0 = 0)
        s2 += P.criterion ? (m > 0.f ? (double)m * log((double)m) : 0.0) : (double)m * (double)m;
        atomicAdd(&hp[float_key(m) >> (32 - kHistBits)], 1u);
      }
      if (want_e) {
        io.pooled_ext[row + t] = me;
        atomicAdd(&he[float_key(me) >> (32 - kHistBits)], 1u);
      }
    }
    if (want_p) {
      s1 = wave_sum(s1);
      s2 = wave_sum(s2);
      if (lane == 0) wst[w] = make_double2(s1, s2);
    }
  }
  __syncthreads();
  if (want_p && threadIdx.x == 0) {
    // one (sum, sum of squares) per work-group: its chunks added in order
    double s1 = 0.0, s2 = 0.0;
    for (int k = 0; k < c1 - c0; ++k) {
      s1 += wst[k].x;
      s2 += wst[k].y;
    }
    io.stats[((int64_t)b * P.H + h) * pool_groups(P) + c0 / kPoolPer] = make_double2(s1, s2);
  }
  uint32_t* gh = io.hist + ((int64_t)b * 2 * P.H) * kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
    if (hp[i]) atomicAdd(&gh[(int64_t)h * kHistBins + i], hp[i]);
    if (he[i]) atomicAdd(&gh[(int64_t)(P.H + h) * kHistBins + i], he[i]);
  }
}

// ---------------------------------------------------------------------------
// prep: grid item (b, h, chunk); 512 threads
// ---------------------------------------------------------------------------
__device__ __forceinline__ void task_prep(const Problem& P, const SelectIO& io, int layer, int b,
                                          int h, int c0, int c1, char* smem) {
  if (h == 0 && c0 == 0) {
    // the selection of this layer ORs its kept tokens into a cleared row
    uint64_t* row = io.bits + ((int64_t)b * P.L + layer) * P.words;
    for (int i = threadIdx.x; i < P.words; i += blockDim.x) row[i] = 0ull;
  }
  int* tmp = reinterpret_cast<int*>(smem);
  // Every load is issued before H_top is known (one memory round trip):
  // both histograms of head h, and both pooled scores and I of this wave's
  // chunk (wave w extracts chunk c0 + w; round k covers tokens
  // [64 k, 64 k + 64) of the chunk, one per lane, so loads coalesce).
  constexpr int per = kHistBins / 512;
  const int tid = threadIdx.x;  // owns bins kHistBins-1-tid*per ... (descending)
  const uint32_t* ghp = io.hist + ((int64_t)b * 2 * P.H + h) * kHistBins;
  const uint32_t* ghe = ghp + (int64_t)P.H * kHistBins;
  int cp[per], ce[per];
#pragma unroll
  for (int e = 0; e < per; ++e) {
    cp[e] = (int)ghp[kHistBins - 1 - (tid * per + e)];
    ce[e] = (int)ghe[kHistBins - 1 - (tid * per + e)];
  }
  static_assert(kPrepChunk == 64 * 16, "one chunk per wave, 16 rounds of 64 tokens");
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int chunk = c0 + w;
  const bool has_chunk = chunk < c1;
  const int t0 = chunk * kPrepChunk;
  const int t1 = min(P.Tc, t0 + kPrepChunk);
  const int64_t hrow = ((int64_t)b * P.H + h) * P.Tc;
  const float* imp = io.imp + (int64_t)b * P.Tc;
  float pp[16], pe[16], im[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int t = has_chunk ? min(t0 + k * 64 + lane, t1 - 1) : 0;
    pp[k] = io.pooled[hrow + t];
    pe[k] = io.pooled_ext[hrow + t];
    im[k] = imp[t];
  }
  const uint32_t top = htop_mask(P, io.stats, b);
  if (h == 0 && c0 == 0 && threadIdx.x == 0 && io.htop_mask) io.htop_mask[b] = top;
  const bool ext = (top >> h) & 1u;
  // Bins holding the Kp-th and the M-th largest key, from one descending
  // prefix sum of the selected histogram.
  int s = 0;
#pragma unroll
  for (int e = 0; e < per; ++e) s += ext ? ce[e] : cp[e];
  if (threadIdx.x == 0) {
    tmp[20] = -1;
    tmp[21] = -1;
  }
  int total;
  const int before = block_excl_scan(s, tmp, total);
  const int ranks[2] = {P.Kp, P.M};
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int k = ranks[q];
    if (k > 0 && before < k && k <= before + s) {
      int run = before, found = -1;
#pragma unroll
      for (int e = 0; e < per; ++e) {
        if (found < 0 && run + (ext ? ce[e] : cp[e]) >= k) found = e;
        run += ext ? ce[e] : cp[e];
      }
      tmp[20 + q] = kHistBins - 1 - (tid * per + found);
    }
  }
  __syncthreads();
  const int bin_kp = tmp[20], bin_m = tmp[21];
  const uint32_t kp_edge = bin_kp < 0 ? 0xffffffffu : (uint32_t)bin_kp << (32 - kHistBits);
  const float c_edge = bin_m < 0 ? INFINITY : key_float((uint32_t)bin_m << (32 - kHistBits));
  const float thr_u = fminf(c_edge, 1.0f);
  const bool has_preserve = bin_kp >= 0;
  if (has_chunk) {
    // members of the chunk in ascending order: round by round, each member's
    // place is the members before it (earlier rounds, then lower lanes)
    const int64_t base = hrow + t0;
    int off = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int t = t0 + k * 64 + lane;
      const float ps = ext ? pe[k] : pp[k];
      const float u = __fadd_rn(ps, __fmul_rn(P.lam, im[k]));
      const bool m = t < t1 && ((has_preserve && float_key(ps) >= kp_edge) || u >= thr_u);
      const uint64_t mask = __ballot(m);
      const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
      if (m) {
        io.mem_t[base + off + before] = t;
        io.mem_ps[base + off + before] = ps;
        io.mem_i[base + off + before] = im[k];
      }
      off += __popcll(mask);
    }
    if (lane == 0) io.mem_n[((int64_t)b * P.H + h) * P.n_prep + chunk] = off;
  }
}

// ---------------------------------------------------------------------------
// select: one work-group per (layer, sequence, head)
// ---------------------------------------------------------------------------

// Block radix select over keys k[0..n) (512 threads): the first `want` keys in
// the order (key desc, index asc) are those > thr plus the first `take` keys
// equal to thr.  Three passes of 11, 11 and 10 bits over an LDS histogram.
__device__ __forceinline__ void block_radix_select(const uint32_t* kb, int n, int want,
                                                   uint32_t* hist, int* tmp, uint32_t& thr,
                                                   int& take) {
  uint32_t prefix = 0, mask = 0;
  int rem = want;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
#pragma unroll
  for (int ps = 0; ps < 3; ++ps) {
    const int shift = shifts[ps], nb = 1 << widths[ps];
    const uint32_t dm = (uint32_t)nb - 1u;
    for (int i = threadIdx.x; i < nb; i += blockDim.x) hist[i] = 0u;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint32_t kk = kb[i];
      if ((kk & mask) == prefix) atomicAdd(&hist[(kk >> shift) & dm], 1u);
    }
    __syncthreads();
    // descending order: thread owns bins nb-1-tid*per .. nb-per-tid*per
    const int per = nb / (int)blockDim.x;
    int cnt[4] = {0, 0, 0, 0}, sum = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (e < per) {
        cnt[e] = (int)hist[nb - 1 - ((int)threadIdx.x * per + e)];
        sum += cnt[e];
      }
    int total;
    const int before = block_excl_scan(sum, tmp, total);
    if (before < rem && rem <= before + sum) {
      int run = before;
      bool found = false;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < per && !found && run + cnt[e] >= rem) {
          tmp[20] = nb - 1 - ((int)threadIdx.x * per + e);
          tmp[21] = rem - run;
          found = true;
        } else if (e < per) {
          run += cnt[e];
        }
    }
    __syncthreads();
    prefix |= (uint32_t)tmp[20] << shift;
    mask |= dm << shift;
    rem = tmp[21];
    __syncthreads();
  }
  thr = prefix;
  take = rem;
}

// Flags of the first `want` members (given thr/take from the radix select),
// in member order, by a blocked prefix count of the keys equal to thr.
// Calls fn(i, selected) for every member i of this thread's block range.
template <class Fn>
__device__ __forceinline__ void block_flags(const uint32_t* kb, int n, int want, uint32_t thr,
                                            int take, int* tmp, Fn fn) {
  const int per = (n + blockDim.x - 1) / blockDim.x;
  const int lo = min(n, (int)threadIdx.x * per), hi = min(n, lo + per);
  int ceq = 0;
  for (int i = lo; i < hi; ++i) ceq += kb[i] == thr;
  int total;
  int e = block_excl_scan(ceq, tmp, total);
  for (int i = lo; i < hi; ++i) {
    const uint32_t kk = kb[i];
    bool sel;
    if (want >= n) {
      sel = true;
    } else if (want <= 0) {
      sel = false;
    } else {
      sel = kk > thr || (kk == thr && e < take);
      e += kk == thr;
    }
    fn(i, sel);
  }
}

// The selection of a layer runs as two tasks one launch apart, both one
// work-group per (sequence, head).  Only the second needs the previous
// layer's bitmap row (n_t), so the first runs while that row is still being
// written, which halves the serial chain from layer to layer.
//
// select A: gathers the head's candidate members (contiguous, ascending t),
// takes the preserve set (first Kp by P_sel desc, t asc) and writes the
// members back compacted into the head's member arrays: t (bitwise
// complemented for preserved members), P_sel, I; their count goes to
// mem_n[.][h][0].
__device__ __forceinline__ void task_select_a(const Problem& P, const SelectIO& io, int b, int h,
                                              char* smem) {
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem);    // [2048]
  int* tmp = reinterpret_cast<int*>(hist + 2048);          // [32]
  int* off = tmp + 32;                                     // [n_prep + 1] member offsets
  char* marr = reinterpret_cast<char*>(off + ((P.n_prep + 1 + 3) & ~3));
  const int64_t hb = (int64_t)b * P.H + h;
  int32_t* mn = io.mem_n + hb * P.n_prep;
  // member offsets of the prep chunks (wave 0, 64 chunks per round)
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int carry = 0;
    for (int c0 = 0; c0 < P.n_prep; c0 += 64) {
      const int c = c0 + lane;
      const int v = c < P.n_prep ? mn[c] : 0;
      const int incl = wave_incl_scan(v);
      if (c < P.n_prep) off[c] = carry + incl - v;
      carry += __shfl(incl, 63);
    }
    if (lane == 0) off[P.n_prep] = carry;
  }
  __syncthreads();
  const int n = off[P.n_prep];
  uint32_t* kb;
  int32_t* mt;
  float *mp, *mi;
  if (n <= P.mcap) {
    kb = reinterpret_cast<uint32_t*>(marr);
    mt = reinterpret_cast<int32_t*>(kb + P.mcap);
    mp = reinterpret_cast<float*>(mt + P.mcap);
    mi = mp + P.mcap;
  } else {
    kb = io.spill_keys + hb * P.Tc;
    mt = io.spill_t + hb * P.Tc;
    mp = io.spill_ps + hb * P.Tc;
    mi = io.spill_i + hb * P.Tc;
  }
  // gather the members contiguously (ascending t), with their preserve keys;
  // kBatch members per thread have their loads in flight together
  constexpr int kBatch = 8;
  int32_t* gt = io.mem_t + hb * P.Tc;
  float* gp = io.mem_ps + hb * P.Tc;
  float* gi = io.mem_i + hb * P.Tc;
  for (int i0 = threadIdx.x; i0 < n; i0 += kBatch * blockDim.x) {
    int g[kBatch];  // member position in the head's chunk arrays
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = i0 + u * (int)blockDim.x;
      int lo = 0, hi = P.n_prep - 1;  // chunk c with off[c] <= i < off[c+1]
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (off[mid] <= i) lo = mid; else hi = mid - 1;
      }
      g[u] = lo * kPrepChunk + (i - off[lo]);
    }
    int32_t vt[kBatch];
    float vp[kBatch], vi[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool ok = i0 + u * (int)blockDim.x < n;
      vt[u] = ok ? gt[g[u]] : 0;
      vp[u] = ok ? gp[g[u]] : 0.f;
      vi[u] = ok ? gi[g[u]] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int i = i0 + u * (int)blockDim.x;
      if (i < n) {
        mt[i] = vt[u];
        mp[i] = vp[u];
        mi[i] = vi[u];
        kb[i] = float_key(vp[u]);
      }
    }
  }
  __syncthreads();
  // preserve set: first Kp members by (P_sel desc, t asc)
  const int kp = min(P.Kp, n);
  uint32_t thr_p = 0xffffffffu;
  int take_p = 0;
  if (kp > 0 && kp < n) block_radix_select(kb, n, kp, hist, tmp, thr_p, take_p);
  // write the members back compacted (every chunk-layout read is done: the
  // gather ended with a barrier), preserved ones marked by ~t
  block_flags(kb, n, kp, thr_p, take_p, tmp, [&](int i, bool pres) {
    gt[i] = pres ? ~mt[i] : mt[i];
    gp[i] = mp[i];
    gi[i] = mi[i];
  });
  if (threadIdx.x == 0) mn[0] = n;
}

// select B: the coverage-aware priority P' of every member (1.0 on the
// preserve set, else P_sel + lambda * I * (1 - n_t/(l+1)) in fp32 op by op),
// the final pick of the first B-O by (P' desc, t asc), its emission in
// ascending order with the window, and the layer's bitmap row.
__device__ __forceinline__ void task_select_b(const Problem& P, const SelectIO& io, int layer, int b,
                                              int h, char* smem) {
  uint32_t* hist = reinterpret_cast<uint32_t*>(smem);    // [2048]
  int* tmp = reinterpret_cast<int*>(hist + 2048);          // [32]
  char* marr = reinterpret_cast<char*>(tmp + 32 + ((P.n_prep + 1 + 3) & ~3));
  const int64_t hb = (int64_t)b * P.H + h;
  const int n = io.mem_n[hb * P.n_prep];
  const int32_t* gt = io.mem_t + hb * P.Tc;
  const float* gp = io.mem_ps + hb * P.Tc;
  const float* gi = io.mem_i + hb * P.Tc;
  uint32_t* kb;
  const int32_t* mt;
  const float *mp, *mi;
  if (n <= P.mcap) {
    kb = reinterpret_cast<uint32_t*>(marr);
    int32_t* lt = reinterpret_cast<int32_t*>(kb + P.mcap);
    float* lp = reinterpret_cast<float*>(lt + P.mcap);
    float* li = lp + P.mcap;
    // members into LDS, kBatch loads per thread in flight together
    constexpr int kBatch = 8;
    for (int i0 = threadIdx.x; i0 < n; i0 += kBatch * blockDim.x) {
      int32_t vt[kBatch];
      float vp[kBatch], vi[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = min(i0 + u * (int)blockDim.x, n - 1);
        vt[u] = gt[i];
        vp[u] = gp[i];
        vi[u] = gi[i];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u * (int)blockDim.x;
        if (i < n) {
          lt[i] = vt[u];
          lp[i] = vp[u];
          li[i] = vi[u];
        }
      }
    }
    __syncthreads();
    mt = lt;
    mp = lp;
    mi = li;
  } else {
    // long member lists stay in global memory; the keys go to this layer's
    // pooled-score array, free once the candidates were extracted
    kb = reinterpret_cast<uint32_t*>(io.pooled) + hb * P.Tc;
    mt = gt;
    mp = gp;
    mi = gi;
  }
  // P' keys: 1.0 on the preserve set, else P_sel + lambda * I * (1 - n_t/(l+1))
  const float f_denom = (float)(layer + 1);
  const uint8_t* cnt = io.cnt_in;
  const uint64_t* prow = io.bits_prev;
  {
    const int per = (n + blockDim.x - 1) / blockDim.x;
    const int lo = min(n, (int)threadIdx.x * per), hi = min(n, lo + per);
    for (int i = lo; i < hi; ++i) {
      const int te = mt[i];
      float pp;
      if (te < 0) {
        pp = 1.0f;
      } else {
        const int t = te;
        int nt = cnt ? (int)cnt[(int64_t)b * P.T + t] : 0;
        if (prow) nt += (int)((prow[(int64_t)b * P.L * P.words + (t >> 6)] >> (t & 63)) & 1ull);
        const float cov = __fdiv_rn((float)nt, f_denom);
        const float focus = __fmul_rn(mi[i], __fsub_rn(1.0f, cov));
        pp = __fadd_rn(mp[i], __fmul_rn(P.lam, focus));
      }
      kb[i] = float_key(pp);
    }
  }
  __syncthreads();
  // final pick: first M members by (P' desc, t asc), emitted in ascending order
  const int m = min(P.M, n);
  uint32_t thr = 0xffffffffu;
  int take = 0;
  if (m > 0 && m < n) block_radix_select(kb, n, m, hist, tmp, thr, take);
  // output positions: blocked count of the selected members, then emission
  const int per = (n + blockDim.x - 1) / blockDim.x;
  const int lo = min(n, (int)threadIdx.x * per), hi = min(n, lo + per);
  int ceq = 0;
  for (int i = lo; i < hi; ++i) ceq += kb[i] == thr;
  int total;
  const int e0 = block_excl_scan(ceq, tmp, total);
  auto selected = [&](uint32_t kk, int& e) {
    if (m >= n) return true;
    if (m <= 0) return false;
    const bool eq = kk == thr;
    const bool sel = kk > thr || (eq && e < take);
    e += eq;
    return sel;
  };
  int csel = 0;
  {
    int e = e0;
    for (int i = lo; i < hi; ++i) csel += selected(kb[i], e);
  }
  int o = block_excl_scan(csel, tmp, total);
  int32_t* out = io.idx + hb * P.B;
  uint64_t* row = io.bits + ((int64_t)b * P.L + layer) * P.words;
  uint64_t word = 0;
  int cur = -1;
  {
    int e = e0;
    for (int i = lo; i < hi; ++i) {
      if (!selected(kb[i], e)) continue;
      const int te = mt[i];
      const int t = te < 0 ? ~te : te;
      out[o++] = t;
      if ((t >> 6) != cur) {
        if (cur >= 0) atomicOr((unsigned long long*)&row[cur], (unsigned long long)word);
        cur = t >> 6;
        word = 0;
      }
      word |= 1ull << (t & 63);
    }
  }
  if (cur >= 0) atomicOr((unsigned long long*)&row[cur], (unsigned long long)word);
  for (int i = threadIdx.x; i < P.O; i += blockDim.x) out[P.M + i] = P.Tc + i;
  if (h == 0) {
    // the observation window is always kept
    for (int t = P.Tc + threadIdx.x; t < P.T; t += blockDim.x)
      atomicOr((unsigned long long*)&row[t >> 6], 1ull << (t & 63));
  }
}

// Running coverage counts of the pipeline: n_t(layer) = n_t(layer-1) + kept
// bit of layer-1, into the buffer of this layer's parity (the next layer's
// selection adds this layer's bitmap row itself).  Part `part` of kCountWords
// bitmap words.
constexpr int kCountWords = 64;

__device__ __forceinline__ void task_count(const Problem& P, const uint8_t* cnt_prev,
                                           const uint64_t* row_prev, uint8_t* cnt_out, int b,
                                           int part) {
  const int w0 = part * kCountWords;
  for (int i = threadIdx.x; i < kCountWords * 64; i += blockDim.x) {
    const int wi = w0 + i / 64, t = wi * 64 + (i & 63);
    if (wi >= P.words || t >= P.T) continue;
    int v = 0;
    if (cnt_prev) v = (int)cnt_prev[(int64_t)b * P.T + t];
    if (row_prev) v += (int)((row_prev[(int64_t)b * P.L * P.words + wi] >> (t & 63)) & 1ull);
    cnt_out[(int64_t)b * P.T + t] = (uint8_t)v;
  }
}

// n_t for a standalone layer call: counts of the caller's bitmap rows < layer.
__device__ __forceinline__ void task_counts_from_bits(const Problem& P, const uint64_t* bits,
                                                      uint8_t* counts, int layer, int b, int wi) {
  const int tlo = wi * 64;
  for (int t = tlo + (int)threadIdx.x; t < min(tlo + 64, P.T); t += blockDim.x) {
    int nt = 0;
    for (int l = 0; l < layer; ++l)
      nt += (int)((bits[((int64_t)b * P.L + l) * P.words + wi] >> (t - tlo)) & 1ull);
    counts[(int64_t)b * P.T + t] = (uint8_t)nt;
  }
}

}  // namespace kvec
