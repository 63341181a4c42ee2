// The eviction step as a software pipeline of fused launches.
//
// Every stage of one layer depends only on earlier stages of the same layer,
// except the coverage-aware selection, which also needs the previous layer's
// selection (its bitmap row defines n_t).  The window rows split in two: the
// last-O rows (P and I, every head) and the rest of the extended window (P
// over O', needed only for the H_top heads, which are known once P is pooled).
// Launch j of the step therefore runs, side by side in one grid of 512-thread
// work-groups:
//
//   select B layer j-10  (one work-group per (sequence, head); the serial chain)
//   count    layer j-10  (running coverage counts for the next selection)
//   select A layer j-9   (members and preserve set; no earlier layer needed)
//   pass 2   layer j-2   last-O rows, every head: P, I
//   pass 2   layer j-6   extended rows, H_top heads: the rest of P over O'
//   pass 1   layer j     last-O rows: row-normaliser partials
//   pass 1   layer j-4   extended rows of the H_top heads
//   lse      layers j-1, j-5 (row normalisers of the two row sets)
//   pool     layer j-3   P: max-pool, sigma sums, histogram, I
//   pool     layer j-7   P over O' of the H_top heads
//   prep     layer j-8   (sigma, H_top, candidate members)
//   gather   layer j-11  (compacted cache)
//
// so L + 11 launches cover the whole step and the serial selection chain
// runs in the shadow of the score passes.  Per-layer scratch lives in a ring
// of kRing slots.
//
// When the caller supplies the window rows' normalisers (the log-sum-exp its
// prefill attention already computed for those query rows), pass 1 and the
// lse stages drop out and the step takes L + 7 launches: pass 2 of the
// last-O rows at j, their pool at j-1, pass 2 of the extended rows at j-2,
// their pool at j-3, prep at j-4, select A at j-5, select B and count at
// j-6, gather at j-7.
//
// Work-group IDs are dispatched round-robin over the 8 XCDs, each with its
// own L2.  Within a stage, consecutive tasks (e.g. the row tiles of one key
// tile, which read the same K rows) are mapped to work-groups on the same
// XCD so that K is fetched once per XCD L2.
#include <string.h>

#include "kvec_step.h"

namespace kvec {
namespace {

using namespace step;

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void counts_kernel(Problem P, const uint64_t* bits, uint8_t* counts, int layer) {
  task_counts_from_bits(P, bits, counts, layer, blockIdx.y, blockIdx.x);
}

// P, P over O', I of one layer from the score partials (fixed order).
__global__ void finalize_kernel(Problem P, const float* psum_base, const float* psum_all,
                                const float* ipart, float* p_raw, float* p_ext, float* imp) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int y = blockIdx.y, b = blockIdx.z;
  if (t >= P.Tc) return;
  if (y < P.H) {
    float sb = 0.f, sa = 0.f;
    for (int rt = 0; rt < P.n_rt; ++rt) {
      const int64_t o = (((int64_t)b * P.n_rt + rt) * P.H + y) * P.Tc + t;
      if (rt < P.n_rt_base) sb += psum_base[o];
      sa += psum_all[o];
    }
    p_raw[((int64_t)b * P.H + y) * P.Tc + t] = sb * P.inv_go;
    p_ext[((int64_t)b * P.H + y) * P.Tc + t] = sa * P.inv_gwn;
  } else {
    float s = 0.f;
    for (int rt = 0; rt < P.n_rt_base; ++rt) s += ipart[((int64_t)b * P.n_rt + rt) * P.Tc + t];
    imp[(int64_t)b * P.Tc + t] = s * P.inv_go;
  }
}

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

// Work-groups of an EXT pass over n_kt key tiles: its (sequence, key tile,
// H_top head, row tile) tasks packed eight to a work-group, one per wave.
int ext_wgs(const Problem& P, int n_kt) {
  return P.n_rt_x ? (int)(((int64_t)P.batch * n_kt * P.delta_eff * P.n_rt_x + 7) / 8) : 0;
}

int seg_count(const Problem& P, int st) {
  const bool ext = P.delta_eff > 0;
  switch (st) {
    case ST_SELECT:
    case ST_SELA: return P.batch * P.H;
    case ST_COUNT: return P.batch * ((P.words + kCountWords - 1) / kCountWords);
    case ST_PASS1: return P.batch * P.n_kt1 * P.n_rtg;
    case ST_P1B: return P.batch * P.n_kt1 * P.n_rtg_base;
    case ST_P1X: return ext_wgs(P, P.n_kt1);
    case ST_LSE:
    case ST_LSEB: return P.batch * lse_tasks_per_seq(P, st);
    case ST_LSEX: return P.n_rt_x ? P.batch * lse_tasks_per_seq(P, st) : 0;
    case ST_PASS2: return P.batch * P.n_kt2 * P.n_rtg;
    case ST_P2B: return P.batch * P.n_kt2 * P.n_rtg_base;
    case ST_P2X: return ext_wgs(P, P.n_kt2);
    case ST_POOL:
    case ST_POOLB: return P.batch * P.H * ((P.n_pool + kPoolPer - 1) / kPoolPer);
    case ST_POOLX: return ext ? P.batch * P.delta_eff * ((P.n_pool + kPoolPer - 1) / kPoolPer) : 0;
    case ST_PREP: return P.batch * P.H * ((P.n_prep + kPrepPer - 1) / kPrepPer);
    case ST_GATHER: return P.batch * P.n_gather;
  }
  return 0;
}

StepFn pick(const Problem& P) {
  if (P.esize == 2) return P.D == 64 ? pick_g<BF16, 64>(P.G) : pick_g<BF16, 128>(P.G);
  return P.D == 64 ? pick_g<F32, 64>(P.G) : pick_g<F32, 128>(P.G);
}

StepArgs base_args(const Geometry& g, char* ws, const Workspace& w) {
  StepArgs a;
  memset(&a, 0, sizeof(a));
  a.P = g.p;
  a.w = w;
  a.ws = ws;
  for (int s = 0; s < ST_N; ++s) a.seg[s] = Seg{-1, 0, 0, 0};
  return a;
}

void set_model(StepArgs& a, const ModelIO& m) {
  a.q = static_cast<const char*>(m.q);
  a.k = static_cast<const char*>(m.k);
  a.v = static_cast<const char*>(m.v);
  for (int i = 0; i < 4; ++i) {
    a.qs[i] = m.qs[i];
    a.ks[i] = m.ks[i];
    a.vs[i] = m.vs[i];
  }
  a.lse = m.lse;
  for (int i = 0; i < 3; ++i) a.ls[i] = m.ls[i];
  a.bits = m.bits;
  a.idx = m.idx;
  a.k_out = static_cast<char*>(m.k_out);
  a.v_out = static_cast<char*>(m.v_out);
  a.sc_p = m.sc_p;
  a.sc_pe = m.sc_pe;
  a.sc_imp = m.sc_imp;
  a.sc_htop = m.sc_htop;
  a.q_step = m.q_step;
  a.k_step = m.k_step;
  a.v_step = m.v_step;
  a.lse_step = m.lse_step;
  a.bits_step = m.bits_step;
  a.idx_step = m.idx_step;
  a.out_step = m.out_step;
}

hipError_t launch(const StepArgs& a, const Workspace& w, hipStream_t s) {
  int total = 0;
  for (int st = 0; st < ST_N; ++st) total += (a.seg[st].count + 7) & ~7;
  if (total == 0) return hipSuccess;
  StepFn fn = pick(a.P);
  static_assert(sizeof(StepArgs) < 4096, "kernel argument block too large");
  hipLaunchKernelGGL(fn, dim3(total), dim3(kThreads), w.lds_bytes, s, a);
  return hipGetLastError();
}

// Stage st of pipeline layer v (layer v % L of step v / L); v outside the
// call's n_steps x L layers leaves the stage out of the launch.
void set_seg(StepArgs& a, int st, int v, int n_steps = 1) {
  if (v < 0 || v >= n_steps * a.P.L) {
    a.seg[st] = Seg{-1, 0, 0, 0};
    return;
  }
  a.seg[st] = Seg{v % a.P.L, v % kRing, seg_count(a.P, st), v / a.P.L};
}

hipError_t fill(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

// Pass 1, row normalisers and pass 2 of one layer into ring slot 0 (pass 2
// alone when the caller gives the row normalisers).
hipError_t score_stages(StepArgs a, const Workspace& w, hipStream_t s) {
  const int order[3] = {ST_PASS1, ST_LSE, ST_PASS2};
  for (int i = a.lse ? 2 : 0; i < 3; ++i) {
    for (int st = 0; st < ST_N; ++st) a.seg[st] = Seg{-1, 0, 0, 0};
    a.seg[order[i]] = Seg{0, 0, seg_count(a.P, order[i]), 0};
    const hipError_t e = launch(a, w, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t set_lds_limit(const Problem& P, const Workspace& w) {
  static_assert(kThreads == 512, "task code assumes 512-thread work-groups");
  if (w.lds_bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(pick(P)),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)w.lds_bytes);
}

}  // namespace

hipError_t run_model(const Geometry& g, const ModelIO& m, char* ws, const Workspace& w,
                     hipStream_t s, hipEvent_t* ev) {
  const Problem& P = g.p;
  hipError_t e = set_lds_limit(P, w);
  if (e != hipSuccess) return e;
  StepArgs a = base_args(g, ws, w);
  set_model(a, m);
  a.idx_layer_stride = (int64_t)P.batch * P.H * P.B;
  a.out_layer = 1;
  a.standalone_counts = 0;
  // several steps: one pipeline over their n_steps x L layers in order (a
  // layer's selection chain only links layers of its own step)
  const int ns = m.n_steps > 0 ? m.n_steps : 1;
  if (m.lse) {
    // The row normalisers come from the caller (the log-sum-exp of the
    // layer's prefill attention): no pass 1, a shorter pipeline.
    const int n_launch = ns * P.L + kPipeDepthLse;
    for (int j = 0; j < n_launch; ++j) {
      set_seg(a, ST_P2B, j, ns);
      set_seg(a, ST_POOLB, j - 1, ns);
      set_seg(a, ST_P2X, j - 2, ns);
      set_seg(a, ST_POOLX, j - 3, ns);
      set_seg(a, ST_PREP, j - 4, ns);
      set_seg(a, ST_SELA, j - 5, ns);
      set_seg(a, ST_SELECT, j - 6, ns);
      set_seg(a, ST_COUNT, j - 6, ns);
      set_seg(a, ST_GATHER, j - 7, ns);
      if (ev) (void)hipEventRecord(ev[j], s);
      if ((e = launch(a, w, s)) != hipSuccess) return e;
    }
    if (ev) (void)hipEventRecord(ev[n_launch], s);
    return hipSuccess;
  }
  const int n_launch = ns * P.L + kPipeDepth;
  for (int j = 0; j < n_launch; ++j) {
    set_seg(a, ST_P1B, j, ns);
    set_seg(a, ST_LSEB, j - 1, ns);
    set_seg(a, ST_P2B, j - 2, ns);
    set_seg(a, ST_POOLB, j - 3, ns);
    set_seg(a, ST_P1X, j - 4, ns);
    set_seg(a, ST_LSEX, j - 5, ns);
    set_seg(a, ST_P2X, j - 6, ns);
    set_seg(a, ST_POOLX, j - 7, ns);
    set_seg(a, ST_PREP, j - 8, ns);
    set_seg(a, ST_SELA, j - 9, ns);
    set_seg(a, ST_SELECT, j - 10, ns);
    set_seg(a, ST_COUNT, j - 10, ns);
    set_seg(a, ST_GATHER, j - 11, ns);
    if (ev) (void)hipEventRecord(ev[j], s);
    if ((e = launch(a, w, s)) != hipSuccess) return e;
  }
  if (ev) (void)hipEventRecord(ev[n_launch], s);
  return hipSuccess;
}

hipError_t run_score(const Geometry& g, const void* q, const int64_t qs[3], const void* k,
                     const int64_t ks[3], const float* lse, const int64_t ls[2], float* p_raw,
                     float* p_ext, float* imp, char* ws, const Workspace& w, hipStream_t s) {
  const Problem& P = g.p;
  hipError_t e = set_lds_limit(P, w);
  if (e != hipSuccess) return e;
  StepArgs a = base_args(g, ws, w);
  a.q = static_cast<const char*>(q);
  a.k = static_cast<const char*>(k);
  for (int i = 0; i < 3; ++i) {
    a.qs[i + 1] = qs[i];
    a.ks[i + 1] = ks[i];
  }
  a.lse = lse;
  if (lse) {
    a.ls[1] = ls[0];
    a.ls[2] = ls[1];
  }
  if ((e = score_stages(a, w, s)) != hipSuccess) return e;
  hipLaunchKernelGGL(finalize_kernel, dim3((P.Tc + 255) / 256, P.H + 1, P.batch), dim3(256), 0, s, P,
                     reinterpret_cast<const float*>(ws + w.psum_base),
                     reinterpret_cast<const float*>(ws + w.psum_all),
                     reinterpret_cast<const float*>(ws + w.ipart), p_raw, p_ext, imp);
  return hipGetLastError();
}

// Selection stages of one layer; scores from the caller (p_raw != null) or
// from the workspace partials of ring slot 0.
static hipError_t select_stages(const Geometry& g, int layer, const float* p_raw, const float* p_ext,
                                const float* imp, uint64_t* bits, int32_t* idx, uint32_t* htop,
                                char* ws, const Workspace& w, hipStream_t s) {
  const Problem& P = g.p;
  hipError_t e;
  // n_t of this layer from the caller's bitmap rows of the earlier layers
  hipLaunchKernelGGL(counts_kernel, dim3(P.words, P.batch), dim3(64), 0, s, P, bits,
                     reinterpret_cast<uint8_t*>(ws + w.counts), layer);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (p_raw && (e = fill(reinterpret_cast<uint32_t*>(ws + w.hist),
                         (int64_t)P.batch * 2 * P.H * kHistBins, 0u, s)) != hipSuccess)
    return e;
  StepArgs a = base_args(g, ws, w);
  a.p_raw = p_raw;
  a.p_ext = p_ext;
  a.imp_in = imp;
  a.bits = bits;
  a.idx = idx;
  a.htop = htop;
  a.standalone_counts = 1;
  const int order[4] = {ST_POOL, ST_PREP, ST_SELA, ST_SELECT};
  for (int i = 0; i < 4; ++i) {
    for (int st = 0; st < ST_N; ++st) a.seg[st] = Seg{-1, 0, 0, 0};
    a.seg[order[i]] = Seg{layer, 0, seg_count(P, order[i]), 0};
    if ((e = launch(a, w, s)) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t run_select(const Geometry& g, int layer, const float* p_raw, const float* p_ext,
                      const float* imp, uint64_t* bits, int32_t* idx, uint32_t* htop, char* ws,
                      const Workspace& w, hipStream_t s) {
  hipError_t e = set_lds_limit(g.p, w);
  if (e != hipSuccess) return e;
  return select_stages(g, layer, p_raw, p_ext, imp, bits, idx, htop, ws, w, s);
}

hipError_t run_evict_layer(const Geometry& g, int layer, const ModelIO& m, char* ws,
                           const Workspace& w, hipStream_t s) {
  const Problem& P = g.p;
  hipError_t e = set_lds_limit(P, w);
  if (e != hipSuccess) return e;
  StepArgs a = base_args(g, ws, w);
  set_model(a, m);
  // scores of this layer into ring slot 0 (the tensors carry no layer dimension)
  if ((e = score_stages(a, w, s)) != hipSuccess) return e;
  if ((e = select_stages(g, layer, nullptr, nullptr, nullptr, m.bits, m.idx, nullptr, ws, w, s)) !=
      hipSuccess)
    return e;
  return run_compact(g, 1, m, s);
}

hipError_t run_compact(const Geometry& g, int n_layers, const ModelIO& m, hipStream_t s) {
  Workspace none;
  memset(&none, 0, sizeof(none));
  StepArgs a = base_args(g, nullptr, none);
  set_model(a, m);
  a.idx_layer_stride = (int64_t)g.p.batch * g.p.H * g.p.B;
  a.out_layer = 1;
  for (int l = 0; l < n_layers; ++l) {
    a.seg[ST_GATHER] = Seg{l, 0, seg_count(g.p, ST_GATHER), 0};
    hipError_t e = launch(a, none, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t run_keep_all(const Geometry& g, int layer, uint64_t* bits, int32_t* idx, hipStream_t s) {
  const Problem& P = g.p;
  const int n = max(P.H * P.B, P.words);
  hipLaunchKernelGGL(keep_all_kernel, dim3((n + 255) / 256, P.batch), dim3(256), 0, s, idx, bits,
                     P.H, P.B, P.T, P.L, P.words, layer);
  return hipGetLastError();
}

hipError_t run_coverage(const Geometry& g, const uint64_t* bits, int upto, int64_t* count,
                        hipStream_t s) {
  hipLaunchKernelGGL(coverage_kernel, dim3(g.p.batch), dim3(256), 0, s, bits, count, g.p.L,
                     g.p.words, upto);
  return hipGetLastError();
}

}  // namespace kvec
