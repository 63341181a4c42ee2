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
//   select   layer j-9   (one work-group per (sequence, head); the serial chain)
//   count    layer j-9   (running coverage counts for the next selection)
//   pass 2   layer j-2   last-O rows, every head: P, I
//   pass 2   layer j-6   extended rows, H_top heads: the rest of P over O'
//   pass 1   layer j     last-O rows: row-normaliser partials
//   pass 1   layer j-4   extended rows of the H_top heads
//   lse      layers j-1, j-5 (row normalisers of the two row sets)
//   pool     layer j-3   P: max-pool, sigma sums, histogram, I
//   pool     layer j-7   P over O' of the H_top heads
//   prep     layer j-8   (sigma, H_top, candidate members)
//   gather   layer j-10  (compacted cache)
//
// so L + 10 launches cover the whole step and the serial selection chain
// runs in the shadow of the score passes.  Per-layer scratch lives in a ring
// of kRing slots.
//
// When the caller supplies the window rows' normalisers (the log-sum-exp its
// prefill attention already computed for those query rows), pass 1 and the
// lse stages drop out and the step takes L + 6 launches: pass 2 of the
// last-O rows at j, their pool at j-1, pass 2 of the extended rows at j-2,
// their pool at j-3, prep at j-4, select and count at j-5, gather at j-6.
//
// Work-group IDs are dispatched round-robin over the 8 XCDs, each with its
// own L2.  Within a stage, consecutive tasks (e.g. the row tiles of one key
// tile, which read the same K rows) are mapped to work-groups on the same
// XCD so that K is fetched once per XCD L2.
#include <string.h>

#include "kvec_score_dev.h"
#include "kvec_select_dev.h"

namespace kvec {
namespace {

// Segments are dispatched in this order (long work-groups first).  *_B and
// *_X are the last-O and the extended-window halves of the layer pipeline;
// the plain stages cover every row and head (per-layer entry points).
enum Stage {
  ST_SELECT = 0, ST_COUNT,
  ST_PASS2, ST_P2B, ST_P2X,
  ST_PASS1, ST_P1B, ST_P1X,
  ST_LSE, ST_LSEB, ST_LSEX,
  ST_POOL, ST_POOLB, ST_POOLX,
  ST_PREP, ST_GATHER, ST_N
};

struct Seg {
  int layer;  // model layer the stage works on
  int slot;   // ring slot of that layer's scratch
  int count;  // tasks of this stage in the launch (work-groups: rounded up to 8)
};

struct StepArgs {
  Problem P;
  Workspace w;
  char* ws;
  const char* q;
  const char* k;
  const char* v;
  int64_t qs[4], ks[4], vs[4];
  const float* lse;          // caller's natural-log row normalisers (else null)
  int64_t ls[3];             // their strides {layer, batch, head}
  uint64_t* bits;
  int32_t* idx;
  int64_t idx_layer_stride;  // elements between layers of idx (0: one layer)
  char* k_out;
  char* v_out;
  int out_layer;             // 1: k_out/v_out have a layer dimension
  const float* p_raw;        // standalone selection inputs (else null)
  const float* p_ext;
  const float* imp_in;
  uint32_t* htop;
  int standalone_counts;     // selection reads complete n_t from the counts buffer
  Seg seg[ST_N];
};

__device__ __forceinline__ ScoreIO score_io(const StepArgs& a, int layer, int slot) {
  ScoreIO io;
  char* sb = a.ws + (size_t)slot * a.w.slot_bytes;
  io.q = a.q + (int64_t)layer * a.qs[0] * a.P.esize;
  io.k = a.k + (int64_t)layer * a.ks[0] * a.P.esize;
  io.qs_b = a.qs[1]; io.qs_h = a.qs[2]; io.qs_r = a.qs[3];
  io.ks_b = a.ks[1]; io.ks_h = a.ks[2]; io.ks_t = a.ks[3];
  io.lse_part = reinterpret_cast<float2*>(sb + a.w.lse_part);
  io.lse2 = reinterpret_cast<float*>(sb + a.w.lse2);
  io.psum_base = reinterpret_cast<float*>(sb + a.w.psum_base);
  io.psum_all = reinterpret_cast<float*>(sb + a.w.psum_all);
  io.ipart = reinterpret_cast<float*>(sb + a.w.ipart);
  io.lse_in = a.lse ? a.lse + (int64_t)layer * a.ls[0] : nullptr;
  io.lse_b = a.ls[1];
  io.lse_h = a.ls[2];
  return io;
}

__device__ __forceinline__ SelectIO select_io(const StepArgs& a, int layer, int slot) {
  SelectIO io;
  char* sb = a.ws + (size_t)slot * a.w.slot_bytes;
  const bool standalone = a.p_raw != nullptr;
  io.psum_base = standalone ? nullptr : reinterpret_cast<const float*>(sb + a.w.psum_base);
  io.psum_all = standalone ? nullptr : reinterpret_cast<const float*>(sb + a.w.psum_all);
  io.ipart = reinterpret_cast<const float*>(sb + a.w.ipart);
  io.p_raw = a.p_raw;
  io.p_ext = a.p_ext;
  io.imp_in = a.imp_in;
  io.imp = standalone ? const_cast<float*>(a.imp_in) : reinterpret_cast<float*>(sb + a.w.imp);
  io.pooled = reinterpret_cast<float*>(sb + a.w.pooled);
  io.pooled_ext = reinterpret_cast<float*>(sb + a.w.pooled_ext);
  io.stats = reinterpret_cast<double2*>(sb + a.w.stats);
  io.hist = reinterpret_cast<uint32_t*>(sb + a.w.hist);
  io.mem_t = reinterpret_cast<int32_t*>(sb + a.w.mem_t);
  io.mem_ps = reinterpret_cast<float*>(sb + a.w.mem_ps);
  io.mem_i = reinterpret_cast<float*>(sb + a.w.mem_i);
  io.mem_n = reinterpret_cast<int32_t*>(sb + a.w.mem_n);
  io.htop_mask = a.htop;
  io.spill_keys = reinterpret_cast<uint32_t*>(a.ws + a.w.spill);
  io.spill_t = reinterpret_cast<int32_t*>(a.ws + a.w.spill + a.w.spill_stride);
  io.spill_ps = reinterpret_cast<float*>(a.ws + a.w.spill + 2 * a.w.spill_stride);
  io.spill_i = reinterpret_cast<float*>(a.ws + a.w.spill + 3 * a.w.spill_stride);
  const uint8_t* cnt = reinterpret_cast<const uint8_t*>(a.ws + a.w.counts);
  if (a.standalone_counts) {
    // counts of the caller's earlier rows, computed for this call
    io.cnt_in = cnt;
    io.bits_prev = nullptr;
  } else {
    // pipeline: n_t(l) = counts(l-1) + kept bit of layer l-1
    io.cnt_in = layer >= 2 ? cnt + (size_t)((layer - 1) & 1) * a.w.counts_stride : nullptr;
    io.bits_prev = layer >= 1 ? a.bits + (int64_t)(layer - 1) * a.P.words : nullptr;
  }
  io.bits = a.bits;
  io.idx = a.idx + (int64_t)layer * a.idx_layer_stride;
  return io;
}

// Cache store (Sec. 4.1): out[b][h][i] = K[b][h][idx[b][h][i]] (and V),
// one 16-byte chunk per thread and round, 4 rounds per work-group; idx
// outside [0, T) -> zeros.  All index loads are issued first, then all row
// loads, then the stores (one memory round trip each).
__device__ __forceinline__ void task_gather(const StepArgs& a, int layer, int b, int part) {
  constexpr int kRounds = 4;
  const Problem& P = a.P;
  const int cpr = P.D * P.esize / 16;
  const int64_t total = (int64_t)P.H * P.B * cpr;
  const int32_t* idx = a.idx + (int64_t)layer * a.idx_layer_stride + (int64_t)b * P.H * P.B;
  const int64_t orow0 = ((int64_t)(a.out_layer ? layer : 0) * P.batch + b) * P.H * P.B;
  int64_t ci[kRounds];
  int id[kRounds];
#pragma unroll
  for (int e = 0; e < kRounds; ++e) {
    ci[e] = ((int64_t)part * kRounds + e) * kThreads + threadIdx.x;
    id[e] = ci[e] < total ? idx[ci[e] / cpr] : -1;
  }
  uint4 kv[kRounds], vv[kRounds];
#pragma unroll
  for (int e = 0; e < kRounds; ++e) {
    kv[e] = make_uint4(0, 0, 0, 0);
    vv[e] = make_uint4(0, 0, 0, 0);
    if (ci[e] < total && id[e] >= 0 && id[e] < P.T) {
      const int ch = (int)(ci[e] % cpr);
      const int h = (int)((ci[e] / cpr) / P.B);
      const int64_t ko = ((int64_t)layer * a.ks[0] + (int64_t)b * a.ks[1] + (int64_t)h * a.ks[2] +
                          (int64_t)id[e] * a.ks[3]) * P.esize;
      const int64_t vo = ((int64_t)layer * a.vs[0] + (int64_t)b * a.vs[1] + (int64_t)h * a.vs[2] +
                          (int64_t)id[e] * a.vs[3]) * P.esize;
      kv[e] = reinterpret_cast<const uint4*>(a.k + ko)[ch];
      vv[e] = reinterpret_cast<const uint4*>(a.v + vo)[ch];
    }
  }
#pragma unroll
  for (int e = 0; e < kRounds; ++e) {
    if (ci[e] < total) {
      const int64_t o = (orow0 + ci[e] / cpr) * cpr + ci[e] % cpr;
      reinterpret_cast<uint4*>(a.k_out)[o] = kv[e];
      reinterpret_cast<uint4*>(a.v_out)[o] = vv[e];
    }
  }
}

// First window row held by the row tiles of the last-O rows.
__host__ __device__ inline int base_row_lo(const Problem& P) { return max(0, P.Wn - P.n_rt_base * P.WR); }

// Row-normaliser tasks per sequence of one LSE stage.
__host__ __device__ inline int lse_tasks_per_seq(const Problem& P, int st) {
  const int rb0 = base_row_lo(P);
  const int nr = st == ST_LSEB ? P.Wn - rb0 : st == ST_LSEX ? rb0 : P.Wn;
  return (P.HQ * nr + kLseRows - 1) / kLseRows;
}

template <class TT, int D, int G>
__global__ __launch_bounds__(kThreads) void step_kernel(StepArgs a) {
  extern __shared__ __align__(16) char smem[];
  const Problem P = a.P;
  int blk = blockIdx.x;
  int st = 0;
  for (; st < ST_N; ++st) {
    const int n8 = (a.seg[st].count + 7) & ~7;
    if (blk < n8) break;
    blk -= n8;
  }
  if (st >= ST_N) return;
  const Seg sg = a.seg[st];
  {
    // XCD-aware remap: segments start at multiples of 8, so blk % 8 is the XCD
    const int n8 = (sg.count + 7) & ~7;
    blk = (blk & 7) * (n8 >> 3) + (blk >> 3);
    if (blk >= sg.count) return;
  }
  switch (st) {
    case ST_SELECT: {
      const int b = blk / P.H, h = blk % P.H;
      task_select(P, select_io(a, sg.layer, sg.slot), sg.layer, b, h, smem);
      break;
    }
    case ST_COUNT: {
      const int parts = (P.words + kCountWords - 1) / kCountWords;
      const int b = blk / parts;
      const int layer = sg.layer;
      const uint8_t* cbase = reinterpret_cast<const uint8_t*>(a.ws + a.w.counts);
      const uint8_t* prev = layer >= 2 ? cbase + (size_t)((layer - 1) & 1) * a.w.counts_stride : nullptr;
      const uint64_t* row = layer >= 1 ? a.bits + (int64_t)(layer - 1) * P.words : nullptr;
      uint8_t* out = reinterpret_cast<uint8_t*>(a.ws + a.w.counts) + (size_t)(layer & 1) * a.w.counts_stride;
      task_count(P, prev, row, out, b, blk % parts);
      break;
    }
    case ST_PASS1:
    case ST_P1B:
    case ST_P1X: {
      const Part part = st == ST_P1B ? PART_BASE : st == ST_P1X ? PART_EXT : PART_ALL;
      const int n_rtg = part == PART_BASE ? P.n_rtg_base : part == PART_EXT ? P.n_rtg_x : P.n_rtg;
      const int per_b = P.n_kt1 * n_rtg;
      const int b = blk / per_b, rem = blk % per_b;
      const uint32_t hm =
          part == PART_EXT ? htop_mask(P, select_io(a, sg.layer, sg.slot).stats, b) : 0u;
      score_tile<TT, D, G, 1>(P, score_io(a, sg.layer, sg.slot), b, rem / n_rtg, rem % n_rtg,
                              reinterpret_cast<float*>(smem), part, hm);
      break;
    }
    case ST_LSE:
    case ST_LSEB:
    case ST_LSEX: {
      const int per_b = lse_tasks_per_seq(P, st);
      const int b = blk / per_b;
      const int rb0 = base_row_lo(P);
      const uint32_t all = (1u << P.H) - 1u;
      const ScoreIO io = score_io(a, sg.layer, sg.slot);
      if (st == ST_LSE)
        task_lse<TT, D, G>(P, io, b, blk % per_b, 0, P.Wn, all);
      else if (st == ST_LSEB)
        task_lse<TT, D, G>(P, io, b, blk % per_b, rb0, P.Wn - rb0, all);
      else
        task_lse<TT, D, G>(P, io, b, blk % per_b, 0, rb0,
                           htop_mask(P, select_io(a, sg.layer, sg.slot).stats, b));
      break;
    }
    case ST_PASS2:
    case ST_P2B:
    case ST_P2X: {
      const Part part = st == ST_P2B ? PART_BASE : st == ST_P2X ? PART_EXT : PART_ALL;
      const int n_rtg = part == PART_BASE ? P.n_rtg_base : part == PART_EXT ? P.n_rtg_x : P.n_rtg;
      const int per_b = P.n_kt2 * n_rtg;
      const int b = blk / per_b, rem = blk % per_b;
      const ScoreIO io = score_io(a, sg.layer, sg.slot);
      const uint32_t hm =
          part == PART_EXT ? htop_mask(P, select_io(a, sg.layer, sg.slot).stats, b) : 0u;
      score_tile<TT, D, G, 2>(P, io, b, rem / n_rtg, rem % n_rtg, reinterpret_cast<float*>(smem),
                              part, hm);
      if (part != PART_EXT) {
        // Clear this sequence's histograms for the pool stages of this layer.
        uint32_t* hist = reinterpret_cast<uint32_t*>(a.ws + (size_t)sg.slot * a.w.slot_bytes + a.w.hist) +
                         (int64_t)b * 2 * P.H * kHistBins;
        const int nwords = 2 * P.H * kHistBins;
        const int per = (nwords + per_b - 1) / per_b;
        for (int i = rem * per + threadIdx.x; i < min(nwords, (rem + 1) * per); i += kThreads) hist[i] = 0u;
      }
      break;
    }
    case ST_PREP: {
      const int nt = (P.n_prep + kPrepPer - 1) / kPrepPer;
      const int per_b = P.H * nt;
      const int b = blk / per_b, rem = blk % per_b;
      const int c0 = (rem % nt) * kPrepPer;
      task_prep(P, select_io(a, sg.layer, sg.slot), sg.layer, b, rem / nt, c0,
                min(P.n_prep, c0 + kPrepPer), smem);
      break;
    }
    case ST_POOL:
    case ST_POOLB: {
      const int nt = (P.n_pool + kPoolPer - 1) / kPoolPer;
      const int per_b = P.H * nt;
      const int b = blk / per_b, rem = blk % per_b;
      const int c0 = (rem % nt) * kPoolPer;
      task_pool(P, select_io(a, sg.layer, sg.slot), b, rem / nt, c0, min(P.n_pool, c0 + kPoolPer),
                smem, true, st == ST_POOL);
      break;
    }
    case ST_POOLX: {
      const int nt = (P.n_pool + kPoolPer - 1) / kPoolPer;
      const int per_b = P.delta_eff * nt;
      const int b = blk / per_b, rem = blk % per_b;
      const SelectIO io = select_io(a, sg.layer, sg.slot);
      const int h = nth_bit(htop_mask(P, io.stats, b), rem / nt);
      const int c0 = (rem % nt) * kPoolPer;
      if (h >= 0) task_pool(P, io, b, h, c0, min(P.n_pool, c0 + kPoolPer), smem, false, true);
      break;
    }
    case ST_GATHER: {
      const int b = blk / P.n_gather;
      task_gather(a, sg.layer, b, blk % P.n_gather);
      break;
    }
  }
}

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

int seg_count(const Problem& P, int st) {
  const bool ext = P.delta_eff > 0;
  switch (st) {
    case ST_SELECT: return P.batch * P.H;
    case ST_COUNT: return P.batch * ((P.words + kCountWords - 1) / kCountWords);
    case ST_PASS1: return P.batch * P.n_kt1 * P.n_rtg;
    case ST_P1B: return P.batch * P.n_kt1 * P.n_rtg_base;
    case ST_P1X: return P.batch * P.n_kt1 * P.n_rtg_x;
    case ST_LSE:
    case ST_LSEB: return P.batch * lse_tasks_per_seq(P, st);
    case ST_LSEX: return P.n_rtg_x ? P.batch * lse_tasks_per_seq(P, st) : 0;
    case ST_PASS2: return P.batch * P.n_kt2 * P.n_rtg;
    case ST_P2B: return P.batch * P.n_kt2 * P.n_rtg_base;
    case ST_P2X: return P.batch * P.n_kt2 * P.n_rtg_x;
    case ST_POOL:
    case ST_POOLB: return P.batch * P.H * ((P.n_pool + kPoolPer - 1) / kPoolPer);
    case ST_POOLX: return ext ? P.batch * P.delta_eff * ((P.n_pool + kPoolPer - 1) / kPoolPer) : 0;
    case ST_PREP: return P.batch * P.H * ((P.n_prep + kPrepPer - 1) / kPrepPer);
    case ST_GATHER: return P.batch * P.n_gather;
  }
  return 0;
}

typedef void (*StepFn)(StepArgs);

template <class TT, int D>
StepFn pick_g(int G) {
  switch (G) {
    case 1: return step_kernel<TT, D, 1>;
    case 2: return step_kernel<TT, D, 2>;
    case 4: return step_kernel<TT, D, 4>;
    default: return step_kernel<TT, D, 8>;
  }
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
  for (int s = 0; s < ST_N; ++s) a.seg[s] = Seg{-1, 0, 0};
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

void set_seg(StepArgs& a, int st, int layer) {
  if (layer < 0 || layer >= a.P.L) {
    a.seg[st] = Seg{-1, 0, 0};
    return;
  }
  a.seg[st] = Seg{layer, layer % kRing, seg_count(a.P, st)};
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
    for (int st = 0; st < ST_N; ++st) a.seg[st] = Seg{-1, 0, 0};
    a.seg[order[i]] = Seg{0, 0, seg_count(a.P, order[i])};
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
  if (m.lse) {
    // The row normalisers come from the caller (the log-sum-exp of the
    // layer's prefill attention): no pass 1, a 6-launch pipeline.
    const int n_launch = P.L + kPipeDepthLse;
    for (int j = 0; j < n_launch; ++j) {
      set_seg(a, ST_P2B, j);
      set_seg(a, ST_POOLB, j - 1);
      set_seg(a, ST_P2X, j - 2);
      set_seg(a, ST_POOLX, j - 3);
      set_seg(a, ST_PREP, j - 4);
      set_seg(a, ST_SELECT, j - 5);
      set_seg(a, ST_COUNT, j - 5);
      set_seg(a, ST_GATHER, j - 6);
      if (ev) (void)hipEventRecord(ev[j], s);
      if ((e = launch(a, w, s)) != hipSuccess) return e;
    }
    if (ev) (void)hipEventRecord(ev[n_launch], s);
    return hipSuccess;
  }
  const int n_launch = P.L + kPipeDepth;
  for (int j = 0; j < n_launch; ++j) {
    set_seg(a, ST_P1B, j);
    set_seg(a, ST_LSEB, j - 1);
    set_seg(a, ST_P2B, j - 2);
    set_seg(a, ST_POOLB, j - 3);
    set_seg(a, ST_P1X, j - 4);
    set_seg(a, ST_LSEX, j - 5);
    set_seg(a, ST_P2X, j - 6);
    set_seg(a, ST_POOLX, j - 7);
    set_seg(a, ST_PREP, j - 8);
    set_seg(a, ST_SELECT, j - 9);
    set_seg(a, ST_COUNT, j - 9);
    set_seg(a, ST_GATHER, j - 10);
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
  const int order[3] = {ST_POOL, ST_PREP, ST_SELECT};
  for (int i = 0; i < 3; ++i) {
    for (int st = 0; st < ST_N; ++st) a.seg[st] = Seg{-1, 0, 0};
    a.seg[order[i]] = Seg{layer, 0, seg_count(P, order[i])};
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
    a.seg[ST_GATHER] = Seg{l, 0, seg_count(g.p, ST_GATHER)};
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
