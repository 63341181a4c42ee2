// Fused step kernel of the eviction pipeline: the argument block, the stage
// dispatch and the cache-store task.  The launchers (kvec_pipeline.hip) see
// only the declarations of pick_g; each (dtype, head_dim) pair is
// instantiated for every group size 1..8 in its own translation unit
// (kvec_step_inst.hip, built once per pair).
#pragma once

#include "kvec_score_dev.h"
#include "kvec_select_dev.h"

namespace kvec {
namespace step {


// Segments are dispatched in this order (long work-groups first).  *_B and
// *_X are the last-O and the extended-window halves of the layer pipeline;
// the plain stages cover every row and head (per-layer entry points).
enum Stage {
  ST_SELECT = 0, ST_SELA, ST_COUNT,
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
  int step;   // which of the call's independent steps the layer belongs to
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
  float* sc_p;               // nullable pipeline score outputs (see ModelIO)
  float* sc_pe;
  float* sc_imp;
  uint32_t* sc_htop;
  int standalone_counts;     // selection reads complete n_t from the counts buffer
  // elements (words for bits) between consecutive steps of a multi-step call
  int64_t q_step, k_step, v_step, lse_step, bits_step, idx_step, out_step;
  Seg seg[ST_N];
};

__device__ __forceinline__ ScoreIO score_io(const StepArgs& a, int layer, int slot, int step = 0) {
  ScoreIO io;
  char* sb = a.ws + (size_t)slot * a.w.slot_bytes;
  io.q = a.q + ((int64_t)step * a.q_step + (int64_t)layer * a.qs[0]) * a.P.esize;
  io.k = a.k + ((int64_t)step * a.k_step + (int64_t)layer * a.ks[0]) * a.P.esize;
  io.qs_b = a.qs[1]; io.qs_h = a.qs[2]; io.qs_r = a.qs[3];
  io.ks_b = a.ks[1]; io.ks_h = a.ks[2]; io.ks_t = a.ks[3];
  io.lse_part = reinterpret_cast<float2*>(sb + a.w.lse_part);
  io.lse2 = reinterpret_cast<float*>(sb + a.w.lse2);
  io.psum_base = reinterpret_cast<float*>(sb + a.w.psum_base);
  io.psum_all = reinterpret_cast<float*>(sb + a.w.psum_all);
  io.ipart = reinterpret_cast<float*>(sb + a.w.ipart);
  io.lse_in = a.lse ? a.lse + (int64_t)step * a.lse_step + (int64_t)layer * a.ls[0] : nullptr;
  io.lse_b = a.ls[1];
  io.lse_h = a.ls[2];
  return io;
}

__device__ __forceinline__ SelectIO select_io(const StepArgs& a, int layer, int slot, int step = 0) {
  SelectIO io;
  uint64_t* const bits = a.bits + (int64_t)step * a.bits_step;
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
  io.htop_mask = a.sc_htop ? a.sc_htop + (int64_t)layer * a.P.batch : a.htop;
  const int64_t per_p = (int64_t)a.P.batch * a.P.H * a.P.Tc;
  io.out_p = a.sc_p ? a.sc_p + (int64_t)layer * per_p : nullptr;
  io.out_pe = a.sc_pe ? a.sc_pe + (int64_t)layer * per_p : nullptr;
  io.out_imp = a.sc_imp ? a.sc_imp + (int64_t)layer * a.P.batch * a.P.Tc : nullptr;
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
    io.bits_prev = layer >= 1 ? bits + (int64_t)(layer - 1) * a.P.words : nullptr;
  }
  io.bits = bits;
  io.idx = a.idx + (int64_t)step * a.idx_step + (int64_t)layer * a.idx_layer_stride;
  return io;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Cache store (Sec. 4.1): out[b][h][i] = K[b][h][idx[b][h][i]] (and V),
// one 16-byte chunk per thread and round, 4 rounds per work-group; idx
// outside [0, T) -> zeros.  All index loads are issued first, then all row
// loads, then the stores (one memory round trip each).  The row reads (the
// last use of those rows in the step) and the stores (not read again by the
// step) are non-temporal, so they do not displace keys that the score
// stages read again.
__device__ __forceinline__ void task_gather(const StepArgs& a, int layer, int step, int b, int part) {
  constexpr int kRounds = 4;
  const Problem& P = a.P;
  const int cpr = P.D * P.esize / 16;
  const int64_t total = (int64_t)P.H * P.B * cpr;
  const int32_t* idx =
      a.idx + (int64_t)step * a.idx_step + (int64_t)layer * a.idx_layer_stride + (int64_t)b * P.H * P.B;
  const int64_t orow0 = ((int64_t)(a.out_layer ? layer : 0) * P.batch + b) * P.H * P.B;
  const char* kin = a.k + (int64_t)step * a.k_step * P.esize;
  const char* vin = a.v + (int64_t)step * a.v_step * P.esize;
  char* kout = a.k_out + (int64_t)step * a.out_step * P.esize;
  char* vout = a.v_out + (int64_t)step * a.out_step * P.esize;
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
      const u32x4 tk = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kin + ko) + ch);
      const u32x4 tv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vin + vo) + ch);
      kv[e] = make_uint4(tk.x, tk.y, tk.z, tk.w);
      vv[e] = make_uint4(tv.x, tv.y, tv.z, tv.w);
    }
  }
#pragma unroll
  for (int e = 0; e < kRounds; ++e) {
    if (ci[e] < total) {
      const int64_t o = (orow0 + ci[e] / cpr) * cpr + ci[e] % cpr;
      const u32x4 tk = {kv[e].x, kv[e].y, kv[e].z, kv[e].w};
      const u32x4 tv = {vv[e].x, vv[e].y, vv[e].z, vv[e].w};
      __builtin_nontemporal_store(tk, reinterpret_cast<u32x4*>(kout) + o);
      __builtin_nontemporal_store(tv, reinterpret_cast<u32x4*>(vout) + o);
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

// EXT passes: wave w of work-group blk takes task blk * 8 + w of the
// (sequence, key tile, H_top head, extended row tile) tasks, in that order
// (the row tiles of one head and key tile, which read the same keys, are
// neighbours).  Returns the sequence; hm gets the task's head as a one-bit
// mask, 0 past the last task.
__device__ __forceinline__ int ext_task(const Problem& P, const StepArgs& a, const Seg& sg, int n_kt,
                                        int blk, int& kt, int& rte, uint32_t& hm) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int per_kt = P.delta_eff * P.n_rt_x;
  const int per_b = n_kt * per_kt;
  const int ti = blk * 8 + w;
  kt = 0;
  rte = 0;
  hm = 0u;
  if (ti >= P.batch * per_b) return 0;
  const int b = ti / per_b, rem = ti % per_b;
  kt = rem / per_kt;
  const int q = rem % per_kt;
  rte = q % P.n_rt_x;
  hm = 1u << nth_bit(htop_mask(P, select_io(a, sg.layer, sg.slot, sg.step).stats, b), q / P.n_rt_x);
  return b;
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
      task_select_b(P, select_io(a, sg.layer, sg.slot, sg.step), sg.layer, b, h, smem);
      break;
    }
    case ST_SELA: {
      const int b = blk / P.H, h = blk % P.H;
      task_select_a(P, select_io(a, sg.layer, sg.slot, sg.step), b, h, smem);
      break;
    }
    case ST_COUNT: {
      const int parts = (P.words + kCountWords - 1) / kCountWords;
      const int b = blk / parts;
      const int layer = sg.layer;
      const uint8_t* cbase = reinterpret_cast<const uint8_t*>(a.ws + a.w.counts);
      const uint8_t* prev = layer >= 2 ? cbase + (size_t)((layer - 1) & 1) * a.w.counts_stride : nullptr;
      const uint64_t* row =
          layer >= 1 ? a.bits + (int64_t)sg.step * a.bits_step + (int64_t)(layer - 1) * P.words : nullptr;
      uint8_t* out = reinterpret_cast<uint8_t*>(a.ws + a.w.counts) + (size_t)(layer & 1) * a.w.counts_stride;
      task_count(P, prev, row, out, b, blk % parts);
      break;
    }
    case ST_PASS1:
    case ST_P1B: {
      const Part part = st == ST_P1B ? PART_BASE : PART_ALL;
      const int n_rtg = part == PART_BASE ? P.n_rtg_base : P.n_rtg;
      const int per_b = P.n_kt1 * n_rtg;
      const int b = blk / per_b, rem = blk % per_b;
      score_tile<TT, D, G, 1>(P, score_io(a, sg.layer, sg.slot, sg.step), b, rem / n_rtg, rem % n_rtg,
                              reinterpret_cast<float*>(smem), part, 0u);
      break;
    }
    case ST_P1X: {
      int kt, rte;
      uint32_t hm;
      const int b = ext_task(P, a, sg, P.n_kt1, blk, kt, rte, hm);
      score_tile<TT, D, G, 1>(P, score_io(a, sg.layer, sg.slot, sg.step), b, kt, rte,
                              reinterpret_cast<float*>(smem), PART_EXT, hm);
      break;
    }
    case ST_LSE:
    case ST_LSEB:
    case ST_LSEX: {
      const int per_b = lse_tasks_per_seq(P, st);
      const int b = blk / per_b;
      const int rb0 = base_row_lo(P);
      const uint32_t all = (1u << P.H) - 1u;
      const ScoreIO io = score_io(a, sg.layer, sg.slot, sg.step);
      if (st == ST_LSE)
        task_lse<TT, D, G>(P, io, b, blk % per_b, 0, P.Wn, all);
      else if (st == ST_LSEB)
        task_lse<TT, D, G>(P, io, b, blk % per_b, rb0, P.Wn - rb0, all);
      else
        task_lse<TT, D, G>(P, io, b, blk % per_b, 0, rb0,
                           htop_mask(P, select_io(a, sg.layer, sg.slot, sg.step).stats, b));
      break;
    }
    case ST_P2X: {
      int kt, rte;
      uint32_t hm;
      const int b = ext_task(P, a, sg, P.n_kt2, blk, kt, rte, hm);
      score_tile<TT, D, G, 2>(P, score_io(a, sg.layer, sg.slot, sg.step), b, kt, rte,
                              reinterpret_cast<float*>(smem), PART_EXT, hm);
      break;
    }
    case ST_PASS2:
    case ST_P2B: {
      const Part part = st == ST_P2B ? PART_BASE : PART_ALL;
      const int n_rtg = part == PART_BASE ? P.n_rtg_base : P.n_rtg;
      const int per_b = P.n_kt2 * n_rtg;
      const int b = blk / per_b, rem = blk % per_b;
      const ScoreIO io = score_io(a, sg.layer, sg.slot, sg.step);
      score_tile<TT, D, G, 2>(P, io, b, rem / n_rtg, rem % n_rtg, reinterpret_cast<float*>(smem),
                              part, 0u);
      {
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
      task_prep(P, select_io(a, sg.layer, sg.slot, sg.step), sg.layer, b, rem / nt, c0,
                min(P.n_prep, c0 + kPrepPer), smem);
      break;
    }
    case ST_POOL:
    case ST_POOLB: {
      const int nt = (P.n_pool + kPoolPer - 1) / kPoolPer;
      const int per_b = P.H * nt;
      const int b = blk / per_b, rem = blk % per_b;
      const int c0 = (rem % nt) * kPoolPer;
      task_pool(P, select_io(a, sg.layer, sg.slot, sg.step), b, rem / nt, c0, min(P.n_pool, c0 + kPoolPer),
                smem, true, st == ST_POOL);
      break;
    }
    case ST_POOLX: {
      const int nt = (P.n_pool + kPoolPer - 1) / kPoolPer;
      const int per_b = P.delta_eff * nt;
      const int b = blk / per_b, rem = blk % per_b;
      const SelectIO io = select_io(a, sg.layer, sg.slot, sg.step);
      const int h = nth_bit(htop_mask(P, io.stats, b), rem / nt);
      const int c0 = (rem % nt) * kPoolPer;
      if (h >= 0) task_pool(P, io, b, h, c0, min(P.n_pool, c0 + kPoolPer), smem, false, true);
      break;
    }
    case ST_GATHER: {
      const int b = blk / P.n_gather;
      task_gather(a, sg.layer, sg.step, b, blk % P.n_gather);
      break;
    }
  }
}

typedef void (*StepFn)(StepArgs);

// The step kernel of one (dtype, head_dim) for group size G (1..8).
template <class TT, int D>
StepFn pick_g(int G);
template <> StepFn pick_g<BF16, 64>(int G);
template <> StepFn pick_g<BF16, 128>(int G);
template <> StepFn pick_g<F32, 64>(int G);
template <> StepFn pick_g<F32, 128>(int G);

}  // namespace step
}  // namespace kvec
