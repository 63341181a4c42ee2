// Internal declarations shared by the libkvec translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kvec.h"

namespace kvec {

constexpr int kThreads = 512;  // every work-group of the step kernel: 8 waves
constexpr int kPipeDepth = 11;         // launches between a layer's first and last stage
constexpr int kPipeDepthLse = 7;       // the same when the row normalisers are given
constexpr int kRing = kPipeDepth + 1;  // layers in flight in the software pipeline

constexpr int kTileMax = 512;     // keys per score work-group at long prefixes
constexpr int kTileMin = 128;     // ... and the least at short ones
constexpr int kPoolChunk = 512;   // tokens per pool statistics entry (one wave)
constexpr int kPrepChunk = 1024;  // tokens per candidate chunk (one wave, 16 per lane)
constexpr int kPoolPer = 8;       // pool chunks per pool work-group (one per wave)
constexpr int kPrepPer = 8;       // candidate chunks per prep work-group (one per wave)
constexpr int kHistBits = 12;     // selection histograms over the top 12 key bits
constexpr int kHistBins = 1 << kHistBits;

// Row tiling of the score passes: a wave computes NB = G * RB blocks of 16
// query rows, i.e. RB 16-row blocks of the window for each of the G query
// heads of its KV head.
template <int G>
struct Tiling {
  static constexpr int RB = G >= 4 ? 1 : 4 / G;
  static constexpr int NB = G * RB;
  static constexpr int WR = 16 * RB;  // window rows per row tile
};

inline int row_blocks_per_tile(int G) { return G >= 4 ? 1 : 4 / G; }

// Key staging of the score passes: each wave streams its keys, 16 per step,
// through a private ring of LDS slots (16 * D * esize bytes each).  Deeper
// rings for small slots; fp32 with d = 128 keeps a single slot.
constexpr int key_ring_slots(int esize, int D) {
  return 16 * D * esize <= 2048 ? 4 : 16 * D * esize <= 4096 ? 3 : 1;
}
constexpr size_t key_ring_bytes(int esize, int D) {
  return (size_t)(kThreads / 64) * key_ring_slots(esize, D) * 16 * D * esize;
}
// Pass-2 LDS floats per row-tile slot of nh heads: the running-max buffers
// [WR][SK + 4] when the slot exchanges the importance over heads (one when
// the exchange period is the whole key tile, else two, used in turn), per-key
// sums of each head (nsum of them: all rows, and the last-O rows when a row
// tile can hold both kinds) and the importance of the key tile.
__host__ __device__ constexpr int exchange_buffers(int SK, int tile2) { return SK >= tile2 ? 1 : 2; }
__host__ __device__ constexpr int p2_slot_floats(int nh, int WR, int SK, int tile2, bool exchange,
                                                 int nsum) {
  return (exchange ? exchange_buffers(SK, tile2) * WR * (SK + 4) : 0) + nsum * nh * tile2 + tile2;
}

// Which window rows and heads a score pass covers.  ALL: every row tile and
// head (the per-layer entry points).  BASE: the row tiles holding the last-O
// rows, every head.  EXT: the remaining row tiles (rows of the extended window
// only), for the heads of H_top only; their rows enter only P over O'.
enum Part { PART_ALL = 0, PART_BASE = 1, PART_EXT = 2 };

// Problem geometry visible to device code.
struct Problem {
  int batch, L, H, HQ, G, D, T, O, Wn, Tc, B, M, Kp, pool, delta_eff;
  float lam, sc, inv_go, inv_gwn;
  int WR, n_rt, n_rt_base, n_rtg, n_kt1, n_kt2, SK, tile1, tile2;
  int sk_shift;    // log2(SK): exchange periods are powers of two
  int nsum;        // pass-2 per-key sums per head: 1 when O is a multiple of WR (no row
                   // tile holds both last-O and earlier rows), else 2
  int n_rtg_base;  // work-groups per key tile of a BASE pass (8/H row tiles each)
  int n_rt_x;      // row tiles of an EXT pass (extended-window rows only; 0: no EXT
                   // pass); its tasks (key tile, H_top head, row tile) go one per wave
  int n_pool, n_prep, words;
  int esize;
  int n_gather;  // gather work-groups per (layer, sequence)
  int mcap;      // selection members per head held in LDS
  int criterion; // H_top criterion: 0 lowest sigma, 1 highest entropy of pooled P
};

struct Geometry {
  Problem p;
  bool keep_all;  // T <= B: every token is kept
};

// Byte offsets of one ring slot (one layer in flight) and of the shared areas.
struct Workspace {
  size_t lse_part, lse2, psum_base, psum_all, ipart, imp, pooled, pooled_ext, stats, hist, mem_t,
      mem_ps, mem_i, mem_n;
  size_t slot_bytes;
  size_t counts, counts_stride;  // two uint8 [b][T] count buffers (layer parity)
  size_t spill, spill_stride;    // four [b][H][Tc] member arrays
  size_t lds_bytes;
  size_t total;
};

kvec_status make_geometry(const kvec_config* cfg, Geometry* g);
Workspace make_workspace(const Geometry& g);

// Host launchers (kvec_pipeline.hip).
struct ModelIO {
  const void* q;          // [layer][b][HQ][Wn][d] with element strides qs
  const void* k;
  const void* v;
  int64_t qs[4], ks[4], vs[4];
  uint64_t* bits;         // [b][L][W]
  int32_t* idx;           // [L][b][H][B] (or [b][H][B] for one layer)
  void* k_out;            // [L][b][H][B][d]
  void* v_out;
  const float* lse;       // nullable: natural-log row normalisers [layer][b][HQ][Wn], strides ls
  int64_t ls[3];
  // nullable score outputs of the layer pipeline (all four or none): P and P
  // over O' before pooling [layer][b][H][Tc] (P over O' for the H_top heads
  // only), I [layer][b][Tc], H_top masks [layer][b]
  float* sc_p;
  float* sc_pe;
  float* sc_imp;
  uint32_t* sc_htop;
  // independent steps run as one pipeline over n_steps x L layers; elements
  // (words for bits) between consecutive steps of each tensor
  int n_steps;
  int64_t q_step, k_step, v_step, lse_step, bits_step, idx_step, out_step;
};

hipError_t run_model(const Geometry& g, const ModelIO& m, char* ws, const Workspace& w,
                     hipStream_t s, hipEvent_t* ev);
hipError_t run_score(const Geometry& g, const void* q, const int64_t qs[3], const void* k,
                     const int64_t ks[3], const float* lse, const int64_t ls[2], float* p_raw,
                     float* p_ext, float* imp, char* ws, const Workspace& w, hipStream_t s);
hipError_t run_select(const Geometry& g, int layer, const float* p_raw, const float* p_ext,
                      const float* imp, uint64_t* bits, int32_t* idx, uint32_t* htop, char* ws,
                      const Workspace& w, hipStream_t s);
hipError_t run_evict_layer(const Geometry& g, int layer, const ModelIO& m, char* ws,
                           const Workspace& w, hipStream_t s);
hipError_t run_compact(const Geometry& g, int n_layers, const ModelIO& m, hipStream_t s);
hipError_t run_keep_all(const Geometry& g, int layer, uint64_t* bits, int32_t* idx, hipStream_t s);
hipError_t run_coverage(const Geometry& g, const uint64_t* bits, int upto, int64_t* count,
                        hipStream_t s);

// Decode attention over the compacted cache (kvec_decode.hip).
struct DecodePlan {
  int chunk;        // cache rows per partial work-group
  int S;            // chunks per (sequence, KV head)
  size_t ws_bytes;  // partial states [b][HQ][S][d + 2] floats
};
DecodePlan decode_plan(const Problem& P, int n_ctx);
// Fixed device scratch of kvec_decode_attention_noalloc (partial states).
constexpr size_t kDecodeScratchBytes = (size_t)4 << 20;
// Device address of that scratch on the current device (set up on first use).
hipError_t decode_scratch(void** ptr);
hipError_t run_decode(const Geometry& g, const void* q, const int64_t qs[2], const void* k,
                      const void* v, const int64_t cs[2], int n_ctx, const int32_t* idx, float* out,
                      void* ws, hipStream_t s);

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

// Order-preserving map of an IEEE float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t float_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive prefix sum over the work-group (blockDim.x a multiple of 64, at
// most 1024).  `tmp` holds >= 17 ints of shared memory.  Returns the
// exclusive prefix; `total` receives the block sum.  Contains barriers.
__device__ __forceinline__ int block_excl_scan(int v, int* tmp, int& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) tmp[wid] = incl;
  __syncthreads();
  if (wid == 0) {
    const int x = lane < nw ? tmp[lane] : 0;
    const int xi = wave_incl_scan(x);
    if (lane < nw) tmp[lane] = xi - x;
    if (lane == nw - 1) tmp[16] = xi;
  }
  __syncthreads();
  const int r = tmp[wid] + incl - v;
  total = tmp[16];
  __syncthreads();
  return r;
}

// Pool work-groups per (sequence, head): each writes one float64 (sum, sum
// of squares) of pooled P over its chunks.
__host__ __device__ inline int pool_groups(const Problem& P) { return (P.n_pool + kPoolPer - 1) / kPoolPer; }

// H_top (Sec. 4.1): bit h set for the delta_eff heads of sequence b with the
// lowest variance of pooled P, or with the highest entropy of pooled P taken
// as a distribution (the ablation's alternative, Sec. 5.4); ties: lower head.
// From the per-work-group float64 sums of the pool stage: (sum, sum of
// squares), or (sum S, sum of x ln x = Q), whence entropy = ln S - Q / S.  Every caller computes it the same way, so
// the score passes of the extended window and the selection agree.  Each wave
// computes it on its own (no LDS, no barrier): a power-of-two group of lanes
// per head adds that head's partials (lane-strided, then a butterfly within
// the group), and each head's rank comes from the group leaders' variances.
__device__ __forceinline__ uint32_t htop_mask(const Problem& P, const double2* stats, int b) {
  const int lane = threadIdx.x & 63;
  const int lph = P.H > 4 ? 8 : P.H > 2 ? 16 : P.H > 1 ? 32 : 64;  // lanes per head
  const int h = lane / lph, j = lane % lph;
  const int ng = pool_groups(P);
  double a1 = 0.0, a2 = 0.0;
  if (h < P.H) {
    const double2* sh = stats + ((int64_t)b * P.H + h) * ng;
    for (int i = j; i < ng; i += lph) {
      const double2 v = sh[i];
      a1 += v.x;
      a2 += v.y;
    }
  }
  for (int o = 1; o < lph; o <<= 1) {
    a1 += __shfl_xor(a1, o);
    a2 += __shfl_xor(a2, o);
  }
  const double mean = a1 / P.Tc;
  // ranking key, lowest first: the variance, or minus the entropy
  const double var = P.criterion ? (a1 > 0.0 ? a2 / a1 - log(a1) : 0.0) : a2 / P.Tc - mean * mean;
  int rank = 0;
  for (int o = 0; o < P.H; ++o) {
    const double vo = __shfl(var, o * lph);
    rank += (vo < var) || (vo == var && o < h);
  }
  const uint64_t sel = __ballot(h < P.H && j == 0 && rank < P.delta_eff);
  uint32_t m = 0;
  for (int g = 0; g < P.H; ++g) m |= (uint32_t)((sel >> (g * lph)) & 1ull) << g;
  return m;
}

// Index of the k-th set bit of m, or -1 when m has at most k set bits.
__device__ __forceinline__ int nth_bit(uint32_t m, int k) {
  for (int i = 0; i < k; ++i) m &= m - 1u;
  return __ffs(m) - 1;
}

}  // namespace kvec
