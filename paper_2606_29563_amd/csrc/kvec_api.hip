// C ABI of libkvec: argument validation, workspace layout and call dispatch.
// Everything here is host code; validation never touches the device.
#include <math.h>
#include <string.h>

#include "kvec_internal.h"

namespace kvec {

constexpr size_t kLdsMax = 163840;  // bytes of LDS per work-group on gfx950
constexpr size_t kLdsStatic = 1024; // reserve for the tasks' static shared variables

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

kvec_status make_geometry(const kvec_config* c, Geometry* g) {
  if (!c || !g) return KVEC_ERR_INVALID;
  if (c->batch < 1 || c->n_layers < 1 || c->n_layers > 255) return KVEC_ERR_INVALID;
  if (c->n_kv_heads < 1 || c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads != 0)
    return KVEC_ERR_INVALID;
  if (c->seq_len < 1) return KVEC_ERR_INVALID;
  if (c->window < 1 || c->window > c->seq_len) return KVEC_ERR_INVALID;
  if (c->window_ext < c->window) return KVEC_ERR_INVALID;
  if (c->budget < c->window) return KVEC_ERR_INVALID;
  if (c->pool_kernel < 1 || (c->pool_kernel % 2) == 0) return KVEC_ERR_INVALID;
  if (c->n_adjust_heads < 0 || c->n_adjust_heads > c->n_kv_heads) return KVEC_ERR_INVALID;
  if (!(c->lambda >= 0.f) || !isfinite(c->lambda)) return KVEC_ERR_INVALID;
  if (!(c->beta >= 0.f && c->beta <= 1.f)) return KVEC_ERR_INVALID;
  if (c->dtype != KVEC_BF16 && c->dtype != KVEC_F32) return KVEC_ERR_INVALID;
  if (c->head_criterion != KVEC_HEADS_STD && c->head_criterion != KVEC_HEADS_ENTROPY)
    return KVEC_ERR_INVALID;
  if (c->head_dim < 1) return KVEC_ERR_INVALID;
  const int H = c->n_kv_heads, G = c->n_q_heads / c->n_kv_heads;
  if (H != 1 && H != 2 && H != 4 && H != 8) return KVEC_ERR_UNSUPPORTED;
  if (G < 1 || G > 8) return KVEC_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return KVEC_ERR_UNSUPPORTED;
  if (c->seq_len > (1 << 18)) return KVEC_ERR_UNSUPPORTED;
  if (c->pool_kernel > 63) return KVEC_ERR_UNSUPPORTED;
  if ((int64_t)c->budget * H > (1 << 26)) return KVEC_ERR_UNSUPPORTED;

  Problem& x = g->p;
  memset(&x, 0, sizeof(x));
  x.batch = c->batch;
  x.L = c->n_layers;
  x.H = H;
  x.HQ = c->n_q_heads;
  x.G = G;
  x.D = c->head_dim;
  x.T = c->seq_len;
  x.O = c->window;
  x.Wn = c->window_ext < c->seq_len ? c->window_ext : c->seq_len;
  x.Tc = c->seq_len - c->window;
  x.B = c->budget;
  x.M = c->budget - c->window;
  const double kp = floor((double)c->beta * (double)c->budget);
  x.Kp = (int)(kp < (double)x.M ? kp : (double)x.M);
  x.pool = c->pool_kernel;
  x.delta_eff = x.Wn > x.O ? c->n_adjust_heads : 0;
  x.lam = c->lambda;
  x.criterion = c->head_criterion;
  x.sc = (float)(1.4426950408889634 / sqrt((double)x.D));
  x.inv_go = (float)(1.0 / ((double)G * x.O));
  x.inv_gwn = (float)(1.0 / ((double)G * x.Wn));
  x.WR = 16 * row_blocks_per_tile(G);
  x.n_rt = (x.Wn + x.WR - 1) / x.WR;
  x.n_rt_base = (x.O + x.WR - 1) / x.WR;
  x.nsum = x.O % x.WR == 0 ? 1 : 2;
  const int tpw = 8 / H;
  x.n_rtg = (x.n_rt + tpw - 1) / tpw;
  // Keys per score work-group: 512 from T = 16384 on, smaller for shorter
  // prefixes (at least 128) so that their launches fill more CUs with
  // shorter work-groups: the largest power of two <= T / 32 in [128, 512].
  int tile_target = kTileMax;
  while (tile_target > kTileMin && tile_target * 32 > x.T) tile_target /= 2;
  x.tile1 = tile_target;
  x.n_kt1 = (x.T + x.tile1 - 1) / x.tile1;
  // pass-2 LDS: the key ring plus, per row tile, the running max over heads
  // (SK keys per exchange period), the staged per-key sums and importance of
  // the key tile.  Prefer the target tile (fewer work-groups, less fixed
  // cost per key) with periods of at least 32 keys at 512, then the widest
  // period; halve the tile only when the LDS budget requires it.
  const size_t ring = key_ring_bytes(c->dtype == KVEC_BF16 ? 2 : 4, x.D);
  // row tiles of the layer pipeline: the last-O rows for every head, the
  // remaining extended-window rows for the delta_eff heads of H_top
  x.n_rtg_base = (x.n_rt_base + tpw - 1) / tpw;
  const int n_rt_ext = x.n_rt - x.n_rt_base;
  x.n_rt_x = x.delta_eff > 0 && n_rt_ext > 0 ? n_rt_ext : 0;
  auto lds_p2 = [&](int sk, int tile) {
    const size_t all = (size_t)tpw * p2_slot_floats(H, x.WR, sk, tile, H > 1, x.nsum);
    // EXT passes: one task per wave, each wave its own slot of one head
    const size_t ext = x.n_rt_x > 0 ? (size_t)8 * p2_slot_floats(1, x.WR, sk, tile, false, x.nsum) : 0;
    return ring + (all > ext ? all : ext) * 4;
  };
  const size_t lds_cap = kLdsMax - kLdsStatic;
  x.tile2 = 0;
  for (int tile = tile_target; tile >= kTileMin && !x.tile2; tile /= 2)
    for (int sk = tile; sk >= (tile == kTileMax ? 32 : 16); sk = (sk == tile && tile > 128) ? 128 : sk / 2)
      if (lds_p2(sk, tile) <= lds_cap) {
        x.tile2 = tile;
        x.SK = sk;  // a power of two
        x.sk_shift = __builtin_ctz((unsigned)sk);
        break;
      }
  if (!x.tile2) return KVEC_ERR_UNSUPPORTED;
  x.n_kt2 = (x.Tc + x.tile2 - 1) / x.tile2;
  x.n_pool = (x.Tc + kPoolChunk - 1) / kPoolChunk;
  x.n_prep = (x.Tc + kPrepChunk - 1) / kPrepChunk;
  x.words = (x.T + 63) / 64;
  x.esize = c->dtype == KVEC_BF16 ? 2 : 4;
  const int64_t chunks = (int64_t)H * x.B * (x.D * x.esize / 16);
  x.n_gather = (int)((chunks + 4 * kThreads - 1) / (4 * kThreads));
  // selection task LDS: 2048-bin histogram, 32 ints, member offsets, then
  // four 4-byte arrays per member
  const size_t sel_fixed = 2048 * 4 + 32 * 4 + (size_t)((x.n_prep + 1 + 3) & ~3) * 4;
  x.mcap = (int)(((kLdsMax - kLdsStatic - sel_fixed) / 16) & ~(size_t)63);
  g->keep_all = x.T <= x.B;
  return KVEC_OK;
}

Workspace make_workspace(const Geometry& g) {
  const Problem& P = g.p;
  Workspace w;
  memset(&w, 0, sizeof(w));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  const size_t bt = (size_t)P.batch, tc = (size_t)(P.Tc > 0 ? P.Tc : 0);
  // one ring slot
  w.lse_part = take(bt * P.HQ * P.Wn * P.n_kt1 * 8);
  w.lse2 = take(bt * P.HQ * P.Wn * 4);
  w.psum_base = take(bt * P.n_rt * P.H * tc * 4);
  w.psum_all = take(bt * P.n_rt * P.H * tc * 4);
  w.ipart = take(bt * P.n_rt * tc * 4);
  w.imp = take(bt * tc * 4);
  w.pooled = take(bt * P.H * tc * 4);
  w.pooled_ext = take(bt * P.H * tc * 4);
  w.stats = take(bt * P.H * pool_groups(P) * 16);
  w.hist = take(bt * 2 * P.H * kHistBins * 4);
  w.mem_t = take(bt * P.H * tc * 4);
  w.mem_ps = take(bt * P.H * tc * 4);
  w.mem_i = take(bt * P.H * tc * 4);
  w.mem_n = take(bt * P.H * P.n_prep * 4);
  w.slot_bytes = off;
  off = w.slot_bytes * kRing;
  w.counts_stride = align256(bt * P.T);
  w.counts = take(2 * w.counts_stride);
  w.spill_stride = align256(bt * P.H * tc * 4);
  w.spill = take(4 * w.spill_stride);
  w.total = off;
  // dynamic LDS: the largest task
  const int tpw = 8 / P.H;
  const size_t p2_all = (size_t)tpw * p2_slot_floats(P.H, P.WR, P.SK, P.tile2, P.H > 1, P.nsum);
  const size_t p2_ext = P.n_rt_x > 0 ? (size_t)8 * p2_slot_floats(1, P.WR, P.SK, P.tile2, false, P.nsum) : 0;
  const size_t lds_p2 = key_ring_bytes(P.esize, P.D) + (p2_all > p2_ext ? p2_all : p2_ext) * 4;
  const size_t lds_pool = (size_t)(2 * (kPoolPer * kPoolChunk + 64) + 2 * kHistBins) * 4 + kPoolPer * 16;
  const size_t lds_prep = 256;
  const size_t lds_sel = 2048 * 4 + 32 * 4 + (size_t)((P.n_prep + 1 + 3) & ~3) * 4 +
                         (size_t)16 * P.mcap;
  size_t lds = lds_p2;
  if (lds_pool > lds) lds = lds_pool;
  if (lds_prep > lds) lds = lds_prep;
  if (lds_sel > lds) lds = lds_sel;
  w.lds_bytes = (lds + 15) & ~(size_t)15;
  return w;
}

}  // namespace kvec

using namespace kvec;

namespace {

bool aligned16(const void* p) { return p && ((uintptr_t)p & 15u) == 0; }

bool strides_ok(const int64_t* s, int n, int esize) {
  if (!s) return false;
  for (int i = 0; i < n; ++i)
    if (s[i] < 0 || (s[i] * esize) % 16 != 0) return false;
  return true;
}

// The score passes address the keys of one (batch, head) with 32-bit buffer
// offsets: T rows of k_strides[t] elements must span less than 2 GiB.
bool keys_addressable(const Problem& P, int64_t t_stride) {
  return (int64_t)P.T * t_stride * P.esize < ((int64_t)1 << 31);
}

kvec_status dev(hipError_t e) { return e == hipSuccess ? KVEC_OK : KVEC_ERR_DEVICE; }

// Caller-supplied row normalisers: fp32, 4-byte aligned, non-negative strides.
bool lse_ok(const float* lse, const int64_t* s, int n) {
  if (!lse || ((uintptr_t)lse & 3u) != 0 || !s) return false;
  for (int i = 0; i < n; ++i)
    if (s[i] < 0) return false;
  return true;
}

kvec_status check_ws(const Geometry& g, void* ws, size_t ws_bytes) {
  const Workspace w = make_workspace(g);
  if (ws_bytes < w.total) return KVEC_ERR_WORKSPACE;
  if (w.total > 0 && !aligned16(ws)) return KVEC_ERR_INVALID;
  return KVEC_OK;
}

void strides4(int64_t out[4], const int64_t* s3) {
  out[0] = 0;
  out[1] = s3[0];
  out[2] = s3[1];
  out[3] = s3[2];
}

}  // namespace

extern "C" {

kvec_status kvec_workspace_size(const kvec_config* cfg, size_t* bytes) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!bytes) return KVEC_ERR_INVALID;
  *bytes = make_workspace(g).total;
  return KVEC_OK;
}

kvec_status kvec_score(const kvec_config* cfg, const void* q_win, const int64_t q_strides[3],
                       const void* k, const int64_t k_strides[3], float* p_raw, float* p_ext_raw,
                       float* imp, void* ws, size_t ws_bytes, hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (g.p.Tc < 1) return KVEC_ERR_INVALID;
  if (!aligned16(q_win) || !aligned16(k) || !strides_ok(q_strides, 3, g.p.esize) ||
      !strides_ok(k_strides, 3, g.p.esize) || !p_raw || !p_ext_raw || !imp)
    return KVEC_ERR_INVALID;
  if (!keys_addressable(g.p, k_strides[2])) return KVEC_ERR_UNSUPPORTED;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  return dev(run_score(g, q_win, q_strides, k, k_strides, nullptr, nullptr, p_raw, p_ext_raw, imp,
                       static_cast<char*>(ws), w, stream));
}

kvec_status kvec_score_lse(const kvec_config* cfg, const void* q_win, const int64_t q_strides[3],
                           const float* lse, const int64_t lse_strides[2], const void* k,
                           const int64_t k_strides[3], float* p_raw, float* p_ext_raw, float* imp,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (g.p.Tc < 1) return KVEC_ERR_INVALID;
  if (!aligned16(q_win) || !aligned16(k) || !strides_ok(q_strides, 3, g.p.esize) ||
      !strides_ok(k_strides, 3, g.p.esize) || !p_raw || !p_ext_raw || !imp)
    return KVEC_ERR_INVALID;
  if (!lse_ok(lse, lse_strides, 2)) return KVEC_ERR_INVALID;
  if (!keys_addressable(g.p, k_strides[2])) return KVEC_ERR_UNSUPPORTED;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  return dev(run_score(g, q_win, q_strides, k, k_strides, lse, lse_strides, p_raw, p_ext_raw, imp,
                       static_cast<char*>(ws), w, stream));
}

kvec_status kvec_select_cover(const kvec_config* cfg, int32_t layer, const float* p_raw,
                              const float* p_ext_raw, const float* imp, uint64_t* cover_bits,
                              int32_t* idx, uint32_t* htop_mask, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (layer < 0 || layer >= g.p.L || !cover_bits || !idx) return KVEC_ERR_INVALID;
  if (g.keep_all) return dev(run_keep_all(g, layer, cover_bits, idx, stream));
  if (!p_raw || !p_ext_raw || !imp) return KVEC_ERR_INVALID;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  return dev(run_select(g, layer, p_raw, p_ext_raw, imp, cover_bits, idx, htop_mask,
                        static_cast<char*>(ws), w, stream));
}

kvec_status kvec_compact(const kvec_config* cfg, const void* k, const int64_t k_strides[3],
                         const void* v, const int64_t v_strides[3], const int32_t* idx,
                         void* k_out, void* v_out, hipStream_t stream) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 3, g.p.esize) ||
      !strides_ok(v_strides, 3, g.p.esize) || !idx || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  ModelIO m;
  memset(&m, 0, sizeof(m));
  m.k = k;
  m.v = v;
  strides4(m.ks, k_strides);
  strides4(m.vs, v_strides);
  m.idx = const_cast<int32_t*>(idx);
  m.k_out = k_out;
  m.v_out = v_out;
  return dev(run_compact(g, 1, m, stream));
}

}  // extern "C"

namespace {

kvec_status evict_layer(const kvec_config* cfg, int32_t layer, const void* q_win,
                        const int64_t q_strides[3], const float* lse, const int64_t lse_strides[2],
                        const void* k, const int64_t k_strides[3], const void* v,
                        const int64_t v_strides[3], uint64_t* cover_bits, int32_t* idx,
                        void* k_out, void* v_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (layer < 0 || layer >= g.p.L || !cover_bits || !idx) return KVEC_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 3, g.p.esize) ||
      !strides_ok(v_strides, 3, g.p.esize) || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && (!aligned16(q_win) || !strides_ok(q_strides, 3, g.p.esize)))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && !keys_addressable(g.p, k_strides[2])) return KVEC_ERR_UNSUPPORTED;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  ModelIO m;
  memset(&m, 0, sizeof(m));
  m.q = q_win;
  m.k = k;
  m.v = v;
  if (q_strides) strides4(m.qs, q_strides);
  strides4(m.ks, k_strides);
  strides4(m.vs, v_strides);
  m.bits = cover_bits;
  m.idx = idx;
  m.k_out = k_out;
  m.v_out = v_out;
  m.lse = lse;
  if (lse) {
    m.ls[1] = lse_strides[0];
    m.ls[2] = lse_strides[1];
  }
  if (g.keep_all) {
    const hipError_t e = run_keep_all(g, layer, cover_bits, idx, stream);
    if (e != hipSuccess) return KVEC_ERR_DEVICE;
    return dev(run_compact(g, 1, m, stream));
  }
  return dev(run_evict_layer(g, layer, m, static_cast<char*>(ws), w, stream));
}

}  // namespace

extern "C" {

kvec_status kvec_evict_layer(const kvec_config* cfg, int32_t layer, const void* q_win,
                             const int64_t q_strides[3], const void* k, const int64_t k_strides[3],
                             const void* v, const int64_t v_strides[3], uint64_t* cover_bits,
                             int32_t* idx, void* k_out, void* v_out, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  return evict_layer(cfg, layer, q_win, q_strides, nullptr, nullptr, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream);
}

kvec_status kvec_evict_layer_lse(const kvec_config* cfg, int32_t layer, const void* q_win,
                                 const int64_t q_strides[3], const float* lse,
                                 const int64_t lse_strides[2], const void* k,
                                 const int64_t k_strides[3], const void* v,
                                 const int64_t v_strides[3], uint64_t* cover_bits, int32_t* idx,
                                 void* k_out, void* v_out, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if (!lse_ok(lse, lse_strides, 2)) return KVEC_ERR_INVALID;
  return evict_layer(cfg, layer, q_win, q_strides, lse, lse_strides, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream);
}

}  // extern "C"

namespace {

kvec_status evict_model(const kvec_config* cfg, const void* q_win, const int64_t q_strides[4],
                        const float* lse, const int64_t lse_strides[3], const void* k,
                        const int64_t k_strides[4], const void* v, const int64_t v_strides[4],
                        uint64_t* cover_bits, int32_t* idx, void* k_out, void* v_out, void* ws,
                        size_t ws_bytes, hipStream_t stream, hipEvent_t* events,
                        const ModelIO* scores = nullptr) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!cover_bits || !idx) return KVEC_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 4, g.p.esize) ||
      !strides_ok(v_strides, 4, g.p.esize) || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && (!aligned16(q_win) || !strides_ok(q_strides, 4, g.p.esize)))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && !keys_addressable(g.p, k_strides[3])) return KVEC_ERR_UNSUPPORTED;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  ModelIO m;
  memset(&m, 0, sizeof(m));
  m.q = q_win;
  m.k = k;
  m.v = v;
  for (int i = 0; i < 4; ++i) {
    m.qs[i] = q_strides ? q_strides[i] : 0;
    m.ks[i] = k_strides[i];
    m.vs[i] = v_strides[i];
  }
  m.bits = cover_bits;
  m.idx = idx;
  m.k_out = k_out;
  m.v_out = v_out;
  m.lse = lse;
  if (lse)
    for (int i = 0; i < 3; ++i) m.ls[i] = lse_strides[i];
  if (scores) {
    m.sc_p = scores->sc_p;
    m.sc_pe = scores->sc_pe;
    m.sc_imp = scores->sc_imp;
    m.sc_htop = scores->sc_htop;
  }
  if (g.keep_all) {
    for (int l = 0; l < g.p.L; ++l) {
      const hipError_t e = run_keep_all(g, l, cover_bits, idx + (int64_t)l * g.p.batch * g.p.H * g.p.B,
                                        stream);
      if (e != hipSuccess) return KVEC_ERR_DEVICE;
    }
    return dev(run_compact(g, g.p.L, m, stream));
  }
  return dev(run_model(g, m, static_cast<char*>(ws), w, stream, events));
}

}  // namespace

extern "C" {

kvec_status kvec_evict_model(const kvec_config* cfg, const void* q_win, const int64_t q_strides[4],
                             const void* k, const int64_t k_strides[4], const void* v,
                             const int64_t v_strides[4], uint64_t* cover_bits, int32_t* idx,
                             void* k_out, void* v_out, void* ws, size_t ws_bytes,
                             hipStream_t stream, hipEvent_t* events) {
  return evict_model(cfg, q_win, q_strides, nullptr, nullptr, k, k_strides, v, v_strides, cover_bits,
                     idx, k_out, v_out, ws, ws_bytes, stream, events);
}

kvec_status kvec_evict_model_lse(const kvec_config* cfg, const void* q_win,
                                 const int64_t q_strides[4], const float* lse,
                                 const int64_t lse_strides[3], const void* k,
                                 const int64_t k_strides[4], const void* v,
                                 const int64_t v_strides[4], uint64_t* cover_bits, int32_t* idx,
                                 void* k_out, void* v_out, void* ws, size_t ws_bytes,
                                 hipStream_t stream, hipEvent_t* events) {
  if (!lse_ok(lse, lse_strides, 3)) return KVEC_ERR_INVALID;
  return evict_model(cfg, q_win, q_strides, lse, lse_strides, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream, events);
}

kvec_status kvec_evict_model_scores(const kvec_config* cfg, const void* q_win,
                                    const int64_t q_strides[4], const void* k,
                                    const int64_t k_strides[4], const void* v,
                                    const int64_t v_strides[4], uint64_t* cover_bits, int32_t* idx,
                                    void* k_out, void* v_out, float* p_raw_out, float* p_ext_out,
                                    float* imp_out, uint32_t* htop_out, void* ws, size_t ws_bytes,
                                    hipStream_t stream) {
  const auto f4 = [](const void* p) { return p && ((uintptr_t)p & 3u) == 0; };
  if (!f4(p_raw_out) || !f4(p_ext_out) || !f4(imp_out) || !f4(htop_out)) return KVEC_ERR_INVALID;
  ModelIO sc;
  memset(&sc, 0, sizeof(sc));
  sc.sc_p = p_raw_out;
  sc.sc_pe = p_ext_out;
  sc.sc_imp = imp_out;
  sc.sc_htop = htop_out;
  return evict_model(cfg, q_win, q_strides, nullptr, nullptr, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream, nullptr, &sc);
}

}  // extern "C"

namespace {

// n_steps independent steps in one pipeline (lse null: the two-pass path).
kvec_status evict_steps(const kvec_config* cfg, int32_t n_steps, const void* q_win,
                        const int64_t q_strides[5], const float* lse, const int64_t lse_strides[4],
                        const void* k, const int64_t k_strides[5], const void* v,
                        const int64_t v_strides[5], uint64_t* cover_bits, int32_t* idx,
                        void* k_out, void* v_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  const Problem& P = g.p;
  if (n_steps < 1 || (int64_t)n_steps * P.L > (1 << 20) || !cover_bits || !idx)
    return KVEC_ERR_INVALID;
  if (!q_strides || !k_strides || !v_strides) return KVEC_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 5, P.esize) ||
      !strides_ok(v_strides, 5, P.esize) || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && (!aligned16(q_win) || !strides_ok(q_strides, 5, P.esize)))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && !keys_addressable(P, k_strides[4])) return KVEC_ERR_UNSUPPORTED;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  // per-step output sizes (elements; words for the bitmap)
  const int64_t bits_step = (int64_t)P.batch * P.L * P.words;
  const int64_t idx_step = (int64_t)P.L * P.batch * P.H * P.B;
  const int64_t out_step = idx_step * P.D;
  if (g.keep_all) {
    // nothing to score: each step is a keep-everything step of its own
    for (int s = 0; s < n_steps; ++s) {
      const char* qs = static_cast<const char*>(q_win);
      st = kvec_evict_model(cfg, qs ? qs + (int64_t)s * q_strides[0] * P.esize : nullptr, q_strides + 1,
                            static_cast<const char*>(k) + (int64_t)s * k_strides[0] * P.esize,
                            k_strides + 1,
                            static_cast<const char*>(v) + (int64_t)s * v_strides[0] * P.esize,
                            v_strides + 1, cover_bits + s * bits_step, idx + s * idx_step,
                            static_cast<char*>(k_out) + s * out_step * P.esize,
                            static_cast<char*>(v_out) + s * out_step * P.esize, ws, ws_bytes, stream,
                            nullptr);
      if (st != KVEC_OK) return st;
    }
    return KVEC_OK;
  }
  const Workspace w = make_workspace(g);
  ModelIO m;
  memset(&m, 0, sizeof(m));
  m.q = q_win;
  m.k = k;
  m.v = v;
  for (int i = 0; i < 4; ++i) {
    m.qs[i] = q_strides[i + 1];
    m.ks[i] = k_strides[i + 1];
    m.vs[i] = v_strides[i + 1];
  }
  if (lse) {
    m.lse = lse;
    for (int i = 0; i < 3; ++i) m.ls[i] = lse_strides[i + 1];
    m.lse_step = lse_strides[0];
  }
  m.bits = cover_bits;
  m.idx = idx;
  m.k_out = k_out;
  m.v_out = v_out;
  m.n_steps = n_steps;
  m.q_step = q_strides[0];
  m.k_step = k_strides[0];
  m.v_step = v_strides[0];
  m.bits_step = bits_step;
  m.idx_step = idx_step;
  m.out_step = out_step;
  return dev(run_model(g, m, static_cast<char*>(ws), w, stream, nullptr));
}

}  // namespace

extern "C" {

kvec_status kvec_evict_model_steps(const kvec_config* cfg, int32_t n_steps, const void* q_win,
                                   const int64_t q_strides[5], const void* k,
                                   const int64_t k_strides[5], const void* v,
                                   const int64_t v_strides[5], uint64_t* cover_bits, int32_t* idx,
                                   void* k_out, void* v_out, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  return evict_steps(cfg, n_steps, q_win, q_strides, nullptr, nullptr, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream);
}

kvec_status kvec_evict_model_lse_steps(const kvec_config* cfg, int32_t n_steps, const void* q_win,
                                       const int64_t q_strides[5], const float* lse,
                                       const int64_t lse_strides[4], const void* k,
                                       const int64_t k_strides[5], const void* v,
                                       const int64_t v_strides[5], uint64_t* cover_bits,
                                       int32_t* idx, void* k_out, void* v_out, void* ws,
                                       size_t ws_bytes, hipStream_t stream) {
  if (!lse_ok(lse, lse_strides, 4)) return KVEC_ERR_INVALID;
  return evict_steps(cfg, n_steps, q_win, q_strides, lse, lse_strides, k, k_strides, v, v_strides,
                     cover_bits, idx, k_out, v_out, ws, ws_bytes, stream);
}

kvec_status kvec_coverage(const kvec_config* cfg, const uint64_t* cover_bits, int32_t upto_layer,
                          int64_t* count_per_seq, hipStream_t stream) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!cover_bits || !count_per_seq || upto_layer < 0 || upto_layer >= g.p.L)
    return KVEC_ERR_INVALID;
  return dev(run_coverage(g, cover_bits, upto_layer, count_per_seq, stream));
}

int32_t kvec_profile_points(const kvec_config* cfg) {
  Geometry g;
  if (make_geometry(cfg, &g) != KVEC_OK) return -1;
  return g.keep_all ? 0 : g.p.L + kPipeDepth + 1;
}

kvec_status kvec_decode_workspace_size(const kvec_config* cfg, int32_t n_ctx, size_t* bytes) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!bytes || n_ctx < 1 || n_ctx > (1 << 20)) return KVEC_ERR_INVALID;
  *bytes = decode_plan(g.p, n_ctx).ws_bytes;
  return KVEC_OK;
}

}  // extern "C"

namespace {

// Validation shared by both decode entry points; fills the plan.
kvec_status decode_check(const kvec_config* cfg, Geometry* g, const void* q,
                         const int64_t q_strides[2], const void* k_cache, const void* v_cache,
                         const int64_t cache_strides[2], int32_t n_ctx, const int32_t* idx,
                         const float* out, DecodePlan* pl) {
  const kvec_status st = make_geometry(cfg, g);
  if (st != KVEC_OK) return st;
  if (n_ctx < 1 || n_ctx > (1 << 20) || (idx && n_ctx < g->p.B)) return KVEC_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !out ||
      ((uintptr_t)out & 3u) != 0 || !strides_ok(q_strides, 2, g->p.esize) ||
      !strides_ok(cache_strides, 2, g->p.esize))
    return KVEC_ERR_INVALID;
  *pl = decode_plan(g->p, n_ctx);
  return KVEC_OK;
}

}  // namespace

extern "C" {

kvec_status kvec_decode_attention(const kvec_config* cfg, const void* q, const int64_t q_strides[2],
                                  const void* k_cache, const void* v_cache,
                                  const int64_t cache_strides[2], int32_t n_ctx,
                                  const int32_t* idx, float* out, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  Geometry g;
  DecodePlan pl;
  const kvec_status st =
      decode_check(cfg, &g, q, q_strides, k_cache, v_cache, cache_strides, n_ctx, idx, out, &pl);
  if (st != KVEC_OK) return st;
  if (ws_bytes < pl.ws_bytes) return KVEC_ERR_WORKSPACE;
  if (!aligned16(ws)) return KVEC_ERR_INVALID;
  return dev(run_decode(g, q, q_strides, k_cache, v_cache, cache_strides, n_ctx, idx, out, ws,
                        stream));
}

kvec_status kvec_decode_attention_noalloc(const kvec_config* cfg, const void* q,
                                          const int64_t q_strides[2], const void* k_cache,
                                          const void* v_cache, const int64_t cache_strides[2],
                                          int32_t n_ctx, const int32_t* idx, float* out,
                                          hipStream_t stream) {
  Geometry g;
  DecodePlan pl;
  const kvec_status st =
      decode_check(cfg, &g, q, q_strides, k_cache, v_cache, cache_strides, n_ctx, idx, out, &pl);
  if (st != KVEC_OK) return st;
  // the partial states must fit the fixed scratch (checked before any device call)
  if (pl.ws_bytes > kDecodeScratchBytes) return KVEC_ERR_WORKSPACE;
  void* scratch = nullptr;
  if (decode_scratch(&scratch) != hipSuccess) return KVEC_ERR_DEVICE;
  return dev(run_decode(g, q, q_strides, k_cache, v_cache, cache_strides, n_ctx, idx, out,
                        scratch, stream));
}

int32_t kvec_profile_points_lse(const kvec_config* cfg) {
  Geometry g;
  if (make_geometry(cfg, &g) != KVEC_OK) return -1;
  return g.keep_all ? 0 : g.p.L + kPipeDepthLse + 1;
}

const char* kvec_status_string(kvec_status s) {
  switch (s) {
    case KVEC_OK: return "ok";
    case KVEC_ERR_INVALID: return "invalid argument";
    case KVEC_ERR_UNSUPPORTED: return "unsupported configuration";
    case KVEC_ERR_WORKSPACE: return "workspace too small";
    case KVEC_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

}  // extern "C"
