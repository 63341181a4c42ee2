// C ABI of libkvec: argument validation, workspace layout and launch order.
// Everything here is host code; validation never touches the device.
#include <math.h>
#include <string.h>

#include "kvec_internal.h"

namespace kvec {

int row_blocks_per_tile(int G);  // kvec_score.hip

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

kvec_status make_geometry(const kvec_config* c, Geometry* g) {
  if (!c || !g) return KVEC_ERR_INVALID;
  if (c->batch < 1 || c->n_layers < 1 || c->n_layers > 255) return KVEC_ERR_INVALID;
  if (c->n_kv_heads < 1 || c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads != 0)
    return KVEC_ERR_INVALID;
  if (c->seq_len < 1 || c->seq_len > (1 << 28)) return KVEC_ERR_INVALID;
  if (c->window < 1 || c->window > c->seq_len) return KVEC_ERR_INVALID;
  if (c->window_ext < c->window) return KVEC_ERR_INVALID;
  if (c->budget < c->window) return KVEC_ERR_INVALID;
  if (c->pool_kernel < 1 || (c->pool_kernel % 2) == 0) return KVEC_ERR_INVALID;
  if (c->n_adjust_heads < 0 || c->n_adjust_heads > c->n_kv_heads) return KVEC_ERR_INVALID;
  if (!(c->lambda >= 0.f) || !isfinite(c->lambda)) return KVEC_ERR_INVALID;
  if (!(c->beta >= 0.f && c->beta <= 1.f)) return KVEC_ERR_INVALID;
  if (c->dtype != KVEC_BF16 && c->dtype != KVEC_F32) return KVEC_ERR_INVALID;
  if (c->head_dim < 1) return KVEC_ERR_INVALID;
  const int G = c->n_q_heads / c->n_kv_heads;
  if (c->n_kv_heads > 16) return KVEC_ERR_UNSUPPORTED;
  if (G != 1 && G != 2 && G != 4 && G != 8) return KVEC_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return KVEC_ERR_UNSUPPORTED;
  if ((int64_t)c->budget * c->n_kv_heads > (1 << 28)) return KVEC_ERR_UNSUPPORTED;

  Geometry& x = *g;
  x.batch = c->batch;
  x.layers = c->n_layers;
  x.H = c->n_kv_heads;
  x.HQ = c->n_q_heads;
  x.G = G;
  x.D = c->head_dim;
  x.T = c->seq_len;
  x.O = c->window;
  x.Wn = c->window_ext < c->seq_len ? c->window_ext : c->seq_len;
  x.Tc = c->seq_len - c->window;
  x.B = c->budget;
  x.pool = c->pool_kernel;
  x.delta = c->n_adjust_heads;
  x.lam = c->lambda;
  x.beta = c->beta;
  x.dtype = c->dtype;
  x.M = c->budget - c->window;
  const double kp = floor((double)c->beta * (double)c->budget);
  x.Kp = (int)(kp < (double)x.M ? kp : (double)x.M);
  x.RB = row_blocks_per_tile(G);
  x.WR = 16 * x.RB;
  x.n_rt = (x.Wn + x.WR - 1) / x.WR;
  x.n_rt_base = (x.O + x.WR - 1) / x.WR;
  x.n_kt1 = (x.T + kTilePass1 - 1) / kTilePass1;
  x.n_kt2 = (x.Tc + kTilePass2 - 1) / kTilePass2;
  x.SK = 64;
  while (x.SK > 16 && ((size_t)x.H * x.WR * x.SK + 64 * x.H) * 4 > 65536) x.SK /= 2;
  x.n_pool_blk = (x.Tc + kPoolBlock - 1) / kPoolBlock;
  x.words = (x.T + 63) / 64;
  x.esize = c->dtype == KVEC_BF16 ? 2 : 4;
  x.keep_all = x.T <= x.B;
  return KVEC_OK;
}

Workspace make_workspace(const Geometry& g) {
  Workspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  const size_t bt = (size_t)g.batch, tc = (size_t)(g.Tc > 0 ? g.Tc : 0);
  w.lse_part = take(bt * g.HQ * g.Wn * g.n_kt1 * 8);
  w.lse2 = take(bt * g.HQ * g.Wn * 4);
  w.psum_base = take(bt * g.n_rt * g.H * tc * 4);
  w.psum_all = take(bt * g.n_rt * g.H * tc * 4);
  w.ipart = take(bt * g.n_rt * tc * 4);
  w.p_raw = take(bt * g.H * tc * 4);
  w.p_ext = take(bt * g.H * tc * 4);
  w.imp = take(bt * tc * 4);
  w.pooled = take(bt * g.H * tc * 4);
  w.pooled_ext = take(bt * g.H * tc * 4);
  w.stats = take(bt * g.H * g.n_pool_blk * 16);
  w.use_ext = take(bt * g.H * 4);
  w.keep = take(bt * g.H * ((tc + 31) / 32) * 4);
  w.keys = take(bt * g.H * tc * 4);
  w.total = off;
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

kvec_status dev(hipError_t e) { return e == hipSuccess ? KVEC_OK : KVEC_ERR_DEVICE; }

kvec_status check_ws(const Geometry& g, void* ws, size_t ws_bytes) {
  const Workspace w = make_workspace(g);
  if (ws_bytes < w.total) return KVEC_ERR_WORKSPACE;
  if (w.total > 0 && !aligned16(ws)) return KVEC_ERR_INVALID;
  return KVEC_OK;
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
  if (g.Tc < 1) return KVEC_ERR_INVALID;
  if (!aligned16(q_win) || !aligned16(k) || !strides_ok(q_strides, 3, g.esize) ||
      !strides_ok(k_strides, 3, g.esize) || !p_raw || !p_ext_raw || !imp)
    return KVEC_ERR_INVALID;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  return dev(launch_score(g, q_win, q_strides, k, k_strides, p_raw, p_ext_raw, imp,
                          static_cast<char*>(ws), w, stream, nullptr));
}

kvec_status kvec_select_cover(const kvec_config* cfg, int32_t layer, const float* p_raw,
                              const float* p_ext_raw, const float* imp, uint64_t* cover_bits,
                              int32_t* idx, uint32_t* htop_mask, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (layer < 0 || layer >= g.layers || !cover_bits || !idx) return KVEC_ERR_INVALID;
  if (g.keep_all) return dev(launch_keep_all(g, layer, cover_bits, idx, stream));
  if (!p_raw || !p_ext_raw || !imp) return KVEC_ERR_INVALID;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  return dev(launch_select(g, layer, p_raw, p_ext_raw, imp, cover_bits, idx, htop_mask,
                           static_cast<char*>(ws), w, stream));
}

kvec_status kvec_compact(const kvec_config* cfg, const void* k, const int64_t k_strides[3],
                         const void* v, const int64_t v_strides[3], const int32_t* idx,
                         void* k_out, void* v_out, hipStream_t stream) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 3, g.esize) ||
      !strides_ok(v_strides, 3, g.esize) || !idx || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  const int64_t ks[4] = {0, k_strides[0], k_strides[1], k_strides[2]};
  const int64_t vs[4] = {0, v_strides[0], v_strides[1], v_strides[2]};
  return dev(launch_compact(g, 1, k, ks, v, vs, idx, k_out, v_out, stream));
}

kvec_status kvec_evict_layer(const kvec_config* cfg, int32_t layer, const void* q_win,
                             const int64_t q_strides[3], const void* k, const int64_t k_strides[3],
                             const void* v, const int64_t v_strides[3], uint64_t* cover_bits,
                             int32_t* idx, void* k_out, void* v_out, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (layer < 0 || layer >= g.layers || !cover_bits || !idx) return KVEC_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 3, g.esize) ||
      !strides_ok(v_strides, 3, g.esize) || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && (!aligned16(q_win) || !strides_ok(q_strides, 3, g.esize)))
    return KVEC_ERR_INVALID;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  char* wsb = static_cast<char*>(ws);
  hipError_t e;
  if (g.keep_all) {
    e = launch_keep_all(g, layer, cover_bits, idx, stream);
  } else {
    float* p_raw = reinterpret_cast<float*>(wsb + w.p_raw);
    float* p_ext = reinterpret_cast<float*>(wsb + w.p_ext);
    float* imp = reinterpret_cast<float*>(wsb + w.imp);
    e = launch_score(g, q_win, q_strides, k, k_strides, p_raw, p_ext, imp, wsb, w, stream, nullptr);
    if (e == hipSuccess)
      e = launch_select(g, layer, p_raw, p_ext, imp, cover_bits, idx, nullptr, wsb, w, stream);
  }
  if (e != hipSuccess) return KVEC_ERR_DEVICE;
  const int64_t ks[4] = {0, k_strides[0], k_strides[1], k_strides[2]};
  const int64_t vs[4] = {0, v_strides[0], v_strides[1], v_strides[2]};
  return dev(launch_compact(g, 1, k, ks, v, vs, idx, k_out, v_out, stream));
}

kvec_status kvec_evict_model(const kvec_config* cfg, const void* q_win, const int64_t q_strides[4],
                             const void* k, const int64_t k_strides[4], const void* v,
                             const int64_t v_strides[4], uint64_t* cover_bits, int32_t* idx,
                             void* k_out, void* v_out, void* ws, size_t ws_bytes,
                             hipStream_t stream, hipEvent_t* events) {
  Geometry g;
  kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!cover_bits || !idx) return KVEC_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !strides_ok(k_strides, 4, g.esize) ||
      !strides_ok(v_strides, 4, g.esize) || !aligned16(k_out) || !aligned16(v_out))
    return KVEC_ERR_INVALID;
  if (!g.keep_all && (!aligned16(q_win) || !strides_ok(q_strides, 4, g.esize)))
    return KVEC_ERR_INVALID;
  if ((st = check_ws(g, ws, ws_bytes)) != KVEC_OK) return st;
  const Workspace w = make_workspace(g);
  char* wsb = static_cast<char*>(ws);
  hipError_t e = launch_zero_bits(g, cover_bits, stream);
  float* p_raw = reinterpret_cast<float*>(wsb + w.p_raw);
  float* p_ext = reinterpret_cast<float*>(wsb + w.p_ext);
  float* imp = reinterpret_cast<float*>(wsb + w.imp);
  const int64_t per_layer_idx = (int64_t)g.batch * g.H * g.B;
  for (int l = 0; l < g.layers && e == hipSuccess; ++l) {
    int32_t* idx_l = idx + l * per_layer_idx;
    if (g.keep_all) {
      e = launch_keep_all(g, l, cover_bits, idx_l, stream);
      continue;
    }
    const char* ql = static_cast<const char*>(q_win) + (int64_t)l * q_strides[0] * g.esize;
    const char* kl = static_cast<const char*>(k) + (int64_t)l * k_strides[0] * g.esize;
    e = launch_score(g, ql, q_strides + 1, kl, k_strides + 1, p_raw, p_ext, imp, wsb, w, stream,
                     events ? events + 4 * l : nullptr);
    if (e == hipSuccess)
      e = launch_select(g, l, p_raw, p_ext, imp, cover_bits, idx_l, nullptr, wsb, w, stream);
  }
  if (e == hipSuccess)
    e = launch_compact(g, g.layers, k, k_strides, v, v_strides, idx, k_out, v_out, stream);
  return dev(e);
}

kvec_status kvec_coverage(const kvec_config* cfg, const uint64_t* cover_bits, int32_t upto_layer,
                          int64_t* count_per_seq, hipStream_t stream) {
  Geometry g;
  const kvec_status st = make_geometry(cfg, &g);
  if (st != KVEC_OK) return st;
  if (!cover_bits || !count_per_seq || upto_layer < 0 || upto_layer >= g.layers)
    return KVEC_ERR_INVALID;
  return dev(launch_coverage(g, cover_bits, upto_layer, count_per_seq, stream));
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
