// Host sanitizer run of the seeded input generator (synth/synth.c) and the
// C++ oracle (oracle/kvec_oracle.cpp): small shapes through every entry
// point, including sliced generation, the keep-everything case, empty
// selections, padding indices and a head with no valid decode row.
// tests/test_sanitize.py builds it with -fsanitize=address,undefined and
// no recovery, so any report ends the run with a non-zero status.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

extern "C" {
typedef struct synth_cfg {
  uint64_t seed;
  int32_t n_layers, batch, n_kv_heads, n_q_heads, head_dim;
  int32_t seq_len;
  int32_t window;
  int32_t window_ext;
  int32_t dtype;
  int32_t rope;
  double rope_theta;
  int32_t hh_count;
  int32_t hh_shared;
  double hh_scale;
  int32_t sink_count;
  double sink_scale;
  int32_t zipf_clusters;
  double zipf_s;
} synth_cfg;
void synth_keys(const synth_cfg* c, int layer, int b, int h0, int h1, int t0, int t1, void* out);
void synth_values(const synth_cfg* c, int layer, int b, int h0, int h1, int t0, int t1, void* out);
void synth_queries(const synth_cfg* c, int layer, int b, int j0, int j1, void* out);
int synth_hh_positions(const synth_cfg* c, int layer, int b, int h, int32_t* out, int cap);

void ko_window_scores(const double* q, const double* k, int hq, int hkv, int wn, int T, int d,
                      int O, int full, double* p, double* pe, double* imp, int threads);
void ko_window_lse(const double* q, const double* k, int hq, int hkv, int wn, int T, int d,
                   double* lse, int threads);
int ko_select_layer(const float* p_raw, const float* p_ext, const float* imp, const int64_t* n_t,
                    int layer, int H, int T, int window, int window_ext, int budget,
                    int pool_kernel, int delta, float lam, float beta, int entropy,
                    int32_t* idx, int64_t* htop, double* sigma, uint8_t* keep, float* p_sel,
                    float* p_adj, uint8_t* bits);
void ko_counts_from_bits(const uint8_t* bits, int n_layers, int T, int64_t* out);
int64_t ko_coverage_count(const uint8_t* bits, int n_layers, int T);
void ko_gather_rows(const uint8_t* x, const int32_t* idx, int H, int T, int B, int row_bytes,
                    uint8_t* out);
void ko_decode_attention(const double* q, const double* k, const double* v, const uint8_t* valid,
                         int hq, int hkv, int n, int d, double* out);
}

static int failures = 0;
#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      ++failures;                                                  \
    }                                                              \
  } while (0)

static double elem(const std::vector<uint8_t>& buf, int dtype, size_t i) {
  if (dtype == 1) {
    float f;
    std::memcpy(&f, buf.data() + 4 * i, 4);
    return f;
  }
  uint16_t u;
  std::memcpy(&u, buf.data() + 2 * i, 2);
  const uint32_t x = (uint32_t)u << 16;
  float f;
  std::memcpy(&f, &x, 4);
  return f;
}

static void run_shape(int dtype, int kv, int qh, int d, int T, int O, int Oe, int budget) {
  synth_cfg c;
  std::memset(&c, 0, sizeof(c));
  c.seed = 11 + dtype;
  c.n_layers = 3;
  c.batch = 2;
  c.n_kv_heads = kv;
  c.n_q_heads = qh;
  c.head_dim = d;
  c.seq_len = T;
  c.window = O;
  c.window_ext = Oe;
  c.dtype = dtype;
  c.rope = 1;
  c.rope_theta = 10000.0;
  c.hh_count = 6;
  c.hh_shared = 2;
  c.hh_scale = 2.0;
  c.sink_count = 2;
  c.sink_scale = 3.0;
  c.zipf_clusters = 3;
  c.zipf_s = 1.1;
  const size_t es = dtype == 1 ? 4 : 2;
  const int wn = Oe < T ? Oe : T;
  std::vector<uint8_t> kb((size_t)kv * T * d * es), vb(kb.size()), qb((size_t)qh * wn * d * es);
  std::vector<uint8_t> part((size_t)kv * T * d * es);
  int32_t pos[4];
  const int npos = synth_hh_positions(&c, 1, 1, kv - 1, pos, 4);
  CHECK(npos >= 0);

  std::vector<double> q((size_t)qh * wn * d), k((size_t)kv * T * d), v(k.size());
  const int H = kv, Tc = T - O;
  std::vector<uint8_t> bits_all;  // [layer][T] of sequence 0
  for (int layer = 0; layer < c.n_layers; ++layer) {
    for (int b = 0; b < c.batch; ++b) {
      synth_keys(&c, layer, b, 0, kv, 0, T, kb.data());
      synth_values(&c, layer, b, 0, kv, 0, T, vb.data());
      synth_queries(&c, layer, b, 0, qh, qb.data());
      // a slice equals the same part of the whole
      const int h0 = kv > 1 ? 1 : 0, t0 = T / 5, t1 = T / 2;
      synth_keys(&c, layer, b, h0, kv, t0, t1, part.data());
      for (int h = h0; h < kv; ++h)
        for (int t = t0; t < t1; ++t)
          CHECK(std::memcmp(part.data() + (((size_t)(h - h0) * (t1 - t0) + (t - t0)) * d) * es,
                            kb.data() + (((size_t)h * T + t) * d) * es, d * es) == 0);
    }
    for (size_t i = 0; i < q.size(); ++i) q[i] = elem(qb, dtype, i);
    for (size_t i = 0; i < k.size(); ++i) {
      k[i] = elem(kb, dtype, i);
      v[i] = elem(vb, dtype, i);
      CHECK(std::isfinite(k[i]) && std::isfinite(v[i]));
    }
    std::vector<double> p((size_t)H * T), pe(p.size()), imp(T), lse((size_t)qh * wn);
    ko_window_scores(q.data(), k.data(), qh, kv, wn, T, d, O, 1, p.data(), pe.data(), imp.data(), 2);
    ko_window_scores(q.data(), k.data(), qh, kv, wn, T, d, O, 0, p.data(), pe.data(), imp.data(), 3);
    ko_window_lse(q.data(), k.data(), qh, kv, wn, T, d, lse.data(), 2);
    std::vector<float> pf((size_t)H * Tc), pef(pf.size()), impf(Tc);
    for (int h = 0; h < H; ++h)
      for (int t = 0; t < Tc; ++t) {
        pf[(size_t)h * Tc + t] = (float)p[(size_t)h * Tc + t];
        pef[(size_t)h * Tc + t] = (float)pe[(size_t)h * Tc + t];
      }
    for (int t = 0; t < Tc; ++t) impf[t] = (float)imp[t];
    std::vector<int64_t> nt(T, 0);
    if (layer > 0) ko_counts_from_bits(bits_all.data(), layer, T, nt.data());
    for (int pol = 0; pol < 3; ++pol) {
      const int B = pol == 2 ? T + 5 : budget;
      std::vector<int32_t> idx((size_t)H * B);
      std::vector<int64_t> htop(H);
      std::vector<double> sigma(H);
      std::vector<uint8_t> keep((size_t)H * (Tc > 0 ? Tc : 1)), bits(T);
      std::vector<float> ps(keep.size()), pa(keep.size());
      const int nh = ko_select_layer(pf.data(), pef.data(), impf.data(), nt.data(), layer, H, T, O, Oe, B,
                                     pol == 1 ? 1 : 7, pol == 1 ? 0 : 1, 1.0f, 0.25f, pol == 1,
                                     idx.data(), htop.data(), sigma.data(), keep.data(), ps.data(),
                                     pa.data(), bits.data());
      CHECK(nh >= 0 && nh <= H);
      for (size_t i = 0; i < idx.size(); ++i) CHECK(idx[i] >= -1 && idx[i] < T);
      if (pol == 0) bits_all.insert(bits_all.end(), bits.begin(), bits.end());
      // the cache store, with the padding indices of the keep-all case
      std::vector<uint8_t> out((size_t)H * B * d * es);
      ko_gather_rows(kb.data(), idx.data(), H, T, B, (int)(d * es), out.data());
    }
    CHECK(ko_coverage_count(bits_all.data(), layer + 1, T) <= T);
    // decode over the kept rows; the last head sees no valid row
    std::vector<double> qd((size_t)qh * d), od(qd.size());
    for (size_t i = 0; i < qd.size(); ++i) qd[i] = q[i];
    std::vector<uint8_t> valid((size_t)kv * T, 1);
    for (int t = 0; t < T; ++t) valid[(size_t)(kv - 1) * T + t] = 0;
    ko_decode_attention(qd.data(), k.data(), v.data(), valid.data(), qh, kv, T, d, od.data());
    ko_decode_attention(qd.data(), k.data(), v.data(), nullptr, qh, kv, T, d, od.data());
    for (double x : od) CHECK(std::isfinite(x));
  }
}

int main() {
  run_shape(0, 2, 8, 16, 120, 8, 16, 24);   // bf16, G = 4
  run_shape(1, 3, 3, 8, 40, 4, 12, 10);     // fp32, G = 1
  run_shape(0, 1, 7, 32, 64, 2, 64, 8);     // bf16, one KV head, G = 7, O' = T
  if (failures) return 1;
  std::printf("ok\n");
  return 0;
}
