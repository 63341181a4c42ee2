// Plain, slow reference of the K-VEC prefill-time eviction step in C++
// (float64 scores, fp32 policy arithmetic), written from the paper's
// definitions independently of kvec_oracle.py: the two oracles are checked
// against each other and against the same closed forms.
//
// TEST INFRASTRUCTURE ONLY: loaded by tests/, by the smoke check and by the
// benchmark's CPU-baseline leg through oracle/cxx.py, never by the product
// path.  It shares no code with the HIP library.  Build (oracle/cxx.py):
//   g++ -O2 -std=c++17 -shared -fPIC -pthread -ffp-contract=off
// (no fused multiply-add contraction: the fp32 steps of Sec. 4.2 round once
// per operation).
//
// Source: "Coverage-Driven KV Cache Eviction for Efficient and Improved
// Inference of LLM" (K-VEC).  Each function names the passage it follows.
// The readings where the paper is silent are the ones kvec_oracle.py lists
// (GQA: a KV head's attention is the mean over its query heads; causal
// softmax with scale 1/sqrt(d); the window [T-O, T) is always kept; max-pool
// along t before sigma; population sigma; ties rank the lower index first;
// the preserve set uses P after the H_top replacement; n_t counts earlier
// layers that kept t in at least one head).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <thread>
#include <vector>

namespace {

// Run f(task) for task in [0, n) on up to `threads` threads.
template <class F>
void parallel_for(int n, int threads, F f) {
  if (threads <= 1 || n <= 1) {
    for (int i = 0; i < n; ++i) f(i);
    return;
  }
  std::atomic<int> next(0);
  std::vector<std::thread> pool;
  const int nt = std::min(threads, n);
  for (int w = 0; w < nt; ++w)
    pool.emplace_back([&]() {
      for (int i = next++; i < n; i = next++) f(i);
    });
  for (auto& t : pool) t.join();
}

// Sec. 4.1, Eq. (eviction): Abar[h][r][t], the causal softmax attention of
// window row r (position T - wn + r, which sees keys 0..p) averaged over the
// G query heads of KV head h (query head j uses KV head j / G).
void window_attention(const double* q, const double* k, int hq, int hkv, int wn, int T, int d,
                      double* abar, int threads) {
  const int g = hq / hkv;
  const double sd = std::sqrt((double)d);
  parallel_for(hkv * wn, threads, [&](int task) {
    const int h = task / wn, r = task % wn;
    const int p = T - wn + r;
    double* out = abar + ((size_t)h * wn + r) * T;
    for (int t = 0; t < T; ++t) out[t] = 0.0;
    std::vector<double> s(p + 1);
    for (int jj = 0; jj < g; ++jj) {
      const int j = h * g + jj;
      const double* qr = q + ((size_t)j * wn + r) * d;
      double m = -INFINITY;
      for (int t = 0; t <= p; ++t) {
        const double* kt = k + ((size_t)h * T + t) * d;
        double dot = 0.0;
        for (int i = 0; i < d; ++i) dot += qr[i] * kt[i];
        s[t] = dot / sd;
        m = std::max(m, s[t]);
      }
      double z = 0.0;
      for (int t = 0; t <= p; ++t) {
        s[t] = std::exp(s[t] - m);
        z += s[t];
      }
      for (int t = 0; t <= p; ++t) out[t] += s[t] / z;
    }
    for (int t = 0; t < T; ++t) out[t] /= g;
  });
}

}  // namespace

extern "C" {

// S1 (Sec. 4.1 Eq. eviction, the extended window of Sec. 4.1, I of Sec. 4.2):
//   P[h][t]     = (1/O)  sum over the last O window rows of Abar[h][r][t]
//   P_ext[h][t] = (1/wn) sum over all wn rows            of Abar[h][r][t]
//   I[t]        = (1/O)  sum over the last O rows of max_h Abar[h][r][t]
// q [hq][wn][d], k [hkv][T][d] (float64); outputs for t < n_out (T - O, or
// T when full): p, pe [hkv][n_out], imp [n_out].
void ko_window_scores(const double* q, const double* k, int hq, int hkv, int wn, int T, int d,
                      int O, int full, double* p, double* pe, double* imp, int threads) {
  std::vector<double> abar((size_t)hkv * wn * T);
  window_attention(q, k, hq, hkv, wn, T, d, abar.data(), threads);
  const int n_out = full ? T : T - O;
  for (int h = 0; h < hkv; ++h)
    for (int t = 0; t < n_out; ++t) {
      double sb = 0.0, sa = 0.0;
      for (int r = 0; r < wn; ++r) {
        const double a = abar[((size_t)h * wn + r) * T + t];
        sa += a;
        if (r >= wn - O) sb += a;
      }
      p[(size_t)h * n_out + t] = sb / O;
      pe[(size_t)h * n_out + t] = sa / wn;
    }
  for (int t = 0; t < n_out; ++t) {
    double s = 0.0;
    for (int r = wn - O; r < wn; ++r) {
      double mx = -INFINITY;
      for (int h = 0; h < hkv; ++h) mx = std::max(mx, abar[((size_t)h * wn + r) * T + t]);
      s += mx;
    }
    imp[t] = s / O;
  }
}

// The softmax denominator of A (Sec. 4.1, Eq. eviction) as a natural log:
// lse[j][r] = ln sum_{t <= p_r} exp(q_{j,r} . k_{j/G,t} / sqrt(d)).
void ko_window_lse(const double* q, const double* k, int hq, int hkv, int wn, int T, int d,
                   double* lse, int threads) {
  const int g = hq / hkv;
  const double sd = std::sqrt((double)d);
  parallel_for(hq * wn, threads, [&](int task) {
    const int j = task / wn, r = task % wn, h = j / g;
    const int p = T - wn + r;
    const double* qr = q + ((size_t)j * wn + r) * d;
    std::vector<double> s(p + 1);
    double m = -INFINITY;
    for (int t = 0; t <= p; ++t) {
      const double* kt = k + ((size_t)h * T + t) * d;
      double dot = 0.0;
      for (int i = 0; i < d; ++i) dot += qr[i] * kt[i];
      s[t] = dot / sd;
      m = std::max(m, s[t]);
    }
    double z = 0.0;
    for (int t = 0; t <= p; ++t) z += std::exp(s[t] - m);
    lse[(size_t)j * wn + r] = m + std::log(z);
  });
}

// S2 (pooling inherited from the SnapKV setting): out[t] = max{ x[u] :
// |u - t| <= kernel/2, 0 <= u < n }, per row.
void ko_maxpool(const float* x, int rows, int n, int kernel, float* out) {
  const int rad = kernel / 2;
  for (int i = 0; i < rows; ++i)
    for (int t = 0; t < n; ++t) {
      float m = -INFINITY;
      for (int u = std::max(0, t - rad); u <= std::min(n - 1, t + rad); ++u) m = std::max(m, x[(size_t)i * n + u]);
      out[(size_t)i * n + t] = m;
    }
}

// S3 (Sec. 4.1): sigma_h = sqrt((1/n) sum_t (x[h][t] - mean_h)^2) in float64.
void ko_head_sigma(const float* x, int H, int n, double* out) {
  for (int h = 0; h < H; ++h) {
    double s = 0.0;
    for (int t = 0; t < n; ++t) s += (double)x[(size_t)h * n + t];
    const double mean = s / n;
    double v = 0.0;
    for (int t = 0; t < n; ++t) {
      const double e = (double)x[(size_t)h * n + t] - mean;
      v += e * e;
    }
    out[h] = std::sqrt(v / n);
  }
}

// Sec. 5.4 (head-selection ablation): Shannon entropy (natural log) of a
// head's scores taken as a distribution over tokens; 0 ln 0 = 0, and a head
// whose scores are all zero has entropy 0.
void ko_head_entropy(const float* x, int H, int n, double* out) {
  for (int h = 0; h < H; ++h) {
    double tot = 0.0;
    for (int t = 0; t < n; ++t) tot += (double)x[(size_t)h * n + t];
    double e = 0.0;
    if (tot > 0.0)
      for (int t = 0; t < n; ++t) {
        const double v = (double)x[(size_t)h * n + t];
        if (v > 0.0) {
          const double q = v / tot;
          e -= q * std::log(q);
        }
      }
    out[h] = e;
  }
}

// H_top (Sec. 4.1): the delta heads with the lowest key (sigma, or minus the
// entropy for the ablation's least-focused heads), ties to the lower head;
// returned in ascending head order.  Returns the number of heads.
int ko_adjusted_heads(const double* key, int H, int delta, int64_t* out) {
  std::vector<int> order(H);
  for (int h = 0; h < H; ++h) order[h] = h;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return key[a] < key[b]; });
  const int n = std::max(0, std::min(delta, H));
  std::vector<int> pick(order.begin(), order.begin() + n);
  std::sort(pick.begin(), pick.end());
  for (int i = 0; i < n; ++i) out[i] = pick[i];
  return n;
}

// Top-B selection and the preserve set (Sec. 4.1, Sec. 4.2): the first k
// tokens in the order (score descending, index ascending).
void ko_rank_first(const float* s, int n, int k, int64_t* out) {
  std::vector<int> order(n);
  for (int t = 0; t < n; ++t) order[t] = t;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return s[a] > s[b]; });
  k = std::max(0, std::min(k, n));
  for (int i = 0; i < k; ++i) out[i] = order[i];
}

// K = beta * B preserved tokens per head (Sec. 4.2), at most the B - O picks.
int ko_preserve_count(int budget, int window, float beta) {
  const double k = std::floor((double)beta * budget);
  return (int)std::min(k, (double)(budget - window));
}

// S5 (Sec. 4.2, Algorithm 1), one fp32 operation per step:
//   coverage = n_t / (l + 1); focus = I * (1 - coverage);
//   P' = P_sel + lambda * focus; P' = 1 on the preserved set (keep != 0).
void ko_adjusted_priority(const float* p_sel, const float* imp, const int64_t* n_t, int layer,
                          float lam, const uint8_t* keep, int H, int n, float* out) {
  const float den = (float)(layer + 1);
  for (int t = 0; t < n; ++t) {
    const float cov = (float)n_t[t] / den;
    const float one_minus = 1.0f - cov;
    const float focus = imp[t] * one_minus;
    const float bonus = lam * focus;
    for (int h = 0; h < H; ++h) {
      const size_t i = (size_t)h * n + t;
      out[i] = keep[i] ? 1.0f : p_sel[i] + bonus;
    }
  }
}

// One layer of the policy on fp32 scores (S2..S7): pooling, H_top and the
// replacement by the extended-window scores (Sec. 4.1), the preserve set and
// the coverage bonus (Sec. 4.2, Algorithm 1), the top B - O prefix tokens in
// ascending order followed by the window (Sec. 4.1), and the layer's kept-token
// bitmap.  p_raw, p_ext [H][T-O], imp [T-O], n_t [T-O].  Outputs: idx [H][B]
// (-1 pads when T <= B), htop (up to H entries, count returned), sigma [H],
// keep [H][T-O], p_sel and p_adj [H][T-O], bits [T].
int ko_select_layer(const float* p_raw, const float* p_ext, const float* imp, const int64_t* n_t,
                    int layer, int H, int T, int window, int window_ext, int budget,
                    int pool_kernel, int delta, float lam, float beta, int entropy,
                    int32_t* idx, int64_t* htop, double* sigma, uint8_t* keep, float* p_sel,
                    float* p_adj, uint8_t* bits) {
  const int O = window, Tc = T - O;
  if (T <= budget) {  // nothing to evict
    for (int h = 0; h < H; ++h) {
      sigma[h] = 0.0;
      for (int i = 0; i < budget; ++i) idx[(size_t)h * budget + i] = i < T ? i : -1;
    }
    for (int t = 0; t < std::max(Tc, 0) * H; ++t) {
      keep[t] = 0;
      p_sel[t] = 0.f;
      p_adj[t] = 0.f;
    }
    for (int t = 0; t < T; ++t) bits[t] = 1;
    return 0;
  }
  std::vector<float> pooled((size_t)H * Tc), pooled_ext((size_t)H * Tc);
  ko_maxpool(p_raw, H, Tc, pool_kernel, pooled.data());
  ko_maxpool(p_ext, H, Tc, pool_kernel, pooled_ext.data());
  ko_head_sigma(pooled.data(), H, Tc, sigma);
  const int wn = std::min(window_ext, T);
  int nh = 0;
  if (wn > O) {
    std::vector<double> key(H);
    if (entropy) {
      ko_head_entropy(pooled.data(), H, Tc, key.data());
      for (auto& v : key) v = -v;
    } else {
      for (int h = 0; h < H; ++h) key[h] = sigma[h];
    }
    nh = ko_adjusted_heads(key.data(), H, delta, htop);
  }
  for (size_t i = 0; i < (size_t)H * Tc; ++i) p_sel[i] = pooled[i];
  for (int a = 0; a < nh; ++a)
    for (int t = 0; t < Tc; ++t) p_sel[(size_t)htop[a] * Tc + t] = pooled_ext[(size_t)htop[a] * Tc + t];
  const int kp = ko_preserve_count(budget, O, beta);
  std::vector<int64_t> pick(std::max(Tc, 1));
  for (size_t i = 0; i < (size_t)H * Tc; ++i) keep[i] = 0;
  for (int h = 0; h < H; ++h) {
    ko_rank_first(p_sel + (size_t)h * Tc, Tc, kp, pick.data());
    for (int i = 0; i < kp; ++i) keep[(size_t)h * Tc + pick[i]] = 1;
  }
  ko_adjusted_priority(p_sel, imp, n_t, layer, lam, keep, H, Tc, p_adj);
  const int m = budget - O;
  for (int t = 0; t < T; ++t) bits[t] = t >= Tc;
  for (int h = 0; h < H; ++h) {
    ko_rank_first(p_adj + (size_t)h * Tc, Tc, m, pick.data());
    std::sort(pick.begin(), pick.begin() + m);
    for (int i = 0; i < m; ++i) {
      idx[(size_t)h * budget + i] = (int32_t)pick[i];
      bits[pick[i]] = 1;
    }
    for (int i = m; i < budget; ++i) idx[(size_t)h * budget + i] = Tc + (i - m);
  }
  return nh;
}

// S7 (Sec. 4.2): n_t = number of the given layers whose kept set contains t;
// bits [n_layers][T] (0/1).
void ko_counts_from_bits(const uint8_t* bits, int n_layers, int T, int64_t* out) {
  for (int t = 0; t < T; ++t) {
    int64_t c = 0;
    for (int l = 0; l < n_layers; ++l) c += bits[(size_t)l * T + t] ? 1 : 0;
    out[t] = c;
  }
}

// Coverage C (Sec. 3.2): the number of unique tokens kept across the layers.
int64_t ko_coverage_count(const uint8_t* bits, int n_layers, int T) {
  int64_t c = 0;
  for (int t = 0; t < T; ++t) {
    bool any = false;
    for (int l = 0; l < n_layers; ++l) any = any || bits[(size_t)l * T + t];
    c += any ? 1 : 0;
  }
  return c;
}

// S8, the cache store (Sec. 4.1): out[h][i] = x[h][idx[h][i]] (row bytes),
// zeros where idx is negative.  x [H][T][row_bytes].
void ko_gather_rows(const uint8_t* x, const int32_t* idx, int H, int T, int B, int row_bytes,
                    uint8_t* out) {
  for (int h = 0; h < H; ++h)
    for (int i = 0; i < B; ++i) {
      const int32_t t = idx[(size_t)h * B + i];
      uint8_t* o = out + ((size_t)h * B + i) * row_bytes;
      if (t < 0) {
        for (int b = 0; b < row_bytes; ++b) o[b] = 0;
      } else {
        const uint8_t* s = x + ((size_t)h * T + t) * row_bytes;
        for (int b = 0; b < row_bytes; ++b) o[b] = s[b];
      }
    }
}

// The decoding phase served by the kept cache (Sec. 4.1): out[j] =
// sum_i softmax_i(q_j . k_{h,i} / sqrt(d)) v_{h,i}, h = j / G, over the rows
// i with valid[h][i] (all rows when valid is null); zeros for a head with no
// valid row.  q [hq][d], k, v [hkv][n][d], out [hq][d], float64.
void ko_decode_attention(const double* q, const double* k, const double* v, const uint8_t* valid,
                         int hq, int hkv, int n, int d, double* out) {
  const int g = hq / hkv;
  const double sd = std::sqrt((double)d);
  for (int j = 0; j < hq; ++j) {
    const int h = j / g;
    double* o = out + (size_t)j * d;
    for (int e = 0; e < d; ++e) o[e] = 0.0;
    std::vector<double> s(n);
    double m = -INFINITY;
    bool any = false;
    for (int i = 0; i < n; ++i) {
      if (valid && !valid[(size_t)h * n + i]) continue;
      double dot = 0.0;
      for (int e = 0; e < d; ++e) dot += k[((size_t)h * n + i) * d + e] * q[(size_t)j * d + e];
      s[i] = dot / sd;
      m = std::max(m, s[i]);
      any = true;
    }
    if (!any) continue;
    double z = 0.0;
    for (int i = 0; i < n; ++i) {
      if (valid && !valid[(size_t)h * n + i]) continue;
      s[i] = std::exp(s[i] - m);
      z += s[i];
    }
    for (int i = 0; i < n; ++i) {
      if (valid && !valid[(size_t)h * n + i]) continue;
      const double w = s[i] / z;
      for (int e = 0; e < d; ++e) o[e] += w * v[((size_t)h * n + i) * d + e];
    }
  }
}

}  // extern "C"
