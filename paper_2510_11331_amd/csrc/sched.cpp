// Serving scheduler: the paper's runtime / pipeline latency model, the
// batching dynamic program and the speculation-length search (Sections II-C,
// II-D and III; see include/sd_sched.h for the model).  Host code only.
#include "sd.h"
#include "sd_sched.h"

#include <algorithm>
#include <cmath>
#include <numeric>
#include <utility>
#include <vector>

namespace {

struct Model {
  double J, h1, h2;
};

struct Ctx {
  Model d, v;
  double c1d, c2d, c1v, c2v, alpha, mem;
  int o_max;
  bool prefill_separate;
};

bool model_ok(const sd_sched_model& m) { return m.n_layers >= 1 && m.d_model >= 1 && m.d_ffn >= 1; }

bool make_ctx(const sd_sched_cfg* c, Ctx& x) {
  if (!c || !model_ok(c->draft) || !model_ok(c->target) || !(c->alpha >= 0.0 && c->alpha <= 1.0) || c->o_max < 1)
    return false;
  if (!(c->c1_draft >= 0 && c->c2_draft >= 0 && c->c1_verify >= 0 && c->c2_verify >= 0)) return false;
  x.d = {(double)c->draft.n_layers, (double)c->draft.d_model, (double)c->draft.d_ffn};
  x.v = {(double)c->target.n_layers, (double)c->target.d_model, (double)c->target.d_ffn};
  x.c1d = c->c1_draft;
  x.c2d = c->c2_draft;
  x.c1v = c->c1_verify;
  x.c2v = c->c2_verify;
  x.alpha = c->alpha;
  x.mem = c->mem_budget;
  x.o_max = c->o_max;
  x.prefill_separate = c->prefill_separate != 0;
  return true;
}

// eq. ol
double emitted(double alpha, int l) { return alpha >= 1.0 ? (double)(l + 1) : (1.0 - std::pow(alpha, l + 1)) / (1.0 - alpha); }

// eq. step_n with O_m = O_max
int steps(int o_max, double alpha, int l) { return (int)std::ceil(o_max / emitted(alpha, l)); }

// eq. flops_d: i-th draft forward of step n, one task
double flops_d(const Model& m, double Im, int i, int n, double L) {
  if (n == 1 && i == 1) return 4.0 * m.J * m.h1 * Im * (2.0 * m.h1 + Im + m.h2);
  const double kv = Im + ((n - 1) * L - 1.0) + i - 1;
  return 4.0 * m.J * m.h1 * (2.0 * m.h1 + kv + 1.0 + m.h2);
}

// eq. flops_v: verify forward of step n, one task
double flops_v(const Model& m, double Im, int l, int n, double L) {
  if (n == 1) return 4.0 * m.J * m.h1 * (Im + l) * (2.0 * m.h1 + Im + l + m.h2);
  const double kv = Im + (n - 1) * L - 1.0;
  return 4.0 * m.J * m.h1 * (1.0 + l) * (2.0 * m.h1 + kv + l + 1.0 + m.h2);
}

// (T^d, T^v) of a batch of b tasks with input length Im at step n
// (eqs. latency_b2, d_latency, v_latency)
// decoding-stage forms: one draft token over kv cached tokens; 1 + l verify
// tokens over kv cached tokens
double flops_d_decode(const Model& m, double kv) { return 4.0 * m.J * m.h1 * (2.0 * m.h1 + kv + 1.0 + m.h2); }
double flops_v_decode(const Model& m, double kv, int l) {
  return 4.0 * m.J * m.h1 * (1.0 + l) * (2.0 * m.h1 + kv + l + 1.0 + m.h2);
}

std::pair<double, double> step_times(const Ctx& x, int b, double Im, int l, int n, double L) {
  double td = 0.0;
  if (x.prefill_separate) {
    // every step is a decoding step: before step n the caches hold the prompt
    // minus one token plus (n - 1) L emitted tokens
    const double base = Im - 1.0 + (n - 1) * L;
    for (int i = 1; i <= l; ++i) td += x.c1d * flops_d_decode(x.d, base + i - 1) * b + x.c2d;
    const double tv = x.c1v * flops_v_decode(x.v, base, l) * b + x.c2v;
    return {td, tv};
  }
  for (int i = 1; i <= l; ++i) td += x.c1d * flops_d(x.d, Im, i, n, L) * b + x.c2d;
  const double tv = x.c1v * flops_v(x.v, Im, l, n, L) * b + x.c2v;
  return {td, tv};
}

// eqs. memory_model + memory_kv
double draft_memory(const Ctx& x, int b, double Im) {
  const Model& m = x.d;
  return m.J * (8.0 * m.h1 * m.h1 + 4.0 * m.h1 * m.h2) + 4.0 * m.J * m.h1 * (Im + x.o_max) * b;
}

bool lengths_ok(int K, const int32_t* len) {
  if (K < 1 || !len) return false;
  for (int k = 0; k < K; ++k)
    if (len[k] < 1) return false;
  return true;
}

std::vector<int> sorted_order(int K, const int32_t* len) {
  std::vector<int> o(K);
  std::iota(o.begin(), o.end(), 0);
  std::stable_sort(o.begin(), o.end(), [&](int a, int b) { return len[a] < len[b]; });
  return o;
}

// Algorithm 1 for one l; returns SD_OK / SD_ENOMEM
int batching(const Ctx& x, int K, const int32_t* len, int l, std::vector<int>& batch_of, int& nb, double& t_inf) {
  const std::vector<int> order = sorted_order(K, len);
  const double L = emitted(x.alpha, l);
  const int N = steps(x.o_max, x.alpha, l);
  // Y[i][n] for the chosen plan of the first i sorted tasks, n = 0..N-1
  std::vector<std::vector<std::pair<double, double>>> Y(K + 1, std::vector<std::pair<double, double>>(N, {0.0, 0.0}));
  std::vector<double> best(K + 1, 0.0);
  std::vector<int> S(K + 1, 0);
  std::vector<std::pair<double, double>> rows(N);
  for (int i = 1; i <= K; ++i) {
    const double Im = (double)len[order[i - 1]];
    bool found = false;
    for (int j = 1; j <= i; ++j) {
      const int b = i - j + 1;
      if (x.mem > 0 && draft_memory(x, b, Im) > x.mem) continue;
      double temp = 0.0;
      for (int n = 1; n <= N; ++n) {
        const std::pair<double, double> t = step_times(x, b, Im, l, n, L);
        const double s0 = Y[j - 1][n - 1].first + t.first;
        const double s1 = std::max(s0, Y[j - 1][n - 1].second) + t.second;
        rows[n - 1] = {s0, s1};
        temp += s1;
      }
      if (!found || best[i] >= temp) {
        found = true;
        best[i] = temp;
        S[i] = j;
        Y[i] = rows;
      }
    }
    if (!found) return SD_ENOMEM;
  }
  // read back: batches are runs [S[i], i] of the sorted order
  std::vector<std::pair<int, int>> runs;
  for (int i = K; i > 0; i = S[i] - 1) runs.push_back({S[i], i});
  std::reverse(runs.begin(), runs.end());
  batch_of.assign(K, 0);
  for (size_t m = 0; m < runs.size(); ++m)
    for (int p = runs[m].first; p <= runs[m].second; ++p) batch_of[order[p - 1]] = (int)m;
  nb = (int)runs.size();
  t_inf = best[K];
  return SD_OK;
}

}  // namespace

extern "C" {

int sd_sched_latency(const sd_sched_cfg* cfg, int K, const int32_t* input_len, int n_batches,
                     const int32_t* batch_of, int l, double* t_inf) {
  Ctx x;
  if (!make_ctx(cfg, x) || !lengths_ok(K, input_len) || !batch_of || !t_inf || l < 1 || n_batches < 1)
    return SD_EINVAL;
  std::vector<int> size(n_batches, 0), Im(n_batches, 0);
  for (int k = 0; k < K; ++k) {
    const int m = batch_of[k];
    if (m < 0 || m >= n_batches) return SD_EINVAL;
    ++size[m];
    Im[m] = std::max(Im[m], (int)input_len[k]);
  }
  for (int m = 0; m < n_batches; ++m)
    if (size[m] == 0) return SD_EINVAL;
  const double L = emitted(x.alpha, l);
  const int N = steps(x.o_max, x.alpha, l);
  double total = 0.0;
  for (int n = 1; n <= N; ++n) {
    double cd = 0.0, c = 0.0;
    for (int m = 0; m < n_batches; ++m) {
      const std::pair<double, double> t = step_times(x, size[m], (double)Im[m], l, n, L);
      cd = cd + t.first;
      c = std::max(cd, c) + t.second;
    }
    total += c;
  }
  *t_inf = total;
  return SD_OK;
}

int sd_sched_batching(const sd_sched_cfg* cfg, int K, const int32_t* input_len, int l, int32_t* batch_of,
                      int* n_batches, double* t_inf) {
  Ctx x;
  if (!make_ctx(cfg, x) || !lengths_ok(K, input_len) || l < 1 || !batch_of || !n_batches || !t_inf) return SD_EINVAL;
  std::vector<int> bo;
  int nb = 0;
  double t = 0.0;
  const int rc = batching(x, K, input_len, l, bo, nb, t);
  if (rc != SD_OK) return rc;
  for (int k = 0; k < K; ++k) batch_of[k] = bo[k];
  *n_batches = nb;
  *t_inf = t;
  return SD_OK;
}

int sd_sched_plan(const sd_sched_cfg* cfg, int K, const int32_t* input_len, int l_max, int32_t* batch_of,
                  int* n_batches, int* l_best, double* t_inf, double* t_inf_by_l) {
  Ctx x;
  if (!make_ctx(cfg, x) || !lengths_ok(K, input_len) || l_max < 1 || !batch_of || !n_batches || !l_best || !t_inf)
    return SD_EINVAL;
  std::vector<int> best_bo, bo;
  int best_nb = 0, best_l = 0;
  double best_t = 0.0;
  std::vector<double> by_l(l_max, 0.0);
  for (int l = 1; l <= l_max; ++l) {
    int nb = 0;
    double t = 0.0;
    const int rc = batching(x, K, input_len, l, bo, nb, t);
    if (rc != SD_OK) return rc;
    by_l[l - 1] = t;
    if (best_l == 0 || t < best_t) {
      best_t = t;
      best_l = l;
      best_nb = nb;
      best_bo = bo;
    }
  }
  for (int k = 0; k < K; ++k) batch_of[k] = best_bo[k];
  *n_batches = best_nb;
  *l_best = best_l;
  *t_inf = best_t;
  if (t_inf_by_l)
    for (int l = 0; l < l_max; ++l) t_inf_by_l[l] = by_l[l];
  return SD_OK;
}

int sd_sched_uplink(int K, const int32_t* input_len, const double* snr, double lambda_bits, double bandwidth_hz,
                    double* w, double* t_com) {
  if (!lengths_ok(K, input_len) || !snr || !w || !t_com || !(lambda_bits > 0) || !(bandwidth_hz > 0)) return SD_EINVAL;
  for (int k = 0; k < K; ++k)
    if (!(snr[k] > 0)) return SD_EINVAL;
  std::vector<double> a(K);
  double tot = 0.0;
  for (int k = 0; k < K; ++k) {
    a[k] = input_len[k] / std::log2(1.0 + snr[k]);
    tot += a[k];
  }
  for (int k = 0; k < K; ++k) w[k] = a[k] / tot;
  *t_com = lambda_bits * tot / bandwidth_hz;
  return SD_OK;
}

}  // extern "C"
