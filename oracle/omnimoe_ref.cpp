// Oracle for the OmniMoE atomic-expert layer forward pass: TEST INFRASTRUCTURE ONLY.
//
// Plain host C++ in double precision, written from the paper (arXiv 2602.05711):
//   Sec. 2.1  atomic expert E_i(x) = act(x . w_in_i) w_out_i (Eq. 4), global tables
//             W, V (Eq. 5), retrieval and assembly y = (g . act(x w_x^T)) v_x (Eq. 6-7)
//   Sec. 2.2  Cartesian Product Router: s_r = x W_r, s_c = x W_c (Eq. 9), the implicit
//             grid S_ij = p_r[i] + p_c[j] (Eq. 11), top-K (Eq. 1) and softmax gates (Eq. 2)
//   Sec. 2.3  Expert-Centric Scheduling: task flatten (Eq. 12), active-expert groups of
//             size B, sort by (group, token) (Eq. 13), per-group compute (Eq. 14)
//   Sec. 2.1  the shared dense branch MLP(x) added to the routed output (Eq. 3, 7), a
//             SwiGLU feed-forward block
//   Sec. 3.3  the router ablation: a dense router scoring all N experts (Table 3)
// It is used only by tests, the smoke check and the benchmark's CPU-baseline leg, and it
// shares no code with the GPU library. Nothing here is blocked, fused or reordered
// beyond what those passages state; library sorts serve as steps where a sort is what
// the passage asks for.
//
// Readings where the paper is silent (the same ones the GPU library follows):
//   * heads: each head has its own sub-key tables and its own top-K and softmax; x, U,
//     V are shared and y sums over heads;
//   * queries: rows score x[0:d_key], columns x[d_key:2 d_key] (split) or both
//     x[0:d_key] (shared); there is no query projection;
//   * expert id of grid cell (i, j) is n = i * n_cols + j;
//   * order: S descending, ties to the lower expert id; the K list is returned in
//     that order and rows/columns rank by (logit descending, index ascending);
//   * LogSoftmax (Eq. 10) subtracts one constant per (token, head, half), so it changes
//     neither the selected set nor the gates; selection uses the raw sums (method 2
//     applies it literally so tests can check that reading);
//   * act is GELU in its erf form (or SiLU); per-token accumulation runs over slots
//     in (head, k) order.
#include "omnimoe_ref.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <thread>
#include <vector>

namespace {

bool valid(const omnimoe_ref_desc* d) {
  if (!d) return false;
  if (d->T < 0 || d->d < 1 || d->n_rows < 1 || d->n_cols < 1 || d->d_key < 1) return false;
  if (d->H < 1 || d->K < 1) return false;
  if ((int64_t)d->K > (int64_t)d->n_rows * d->n_cols) return false;
  if (d->query_mode == 0 && 2 * (int64_t)d->d_key > d->d) return false;
  if (d->query_mode == 1 && d->d_key > d->d) return false;
  if (d->query_mode != 0 && d->query_mode != 1) return false;
  if (d->act != 0 && d->act != 1) return false;
  if (d->group_size < 1) return false;
  return true;
}

// Runs body(begin, end) over [0, n) split into contiguous chunks, one per thread.
void parallel_for(int64_t n, int n_threads, const std::function<void(int64_t, int64_t)>& body) {
  if (n <= 0) return;
  if (n_threads < 1) n_threads = 1;
  if ((int64_t)n_threads > n) n_threads = (int)n;
  if (n_threads == 1) {
    body(0, n);
    return;
  }
  std::vector<std::thread> pool;
  for (int i = 0; i < n_threads; ++i) {
    int64_t b = n * i / n_threads, e = n * (i + 1) / n_threads;
    pool.emplace_back([&body, b, e] { body(b, e); });
  }
  for (auto& th : pool) th.join();
}

// True when a + b is exact in double (the error term of TwoSum is zero).
bool sum_is_exact(double a, double b) {
  double s = a + b;
  double bb = s - a;
  double err = (a - (s - bb)) + (b - bb);
  return err == 0.0;
}

struct Cand {
  double s;   // score S
  int64_t n;  // expert id
};

// (S descending, id ascending)
bool cand_before(const Cand& a, const Cand& b) {
  if (a.s != b.s) return a.s > b.s;
  return a.n < b.n;
}

// First k entries of `c` in (S desc, id asc) order.
void top_k(std::vector<Cand>& c, int k) {
  std::partial_sort(c.begin(), c.begin() + k, c.end(), cand_before);
}

// Softmax of the selected scores (Eq. 2), s[0] being the largest.
void softmax_gates(const double* s, int k, double* g) {
  double z = 0.0;
  for (int i = 0; i < k; ++i) z += std::exp(s[i] - s[0]);
  for (int i = 0; i < k; ++i) g[i] = std::exp(s[i] - s[0]) / z;
}

// log-sum-exp of one half's logits, for the literal LogSoftmax of Eq. 10.
double log_sum_exp(const double* s, int n) {
  double m = s[0];
  for (int i = 1; i < n; ++i) m = std::max(m, s[i]);
  double z = 0.0;
  for (int i = 0; i < n; ++i) z += std::exp(s[i] - m);
  return m + std::log(z);
}

// Selection for one (token, head) row.
int64_t select_row(const omnimoe_ref_desc* d, const double* sr, const double* sc, int method,
                   int32_t* idx, double* sel, double* gates) {
  const int nr = d->n_rows, nc = d->n_cols, K = d->K;
  int64_t inexact = 0;
  std::vector<Cand> cand;
  if (method == 0 || method == 2) {
    // Definition: every cell of the grid is a candidate.
    std::vector<double> pr(sr, sr + nr), pc(sc, sc + nc);
    if (method == 2) {
      double lr = log_sum_exp(sr, nr), lc = log_sum_exp(sc, nc);
      for (auto& v : pr) v -= lr;
      for (auto& v : pc) v -= lc;
    }
    cand.resize((size_t)nr * nc);
    for (int i = 0; i < nr; ++i)
      for (int j = 0; j < nc; ++j) {
        if (!sum_is_exact(pr[i], pc[j])) ++inexact;
        cand[(size_t)i * nc + j] = Cand{pr[i] + pc[j], (int64_t)i * nc + j};
      }
  } else {
    // Method: rank rows and columns, keep the cells (a, b) of rank with (a+1)(b+1) <= K.
    // Cell (i, j) is preceded in (S desc, n asc) order by every other cell whose row and
    // column ranks are both no worse, so it can only be in the top K when
    // (rank_i + 1)(rank_j + 1) <= K; the sums must be exact for that argument.
    const int kr = std::min(K, nr), kc = std::min(K, nc);
    std::vector<Cand> rows(nr), cols(nc);
    for (int i = 0; i < nr; ++i) rows[i] = Cand{sr[i], i};
    for (int j = 0; j < nc; ++j) cols[j] = Cand{sc[j], j};
    top_k(rows, kr);
    top_k(cols, kc);
    for (int a = 0; a < kr; ++a)
      for (int b = 0; b < kc && (int64_t)(a + 1) * (b + 1) <= K; ++b) {
        double x = rows[a].s, y = cols[b].s;
        if (!sum_is_exact(x, y)) ++inexact;
        cand.push_back(Cand{x + y, rows[a].n * nc + cols[b].n});
      }
  }
  top_k(cand, K);
  std::vector<double> s(K);
  for (int k = 0; k < K; ++k) {
    idx[k] = (int32_t)cand[k].n;
    s[k] = cand[k].s;
    if (sel) sel[k] = s[k];
  }
  softmax_gates(s.data(), K, gates);
  return inexact;
}

// Dense selection for one (token, head) row of N logits: the plain definition of Eq. 1.
void select_dense_row(const double* L, int64_t N, int K, int32_t* idx, double* gates) {
  std::vector<Cand> cand((size_t)N);
  for (int64_t n = 0; n < N; ++n) cand[(size_t)n] = Cand{L[n], n};
  top_k(cand, K);
  std::vector<double> s(K);
  for (int k = 0; k < K; ++k) {
    idx[k] = (int32_t)cand[k].n;
    s[k] = cand[k].s;
  }
  softmax_gates(s.data(), K, gates);
}

double gelu_erf(double z) { return 0.5 * z * (1.0 + std::erf(z / std::sqrt(2.0))); }
double silu(double z) { return z / (1.0 + std::exp(-z)); }
// d/dz of z Phi(z) = Phi(z) + z phi(z); d/dz of z s(z) = s(z) (1 + z (1 - s(z))).
double gelu_erf_grad(double z) {
  const double pi = 3.14159265358979323846;
  return 0.5 * (1.0 + std::erf(z / std::sqrt(2.0))) + z * std::exp(-0.5 * z * z) / std::sqrt(2.0 * pi);
}
double silu_grad(double z) {
  const double sg = 1.0 / (1.0 + std::exp(-z));
  return sg * (1.0 + z * (1.0 - sg));
}

double dot_row(const float* a, const float* b, int n) {
  double s = 0.0;
  for (int m = 0; m < n; ++m) s += (double)a[m] * (double)b[m];
  return s;
}

}  // namespace

extern "C" {

double omnimoe_ref_act(int act, double z) { return act == 1 ? silu(z) : gelu_erf(z); }
double omnimoe_ref_act_grad(int act, double z) { return act == 1 ? silu_grad(z) : gelu_erf_grad(z); }

int omnimoe_ref_half_scores(const omnimoe_ref_desc* d, const float* x, const float* keys_row,
                            const float* keys_col, double* sr, double* sc, int n_threads) {
  if (!valid(d)) return -1;
  const int H = d->H, nr = d->n_rows, nc = d->n_cols, dk = d->d_key;
  const int c0 = d->query_mode == 0 ? dk : 0;
  parallel_for(d->T * H, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t th = b; th < e; ++th) {
      int64_t t = th / H;
      int h = (int)(th % H);
      const float* xt = x + t * d->d;
      for (int i = 0; i < nr; ++i)
        sr[th * nr + i] = dot_row(xt, keys_row + ((int64_t)h * nr + i) * dk, dk);
      for (int j = 0; j < nc; ++j)
        sc[th * nc + j] = dot_row(xt + c0, keys_col + ((int64_t)h * nc + j) * dk, dk);
    }
  });
  return 0;
}

int omnimoe_ref_select(const omnimoe_ref_desc* d, const double* sr, const double* sc, int method,
                       int32_t* idx, double* sel_scores, double* gates, int64_t* inexact_sums,
                       int n_threads) {
  if (!valid(d) || method < 0 || method > 2) return -1;
  const int H = d->H, nr = d->n_rows, nc = d->n_cols, K = d->K;
  const int64_t rows = d->T * H;
  std::vector<int64_t> inexact(std::max(1, n_threads), 0);
  int nt = std::max(1, n_threads);
  std::vector<std::thread> pool;
  for (int w = 0; w < nt; ++w) {
    int64_t b = rows * w / nt, e = rows * (w + 1) / nt;
    pool.emplace_back([&, w, b, e] {
      for (int64_t r = b; r < e; ++r)
        inexact[w] += select_row(d, sr + r * nr, sc + r * nc, method, idx + r * K,
                                 sel_scores ? sel_scores + r * K : nullptr, gates + r * K);
    });
  }
  for (auto& th : pool) th.join();
  if (inexact_sums) {
    int64_t s = 0;
    for (auto v : inexact) s += v;
    *inexact_sums = s;
  }
  return 0;
}

int omnimoe_ref_select_f32(const omnimoe_ref_desc* d, const float* hs, int method, int32_t* idx,
                           double* sel_scores, double* gates, int64_t* inexact_sums,
                           int n_threads) {
  if (!valid(d)) return -1;
  const int nr = d->n_rows, nc = d->n_cols;
  const int64_t rows = d->T * d->H;
  std::vector<double> sr((size_t)rows * nr), sc((size_t)rows * nc);
  for (int64_t r = 0; r < rows; ++r) {
    const float* row = hs + r * (nr + nc);
    for (int i = 0; i < nr; ++i) sr[r * nr + i] = (double)row[i];
    for (int j = 0; j < nc; ++j) sc[r * nc + j] = (double)row[nr + j];
  }
  return omnimoe_ref_select(d, sr.data(), sc.data(), method, idx, sel_scores, gates,
                            inexact_sums, n_threads);
}

int omnimoe_ref_schedule(const omnimoe_ref_desc* d, const int32_t* idx, int32_t* perm,
                         int32_t* active, int32_t* active_offsets, int32_t* n_active,
                         int32_t* dense_offsets) {
  if (!valid(d)) return -1;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  const int64_t M = d->T * d->H * d->K;
  // Task flatten (Eq. 12): pair p = (t * H + h) * K + k carries expert idx[p].
  std::vector<int64_t> count(N, 0);
  for (int64_t p = 0; p < M; ++p) {
    if (idx[p] < 0 || idx[p] >= N) return -2;
    ++count[idx[p]];
  }
  // Active experts in ascending id order, and their group q = rank / B.
  std::vector<int64_t> rank(N, -1);
  int64_t A = 0;
  for (int64_t e = 0; e < N; ++e)
    if (count[e] > 0) {
      active[A] = (int32_t)e;
      rank[e] = A++;
    }
  *n_active = (int32_t)A;
  int64_t acc = 0;
  for (int64_t a = 0; a < A; ++a) {
    active_offsets[a] = (int32_t)acc;
    acc += count[active[a]];
  }
  active_offsets[A] = (int32_t)acc;
  if (dense_offsets) {
    acc = 0;
    for (int64_t e = 0; e < N; ++e) {
      dense_offsets[e] = (int32_t)acc;
      acc += count[e];
    }
    dense_offsets[N] = (int32_t)acc;
  }
  // Sort by (group, token) (Eq. 13): a stable counting sort of the pair ids by group.
  // Pair ids are token-major, so within a group the order is (token, head, k).
  const int64_t B = d->group_size;
  const int64_t G = (A + B - 1) / B;
  std::vector<int64_t> gstart(G + 1, 0);
  for (int64_t p = 0; p < M; ++p) ++gstart[rank[idx[p]] / B + 1];
  for (int64_t g = 0; g < G; ++g) gstart[g + 1] += gstart[g];
  for (int64_t p = 0; p < M; ++p) perm[gstart[rank[idx[p]] / B]++] = (int32_t)p;
  return 0;
}

int omnimoe_ref_expert_forward(const omnimoe_ref_desc* d, const float* x, const float* u,
                               const float* v, const int32_t* idx, const double* gates,
                               int scheduled, double* y, int n_threads) {
  if (!valid(d)) return -1;
  const int D = d->d;
  const int64_t HK = (int64_t)d->H * d->K;
  const int64_t M = d->T * HK;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  for (int64_t p = 0; p < M; ++p)
    if (idx[p] < 0 || idx[p] >= N) return -2;
  if (!scheduled) {
    // Token-centric: each token gathers its own experts (Eq. 6-7).
    parallel_for(d->T, n_threads, [&](int64_t b, int64_t e) {
      for (int64_t t = b; t < e; ++t) {
        double* yt = y + t * D;
        for (int m = 0; m < D; ++m) yt[m] = 0.0;
        for (int64_t s = 0; s < HK; ++s) {
          int64_t p = t * HK + s;
          int64_t ex = idx[p];
          double a = gates[p] * omnimoe_ref_act(d->act, dot_row(x + t * D, u + ex * D, D));
          for (int m = 0; m < D; ++m) yt[m] += a * (double)v[ex * D + m];
        }
      }
    });
    return 0;
  }
  // Expert-centric: walk the schedule group by group, expert by expert, forming
  // a[p] = g_p * act(x_t . u_e) (the G (.) act(X W^T) factor of Eq. 14), then add
  // a[p] * v_e into its token in slot order.
  std::vector<int32_t> perm(M), active(std::min(M, N) + 1), off(std::min(M, N) + 2);
  int32_t A = 0;
  int rc = omnimoe_ref_schedule(d, idx, perm.data(), active.data(), off.data(), &A, nullptr);
  if (rc) return rc;
  std::vector<double> a(M);
  parallel_for(M, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t tau = b; tau < e; ++tau) {
      int64_t p = perm[tau];
      int64_t t = p / HK;
      int64_t ex = idx[p];
      a[p] = gates[p] * omnimoe_ref_act(d->act, dot_row(x + t * D, u + ex * D, D));
    }
  });
  parallel_for(d->T, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t t = b; t < e; ++t) {
      double* yt = y + t * D;
      for (int m = 0; m < D; ++m) yt[m] = 0.0;
      for (int64_t s = 0; s < HK; ++s) {
        int64_t p = t * HK + s;
        int64_t ex = idx[p];
        for (int m = 0; m < D; ++m) yt[m] += a[p] * (double)v[ex * D + m];
      }
    }
  });
  return 0;
}

int omnimoe_ref_layer_forward(const omnimoe_ref_desc* d, const float* x, const float* keys_row,
                              const float* keys_col, const float* u, const float* v, int method,
                              double* y, int32_t* idx, double* gates, int n_threads) {
  if (!valid(d)) return -1;
  const int64_t rows = d->T * d->H;
  const int64_t M = rows * d->K;
  std::vector<double> sr((size_t)rows * d->n_rows), sc((size_t)rows * d->n_cols);
  int rc = omnimoe_ref_half_scores(d, x, keys_row, keys_col, sr.data(), sc.data(), n_threads);
  if (rc) return rc;
  std::vector<int32_t> idx_buf(idx ? 0 : M);
  std::vector<double> g_buf(gates ? 0 : M);
  int32_t* I = idx ? idx : idx_buf.data();
  double* G = gates ? gates : g_buf.data();
  rc = omnimoe_ref_select(d, sr.data(), sc.data(), method, I, nullptr, G, nullptr, n_threads);
  if (rc) return rc;
  return omnimoe_ref_expert_forward(d, x, u, v, I, G, 1, y, n_threads);
}

int omnimoe_ref_route_dense(const omnimoe_ref_desc* d, const float* x, const float* w_gate,
                            int32_t* idx, double* gates, double* logits, int n_threads) {
  if (!valid(d)) return -1;
  const int H = d->H, K = d->K, D = d->d;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  parallel_for(d->T * H, n_threads, [&](int64_t b, int64_t e) {
    std::vector<double> L((size_t)N);
    for (int64_t th = b; th < e; ++th) {
      const int64_t t = th / H;
      const int h = (int)(th % H);
      for (int64_t n = 0; n < N; ++n)
        L[(size_t)n] = dot_row(x + t * D, w_gate + ((int64_t)h * N + n) * D, D);
      if (logits) std::copy(L.begin(), L.end(), logits + th * N);
      select_dense_row(L.data(), N, K, idx + th * K, gates + th * K);
    }
  });
  return 0;
}

int omnimoe_ref_select_dense_f32(const omnimoe_ref_desc* d, const float* logits, int32_t* idx,
                                 double* gates, int n_threads) {
  if (!valid(d)) return -1;
  const int K = d->K;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  parallel_for(d->T * d->H, n_threads, [&](int64_t b, int64_t e) {
    std::vector<double> L((size_t)N);
    for (int64_t th = b; th < e; ++th) {
      for (int64_t n = 0; n < N; ++n) L[(size_t)n] = (double)logits[th * N + n];
      select_dense_row(L.data(), N, K, idx + th * K, gates + th * K);
    }
  });
  return 0;
}

int omnimoe_ref_shared_mlp(const omnimoe_ref_desc* d, int32_t d_ff, const float* x,
                           const float* w_gu, const float* w_down, double* y, int n_threads) {
  if (!valid(d) || d_ff < 1) return -1;
  const int D = d->d;
  parallel_for(d->T, n_threads, [&](int64_t b, int64_t e) {
    std::vector<double> a((size_t)d_ff);
    for (int64_t t = b; t < e; ++t) {
      const float* xt = x + t * D;
      for (int f = 0; f < d_ff; ++f) {
        const double g = dot_row(xt, w_gu + (int64_t)f * D, D);
        const double u = dot_row(xt, w_gu + ((int64_t)d_ff + f) * D, D);
        a[(size_t)f] = silu(g) * u;
      }
      for (int c = 0; c < D; ++c) {
        double s = 0.0;
        for (int f = 0; f < d_ff; ++f) s += (double)w_down[(int64_t)c * d_ff + f] * a[(size_t)f];
        y[t * D + c] += s;
      }
    }
  });
  return 0;
}

int omnimoe_ref_expert_backward(const omnimoe_ref_desc* d, const float* x, const float* u,
                                const float* v, const int32_t* idx, const double* gates,
                                const double* dy, double* dx, double* du_rows, double* dv_rows,
                                int32_t* active, int32_t* n_active, double* dgates,
                                double* dscores, int n_threads) {
  if (!valid(d)) return -1;
  const int D = d->d, K = d->K;
  const int64_t HK = (int64_t)d->H * K;
  const int64_t M = d->T * HK;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  for (int64_t p = 0; p < M; ++p)
    if (idx[p] < 0 || idx[p] >= N) return -2;
  // per task: a_p and dh_p = da_p g_p act'(h_p); gate and score gradients per (t, h) row
  std::vector<double> a(M), dh(M);
  parallel_for(d->T * d->H, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t th = b; th < e; ++th) {
      const int64_t t = th / d->H;
      double sgd = 0.0;
      for (int k = 0; k < K; ++k) {
        const int64_t p = th * K + k;
        const int64_t ex = idx[p];
        const double h = dot_row(x + t * D, u + ex * D, D);
        double da = 0.0;
        for (int m = 0; m < D; ++m) da += dy[t * D + m] * (double)v[ex * D + m];
        a[p] = gates[p] * omnimoe_ref_act(d->act, h);
        dh[p] = da * gates[p] * omnimoe_ref_act_grad(d->act, h);
        dgates[p] = da * omnimoe_ref_act(d->act, h);
        sgd += gates[p] * dgates[p];
      }
      for (int k = 0; k < K; ++k) {
        const int64_t p = th * K + k;
        dscores[p] = gates[p] * (dgates[p] - sgd);
      }
    }
  });
  // dx: token by token over the slots
  parallel_for(d->T, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t t = b; t < e; ++t) {
      double* dxt = dx + t * D;
      for (int m = 0; m < D; ++m) dxt[m] = 0.0;
      for (int64_t s = 0; s < HK; ++s) {
        const int64_t p = t * HK + s;
        const int64_t ex = idx[p];
        for (int m = 0; m < D; ++m) dxt[m] += dh[p] * (double)u[ex * D + m];
      }
    }
  });
  // du, dv: expert by expert over the schedule's segments (tasks in id order)
  const int64_t cap = std::min(M, N);
  std::vector<int32_t> perm(M), off(cap + 2);
  int32_t A = 0;
  omnimoe_ref_desc d1 = *d;
  d1.group_size = 1;
  int rc = omnimoe_ref_schedule(&d1, idx, perm.data(), active, off.data(), &A, nullptr);
  if (rc) return rc;
  *n_active = A;
  parallel_for(A, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t r = b; r < e; ++r) {
      double* du = du_rows + r * D;
      double* dv = dv_rows + r * D;
      for (int m = 0; m < D; ++m) du[m] = dv[m] = 0.0;
      for (int64_t tau = off[r]; tau < off[r + 1]; ++tau) {
        const int64_t p = perm[tau];
        const int64_t t = p / HK;
        for (int m = 0; m < D; ++m) {
          du[m] += dh[p] * (double)x[t * D + m];
          dv[m] += a[p] * dy[t * D + m];
        }
      }
    }
  });
  return 0;
}

int omnimoe_ref_route_backward(const omnimoe_ref_desc* d, const float* x, const float* keys_row,
                               const float* keys_col, const int32_t* idx, const double* dscores,
                               double* dx, double* dkeys_row, double* dkeys_col, int n_threads) {
  if (!valid(d)) return -1;
  const int H = d->H, K = d->K, D = d->d, dk = d->d_key, nr = d->n_rows, nc = d->n_cols;
  const int c0 = d->query_mode == 0 ? dk : 0;
  const int64_t rows = d->T * H;
  const int64_t N = (int64_t)nr * nc;
  for (int64_t p = 0; p < rows * K; ++p)
    if (idx[p] < 0 || idx[p] >= N) return -2;
  // sub-key gradients: one head at a time (each head's tables are independent)
  parallel_for(H, n_threads, [&](int64_t hb, int64_t he) {
    for (int64_t h = hb; h < he; ++h) {
      double* dr = dkeys_row + h * nr * dk;
      double* dc = dkeys_col + h * nc * dk;
      std::fill(dr, dr + (int64_t)nr * dk, 0.0);
      std::fill(dc, dc + (int64_t)nc * dk, 0.0);
      for (int64_t t = 0; t < d->T; ++t)
        for (int k = 0; k < K; ++k) {
          const int64_t p = (t * H + h) * K + k;
          const int64_t i = idx[p] / nc, j = idx[p] % nc;
          for (int m = 0; m < dk; ++m) {
            dr[i * dk + m] += dscores[p] * (double)x[t * D + m];
            dc[j * dk + m] += dscores[p] * (double)x[t * D + c0 + m];
          }
        }
    }
  });
  // input gradient, token by token
  parallel_for(d->T, n_threads, [&](int64_t b, int64_t e) {
    for (int64_t t = b; t < e; ++t)
      for (int h = 0; h < H; ++h)
        for (int k = 0; k < K; ++k) {
          const int64_t p = (t * H + h) * K + k;
          const int64_t i = idx[p] / nc, j = idx[p] % nc;
          for (int m = 0; m < dk; ++m) {
            dx[t * D + m] += dscores[p] * (double)keys_row[((int64_t)h * nr + i) * dk + m];
            dx[t * D + c0 + m] += dscores[p] * (double)keys_col[((int64_t)h * nc + j) * dk + m];
          }
        }
  });
  return 0;
}

}  // extern "C"
