// Host side of libsaki: float64 calibration (Sec. 6, Eq. 2-4, Appendix A),
// the weight-SVD baseline factors, status strings and size helpers.
//
// Calibration is O(d^3) per head and runs once per model; it uses its own
// symmetric eigensolver (Householder tridiagonalisation followed by the
// implicit QL iteration with Wilkinson-type shifts, as in Golub & Van Loan,
// "Matrix Computations", Sec. 8.3) so that the library depends on no LAPACK.
// The SVD of C is taken from the eigendecomposition of C^T C: V are its
// eigenvectors, sigma_i^2 its eigenvalues, and U_r = C V_r diag(sigma_r)^-1.

#include "saki.h"
#include "saki_internal.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <limits>
#include <new>
#include <thread>
#include <vector>

namespace {

using Mat = std::vector<double>;  // row-major square matrix

// C = A * B for n x n row-major matrices (i-k-j order, contiguous inner loop).
void matmul(int n, const double* A, const double* B, double* C) {
  std::fill(C, C + (size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) {
    double* ci = C + (size_t)i * n;
    for (int k = 0; k < n; ++k) {
      const double a = A[(size_t)i * n + k];
      const double* bk = B + (size_t)k * n;
      for (int j = 0; j < n; ++j) ci[j] += a * bk[j];
    }
  }
}

// Reduce symmetric `a` (n x n, overwritten) to tridiagonal form T = Q^T A Q.
// On return diag/off hold T's diagonal and sub-diagonal (off[n-1] = 0) and
// `q` (n x n row-major) holds Q.
void tridiagonalize(int n, double* a, double* diag, double* off, double* q) {
  std::fill(q, q + (size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) q[(size_t)i * n + i] = 1.0;
  std::vector<double> v(n), p(n), w(n);
  for (int k = 0; k + 2 < n; ++k) {
    const int m = n - k - 1;  // length of the column part below the diagonal
    double sumsq = 0.0;
    for (int i = 0; i < m; ++i) {
      const double x = a[(size_t)(k + 1 + i) * n + k];
      v[i] = x;
      sumsq += x * x;
    }
    const double x0 = v[0];
    double alpha = std::sqrt(sumsq);
    if (alpha == 0.0) continue;              // column already reduced
    if (x0 > 0) alpha = -alpha;              // reflect away from x0's sign
    v[0] = x0 - alpha;
    const double vv = sumsq - x0 * x0 + v[0] * v[0];
    if (vv == 0.0) continue;
    const double beta = 2.0 / vv;
    // p = beta * A22 v,  K = beta/2 * v.p,  w = p - K v
    for (int i = 0; i < m; ++i) {
      const double* ai = a + (size_t)(k + 1 + i) * n + (k + 1);
      double s = 0.0;
      for (int j = 0; j < m; ++j) s += ai[j] * v[j];
      p[i] = beta * s;
    }
    double vp = 0.0;
    for (int i = 0; i < m; ++i) vp += v[i] * p[i];
    const double K = 0.5 * beta * vp;
    for (int i = 0; i < m; ++i) w[i] = p[i] - K * v[i];
    // A22 -= v w^T + w v^T
    for (int i = 0; i < m; ++i) {
      double* ai = a + (size_t)(k + 1 + i) * n + (k + 1);
      const double vi = v[i], wi = w[i];
      for (int j = 0; j < m; ++j) ai[j] -= vi * w[j] + wi * v[j];
    }
    // column/row k now has a single sub-diagonal entry alpha
    for (int i = 0; i < m; ++i) {
      a[(size_t)(k + 1 + i) * n + k] = (i == 0) ? alpha : 0.0;
      a[(size_t)k * n + (k + 1 + i)] = (i == 0) ? alpha : 0.0;
    }
    // Q <- Q (I - beta v v^T) on columns k+1 .. n-1
    for (int r = 0; r < n; ++r) {
      double* qr = q + (size_t)r * n + (k + 1);
      double s = 0.0;
      for (int j = 0; j < m; ++j) s += qr[j] * v[j];
      s *= beta;
      for (int j = 0; j < m; ++j) qr[j] -= s * v[j];
    }
  }
  for (int i = 0; i < n; ++i) diag[i] = a[(size_t)i * n + i];
  for (int i = 0; i + 1 < n; ++i) off[i] = a[(size_t)(i + 1) * n + i];
  off[n - 1] = 0.0;
}

// Implicit QL on the tridiagonal (diag, off).  zt holds the transpose of the
// accumulated orthogonal matrix (row i = current column i), so that the
// rotations update two contiguous rows.  Returns false without convergence.
bool tridiag_ql(int n, double* diag, double* off, double* zt) {
  const double eps = std::numeric_limits<double>::epsilon();
  // Deflation test: relative to the neighbouring diagonal entries, or
  // absolute at eps * ||T|| (an off-diagonal that small moves any eigenvalue
  // by at most eps * ||T||); the absolute test ends the iteration on blocks
  // of (near-)zero eigenvalues, where a purely relative test never does.
  double tnorm = 0.0;
  for (int i = 0; i < n; ++i) tnorm = std::max(tnorm, std::fabs(diag[i]) + std::fabs(off[i]));
  const double abs_tol = eps * tnorm;
  for (int l = 0; l < n; ++l) {
    int iter = 0;
    for (;;) {
      int m = l;
      for (; m + 1 < n; ++m) {
        const double scale = std::fabs(diag[m]) + std::fabs(diag[m + 1]);
        if (std::fabs(off[m]) <= std::max(eps * scale, abs_tol)) break;
      }
      if (m == l) break;
      if (++iter > 80) return false;
      // shift from the leading 2x2 block of the unreduced part
      double g = (diag[l + 1] - diag[l]) / (2.0 * off[l]);
      double rad = std::hypot(g, 1.0);
      g = diag[m] - diag[l] + off[l] / (g + std::copysign(rad, g));
      double s = 1.0, c = 1.0, p = 0.0;
      bool split = false;
      for (int i = m - 1; i >= l; --i) {
        const double f = s * off[i];
        const double b = c * off[i];
        rad = std::hypot(f, g);
        off[i + 1] = rad;
        if (rad == 0.0) {  // an off-diagonal underflowed: deflate and restart
          diag[i + 1] -= p;
          off[m] = 0.0;
          split = true;
          break;
        }
        s = f / rad;
        c = g / rad;
        g = diag[i + 1] - p;
        rad = (diag[i] - g) * s + 2.0 * c * b;
        p = s * rad;
        diag[i + 1] = g + p;
        g = c * rad - b;
        double* zi = zt + (size_t)i * n;
        double* zj = zt + (size_t)(i + 1) * n;
        for (int k = 0; k < n; ++k) {
          const double zik = zi[k], zjk = zj[k];
          zj[k] = s * zik + c * zjk;
          zi[k] = c * zik - s * zjk;
        }
      }
      if (split) continue;
      diag[l] -= p;
      off[l] = g;
      off[m] = 0.0;
    }
  }
  return true;
}

// Eigen-decomposition of symmetric A (n x n row-major).  w ascending; vt row j
// = eigenvector j.  Returns false on non-convergence or non-finite input.
bool sym_eig_rows(int n, const double* A, double* w, double* vt) {
  for (size_t i = 0; i < (size_t)n * n; ++i)
    if (!std::isfinite(A[i])) return false;
  Mat a(A, A + (size_t)n * n), q((size_t)n * n), zt((size_t)n * n);
  // symmetrise exactly
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < i; ++j) {
      const double s = 0.5 * (a[(size_t)i * n + j] + a[(size_t)j * n + i]);
      a[(size_t)i * n + j] = a[(size_t)j * n + i] = s;
    }
  std::vector<double> diag(n), off(n);
  tridiagonalize(n, a.data(), diag.data(), off.data(), q.data());
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < n; ++j) zt[(size_t)j * n + i] = q[(size_t)i * n + j];
  if (!tridiag_ql(n, diag.data(), off.data(), zt.data())) return false;
  std::vector<int> order(n);
  for (int i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int x, int y) { return diag[x] < diag[y]; });
  for (int i = 0; i < n; ++i) {
    w[i] = diag[order[i]];
    std::memcpy(vt + (size_t)i * n, zt.data() + (size_t)order[i] * n, sizeof(double) * n);
  }
  return true;
}

// Flip the sign of row `v` (length n) -- and of `u` if given -- so that its
// largest-magnitude entry (lowest index on ties) is positive.
void canonical_sign(int n, double* v, double* u) {
  int jmax = 0;
  double amax = std::fabs(v[0]);
  for (int j = 1; j < n; ++j)
    if (std::fabs(v[j]) > amax) { amax = std::fabs(v[j]); jmax = j; }
  if (v[jmax] < 0) {
    for (int j = 0; j < n; ++j) v[j] = -v[j];
    if (u)
      for (int j = 0; j < n; ++j) u[j] = -u[j];
  }
}

// Clamped symmetric roots of a PSD moment (Appendix A, reading: clamp).
bool clamped_roots(int n, const double* S, double floor_rel, double* half,
                   double* ihalf, int* n_clamped) {
  std::vector<double> w(n), vt((size_t)n * n);
  if (!sym_eig_rows(n, S, w.data(), vt.data())) return false;
  const double lmax = w[n - 1];
  int cnt = 0;
  if (!(lmax > 0.0)) {
    for (int i = 0; i < n; ++i) w[i] = 1.0;
    cnt = n;
  } else {
    const double floor = floor_rel * lmax;
    for (int i = 0; i < n; ++i)
      if (w[i] < floor) { w[i] = floor; ++cnt; }
  }
  // half = V diag(sqrt w) V^T = sum_i sqrt(w_i) v_i v_i^T
  std::fill(half, half + (size_t)n * n, 0.0);
  std::fill(ihalf, ihalf + (size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) {
    const double sw = std::sqrt(w[i]), isw = 1.0 / sw;
    const double* v = vt.data() + (size_t)i * n;
    for (int a = 0; a < n; ++a) {
      const double va = v[a];
      double* h = half + (size_t)a * n;
      double* ih = ihalf + (size_t)a * n;
      const double sa = sw * va, ia = isw * va;
      for (int b = 0; b < n; ++b) { h[b] += sa * v[b]; ih[b] += ia * v[b]; }
    }
  }
  if (n_clamped) *n_clamped = cnt;
  return true;
}

// Run fn(i) for i in [0, count) on up to n_threads threads.
template <class F>
void parallel_for(int count, int n_threads, F fn) {
  int nt = n_threads > 0 ? n_threads : (int)std::thread::hardware_concurrency();
  if (n_threads <= 0) nt = std::min(nt, 16);
  nt = std::max(1, std::min(nt, count));
  if (nt == 1) {
    for (int i = 0; i < count; ++i) fn(i);
    return;
  }
  std::atomic<int> next(0);
  std::vector<std::thread> pool;
  pool.reserve(nt);
  for (int t = 0; t < nt; ++t)
    pool.emplace_back([&]() {
      for (int i = next.fetch_add(1); i < count; i = next.fetch_add(1)) fn(i);
    });
  for (auto& th : pool) th.join();
}

struct KvState {
  Mat half, ihalf;         // Sigma_k^{1/2}, Sigma_k^{-1/2}
  std::vector<double> mu;  // key mean
  Mat sk;                  // Sigma_k
  int n_clamped = 0;
  bool ok = false;
};

}  // namespace

extern "C" {

const char* saki_status_string(int status) {
  switch (status) {
    case SAKI_OK: return "ok";
    case SAKI_ERR_ARG: return "invalid argument (null pointer or inconsistent size)";
    case SAKI_ERR_UNSUPPORTED: return "unsupported size or dtype (GPU path: d=128, r in {16,32,64,128}, 1<=k<=64)";
    case SAKI_ERR_WORKSPACE: return "workspace or index buffer too small";
    case SAKI_ERR_NOMEM: return "host allocation failed or size overflow";
    case SAKI_ERR_HIP: return "HIP runtime or kernel launch error";
    case SAKI_ERR_NUMERIC: return "non-finite input or eigensolver did not converge";
    default: return "unknown status";
  }
}

int saki_version(void) { return 1; }

int saki_sym_eig(int n, const double* A, double* w, double* V) {
  if (n <= 0 || n > 4096 || !A || !w || !V) return SAKI_ERR_ARG;
  try {
    std::vector<double> vt((size_t)n * n);
    if (!sym_eig_rows(n, A, w, vt.data())) return SAKI_ERR_NUMERIC;
    for (int i = 0; i < n; ++i)
      for (int j = 0; j < n; ++j) V[(size_t)j * n + i] = vt[(size_t)i * n + j];
  } catch (const std::bad_alloc&) {
    return SAKI_ERR_NOMEM;
  }
  return SAKI_OK;
}

int saki_calibrate(const float* q_cal, const float* k_cal, int H_q, int H_kv,
                   int T, int d, int r, int method, double floor_rel,
                   float* B_q, float* B_k, float* mu, double* sigma,
                   int* n_clamped, int n_threads) {
  if (!q_cal || !k_cal || !B_q || !B_k || !mu) return SAKI_ERR_ARG;
  if (H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || T <= 0 || d <= 0 || d > 4096 ||
      r <= 0 || r > d || !(floor_rel >= 0.0))
    return SAKI_ERR_ARG;
  if (method != SAKI_METHOD_OPT && method != SAKI_METHOD_KEY_PCA) return SAKI_ERR_UNSUPPORTED;
  const int G = H_q / H_kv;
  const size_t dd = (size_t)d * d;
  try {
    // ---- per KV head: key mean, centred key moment and its clamped roots
    std::vector<KvState> kv(H_kv);
    parallel_for(H_kv, n_threads, [&](int g) {
      KvState& st = kv[g];
      const float* k = k_cal + (size_t)g * T * d;
      st.mu.assign(d, 0.0);
      for (int t = 0; t < T; ++t)
        for (int i = 0; i < d; ++i) st.mu[i] += (double)k[(size_t)t * d + i];
      for (int i = 0; i < d; ++i) st.mu[i] /= (double)T;
      st.sk.assign(dd, 0.0);
      std::vector<double> kc(d);
      for (int t = 0; t < T; ++t) {
        for (int i = 0; i < d; ++i) kc[i] = (double)k[(size_t)t * d + i] - st.mu[i];
        for (int i = 0; i < d; ++i) {
          double* row = st.sk.data() + (size_t)i * d;
          const double ki = kc[i];
          for (int j = 0; j <= i; ++j) row[j] += ki * kc[j];
        }
      }
      for (int i = 0; i < d; ++i)
        for (int j = 0; j <= i; ++j) {
          const double v = st.sk[(size_t)i * d + j] / (double)T;
          st.sk[(size_t)i * d + j] = v;
          st.sk[(size_t)j * d + i] = v;
        }
      if (method == SAKI_METHOD_OPT) {
        st.half.resize(dd);
        st.ihalf.resize(dd);
        st.ok = clamped_roots(d, st.sk.data(), floor_rel, st.half.data(),
                              st.ihalf.data(), &st.n_clamped);
      } else {
        st.ok = true;
      }
      for (int i = 0; i < d; ++i) mu[(size_t)g * d + i] = (float)st.mu[i];
    });
    for (int g = 0; g < H_kv; ++g)
      if (!kv[g].ok) return SAKI_ERR_NUMERIC;

    std::atomic<int> failed(0);
    parallel_for(H_q, n_threads, [&](int h) {
      const KvState& st = kv[h / G];
      float* bq = B_q + (size_t)h * d * r;
      float* bk = B_k + (size_t)h * d * r;
      if (method == SAKI_METHOD_KEY_PCA) {
        std::vector<double> w(d), vt(dd);
        if (!sym_eig_rows(d, st.sk.data(), w.data(), vt.data())) { failed = 1; return; }
        for (int m = 0; m < r; ++m) {
          double* v = vt.data() + (size_t)(d - 1 - m) * d;  // m-th largest
          canonical_sign(d, v, nullptr);
          for (int i = 0; i < d; ++i) bq[(size_t)i * r + m] = bk[(size_t)i * r + m] = (float)v[i];
        }
        if (sigma)
          for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = w[d - 1 - m];
        if (n_clamped) { n_clamped[2 * h] = 0; n_clamped[2 * h + 1] = 0; }
        return;
      }
      // Sigma_q (uncentred) and its clamped roots
      const float* q = q_cal + (size_t)h * T * d;
      Mat sq(dd, 0.0);
      std::vector<double> qt(d);
      for (int t = 0; t < T; ++t) {
        for (int i = 0; i < d; ++i) qt[i] = (double)q[(size_t)t * d + i];
        for (int i = 0; i < d; ++i) {
          double* row = sq.data() + (size_t)i * d;
          const double qi = qt[i];
          for (int j = 0; j <= i; ++j) row[j] += qi * qt[j];
        }
      }
      for (int i = 0; i < d; ++i)
        for (int j = 0; j <= i; ++j) {
          const double v = sq[(size_t)i * d + j] / (double)T;
          sq[(size_t)i * d + j] = v;
          sq[(size_t)j * d + i] = v;
        }
      Mat qh(dd), qih(dd);
      int nq = 0;
      if (!clamped_roots(d, sq.data(), floor_rel, qh.data(), qih.data(), &nq)) { failed = 1; return; }
      // C = Sigma_q^{1/2} Sigma_k^{1/2};  C^T C -> V, sigma^2
      Mat C(dd), Ct(dd), CtC(dd);
      matmul(d, qh.data(), st.half.data(), C.data());
      for (int i = 0; i < d; ++i)
        for (int j = 0; j < d; ++j) Ct[(size_t)j * d + i] = C[(size_t)i * d + j];
      matmul(d, Ct.data(), C.data(), CtC.data());
      std::vector<double> w(d), vt(dd);
      if (!sym_eig_rows(d, CtC.data(), w.data(), vt.data())) { failed = 1; return; }
      std::vector<double> sig(d);
      for (int m = 0; m < d; ++m) sig[m] = std::sqrt(std::max(w[d - 1 - m], 0.0));
      if (sigma)
        for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
      if (n_clamped) { n_clamped[2 * h] = nq; n_clamped[2 * h + 1] = st.n_clamped; }
      // top-r pairs: v_m (row of vt), u_m = C v_m / sigma_m
      std::vector<double> v(d), u(d), colq(d), colk(d);
      for (int m = 0; m < r; ++m) {
        std::memcpy(v.data(), vt.data() + (size_t)(d - 1 - m) * d, sizeof(double) * d);
        const double s = sig[m];
        if (s > 0.0) {
          for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            const double* ci = C.data() + (size_t)i * d;
            for (int j = 0; j < d; ++j) acc += ci[j] * v[j];
            u[i] = acc / s;
          }
        } else {
          std::fill(u.begin(), u.end(), 0.0);
        }
        canonical_sign(d, v.data(), u.data());
        const double rs = std::sqrt(s);
        // B_q[:, m] = Sigma_q^{-1/2} u sqrt(s);  B_k[:, m] = Sigma_k^{-1/2} v sqrt(s)
        for (int i = 0; i < d; ++i) {
          const double* ai = qih.data() + (size_t)i * d;
          const double* bi = st.ihalf.data() + (size_t)i * d;
          double aq = 0.0, ak = 0.0;
          for (int j = 0; j < d; ++j) { aq += ai[j] * u[j]; ak += bi[j] * v[j]; }
          bq[(size_t)i * r + m] = (float)(aq * rs);
          bk[(size_t)i * r + m] = (float)(ak * rs);
        }
      }
    });
    if (failed) return SAKI_ERR_NUMERIC;
  } catch (const std::bad_alloc&) {
    return SAKI_ERR_NOMEM;
  }
  return SAKI_OK;
}

int saki_weight_svd_factors(const double* W_K, int H_q, int H_kv, int d, int D,
                            int r, float* B_q, float* B_k) {
  if (!W_K || !B_q || !B_k) return SAKI_ERR_ARG;
  if (H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || d <= 0 || d > 4096 || D <= 0 ||
      r <= 0 || r > d)
    return SAKI_ERR_ARG;
  const int G = H_q / H_kv;
  try {
    for (int g = 0; g < H_kv; ++g) {
      const double* w = W_K + (size_t)g * d * D;
      Mat wwt((size_t)d * d, 0.0);
      for (int i = 0; i < d; ++i)
        for (int j = 0; j <= i; ++j) {
          double acc = 0.0;
          for (int c = 0; c < D; ++c) acc += w[(size_t)i * D + c] * w[(size_t)j * D + c];
          wwt[(size_t)i * d + j] = wwt[(size_t)j * d + i] = acc;
        }
      std::vector<double> ev(d), vt((size_t)d * d);
      if (!sym_eig_rows(d, wwt.data(), ev.data(), vt.data())) return SAKI_ERR_NUMERIC;
      for (int m = 0; m < r; ++m) {
        double* v = vt.data() + (size_t)(d - 1 - m) * d;
        canonical_sign(d, v, nullptr);
        for (int h = g * G; h < (g + 1) * G; ++h)
          for (int i = 0; i < d; ++i)
            B_q[((size_t)h * d + i) * r + m] = B_k[((size_t)h * d + i) * r + m] = (float)v[i];
      }
    }
  } catch (const std::bad_alloc&) {
    return SAKI_ERR_NOMEM;
  }
  return SAKI_OK;
}

size_t saki_index_bytes(int B, int H_q, int N_cap, int r, int sketch_dtype) {
  if (B <= 0 || H_q <= 0 || N_cap < 0 || !saki::rank_supported(r) ||
      (sketch_dtype != SAKI_F32 && sketch_dtype != SAKI_BF16))
    return 0;
  return saki::index_bytes(B, H_q, N_cap, r, sketch_dtype);
}

size_t saki_score_topk_workspace_bytes(int B, int H_q, int Q, int N_valid, int r,
                                       int k, int sketch_dtype) {
  if (B <= 0 || H_q <= 0 || Q < 0 || N_valid < 0 || !saki::rank_supported(r) ||
      k < 1 || k > saki::kMaxK || (sketch_dtype != SAKI_F32 && sketch_dtype != SAKI_BF16))
    return 0;
  return saki::score_plan(B, H_q, Q, N_valid, r).ws_bytes;
}

size_t saki_recall_workspace_bytes(int B, int H_q, int Q, int N_valid, int d, int k) {
  if (B <= 0 || H_q <= 0 || Q < 0 || N_valid < 0 || d != saki::kHeadDim || k < 1 ||
      k > saki::kMaxK)
    return 0;
  return saki::recall_plan(B, H_q, Q, N_valid).ws_bytes;
}

}  // extern "C"
