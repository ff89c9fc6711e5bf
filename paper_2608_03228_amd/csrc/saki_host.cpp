// Host side of libsaki: float64 calibration (Sec. 6, Eq. 2-4, Appendix A),
// the weight-SVD baseline factors, status strings and size helpers.
//
// Calibration is O(d^3) per head and runs once per model; it uses its own
// symmetric eigensolver (Householder tridiagonalisation followed by the
// implicit QL iteration with Wilkinson-type shifts, as in Golub & Van Loan,
// "Matrix Computations", Sec. 8.3) so that the library depends on no LAPACK.
//
// Two mathematically identical routes compute the factors:
//  * Cholesky route, used when the eigenvalue floor provably does not bind on
//    either moment (Cholesky of Sigma - floor_rel * ||Sigma||_F * I succeeds;
//    ||Sigma||_F >= lambda_max, so every eigenvalue is above the floor).  With
//    Sigma_k = L L^T, C' = L_q^T L has the singular values of C, and
//    M = C'^T C' = L^T Sigma_q L has eigenvectors V' = O V for the orthogonal
//    O relating L to Sigma_k^{1/2}.  Then B_q = L V'_r diag(sigma_r)^-1/2 and
//    B_k = L^{-T} V'_r diag(sigma_r)^1/2 are exactly Eq. 4's factors (the
//    square root chosen does not matter) at one eigendecomposition per head.
//  * Symmetric route otherwise: clamped eigendecompositions of both moments,
//    C = Sigma_q^{1/2} Sigma_k^{1/2}, V and sigma^2 from the eigenvalues of
//    C^T C, U_r = C V_r diag(sigma_r)^-1.
// Either way each singular pair is signed so that the largest-magnitude
// entry of its B_k column is positive (lowest index on ties).

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

// S = (1/T) sum_t (x_t - mu)(x_t - mu)^T for the T rows of X (float, T x d);
// mu may be null (uncentred).  Four tokens per sweep over the triangle.
void moment(int T, int d, const float* X, const double* mu, double* S) {
  std::fill(S, S + (size_t)d * d, 0.0);
  std::vector<double> x((size_t)4 * d);
  for (int t0 = 0; t0 < T; t0 += 4) {
    const int nb = std::min(4, T - t0);
    for (int b = 0; b < 4; ++b)
      for (int i = 0; i < d; ++i)
        x[(size_t)b * d + i] = b < nb ? (double)X[(size_t)(t0 + b) * d + i] - (mu ? mu[i] : 0.0) : 0.0;
    const double *x0 = x.data(), *x1 = x0 + d, *x2 = x1 + d, *x3 = x2 + d;
    for (int i = 0; i < d; ++i) {
      double* row = S + (size_t)i * d;
      const double a0 = x0[i], a1 = x1[i], a2 = x2[i], a3 = x3[i];
      for (int j = 0; j <= i; ++j) row[j] += a0 * x0[j] + a1 * x1[j] + a2 * x2[j] + a3 * x3[j];
    }
  }
  for (int i = 0; i < d; ++i)
    for (int j = 0; j <= i; ++j) {
      const double v = S[(size_t)i * d + j] / (double)T;
      S[(size_t)i * d + j] = v;
      S[(size_t)j * d + i] = v;
    }
}

// Lower Cholesky factor of S - shift * I (row-major, upper part zero).
// Returns false unless every pivot is positive.
bool cholesky(int n, const double* S, double shift, double* L) {
  std::fill(L, L + (size_t)n * n, 0.0);
  for (int j = 0; j < n; ++j) {
    const double* lj = L + (size_t)j * n;
    double dsum = S[(size_t)j * n + j] - shift;
    for (int k = 0; k < j; ++k) dsum -= lj[k] * lj[k];
    if (!(dsum > 0.0) || !std::isfinite(dsum)) return false;
    const double piv = std::sqrt(dsum);
    L[(size_t)j * n + j] = piv;
    for (int i = j + 1; i < n; ++i) {
      const double* li = L + (size_t)i * n;
      double acc = S[(size_t)i * n + j];
      for (int k = 0; k < j; ++k) acc -= li[k] * lj[k];
      L[(size_t)i * n + j] = acc / piv;
    }
  }
  return true;
}

double frobenius(int n, const double* S) {
  double acc = 0.0;
  for (size_t i = 0; i < (size_t)n * n; ++i) acc += S[i] * S[i];
  return std::sqrt(acc);
}

// True when no eigenvalue of the PSD moment lies below floor_rel * lambda_max
// (sufficient test); L then holds the Cholesky factor of S itself.
bool unclamped_cholesky(int n, const double* S, double floor_rel, double* L) {
  const double f = frobenius(n, S);
  if (!(f > 0.0) || !std::isfinite(f)) return false;
  if (!cholesky(n, S, floor_rel * f, L)) return false;
  return cholesky(n, S, 0.0, L);
}

// Flip column m of both factors (d x r, row-major, float output) when the
// largest-magnitude entry of the B_k column is negative.
void store_pair(int d, int r, int m, const double* bq, const double* bk, float* Bq, float* Bk) {
  int jmax = 0;
  double amax = std::fabs(bk[0]);
  for (int j = 1; j < d; ++j)
    if (std::fabs(bk[j]) > amax) { amax = std::fabs(bk[j]); jmax = j; }
  const double sgn = bk[jmax] < 0 ? -1.0 : 1.0;
  for (int i = 0; i < d; ++i) {
    Bq[(size_t)i * r + m] = (float)(sgn * bq[i]);
    Bk[(size_t)i * r + m] = (float)(sgn * bk[i]);
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
  Mat half, ihalf;         // Sigma_k^{1/2}, Sigma_k^{-1/2} (symmetric route)
  Mat L;                   // Cholesky factor of Sigma_k (Cholesky route)
  std::vector<double> mu;  // key mean
  Mat sk;                  // Sigma_k
  int n_clamped = 0;
  bool chol = false;       // the floor provably does not bind on Sigma_k
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
    // ---- per KV head: key mean, centred key moment, and either its Cholesky
    //      factor or its clamped symmetric roots
    std::vector<KvState> kv(H_kv);
    parallel_for(H_kv, n_threads, [&](int g) {
      KvState& st = kv[g];
      const float* k = k_cal + (size_t)g * T * d;
      st.mu.assign(d, 0.0);
      for (int t = 0; t < T; ++t)
        for (int i = 0; i < d; ++i) st.mu[i] += (double)k[(size_t)t * d + i];
      for (int i = 0; i < d; ++i) st.mu[i] /= (double)T;
      st.sk.resize(dd);
      moment(T, d, k, st.mu.data(), st.sk.data());
      if (method == SAKI_METHOD_OPT) {
        st.L.resize(dd);
        st.chol = unclamped_cholesky(d, st.sk.data(), floor_rel, st.L.data());
        if (st.chol) {
          st.ok = true;
        } else {
          st.half.resize(dd);
          st.ihalf.resize(dd);
          st.ok = clamped_roots(d, st.sk.data(), floor_rel, st.half.data(), st.ihalf.data(),
                                &st.n_clamped);
        }
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
      // Sigma_q (uncentred)
      const float* q = q_cal + (size_t)h * T * d;
      Mat sq(dd);
      moment(T, d, q, nullptr, sq.data());
      std::vector<double> sig(d), bqc(d), bkc(d);
      Mat scratch(dd);
      if (st.chol && unclamped_cholesky(d, sq.data(), floor_rel, scratch.data())) {
        // ---- Cholesky route: M = L^T Sigma_q L, B_q = L v / sqrt(s), B_k = L^-T v sqrt(s)
        const double* L = st.L.data();
        Mat W(dd, 0.0), M(dd, 0.0);
        for (int i = 0; i < d; ++i) {  // W = Sigma_q L  (L lower: column j uses rows k >= j)
          const double* si = sq.data() + (size_t)i * d;
          double* wi = W.data() + (size_t)i * d;
          for (int k = 0; k < d; ++k) {
            const double a = si[k];
            const double* lk = L + (size_t)k * d;
            for (int j = 0; j <= k; ++j) wi[j] += a * lk[j];
          }
        }
        for (int k = 0; k < d; ++k) {  // M = L^T W: row i gathers rows k >= i of W
          const double* lk = L + (size_t)k * d;
          const double* wk = W.data() + (size_t)k * d;
          for (int i = 0; i <= k; ++i) {
            const double a = lk[i];
            double* mi = M.data() + (size_t)i * d;
            for (int j = 0; j < d; ++j) mi[j] += a * wk[j];
          }
        }
        std::vector<double> w(d), vt(dd);
        if (!sym_eig_rows(d, M.data(), w.data(), vt.data())) { failed = 1; return; }
        for (int m = 0; m < d; ++m) sig[m] = std::sqrt(std::max(w[d - 1 - m], 0.0));
        for (int m = 0; m < r; ++m) {
          const double* v = vt.data() + (size_t)(d - 1 - m) * d;
          const double sm = sig[m], rs = std::sqrt(sm);
          for (int i = 0; i < d; ++i) {  // L v
            const double* li = L + (size_t)i * d;
            double acc = 0.0;
            for (int j = 0; j <= i; ++j) acc += li[j] * v[j];
            bqc[i] = sm > 0.0 ? acc / rs : 0.0;
          }
          for (int i = d - 1; i >= 0; --i) {  // L^T x = v (back substitution)
            double acc = v[i];
            for (int k = i + 1; k < d; ++k) acc -= L[(size_t)k * d + i] * bkc[k];
            bkc[i] = acc / L[(size_t)i * d + i];
          }
          for (int i = 0; i < d; ++i) bkc[i] *= rs;
          store_pair(d, r, m, bqc.data(), bkc.data(), bq, bk);
        }
        if (sigma)
          for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
        if (n_clamped) { n_clamped[2 * h] = 0; n_clamped[2 * h + 1] = 0; }
        return;
      }
      // ---- symmetric route: clamped roots of both moments
      Mat qh(dd), qih(dd);
      int nq = 0;
      if (!clamped_roots(d, sq.data(), floor_rel, qh.data(), qih.data(), &nq)) { failed = 1; return; }
      Mat kh_local, kih_local;
      const double* khalf = st.half.data();
      const double* kihalf = st.ihalf.data();
      int nk = st.n_clamped;
      if (st.chol) {  // Sigma_k took the Cholesky route: its roots are needed here only
        kh_local.resize(dd);
        kih_local.resize(dd);
        if (!clamped_roots(d, st.sk.data(), floor_rel, kh_local.data(), kih_local.data(), &nk)) {
          failed = 1;
          return;
        }
        khalf = kh_local.data();
        kihalf = kih_local.data();
      }
      // C = Sigma_q^{1/2} Sigma_k^{1/2};  C^T C -> V, sigma^2
      Mat C(dd), Ct(dd), CtC(dd);
      matmul(d, qh.data(), khalf, C.data());
      for (int i = 0; i < d; ++i)
        for (int j = 0; j < d; ++j) Ct[(size_t)j * d + i] = C[(size_t)i * d + j];
      matmul(d, Ct.data(), C.data(), CtC.data());
      std::vector<double> w(d), vt(dd);
      if (!sym_eig_rows(d, CtC.data(), w.data(), vt.data())) { failed = 1; return; }
      for (int m = 0; m < d; ++m) sig[m] = std::sqrt(std::max(w[d - 1 - m], 0.0));
      if (sigma)
        for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
      if (n_clamped) { n_clamped[2 * h] = nq; n_clamped[2 * h + 1] = nk; }
      // top-r pairs: v_m (row of vt), u_m = C v_m / sigma_m
      std::vector<double> u(d);
      for (int m = 0; m < r; ++m) {
        const double* v = vt.data() + (size_t)(d - 1 - m) * d;
        const double sm = sig[m];
        for (int i = 0; i < d; ++i) {
          double acc = 0.0;
          const double* ci = C.data() + (size_t)i * d;
          for (int j = 0; j < d; ++j) acc += ci[j] * v[j];
          u[i] = sm > 0.0 ? acc / sm : 0.0;
        }
        const double rs = std::sqrt(sm);
        // B_q[:, m] = Sigma_q^{-1/2} u sqrt(s);  B_k[:, m] = Sigma_k^{-1/2} v sqrt(s)
        for (int i = 0; i < d; ++i) {
          const double* ai = qih.data() + (size_t)i * d;
          const double* bi = kihalf + (size_t)i * d;
          double aq = 0.0, ak = 0.0;
          for (int j = 0; j < d; ++j) { aq += ai[j] * u[j]; ak += bi[j] * v[j]; }
          bqc[i] = aq * rs;
          bkc[i] = ak * rs;
        }
        store_pair(d, r, m, bqc.data(), bkc.data(), bq, bk);
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

size_t saki_recall_workspace_bytes(int B, int H_q, int H_kv, int Q, int N_valid, int d, int k) {
  if (B <= 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || Q < 0 || N_valid < 0 ||
      d != saki::kHeadDim || k < 1 || k > saki::kMaxK)
    return 0;
  return saki::recall_plan(B, H_q, H_kv, Q, N_valid).ws_bytes;
}

}  // extern "C"
