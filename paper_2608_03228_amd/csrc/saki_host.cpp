// Host side of libsaki: float64 calibration (Sec. 6, Eq. 2-4, Appendix A),
// the weight-SVD baseline factors, status strings and size helpers.
//
// Calibration is O(d^3) per head and runs once per model; it uses its own
// symmetric eigensolver (Householder tridiagonalisation followed by implicit
// symmetric QR steps with the Wilkinson shift, Golub & Van Loan, "Matrix
// Computations", Sec. 8.3) so that the library depends on no LAPACK.
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

#include <immintrin.h>

#include <algorithm>
#include <unistd.h>

#include <atomic>
#include <condition_variable>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <functional>
#include <limits>
#include <memory>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

namespace {

using Mat = std::vector<double>;  // row-major square matrix

// A matrix buffer owned by the calling thread and kept between calls (the
// pool's workers live on), so the per-head d x d temporaries are not
// allocated, page-faulted and returned to the system on every call.  Slots
// 0-1 belong to the per-head calibration steps, 2-3 to sym_eig_top and 4
// to congruence_lower.
double* thread_buffer(int slot, size_t n) {
  thread_local std::vector<double> buf[5];
  if (buf[slot].size() < n) buf[slot].resize(n);
  return buf[slot].data();
}

// Per-call buffers larger than one matrix (a d x d block per head) come
// from this process-wide cache and go back to it when the call ends, so
// their pages are touched once, not on every call.  At most four are kept.
class BufferCache {
 public:
  struct Buf {
    std::unique_ptr<double[]> p;
    size_t n = 0;
  };
  static Buf take(size_t n) {
    {
      std::lock_guard<std::mutex> lk(mutex());
      auto& f = list();
      for (size_t i = 0; i < f.size(); ++i)
        if (f[i].n >= n) {
          Buf b = std::move(f[i]);
          f.erase(f.begin() + (long)i);
          return b;
        }
    }
    Buf b;
    b.p.reset(new double[n]);
    b.n = n;
    return b;
  }
  static void give(Buf b) {
    std::lock_guard<std::mutex> lk(mutex());
    auto& f = list();
    if (f.size() < 4) f.push_back(std::move(b));
  }

 private:
  static std::mutex& mutex() {
    static std::mutex m;
    return m;
  }
  static std::vector<Buf>& list() {
    static std::vector<Buf> f;
    return f;
  }
};

// A cached buffer for the lifetime of a scope.
struct ScopedBuffer {
  BufferCache::Buf b;
  explicit ScopedBuffer(size_t n) : b(BufferCache::take(n)) {}
  ~ScopedBuffer() { BufferCache::give(std::move(b)); }
  double* data() { return b.p.get(); }
};


// ---------------------------------------------------------------- AVX2 kernels
// The library is built for x86-64-v3 hosts (AVX2 + FMA); these helpers keep
// the O(T d^2) and O(d^3) steps of the calibration in 256-bit registers.

inline double hsum(__m256d v) {
  const __m128d lo = _mm256_castpd256_pd128(v), hi = _mm256_extractf128_pd(v, 1);
  const __m128d s = _mm_add_pd(lo, hi);
  return _mm_cvtsd_f64(_mm_add_sd(s, _mm_unpackhi_pd(s, s)));
}

// True when every x[i] is finite: x * 0 is NaN exactly for infinities and
// NaNs, and a NaN survives the sum.
bool all_finite(const double* x, size_t n) {
  __m256d s0 = _mm256_setzero_pd(), s1 = _mm256_setzero_pd();
  const __m256d zero = _mm256_setzero_pd();
  size_t i = 0;
  for (; i + 8 <= n; i += 8) {
    s0 = _mm256_add_pd(s0, _mm256_mul_pd(_mm256_loadu_pd(x + i), zero));
    s1 = _mm256_add_pd(s1, _mm256_mul_pd(_mm256_loadu_pd(x + i + 4), zero));
  }
  double acc = hsum(_mm256_add_pd(s0, s1));
  for (; i < n; ++i) acc += x[i] * 0.0;
  return acc == 0.0;
}

// sum_i a[i] * b[i]
double dot(const double* a, const double* b, int n) {
  __m256d s0 = _mm256_setzero_pd(), s1 = _mm256_setzero_pd();
  int i = 0;
  for (; i + 8 <= n; i += 8) {
    s0 = _mm256_fmadd_pd(_mm256_loadu_pd(a + i), _mm256_loadu_pd(b + i), s0);
    s1 = _mm256_fmadd_pd(_mm256_loadu_pd(a + i + 4), _mm256_loadu_pd(b + i + 4), s1);
  }
  double acc = hsum(_mm256_add_pd(s0, s1));
  for (; i < n; ++i) acc += a[i] * b[i];
  return acc;
}

// y[i] += alpha * x[i]
void axpy(double alpha, const double* x, double* y, int n) {
  const __m256d a = _mm256_set1_pd(alpha);
  int i = 0;
  for (; i + 4 <= n; i += 4)
    _mm256_storeu_pd(y + i, _mm256_fmadd_pd(a, _mm256_loadu_pd(x + i), _mm256_loadu_pd(y + i)));
  for (; i < n; ++i) y[i] += alpha * x[i];
}

// y[i] += a * x[i] + b * z[i]
void axpy2(double a, const double* x, double b, const double* z, double* y, int n) {
  const __m256d va = _mm256_set1_pd(a), vb = _mm256_set1_pd(b);
  int i = 0;
  for (; i + 4 <= n; i += 4) {
    __m256d t = _mm256_fmadd_pd(va, _mm256_loadu_pd(x + i), _mm256_loadu_pd(y + i));
    _mm256_storeu_pd(y + i, _mm256_fmadd_pd(vb, _mm256_loadu_pd(z + i), t));
  }
  for (; i < n; ++i) y[i] += a * x[i] + b * z[i];
}

// One row of a symmetric product over a stored triangle: returns
// sum_{j<n} a[j] * v[j] and adds vi * a[j] to p[j] (j < n), in one pass.
double dot_axpy(const double* a, const double* v, double vi, double* p, int n) {
  const __m256d b = _mm256_set1_pd(vi);
  __m256d s0 = _mm256_setzero_pd(), s1 = _mm256_setzero_pd();
  int j = 0;
  for (; j + 8 <= n; j += 8) {
    const __m256d a0 = _mm256_loadu_pd(a + j), a1 = _mm256_loadu_pd(a + j + 4);
    s0 = _mm256_fmadd_pd(a0, _mm256_loadu_pd(v + j), s0);
    s1 = _mm256_fmadd_pd(a1, _mm256_loadu_pd(v + j + 4), s1);
    _mm256_storeu_pd(p + j, _mm256_fmadd_pd(b, a0, _mm256_loadu_pd(p + j)));
    _mm256_storeu_pd(p + j + 4, _mm256_fmadd_pd(b, a1, _mm256_loadu_pd(p + j + 4)));
  }
  double acc = hsum(_mm256_add_pd(s0, s1));
  for (; j < n; ++j) {
    acc += a[j] * v[j];
    p[j] += vi * a[j];
  }
  return acc;
}

// sqrt(a^2 + b^2); the plain formula where it cannot over- or underflow.
inline double hypot2(double a, double b) {
  const double m = std::max(std::fabs(a), std::fabs(b));
  if (m > 1e-150 && m < 1e150) return std::sqrt(a * a + b * b);
  return std::hypot(a, b);
}

// C[i][j] += sum_{k in [kb(i0,j0), ke(i0,j0))} A(i, k) * B[k][j] for one 4 x 8
// block (i0.., j0..) of row-major n x n matrices; A(i, k) = A[i*sai + k*sak]
// so that a transposed operand needs no copy.
inline void block4x8(int n, const double* A, long sai, long sak, const double* B, double* C,
                     int i0, int j0, int kb, int ke) {
  __m256d c[4][2];
  for (int a = 0; a < 4; ++a) c[a][0] = c[a][1] = _mm256_setzero_pd();
  for (int k = kb; k < ke; ++k) {
    const __m256d b0 = _mm256_loadu_pd(B + (size_t)k * n + j0);
    const __m256d b1 = _mm256_loadu_pd(B + (size_t)k * n + j0 + 4);
    for (int a = 0; a < 4; ++a) {
      const __m256d x = _mm256_broadcast_sd(A + (i0 + a) * sai + k * sak);
      c[a][0] = _mm256_fmadd_pd(x, b0, c[a][0]);
      c[a][1] = _mm256_fmadd_pd(x, b1, c[a][1]);
    }
  }
  for (int a = 0; a < 4; ++a) {
    double* ci = C + (size_t)(i0 + a) * n + j0;
    _mm256_storeu_pd(ci, _mm256_add_pd(_mm256_loadu_pd(ci), c[a][0]));
    _mm256_storeu_pd(ci + 4, _mm256_add_pd(_mm256_loadu_pd(ci + 4), c[a][1]));
  }
}

// C0[a*ldc + j0 ..+7] += sum_{k in [kb, ke)} A0[a*sai + k*sak] * B[k*ldb + j0 ..+7]
// for a < 4: one 4 x 8 block of a product whose operands have their own row
// strides (A0 and C0 point at the block's first row).
inline void block4x8s(const double* A0, long sai, long sak, const double* B, long ldb,
                      double* C0, long ldc, int j0, int kb, int ke) {
  __m256d c[4][2];
  for (int a = 0; a < 4; ++a) c[a][0] = c[a][1] = _mm256_setzero_pd();
  for (int k = kb; k < ke; ++k) {
    const __m256d b0 = _mm256_loadu_pd(B + (size_t)k * ldb + j0);
    const __m256d b1 = _mm256_loadu_pd(B + (size_t)k * ldb + j0 + 4);
    for (int a = 0; a < 4; ++a) {
      const __m256d x = _mm256_broadcast_sd(A0 + a * sai + k * sak);
      c[a][0] = _mm256_fmadd_pd(x, b0, c[a][0]);
      c[a][1] = _mm256_fmadd_pd(x, b1, c[a][1]);
    }
  }
  for (int a = 0; a < 4; ++a) {
    double* ci = C0 + (size_t)a * ldc + j0;
    _mm256_storeu_pd(ci, _mm256_add_pd(_mm256_loadu_pd(ci), c[a][0]));
    _mm256_storeu_pd(ci + 4, _mm256_add_pd(_mm256_loadu_pd(ci + 4), c[a][1]));
  }
}

// P = L V (d x r, row-major) for lower-triangular L (d x d, upper part zero).
void lower_times(int d, int r, const double* L, const double* V, double* P) {
  std::fill(P, P + (size_t)d * r, 0.0);
  if (d % 4 == 0 && r % 8 == 0) {
    for (int i0 = 0; i0 < d; i0 += 4)
      for (int j0 = 0; j0 < r; j0 += 8)
        block4x8s(L + (size_t)i0 * d, d, 1, V, r, P + (size_t)i0 * r, r, j0, 0, i0 + 4);
    return;
  }
  for (int i = 0; i < d; ++i)
    for (int j = 0; j <= i; ++j) axpy(L[(size_t)i * d + j], V + (size_t)j * r, P + (size_t)i * r, r);
}

// X = L^-T V (d x r, row-major): solves L^T X = V for lower-triangular L.
// Rows are solved from the last, four at a time: the sum over the rows already
// solved runs through the 4 x 8 block kernel, then the 4 x 4 diagonal block.
void lower_t_solve(int d, int r, const double* L, const double* V, double* X) {
  if (d % 4 == 0 && r % 8 == 0) {
    std::vector<double> T((size_t)4 * r);
    for (int i0 = d - 4; i0 >= 0; i0 -= 4) {
      std::fill(T.begin(), T.end(), 0.0);
      // T[a] = sum_{j >= i0+4} L[j][i0+a] X[j]
      for (int j0 = 0; j0 < r; j0 += 8)
        block4x8s(L + i0, 1, d, X, r, T.data(), r, j0, i0 + 4, d);
      for (int a = 3; a >= 0; --a) {
        const int i = i0 + a;
        const double rl = 1.0 / L[(size_t)i * d + i];
        double* xi = X + (size_t)i * r;
        for (int m = 0; m < r; ++m) {
          double v = V[(size_t)i * r + m] - T[(size_t)a * r + m];
          for (int b = a + 1; b < 4; ++b) v -= L[(size_t)(i0 + b) * d + i] * X[(size_t)(i0 + b) * r + m];
          xi[m] = v * rl;
        }
      }
    }
    return;
  }
  std::vector<double> W(V, V + (size_t)d * r);
  for (int i = d - 1; i >= 0; --i) {  // row i of L at a time
    double* xi = X + (size_t)i * r;
    const double rl = 1.0 / L[(size_t)i * d + i];
    for (int m = 0; m < r; ++m) xi[m] = W[(size_t)i * r + m] * rl;
    for (int j = 0; j < i; ++j) axpy(-L[(size_t)i * d + j], xi, W.data() + (size_t)j * r, r);
  }
}

// C = A * B for n x n row-major matrices (i-k-j order, contiguous inner loop).
void matmul(int n, const double* A, const double* B, double* C) {
  std::fill(C, C + (size_t)n * n, 0.0);
  if (n % 8 == 0) {
    for (int i0 = 0; i0 < n; i0 += 4)
      for (int j0 = 0; j0 < n; j0 += 8) block4x8(n, A, n, 1, B, C, i0, j0, 0, n);
    return;
  }
  for (int i = 0; i < n; ++i) {
    double* ci = C + (size_t)i * n;
    for (int k = 0; k < n; ++k) axpy(A[(size_t)i * n + k], B + (size_t)k * n, ci, n);
  }
}

// M = L^T S L for lower-triangular L and symmetric S (n x n row-major).
// W = S L skips the zero upper part of L (column block j0 needs k >= j0);
// M = L^T W needs k >= i for row i, and only blocks on or below the diagonal
// are formed before mirroring.
void congruence_lower(int n, const double* S, const double* L, double* M) {
  double* W = thread_buffer(4, (size_t)n * n);
  std::fill(W, W + (size_t)n * n, 0.0);
  std::fill(M, M + (size_t)n * n, 0.0);
  if (n % 8 == 0) {
    for (int i0 = 0; i0 < n; i0 += 4)
      for (int j0 = 0; j0 < n; j0 += 8) block4x8(n, S, n, 1, L, W, i0, j0, j0, n);
    for (int i0 = 0; i0 < n; i0 += 4)
      for (int j0 = 0; j0 < i0 + 4; j0 += 8) block4x8(n, L, 1, n, W, M, i0, j0, i0, n);
  } else {
    for (int i = 0; i < n; ++i)
      for (int k = 0; k < n; ++k) axpy(S[(size_t)i * n + k], L + (size_t)k * n, W + (size_t)i * n, k + 1);
    for (int k = 0; k < n; ++k)
      for (int i = 0; i <= k; ++i) axpy(L[(size_t)k * n + i], W + (size_t)k * n, M + (size_t)i * n, n);
  }
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < i; ++j) M[(size_t)j * n + i] = M[(size_t)i * n + j];
}

// S = (1/T) sum_t (x_t - mu)(x_t - mu)^T for the T rows of X (float, T x d);
// mu may be null (uncentred).  Tokens are converted to float64 in blocks and
// the lower triangle is accumulated in 4 x 8 register blocks.
void moment(int T, int d, const float* X, const double* mu, double* S) {
  std::fill(S, S + (size_t)d * d, 0.0);
  constexpr int TB = 128;
  std::vector<double> x((size_t)TB * d);
  for (int t0 = 0; t0 < T; t0 += TB) {
    const int nb = std::min(TB, T - t0);
    for (int b = 0; b < nb; ++b)
      for (int i = 0; i < d; ++i)
        x[(size_t)b * d + i] = (double)X[(size_t)(t0 + b) * d + i] - (mu ? mu[i] : 0.0);
    if (d % 8 == 0) {
      // the transposed token block: A(i, t) = x[t][i]
      for (int i0 = 0; i0 < d; i0 += 4)
        for (int j0 = 0; j0 < i0 + 4; j0 += 8) block4x8(d, x.data(), 1, d, x.data(), S, i0, j0, 0, nb);
    } else {
      for (int b = 0; b < nb; ++b) {
        const double* xb = x.data() + (size_t)b * d;
        for (int i = 0; i < d; ++i) axpy(xb[i], xb, S + (size_t)i * d, i + 1);
      }
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
    const double dsum = S[(size_t)j * n + j] - shift - dot(lj, lj, j);
    if (!(dsum > 0.0) || !std::isfinite(dsum)) return false;
    const double piv = std::sqrt(dsum);
    L[(size_t)j * n + j] = piv;
    for (int i = j + 1; i < n; ++i) {
      const double* li = L + (size_t)i * n;
      L[(size_t)i * n + j] = (S[(size_t)i * n + j] - dot(li, lj, j)) / piv;
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
// (sufficient test: S - floor_rel ||S||_F I is positive definite and
// ||S||_F >= lambda_max).  With want_factor, L then holds the Cholesky factor
// of S itself; otherwise L is scratch.
bool unclamped_cholesky(int n, const double* S, double floor_rel, double* L, bool want_factor) {
  const double f = frobenius(n, S);
  if (!(f > 0.0) || !std::isfinite(f)) return false;
  if (!cholesky(n, S, floor_rel * f, L)) return false;
  return !want_factor || cholesky(n, S, 0.0, L);
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

// Orthonormalise the r vectors stored as the rows of A (r x d) in place, in
// row order, by modified Gram-Schmidt with each vector orthogonalised twice
// against the earlier ones; then sign each vector so that its
// largest-magnitude entry is positive (lowest index on ties).  Returns false
// when a vector is numerically in the span of the earlier ones.
bool orthonormal_rows(int d, int r, double* A) {
  for (int m = 0; m < r; ++m) {
    double* a = A + (size_t)m * d;
    const double n0 = std::sqrt(dot(a, a, d));
    for (int pass = 0; pass < 2; ++pass)
      for (int p = 0; p < m; ++p) {
        const double* b = A + (size_t)p * d;
        axpy(-dot(b, a, d), b, a, d);
      }
    const double nrm = std::sqrt(dot(a, a, d));
    if (!(nrm > 1e-12 * n0) || !std::isfinite(nrm)) return false;
    for (int i = 0; i < d; ++i) a[i] /= nrm;
    int jmax = 0;
    for (int i = 1; i < d; ++i)
      if (std::fabs(a[i]) > std::fabs(a[jmax])) jmax = i;
    if (a[jmax] < 0)
      for (int i = 0; i < d; ++i) a[i] = -a[i];
  }
  return true;
}

// B_q = B_k = Q (d x r, row-major float) from the r basis vectors (rows of Qr).
void store_basis(int d, int r, const double* Qr, float* Bq, float* Bk) {
  for (int m = 0; m < r; ++m)
    for (int i = 0; i < d; ++i)
      Bq[(size_t)i * r + m] = Bk[(size_t)i * r + m] = (float)Qr[(size_t)m * d + i];
}

// The Householder reflector of x (m entries, contiguous) into v: H = I -
// beta v v^T maps x to alpha e_0.  Returns beta (0, with v = 0 and alpha = 0,
// for x = 0).
double householder_vec(const double* x, int m, double* v, double* alpha_out) {
  std::copy(x, x + m, v);
  const double sumsq = dot(v, v, m);
  const double x0 = v[0];
  double alpha = std::sqrt(sumsq);
  *alpha_out = 0.0;
  if (alpha == 0.0) { std::fill(v, v + m, 0.0); return 0.0; }
  if (x0 > 0) alpha = -alpha;  // reflect away from x0's sign
  v[0] = x0 - alpha;
  const double vv = sumsq - x0 * x0 + v[0] * v[0];
  if (vv == 0.0) { std::fill(v, v + m, 0.0); return 0.0; }
  *alpha_out = alpha;
  return 2.0 / vv;
}

// One row of the trailing block in the fused pass, from its diagonal (len
// entries r[t] = a(i, i+t)): r -= vi*w + wi*v (v, w from index i), then the
// row's part of the next product pn = A v_next over the upper triangle (vn,
// pn from the row's index in the next block): pn[0] gets the row times vn,
// pn[t] (t >= 1) gets vn[0] * r[t].
void update_row_and_product(double* r, const double* v, const double* w, double vi, double wi,
                            const double* vn, double* pn, int len) {
  const double vni = vn[0];
  const double x0 = std::fma(-wi, v[0], std::fma(-vi, w[0], r[0]));
  r[0] = x0;
  double acc = x0 * vni;
  const __m256d nvi = _mm256_set1_pd(-vi), nwi = _mm256_set1_pd(-wi), bn = _mm256_set1_pd(vni);
  __m256d s0 = _mm256_setzero_pd();
  int t = 1;
  for (; t + 4 <= len; t += 4) {
    const __m256d x = _mm256_fmadd_pd(nwi, _mm256_loadu_pd(v + t),
                                      _mm256_fmadd_pd(nvi, _mm256_loadu_pd(w + t), _mm256_loadu_pd(r + t)));
    _mm256_storeu_pd(r + t, x);
    s0 = _mm256_fmadd_pd(x, _mm256_loadu_pd(vn + t), s0);
    _mm256_storeu_pd(pn + t, _mm256_fmadd_pd(bn, x, _mm256_loadu_pd(pn + t)));
  }
  acc += hsum(s0);
  for (; t < len; ++t) {
    const double x = std::fma(-wi, v[t], std::fma(-vi, w[t], r[t]));
    r[t] = x;
    acc += x * vn[t];
    pn[t] += vni * x;
  }
  pn[0] += acc;
}

// Householder reduction of symmetric `a` (n x n, upper triangle read and
// overwritten; the lower triangle is ignored) to tridiagonal
// form T = Q^T A Q, Q = H_0 H_1 ... H_{n-3} with H_k = I - beta_k v_k v_k^T
// acting on indices k+1 .. n-1 (Golub & Van Loan, Sec. 8.3.1).  diag/off
// receive T's diagonal and sub-diagonal (off[n-1] = 0); row k of `hv` holds
// v_k in its entries k+1 .. n-1 and beta[k] its factor (0 when H_k = I).
// The upper triangle keeps every column below the diagonal contiguous (as
// the row right of it).  Each step's rank-2 update of the trailing block runs
// in one pass with the next step's product A v_next: the block's first row is
// updated first, the next reflector is formed from it, then every row is
// updated and multiplied while it is at hand.
void householder_tridiag(int n, double* a, double* diag, double* off, double* hv, double* beta) {
  std::fill(hv, hv + (size_t)n * n, 0.0);
  std::fill(beta, beta + n, 0.0);
  std::vector<double> p(n), w(n), pn(n);
  auto row = [&](int i) { return a + (size_t)i * n + i; };  // row i from its diagonal
  double alpha = 0.0;
  if (n >= 3) beta[0] = householder_vec(row(0) + 1, n - 1, hv + 1, &alpha);
  bool p_ready = false;  // p holds A22 v_k, accumulated in the previous step's pass
  for (int k = 0; k + 2 < n; ++k) {
    const int m = n - k - 1;  // order of the trailing block A22 (rows/cols k+1..)
    const double* v = hv + (size_t)k * n + (k + 1);
    const double bk = beta[k];
    const double alpha_k = alpha;
    if (bk != 0.0) {
      if (!p_ready) {  // p = A22 v over the upper triangle
        std::fill(p.begin(), p.begin() + m, 0.0);
        for (int i = 0; i < m; ++i) {
          const double* r = row(k + 1 + i);
          p[i] += r[0] * v[i] + dot_axpy(r + 1, v + i + 1, v[i], p.data() + i + 1, m - i - 1);
        }
      }
      // p = beta A22 v,  K = beta/2 v.p,  w = p - K v
      for (int i = 0; i < m; ++i) p[i] *= bk;
      const double K = 0.5 * bk * dot(v, p.data(), m);
      for (int i = 0; i < m; ++i) w[i] = p[i] - K * v[i];
      double* r0 = row(k + 1);  // the block's first row
      for (int t = 0; t < m; ++t) r0[t] = std::fma(-w[0], v[t], std::fma(-v[0], w[t], r0[t]));
    }
    p_ready = false;
    const bool next = k + 3 < n;
    double* vn = next ? hv + (size_t)(k + 1) * n + (k + 2) : nullptr;
    if (next) beta[k + 1] = householder_vec(row(k + 1) + 1, m - 1, vn, &alpha);
    const bool fuse = next && beta[k + 1] != 0.0;
    if (fuse) std::fill(pn.begin(), pn.begin() + (m - 1), 0.0);
    if (bk != 0.0 || fuse) {
      for (int i = 1; i < m; ++i) {
        double* r = row(k + 1 + i);  // entries j = i .. m-1 of the block's row i
        const int ii = i - 1;        // its row in the next block
        if (bk != 0.0 && fuse) {
          update_row_and_product(r, v + i, w.data() + i, v[i], w[i], vn + ii, pn.data() + ii, m - i);
        } else if (bk != 0.0) {
          axpy2(-v[i], w.data() + i, -w[i], v + i, r, m - i);
        } else {
          pn[ii] += r[0] * vn[ii] + dot_axpy(r + 1, vn + ii + 1, vn[ii], pn.data() + ii + 1, m - i - 1);
        }
      }
      if (fuse) {
        std::swap(p, pn);
        p_ready = true;
      }
    }
    // column k below its diagonal (row k right of it) is now alpha e_0
    double* rk = row(k) + 1;
    for (int t = 0; t < m; ++t) rk[t] = t == 0 ? alpha_k : 0.0;
  }
  for (int i = 0; i < n; ++i) diag[i] = a[(size_t)i * n + i];
  for (int i = 0; i + 1 < n; ++i) off[i] = a[(size_t)i * n + i + 1];
  off[n - 1] = 0.0;
}

// X <- Q X for the Q of householder_tridiag; X is n x c row-major (c
// vectors side by side), so each reflector is two passes of row axpys.
void apply_q(int n, const double* hv, const double* beta, double* X, int c) {
  std::vector<double> t(c);
  for (int k = n - 3; k >= 0; --k) {
    if (beta[k] == 0.0) continue;
    const double* v = hv + (size_t)k * n + (k + 1);
    const int m = n - k - 1;
    double* xk = X + (size_t)(k + 1) * c;
    std::fill(t.begin(), t.end(), 0.0);
    for (int i = 0; i < m; ++i) axpy(v[i], xk + (size_t)i * c, t.data(), c);  // t = v^T X
    for (int i = 0; i < m; ++i) axpy(-beta[k] * v[i], t.data(), xk + (size_t)i * c, c);
  }
}

// zt <- Q^T = H_{n-3} ... H_0 (row-major n x n), the starting point of the
// eigenvector accumulation of the QR steps.
void form_qt(int n, const double* hv, const double* beta, double* zt) {
  std::fill(zt, zt + (size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) zt[(size_t)i * n + i] = 1.0;
  std::vector<double> w(n);
  for (int k = 0; k + 2 < n; ++k) {
    if (beta[k] == 0.0) continue;
    const double* v = hv + (size_t)k * n + (k + 1);
    const int m = n - k - 1;
    // rows k+1.. of zt: row_i -= beta v_i (sum_l v_l row_l)
    std::fill(w.begin(), w.end(), 0.0);
    for (int l = 0; l < m; ++l) axpy(v[l], zt + (size_t)(k + 1 + l) * n, w.data(), n);
    for (int i = 0; i < m; ++i) axpy(-beta[k] * v[i], w.data(), zt + (size_t)(k + 1 + i) * n, n);
  }
}

// One implicit symmetric QR step with the Wilkinson shift on the unreduced
// block [l, m] of the tridiagonal (a: diagonal, b[i]: the entry coupling i and
// i + 1), after Golub & Van Loan, "Matrix Computations", Algorithm 8.3.2.  The
// shift mu is the eigenvalue of the block's trailing 2 x 2 nearer a[m]; the
// first rotation acts on (a[l] - mu, b[l]) and each later one, on rows and
// columns (k, k + 1), removes the bulge the previous one left at (k + 1, k - 1).
// With rows (k, k+1) mixed as (c, s; -s, c) and the columns alike, the 2 x 2
// block (p, r; r, q) becomes
//   p' = c^2 p + 2cs r + s^2 q,  q' = s^2 p - 2cs r + c^2 q,
//   r' = cs (q - p) + (c^2 - s^2) r,
// and the next coupling b[k+1] splits into c b[k+1] and the new bulge s b[k+1].
// zt (rows = columns of the accumulated orthogonal matrix) takes the same
// rotations when not null.
void qr_step(int n, int l, int m, double* a, double* b, double* zt) {
  const double d = 0.5 * (a[m - 1] - a[m]);
  const double e = b[m - 1];
  const double den = d + std::copysign(hypot2(d, e), d);
  const double mu = den != 0.0 ? a[m] - e * e / den : a[m];
  double x = a[l] - mu, z = b[l];
  for (int k = l; k < m; ++k) {
    const double rad = hypot2(x, z);
    const double c = rad > 0.0 ? x / rad : 1.0, s = rad > 0.0 ? z / rad : 0.0;
    if (k > l) b[k - 1] = rad;
    const double p = a[k], q = a[k + 1], r = b[k];
    const double cc = c * c, ss = s * s, cs = c * s;
    a[k] = cc * p + 2.0 * cs * r + ss * q;
    a[k + 1] = ss * p - 2.0 * cs * r + cc * q;
    b[k] = cs * (q - p) + (cc - ss) * r;
    if (k + 1 < m) {
      z = s * b[k + 1];
      b[k + 1] *= c;
      x = b[k];
    }
    if (zt) {
      double* zk = zt + (size_t)k * n;
      double* zk1 = zt + (size_t)(k + 1) * n;
      for (int i = 0; i < n; ++i) {
        const double u = zk[i], v = zk1[i];
        zk[i] = c * u + s * v;
        zk1[i] = c * v - s * u;
      }
    }
  }
}

// Eigenvalues (left in a) and, with zt, eigenvectors of the symmetric
// tridiagonal (a, b) by implicit QR steps (Golub & Van Loan, Algorithm 8.3.3):
// couplings that have become negligible are set to zero, and a step is
// applied to the unreduced block that ends at the lowest row not yet split
// off.  A coupling is negligible relative to its two diagonal entries, or
// absolutely at eps * ||T|| (which moves any eigenvalue by at most that
// much; the absolute test ends the iteration on blocks of (near-)zero
// eigenvalues, where a purely relative one never does).  Returns false
// without convergence.
bool tridiag_qr(int n, double* a, double* b, double* zt) {
  const double eps = std::numeric_limits<double>::epsilon();
  double tnorm = 0.0;
  for (int i = 0; i < n; ++i)
    tnorm = std::max(tnorm, std::fabs(a[i]) + (i + 1 < n ? std::fabs(b[i]) : 0.0));
  const double abs_tol = eps * tnorm;
  auto negligible = [&](int i) {  // b[i], between rows i and i + 1
    return std::fabs(b[i]) <= std::max(eps * (std::fabs(a[i]) + std::fabs(a[i + 1])), abs_tol);
  };
  long long steps = 0;
  for (int m = n - 1; m > 0;) {
    if (negligible(m - 1)) {
      b[m - 1] = 0.0;
      --m;
      continue;
    }
    int l = m - 1;
    while (l > 0 && !negligible(l - 1)) --l;
    if (++steps > 80LL * n) return false;
    qr_step(n, l, m, a, b, zt);
  }
  if (n > 0) b[n - 1] = 0.0;
  return true;
}

// Eigen-decomposition of symmetric A (n x n row-major).  w ascending; vt row j
// = eigenvector j.  Returns false on non-convergence or non-finite input.
bool sym_eig_rows(int n, const double* A, double* w, double* vt) {
  if (!all_finite(A, (size_t)n * n)) return false;
  Mat a(A, A + (size_t)n * n), q((size_t)n * n), zt((size_t)n * n);
  // symmetrise exactly
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < i; ++j) {
      const double s = 0.5 * (a[(size_t)i * n + j] + a[(size_t)j * n + i]);
      a[(size_t)i * n + j] = a[(size_t)j * n + i] = s;
    }
  std::vector<double> diag(n), off(n), beta(n);
  householder_tridiag(n, a.data(), diag.data(), off.data(), q.data(), beta.data());
  form_qt(n, q.data(), beta.data(), zt.data());
  if (!tridiag_qr(n, diag.data(), off.data(), zt.data())) return false;
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

// LU factorisation with partial pivoting of T - lambda_l I for four shifts
// at once, one per AVX2 lane, for the symmetric tridiagonal T (diag, off).
// Each lane takes the steps of the one-shift factorisation, its row exchange
// chosen by a blend; pivots smaller than `tiny` are replaced by +-tiny, as
// inverse iteration requires, and stored as reciprocals.
struct ShiftedTridiagLU4 {
  // row i of each array: its four lanes at [4i, 4i + 4)
  std::vector<double> rdg, du, du2, dl, sw;
  explicit ShiftedTridiagLU4(int n) : rdg(4 * n), du(4 * n), du2(4 * n), dl(4 * n), sw(4 * n) {}
  static __m256d ld(const std::vector<double>& v, int i) { return _mm256_loadu_pd(v.data() + 4 * i); }
  static void st(std::vector<double>& v, int i, __m256d x) { _mm256_storeu_pd(v.data() + 4 * i, x); }

  void factor(int n, const double* diag, const double* off, const double* lambda, double tiny) {
    const __m256d lam = _mm256_loadu_pd(lambda), vtiny = _mm256_set1_pd(tiny);
    const __m256d absmask = _mm256_castsi256_pd(_mm256_set1_epi64x(0x7fffffffffffffffll));
    const __m256d zero = _mm256_setzero_pd();
    std::vector<double>& dg = rdg;
    for (int i = 0; i < n; ++i) st(dg, i, _mm256_sub_pd(_mm256_set1_pd(diag[i]), lam));
    for (int i = 0; i + 1 < n; ++i) st(du, i, _mm256_set1_pd(off[i]));
    st(du, n - 1, zero);
    st(du2, n - 1, zero);
    st(dl, n - 1, zero);
    st(sw, n - 1, zero);
    for (int i = 0; i + 1 < n; ++i) {
      const __m256d a = ld(dg, i), o = _mm256_set1_pd(off[i]), d1 = ld(dg, i + 1), t = ld(du, i);
      // exchange rows i and i+1 where |dg_i| < |off_i|
      const __m256d s = _mm256_cmp_pd(_mm256_and_pd(a, absmask), _mm256_and_pd(o, absmask), _CMP_LT_OQ);
      const __m256d piv = _mm256_blendv_pd(a, vtiny, _mm256_cmp_pd(a, zero, _CMP_EQ_OQ));
      const __m256d f = _mm256_div_pd(_mm256_blendv_pd(o, a, s), _mm256_blendv_pd(piv, o, s));
      st(dl, i, f);
      st(dg, i, _mm256_blendv_pd(a, o, s));
      st(du, i, _mm256_blendv_pd(t, d1, s));
      st(dg, i + 1, _mm256_blendv_pd(_mm256_fnmadd_pd(f, t, d1), _mm256_fnmadd_pd(f, d1, t), s));
      if (i + 2 < n) {
        const __m256d u1 = ld(du, i + 1);
        st(du2, i, _mm256_and_pd(s, u1));
        st(du, i + 1, _mm256_blendv_pd(u1, _mm256_sub_pd(zero, _mm256_mul_pd(f, u1)), s));
      } else {
        st(du2, i, zero);
      }
      st(sw, i, s);
    }
    const __m256d one = _mm256_set1_pd(1.0);
    for (int i = 0; i < n; ++i) {
      const __m256d x = ld(dg, i);
      const __m256d small = _mm256_cmp_pd(_mm256_and_pd(x, absmask), vtiny, _CMP_LT_OQ);
      const __m256d tt = _mm256_blendv_pd(vtiny, _mm256_sub_pd(zero, vtiny), _mm256_cmp_pd(x, zero, _CMP_LT_OQ));
      st(dg, i, _mm256_div_pd(one, _mm256_blendv_pd(x, tt, small)));
    }
  }

  // b <- (T - lambda_l I)^{-1} b in each lane (b[4i + l]: lane l's element i)
  void solve(int n, double* b) const {
    auto bl = [&](int i) { return _mm256_loadu_pd(b + 4 * i); };
    auto bs = [&](int i, __m256d x) { _mm256_storeu_pd(b + 4 * i, x); };
    for (int i = 0; i + 1 < n; ++i) {  // L y = P b
      const __m256d bi = bl(i), bi1 = bl(i + 1), s = ld(sw, i), l = ld(dl, i);
      bs(i, _mm256_blendv_pd(bi, bi1, s));
      bs(i + 1, _mm256_blendv_pd(_mm256_fnmadd_pd(l, bi, bi1), _mm256_fnmadd_pd(l, bi1, bi), s));
    }
    bs(n - 1, _mm256_mul_pd(bl(n - 1), ld(rdg, n - 1)));  // U x = y
    if (n > 1) bs(n - 2, _mm256_mul_pd(_mm256_fnmadd_pd(ld(du, n - 2), bl(n - 1), bl(n - 2)), ld(rdg, n - 2)));
    for (int i = n - 3; i >= 0; --i)
      bs(i, _mm256_mul_pd(_mm256_fnmadd_pd(ld(du2, i), bl(i + 2), _mm256_fnmadd_pd(ld(du, i), bl(i + 1), bl(i))),
                          ld(rdg, i)));
  }
};

// Sturm counts of the symmetric tridiagonal (diag, off2 = off^2): cnt[e] =
// the number of eigenvalues below x[e] for the kBisectShifts points, in
// independent 4-wide sequences so that their divisions overlap (Golub & Van
// Loan, Sec. 8.4.1).  A pivot smaller in magnitude than pivmin is replaced by
// -pivmin.
constexpr int kBisectShifts = 16;
void sturm_counts(int n, const double* diag, const double* off2, double pivmin, const double* x,
                  int* cnt_out) {
  constexpr int V = kBisectShifts / 4;
  const __m256d one = _mm256_set1_pd(1.0), zero = _mm256_setzero_pd();
  const __m256d npm = _mm256_set1_pd(-pivmin), pm = _mm256_set1_pd(pivmin);
  const __m256d absmask = _mm256_castsi256_pd(_mm256_set1_epi64x(0x7fffffffffffffffll));
  __m256d xv[V], q[V], cnt[V];
  const __m256d d0 = _mm256_set1_pd(diag[0]);
  for (int v = 0; v < V; ++v) {
    xv[v] = _mm256_loadu_pd(x + 4 * v);
    q[v] = _mm256_sub_pd(d0, xv[v]);
    q[v] = _mm256_blendv_pd(q[v], npm, _mm256_cmp_pd(_mm256_and_pd(q[v], absmask), pm, _CMP_LT_OQ));
    cnt[v] = _mm256_and_pd(_mm256_cmp_pd(q[v], zero, _CMP_LT_OQ), one);
  }
  for (int i = 1; i < n; ++i) {
    const __m256d di = _mm256_set1_pd(diag[i]), ei = _mm256_set1_pd(off2[i - 1]);
    for (int v = 0; v < V; ++v) {
      q[v] = _mm256_sub_pd(_mm256_sub_pd(di, xv[v]), _mm256_div_pd(ei, q[v]));
      q[v] = _mm256_blendv_pd(q[v], npm, _mm256_cmp_pd(_mm256_and_pd(q[v], absmask), pm, _CMP_LT_OQ));
      cnt[v] = _mm256_add_pd(cnt[v], _mm256_and_pd(_mm256_cmp_pd(q[v], zero, _CMP_LT_OQ), one));
    }
  }
  alignas(32) double c[kBisectShifts];
  for (int v = 0; v < V; ++v) _mm256_store_pd(c + 4 * v, cnt[v]);
  for (int e = 0; e < kBisectShifts; ++e) cnt_out[e] = (int)c[e];
}

// The eigenvalues with ascending indices i_lo .. n-1 (the n - i_lo largest)
// of the symmetric tridiagonal (diag, off2), by multisection on Sturm counts
// over [glo, ghi) (count(glo) = 0, count(ghi) = n).  A bracket [a, b) with
// counts ca = count(a), cb = count(b) holds eigenvalues ca .. cb-1.  Each
// round spends the kBisectShifts evaluation points on the open brackets that
// hold wanted eigenvalues: several points per bracket, equally spaced, while
// fewer brackets are open, one (the midpoint) once there are more.  A bracket
// no wider than tol closes, and its eigenvalues take its midpoint.  out[i -
// i_lo] receives eigenvalue i.
void multisect_eigs(int n, const double* diag, const double* off2, double pivmin, double glo,
                    double ghi, double tol, int i_lo, double* out) {
  struct Bracket {
    double a, b;
    int ca, cb;
  };
  std::vector<Bracket> open{{glo, ghi, 0, n}}, act;
  while (!open.empty()) {
    act.clear();
    for (const Bracket& B : open) {
      const int t0 = std::max(B.ca, i_lo), t1 = B.cb;  // wanted eigenvalues in the bracket
      if (t0 >= t1) continue;
      if (B.b - B.a <= tol) {
        for (int i = t0; i < t1; ++i) out[i - i_lo] = 0.5 * (B.a + B.b);
        continue;
      }
      act.push_back(B);
    }
    open.clear();
    for (size_t s = 0; s < act.size(); s += kBisectShifts) {
      const int m = (int)std::min<size_t>(kBisectShifts, act.size() - s);
      const int per = kBisectShifts / m;  // points per bracket this round
      alignas(32) double x[kBisectShifts];
      int cnt[kBisectShifts];
      int np = 0;
      for (int j = 0; j < m; ++j) {
        const Bracket& B = act[s + j];
        for (int u = 1; u <= per; ++u) x[np++] = B.a + (B.b - B.a) * ((double)u / (per + 1));
      }
      for (int e = np; e < kBisectShifts; ++e) x[e] = x[0];  // unused lanes
      sturm_counts(n, diag, off2, pivmin, x, cnt);
      for (int j = 0, e = 0; j < m; ++j) {
        const Bracket& B = act[s + j];
        double a = B.a;
        int ca = B.ca;
        bool stuck = false;
        for (int u = 0; u < per; ++u, ++e) {
          if (!(x[e] > a && x[e] < B.b)) stuck = true;  // no room left between doubles
          const int c = std::min(std::max(cnt[e], ca), B.cb);  // counts rise with x
          if (!stuck) {
            open.push_back({a, x[e], ca, c});
            a = x[e];
            ca = c;
          }
        }
        if (stuck) {  // close what is left at its midpoint
          for (int i = std::max(ca, i_lo); i < B.cb; ++i) out[i - i_lo] = 0.5 * (a + B.b);
        } else {
          open.push_back({a, B.b, ca, B.cb});
        }
      }
    }
  }
}

// Tridiagonal form of symmetric A (n x n row-major, read from its lower
// triangle) and its reflectors, as householder_tridiag returns them.
bool tridiag_of(int n, const double* A, double* diag, double* off, double* hv, double* beta) {
  if (!all_finite(A, (size_t)n * n)) return false;
  double* a = thread_buffer(2, (size_t)n * n);
  for (int i = 0; i < n; ++i)  // A's lower triangle, transposed into the upper one
    for (int j = i; j < n; ++j) a[(size_t)i * n + j] = A[(size_t)j * n + i];
  householder_tridiag(n, a, diag, off, hv, beta);
  return true;
}

// The r largest eigenpairs of the symmetric matrix whose tridiagonal form
// (diag, off) and reflectors (hv, beta) tridiag_of produced: w receives the
// r largest eigenvalues in descending order (all n with all_values), row m
// of `vecs` (r x n) the unit eigenvector of w[m].  Eigenvalues by QR steps without
// vectors (all_values) or by multisection on Sturm counts (only the r
// largest), then inverse iteration on the tridiagonal for the r vectors
// (Golub & Van Loan, Sec. 8.2.2 and 8.4), four shifts at a time,
// re-orthogonalised within clusters of close eigenvalues, and
// back-transformation by the reflectors.  With the reduction this costs
// 2n^3 + O(n^2 r) flops instead of the roughly 9n^3 of the full solver.
bool top_eigpairs(int n, const double* diag, const double* off, const double* hv,
                  const double* beta, int r, double* w, double* vecs, bool all_values) {
  std::vector<double> ev(n);
  if (all_values) {
    std::vector<double> eo(off, off + n);
    std::copy(diag, diag + n, ev.begin());
    if (!tridiag_qr(n, ev.data(), eo.data(), nullptr)) return false;
    std::sort(ev.begin(), ev.end(), [](double x, double y) { return x > y; });
  } else {  // only the r largest, by multisection
    std::vector<double> off2(n, 0.0);
    double glo = diag[0], ghi = diag[0], emax = 0.0;
    for (int i = 0; i < n; ++i) {
      const double rad = (i > 0 ? std::fabs(off[i - 1]) : 0.0) + (i + 1 < n ? std::fabs(off[i]) : 0.0);
      glo = std::min(glo, diag[i] - rad);
      ghi = std::max(ghi, diag[i] + rad);
      if (i + 1 < n) {
        off2[i] = off[i] * off[i];
        emax = std::max(emax, off2[i]);
      }
    }
    const double pivmin = std::numeric_limits<double>::min() * std::max(1.0, emax);
    const double pad = 2.0 * std::numeric_limits<double>::epsilon() * std::max(std::fabs(glo), std::fabs(ghi)) + pivmin;
    // narrow the Gershgorin interval down to 2^-46 of the spectrum's scale:
    // the factors are stored in float32, 2^-46 |T| is far below their rounding
    const double scale = std::max(std::fabs(glo), std::fabs(ghi));
    const double tol = std::ldexp(scale, -46);
    std::vector<double> asc(r);  // eigenvalues n-r .. n-1 in ascending index order
    multisect_eigs(n, diag, off2.data(), pivmin, glo - pad, ghi + pad, tol, n - r, asc.data());
    for (int m = 0; m < r; ++m) ev[m] = asc[r - 1 - m];  // descending
  }
  std::copy(ev.begin(), ev.begin() + (all_values ? n : r), w);

  const double eps = std::numeric_limits<double>::epsilon();
  double tnorm = 0.0;  // 1-norm of T
  for (int i = 0; i < n; ++i)
    tnorm = std::max(tnorm, std::fabs(diag[i]) + std::fabs(off[i]) + (i ? std::fabs(off[i - 1]) : 0.0));
  if (tnorm == 0.0) tnorm = 1.0;
  const double cluster_gap = 1e-3 * tnorm;  // re-orthogonalise closer eigenvalues
  const double tiny = eps * tnorm;
  const double converged = std::sqrt(0.1 / n);
  // shifts, clusters and start vectors of the r vectors, in order
  std::vector<double> shift(r), start((size_t)r * n);
  std::vector<int> cbeg(r);
  {
    int cluster_begin = 0;
    double shift_prev = 0.0;
    uint64_t seed = 0x9E3779B97F4A7C15ull;
    for (int m = 0; m < r; ++m) {
      double lambda = ev[m];
      if (m > 0) {
        if (shift_prev - lambda > cluster_gap) cluster_begin = m;
        // equal eigenvalues get distinct shifts so the iterations separate them
        const double sep = 10.0 * eps * std::max(std::fabs(shift_prev), tnorm * eps);
        if (lambda > shift_prev - sep) lambda = shift_prev - sep;
      }
      shift_prev = lambda;
      shift[m] = lambda;
      cbeg[m] = cluster_begin;
      for (int i = 0; i < n; ++i) {  // fixed pseudo-random start in [-1, 1)
        seed = seed * 6364136223846793005ull + 1442695040888963407ull;
        start[(size_t)m * n + i] = (double)(seed >> 11) * (2.0 / 9007199254740992.0) - 1.0;
      }
    }
  }
  // four vectors at a time, one per lane of the factorisation and solve; a
  // vector is re-orthogonalised after each solve against the finished
  // vectors of its cluster and against the earlier lanes of its group (block
  // Gram-Schmidt), and is kept once it has converged
  ShiftedTridiagLU4 lu(n);
  std::vector<double> xb((size_t)4 * n);
  std::vector<double> x4((size_t)4 * n);  // lane l's vector at x4[l * n ...]
  for (int m0 = 0; m0 < r; m0 += 4) {
    const int nl = std::min(4, r - m0);
    double lam[4];
    for (int l = 0; l < 4; ++l) lam[l] = l < nl ? shift[m0 + l] : shift[m0] + (l + 1) * tnorm;  // idle lanes: any shift
    lu.factor(n, diag, off, lam, tiny);
    for (int l = 0; l < 4; ++l)
      std::copy(start.begin() + (size_t)(m0 + std::min(l, nl - 1)) * n,
                start.begin() + (size_t)(m0 + std::min(l, nl - 1) + 1) * n, x4.begin() + (size_t)l * n);
    int extra[4] = {0, 0, 0, 0};
    bool done[4];
    for (int l = 0; l < 4; ++l) done[l] = l >= nl;
    auto finish = [&](int l) {
      const double* xl = x4.data() + (size_t)l * n;
      const double nrm = std::sqrt(dot(xl, xl, n));
      double* vm = vecs + (size_t)(m0 + l) * n;
      for (int i = 0; i < n; ++i) vm[i] = xl[i] / nrm;
    };
    for (int it = 0; it < 6; ++it) {
      if (done[0] && done[1] && done[2] && done[3]) break;
      for (int l = 0; l < 4; ++l) {  // start small: a converged solve then grows by about 1 / (eps n)
        double* xl = x4.data() + (size_t)l * n;
        double l1 = 0.0;
        for (int i = 0; i < n; ++i) l1 += std::fabs(xl[i]);
        const double sc = l1 > 0.0 ? n * tnorm * eps / l1 : 1.0;
        for (int i = 0; i < n; ++i) xl[i] *= sc;
      }
      for (int i = 0; i < n; ++i)
        for (int l = 0; l < 4; ++l) xb[(size_t)4 * i + l] = x4[(size_t)l * n + i];
      lu.solve(n, xb.data());
      for (int l = 0; l < 4; ++l)
        if (!done[l])
          for (int i = 0; i < n; ++i) x4[(size_t)l * n + i] = xb[(size_t)4 * i + l];
      for (int l = 0; l < nl; ++l) {
        if (done[l]) continue;
        double* xl = x4.data() + (size_t)l * n;
        const int m = m0 + l;
        for (int p = cbeg[m]; p < m; ++p) {
          if (p < m0 || done[p - m0]) {  // a finished unit vector, still in the tridiagonal basis
            const double* vp = vecs + (size_t)p * n;
            axpy(-dot(vp, xl, n), vp, xl, n);
          } else {  // an earlier lane of this group, not yet finished
            const double* xp = x4.data() + (size_t)(p - m0) * n;
            const double pp = dot(xp, xp, n);
            if (pp > 0.0) axpy(-dot(xp, xl, n) / pp, xp, xl, n);
          }
        }
        double amax = 0.0;
        for (int i = 0; i < n; ++i) amax = std::max(amax, std::fabs(xl[i]));
        if (!std::isfinite(amax) || amax == 0.0) return false;
        if (amax >= converged && ++extra[l] >= 2) {
          done[l] = true;
          finish(l);
        }
      }
    }
    for (int l = 0; l < nl; ++l)
      if (!done[l]) finish(l);
  }
  // back to the basis of A, all r vectors at once (n x r, then transposed)
  std::vector<double> X((size_t)n * r);
  for (int m = 0; m < r; ++m)
    for (int i = 0; i < n; ++i) X[(size_t)i * r + m] = vecs[(size_t)m * n + i];
  apply_q(n, hv, beta, X.data(), r);
  for (int m = 0; m < r; ++m)
    for (int i = 0; i < n; ++i) vecs[(size_t)m * n + i] = X[(size_t)i * r + m];
  return true;
}

// The r largest eigenpairs of symmetric A (n x n row-major, read from its
// lower triangle); w, vecs and all_values as for top_eigpairs.
bool sym_eig_top(int n, const double* A, int r, double* w, double* vecs, bool all_values) {
  double* hv = thread_buffer(3, (size_t)n * n);
  std::vector<double> diag(n), off(n), beta(n);
  return tridiag_of(n, A, diag.data(), off.data(), hv, beta.data()) &&
         top_eigpairs(n, diag.data(), off.data(), hv, beta.data(), r, w, vecs, all_values);
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

// Worker threads kept for the life of the process.  A calibration call runs
// two parallel phases over heads; starting threads for each phase would cost
// tens of microseconds per thread, a large share of a call that takes a few
// milliseconds.  Jobs are serialised: concurrent callers wait for the pool,
// and a job started from inside a worker (nesting) runs inline.  The workers
// are detached and the pool is never destroyed, so process exit does not
// wait for them; a child of fork() builds its own pool.
class WorkerPool {
 public:
  static WorkerPool& get() {
    static std::mutex m;
    static WorkerPool* pool = nullptr;
    std::lock_guard<std::mutex> lk(m);
    if (!pool || pool->pid_ != getpid()) pool = new WorkerPool();  // old one leaks after fork
    return *pool;
  }

  // fn(i) for i in [0, count) on nt threads (the caller is one of them).
  // Returns false if some fn(i) threw std::bad_alloc.
  template <class F>
  bool run(int count, int nt, F& fn) {
    if (t_in_worker) return run_inline(count, fn);
    std::lock_guard<std::mutex> job(job_mutex_);
    grow(nt - 1);
    std::atomic<int> next(0);
    std::atomic<bool> oom(false);
    Body body = [&]() {
      for (int i = next.fetch_add(1); i < count; i = next.fetch_add(1)) {
        try {
          fn(i);
        } catch (const std::bad_alloc&) {
          oom = true;
        }
      }
    };
    {
      std::lock_guard<std::mutex> lk(m_);
      body_ = &body;
      helpers_ = nt - 1;
      done_ = 0;
      ++generation_;
    }
    cv_start_.notify_all();
    t_in_worker = true;
    body();
    t_in_worker = false;
    std::unique_lock<std::mutex> lk(m_);
    cv_done_.wait(lk, [&] { return done_ == helpers_; });
    body_ = nullptr;
    return !oom;
  }

 private:
  using Body = std::function<void()>;
  static thread_local bool t_in_worker;

  WorkerPool() : pid_(getpid()) {}

  template <class F>
  static bool run_inline(int count, F& fn) {
    try {
      for (int i = 0; i < count; ++i) fn(i);
    } catch (const std::bad_alloc&) {
      return false;
    }
    return true;
  }

  void grow(int n) {
    while ((int)n_workers_ < n) {
      const int id = n_workers_++;
      std::thread([this, id] { loop(id); }).detach();
    }
  }

  void loop(int id) {
    t_in_worker = true;
    uint64_t seen = 0;
    for (;;) {
      Body* body;
      {
        std::unique_lock<std::mutex> lk(m_);
        cv_start_.wait(lk, [&] { return generation_ != seen; });
        seen = generation_;
        if (id >= helpers_) continue;  // not needed for this job
        body = body_;
      }
      (*body)();
      {
        std::lock_guard<std::mutex> lk(m_);
        ++done_;
      }
      cv_done_.notify_one();
    }
  }

  const pid_t pid_;
  std::mutex job_mutex_;  // one job at a time
  std::mutex m_;
  std::condition_variable cv_start_, cv_done_;
  Body* body_ = nullptr;
  int helpers_ = 0, done_ = 0, n_workers_ = 0;
  uint64_t generation_ = 0;
};

thread_local bool WorkerPool::t_in_worker = false;

// Run fn(i) for i in [0, count) on up to n_threads threads (0: the host's
// hardware threads, at most 16).  Throws std::bad_alloc if a task did.
template <class F>
void parallel_for(int count, int n_threads, F fn) {
  int nt = n_threads > 0 ? n_threads : (int)std::thread::hardware_concurrency();
  if (n_threads <= 0) nt = std::min(nt, 16);
  nt = std::max(1, std::min({nt, count, 256}));
  const bool ok = nt == 1 ? [&] {
    for (int i = 0; i < count; ++i) fn(i);
    return true;
  }() : WorkerPool::get().run(count, nt, fn);
  if (!ok) throw std::bad_alloc();
}

struct KvState {
  Mat half, ihalf;         // Sigma_k^{1/2}, Sigma_k^{-1/2} (symmetric route)
  Mat L;                   // Cholesky factor of Sigma_k (Cholesky route)
  std::vector<double> mu;  // key mean
  Mat sk;                  // Sigma_k, when computed here
  const double* skp = nullptr;  // Sigma_k (sk, or the caller's moment)
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

int saki_version(void) { return 2; }

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

}  // extern "C"

namespace {

// Both calibration entry points: the moments either come in (Sq_in, Sk_in,
// mu_in, float64) or are computed here from the calibration tokens.
int calibrate_core(const float* q_cal, const float* k_cal, const double* Sq_in,
                   const double* Sk_in, const double* mu_in, int H_q, int H_kv, int T, int d,
                   int r, int method, double floor_rel, float* B_q, float* B_k, float* mu,
                   double* sigma, int* n_clamped, int n_threads) {
  const bool given = Sq_in != nullptr;
  if (!B_q || !B_k || !mu) return SAKI_ERR_ARG;
  if (given ? (!Sk_in || !mu_in) : (!q_cal || !k_cal)) return SAKI_ERR_ARG;
  if (H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || (!given && T <= 0) || d <= 0 || d > 4096 ||
      r <= 0 || r > d || !(floor_rel >= 0.0))
    return SAKI_ERR_ARG;
  if (method != SAKI_METHOD_OPT && method != SAKI_METHOD_KEY_PCA && method != SAKI_METHOD_SHARED &&
      method != SAKI_METHOD_SAP_MAP && method != SAKI_METHOD_SAP_SVD)
    return SAKI_ERR_UNSUPPORTED;
  const int G = H_q / H_kv;
  const size_t dd = (size_t)d * d;
  try {
    // ---- per KV head: key mean, centred key moment, and either its Cholesky
    //      factor or its clamped symmetric roots
    std::vector<KvState> kv(H_kv);
    // every method but key PCA goes through C = Sigma_q^{1/2} Sigma_k^{1/2}
    const bool opt = method != SAKI_METHOD_KEY_PCA;
    // Sigma_q per head: the caller's moments, or computed here
    std::vector<const double*> sq_of(opt ? H_q : 0);
    std::vector<Mat> sq_own(opt && !given ? H_q : 0);
    for (int h = 0; h < (int)sq_of.size(); ++h) sq_of[h] = given ? Sq_in + (size_t)h * dd : nullptr;
    const bool shared = method == SAKI_METHOD_SHARED;
    std::vector<Mat> pooled(shared ? H_kv : 0);
    auto kv_task = [&](int g) {
      KvState& st = kv[g];
      if (given) {
        st.mu.assign(mu_in + (size_t)g * d, mu_in + (size_t)(g + 1) * d);
        st.skp = Sk_in + (size_t)g * dd;
        if (!all_finite(st.mu.data(), d) || !all_finite(st.skp, dd)) return;  // st.ok stays false
      } else {
        const float* k = k_cal + (size_t)g * T * d;
        st.mu.assign(d, 0.0);
        for (int t = 0; t < T; ++t)
          for (int i = 0; i < d; ++i) st.mu[i] += (double)k[(size_t)t * d + i];
        for (int i = 0; i < d; ++i) st.mu[i] /= (double)T;
        st.sk.resize(dd);
        moment(T, d, k, st.mu.data(), st.sk.data());
        st.skp = st.sk.data();
      }
      if (opt) {
        st.L.resize(dd);
        st.chol = unclamped_cholesky(d, st.skp, floor_rel, st.L.data(), true);
        if (st.chol) {
          st.ok = true;
        } else {
          st.half.resize(dd);
          st.ihalf.resize(dd);
          st.ok = clamped_roots(d, st.skp, floor_rel, st.half.data(), st.ihalf.data(),
                                &st.n_clamped);
        }
      } else {
        st.ok = true;
      }
      for (int i = 0; i < d; ++i) mu[(size_t)g * d + i] = (float)st.mu[i];
    };
    auto qm_task = [&](int h) {  // uncentred query moment from the tokens
      sq_own[h].resize(dd);
      moment(T, d, q_cal + (size_t)h * T * d, nullptr, sq_own[h].data());
      sq_of[h] = sq_own[h].data();
    };
    // one shared map per KV group: the group's pooled query moment
    // (1/G) sum_h Sigma_q^(h) goes through the per-head steps once, for the
    // group's first head, and the factors are copied to the others
    auto pool_task = [&](int g) {
      for (int hh = 0; hh < G; ++hh)
        if (!sq_of[(size_t)g * G + hh]) return;  // a moment failed: sq_of stays unpooled
      Mat& pool = pooled[g];
      pool.assign(sq_of[(size_t)g * G], sq_of[(size_t)g * G] + dd);
      for (int hh = 1; hh < G; ++hh) {
        const double* o = sq_of[(size_t)g * G + hh];
        for (size_t i = 0; i < dd; ++i) pool[i] += o[i];
      }
      for (size_t i = 0; i < dd; ++i) pool[i] /= (double)G;
    };

    // One task list, claimed in this order: KV heads, query moments (tokens
    // given), pooled group moments (shared map), then the per-head factors.
    // A task waits only for earlier tasks whose results it reads; those are
    // already claimed by threads that never wait on later tasks, so the
    // kinds overlap without a barrier and the waits always end.
    // A head on the Cholesky route takes two tasks: the reduction of M to
    // tridiagonal form, then its eigenpairs and factor columns (halves of
    // about equal cost, so that threads slowed by other work on the host
    // hold up less of the call).
    const int n_qm = (int)sq_own.size(), n_pool = (int)pooled.size();
    const int n_pre = H_kv + n_qm + n_pool;
    const int n_head = shared ? H_kv : H_q;
    std::unique_ptr<std::atomic<int>[]> done(new std::atomic<int>[n_pre + n_head]);
    for (int t = 0; t < n_pre + n_head; ++t) done[t].store(0, std::memory_order_relaxed);
    struct Reduced {  // a head's M in tridiagonal form, between its two tasks
      std::vector<double> diag, off, beta;
      bool pending = false;
    };
    std::vector<Reduced> red(n_head);
    ScopedBuffer hv_all(opt ? (size_t)n_head * dd : 1);
    auto wait_for = [&](int t) {
      while (done[t].load(std::memory_order_acquire) == 0) _mm_pause();
    };
    struct Finish {  // marks a task done however it ends (bad_alloc included)
      std::atomic<int>& flag;
      ~Finish() { flag.store(1, std::memory_order_release); }
    };
    std::atomic<int> failed(0);
    // Cholesky route, second half: B_q = L v / sqrt(s), B_k = L^-T v sqrt(s)
    // for the top-r eigenpairs (s, v) of M = L^T Sigma_q L
    auto chol_factors = [&](int h, int task) {
      const Reduced& rd = red[task];
      const double* L = kv[h / G].L.data();
      float* bq = B_q + (size_t)h * d * r;
      float* bk = B_k + (size_t)h * d * r;
      std::vector<double> sig(d), bqc(d), bkc(d);
      std::vector<double> w(d), vt((size_t)r * d);
      if (!top_eigpairs(d, rd.diag.data(), rd.off.data(), hv_all.data() + (size_t)task * dd,
                        rd.beta.data(), r, w.data(), vt.data(), sigma != nullptr)) {
        failed = 1;
        return;
      }
      for (int m = 0; m < (sigma ? d : r); ++m) sig[m] = std::sqrt(std::max(w[m], 0.0));
      // all r columns at once (d x r, row-major): P = L V', X = L^-T V'
      Mat V((size_t)d * r), P((size_t)d * r), X((size_t)d * r);
      for (int m = 0; m < r; ++m)
        for (int i = 0; i < d; ++i) V[(size_t)i * r + m] = vt[(size_t)m * d + i];
      lower_times(d, r, L, V.data(), P.data());
      if (method == SAKI_METHOD_SAP_MAP) {  // column m of P = L V' is Sigma_k^{1/2} v_m
        Mat Qr((size_t)r * d);
        for (int m = 0; m < r; ++m)
          for (int i = 0; i < d; ++i) Qr[(size_t)m * d + i] = P[(size_t)i * r + m];
        if (!orthonormal_rows(d, r, Qr.data())) { failed = 1; return; }
        store_basis(d, r, Qr.data(), bq, bk);
        if (sigma)
          for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
        if (n_clamped) { n_clamped[2 * h] = 0; n_clamped[2 * h + 1] = 0; }
        return;
      }
      lower_t_solve(d, r, L, V.data(), X.data());  // L^T X = V
      for (int m = 0; m < r; ++m) {
        const double sm = sig[m], rs = std::sqrt(sm);
        for (int i = 0; i < d; ++i) {
          bqc[i] = sm > 0.0 ? P[(size_t)i * r + m] / rs : 0.0;
          bkc[i] = X[(size_t)i * r + m] * rs;
        }
        store_pair(d, r, m, bqc.data(), bkc.data(), bq, bk);
      }
      if (sigma)
        for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
      if (n_clamped) { n_clamped[2 * h] = 0; n_clamped[2 * h + 1] = 0; }
    };
    parallel_for(n_pre + 2 * n_head, n_threads, [&](int t) {
      if (t < n_pre) {
        Finish fin{done[t]};
        if (t < H_kv) {
          kv_task(t);
        } else if (t < H_kv + n_qm) {
          qm_task(t - H_kv);
        } else {
          const int g = t - H_kv - n_qm;
          if (!given)
            for (int hh = 0; hh < G; ++hh) wait_for(H_kv + g * G + hh);
          pool_task(g);
        }
        return;
      }
      if (t >= n_pre + n_head) {  // second half of a Cholesky-route head
        const int task = t - n_pre - n_head;
        wait_for(n_pre + task);
        if (!red[task].pending) return;
        const int h = shared ? task * G : task;
        chol_factors(h, task);
        return;
      }
      const int task = t - n_pre;
      Finish fin{done[t]};
      const int h = shared ? task * G : task;
      wait_for(h / G);
      const KvState& st = kv[h / G];
      if (!st.ok) { failed = 1; return; }
      float* bq = B_q + (size_t)h * d * r;
      float* bk = B_k + (size_t)h * d * r;
      if (method == SAKI_METHOD_KEY_PCA) {
        std::vector<double> w(d), vt(dd);
        if (!sym_eig_rows(d, st.skp, w.data(), vt.data())) { failed = 1; return; }
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
      // Sigma_q (uncentred): the caller's, this head's moment task, or the pool
      if (shared)
        wait_for(H_kv + n_qm + task);
      else if (!given)
        wait_for(H_kv + h);
      const double* sq = shared ? (pooled[task].empty() ? nullptr : pooled[task].data()) : sq_of[h];
      if (!sq) { failed = 1; return; }
      if (given && !all_finite(sq, dd)) { failed = 1; return; }
      std::vector<double> sig(d), bqc(d), bkc(d);
      // (SAP-svd needs the singular vectors of C with symmetric roots)
      if (st.chol && method != SAKI_METHOD_SAP_SVD &&
          unclamped_cholesky(d, sq, floor_rel, thread_buffer(0, dd), false)) {
        // ---- Cholesky route: M = L^T Sigma_q L, reduced to tridiagonal form here;
        //      the eigenpairs and columns are the head's second task
        double* M = thread_buffer(1, dd);
        congruence_lower(d, sq, st.L.data(), M);
        Reduced& rd = red[task];
        rd.diag.resize(d);
        rd.off.resize(d);
        rd.beta.resize(d);
        if (!tridiag_of(d, M, rd.diag.data(), rd.off.data(), hv_all.data() + (size_t)task * dd,
                        rd.beta.data())) {
          failed = 1;
          return;
        }
        rd.pending = true;
        return;
      }
      // ---- symmetric route: clamped roots of both moments
      Mat qh(dd), qih(dd);
      int nq = 0;
      if (!clamped_roots(d, sq, floor_rel, qh.data(), qih.data(), &nq)) { failed = 1; return; }
      Mat kh_local, kih_local;
      const double* khalf = st.half.data();
      const double* kihalf = st.ihalf.data();
      int nk = st.n_clamped;
      if (st.chol) {  // Sigma_k took the Cholesky route: its roots are needed here only
        kh_local.resize(dd);
        kih_local.resize(dd);
        if (!clamped_roots(d, st.skp, floor_rel, kh_local.data(), kih_local.data(), &nk)) {
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
      std::vector<double> w(d), vt((size_t)r * d);
      if (!sym_eig_top(d, CtC.data(), r, w.data(), vt.data(), sigma != nullptr)) { failed = 1; return; }
      for (int m = 0; m < (sigma ? d : r); ++m) sig[m] = std::sqrt(std::max(w[m], 0.0));
      if (sigma)
        for (int m = 0; m < d; ++m) sigma[(size_t)h * d + m] = sig[m];
      if (n_clamped) { n_clamped[2 * h] = nq; n_clamped[2 * h + 1] = nk; }
      if (method == SAKI_METHOD_SAP_SVD || method == SAKI_METHOD_SAP_MAP) {
        Mat Qr((size_t)r * d);
        for (int m = 0; m < r; ++m) {
          const double* v = vt.data() + (size_t)m * d;
          double* qm = Qr.data() + (size_t)m * d;
          if (method == SAKI_METHOD_SAP_SVD) {
            std::copy(v, v + d, qm);
          } else {  // Sigma_k^{1/2} v_m
            for (int i = 0; i < d; ++i) qm[i] = dot(khalf + (size_t)i * d, v, d);
          }
        }
        if (!orthonormal_rows(d, r, Qr.data())) { failed = 1; return; }
        store_basis(d, r, Qr.data(), bq, bk);
        return;
      }
      // top-r pairs: v_m (row of vt), u_m = C v_m / sigma_m
      std::vector<double> u(d);
      for (int m = 0; m < r; ++m) {
        const double* v = vt.data() + (size_t)m * d;
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
    if (shared && !failed) {  // the group's other heads get its factors
      for (int g = 0; g < H_kv; ++g)
        for (int hh = 1; hh < G; ++hh) {
          const size_t h0 = (size_t)g * G, h1 = h0 + hh;
          std::copy(B_q + h0 * d * r, B_q + (h0 + 1) * d * r, B_q + h1 * d * r);
          std::copy(B_k + h0 * d * r, B_k + (h0 + 1) * d * r, B_k + h1 * d * r);
          if (sigma) std::copy(sigma + h0 * d, sigma + (h0 + 1) * d, sigma + h1 * d);
          if (n_clamped) {
            n_clamped[2 * h1] = n_clamped[2 * h0];
            n_clamped[2 * h1 + 1] = n_clamped[2 * h0 + 1];
          }
        }
    }
    if (failed) return SAKI_ERR_NUMERIC;
  } catch (const std::bad_alloc&) {
    return SAKI_ERR_NOMEM;
  }
  return SAKI_OK;
}

}  // namespace

extern "C" {

int saki_calibrate(const float* q_cal, const float* k_cal, int H_q, int H_kv,
                   int T, int d, int r, int method, double floor_rel,
                   float* B_q, float* B_k, float* mu, double* sigma,
                   int* n_clamped, int n_threads) {
  if (!q_cal || !k_cal) return SAKI_ERR_ARG;
  return calibrate_core(q_cal, k_cal, nullptr, nullptr, nullptr, H_q, H_kv, T, d, r, method,
                        floor_rel, B_q, B_k, mu, sigma, n_clamped, n_threads);
}

int saki_calibrate_from_moments(const double* Sigma_q, const double* Sigma_k,
                                const double* key_mean, int H_q, int H_kv, int d, int r,
                                int method, double floor_rel, float* B_q, float* B_k, float* mu,
                                double* sigma, int* n_clamped, int n_threads) {
  if (!Sigma_q || !Sigma_k || !key_mean) return SAKI_ERR_ARG;
  return calibrate_core(nullptr, nullptr, Sigma_q, Sigma_k, key_mean, H_q, H_kv, 0, d, r,
                        method, floor_rel, B_q, B_k, mu, sigma, n_clamped, n_threads);
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
      (sketch_dtype != SAKI_F32 && sketch_dtype != SAKI_BF16 && sketch_dtype != SAKI_FP8))
    return 0;
  return saki::index_bytes(B, H_q, N_cap, r, sketch_dtype);
}

size_t saki_score_topk_workspace_bytes(int B, int H_q, int index_heads, int Q, int N_valid,
                                       int r, int k, int sketch_dtype) {
  if (B <= 0 || H_q <= 0 || index_heads <= 0 || H_q % index_heads != 0 || Q < 0 ||
      N_valid < 0 || !saki::rank_supported(r) || k < 1 || k > saki::kMaxK ||
      (sketch_dtype != SAKI_F32 && sketch_dtype != SAKI_BF16 && sketch_dtype != SAKI_FP8))
    return 0;
  return saki::score_plan(B, H_q, index_heads, Q, N_valid, r, sketch_dtype).ws_bytes;
}

size_t saki_recall_workspace_bytes(int B, int H_q, int H_kv, int Q, int N_valid, int d, int k) {
  if (B <= 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || Q < 0 || N_valid < 0 ||
      d != saki::kHeadDim || k < 1 || k > saki::kMaxK)
    return 0;
  return saki::recall_plan(B, H_q, H_kv, Q, N_valid).ws_bytes;
}

}  // extern "C"
