// Offline construction of the codec's shared objects: the Haar rotation and
// the radial-angular codebook (Sec. 3 overview; Sec. 3.3; App. A
// codebook-construction table), plus the codebook file.  Host code only.
//
// Random draws: Philox4x32-10 (Salmon et al., SC'11) turned into standard
// normals by Box-Muller.  Normal n of stream (seed, tag) comes from block
// j = n / 2 with counter (j lo, j hi, tag, 0) and key (seed lo, seed hi);
// 53-bit uniforms u1 = (((w0 << 21) | (w1 >> 11)) + 0.5) / 2^53 and
// u2 likewise from (w2, w3); r = sqrt(-2 ln u1); normal 2j = r cos(2 pi u2),
// normal 2j + 1 = r sin(2 pi u2).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <thread>
#include <vector>

#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace host {

// ------------------------------------------------------------ Philox -------
static inline void philox_round(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
  const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
  const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    philox_round(c, k0, k1);
  }
  for (int i = 0; i < 4; ++i) out[i] = c[i];
}

void normals(uint64_t seed, uint32_t tag, uint64_t start, uint64_t count, double* out) {
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  const double two53 = 9007199254740992.0;
  uint64_t n = start;
  const uint64_t end = start + count;
  while (n < end) {
    const uint64_t j = n >> 1;
    const uint32_t ctr[4] = {(uint32_t)j, (uint32_t)(j >> 32), tag, 0u};
    uint32_t w[4];
    philox4x32_10(ctr, key, w);
    const uint64_t a = ((uint64_t)w[0] << 21) | (w[1] >> 11);
    const uint64_t b = ((uint64_t)w[2] << 21) | (w[3] >> 11);
    const double u1 = ((double)a + 0.5) / two53;
    const double u2 = ((double)b + 0.5) / two53;
    const double r = std::sqrt(-2.0 * std::log(u1));
    const double ang = 2.0 * M_PI * u2;
    if ((n & 1) == 0) {
      out[n - start] = r * std::cos(ang);
      if (n + 1 < end) out[n + 1 - start] = r * std::sin(ang);
      n += 2;
    } else {
      out[n - start] = r * std::sin(ang);
      n += 1;
    }
  }
}

// --------------------------------------------------- Haar via Householder ---
// Q of A = QR with diag(R) > 0, A row-major n x n; Q written row-major.
void haar_q(int n, const double* A, double* Q) {
  std::vector<double> R(A, A + (size_t)n * n);
  std::vector<double> V((size_t)n * n, 0.0);  // Householder vectors, column j in V[:, j]
  std::vector<double> beta(n, 0.0);
  for (int j = 0; j < n; ++j) {
    double norm2 = 0.0;
    for (int i = j; i < n; ++i) norm2 += R[(size_t)i * n + j] * R[(size_t)i * n + j];
    const double norm = std::sqrt(norm2);
    const double x0 = R[(size_t)j * n + j];
    const double alpha = (x0 >= 0.0) ? -norm : norm;  // avoids cancellation
    for (int i = j; i < n; ++i) V[(size_t)i * n + j] = R[(size_t)i * n + j];
    V[(size_t)j * n + j] = x0 - alpha;
    double vnorm2 = 0.0;
    for (int i = j; i < n; ++i) vnorm2 += V[(size_t)i * n + j] * V[(size_t)i * n + j];
    beta[j] = (vnorm2 > 0.0) ? 2.0 / vnorm2 : 0.0;
    for (int c = j; c < n; ++c) {  // R <- (I - beta v v^T) R
      double s = 0.0;
      for (int i = j; i < n; ++i) s += V[(size_t)i * n + j] * R[(size_t)i * n + c];
      s *= beta[j];
      for (int i = j; i < n; ++i) R[(size_t)i * n + c] -= s * V[(size_t)i * n + j];
    }
  }
  // Q = H_0 H_1 ... H_{n-1}: apply to the identity from the right-most factor.
  for (size_t i = 0; i < (size_t)n * n; ++i) Q[i] = 0.0;
  for (int i = 0; i < n; ++i) Q[(size_t)i * n + i] = 1.0;
  for (int j = n - 1; j >= 0; --j) {
    for (int c = 0; c < n; ++c) {
      double s = 0.0;
      for (int i = j; i < n; ++i) s += V[(size_t)i * n + j] * Q[(size_t)i * n + c];
      s *= beta[j];
      for (int i = j; i < n; ++i) Q[(size_t)i * n + c] -= s * V[(size_t)i * n + j];
    }
  }
  // Sign fix: Q <- Q diag(sign(diag R)), making the factorisation unique.
  for (int c = 0; c < n; ++c) {
    if (R[(size_t)c * n + c] < 0.0)
      for (int i = 0; i < n; ++i) Q[(size_t)i * n + c] = -Q[(size_t)i * n + c];
  }
}

// ------------------------------------------------- regularised beta -------
// I_x(a, b) by the continued fraction of the incomplete beta function
// (modified Lentz), with the symmetry I_x(a,b) = 1 - I_{1-x}(b,a).
static double betacf(double a, double b, double x) {
  const double tiny = 1e-300, eps = 1e-16;
  double c = 1.0, d = 1.0 - (a + b) * x / (a + 1.0);
  if (std::fabs(d) < tiny) d = tiny;
  d = 1.0 / d;
  double h = d;
  for (int m = 1; m <= 10000; ++m) {
    const double m2 = 2.0 * m;
    double aa = m * (b - m) * x / ((a + m2 - 1.0) * (a + m2));
    d = 1.0 + aa * d;
    if (std::fabs(d) < tiny) d = tiny;
    c = 1.0 + aa / c;
    if (std::fabs(c) < tiny) c = tiny;
    d = 1.0 / d;
    h *= d * c;
    aa = -(a + m) * (a + b + m) * x / ((a + m2) * (a + m2 + 1.0));
    d = 1.0 + aa * d;
    if (std::fabs(d) < tiny) d = tiny;
    c = 1.0 + aa / c;
    if (std::fabs(c) < tiny) c = tiny;
    d = 1.0 / d;
    const double del = d * c;
    h *= del;
    if (std::fabs(del - 1.0) < eps) break;
  }
  return h;
}

double beta_inc(double a, double b, double x) {
  if (x <= 0.0) return 0.0;
  if (x >= 1.0) return 1.0;
  const double lbt = std::lgamma(a + b) - std::lgamma(a) - std::lgamma(b) + a * std::log(x) +
                     b * std::log1p(-x);
  const double bt = std::exp(lbt);
  if (x < (a + 1.0) / (a + b + 2.0)) return bt * betacf(a, b, x) / a;
  return 1.0 - bt * betacf(b, a, 1.0 - x) / b;
}

// Inverse of I_x(a, b) in x: bisection to a bracket, then Newton steps with
// the Beta density, each kept inside the bracket.
double beta_inc_inv(double a, double b, double p) {
  if (p <= 0.0) return 0.0;
  if (p >= 1.0) return 1.0;
  double lo = 0.0, hi = 1.0, x = 0.5;
  for (int it = 0; it < 60; ++it) {
    x = 0.5 * (lo + hi);
    if (beta_inc(a, b, x) < p) lo = x; else hi = x;
  }
  const double lbeta = std::lgamma(a) + std::lgamma(b) - std::lgamma(a + b);
  for (int it = 0; it < 50; ++it) {
    const double f = beta_inc(a, b, x) - p;
    if (f < 0.0) lo = x; else hi = x;
    const double dens = std::exp((a - 1.0) * std::log(x) + (b - 1.0) * std::log1p(-x) - lbeta);
    double xn = (dens > 0.0) ? x - f / dens : 0.5 * (lo + hi);
    if (!(xn > lo && xn < hi)) xn = 0.5 * (lo + hi);
    if (std::fabs(xn - x) <= 1e-17 * std::max(1.0, x)) { x = xn; break; }
    x = xn;
  }
  return x;
}

// Standard-normal quantile: bisection-bracketed Newton on Phi(z) = erfc(-z/sqrt2)/2.
double norm_inv(double p) {
  double lo = -40.0, hi = 40.0, z = 0.0;
  for (int it = 0; it < 200; ++it) {
    const double f = 0.5 * std::erfc(-z / M_SQRT2) - p;
    if (f < 0.0) lo = z; else hi = z;
    const double dens = std::exp(-0.5 * z * z) / std::sqrt(2.0 * M_PI);
    double zn = (dens > 1e-300) ? z - f / dens : 0.5 * (lo + hi);
    if (!(zn > lo && zn < hi)) zn = 0.5 * (lo + hi);
    if (std::fabs(zn - z) < 1e-15 * std::max(1.0, std::fabs(z))) { z = zn; break; }
    z = zn;
  }
  return z;
}

// ------------------------------------------------------- radii, directions --
void radii(int d, int k, int N, double* r) {
  const double beta_dk = (double)k / (k + 2.0) * (d - k - 2.0) / 2.0 + 1.0;
  for (int n = 1; n <= N; ++n) {
    const double q = (n - 0.5) / N;
    if (k == 2) r[n - 1] = std::sqrt(1.0 - std::pow(1.0 - q, 4.0 / d));  // Eq. radii_k2
    else r[n - 1] = std::sqrt(beta_inc_inv(0.5 * k, beta_dk, q));        // Eq. radii_main
  }
}

double roberts_phi(int k) {
  double lo = 1.0, hi = 2.0;
  for (int it = 0; it < 200; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (std::pow(mid, k + 1) - mid - 1.0 > 0.0) hi = mid; else lo = mid;
  }
  return 0.5 * (lo + hi);
}

// Directions u_n for n = offset+1 .. offset+N.  A positive offset continues
// the sequence, which gives each shell of the multi-shell codebook its own
// set (App. E); at k = 3 the latitude bands restart, only the azimuth continues.
void directions(int k, int N, double* u, int64_t offset) {
  const double golden = (1.0 + std::sqrt(5.0)) / 2.0;
  for (int64_t n = offset + 1; n <= offset + N; ++n) {
    double* un = u + (size_t)(n - offset - 1) * k;
    if (k == 1) {
      un[0] = (n % 2 == 1) ? 1.0 : -1.0;
    } else if (k == 2) {  // planar Fibonacci spiral
      const double th = 2.0 * M_PI * ((double)n - 1.0) * (1.0 - 1.0 / golden);
      un[0] = std::cos(th);
      un[1] = std::sin(th);
    } else if (k == 3) {  // Fibonacci sphere (App. E)
      const double z = 1.0 - (2.0 * (double)(n - offset) - 1.0) / N;
      const double th = 2.0 * M_PI * ((double)n - 1.0) * (1.0 - 1.0 / golden);
      const double rho = std::sqrt(1.0 - z * z);
      un[0] = rho * std::cos(th);
      un[1] = rho * std::sin(th);
      un[2] = z;
    } else {  // Roberts-Kronecker rank-one sequence, Gaussianised and projected
      const double phi = roberts_phi(k);
      double s = 0.0;
      for (int j = 1; j <= k; ++j) {
        double xi = std::fmod(((double)n - 0.5) * std::pow(phi, -(double)j), 1.0);
        un[j - 1] = norm_inv(xi);
        s += un[j - 1] * un[j - 1];
      }
      s = std::sqrt(s);
      for (int j = 0; j < k; ++j) un[j] /= s;
    }
  }
}

// ------------------------------------------------------------- Lloyd-Max ---
namespace {

constexpr int64_t kChunk = 8192;  // fixed partition: results independent of threads

struct Pool {
  int nt;
  explicit Pool(int n) : nt(n) {}
  template <class F>
  void run(int64_t nchunks, F f) const {
    if (nt <= 1 || nchunks <= 1) {
      for (int64_t c = 0; c < nchunks; ++c) f(c);
      return;
    }
    std::vector<std::thread> th;
    const int use = (int)std::min<int64_t>(nt, nchunks);
    for (int t = 0; t < use; ++t)
      th.emplace_back([&, t] {
        for (int64_t c = t; c < nchunks; c += use) f(c);
      });
    for (auto& x : th) x.join();
  }
};

// nearest codeword by brute force (direct form, ties -> lowest index)
inline int nearest(const double* x, const double* c, int N, int k, double* dist) {
  int best = 0;
  double bd = 0.0;
  for (int n = 0; n < N; ++n) {
    const double* cn = c + (size_t)n * k;
    double s = 0.0;
    for (int i = 0; i < k; ++i) {
      const double t = x[i] - cn[i];
      s += t * t;
    }
    if (n == 0 || s < bd) { bd = s; best = n; }
  }
  *dist = bd;
  return best;
}

// (x - c)^T M (x - c) for a k x k metric M (row-major), summed over (i, j)
// with i outer; nearest codeword in that metric, ties -> lowest index.
inline double metric_dist(const double* x, const double* c, int k, const double* M) {
  double s = 0.0;
  for (int i = 0; i < k; ++i) {
    const double ti = x[i] - c[i];
    for (int j = 0; j < k; ++j) s += ti * M[(size_t)i * k + j] * (x[j] - c[j]);
  }
  return s;
}
inline int nearest_metric(const double* x, const double* c, int N, int k, const double* M,
                          double* dist) {
  int best = 0;
  double bd = 0.0;
  for (int n = 0; n < N; ++n) {
    const double s = metric_dist(x, c + (size_t)n * k, k, M);
    if (n == 0 || s < bd) { bd = s; best = n; }
  }
  *dist = bd;
  return best;
}

}  // namespace

double round_to_binary16(double x) {
  if (!(std::fabs(x) < 65504.0)) return x;  // out of the codeword range: unchanged
  const double ax = std::fabs(x);
  double q;  // quantum of binary16 at |x|
  if (ax < 6.103515625e-05) {
    q = 5.9604644775390625e-08;  // 2^-24 (subnormal spacing)
  } else {
    int e;
    std::frexp(ax, &e);  // ax in [2^(e-1), 2^e)
    q = std::ldexp(1.0, e - 11);
  }
  return std::nearbyint(x / q) * q;  // round half to even (default rounding mode)
}

int build_codebook(int d, int k, int N, uint64_t seed, int64_t M, int restarts, int iters,
                   int n_threads, int init, int fixed_shells, const double* metric, float* C_out,
                   double* mse_out, int* shells_out) {
  if (n_threads <= 0) n_threads = (int)std::max(1u, std::thread::hardware_concurrency());
  Pool pool(n_threads);

  // training samples: first k coordinates of normalised d-dim Gaussians
  std::vector<double> X((size_t)M * k);
  const int64_t nchunks = (M + kChunk - 1) / kChunk;
  pool.run(nchunks, [&](int64_t ch) {
    const int64_t s0 = ch * kChunk, s1 = std::min<int64_t>(M, s0 + kChunk);
    std::vector<double> g((size_t)d);
    for (int64_t s = s0; s < s1; ++s) {
      normals(seed, kTagTrain, (uint64_t)s * d, (uint64_t)d, g.data());
      double nn = 0.0;
      for (int i = 0; i < d; ++i) nn += g[i] * g[i];
      nn = std::sqrt(nn);
      for (int i = 0; i < k; ++i) X[(size_t)s * k + i] = g[i] / nn;
    }
  });

  std::vector<int> assign((size_t)M);
  std::vector<double> err((size_t)M);
  std::vector<double> c((size_t)N * k);

  auto assign_all = [&]() {
    pool.run(nchunks, [&](int64_t ch) {
      const int64_t s0 = ch * kChunk, s1 = std::min<int64_t>(M, s0 + kChunk);
      for (int64_t s = s0; s < s1; ++s)
        assign[s] = metric ? nearest_metric(&X[(size_t)s * k], c.data(), N, k, metric, &err[s])
                           : nearest(&X[(size_t)s * k], c.data(), N, k, &err[s]);
    });
  };
  auto train_mse = [&]() {  // assign, then the mean squared error summed in sample order
    assign_all();
    double tot = 0.0;
    for (int64_t s = 0; s < M; ++s) tot += err[s];
    return tot / (double)M;
  };
  // C(S, M_a) of App. E Eq. multishell: S Beta-quantile shells, shell s
  // carrying the next M_a directions of the sequence; the single shell of
  // App. D uses the radius sqrt(k/d) instead.
  auto shells = [&](int S, bool typical_radius, double* out) {
    const int Ma = N / S;
    std::vector<double> r(S), u((size_t)Ma * k);
    if (typical_radius) r[0] = std::sqrt((double)k / d);
    else radii(d, k, S, r.data());
    for (int sh = 0; sh < S; ++sh) {
      directions(k, Ma, u.data(), (int64_t)sh * Ma);
      for (size_t i = 0; i < (size_t)Ma * k; ++i) out[(size_t)sh * Ma * k + i] = r[sh] * u[i];
    }
  };

  std::vector<double> c0((size_t)N * k);
  int n_shells = N;
  if (init == FIBQ_INIT_SHELL) {
    shells(1, true, c0.data());
    n_shells = 1;
  } else if (init == FIBQ_INIT_MULTISHELL && fixed_shells > 0) {  // C(S, N / S), S given
    shells(fixed_shells, false, c0.data());
    n_shells = fixed_shells;
  } else if (init == FIBQ_INIT_MULTISHELL) {  // every factor pair S * M_a = N, lowest training MSE
    double best = INFINITY;
    for (int S = 1; S <= N; ++S) {
      if (N % S) continue;
      shells(S, false, c.data());
      const double m = train_mse();
      if (m < best) {
        best = m;
        n_shells = S;
        c0 = c;
      }
    }
  } else {  // Eq. radii_main: N radii, one direction each (C(N, 1) except at k = 3)
    std::vector<double> r(N), u((size_t)N * k);
    radii(d, k, N, r.data());
    directions(k, N, u.data());
    for (int n = 0; n < N; ++n)
      for (int i = 0; i < k; ++i) c0[(size_t)n * k + i] = r[n] * u[(size_t)n * k + i];
  }

  std::vector<double> best_c(c0);
  double best_d = INFINITY;
  uint64_t repair_events = 0;
  std::vector<double> part_sum((size_t)nchunks * N * k), part_sse((size_t)nchunks * N);
  std::vector<int64_t> part_cnt((size_t)nchunks * N);

  for (int j = 0; j < restarts; ++j) {
    std::vector<double> g((size_t)k * k), om((size_t)k * k);
    normals(seed, kTagRestart, (uint64_t)j * k * k, (uint64_t)k * k, g.data());
    haar_q(k, g.data(), om.data());
    for (int n = 0; n < N; ++n)  // c_n <- Omega_j c_n
      for (int a = 0; a < k; ++a) {
        double s = 0.0;
        for (int bb = 0; bb < k; ++bb) s += om[(size_t)a * k + bb] * c0[(size_t)n * k + bb];
        c[(size_t)n * k + a] = s;
      }
    for (int t = 0; t < iters; ++t) {
      assign_all();
      // per-chunk partial sums, reduced in chunk order
      pool.run(nchunks, [&](int64_t ch) {
        const int64_t s0 = ch * kChunk, s1 = std::min<int64_t>(M, s0 + kChunk);
        double* ps = &part_sum[(size_t)ch * N * k];
        int64_t* pc = &part_cnt[(size_t)ch * N];
        std::fill(ps, ps + (size_t)N * k, 0.0);
        std::fill(pc, pc + N, 0);
        for (int64_t s = s0; s < s1; ++s) {
          const int a = assign[s];
          pc[a] += 1;
          for (int i = 0; i < k; ++i) ps[(size_t)a * k + i] += X[(size_t)s * k + i];
        }
      });
      std::vector<int64_t> cnt(N, 0);
      std::vector<double> sum((size_t)N * k, 0.0);
      for (int64_t ch = 0; ch < nchunks; ++ch)
        for (int n = 0; n < N; ++n) {
          cnt[n] += part_cnt[(size_t)ch * N + n];
          for (int i = 0; i < k; ++i) sum[(size_t)n * k + i] += part_sum[((size_t)ch * N + n) * k + i];
        }
      for (int n = 0; n < N; ++n)
        if (cnt[n] > 0)
          for (int i = 0; i < k; ++i) c[(size_t)n * k + i] = sum[(size_t)n * k + i] / (double)cnt[n];
      // within-cell squared error about the updated centroids
      pool.run(nchunks, [&](int64_t ch) {
        const int64_t s0 = ch * kChunk, s1 = std::min<int64_t>(M, s0 + kChunk);
        double* pe = &part_sse[(size_t)ch * N];
        std::fill(pe, pe + N, 0.0);
        for (int64_t s = s0; s < s1; ++s) {
          const int a = assign[s];
          double e = 0.0;
          if (metric) {
            e = metric_dist(&X[(size_t)s * k], &c[(size_t)a * k], k, metric);
          } else {
            for (int i = 0; i < k; ++i) {
              const double t2 = X[(size_t)s * k + i] - c[(size_t)a * k + i];
              e += t2 * t2;
            }
          }
          pe[a] += e;
        }
      });
      std::vector<double> sse(N, 0.0);
      for (int64_t ch = 0; ch < nchunks; ++ch)
        for (int n = 0; n < N; ++n) sse[n] += part_sse[(size_t)ch * N + n];
      // empty-cell repair: split the occupied cell with the largest SSE
      for (int e = 0; e < N; ++e) {
        if (cnt[e] > 0) continue;
        int donor = -1;
        double bv = -1.0;
        for (int n = 0; n < N; ++n) {
          const double v = (cnt[n] >= 2) ? sse[n] : -1.0;
          if (v > bv) { bv = v; donor = n; }
        }
        if (donor < 0 || bv < 0.0) break;
        std::vector<double> gg((size_t)k);
        normals(seed, kTagRepair, repair_events * (uint64_t)k, (uint64_t)k, gg.data());
        repair_events++;
        double gn = 0.0;
        for (int i = 0; i < k; ++i) gn += gg[i] * gg[i];
        gn = std::sqrt(gn);
        const double scale = 1e-2 * std::sqrt(sse[donor] / (double)cnt[donor]);
        for (int i = 0; i < k; ++i) {
          const double ui = (gn > 0.0) ? gg[i] / gn : (i == 0 ? 1.0 : 0.0);
          const double delta = scale * ui;
          c[(size_t)e * k + i] = c[(size_t)donor * k + i] + delta;
          c[(size_t)donor * k + i] = c[(size_t)donor * k + i] - delta;
        }
        sse[donor] *= 0.5;
        const int64_t half = cnt[donor] / 2;
        cnt[e] = half;
        cnt[donor] -= half;
      }
    }
    const double dj = train_mse();
    if (dj < best_d) {
      best_d = dj;
      best_c = c;
    }
  }
  // Codewords are stored as binary16-representable values (round to nearest,
  // ties to even, on 11 significant bits; quantum 2^-24 below 2^-14): the
  // fused attention reads an fp16 copy of the codebook, which is then exact.
  for (size_t i = 0; i < (size_t)N * k; ++i) C_out[i] = (float)round_to_binary16(best_c[i]);
  if (mse_out) *mse_out = best_d;
  if (shells_out) *shells_out = n_shells;
  return FIBQ_OK;
}

// Stage 2 tables of the list-decoding encoder (App. F): per shell of a
// shell-major codebook, spherical k-means of the codeword directions into K
// parents started from every (M_a / K)-th codeword, `rounds` rounds
// (assignment by the largest inner product, first parent on ties; a parent
// that empties keeps its direction), then a final assignment.  Outputs: mu
// [L][K][k] parent directions, offsets [L][K + 1] and members [N]: the local
// indices of each parent's codewords in increasing order, shell by shell.
int build_parent_lists(const float* C, int N, int k, int L, int K, int rounds, double* mu,
                       int32_t* offsets, int32_t* members) {
  const int Ma = N / L, step = Ma / K;
  std::vector<double> U((size_t)Ma * k), m((size_t)k);
  std::vector<int> g(Ma);
  for (int l = 0; l < L; ++l) {
    for (int n = 0; n < Ma; ++n) {
      const float* c = C + (size_t)(l * Ma + n) * k;
      double s = 0.0;
      for (int i = 0; i < k; ++i) s += (double)c[i] * (double)c[i];
      s = std::sqrt(s);
      for (int i = 0; i < k; ++i) U[(size_t)n * k + i] = s > 0.0 ? (double)c[i] / s : 0.0;
    }
    double* mul = mu + (size_t)l * K * k;
    for (int j = 0; j < K; ++j)
      for (int i = 0; i < k; ++i) mul[(size_t)j * k + i] = U[(size_t)(j * step) * k + i];
    auto assign = [&]() {
      for (int n = 0; n < Ma; ++n) {
        int best = 0;
        double bs = 0.0;
        for (int j = 0; j < K; ++j) {
          double sc = 0.0;
          for (int i = 0; i < k; ++i) sc += U[(size_t)n * k + i] * mul[(size_t)j * k + i];
          if (j == 0 || sc > bs) { bs = sc; best = j; }
        }
        g[n] = best;
      }
    };
    for (int it = 0; it < rounds; ++it) {
      assign();
      for (int j = 0; j < K; ++j) {
        std::fill(m.begin(), m.end(), 0.0);
        for (int n = 0; n < Ma; ++n)
          if (g[n] == j)
            for (int i = 0; i < k; ++i) m[i] += U[(size_t)n * k + i];
        double nn = 0.0;
        for (int i = 0; i < k; ++i) nn += m[i] * m[i];
        nn = std::sqrt(nn);
        if (nn > 0.0)
          for (int i = 0; i < k; ++i) mul[(size_t)j * k + i] = m[i] / nn;
      }
    }
    assign();
    int32_t* off = offsets + (size_t)l * (K + 1);
    int pos = 0;
    for (int j = 0; j < K; ++j) {
      off[j] = pos;
      for (int n = 0; n < Ma; ++n)
        if (g[n] == j) members[(size_t)l * Ma + pos++] = n;
    }
    off[K] = pos;
  }
  return FIBQ_OK;
}

int build_rotation(int d, uint64_t seed, float* R_out) {
  std::vector<double> g((size_t)d * d), q((size_t)d * d);
  normals(seed, kTagRotation, 0, (uint64_t)d * d, g.data());
  haar_q(d, g.data(), q.data());
  for (size_t i = 0; i < (size_t)d * d; ++i) R_out[i] = (float)q[i];
  return FIBQ_OK;
}

// ------------------------------------------------------------- file I/O ----
static uint64_t fnv1a64(const unsigned char* p, size_t n) {
  uint64_t h = 0xCBF29CE484222325ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 0x100000001B3ull;
  }
  return h;
}

static void put32(std::vector<unsigned char>& v, uint32_t x) {
  for (int i = 0; i < 4; ++i) v.push_back((unsigned char)(x >> (8 * i)));
}
static void put64(std::vector<unsigned char>& v, uint64_t x) {
  for (int i = 0; i < 8; ++i) v.push_back((unsigned char)(x >> (8 * i)));
}
static uint32_t get32(const unsigned char* p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}
static uint64_t get64(const unsigned char* p) {
  return (uint64_t)get32(p) | ((uint64_t)get32(p + 4) << 32);
}

int save_codebook(const char* path, int d, int k, int N, const float* C, const float* R,
                  uint64_t s0, uint64_t s1) {
  std::vector<unsigned char> v;
  const char magic[9] = "FIBQCB01";
  v.insert(v.end(), magic, magic + 8);
  put32(v, (uint32_t)d);
  put32(v, (uint32_t)k);
  put32(v, (uint32_t)N);
  put32(v, 0u);
  put64(v, s0);
  put64(v, s1);
  auto putf = [&](const float* a, size_t n) {
    for (size_t i = 0; i < n; ++i) {
      uint32_t b;
      std::memcpy(&b, &a[i], 4);
      put32(v, b);
    }
  };
  putf(C, (size_t)N * k);
  putf(R, (size_t)d * d);
  put64(v, fnv1a64(v.data(), v.size()));
  FILE* f = std::fopen(path, "wb");
  if (!f) return FIBQ_EIO;
  const size_t w = std::fwrite(v.data(), 1, v.size(), f);
  const int rc = std::fclose(f);
  return (w == v.size() && rc == 0) ? FIBQ_OK : FIBQ_EIO;
}

int load_codebook(const char* path, int* d, int* k, int* N, float* C, float* R, uint64_t* seeds) {
  FILE* f = std::fopen(path, "rb");
  if (!f) return FIBQ_EIO;
  std::vector<unsigned char> v;
  unsigned char buf[65536];
  size_t got;
  while ((got = std::fread(buf, 1, sizeof(buf), f)) > 0) v.insert(v.end(), buf, buf + got);
  std::fclose(f);
  if (v.size() < 48 || std::memcmp(v.data(), "FIBQCB01", 8) != 0) return FIBQ_EIO;
  const uint32_t dd = get32(&v[8]), kk = get32(&v[12]), nn = get32(&v[16]);
  if (dd == 0 || kk == 0 || nn == 0 || dd > 4096 || kk > 4096 || nn > (1u << 20)) return FIBQ_EIO;
  const size_t need = 40 + 4 * ((size_t)nn * kk + (size_t)dd * dd) + 8;
  if (v.size() != need) return FIBQ_EIO;
  if (get64(&v[need - 8]) != fnv1a64(v.data(), need - 8)) return FIBQ_EIO;
  *d = (int)dd;
  *k = (int)kk;
  *N = (int)nn;
  if (seeds) {
    seeds[0] = get64(&v[24]);
    seeds[1] = get64(&v[32]);
  }
  if (C && R) {
    std::memcpy(C, &v[40], 4 * (size_t)nn * kk);
    std::memcpy(R, &v[40 + 4 * (size_t)nn * kk], 4 * (size_t)dd * dd);
  }
  return FIBQ_OK;
}

}  // namespace host
}  // namespace fibq
