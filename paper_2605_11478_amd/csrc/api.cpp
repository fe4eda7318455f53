// C ABI of libfibq.so: argument validation and dispatch.  Every entry point
// validates synchronously and returns a status; nothing throws across the ABI.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <exception>

#include <vector>

#include "fibq.h"
#include "fibq_internal.h"

using fibq::dev::Shape;

namespace {

int log2_exact(int N) {
  if (N < 2 || N > 65536 || (N & (N - 1)) != 0) return -1;
  int w = 0;
  while ((1 << w) < N) ++w;
  return w;
}

// Shape validity (Sec. 3.1): k | d, N = 2^w; rate b = w / k.
int check_shape(int d, int k, int N, Shape* s) {
  if (d <= 0 || k <= 0 || k > d || d % k != 0) return FIBQ_EINVAL;
  const int w = log2_exact(N);
  if (w < 1 || w > 16) return FIBQ_EINVAL;
  s->d = d;
  s->k = k;
  s->N = N;
  s->w = w;
  s->P = ((d / k) * w + 7) / 8;
  return FIBQ_OK;
}

int check_rate(double b, const Shape& s) {
  if (!std::isfinite(b) || std::fabs(b * s.k - s.w) > 1e-9) return FIBQ_EINVAL;
  return FIBQ_OK;
}

int check_supported(const Shape& s) {
  if (s.d != 64 && s.d != 128) return FIBQ_EUNSUPPORTED;
  const bool small_k = s.k == 1 || s.k == 2 || s.k == 4 || s.k == 8 || s.k == 16;
  const bool large_k = (s.k == 32 || s.k == 64) && s.d == 64;  // large-block codes
  if (!small_k && !large_k) return FIBQ_EUNSUPPORTED;
  if (s.N > 16384 || (int64_t)s.N * s.k > (1 << 20)) return FIBQ_EUNSUPPORTED;
  return FIBQ_OK;
}

int hip_status(int rc) { return rc == 0 ? FIBQ_OK : FIBQ_EHIP; }

}  // namespace

extern "C" {

const char* fibq_strerror(int status) {
  switch (status) {
    case FIBQ_OK: return "ok";
    case FIBQ_EINVAL: return "invalid argument (shape, rate, pointer or size)";
    case FIBQ_EUNSUPPORTED: return "valid shape without a kernel instantiation";
    case FIBQ_EHIP: return "HIP launch or runtime error";
    case FIBQ_EIO: return "codebook file missing, short or corrupt";
    case FIBQ_EWORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

int fibq_version(void) { return 100; }

int fibq_payload_bytes(int d, int k, int N) {
  Shape s;
  const int rc = check_shape(d, k, N, &s);
  return rc == FIBQ_OK ? s.P : rc;
}

int fibq_supported(int d, int k, int N) {
  Shape s;
  const int rc = check_shape(d, k, N, &s);
  return rc == FIBQ_OK ? check_supported(s) : rc;
}

int fibq_build_rotation(int d, uint64_t seed, float* R_out) {
  if (d < 1 || d > 1024 || !R_out) return FIBQ_EINVAL;
  try {
    return fibq::host::build_rotation(d, seed, R_out);
  } catch (const std::exception&) {
    return FIBQ_EINVAL;
  }
}

// Symmetric (to 1e-12 of its largest entry) and positive definite (Cholesky).
static bool spd(const double* A, int k) {
  double mx = 0.0;
  for (int i = 0; i < k * k; ++i) {
    if (!std::isfinite(A[i])) return false;
    mx = std::max(mx, std::fabs(A[i]));
  }
  for (int i = 0; i < k; ++i)
    for (int j = 0; j < i; ++j)
      if (std::fabs(A[i * k + j] - A[j * k + i]) > 1e-12 * mx) return false;
  std::vector<double> L((size_t)k * k, 0.0);
  for (int j = 0; j < k; ++j) {
    double s = A[j * k + j];
    for (int p = 0; p < j; ++p) s -= L[j * k + p] * L[j * k + p];
    if (!(s > 0.0)) return false;
    L[j * k + j] = std::sqrt(s);
    for (int i = j + 1; i < k; ++i) {
      double t = A[i * k + j];
      for (int p = 0; p < j; ++p) t -= L[i * k + p] * L[j * k + p];
      L[i * k + j] = t / L[j * k + j];
    }
  }
  return true;
}

int fibq_build_codebook_init(int d, int k, double b, int N, uint64_t seed, int64_t M,
                             int restarts, int iters, int n_threads, int init, int shells,
                             const double* metric, float* C_out, double* train_mse_out,
                             int* shells_out) {
  Shape s;
  int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, s)) != FIBQ_OK) return rc;
  if (restarts < 1 || iters < 0 || !C_out) return FIBQ_EINVAL;
  if (init != FIBQ_INIT_BETA && init != FIBQ_INIT_SHELL && init != FIBQ_INIT_MULTISHELL)
    return FIBQ_EINVAL;
  if (shells < 0 || (shells > 0 && (init != FIBQ_INIT_MULTISHELL || N % shells != 0)))
    return FIBQ_EINVAL;
  if (metric && !spd(metric, k)) return FIBQ_EINVAL;
  if (M <= 0) M = (30LL * N > 100000) ? 30LL * N : 100000;
  if (M > (1LL << 31)) return FIBQ_EINVAL;
  try {
    return fibq::host::build_codebook(d, k, N, seed, M, restarts, iters, n_threads, init, shells,
                                      metric, C_out, train_mse_out, shells_out);
  } catch (const std::exception&) {
    return FIBQ_EINVAL;
  }
}

int fibq_build_codebook(int d, int k, double b, int N, uint64_t seed, int64_t M, int restarts,
                        int iters, int n_threads, float* C_out, double* train_mse_out) {
  return fibq_build_codebook_init(d, k, b, N, seed, M, restarts, iters, n_threads, FIBQ_INIT_BETA,
                                  0, nullptr, C_out, train_mse_out, nullptr);
}

int fibq_save_codebook(const char* path, int d, int k, int N, const float* C, const float* R,
                       uint64_t rotation_seed, uint64_t codebook_seed) {
  Shape s;
  if (!path || !C || !R) return FIBQ_EINVAL;
  const int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  try {
    return fibq::host::save_codebook(path, d, k, N, C, R, rotation_seed, codebook_seed);
  } catch (const std::exception&) {
    return FIBQ_EIO;
  }
}

int fibq_load_codebook(const char* path, int* d, int* k, int* N, float* C, float* R,
                       uint64_t* seeds) {
  if (!path || !d || !k || !N) return FIBQ_EINVAL;
  try {
    return fibq::host::load_codebook(path, d, k, N, C, R, seeds);
  } catch (const std::exception&) {
    return FIBQ_EIO;
  }
}

int fibq_encode(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride, int d, int k,
                double b, int N, const float* R, const float* C, uint8_t* payload,
                uint16_t* norms, void* stream) {
  Shape s;
  int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, s)) != FIBQ_OK) return rc;
  if (dtype != FIBQ_F32 && dtype != FIBQ_F16 && dtype != FIBQ_BF16) return FIBQ_EINVAL;
  if (n_vec < 0 || x_row_stride < d) return FIBQ_EINVAL;
  if ((rc = check_supported(s)) != FIBQ_OK) return rc;
  if (n_vec == 0) return FIBQ_OK;
  if (!x || !R || !C || !payload || !norms) return FIBQ_EINVAL;
  return hip_status(fibq::dev::launch_encode(x, dtype, n_vec, x_row_stride, s, R, C, payload,
                                             norms, stream));
}

// Eq. multishell's L shell radii for (d, k), kept per thread for the last
// (d, k, L) asked for: the inverse incomplete Beta quantiles cost more host
// time than a small launch.
static const double* shell_radii(int d, int k, int L) {
  thread_local int key[3] = {0, 0, 0};
  thread_local double r[256];
  if (key[0] != d || key[1] != k || key[2] != L) {
    fibq::host::radii(d, k, L, r);
    key[0] = d;
    key[1] = k;
    key[2] = L;
  }
  return r;
}

int fibq_encode_radius_first(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride, int d,
                             int k, double b, int N, int L, const float* R, const float* C,
                             uint8_t* payload, uint16_t* norms, void* stream) {
  Shape s;
  int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, s)) != FIBQ_OK) return rc;
  if (dtype != FIBQ_F32 && dtype != FIBQ_F16 && dtype != FIBQ_BF16) return FIBQ_EINVAL;
  if (n_vec < 0 || x_row_stride < d) return FIBQ_EINVAL;
  if (L < 1 || L > 256 || (L & (L - 1)) != 0 || N % L != 0) return FIBQ_EINVAL;
  if ((rc = check_supported(s)) != FIBQ_OK) return rc;
  if (n_vec == 0) return FIBQ_OK;
  if (!x || !R || !C || !payload || !norms) return FIBQ_EINVAL;
  return hip_status(fibq::dev::launch_encode_shells(x, dtype, n_vec, x_row_stride, s, L,
                                                    shell_radii(d, k, L), R, C, payload, norms,
                                                    stream));
}

int fibq_build_parent_lists(const float* C, int N, int k, int L, int K, int rounds,
                            double* mu_out, int32_t* offsets_out, int32_t* members_out) {
  if (!C || !mu_out || !offsets_out || !members_out) return FIBQ_EINVAL;
  if (N < 2 || k < 1 || L < 1 || N % L != 0 || K < 1 || K > N / L || K > 64 || rounds < 0)
    return FIBQ_EINVAL;
  try {
    return fibq::host::build_parent_lists(C, N, k, L, K, rounds, mu_out, offsets_out,
                                          members_out);
  } catch (const std::exception&) {
    return FIBQ_EINVAL;
  }
}

int fibq_encode_list(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride, int d, int k,
                     double b, int N, int L, int K, int T, const double* mu,
                     const int32_t* offsets, const int32_t* members, const float* R,
                     const float* C, uint8_t* payload, uint16_t* norms, void* stream) {
  Shape s;
  int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, s)) != FIBQ_OK) return rc;
  if (dtype != FIBQ_F32 && dtype != FIBQ_F16 && dtype != FIBQ_BF16) return FIBQ_EINVAL;
  if (n_vec < 0 || x_row_stride < d) return FIBQ_EINVAL;
  if (L < 1 || L > 256 || (L & (L - 1)) != 0 || N % L != 0) return FIBQ_EINVAL;
  if (K < 1 || K > N / L || K > 64 || T < 1 || T > 8 || T > K) return FIBQ_EINVAL;
  if (!((d == 64 && (k == 4 || k == 8 || k == 16 || k == 32)) ||
        (d == 128 && (k == 4 || k == 8 || k == 16))))
    return FIBQ_EUNSUPPORTED;
  if ((rc = check_supported(s)) != FIBQ_OK) return rc;
  if (n_vec == 0) return FIBQ_OK;
  if (!x || !R || !C || !payload || !norms || !mu || !offsets || !members) return FIBQ_EINVAL;
  return hip_status(fibq::dev::launch_encode_list(x, dtype, n_vec, x_row_stride, s, L,
                                                  shell_radii(d, k, L), K,
                                                  T, mu, offsets, members, R, C, payload, norms,
                                                  stream));
}

int fibq_decode(const uint8_t* payload, const uint16_t* norms, const int64_t* token_ids,
                int64_t n_vec, int64_t n_cache, int d, int k, double b, int N, const float* R,
                const float* C, float* x_hat, void* stream) {
  Shape s;
  int rc = check_shape(d, k, N, &s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, s)) != FIBQ_OK) return rc;
  if (n_vec < 0 || n_cache < 0) return FIBQ_EINVAL;
  if (!token_ids && n_vec > n_cache) return FIBQ_EINVAL;
  if ((rc = check_supported(s)) != FIBQ_OK) return rc;
  if (n_vec == 0) return FIBQ_OK;
  if (!payload || !norms || !R || !C || !x_hat) return FIBQ_EINVAL;
  if (reinterpret_cast<uintptr_t>(x_hat) % 16 != 0) return FIBQ_EINVAL;  // float4 row stores
  return hip_status(fibq::dev::launch_decode(payload, norms, token_ids, n_vec, n_cache, s, R, C,
                                             x_hat, stream));
}

size_t fibq_attn_workspace_bytes(int64_t n_groups, int G, int64_t T, int d, int k, int N) {
  Shape s;
  if (check_shape(d, k, N, &s) != FIBQ_OK || check_supported(s) != FIBQ_OK) return 0;
  if (n_groups < 0 || G < 1 || G > 16 || T < 0) return 0;
  return fibq::dev::attn_workspace_bytes(n_groups, G, T, s);
}

// Synchronous checks shared by both attention entry points.  On FIBQ_OK,
// *done tells whether the call is already complete (no groups).
static int attn_check(const void* q, int q_dtype, const uint8_t* k_payload,
                      const uint16_t* k_norms, const uint8_t* v_payload,
                      const uint16_t* v_norms, int64_t n_groups, int G, int64_t T,
                      int64_t T_stride, int d, int k, double b, int N, const float* R,
                      const float* C, float scale, const float* out, Shape* s, bool* done) {
  *done = false;
  int rc = check_shape(d, k, N, s);
  if (rc != FIBQ_OK) return rc;
  if ((rc = check_rate(b, *s)) != FIBQ_OK) return rc;
  if (q_dtype != FIBQ_F32 && q_dtype != FIBQ_F16 && q_dtype != FIBQ_BF16) return FIBQ_EINVAL;
  if (n_groups < 0 || G < 1 || G > 16 || T < 0 || T_stride < T) return FIBQ_EINVAL;
  if (!std::isfinite(scale)) return FIBQ_EINVAL;
  if ((rc = check_supported(*s)) != FIBQ_OK) return rc;
  if (n_groups == 0) {
    *done = true;
    return FIBQ_OK;
  }
  if (!q || !R || !C || !out) return FIBQ_EINVAL;
  if (T > 0 && (!k_payload || !k_norms || !v_payload || !v_norms)) return FIBQ_EINVAL;
  return FIBQ_OK;
}

int fibq_attn_decode(const void* q, int q_dtype, const uint8_t* k_payload,
                     const uint16_t* k_norms, const uint8_t* v_payload, const uint16_t* v_norms,
                     int64_t n_groups, int G, int64_t T, int64_t T_stride, int d, int k,
                     double b, int N, const float* R, const float* C, float scale, float* out,
                     void* workspace, size_t workspace_bytes, void* stream) {
  Shape s;
  bool done = false;
  const int rc = attn_check(q, q_dtype, k_payload, k_norms, v_payload, v_norms, n_groups, G, T,
                            T_stride, d, k, b, N, R, C, scale, out, &s, &done);
  if (rc != FIBQ_OK || done) return rc;
  const size_t need = fibq::dev::attn_workspace_bytes(n_groups, G, T, s);
  if (need > 0 && (!workspace || workspace_bytes < need)) return FIBQ_EWORKSPACE;
  if (scale <= 0.0f) scale = 1.0f / std::sqrt((float)d);
  return hip_status(fibq::dev::launch_attn(q, q_dtype, k_payload, k_norms, v_payload, v_norms,
                                           n_groups, G, T, T_stride, s, R, C, scale, out,
                                           workspace, workspace_bytes, stream));
}

int fibq_attn_decode_noalloc(const void* q, int q_dtype, const uint8_t* k_payload,
                             const uint16_t* k_norms, const uint8_t* v_payload,
                             const uint16_t* v_norms, int64_t n_groups, int G, int64_t T,
                             int64_t T_stride, int d, int k, double b, int N, const float* R,
                             const float* C, float scale, float* out, void* stream) {
  Shape s;
  bool done = false;
  const int rc = attn_check(q, q_dtype, k_payload, k_norms, v_payload, v_norms, n_groups, G, T,
                            T_stride, d, k, b, N, R, C, scale, out, &s, &done);
  if (rc != FIBQ_OK || done) return rc;
  if (fibq::dev::attn_workspace_bytes(n_groups, G, T, s) > FIBQ_ATTN_SCRATCH_BYTES)
    return FIBQ_EWORKSPACE;
  void* ws = nullptr;
  if (fibq::dev::static_attn_scratch(&ws) != 0) return FIBQ_EHIP;
  if (scale <= 0.0f) scale = 1.0f / std::sqrt((float)d);
  return hip_status(fibq::dev::launch_attn(q, q_dtype, k_payload, k_norms, v_payload, v_norms,
                                           n_groups, G, T, T_stride, s, R, C, scale, out, ws,
                                           FIBQ_ATTN_SCRATCH_BYTES, stream));
}

}  // extern "C"
