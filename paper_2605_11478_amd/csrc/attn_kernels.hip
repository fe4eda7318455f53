// Fused dequantisation + single-query decode attention (Eq. lattn over the
// decoded cache of Sec. 3.1), general kernels for every supported shape.
//
// Three launches on the caller's stream:
//   prep : q~_h = Pi q_h per (group, head); when the table fits (<= 64 KB per
//          group) and N <= T / 4 also LUT[h][m][n] = <q~_h^(m), c_n>, so a score is a sum of
//          d/k table entries: <q, K_hat_t> = nu_t sum_m LUT[h][m][i_{t,m}]
//          (Pi orthogonal, so <q, Pi^T c> = <Pi q, c>);
//   main : one workgroup per (split, group); 64-token tiles; scores by table
//          lookup (or by gathering codewords and dotting with q~ when the
//          table is too large), online softmax per head with wavefront
//          reductions, value accumulation sum_t p_t nu_t c_(t) in rotated
//          space; writes the split's (max, sum, acc) partial state;
//   merge: log-sum-exp merge of the splits and one inverse rotation Pi^T
//          per head.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {

constexpr int kAT = 256;                 // threads per workgroup
constexpr int kTT = 64;                  // tokens per tile (= wavefront size)
constexpr size_t kLutMax = 64 * 1024;    // LUT bytes per group held in LDS
constexpr int kTargetWGs = 2048;         // split-K target across the device
constexpr size_t kLdsMax = 160 * 1024;

static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct AttnPlan {
  bool lut;
  int n_split;
  int64_t chunk;
  size_t off_qrot, off_lut, off_ml, off_acc, total;
};

static AttnPlan make_plan(int64_t n_groups, int G, int64_t T, const Shape& s) {
  AttnPlan p{};
  const int NB = s.d / s.k;
  // the table pays off when it is small against the tokens it serves: every
  // split block stages it in LDS, and building it costs N dot products per
  // (head, block) against T per (head, block) when gathering codewords
  p.lut = (size_t)G * NB * s.N * sizeof(float) <= kLutMax && 4 * (int64_t)s.N <= T;
  int64_t ntiles = (T + kTT - 1) / kTT;
  if (ntiles < 1) ntiles = 1;
  int64_t ns = (kTargetWGs + n_groups - 1) / (n_groups > 0 ? n_groups : 1);
  if (ns < 1) ns = 1;
  if (ns > ntiles) ns = ntiles;
  const int64_t tiles_per = (ntiles + ns - 1) / ns;
  p.chunk = tiles_per * kTT;
  p.n_split = (int)((ntiles + tiles_per - 1) / tiles_per);
  size_t off = 0;
  p.off_qrot = off;
  off = align256(off + (size_t)n_groups * G * s.d * sizeof(float));
  p.off_lut = off;
  if (p.lut) off = align256(off + (size_t)n_groups * G * NB * s.N * sizeof(float));
  p.off_ml = off;
  off = align256(off + (size_t)n_groups * p.n_split * G * 2 * sizeof(float));
  p.off_acc = off;
  off = align256(off + (size_t)n_groups * p.n_split * G * s.d * sizeof(float));
  p.total = off;
  return p;
}

size_t attn_workspace_bytes(int64_t n_groups, int G, int64_t T, Shape s) {
  size_t b = make_plan(n_groups, G, T, s).total;
  if (attn_fast_applies(G, s)) {
    const size_t f = attn_fast_workspace_bytes(n_groups, T);
    if (f > b) b = f;
  }
  if (attn_w4_applies(G, s)) {
    const size_t f = attn_w4_workspace_bytes(n_groups, T);
    if (f > b) b = f;
  }
  if (attn_k4_applies(G, s)) {
    const size_t f = attn_k4_workspace_bytes(n_groups, T, s);
    if (f > b) b = f;
  }
  return b;
}

int launch_attn_fast(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                     const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int64_t T,
                     int64_t T_stride, const Shape& s, const float* R, const float* C,
                     float scale, float* out, void* ws, hipStream_t st);
int launch_attn_k4(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                   const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int G, int64_t T,
                   int64_t T_stride, const Shape& s, const float* R, const float* C, float scale,
                   float* out, void* ws, hipStream_t st);
int launch_attn_w4(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                   const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int64_t T,
                   int64_t T_stride, const float* R, const float* C, float scale, float* out,
                   void* ws, hipStream_t st);

__device__ __forceinline__ float load_q(const void* q, int dtype, int64_t i) {
  if (dtype == FIBQ_F32) return static_cast<const float*>(q)[i];
  if (dtype == FIBQ_F16) return to_float(static_cast<const f16_t*>(q)[i]);
  return to_float(static_cast<const bf16_t*>(q)[i]);
}

template <int D, int K>
__global__ __launch_bounds__(kAT) void attn_prep_kernel(const void* __restrict__ q, int q_dtype,
                                                        int G, const float* __restrict__ R,
                                                        const float* __restrict__ C, int N,
                                                        bool lut, float* __restrict__ qrot,
                                                        float* __restrict__ lutg) {
  constexpr int NB = D / K;
  __shared__ float qs[16 * D];
  __shared__ float qt[16 * D];
  const int64_t g = blockIdx.x;
  for (int i = threadIdx.x; i < G * D; i += kAT) qs[i] = load_q(q, q_dtype, g * G * D + i);
  __syncthreads();
  for (int e = threadIdx.x; e < G * D; e += kAT) {
    const int h = e / D, i = e % D;
    float s = 0.0f;
    for (int j = 0; j < D; ++j) s = fmaf(R[i * D + j], qs[h * D + j], s);
    qt[e] = s;
    qrot[g * G * D + e] = s;
  }
  if (!lut) return;
  __syncthreads();
  const int tot = G * NB * N;
  for (int e = threadIdx.x; e < tot; e += kAT) {
    const int n = e % N, hm = e / N, m = hm % NB, h = hm / NB;
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < K; ++r) s = fmaf(qt[h * D + m * K + r], C[n * K + r], s);
    lutg[(int64_t)g * tot + e] = s;
  }
}

struct MainLds {
  size_t lut, qt, cs, kidx, vidx, kn, vn, st, wt, vhat, stats, total;
};

static MainLds main_lds(int G, const Shape& s, bool lut, bool cg) {
  MainLds L{};
  const int NB = s.d / s.k;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (off + bytes + 15) & ~(size_t)15;
    return o;
  };
  L.lut = take(lut ? (size_t)G * NB * s.N * 4 : 0);
  L.qt = take(lut ? 0 : (size_t)G * s.d * 4);
  L.cs = take(cg ? 0 : (size_t)s.N * s.k * 4);
  L.kidx = take((size_t)kTT * NB * 2);
  L.vidx = take((size_t)kTT * NB * 2);
  L.kn = take(kTT * 4);
  L.vn = take(kTT * 4);
  L.st = take((size_t)G * kTT * 4);
  L.wt = take((size_t)G * kTT * 4);
  L.vhat = take((size_t)kTT * s.d * 4);
  L.stats = take((size_t)3 * G * 4);
  L.total = off;
  return L;
}

// Codebooks of more than kCbLds floats (N k > 16384) are read from global
// memory (cache-resident) instead of LDS (CG).
constexpr int kCbLds = 16384;

template <int D, int K, bool LUT, bool CG>
__global__ __launch_bounds__(kAT) void attn_main_kernel(
    const uint8_t* __restrict__ kp, const uint16_t* __restrict__ kn,
    const uint8_t* __restrict__ vp, const uint16_t* __restrict__ vn, int G, int64_t T,
    int64_t T_stride, int N, int W, int P, int64_t chunk, int n_split,
    const float* __restrict__ C, float scale, const float* __restrict__ qrot,
    const float* __restrict__ lutg, float* __restrict__ ml, float* __restrict__ accws,
    MainLds L) {
  constexpr int NB = D / K;
  extern __shared__ __align__(16) unsigned char smem[];
  float* lut_s = reinterpret_cast<float*>(smem + L.lut);
  float* qt_s = reinterpret_cast<float*>(smem + L.qt);
  float* cs = reinterpret_cast<float*>(smem + L.cs);
  uint16_t* kidx = reinterpret_cast<uint16_t*>(smem + L.kidx);
  uint16_t* vidx = reinterpret_cast<uint16_t*>(smem + L.vidx);
  float* kn_s = reinterpret_cast<float*>(smem + L.kn);
  float* vn_s = reinterpret_cast<float*>(smem + L.vn);
  float* s_t = reinterpret_cast<float*>(smem + L.st);
  float* w_t = reinterpret_cast<float*>(smem + L.wt);
  float* vhat = reinterpret_cast<float*>(smem + L.vhat);
  float* st_m = reinterpret_cast<float*>(smem + L.stats);
  float* st_l = st_m + G;
  float* st_a = st_l + G;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t g = blockIdx.y;
  const int sidx = blockIdx.x;
  const int64_t t0 = (int64_t)sidx * chunk;
  const int64_t t1 = (t0 + chunk < T) ? t0 + chunk : T;

  if (LUT) {
    const int tot = G * NB * N;
    for (int i = tid; i < tot; i += kAT) lut_s[i] = lutg[g * tot + i];
  } else {
    for (int i = tid; i < G * D; i += kAT) qt_s[i] = qrot[g * G * D + i];
  }
  if (!CG)
    for (int i = tid; i < N * K; i += kAT) cs[i] = C[i];
  const float* cb = CG ? C : cs;
  if (tid < G) {
    st_m[tid] = -INFINITY;
    st_l[tid] = 0.0f;
    st_a[tid] = 1.0f;
  }
  constexpr int kMaxOwn = 16 * D / kAT;  // G <= 16
  float acc[kMaxOwn];
#pragma unroll
  for (int i = 0; i < kMaxOwn; ++i) acc[i] = 0.0f;
  const int GD = G * D;
  __syncthreads();

  const uint8_t* kpg = kp + g * T_stride * (int64_t)P;
  const uint8_t* vpg = vp + g * T_stride * (int64_t)P;
  const uint16_t* kng = kn + g * T_stride;
  const uint16_t* vng = vn + g * T_stride;

  for (int64_t t = t0; t < t1; t += kTT) {
    const int nt = (int)((t1 - t) < kTT ? (t1 - t) : kTT);
    // 1. indices and norms of the tile
    for (int e = tid; e < kTT * NB; e += kAT) {
      const int tt = e / NB, m = e % NB;
      uint16_t ki = 0, vi = 0;
      if (tt < nt) {
        ki = (uint16_t)extract_index(kpg + (t + tt) * P, m, W);
        vi = (uint16_t)extract_index(vpg + (t + tt) * P, m, W);
      }
      kidx[e] = ki;
      vidx[e] = vi;
    }
    if (tid < kTT) {
      kn_s[tid] = tid < nt ? half_bits_to_float(kng[t + tid]) : 0.0f;
      vn_s[tid] = tid < nt ? half_bits_to_float(vng[t + tid]) : 0.0f;
    }
    __syncthreads();
    // 2. scores
    for (int e = tid; e < G * kTT; e += kAT) {
      const int h = e / kTT, tt = e % kTT;
      float s = -INFINITY;
      if (tt < nt) {
        float a = 0.0f;
        if (LUT) {
#pragma unroll
          for (int m = 0; m < NB; ++m) a += lut_s[(h * NB + m) * N + kidx[tt * NB + m]];
        } else {
#pragma unroll
          for (int m = 0; m < NB; ++m) {
            const float* c = cb + kidx[tt * NB + m] * K;
            const float* qq = qt_s + h * D + m * K;
#pragma unroll
            for (int r = 0; r < K; ++r) a = fmaf(qq[r], c[r], a);
          }
        }
        s = a * kn_s[tt] * scale;
      }
      s_t[e] = s;
    }
    __syncthreads();
    // 3. online softmax statistics, one wavefront per head (lane = token)
    for (int h = wave; h < G; h += kAT / 64) {
      const float s = s_t[h * kTT + lane];
      const float M = wave_max(s);
      const float m_old = st_m[h];
      const float m_new = fmaxf(m_old, M);
      float p, alpha;
      if (m_new == -INFINITY) {
        p = 0.0f;
        alpha = 1.0f;
      } else {
        p = __expf(s - m_new);
        alpha = __expf(m_old - m_new);
      }
      const float lsum = wave_sum(p);
      w_t[h * kTT + lane] = p * vn_s[lane];
      if (lane == 0) {
        st_m[h] = m_new;
        st_l[h] = st_l[h] * alpha + lsum;
        st_a[h] = alpha;
      }
    }
    // 4. decode the value tile (rotated space)
    for (int e = tid; e < kTT * D; e += kAT) {
      const int tt = e / D, j = e % D;
      vhat[e] = cb[vidx[tt * NB + j / K] * K + (j % K)];
    }
    __syncthreads();
    // 5. accumulate sum_t w_t c_(t) per owned (head, coordinate)
#pragma unroll
    for (int i = 0; i < kMaxOwn; ++i) {
      const int o = tid + i * kAT;
      if (o < GD) {
        const int h = o / D, j = o % D;
        float a = acc[i] * st_a[h];
        for (int tt = 0; tt < nt; ++tt) a = fmaf(w_t[h * kTT + tt], vhat[tt * D + j], a);
        acc[i] = a;
      }
    }
    __syncthreads();
  }
  const int64_t base = (g * n_split + sidx) * G;
#pragma unroll
  for (int i = 0; i < kMaxOwn; ++i) {
    const int o = tid + i * kAT;
    if (o < GD) accws[base * D + o] = acc[i];
  }
  if (tid < G) {
    ml[(base + tid) * 2 + 0] = st_m[tid];
    ml[(base + tid) * 2 + 1] = st_l[tid];
  }
}

template <int D>
__global__ __launch_bounds__(kAT) void attn_merge_kernel(const float* __restrict__ ml,
                                                         const float* __restrict__ accws,
                                                         int n_split, int G,
                                                         const float* __restrict__ R,
                                                         float* __restrict__ out) {
  __shared__ float ar[16 * D];
  const int64_t g = blockIdx.x;
  for (int e = threadIdx.x; e < G * D; e += kAT) {
    const int h = e / D, i = e % D;
    float M = -INFINITY;
    for (int s = 0; s < n_split; ++s) M = fmaxf(M, ml[((g * n_split + s) * G + h) * 2]);
    float a = 0.0f, l = 0.0f;
    if (M != -INFINITY) {
      for (int s = 0; s < n_split; ++s) {
        const int64_t b = (g * n_split + s) * G + h;
        const float ms = ml[b * 2];
        const float f = (ms == -INFINITY) ? 0.0f : __expf(ms - M);
        l = fmaf(ml[b * 2 + 1], f, l);
        a = fmaf(accws[b * D + i], f, a);
      }
    }
    ar[e] = (l > 0.0f) ? a / l : 0.0f;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * D; e += kAT) {  // o = Pi^T a
    const int h = e / D, j = e % D;
    float s = 0.0f;
    for (int i = 0; i < D; ++i) s = fmaf(R[i * D + j], ar[h * D + i], s);
    out[g * G * D + e] = s;
  }
}

template <int D, int K>
static int launch_attn_t(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                         const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int G,
                         int64_t T, int64_t T_stride, const Shape& s, const float* R,
                         const float* C, float scale, float* out, void* ws, hipStream_t st) {
  const AttnPlan p = make_plan(n_groups, G, T, s);
  unsigned char* wsb = static_cast<unsigned char*>(ws);
  float* qrot = reinterpret_cast<float*>(wsb + p.off_qrot);
  float* lutg = reinterpret_cast<float*>(wsb + p.off_lut);
  float* ml = reinterpret_cast<float*>(wsb + p.off_ml);
  float* accws = reinterpret_cast<float*>(wsb + p.off_acc);
  if (n_groups > 2147483647LL) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL((attn_prep_kernel<D, K>), dim3((unsigned)n_groups), dim3(kAT), 0, st, q,
                     q_dtype, G, R, C, s.N, p.lut, qrot, lutg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  const bool cg = s.N * K > kCbLds;
  const MainLds L = main_lds(G, s, p.lut, cg);
  if (L.total > kLdsMax) return (int)hipErrorInvalidValue;
  dim3 grid((unsigned)p.n_split, (unsigned)n_groups);
  auto launch = [&](auto kern) -> hipError_t {
    hipError_t r = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)L.total);
    if (r != hipSuccess) return r;
    hipLaunchKernelGGL(kern, grid, dim3(kAT), L.total, st, kp, kn, vp, vn, G, T, T_stride, s.N,
                       s.w, s.P, p.chunk, p.n_split, C, scale, qrot, lutg, ml, accws, L);
    return hipSuccess;
  };
  if (p.lut) e = cg ? launch(attn_main_kernel<D, K, true, true>) : launch(attn_main_kernel<D, K, true, false>);
  else e = cg ? launch(attn_main_kernel<D, K, false, true>) : launch(attn_main_kernel<D, K, false, false>);
  if (e != hipSuccess) return (int)e;
  e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  hipLaunchKernelGGL((attn_merge_kernel<D>), dim3((unsigned)n_groups), dim3(kAT), 0, st, ml,
                     accws, p.n_split, G, R, out);
  return (int)hipGetLastError();
}

int launch_attn(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int G, int64_t T,
                int64_t T_stride, Shape s, const float* R, const float* C, float scale,
                float* out, void* ws, size_t ws_bytes, void* stream) {
  (void)ws_bytes;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // matrix-core kernel for the sub-one-bit shapes; its payload loads need
  // 4-byte (P = 4) or 2-byte (P = 6) aligned payload pointers
  const uintptr_t align = (s.w == 4) ? 3u : 1u;
  if (attn_w4_applies(G, s) && T < (1LL << 30) &&
      ((reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn)) & 1u) == 0)
    return launch_attn_w4(q, q_dtype, kp, kn, vp, vn, n_groups, T, T_stride, R, C, scale, out, ws,
                          st);
  if (attn_fast_applies(G, s) && T < (1LL << 30) &&  // 32-bit token indices
      ((reinterpret_cast<uintptr_t>(kp) | reinterpret_cast<uintptr_t>(vp)) & align) == 0 &&
      ((reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn)) & 1u) == 0)
    return launch_attn_fast(q, q_dtype, kp, kn, vp, vn, n_groups, T, T_stride, s, R, C, scale, out,
                            ws, st);
  // matrix-core kernel for k = 4 (and k = 2, w = 4 or 6, read as pairs of
  // blocks); payload quarters are read as dwords or 16-bit halves
  if (attn_k4_applies(G, s) && T < (1LL << 30) &&
      ((reinterpret_cast<uintptr_t>(kp) | reinterpret_cast<uintptr_t>(vp)) & 3u) == 0 &&
      ((reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn)) & 1u) == 0)
    return launch_attn_k4(q, q_dtype, kp, kn, vp, vn, n_groups, G, T, T_stride, s, R, C, scale,
                          out, ws, st);
#define FIBQ_ATTN_CASE(DD, KK)                                                                 \
  if (s.d == DD && s.k == KK)                                                               \
    return launch_attn_t<DD, KK>(q, q_dtype, kp, kn, vp, vn, n_groups, G, T, T_stride, s, R, C, \
                                 scale, out, ws, st);
  FIBQ_ATTN_CASE(64, 1) FIBQ_ATTN_CASE(64, 2) FIBQ_ATTN_CASE(64, 4) FIBQ_ATTN_CASE(64, 8)
  FIBQ_ATTN_CASE(64, 16) FIBQ_ATTN_CASE(128, 1) FIBQ_ATTN_CASE(128, 2) FIBQ_ATTN_CASE(128, 4)
  FIBQ_ATTN_CASE(128, 8) FIBQ_ATTN_CASE(128, 16) FIBQ_ATTN_CASE(64, 32) FIBQ_ATTN_CASE(64, 64)
#undef FIBQ_ATTN_CASE
  return (int)hipErrorInvalidValue;
}

}  // namespace dev
}  // namespace fibq
