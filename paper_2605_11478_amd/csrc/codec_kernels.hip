// Encoder and random-access decoder kernels (Sec. 3.1, Eq. encode; decoder).
//
// Encoder, one thread per vector, persistent grid over 256-vector tiles:
//   - the row is read in its own dtype and held exactly (fp32 registers);
//   - nu^2 = sum x^2 in float64 (exact products), nu = sqrt, the header is
//     rounded once from float64 to binary16 (round-to-nearest-even);
//   - y = Pi x / nu in float64 (Pi staged in LDS, read by broadcast);
//   - nearest codeword per block: a float32 screen in the expanded form
//     ||c||^2 - 2 <y, c> (codebook in LDS) keeps the best two values; when
//     they are closer than a bound on the float32 rounding error, the block
//     is re-scored over all N codewords in float64 in the direct form
//     ||y - c||^2, so the chosen index is the float64 argmin (lowest index on
//     ties) in every case;
//   - the d/k indices are bit-packed into P bytes, staged in LDS and stored
//     with coalesced dword writes; the fp16 header is a coalesced u16 store.
// Decoder, d / 16 threads per output vector: unpack, gather codewords from
// LDS, x_hat = nu Pi^T y_hat in float32 (Pi in LDS), 16 consecutive outputs
// per thread stored as float4 (coalesced rows).
#include <hip/hip_runtime.h>
#include <atomic>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {

constexpr int kEncThreads = 256;

template <int D>
struct EncPi {  // rotation element type held in LDS
  using T = typename std::conditional<(D <= 64), double, float>::type;
};

// Codebooks of more than kCbLds floats (N k > 16384: up to 256 KB) are read
// from global memory, where they stay cache-resident, instead of LDS (CG).
constexpr int kCbLds = 16384;

// A row of the input for the one-thread-per-vector encoders, either held in
// registers or re-read from cache in 8-element pieces (16-byte loads when the
// rows are 16-byte aligned).  Either way get8 returns the exact values, so
// the float64 sums below take the same terms in the same order.  Measured:
// holding pays at d = 64 with k < 8 (many blocks, each re-read would cost a
// row), streaming at k >= 8 and at d = 128 (128 held registers spill).
template <int D, int K>
constexpr bool hold_row() { return D <= 64 && K < 8; }

template <typename IN, int D, bool HOLD>
struct RowX {
  static constexpr bool kHold = HOLD;
  const IN* p;
  bool al16;
  float xf[kHold ? D : 1];
  __device__ __forceinline__ RowX(const IN* row, bool aligned) : p(row), al16(aligned) {
    if constexpr (kHold) {
#pragma unroll
      for (int j = 0; j < D; ++j) xf[j] = to_float(row[j]);
    }
  }
  __device__ __forceinline__ void get8(int j0, float c[8]) const {
    if constexpr (kHold) {
#pragma unroll
      for (int e = 0; e < 8; ++e) c[e] = xf[j0 + e];
    } else if constexpr (sizeof(IN) == 2) {
      if (al16) {
        const uint4 w = *reinterpret_cast<const uint4*>(p + j0);
        const IN* h = reinterpret_cast<const IN*>(&w);
#pragma unroll
        for (int e = 0; e < 8; ++e) c[e] = to_float(h[e]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) c[e] = to_float(p[j0 + e]);
      }
    } else {
      if (al16) {
        const float4 a = *reinterpret_cast<const float4*>(p + j0);
        const float4 b = *reinterpret_cast<const float4*>(p + j0 + 4);
        c[0] = a.x; c[1] = a.y; c[2] = a.z; c[3] = a.w;
        c[4] = b.x; c[5] = b.y; c[6] = b.z; c[7] = b.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) c[e] = to_float(p[j0 + e]);
      }
    }
  }
};

// y rows m K .. m K + K - 1 of Pi x (float64, each a sum over j in order).
template <typename IN, int D, int K, typename PT, bool HOLD>
__device__ __forceinline__ void rotate_block(const RowX<IN, D, HOLD>& xr, const PT* Rs, int m,
                                             double s[K]) {
#pragma unroll
  for (int r = 0; r < K; ++r) s[r] = 0.0;
  auto piece = [&](int j0) {
    float c[8];
    xr.get8(j0, c);
#pragma unroll
    for (int r = 0; r < K; ++r) {
      const PT* Rrow = Rs + (m * K + r) * D + j0;
#pragma unroll
      for (int e = 0; e < 8; ++e) s[r] = fma((double)Rrow[e], (double)c[e], s[r]);
    }
  };
  if constexpr (HOLD) {  // static indices into the held row
#pragma unroll
    for (int j0 = 0; j0 < D; j0 += 8) piece(j0);
  } else {  // a rolled loop keeps the Pi loads from being hoisted into registers
#pragma unroll 1
    for (int j0 = 0; j0 < D; j0 += 8) piece(j0);
  }
}

template <typename IN, int D, bool HOLD>
__device__ __forceinline__ double row_norm2(const RowX<IN, D, HOLD>& xr) {
  double nu2 = 0.0;
  auto piece = [&](int j0) {
    float c[8];
    xr.get8(j0, c);
#pragma unroll
    for (int e = 0; e < 8; ++e) nu2 = fma((double)c[e], (double)c[e], nu2);
  };
  if constexpr (HOLD) {
#pragma unroll
    for (int j0 = 0; j0 < D; j0 += 8) piece(j0);
  } else {
#pragma unroll 1
    for (int j0 = 0; j0 < D; j0 += 8) piece(j0);
  }
  return nu2;
}

// Radius-first search (App. F, Stage 1): the codebook holds L shells of N / L
// codewords, shell-major; a block takes the shell whose radius r_l is nearest
// to its norm rho (lower shell on ties) and is searched against that shell
// alone.  The L - 1 midpoints (r_l + r_{l+1}) / 2 travel by value.
constexpr int kMaxShells = 256;
struct ShellMids {
  double m[kMaxShells - 1];
};

template <typename IN, int D, int K, bool CG, bool SH>
__device__ __forceinline__ void encode_body(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms, int L, const ShellMids* __restrict__ sm) {
  using PT = typename EncPi<D>::T;
  constexpr int NB = D / K;
  extern __shared__ __align__(16) unsigned char smem[];
  PT* Rs = reinterpret_cast<PT*>(smem);
  double* mids = reinterpret_cast<double*>(smem + sizeof(PT) * D * D);  // SH: L - 1 midpoints
  float* Cs = reinterpret_cast<float*>(smem + sizeof(PT) * D * D + (SH ? 8 * kMaxShells : 0));
  float* cc = Cs + (CG ? 0 : N * K);
  const float* Cb = CG ? C : Cs;  // codebook rows (wave-uniform reads in the screen)
  float* red = cc + N;                                   // 1 float: max ||c||^2
  uint8_t* stage = reinterpret_cast<uint8_t*>(red + 4);  // kEncThreads * P bytes

  const int tid = threadIdx.x;
  for (int i = tid; i < D * D; i += kEncThreads) Rs[i] = (PT)R[i];
  if (SH)
    for (int i = tid; i < L - 1; i += kEncThreads) mids[i] = sm->m[i];
  if (!CG)
    for (int i = tid; i < N * K; i += kEncThreads) Cs[i] = C[i];
  if (tid == 0) red[0] = 1.0f;
  __syncthreads();
  float my_max = 0.0f;
  for (int j = tid; j < N; j += kEncThreads) {
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < K; ++r) s = fmaf(Cb[j * K + r], Cb[j * K + r], s);
    cc[j] = s;
    my_max = fmaxf(my_max, s);
  }
  my_max = wave_max(my_max);
  if ((tid & 63) == 0) atomicMax(reinterpret_cast<int*>(red), __float_as_int(my_max));
  __syncthreads();
  // Bound on the float32 screen's error for the gap between two candidates
  // (|y| <= 1, |c|^2 <= S): 2 (3K + 8) S 2^-24.
  const float eps = (6.0f * K + 16.0f) * fmaxf(1.0f, red[0]) * 5.9604645e-8f;

  const bool aligned = reinterpret_cast<uintptr_t>(x) % 16 == 0 && (stride * sizeof(IN)) % 16 == 0;
  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t v = tile * kEncThreads + tid;
    const bool live = v < n_vec;
    uint64_t acc = 0;  // bit accumulator, flushed to the LDS stage per 32 bits
    int nbits = 0, wi = 0;
    if (live) {
      const RowX<IN, D, hold_row<D, K>()> xr(x + v * stride, aligned);
      const double nu = sqrt(row_norm2(xr));
      const double inv = nu > 0.0 ? 1.0 / nu : 0.0;
      norms[v] = nu > 0.0 ? f64_to_f16_bits(nu) : (uint16_t)0;

      for (int m = 0; m < NB; ++m) {
        double yb[K];
        float yf[K];
        rotate_block<IN, D, K, PT, hold_row<D, K>()>(xr, Rs, m, yb);
#pragma unroll
        for (int r = 0; r < K; ++r) {
          yb[r] *= inv;
          yf[r] = (float)yb[r];
        }
        int j0 = 0, nc = N;  // candidate range [j0, j0 + nc)
        if (SH) {
          double rho2 = 0.0;
#pragma unroll
          for (int r = 0; r < K; ++r) rho2 = fma(yb[r], yb[r], rho2);
          const double rho = sqrt(rho2);
          int l = 0;  // number of midpoints below rho (L is a power of two)
          for (int step = L >> 1; step >= 1; step >>= 1)
            if (rho > mids[l + step - 1]) l += step;
          nc = N / L;
          j0 = l * nc;
        }
        float b1 = INFINITY, b2 = INFINITY;
        int i1 = j0;
#pragma unroll 4
        for (int j = j0; j < j0 + nc; ++j) {
          float dot = 0.0f;
#pragma unroll
          for (int r = 0; r < K; ++r) dot = fmaf(yf[r], Cb[j * K + r], dot);
          const float dp = fmaf(-2.0f, dot, cc[j]);
          const bool lt = dp < b1;
          b2 = lt ? b1 : fminf(b2, dp);
          i1 = lt ? j : i1;
          b1 = lt ? dp : b1;
        }
        if (b2 - b1 <= eps) {  // near tie: exact float64 re-score (rare)
          double bd = INFINITY;
          int bi = j0;
          for (int j = j0; j < j0 + nc; ++j) {
            double s = 0.0;
#pragma unroll
            for (int r = 0; r < K; ++r) {
              const double t = yb[r] - (double)Cb[j * K + r];
              s = fma(t, t, s);
            }
            if (s < bd) {
              bd = s;
              bi = j;
            }
          }
          i1 = bi;
        }
        if (!(nu > 0.0)) i1 = 0;
        acc |= (uint64_t)(uint32_t)i1 << nbits;
        nbits += W;
        if (nbits >= 32) {
          const uint32_t wv = (uint32_t)acc;
#pragma unroll
          for (int b = 0; b < 4; ++b)
            if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
          ++wi;
          acc >>= 32;
          nbits -= 32;
        }
      }
      if (nbits > 0) {
        const uint32_t wv = (uint32_t)acc;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
      }
    }
    __syncthreads();
    // coalesced copy of the tile's payload: the tile start tile*256*P is a
    // multiple of 4 bytes, so whole dwords are aligned.
    const int64_t nv = (n_vec - tile * kEncThreads) < kEncThreads ? (n_vec - tile * kEncThreads)
                                                                  : kEncThreads;
    const int64_t nbytes = nv * P;
    uint8_t* dst = payload + tile * kEncThreads * (int64_t)P;
    const int64_t ndw = nbytes >> 2;
    for (int64_t i = tid; i < ndw; i += kEncThreads) {
      uint32_t wv = (uint32_t)stage[4 * i] | ((uint32_t)stage[4 * i + 1] << 8) |
                    ((uint32_t)stage[4 * i + 2] << 16) | ((uint32_t)stage[4 * i + 3] << 24);
      reinterpret_cast<uint32_t*>(dst)[i] = wv;
    }
    for (int64_t i = (ndw << 2) + tid; i < nbytes; i += kEncThreads) dst[i] = stage[i];
    __syncthreads();
  }
}

template <typename IN, int D, int K, bool CG>
__global__ __launch_bounds__(kEncThreads) void encode_kernel(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms) {
  encode_body<IN, D, K, CG, false>(x, n_vec, stride, R, C, N, W, P, payload, norms, 1, nullptr);
}
template <typename IN, int D, int K, bool CG>
__global__ __launch_bounds__(kEncThreads) void encode_shells_kernel(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms, int L, ShellMids sm) {
  encode_body<IN, D, K, CG, true>(x, n_vec, stride, R, C, N, W, P, payload, norms, L, &sm);
}

// Exhaustive encoder for codebooks read from global memory at d = 64 and
// k >= 32 (one or two blocks per vector; at k = 8, 16 the general kernel's
// scalar-load scan measured faster).  The general kernel's wavefronts each
// stream the whole codebook once per block through scalar loads; here a
// workgroup stages the codebook in 32 KB chunks in LDS with coalesced loads
// and its 256 vectors scan every chunk, each thread keeping the best two
// float32 screen values of each of its blocks.  The rotation, the screen
// arithmetic, its error bound and the float64 near-tie re-score (over all N
// codewords, from global memory) are the general kernel's.
template <typename IN, int D, int K>
__global__ __launch_bounds__(kEncThreads) __attribute__((amdgpu_waves_per_eu(2))) void encode_chunked_kernel(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms) {
  using PT = typename EncPi<D>::T;
  constexpr int NB = D / K;
  constexpr int CH = 8192 / K;  // codewords per chunk (32 KB of float32)
  extern __shared__ __align__(16) unsigned char smem[];
  PT* Rs = reinterpret_cast<PT*>(smem);
  float* Cc = reinterpret_cast<float*>(smem + sizeof(PT) * D * D);  // CH * K
  float* ccs = Cc + CH * K;                                           // CH norms ||c||^2
  float* red = ccs + CH;                                              // max ||c||^2
  uint8_t* stage = reinterpret_cast<uint8_t*>(red + 4);              // kEncThreads * P

  const int tid = threadIdx.x;
  for (int i = tid; i < D * D; i += kEncThreads) Rs[i] = (PT)R[i];
  if (tid == 0) red[0] = 1.0f;
  __syncthreads();
  float my_max = 0.0f;
  for (int j = tid; j < N; j += kEncThreads) {
    float sq = 0.0f;
#pragma unroll
    for (int r = 0; r < K; ++r) sq = fmaf(C[j * K + r], C[j * K + r], sq);
    my_max = fmaxf(my_max, sq);
  }
  my_max = wave_max(my_max);
  if ((tid & 63) == 0) atomicMax(reinterpret_cast<int*>(red), __float_as_int(my_max));
  __syncthreads();
  const float eps = (6.0f * K + 16.0f) * fmaxf(1.0f, red[0]) * 5.9604645e-8f;

  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t v = tile * kEncThreads + tid;
    const bool live = v < n_vec;
    float yf[D];
    double nu = 0.0;
    if (live) {
      const IN* row = x + v * stride;
      float xf[D];
#pragma unroll
      for (int j = 0; j < D; ++j) xf[j] = to_float(row[j]);
      double nu2 = 0.0;
#pragma unroll
      for (int j = 0; j < D; ++j) nu2 = fma((double)xf[j], (double)xf[j], nu2);
      nu = sqrt(nu2);
      const double inv = nu > 0.0 ? 1.0 / nu : 0.0;
      norms[v] = nu > 0.0 ? f64_to_f16_bits(nu) : (uint16_t)0;
#pragma unroll
      for (int i = 0; i < D; ++i) {
        const PT* Rrow = Rs + i * D;
        double sacc = 0.0;
#pragma unroll
        for (int j = 0; j < D; ++j) sacc = fma((double)Rrow[j], (double)xf[j], sacc);
        yf[i] = (float)(sacc * inv);
      }
    } else {
#pragma unroll
      for (int i = 0; i < D; ++i) yf[i] = 0.0f;
    }
    float b1[NB], b2[NB];
    int i1[NB];
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      b1[m] = INFINITY;
      b2[m] = INFINITY;
      i1[m] = 0;
    }
    for (int c0 = 0; c0 < N; c0 += CH) {  // uniform trip count: every thread reaches the barriers
      __syncthreads();
      const float4* src = reinterpret_cast<const float4*>(C + (size_t)c0 * K);
      for (int i = tid; i < CH * K / 4; i += kEncThreads) reinterpret_cast<float4*>(Cc)[i] = src[i];
      for (int j = tid; j < CH; j += kEncThreads) {
        float sq = 0.0f;
#pragma unroll
        for (int r = 0; r < K; ++r) sq = fmaf(C[(size_t)(c0 + j) * K + r], C[(size_t)(c0 + j) * K + r], sq);
        ccs[j] = sq;
      }
      __syncthreads();
#pragma unroll
      for (int m = 0; m < NB; ++m) {
#pragma unroll 2
        for (int j = 0; j < CH; ++j) {
          float dot = 0.0f;
#pragma unroll
          for (int r = 0; r < K; ++r) dot = fmaf(yf[m * K + r], Cc[j * K + r], dot);
          const float dp = fmaf(-2.0f, dot, ccs[j]);
          const bool lt = dp < b1[m];
          b2[m] = lt ? b1[m] : fminf(b2[m], dp);
          i1[m] = lt ? c0 + j : i1[m];
          b1[m] = lt ? dp : b1[m];
        }
      }
    }
    uint64_t acc = 0;
    int nbits = 0, wi = 0;
    if (live) {
#pragma unroll
      for (int m = 0; m < NB; ++m) {
        int im = i1[m];
        if (b2[m] - b1[m] <= eps) {  // near tie: float64 re-score over all N (rare)
          const IN* row = x + v * stride;
          const double inv = nu > 0.0 ? 1.0 / nu : 0.0;
          double yb[K];
#pragma unroll
          for (int r = 0; r < K; ++r) {
            const PT* Rrow = Rs + (m * K + r) * D;
            double sacc = 0.0;
            for (int j = 0; j < D; ++j) sacc = fma((double)Rrow[j], (double)to_float(row[j]), sacc);
            yb[r] = sacc * inv;
          }
          double bd = INFINITY;
          int bi = 0;
          for (int j = 0; j < N; ++j) {
            double sd = 0.0;
#pragma unroll
            for (int r = 0; r < K; ++r) {
              const double t = yb[r] - (double)C[(size_t)j * K + r];
              sd = fma(t, t, sd);
            }
            if (sd < bd) {
              bd = sd;
              bi = j;
            }
          }
          im = bi;
        }
        if (!(nu > 0.0)) im = 0;
        acc |= (uint64_t)(uint32_t)im << nbits;
        nbits += W;
        if (nbits >= 32) {
          const uint32_t wv = (uint32_t)acc;
#pragma unroll
          for (int b = 0; b < 4; ++b)
            if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
          ++wi;
          acc >>= 32;
          nbits -= 32;
        }
      }
      if (nbits > 0) {
        const uint32_t wv = (uint32_t)acc;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
      }
    }
    __syncthreads();
    const int64_t nv = (n_vec - tile * kEncThreads) < kEncThreads ? (n_vec - tile * kEncThreads)
                                                                  : kEncThreads;
    const int64_t nbytes = nv * P;
    uint8_t* dst = payload + tile * kEncThreads * (int64_t)P;
    const int64_t ndw = nbytes >> 2;
    for (int64_t i = tid; i < ndw; i += kEncThreads) {
      uint32_t wv = (uint32_t)stage[4 * i] | ((uint32_t)stage[4 * i + 1] << 8) |
                    ((uint32_t)stage[4 * i + 2] << 16) | ((uint32_t)stage[4 * i + 3] << 24);
      reinterpret_cast<uint32_t*>(dst)[i] = wv;
    }
    for (int64_t i = (ndw << 2) + tid; i < nbytes; i += kEncThreads) dst[i] = stage[i];
  }
}

// List decoding inside the radius-chosen shell (App. F, Stages 1 + 2): the
// block's shell as in the radius-first search, then its NP parents ranked by
// <y, mu_p> in float64 (first parent on ties), and the children of the best T
// parents searched: float32 screen of ||c||^2 - 2 <y, c> with the general
// kernel's error bound, float64 direct-form re-score of the same lists on a
// near tie; the lowest index wins a tie.  Tables and codebook are read from
// global memory (per-lane gathers); Pi and the radius midpoints from LDS.
constexpr int kMaxList = 8;  // T <= 8

template <typename IN, int D, int K>
__global__ __launch_bounds__(kEncThreads) void encode_list_kernel(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms, int L, ShellMids sm, int NP, int T,
    const double* __restrict__ mu, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ members) {
  using PT = typename EncPi<D>::T;
  constexpr int NB = D / K;
  extern __shared__ __align__(16) unsigned char smem[];
  PT* Rs = reinterpret_cast<PT*>(smem);
  double* mids = reinterpret_cast<double*>(smem + sizeof(PT) * D * D);
  float* red = reinterpret_cast<float*>(mids + kMaxShells);
  uint8_t* stage = reinterpret_cast<uint8_t*>(red + 4);  // kEncThreads * P bytes
  const int tid = threadIdx.x;
  const int Ma = N / L;
  for (int i = tid; i < D * D; i += kEncThreads) Rs[i] = (PT)R[i];
  for (int i = tid; i < L - 1; i += kEncThreads) mids[i] = sm.m[i];
  if (tid == 0) red[0] = 1.0f;
  __syncthreads();
  float my_max = 0.0f;
  for (int j = tid; j < N; j += kEncThreads) {
    float sq = 0.0f;
#pragma unroll
    for (int r = 0; r < K; ++r) sq = fmaf(C[(size_t)j * K + r], C[(size_t)j * K + r], sq);
    my_max = fmaxf(my_max, sq);
  }
  my_max = wave_max(my_max);
  if ((tid & 63) == 0) atomicMax(reinterpret_cast<int*>(red), __float_as_int(my_max));
  __syncthreads();
  const float eps = (6.0f * K + 16.0f) * fmaxf(1.0f, red[0]) * 5.9604645e-8f;

  const bool aligned = reinterpret_cast<uintptr_t>(x) % 16 == 0 && (stride * sizeof(IN)) % 16 == 0;
  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t v = tile * kEncThreads + tid;
    const bool live = v < n_vec;
    uint64_t acc = 0;
    int nbits = 0, wi = 0;
    if (live) {
      const RowX<IN, D, hold_row<D, K>()> xr(x + v * stride, aligned);
      const double nu = sqrt(row_norm2(xr));
      const double inv = nu > 0.0 ? 1.0 / nu : 0.0;
      norms[v] = nu > 0.0 ? f64_to_f16_bits(nu) : (uint16_t)0;
      for (int m = 0; m < NB; ++m) {
        double yb[K];
        float yf[K];
        rotate_block<IN, D, K, PT, hold_row<D, K>()>(xr, Rs, m, yb);
#pragma unroll
        for (int r = 0; r < K; ++r) {
          yb[r] *= inv;
          yf[r] = (float)yb[r];
        }
        double rho2 = 0.0;
#pragma unroll
        for (int r = 0; r < K; ++r) rho2 = fma(yb[r], yb[r], rho2);
        const double rho = sqrt(rho2);
        int l = 0;
        for (int step = L >> 1; step >= 1; step >>= 1)
          if (rho > mids[l + step - 1]) l += step;
        // the T best parents of shell l (strictly better displaces: first on ties)
        double ts[kMaxList];
        int tp[kMaxList];
        for (int t = 0; t < T; ++t) { ts[t] = -INFINITY; tp[t] = 0; }
        const double* mul = mu + (size_t)l * NP * K;
        for (int p = 0; p < NP; ++p) {
          double sc = 0.0;
#pragma unroll
          for (int r = 0; r < K; ++r) sc = fma(yb[r], mul[(size_t)p * K + r], sc);
          if (sc > ts[T - 1]) {
            int t = T - 1;
            while (t > 0 && sc > ts[t - 1]) {
              ts[t] = ts[t - 1];
              tp[t] = tp[t - 1];
              --t;
            }
            ts[t] = sc;
            tp[t] = p;
          }
        }
        const int32_t* offl = offsets + (size_t)l * (NP + 1);
        const int32_t* meml = members + (size_t)l * Ma;
        float b1 = INFINITY, b2 = INFINITY;
        int i1 = N;
        // table entries are clamped into the shell, so any table stays in bounds
        auto lo_of = [&](int t) { return min(max(offl[tp[t]], 0), Ma); };
        auto hi_of = [&](int t) { return min(max(offl[tp[t] + 1], lo_of(t)), Ma); };
        auto code_of = [&](int e) { return l * Ma + min(max(meml[e], 0), Ma - 1); };
        for (int t = 0; t < T; ++t) {
          const int e1 = hi_of(t);
          for (int e = lo_of(t); e < e1; ++e) {
            const int j = code_of(e);
            const float* cj = C + (size_t)j * K;
            float dot = 0.0f, sq = 0.0f;
#pragma unroll
            for (int r = 0; r < K; ++r) {
              dot = fmaf(yf[r], cj[r], dot);
              sq = fmaf(cj[r], cj[r], sq);
            }
            const float dp = fmaf(-2.0f, dot, sq);
            if (dp < b1 || (dp == b1 && j < i1)) {
              b2 = b1;
              b1 = dp;
              i1 = j;
            } else {
              b2 = fminf(b2, dp);
            }
          }
        }
        if (b2 - b1 <= eps) {  // near tie: float64 re-score of the same lists
          double bd = INFINITY;
          int bi = N;
          for (int t = 0; t < T; ++t) {
            const int e1 = hi_of(t);
            for (int e = lo_of(t); e < e1; ++e) {
              const int j = code_of(e);
              double sd = 0.0;
#pragma unroll
              for (int r = 0; r < K; ++r) {
                const double tt = yb[r] - (double)C[(size_t)j * K + r];
                sd = fma(tt, tt, sd);
              }
              if (sd < bd || (sd == bd && j < bi)) {
                bd = sd;
                bi = j;
              }
            }
          }
          i1 = bi;
        }
        if (!(nu > 0.0) || i1 >= N) i1 = 0;
        acc |= (uint64_t)(uint32_t)i1 << nbits;
        nbits += W;
        if (nbits >= 32) {
          const uint32_t wv = (uint32_t)acc;
#pragma unroll
          for (int b = 0; b < 4; ++b)
            if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
          ++wi;
          acc >>= 32;
          nbits -= 32;
        }
      }
      if (nbits > 0) {
        const uint32_t wv = (uint32_t)acc;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if (wi * 4 + b < P) stage[tid * P + wi * 4 + b] = (uint8_t)(wv >> (8 * b));
      }
    }
    __syncthreads();
    const int64_t nv = (n_vec - tile * kEncThreads) < kEncThreads ? (n_vec - tile * kEncThreads)
                                                                  : kEncThreads;
    const int64_t nbytes = nv * P;
    uint8_t* dst = payload + tile * kEncThreads * (int64_t)P;
    const int64_t ndw = nbytes >> 2;
    for (int64_t i = tid; i < ndw; i += kEncThreads) {
      uint32_t wv = (uint32_t)stage[4 * i] | ((uint32_t)stage[4 * i + 1] << 8) |
                    ((uint32_t)stage[4 * i + 2] << 16) | ((uint32_t)stage[4 * i + 3] << 24);
      reinterpret_cast<uint32_t*>(dst)[i] = wv;
    }
    for (int64_t i = (ndw << 2) + tid; i < nbytes; i += kEncThreads) dst[i] = stage[i];
    __syncthreads();
  }
}

// D / 16 lanes per output row, each producing 16 consecutive floats, so a
// wavefront's float4 stores cover whole contiguous rows.
template <int D, int K, bool CG>
__global__ __launch_bounds__(256) void decode_kernel(const uint8_t* __restrict__ payload,
                                                     const uint16_t* __restrict__ norms,
                                                     const int64_t* __restrict__ ids,
                                                     int64_t n_vec, int64_t n_cache,
                                                     const float* __restrict__ R,
                                                     const float* __restrict__ C, int N, int W,
                                                     int P, float* __restrict__ out) {
  constexpr int NB = D / K;
  constexpr int TPV = D / 16;  // lanes per row
  extern __shared__ __align__(16) unsigned char smem[];
  float* Rs = reinterpret_cast<float*>(smem);
  float* Cs = Rs + D * D;
  const float* Cb = CG ? C : Cs;  // large codebooks: gathered from global memory
  for (int i = threadIdx.x; i < D * D; i += blockDim.x) Rs[i] = R[i];
  if (!CG)
    for (int i = threadIdx.x; i < N * K; i += blockDim.x) Cs[i] = C[i];
  __syncthreads();
  const int q = threadIdx.x % TPV;  // this lane's 16 dims: 16 q .. 16 q + 15
  for (int64_t gv = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / TPV; gv < n_vec;
       gv += (int64_t)gridDim.x * blockDim.x / TPV) {
    const int64_t t = ids ? ids[gv] : gv;
    float4* o = reinterpret_cast<float4*>(out + gv * D + 16 * q);
    if (t < 0 || t >= n_cache) {
      const float nan = __int_as_float(0x7FC00000);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = make_float4(nan, nan, nan, nan);
      continue;
    }
    const uint8_t* p = payload + t * (int64_t)P;
    float yh[D];
#pragma unroll
    for (int m = 0; m < NB; ++m) {
      const uint32_t id = extract_index(p, m, W);
#pragma unroll
      for (int r = 0; r < K; ++r) yh[m * K + r] = Cb[id * K + r];
    }
    const float h = half_bits_to_float(norms[t]);
    float acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0.0f;
    // (fully unrolled: a partly unrolled loop indexes y_hat at run time,
    // which puts the array in scratch memory)
#pragma unroll
    for (int i = 0; i < D; ++i) {  // x_hat = nu Pi^T y_hat: row i of Pi times y_hat_i
      const float4* row = reinterpret_cast<const float4*>(Rs + i * D + 16 * q);
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        const float4 r4 = row[j4];
        acc[4 * j4 + 0] = fmaf(r4.x, yh[i], acc[4 * j4 + 0]);
        acc[4 * j4 + 1] = fmaf(r4.y, yh[i], acc[4 * j4 + 1]);
        acc[4 * j4 + 2] = fmaf(r4.z, yh[i], acc[4 * j4 + 2]);
        acc[4 * j4 + 3] = fmaf(r4.w, yh[i], acc[4 * j4 + 3]);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = make_float4(h * acc[4 * j], h * acc[4 * j + 1], h * acc[4 * j + 2], h * acc[4 * j + 3]);
  }
}

// Small codebooks (d/k * N * d floats <= 64 KB): x_hat = nu Pi^T y_hat is a sum
// of d/k rows of the table T[m][j] = Pi_m^T c_j (Pi_m: the k rows of Pi of
// block m), which each workgroup builds once in LDS; a row then costs d/k
// gathers of its 16 dims per lane instead of the d x d product.
constexpr int kDecTab = 16384;  // floats

template <int D, int K>
__global__ __launch_bounds__(256) void decode_table_kernel(const uint8_t* __restrict__ payload,
                                                           const uint16_t* __restrict__ norms,
                                                           const int64_t* __restrict__ ids,
                                                           int64_t n_vec, int64_t n_cache,
                                                           const float* __restrict__ R,
                                                           const float* __restrict__ C, int N,
                                                           int W, int P, float* __restrict__ out) {
  constexpr int NB = D / K;
  constexpr int TPV = D / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  float* tab = reinterpret_cast<float*>(smem);  // [NB][N][D]
  // one (block m, column) per thread: the K entries of Pi's column are read
  // once (coalesced across the threads) and serve all N codewords
  for (int mc = threadIdx.x; mc < NB * D; mc += blockDim.x) {
    const int col = mc % D, m = mc / D;
    float rv[K];
#pragma unroll
    for (int r = 0; r < K; ++r) rv[r] = R[(m * K + r) * D + col];
    for (int j = 0; j < N; ++j) {
      float sacc = 0.0f;
#pragma unroll
      for (int r = 0; r < K; ++r) sacc = fmaf(C[j * K + r], rv[r], sacc);
      tab[(m * N + j) * D + col] = sacc;
    }
  }
  __syncthreads();
  const int q = threadIdx.x % TPV;
  for (int64_t gv = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / TPV; gv < n_vec;
       gv += (int64_t)gridDim.x * blockDim.x / TPV) {
    const int64_t t = ids ? ids[gv] : gv;
    float4* o = reinterpret_cast<float4*>(out + gv * D + 16 * q);
    if (t < 0 || t >= n_cache) {
      const float nan = __int_as_float(0x7FC00000);
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = make_float4(nan, nan, nan, nan);
      continue;
    }
    const uint8_t* p = payload + t * (int64_t)P;
    float4 acc[4] = {};
#pragma unroll 4
    for (int m = 0; m < NB; ++m) {
      const uint32_t id = extract_index(p, m, W);
      const float4* tr = reinterpret_cast<const float4*>(tab + ((size_t)m * N + id) * D + 16 * q);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 v = tr[j];
        acc[j].x += v.x;
        acc[j].y += v.y;
        acc[j].z += v.z;
        acc[j].w += v.w;
      }
    }
    const float h = half_bits_to_float(norms[t]);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = make_float4(h * acc[j].x, h * acc[j].y, h * acc[j].z, h * acc[j].w);
  }
}

// ----------------------------------------------------------------- launch ---
// Compute units of the current device.  The attribute query costs more host
// time than a small launch, so each device's count (a fixed property of the
// hardware) is read once and kept; racing first calls store the same value.
static int num_cus() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < kMaxDevices && (n = cache[dev].load(std::memory_order_relaxed)) > 0)
    return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return 256;
  if (dev >= 0 && dev < kMaxDevices) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

template <typename IN, int D, int K, bool CG>
static int launch_encode_cg(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                            const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                            int L, const ShellMids* sm, hipStream_t st) {
  using PT = typename EncPi<D>::T;
  const size_t lds = sizeof(PT) * D * D + (sm ? 8 * kMaxShells : 0) +
                     sizeof(float) * (size_t)((CG ? 0 : s.N * K) + s.N + 4) +
                     (size_t)kEncThreads * s.P;
  const void* kern = sm ? reinterpret_cast<const void*>(&encode_shells_kernel<IN, D, K, CG>)
                        : reinterpret_cast<const void*>(&encode_kernel<IN, D, K, CG>);
  hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return (int)e;
  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  const int64_t cap = (int64_t)num_cus() * 4;
  const int grid = (int)(ntiles < cap ? ntiles : cap);
  if (sm)
    hipLaunchKernelGGL((encode_shells_kernel<IN, D, K, CG>), dim3(grid), dim3(kEncThreads), lds,
                       st, static_cast<const IN*>(x), n_vec, stride, R, C, s.N, s.w, s.P, payload,
                       norms, L, *sm);
  else
    hipLaunchKernelGGL((encode_kernel<IN, D, K, CG>), dim3(grid), dim3(kEncThreads), lds, st,
                       static_cast<const IN*>(x), n_vec, stride, R, C, s.N, s.w, s.P, payload,
                       norms);
  return (int)hipGetLastError();
}

template <typename IN, int D, int K>
static int launch_encode_chunked(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                                 const float* R, const float* C, uint8_t* payload,
                                 uint16_t* norms, hipStream_t st) {
  using PT = typename EncPi<D>::T;
  constexpr int CH = 8192 / K;
  const size_t lds = sizeof(PT) * D * D + sizeof(float) * (size_t)(CH * K + CH + 4) +
                     (size_t)kEncThreads * s.P;
  auto kern = encode_chunked_kernel<IN, D, K>;
  hipError_t e = hipFuncSetAttribute((const void*)kern,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return (int)e;
  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  const int64_t cap = (int64_t)num_cus() * 2;
  const int grid = (int)(ntiles < cap ? ntiles : cap);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kEncThreads), lds, st, static_cast<const IN*>(x),
                     n_vec, stride, R, C, s.N, s.w, s.P, payload, norms);
  return (int)hipGetLastError();
}

template <typename IN, int D, int K>
static int launch_encode_t(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                           const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                           int L, const ShellMids* sm, hipStream_t st) {
  if constexpr (D == 64 && K >= 32) {  // large blocks and codebooks: chunked through LDS
    if (!sm && s.N * K > kCbLds && s.N % (8192 / K) == 0 &&
        reinterpret_cast<uintptr_t>(C) % 16 == 0)
      return launch_encode_chunked<IN, D, K>(x, n_vec, stride, s, R, C, payload, norms, st);
  }
  if (s.N * K > kCbLds)
    return launch_encode_cg<IN, D, K, true>(x, n_vec, stride, s, R, C, payload, norms, L, sm, st);
  return launch_encode_cg<IN, D, K, false>(x, n_vec, stride, s, R, C, payload, norms, L, sm, st);
}

template <typename IN>
static int dispatch_encode(const void* x, int64_t n, int64_t stride, const Shape& s,
                           const float* R, const float* C, uint8_t* p, uint16_t* nm, int L,
                           const ShellMids* sm, hipStream_t st) {
#define FIBQ_ENC_CASE(DD, KK)                                                                  \
  if (s.d == DD && s.k == KK)                                                                  \
    return launch_encode_t<IN, DD, KK>(x, n, stride, s, R, C, p, nm, L, sm, st);
  FIBQ_ENC_CASE(64, 1) FIBQ_ENC_CASE(64, 2) FIBQ_ENC_CASE(64, 4) FIBQ_ENC_CASE(64, 8)
  FIBQ_ENC_CASE(64, 16) FIBQ_ENC_CASE(128, 1) FIBQ_ENC_CASE(128, 2) FIBQ_ENC_CASE(128, 4)
  FIBQ_ENC_CASE(128, 8) FIBQ_ENC_CASE(128, 16) FIBQ_ENC_CASE(64, 32) FIBQ_ENC_CASE(64, 64)
#undef FIBQ_ENC_CASE
  return (int)hipErrorInvalidValue;
}

static int dispatch_dtype(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                          const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                          int L, const ShellMids* sm, hipStream_t st) {
  switch (dtype) {
    case FIBQ_F32:
      return dispatch_encode<float>(x, n_vec, stride, s, R, C, payload, norms, L, sm, st);
    case FIBQ_F16:
      return dispatch_encode<f16_t>(x, n_vec, stride, s, R, C, payload, norms, L, sm, st);
    case FIBQ_BF16:
      return dispatch_encode<bf16_t>(x, n_vec, stride, s, R, C, payload, norms, L, sm, st);
  }
  return (int)hipErrorInvalidValue;
}

int launch_encode(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s,
                  const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                  void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (encode_mfma_applies(dtype, s, x, stride, R, payload, norms))
    return launch_encode_mfma(x, n_vec, stride, s, R, C, payload, norms, stream, num_cus());
  if (encode_mf4_applies(dtype, s, x, stride, R, payload, norms))
    return launch_encode_mf4(x, dtype, n_vec, stride, s, R, C, payload, norms, stream, num_cus());
  if (encode_big_applies(dtype, s, x, stride, R, C, payload))
    return launch_encode_big(x, dtype, n_vec, stride, s, R, C, payload, norms, stream, num_cus());
  return dispatch_dtype(x, dtype, n_vec, stride, s, R, C, payload, norms, 1, nullptr, st);
}

int launch_encode_shells(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s, int L,
                         const double* radii, const float* R, const float* C, uint8_t* payload,
                         uint16_t* norms, void* stream) {
  if (L < 1 || L > kMaxShells) return (int)hipErrorInvalidValue;
  ShellMids sm{};
  for (int l = 0; l + 1 < L; ++l) sm.m[l] = 0.5 * (radii[l] + radii[l + 1]);
  return dispatch_dtype(x, dtype, n_vec, stride, s, R, C, payload, norms, L, &sm,
                        static_cast<hipStream_t>(stream));
}

template <typename IN, int D, int K>
static int launch_list_t(const void* x, int64_t n_vec, int64_t stride, const Shape& s, int L,
                         const ShellMids& sm, int NP, int T, const double* mu,
                         const int32_t* offsets, const int32_t* members, const float* R,
                         const float* C, uint8_t* payload, uint16_t* norms, hipStream_t st) {
  using PT = typename EncPi<D>::T;
  const size_t lds = sizeof(PT) * D * D + 8 * kMaxShells + 16 + (size_t)kEncThreads * s.P;
  auto kern = encode_list_kernel<IN, D, K>;
  hipError_t e = hipFuncSetAttribute((const void*)kern,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return (int)e;
  const int64_t ntiles = (n_vec + kEncThreads - 1) / kEncThreads;
  const int64_t cap = (int64_t)num_cus() * 4;
  const int grid = (int)(ntiles < cap ? ntiles : cap);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kEncThreads), lds, st, static_cast<const IN*>(x),
                     n_vec, stride, R, C, s.N, s.w, s.P, payload, norms, L, sm, NP, T, mu,
                     offsets, members);
  return (int)hipGetLastError();
}

template <typename IN>
static int dispatch_list(const void* x, int64_t n, int64_t stride, const Shape& s, int L,
                         const ShellMids& sm, int NP, int T, const double* mu,
                         const int32_t* off, const int32_t* mem, const float* R, const float* C,
                         uint8_t* p, uint16_t* nm, hipStream_t st) {
#define FIBQ_LIST_CASE(DD, KK)                                                                  \
  if (s.d == DD && s.k == KK)                                                                   \
    return launch_list_t<IN, DD, KK>(x, n, stride, s, L, sm, NP, T, mu, off, mem, R, C, p, nm, st);
  FIBQ_LIST_CASE(64, 4) FIBQ_LIST_CASE(64, 8) FIBQ_LIST_CASE(64, 16) FIBQ_LIST_CASE(64, 32)
  FIBQ_LIST_CASE(128, 4) FIBQ_LIST_CASE(128, 8) FIBQ_LIST_CASE(128, 16)
#undef FIBQ_LIST_CASE
  return (int)hipErrorInvalidValue;
}

int launch_encode_list(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s, int L,
                       const double* radii, int K, int T, const double* mu,
                       const int32_t* offsets, const int32_t* members, const float* R,
                       const float* C, uint8_t* payload, uint16_t* norms, void* stream) {
  if (L < 1 || L > kMaxShells || T < 1 || T > kMaxList || T > K) return (int)hipErrorInvalidValue;
  ShellMids sm{};
  for (int l = 0; l + 1 < L; ++l) sm.m[l] = 0.5 * (radii[l] + radii[l + 1]);
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (dtype) {
    case FIBQ_F32:
      return dispatch_list<float>(x, n_vec, stride, s, L, sm, K, T, mu, offsets, members, R, C,
                                  payload, norms, st);
    case FIBQ_F16:
      return dispatch_list<f16_t>(x, n_vec, stride, s, L, sm, K, T, mu, offsets, members, R, C,
                                  payload, norms, st);
    case FIBQ_BF16:
      return dispatch_list<bf16_t>(x, n_vec, stride, s, L, sm, K, T, mu, offsets, members, R, C,
                                   payload, norms, st);
  }
  return (int)hipErrorInvalidValue;
}

template <int D, int K, bool CG>
static int launch_decode_cg(const uint8_t* payload, const uint16_t* norms, const int64_t* ids,
                            int64_t n_vec, int64_t n_cache, const Shape& s, const float* R,
                            const float* C, float* out, hipStream_t st) {
  const size_t lds = sizeof(float) * ((size_t)D * D + (CG ? 0 : (size_t)s.N * K));
  auto kern = decode_kernel<D, K, CG>;
  hipError_t e = hipFuncSetAttribute((const void*)kern,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return (int)e;
  const int64_t nb = (n_vec * (D / 16) + 255) / 256;
  // every workgroup stages Pi (and a small codebook) in LDS: no more
  // workgroups than fit on the compute units at once, so large stagings
  // (d = 128 with 64 KB codebooks: 128 KB) are not repeated per batch of rows
  const int64_t per_cu = (int64_t)(160 * 1024 / lds) < 8 ? (int64_t)(160 * 1024 / lds) : 8;
  const int64_t cap = (int64_t)num_cus() * (per_cu > 0 ? per_cu : 1);
  const int grid = (int)(nb < cap ? nb : cap);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, payload, norms, ids, n_vec, n_cache, R,
                     C, s.N, s.w, s.P, out);
  return (int)hipGetLastError();
}

template <int D, int K>
static int launch_decode_t(const uint8_t* payload, const uint16_t* norms, const int64_t* ids,
                           int64_t n_vec, int64_t n_cache, const Shape& s, const float* R,
                           const float* C, float* out, hipStream_t st) {
  if ((int64_t)(D / K) * s.N * D <= kDecTab) {
    const size_t lds = sizeof(float) * (size_t)(D / K) * s.N * D;
    auto kern = decode_table_kernel<D, K>;
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return (int)e;
    const int64_t nb = (n_vec * (D / 16) + 255) / 256;
    const int64_t cap = (int64_t)num_cus() * 4;  // the table is built once per workgroup
    const int grid = (int)(nb < cap ? nb : cap);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, st, payload, norms, ids, n_vec, n_cache,
                       R, C, s.N, s.w, s.P, out);
    return (int)hipGetLastError();
  }
  // codebooks gathered from global memory (L2) when they do not fit beside Pi
  // in a third of the LDS (d = 128 with 64 KB codebooks: two workgroups per
  // compute unit instead of one)
  if (s.N * K > kCbLds || (int64_t)(D * D + s.N * K) * 4 > 96 * 1024)
    return launch_decode_cg<D, K, true>(payload, norms, ids, n_vec, n_cache, s, R, C, out, st);
  return launch_decode_cg<D, K, false>(payload, norms, ids, n_vec, n_cache, s, R, C, out, st);
}

int launch_decode(const uint8_t* payload, const uint16_t* norms, const int64_t* ids,
                  int64_t n_vec, int64_t n_cache, Shape s, const float* R, const float* C,
                  float* out, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
#define FIBQ_DEC_CASE(DD, KK)    \
  if (s.d == DD && s.k == KK) \
    return launch_decode_t<DD, KK>(payload, norms, ids, n_vec, n_cache, s, R, C, out, st);
  FIBQ_DEC_CASE(64, 1) FIBQ_DEC_CASE(64, 2) FIBQ_DEC_CASE(64, 4) FIBQ_DEC_CASE(64, 8)
  FIBQ_DEC_CASE(64, 16) FIBQ_DEC_CASE(128, 1) FIBQ_DEC_CASE(128, 2) FIBQ_DEC_CASE(128, 4)
  FIBQ_DEC_CASE(128, 8) FIBQ_DEC_CASE(128, 16) FIBQ_DEC_CASE(64, 32) FIBQ_DEC_CASE(64, 64)
#undef FIBQ_DEC_CASE
  return (int)hipErrorInvalidValue;
}

}  // namespace dev
}  // namespace fibq
