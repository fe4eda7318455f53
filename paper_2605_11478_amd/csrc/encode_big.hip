// Encoder for large codebooks at block dimension k = 4 (d = 128 with N = 1024,
// 2048 or 4096; d = 64 with N = 256, 1024 or 4096): Eq. encode of Sec. 3.1
// with the nearest-codeword search as a dense contraction on the matrix cores.
//
// A wavefront encodes 16 vectors per batch:
//
//   norm     nu^2 = sum x^2 in float64 (exact squares), header = binary16(nu)
//            rounded once, to nearest even;
//   rotate   y = Pi x / nu with v_mfma_f64_16x16x4_f64 (A = rows of Pi, B =
//            the 16 vectors; Pi is read as fp32 and converted exactly, its
//            rows permuted to match the output layout), so y carries only
//            float64 rounding.  Lane l then holds the k-blocks 4 rt + l / 16
//            (rt = 0 .. d/16 - 1) of vector l % 16;
//   screen   S_j = 2^24 (<y_b, c_j> - |c_j|^2 / 2) for 32 codewords x 32
//            blocks per v_mfma_f32_32x32x16_f16.  The 16 K slots carry the
//            binary16 hi / lo parts: c_lo y_hi + c_hi y_hi (lanes 0-31) and
//            c_hi y_lo - |c|^2 / 2 (lanes 32-63); y and c are scaled by 2^12
//            and |c|^2 / 2 by 2^14 (times B entries 2^10) so that no low part
//            leaves the binary16 normal range by much.  The codebook operand
//            table (24 bytes per codeword) lives in LDS;
//   select   each lane keeps, per block column, the best screen value B1, the
//            32-codeword tile T1 where it occurred and the best value B2 of
//            the other tiles (max / med3 per tile);
//   certify  the rows of tile T1 are re-scored in float64 in the direct form
//            |y - c|^2 (both half-wavefronts, lowest index on ties).  If the
//            best of them beats B2 by more than a bound E on the screen's
//            error, it is the float64 argmin over all N; otherwise the whole
//            wavefront re-scores all N codewords of that block in float64;
//   pack     w-bit indices, little-endian bit stream of P = 4 w bytes.
//
// Screen error bound (unscaled units): binary16 hi + lo represents y and c to
// 2^-22 relative plus 2^-26 absolute (low parts below the binary16 normal
// range may be flushed), the dropped c_lo y_lo term is below 2^-22 |c_i y_i|,
// products of binary16 numbers are exact in fp32, and the accumulation of the
// 16 terms is taken to lose at most 32 fp32 ulps of the sum of their
// magnitudes.  With sum |c_i y_i| <= min(|c|_inf |y_b|_1, |c|_2 |y_b|_2):
//   E = 1.25 [ (2^-18 + 2^-20) (sum |c_i y_i|) + (2^-18 + 2^-22) |c|^2_max / 2
//             + 2^-26 (|c|_1,max + |y_b|_1) + 2^-28 ] + 2^-40.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace big {

constexpr int K = 4;
constexpr int kWaves = 8;       // wavefronts per workgroup, large codebooks
constexpr int kWavesSmall = 4;  // small codebooks (N <= kSmallN): three workgroups per CU
constexpr int kSmallN = 1024;
constexpr int kVec = 16;        // vectors per wavefront batch
constexpr int kNmax = 4096;
constexpr int kRow = 24;        // LDS bytes per codeword: c_lo[4], c_hi[4], -n_hi, -n_lo, 0, 0
constexpr float kScale = 4096.0f;         // 2^12: y and c
constexpr double kNScale = 16384.0;       // 2^14: |c|^2 / 2
constexpr uint32_t kB1024 = 0x64006400u;  // binary16 pair (1024, 1024)
constexpr float kUnscale = 5.9604644775390625e-08f;  // 2^-24

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef double d4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t pack2(_Float16 a, _Float16 b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}
__device__ __forceinline__ double shfl64(double v, int src) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)u, src, 64);
  const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(u >> 32), src, 64);
  return __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
}
__device__ __forceinline__ double xor64(double v, int m) {
  return shfl64(v, (int)(threadIdx.x & 63) ^ m);
}
__device__ __forceinline__ double readlane64(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
}
// float64 squared distance |y - c|^2 in the direct form (coordinates in order)
__device__ __forceinline__ double dist64(const double y[4], float4 c) {
  double t = y[0] - (double)c.x, s = t * t;
  t = y[1] - (double)c.y; s = fma(t, t, s);
  t = y[2] - (double)c.z; s = fma(t, t, s);
  t = y[3] - (double)c.w; s = fma(t, t, s);
  return s;
}
__device__ __forceinline__ float fmax3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
// (d, j) is better than (bd, bj): smaller distance, lower index on ties
__device__ __forceinline__ bool better(double d, int j, double bd, int bj) {
  return d < bd || (d == bd && j < bj);
}

// NQ input elements (one quarter of a row) converted exactly to float
template <int NQ, typename IN>
__device__ __forceinline__ void loadq(const IN* p, float* xf);
template <int NQ>
__device__ __forceinline__ void loadq(const float* p, float* xf) {
#pragma unroll
  for (int i = 0; i < NQ / 4; ++i) {
    const float4 v = reinterpret_cast<const float4*>(p)[i];
    xf[4 * i] = v.x; xf[4 * i + 1] = v.y; xf[4 * i + 2] = v.z; xf[4 * i + 3] = v.w;
  }
}
template <int NQ>
__device__ __forceinline__ void loadq(const bf16_t* p, float* xf) {
#pragma unroll
  for (int i = 0; i < NQ / 8; ++i) {
    const uint4 v = reinterpret_cast<const uint4*>(p)[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xf[8 * i + 2 * j] = __uint_as_float(w[j] << 16);
      xf[8 * i + 2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
}
template <int NQ>
__device__ __forceinline__ void loadq(const f16_t* p, float* xf) {
#pragma unroll
  for (int i = 0; i < NQ / 8; ++i) {
    const uint4 v = reinterpret_cast<const uint4*>(p)[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xf[8 * i + 2 * j] = half_bits_to_float((uint16_t)(w[j] & 0xFFFFu));
      xf[8 * i + 2 * j + 1] = half_bits_to_float((uint16_t)(w[j] >> 16));
    }
  }
}

template <int D, typename IN, int WAVES>
__device__ __forceinline__ void encode_big_body(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms) {
  extern __shared__ __align__(16) unsigned char tab[];  // N * kRow bytes (launch argument)
  __shared__ uint32_t cst[4];  // float bits of max |c|_inf, max |c|_1, max |c|^2; bad flag
  __shared__ uint16_t stage[WAVES][kVec][D / K];  // chosen indices of a batch
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid < 4) cst[tid] = 0u;
  __syncthreads();
  {  // codebook operand table and the codebook's constants for the bound
    float ci = 0.0f, c1 = 0.0f, c2 = 0.0f;
    uint32_t bad = 0u;
    for (int j = tid; j < N; j += 64 * WAVES) {
      const float4 c4 = reinterpret_cast<const float4*>(C)[j];
      const float cv[4] = {c4.x, c4.y, c4.z, c4.w};
      _Float16 hi[4], lo[4];
      double n2 = 0.0;
      float a1 = 0.0f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float cs = cv[r] * kScale;  // exact
        hi[r] = (_Float16)cs;
        lo[r] = (_Float16)(cs - (float)hi[r]);
        n2 = fma((double)cv[r], (double)cv[r], n2);
        ci = fmaxf(ci, fabsf(cv[r]));
        a1 += fabsf(cv[r]);
      }
      c1 = fmaxf(c1, a1);
      c2 = fmaxf(c2, (float)n2);
      if (!(n2 <= 4.0)) bad = 1u;  // |c| <= 2 keeps every operand in binary16 range
      const double ns = 0.5 * n2 * kNScale;
      const _Float16 nh = (_Float16)(float)ns;
      const _Float16 nl = (_Float16)(float)(ns - (double)nh);
      uint32_t* row = reinterpret_cast<uint32_t*>(tab + (size_t)j * kRow);
      row[0] = pack2(lo[0], lo[1]);
      row[1] = pack2(lo[2], lo[3]);
      row[2] = pack2(hi[0], hi[1]);
      row[3] = pack2(hi[2], hi[3]);
      row[4] = pack2(-nh, -nl);
      row[5] = 0u;
    }
    ci = wave_max(ci);
    c1 = wave_max(c1);
    c2 = wave_max(c2);
    bad = __any(bad) ? 1u : 0u;
    if (lane == 0) {
      atomicMax(&cst[0], __float_as_uint(ci));
      atomicMax(&cst[1], __float_as_uint(c1));
      atomicMax(&cst[2], __float_as_uint(c2));
      atomicOr(&cst[3], bad);
    }
  }
  __syncthreads();
  const double cinf = (double)__uint_as_float(cst[0]);
  const double c1max = (double)__uint_as_float(cst[1]);
  const double c2max = (double)__uint_as_float(cst[2]);
  const double cnorm = sqrt(c2max);
  const bool bad = cst[3] != 0u;
  const double kE1 = 0x1p-18 + 0x1p-20, kE2 = 0x1p-18 + 0x1p-22;
  const double econst = 1.25 * (kE2 * 0.5 * c2max + 0x1p-26 * c1max + 0x1p-28) + 0x1p-40;

  const int h = lane >> 5, c32 = lane & 31, g = lane >> 4, v16 = lane & 15;
  const int ntile = N >> 5;
  const float4* C4 = reinterpret_cast<const float4*>(C);
  const unsigned char* arow = tab + (size_t)c32 * kRow + 8 * h;
  const int64_t nbatch = (n_vec + kVec - 1) / kVec;
  const int64_t nw = (int64_t)gridDim.x * WAVES;

  for (int64_t bt = (int64_t)blockIdx.x * WAVES + wave; bt < nbatch; bt += nw) {
    const int64_t v0 = bt * kVec;
    const int64_t vl = v0 + v16 < n_vec ? v0 + v16 : n_vec - 1;  // clamped (ragged batch)
    constexpr int NQ = D / 4;  // elements of a row per lane
    float xf[NQ];
    loadq<NQ>(x + vl * stride + NQ * g, xf);
    double ss = 0.0;
#pragma unroll
    for (int s = 0; s < NQ; ++s) ss = fma((double)xf[s], (double)xf[s], ss);
    ss += xor64(ss, 16);
    ss += xor64(ss, 32);
    const double nu = sqrt(ss);
    const double inv = nu > 0.0 ? 1.0 / nu : 0.0;
    if (g == 0 && v0 + v16 < n_vec) norms[v0 + v16] = nu > 0.0 ? f64_to_f16_bits(nu) : (uint16_t)0;

#pragma unroll 1
    for (int pass = 0; pass < D / 32; ++pass) {
      // ---- rotation of row tiles rt = 2 pass + q: y[q][i] = row 16 rt + 4 g + i of
      //      Pi x / nu, i.e. coordinate i of block 4 rt + g of vector lane % 16.
      //      The float64 MFMA leaves output row 4 i + g of a tile in register i
      //      of lanes 16 g .. 16 g + 15, so A row p (lanes with lane % 16 = p)
      //      is row 16 rt + 4 (p % 4) + p / 4 of Pi.
      d4 y[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int rt = 2 * pass + q;
        const int prw = 16 * rt + 4 * (v16 & 3) + (v16 >> 2);
        const float4* prow = reinterpret_cast<const float4*>(R + (size_t)prw * D + NQ * g);
        d4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int q4 = 0; q4 < NQ / 4; ++q4) {
          const float4 p = prow[q4];
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)p.x, (double)xf[4 * q4], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)p.y, (double)xf[4 * q4 + 1], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)p.z, (double)xf[4 * q4 + 2], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)p.w, (double)xf[4 * q4 + 3], acc, 0, 0, 0);
        }
        y[q] = acc * inv;
      }
      // B operands o = 2 q + s: row tile rt = 2 pass + q, column c = pair of lane c + 32 s
      h8 bop[4];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const d4 yr = y[q];
        _Float16 yh[4], yl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const double Y = yr[i] * (double)kScale;
          yh[i] = (_Float16)(float)Y;
          yl[i] = (_Float16)(float)(Y - (double)yh[i]);
        }
        const uint32_t oh0 = pack2(yh[0], yh[1]), oh1 = pack2(yh[2], yh[3]);
        const uint32_t ol0 = pack2(yl[0], yl[1]), ol1 = pack2(yl[2], yl[3]);
        // half 0 needs the partner's hi parts, half 1 the partner's lo parts
        const uint32_t r0 = (uint32_t)__shfl_xor((int)(h ? oh0 : ol0), 32, 64);
        const uint32_t r1 = (uint32_t)__shfl_xor((int)(h ? oh1 : ol1), 32, 64);
        u4 b0, b1;
        if (h == 0) {
          b0 = u4{oh0, oh1, oh0, oh1};
          b1 = u4{r0, r1, r0, r1};
        } else {
          b0 = u4{r0, r1, kB1024, 0u};
          b1 = u4{ol0, ol1, kB1024, 0u};
        }
        bop[2 * q] = __builtin_bit_cast(h8, b0);
        bop[2 * q + 1] = __builtin_bit_cast(h8, b1);
      }

      // ---- screen: best value, its tile, best value of the other tiles.
      // A tile's maximum carries the tile number in its 7 low mantissa bits
      // (one and-or against a mask held in a register; moves it by < 128 of
      // its ulps, a term of the certificate's bound), so the best key also
      // names its tile.
      float b1v[4], b2v[4];
      int t1[4];
#pragma unroll
      for (int o = 0; o < 4; ++o) { b1v[o] = -INFINITY; b2v[o] = -INFINITY; }
      uint32_t kmask = ~127u;
      asm volatile("" : "+v"(kmask));
      // (maximum3 instead of max: no canonicalising moves; scores are finite)
      uint2 a0 = *reinterpret_cast<const uint2*>(arow);
      uint2 a1 = *reinterpret_cast<const uint2*>(arow + 8);
#pragma unroll 2
      for (int t = 0; t < ntile; ++t) {
        const h8 A = __builtin_bit_cast(h8, u4{a0.x, a0.y, a1.x, a1.y});
        {  // next tile's operand (the last tile re-reads itself)
          const unsigned char* ap = arow + (size_t)(t + 1 < ntile ? t + 1 : t) * (32 * kRow);
          a0 = *reinterpret_cast<const uint2*>(ap);
          a1 = *reinterpret_cast<const uint2*>(ap + 8);
        }
#pragma unroll
        for (int o = 0; o < 4; ++o) {
          const f16v s = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, bop[o], f16v{}, 0, 0, 0);
          float m = fmax3(s[0], s[1], s[2]);
          m = fmax3(m, s[3], s[4]);
          m = fmax3(m, s[5], s[6]);
          m = fmax3(m, s[7], s[8]);
          m = fmax3(m, s[9], s[10]);
          m = fmax3(m, s[11], s[12]);
          m = fmax3(m, s[13], s[14]);
          m = __builtin_elementwise_maximum(m, s[15]);
          const float mk = __uint_as_float((__float_as_uint(m) & kmask) | (uint32_t)t);
          b2v[o] = __builtin_amdgcn_fmed3f(b1v[o], b2v[o], mk);
          b1v[o] = __builtin_elementwise_maximum(b1v[o], mk);
        }
      }
#pragma unroll
      for (int o = 0; o < 4; ++o) t1[o] = (int)(__float_as_uint(b1v[o]) & 127u);

      // ---- certificate per column, float64 fallback over all N when needed
#pragma unroll
      for (int o = 0; o < 4; ++o) {
        const int rt = 2 * pass + (o >> 1), s = o & 1;
        double yc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const double other = xor64(y[o >> 1][i], 32);
          yc[i] = (s == h) ? y[o >> 1][i] : other;
        }
        // rows of tile t1 in this half: codewords 32 t1 + 8 (r / 4) + 4 h + r % 4
        double bd = INFINITY;
        int bj = 0;
        const int jb = 32 * t1[o] + 4 * h;
#pragma unroll 4
        for (int r = 0; r < 16; ++r) {
          const int j = jb + 8 * (r >> 2) + (r & 3);
          const double dd = dist64(yc, C4[j]);
          if (dd < bd) { bd = dd; bj = j; }
        }
        const double od = xor64(bd, 32);
        const int oj = __shfl_xor(bj, 32, 64);
        if (better(od, oj, bd, bj)) { bd = od; bj = oj; }
        const float b2 = fmaxf(b2v[o], __shfl_xor(b2v[o], 32, 64));
        const double yn2 = yc[0] * yc[0] + yc[1] * yc[1] + yc[2] * yc[2] + yc[3] * yc[3];
        const double y1 = fabs(yc[0]) + fabs(yc[1]) + fabs(yc[2]) + fabs(yc[3]);
        const double cy = fmin(cinf * y1, cnorm * sqrt(yn2));
        const double E = 1.25 * kE1 * cy + 1.25 * 0x1p-26 * y1 + econst +
                         1.25 * 0x1p-16 * fabs((double)b2 * (double)kUnscale);  // packed bits
        const bool cert = !bad && 0.5 * (yn2 - bd) > (double)b2 * (double)kUnscale + E;
        // full float64 re-score of the uncertified columns, one at a time
        uint64_t pend = __ballot(!cert && h == 0);
        while (pend) {
          const int cl = __builtin_ctzll(pend);
          pend &= pend - 1;
          const double yb[4] = {readlane64(yc[0], cl), readlane64(yc[1], cl),
                                readlane64(yc[2], cl), readlane64(yc[3], cl)};
          double fd = INFINITY;
          int fj = 0;
#pragma unroll 1
          for (int j = lane; j < N; j += 64) {
            const double dd = dist64(yb, C4[j]);
            if (dd < fd) { fd = dd; fj = j; }
          }
#pragma unroll
          for (int m = 32; m > 0; m >>= 1) {
            const double od2 = xor64(fd, m);
            const int oj2 = __shfl_xor(fj, m, 64);
            if (better(od2, oj2, fd, fj)) { fd = od2; fj = oj2; }
          }
          if (c32 == cl) bj = fj;
        }
        // column c32 of operand o is block 4 rt + 2 s + c32 / 16 of vector c32 % 16
        if (h == 0) stage[wave][v16][4 * rt + 2 * s + (c32 >> 4)] = (uint16_t)bj;
      }
    }

    // ---- pack: lane v < 16 writes the bit stream of vector v (this wavefront's
    //      own LDS writes precede its reads)
    if (lane < 16 && v0 + lane < n_vec) {
      uint32_t* dst = reinterpret_cast<uint32_t*>(payload + (v0 + lane) * (int64_t)P);
      const bool zero = !(nu > 0.0);
      uint64_t bits = 0;
      int nb = 0, wd = 0;
#pragma unroll
      for (int m = 0; m < D / K; ++m) {
        const uint32_t id = zero ? 0u : (uint32_t)stage[wave][lane][m];
        bits |= (uint64_t)id << nb;
        nb += W;
        if (nb >= 32) {
          dst[wd++] = (uint32_t)bits;
          bits >>= 32;
          nb -= 32;
        }
      }
    }
  }
}

// At d = 64, small codebooks (N <= 1024: an operand table of at most 24 KB)
// run in 4-wavefront workgroups, three per compute unit (three wavefronts per
// SIMD, <= 168 VGPRs); larger tables, and d = 128 (whose registers do not fit
// that budget), run one 8-wavefront workgroup per compute unit.
template <int D, typename IN>
__global__ __launch_bounds__(64 * kWavesSmall) __attribute__((amdgpu_waves_per_eu(3))) void
encode_big_kernel_s(const IN* __restrict__ x, int64_t n_vec, int64_t stride,
                    const float* __restrict__ R, const float* __restrict__ C, int N, int W, int P,
                    uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_big_body<D, IN, kWavesSmall>(x, n_vec, stride, R, C, N, W, P, payload, norms);
}
template <int D, typename IN>
__global__ __launch_bounds__(64 * kWaves) void encode_big_kernel(
    const IN* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, int N, int W, int P, uint8_t* __restrict__ payload,
    uint16_t* __restrict__ norms) {
  encode_big_body<D, IN, kWaves>(x, n_vec, stride, R, C, N, W, P, payload, norms);
}

}  // namespace big

bool encode_big_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                        const float* R, const float* C, const uint8_t* payload) {
  if (s.k != big::K || s.N > big::kNmax) return false;
  if (s.d == 128) {
    if (s.N < 1024) return false;
  } else if (s.d == 64) {
    // the packer stores whole 32-bit words: 16 blocks x w bits must fill them
    if (s.N < 256 || (16 * s.w) % 32 != 0) return false;
  } else {
    return false;
  }
  const int esz = dtype == FIBQ_F32 ? 4 : 2;
  const auto al = [](const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; };
  return al(x, 16) && (stride * esz) % 16 == 0 && al(R, 16) && al(C, 16) && al(payload, 4);
}

template <int D, typename IN>
static int launch_big_t(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                        const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                        int n_cu, hipStream_t st) {
  const size_t lds = (size_t)s.N * big::kRow;
  const int64_t nbatch = (n_vec + big::kVec - 1) / big::kVec;
  const IN* xi = static_cast<const IN*>(x);
  if constexpr (D == 64) {
    if (s.N <= big::kSmallN) {
      const int64_t want = (nbatch + big::kWavesSmall - 1) / big::kWavesSmall;
      const int grid = (int)(want < 3LL * n_cu ? want : 3LL * n_cu);
      hipLaunchKernelGGL((big::encode_big_kernel_s<D, IN>), dim3(grid),
                         dim3(64 * big::kWavesSmall), lds, st, xi, n_vec, stride, R, C, s.N, s.w,
                         s.P, payload, norms);
      return (int)hipGetLastError();
    }
  }
  auto kern = big::encode_big_kernel<D, IN>;
  if (lds > 65536) {  // above the default dynamic LDS limit
    const hipError_t e = hipFuncSetAttribute(
        (const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return (int)e;
  }
  const int64_t want = (nbatch + big::kWaves - 1) / big::kWaves;
  const int grid = (int)(want < n_cu ? want : n_cu);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * big::kWaves), lds, st, xi, n_vec, stride, R, C,
                     s.N, s.w, s.P, payload, norms);
  return (int)hipGetLastError();
}

template <int D>
static int launch_big_d(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                        const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                        int n_cu, hipStream_t st) {
  switch (dtype) {
    case FIBQ_F32:
      return launch_big_t<D, float>(x, n_vec, stride, s, R, C, payload, norms, n_cu, st);
    case FIBQ_F16:
      return launch_big_t<D, f16_t>(x, n_vec, stride, s, R, C, payload, norms, n_cu, st);
    default:
      return launch_big_t<D, bf16_t>(x, n_vec, stride, s, R, C, payload, norms, n_cu, st);
  }
}

int launch_encode_big(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                      const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                      void* stream, int n_cu) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s.d == 128) return launch_big_d<128>(x, dtype, n_vec, stride, s, R, C, payload, norms, n_cu, st);
  return launch_big_d<64>(x, dtype, n_vec, stride, s, R, C, payload, norms, n_cu, st);
}

}  // namespace dev
}  // namespace fibq
