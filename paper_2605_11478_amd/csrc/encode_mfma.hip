// Encoder on the matrix cores for bf16 caches with d = 64, k = 8 and
// N in {16, 64} (the sub-one-bit long-context rates; Sec. 3.1, Eq. encode).
//
// One wavefront encodes 16 vectors per step:
//   norm      nu^2 = sum x^2 in float32 (packed bf16 dot products), nu = sqrt;
//             the binary16 header is certified by rounding nu (1 -+ delta),
//             delta above the float32 error; an uncertain header is redone in
//             float64 from the exact squares;
//   rotation  z = Pi x on v_mfma_f32_16x16x32_bf16: x is exact in bf16 and Pi
//             is split into three bf16 parts (hi + mid + lo == Pi), so the
//             products are exact and only the float32 accumulation rounds.
//             The rows of Pi are permuted so that the lane holding a vector's
//             result holds all 8 coordinates of one block (no shuffles);
//   screen    G_j = <y, c_j> - |c_j|^2 / 2 + K0 for every codeword (the
//             argmin of |y - c_j|^2 is the argmax of G_j), one
//             v_mfma_f32_16x16x32_f16 per 4 codewords x 4 blocks: y = z / nu
//             enters as fp16 hi + lo of 2^8 y (two products), the codebook
//             as fp16 2^10 c (a codebook that is not fp16-exact adds its
//             residual); the scalings keep the fp16 low parts in the normal
//             range, so the result does not depend on how the matrix cores
//             treat fp16 subnormals.  The accumulator starts at
//             2^18 (K0 - |c_j|^2 / 2) > 0.  Each lane sees all
//             N candidates of one (vector, block) pair and keeps the best two
//             with the codeword number packed into the low mantissa bits
//             (positive floats compare as integers);
//   exact     when the best two are closer than a rigorous bound on the
//             screen's error, the block is redone in float64 in the direct
//             form |y - c|^2 by the whole wavefront (rare), so every index is
//             the float64 argmin (lowest index on ties).
// Payload words are assembled across the four lanes of a vector and stored
// with coalesced writes; the headers likewise.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace encmf {

constexpr int D = 64, K = 8;
constexpr int kThreads = 256;
constexpr int kDepth = 6;  // input tiles in flight per wavefront

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// bf16 bits of a float, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float v) {
  const uint32_t b = __float_as_uint(v);
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_val(uint32_t bits) { return __uint_as_float(bits << 16); }

// Asynchronous 16-byte-per-lane copy global -> LDS (global_load_lds_dwordx4):
// lane l's 16 bytes land at lds_base + 16 l.  Issued from inline assembly so
// that the compiler does not serialise it with a blanket wait before every
// LDS read; completion is awaited explicitly with vm_wait (vector-memory
// operations complete in issue order).  M0 (the LDS base) is saved and
// restored around the instruction.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
  uint32_t keep;
  const uint32_t b = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(gptr), "s"(b)
      : "memory");
}
template <int CNT>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CNT) : "memory");
}

// x + (partner in the other half-wave), and the same over 16-lane rows:
// symmetric sums over the four lane groups holding one vector.
__device__ __forceinline__ float sum_groups(float v) {
  auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ uint32_t or_groups(uint32_t v) {
  auto a = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = a[0] | a[1];
  auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return b[0] | b[1];
}
__device__ __forceinline__ double sum_groups64(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)u, (uint32_t)u, false, false);
  auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  v = __longlong_as_double((long long)((uint64_t)lo[0] | ((uint64_t)hi[0] << 32))) +
      __longlong_as_double((long long)((uint64_t)lo[1] | ((uint64_t)hi[1] << 32)));
  const uint64_t w = (uint64_t)__double_as_longlong(v);
  auto lo2 = __builtin_amdgcn_permlane16_swap((uint32_t)w, (uint32_t)w, false, false);
  auto hi2 = __builtin_amdgcn_permlane16_swap((uint32_t)(w >> 32), (uint32_t)(w >> 32), false, false);
  return __longlong_as_double((long long)((uint64_t)lo2[0] | ((uint64_t)hi2[0] << 32))) +
         __longlong_as_double((long long)((uint64_t)lo2[1] | ((uint64_t)hi2[1] << 32)));
}

// Register-only cross-lane moves for the float64 path (DPP within 16-lane
// rows; v_permlane*_swap across rows), so that it does not wait on LDS.
__device__ __forceinline__ uint32_t dpp32(uint32_t v, int ctrl) {
  switch (ctrl) {  // the control must be an immediate
    case 0xB1: return __builtin_amdgcn_update_dpp(0u, v, 0xB1, 0xF, 0xF, false);   // lane ^ 1
    case 0x4E: return __builtin_amdgcn_update_dpp(0u, v, 0x4E, 0xF, 0xF, false);   // lane ^ 2
    case 0x141: return __builtin_amdgcn_update_dpp(0u, v, 0x141, 0xF, 0xF, false); // 7 - lane in 8
    default: return __builtin_amdgcn_update_dpp(0u, v, 0x140, 0xF, 0xF, false);    // 15 - lane in 16
  }
}
__device__ __forceinline__ double dpp64(double v, int ctrl) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint64_t r = (uint64_t)dpp32((uint32_t)u, ctrl) | ((uint64_t)dpp32((uint32_t)(u >> 32), ctrl) << 32);
  return __longlong_as_double((long long)r);
}
// sum over the aligned group of 8 lanes (identical in all 8)
__device__ __forceinline__ double sum8(double v) {
  v += dpp64(v, 0xB1);
  v += dpp64(v, 0x4E);
  return v + dpp64(v, 0x141);
}
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t perm64(uint64_t v, bool p16) {
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  if (p16) {
    auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    return umin64((uint64_t)a[0] | ((uint64_t)b[0] << 32), (uint64_t)a[1] | ((uint64_t)b[1] << 32));
  }
  auto a = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  auto b = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  return umin64((uint64_t)a[0] | ((uint64_t)b[0] << 32), (uint64_t)a[1] | ((uint64_t)b[1] << 32));
}
// minimum over the wavefront (identical in all lanes)
__device__ __forceinline__ uint64_t wave_min64(uint64_t k) {
  auto step = [](uint64_t v, int ctrl) {
    const uint64_t o = (uint64_t)dpp32((uint32_t)v, ctrl) | ((uint64_t)dpp32((uint32_t)(v >> 32), ctrl) << 32);
    return umin64(v, o);
  };
  k = step(k, 0xB1);
  k = step(k, 0x4E);
  k = step(k, 0x141);
  k = step(k, 0x140);
  k = perm64(k, true);
  return perm64(k, false);
}

// Float64 nearest codeword of block m of one vector (direct form), computed
// by the whole wavefront: lane (r, c) = (l / 8, l % 8) forms the partial sum
// of row 8m + r of Pi x over dims 8c .. 8c+7 (x read from the LDS tile,
// chunk c of the row sits at position c xor (row % 8)); lane j then scores
// codeword j.  The minimum is taken over (D_j with its 6 lowest bits
// replaced by j): equal keys pick the lowest index, and D_j agreeing to
// within 2^-46 relative (far inside the near-tie window) count as ties.
// All 64 lanes must be active.
__device__ __forceinline__ uint32_t exact_block(const unsigned char* tile, int vl,
                                                const float* __restrict__ R,
                                                const float* __restrict__ C, int N, int m,
                                                int l) {
  const int r = l >> 3, c = l & 7;
  const uint4 raw = *reinterpret_cast<const uint4*>(tile + (vl >> 3) * 1024 + (vl & 7) * 128 +
                                                    16 * (c ^ (vl & 7)));
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  const float4 pa = *reinterpret_cast<const float4*>(R + (8 * m + r) * D + 8 * c);
  const float4 pb = *reinterpret_cast<const float4*>(R + (8 * m + r) * D + 8 * c + 4);
  const float pr[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
  double ss = 0.0, p = 0.0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const double x0 = (double)__uint_as_float(w[i] << 16);
    const double x1 = (double)__uint_as_float(w[i] & 0xFFFF0000u);
    ss = fma(x0, x0, ss);
    ss = fma(x1, x1, ss);
    p = fma((double)pr[2 * i], x0, p);
    p = fma((double)pr[2 * i + 1], x1, p);
  }
  ss = sum8(ss);
  p = sum8(p);
  const double nu = sqrt(ss);
  if (!(nu > 0.0)) return 0u;  // uniform: zero or NaN norm stores index 0
  const double yr = p / nu;    // y_{8m + r}, identical in lanes 8r .. 8r+7
  const uint64_t yu = (uint64_t)__double_as_longlong(yr);
  double dj = 0.0;
#pragma unroll
  for (int rr = 0; rr < K; ++rr) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)yu, 8 * rr);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(yu >> 32), 8 * rr);
    const double yb = __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
    const double t = yb - (double)C[(l < N ? l : 0) * K + rr];
    dj = fma(t, t, dj);
  }
  uint64_t key = ((uint64_t)__double_as_longlong(dj) & ~(uint64_t)63) | (uint64_t)l;
  if (l >= N) key = ~(uint64_t)0;
  key = wave_min64(key);
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)(key & 63));
}

template <int N>
__device__ __forceinline__ void encode_body(const uint16_t* __restrict__ x, int64_t n_vec,
                                            int64_t stride, const float* __restrict__ R,
                                            const float* __restrict__ C,
                                            uint8_t* __restrict__ payload,
                                            uint16_t* __restrict__ norms) {
  constexpr int NSET = N / 4;       // codeword sets of 4 (one MFMA row group each)
  constexpr int W = (N == 16) ? 4 : 6;
  const int l = threadIdx.x & 63;
  const int g = l >> 4, col = l & 15;

  // LDS: per-wavefront rings of kDepth 2 KB input tiles (the first 16 KB
  // hold Pi while the per-lane constants are built, before any tile is
  // requested), the codebook, and the residual rows of a codebook that is not
  // fp16-exact.
  constexpr int kRing = (kThreads / 64) * kDepth * 2048;
  __shared__ __align__(16) unsigned char smem[kRing + N * K * 4 + (kThreads / 64) * NSET * 64 * 16];
  float* Rs = reinterpret_cast<float*>(smem);
  float* Cs = reinterpret_cast<float*>(smem + kRing);
  h8(*alo_lds)[NSET][64] = reinterpret_cast<h8(*)[NSET][64]>(smem + kRing + N * K * 4);
  for (int i = threadIdx.x; i < D * D / 4; i += kThreads)
    reinterpret_cast<float4*>(Rs)[i] = reinterpret_cast<const float4*>(R)[i];
  for (int i = threadIdx.x; i < N * K; i += kThreads) Cs[i] = C[i];
  __syncthreads();
  const float* Rg = R;  // global copies for the float64 path (the ring reuses Rs)
  R = Rs;
  C = Cs;

  // ---- rotation operands: A = rows of Pi in the permuted order, three bf16
  // parts.  Output row rho of tile r is dimension
  // 8 (4 (r >> 1) + rho / 4) + 4 (r & 1) + rho % 4.
  bf8 Api[4][2][3];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int rho = l & 15;
    const int dim = 8 * (4 * (r >> 1) + (rho >> 2)) + 4 * (r & 1) + (rho & 3);
#pragma unroll
    for (int kap = 0; kap < 2; ++kap) {
      const float* src = R + dim * D + 32 * kap + 8 * g;
      const float4 a = *reinterpret_cast<const float4*>(src);
      const float4 b = *reinterpret_cast<const float4*>(src + 4);
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      uint32_t part[3][4];
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        uint32_t hb[2], mb[2], lb[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const float vv = v[i + t];
          hb[t] = bf16_rne(vv);
          const float r1 = vv - bf16_val(hb[t]);  // exact
          mb[t] = bf16_rne(r1);
          const float r2 = r1 - bf16_val(mb[t]);  // exact
          lb[t] = bf16_rne(r2);
        }
        part[0][i / 2] = hb[0] | (hb[1] << 16);
        part[1][i / 2] = mb[0] | (mb[1] << 16);
        part[2][i / 2] = lb[0] | (lb[1] << 16);
      }
#pragma unroll
      for (int s = 0; s < 3; ++s)
        Api[r][kap][s] = __builtin_bit_cast(bf8, u4v{part[s][0], part[s][1], part[s][2], part[s][3]});
    }
  }

  // ---- screen operands: A_s = codewords 4s + rho % 4 on the K range of block
  // rho / 4 of the quad (zero elsewhere); accumulator init K0 - |c|^2 / 2.
  float cmax2 = 0.0f, l1max = 0.0f;
  bool lo_any = false;
  for (int j = l; j < N; j += 64) {
    float s2 = 0.0f;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const float cv = C[j * K + i];
      s2 = fmaf(cv, cv, s2);
      lo_any |= (float)(_Float16)cv != cv;
    }
    cmax2 = fmaxf(cmax2, s2);
  }
  for (int pr = l; pr < N * N; pr += 64) {  // max over pairs of |c_i - c_j|_1
    const int i = pr / N, j = pr % N;
    if (i < j) {
      float s1 = 0.0f;
#pragma unroll
      for (int t = 0; t < K; ++t) s1 += fabsf(C[i * K + t] - C[j * K + t]);
      l1max = fmaxf(l1max, s1);
    }
  }
  cmax2 = wave_max(cmax2) * (1.0f + 1e-6f);
  l1max = wave_max(l1max) * (1.0f + 1e-6f);
  const bool has_lo = __any(lo_any);
  const float cmax = sqrtf(cmax2) * (1.0f + 1e-6f);
  const float K0 = cmax + 0.5f * cmax2 + 0x1p-10f;  // G_j >= 2^-10 for |y| <= 1
  // Bound on the screen's error for the difference of two candidates' G
  // (y = Pi x / nu per block has |y| <= 1):
  //   rotation: bf16 x and Pi parts give exact products, <= 128 float32
  //     roundings (at most 2 ulp each) per output: |dy| <= 2^-17 per dim,
  //     times max |c_i - c_j|_1;
  //   nu, hi/lo split: relative 2^-19 + 2^-22 of y, times max |c_i - c_j|;
  //   screen accumulation (<= 40 roundings of values <= K0 + 2 cmax), the
  //     fp16 codebook residual and the packed index bits (log2 N of 23).
  //   fp16 low parts of 2^8 y below the normal range: 2^-22 per dim.
  // Everything in units of G; the screen works in units of 2^18 G.
  const float gmax = K0 + 2.0f * cmax + cmax2;
  const float e_rot = (1.02f * 0x1p-17f + 0x1p-25f + 0x1p-22f) * l1max;
  const float e_nu = (0x1p-19f + 0x1p-22f) * 2.0f * cmax;
  const float e_acc = 100.0f * 0x1p-24f * gmax + (has_lo ? 0x1p-21f * cmax : 0.0f);
  const float e_pack = 2.0f * gmax * (float)N * 0x1p-23f;
  const float margin =
      0x1p18f * (1.25f * (e_rot + e_nu + e_acc + e_pack) + 4.0f * 0x1p-24f * gmax);

  h8 Acb[NSET];
  f4 init[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    const int rho = l & 15;
    const int j = 4 * s + (rho & 3);
    const bool on = (rho >> 2) == g;
    h8 a, al;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const float cv = C[j * K + i];
      const _Float16 hi = (_Float16)cv;
      a[i] = on ? (_Float16)((float)hi * 0x1p10f) : (_Float16)0.0f;
      al[i] = on ? (_Float16)((cv - (float)hi) * 0x1p10f) : (_Float16)0.0f;
    }
    Acb[s] = a;
    alo_lds[threadIdx.x >> 6][s][l] = al;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int jj = 4 * s + e;
      float s2 = 0.0f;
#pragma unroll
      for (int i = 0; i < K; ++i) s2 = fmaf(C[jj * K + i], C[jj * K + i], s2);
      init[s][e] = 0x1p18f * (K0 - 0.5f * s2);
    }
  }

  // ---- persistent loop over 16-vector tiles, one wavefront per tile.
  // Tile loads run kDepth - 1 tiles ahead through the LDS ring: lane l copies
  // 16 bytes of row 8 h + l / 8 (h = half of the tile) into slot position l;
  // the chunk it takes is (l % 8) xor (l / 8), so the transposed operand
  // reads below spread over the LDS banks while each row stays one 128-byte
  // burst.  The last tile clamps its rows into [0, n_vec).
  const int64_t ntiles = (n_vec + 15) >> 4;
  const int64_t nwaves = (int64_t)gridDim.x * (kThreads / 64);
  const int64_t wid = (int64_t)blockIdx.x * (kThreads / 64) +
                      __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  R = Rg;  // Pi from global memory from here on (LDS copy is overwritten)
  __syncthreads();  // every wavefront has built its constants from Rs
  const uint32_t ring = (uint32_t)(uintptr_t)(smem + (threadIdx.x >> 6) * kDepth * 2048);
  const int rih = l >> 3, pos = l & 7;
  const int chunk = pos ^ rih;
  auto issue = [&](int64_t tile, int slot) {
    int64_t ra = tile * 16 + rih, rb = ra + 8;
    ra = ra < n_vec ? ra : n_vec - 1;
    rb = rb < n_vec ? rb : n_vec - 1;
    dma16(x + ra * stride + 8 * chunk, ring + slot * 2048);
    dma16(x + rb * stride + 8 * chunk, ring + slot * 2048 + 1024);
  };
  // operand chunks of this lane: row col, chunks g and 4 + g
  const uint32_t rd0 = (col >> 3) * 1024 + (col & 7) * 128 + 16 * (g ^ (col & 7));
  const uint32_t rd1 = (col >> 3) * 1024 + (col & 7) * 128 + 16 * ((4 + g) ^ (col & 7));
#pragma unroll
  for (int d = 0; d < kDepth; ++d)
    if (wid + d * nwaves < ntiles) issue(wid + d * nwaves, d);
  int slot = 0;
  for (int64_t tile = wid; tile < ntiles; tile += nwaves) {
    // the tile's copies are older than the 2 (kDepth - 1) copies of the
    // tiles requested after it (when all of those exist; else wait for all)
    if (tile + (kDepth - 1) * nwaves < ntiles) vm_wait<2 * (kDepth - 1)>();
    else vm_wait<0>();
    const unsigned char* sl = smem + (threadIdx.x >> 6) * kDepth * 2048 + slot * 2048;
    const uint4 ca = *reinterpret_cast<const uint4*>(sl + rd0);
    const uint4 cb = *reinterpret_cast<const uint4*>(sl + rd1);
    const int64_t v = tile * 16 + col;
    const bool live = v < n_vec;
    const bf8 x0 = __builtin_bit_cast(bf8, u4v{ca.x, ca.y, ca.z, ca.w});
    const bf8 x1 = __builtin_bit_cast(bf8, u4v{cb.x, cb.y, cb.z, cb.w});

    // norm (float32) and its certified binary16 header
    float ss = 0.0f;
    {
      const uint32_t w0[4] = {ca.x, ca.y, ca.z, ca.w}, w1[4] = {cb.x, cb.y, cb.z, cb.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf2 p0 = __builtin_bit_cast(bf2, w0[i]), p1 = __builtin_bit_cast(bf2, w1[i]);
        ss = __builtin_amdgcn_fdot2_f32_bf16(p0, p0, ss, false);
        ss = __builtin_amdgcn_fdot2_f32_bf16(p1, p1, ss, false);
      }
    }
    ss = sum_groups(ss);
    // hardware sqrt and reciprocal (1 ulp each; the bounds above allow 2^-19)
    const float nu = __builtin_amdgcn_sqrtf(ss);
    const float inv = 0x1p8f * __builtin_amdgcn_rcpf(nu);  // 2^8 / nu: the screen's scaling of y
    const uint16_t h_a = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f - 0x1p-19f)));
    const uint16_t h_b = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f + 0x1p-19f)));
    uint32_t hdr = h_a;
    bool zero = false;
    if (__any(ss == 0.0f)) {  // the float32 sum can underflow: test the bits
      const uint32_t o = (ca.x | ca.y | ca.z | ca.w | cb.x | cb.y | cb.z | cb.w) & 0x7FFF7FFFu;
      zero = or_groups(o) == 0u;
    }
    // float32 range where the error bounds hold; outside it (or for
    // non-finite input) the whole vector is redone in float64
    const bool wild = !(ss >= 0x1p-100f && ss <= 0x1p100f) && !zero;
    bool hdr_unsure = (h_a != h_b) && !wild && !zero;
    if (zero) hdr = 0;

    // rotation: z[r] = rows of (Pi x) for tile r (small parts first)
    f4 z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      f4 a = {0, 0, 0, 0};
#pragma unroll
      for (int s = 2; s >= 0; --s) {
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Api[r][0][s], x0, a, 0, 0, 0);
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Api[r][1][s], x1, a, 0, 0, 0);
      }
      z[r] = a;
    }

    // screen, per block quad q: this lane sees block 4q + g of vector col
    uint32_t idx[2];
    bool unsure[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      h8 yh, yl;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float zz = z[2 * q + (i >> 2)][i & 3];
        const _Float16 hi = (_Float16)__builtin_fmaf(zz, inv, 0.0f);  // one mixed fma
        yh[i] = hi;
        yl[i] = (_Float16)__builtin_fmaf(zz, inv, -(float)hi);
      }
      uint32_t t1 = 0, t2 = 0;
#pragma unroll
      for (int s = 0; s < NSET; ++s) {
        f4 gq = __builtin_amdgcn_mfma_f32_16x16x32_f16(Acb[s], yh, init[s], 0, 0, 0);
        gq = __builtin_amdgcn_mfma_f32_16x16x32_f16(Acb[s], yl, gq, 0, 0, 0);
        if (has_lo)
          gq = __builtin_amdgcn_mfma_f32_16x16x32_f16(alo_lds[threadIdx.x >> 6][s][l], yh, gq, 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t p = (__float_as_uint(gq[e]) & ~(uint32_t)(N - 1)) | (uint32_t)(4 * s + e);
          t2 = max(min(t1, t2), min(max(t1, t2), p));  // second largest of {t1, t2, p}
          t1 = max(t1, p);
        }
      }
      idx[q] = t1 & (uint32_t)(N - 1);
      const float gap = __uint_as_float(t1) - __uint_as_float(t2);
      unsure[q] = !(gap >= margin) && live && !zero;
      if (zero) idx[q] = 0;
    }

    // ---- rare exact paths (wave-uniform loops).  A vector outside the
    // float32 range has its header and all 8 blocks redone in float64.
    if (wild && live) {
      hdr_unsure = true;
      unsure[0] = unsure[1] = true;
    }
    if (__any(hdr_unsure && live)) {
      // float64 sum of the exact squares over this lane's 16 values
      double s64 = 0.0;
      const uint32_t w0[4] = {ca.x, ca.y, ca.z, ca.w}, w1[4] = {cb.x, cb.y, cb.z, cb.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double a0 = __uint_as_float(w0[i] << 16), a1 = __uint_as_float(w0[i] & 0xFFFF0000u);
        const double b0 = __uint_as_float(w1[i] << 16), b1 = __uint_as_float(w1[i] & 0xFFFF0000u);
        s64 = fma(a0, a0, s64);
        s64 = fma(a1, a1, s64);
        s64 = fma(b0, b0, s64);
        s64 = fma(b1, b1, s64);
      }
      s64 = sum_groups64(s64);
      if (hdr_unsure) hdr = s64 > 0.0 ? f64_to_f16_bits(sqrt(s64)) : 0u;
    }
    uint64_t todo = __ballot(unsure[0] || unsure[1]);
    while (todo) {  // near ties: the block in float64
      const int ln = __builtin_ctzll(todo);
      todo &= todo - 1;
      const int lg = ln >> 4;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (__builtin_amdgcn_readlane((int)unsure[q], ln)) {
          const uint32_t bi = exact_block(sl, ln & 15, R, C, N, 4 * q + lg, l);
          if (l == ln) idx[q] = bi;
        }
      }
    }

    // ---- payload (little-endian bit stream, index m at bits [m W, (m+1) W))
    //      and header stores
    if (W == 4) {
      const uint32_t word = or_groups((idx[0] << (4 * g)) | (idx[1] << (16 + 4 * g)));
      if (live && g == 0) reinterpret_cast<uint32_t*>(payload)[v] = word;
    } else {
      const uint64_t part = ((uint64_t)idx[0] << (6 * g)) | ((uint64_t)idx[1] << (24 + 6 * g));
      const uint32_t lo = or_groups((uint32_t)part), hi = or_groups((uint32_t)(part >> 32));
      if (live && g < 3) {
        const uint32_t half = g == 0 ? (lo & 0xFFFFu) : (g == 1 ? (lo >> 16) : (hi & 0xFFFFu));
        reinterpret_cast<uint16_t*>(payload)[3 * v + g] = (uint16_t)half;
      }
    }
    if (live && g == 3) norms[v] = (uint16_t)hdr;
    // request tile + kDepth waves into the slot read in this iteration (its
    // LDS reads have completed: their values fed this tile's work)
    const int64_t nt = tile + kDepth * nwaves;
    if (nt < ntiles) issue(nt, slot);
    slot = slot + 1 == kDepth ? 0 : slot + 1;
  }
}

// N = 16 fits two wavefronts per SIMD (<= 256 VGPRs); N = 64 holds four
// times the codebook operands and runs one.
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void encode_kernel16(
    const uint16_t* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_body<16>(x, n_vec, stride, R, C, payload, norms);
}
__global__ __launch_bounds__(kThreads) void encode_kernel64(
    const uint16_t* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_body<64>(x, n_vec, stride, R, C, payload, norms);
}

}  // namespace encmf

bool encode_mfma_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                         const float* R, const uint8_t* payload, const uint16_t* norms) {
  if (dtype != FIBQ_BF16 || s.d != 64 || s.k != 8 || !(s.N == 16 || s.N == 64)) return false;
  const uintptr_t ax = reinterpret_cast<uintptr_t>(x), ar = reinterpret_cast<uintptr_t>(R);
  const uintptr_t ap = reinterpret_cast<uintptr_t>(payload), an = reinterpret_cast<uintptr_t>(norms);
  return (ax % 16 == 0) && (stride % 8 == 0) && (ar % 16 == 0) && (ap % 4 == 0) && (an % 2 == 0);
}

int launch_encode_mfma(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                       const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                       void* stream, int n_cu) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t ntiles = (n_vec + 15) / 16;
  const int64_t waves_cap = (int64_t)n_cu * (s.N == 16 ? 8 : 4);
  const int64_t waves = ntiles < waves_cap ? ntiles : waves_cap;
  const int grid = (int)((waves + 3) / 4);
  const uint16_t* xb = static_cast<const uint16_t*>(x);
  if (s.N == 16)
    hipLaunchKernelGGL(encmf::encode_kernel16, dim3(grid), dim3(encmf::kThreads), 0, st, xb,
                       n_vec, stride, R, C, payload, norms);
  else
    hipLaunchKernelGGL(encmf::encode_kernel64, dim3(grid), dim3(encmf::kThreads), 0, st, xb,
                       n_vec, stride, R, C, payload, norms);
  return (int)hipGetLastError();
}

}  // namespace dev
}  // namespace fibq
