// Fused dequantisation + decode attention on the matrix cores, for the
// 6-bit sub-one-bit shape: d = 64, k = 8 (eight 8-dim blocks), G = 8 query
// heads per KV head, N = 64 codewords (Eq. lattn over the decoded cache of
// Sec. 3.1; scores and values in rotated space).  The 4-bit shape (N = 16)
// has its own kernel in attn_w4.hip.
//
// Per wavefront, 32 cached tokens per step (two 16-token tiles):
//   scores  S[t][.] = K_hat[t][:] . [q~_hi | q~_lo]  (v_mfma_f32_16x16x32_f16,
//           A = codeword rows gathered from an fp16 copy of the codebook in
//           LDS, 16 bytes per (token, block); the 16 output columns hold the
//           8 heads' products with the high and the low fp16 halves of the
//           rotated query, summed by one DPP add), so scores keep ~fp32
//           accuracy; a codebook that is not exactly representable in fp16
//           adds its residual rows (C - fp16(C)) times q~_hi;
//   softmax online, base 2 (q~ is pre-scaled by scale * log2 e); the running
//           maximum only moves when a token exceeds it (rare after the first
//           tiles); the norms enter through mixed-precision FMAs;
//   values  acc[(tile, h)][dims] += W[(tile, h)][tokens] V_hat[tokens][dims]
//           (v_mfma_f32_16x16x32_f16); rows 0-7 take the first tile's tokens,
//           rows 8-15 the second's, so every lane's softmax work is used; the
//           B operand (8 consecutive tokens of one dim) comes straight from
//           transposing LDS reads (ds_read_b64_tr_b16) of codeword rows.  The
//           value tiles' columns are the first (second) halves of four blocks,
//           so one row address serves two reads.
// Work is split into (group, 256-token chunk) items assigned contiguously to a
// persistent grid; a workgroup emits one partial state (m, l, acc) per group
// it touches, merged by log-sum-exp with one inverse rotation per head.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {

namespace fast {

constexpr int D = 64, K = 8, G = 8;
constexpr int kThreads = 256;   // 4 wavefronts
constexpr int kChunk = 256;     // tokens per work item (64 per wavefront)
constexpr int kMaxN = 64;
// persistent workgroups per compute unit: all must be resident at once; at
// ~136 VGPRs three wavefronts fit per SIMD, i.e. three 4-wavefront groups
constexpr int kWgPerCu = 3;
constexpr int kRec = G * (D + 2);  // floats per partial record: m[G], l[G], acc[G][D]

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

struct Plan {
  int64_t items, chunks_per_group;
  int wgs, slots;  // slots = partial records per workgroup
  size_t off_bq, off_qs, off_cb, off_rec, total;
};

static inline size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

static Plan make_plan(int64_t n_groups, int64_t T, int n_cu) {
  Plan p{};
  p.chunks_per_group = (T + kChunk - 1) / kChunk;
  if (p.chunks_per_group < 1) p.chunks_per_group = 1;
  p.items = n_groups * p.chunks_per_group;
  const int64_t cap = (int64_t)n_cu * kWgPerCu;
  p.wgs = (int)(p.items < cap ? p.items : cap);
  const int64_t per = (p.items + p.wgs - 1) / p.wgs;
  p.slots = (int)((per + p.chunks_per_group - 1) / p.chunks_per_group + 1);
  size_t off = 0;
  p.off_bq = off;
  off = al(off + (size_t)n_groups * 2 * 64 * 8 * 2);      // B operands of the rotated query
  p.off_qs = off;
  off = al(off + (size_t)n_groups * 4);                    // power-of-two query divisors
  p.off_cb = off;
  off = al(off + 2 * kMaxN * 8 * 2 + 16);                  // fp16 codebook hi, lo, flag
  p.off_rec = off;
  off = al(off + (size_t)p.wgs * p.slots * kRec * 4);
  p.total = off;
  return p;
}

// first item of workgroup w (contiguous, balanced assignment)
__host__ __device__ inline int64_t wg_first(int64_t w, int64_t items, int wgs) {
  return (w * items) / wgs;
}

// ----------------------------------------------------------------- prep ----
// One block per group: q~ = Pi q scaled by scale*log2(e), split into fp16
// hi + lo and written in the MFMA B-operand order; block 0 also writes the
// fp16 codebook (hi, residual lo) and a flag telling whether lo is nonzero.
__global__ __launch_bounds__(256) void prep_kernel(const void* __restrict__ q, int q_dtype,
                                                   const float* __restrict__ R,
                                                   const float* __restrict__ C, int N,
                                                   float qscale, _Float16* __restrict__ bq,
                                                   float* __restrict__ qsc,
                                                   _Float16* __restrict__ cb) {
  __shared__ float Rs[D][D + 1];  // padded: row reads by different threads hit different banks
  __shared__ float qs[G * D];
  __shared__ float qt[G * D];
  __shared__ float red[4];
  __shared__ int any_lo;
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  for (int i = tid; i < D * D; i += 256) Rs[i / D][i % D] = R[i];
  for (int i = tid; i < G * D; i += 256) {
    const int64_t src = g * G * D + i;
    float v;
    if (q_dtype == FIBQ_F32) v = static_cast<const float*>(q)[src];
    else if (q_dtype == FIBQ_F16) v = to_float(static_cast<const f16_t*>(q)[src]);
    else v = to_float(static_cast<const bf16_t*>(q)[src]);
    qs[i] = v;
  }
  if (tid == 0) any_lo = 0;
  __syncthreads();
  float amax = 0.0f;
  for (int e = tid; e < G * D; e += 256) {
    const int h = e / D, i = e % D;
    float s = 0.0f;
#pragma unroll 8
    for (int j = 0; j < D; ++j) s = fmaf(Rs[i][j], qs[h * D + j], s);
    qt[e] = s * qscale;
    amax = fmaxf(amax, fabsf(qt[e]));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  // power-of-two divisor keeping the binary16 parts of q~ in range (1 if none);
  // scores are then in units of 1 / sc and multiplied back before exp2
  const float top = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sc = 1.0f;
  if (top > 16384.0f) {
    int e2 = 0;
    frexpf(top / 16384.0f, &e2);
    sc = ldexpf(1.0f, e2);
  }
  const float inv = 1.0f / sc;
  if (tid == 0) qsc[g] = sc;
  // B operand of v_mfma_f32_16x16x32_f16 for K-step kappa (dims 32 kappa ..):
  // lane l holds B[k = 8 (l/16) + e][n = l % 16], column n < 8 -> hi of head n,
  // n >= 8 -> lo of head n - 8.
  for (int e = tid; e < 2 * 64 * 8; e += 256) {
    const int kap = e / 512, l = (e / 8) % 64, j = e % 8;
    const int n = l % 16, dim = 32 * kap + 8 * (l / 16) + j;
    const float v = qt[(n & 7) * D + dim] * inv;
    const _Float16 hi = (_Float16)v;
    const _Float16 out = (n < 8) ? hi : (_Float16)(v - (float)hi);
    bq[g * 1024 + e] = out;
  }
  if (g == 0) {
    for (int i = tid; i < kMaxN * K; i += 256) {
      const float c = (i < N * K) ? C[i] : 0.0f;
      const _Float16 hi = (_Float16)c;
      const _Float16 lo = (_Float16)(c - (float)hi);
      cb[i] = hi;
      cb[kMaxN * K + i] = lo;
      if ((float)lo != 0.0f) any_lo = 1;
    }
    __syncthreads();
    if (tid == 0) reinterpret_cast<int*>(cb + 2 * kMaxN * K)[0] = any_lo;
  }
}

__device__ __forceinline__ float dpp_ror8(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
}

__device__ __forceinline__ h4 tr_read(const unsigned char* lds_byte_addr) {
  s4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s4*)(lds_byte_addr));
  return __builtin_bit_cast(h4, r);
}

__device__ __forceinline__ float xmax(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, 64));
}
__device__ __forceinline__ float xsum(float v, int mask) { return v + __shfl_xor(v, mask, 64); }

// ----------------------------------------------------------------- main ----
// Raw loads of one wavefront's 64 tokens of a work item (two 32-token steps):
// payload words of the tokens whose codeword rows this lane gathers for the
// score MFMA (A rows) and for the transposing value reads (TR rows), and the
// fp16 norms of the four tokens whose softmax this lane computes.
struct Blk {
  uint32_t ka[4], kah[4], vr[4], vrh[4];  // [step * 2 + tile]
  uint32_t nk[4], nv[4];                  // [step * 2 + {0,1}] two fp16 norms per word
};

// Byte offset (index * 16) of the codeword row of block m.
// W = 4: rotate bits 4m .. 4m+3 onto bits 4 .. 7 and mask; sh = (4m - 4) mod 32.
__device__ __forceinline__ uint32_t row4(uint32_t v, uint32_t sh) {
  return __builtin_amdgcn_alignbit(v, v, sh) & 0xF0u;
}
__device__ __forceinline__ uint32_t row6(uint32_t lo, uint32_t hi, int m) {
  const uint64_t v = (uint64_t)lo | ((uint64_t)hi << 32);
  return ((uint32_t)(v >> (6 * m)) << 4) & 0x3F0u;
}

template <int W>
__device__ __forceinline__ uint32_t pay_lo(const uint8_t* base, int t, uint32_t& hi) {
  if (W == 4) {
    hi = 0;
    return reinterpret_cast<const uint32_t*>(base)[t];
  }
  const uint16_t* p = reinterpret_cast<const uint16_t*>(base) + 3 * t;
  hi = p[2];
  return (uint32_t)p[0] | ((uint32_t)p[1] << 16);
}

template <int W>
__global__ __launch_bounds__(kThreads) void main_kernel(
    const uint8_t* __restrict__ kp, const uint16_t* __restrict__ kn,
    const uint8_t* __restrict__ vp, const uint16_t* __restrict__ vn, int T, int64_t T_stride,
    int64_t items, int64_t cpg, int slots, const _Float16* __restrict__ bq,
    const float* __restrict__ qsc,
    const _Float16* __restrict__ cbg, float* __restrict__ rec) {
  constexpr int P = (W == 4) ? 4 : 6;
  __shared__ __align__(16) _Float16 cb[2 * kMaxN * K];     // hi rows, lo rows
  __shared__ float mstate[4][G], lstate[4][G];
  __shared__ float astate[4][G][D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g16 = lane >> 4, c = lane & 15;
  for (int i = tid; i < 2 * kMaxN * K; i += kThreads) cb[i] = cbg[i];
  const bool has_lo = reinterpret_cast<const int*>(cbg + 2 * kMaxN * K)[0] != 0;
  __syncthreads();

  const int64_t w = blockIdx.x;
  const int64_t i0 = wg_first(w, items, gridDim.x), i1 = wg_first(w + 1, items, gridDim.x);
  if (i0 >= i1) return;
  const int64_t first_group = i0 / cpg;
  // group bases of the norm planes are 8-byte aligned when T_stride % 4 == 0
  const bool norms_aligned = ((T_stride & 3) == 0) &&
                             ((reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn)) & 7) == 0;

  const int mytile = c >> 3;  // tile whose tokens this lane's softmax covers
  const unsigned char* cbhi = reinterpret_cast<const unsigned char*>(cb);
  const unsigned char* cblo = cbhi + kMaxN * K * 2;
  // lane constants: score rows use blocks g16, 4 + g16; value rows use blocks
  // (c & 3) and 4 + (c & 3) of the tokens 4 g16 + (c >> 2) (+16)
  const uint32_t shA = (4u * g16 - 4u) & 31u, shB = (4u * g16 + 12u) & 31u;
  const uint32_t shV0 = (4u * (c & 3) - 4u) & 31u, shV1 = (4u * (c & 3) + 12u) & 31u;
  const int offA = c, offT = 4 * g16 + (c >> 2), offS = 16 * mytile + 4 * g16;
  const int tmax = T - 1;

  // work items are visited in order; (group, chunk) advance incrementally
  // (no 64-bit division inside the loop)
  auto load = [&](int64_t grp, int chunk) -> Blk {
    Blk b;
    const int tok0 = chunk * kChunk + wave * (kChunk / 4);
    const uint8_t* kpg = kp + grp * T_stride * (int64_t)P;
    const uint8_t* vpg = vp + grp * T_stride * (int64_t)P;
    const uint16_t* kng = kn + grp * T_stride;
    const uint16_t* vng = vn + grp * T_stride;
    if (tok0 + 64 <= T) {  // whole block inside the group: no clamping
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int tb = tok0 + 32 * st;
        const uint8_t* kb = kpg + (size_t)tb * P;
        const uint8_t* vb = vpg + (size_t)tb * P;
        b.ka[2 * st] = pay_lo<W>(kb, offA, b.kah[2 * st]);
        b.ka[2 * st + 1] = pay_lo<W>(kb, offA + 16, b.kah[2 * st + 1]);
        b.vr[2 * st] = pay_lo<W>(vb, offT, b.vrh[2 * st]);
        b.vr[2 * st + 1] = pay_lo<W>(vb, offT + 16, b.vrh[2 * st + 1]);
        if (norms_aligned) {
          const uint2 k4 = *reinterpret_cast<const uint2*>(kng + tb + offS);
          const uint2 v4 = *reinterpret_cast<const uint2*>(vng + tb + offS);
          b.nk[2 * st] = k4.x; b.nk[2 * st + 1] = k4.y;
          b.nv[2 * st] = v4.x; b.nv[2 * st + 1] = v4.y;
        } else {
          const uint16_t* kk = kng + tb + offS;
          const uint16_t* vv = vng + tb + offS;
          b.nk[2 * st] = kk[0] | ((uint32_t)kk[1] << 16); b.nk[2 * st + 1] = kk[2] | ((uint32_t)kk[3] << 16);
          b.nv[2 * st] = vv[0] | ((uint32_t)vv[1] << 16); b.nv[2 * st + 1] = vv[2] | ((uint32_t)vv[3] << 16);
        }
      }
    } else {  // ragged end of a group: clamp every token into [0, T)
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int tb = tok0 + 32 * st;
        b.ka[2 * st] = pay_lo<W>(kpg, min(tb + offA, tmax), b.kah[2 * st]);
        b.ka[2 * st + 1] = pay_lo<W>(kpg, min(tb + offA + 16, tmax), b.kah[2 * st + 1]);
        b.vr[2 * st] = pay_lo<W>(vpg, min(tb + offT, tmax), b.vrh[2 * st]);
        b.vr[2 * st + 1] = pay_lo<W>(vpg, min(tb + offT + 16, tmax), b.vrh[2 * st + 1]);
        uint32_t kk[4], vv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int t = min(tb + offS + e, tmax);
          kk[e] = kng[t];
          vv[e] = vng[t];
        }
        b.nk[2 * st] = kk[0] | (kk[1] << 16); b.nk[2 * st + 1] = kk[2] | (kk[3] << 16);
        b.nv[2 * st] = vv[0] | (vv[1] << 16); b.nv[2 * st + 1] = vv[2] | (vv[3] << 16);
      }
    }
    return b;
  };

  int64_t cur_group = -1;
  h8 bq0 = {}, bq1 = {}, bqh0 = {}, bqh1 = {};
  f4 acc[4];  // [pair p = block quartet, half h of each block]: index 2p + h
  float m_run = -INFINITY, l_run = 0.0f;
  float qsg = 1.0f;  // the group's query divisor: scores are in units of 1 / qsg

  auto flush = [&](int64_t grp) {
    // combine rows (tile 0, h) and (tile 1, h): lanes g16 and g16 ^ 2
    float a[4][4];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
#pragma unroll
      for (int e = 0; e < 4; ++e) a[ti][e] = acc[ti][e] + __shfl_xor(acc[ti][e], 32, 64);
    // l: sum over the 8 lanes of each head (c and c^8, four row groups)
    float l = l_run;
    l = xsum(l, 8);
    l = xsum(l, 16);
    l = xsum(l, 32);
    if (g16 < 2) {  // rows 4 g16 + e = heads; column c of tile (p, h) is dim
                    // 8 (4p + c/4) + 4h + c%4
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            astate[wave][4 * g16 + e][8 * (4 * p + (c >> 2)) + 4 * hh + (c & 3)] = a[2 * p + hh][e];
    }
    if (lane < G) {
      mstate[wave][lane] = m_run * qsg;  // true log2 units
      lstate[wave][lane] = l;
    }
    __syncthreads();
    // merge the four wavefronts and write the record
    const int64_t slot = w * slots + (grp - first_group);
    float* r = rec + slot * kRec;
    for (int e = tid; e < G * D; e += kThreads) {
      const int h = e / D, dd = e % D;
      float M = -INFINITY;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) M = fmaxf(M, mstate[q4][h]);
      float s = 0.0f;
      if (M != -INFINITY) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float mq = mstate[q4][h];
          if (mq != -INFINITY) s = fmaf(astate[q4][h][dd], __builtin_amdgcn_exp2f(mq - M), s);
        }
      }
      r[2 * G + e] = s;
    }
    if (tid < G) {
      float M = -INFINITY;
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) M = fmaxf(M, mstate[q4][tid]);
      float s = 0.0f;
      if (M != -INFINITY) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float mq = mstate[q4][tid];
          if (mq != -INFINITY) s = fmaf(lstate[q4][tid], __builtin_amdgcn_exp2f(mq - M), s);
        }
      }
      r[tid] = M;
      r[G + tid] = s;
    }
    __syncthreads();
  };

  // compiled once per codebook kind (residual rows or not): the hot body
  // has no branch on it
  auto compute = [&](const Blk& b, int tok0, auto lo_tag) {
    constexpr bool HL = decltype(lo_tag)::value;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int tb = tok0 + 32 * st;
      if (tb >= T) break;
      const bool full = tb + 32 <= T;
      // ---- scores: two tiles x two K-steps (blocks g16 and 4 + g16)
      f4 s0 = {0, 0, 0, 0}, s1 = {0, 0, 0, 0};
      {
        const uint32_t k0 = b.ka[2 * st], k0h = b.kah[2 * st];
        const uint32_t k1 = b.ka[2 * st + 1], k1h = b.kah[2 * st + 1];
        uint32_t n00, n01, n10, n11;  // byte offsets of the rows
        if (W == 4) {
          n00 = row4(k0, shA); n01 = row4(k0, shB); n10 = row4(k1, shA); n11 = row4(k1, shB);
        } else {
          n00 = row6(k0, k0h, g16); n01 = row6(k0, k0h, 4 + g16);
          n10 = row6(k1, k1h, g16); n11 = row6(k1, k1h, 4 + g16);
        }
        const h8 a00 = *reinterpret_cast<const h8*>(cbhi + n00);
        const h8 a01 = *reinterpret_cast<const h8*>(cbhi + n01);
        const h8 a10 = *reinterpret_cast<const h8*>(cbhi + n10);
        const h8 a11 = *reinterpret_cast<const h8*>(cbhi + n11);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a00, bq0, s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a10, bq0, s1, 0, 0, 0);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a01, bq1, s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a11, bq1, s1, 0, 0, 0);
        if (HL) {
          const h8 b00 = *reinterpret_cast<const h8*>(cblo + n00);
          const h8 b01 = *reinterpret_cast<const h8*>(cblo + n01);
          const h8 b10 = *reinterpret_cast<const h8*>(cblo + n10);
          const h8 b11 = *reinterpret_cast<const h8*>(cblo + n11);
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b00, bqh0, s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b10, bqh0, s1, 0, 0, 0);
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b01, bqh1, s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_f16(b11, bqh1, s1, 0, 0, 0);
        }
      }
      // ---- this lane's (tile, head) scores for tokens ts .. ts+3, relative
      //      to the running maximum: t = S nu_K - m
      const int ts = tb + offS;
      float f4s[4], t4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float own = mytile ? s1[e] : s0[e];
        const float oth = mytile ? s0[e] : s1[e];
        f4s[e] = own + dpp_ror8(oth);  // hi + lo of the head
        const h2 nk2 = __builtin_bit_cast(h2, b.nk[2 * st + (e >> 1)]);
        t4[e] = fmaf(f4s[e], (float)nk2[e & 1], -m_run);
      }
      if (!full) {
#pragma unroll
        for (int e = 0; e < 4; ++e) t4[e] = (ts + e < T) ? t4[e] : -INFINITY;
      }
      const float tmx = fmaxf(fmaxf(t4[0], t4[1]), fmaxf(t4[2], t4[3]));
      if (__any(tmx > 0.0f)) {  // a token beats the running maximum (rare)
        float delta;
        if (m_run == -INFINITY) {  // first tokens of this group: t holds +inf
          float s[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const h2 nk2 = __builtin_bit_cast(h2, b.nk[2 * st + (e >> 1)]);
            s[e] = (full || ts + e < T) ? f4s[e] * (float)nk2[e & 1] : -INFINITY;
          }
          float mh = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
          mh = xmax(mh, 8);
          mh = xmax(mh, 16);
          mh = xmax(mh, 32);
#pragma unroll
          for (int e = 0; e < 4; ++e) t4[e] = s[e] - mh;
          m_run = mh;
          delta = INFINITY;  // alpha = 0 (nothing accumulated yet)
        } else {
          float mh = tmx;  // max over the 8 lanes of this head
          mh = xmax(mh, 8);
          mh = xmax(mh, 16);
          mh = xmax(mh, 32);
          delta = fmaxf(mh, 0.0f);
          m_run += delta;
#pragma unroll
          for (int e = 0; e < 4; ++e) t4[e] -= delta;
        }
        const float alpha = __builtin_amdgcn_exp2f(-delta * qsg);
        l_run *= alpha;
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // acc row 4 g16 + e belongs to head (4 g16 + e) & 7
          const float ar = __shfl(alpha, (4 * g16 + e) & 7, 64);
#pragma unroll
          for (int ti = 0; ti < 4; ++ti) acc[ti][e] *= ar;
        }
      }
      // ---- weights p nu_V as the value MFMA's A operand
      h2 w01, w23;
      {
        float p[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p[e] = __builtin_amdgcn_exp2f(t4[e] * qsg);  // exp2(-inf) = 0
          l_run += p[e];
        }
        const h2 nv01 = __builtin_bit_cast(h2, b.nv[2 * st]);
        const h2 nv23 = __builtin_bit_cast(h2, b.nv[2 * st + 1]);
        w01 = h2{(_Float16)(p[0] * (float)nv01[0]), (_Float16)(p[1] * (float)nv01[1])};
        w23 = h2{(_Float16)(p[2] * (float)nv23[0]), (_Float16)(p[3] * (float)nv23[1])};
      }
      const uint32_t u01 = __builtin_bit_cast(uint32_t, w01), u23 = __builtin_bit_cast(uint32_t, w23);
      const u4v awu = mytile ? u4v{0u, 0u, u01, u23} : u4v{u01, u23, 0u, 0u};
      const h8 aw = __builtin_bit_cast(h8, awu);
      // ---- values: tiles (pair p, half h); B from transposing reads, one row
      //      address per (token, pair) serving both halves
      {
        const uint32_t v0 = b.vr[2 * st], v0h = b.vrh[2 * st];
        const uint32_t v1 = b.vr[2 * st + 1], v1h = b.vrh[2 * st + 1];
        uint32_t r00, r01, r10, r11;  // [tile token][pair]
        if (W == 4) {
          r00 = row4(v0, shV0); r01 = row4(v0, shV1); r10 = row4(v1, shV0); r11 = row4(v1, shV1);
        } else {
          r00 = row6(v0, v0h, c & 3); r01 = row6(v0, v0h, 4 + (c & 3));
          r10 = row6(v1, v1h, c & 3); r11 = row6(v1, v1h, 4 + (c & 3));
        }
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          const uint32_t ra = pp ? r01 : r00, rb = pp ? r11 : r10;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const h4 b0 = tr_read(cbhi + ra + 8 * hh);
            const h4 b1 = tr_read(cbhi + rb + 8 * hh);
            const h8 bv = h8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
            acc[2 * pp + hh] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, bv, acc[2 * pp + hh], 0, 0, 0);
            if (HL) {  // residual rows of a codebook that is not binary16-exact
              const h4 d0 = tr_read(cblo + ra + 8 * hh);
              const h4 d1 = tr_read(cblo + rb + 8 * hh);
              const h8 dv = h8{d0[0], d0[1], d0[2], d0[3], d1[0], d1[1], d1[2], d1[3]};
              acc[2 * pp + hh] =
                  __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, dv, acc[2 * pp + hh], 0, 0, 0);
            }
          }
        }
      }
    }
  };

  int64_t grp = first_group;
  int chunk = (int)(i0 - first_group * cpg);
  Blk cur = load(grp, chunk);
  for (int64_t it = i0; it < i1; ++it) {
    if (grp != cur_group) {
      if (cur_group >= 0) flush(cur_group);
      cur_group = grp;
      qsg = qsc[grp];
      const _Float16* bqg = bq + grp * 1024;
      bq0 = *reinterpret_cast<const h8*>(bqg + lane * 8);
      bq1 = *reinterpret_cast<const h8*>(bqg + 512 + lane * 8);
      bqh0 = (c < 8) ? bq0 : h8{};  // hi columns only (for the residual rows)
      bqh1 = (c < 8) ? bq1 : h8{};
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) acc[ti] = f4{0, 0, 0, 0};
      m_run = -INFINITY;
      l_run = 0.0f;
    }
    int64_t ngrp = grp;
    int nchunk = chunk + 1;
    if (nchunk == cpg) {
      nchunk = 0;
      ++ngrp;
    }
    Blk nxt = cur;
    if (it + 1 < i1) nxt = load(ngrp, nchunk);  // prefetch the next item
    if (has_lo) compute(cur, chunk * kChunk + wave * (kChunk / 4), std::true_type{});
    else compute(cur, chunk * kChunk + wave * (kChunk / 4), std::false_type{});
    cur = nxt;
    grp = ngrp;
    chunk = nchunk;
  }
  flush(cur_group);
}

// ---------------------------------------------------------------- merge ----

__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ rec, int64_t items,
                                                    int wgs, int slots, int64_t cpg,
                                                    const float* __restrict__ R,
                                                    float* __restrict__ out) {
  // One block per group: log-sum-exp over the records of the workgroups whose
  // item ranges meet the group, then o = Pi^T (acc / l).  Thread t owns
  // outputs t + 256 u; for each chunk of kMergeMax contributors it loads every
  // value it needs before using any (one round of memory requests per chunk);
  // Pi is staged in LDS.
  constexpr int EPT = G * D / 256;  // output elements per thread
  constexpr int kMergeMax = 32 / EPT;  // contributors per round: as many as registers allow
  __shared__ __align__(16) float rs[D * D];
  __shared__ float ar[G * D];
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  if (items == 0) {  // no cached tokens: the output is zero
    for (int e = tid; e < G * D; e += 256) out[g * G * D + e] = 0.0f;
    return;
  }
  for (int e = tid; e < D * D / 4; e += 256)
    reinterpret_cast<float4*>(rs)[e] = reinterpret_cast<const float4*>(R)[e];
  // workgroups whose item range intersects [g cpg, (g + 1) cpg)
  int64_t wlo = (g * cpg * wgs) / items;
  while (wlo > 0 && wg_first(wlo, items, wgs) > g * cpg) --wlo;
  while (wlo + 1 < wgs && wg_first(wlo + 1, items, wgs) <= g * cpg) ++wlo;
  int64_t whi = wlo;
  while (whi + 1 < wgs && wg_first(whi + 1, items, wgs) < (g + 1) * cpg) ++whi;
  float M[EPT], L[EPT], a[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) { M[u] = -INFINITY; L[u] = 0.0f; a[u] = 0.0f; }
  for (int64_t base = wlo; base <= whi; base += kMergeMax) {
    float mk[kMergeMax][EPT], lk[kMergeMax][EPT], xk[kMergeMax][EPT];
#pragma unroll
    for (int k = 0; k < kMergeMax; ++k) {
      const int64_t w = base + k;
      const bool has = w <= whi;
      const float* rr =
          rec + ((int64_t)(has ? w : wlo) * slots + (g - wg_first(has ? w : wlo, items, wgs) / cpg)) * kRec;
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + 256 * u, h = e / D;
        mk[k][u] = has ? rr[h] : -INFINITY;
        lk[k][u] = has ? rr[G + h] : 0.0f;
        xk[k][u] = has ? rr[2 * G + e] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      float Mn = M[u];
#pragma unroll
      for (int k = 0; k < kMergeMax; ++k) Mn = fmaxf(Mn, mk[k][u]);
      if (Mn == -INFINITY) continue;
      const float fo = (M[u] == -INFINITY) ? 0.0f : exp2f(M[u] - Mn);
      L[u] *= fo;
      a[u] *= fo;
#pragma unroll
      for (int k = 0; k < kMergeMax; ++k) {
        const float f = (mk[k][u] == -INFINITY) ? 0.0f : exp2f(mk[k][u] - Mn);
        L[u] = fmaf(lk[k][u], f, L[u]);
        a[u] = fmaf(xk[k][u], f, a[u]);
      }
      M[u] = Mn;
    }
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int e = tid + 256 * u;
    ar[e] = (L[u] > 0.0f) ? a[u] / L[u] : 0.0f;
  }
  __syncthreads();
  for (int e = tid; e < G * D; e += 256) {  // o = Pi^T a; Pi columns read without conflicts
    const int h = e / D, j = e % D;
    float sacc = 0.0f;
#pragma unroll 16
    for (int i = 0; i < D; ++i) sacc = fmaf(rs[i * D + j], ar[h * D + i], sacc);
    out[g * G * D + e] = sacc;
  }
}

}  // namespace fast

bool attn_fast_applies(int G, const Shape& s) {
  // the 4-bit shape has its own kernel (attn_w4.hip)
  return s.d == 64 && s.k == 8 && G == 8 && s.w == 6;
}

// The grid is fixed at (at most) 256 x 4 workgroups, so the workspace size
// does not depend on the device.
size_t attn_fast_workspace_bytes(int64_t n_groups, int64_t T) {
  return fast::make_plan(n_groups, T, 256).total;
}

int launch_attn_fast(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                     const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int64_t T,
                     int64_t T_stride, const Shape& s, const float* R, const float* C,
                     float scale, float* out, void* ws, hipStream_t st) {
  // the same plan as the workspace query (sized for 256 CUs), so the record
  // slots always fit the caller's workspace
  const fast::Plan p = fast::make_plan(n_groups, T, 256);
  unsigned char* b = static_cast<unsigned char*>(ws);
  _Float16* bq = reinterpret_cast<_Float16*>(b + p.off_bq);
  float* qsc = reinterpret_cast<float*>(b + p.off_qs);
  _Float16* cb = reinterpret_cast<_Float16*>(b + p.off_cb);
  float* rec = reinterpret_cast<float*>(b + p.off_rec);
  const float qscale = scale * 1.4426950408889634f;  // base-2 softmax
  hipLaunchKernelGGL(fast::prep_kernel, dim3((unsigned)n_groups), dim3(256), 0, st, q, q_dtype, R,
                     C, s.N, qscale, bq, qsc, cb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  if (T > 0) {
    hipLaunchKernelGGL(fast::main_kernel<6>, dim3((unsigned)p.wgs), dim3(fast::kThreads), 0, st, kp,
                       kn, vp, vn, (int)T, T_stride, p.items, p.chunks_per_group, p.slots, bq, qsc,
                       cb, rec);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
  }
  hipLaunchKernelGGL(fast::merge_kernel, dim3((unsigned)n_groups), dim3(256), 0, st, rec,
                     T > 0 ? p.items : 0, T > 0 ? p.wgs : 0, p.slots, p.chunks_per_group, R, out);
  return (int)hipGetLastError();
}

}  // namespace dev
}  // namespace fibq
