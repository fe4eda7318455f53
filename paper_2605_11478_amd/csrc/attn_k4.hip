// Fused dequantisation + single-query decode attention on the matrix cores
// for block dimension k = 4 (Eq. lattn over the decoded cache of Sec. 3.1,
// evaluated in rotated space): d = 64 or 128 with 8- or 12-bit indices
// (N = 256 or 4096), G <= 8 query heads per KV head.
//
// Block dimension k = 2 with w = 4 or 6 bits (N = 16 or 64) runs through the
// same kernels: its payload, read as a stream of 2w-bit indices, is exactly
// the payload of a k = 4 code over the pair codebook whose row i + N j is
// (c_i, c_j) (index i of block 2p sits in the low w bits of pair p).  The
// prep kernel writes that N^2-row table instead of the codebook.
//
// Per wavefront, 32 cached tokens per step (two 16-token tiles):
//   loads   the payload of a token is read as four contiguous quarters of
//           P / 4 bytes, one per lane of a 4-lane set, so a wavefront's loads
//           cover 16 whole payloads per instruction (no lane reads bytes it
//           does not use).  The MFMA K slots are assigned to dimensions to
//           match: in the score product, lane group g (lanes 16 g .. 16 g + 15)
//           owns the blocks of quarter g; in the value product, the lane with
//           lane % 4 = a supplies rows of quarter a;
//   scores  S[t][.] = K_hat[t][:] . [q~_hi | q~_lo]  (v_mfma_f32_16x16x32_f16,
//           A = two gathered 4-dim codeword rows per lane from an fp16 copy of
//           the codebook in LDS; the 16 columns are the heads' products with
//           the binary16 high and low parts of the rotated query, summed by
//           one DPP add; a codebook that is not binary16-exact adds its
//           residual rows times q~_hi);
//   softmax online, base 2 (q~ carries scale * log2 e and, if needed, a power
//           of two that keeps it in binary16 range); the running maximum of a
//           head moves only when a token exceeds it;
//   values  acc[(tile, h)][dims] += W[(tile, h)][tokens] V_hat[tokens][dims]
//           (v_mfma_f32_16x16x32_f16; plus the residual rows when the
//           codebook is not binary16-exact), B from transposing LDS reads
//           (ds_read_b64_tr_b16: in each 16-lane row, lane 4 a + e receives
//           element e of the rows addressed by lanes a, a + 4, a + 8, a + 12).
// Units of 32 tokens over all groups laid end to end are split into equal
// contiguous ranges, one per wavefront; a wavefront writes one partial state
// (m, l, acc) per group it touches; the merge kernel combines them by
// log-sum-exp and applies Pi^T once per head.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace k4 {

constexpr int K = 4;
constexpr int kMaxG = 8;
constexpr int kMaxN = 4096;
constexpr int kWaves = 8, kThreads = 64 * kWaves;
constexpr int kStep = 32;  // tokens per unit
constexpr int kMinUnits = 1;

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

struct Plan {
  int64_t units;  // 32-token units over all groups
  int upg;        // units per group
  int waves, slots;
  size_t off_bq, off_qs, off_cb, off_rec, total;
};

static inline size_t al(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr int rec_floats(int D) { return kMaxG * (D + 2); }

static Plan make_plan(int64_t n_groups, int64_t T, int D, int N, int n_cu) {
  Plan p{};
  p.upg = (int)((T + kStep - 1) / kStep);
  if (p.upg < 1) p.upg = 1;
  p.units = n_groups * p.upg;
  // whole workgroups of kWaves wavefronts, at most two per compute unit, and
  // at least kMinUnits units per wavefront (fewer partial records to merge
  // for small caches)
  int64_t wgs = (p.units + kWaves * kMinUnits - 1) / (kWaves * kMinUnits);
  if (wgs > (int64_t)n_cu * 2) wgs = (int64_t)n_cu * 2;
  if (wgs < 1) wgs = 1;
  p.waves = (int)(wgs * kWaves);
  const int64_t per = (p.units + p.waves - 1) / p.waves;
  p.slots = (int)((per + p.upg - 1) / p.upg + 1);
  size_t off = 0;
  p.off_bq = off;
  off = al(off + (size_t)n_groups * (D / 32) * 64 * 8 * 2);
  p.off_qs = off;
  off = al(off + (size_t)n_groups * 4);
  p.off_cb = off;
  off = al(off + 2 * (size_t)N * K * 2 + 16);
  p.off_rec = off;
  off = al(off + (size_t)p.waves * p.slots * rec_floats(D) * 4);
  p.total = off;
  return p;
}

__host__ __device__ inline int64_t first_unit(int64_t w, int64_t units, int waves) {
  return (w * units) / waves;
}

// the wavefront whose unit range [first_unit(w), first_unit(w + 1)) holds u
__device__ inline int wave_of(int64_t u, int64_t units, int waves) {
  int64_t w = (u * waves) / units;
  while (w + 1 < waves && first_unit(w + 1, units, waves) <= u) ++w;
  while (w > 0 && first_unit(w, units, waves) > u) --w;
  return (int)w;
}

// ----------------------------------------------------------------- prep ----
// One block per group: q~ = Pi q * scale * log2(e) (divided by a power of two
// when an entry would exceed 2^14), split into binary16 hi + lo and written
// in the B-operand order of the score MFMA; block 0 also writes the binary16
// codebook (rows and residual rows) and a flag telling whether the residual
// is nonzero.
template <int D>
__global__ __launch_bounds__(256) void prep_kernel(const void* __restrict__ q, int q_dtype, int G,
                                                   const float* __restrict__ R,
                                                   const float* __restrict__ C, int N, int pair_n,
                                                   float qscale, _Float16* __restrict__ bq,
                                                   float* __restrict__ qsc,
                                                   _Float16* __restrict__ cb) {
  constexpr int NB = D / K, Q = NB / 4;  // blocks per payload quarter
  __shared__ float qs[kMaxG * D];
  __shared__ float qt[kMaxG * D];
  __shared__ float rt[D * (D + 1)];  // Pi^T, rows padded: conflict-free column reads
  __shared__ float red[4];
  __shared__ int any_lo;
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  for (int e = tid; e < D * D / 4; e += 256) {  // coalesced 16-byte reads of Pi's rows
    const float4 r4 = reinterpret_cast<const float4*>(R)[e];
    const int ri = (4 * e) / D, rj = (4 * e) % D;
    rt[(rj + 0) * (D + 1) + ri] = r4.x;
    rt[(rj + 1) * (D + 1) + ri] = r4.y;
    rt[(rj + 2) * (D + 1) + ri] = r4.z;
    rt[(rj + 3) * (D + 1) + ri] = r4.w;
  }
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
#pragma unroll 16
    for (int j = 0; j < D; ++j) s = fmaf(rt[j * (D + 1) + i], qs[h * D + j], s);
    qt[e] = s * qscale;
    amax = fmaxf(amax, fabsf(qt[e]));
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  const float top = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float sc = 1.0f;
  if (top > 16384.0f) {
    int e2 = 0;
    frexpf(top / 16384.0f, &e2);
    sc = ldexpf(1.0f, e2);
  }
  const float inv = 1.0f / sc;  // exact (power of two)
  if (tid == 0) qsc[g] = sc;
  // B operand of K-step kap: lane l holds B[k = 8 (l / 16) + e][n = l % 16];
  // the K slots of lane group gq are dims 4 (gq Q + 2 kap + e / 4) + e % 4;
  // column n < 8 is the high part of head n, n >= 8 the low part of head n - 8
  for (int x = tid; x < (D / 32) * 64 * 8; x += 256) {
    const int kap = x / 512, l = (x / 8) % 64, e = x % 8;
    const int n = l % 16, gq = l / 16, h = n & 7;
    const int dim = 4 * (gq * Q + 2 * kap + e / 4) + (e % 4);
    _Float16 o = (_Float16)0.0f;
    if (h < G) {
      const float v = qt[h * D + dim] * inv;
      const _Float16 hi = (_Float16)v;
      o = (n < 8) ? hi : (_Float16)(v - (float)hi);
    }
    bq[g * (D / 32) * 512 + x] = o;
  }
  // The binary16 table: N rows of 4 (k = 4), or the pair table of a k = 2
  // codebook with pair_n rows (entry e of row j is dim e % 2 of codeword
  // (e < 2 ? j % pair_n : j / pair_n)), converted by all blocks in slices.
  for (int64_t i = g * 256 + tid; i < (int64_t)N * K; i += (int64_t)gridDim.x * 256) {
    float c;
    if (pair_n > 0) {
      const int j = (int)(i >> 2), e = (int)(i & 3);
      const int src = (e < 2) ? (j % pair_n) : (j / pair_n);
      c = C[2 * src + (e & 1)];
    } else {
      c = C[i];
    }
    const _Float16 hi = (_Float16)c;
    cb[i] = hi;
    cb[N * K + i] = (_Float16)(c - (float)hi);
  }
  if (g == 0) {  // whether any residual row is nonzero: from the codebook itself
    const int n_c = pair_n > 0 ? 2 * pair_n : N * K;
    for (int i = tid; i < n_c; i += 256) {
      const float c = C[i];
      if ((float)(_Float16)(c - (float)(_Float16)c) != 0.0f) any_lo = 1;
    }
    __syncthreads();
    if (tid == 0) reinterpret_cast<int*>(cb + 2 * N * K)[0] = any_lo;
  }
}

// ----------------------------------------------------------------- main ----
__device__ __forceinline__ h4 tr_read(const unsigned char* lds_byte_addr) {
  s4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s4*)(lds_byte_addr));
  return __builtin_bit_cast(h4, r);
}
__device__ __forceinline__ float dpp_ror8(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
}
__device__ __forceinline__ float xmax(float v, int mask) {
  return fmaxf(v, __shfl_xor(v, mask, 64));
}
__device__ __forceinline__ float xsum(float v, int mask) { return v + __shfl_xor(v, mask, 64); }

// One lane's raw loads of a unit: a payload quarter of the token whose K rows
// it gathers in each tile, a quarter of the token whose V rows it addresses
// in each tile, and the binary16 norms of the four tokens of its softmax work.
template <int QW>
struct Unit {
  uint32_t kq[2][QW], vq[2][QW];  // [tile][dword of the quarter]
  uint32_t nk[2], nv[2];          // two binary16 norms per word
};

// index of local block b of a quarter (w-bit indices, little-endian)
template <int QW, int W>
__device__ __forceinline__ uint32_t qidx(const uint32_t (&qq)[QW], int b) {
  if (W == 8) return (qq[b >> 2] >> (8 * (b & 3))) & 0xFFu;
  // W == 12: bits 12 b .. 12 b + 11 of the quarter
  const int bit = 12 * b, wd = bit >> 5, sh = bit & 31;
  uint32_t v = qq[wd] >> sh;
  if (sh > 20) v |= qq[wd + 1] << (32 - sh);
  return v & 0xFFFu;
}

template <int D, int W>
__global__ __launch_bounds__(kThreads) void main_kernel(
    const uint8_t* __restrict__ kp, const uint16_t* __restrict__ kn,
    const uint8_t* __restrict__ vp, const uint16_t* __restrict__ vn, int G, int T,
    int64_t T_stride, int N, int64_t units, int upg, int slots,
    const _Float16* __restrict__ bq, const float* __restrict__ qsc,
    const _Float16* __restrict__ cbg, float* __restrict__ rec) {
  constexpr int NB = D / K, Q = NB / 4;     // blocks per quarter
  constexpr int P = NB * W / 8, QB = P / 4;  // payload bytes, bytes per quarter
  constexpr int QW = (QB + 3) / 4;           // dwords holding a quarter
  constexpr int KS = D / 32;                 // score K-steps
  constexpr int VM = D / 16;                 // value MFMAs (16 dims each)
  constexpr int REC = rec_floats(D);
  // quarters are whole dwords, except d = 64 with 12-bit indices (6 bytes,
  // read as three 16-bit halves)
  static_assert(QB % 4 == 0 || QB == 6, "unsupported payload quarter");
  extern __shared__ __align__(16) unsigned char smem[];  // codebook rows hi [N][4], lo [N][4]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g16 = lane >> 4, c = lane & 15;
  for (int i = tid; i < N; i += kThreads)
    reinterpret_cast<uint4*>(smem)[i] = reinterpret_cast<const uint4*>(cbg)[i];
  const bool has_lo = reinterpret_cast<const int*>(cbg + 2 * N * K)[0] != 0;
  __syncthreads();
  const unsigned char* cbhi = smem;
  const unsigned char* cblo = smem + (size_t)N * K * 2;

  const int nwaves = gridDim.x * kWaves;
  const int64_t w = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t u0 = first_unit(w, units, nwaves), u1 = first_unit(w + 1, units, nwaves);
  if (u0 >= u1) return;
  const int64_t g_first = u0 / upg;
  const bool norms_aligned = ((T_stride & 3) == 0) &&
                             ((reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn)) & 7) == 0;
  const int mytile = c >> 3;                     // tile of this lane's softmax tokens
  const int sm_tok = 16 * mytile + 4 * g16;      // first of its four tokens (unit-relative)
  const int kq_tok = c, kq_q = g16;              // K loads: token c of each tile, quarter g16
  const int vq_tok = 4 * g16 + (c >> 2), vq_q = c & 3;  // V loads: quarter c % 4

  auto load = [&](int64_t grp, int step) -> Unit<QW> {
    Unit<QW> b;
    const int tb = step * kStep;
    const uint8_t* kpg = kp + grp * T_stride * (int64_t)P;
    const uint8_t* vpg = vp + grp * T_stride * (int64_t)P;
    const uint16_t* kng = kn + grp * T_stride;
    const uint16_t* vng = vn + grp * T_stride;
    const int tm = T - 1;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int tk = min(tb + 16 * t + kq_tok, tm), tv = min(tb + 16 * t + vq_tok, tm);
      if (QB % 4 == 0) {
        const uint32_t* ks = reinterpret_cast<const uint32_t*>(kpg + (size_t)tk * P + kq_q * QB);
        const uint32_t* vs = reinterpret_cast<const uint32_t*>(vpg + (size_t)tv * P + vq_q * QB);
#pragma unroll
        for (int i = 0; i < QW; ++i) { b.kq[t][i] = ks[i]; b.vq[t][i] = vs[i]; }
      } else {
        const uint16_t* ks = reinterpret_cast<const uint16_t*>(kpg + (size_t)tk * P + kq_q * QB);
        const uint16_t* vs = reinterpret_cast<const uint16_t*>(vpg + (size_t)tv * P + vq_q * QB);
        b.kq[t][0] = (uint32_t)ks[0] | ((uint32_t)ks[1] << 16);
        b.kq[t][1] = ks[2];
        b.vq[t][0] = (uint32_t)vs[0] | ((uint32_t)vs[1] << 16);
        b.vq[t][1] = vs[2];
      }
    }
    const int ts = tb + sm_tok;
    if (norms_aligned && ts + 4 <= T) {
      const uint2 k4v = *reinterpret_cast<const uint2*>(kng + ts);
      const uint2 v4v = *reinterpret_cast<const uint2*>(vng + ts);
      b.nk[0] = k4v.x; b.nk[1] = k4v.y; b.nv[0] = v4v.x; b.nv[1] = v4v.y;
    } else {
      uint32_t kk[4], vv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = min(ts + e, tm);
        kk[e] = kng[t];
        vv[e] = vng[t];
      }
      b.nk[0] = kk[0] | (kk[1] << 16); b.nk[1] = kk[2] | (kk[3] << 16);
      b.nv[0] = vv[0] | (vv[1] << 16); b.nv[1] = vv[2] | (vv[3] << 16);
    }
    return b;
  };

  h8 bqv[KS], bqh[KS];
  f4 acc[VM];
  float m_run = -INFINITY, l_run = 0.0f, qsg = 1.0f;
  int64_t cur_group = -1;

  auto flush = [&](int64_t grp) {
    // rows (tile 0, h) and (tile 1, h) sit in lanes l and l ^ 32
    float l = l_run;
    l = xsum(l, 8);
    l = xsum(l, 16);
    l = xsum(l, 32);
    float* r = rec + ((size_t)w * slots + (size_t)(grp - g_first)) * REC;
#pragma unroll
    for (int mu = 0; mu < VM; ++mu) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = acc[mu][e] + __shfl_xor(acc[mu][e], 32, 64);
        // row 4 g16 + e is head 4 g16 + e; column c is dim
        // 4 ((c / 4) (D / 16) + mu) + c % 4
        const int h = 4 * g16 + e;
        if (g16 < 2 && h < G) r[2 * kMaxG + h * D + 4 * ((c >> 2) * (D / 16) + mu) + (c & 3)] = a;
      }
    }
    if (lane < G) {
      r[lane] = m_run * qsg;  // true log2 units
      r[kMaxG + lane] = l;
    }
  };

  // compiled once per codebook kind (residual rows or not): the hot body
  // has no branch on it
  auto compute = [&](const Unit<QW>& b, int tb, auto lo_tag) {
    constexpr bool HL = decltype(lo_tag)::value;
    const bool full = tb + kStep <= T;
    // ---- scores: two tiles x KS K-steps
    f4 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      s[t] = f4{0, 0, 0, 0};
#pragma unroll
      for (int kap = 0; kap < KS; ++kap) {
        const uint32_t r0 = qidx<QW, W>(b.kq[t], 2 * kap) * 8u;
        const uint32_t r1 = qidx<QW, W>(b.kq[t], 2 * kap + 1) * 8u;
        const h4 a0 = *reinterpret_cast<const h4*>(cbhi + r0);
        const h4 a1 = *reinterpret_cast<const h4*>(cbhi + r1);
        const h8 av = h8{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
        s[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bqv[kap], s[t], 0, 0, 0);
        if (HL) {
          const h4 d0 = *reinterpret_cast<const h4*>(cblo + r0);
          const h4 d1 = *reinterpret_cast<const h4*>(cblo + r1);
          const h8 dv = h8{d0[0], d0[1], d0[2], d0[3], d1[0], d1[1], d1[2], d1[3]};
          s[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(dv, bqh[kap], s[t], 0, 0, 0);
        }
      }
    }
    // ---- this lane's (tile, head) scores for its four tokens, relative to
    //      the running maximum: t = S nu_K - m
    const int ts = tb + sm_tok;
    float f4s[4], t4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float own = mytile ? s[1][e] : s[0][e];
      const float oth = mytile ? s[0][e] : s[1][e];
      f4s[e] = own + dpp_ror8(oth);  // hi + lo parts of the head
      const h2 nk2 = __builtin_bit_cast(h2, b.nk[e >> 1]);
      t4[e] = fmaf(f4s[e], (float)nk2[e & 1], -m_run);
    }
    if (!full) {
#pragma unroll
      for (int e = 0; e < 4; ++e) t4[e] = (ts + e < T) ? t4[e] : -INFINITY;
    }
    const float tmx = fmaxf(fmaxf(t4[0], t4[1]), fmaxf(t4[2], t4[3]));
    if (__any(tmx > 0.0f)) {  // a token beats the running maximum
      float delta;
      if (m_run == -INFINITY) {  // first tokens of this group for this wavefront
        float sv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const h2 nk2 = __builtin_bit_cast(h2, b.nk[e >> 1]);
          sv[e] = (full || ts + e < T) ? f4s[e] * (float)nk2[e & 1] : -INFINITY;
        }
        float mh = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
        mh = xmax(mh, 8);
        mh = xmax(mh, 16);
        mh = xmax(mh, 32);
#pragma unroll
        for (int e = 0; e < 4; ++e) t4[e] = sv[e] - mh;
        m_run = mh;
        delta = INFINITY;  // nothing accumulated yet
      } else {
        float mh = tmx;
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
      for (int e = 0; e < 4; ++e) {  // accumulator row 4 g16 + e belongs to head (4 g16 + e) & 7
        const float ar = __shfl(alpha, (4 * g16 + e) & 7, 64);
#pragma unroll
        for (int mu = 0; mu < VM; ++mu) acc[mu][e] *= ar;
      }
    }
    // ---- weights p nu_V (binary16) as the value MFMA's A operand
    float p[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p[e] = __builtin_amdgcn_exp2f(t4[e] * qsg);  // exp2(-inf) = 0
      l_run += p[e];
    }
    const h2 nv01 = __builtin_bit_cast(h2, b.nv[0]);
    const h2 nv23 = __builtin_bit_cast(h2, b.nv[1]);
    const h2 w01 = h2{(_Float16)(p[0] * (float)nv01[0]), (_Float16)(p[1] * (float)nv01[1])};
    const h2 w23 = h2{(_Float16)(p[2] * (float)nv23[0]), (_Float16)(p[3] * (float)nv23[1])};
    const uint32_t u01 = __builtin_bit_cast(uint32_t, w01), u23 = __builtin_bit_cast(uint32_t, w23);
    const h8 aw = __builtin_bit_cast(h8, mytile ? u4v{0u, 0u, u01, u23} : u4v{u01, u23, 0u, 0u});
    // ---- values: MFMA mu covers local block mu of every quarter
#pragma unroll
    for (int mu = 0; mu < VM; ++mu) {
      const uint32_t ra = qidx<QW, W>(b.vq[0], mu) * 8u;
      const uint32_t rb = qidx<QW, W>(b.vq[1], mu) * 8u;
      const h4 b0 = tr_read(cbhi + ra);
      const h4 b1 = tr_read(cbhi + rb);
      const h8 bv = h8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
      acc[mu] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, bv, acc[mu], 0, 0, 0);
      if (HL) {  // residual rows of a codebook that is not binary16-exact
        const h4 d0 = tr_read(cblo + ra);
        const h4 d1 = tr_read(cblo + rb);
        const h8 dv = h8{d0[0], d0[1], d0[2], d0[3], d1[0], d1[1], d1[2], d1[3]};
        acc[mu] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, dv, acc[mu], 0, 0, 0);
      }
    }
  };

  int64_t grp = g_first;
  int step = (int)(u0 - g_first * upg);
  Unit<QW> cur = load(grp, step);
  for (int64_t it = u0; it < u1; ++it) {
    if (grp != cur_group) {
      if (cur_group >= 0) flush(cur_group);
      cur_group = grp;
      qsg = qsc[grp];
      const _Float16* bqg = bq + grp * KS * 512;
#pragma unroll
      for (int kap = 0; kap < KS; ++kap) {
        bqv[kap] = *reinterpret_cast<const h8*>(bqg + kap * 512 + lane * 8);
        bqh[kap] = (c < 8) ? bqv[kap] : h8{};  // high parts only (residual rows)
      }
#pragma unroll
      for (int mu = 0; mu < VM; ++mu) acc[mu] = f4{0, 0, 0, 0};
      m_run = -INFINITY;
      l_run = 0.0f;
    }
    int64_t ngrp = grp;
    int nstep = step + 1;
    if (nstep == upg) {
      nstep = 0;
      ++ngrp;
    }
    Unit<QW> nxt = cur;
    if (it + 1 < u1) nxt = load(ngrp, nstep);  // prefetch the next unit
    if (has_lo) compute(cur, step * kStep, std::true_type{});
    else compute(cur, step * kStep, std::false_type{});
    cur = nxt;
    grp = ngrp;
    step = nstep;
  }
  flush(cur_group);
}

// ---------------------------------------------------------------- merge ----

template <int D>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ rec, int64_t units,
                                                    int waves, int slots, int upg, int G,
                                                    const float* __restrict__ R,
                                                    float* __restrict__ out) {
  // One block per group: log-sum-exp over the records of the wavefronts whose
  // unit ranges meet the group, then o = Pi^T (acc / l).  The threads form S
  // stripes of 256 / S (S = 4, 2, 1 as G D <= 64, <= 128, larger); stripe s
  // takes contributors s, s + S, ... and its thread t owns outputs
  // t + (256 / S) u; the stripes' partial states are then combined in LDS.
  // For each round of kMergeMax contributors a thread loads every value it
  // needs (m and l of its heads, its acc entries) before using any, so a
  // round costs one trip to memory; absent contributors are skipped; Pi is
  // staged in LDS.
  constexpr int REC = rec_floats(D);
  constexpr int EPT = kMaxG * D / 256;  // output elements per thread (at most)
  constexpr int kMergeMax = 32 / EPT;  // contributors per round: as many as registers allow
  __shared__ __align__(16) float rs[D * D];
  __shared__ float ar[kMaxG * D];
  __shared__ float sp[3][256];  // stripes' (m, l, acc) when S > 1 (S G D <= 256)
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  if (units == 0) {  // no cached tokens: the output is zero
    for (int e = tid; e < G * D; e += 256) out[g * G * D + e] = 0.0f;
    return;
  }
  for (int e = tid; e < D * D / 4; e += 256)
    reinterpret_cast<float4*>(rs)[e] = reinterpret_cast<const float4*>(R)[e];
  const int GD = G * D;
  const int S = GD <= 64 ? 4 : (GD <= 128 ? 2 : 1);
  const int TS = 256 / S, st = tid / TS, lt = tid % TS;
  const int wlo = wave_of(g * upg, units, waves), whi = wave_of((g + 1) * upg - 1, units, waves);
  // the first contributor's record slot (the fallback for contributors past
  // the last one, so that no address leaves the workspace)
  const int64_t slot_lo =
      (int64_t)wlo * slots + (g - first_unit(wlo, units, waves) / upg);
  float M[EPT], L[EPT], a[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) { M[u] = -INFINITY; L[u] = 0.0f; a[u] = 0.0f; }
  for (int base = wlo + st; base <= whi; base += S * kMergeMax) {
    float mk[kMergeMax][EPT], lk[kMergeMax][EPT], xk[kMergeMax][EPT];
    const int nk = (whi - base) / S + 1;  // contributors left for this stripe (uniform)
#pragma unroll
    for (int k = 0; k < kMergeMax; ++k) {
      if (k >= nk) {
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
          mk[k][u] = -INFINITY;
          lk[k][u] = 0.0f;
          xk[k][u] = 0.0f;
        }
        continue;
      }
      const int wv = base + S * k;
      const int64_t f0 = ((int64_t)wv * units) / waves;
      const int64_t f1 = ((int64_t)(wv + 1) * units) / waves;
      const bool has = wv <= whi && f0 < f1;  // a wavefront with an empty range wrote nothing
      const float* rr =
          rec + (has ? (int64_t)wv * slots + (g - f0 / upg) : slot_lo) * REC;
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = lt + TS * u, h = e / D;
        const bool ok = has && e < GD;
        mk[k][u] = ok ? rr[h] : -INFINITY;
        lk[k][u] = ok ? rr[kMaxG + h] : 0.0f;
        xk[k][u] = ok ? rr[2 * kMaxG + e] : 0.0f;
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
  if (S == 1) {
#pragma unroll
    for (int u = 0; u < EPT; ++u) {
      const int e = lt + TS * u;
      if (e < GD) ar[e] = (L[u] > 0.0f) ? a[u] / L[u] : 0.0f;
    }
  } else {
    // S G D <= 256 and G D <= TS: one element per thread (u = 0)
    if (lt < GD) {
      sp[0][st * GD + lt] = M[0];
      sp[1][st * GD + lt] = L[0];
      sp[2][st * GD + lt] = a[0];
    }
    __syncthreads();
    if (st == 0 && lt < GD) {
      float Mn = -INFINITY;
      for (int q = 0; q < S; ++q) Mn = fmaxf(Mn, sp[0][q * GD + lt]);
      float Ls = 0.0f, As = 0.0f;
      if (Mn != -INFINITY) {
        for (int q = 0; q < S; ++q) {
          const float mq = sp[0][q * GD + lt];
          const float f = (mq == -INFINITY) ? 0.0f : exp2f(mq - Mn);
          Ls = fmaf(sp[1][q * GD + lt], f, Ls);
          As = fmaf(sp[2][q * GD + lt], f, As);
        }
      }
      ar[lt] = (Ls > 0.0f) ? As / Ls : 0.0f;
    }
  }
  __syncthreads();
  for (int e = tid; e < GD; e += 256) {  // o = Pi^T a; Pi columns read without conflicts
    const int h = e / D, j = e % D;
    float sacc = 0.0f;
#pragma unroll 16
    for (int i = 0; i < D; ++i) sacc = fmaf(rs[i * D + j], ar[h * D + i], sacc);
    out[g * G * D + e] = sacc;
  }
}

}  // namespace k4

// the k = 4 shape a k = 2 code (w = 4 or 6) is read as: pairs of blocks with
// 2w-bit indices over the N^2-row pair codebook
static Shape k4_shape(const Shape& s) {
  if (s.k != 2) return s;
  return Shape{s.d, 4, s.N * s.N, 2 * s.w, s.P};
}

bool attn_k4_applies(int G, const Shape& s0) {
  if (G < 1 || G > k4::kMaxG) return false;
  if (s0.k == 2 && !(s0.w == 4 || s0.w == 6)) return false;
  const Shape s = k4_shape(s0);
  if (s.k != 4 || s.N > k4::kMaxN) return false;
  return (s.d == 64 || s.d == 128) && (s.w == 8 || s.w == 12);
}

size_t attn_k4_workspace_bytes(int64_t n_groups, int64_t T, const Shape& s0) {
  const Shape s = k4_shape(s0);
  return k4::make_plan(n_groups, T, s.d, s.N, 256).total;
}

int launch_attn_k4(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                   const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int G, int64_t T,
                   int64_t T_stride, const Shape& s0, const float* R, const float* C, float scale,
                   float* out, void* ws, hipStream_t st) {
  const Shape s = k4_shape(s0);
  const int pair_n = s0.k == 2 ? s0.N : 0;
  // the same plan as the workspace query (sized for 256 CUs)
  const k4::Plan p = k4::make_plan(n_groups, T, s.d, s.N, 256);
  unsigned char* b = static_cast<unsigned char*>(ws);
  _Float16* bq = reinterpret_cast<_Float16*>(b + p.off_bq);
  float* qsc = reinterpret_cast<float*>(b + p.off_qs);
  _Float16* cb = reinterpret_cast<_Float16*>(b + p.off_cb);
  float* rec = reinterpret_cast<float*>(b + p.off_rec);
  const float qscale = scale * 1.4426950408889634f;  // base-2 softmax
  const unsigned ng = (unsigned)n_groups;
  const int wgs = p.waves / k4::kWaves;
  const size_t lds = 2 * (size_t)s.N * k4::K * 2;
  hipError_t e = hipSuccess;
#define FIBQ_K4_CASE(DD, WW)                                                                     \
  if (s.d == DD && s.w == WW) {                                                                  \
    hipLaunchKernelGGL(k4::prep_kernel<DD>, dim3(ng), dim3(256), 0, st, q, q_dtype, G, R, C, s.N, \
                       pair_n, qscale, bq, qsc, cb);                                              \
    if ((e = hipGetLastError()) != hipSuccess) return (int)e;                                    \
    if (T > 0) {                                                                                  \
      auto kern = k4::main_kernel<DD, WW>;                                                        \
      if (lds > 65536) { /* above the default dynamic LDS limit */                                \
        e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,    \
                                (int)lds);                                                        \
        if (e != hipSuccess) return (int)e;                                                       \
      }                                                                                           \
      hipLaunchKernelGGL(kern, dim3((unsigned)wgs), dim3(k4::kThreads), lds, st, kp, kn, vp, vn,  \
                         G, (int)T, T_stride, s.N, p.units, p.upg, p.slots, bq, qsc, cb, rec);    \
      if ((e = hipGetLastError()) != hipSuccess) return (int)e;                                  \
    }                                                                                             \
    hipLaunchKernelGGL(k4::merge_kernel<DD>, dim3(ng), dim3(256), 0, st, rec, T > 0 ? p.units : 0, \
                       p.waves, p.slots, p.upg, G, R, out);                                       \
    return (int)hipGetLastError();                                                                \
  }
  FIBQ_K4_CASE(64, 8) FIBQ_K4_CASE(64, 12) FIBQ_K4_CASE(128, 8) FIBQ_K4_CASE(128, 12)
#undef FIBQ_K4_CASE
  return (int)hipErrorInvalidValue;
}

}  // namespace dev
}  // namespace fibq
