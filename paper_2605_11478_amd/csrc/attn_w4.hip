// Fused dequantisation + single-query decode attention for the 4-bit shape
// d = 64, k = 8, N = 16 (b = 1/2), G = 8 query heads per KV head: Eq. lattn
// over the decoded cache of Sec. 3.1, evaluated in rotated space (the rotated
// query against codeword rows scaled by the stored norms; one inverse
// rotation per head at the end).
//
// One 1024-thread workgroup per compute unit owns a contiguous range of
// 64-token units (all groups laid end to end); its 16 wavefronts claim units
// from an LDS counter.  Per 32-token step of a wavefront:
//
//   scores   S^T[r][t] = Q[r][:] . C_hat[t][:]  (v_mfma_f32_16x16x32_f16):
//            A = the rotated query, row r = (head r/2, part r%2) with part 0
//            its binary16 rounding and part 1 the binary16 rounding of the
//            remainder; B = codeword rows gathered from a 256-byte table in
//            LDS (every row occupies its own banks, so any gather is
//            conflict-free).  Each lane ends up with both parts of two heads
//            for one token, so the two parts are summed in-lane.
//            Addresses: each lane loads the payload byte that holds its two
//            blocks' 4-bit indices; high nibble -> (x & 0xF0), low nibble ->
//            (x << 4) & 0xF0, i.e. one instruction per row address.
//   softmax  base 2 (the query carries scale * log2 e), online; the norms
//            enter through mixed-precision FMAs; weights p are rounded to
//            binary16 once, and both the value weights (p * nu_V, packed
//            binary16 multiply) and the running sum l (fp32 dot of the
//            rounded p) use that rounded p.
//   values   O[h][:] += W[h][t] V_hat[t][:]  (v_mfma_f32_16x16x32_f16):
//            the weights go through a 512-byte per-wavefront LDS buffer
//            (written as packed pairs, read back as matrix rows), B comes
//            from transposing reads (ds_read_b64_tr_b16) of codeword rows.
//
// Loads: one global_load_lds_dwordx4 per unit moves its K and V payload
// words and both norm planes (768 bytes) into a 4-slot per-wavefront LDS
// ring; lanes then read their bytes from LDS.  (Per-lane byte loads from
// HBM cost one vector-memory instruction per 64 bytes and cap the stream
// far below the memory bandwidth.)  Units at a ragged group end, or strides
// that break the 16-byte alignment of the copies, are loaded per lane.
//
// At the end of each group segment the workgroup merges its 16 wavefront
// states (log-sum-exp) and writes one record; the merge kernel combines the
// records of a group and applies Pi^T.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace w4 {

constexpr int D = 64, K = 8, G = 8, NC = 16;
constexpr int kWaves = 16;                // at most 16 (two per lane group in the state merge)
constexpr int kThreads = 64 * kWaves;
constexpr int kUnit = 128;                // tokens per claim (two 64-token sub-units)
constexpr int kSub = 64;                  // tokens per sub-unit (two 32-token steps)
constexpr int kRec = G * (D + 2);         // floats per record: m[G], l[G], acc[G][D]
constexpr int kMaxWgs = 256;              // workgroups (one per compute unit)
constexpr int kQop = 2 * 64 * 8;          // binary16 query operand entries per group
// Loaded HBM latency is several microseconds, so each compute unit keeps
// about 100 KB of copies in flight: 4 slots of one unit per wavefront.
constexpr int kDepth = 4;                 // LDS ring slots per wavefront
constexpr int kSlot = kUnit * 12;         // K, V words (4 B) and K, V norms (2 B) per token
constexpr int kWRow = 80;                 // bytes per row of a weight buffer (64 + pad)
constexpr int kWBuf = G * kWRow;          // one weight buffer W[h][t] (binary16)
// The running maximum m of a head is a reference, not necessarily the true
// maximum: it is only raised when a score exceeds it by more than kLag (log2
// units), so weights p = 2^(s - m) stay below 2^kLag (exact in binary16) and
// the costly rescaling is rare.  Units whose V norms could overflow p * nu_V
// in binary16 use a zero lag.
constexpr float kLag = 8.0f;
constexpr unsigned short kNuLagBits = 0x5BF8;  // binary16 255.0 (<= 65504 / 2^kLag)
constexpr float kQMax = 16384.0f;         // query entries are scaled below this
constexpr int kFusedGroups = 4;           // groups per workgroup in the one-launch form

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

struct Plan {
  int64_t units;  // 64-token units over all groups
  int upg;        // units per group
  int wgs, slots; // workgroups, records per workgroup
  size_t off_q, off_qs, off_cb, off_rec, total;
};

static inline size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

static Plan make_plan(int64_t n_groups, int64_t T) {
  Plan p{};
  p.upg = (int)((T + kUnit - 1) / kUnit);
  if (p.upg < 1) p.upg = 1;
  p.units = n_groups * p.upg;
  p.wgs = (int)(p.units < kMaxWgs ? p.units : kMaxWgs);
  if (p.wgs < 1) p.wgs = 1;
  const int64_t upw = (p.units + p.wgs - 1) / p.wgs;
  p.slots = (int)((upw + p.upg - 1) / p.upg + 1);
  size_t off = 0;
  p.off_q = off;
  off = al(off + (size_t)n_groups * kQop * 2);
  p.off_qs = off;
  off = al(off + (size_t)n_groups * 4);
  p.off_cb = off;
  off = al(off + 2 * NC * K * 2 + 16);
  p.off_rec = off;
  off = al(off + (size_t)p.wgs * p.slots * kRec * 4);
  p.total = off;
  return p;
}

__host__ __device__ inline int64_t first_unit(int64_t w, int64_t units, int wgs) {
  return (w * units) / wgs;
}

// workgroup whose unit range contains unit u
__device__ inline int wg_of(int64_t u, int64_t units, int wgs) {
  int64_t w = (u * wgs) / units;
  while (w + 1 < wgs && first_unit(w + 1, units, wgs) <= u) ++w;
  while (w > 0 && first_unit(w, units, wgs) > u) --w;
  return (int)w;
}

// ----------------------------------------------------------------- prep ----
// One block per group: q~ = Pi q * scale * log2(e) (divided by a power of two
// 2^s when an entry would exceed kQMax in binary16), split into binary16
// parts and written in the A-operand order of the score MFMA.  Block 0 also
// writes the binary16 codebook (rows and
// residual rows) and a flag telling whether the residual is nonzero.
__global__ __launch_bounds__(256) void prep_kernel(const void* __restrict__ q, int q_dtype,
                                                   const float* __restrict__ R,
                                                   const float* __restrict__ C, float qscale,
                                                   _Float16* __restrict__ qop,
                                                   float* __restrict__ qsc,
                                                   _Float16* __restrict__ cb,
                                                   float* __restrict__ out, int zero_out) {
  __shared__ __align__(16) float qs[G * D];
  __shared__ float qt[G * D];
  __shared__ float rt[D * (D + 1)];  // Pi^T, rows padded: conflict-free column reads
  __shared__ float red[4];
  __shared__ int any_lo;
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  // this thread's outputs: dim i of heads hq and hq + 4, from row i of Pi
  const int i = tid & (D - 1), hq = tid >> 6;
  for (int e = tid; e < D * D / 4; e += 256) {  // coalesced 16-byte reads of Pi's rows
    const float4 r4 = reinterpret_cast<const float4*>(R)[e];
    const int ri = e >> 4, rj = 4 * (e & 15);
    rt[(rj + 0) * (D + 1) + ri] = r4.x;
    rt[(rj + 1) * (D + 1) + ri] = r4.y;
    rt[(rj + 2) * (D + 1) + ri] = r4.z;
    rt[(rj + 3) * (D + 1) + ri] = r4.w;
  }
  for (int e = tid; e < G * D; e += 256) {
    const int64_t src = g * G * D + e;
    float v;
    if (q_dtype == FIBQ_F32) v = static_cast<const float*>(q)[src];
    else if (q_dtype == FIBQ_F16) v = to_float(static_cast<const f16_t*>(q)[src]);
    else v = to_float(static_cast<const bf16_t*>(q)[src]);
    qs[e] = v;
  }
  if (tid == 0) any_lo = 0;
  __syncthreads();
  float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
  for (int k = 0; k < D / 4; ++k) {
    const float4 a = reinterpret_cast<const float4*>(qs + hq * D)[k];
    const float4 b = reinterpret_cast<const float4*>(qs + (hq + 4) * D)[k];
    const float r0 = rt[(4 * k + 0) * (D + 1) + i], r1 = rt[(4 * k + 1) * (D + 1) + i];
    const float r2 = rt[(4 * k + 2) * (D + 1) + i], r3 = rt[(4 * k + 3) * (D + 1) + i];
    s0 = fmaf(r0, a.x, s0); s0 = fmaf(r1, a.y, s0);
    s0 = fmaf(r2, a.z, s0); s0 = fmaf(r3, a.w, s0);
    s1 = fmaf(r0, b.x, s1); s1 = fmaf(r1, b.y, s1);
    s1 = fmaf(r2, b.z, s1); s1 = fmaf(r3, b.w, s1);
  }
  s0 *= qscale;
  s1 *= qscale;
  qt[hq * D + i] = s0;
  qt[(hq + 4) * D + i] = s1;
  float amax = fmaxf(fabsf(s0), fabsf(s1));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  const float top = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  // power-of-two divisor that brings every entry to at most kQMax (1 if none)
  float sc = 1.0f;
  if (top > kQMax) {
    int e2 = 0;
    frexpf(top / kQMax, &e2);
    sc = ldexpf(1.0f, e2);
  }
  const float inv = 1.0f / sc;  // exact (power of two)
  // A operand of v_mfma_f32_16x16x32_f16 for K-step kap: lane ln holds row
  // r = ln % 16 (head r / 2, part r % 2) and K entries 8 (ln / 16) .. +7, which
  // are dims 0..7 of block 2 (ln / 16) + kap.  Four entries per thread.
  {
    const int e0 = 4 * tid;
    const int kap = e0 >> 9, ln = (e0 >> 3) & 63, j0 = e0 & 7;
    const int r = ln & 15, gq = ln >> 4;
    const float* src = qt + (r >> 1) * D + 8 * (2 * gq + kap) + j0;
    h4 o;
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const float v = src[y] * inv;
      const _Float16 hi = (_Float16)v;
      o[y] = (r & 1) ? (_Float16)(v - (float)hi) : hi;
    }
    *reinterpret_cast<h4*>(qop + g * kQop + e0) = o;
  }
  if (tid == 0) qsc[g] = sc;
  if (zero_out)
    for (int e = tid; e < G * D; e += 256) out[g * G * D + e] = 0.0f;
  if (g == 0) {
    for (int k = tid; k < NC * K; k += 256) {
      const float c = C[k];
      const _Float16 hi = (_Float16)c;
      const _Float16 lo = (_Float16)(c - (float)hi);
      cb[k] = hi;
      cb[NC * K + k] = lo;
      if ((float)lo != 0.0f) any_lo = 1;
    }
    __syncthreads();
    if (tid == 0) reinterpret_cast<int*>(cb + 2 * NC * K)[0] = any_lo;
  }
}

// ----------------------------------------------------------------- main ----
__device__ __forceinline__ h4 tr_read(const unsigned char* lds_byte_addr) {
  s4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s4*)(lds_byte_addr));
  return __builtin_bit_cast(h4, r);
}

// byte offset of the codeword row of the low nibble of byte x: (x & 15) * 16
__device__ __forceinline__ uint32_t row_lo(uint32_t x) {
  uint32_t r;
  asm("v_lshlrev_b32_sdwa %0, 4, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD "
      "src1_sel:BYTE_0"
      : "=v"(r)
      : "v"(x));
  return r;
}
// ... of the high nibble: (x >> 4) * 16
__device__ __forceinline__ uint32_t row_hi(uint32_t x) { return x & 0xF0u; }

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
// max over the 16 lanes of a row: quad xor 1, quad xor 2, half-row mirror, row mirror
__device__ __forceinline__ float xmax16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}
__device__ __forceinline__ float xsum16(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  return v;
}

// Copy of 16 bytes per lane from global memory into LDS at lds_base + 16 *
// lane (global_load_lds_dwordx4); the wait for its completion is explicit
// (vm_wait), since vector-memory loads complete in issue order.  M0 (the LDS
// base) is saved and restored around the instruction.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_base) {
  uint32_t keep;
  const uint32_t bb = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(gptr), "s"(bb)
      : "memory");
}
template <int CNT>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CNT) : "memory");
}
// One lane's bytes of a 64-token sub-unit (tokens are sub-unit-relative):
//   kb[i]  byte (lane / 16) of the K payload word of token 4 (lane % 16) + i;
//   vb[2j + s]  byte (lane % 4) of the V word of token tv + 2j + 8s, with
//          tv = 16 (lane / 16) + 4 ((lane % 16) / 8) + ((lane % 16) / 4) % 2;
//   nk, nv  the binary16 norms of tokens 4 (lane % 16) .. +3.
struct Unit {
  uint32_t kb[4], vb[4];
  uint32_t nk[2], nv[2];
};

// Inputs of the form without a preparation launch: the workgroup builds the
// binary16 codebook table and the query operands of its groups itself.
struct Fused {
  const void* q;          // [n_groups][G][D] queries of q_dtype
  int q_dtype;
  const float* R;         // Pi, D x D row-major
  const float* C;         // codebook, NC x K
  float qscale;           // scale * log2(e)
};

template <bool FUSED>
__global__ __launch_bounds__(kThreads) void main_kernel(
    const uint8_t* __restrict__ kp, const uint16_t* __restrict__ kn,
    const uint8_t* __restrict__ vp, const uint16_t* __restrict__ vn, int T, int64_t T_stride,
    int64_t units, int upg, int slots, int ring_ok, const _Float16* __restrict__ qop,
    const float* __restrict__ qsc, const _Float16* __restrict__ cbg, float* __restrict__ rec,
    Fused fz) {
  // LDS: the codebook tables first (their row offsets then need no base),
  // then per-wavefront weight buffers, flush scratch, the claim counter, the
  // per-wavefront copy rings and the wavefront states of a flush.  Each
  // 16-byte codeword row occupies its own four banks, so any gather of rows
  // is free of bank conflicts (lanes reading one row share the access); a
  // table indexed by a whole payload byte would not be.  A ring slot holds
  // one unit: K words [0, 512), V words [512, 1024), K norms [1024, 1280),
  // V norms [1280, 1536); token t at 4t (words) or 2t (norms).
  constexpr int kOffW = 2 * NC * K * 2;
  constexpr int kOffSm = kOffW + kWaves * 2 * kWBuf;  // two weight buffers per wavefront
  constexpr int kOffCtr = kOffSm + 2 * kWaves * G * 4;
  constexpr int kOffFac = kOffCtr + 16;  // merge factors [G][kWaves], then M[G], L[G]
  constexpr int kOffRing = kOffFac + (G * kWaves + 2 * G) * 4;
  constexpr int kOffSacc = kOffRing + kWaves * kDepth * kSlot;
  // fused form: the query operands of up to kFusedGroups groups, their
  // divisors and the codebook's residual flag
  constexpr int kOffQop = kOffSacc + kWaves * G * D * 4;
  constexpr int kOffQsc = kOffQop + (FUSED ? kFusedGroups * kQop * 2 : 0);
  constexpr int kSmem = kOffQsc + (FUSED ? kFusedGroups * 4 + 32 : 0);
  __shared__ __align__(16) unsigned char smem[kSmem];
  _Float16* cb = reinterpret_cast<_Float16*>(smem);
  float (*sm)[G] = reinterpret_cast<float (*)[G]>(smem + kOffSm);
  float (*sl)[G] = reinterpret_cast<float (*)[G]>(smem + kOffSm + kWaves * G * 4);
  int& ctr = *reinterpret_cast<int*>(smem + kOffCtr);         // claims handed out
  int* seg_done = reinterpret_cast<int*>(smem + kOffCtr + 4);   // wavefronts done with the segment
  int* seg_merged = reinterpret_cast<int*>(smem + kOffCtr + 8); // segments merged so far
  float* fac = reinterpret_cast<float*>(smem + kOffFac);
  unsigned char* ring = smem + kOffRing;
  float* sacc = reinterpret_cast<float*>(smem + kOffSacc);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, c = lane & 15;
  _Float16* lqop = reinterpret_cast<_Float16*>(smem + kOffQop);
  float* lqsc = reinterpret_cast<float*>(smem + kOffQsc);
  int* lflag = reinterpret_cast<int*>(smem + kOffQsc + kFusedGroups * 4);  // residual flag, amax[4]
  if (!FUSED) {
    if (tid < 2 * NC * K / 8)
      reinterpret_cast<uint4*>(cb)[tid] = reinterpret_cast<const uint4*>(cbg)[tid];
  }
  if (tid == 0) {
    ctr = 0;
    seg_done[0] = 0;
    seg_merged[0] = 0;
    if (FUSED) lflag[0] = 0;
  }
  __syncthreads();

  const int wgs = gridDim.x;
  const int64_t w = blockIdx.x;
  const int64_t u0 = first_unit(w, units, wgs), u1 = first_unit(w + 1, units, wgs);
  const int64_t g_first = u0 / upg, g_last = (u1 - 1) / upg;
  const unsigned char* cbb = reinterpret_cast<const unsigned char*>(cb);
  const unsigned char* cbl = cbb + NC * K * 2;
  unsigned char* wb = smem + kOffW + wave * 2 * kWBuf;
  unsigned char* myring = ring + wave * kDepth * kSlot;
  const uint32_t ring_lds = (uint32_t)(uintptr_t)myring;

  // lane constants (see Unit)
  const int tk = 4 * c;
  const int tv = 16 * g4 + 4 * (c >> 3) + ((c >> 2) & 1);
  const uint32_t kbyte = (uint32_t)g4, vbyte = (uint32_t)(c & 3);
  const uint32_t w_wr = (uint32_t)(2 * g4) * kWRow + 4u * c;       // W[2 g4][2c] byte offset
  const uint32_t w_rd = (uint32_t)(c & 7) * kWRow + 16u * g4;      // W[c % 8][8 g4] byte offset
  const uint32_t rk = (uint32_t)tk * 4u + kbyte;                   // ring offsets of this lane
  const uint32_t rv = 512u + (uint32_t)tv * 4u + vbyte;            // (sub-unit 0)
  const uint32_t rn = 1024u + (uint32_t)tk * 2u;
  // ring copy sources: copy 1 moves 16 bytes of K words (lanes 0-31) or V
  // words (32-63), copy 2 moves K norms (lanes 0-15) or V norms (16-31)
  const unsigned char* cp1 = (lane < 32 ? kp : vp) + 16 * (lane & 31);
  const unsigned char* cp2 = reinterpret_cast<const unsigned char*>(lane < 16 ? kn : vn) +
                             16 * (lane & 15);

  // claims: positions relative to the first unit of group g_first; the
  // group of the latest claim (index ck relative to g_first, first position
  // cbase, first token row crow) is tracked incrementally
  const int pos0 = (int)(u0 - g_first * upg);
  const int n_w = (int)(u1 - u0);
  int ck = 0, cbase = 0;
  int64_t crow = g_first * T_stride;
  auto claim = [&]() -> int {
    int v = 0;
    if (lane == 0) v = atomicAdd(&ctr, 1);
    v = __builtin_amdgcn_readfirstlane(v);
    if (v >= n_w) return -1;
    const int pos = pos0 + v;
    while (pos - cbase >= upg) { cbase += upg; ++ck; crow += T_stride; }
    return pos;
  };
  // copies of the latest claim into a slot, if it is a whole unit and the
  // planes are aligned for them; returns the number of copies issued
  auto issue = [&](int pos, int slot) -> int {
    const int tb = (pos - cbase) * kUnit;
    if (!ring_ok || tb + kUnit > T) return 0;
    const int64_t row0 = crow + tb;
    const uint32_t dst = ring_lds + slot * kSlot;
    dma16(cp1 + (row0 << 2), dst);
    if (lane < 32) dma16(cp2 + (row0 << 1), dst + 1024);
    return 2;
  };
  auto read_ring = [&](const unsigned char* sb, int sub) -> Unit {
    Unit b;
#pragma unroll
    for (int i = 0; i < 4; ++i) b.kb[i] = sb[rk + 256 * sub + 4 * i];
#pragma unroll
    for (int i = 0; i < 4; ++i) b.vb[i] = sb[rv + 256 * sub + 8 * (i >> 1) + 32 * (i & 1)];
    // the bytes are used as whole registers from here on (the empty asm keeps
    // the compiler from narrowing them and re-masking in later blocks)
#pragma unroll
    for (int i = 0; i < 4; ++i) asm("" : "+v"(b.kb[i]), "+v"(b.vb[i]));
    const uint2 a = *reinterpret_cast<const uint2*>(sb + rn + 128 * sub);
    const uint2 v = *reinterpret_cast<const uint2*>(sb + rn + 128 * sub + 256);
    b.nk[0] = a.x; b.nk[1] = a.y; b.nv[0] = v.x; b.nv[1] = v.y;
    return b;
  };
  // per-lane fill of a ring slot from global memory, for units the copies
  // cannot move (ragged group ends, unaligned planes or strides): same
  // layout, tokens clamped into [0, T)
  auto fill_direct = [&](int pos, int gbase, int64_t grow, int slot) {
    const int tb = (pos - gbase) * kUnit;
    const int tm = T - 1 - tb;  // last valid unit-relative token
    const int64_t row0 = grow + tb;
    unsigned char* sb = myring + slot * kSlot;
    {  // payload words of tokens 4 (lane % 32) .. +3
      const uint8_t* src = (lane < 32 ? kp : vp) + row0 * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = min(4 * (lane & 31) + i, tm);
#pragma unroll
        for (int y = 0; y < 4; ++y) sb[16 * lane + 4 * i + y] = src[(int64_t)t * 4 + y];
      }
    }
    if (lane < 32) {  // norms of tokens 8 (lane % 16) .. +7
      const uint16_t* src = (lane < 16 ? kn : vn) + row0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int t = min(8 * (lane & 15) + i, tm);
        reinterpret_cast<uint16_t*>(sb + 1024 + 16 * lane)[i] = src[t];
      }
    }
  };

  // the claim queue: q[0] is the next unit to process, in ring slot `slot`;
  // `inflight` counts copies issued and not yet waited for
  int q[kDepth];
  int inflight = 0;
#pragma unroll
  for (int d = 0; d < kDepth; ++d) {
    q[d] = claim();
    if (q[d] >= 0) inflight += issue(q[d], d);
  }
  int slot = 0;
  // fused form: while the first copies are in flight, the workgroup builds
  // the binary16 codebook tables and the query operands of its groups (as
  // prep_kernel does for all groups)
  if (FUSED) {
    const int ng = (int)(g_last - g_first + 1);  // <= kFusedGroups (checked at launch)
    if (tid < NC * K) {
      const float cv = fz.C[tid];
      const _Float16 hi = (_Float16)cv;
      const _Float16 lo = (_Float16)(cv - (float)hi);
      cb[tid] = hi;
      cb[NC * K + tid] = lo;
      if ((float)lo != 0.0f) atomicOr(lflag, 1);
    }
    // scratch of the prologue: Pi^T in the state area, rows padded to D + 1
    // floats (loaded with coalesced 16-byte reads of Pi's rows, read back a
    // column per lane without bank conflicts), followed by the queries; the
    // rotated, scaled queries [ng][G][D] in the weight buffers.  Both areas
    // are free until the main loop.
    static_assert(kWaves * G * D >= D * (D + 1) + kFusedGroups * G * D,
                  "state area too small for Pi^T and the queries");
    static_assert(kWaves * 2 * kWBuf >= kFusedGroups * G * D * 4, "weight buffers too small");
    float* rt = sacc;
    float* qs32 = sacc + D * (D + 1);  // [ng][G][D] queries as float
    float* qt = reinterpret_cast<float*>(smem + kOffW);
    for (int e = tid; e < ng * G * D; e += kThreads) {
      const int64_t src = g_first * G * D + e;
      float v;
      if (fz.q_dtype == FIBQ_F32) v = static_cast<const float*>(fz.q)[src];
      else if (fz.q_dtype == FIBQ_F16) v = to_float(static_cast<const f16_t*>(fz.q)[src]);
      else v = to_float(static_cast<const bf16_t*>(fz.q)[src]);
      qs32[e] = v;
    }
    for (int e = tid; e < D * D / 4; e += kThreads) {
      const float4 r4 = reinterpret_cast<const float4*>(fz.R)[e];
      const int ri = e >> 4, rj = 4 * (e & 15);
      rt[(rj + 0) * (D + 1) + ri] = r4.x;
      rt[(rj + 1) * (D + 1) + ri] = r4.y;
      rt[(rj + 2) * (D + 1) + ri] = r4.z;
      rt[(rj + 3) * (D + 1) + ri] = r4.w;
    }
    if (tid < kFusedGroups) lflag[1 + tid] = 0;  // per-group max |entry| (float bits)
    __syncthreads();
    for (int o = tid; o < ng * G * D; o += kThreads) {  // o = (group j, head h, dim i)
      const int i = o & (D - 1), jh = o >> 6;
      const float4* qq = reinterpret_cast<const float4*>(qs32 + jh * D);  // broadcast reads
      float sacc_o = 0.0f;
#pragma unroll
      for (int k4 = 0; k4 < D / 4; ++k4) {
        const float4 b = qq[k4];
        sacc_o = fmaf(rt[(4 * k4 + 0) * (D + 1) + i], b.x, sacc_o);
        sacc_o = fmaf(rt[(4 * k4 + 1) * (D + 1) + i], b.y, sacc_o);
        sacc_o = fmaf(rt[(4 * k4 + 2) * (D + 1) + i], b.z, sacc_o);
        sacc_o = fmaf(rt[(4 * k4 + 3) * (D + 1) + i], b.w, sacc_o);
      }
      sacc_o *= fz.qscale;
      qt[o] = sacc_o;
      float amax = fabsf(sacc_o);
#pragma unroll
      for (int sh = 32; sh > 0; sh >>= 1) amax = fmaxf(amax, __shfl_xor(amax, sh, 64));
      if (lane == 0) atomicMax(lflag + 1 + (o >> 9), __float_as_int(amax));
    }
    __syncthreads();
    for (int eo = tid; eo < ng * 256; eo += kThreads) {  // entries 4 (eo % 256) .. +3 of group eo / 256
      const int j = eo >> 8;
      {
        const float top = __int_as_float(lflag[1 + j]);
        float sc = 1.0f;
        if (top > kQMax) {
          int e2 = 0;
          frexpf(top / kQMax, &e2);
          sc = ldexpf(1.0f, e2);
        }
        const float inv = 1.0f / sc;  // exact (power of two)
        const int e0 = 4 * (eo & 255);
        const int kap = e0 >> 9, ln = (e0 >> 3) & 63, j0 = e0 & 7;
        const int r = ln & 15, gq = ln >> 4;
        const float* src = qt + j * G * D + (r >> 1) * D + 8 * (2 * gq + kap) + j0;
        h4 o4;
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          const float v = src[y] * inv;
          const _Float16 hi = (_Float16)v;
          o4[y] = (r & 1) ? (_Float16)(v - (float)hi) : hi;
        }
        *reinterpret_cast<h4*>(lqop + j * kQop + e0) = o4;
        if ((eo & 255) == 0) lqsc[j] = sc;
      }
    }
    __syncthreads();
  }
  const bool has_lo = FUSED ? (lflag[0] != 0)
                            : (reinterpret_cast<const int*>(cbg + 2 * NC * K)[0] != 0);

  for (int64_t grp = g_first; grp <= g_last; ++grp) {
    const int gk = (int)(grp - g_first);
    const int gbase = gk * upg, gend = gbase + upg;  // positions of this group
    const int64_t grow = grp * T_stride;
    const float qs = FUSED ? lqsc[gk] : qsc[grp];
    const bool scaled = qs != 1.0f;
    const _Float16* qg = FUSED ? lqop + gk * kQop : qop + grp * kQop;
    const h8 qa0 = reinterpret_cast<const h8*>(qg)[lane];
    const h8 qa1 = reinterpret_cast<const h8*>(qg + 512)[lane];
    f4 acc[4] = {f4{0, 0, 0, 0}, f4{0, 0, 0, 0}, f4{0, 0, 0, 0}, f4{0, 0, 0, 0}};
    float m0 = -INFINITY, m1 = -INFINITY, l0 = 0.0f, l1 = 0.0f;

    auto run = [&](auto lo_tag, auto sc_tag) {
    constexpr bool HAS_LO = decltype(lo_tag)::value;
    constexpr bool SCALED = decltype(sc_tag)::value;
    const h8 qh0 = (HAS_LO && !(lane & 1)) ? qa0 : h8{};  // part-0 rows (residual codebook rows)
    const h8 qh1 = (HAS_LO && !(lane & 1)) ? qa1 : h8{};
    // the lag in the units of t (scores carry a factor 1 / qs when scaled)
    const int lag_bits = __float_as_int(SCALED ? kLag / qs : kLag);
    // Both 32-token steps of a 64-token sub-unit at once (one basic block on
    // the common path, so that the two steps' LDS and matrix-core latencies
    // overlap).  Step j covers tokens tk + 2j (tile 0) and tk + 2j + 1 (tile 1).
    auto step2 = [&](const Unit& b, int tb, bool full, int thr_bits) {
      // ---- scores
      f4 s[2][2];  // [step][tile]: rows 4 g4 .. +3 = (h0 part 0, h0 part 1, h1 part 0,
                   // h1 part 1) with h0 = 2 g4, h1 = 2 g4 + 1; column c = the token
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint32_t x0 = b.kb[2 * j], x1 = b.kb[2 * j + 1];
        const uint32_t a0l = row_lo(x0), a0h = row_hi(x0), a1l = row_lo(x1), a1h = row_hi(x1);
        const h8 c00 = *reinterpret_cast<const h8*>(cbb + a0l);
        const h8 c01 = *reinterpret_cast<const h8*>(cbb + a0h);
        const h8 c10 = *reinterpret_cast<const h8*>(cbb + a1l);
        const h8 c11 = *reinterpret_cast<const h8*>(cbb + a1h);
        s[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa0, c00, f4{0, 0, 0, 0}, 0, 0, 0);
        s[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa0, c10, f4{0, 0, 0, 0}, 0, 0, 0);
        s[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa1, c01, s[j][0], 0, 0, 0);
        s[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa1, c11, s[j][1], 0, 0, 0);
        if (HAS_LO) {
          const h8 d00 = *reinterpret_cast<const h8*>(cbl + a0l);
          const h8 d01 = *reinterpret_cast<const h8*>(cbl + a0h);
          const h8 d10 = *reinterpret_cast<const h8*>(cbl + a1l);
          const h8 d11 = *reinterpret_cast<const h8*>(cbl + a1h);
          s[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qh0, d00, s[j][0], 0, 0, 0);
          s[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qh0, d10, s[j][1], 0, 0, 0);
          s[j][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qh1, d01, s[j][0], 0, 0, 0);
          s[j][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(qh1, d11, s[j][1], 0, 0, 0);
        }
      }
      // t = S nu_K - m, [step][head][tile]
      float t[2][2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const h2 nk2 = __builtin_bit_cast(h2, b.nk[j]);
#pragma unroll
        for (int tl = 0; tl < 2; ++tl) {
          t[j][0][tl] = fmaf(s[j][tl][0] + s[j][tl][1], (float)nk2[tl], -m0);
          t[j][1][tl] = fmaf(s[j][tl][2] + s[j][tl][3], (float)nk2[tl], -m1);
        }
      }
      if (!full) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int tl = 0; tl < 2; ++tl)
            if (tb + tk + 2 * j + tl >= T) { t[j][0][tl] = -INFINITY; t[j][1][tl] = -INFINITY; }
      }
      // a score more than the lag above the reference (compared as integers:
      // the lag is positive or zero, and negative floats are negative ints)
      int tmx = __float_as_int(t[0][0][0]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int tl = 0; tl < 2; ++tl) tmx = max(tmx, __float_as_int(t[j][h][tl]));
      if (__any(tmx > thr_bits)) {  // rare after the first sub-unit
        if (m0 == -INFINITY) {  // first sub-unit of this wavefront in the group
          float u[2][2][2];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const h2 nk2 = __builtin_bit_cast(h2, b.nk[j]);
#pragma unroll
            for (int tl = 0; tl < 2; ++tl) {
              const bool live = full || tb + tk + 2 * j + tl < T;
              u[j][0][tl] = live ? (s[j][tl][0] + s[j][tl][1]) * (float)nk2[tl] : -INFINITY;
              u[j][1][tl] = live ? (s[j][tl][2] + s[j][tl][3]) * (float)nk2[tl] : -INFINITY;
            }
          }
          m0 = xmax16(fmaxf(fmaxf(u[0][0][0], u[0][0][1]), fmaxf(u[1][0][0], u[1][0][1])));
          m1 = xmax16(fmaxf(fmaxf(u[0][1][0], u[0][1][1]), fmaxf(u[1][1][0], u[1][1][1])));
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int tl = 0; tl < 2; ++tl) {
              t[j][0][tl] = u[j][0][tl] - m0;
              t[j][1][tl] = u[j][1][tl] - m1;
            }
          // nothing accumulated yet: acc and l stay zero
        } else {
          const float d0 = fmaxf(xmax16(fmaxf(fmaxf(t[0][0][0], t[0][0][1]),
                                              fmaxf(t[1][0][0], t[1][0][1]))), 0.0f);
          const float d1 = fmaxf(xmax16(fmaxf(fmaxf(t[0][1][0], t[0][1][1]),
                                              fmaxf(t[1][1][0], t[1][1][1]))), 0.0f);
          m0 += d0; m1 += d1;
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int tl = 0; tl < 2; ++tl) {
              t[j][0][tl] -= d0;
              t[j][1][tl] -= d1;
            }
          const float a0 = __builtin_amdgcn_exp2f(SCALED ? -d0 * qs : -d0);
          const float a1 = __builtin_amdgcn_exp2f(SCALED ? -d1 * qs : -d1);
          l0 *= a0; l1 *= a1;
          // accumulator row 4 g4 + e (g4 < 2) is head 4 g4 + e, whose factor
          // sits in lanes 16 ((4 g4 + e) / 2) (element e % 2)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int src = 16 * (((4 * g4 + e) & 7) >> 1);
            const float f = (e & 1) ? __shfl(a1, src, 64) : __shfl(a0, src, 64);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) acc[qq][e] *= f;
          }
        }
      }
      // ---- weights: p rounded to binary16 once; W[h][2c], W[h][2c+1] for
      //      h = 2 g4, 2 g4 + 1 into the step's weight buffer
      const h2 ones = h2{(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if (SCALED) {
#pragma unroll
          for (int h = 0; h < 2; ++h) { t[j][h][0] *= qs; t[j][h][1] *= qs; }
        }
        const h2 p0 = h2{(_Float16)__builtin_amdgcn_exp2f(t[j][0][0]),
                         (_Float16)__builtin_amdgcn_exp2f(t[j][0][1])};
        const h2 p1 = h2{(_Float16)__builtin_amdgcn_exp2f(t[j][1][0]),
                         (_Float16)__builtin_amdgcn_exp2f(t[j][1][1])};
        l0 = __builtin_amdgcn_fdot2(p0, ones, l0, false);
        l1 = __builtin_amdgcn_fdot2(p1, ones, l1, false);
        const h2 nv2 = __builtin_bit_cast(h2, b.nv[j]);
        *reinterpret_cast<h2*>(wb + j * kWBuf + w_wr) = p0 * nv2;
        *reinterpret_cast<h2*>(wb + j * kWBuf + w_wr + kWRow) = p1 * nv2;
      }
      // ---- values: O[h][:] += W[h][t] V_hat[t][:].  A = W (rows 0..7; rows
      //      8..15 repeat them at the same addresses, so the LDS broadcasts,
      //      and feed accumulator rows never read).  B: K entries 8 g4 .. +7
      //      of the value MFMA (hn, hh) are step tokens tv + 2j + {0, 1, 2, 3
      //      from the transposing read} (+8 for the second read); column c is
      //      dim 8 (2 (c / 4) + hn) + 4 hh + c % 4.
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        // rows 8..15 of the operand feed accumulator rows that are never read:
        // only the lanes of rows 0..7 read the buffer (half the LDS traffic)
        h8 aw = h8{};
        if ((lane & 15) < 8) aw = *reinterpret_cast<const h8*>(wb + j * kWBuf + w_rd);
        const uint32_t y0 = b.vb[2 * j], y1 = b.vb[2 * j + 1];
        const uint32_t r0l = row_lo(y0), r0h = row_hi(y0), r1l = row_lo(y1), r1h = row_hi(y1);
#pragma unroll
        for (int hn = 0; hn < 2; ++hn)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const h4 b0 = tr_read(cbb + (hn ? r0h : r0l) + 8 * hh);
            const h4 b1 = tr_read(cbb + (hn ? r1h : r1l) + 8 * hh);
            const h8 bv = h8{b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
            acc[2 * hn + hh] = __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, bv, acc[2 * hn + hh], 0, 0, 0);
            if (HAS_LO) {  // residual rows of a codebook that is not binary16-exact
              const h4 d0 = tr_read(cbl + (hn ? r0h : r0l) + 8 * hh);
              const h4 d1 = tr_read(cbl + (hn ? r1h : r1l) + 8 * hh);
              const h8 dv = h8{d0[0], d0[1], d0[2], d0[3], d1[0], d1[1], d1[2], d1[3]};
              acc[2 * hn + hh] =
                  __builtin_amdgcn_mfma_f32_16x16x32_f16(aw, dv, acc[2 * hn + hh], 0, 0, 0);
            }
          }
      }
    };

    // one 64-token sub-unit starting at token tb of the group
    auto sub_unit = [&](const unsigned char* sb, int sub, int tb) {
      const Unit b = read_ring(sb, sub);
      const bool full = tb + kSub <= T;
      // lag of this sub-unit: zero if some V norm could overflow p * nu_V
      // (the norms are non-negative binary16, ordered like their bit patterns)
      const u16x2 nvm = __builtin_elementwise_max(__builtin_bit_cast(u16x2, b.nv[0]),
                                                  __builtin_bit_cast(u16x2, b.nv[1]));
      const u16x2 over = __builtin_elementwise_sub_sat(nvm, u16x2{kNuLagBits, kNuLagBits});
      const int thr_bits = __any(__builtin_bit_cast(uint32_t, over) != 0u) ? 0 : lag_bits;
      step2(b, tb, full, thr_bits);
    };
    // units of this group: the head of the queue while it lies here
    while (q[0] >= 0 && q[0] < gend) {
      const int head = q[0];
      const int tb = (head - gbase) * kUnit;
      if (ring_ok && tb + kUnit <= T) {
        // the head's two copies are the oldest in flight (copies complete in issue order)
        inflight -= 2;
        // steady state: the three younger units' copies stay in flight
        if (inflight == 2 * (kDepth - 1)) vm_wait<2 * (kDepth - 1)>();
        else vm_wait<0>();
      } else {
        fill_direct(head, gbase, grow, slot);  // this wavefront's LDS writes precede its reads
      }
      const unsigned char* sb = myring + slot * kSlot;
      sub_unit(sb, 0, tb);
      if (tb + kSub < T) sub_unit(sb, 1, tb + kSub);
      // refill the slot just read (its LDS reads have completed: their
      // values fed this unit's steps)
#pragma unroll
      for (int d = 0; d + 1 < kDepth; ++d) q[d] = q[d + 1];
      q[kDepth - 1] = claim();
      if (q[kDepth - 1] >= 0) inflight += issue(q[kDepth - 1], slot);
      slot = (slot + 1) & (kDepth - 1);
    }
    };
    if (has_lo) {
      if (scaled) run(std::true_type{}, std::true_type{});
      else run(std::true_type{}, std::false_type{});
    } else {
      if (scaled) run(std::false_type{}, std::true_type{});
      else run(std::false_type{}, std::false_type{});
    }

    // ---- segment end, without a workgroup barrier: the wavefront parks its
    // state in its LDS slot (once the previous segment's states have been
    // merged) and counts itself done; the last one merges the 16 states and
    // writes the record
    const float ml0 = scaled ? m0 * qs : m0, ml1 = scaled ? m1 * qs : m1;  // true log2 units
    l0 = xsum16(l0);
    l1 = xsum16(l1);
    // Why this wait ends: the segment loop's bounds depend on the workgroup
    // only and nothing between its head and this point leaves it, so every
    // one of the kWaves wavefronts reaches every segment end, in order (the
    // unit loop above ends: claims only grow and run out after n_w).  The
    // wavefront that arrives last at the end of segment gk - 1 has seen all
    // kWaves states of it; it merges them, resets seg_done and then (release)
    // sets seg_merged to gk.  A wavefront waiting here for segment gk has
    // itself arrived at segment gk - 1, so that merge never waits on it, and
    // all waves of a workgroup are resident on one compute unit together
    // (s_sleep hands over the issue slots).  The acquire pairs with that
    // release: the slots sm/sl/sacc are free again and seg_done is zero
    // before this wavefront writes them or counts itself.
    while (__hip_atomic_load(seg_merged, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < gk)
      __builtin_amdgcn_s_sleep(2);
    if (c == 0) {
      sm[wave][2 * g4] = ml0;
      sm[wave][2 * g4 + 1] = ml1;
      sl[wave][2 * g4] = l0;
      sl[wave][2 * g4 + 1] = l1;
    }
    if (g4 < 2) {
      // accumulator (hn, hh): column c is dim 8 (2 (c / 4) + hn) + 4 hh + c % 4
#pragma unroll
      for (int hn = 0; hn < 2; ++hn)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            sacc[(wave * G + 4 * g4 + e) * D + 8 * (2 * (c >> 2) + hn) + 4 * hh + (c & 3)] =
                acc[2 * hn + hh][e];
    }
    int arrived = 0;
    if (lane == 0)
      arrived = __hip_atomic_fetch_add(seg_done, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
    arrived = __builtin_amdgcn_readfirstlane(arrived);
    if (arrived == kWaves - 1) {  // the last wavefront of this segment merges it
      // factors 2^(m_w - M) per (head, wavefront): lane l covers head l / 8,
      // wavefronts 2 (l % 8) and 2 (l % 8) + 1
      {
        const int h = lane >> 3, w0 = 2 * (lane & 7);
        float M = -INFINITY;
#pragma unroll
        for (int q4 = 0; q4 < kWaves; ++q4) M = fmaxf(M, sm[q4][h]);
        float L = 0.0f;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          if (w0 + k < kWaves) {
            const float mq = sm[w0 + k][h];
            const float f = (mq == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mq - M);
            fac[h * kWaves + w0 + k] = f;
            L = fmaf(sl[w0 + k][h], f, L);
          }
        }
        L += __shfl_xor(L, 1, 64);
        L += __shfl_xor(L, 2, 64);
        L += __shfl_xor(L, 4, 64);
        if ((lane & 7) == 0) {
          fac[G * kWaves + h] = M;
          fac[G * kWaves + G + h] = L;
        }
      }
      float* r = rec + ((int64_t)w * slots + gk) * kRec;
#pragma unroll
      for (int k = 0; k < G; ++k) {  // output k * 64 + lane: head k, dim lane
        float sacc_k = 0.0f;
#pragma unroll
        for (int q4 = 0; q4 < kWaves; ++q4)
          sacc_k = fmaf(sacc[(q4 * G + k) * D + lane], fac[k * kWaves + q4], sacc_k);
        r[2 * G + k * D + lane] = sacc_k;
      }
      if (lane < 2 * G) r[lane] = fac[G * kWaves + lane];  // M[G], then L[G]
      if (lane == 0) {
        __hip_atomic_store(seg_done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __hip_atomic_store(seg_merged, gk + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }
}

// ---------------------------------------------------------------- merge ----
// One block per group: log-sum-exp over the records of the workgroups whose
// unit ranges meet the group, then o = Pi^T (acc / l).  Thread t owns dim
// t % 64 of heads t / 64 and t / 64 + 4.  Pi is staged in LDS and the
// records of up to kMergeMax contributors are loaded in the same round of
// memory requests, before any of their values is used.
constexpr int kMergeThreads = 256;
constexpr int kMergeMax = 4;   // contributors per pass over the records

__global__ __launch_bounds__(kMergeThreads) void merge_kernel(const float* __restrict__ rec,
                                                              int64_t units, int upg, int wgs,
                                                              int slots,
                                                              const float* __restrict__ R,
                                                              float* __restrict__ out) {
  __shared__ __align__(16) float rs[D * D];  // Pi row-major: column reads are conflict-free
  __shared__ __align__(16) float ra[G * D];
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x, j = tid & (D - 1), h0 = tid >> 6, h1 = h0 + 4;
  float4 r4[D * D / 4 / kMergeThreads];
#pragma unroll
  for (int e = 0; e < D * D / 4 / kMergeThreads; ++e)
    r4[e] = reinterpret_cast<const float4*>(R)[tid + e * kMergeThreads];
  const int wlo = wg_of(g * upg, units, wgs), whi = wg_of((g + 1) * upg - 1, units, wgs);
  float M0 = -INFINITY, L0 = 0.0f, a0 = 0.0f, M1 = -INFINITY, L1 = 0.0f, a1 = 0.0f;
  for (int base = wlo; base <= whi; base += kMergeMax) {
    float m0[kMergeMax], l0[kMergeMax], x0[kMergeMax], m1[kMergeMax], l1[kMergeMax],
        x1[kMergeMax];
#pragma unroll
    for (int k = 0; k < kMergeMax; ++k) {
      const int ww = base + k;
      if (ww <= whi) {
        const int64_t fg = first_unit(ww, units, wgs) / upg;
        const float* rr = rec + ((int64_t)ww * slots + (g - fg)) * kRec;
        m0[k] = rr[h0]; l0[k] = rr[G + h0]; x0[k] = rr[2 * G + h0 * D + j];
        m1[k] = rr[h1]; l1[k] = rr[G + h1]; x1[k] = rr[2 * G + h1 * D + j];
      } else {
        m0[k] = m1[k] = -INFINITY;
        l0[k] = l1[k] = x0[k] = x1[k] = 0.0f;
      }
    }
    auto fold = [&](float& M, float& L, float& a, const float* mk, const float* lk,
                    const float* xk) {
      float Mn = M;
#pragma unroll
      for (int k = 0; k < kMergeMax; ++k) Mn = fmaxf(Mn, mk[k]);
      if (Mn == -INFINITY) return;
      const float fo = (M == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(M - Mn);
      L *= fo;
      a *= fo;
#pragma unroll
      for (int k = 0; k < kMergeMax; ++k) {
        const float f = (mk[k] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mk[k] - Mn);
        L = fmaf(lk[k], f, L);
        a = fmaf(xk[k], f, a);
      }
      M = Mn;
    };
    fold(M0, L0, a0, m0, l0, x0);
    fold(M1, L1, a1, m1, l1, x1);
  }
#pragma unroll
  for (int e = 0; e < D * D / 4 / kMergeThreads; ++e)
    reinterpret_cast<float4*>(rs)[tid + e * kMergeThreads] = r4[e];
  ra[h0 * D + j] = (L0 > 0.0f) ? a0 / L0 : 0.0f;
  ra[h1 * D + j] = (L1 > 0.0f) ? a1 / L1 : 0.0f;
  __syncthreads();
  float o0 = 0.0f, o1 = 0.0f;  // o[h][j] = sum_i Pi[i][j] a[h][i]
#pragma unroll 16
  for (int i = 0; i < D; ++i) {
    const float r = rs[i * D + j];
    o0 = fmaf(r, ra[h0 * D + i], o0);
    o1 = fmaf(r, ra[h1 * D + i], o1);
  }
  out[g * G * D + h0 * D + j] = o0;
  out[g * G * D + h1 * D + j] = o1;
}

}  // namespace w4

bool attn_w4_applies(int G, const Shape& s) {
  return s.d == 64 && s.k == 8 && G == 8 && s.w == 4;
}

size_t attn_w4_workspace_bytes(int64_t n_groups, int64_t T) {
  return w4::make_plan(n_groups, T).total;
}

int launch_attn_w4(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                   const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int64_t T,
                   int64_t T_stride, const float* R, const float* C, float scale, float* out,
                   void* ws, hipStream_t st) {
  const w4::Plan p = w4::make_plan(n_groups, T);
  unsigned char* b = static_cast<unsigned char*>(ws);
  _Float16* qop = reinterpret_cast<_Float16*>(b + p.off_q);
  float* qsc = reinterpret_cast<float*>(b + p.off_qs);
  _Float16* cb = reinterpret_cast<_Float16*>(b + p.off_cb);
  float* rec = reinterpret_cast<float*>(b + p.off_rec);
  const float qscale = scale * 1.4426950408889634f;  // base-2 softmax
  // the ring copies move 16-byte chunks: 16-byte aligned planes and a stride
  // that keeps every unit's payload and norm rows 16-byte aligned
  const uintptr_t mis = reinterpret_cast<uintptr_t>(kp) | reinterpret_cast<uintptr_t>(vp) |
                        reinterpret_cast<uintptr_t>(kn) | reinterpret_cast<uintptr_t>(vn);
  const int ring_ok = ((mis & 15) == 0 && (T_stride & 7) == 0) ? 1 : 0;
  const w4::Fused fz{q, q_dtype, R, C, qscale};
  hipError_t e;
  if (T > 0 && p.slots <= w4::kFusedGroups) {
    // the main kernel prepares its own groups' query operands
    hipLaunchKernelGGL(w4::main_kernel<true>, dim3((unsigned)p.wgs), dim3(w4::kThreads), 0, st, kp,
                       kn, vp, vn, (int)T, T_stride, p.units, p.upg, p.slots, ring_ok, qop, qsc,
                       cb, rec, fz);
  } else {
    hipLaunchKernelGGL(w4::prep_kernel, dim3((unsigned)n_groups), dim3(256), 0, st, q, q_dtype, R,
                       C, qscale, qop, qsc, cb, out, T == 0 ? 1 : 0);
    e = hipGetLastError();
    if (e != hipSuccess || T == 0) return (int)e;
    hipLaunchKernelGGL(w4::main_kernel<false>, dim3((unsigned)p.wgs), dim3(w4::kThreads), 0, st,
                       kp, kn, vp, vn, (int)T, T_stride, p.units, p.upg, p.slots, ring_ok, qop,
                       qsc, cb, rec, fz);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  hipLaunchKernelGGL(w4::merge_kernel, dim3((unsigned)n_groups), dim3(w4::kMergeThreads), 0, st,
                     rec, p.units, p.upg, p.wgs, p.slots, R, out);
  return (int)hipGetLastError();
}

}  // namespace dev
}  // namespace fibq
