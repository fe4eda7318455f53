// Encoder on the matrix cores for d = 64 with block dimension k = 2 or 4 and
// N in {16, 64, 256}, bf16 or fp16 caches (Sec. 3.1, Eq. encode): the
// TinyLlama- and GPT-2-shaped rates (k = 4, N = 256; k = 2, N = 64).
//
// One wavefront encodes 32 vectors per step; lane l works on vector l % 32
// and the two half-wavefronts split the blocks:
//   input     32-row tiles stream through a per-wavefront LDS ring (two 4 KB
//             slots) filled by global_load_lds_dwordx4;
//   norm      nu^2 = sum x^2 in float32 (dot products of exact products), the
//             binary16 header certified by rounding nu (1 -+ 2^-20) and
//             redone in float64 from the exact squares when uncertain;
//   rotation  z = Pi x on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16):
//             Pi as its three bf16 parts hi + mid + lo (their sum is Pi
//             exactly), x exact in bf16 (an fp16 row is split into bf16
//             hi + lo, also exact), so products are exact and only the
//             float32 accumulation rounds.  Each lane ends with 32 dimensions
//             of its vector (8 blocks of k = 4, or 16 of k = 2);
//   screen    G_j = <y_b, c_j> - |c_j|^2 / 2 (argmax G = argmin |y_b - c|^2)
//             with v_mfma_f32_32x32x16_f16 over 16 codewords x 2 blocks x 32
//             vectors: the two K halves carry one block each (A holds the
//             codeword on its half and zeros on the other).  In a half, k = 4
//             puts [2^8 y hi | 2^8 y lo] against [2^10 c hi | 2^10 c hi] (a
//             residual codebook adds a second product c lo * y hi) and the
//             accumulator starts at -2^17 |c|^2; k = 2 puts [y hi | y lo |
//             y hi | 2^8, 2^8] against [c hi | c hi | c lo | -n hi, -n lo]
//             with n = 2^9 |c|^2 (binary16 hi + lo), accumulator zero.  Codeword
//             sets are the outer loop, so the per-set operands are read from
//             LDS once and serve 8 (k = 4) or 4 (k = 2) blocks;
//   select    k = 2 (and N = 16): per block, the best two keys (float
//             max3 / med3, four candidates per step) with the codeword's
//             number within its set in the 4 low mantissa bits (which move a
//             key by less than 16 of its own ulps: that term of the bound
//             uses the two keys' magnitudes) and the set of the best tracked
//             beside it.  k = 4 with N >= 64 in two phases: the matrix cores'
//             scores give each set's maximum (the set number in its low bits)
//             and the best two set maxima; then the best set's 16 codewords
//             are scored again in float32 from 2^18 y and the fp32 codebook,
//             which gives the index and this set's second; the second best
//             overall is the larger of that and the second set maximum.  The
//             bound covers keys of either kind, and a best set chosen wrongly
//             (set maxima within the bound) leaves the gap below it;
//   grid      k = 2 with N = 64 skips the screen: a table built by each
//             workgroup lists, for each cell of a 32 x 32 grid over the block
//             plane, the codewords that can be nearest to a point of the cell;
//             a block scores only its cell's (at most 6) candidates in
//             float32, as in the second phase above, under the same bound;
//   exact     a block whose best two are closer than a rigorous bound on
//             the screen's error is redone in float64 (|z - nu c_j|^2 over
//             all N codewords; lowest index on ties), so every index is the
//             float64 argmin.  They wait in a per-wavefront queue and are
//             redone eight at a time; a tile with more takes them 2 (k = 4)
//             or 4 (k = 2) per pass of the whole wavefront.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device_common.h"
#include "encode_mf_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace encmf4 {

using namespace mfc;

constexpr int D = 64;
constexpr int kTile = 32;            // vectors per wavefront step
constexpr int kSlot = kTile * 128;   // bytes of one input tile
constexpr int kWaves = 12, kDepth = 2;

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// k = 4 with N >= 64 screens in two phases (set maxima on the matrix cores,
// then the best set's 16 codewords in float32); its LDS tables are padded per
// set of 16 codewords (+16 bytes) so that lanes reading different sets meet
// in different banks
template <int KB, int N>
constexpr bool two_phase() { return KB == 4 && N >= 64; }
template <int KB, int N>
constexpr int cs_stride() { return 16 * KB + (two_phase<KB, N>() ? 4 : 0); }  // floats per set
template <int KB, int N>
__device__ __forceinline__ int cs_at(int j) { return (j >> 4) * cs_stride<KB, N>() + (j & 15) * KB; }

// k = 2 with N = 64 takes its nearest codewords from a grid over the block
// plane instead of the matrix-core screen: each of kGS x kGS cells covering
// [-kGR, kGR]^2 lists the codewords that can be nearest to a point of the
// cell (at most kGCap; the workgroup builds the table from the codebook).
// Blocks of a unit vector in 64 dimensions leave that square with
// probability ~3e-6; those, and cells with more candidates, take the float64
// path.
template <int KB, int N>
constexpr bool grid_mode() { return KB == 2 && N == 64; }
constexpr int kGS = 32;
constexpr float kGR = 0.55f;
constexpr int kGCap = 6;

__device__ __forceinline__ double bcast64(double v, int lane) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), lane);
  return __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
}

template <int DT>  // 0: bf16, 1: fp16
__device__ __forceinline__ float elem(uint32_t bits16) {
  if (DT == 0) return __uint_as_float(bits16 << 16);
  return half_bits_to_float((uint16_t)bits16);
}

__device__ __forceinline__ double shfl64(double v, int src) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)u, src, 64);
  const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(u >> 32), src, 64);
  return __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
}

// Float64 nearest codewords of B = 64 / GL blocks at once (B = 2 for k = 4,
// 4 for k = 2), by the whole wavefront: lane group g = l / GL takes block
// bg[g] of tile vector vlg[g]; its lane (r, c) = ((l % GL) / 8, l % 8) forms
// the partial sum of row k b + r of z = Pi x over dims 8c .. 8c + 7 (x from
// the LDS tile; Pi as the exact sum of its three bf16 parts from the
// rotation's operand table), summed over the 8 lanes of the row; the group's
// lanes then score codewords l % GL, l % GL + GL, ... as
// |z - nu c_j|^2 = nu^2 |y - c_j|^2.  Keys carry the codeword number in their
// 8 low bits (scores agreeing to 2^-44 relative count as ties; equal keys
// pick the lowest index).  A zero or NaN norm gives index 0.  All 64 lanes
// must be active; res[g] is uniform.
template <int KB, int N, int DT>
__device__ __forceinline__ void exact_batch(const unsigned char* tile, const uint4* Pops,
                                            const float* Cl, int l, int vb0, int vb1, int vb2,
                                            int vb3, uint32_t (&res)[64 / (8 * KB)]) {
  constexpr int GL = 8 * KB, B = 64 / GL;
  const int g = l / GL, lg = l % GL, r = lg >> 3, c = l & 7;
  // this lane's group's (vector, block), packed as vector + 32 block: plain
  // selects between scalars
  const int s01 = (g & 1) ? vb1 : vb0;
  const int vb = (B == 4) ? ((g & 2) ? ((g & 1) ? vb3 : vb2) : s01) : s01;
  const int vl = vb & 31, b = vb >> 5;
  const uint4 raw = *reinterpret_cast<const uint4*>(tile + (vl >> 3) * 1024 + (vl & 7) * 128 +
                                                    16 * (c ^ (vl & 7)));
  // row dim = k b + r of Pi in the operand table: entry (t, kap, ln) holds,
  // for output row rho = ln % 32 of tile t, columns 16 kap + 8 (ln / 32) ..
  // + 7, where dim = 8 (4 t + 2 (i / 2) + hh) + 4 (i % 2) + e and
  // rho = 8 i + 4 hh + e
  const int dim = KB * b + r;
  const int b8 = dim >> 3, t = b8 >> 2, rem = b8 & 3, hh = rem & 1;
  const int i = 2 * (rem >> 1) + ((dim & 7) >> 2), rho = 8 * i + 4 * hh + (dim & 3);
  const int kap = c >> 1, kh = c & 1;
  // hi + mid + lo == Pi exactly: the parts of a float32 value, summed small
  // first, give it back exactly in float32
  float pv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) pv[u] = 0.0f;
#pragma unroll
  for (int sp = 2; sp >= 0; --sp) {
    const uint4 q = Pops[((t * 4 + kap) * 3 + sp) * 64 + 32 * kh + rho];
    const uint32_t pw[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int u = 0; u < 8; ++u) pv[u] += bf16_val((pw[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
  }
  const uint32_t xw[4] = {raw.x, raw.y, raw.z, raw.w};
  double ss = 0.0, p = 0.0;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const double xv = (double)elem<DT>((xw[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
    ss = fma(xv, xv, ss);
    p = fma((double)pv[u], xv, p);
  }
  ss = sum8(ss);
  p = sum8(p);
  const double nu = sqrt(ss);
  double z[KB];
#pragma unroll
  for (int rr = 0; rr < KB; ++rr) z[rr] = shfl64(p, g * GL + 8 * rr);
  uint64_t key = ~(uint64_t)0;
#pragma unroll
  for (int m = 0; m < (N + GL - 1) / GL; ++m) {
    const int j = lg + GL * m;
    if (j < N) {
      double dj = 0.0;
#pragma unroll
      for (int rr = 0; rr < KB; ++rr) {
        const double tt = fma(-nu, (double)Cl[cs_at<KB, N>(j) + rr], z[rr]);
        dj = fma(tt, tt, dj);
      }
      key = umin64(key, ((uint64_t)__double_as_longlong(dj) & ~(uint64_t)255) | (uint64_t)j);
    }
  }
  key = min16_64(key);
  if (GL == 32) key = perm64(key, true);  // the other 16-lane row of the half
  const uint32_t ix = nu > 0.0 ? (uint32_t)(key & 255) : 0u;
#pragma unroll
  for (int gg = 0; gg < B; ++gg) res[gg] = (uint32_t)__builtin_amdgcn_readlane((int)ix, gg * GL);
}

__device__ __forceinline__ double wave_max64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// A deferred near tie of the tile loop below, eight lanes each (all 64
// lanes active): ent = (vector << 5) | block is the queue entry of this
// lane's group l / 8, act whether that entry is a real one.  Lane c = l % 8
// reads dims 8c .. 8c + 7 of the vector's row and Pi's fp32 entries for them
// from global memory and forms their share of the block's k rows of z = Pi x
// and of |x|^2 in float64 (the order of exact_batch, whose results it
// repeats bit for bit); the eight lanes' sums give z and nu, then codewords
// c, c + 8, ... are scored as |z - nu c_j|^2 with the same keys.  The stored
// index is replaced with atomic and / or on the 32-bit word(s) of the
// vector's payload holding its W bits, after the wavefront's stores have
// completed (P is a multiple of 4: the words are the vector's own).  Not
// inlined: its registers are needed only at the rare drain points.
template <int KB, int N, int DT>
__device__ __attribute__((noinline)) void defer_pass(int64_t ent, bool act, int l,
                                                     const uint16_t* __restrict__ x,
                                                     int64_t stride, const float* __restrict__ R,
                                                     const float* Cs, uint8_t* __restrict__ payload) {
  constexpr int W = N == 16 ? 4 : (N == 64 ? 6 : 8);
  constexpr int P = (D / KB) * W / 8;
  const int c = l & 7;
  const int64_t dv = ent >> 5;
  const int b = (int)(ent & 31);
  const uint4 raw = *reinterpret_cast<const uint4*>(x + dv * stride + 8 * c);
  const uint32_t xw[4] = {raw.x, raw.y, raw.z, raw.w};
  double xv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) xv[u] = (double)elem<DT>((xw[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
  double ss = 0.0;
#pragma unroll
  for (int u = 0; u < 8; ++u) ss = fma(xv[u], xv[u], ss);
  double zr[KB];
#pragma unroll
  for (int r = 0; r < KB; ++r) {
    const float* row = R + (KB * b + r) * D + 8 * c;
    double pz = 0.0;
#pragma unroll
    for (int u = 0; u < 8; ++u) pz = fma((double)row[u], xv[u], pz);
    zr[r] = sum8(pz);
  }
  const double nu = sqrt(sum8(ss));
  uint64_t key = ~(uint64_t)0;
#pragma unroll
  for (int i = 0; i < N / 8; ++i) {
    const int j = c + 8 * i;
    double dj = 0.0;
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const double tt = fma(-nu, (double)Cs[cs_at<KB, N>(j) + r], zr[r]);
      dj = fma(tt, tt, dj);
    }
    key = umin64(key, ((uint64_t)__double_as_longlong(dj) & ~(uint64_t)255) | (uint64_t)j);
  }
  key = min_step(key, 0xB1);  // minimum over the eight lanes of the entry
  key = min_step(key, 0x4E);
  key = min_step(key, 0x141);
  const uint32_t bi = nu > 0.0 ? (uint32_t)(key & 255) : 0u;
  vm_wait<0>();  // this wavefront's payload stores have completed
  if (c == 0 && act) {
    constexpr uint32_t msk = (1u << W) - 1u;
    const int64_t bit = dv * (int64_t)(8 * P) + W * b;
    uint32_t* pw = reinterpret_cast<uint32_t*>(payload) + (bit >> 5);
    const int sh = (int)(bit & 31);
    atomicAnd(pw, ~(msk << sh));
    atomicOr(pw, bi << sh);
    if (sh + W > 32) {  // the upper bits in the next word
      atomicAnd(pw + 1, ~(msk >> (32 - sh)));
      atomicOr(pw + 1, bi >> (32 - sh));
    }
  }
}

template <int KB, int N, int DT>
__device__ __forceinline__ void encode_body(const uint16_t* __restrict__ x, int64_t n_vec,
                                            int64_t stride, const float* __restrict__ R,
                                            const float* __restrict__ C,
                                            uint8_t* __restrict__ payload,
                                            uint16_t* __restrict__ norms) {
  constexpr int NSET = N / 16;                       // codeword sets of 16
  constexpr int W = N == 16 ? 4 : (N == 64 ? 6 : 8);  // index bits
  constexpr int NBL = 32 / KB;                       // blocks per lane
  constexpr int P = (D / KB) * W / 8;                // payload bytes per vector
  constexpr int PW = P / 4;                          // payload words
  constexpr int GB = KB == 4 ? 8 : 4;                 // blocks per screen group
  static_assert(P % 4 == 0 && NBL % GB == 0, "layout");
  const int l = threadIdx.x & 63;
  const int h = l >> 5, v = l & 31;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  constexpr int kThr = kWaves * 64;

  // LDS: input rings; rotation A operands (Pi hi, mid, lo, lane order); screen
  // A operands per codeword set (lane order) and, for k = 4, the residual
  // rows and the accumulator start per set; the codebook in fp32.
  constexpr int kRing = kWaves * kDepth * kSlot;
  constexpr int kOps = 2 * 4 * 3 * 64 * 16;
  constexpr bool GRID = grid_mode<KB, N>();
  constexpr int kA = GRID ? 0 : NSET * 64 * 16;
  constexpr int kAlo = KB == 4 ? kA : 0;
  constexpr bool TP = two_phase<KB, N>();
  constexpr int kIStr = TP ? 20 : 16;  // floats per set in Ini (padded as the codebook)
  constexpr int kInit = (KB == 4 || TP) ? NSET * kIStr * 4 : 0;
  constexpr int kCs = NSET * cs_stride<KB, N>() * 4;
  // grid mode: the cell table (kGCap codeword numbers per cell, bytes 0 .. 5,
  // unused ones N; byte 6 flags a cell with more candidates) and the
  // codewords as (c_0, c_1, -2^17 |c|^2, number), entry N a sentinel that
  // never wins
  constexpr int kTab = GRID ? kGS * kGS * 8 : 0;
  constexpr int kCw = GRID ? (N + 1) * 16 : 0;
  __shared__ __align__(16) unsigned char smem[kRing + kOps + kA + kAlo + kInit + kCs + kTab + kCw];
  uint4* Pops = reinterpret_cast<uint4*>(smem + kRing);
  uint4* Ascr = reinterpret_cast<uint4*>(smem + kRing + kOps);
  uint4* Alos = reinterpret_cast<uint4*>(smem + kRing + kOps + kA);
  float* Ini = reinterpret_cast<float*>(smem + kRing + kOps + kA + kAlo);
  float* Cs = reinterpret_cast<float*>(smem + kRing + kOps + kA + kAlo + kInit);
  uint2* Tab = reinterpret_cast<uint2*>(smem + kRing + kOps + kA + kAlo + kInit + kCs);
  f4* Cw = reinterpret_cast<f4*>(smem + kRing + kOps + kA + kAlo + kInit + kCs + kTab);
  __shared__ int claim_ctr;
  __shared__ uint32_t cst[3];    // float bits of max |c|^2 and max |c|_1; residual flag
  // near ties wait in a per-wavefront queue, (vector << 5) | block, and are
  // redone eight at a time (defer_pass)
  constexpr int kQ = 16;
  __shared__ int64_t dq[kWaves * kQ];
  if (threadIdx.x == 0) {
    claim_ctr = 0;
    cst[0] = cst[1] = cst[2] = 0u;
  }
  for (int i = threadIdx.x; i < N * KB; i += kThr) Cs[cs_at<KB, N>(i / KB) + i % KB] = C[i];
  // ---- rotation operands (read only Pi, so their loads overlap the
  // codebook's): output row rho = 8 i + 4 hh + e of tile t is
  // dimension 8 (4 t + 2 (i / 2) + hh) + 4 (i % 2) + e
  for (int e = threadIdx.x; e < 2 * 4 * 64; e += kThr) {
    const int t = e >> 8, kap = (e >> 6) & 3, ln = e & 63;
    const int rho = ln & 31, i = rho >> 3, hh = (rho >> 2) & 1, ee = rho & 3;
    const int dim = 8 * (4 * t + 2 * (i >> 1) + hh) + 4 * (i & 1) + ee;
    const float* src = R + dim * D + 16 * kap + 8 * (ln >> 5);
    uint32_t part[3][4];
#pragma unroll
    for (int q = 0; q < 8; q += 2) {
      uint32_t hb[2], mb[2], lb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float vv = src[q + u];
        hb[u] = bf16_rne(vv);
        const float r1 = vv - bf16_val(hb[u]);  // exact
        mb[u] = bf16_rne(r1);
        lb[u] = bf16_rne(r1 - bf16_val(mb[u]));  // exact: r1 - mid is a bf16 value
      }
      part[0][q / 2] = hb[0] | (hb[1] << 16);
      part[1][q / 2] = mb[0] | (mb[1] << 16);
      part[2][q / 2] = lb[0] | (lb[1] << 16);
    }
#pragma unroll
    for (int sp = 0; sp < 3; ++sp)
      Pops[((t * 4 + kap) * 3 + sp) * 64 + ln] = uint4{part[sp][0], part[sp][1], part[sp][2], part[sp][3]};
  }

  __syncthreads();

  // ---- persistent loop over 32-vector tiles (as the k = 8 encoder: equal
  // contiguous ranges per workgroup, claimed one at a time from an LDS
  // counter; copies kDepth tiles ahead; the last tile clamps its rows).  The
  // first copies are issued here, so that their latency overlaps the rest of
  // the set-up (the ring is apart from the tables built below)
  const int64_t ntiles = (n_vec + kTile - 1) / kTile;
  const int64_t tb = ((int64_t)blockIdx.x * ntiles) / gridDim.x;
  const int64_t te = ((int64_t)(blockIdx.x + 1) * ntiles) / gridDim.x;
  auto claim = [&]() -> int64_t {
    int cc = 0;
    if (l == 0) cc = atomicAdd(&claim_ctr, 1);
    cc = __builtin_amdgcn_readfirstlane(cc);
    return tb + cc < te ? tb + cc : -1;
  };
  unsigned char* myring = smem + wave * kDepth * kSlot;
  const uint32_t ring = (uint32_t)(uintptr_t)myring;
  const int rih = l >> 3, chunk = (l & 7) ^ rih;
  const uint32_t loff = (uint32_t)(((int64_t)rih * stride + 8 * chunk) * 2);
  auto issue = [&](int64_t tile, int slot) {
    const uint16_t* base = x + tile * kTile * stride;
    if ((tile + 1) * kTile <= n_vec) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        dma16s(loff, base + 8 * q * stride, ring + slot * kSlot + 1024 * q);
    } else {
      const int lim = (int)(n_vec - 1 - tile * kTile);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = min(8 * q + rih, lim);
        dma16s((uint32_t)((r * stride + 8 * chunk) * 2), base, ring + slot * kSlot + 1024 * q);
      }
    }
  };
  // this lane's chunks of its row (2 kap + h, swizzled by v % 8) sit at
  // rrow + ((32 kap) ^ rsw); recomputed per tile from two registers
  const uint32_t rrow = (v >> 3) * 1024 + (v & 7) * 128 + 16 * (h ^ (v & 1));
  const uint32_t rsw = 32 * ((v & 7) >> 1);
  int64_t queue[kDepth];
#pragma unroll
  for (int d = 0; d < kDepth; ++d) {
    queue[d] = claim();
    if (queue[d] >= 0) issue(queue[d], d);
  }

  // ---- codebook constants for the bound: max |c|^2, max over pairs of
  // |c_a - c_b|_1 and whether some entry is not binary16-exact.  Since
  // |u|_1 = max over sign vectors s of s.u, the pair maximum is the maximum
  // over s of max_a s.c_a - min_b s.c_b (the pair s, -s together): 2^(k-1)
  // sign vectors, one per wavefront, instead of N^2 / 2 pairs.  The sums are
  // taken in float64, where k float32 terms add exactly or within
  // 2^-52 |c|_1 (the additive term where the bound is formed).
  __shared__ double pspan[8];
  {
    constexpr int NS = 1 << KB;
    static_assert(NS / 2 <= 8 && NS / 2 <= kWaves, "one sign vector per wavefront");
    if (wave < NS / 2) {
      double mx = -INFINITY, mn = INFINITY;
      float c2 = 0.0f, a1 = 0.0f;
      bool lo_any = false;
      for (int j = l; j < N; j += 64) {
        double sd = 0.0;
        float s2 = 0.0f, n1 = 0.0f;
#pragma unroll
        for (int q = 0; q < KB; ++q) {
          const float cv = Cs[cs_at<KB, N>(j) + q];
          sd += ((wave >> q) & 1) ? -(double)cv : (double)cv;
          s2 = fmaf(cv, cv, s2);
          n1 += fabsf(cv);
          lo_any |= (float)(_Float16)cv != cv;
        }
        mx = fmax(mx, sd);
        mn = fmin(mn, sd);
        c2 = fmaxf(c2, s2);
        a1 = fmaxf(a1, n1);
      }
      const double span = wave_max64(mx) + wave_max64(-mn);
      if (l == 0) pspan[wave] = span;
      if (wave == 0) {
        c2 = wave_max(c2);
        a1 = wave_max(a1);
        const bool la = __any(lo_any);
        if (l == 0) {
          cst[0] = __float_as_uint(c2);
          cst[1] = __float_as_uint(a1);  // max |c|_1
          cst[2] = la ? 1u : 0u;
        }
      }
    }
  }
  // the screen's A operands: row rho = 8 i + 4 hh + e of set s is codeword
  // 16 s + 4 i + e of the block on K half hh
  for (int e = threadIdx.x; e < (GRID ? 0 : NSET * 64); e += kThr) {
    const int s = e >> 6, ln = e & 63;
    const int rho = ln & 31, kh = ln >> 5;
    const int j = 16 * s + 4 * (rho >> 3) + (rho & 3);
    const bool on = kh == ((rho >> 2) & 1);
    _Float16 hi[KB], lo[KB];
    float s2 = 0.0f;
#pragma unroll
    for (int q = 0; q < KB; ++q) {
      const float cv = Cs[cs_at<KB, N>(j) + q];
      const _Float16 c16 = (_Float16)cv;
      hi[q] = (_Float16)((float)c16 * 0x1p10f);
      lo[q] = (_Float16)((cv - (float)c16) * 0x1p10f);
      s2 = fmaf(cv, cv, s2);
    }
    _Float16 a[8], b[8];
    if (KB == 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = hi[q];
        a[4 + q] = hi[q];
        b[q] = lo[q];
        b[4 + q] = (_Float16)0.0f;
      }
    } else {
      const float n = s2 * 0x1p9f;  // 2^10 |c|^2 / 2
      const _Float16 nh = (_Float16)n;
      const _Float16 nl = (_Float16)(n - (float)nh);
      a[0] = hi[0]; a[1] = hi[1]; a[2] = hi[0]; a[3] = hi[1];
      a[4] = lo[0]; a[5] = lo[1]; a[6] = -nh;   a[7] = -nl;
#pragma unroll
      for (int q = 0; q < 8; ++q) b[q] = (_Float16)0.0f;
    }
    uint32_t wa[4], wb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const _Float16 z0 = (_Float16)0.0f;
      wa[q] = (uint32_t)__builtin_bit_cast(uint16_t, on ? a[2 * q] : z0) |
              ((uint32_t)__builtin_bit_cast(uint16_t, on ? a[2 * q + 1] : z0) << 16);
      wb[q] = (uint32_t)__builtin_bit_cast(uint16_t, on ? b[2 * q] : z0) |
              ((uint32_t)__builtin_bit_cast(uint16_t, on ? b[2 * q + 1] : z0) << 16);
    }
    Ascr[e] = uint4{wa[0], wa[1], wa[2], wa[3]};
    if (KB == 4) Alos[e] = uint4{wb[0], wb[1], wb[2], wb[3]};
  }
  if (KB == 4 || TP) {
    for (int j = threadIdx.x; j < N; j += kThr) {
      float s2 = 0.0f;
#pragma unroll
      for (int q = 0; q < KB; ++q) s2 = fmaf(Cs[cs_at<KB, N>(j) + q], Cs[cs_at<KB, N>(j) + q], s2);
      Ini[(j >> 4) * kIStr + (j & 15)] = -0x1p17f * s2;  // codeword 16 s + r
    }
  }
  __syncthreads();
  C = Cs;
  if constexpr (GRID) {
    // Candidates of a cell: a codeword b is left out when the codeword a
    // nearest the cell's centre is closer than b to every point of the cell
    // widened by 2^-14 (more than the error of y, so that the exact block
    // lies in the widened cell of the computed one).  |p - a|^2 - |p - b|^2 =
    // |a|^2 - |b|^2 - 2 p.(a - b) is linear in p: its maximum over the box is
    // the value at the centre plus 2 h (|a_0 - b_0| + |a_1 - b_1|).  The
    // float32 evaluation errs by far less than tau, so no candidate is lost.
    const float gc2 = __uint_as_float(cst[0]);
    const float tau = 0x1p-16f * (1.0f + 2.0f * gc2 + 8.0f * sqrtf(gc2));
    constexpr float hw = kGR / kGS;
    const float he = hw + 0x1p-14f;
    for (int j = threadIdx.x; j <= N; j += kThr) {
      if (j < N) {
        const float c0 = Cs[cs_at<KB, N>(j)], c1 = Cs[cs_at<KB, N>(j) + 1];
        float s2 = 0.0f;
        s2 = fmaf(c0, c0, s2);
        s2 = fmaf(c1, c1, s2);
        Cw[j] = f4{c0, c1, -0x1p17f * s2, __uint_as_float((uint32_t)j)};
      } else {
        Cw[j] = f4{0.0f, 0.0f, -0x1p120f, __uint_as_float((uint32_t)N)};
      }
    }
    for (int cell = threadIdx.x; cell < kGS * kGS; cell += kThr) {
      const float cx = -kGR + (float)(2 * (cell / kGS) + 1) * hw;
      const float cy = -kGR + (float)(2 * (cell % kGS) + 1) * hw;
      float bd = INFINITY;
      int bi = 0;
      for (int j = 0; j < N; ++j) {
        const float dx = cx - Cs[cs_at<KB, N>(j)], dy = cy - Cs[cs_at<KB, N>(j) + 1];
        const float dd = fmaf(dx, dx, dy * dy);
        if (dd < bd) { bd = dd; bi = j; }
      }
      const float a0 = Cs[cs_at<KB, N>(bi)], a1 = Cs[cs_at<KB, N>(bi) + 1];
      const float an = fmaf(a0, a0, a1 * a1);
      uint32_t w0 = 0x01010101u * (uint32_t)N, w1 = 0x0101u * (uint32_t)N;
      int cnt = 0;
      for (int j = 0; j < N; ++j) {
        const float b0 = Cs[cs_at<KB, N>(j)], b1 = Cs[cs_at<KB, N>(j) + 1];
        const float dx = a0 - b0, dy = a1 - b1;
        const float f = (an - fmaf(b0, b0, b1 * b1)) - 2.0f * fmaf(cx, dx, cy * dy) +
                        2.0f * he * (fabsf(dx) + fabsf(dy));
        if (!(f < -tau)) {
          if (cnt < 4) w0 = (w0 & ~(0xFFu << (8 * cnt))) | ((uint32_t)j << (8 * cnt));
          else if (cnt < kGCap) w1 = (w1 & ~(0xFFu << (8 * (cnt - 4)))) | ((uint32_t)j << (8 * (cnt - 4)));
          ++cnt;
        }
      }
      if (cnt > kGCap) w1 |= 1u << 16;
      Tab[cell] = uint2{w0, w1};
    }
    __syncthreads();
  }

  // ---- bound on the screen's error for the difference of two candidates'
  // G (|y| <= 1): rotation accumulation times max |c_a - c_b|_1 (per output
  // the hi x hi products of one K step pass through one matrix-core
  // accumulation of 16 terms, <= 1 ulp each, and three float32 additions; the
  // parts below 2^-8 of them through <= 6 accumulations, ~1 ulp more; with
  // sum_j |Pi_ij x_j| <= |x|: < 21 ulp of |x|); nu (the sum of squares in
  // four chains of four dot products, <= 2 ulp each, and three additions:
  // < 10 ulp, so nu < 2^-20.6 relative), reciprocal and the hi/lo split of y
  // (2^-20 + 2^-22 relative) times 2 cmax; the screen accumulation, per key
  // <= (terms + 1) ulp of the largest partial magnitude gabs =
  // cmax + cmax^2 / 2 (k = 4: 8 products and the start, plus a residual
  // product pass of 4; the float32 rescore of phase two: 5 roundings; k = 2:
  // 8 products), for the two keys of a gap; the binary16 norm term and a
  // residual codebook; 25 %.  The packed index bits (< 16 ulp of each of the
  // two keys) are added per block, from the keys.
  const float cmax2 = __uint_as_float(cst[0]) * (1.0f + 1e-6f);
  double pmax = 0.0;
#pragma unroll
  for (int w = 0; w < (1 << KB) / 2; ++w) pmax = fmax(pmax, pspan[w]);
  const float l1max = (float)(pmax + 0x1p-50 * (double)__uint_as_float(cst[1])) * (1.0f + 1e-6f);
  const bool has_lo = cst[2] != 0u;
  const float cmax = sqrtf(cmax2) * (1.0f + 1e-6f);
  const float gabs = (cmax + 0.5f * cmax2) * (1.0f + 1e-6f);
  const float e_rot = (1.02f * 21.0f * 0x1p-23f + 0x1p-25f + 0x1p-22f) * l1max;
  const float e_nu = (0x1p-20f + 0x1p-22f) * 2.0f * cmax;
  const float kAcc = KB == 4 ? (has_lo ? 72.0f : 48.0f) : 40.0f;  // half-ulps of gabs, two keys
  const float e_acc = kAcc * 0x1p-24f * gabs + 0x1p-21f * cmax2 + (has_lo ? 0x1p-21f * cmax : 0.0f);
  // operands stay inside the binary16 range for |c| <= 8; beyond it every
  // block takes the float64 path
  const float margin = cmax2 <= 64.0f
                           ? 0x1p18f * (1.25f * (e_rot + e_nu + e_acc) + 4.0f * 0x1p-24f * gabs)
                           : INFINITY;
  constexpr float kPack = 1.25f * 16.0f * 0x1p-23f;  // per unit of key magnitude


  auto run = [&](auto has_lo_tag) {
  constexpr bool HL = decltype(has_lo_tag)::value && KB == 4;
  int qn = 0;  // deferred near ties in this wavefront's queue
  // the key mask in a register (an and-or takes no literal beside an
  // inline constant)
  uint32_t kmask = ~15u;
  asm volatile("" : "+v"(kmask));
  int slot = 0;
  while (queue[0] >= 0) {
    const int64_t tile = queue[0];
    if (queue[kDepth - 1] >= 0) vm_wait<4 * (kDepth - 1)>();
    else vm_wait<0>();
    const unsigned char* sl = myring + slot * kSlot;
    const int64_t vg = tile * kTile + v;
    const bool live = vg < n_vec;
    uint32_t rdo[4];
    {
      uint32_t rr = rrow, rx = rsw;
      asm volatile("" : "+v"(rr), "+v"(rx));  // not hoisted out of the loop
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) rdo[kap] = rr + ((32u * kap) ^ rx);
    }
    f16v z[2];
    float ss;
    {
      uint4 xc[4];
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) xc[kap] = *reinterpret_cast<const uint4*>(sl + rdo[kap]);
      // norm: dot products of exact products, float32 accumulation in four
      // chains of four (then two additions, and one across the halves)
      float sk[4];
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) {
        const uint32_t w4[4] = {xc[kap].x, xc[kap].y, xc[kap].z, xc[kap].w};
        sk[kap] = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (DT == 0) {
            const bf2 p2 = __builtin_bit_cast(bf2, w4[q]);
            sk[kap] = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, sk[kap], false);
          } else {
            const h2 p2 = __builtin_bit_cast(h2, w4[q]);
            sk[kap] = __builtin_amdgcn_fdot2(p2, p2, sk[kap], false);
          }
        }
      }
      ss = (sk[0] + sk[1]) + (sk[2] + sk[3]);
      // rotation: z[t] = rows of (Pi x) for tile t.  One accumulator per
      // 16-column K step, small parts first and the hi x hi products last, so
      // that those (nearly all of |Pi x|) pass through one matrix-core
      // accumulation and three float32 additions only
      z[0] = f16v{};
      z[1] = f16v{};
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) {
        bf8 xh, xl;
        if (DT == 0) {
          xh = __builtin_bit_cast(bf8, xc[kap]);
          xl = xh;  // unused
        } else {
          // an fp16 row as bf16 hi + lo (exact)
          const uint32_t w4[4] = {xc[kap].x, xc[kap].y, xc[kap].z, xc[kap].w};
          uint32_t hw[4], lw[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            // the hardware's packed conversion rounds to nearest even, as the
            // integer rounding of the rotation operands does; the remainders
            // are bf16 values, so their conversion is exact
            const float f0 = half_bits_to_float((uint16_t)(w4[q] & 0xFFFFu));
            const float f1 = half_bits_to_float((uint16_t)(w4[q] >> 16));
            const uint32_t hb = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)f0, (__bf16)f1});
            const float r0 = f0 - __uint_as_float(hb << 16);
            const float r1 = f1 - __uint_as_float(hb & 0xFFFF0000u);
            hw[q] = hb;
            lw[q] = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)r0, (__bf16)r1});
          }
          xh = __builtin_bit_cast(bf8, u4v{hw[0], hw[1], hw[2], hw[3]});
          xl = __builtin_bit_cast(bf8, u4v{lw[0], lw[1], lw[2], lw[3]});
        }
        f16v acc[2] = {f16v{}, f16v{}};
        // stages (Pi part, x part): (lo, mid, hi) x lo for fp16 rows, then
        // (lo, mid) x hi, then hi x hi
#pragma unroll
        for (int st = (DT == 0 ? 3 : 0); st < 6; ++st) {
          const int sp = 2 - st % 3;
#pragma unroll
          for (int t = 0; t < 2; ++t)
            acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf8, Pops[((t * 4 + kap) * 3 + sp) * 64 + l]),
                st < 3 ? xl : xh, acc[t], 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) z[t] += acc[t];
        // keep the scheduler from hoisting the next K step's operands
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    ss = sum_halves(ss);
    const float nu = __builtin_amdgcn_sqrtf(ss);
    const float inv = 0x1p8f * __builtin_amdgcn_rcpf(nu);  // 2^8 / nu
    const float inv1024 = inv * 0x1p10f;                     // exact
    const uint16_t h_a = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f - 0x1p-20f)));
    const uint16_t h_b = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f + 0x1p-20f)));
    uint32_t hdr = h_a;

    // ---- screen: 8 blocks of this lane at a time, codeword sets outermost
    // indices go straight into this lane's payload words (index m at bits
    // [m W, (m + 1) W), this lane's blocks placed as for the lower half; the
    // upper half's are moved up by W (8 / k) bits at the store); um marks the
    // near-tie blocks
    uint32_t wd[PW];
#pragma unroll
    for (int w = 0; w < PW; ++w) wd[w] = 0u;
    auto put = [&](int q, uint32_t val) {  // q compile-time after unrolling
      const int t = q / (NBL / 2), rq = q % (NBL / 2);
      const int i = rq / (4 / KB), j = rq % (4 / KB);
      const int b0 = (8 / KB) * (4 * t + 2 * (i >> 1)) + (4 / KB) * (i & 1) + j;
      const int bit = W * b0, w0 = bit >> 5, sh = bit & 31;
      constexpr uint32_t msk = (1u << W) - 1u;
      wd[w0] = (wd[w0] & ~(msk << sh)) | (val << sh);
      if (sh + W > 32) wd[w0 + 1] = (wd[w0 + 1] & ~(msk >> (32 - sh))) | (val >> (32 - sh));
    };
    uint32_t um = 0u;
    if constexpr (GRID) {
      // per block: the cell of 2^18 y, its candidates scored in float32 as
      // 2^18 (<y, c> - |c|^2 / 2) (the codeword number in the keys' 6 low
      // bits) and the best two; a block outside the grid or in a cell with
      // more than kGCap candidates is a near tie (float64)
      constexpr float gsc = 0x1p-18f * (float)kGS / (2.0f * kGR);
      constexpr float goff = 0.5f * (float)kGS;
      constexpr float kPackG = 1.25f * 64.0f * 0x1p-23f;  // 6 index bits
      uint32_t km = ~63u;
      asm volatile("" : "+v"(km));
#pragma unroll
      for (int q = 0; q < NBL; ++q) {
        const int t = q / (NBL / 2), rq = q % (NBL / 2);
        const int i = rq / (4 / KB), j = rq % (4 / KB);
        const float y0 = z[t][4 * i + KB * j] * inv1024;
        const float y1 = z[t][4 * i + KB * j + 1] * inv1024;
        const float u0 = fmaf(y0, gsc, goff), u1 = fmaf(y1, gsc, goff);
        const bool in = u0 >= 0.0f && u0 < (float)kGS && u1 >= 0.0f && u1 < (float)kGS;
        const int cell = in ? (int)u0 * kGS + (int)u1 : 0;
        const uint2 ent = Tab[cell];
        float t1 = -INFINITY, t2 = -INFINITY;
#pragma unroll
        for (int e = 0; e < kGCap; ++e) {
          const uint32_t cj = ((e < 4 ? ent.x : ent.y) >> (8 * (e & 3))) & 255u;
          const f4 cw = Cw[cj];
          const float g = fmaf(y0, cw[0], fmaf(y1, cw[1], cw[2]));
          const float key = __uint_as_float((__float_as_uint(g) & km) | __float_as_uint(cw[3]));
          t2 = __builtin_amdgcn_fmed3f(t1, t2, key);
          t1 = fmaxf(t1, key);
        }
        put(q, __float_as_uint(t1) & 63u);
        const float mq = fmaf(kPackG, fabsf(t1) + fabsf(t2), margin);
        const bool bad = !in || (ent.y & 0x10000u) != 0u;
        um |= (uint32_t)((!(t1 - t2 >= mq) || bad) && live) << q;
      }
    } else {
#pragma unroll
    for (int grp = 0; grp < NBL / GB; ++grp) {
      h8 yb[GB];
      float t1[GB], t2[GB];
      uint32_t bs[GB];  // codeword set of t1
#pragma unroll
      for (int qq = 0; qq < GB; ++qq) {
        const int q = grp * GB + qq;
        // lane block q: tile t, row group i, pair j (k = 2)
        const int t = q / (NBL / 2), rq = q % (NBL / 2);
        const int i = rq / (4 / KB), j = rq % (4 / KB);
        _Float16 yh[KB], yl[KB];
#pragma unroll
        for (int dd = 0; dd < KB; ++dd) {
          const float zz = z[t][4 * i + KB * j + dd];
          const _Float16 hi = (_Float16)__builtin_fmaf(zz, inv, 0.0f);
          yh[dd] = hi;
          yl[dd] = (_Float16)__builtin_fmaf(zz, inv, -(float)hi);
        }
        if (KB == 4) {
          yb[qq] = h8{yh[0], yh[1], yh[2], yh[3], yl[0], yl[1], yl[2], yl[3]};
        } else {
          const _Float16 s8 = (_Float16)256.0f;
          yb[qq] = h8{yh[0], yh[1], yl[0], yl[1], yh[0], yh[1], s8, s8};
        }
        t1[qq] = -INFINITY;
        t2[qq] = -INFINITY;
        bs[qq] = 0u;
      }
#pragma unroll 2
      for (int s = 0; s < NSET; ++s) {
        const h8 A = __builtin_bit_cast(h8, Ascr[s * 64 + l]);
        h8 Al = {};
        if (HL) Al = __builtin_bit_cast(h8, Alos[s * 64 + l]);
        f16v ini = {};
        if (KB == 4) ini = *reinterpret_cast<const f16v*>(Ini + kIStr * s);
#pragma unroll
        for (int qq = 0; qq < GB; ++qq) {
          f16v gq = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, yb[qq], ini, 0, 0, 0);
          if (HL) gq = __builtin_amdgcn_mfma_f32_32x32x16_f16(Al, yb[qq], gq, 0, 0, 0);
          // keys: the codeword's number within the set in the 4 low
          // mantissa bits (one and-or with a register mask and an inline
          // constant); the set of the best is tracked beside it.  Four
          // candidates at a time: with t1 >= t2 the best two of
          // {t1, t2, a, b} are u = max3(t1, a, b) and max(t2, med3(t1, a, b));
          // adding c, d the best is max3(u, c, d) and the second
          // max3(t2, med3(t1, a, b), med3(u, c, d))
          if constexpr (TP) {
            // phase 1: the set's largest score, its set number in the key's
            // 4 low bits; best two set maxima per block
            // (med3(a, b, 2^100) = max(a, b) for keys far below 2^100 takes
            // the matrix-core results without the quieting fmaxf would add)
            float m = __builtin_amdgcn_fmed3f(gq[0], gq[1], 0x1p100f);
#pragma unroll
            for (int r = 2; r < 16; r += 2) m = fmaxf(fmaxf(m, gq[r]), gq[r + 1]);
            const float mk = __uint_as_float((__float_as_uint(m) & kmask) | (uint32_t)s);
            t2[qq] = __builtin_amdgcn_fmed3f(t1[qq], t2[qq], mk);
            t1[qq] = __builtin_amdgcn_fmed3f(t1[qq], mk, 0x1p100f);
          } else {
            const float t1o = t1[qq];
#pragma unroll
            for (int r = 0; r < 16; r += 4) {
              float kc[4];
#pragma unroll
              for (int e = 0; e < 4; ++e)
                kc[e] = __uint_as_float((__float_as_uint(gq[r + e]) & kmask) | (uint32_t)(r + e));
              const float u = fmaxf(fmaxf(t1[qq], kc[0]), kc[1]);
              const float m1 = __builtin_amdgcn_fmed3f(t1[qq], kc[0], kc[1]);
              const float m2 = __builtin_amdgcn_fmed3f(u, kc[2], kc[3]);
              t1[qq] = fmaxf(fmaxf(u, kc[2]), kc[3]);
              t2[qq] = fmaxf(fmaxf(t2[qq], m1), m2);
            }
            // equal keys from two sets keep the earlier set (and give a zero
            // gap, so the block is redone in float64)
            if (NSET > 1) bs[qq] = t1[qq] != t1o ? (uint32_t)s : bs[qq];
          }
        }
      }
#pragma unroll
      for (int qq = 0; qq < GB; ++qq) {
        if constexpr (TP) {
          // phase 2: the 16 codewords of the best set in float32,
          // 2^18 (<y, c> - |c|^2 / 2) from 2^18 y = z 2^18 / nu; the second
          // best overall is the better of this set's second and the second
          // set maximum.  A wrong best set (set maxima within the bound)
          // leaves the gap below the bound.
          const int q = grp * GB + qq;
          const int t = q / (NBL / 2), rq = q % (NBL / 2);
          const int i = rq / (4 / KB), j = rq % (4 / KB);
          const uint32_t sb = __float_as_uint(t1[qq]) & 15u;
          float y8[KB];
#pragma unroll
          for (int dd = 0; dd < KB; ++dd) y8[dd] = z[t][4 * i + KB * j + dd] * inv1024;
          const float* cb = Cs + sb * cs_stride<KB, N>();
          const float* ib = Ini + sb * kIStr;
          float u1 = -INFINITY, u2 = -INFINITY;
#pragma unroll
          for (int r = 0; r < 16; r += 4) {
            const f4 iv = *reinterpret_cast<const f4*>(ib + r);
            float kc[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float g = iv[e];
              if (KB == 4) {
                const f4 cv = *reinterpret_cast<const f4*>(cb + (r + e) * 4);
#pragma unroll
                for (int dd = 0; dd < 4; ++dd) g = fmaf(y8[dd], cv[dd], g);
              } else {
                const float2 cv = *reinterpret_cast<const float2*>(cb + (r + e) * 2);
                g = fmaf(y8[0], cv.x, g);
                g = fmaf(y8[1], cv.y, g);
              }
              kc[e] = __uint_as_float((__float_as_uint(g) & kmask) | (uint32_t)(r + e));
            }
            const float u = fmaxf(fmaxf(u1, kc[0]), kc[1]);
            const float m1 = __builtin_amdgcn_fmed3f(u1, kc[0], kc[1]);
            const float m2 = __builtin_amdgcn_fmed3f(u, kc[2], kc[3]);
            u1 = fmaxf(fmaxf(u, kc[2]), kc[3]);
            u2 = fmaxf(fmaxf(u2, m1), m2);
          }
          put(q, (sb << 4) | (__float_as_uint(u1) & 15u));
          const float s2 = fmaxf(u2, t2[qq]);
          const float mq = fmaf(kPack, fabsf(u1) + fabsf(s2), margin);
          um |= (uint32_t)(!(u1 - s2 >= mq) && live) << q;
        } else {
          put(grp * GB + qq, (bs[qq] << 4) | (__float_as_uint(t1[qq]) & 15u));
          const float mq = fmaf(kPack, fabsf(t1[qq]) + fabsf(t2[qq]), margin);
          um |= (uint32_t)(!(t1[qq] - t2[qq] >= mq) && live) << (grp * GB + qq);
        }
      }
      // one group's work at a time (the scheduler would otherwise overlap
      // the groups and run out of registers)
      if (TP) __builtin_amdgcn_sched_barrier(0);
    }
    }

    // ---- fix-ups (the rare paths re-read this lane's row from the slot)
    bool zero = false;
    if (__any(ss == 0.0f)) {
      uint32_t o = 0;
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) {
        const uint4 xw = *reinterpret_cast<const uint4*>(sl + rdo[kap]);
        o |= xw.x | xw.y | xw.z | xw.w;
      }
      zero = or_halves(o & 0x7FFF7FFFu) == 0u;
      if (zero) {
        hdr = 0;
#pragma unroll
        for (int w = 0; w < PW; ++w) wd[w] = 0u;
        um = 0u;
      }
    }
    const bool wild = !(ss >= 0x1p-100f && ss <= 0x1p100f) && !zero;
    bool hdr_unsure = (h_a != h_b) && !wild && !zero;
    if (wild && live) {
      hdr_unsure = true;
      um = (NBL == 32) ? ~0u : ((1u << NBL) - 1u);
    }
    if (__any(hdr_unsure && live)) {
      double s64 = 0.0;
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) {
        const uint4 xw = *reinterpret_cast<const uint4*>(sl + rdo[kap]);
        const uint32_t w4[4] = {xw.x, xw.y, xw.z, xw.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const double a0 = (double)elem<DT>(w4[q] & 0xFFFFu), a1 = (double)elem<DT>(w4[q] >> 16);
          s64 = fma(a0, a0, s64);
          s64 = fma(a1, a1, s64);
        }
      }
      s64 = sum_halves64(s64);
      if (hdr_unsure) hdr = s64 > 0.0 ? f64_to_f16_bits(sqrt(s64)) : 0u;
    }
    // near ties: queued for a later batch when they fit (their stored indices
    // are patched when the queue is drained); else the inline pass below
    bool inline_pass = __ballot(um != 0u) != 0;
    if (inline_pass) {
      int cnt = 0;
#pragma unroll
      for (int q = 0; q < NBL; ++q) cnt += __popcll(__ballot((um >> q) & 1u));
      if (qn + cnt <= kQ) {
#pragma unroll
        for (int q = 0; q < NBL; ++q) {
          const uint64_t mk = __ballot((um >> q) & 1u);
          const int below = (int)__builtin_amdgcn_mbcnt_hi(
              (uint32_t)(mk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0u));
          if ((um >> q) & 1u) {
            const int t = q / (NBL / 2), rq = q % (NBL / 2);
            const int i = rq / (4 / KB), j = rq % (4 / KB);
            const int b0 = (8 / KB) * (4 * t + 2 * (i >> 1)) + (4 / KB) * (i & 1) + j;
            dq[wave * kQ + qn + below] = (vg << 5) | (int64_t)(b0 + (8 / KB) * h);
          }
          qn += __popcll(mk);
        }
        inline_pass = false;
      }
    }
    // the inline pass: B at a time (lane, block) pairs in lane-block order
    if (inline_pass) {
      constexpr int B = 64 / (8 * KB);
      int lng[B], qg[B];
#pragma unroll
      for (int gg = 0; gg < B; ++gg) { lng[gg] = 0; qg[gg] = 0; }
      int filled = 0, q = 0;
      uint64_t m = __ballot(um & 1u);
      for (;;) {
        while (filled < B && q < NBL) {  // the next (lane, block) pairs, in order
          if (m == 0) {
            if (++q < NBL) m = __ballot((um >> q) & 1u);
            continue;
          }
          const int ln = __builtin_ctzll(m);
          m &= m - 1;
#pragma unroll
          for (int gg = 0; gg < B; ++gg)
            if (filled == gg) {
              lng[gg] = ln;
              qg[gg] = q;
            }
          ++filled;
        }
        if (filled == 0) break;
        int vbg[4], bitg[B];
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) {
          const int ln = gg < filled && gg < B ? lng[gg < B ? gg : 0] : lng[0];
          const int qq = gg < filled && gg < B ? qg[gg < B ? gg : 0] : qg[0];
          const int t = qq / (NBL / 2), rq = qq % (NBL / 2);
          const int i = rq / (4 / KB), j = rq % (4 / KB);
          const int b0 = (8 / KB) * (4 * t + 2 * (i >> 1)) + (4 / KB) * (i & 1) + j;
          vbg[gg] = (ln & 31) + 32 * (b0 + (8 / KB) * (ln >> 5));
          if (gg < B) bitg[gg] = W * b0;  // position in this lane's (lower-half) words
        }
        uint32_t res[B];
        exact_batch<KB, N, DT>(sl, Pops, C, l, vbg[0], vbg[1], vbg[2], vbg[3], res);
        // the owning lane replaces the block's W bits (uniform shifts)
#pragma unroll
        for (int gg = 0; gg < B; ++gg) {
          const bool me = gg < filled && l == lng[gg];
          constexpr uint32_t msk = (1u << W) - 1u;
#pragma unroll
          for (int w = 0; w < PW; ++w) {
            const int sh = bitg[gg] - 32 * w;
            if (sh >= 32 || sh <= -W) continue;
            const uint32_t mk = sh >= 0 ? msk << sh : msk >> -sh;
            const uint32_t vv = sh >= 0 ? res[gg] << sh : res[gg] >> -sh;
            wd[w] = me ? ((wd[w] & ~mk) | vv) : wd[w];
          }
        }
        filled = 0;
      }
    }

    // ---- payload words of the vector (the upper half's blocks moved up)
    constexpr int S1 = W * (8 / KB);  // bit offset of the upper half's blocks
    constexpr int S1w = S1 >> 5, S1b = S1 & 31;
    uint32_t out[PW];
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      uint32_t up = 0u;
      if (w - S1w >= 0) up = S1b ? (wd[w - S1w] << S1b) : wd[w - S1w];
      if (S1b && w - S1w - 1 >= 0) up |= wd[w - S1w - 1] >> (32 - S1b);
      out[w] = or_halves(h ? up : wd[w]);
    }
    if (live) {
      uint32_t* dst = reinterpret_cast<uint32_t*>(payload + vg * P);
#pragma unroll
      for (int w = 0; w < PW; ++w)
        if ((w & 1) == h) dst[w] = out[w];
      if (h == 1) norms[vg] = (uint16_t)hdr;
    }
    while (qn >= 8) {
      defer_pass<KB, N, DT>(dq[wave * kQ + (l >> 3)], true, l, x, stride, R, Cs, payload);
      const int rest = qn - 8;  // move the queue's tail to its head
      int64_t te = 0;
      if (l < rest) te = dq[wave * kQ + 8 + l];
      if (l < rest) dq[wave * kQ + l] = te;
      qn = rest;
    }
#pragma unroll
    for (int d = 0; d + 1 < kDepth; ++d) queue[d] = queue[d + 1];
    queue[kDepth - 1] = claim();
    if (queue[kDepth - 1] >= 0) issue(queue[kDepth - 1], slot);
    slot = slot + 1 == kDepth ? 0 : slot + 1;
  }
  if (qn > 0) {  // qn < 8
    const int e = l >> 3;
    defer_pass<KB, N, DT>(dq[wave * kQ + (e < qn ? e : 0)], e < qn, l, x, stride, R, Cs, payload);
  }
  };
  if (has_lo) run(std::true_type{});
  else run(std::false_type{});
}

template <int KB, int N, int DT>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(3))) void encode_kernel(
    const uint16_t* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_body<KB, N, DT>(x, n_vec, stride, R, C, payload, norms);
}

}  // namespace encmf4

bool encode_mf4_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                        const float* R, const uint8_t* payload, const uint16_t* norms) {
  if (!(dtype == FIBQ_BF16 || dtype == FIBQ_F16) || s.d != 64) return false;
  if (!(s.k == 2 || s.k == 4) || !(s.N == 16 || s.N == 64 || s.N == 256)) return false;
  const uintptr_t ax = reinterpret_cast<uintptr_t>(x), ar = reinterpret_cast<uintptr_t>(R);
  const uintptr_t ap = reinterpret_cast<uintptr_t>(payload), an = reinterpret_cast<uintptr_t>(norms);
  // 32 rows of the input must lie within 2^31 bytes (32-bit copy offsets)
  return (ax % 16 == 0) && (stride % 8 == 0) && stride <= ((int64_t)1 << 24) && (ar % 4 == 0) &&
         (ap % 4 == 0) && (an % 2 == 0);
}

template <int KB, int N, int DT>
static int launch_mf4_t(const void* x, int64_t n_vec, int64_t stride, const float* R,
                        const float* C, uint8_t* payload, uint16_t* norms, int n_cu,
                        hipStream_t st) {
  const int64_t ntiles = (n_vec + encmf4::kTile - 1) / encmf4::kTile;
  const int64_t wgs = (ntiles + encmf4::kWaves - 1) / encmf4::kWaves;  // one per CU at most
  const int grid = (int)(wgs < n_cu ? wgs : n_cu);
  hipLaunchKernelGGL((encmf4::encode_kernel<KB, N, DT>), dim3(grid), dim3(encmf4::kWaves * 64), 0,
                     st, static_cast<const uint16_t*>(x), n_vec, stride, R, C, payload, norms);
  return (int)hipGetLastError();
}

int launch_encode_mf4(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                      const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                      void* stream, int n_cu) {
  hipStream_t st = static_cast<hipStream_t>(stream);
#define FIBQ_MF4(KK, NN)                                                                        \
  if (s.k == KK && s.N == NN)                                                                   \
    return dtype == FIBQ_BF16                                                                   \
               ? launch_mf4_t<KK, NN, 0>(x, n_vec, stride, R, C, payload, norms, n_cu, st)      \
               : launch_mf4_t<KK, NN, 1>(x, n_vec, stride, R, C, payload, norms, n_cu, st);
  FIBQ_MF4(4, 256) FIBQ_MF4(4, 64) FIBQ_MF4(4, 16) FIBQ_MF4(2, 256) FIBQ_MF4(2, 64) FIBQ_MF4(2, 16)
#undef FIBQ_MF4
  return (int)hipErrorInvalidValue;
}

}  // namespace dev
}  // namespace fibq
