// Encoder on the matrix cores for bf16 caches with d = 64, k = 8 and
// N in {16, 64} (the sub-one-bit long-context rates; Sec. 3.1, Eq. encode).
//
// One wavefront encodes 32 vectors per step (v_mfma_f32_32x32x16_*: lane l
// works on vector l % 32; the two half-wavefronts split the blocks):
//   input     tiles of 32 rows stream through a per-wavefront LDS ring filled
//             by global_load_lds_dwordx4 several tiles ahead;
//   norm      nu^2 = sum x^2 in float32 (packed bf16 dot products), nu = sqrt;
//             the binary16 header is certified by rounding nu (1 -+ delta),
//             delta above the float32 error; an uncertain header is redone in
//             float64 from the exact squares;
//   rotation  z = Pi x on the bf16 matrix cores: x is exact in bf16 and Pi
//             enters as two bf16 parts hi + mid (Pi = hi + mid + lo exactly),
//             so the products are exact and the float32 accumulation rounds;
//             the dropped part moves coordinate i of y = z / nu by at most
//             |lo_i|_2 (Cauchy-Schwarz with |x| = nu), and the largest row
//             norm of lo, computed from the same split, enters the bound.
//             The rows of Pi are permuted so that each lane ends up holding
//             four whole blocks of its vector (no shuffles);
//   screen    G_j = <y, c_j> - |c_j|^2 / 2 for every codeword (the
//             argmin of |y - c_j|^2 is the argmax of G_j), one fp16 MFMA per
//             16 codewords x 2 blocks: y = z / nu enters as fp16 hi + lo of
//             2^8 y (two products), the codebook as fp16 2^10 c (a codebook
//             that is not fp16-exact adds its residual); the scalings keep the
//             fp16 low parts in the normal range, so the result does not
//             depend on how the matrix cores treat fp16 subnormals.  The
//             accumulator starts at -2^18 |c_j|^2 / 2.  Each lane sees all N
//             candidates of its (vector, block) pairs and keeps the best two
//             (float max3 / med3) with the codeword number packed into the
//             low mantissa bits, which moves a key by less than N ulp;
//   exact     when the best two are closer than a rigorous bound on the
//             screen's error, the block is redone in float64 in the direct
//             form |y - c|^2 by the whole wavefront (rare), so every index is
//             the float64 argmin (lowest index on ties).
// Payload words are assembled across the two lanes of a vector and stored
// with coalesced writes; the headers likewise.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device_common.h"
#include "encode_mf_common.h"
#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {
namespace encmf {

constexpr int D = 64, K = 8;
constexpr int kTile = 32;   // vectors per wavefront step
constexpr int kSlot = kTile * 128;  // bytes of one input tile

using namespace mfc;

// Float64 nearest codeword of block m of one vector, computed by the whole
// wavefront: lane (r, c) = (l / 8, l % 8) forms the partial sums of row
// 8m + r of z = Pi x over dims 8c .. 8c+7 (x from the LDS tile, chunk c of a
// row at position c xor (row % 8); Pi and C from LDS); lane j then scores
// codeword j as |z - nu c_j|^2 = nu^2 |y - c_j|^2 (same argmin, no division).
// The minimum is taken over (score with its 6 lowest bits replaced by j):
// equal keys pick the lowest index, and scores agreeing to within 2^-46
// relative (far inside the near-tie window) count as ties.  All 64 lanes must
// be active.
template <int N>
__device__ __forceinline__ uint32_t exact_block(const unsigned char* tile, int vl,
                                                const float* Rl, const float* Cl, int m, int l) {
  const int r = l >> 3, c = l & 7;
  const uint4 raw = *reinterpret_cast<const uint4*>(tile + (vl >> 3) * 1024 + (vl & 7) * 128 +
                                                    16 * (c ^ (vl & 7)));
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  const float4 pa = *reinterpret_cast<const float4*>(Rl + (8 * m + r) * D + 8 * c);
  const float4 pb = *reinterpret_cast<const float4*>(Rl + (8 * m + r) * D + 8 * c + 4);
  const float pr[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
  double ss0 = 0.0, ss1 = 0.0, p0 = 0.0, p1 = 0.0;  // two short chains each
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const double x0 = (double)__uint_as_float(w[i] << 16);
    const double x1 = (double)__uint_as_float(w[i] & 0xFFFF0000u);
    ss0 = fma(x0, x0, ss0);
    ss1 = fma(x1, x1, ss1);
    p0 = fma((double)pr[2 * i], x0, p0);
    p1 = fma((double)pr[2 * i + 1], x1, p1);
  }
  const double ss = sum8(ss0 + ss1);
  const double zr = sum8(p0 + p1);  // z_{8m + r}, identical in lanes 8r .. 8r+7
  const double nu = sqrt(ss);
  if (!(nu > 0.0)) return 0u;  // uniform: zero or NaN norm stores index 0
  const uint64_t zu = (uint64_t)__double_as_longlong(zr);
  const int j = l < N ? l : 0;
  double dj = 0.0;
#pragma unroll
  for (int rr = 0; rr < K; ++rr) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)zu, 8 * rr);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(zu >> 32), 8 * rr);
    const double zb = __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
    const double t = fma(-nu, (double)Cl[j * K + rr], zb);
    dj = fma(t, t, dj);
  }
  uint64_t key = ((uint64_t)__double_as_longlong(dj) & ~(uint64_t)63) | (uint64_t)l;
  if (l >= N) key = ~(uint64_t)0;
  if (N <= 16) key = min16_64(key);  // candidates live in lanes 0 .. 15
  else key = wave_min64(key);
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)(key & 63));
}

template <int N, int WAVES, int DEPTH>
__device__ __forceinline__ void encode_body(const uint16_t* __restrict__ x, int64_t n_vec,
                                            int64_t stride, const float* __restrict__ R,
                                            const float* __restrict__ C,
                                            uint8_t* __restrict__ payload,
                                            uint16_t* __restrict__ norms) {
  constexpr int NSET = N / 16;  // codeword sets of 16 (one screen MFMA per block pair each)
  constexpr int W = (N == 16) ? 4 : 6;
  const int l = threadIdx.x & 63;
  const int h = l >> 5, v = l & 31;  // K half / row group, and vector (column) of this lane
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  constexpr int kThr = WAVES * 64;
  constexpr int kDepth = DEPTH;
  // LDS: per-wavefront rings of kDepth 4 KB input tiles; the rotation's MFMA
  // A operands (two bf16 parts of Pi in lane order, read per tile so that
  // they do not occupy registers); Pi and the codebook in fp32.
  constexpr int kRing = WAVES * kDepth * kSlot;
  constexpr int kOps = 2 * 4 * 2 * 64 * 16;
  __shared__ __align__(16) unsigned char smem[kRing + kOps + D * D * 4 + N * K * 4];
  uint4* Pops = reinterpret_cast<uint4*>(smem + kRing);
  float* Rs = reinterpret_cast<float*>(smem + kRing + kOps);
  float* Cs = reinterpret_cast<float*>(smem + kRing + kOps + D * D * 4);
  for (int i = threadIdx.x; i < D * D / 4; i += kThr)
    reinterpret_cast<float4*>(Rs)[i] = reinterpret_cast<const float4*>(R)[i];
  for (int i = threadIdx.x; i < N * K; i += kThr) Cs[i] = C[i];
  __shared__ int claim_ctr;  // tiles of this workgroup handed out so far
  __shared__ float lo2[D];   // |lo_i|_2^2 per row of Pi (the dropped third part)
  // near ties wait in a per-wavefront queue (vector, block) and are redone
  // eight at a time (see defer_pass below)
  constexpr bool kDefer = true;
  constexpr int kQ = 32;
  __shared__ int64_t dq_v[kDefer ? WAVES * kQ : 1];
  __shared__ int dq_m[kDefer ? WAVES * kQ : 1];
  const float* const Rg = R;  // Pi in global memory (the deferred pass reads it there)
  if (threadIdx.x == 0) claim_ctr = 0;
  for (int i = threadIdx.x; i < D; i += kThr) lo2[i] = 0.0f;
  __syncthreads();
  C = Cs;

  // ---- rotation operands (v_mfma_f32_32x32x16_bf16, A = rows of Pi in a
  // permuted order, the bf16 parts hi and mid).  Output row rho = 8 i + 4 hh + e
  // of tile t is dimension 8 (4 t + 2 (i / 2) + hh) + 4 (i % 2) + e, so the
  // lane of row group hh holds blocks hh, 2 + hh, 4 + hh, 6 + hh whole.
  for (int e = threadIdx.x; e < 2 * 4 * 64; e += kThr) {
    const int t = e >> 8, kap = (e >> 6) & 3, ln = e & 63;
    const int rho = ln & 31, i = rho >> 3, hh = (rho >> 2) & 1, ee = rho & 3;
    const int dim = 8 * (4 * t + 2 * (i >> 1) + hh) + 4 * (i & 1) + ee;
    const float* src = Rs + dim * D + 16 * kap + 8 * (ln >> 5);
    uint32_t part[2][4];
    float sq = 0.0f;  // squares of lo: exact (bf16 values), 8 terms
#pragma unroll
    for (int q = 0; q < 8; q += 2) {
      uint32_t hb[2], mb[2], lb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float vv = src[q + u];
        hb[u] = bf16_rne(vv);
        const float r1 = vv - bf16_val(hb[u]);  // exact
        mb[u] = bf16_rne(r1);
        const float r2 = r1 - bf16_val(mb[u]);  // exact, and exactly bf16
        lb[u] = bf16_rne(r2);
        sq = fmaf(bf16_val(lb[u]), bf16_val(lb[u]), sq);
      }
      part[0][q / 2] = hb[0] | (hb[1] << 16);
      part[1][q / 2] = mb[0] | (mb[1] << 16);
    }
#pragma unroll
    for (int sp = 0; sp < 2; ++sp)
      Pops[((t * 4 + kap) * 2 + sp) * 64 + ln] = uint4{part[sp][0], part[sp][1], part[sp][2], part[sp][3]};
    atomicAdd(&lo2[dim], sq);
  }
  __syncthreads();
  // largest |lo_i|_2 over the rows (64 exact squares summed in float32:
  // relative error below 2^-18, covered by the factor)
  const float lrot = sqrtf(wave_max(lo2[l])) * (1.0f + 0x1p-10f);

  // ---- screen operands (v_mfma_f32_32x32x16_f16 over a block pair: K half
  // hh of the B operand is the block 2p + hh).  Row rho = 8 i + 4 hh + e of
  // set s is codeword 16 s + 4 i + e of block 2p + hh: A holds it on K half
  // hh and zeros on the other; the accumulator starts at
  // -2^18 |c|^2 / 2; each lane's 16 accumulators are then all the
  // candidates 16 s + r (r = 4 i + e) of its own block.
  float cmax2 = 0.0f, l1max = 0.0f;
  bool lo_any = false;
  for (int j = l; j < N; j += 64) {
    float s2 = 0.0f;
#pragma unroll
    for (int q = 0; q < K; ++q) {
      const float cv = C[j * K + q];
      s2 = fmaf(cv, cv, s2);
      lo_any |= (float)(_Float16)cv != cv;
    }
    cmax2 = fmaxf(cmax2, s2);
  }
  for (int pr = l; pr < N * N; pr += 64) {  // max over pairs of |c_i - c_j|_1
    const int a = pr / N, b = pr % N;
    if (a < b) {
      float s1 = 0.0f;
#pragma unroll
      for (int q = 0; q < K; ++q) s1 += fabsf(C[a * K + q] - C[b * K + q]);
      l1max = fmaxf(l1max, s1);
    }
  }
  cmax2 = wave_max(cmax2) * (1.0f + 1e-6f);
  l1max = wave_max(l1max) * (1.0f + 1e-6f);
  const bool has_lo = __any(lo_any);
  const float cmax = sqrtf(cmax2) * (1.0f + 1e-6f);
  // Bound on the screen's error for the difference of two candidates' G
  // (y = Pi x / nu per block has |y| <= 1):
  //   rotation: bf16 x and Pi parts give exact products, <= 128 float32
  //     roundings (at most 2 ulp each) per output: |dy| <= 2^-17 per dim,
  //     plus the dropped part lo: |dy_i| <= |lo_i|_2 <= lrot; times
  //     max |c_i - c_j|_1;
  //   nu, hi/lo split: relative 2^-19 + 2^-22 of y, times max |c_i - c_j|;
  //   screen accumulation (<= 50 roundings of partial sums of magnitude
  //     <= gabs = cmax + cmax^2 / 2), the fp16 codebook residual and the
  //     packed index bits (< N ulp of a key of magnitude <= gabs);
  //   fp16 low parts of 2^8 y below the normal range: 2^-22 per dim.
  // Everything in units of G; the screen works in units of 2^18 G.
  const float gabs = (cmax + 0.5f * cmax2) * (1.0f + 1e-6f);
  const float e_rot = (1.02f * 0x1p-17f + 0x1p-25f + 0x1p-22f + lrot) * l1max;
  const float e_nu = (0x1p-19f + 0x1p-22f) * 2.0f * cmax;
  const float e_acc = 100.0f * 0x1p-24f * gabs + (has_lo ? 0x1p-21f * cmax : 0.0f);
  const float e_pack = 2.0f * gabs * (float)N * 0x1p-23f;
  const float margin =
      0x1p18f * (1.25f * (e_rot + e_nu + e_acc + e_pack) + 4.0f * 0x1p-24f * gabs);

  h8 Acb[NSET], Alo[NSET];
  f16v init[NSET];
#pragma unroll
  for (int s = 0; s < NSET; ++s) {
    const int rho = l & 31;
    const int j = 16 * s + 4 * (rho >> 3) + (rho & 3);
    const bool on = ((rho >> 2) & 1) == h;
#pragma unroll
    for (int q = 0; q < K; ++q) {
      const float cv = C[j * K + q];
      const _Float16 hi = (_Float16)cv;
      Acb[s][q] = on ? (_Float16)((float)hi * 0x1p10f) : (_Float16)0.0f;
      Alo[s][q] = on ? (_Float16)((cv - (float)hi) * 0x1p10f) : (_Float16)0.0f;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int jj = 16 * s + r;
      float s2 = 0.0f;
#pragma unroll
      for (int q = 0; q < K; ++q) s2 = fmaf(C[jj * K + q], C[jj * K + q], s2);
      init[s][r] = -0x1p17f * s2;
    }
  }

  // ---- persistent loop over 32-vector tiles, one wavefront per tile.
  // Each workgroup owns an equal contiguous range of tiles; its wavefronts
  // claim tiles one at a time from an LDS counter (the issue arbiter favours
  // older wavefronts, so a fixed split would leave a SIMD running a single
  // wavefront at the end).  Tile loads run kDepth tiles ahead through the
  // LDS ring: copy q of a tile moves rows 8q .. 8q+7; lane l takes 16 bytes
  // of row 8q + l / 8, chunk (l % 8) xor (l / 8), into position l, so each
  // row is one 128-byte burst and the transposed operand reads spread over
  // the LDS banks.  The last tile clamps its rows into [0, n_vec).
  const int64_t ntiles = (n_vec + kTile - 1) / kTile;
  const int64_t tb = ((int64_t)blockIdx.x * ntiles) / gridDim.x;
  const int64_t te = ((int64_t)(blockIdx.x + 1) * ntiles) / gridDim.x;
  auto claim = [&]() -> int64_t {
    int c = 0;
    if (l == 0) c = atomicAdd(&claim_ctr, 1);
    c = __builtin_amdgcn_readfirstlane(c);
    return tb + c < te ? tb + c : -1;
  };
  unsigned char* myring = smem + wave * kDepth * kSlot;
  const uint32_t ring = (uint32_t)(uintptr_t)myring;
  const int rih = l >> 3, chunk = (l & 7) ^ rih;
  // Copy q of a tile reads row 8q + rih at byte offset loff from the tile's
  // row 8q (the host keeps 32 rows of the input within 2^31 bytes, so the
  // offsets are 32-bit and the row addresses are wave-uniform).
  const uint32_t loff = (uint32_t)(((int64_t)rih * stride + 8 * chunk) * 2);
  auto issue = [&](int64_t tile, int slot) {
    const uint16_t* base = x + tile * kTile * stride;
    if ((tile + 1) * kTile <= n_vec) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        dma16s(loff, base + 8 * q * stride, ring + slot * kSlot + 1024 * q);
    } else {  // the ragged last tile clamps its rows into [0, n_vec)
      const int lim = (int)(n_vec - 1 - tile * kTile);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = min(8 * q + rih, lim);
        dma16s((uint32_t)((r * stride + 8 * chunk) * 2), base, ring + slot * kSlot + 1024 * q);
      }
    }
  };
  // operand chunks of this lane: row v, chunks 2 kap + h
  uint32_t rdo[4];
#pragma unroll
  for (int kap = 0; kap < 4; ++kap)
    rdo[kap] = (v >> 3) * 1024 + (v & 7) * 128 + 16 * ((2 * kap + h) ^ (v & 7));
  int64_t queue[kDepth];  // claimed tiles, in claim order (slot of queue[0] is `slot`)
#pragma unroll
  for (int d = 0; d < kDepth; ++d) {
    queue[d] = claim();
    if (queue[d] >= 0) issue(queue[d], d);
  }
  // the tile loop, compiled once per codebook kind (residual rows or not), so
  // that the hot part of a tile is one basic block
  // Deferred near ties: entries 0 .. n - 1 (n <= 8) of this wavefront's
  // queue, eight lanes each (all 64 lanes active).  Lane (e, c) =
  // (l / 8, l % 8) reads dims 8c .. 8c + 7 of entry e's row from global
  // memory and forms their share of z_{8m + r} (r = 0 .. 7, Pi's fp32 rows
  // from global memory) and of |x|^2 in float64; the eight lanes' sums give
  // z and nu, then codewords c, c + 8, ... are scored as |z - nu c_j|^2
  // (keys as in exact_block: ties within 2^-46 relative take the lowest
  // index; a zero or NaN norm gives index 0).  The stored index is replaced
  // with atomic and / or on the aligned 32-bit word(s) holding its W bits,
  // after the wavefront's earlier stores have completed: the atomics clear
  // and set only those bits, and a neighbour's plain stores touch only its
  // own bytes.
  auto defer_pass = [&](int n) {
    const int e = l >> 3, c = l & 7;
    const int ei = e < n ? e : 0;
    const int64_t dv = dq_v[wave * kQ + ei];
    const int m = dq_m[wave * kQ + ei];
    const uint4 raw = *reinterpret_cast<const uint4*>(x + dv * stride + 8 * c);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
    double xv[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xv[2 * i] = (double)__uint_as_float(w[i] << 16);
      xv[2 * i + 1] = (double)__uint_as_float(w[i] & 0xFFFF0000u);
    }
    double ss = 0.0;
#pragma unroll
    for (int u = 0; u < 8; ++u) ss = fma(xv[u], xv[u], ss);
    double z[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const float4 pa = *reinterpret_cast<const float4*>(Rg + (8 * m + r) * D + 8 * c);
      const float4 pb = *reinterpret_cast<const float4*>(Rg + (8 * m + r) * D + 8 * c + 4);
      const float pr[8] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
      double pz = 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u) pz = fma((double)pr[u], xv[u], pz);
      z[r] = sum8(pz);
    }
    const double nu = sqrt(sum8(ss));
    uint64_t key = ~(uint64_t)0;
#pragma unroll
    for (int jj = 0; jj < N / 8; ++jj) {
      const int j = c + 8 * jj;
      double dj = 0.0;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const double t = fma(-nu, (double)C[j * K + r], z[r]);
        dj = fma(t, t, dj);
      }
      key = umin64(key, ((uint64_t)__double_as_longlong(dj) & ~(uint64_t)63) | (uint64_t)j);
    }
    key = min_step(key, 0xB1);  // minimum over the eight lanes of the entry
    key = min_step(key, 0x4E);
    key = min_step(key, 0x141);
    const uint32_t bi = nu > 0.0 ? (uint32_t)(key & 63) : 0u;
    vm_wait<0>();  // this wavefront's payload stores have completed
    if (c == 0 && e < n) {
      constexpr uint32_t msk = (1u << W) - 1u;
      const int64_t bit = dv * (int64_t)(8 * W) + W * m;  // index m of vector dv
      uint32_t* pw = reinterpret_cast<uint32_t*>(payload) + (bit >> 5);
      const int sh = (int)(bit & 31);
      atomicAnd(pw, ~(msk << sh));
      atomicOr(pw, bi << sh);
      if (sh + W > 32) {  // the upper bits in the next word
        atomicAnd(pw + 1, ~(msk >> (32 - sh)));
        atomicOr(pw + 1, bi >> (32 - sh));
      }
    }
  };
  auto run = [&](auto has_lo_tag) {
  constexpr bool HAS_LO = decltype(has_lo_tag)::value;
  int slot = 0;
  int qn = 0;  // deferred near ties in this wavefront's queue
  while (queue[0] >= 0) {
    const int64_t tile = queue[0];
    // the tile's copies are older than the 4 (kDepth - 1) copies of the
    // tiles claimed after it (when all of those exist; else wait for all)
    if (queue[kDepth - 1] >= 0) vm_wait<4 * (kDepth - 1)>();
    else vm_wait<0>();
    const unsigned char* sl = myring + slot * kSlot;
    uint4 xc[4];
#pragma unroll
    for (int kap = 0; kap < 4; ++kap) xc[kap] = *reinterpret_cast<const uint4*>(sl + rdo[kap]);
    const int64_t vg = tile * kTile + v;
    const bool live = vg < n_vec;

    // norm (float32) and its certified binary16 header
    float ss = 0.0f;
#pragma unroll
    for (int kap = 0; kap < 4; ++kap) {
      const uint32_t w4[4] = {xc[kap].x, xc[kap].y, xc[kap].z, xc[kap].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bf2 p2 = __builtin_bit_cast(bf2, w4[q]);
        ss = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, ss, false);
      }
    }
    ss = sum_halves(ss);
    // hardware sqrt and reciprocal (1 ulp each; the bounds above allow 2^-19)
    const float nu = __builtin_amdgcn_sqrtf(ss);
    const float inv = 0x1p8f * __builtin_amdgcn_rcpf(nu);  // 2^8 / nu: the screen's scaling of y
    const uint16_t h_a = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f - 0x1p-19f)));
    const uint16_t h_b = __builtin_bit_cast(uint16_t, (_Float16)(nu * (1.0f + 0x1p-19f)));
    uint32_t hdr = h_a;

    // rotation: z[t] = rows of (Pi x) for tile t (small part first)
    f16v z[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      f16v a = {};
#pragma unroll
      for (int sp = 1; sp >= 0; --sp)
#pragma unroll
        for (int kap = 0; kap < 4; ++kap)
          a = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf8, Pops[((t * 4 + kap) * 2 + sp) * 64 + l]),
              __builtin_bit_cast(bf8, xc[kap]), a, 0, 0, 0);
      z[t] = a;
    }

    // screen, per block pair p: this lane sees block 2p + h of vector v
    uint32_t idx[4];
    bool unsure[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      h8 yh, yl;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float zz = z[p >> 1][4 * (2 * (p & 1) + (q >> 2)) + (q & 3)];
        const _Float16 hi = (_Float16)__builtin_fmaf(zz, inv, 0.0f);  // one mixed fma
        yh[q] = hi;
        yl[q] = (_Float16)__builtin_fmaf(zz, inv, -(float)hi);
      }
      float t1 = -INFINITY, t2 = -INFINITY;
#pragma unroll
      for (int s = 0; s < NSET; ++s) {
        f16v gq = __builtin_amdgcn_mfma_f32_32x32x16_f16(Acb[s], yh, init[s], 0, 0, 0);
        gq = __builtin_amdgcn_mfma_f32_32x32x16_f16(Acb[s], yl, gq, 0, 0, 0);
        if (HAS_LO) gq = __builtin_amdgcn_mfma_f32_32x32x16_f16(Alo[s], yh, gq, 0, 0, 0);
        // four candidates a, b, c, d at a time (the keys are distinct: the
        // low bits hold the codeword number): with t1 >= t2, the largest two
        // of {t1, t2, a, b} are u = max3(t1, a, b) and
        // max(t2, med3(t1, a, b)); adding c, d the largest is max3(u, c, d)
        // and the second max3(t2, med3(t1, a, b), med3(u, c, d))
#pragma unroll
        for (int r = 0; r < 16; r += 4) {
          float kc[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            kc[e] = __uint_as_float((__float_as_uint(gq[r + e]) & ~(uint32_t)(N - 1)) |
                                    (uint32_t)(16 * s + r + e));
          const float u = fmaxf(fmaxf(t1, kc[0]), kc[1]);
          const float m1 = __builtin_amdgcn_fmed3f(t1, kc[0], kc[1]);
          const float m2 = __builtin_amdgcn_fmed3f(u, kc[2], kc[3]);
          t1 = fmaxf(fmaxf(u, kc[2]), kc[3]);
          t2 = fmaxf(fmaxf(t2, m1), m2);
        }
      }
      idx[p] = __float_as_uint(t1) & (uint32_t)(N - 1);
      const float gap = t1 - t2;
      unsure[p] = !(gap >= margin) && live;
    }

    // ---- fix-ups after the branch-free part.  An all-zero row stores header
    // 0 and indices 0 (the float32 sum can underflow: test the bits).  A row
    // outside the float32 range where the bounds hold (or non-finite) has its
    // header and all 8 blocks redone in float64.
    bool zero = false;
    if (__any(ss == 0.0f)) {
      uint32_t o = 0;
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) o |= xc[kap].x | xc[kap].y | xc[kap].z | xc[kap].w;
      zero = or_halves(o & 0x7FFF7FFFu) == 0u;
      if (zero) {
        hdr = 0;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          idx[p] = 0;
          unsure[p] = false;
        }
      }
    }
    const bool wild = !(ss >= 0x1p-100f && ss <= 0x1p100f) && !zero;
    bool hdr_unsure = (h_a != h_b) && !wild && !zero;
    // ---- rare exact paths (wave-uniform loops)
    if (wild && live) {
      hdr_unsure = true;
#pragma unroll
      for (int p = 0; p < 4; ++p) unsure[p] = true;
    }
    if (__any(hdr_unsure && live)) {
      // float64 sum of the exact squares over this lane's 32 values
      double s64 = 0.0;
#pragma unroll
      for (int kap = 0; kap < 4; ++kap) {
        const uint32_t w4[4] = {xc[kap].x, xc[kap].y, xc[kap].z, xc[kap].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const double a0 = __uint_as_float(w4[q] << 16), a1 = __uint_as_float(w4[q] & 0xFFFF0000u);
          s64 = fma(a0, a0, s64);
          s64 = fma(a1, a1, s64);
        }
      }
      s64 = sum_halves64(s64);
      if (hdr_unsure) hdr = s64 > 0.0 ? f64_to_f16_bits(sqrt(s64)) : 0u;
    }
    uint64_t todo = __ballot(unsure[0] || unsure[1] || unsure[2] || unsure[3]);
    // (the tile of the last vector keeps the inline pass: at N = 64 the
    // 32-bit word holding its last index bits can reach past the payload)
    if (kDefer && todo && (tile + 1) * kTile < n_vec) {
      // near ties join this wavefront's queue (their stored indices are
      // patched when it is drained); a tile with more than the queue holds
      // (out-of-range rows) takes the inline pass below
      uint64_t mk[4];
      int cnt = 0;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        mk[p] = __ballot(unsure[p]);
        cnt += __popcll(mk[p]);
      }
      if (qn + cnt <= kQ) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int below = (int)__builtin_amdgcn_mbcnt_hi(
              (uint32_t)(mk[p] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mk[p], 0u));
          if (unsure[p]) {
            dq_v[wave * kQ + qn + below] = vg;
            dq_m[wave * kQ + qn + below] = 2 * p + h;
          }
          qn += __popcll(mk[p]);
        }
        todo = 0;
      }
    }
    while (todo) {  // near ties: the block in float64
      const int ln = __builtin_ctzll(todo);
      todo &= todo - 1;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if (__builtin_amdgcn_readlane((int)unsure[p], ln)) {
          const uint32_t bi = exact_block<N>(sl, ln & 31, Rs, C, 2 * p + (ln >> 5), l);
          if (l == ln) idx[p] = bi;
        }
      }
    }

    // ---- payload (little-endian bit stream, index m at bits [m W, (m+1) W))
    //      and header stores
    if (W == 4) {
      uint32_t part = 0;
#pragma unroll
      for (int p = 0; p < 4; ++p) part |= idx[p] << (4 * (2 * p + h));
      const uint32_t word = or_halves(part);
      if (live && h == 0) reinterpret_cast<uint32_t*>(payload)[vg] = word;
      if (live && h == 1) norms[vg] = (uint16_t)hdr;
    } else {
      uint64_t part = 0;
#pragma unroll
      for (int p = 0; p < 4; ++p) part |= (uint64_t)idx[p] << (6 * (2 * p + h));
      const uint32_t lo = or_halves((uint32_t)part), hi = or_halves((uint32_t)(part >> 32));
      uint16_t* p16 = reinterpret_cast<uint16_t*>(payload) + 3 * vg;
      if (live && h == 0) {
        p16[0] = (uint16_t)lo;
        p16[1] = (uint16_t)(lo >> 16);
      }
      if (live && h == 1) {
        p16[2] = (uint16_t)hi;
        norms[vg] = (uint16_t)hdr;
      }
    }
    if (kDefer) {
      while (qn >= 8) {
        defer_pass(8);
        const int rest = qn - 8;  // move the queue's tail to its head
        int64_t tv = 0;
        int tm = 0;
        if (l < rest) {
          tv = dq_v[wave * kQ + 8 + l];
          tm = dq_m[wave * kQ + 8 + l];
        }
        if (l < rest) {
          dq_v[wave * kQ + l] = tv;
          dq_m[wave * kQ + l] = tm;
        }
        qn = rest;
      }
    }
    // claim the next tile into the slot read in this iteration (its LDS reads
    // have completed: their values fed this tile's work)
#pragma unroll
    for (int d = 0; d + 1 < kDepth; ++d) queue[d] = queue[d + 1];
    queue[kDepth - 1] = claim();
    if (queue[kDepth - 1] >= 0) issue(queue[kDepth - 1], slot);
    slot = slot + 1 == kDepth ? 0 : slot + 1;
  }
  if (kDefer && qn > 0) defer_pass(qn);  // qn < 8 here
  };
  if (has_lo) run(std::true_type{});
  else run(std::false_type{});
}

// N = 16: one 768-thread workgroup per CU, three wavefronts per SIMD
// (<= 168 VGPRs), two tiles in flight per wavefront.  N = 64 holds four times
// the codebook operands: two wavefronts per SIMD (<= 256 VGPRs; the matrix
// and vector work of the two overlap), three ring slots each; at three per
// SIMD the compiler spills inside the tile loop.
constexpr int kWaves16 = 12, kDepth16 = 2, kWaves64 = 8, kDepth64 = 3;
__global__ __launch_bounds__(kWaves16 * 64) __attribute__((amdgpu_waves_per_eu(3))) void encode_kernel16(
    const uint16_t* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_body<16, kWaves16, kDepth16>(x, n_vec, stride, R, C, payload, norms);
}
__global__ __launch_bounds__(kWaves64 * 64) __attribute__((amdgpu_waves_per_eu(2))) void encode_kernel64(
    const uint16_t* __restrict__ x, int64_t n_vec, int64_t stride, const float* __restrict__ R,
    const float* __restrict__ C, uint8_t* __restrict__ payload, uint16_t* __restrict__ norms) {
  encode_body<64, kWaves64, kDepth64>(x, n_vec, stride, R, C, payload, norms);
}

}  // namespace encmf

bool encode_mfma_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                         const float* R, const uint8_t* payload, const uint16_t* norms) {
  if (dtype != FIBQ_BF16 || s.d != 64 || s.k != 8 || !(s.N == 16 || s.N == 64)) return false;
  const uintptr_t ax = reinterpret_cast<uintptr_t>(x), ar = reinterpret_cast<uintptr_t>(R);
  const uintptr_t ap = reinterpret_cast<uintptr_t>(payload), an = reinterpret_cast<uintptr_t>(norms);
  // 32 rows of the input must lie within 2^31 bytes (32-bit copy offsets)
  return (ax % 16 == 0) && (stride % 8 == 0) && stride <= ((int64_t)1 << 24) && (ar % 16 == 0) &&
         (ap % 4 == 0) && (an % 2 == 0);
}

int launch_encode_mfma(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                       const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                       void* stream, int n_cu) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t ntiles = (n_vec + encmf::kTile - 1) / encmf::kTile;
  const int wg_waves = s.N == 16 ? encmf::kWaves16 : encmf::kWaves64;
  const int64_t wgs = (ntiles + wg_waves - 1) / wg_waves;  // one workgroup per CU at most
  const int grid = (int)(wgs < n_cu ? wgs : n_cu);
  const uint16_t* xb = static_cast<const uint16_t*>(x);
  if (s.N == 16)
    hipLaunchKernelGGL(encmf::encode_kernel16, dim3(grid), dim3(encmf::kWaves16 * 64), 0, st, xb,
                       n_vec, stride, R, C, payload, norms);
  else
    hipLaunchKernelGGL(encmf::encode_kernel64, dim3(grid), dim3(encmf::kWaves64 * 64), 0, st, xb,
                       n_vec, stride, R, C, payload, norms);
  return (int)hipGetLastError();
}

}  // namespace dev
}  // namespace fibq
