/*
 * fibq.h -- C ABI of libfibq.so, the MI355X (gfx950) implementation of the
 * FibQuant random-access KV-cache codec (arXiv 2605.11478, "FibQuant:
 * Universal Vector Quantization for Random-Access KV-Cache Compression").
 *
 * Notation (Sec. 3.1): head dimension d, block dimension k (k | d), codebook
 * size N = 2^w, index width w = log2 N bits, rate b = w / k bits per
 * coordinate, shared orthogonal rotation Pi (d x d), shared codebook
 * C = {c_1..c_N} in the unit ball of R^k.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every function returns an int status (FIBQ_OK or a negative FIBQ_E*).
 *   Arguments are validated synchronously before anything is enqueued; on an
 *   error nothing is launched and no output is touched.  No C++ exception
 *   crosses the ABI and nothing aborts.
 * - (d, k, b, N) must satisfy: N a power of two with 1 <= w <= 16,
 *   |b * k - w| < 1e-9, 1 <= k <= d, d % k == 0.  Violations give
 *   FIBQ_EINVAL; valid shapes that have no kernel instantiation (see
 *   fibq_supported) give FIBQ_EUNSUPPORTED.
 * - Device entry points take device pointers (memory the caller allocated on
 *   the current HIP device and owns), enqueue their kernels on `stream`
 *   (a hipStream_t passed as void*, NULL = the default stream) and return
 *   without synchronising.  A launch failure is reported as FIBQ_EHIP.
 *   They allocate no device memory.
 * - Layouts are row-major and dense unless a stride argument says otherwise.
 * - The payload of one vector is P = ceil((d / k) * w / 8) bytes: a
 *   little-endian bit stream in which the index of block m occupies bits
 *   [m w, (m + 1) w) (byte j holds bits 8j .. 8j + 7, bit 0 least
 *   significant), trailing bits zero.  Indices are 0-based.  Vector v of a
 *   cache owns bytes [v P, (v + 1) P) of the payload array and element v of
 *   the norm array (IEEE binary16 bits): fixed rate, affine addresses
 *   (Sec. 3.1, Fig. 1 caption).
 * - The library keeps no global mutable state; concurrent calls on different
 *   streams are safe.
 */
#ifndef FIBQ_H
#define FIBQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FIBQ_OK 0
#define FIBQ_EINVAL (-1)        /* bad shape, rate, pointer or argument      */
#define FIBQ_EUNSUPPORTED (-2)  /* valid, but no kernel for this shape        */
#define FIBQ_EHIP (-3)          /* HIP launch / runtime error                 */
#define FIBQ_EIO (-4)           /* codebook file missing, short or corrupt    */
#define FIBQ_EWORKSPACE (-5)    /* workspace missing or too small             */

#define FIBQ_F32 0
#define FIBQ_F16 1
#define FIBQ_BF16 2

/* Human-readable text for a status code (static storage, never NULL). */
const char* fibq_strerror(int status);

/* Library version as major * 10000 + minor * 100 + patch. */
int fibq_version(void);

/* Payload bytes per vector, P = ceil((d/k) * log2(N) / 8) (Sec. 3.1: the
 * fixed-rate (d log2 N)/k-bit payload).  Returns P > 0, or FIBQ_EINVAL for an
 * invalid (d, k, N) (N must be a power of two, 2 <= N <= 65536, k | d). */
int fibq_payload_bytes(int d, int k, int N);

/* FIBQ_OK if (d, k, N) has device kernels for encode, decode and attention,
 * FIBQ_EUNSUPPORTED if the shape is valid but not instantiated, FIBQ_EINVAL
 * if it is invalid.  Instantiated: d in {64, 128} with k in {1, 2, 4, 8, 16},
 * and d = 64 with the large-block codes k in {32, 64}; 2 <= N <= 16384 and
 * N k <= 2^20 (codebooks up to 4 MB; those above 64 KB are read from global
 * memory instead of LDS). */
int fibq_supported(int d, int k, int N);

/* ------------------------------------------------------------------ host --
 * Offline construction of the two shared objects.  Host memory only, no GPU
 * needed.  Random draws come from Philox4x32-10 normals (the stream is
 * defined in the design notes); results are deterministic for a seed and do
 * not depend on n_threads. */

/* Haar-random orthogonal rotation Pi (Sec. 3 overview, Fig. 1 caption: one
 * matrix shared by all layers, heads, tokens, K and V): Q of the QR
 * factorisation of a d x d standard-normal matrix with diag(R) > 0, computed
 * in float64 and rounded once to float.  R_out: host, d*d floats, row-major,
 * y_i = sum_j Pi[i*d + j] x_j.  1 <= d <= 1024, else FIBQ_EINVAL. */
int fibq_build_rotation(int d, uint64_t seed, float* R_out);

/* Radial-angular codebook (Sec. 3.3; App. A codebook-construction table):
 * Beta-quantile radii (Eq. radii_main; closed form Eq. radii_k2 at k = 2)
 * times quasi-uniform directions (planar Fibonacci spiral at k = 2,
 * Fibonacci sphere at k = 3, Roberts-Kronecker at k >= 4, +/-1 at k = 1),
 * then `restarts` Lloyd-Max runs of `iters` rounds on M samples of the
 * spherical-Beta source f_{d,k} (Lemma 1), each run starting from the
 * initial codebook rotated by its own Haar k x k matrix; the run with the
 * lowest training MSE is kept; its codewords are finally rounded to
 * binary16-representable values (round to nearest, ties to even), which the
 * fused attention kernel reads exactly from an fp16 table (the effect on the
 * distortion is below 1e-4 dB).  M <= 0 selects max(100000, 30 N).
 * n_threads <= 0 uses all hardware threads.
 * C_out: host, N*k floats (codeword n at n*k).  train_mse_out (nullable):
 * per-block training MSE of the kept codebook.
 * k = d is the full-vector code (Sec. 5, "why a full-vector code can win"):
 * the source is then the whole normalised vector and the same steps apply.
 * Same as fibq_build_codebook_init with init = FIBQ_INIT_BETA. */
int fibq_build_codebook(int d, int k, double b, int N, uint64_t seed, int64_t M,
                        int restarts, int iters, int n_threads, float* C_out,
                        double* train_mse_out);

/* Starting codebooks for the same Lloyd-Max polish.
 * FIBQ_INIT_BETA: N Beta-quantile shells, one direction each (Eq. radii_main).
 * FIBQ_INIT_SHELL: the large-d shortcut of App. D (App. A table, last row):
 *   every codeword at the typical radius sqrt(k/d).
 * FIBQ_INIT_MULTISHELL: C(S, M_a) of App. E Eq. multishell, S shells at the
 *   Beta quantiles (s - 1/2)/S, shell s holding directions s*M_a+1 .. (s+1)*M_a
 *   of the sequence above (at k = 3 the latitude bands restart per shell, the
 *   azimuth continues); every factor pair S * M_a = N is tried on the training
 *   sample and the one with the lowest training MSE starts the polish (ties:
 *   the smaller S).  Codewords are shell-major. */
#define FIBQ_INIT_BETA 0
#define FIBQ_INIT_SHELL 1
#define FIBQ_INIT_MULTISHELL 2

/* fibq_build_codebook with a choice of starting codebook (`init`, one of the
 * FIBQ_INIT_* values, else FIBQ_EINVAL).  `shells` > 0 fixes S for
 * FIBQ_INIT_MULTISHELL (it must divide N; e.g. S = sqrt(N) for
 * fibq_encode_radius_first); 0 searches all factor pairs; any other use is
 * FIBQ_EINVAL.  `metric` (host, k*k doubles, row-major; NULL for the squared
 * Euclidean error) replaces ||x - c||^2 by (x - c)^T M (x - c) throughout
 * the Lloyd-Max polish: the task-weighted / Mahalanobis objective of Sec. 3
 * (the discussion after Eq. lattn); the cell mean stays the optimal centroid,
 * the payload and decoder are unchanged.  M must be symmetric (to 1e-12 of
 * its largest entry) and positive definite, else FIBQ_EINVAL.  shells_out
 * (nullable) receives the number of radial shells of the starting codebook
 * (N, 1 or S). */
int fibq_build_codebook_init(int d, int k, double b, int N, uint64_t seed, int64_t M,
                             int restarts, int iters, int n_threads, int init, int shells,
                             const double* metric, float* C_out, double* train_mse_out,
                             int* shells_out);

/* Write / read the codebook file (C, Pi and the two seeds; little-endian;
 * magic "FIBQCB01", u32 d, k, N, 0, u64 seeds, f32 C, f32 Pi, u64 FNV-1a-64
 * of all preceding bytes).  fibq_load_codebook with C == NULL or R == NULL
 * only reports the shape (query mode); `seeds` (nullable) receives 2 values.
 * Errors: FIBQ_EIO (cannot open, short, bad magic or checksum),
 * FIBQ_EINVAL (NULL path / shape pointers). */
int fibq_save_codebook(const char* path, int d, int k, int N, const float* C,
                       const float* R, uint64_t rotation_seed,
                       uint64_t codebook_seed);
int fibq_load_codebook(const char* path, int* d, int* k, int* N, float* C,
                       float* R, uint64_t* seeds);

/* ---------------------------------------------------------------- device -- */

/* Encoder (Sec. 3.1, Eq. encode): for each of n_vec vectors x_v (row v of
 * `x`, d elements of `dtype`, rows x_row_stride elements apart,
 * x_row_stride >= d):
 *   nu = ||x_v||_2, stored as binary16 (round-to-nearest-even) in norms[v];
 *   y = Pi (x_v / nu) (unrounded nu), cut into d/k blocks y^(m);
 *   i_m = argmin_j ||y^(m) - c_j||^2 (ties: lowest index), packed into
 *   payload[v*P .. v*P + P).
 * An all-zero vector stores norm 0 and indices 0.  Norms above the binary16
 * range store +inf.  R: device, d*d floats (row-major, as built above).
 * C: device, N*k floats.  payload: device, n_vec*P bytes.  norms: device,
 * n_vec uint16.  n_vec == 0 is a no-op. */
int fibq_encode(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride,
                int d, int k, double b, int N, const float* R, const float* C,
                uint8_t* payload, uint16_t* norms, void* stream);

/* Radius-first encoder (App. F, Stage 1), an approximate search for
 * multi-shell codebooks built with FIBQ_INIT_MULTISHELL and S = L shells
 * (C shell-major: shell l holds codewords l*N/L .. (l+1)*N/L - 1).  Block m
 * of y takes the shell l* whose radius r_l = sqrt(BetaInv((l + 1/2)/L; k/2,
 * beta_dk)) (Eq. multishell, the same radii as the builder) is nearest to
 * ||y^(m)||_2 (lower shell on ties) and stores l* N/L + the index of the
 * nearest codeword of that shell alone (ties: lowest index): O(L + N/L)
 * work per block instead of O(N).  Header, payload layout and the decoder
 * are those of fibq_encode; L = 1 is exactly fibq_encode's search.
 * L: a power of two dividing N, 1 <= L <= 256, else FIBQ_EINVAL.  Other
 * arguments, ownership and errors as fibq_encode. */
int fibq_encode_radius_first(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride,
                             int d, int k, double b, int N, int L, const float* R,
                             const float* C, uint8_t* payload, uint16_t* norms, void* stream);

/* Stage 2 tables for fibq_encode_list (App. F, hierarchical direction code),
 * host side: for each of the L shells of the shell-major codebook C (host,
 * N*k floats), spherical k-means of the shell's codeword directions into K
 * parents, started from codewords 0, s, 2s, .. (s = (N/L)/K), `rounds`
 * rounds of assignment by the largest inner product (first parent on ties)
 * and mean-direction update (a parent that empties keeps its direction),
 * then a final assignment.  mu_out: L*K*k doubles (parent p of shell l at
 * (l*K + p)*k); offsets_out: L*(K+1) ints, members_out: N ints: parent p of
 * shell l owns members_out[l*N/L + offsets_out[l*(K+1) + p] ..
 * l*N/L + offsets_out[l*(K+1) + p + 1]), the shell-local indices of its
 * codewords in increasing order.  Requires L | N, 1 <= K <= min(N/L, 64),
 * rounds >= 0, non-NULL pointers; else FIBQ_EINVAL. */
int fibq_build_parent_lists(const float* C, int N, int k, int L, int K, int rounds,
                            double* mu_out, int32_t* offsets_out, int32_t* members_out);

/* List-decoding encoder (App. F, Stages 1 + 2 composed), approximate: the
 * shell is chosen as in fibq_encode_radius_first; the shell's K parents are
 * ranked by <y^(m), mu_p> (float64, first parent on ties) and the codewords
 * of the best T parents are searched (float32 screen, float64 re-score of
 * near ties; lowest index on ties); the index is l* N/L + the shell-local
 * index.  T = K searches the whole shell (the radius-first result).  mu,
 * offsets, members: device copies of fibq_build_parent_lists' outputs for
 * the same C, L and K (L*K*k doubles, L*(K+1) and N ints).  Offsets and
 * members are clamped into their shell on the device, so other table
 * contents cannot read out of bounds (they only give a different search).  d = 64 with k in {4, 8, 16, 32} or d = 128 with k in
 * {4, 8, 16} (else FIBQ_EUNSUPPORTED); 1 <= T <= min(K, 8); L as in
 * fibq_encode_radius_first.  Other arguments, ownership and errors as
 * fibq_encode. */
int fibq_encode_list(const void* x, int dtype, int64_t n_vec, int64_t x_row_stride, int d, int k,
                     double b, int N, int L, int K, int T, const double* mu,
                     const int32_t* offsets, const int32_t* members, const float* R,
                     const float* C, uint8_t* payload, uint16_t* norms, void* stream);

/* Random-access decoder (Sec. 3.1 decoder; Sec. 6 "table lookup followed by
 * inverse rotation"): x_hat_i = nu * Pi^T (c_{i_1}, ..., c_{i_{d/k}}) with nu
 * the stored binary16 norm.  Output row i (d floats of x_hat, device) is
 * the vector t = token_ids[i] of the cache (payload row t, norms[t]), or
 * t = i when token_ids is NULL.  payload/norms hold n_cache vectors;
 * token_ids (device, nullable) holds n_vec int64 ids.  An id outside
 * [0, n_cache) yields a row of NaNs (the kernel checks every id).  With
 * token_ids == NULL, n_vec <= n_cache is required.  x_hat must be 16-byte
 * aligned (rows are stored as float4).  Violations give FIBQ_EINVAL. */
int fibq_decode(const uint8_t* payload, const uint16_t* norms,
                const int64_t* token_ids, int64_t n_vec, int64_t n_cache,
                int d, int k, double b, int N, const float* R, const float* C,
                float* x_hat, void* stream);

/* Workspace bytes fibq_attn_decode needs for this problem (0 for an invalid
 * one).  The workspace holds the rotated queries, the per-block query-codeword
 * tables and the split-K partial softmax states. */
size_t fibq_attn_workspace_bytes(int64_t n_groups, int G, int64_t T, int d,
                                 int k, int N);

/* Fused dequantisation + single-query decode attention (Eq. lattn with K, V
 * replaced by the decoded cache; Sec. 3.1 decoder; random access makes the
 * fusion possible, Sec. 1 and App. F):
 *   for group g (a (layer, batch, kv-head) triple, flattened by the caller)
 *   and its G query heads h (GQA: q-head h of the group shares its K, V):
 *   o_{g,h} = sum_t softmax_t(scale * <q_{g,h}, K_hat_{g,t}>) V_hat_{g,t},
 *   t = 0 .. T-1, no mask.  scale <= 0 selects 1/sqrt(d).
 * Computed in rotated space: the query is rotated once (q~ = Pi q, so
 * <q, K_hat_t> = nu_t <q~, c_(t)>), scores are sums of per-block
 * query-codeword dot products, values are accumulated as
 * sum_t p_t nu_t c_(t) and rotated back once (Pi^T) per head.
 * q: device [n_groups][G][d] of q_dtype.  k_payload/v_payload: device
 * [n_groups][T_stride][P] bytes; k_norms/v_norms: device
 * [n_groups][T_stride] binary16 bits (T <= T_stride: only the first T
 * tokens of each group are read).  out: device [n_groups][G][d] float.
 * workspace: device, at least fibq_attn_workspace_bytes(...) bytes, else
 * FIBQ_EWORKSPACE.  T == 0 writes zeros.  1 <= G <= 16. */
int fibq_attn_decode(const void* q, int q_dtype, const uint8_t* k_payload,
                     const uint16_t* k_norms, const uint8_t* v_payload,
                     const uint16_t* v_norms, int64_t n_groups, int G,
                     int64_t T, int64_t T_stride, int d, int k, double b,
                     int N, const float* R, const float* C, float scale,
                     float* out, void* workspace, size_t workspace_bytes,
                     void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid hipMalloc): the same
 * computation as fibq_attn_decode, with the same arguments, layouts, results
 * and errors, but without a workspace argument.  The workspace comes from a
 * static device array of FIBQ_ATTN_SCRATCH_BYTES bytes that the library owns:
 * one per GPU it runs on, held until the process ends, located on the first
 * call on each device.  The call allocates nothing (no hipMalloc / hipFree).
 * A problem whose fibq_attn_workspace_bytes exceeds FIBQ_ATTN_SCRATCH_BYTES
 * returns FIBQ_EWORKSPACE before anything is enqueued.  All calls on one GPU
 * share that GPU's array: calls that overlap in time on one GPU (different
 * streams or host threads without ordering) race and give wrong results;
 * calls ordered on one stream are safe. */
#define FIBQ_ATTN_SCRATCH_BYTES ((size_t)64 << 20)
int fibq_attn_decode_noalloc(const void* q, int q_dtype, const uint8_t* k_payload,
                             const uint16_t* k_norms, const uint8_t* v_payload,
                             const uint16_t* v_norms, int64_t n_groups, int G, int64_t T,
                             int64_t T_stride, int d, int k, double b, int N, const float* R,
                             const float* C, float scale, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FIBQ_H */
