// Internal declarations shared by the library's translation units.
#ifndef FIBQ_INTERNAL_H
#define FIBQ_INTERNAL_H

#include <stddef.h>
#include <stdint.h>

namespace fibq {

// Philox stream tags of the codebook construction.
constexpr uint32_t kTagRotation = 1;
constexpr uint32_t kTagTrain = 2;
constexpr uint32_t kTagRestart = 3;
constexpr uint32_t kTagRepair = 4;

namespace host {
void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
void normals(uint64_t seed, uint32_t tag, uint64_t start, uint64_t count, double* out);
void haar_q(int n, const double* A, double* Q);
double beta_inc(double a, double b, double x);
double beta_inc_inv(double a, double b, double p);
double norm_inv(double p);
void radii(int d, int k, int N, double* r);
void directions(int k, int N, double* u, int64_t offset = 0);
int build_rotation(int d, uint64_t seed, float* R_out);
int build_parent_lists(const float* C, int N, int k, int L, int K, int rounds, double* mu,
                       int32_t* offsets, int32_t* members);
double round_to_binary16(double x);
int build_codebook(int d, int k, int N, uint64_t seed, int64_t M, int restarts, int iters,
                   int n_threads, int init, int fixed_shells, const double* metric, float* C_out,
                   double* mse_out, int* shells_out);
int save_codebook(const char* path, int d, int k, int N, const float* C, const float* R,
                  uint64_t s0, uint64_t s1);
int load_codebook(const char* path, int* d, int* k, int* N, float* C, float* R, uint64_t* seeds);
}  // namespace host

// Device launchers (defined in the .hip files).  They assume validated
// arguments and return 0 or a HIP error code.
namespace dev {
struct Shape {
  int d, k, N, w, P;
};
int launch_encode(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s,
                  const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                  void* stream);
// Radius-first search over L shells (App. F Stage 1); radii: host, L values,
// increasing; L a power of two dividing N, at most 256.
int launch_encode_shells(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s, int L,
                         const double* radii, const float* R, const float* C, uint8_t* payload,
                         uint16_t* norms, void* stream);
// List decoding inside the radius-chosen shell (App. F Stage 2); mu, offsets,
// members: device tables of build_parent_lists.
int launch_encode_list(const void* x, int dtype, int64_t n_vec, int64_t stride, Shape s, int L,
                       const double* radii, int K, int T, const double* mu,
                       const int32_t* offsets, const int32_t* members, const float* R,
                       const float* C, uint8_t* payload, uint16_t* norms, void* stream);
int launch_decode(const uint8_t* payload, const uint16_t* norms, const int64_t* ids,
                  int64_t n_vec, int64_t n_cache, Shape s, const float* R, const float* C,
                  float* out, void* stream);
bool encode_mfma_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                         const float* R, const uint8_t* payload, const uint16_t* norms);
int launch_encode_mfma(const void* x, int64_t n_vec, int64_t stride, const Shape& s,
                       const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                       void* stream, int n_cu);
bool encode_mf4_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                        const float* R, const uint8_t* payload, const uint16_t* norms);
int launch_encode_mf4(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                      const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                      void* stream, int n_cu);
bool encode_big_applies(int dtype, const Shape& s, const void* x, int64_t stride,
                        const float* R, const float* C, const uint8_t* payload);
int launch_encode_big(const void* x, int dtype, int64_t n_vec, int64_t stride, const Shape& s,
                      const float* R, const float* C, uint8_t* payload, uint16_t* norms,
                      void* stream, int n_cu);
size_t attn_workspace_bytes(int64_t n_groups, int G, int64_t T, Shape s);
bool attn_fast_applies(int G, const Shape& s);
size_t attn_fast_workspace_bytes(int64_t n_groups, int64_t T);
bool attn_w4_applies(int G, const Shape& s);
bool attn_k4_applies(int G, const Shape& s);
size_t attn_k4_workspace_bytes(int64_t n_groups, int64_t T, const Shape& s);
size_t attn_w4_workspace_bytes(int64_t n_groups, int64_t T);
// The library's static attention scratch on the current device (its address
// is looked up once per device); 0 or a HIP error code.
int static_attn_scratch(void** ptr);
int launch_attn(const void* q, int q_dtype, const uint8_t* kp, const uint16_t* kn,
                const uint8_t* vp, const uint16_t* vn, int64_t n_groups, int G, int64_t T,
                int64_t T_stride, Shape s, const float* R, const float* C, float scale,
                float* out, void* ws, size_t ws_bytes, void* stream);
}  // namespace dev

}  // namespace fibq

#endif
