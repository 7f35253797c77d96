// Shared device-side definitions of the MoARa HIP library (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

enum { SIDE_LEFT = 1, SIDE_RIGHT = 2 };

// ---------------------------------------------------------------- descriptors
// One projected matrix as seen by the step kernels. Rebuilt on the host for
// every call (pointers to W and G change between calls) and uploaded as one
// array; per-kernel tile prefixes let one launch cover every matrix.
struct MatDev {
  const float* G;      // m x n fp32, row-major
  void* W;             // m x n, weight dtype
  int64_t m, n;        // rows, cols
  int32_t k;           // blocks per row = ceil(n / B)
  int32_t r;           // rank
  int32_t side;        // SIDE_LEFT (P is m x r) or SIDE_RIGHT (Q is n x r)
  int32_t L, s;        // L = uncompressed state dim, s = projected dim
  float* inv;          // m x k: 1 / (M + eps_d)
  float* dM;           // m x k: Optimizer_M output
  float* mag1;         // m x k: Optimizer_M moments
  float* mag2;
  float* exp1;         // L x r: Optimizer_V moments (row l, column j)
  float* exp2;
  void* N;             // L x r: Optimizer_V output in operand dtype
  const void* Pop;     // s x r projector, operand dtype
  const void* Ptop;    // r x s projector (transposed copy), operand dtype
  float bc1, bc2;      // 1 - beta1^t, 1 - beta2^t for this step
  uint32_t tile_dec;   // first WG index of this matrix in the decompose launch
  uint32_t tile_proj;  // ... in the projection launch
  uint32_t tile_back;  // ... in the back-projection launch
  int32_t vt;          // V output layout: 0 row-major m x n, 1 transposed n x m
  bf16* Vb;            // bf16 direction tensor V written by the decomposition (nullptr: none)
  int32_t n_bf16;      // zero-gradient step: N is bf16 (else fp32) ...
  int32_t n_kp;        // ... in the blocked layout kp_index(l, j, L)
  int32_t mom_bf16;    // zero-gradient step: exp1 / exp2 hold bf16 values
  int32_t pad_;
};

struct StepParams {
  int32_t B;            // block size
  int32_t nmat;
  int32_t decompose;    // 0: V = G, dM = 1
  int32_t weight_bf16;  // 1: W is bf16
  float beta1, beta2, adam_eps, decomp_eps;
  float lr, scale;
  uint32_t total_dec, total_proj, total_back;
};

// ---------------------------------------------------------------- helpers
// Blocked ("K-panel") layout of a bf16 GEMM operand with `rows` rows and reduction
// length K (a multiple of 32): element (i, k) sits at ((k / 32) * rows + i) * 32 + k % 32.
// The 64-byte row segments of one 32-wide K step of consecutive rows are then one
// contiguous run, which the large-tile GEMM streams with whole-line DMA loads.
__host__ __device__ __forceinline__ int64_t kp_index(int64_t i, int64_t k, int64_t rows) {
  return ((k >> 5) * rows + i) * 32 + (k & 31);
}

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }   // round to nearest even

// Bijective remap of the hardware dispatch order (round-robin over the 8 XCDs)
// so that consecutive logical tiles run on the same XCD and share its L2.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t nblk) {
  const uint32_t X = 8;
  uint32_t xcd = bid % X, idx = bid / X;
  uint32_t per = nblk / X, rem = nblk % X;
  return (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}

// Largest i with prefix(i) <= t, prefix read through a member pointer of MatDev.
template <typename F>
__device__ __forceinline__ int find_mat(const MatDev* mats, int nmat, uint32_t t, F prefix) {
  int lo = 0, hi = nmat - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (prefix(mats[mid]) <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Adam step of Kingma & Ba with bias correction terms passed in (no weight decay).
__device__ __forceinline__ float adam_out(float x, float& e, float& q, float b1, float b2,
                                          float eps, float bc1, float bc2) {
  e = b1 * e + (1.0f - b1) * x;
  q = b2 * q + (1.0f - b2) * x * x;
  return (e / bc1) / (sqrtf(q / bc2) + eps);
}

// The same step with the moments stored in bf16: the updated moments are rounded to bf16
// (nearest even) for storage and the output is formed from the stored values.
__device__ __forceinline__ float adam_out_bf16(float x, bf16& e, bf16& q, float b1, float b2, float eps,
                                               float bc1, float bc2) {
  const float e1 = bf2f(f2bf(b1 * bf2f(e) + (1.0f - b1) * x));
  const float q1 = bf2f(f2bf(b2 * bf2f(q) + (1.0f - b2) * x * x));
  e = f2bf(e1);
  q = f2bf(q1);
  return (e1 / bc1) / (sqrtf(q1 / bc2) + eps);
}

// ---------------------------------------------------------------- launchers
// All launchers return hipError_t from hipGetLastError after the launch.
struct GemmProb;
hipError_t launch_decompose(const MatDev* mats_dev, const StepParams& p, hipStream_t st);
hipError_t launch_decompose_inv_only(const MatDev* mats_dev, const StepParams& p, hipStream_t st);
hipError_t launch_decompose_vt(const MatDev* mats_dev, const StepParams& p, int adam_m, hipStream_t st);
int decompose_tiles(int64_t m);
int decompose_vt_tiles(int64_t m);
// Optimizer_M and Optimizer_V of a matrix whose gradient is exactly zero (no G is read):
// magnitude moments -> dM (when p.decompose), direction moments -> N; tile_dec holds the
// matrix's first workgroup, zero_grad_tiles(...) workgroups per matrix.
uint32_t zero_grad_tiles(int64_t mk, int64_t Lr);
hipError_t launch_zero_grad(const MatDev* mats_dev, const StepParams& p, hipStream_t st);
// limits of the V-writing decomposition paths (blocks per row)
constexpr int DEC_VT_MAX_K = 160;    // transposed path, 64 rows per workgroup
constexpr int DEC_ROW_MAX_K = 512;   // row-major path, 16 rows per workgroup
hipError_t launch_project(const MatDev* mats_dev, const StepParams& p, int operand_bf16, hipStream_t st);
hipError_t launch_backproject(const MatDev* mats_dev, const StepParams& p, int operand_bf16, hipStream_t st);
