// Grouped MFMA GEMM used by every dense contraction of the library.
//
//   C[M x N] = sum_k A[i][k] * B[j][k]     (i < M, j < N, k < K)
//
// One launch covers a list of independent problems (e.g. every matrix of a
// layer stack); each workgroup finds its problem by binary search over the
// problems' tile prefixes, then computes one BM x BN tile.
#pragma once
#include "common.h"

enum { KIND_BF16 = 0, KIND_F32 = 1 };
// A access modes:
//   A_G_ROW   : A[i][k] = G[i*lda + k]   * inv[i*inv_ld + k/B]   (direction V, rows)
//   A_G_TRANS : A[i][k] = G[k*lda + i]   * inv[k*inv_ld + i/B]   (direction V^T)
//   A_KC      : A[i][k] = a[i*lda + k]   (operand dtype)
// B access modes:
//   B_KC      : B[j][k] = b[j*ldb + k]   (operand dtype)
//   B_NC      : B[j][k] = b[k*ldb + j]   (fp32 kind only)
enum { A_G_ROW = 0, A_G_TRANS = 1, A_KC = 2 };
enum { B_KC = 0, B_NC = 1 };
// Epilogues:
//   EP_ADAM   : Optimizer_V on the projected tile; moments e1/e2 and output c are [M][N]
//               (e1/e2 hold bf16 values when GemmUniform::moment_bf16 is set)
//   EP_UPDATE : W[i][j] -= lr * scale * dM[i][j/B] * C[i][j] (bf16 or fp32 W in c)
//   EP_STORE  : c[i*ldc + j] = C[i][j] (fp32)
//   EP_STORE_BF16: c[i*ldc + j] = bf16(C[i][j])   (large-tile path only)
//   EP_ALIGN  : alignment sums (fp32 kind): with R[i][j] = M[i][j/B] * C[i][j], M = 1 / inv - eps
//               (inv = nullptr: M = 1) and G[i][j] = c[i*ldc + j] (read only), adds
//               sum G R, sum R^2 and sum G^2 of the tile to red[0..2] (fp64 atomics)
enum { EP_ADAM = 0, EP_UPDATE = 1, EP_STORE = 2, EP_STORE_BF16 = 3, EP_ALIGN = 4,
       EP_ADAM_B16 = 5 };   // large-tile kernel only: EP_ADAM with bf16 moments (GemmUniform::moment_bf16)

struct GemmProb {
  int64_t M, N, K;
  const void* a;
  int64_t lda;
  const float* inv;   // A_G_* only; nullptr = no scaling (V = G)
  int64_t inv_ld;
  const void* b;
  int64_t ldb;
  void* c;
  int64_t ldc;
  float* e1;          // EP_ADAM moments
  float* e2;
  const float* dM;    // EP_UPDATE magnitudes (nullptr = 1)
  int64_t dM_ld;
  float bc1, bc2;     // EP_ADAM bias corrections
  uint32_t tile_start;
  uint32_t tiles_n;
  int32_t vec;        // bit0: A may use 16-byte loads, bit1: B may
  int32_t kp;         // blocked layout (kp_index, bf16 only): bit0 A (rows M), bit1 B (rows N),
                      // bit2 the EP_ADAM output c (rows M); K a multiple of 32
  uint32_t a_bytes;   // extent of the A array (buffer loads past it return 0); 0 = unknown
  uint32_t b_bytes;   // extent of the B array
  uint32_t inv_bytes; // extent of the inv array
  uint32_t tri_b;     // fp32 kind: 1 = B[j][k] is zero for k > j (upper triangular right factor),
                      // so a tile's K loop stops after its last column; large-tile plain-store
                      // path: 2 = A[i][k] is zero for k > i, so it stops after the tile's last row
  double* red;        // EP_ALIGN accumulators (three per problem)
  // Large-tile path, split operands: the K loop runs nseg (1 .. 6) segments of K each,
  // segment 0 on (a, b), segment i > 0 on (seg_a[i-1], seg_b[i-1]), all with the layouts
  // and extents of a and b; with the operands split into bf16 parts (x = x_h + x_m + x_l)
  // this forms a product near fp32 accuracy from bf16 MFMA work. nseg 0 means 1.
  const void* seg_a[5];
  const void* seg_b[5];
  int32_t nseg;
  int32_t pad2_;
  void* c_lo;         // EP_STORE_BF16: also store the residual bf16(C - bf16(C)) here (nullable)
  void* c_parts;      // EP_STORE (large-tile path): also store C's three bf16 parts
                      // c_h = bf16(C), c_m = bf16(C - c_h), c_l = bf16(C - c_h - c_m) as three
                      // consecutive M x N arrays in the blocked layout (rows M, K = N) (nullable)
};

struct GemmUniform {
  int32_t B;            // decomposition block size (A_G_* scaling, EP_UPDATE)
  int32_t nprob;
  int32_t weight_bf16;  // EP_UPDATE
  float decomp_eps;     // EP_ALIGN
  float beta1, beta2, adam_eps;
  float lr, scale;
  int32_t moment_bf16;  // EP_ADAM: the moments are stored in bf16
  int32_t pad_;
};

template <int KIND> struct GemmTile;
template <> struct GemmTile<KIND_BF16> { static constexpr int BM = 128, BN = 128, BK = 64; };
template <> struct GemmTile<KIND_F32> { static constexpr int BM = 128, BN = 128, BK = 32; };

// GROUP_M swizzle: consecutive tiles walk GM tile-rows for one tile-column before
// moving on, so the workgroups resident on one XCD share B tiles in its L2 while
// the GM A tile-rows stay resident too.
constexpr int GM = 8;
__device__ __forceinline__ void tile_coords(uint32_t lt, uint32_t tiles_m, uint32_t tiles_n, uint32_t& tm,
                                            uint32_t& tn, uint32_t gm = GM) {
  const uint32_t per_group = gm * tiles_n;
  const uint32_t group = lt / per_group;
  const uint32_t first = group * gm;
  const uint32_t gsz = (tiles_m - first < gm) ? tiles_m - first : gm;
  const uint32_t idx = lt - group * per_group;
  tm = first + idx % gsz;
  tn = idx / gsz;
}

// Host helpers (gemm.hip).
uint32_t gemm_tiles_m(int kind, int64_t M);
uint32_t gemm_tiles_n(int kind, int64_t N);
hipError_t launch_gemm(int kind, int amode, int bmode, int ep, const GemmProb* probs_dev, int nprob,
                       uint32_t total_tiles, const GemmUniform& u, hipStream_t st);

// Large-tile bf16 path (gemm_nt.hip): A (M x K) and B (N x K) bf16, K-contiguous,
// EP_ADAM, EP_UPDATE, EP_STORE or EP_STORE_BF16; 256-row tiles.
uint32_t gemm_nt_tiles_m(int64_t M);
uint32_t gemm_nt_tiles_n(int64_t N);
bool gemm_nt_eligible(int ep, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc,
                      const void* a, const void* b, const void* c, int weight_bf16);
hipError_t launch_gemm_nt(int ep, const GemmProb* probs_dev, int nprob, uint32_t total_tiles, const GemmUniform& u,
                          hipStream_t st);
