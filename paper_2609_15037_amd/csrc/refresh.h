// Projector refresh (Algorithm 1: P <- TruncatedSVD(V, r)) kernels.
#pragma once
#include "common.h"

// Per-matrix refresh descriptor (device array, one entry per refreshed matrix).
struct RefDev {
  int64_t s;          // projected dimension (rows of P)
  int64_t L;          // other dimension
  int32_t w;          // subspace width r + p (<= s)
  int32_t wpad;       // w rounded up to a multiple of JB (Jacobi block)
  int32_t r;
  int32_t operand_bf16;
  uint64_t seed;      // Philox key for the Gaussian start block
  float* Z;           // s x w fp32 (iterate, row-major)
  float* Z0;          // s x w fp32: where the Gaussian start block goes (Z, or Z2 when it is orthonormalised first)
  double* C;          // w x w fp64 Gram, factorised in place into R (upper)
  double* X;          // w x w fp64 R^{-1} (upper)
  double* cmax;       // max diagonal of the Gram (pivot floor), one value
  float* Rinv;        // w x w fp32 inverse Cholesky factor
  double* Zc;         // wpad x w fp64, column-major copy of the Cholesky factor R of the final
                      // iterate (Z2 = Q R), rotated in place by the Jacobi sweeps
  int64_t jl;         // column length of Zc (= w)
  const float* Q;     // s x w fp32 orthonormal factor Q of the final iterate
  float* Pw;          // s x r fp32: Q (R J)_top before signs
  float* Bt;          // r x w fp32: (R J)_top^T, columns normalised
  float* P32;         // s x r fp32 master projector
  void* Pop;          // s x r operand dtype
  void* Ptop;         // r x s operand dtype
  int32_t kp;         // 1: Pop and Ptop in the blocked operand layout (kp_index; bf16)
  int32_t pad_kp;
  uint32_t* off;      // per-sweep max off-diagonal (float bits), >= n_sweeps entries
  int32_t* order;     // wpad scratch: column order by norm
  double* norms;      // wpad scratch
  uint32_t tile_gauss, tile_jac, tile_cm, tile_norm;   // per-launch workgroup prefixes
  int32_t has_prev;   // 1: a projector exists (an all-zero V keeps it)
  int32_t max_sweeps; // Jacobi sweeps launched
  int32_t* info;      // 4 ints of the state, written by the refresh: [0] Jacobi sweeps run,
                      // [1] 1 = converged, [2] numerical rank (kept Ritz directions, <= r),
                      // [3] largest pair cosine of the last sweep measured (float bits)
  double* cw;         // basis completion workspace: s x 64 block, r x 64 coefficients, s row norms
  int32_t* sidx;      // basis completion: the r canonical indices, by increasing row norm
  // Jacobi pair records: for the pair visited in round rr at position p (index
  // rr * nb / 2 + p, nb = wpad / JB blocks) the sweep + 1 of its last visit that measured
  // it converged (0: rotated), and that measurement; per block, 1 + the global round
  // index (sweep * (nb - 1) + round) of its last rotation (0: none yet)
  uint32_t* jconv;
  float* jmx;
  uint32_t* jmod;
};

// Ritz directions whose value is not above this fraction of the largest one are
// numerically null: an fp32 subspace iteration cannot resolve them (its GEMMs carry
// relative errors of order 1e-6), so their columns are completed to an orthonormal basis.
constexpr double RITZ_NULL_REL = 1e-5;

constexpr int JB = 32;   // Jacobi column block; a pair holds 2*JB columns

// Gram problem: C = A^T A for A (rows x w, row stride lda), fp64 accumulation.
struct GramProb {
  const float* A;
  int64_t rows, lda;
  double* C;
  int32_t w, tiles;     // tiles per dimension (64-wide)
  uint32_t tile_start, pad_;
};

// Transpose (and convert to bf16): out[c][r] = bf16(in[r][c]) for r < rows, c < cols.
struct TransProb {
  const void* in;       // rows x cols, row stride ldi, fp32 (in_f32) or bf16
  void* out;            // cols x rows bf16, row stride ldo
  int64_t rows, cols, ldi, ldo;
  int32_t in_f32, tiles_c;   // tiles_c: 64-wide tiles along cols
  uint32_t tile_start;
  int32_t in_kp;             // 1: bf16 input in the blocked layout (kp_index(r, c, rows))
  int32_t out_kp;            // 1: output in the blocked layout (kp_index(c, r, cols))
  int32_t pad_;
  void* out_lo;              // fp32 input: also x_m = bf16(x - x_h), x_h = bf16(x), same layout (nullable)
  void* out_lo2;             // ... and x_l = bf16(x - x_h - x_m) (nullable; needs out_lo)
};
uint32_t transpose_tiles(int64_t rows, int64_t cols);
hipError_t launch_transpose(const TransProb* t, int n, uint32_t total, hipStream_t st);

// The bf16 parts of the direction tensor beyond its bf16 value v_h = bf16(v), for the split
// products of the last subspace iterations: v_m = bf16(v - v_h) and v_l = bf16(v - v_h - v_m)
// (v = v_h + v_m + v_l to about 2^-24 relative), with v = G * inv in fp32 as the
// decomposition and the fp32 products form V (inv = nullptr: v = G); each stored in the
// blocked layout both as the m x n operand (K = n) and as the n x m one (K = m).
struct SplitProb {
  const float* g;       // m x n, row stride n
  const float* inv;     // m x k, row stride inv_ld (nullable)
  void* out_n[2];       // v_m, v_l as m x n
  void* out_t[2];       // v_m, v_l as n x m
  int64_t m, n;
  int32_t inv_ld, B;
  int32_t tiles_c;      // 64-wide tiles along n
  uint32_t tile_start;
};
uint32_t split_lo_tiles(int64_t m, int64_t n);
hipError_t launch_split_lo(const SplitProb* p, int n, uint32_t total, hipStream_t st);

hipError_t launch_gauss(const RefDev* d, int n, uint32_t total, hipStream_t st);
hipError_t launch_gram(const GramProb* g, int n, uint32_t total, hipStream_t st);
int chol_blocks(int32_t w);
hipError_t launch_chol_diag(const RefDev* d, int n, hipStream_t st);   // block 0
hipError_t launch_chol_panel(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int k, hipStream_t st);
hipError_t launch_chol_row(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int k,
                           hipStream_t st);   // k >= 1, factors block k too
int trtri_levels(int32_t nbmax);
uint32_t trtri_tiles(int32_t w, int l);
hipError_t launch_trtri(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int l, int phase, hipStream_t st);
hipError_t launch_jacobi_round(const RefDev* d, int n, uint32_t total, int round, int sweep, hipStream_t st);
hipError_t launch_r_colmajor(const RefDev* d, int n, uint32_t total, hipStream_t st);
uint32_t r_colmajor_tiles(int32_t w, int32_t wpad);
uint32_t norm_tiles(int32_t wpad);
hipError_t launch_finalize_order(const RefDev* d, int n, uint32_t norm_total, hipStream_t st);
hipError_t launch_finalize_out(const RefDev* d, int n, int32_t rmax, hipStream_t st);
hipError_t launch_complete_basis(const RefDev* d, int n, hipStream_t st);
hipError_t launch_convert_projector(const float* P32, void* Pop, void* Ptop, int64_t s, int64_t r,
                                    int operand_bf16, int kp, hipStream_t st);
// P = the first r canonical basis vectors (the projector of an all-zero V with none before)
hipError_t launch_canonical_projector(float* P32, void* Pop, void* Ptop, int64_t s, int64_t r, int operand_bf16,
                                      int kp, hipStream_t st);
uint32_t gauss_tiles(int64_t s, int32_t w);
uint32_t gram_tiles(int32_t w);
uint32_t jacobi_tiles(int32_t wpad);
