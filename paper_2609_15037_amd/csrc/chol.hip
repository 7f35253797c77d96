// Blocked Cholesky factorisation and triangular inverse of the fp64 Gram
// matrices of a refresh batch (CholeskyQR: Z = Q R with R^T R = Z^T Z, then
// Q = Z R^{-1}). 64 x 64 blocks; every launch covers all matrices of the batch:
//   block row 0:   diag      factor C_00 = R_00^T R_00 and invert R_00 (one wave per matrix)
//   block row k:   row(k)    C_kc -= sum_{j<k} R_jk^T R_jc for c >= k (one WG per block, k >= 1);
//                            the WG of the diagonal block then factors C_kk and inverts
//                            R_kk while the launch's other WGs still run
//                  panel(k)  R_kc = R_kk^{-T} C_kc for c > k           (one WG per block)
//   then X = R^{-1} by recursive doubling over the blocks (k_trtri).
// A pivot not above 1e-13 * max(diag C) marks a numerically dependent column (a
// rank-deficient iterate): its row of R and its row and column of X = R^{-1} are set to
// zero, which is the Cholesky factor and inverse of the independent columns alone, so
// Q = Z X has orthonormal independent columns and zero dependent ones (raising such a
// pivot to a floor instead leaves chains of 1 / sqrt(floor) factors in R^{-1} that
// overflow its fp32 copy). An all-zero Gram gives R = I.
#include <algorithm>

#include "refresh.h"

namespace {

constexpr int NB = 64;
constexpr int LDB = NB + 1;

__device__ __forceinline__ int find_pref(const uint32_t* pref, int n, uint32_t t) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pref[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ int nblk(int w) { return (w + NB - 1) / NB; }
__device__ __forceinline__ int bsz(int w, int b) { return min(NB, w - b * NB); }

// load a kb_r x kb_c block (zero padded to 64 x 64) of a w x w row-major matrix into LDS
__device__ __forceinline__ void load_blk(double (*dst)[LDB], const double* M, int w, int br, int bc) {
  const int r0 = br * NB, c0 = bc * NB;
  for (int e = threadIdx.x; e < NB * NB; e += 256) {
    const int i = e >> 6, j = e & 63;
    dst[i][j] = (r0 + i < w && c0 + j < w) ? M[(int64_t)(r0 + i) * w + c0 + j] : 0.0;
  }
}

// fp64 MFMA form of the 64 x 64 block products (v_mfma_f64_16x16x4: lane l supplies
// A[l%16][l/16] and B[l/16][l%16] and receives D[4r + l/16][l%16] in register r).
// Wave w accumulates rows [16w, 16w+16) of the product, all 64 columns (four 16 x 16
// tiles): acc[jt] += op(A)[rows][t] * B[t][16 jt ..], op(A) = A^T when TA.
typedef double f64x4 __attribute__((ext_vector_type(4)));
template <bool TA>
__device__ __forceinline__ void mfma_blk(const double (*A)[LDB], const double (*Bm)[LDB], f64x4 (&acc)[4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = 16 * wave + (lane & 15);
#pragma unroll 4
  for (int ks = 0; ks < NB / 4; ++ks) {
    const int t = 4 * ks + (lane >> 4);
    const double a = TA ? A[t][i] : A[i][t];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
      acc[jt] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, Bm[t][16 * jt + (lane & 15)], acc[jt], 0, 0, 0);
  }
}
// element (row, col) of the 64 x 64 block held in acc[jt][r]
__device__ __forceinline__ int mfma_row(int r) { return 16 * (threadIdx.x >> 6) + 4 * r + ((threadIdx.x & 63) >> 4); }
__device__ __forceinline__ int mfma_col(int jt) { return 16 * jt + (threadIdx.x & 15); }

// One wave factors a 64 x 64 diagonal block held in LDS (D_ic at Dl[i * LD + c]) and
// inverts its factor; it writes R_kk, X_kk = R_kk^{-1} and its fp32 copy. Lane c keeps
// column c in registers (col[i] = D_ic); row j of R, which every column's update needs,
// goes through LDS (over the block's own rows, which are in registers by then), where
// all lanes read one address at a time (a broadcast). The LDS operations of one wave
// take effect in program order, so no step needs a workgroup barrier. A ragged block is
// padded with the identity, which factors and inverts to itself; take = 0 (an all-zero
// Gram) gives R_kk = X_kk = I.
//   factor, right-looking, column j = 0 .. kb-1:
//     R_jj = sqrt(D_jj) (0 for a dependent column), R_jc = D_jc / R_jj (c > j),
//     D_ac -= R_ja R_jc for a > j (lane c; for a > c this is the lower triangle,
//     which follows the symmetric Schur complement and is not read);
//   invert from the last row up, lane c: a_ic = sum_{t > i} R_it X_tc accumulated as
//     the rows of X below i are finished (X_tc = 0 for t > c),
//     X_cc = 1 / R_cc, X_ic = -a_ic / R_ii (i < c); a zero R_ii gives a zero row of X.
// Each step's updates are kept inside the step (a wave-uniform branch per step ends its
// basic block): left free, the compiler defers them into long chains that spill.
template <int LD>
__device__ __forceinline__ void diag_factor(double* Dl, int kb, bool take, double floor_piv, const RefDev& d,
                                            int r0) {
  const int w = d.w;
  const int lane = threadIdx.x & 63;
  const bool live = lane < kb;
  double col[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const double c = Dl[i * LD + lane];
    col[i] = (take && live && i < kb) ? c : (i == lane ? 1.0 : 0.0);
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (j >= kb) continue;
    const double v = __shfl(col[j], j, 64);
    const double rjj = v > floor_piv ? sqrt(v) : 0.0;   // 0: dependent column
    const double q = col[j] / (rjj > 0.0 ? rjj : 1.0);
    const double rjc = lane == j ? rjj : (lane > j && rjj > 0.0 ? q : 0.0);
    col[j] = rjc;
    Dl[j * LD + lane] = rjc;
#pragma unroll
    for (int a = j + 1; a < NB; ++a) col[a] -= Dl[j * LD + a] * rjc;
  }
  if (live) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (i < kb) d.C[(int64_t)(r0 + i) * w + r0 + lane] = col[i];
  }
  double* acc = col;   // a_ic, accumulated from the bottom row up
#pragma unroll
  for (int i = 0; i < NB; ++i) acc[i] = 0.0;
#pragma unroll
  for (int t = NB - 1; t >= 0; --t) {
    if (t >= kb) continue;
    const double rtt = Dl[t * LD + t];
    const double num = lane == t ? 1.0 : -acc[t];
    const double q = num / (rtt > 0.0 ? rtt : 1.0);
    const double x = (lane >= t && rtt > 0.0) ? q : 0.0;
    acc[t] = x;
#pragma unroll
    for (int i = 0; i < t; ++i) acc[i] += Dl[i * LD + t] * x;
  }
  if (live) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (i < kb) {
        const int64_t g = (int64_t)(r0 + i) * w + r0 + lane;
        d.X[g] = acc[i];
        d.Rinv[g] = (float)acc[i];
      }
  }
}

// Block 0 (no update before it): one wave per matrix; also records the pivot floor's
// reference, the largest diagonal entry of the untouched Gram.
__global__ __launch_bounds__(64) void k_chol_diag(const RefDev* __restrict__ ds) {
  __shared__ double Dl[NB][NB];
  const RefDev& d = ds[blockIdx.x];
  const int w = d.w;
  const int lane = threadIdx.x;
  double mx = 0.0;
  for (int i = lane; i < w; i += 64) mx = fmax(mx, d.C[(int64_t)i * w + i]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) d.cmax[0] = mx;
  const int kb = bsz(w, 0);
  const int lc = min(lane, kb - 1);   // clamped: every lane loads in bounds
  for (int i = 0; i < NB; ++i) Dl[i][lane] = d.C[(int64_t)min(i, kb - 1) * w + lc];
  diag_factor<NB>(&Dl[0][0], kb, mx > 0.0, mx * 1e-13, d, 0);
}

__global__ __launch_bounds__(256, 4) void k_chol_panel(const RefDev* __restrict__ ds, const uint32_t* __restrict__ pref,
                                                       int n, int k) {
  const uint32_t t = blockIdx.x;
  const int mi = find_pref(pref, n, t);
  const RefDev& d = ds[mi];
  const int w = d.w;
  const int j = k + 1 + (int)(t - pref[mi]);
  // R_kj = X_kk^T C_kj: C_kj in LDS, each wave's 16 columns of X_kk straight into its MFMA
  // operand registers (A[i][t] = X_kk[t][16 w + i])
  __shared__ double Cb[NB][LDB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double av[NB / 4];
  {
    const int col = k * NB + 16 * wave + (lane & 15);
#pragma unroll
    for (int ks = 0; ks < NB / 4; ++ks) {
      const int row = k * NB + 4 * ks + (lane >> 4);
      av[ks] = (row < w && col < w) ? d.X[(int64_t)row * w + col] : 0.0;
    }
  }
  load_blk(Cb, d.C, w, k, j);
  __syncthreads();
  f64x4 acc[4];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) acc[jt] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int ks = 0; ks < NB / 4; ++ks) {
    const int tr = 4 * ks + (lane >> 4);
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
      acc[jt] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[ks], Cb[tr][16 * jt + (lane & 15)], acc[jt], 0, 0, 0);
  }
  const bool zero = !(d.cmax[0] > 0.0);
#pragma unroll
  for (int jt = 0; jt < 4; ++jt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = k * NB + mfma_row(r), col = j * NB + mfma_col(jt);
      if (row < w && col < w) d.C[(int64_t)row * w + col] = zero ? 0.0 : acc[jt][r];
    }
}

// Left-looking update of block row k before its factorisation (k >= 1):
//   C_kc -= sum_{j < k} R_jk^T R_jc     for every block column c >= k
// One workgroup per (matrix, c); its K loop runs over the factored block rows j < k,
// with the next pair of blocks loaded into registers while the current one is
// multiplied (R_jc from LDS, R_jk's 16 columns of each wave straight into its MFMA
// operand registers: A[i][t] = R_jk[t][16 w + i]). Every block of C is read and written
// once here, where a right-looking update would rewrite the trailing matrix after every
// panel; the factored rows R_j. are shared by all workgroups of a matrix (L2 hits).
__global__ __launch_bounds__(256, 2) void k_chol_row(const RefDev* __restrict__ ds, const uint32_t* __restrict__ pref,
                                                     int n, int k) {
  // workgroups 0 .. n-1: the diagonal block of matrix t (updated, then factored here);
  // the rest: the blocks c > k, matrices by prefix
  const uint32_t t = blockIdx.x;
  const bool diag = t < (uint32_t)n;
  const int mi = diag ? (int)t : find_pref(pref, n, t - n);
  const RefDev& d = ds[mi];
  const int w = d.w;
  if (diag && k >= nblk(w)) return;
  const int c = diag ? k : k + 1 + (int)(t - n - pref[mi]);
  __shared__ double Rb[NB][LDB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double av[NB / 4], an[NB / 4], pb[16];
  auto fetch = [&](int j, double (&a)[NB / 4]) {
    const int col = k * NB + 16 * wave + (lane & 15);
#pragma unroll
    for (int ks = 0; ks < NB / 4; ++ks) {
      const int row = j * NB + 4 * ks + (lane >> 4);
      a[ks] = (row < w && col < w) ? d.C[(int64_t)row * w + col] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = threadIdx.x + 256 * q, i = e >> 6, jj = e & 63;
      const int row = j * NB + i, col2 = c * NB + jj;
      pb[q] = (row < w && col2 < w) ? d.C[(int64_t)row * w + col2] : 0.0;
    }
  };
  auto publish = [&]() {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = threadIdx.x + 256 * q;
      Rb[e >> 6][e & 63] = pb[q];
    }
  };
  f64x4 acc[4];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) acc[jt] = f64x4{0.0, 0.0, 0.0, 0.0};
  fetch(0, av);
  publish();
  __syncthreads();
  for (int j = 0; j < k; ++j) {
    if (j + 1 < k) fetch(j + 1, an);
#pragma unroll
    for (int ks = 0; ks < NB / 4; ++ks) {
      const int tr = 4 * ks + (lane >> 4);
#pragma unroll
      for (int jt = 0; jt < 4; ++jt)
        acc[jt] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[ks], Rb[tr][16 * jt + (lane & 15)], acc[jt], 0, 0, 0);
    }
    __syncthreads();
    if (j + 1 < k) {
      publish();
#pragma unroll
      for (int ks = 0; ks < NB / 4; ++ks) av[ks] = an[ks];
      __syncthreads();
    }
  }
  if (!diag) {
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = k * NB + mfma_row(r), col = c * NB + mfma_col(jt);
        if (row < w && col < w) d.C[(int64_t)row * w + col] -= acc[jt][r];
      }
    return;
  }
  // diagonal block: the updated C_kk goes to LDS (Rb is free: the K loop ended with a
  // barrier) and wave 0 factors it while the other workgroups of the launch run on
  const double cmax = d.cmax[0];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = mfma_row(r), j = mfma_col(jt), row = k * NB + i, col = k * NB + j;
      Rb[i][j] = (row < w && col < w) ? d.C[(int64_t)row * w + col] - acc[jt][r] : 0.0;
    }
  __syncthreads();
  if (wave == 0) diag_factor<LDB>(&Rb[0][0], bsz(w, k), cmax > 0.0, cmax * 1e-13, d, k * NB);
}

// Triangular inverse X = R^{-1} by recursive doubling over the 64 x 64 blocks. Level l
// (l = 1, 2, ...) pairs the already inverted halves A = blocks [p 2^l, p 2^l + 2^(l-1))
// and B = [p 2^l + 2^(l-1), min((p + 1) 2^l, nb)) of every super-block p and forms
//   X_AB = -X_AA R_AB X_BB
// in two launches: phase 0 T = R_AB X_BB, phase 1 X_AB = -X_AA T. T waits in the
// (otherwise unused) strictly lower part of X, its block (i, j) transposed at block
// (j, i), which holds exactly the rows and columns of T's block even at a partial edge block. The
// diagonal blocks X_kk come from k_chol_diag. A dependency chain is at most 2^(l-1)
// block products long, against up to nb - 1 for a column-by-column inverse. One
// workgroup per 64 x 64 output block; its K loop loads the next block pair into
// registers while the current one is multiplied from LDS.
__global__ __launch_bounds__(256, 2) void k_trtri(const RefDev* __restrict__ ds, const uint32_t* __restrict__ pref,
                                               int n, int l, int phase) {
  const uint32_t t = blockIdx.x;
  const int mi = find_pref(pref, n, t);
  const RefDev& d = ds[mi];
  const int w = d.w, nb = nblk(w);
  const int h = 1 << (l - 1);
  int rem = (int)(t - pref[mi]), A0 = 0, nB = 1;
  for (int p = 0; p * 2 * h + h < nb; ++p) {   // pairs with a non-empty B half
    const int a0 = p * 2 * h, cnt = h * (min(a0 + 2 * h, nb) - a0 - h);
    if (rem < cnt) { A0 = a0; nB = min(a0 + 2 * h, nb) - a0 - h; break; }
    rem -= cnt;
  }
  const int B0 = A0 + h;
  const int I = A0 + rem / nB, J = B0 + rem % nB;
  // phase 0: sum over tb = B0 .. J of R_{I,tb} X_{tb,J}   (R in the upper part of C)
  // phase 1: sum over tb = I .. B0-1 of X_{I,tb} T_{tb,J} (T_{tb,J}^T parked at X block (J, tb))
  const int tlo = phase == 0 ? B0 : I, thi = phase == 0 ? J : B0 - 1;
  __shared__ double Ab[NB][LDB];
  __shared__ double Bb[NB][LDB];
  f64x4 acc[4];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) acc[jt] = f64x4{0.0, 0.0, 0.0, 0.0};
  double pa[16], pb[16];
  auto fetch = [&](int tb) {
    const double* Am = phase == 0 ? d.C : d.X;
    const int ar = I, ac = tb;                       // A block (I, tb)
    const int br = phase == 0 ? tb : J, bc = phase == 0 ? J : tb;   // B block (phase 1: transposed)
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = threadIdx.x + 256 * q, i = e >> 6, j = e & 63;
      const int ra = ar * NB + i, ca = ac * NB + j, rb = br * NB + i, cb = bc * NB + j;
      pa[q] = (ra < w && ca < w) ? Am[(int64_t)ra * w + ca] : 0.0;
      pb[q] = (rb < w && cb < w) ? d.X[(int64_t)rb * w + cb] : 0.0;
    }
  };
  auto publish = [&]() {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e = threadIdx.x + 256 * q, i = e >> 6, j = e & 63;
      Ab[i][j] = pa[q];
      if (phase == 0) Bb[i][j] = pb[q];
      else Bb[j][i] = pb[q];   // X block (J, tb) holds T_{tb,J}^T
    }
  };
  fetch(tlo);
  publish();
  __syncthreads();
  for (int tb = tlo; tb <= thi; ++tb) {
    if (tb < thi) fetch(tb + 1);
    mfma_blk<false>(Ab, Bb, acc);
    __syncthreads();
    if (tb < thi) {
      publish();
      __syncthreads();
    }
  }
  if (phase == 0) {   // park T_{I,J}^T at block (J, I), transposed through LDS
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) Ab[mfma_col(jt)][mfma_row(r)] = acc[jt][r];
    __syncthreads();
    for (int e = threadIdx.x; e < NB * NB; e += 256) {
      const int i = e >> 6, j = e & 63, row = J * NB + i, col = I * NB + j;
      if (row < w && col < w) d.X[(int64_t)row * w + col] = Ab[i][j];
    }
  } else {
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = I * NB + mfma_row(r), col = J * NB + mfma_col(jt);
        if (row < w && col < w) {
          const int64_t g = (int64_t)row * w + col;
          d.X[g] = -acc[jt][r];
          d.Rinv[g] = (float)(-acc[jt][r]);
        }
      }
  }
}

}  // namespace

int chol_blocks(int32_t w) { return (w + NB - 1) / NB; }

hipError_t launch_chol_diag(const RefDev* d, int n, hipStream_t st) {
  if (!n) return hipSuccess;
  hipLaunchKernelGGL(k_chol_diag, dim3(n), dim3(64), 0, st, d);
  return hipGetLastError();
}
hipError_t launch_chol_panel(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int k, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_chol_panel, dim3(total), dim3(256), 0, st, d, pref, n, k);
  return hipGetLastError();
}
hipError_t launch_chol_row(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int k, hipStream_t st) {
  if (!n || k < 1 || total < (uint32_t)n) return hipSuccess;
  hipLaunchKernelGGL(k_chol_row, dim3(total), dim3(256), 0, st, d, pref, n, k);
  return hipGetLastError();
}
int trtri_levels(int32_t nbmax) { int l = 0; while ((1 << l) < nbmax) ++l; return l; }
uint32_t trtri_tiles(int32_t w, int l) {
  const int nb = (w + NB - 1) / NB, h = 1 << (l - 1);
  uint32_t c = 0;
  for (int a0 = 0; a0 + h < nb; a0 += 2 * h) c += (uint32_t)(h * (std::min(a0 + 2 * h, nb) - a0 - h));
  return c;
}
hipError_t launch_trtri(const RefDev* d, const uint32_t* pref, int n, uint32_t total, int l, int phase, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_trtri, dim3(total), dim3(256), 0, st, d, pref, n, l, phase);
  return hipGetLastError();
}
