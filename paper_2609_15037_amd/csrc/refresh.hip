// Projector refresh kernels: P <- TruncatedSVD(V, r) (Algorithm 1).
//
// Method (randomised subspace iteration with Rayleigh-Ritz, all on the device):
//   Z = seeded Gaussian s x w block (w = r + p; for w <= s / 2 its condition number
//       stays below 6 and it is used as it is, else Z = orth(Gaussian))
//   repeat q times:  Y = X Z;  Zn = X^T Y;  Z = orth(Zn)      (last time: Y = orth(Y) first)
//   Rayleigh-Ritz:   one-sided Jacobi on Zn = X^T Y (fp64) orthogonalises its columns
//                    into (right singular vectors of X) x (singular values); the r
//                    columns of largest norm, normalised, are P.
// X is V (RIGHT, s = n) or V^T (LEFT, s = m); the big GEMMs live in gemm.hip.
// orth() is CholeskyQR with an fp64 Gram and an fp64 Cholesky factor.
//
// Kernels here: Philox-4x32-10 Gaussian start (Salmon et al., SC'11, with the
// Box-Muller transform), fp64 Gram, the Jacobi sweep rounds and the final
// ordering / sign fixing; the blocked Cholesky and inverse live in chol.hip.
#include "refresh.h"

namespace {

// ------------------------------------------------------------------ Philox 4x32-10
__device__ __forceinline__ void philox_round(uint32_t c[4], uint32_t k[2]) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t lo0 = M0 * c[0], hi0 = __umulhi(M0, c[0]);
  const uint32_t lo1 = M1 * c[2], hi1 = __umulhi(M1, c[2]);
  const uint32_t n0 = hi1 ^ c[1] ^ k[0], n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
  k[0] += 0x9E3779B9u; k[1] += 0xBB67AE85u;
}

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint64_t key) {
  uint32_t k[2] = {(uint32_t)key, (uint32_t)(key >> 32)};
#pragma unroll
  for (int i = 0; i < 10; ++i) philox_round(c, k);
}

__device__ __forceinline__ float u01(uint32_t x) {   // (0, 1]
  return ((float)(x >> 8) + 1.0f) * (1.0f / 16777216.0f);
}

constexpr int GAUSS_PER_WG = 1024;   // elements (4 per thread)

__global__ __launch_bounds__(256) void k_gauss(const RefDev* __restrict__ ds, int n) {
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ds[mid].tile_gauss <= t) lo = mid; else hi = mid - 1; }
  const RefDev& d = ds[lo];
  const int64_t total = d.s * d.w;
  const int64_t e0 = ((int64_t)(t - d.tile_gauss) * GAUSS_PER_WG) + threadIdx.x * 4;
  if (t == d.tile_gauss && threadIdx.x < 64) d.off[threadIdx.x] = 0u;   // per-sweep Jacobi measures
  if (e0 >= total) return;
  uint32_t c[4] = {(uint32_t)(e0 >> 2), (uint32_t)(e0 >> 34), 0x4D6F4152u, 0x52656672u};
  philox4x32_10(c, d.seed);
  const float r0 = sqrtf(-2.0f * logf(u01(c[0]))), r1 = sqrtf(-2.0f * logf(u01(c[2])));
  const float a0 = 6.283185307179586f * u01(c[1]), a1 = 6.283185307179586f * u01(c[3]);
  float v[4] = {r0 * cosf(a0), r0 * sinf(a0), r1 * cosf(a1), r1 * sinf(a1)};
  for (int q = 0; q < 4 && e0 + q < total; ++q) d.Z0[e0 + q] = v[q];
  // the same launch clears what later kernels expect at zero, saving separate memsets:
  // the measures above and the blocks of the fp32 R^{-1} below its diagonal, which the
  // factorisation never writes (w^2 <= s w)
  const int64_t ww = (int64_t)d.w * d.w;
  for (int q = 0; q < 4; ++q)
    if (e0 + q < ww) d.Rinv[e0 + q] = 0.f;
}

// ------------------------------------------------------------------ fp64 Gram C = A^T A
// One workgroup per 64 x 64 tile of the upper triangle. fp32 rows are staged in
// LDS as fp64 (32 rows per chunk, the next two chunks in flight in registers) and
// multiplied on v_mfma_f64_16x16x4; wave w owns tile rows [16w, 16w+16).
typedef double f64x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256, 4) void k_gram(const GramProb* __restrict__ gs, int n) {
  // One LDS buffer per operand (34 KB in all, four workgroups per CU); row stride 66
  // doubles keeps every 4-column group 16-byte aligned for b128 stores.
  __shared__ __attribute__((aligned(16))) double Ai[32][64 + 2];
  __shared__ __attribute__((aligned(16))) double Aj[32][64 + 2];
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (gs[mid].tile_start <= t) lo = mid; else hi = mid - 1; }
  const GramProb& g = gs[lo];
  int rem = (int)(t - g.tile_start), ti = 0;
  while (rem >= g.tiles - ti) { rem -= g.tiles - ti; ++ti; }
  const int tj = ti + rem;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (int)((g.rows + 31) / 32);
  // 16-byte loads of four columns when rows and the width allow them
  const bool vec = (g.lda & 3) == 0 && (g.w & 3) == 0 && (((uintptr_t)g.A) & 15) == 0;
  // Two chunks of global loads stay in flight in a register ring while the current
  // chunk is multiplied from LDS: chunk c + 1 in slot (c + 1) & 1, chunk c + 2 in slot c & 1.
  // Thread e of a chunk (two per thread) covers row e / 16, columns 4 (e % 16) .. + 3.
  float4 pi[2][2], pj[2][2];
  auto load4 = [&](int64_t row, int col) -> float4 {
    if (row >= g.rows || col >= g.w) return make_float4(0.f, 0.f, 0.f, 0.f);
    const float* src = g.A + row * g.lda + col;
    if (vec) return *reinterpret_cast<const float4*>(src);
    return make_float4(src[0], col + 1 < g.w ? src[1] : 0.f, col + 2 < g.w ? src[2] : 0.f, col + 3 < g.w ? src[3] : 0.f);
  };
  auto load_chunk = [&](int c, float4 (&xi)[2], float4 (&xj)[2]) {
    const int64_t l0 = (int64_t)c * 32;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = tid + 256 * q, l = e >> 4, c4 = (e & 15) * 4;
      xi[q] = load4(l0 + l, ti * 64 + c4);
      xj[q] = load4(l0 + l, tj * 64 + c4);
    }
  };
  auto store_chunk = [&](const float4 (&xi)[2], const float4 (&xj)[2]) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = tid + 256 * q, l = e >> 4, c4 = (e & 15) * 4;
      double2* di = reinterpret_cast<double2*>(&Ai[l][c4]);
      double2* dj = reinterpret_cast<double2*>(&Aj[l][c4]);
      di[0] = make_double2(xi[q].x, xi[q].y); di[1] = make_double2(xi[q].z, xi[q].w);
      dj[0] = make_double2(xj[q].x, xj[q].y); dj[1] = make_double2(xj[q].z, xj[q].w);
    }
  };
  f64x4 acc[4];
#pragma unroll
  for (int jt = 0; jt < 4; ++jt) acc[jt] = f64x4{0.0, 0.0, 0.0, 0.0};
  auto mult = [&]() {
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const int kr = 4 * ks + (lane >> 4);
      const double a = Ai[kr][16 * wave + (lane & 15)];
#pragma unroll
      for (int jt = 0; jt < 4; ++jt)
        acc[jt] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, Aj[kr][16 * jt + (lane & 15)], acc[jt], 0, 0, 0);
    }
  };
  load_chunk(0, pi[0], pj[0]);
  store_chunk(pi[0], pj[0]);
  if (1 < nch) load_chunk(1, pi[1], pj[1]);
  if (2 < nch) load_chunk(2, pi[0], pj[0]);
  __syncthreads();
  for (int c = 0; c < nch; c += 2) {   // unrolled by two so that the ring slots stay static
    mult();                                                // chunk c
    __syncthreads();
    if (c + 1 < nch) store_chunk(pi[1], pj[1]);
    if (c + 3 < nch) load_chunk(c + 3, pi[1], pj[1]);
    __syncthreads();
    if (c + 1 >= nch) break;
    mult();                                                // chunk c + 1
    __syncthreads();
    if (c + 2 < nch) store_chunk(pi[0], pj[0]);
    if (c + 4 < nch) load_chunk(c + 4, pi[0], pj[0]);
    __syncthreads();
  }
#pragma unroll
  for (int jt = 0; jt < 4; ++jt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = ti * 64 + 16 * wave + 4 * r + (lane >> 4), j = tj * 64 + 16 * jt + (lane & 15);
      if (i < g.w && j < g.w && (ti != tj || i <= j)) {   // diagonal tiles: one writer per pair
        g.C[(int64_t)i * g.w + j] = acc[jt][r];
        g.C[(int64_t)j * g.w + i] = acc[jt][r];
      }
    }
}

// ------------------------------------------------------------------ Zn (s x w fp32) -> Zc (wpad x s fp64)
// ------------------------------------------------------------------ one Jacobi round
// Workgroup = (matrix, block pair). Blocks of JB columns are paired by the
// circle method: over nb-1 rounds every pair of the nb blocks meets once.
__device__ __forceinline__ int circle(int pos, int round, int nb) {
  return pos == 0 ? 0 : 1 + ((pos - 1 + round) % (nb - 1));
}

constexpr int PW = 2 * JB;   // 64 columns per pair
// Convergence: a pair whose largest column cosine is below JAC_TOL is not rotated, and a
// matrix stops once a whole sweep measured below it. Cosines c between columns with
// relative singular-value gap g perturb the singular subspaces by about c / (2 g); at
// 1e-8 that stays below 5e-5 rad for gaps down to 1e-4 (well inside what the subspace
// iteration itself resolves) and below fp32 rounding for gaps above 0.1. A tolerance
// of 1e-10 cost about 5 % more sweep time for digits the fp32 projector does not keep.
#ifndef MOARA_JAC_TOL
#define MOARA_JAC_TOL 1e-7
#endif
constexpr double JAC_TOL = MOARA_JAC_TOL;
// Inner Jacobi sweeps per pair visit. The pair's Gram need not be diagonalised
// exactly on every visit: with one inner sweep the outer iteration needs about one
// more sweep to reach the same off-diagonal level, but every visit is much cheaper
// and the visits of one round take about the same time (measured fastest of 1-3).
#ifndef JAC_INNER_SWEEPS
#define JAC_INNER_SWEEPS 1
#endif

// LDS: two 64 x 65 fp64 regions. Region A holds the pair's Gram G during the inner
// solve; during the column passes it holds the current 32-row chunk of the 64 columns
// (rows 0-31) and, in the rotation pass, the rotated chunk (rows 32-63). Region B holds
// the rotation J (and the convergence reduction's scratch before J is built). 67 KB,
// so two workgroups share a CU and one's LDS-bound inner solve overlaps the other's
// MFMA / memory phases.
constexpr int JR = 32;   // rows per column chunk
#ifndef JAC_RING
#define JAC_RING 2
#endif
#ifndef JAC_WAVES
#define JAC_WAVES 8
#endif
constexpr int JNT = 64 * JAC_WAVES;    // threads per workgroup
constexpr int JEPT = JR * PW / JNT;    // chunk elements per thread
static_assert(2 * JR == PW && JEPT * JNT == JR * PW && (JAC_WAVES == 4 || JAC_WAVES == 8), "chunk mapping");
// Gram tiles (it, jt), it <= jt, of each wave, packed as it * 4 + jt per byte (0xFF = none).
// Waves w and w + 4 share a SIMD; the per-SIMD counts are 3, 3, 2, 2 in both layouts.
__device__ __forceinline__ uint32_t jac_gram_tiles(int wave) {
  if (JAC_WAVES == 4)
    return wave == 0 ? 0xFF020100u : wave == 1 ? 0xFF060503u : wave == 2 ? 0xFFFF0A07u : 0xFFFF0F0Bu;
  constexpr uint32_t tab[8] = {0xFFFF0100u, 0xFFFF0605u, 0xFFFFFF02u, 0xFFFFFF03u,
                               0xFFFFFF07u, 0xFFFFFF0Au, 0xFFFFFF0Bu, 0xFFFFFF0Fu};
  return tab[wave];
}
__global__ __launch_bounds__(JNT, 2) void k_jacobi_round(const RefDev* __restrict__ ds, int n, int round, int sweep) {
  __shared__ double Am[PW][PW + 1];
  __shared__ double Jm[PW][PW + 1];
  __shared__ double CS[PW / 2][2];   // the round's rotations (cosine, sine) of the inner solve
  double (*Gm)[PW + 1] = Am;         // inner solve
  double (*T)[PW + 1] = Am;          // column chunk (rows 0 .. JR-1)
  double (*O)[PW + 1] = Am + JR;     // rotated chunk (rows JR .. 2 JR-1)
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ds[mid].tile_jac <= t) lo = mid; else hi = mid - 1; }
  const RefDev& d = ds[lo];
  const int nb = d.wpad / JB;
  const int pair = (int)(t - d.tile_jac);
  if (round >= nb - 1) return;   // this matrix has fewer blocks than the widest one
  if (sweep > 0 && __uint_as_float(d.off[sweep - 1]) < (float)JAC_TOL) return;   // converged
  const int ba = circle(pair, round, nb), bb = circle(nb - 1 - pair, round, nb);
  const int tid = threadIdx.x;
  // The circle schedule brings this pair back at the same round of every sweep. If its
  // last visit measured it converged and neither block was rotated since, its columns,
  // hence its Gram and measure, are what they were: record that measure again and skip
  // the visit (the sweeps' results are exactly those of visiting it).
  const uint32_t pidx = (uint32_t)round * (uint32_t)(nb / 2) + (uint32_t)pair;
  const uint32_t gnow = (uint32_t)sweep * (uint32_t)(nb - 1) + (uint32_t)round;
  if (sweep == 0) {
    if (round == 0 && tid == 0) { d.jmod[ba] = 0; d.jmod[bb] = 0; }   // round 0 covers every block
  } else {
    const uint32_t gprev = gnow - (uint32_t)(nb - 1);
    if (d.jconv[pidx] == (uint32_t)sweep && d.jmod[ba] <= gprev && d.jmod[bb] <= gprev) {
      if (tid == 0) {
        atomicMax(&d.off[sweep], __float_as_uint(d.jmx[pidx]));
        d.jconv[pidx] = (uint32_t)sweep + 1;
      }
      return;
    }
  }
  const int64_t s = d.jl;   // column length
  auto colp = [&](int x) -> double* { return d.Zc + (int64_t)((x < JB) ? ba * JB + x : bb * JB + (x - JB)) * s; };
  const int lane = tid & 63, wave = tid >> 6;
  const int nch = (int)((s + JR - 1) / JR);

  // Column chunks: JR rows x 64 columns; thread e = tid + JNT q covers column e / JR,
  // row e % JR (a wave reads two whole 256-byte column segments per instruction).
  // While chunk c is used from LDS, chunks c + 1 .. c + JAC_RING are in flight in a
  // register ring (chunk x in slot x % JAC_RING).
  double pre[JAC_RING][JEPT];
  auto load_chunk = [&](int c, double (&x8)[JEPT]) {
    const int64_t r0 = (int64_t)c * JR;
#pragma unroll
    for (int q = 0; q < JEPT; ++q) {
      const int e = tid + JNT * q, x = e / JR, l = e % JR;
      x8[q] = (r0 + l < s) ? colp(x)[r0 + l] : 0.0;
    }
  };
  auto store_chunk = [&](const double (&x8)[JEPT]) {
#pragma unroll
    for (int q = 0; q < JEPT; ++q) {
      const int e = tid + JNT * q;
      T[e % JR][e / JR] = x8[q];
    }
  };
  auto prime = [&]() {   // chunk 0 -> T; chunks 1 .. JAC_RING in flight
#pragma unroll
    for (int k = 0; k < JAC_RING; ++k)
      if (k < nch) load_chunk(k, pre[k]);
    store_chunk(pre[0]);
    if (JAC_RING < nch) load_chunk(JAC_RING, pre[0]);
    __syncthreads();
  };
  // after every wave is done with chunk c in T: publish chunk c + 1 from its slot and
  // refill that slot with chunk c + 1 + JAC_RING
  auto advance = [&](int c, double (&slot)[JEPT]) {
    if (c + 1 < nch) store_chunk(slot);
    if (c + 1 + JAC_RING < nch) load_chunk(c + 1 + JAC_RING, slot);
  };

  // (1) Gram of the 64 columns on fp64 MFMA (v_mfma_f64_16x16x4: lane l supplies
  // A[l%16][l/16] and B[l/16][l%16] and receives D[4r + l/16][l%16] in register r).
  // G is symmetric: only its ten 16 x 16 tiles (it, jt) with it <= jt are computed
  // (jac_gram_tiles) and mirrored when G is written.
  {
    const uint32_t tiles = jac_gram_tiles(wave);
    const int nt = ((tiles & 0xFF) != 0xFF) + ((tiles >> 8 & 0xFF) != 0xFF) + ((tiles >> 16 & 0xFF) != 0xFF);
    f64x4 acc[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) acc[k] = f64x4{0.0, 0.0, 0.0, 0.0};
    auto mult = [&]() {
#pragma unroll
      for (int ks = 0; ks < JR / 4; ++ks) {
        const int kr = 4 * ks + (lane >> 4);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          if (k < nt) {
            const int tl = (tiles >> (8 * k)) & 0xFF, it = tl >> 2, jt = tl & 3;
            acc[k] = __builtin_amdgcn_mfma_f64_16x16x4f64(T[kr][16 * it + (lane & 15)], T[kr][16 * jt + (lane & 15)],
                                                         acc[k], 0, 0, 0);
          }
        }
      }
    };
    prime();
    for (int c0 = 0; c0 < nch; c0 += JAC_RING) {   // unrolled by the ring size: static slots
#pragma unroll
      for (int k = 0; k < JAC_RING; ++k) {
        if (c0 + k >= nch) break;
        mult();
        __syncthreads();
        advance(c0 + k, pre[(k + 1) % JAC_RING]);
        __syncthreads();
      }
    }
    // T is idle now (the last pass ended with a barrier): write G over it
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      if (k < nt) {
        const int tl = (tiles >> (8 * k)) & 0xFF, it = tl >> 2, jt = tl & 3;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = 16 * it + 4 * r + (lane >> 4), j = 16 * jt + (lane & 15);
          Gm[i][j] = acc[k][r];
          if (it != jt) Gm[j][i] = acc[k][r];
        }
      }
    }
  }
  __syncthreads();
  // convergence measure of this pair (before rotating): max |g_xy| / sqrt(g_xx g_yy)
  {
    double* red = &Jm[0][0];   // J is built after this reduction
    double m = 0.0;
    for (int e = tid; e < PW * PW; e += JNT) {
      const int x = e / PW, y = e % PW;
      if (x < y) {
        const double den = sqrt(Gm[x][x] * Gm[y][y]);
        if (den > 0.0) m = fmax(m, fabs(Gm[x][y]) / den);
      }
    }
    red[tid] = m;
    __syncthreads();
    for (int o = JNT / 2; o > 0; o >>= 1) { if (tid < o) red[tid] = fmax(red[tid], red[tid + o]); __syncthreads(); }
    const double mx = red[0];
    const bool conv = mx < JAC_TOL;
    if (tid == 0) {
      atomicMax(&d.off[sweep], __float_as_uint((float)mx));
      d.jconv[pidx] = conv ? (uint32_t)sweep + 1 : 0u;
      d.jmx[pidx] = (float)mx;
      if (!conv) { d.jmod[ba] = gnow + 1; d.jmod[bb] = gnow + 1; }
    }
    if (conv) return;   // already orthogonal: nothing to rotate (uniform branch)
    __syncthreads();            // red[0] is read by every thread before J overwrites it
  }
  for (int e = tid; e < PW * PW; e += JNT) Jm[e / PW][e % PW] = (e / PW == e % PW) ? 1.0 : 0.0;
  __syncthreads();

  // (2) JAC_INNER_SWEEPS sweeps of parallel cyclic Jacobi on the 64 x 64 Gram, in place.
  // One round rotates 32 disjoint pairs (circle method) on both sides at once,
  // G' = R^T G R: lanes 0-31 of wave 0 compute the 32 rotations from the current G into
  // CS (once per round, not redundantly in every wave: the fp64 square roots and
  // divisions were 40 % of a round); after a barrier (every rotation computed from G
  // before any entry changes) each lane reads rotation beta = l % 32 and the rotations
  // of its row pairs alpha from CS, rewrites 16 / JAC_WAVES 2 x 2 blocks of G, which no
  // other lane touches, and applies rotation beta to 32 / JAC_WAVES rows of the
  // accumulated J. The barrier closing the round orders these writes before the next
  // round's reads of G and CS.
  {
    const int beta = lane & 31, half = lane >> 5;
    for (int isw = 0; isw < JAC_INNER_SWEEPS; ++isw) {
      for (int rr = 0; rr < PW - 1; ++rr) {
        int pb = circle(beta, rr, PW), qb = circle(PW - 1 - beta, rr, PW);
        if (pb > qb) { const int tmp = pb; pb = qb; qb = tmp; }
        if (tid < 32) {
          double c = 1.0, sn = 0.0;
          const double app = Gm[pb][pb], aqq = Gm[qb][qb], apq = Gm[pb][qb];
          const double den = sqrt(app * aqq);
          if (den > 0.0 && fabs(apq) > 1e-16 * den) {
            const double zeta = (aqq - app) / (2.0 * apq);
            const double tt = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            c = 1.0 / sqrt(1.0 + tt * tt);
            sn = c * tt;
          }
          CS[tid][0] = c;
          CS[tid][1] = sn;
        }
        __syncthreads();
        const double cb = CS[beta][0], sb = CS[beta][1];
#pragma unroll
        for (int i = 0; i < 16 / JAC_WAVES; ++i) {
          const int alpha = 2 * (16 / JAC_WAVES * wave + i) + half;
          int pa = circle(alpha, rr, PW), qa = circle(PW - 1 - alpha, rr, PW);
          if (pa > qa) { const int tmp = pa; pa = qa; qa = tmp; }
          const double ca = CS[alpha][0], sa = CS[alpha][1];
          const double g_pp = Gm[pa][pb], g_pq = Gm[pa][qb], g_qp = Gm[qa][pb], g_qq = Gm[qa][qb];
          const double r_pp = ca * g_pp - sa * g_qp, r_pq = ca * g_pq - sa * g_qq;   // rows
          const double r_qp = sa * g_pp + ca * g_qp, r_qq = sa * g_pq + ca * g_qq;
          Gm[pa][pb] = cb * r_pp - sb * r_pq;                                          // columns
          Gm[pa][qb] = sb * r_pp + cb * r_pq;
          Gm[qa][pb] = cb * r_qp - sb * r_qq;
          Gm[qa][qb] = sb * r_qp + cb * r_qq;
        }
#pragma unroll
        for (int i = 0; i < 32 / JAC_WAVES; ++i) {
          const int a = half + 2 * (wave + JAC_WAVES * i);
          const double jp = Jm[a][pb], jq = Jm[a][qb];
          Jm[a][pb] = cb * jp - sb * jq;
          Jm[a][qb] = sb * jp + cb * jq;
        }
        __syncthreads();
      }
    }
  }

  // (3) rotate the 64 columns: Zc[:, pair] <- Zc[:, pair] J, JR rows at a time on
  // fp64 MFMA; wave w computes columns [16 (w % 4), +16) of the chunk's 16-row halves
  // h = w / 4, w / 4 + 4, ... (with four waves both halves share J's fragment). The
  // result goes through LDS (region A's upper half) so the write-back is
  // column-contiguous.
  constexpr int NH = 8 / JAC_WAVES;   // 16-row halves per wave
  const int cbk = wave & 3, h0 = wave >> 2;
  // J is fixed for the whole pass: each wave keeps its 64 x 16 column slice of it as
  // MFMA B fragments in registers, so only the chunk operand is read from LDS
  double jf[PW / 4];
#pragma unroll
  for (int ks = 0; ks < PW / 4; ++ks) jf[ks] = Jm[4 * ks + (lane >> 4)][16 * cbk + (lane & 15)];
  auto rotate = [&]() {
    f64x4 o[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) o[h] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int ks = 0; ks < PW / 4; ++ks) {
      const int y = 4 * ks + (lane >> 4);
#pragma unroll
      for (int h = 0; h < NH; ++h)
        o[h] = __builtin_amdgcn_mfma_f64_16x16x4f64(T[16 * (h0 + h) + (lane & 15)][y], jf[ks], o[h], 0, 0, 0);
    }
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) O[16 * (h0 + h) + 4 * r + (lane >> 4)][16 * cbk + (lane & 15)] = o[h][r];
  };
  auto write_out = [&](int c) {
    const int64_t r0 = (int64_t)c * JR;
#pragma unroll
    for (int q = 0; q < JEPT; ++q) {
      const int e = tid + JNT * q, x = e / JR, l = e % JR;
      if (r0 + l < s) colp(x)[r0 + l] = O[l][x];
    }
  };
  prime();
  for (int c0 = 0; c0 < nch; c0 += JAC_RING) {   // unrolled by the ring size: static slots
#pragma unroll
    for (int k = 0; k < JAC_RING; ++k) {
      if (c0 + k >= nch) break;
      rotate();
      __syncthreads();
      write_out(c0 + k);
      advance(c0 + k, pre[(k + 1) % JAC_RING]);
      __syncthreads();
    }
  }
}

// ------------------------------------------------------------------ transpose
// One workgroup per 64 x 64 tile: coalesced row reads into LDS, coalesced row
// writes of the transposed tile (bf16 output).
__global__ __launch_bounds__(256) void k_transpose(const TransProb* __restrict__ ts, int n) {
  __shared__ float T[64][65];
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ts[mid].tile_start <= t) lo = mid; else hi = mid - 1; }
  const TransProb& P = ts[lo];
  const int rel = (int)(t - P.tile_start);
  const int64_t r0 = (int64_t)(rel / P.tiles_c) * 64, c0 = (int64_t)(rel % P.tiles_c) * 64;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e >> 6, c = e & 63;
    float v = 0.f;
    if (r0 + r < P.rows && c0 + c < P.cols) {
      const int64_t i = (r0 + r) * P.ldi + c0 + c;
      v = P.in_f32 ? ((const float*)P.in)[i]
                   : (float)((const bf16*)P.in)[P.in_kp ? kp_index(r0 + r, c0 + c, P.rows) : i];
    }
    T[r][c] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int c = e >> 6, r = e & 63;
    if (r0 + r < P.rows && c0 + c < P.cols) {
      const int64_t o = P.out_kp ? kp_index(c0 + c, r0 + r, P.cols) : (c0 + c) * P.ldo + r0 + r;
      const bf16 h = f2bf(T[r][c]);
      ((bf16*)P.out)[o] = h;
      if (P.out_lo) {
        const float d = T[r][c] - bf2f(h);   // exact
        const bf16 m = f2bf(d);
        ((bf16*)P.out_lo)[o] = m;
        if (P.out_lo2) ((bf16*)P.out_lo2)[o] = f2bf(d - bf2f(m));
      }
    }
  }
}

// ------------------------------------------------------------------ bf16 parts of V
// One workgroup per 64 x 64 tile of G: read along rows (coalesced), form v and its parts
// v_m, v_l (each difference is exact in fp32), store them straight (blocked, rows m) and,
// through LDS, transposed (blocked, rows n); both stores run along the K index of their
// layout.
__global__ __launch_bounds__(256) void k_split_lo(const SplitProb* __restrict__ ps, int np) {
  __shared__ float T[2][64][65];
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = np - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ps[mid].tile_start <= t) lo = mid; else hi = mid - 1; }
  const SplitProb& P = ps[lo];
  const int rel = (int)(t - P.tile_start);
  const int64_t r0 = (int64_t)(rel / P.tiles_c) * 64, c0 = (int64_t)(rel % P.tiles_c) * 64;
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int r = e >> 6, c = e & 63;
    float xm = 0.f, xl = 0.f;
    if (r0 + r < P.m && c0 + c < P.n) {
      const float g = P.g[(r0 + r) * P.n + c0 + c];
      const float v = P.inv ? g * P.inv[(r0 + r) * P.inv_ld + (c0 + c) / P.B] : g;
      const float d = v - bf2f(f2bf(v));
      const bf16 m = f2bf(d);
      xm = bf2f(m);
      xl = d - xm;
      const int64_t o = kp_index(r0 + r, c0 + c, P.m);
      ((bf16*)P.out_n[0])[o] = m;
      ((bf16*)P.out_n[1])[o] = f2bf(xl);
    }
    T[0][r][c] = xm;
    T[1][r][c] = xl;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int c = e >> 6, r = e & 63;
    if (r0 + r < P.m && c0 + c < P.n) {
      const int64_t o = kp_index(c0 + c, r0 + r, P.n);
      ((bf16*)P.out_t[0])[o] = f2bf(T[0][r][c]);
      ((bf16*)P.out_t[1])[o] = f2bf(T[1][r][c]);
    }
  }
}

// ------------------------------------------------------------------ R -> column-major
// Zc[j][i] = R[i][j] for i <= j < w (R: upper Cholesky factor left in C, row-major);
// zero below the diagonal (C still holds Gram entries there) and in padded columns.
__global__ __launch_bounds__(256) void k_r_colmajor(const RefDev* __restrict__ ds, int n) {
  __shared__ double tile[32][33];
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ds[mid].tile_cm <= t) lo = mid; else hi = mid - 1; }
  const RefDev& d = ds[lo];
  const int w = d.w;
  const int64_t tiles_i = (w + 31) / 32;
  const int64_t lt = t - d.tile_cm;
  const int64_t ti = lt % tiles_i, tj = lt / tiles_i;
  const int x = threadIdx.x & 31, y = threadIdx.x >> 5;
  for (int yy = y; yy < 32; yy += 8) {
    const int64_t i = ti * 32 + yy, j = tj * 32 + x;
    tile[yy][x] = (i < w && j < w && i <= j) ? d.C[i * w + j] : 0.0;
  }
  __syncthreads();
  for (int yy = y; yy < 32; yy += 8) {
    const int64_t j = tj * 32 + yy, i = ti * 32 + x;
    if (j < d.wpad && i < w) d.Zc[j * d.jl + i] = tile[x][yy];
  }
}

// ------------------------------------------------------------------ finalize
// After the Jacobi sweeps Zc = R J has orthogonal columns whose norms are the Ritz
// values; the Ritz vectors are Q (R J) / norm. k_finalize_order (one workgroup per
// matrix): column norms, order by decreasing norm, Bt = the first r columns,
// normalised (zero for numerically null directions). A GEMM then forms Pw = Q Bt^T.
// k_finalize_out: make each column's largest-magnitude entry positive (lowest index on
// ties) and write P (fp32 master and both operand copies). An all-zero iterate (V == 0) keeps the previous projector, or yields the
// first r canonical basis vectors when there is none; numerically null directions
// (Ritz value not above RITZ_NULL_REL of the largest) are written as e_j here and
// replaced by an orthonormal completion (k_complete_basis) when some directions were kept.
// Column norms of R J (the Ritz values): NORM_COLS columns per workgroup, one wave per
// column at a time (butterfly sum).
__device__ __forceinline__ bool null_dir(double nrm, double nmax) {
  return !(nrm > 1e-300) || !(nrm > RITZ_NULL_REL * nmax);
}
constexpr int NORM_COLS = 16;
__global__ __launch_bounds__(256) void k_col_norms(const RefDev* __restrict__ ds, int n) {
  const uint32_t t = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) { int mid = (lo + hi + 1) >> 1; if (ds[mid].tile_norm <= t) lo = mid; else hi = mid - 1; }
  const RefDev& d = ds[lo];
  const int c0 = (int)(t - d.tile_norm) * NORM_COLS;
  const int64_t L = d.jl;
  // an all-zero final iterate has R = I (zero-Gram fallback of the factorisation):
  // its Ritz values are all zero
  const bool zero = !(d.cmax[0] > 0.0);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int c = c0 + wave; c < c0 + NORM_COLS && c < d.wpad; c += 4) {
    const double* col = d.Zc + (int64_t)c * L;
    double a = 0.0;
    for (int64_t i = lane; i < L; i += 64) a = fma(col[i], col[i], a);
    a = wave_sum_d(a);
    if (lane == 0) d.norms[c] = zero ? 0.0 : sqrt(a);
  }
}

__global__ __launch_bounds__(256) void k_finalize_order(const RefDev* __restrict__ ds) {
  const RefDev& d = ds[blockIdx.x];
  const int tid = threadIdx.x;
  const int64_t L = d.jl;
  // rank of every column by decreasing norm (ties by index), norms read from LDS
  __shared__ double nl[2048];
  const bool in_lds = d.wpad <= 2048;
  // a norm that is not a finite number >= 0 ranks as -1, so the keys are totally ordered
  // and the ranks form a permutation of 0 .. wpad-1 (every entry of order is written)
  auto key = [](double v) { return (v >= 0.0 && v <= 1.7976931348623157e308) ? v : -1.0; };
  if (in_lds)
    for (int c = tid; c < d.wpad; c += 256) nl[c] = key(d.norms[c]);
  __syncthreads();
  for (int c = tid; c < d.wpad; c += 256) {
    const double nc = in_lds ? nl[c] : key(d.norms[c]);
    int rank = 0;
    for (int c2 = 0; c2 < d.wpad; ++c2) {
      const double n2 = in_lds ? nl[c2] : key(d.norms[c2]);
      rank += (n2 > nc) || (n2 == nc && c2 < c);
    }
    d.order[rank] = c;
  }
  __syncthreads();
  const double nmax = d.norms[d.order[0]];
  int kept = 0;
  for (int j = 0; j < d.r; ++j) {
    const int src = d.order[j];
    const double nrm = d.norms[src];
    const bool deg = null_dir(nrm, nmax);
    kept += deg ? 0 : 1;
    const double* col = d.Zc + (int64_t)src * L;
    for (int64_t i = tid; i < d.w; i += 256) d.Bt[(int64_t)j * d.w + i] = deg ? 0.f : (float)(col[i] / nrm);
  }
  if (tid == 0) {
    // the first sweep whose measured pair cosines all fell below the tolerance ended the
    // iteration (later sweeps returned at once and left their entries at zero)
    int sw = 0;
    while (sw < d.max_sweeps && !(__uint_as_float(d.off[sw]) < (float)JAC_TOL)) ++sw;
    const bool conv = sw < d.max_sweeps;
    d.info[0] = conv ? sw + 1 : d.max_sweeps;
    d.info[1] = conv ? 1 : 0;
    d.info[2] = kept;
    d.info[3] = (int32_t)d.off[conv ? sw : d.max_sweeps - 1];
  }
}

// k_finalize_out: one workgroup per (matrix, block of FO_COLS projector columns). Pass 1
// finds each column's entry of largest magnitude (lowest index on ties) with row-wise,
// coalesced reads; pass 2 writes the column block with that entry made positive: P
// (fp32 master) and the operand copy row by row, the transposed operand copy through a
// 32-row LDS tile so that its writes also run along its rows.
constexpr int FO_COLS = 64;
__global__ __launch_bounds__(256) void k_finalize_out(const RefDev* __restrict__ ds, int cblocks) {
  const RefDev& d = ds[blockIdx.x / cblocks];
  const int j0 = (int)(blockIdx.x % cblocks) * FO_COLS;
  const int r = d.r;
  if (j0 >= r) return;
  const double nmax = d.norms[d.order[0]];
  if (!(nmax > 0.0) && d.has_prev) return;   // V == 0: keep the previous projector
  __shared__ float bv[4][FO_COLS];
  __shared__ int bix[4][FO_COLS];
  __shared__ float sg[FO_COLS];              // column sign; 0 = null direction (e_j)
  __shared__ float tile[32][FO_COLS + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t s = d.s;
  const int j = j0 + lane;
  const bool jin = j < r;
  {
    float best = -1.f;
    int bi = 0;
    if (jin)
      for (int64_t i = wave; i < s; i += 4) {   // increasing rows: ties keep the lowest index
        const float v = fabsf(d.Pw[i * r + j]);
        if (v > best) { best = v; bi = (int)i; }
      }
    bv[wave][lane] = best;
    bix[wave][lane] = bi;
    __syncthreads();
    if (wave == 0) {
      for (int w2 = 1; w2 < 4; ++w2) {
        const float ob = bv[w2][lane];
        const int oi = bix[w2][lane];
        if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
      }
      float g = 1.f;
      if (jin) {
        const double nrm = d.norms[d.order[j]];
        g = null_dir(nrm, nmax) ? 0.f : ((d.Pw[(int64_t)bi * r + j] < 0.f) ? -1.f : 1.f);
      }
      sg[lane] = g;
    }
    __syncthreads();
  }
  const float g = sg[lane];
  for (int64_t i0 = 0; i0 < s; i0 += 32) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {   // row-major outputs: rows i0 + wave + 4 k, column j
      const int li = wave + 4 * k;
      const int64_t i = i0 + li;
      if (i < s && jin) {
        const float v = g == 0.f ? (i == (j % s) ? 1.f : 0.f) : g * d.Pw[i * r + j];
        d.P32[i * r + j] = v;
        if (d.operand_bf16) ((bf16*)d.Pop)[d.kp ? kp_index(i, j, s) : i * r + j] = f2bf(v);
        else ((float*)d.Pop)[i * r + j] = v;
        tile[li][lane] = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {   // transposed copy: row j0 + (tid >> 5) + 8 k, columns i0 ..
      const int lj = (tid >> 5) + 8 * k, li = tid & 31;
      const int jj = j0 + lj;
      const int64_t i = i0 + li;
      if (i < s && jj < r) {
        const float v = tile[li][lj];
        if (d.operand_bf16) ((bf16*)d.Ptop)[d.kp ? kp_index(jj, i, r) : (int64_t)jj * s + i] = f2bf(v);
        else ((float*)d.Ptop)[(int64_t)jj * s + i] = v;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ basis completion
// When only rho < r Ritz directions lie above the null level (V of rank below r), the
// remaining r - rho columns of P are completed to an orthonormal basis of the complement
// of the kept ones; any such completion is a top-r singular basis of a rank-deficient V.
// Candidates are the canonical vectors e_c at which the kept columns are smallest (rows
// of P by increasing squared norm, ties by index). Blocks of up to CB of them are
// projected off every column written so far, twice (classical Gram-Schmidt with
// reorthogonalisation), orthonormalised by the Cholesky factor of their CB x CB Gram
// matrix (after each projection), signed like the Ritz vectors (largest-magnitude entry
// positive, lowest index on ties) and appended to P and its operand copies. fp64
// arithmetic, one workgroup per matrix; a matrix whose directions were all kept (or
// whose V is zero) returns at once.
constexpr int CB = 64;
typedef double CbTile[CB + 1];

// acc (4 x 4 per thread: rows 4 (tid >> 4) + x, columns 4 (tid & 15) + y of a CB x CB
// tile) += sum_{k < K} fa(i, k) fb(k, j). ACOL: A is staged column by column (fa reads
// consecutive i at consecutive addresses).
template <bool ACOL, class FA, class FB>
__device__ void cb_mm(double (&acc)[4][4], int64_t K, FA fa, FB fb, CbTile* As, CbTile* Bs) {
  const int tid = threadIdx.x, ti = tid >> 4, tj = tid & 15;
  for (int64_t k0 = 0; k0 < K; k0 += CB) {
    __syncthreads();   // earlier readers of As / Bs are done
    for (int e = tid; e < CB * CB; e += 256) {
      const int i = ACOL ? (e & (CB - 1)) : (e / CB), k = ACOL ? (e / CB) : (e & (CB - 1));
      As[i][k] = (k0 + k < K) ? fa(i, k0 + k) : 0.0;
    }
    for (int e = tid; e < CB * CB; e += 256) {
      const int k = e / CB, j = e & (CB - 1);
      Bs[k][j] = (k0 + k < K) ? fb(k0 + k, j) : 0.0;
    }
    __syncthreads();
    const int kk = (int)((K - k0) < CB ? (K - k0) : CB);
    for (int k = 0; k < kk; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) { a[x] = As[4 * ti + x][k]; b[x] = Bs[k][4 * tj + x]; }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = fma(a[x], b[y], acc[x][y]);
    }
  }
}

__global__ __launch_bounds__(256) void k_complete_basis(const RefDev* __restrict__ ds) {
  const RefDev& d = ds[blockIdx.x];
  const int r = d.r, rho = d.info[2];
  if (rho <= 0 || rho >= r) return;
  __shared__ CbTile As[CB], Bs[CB], Hs[CB], Xs[CB];
  __shared__ double bvl[4][CB];
  __shared__ int bil[4][CB];
  __shared__ double sgn[CB];
  const int tid = threadIdx.x, ti = tid >> 4, tj = tid & 15;
  const int64_t s = d.s;
  float* P = d.P32;
  double* Cb = d.cw;                     // s x CB
  double* T = d.cw + s * CB;             // r x CB
  double* rn = T + (int64_t)r * CB;      // s
  const int q = r - rho;
  for (int64_t i = tid; i < s; i += 256) {
    double a = 0.0;
    for (int k = 0; k < rho; ++k) { const double v = P[i * r + k]; a = fma(v, v, a); }
    rn[i] = a;
  }
  __syncthreads();
  for (int64_t i = tid; i < s; i += 256) {
    const double v = rn[i];
    int64_t rank = 0;
    for (int64_t c = 0; c < s; ++c) { const double u = rn[c]; rank += (u < v) || (u == v && c < i); }
    if (rank < q) d.sidx[rank] = (int32_t)i;
  }
  __syncthreads();
  for (int b0 = 0; b0 < q; b0 += CB) {
    const int nb = (q - b0) < CB ? (q - b0) : CB;
    const int J = rho + b0;              // columns of P written so far
    const int32_t* S = d.sidx + b0;
    // Cb = E_S - P_J P_J[S, :]^T  (columns >= nb stay zero)
    for (int64_t r0 = 0; r0 < s; r0 += CB) {
      double acc[4][4] = {};
      cb_mm<false>(acc, J, [&](int i, int64_t k) { return r0 + i < s ? (double)P[(r0 + i) * r + k] : 0.0; },
                   [&](int64_t k, int j) { return j < nb ? (double)P[(int64_t)S[j] * r + k] : 0.0; }, As, Bs);
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          const int64_t i = r0 + 4 * ti + x;
          const int j = 4 * tj + y;
          if (i < s) Cb[i * CB + j] = j < nb ? ((i == S[j]) ? 1.0 : 0.0) - acc[x][y] : 0.0;
        }
    }
    for (int pass = 0; pass < 2; ++pass) {
      // T = P_J^T Cb ; Cb -= P_J T
      for (int t0 = 0; t0 < J; t0 += CB) {
        double acc[4][4] = {};
        cb_mm<true>(acc, s, [&](int i, int64_t k) { return t0 + i < J ? (double)P[k * r + t0 + i] : 0.0; },
                    [&](int64_t k, int j) { return Cb[k * CB + j]; }, As, Bs);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y)
            if (t0 + 4 * ti + x < J) T[(int64_t)(t0 + 4 * ti + x) * CB + 4 * tj + y] = acc[x][y];
      }
      __syncthreads();
      for (int64_t r0 = 0; r0 < s; r0 += CB) {
        double acc[4][4] = {};
        cb_mm<false>(acc, J, [&](int i, int64_t k) { return r0 + i < s ? (double)P[(r0 + i) * r + k] : 0.0; },
                     [&](int64_t k, int j) { return T[k * CB + j]; }, As, Bs);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) {
            const int64_t i = r0 + 4 * ti + x;
            if (i < s) Cb[i * CB + 4 * tj + y] -= acc[x][y];
          }
      }
      // Gram H = Cb^T Cb, unit diagonal past nb
      {
        double acc[4][4] = {};
        cb_mm<true>(acc, s, [&](int i, int64_t k) { return Cb[k * CB + i]; },
                    [&](int64_t k, int j) { return Cb[k * CB + j]; }, As, Bs);
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) {
            const int i = 4 * ti + x, j = 4 * tj + y;
            Hs[i][j] = (i < nb && j < nb) ? acc[x][y] : (i == j ? 1.0 : 0.0);
          }
      }
      __syncthreads();
      // Cholesky H = R^T R in place (upper triangle), pivots floored at 1e-28 of the largest
      double hmax = 0.0;
      for (int k = 0; k < CB; ++k) hmax = fmax(hmax, Hs[k][k]);
      const double floor_piv = 1e-28 * hmax + 1e-300;
      for (int k = 0; k < CB; ++k) {
        const double pk = Hs[k][k] > floor_piv ? Hs[k][k] : floor_piv;
        const double dk = sqrt(pk);
        __syncthreads();   // every thread has read Hs[k][k]
        for (int j = k + tid; j < CB; j += 256) Hs[k][j] = (j == k) ? dk : Hs[k][j] / dk;
        __syncthreads();
        for (int e = tid; e < CB * CB; e += 256) {
          const int i = e / CB, j = e & (CB - 1);
          if (i > k && j >= i) Hs[i][j] -= Hs[k][i] * Hs[k][j];
        }
        __syncthreads();
      }
      // X = R^{-1} (upper triangular), one column per thread
      for (int e = tid; e < CB * CB; e += 256) Xs[e / CB][e & (CB - 1)] = 0.0;
      __syncthreads();
      if (tid < CB) {
        const int j = tid;
        Xs[j][j] = 1.0 / Hs[j][j];
        for (int i = j - 1; i >= 0; --i) {
          double a = 0.0;
          for (int k = i + 1; k <= j; ++k) a = fma(Hs[i][k], Xs[k][j], a);
          Xs[i][j] = -a / Hs[i][i];
        }
      }
      __syncthreads();
      // Cb <- Cb X
      for (int64_t r0 = 0; r0 < s; r0 += CB) {
        double acc[4][4] = {};
        cb_mm<false>(acc, CB, [&](int i, int64_t k) { return r0 + i < s ? Cb[(r0 + i) * CB + k] : 0.0; },
                     [&](int64_t k, int j) { return Xs[k][j]; }, As, Bs);
        __syncthreads();   // the whole row block is staged before it is overwritten
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) {
            const int64_t i = r0 + 4 * ti + x;
            if (i < s) Cb[i * CB + 4 * tj + y] = acc[x][y];
          }
      }
      __syncthreads();
    }
    // signs: each column's largest-magnitude entry positive (lowest index on ties)
    {
      const int j = tid & (CB - 1), part = tid >> 6;
      double best = -1.0;
      int bi = 0;
      for (int64_t i = part; i < s; i += 4) {
        const double v = fabs(Cb[i * CB + j]);
        if (v > best) { best = v; bi = (int)i; }
      }
      bvl[part][j] = best;
      bil[part][j] = bi;
      __syncthreads();
      if (tid < CB) {
        for (int p2 = 1; p2 < 4; ++p2)
          if (bvl[p2][j] > best || (bvl[p2][j] == best && bil[p2][j] < bi)) { best = bvl[p2][j]; bi = bil[p2][j]; }
        sgn[j] = Cb[(int64_t)bi * CB + j] < 0.0 ? -1.0 : 1.0;
      }
      __syncthreads();
    }
    for (int64_t e = tid; e < s * nb; e += 256) {
      const int64_t i = e / nb;
      const int j = (int)(e % nb), col = J + j;
      const float v = (float)(sgn[j] * Cb[i * CB + j]);
      P[i * r + col] = v;
      if (d.operand_bf16) {
        ((bf16*)d.Pop)[d.kp ? kp_index(i, col, s) : i * r + col] = f2bf(v);
        ((bf16*)d.Ptop)[d.kp ? kp_index(col, i, r) : (int64_t)col * s + i] = f2bf(v);
      } else {
        ((float*)d.Pop)[i * r + col] = v;
        ((float*)d.Ptop)[(int64_t)col * s + i] = v;
      }
    }
    __syncthreads();   // the next block reads these columns
  }
}

__global__ __launch_bounds__(256) void k_convert_projector(const float* __restrict__ P32, void* Pop, void* Ptop,
                                                           int64_t s, int64_t r, int bf, int kp) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= s * r) return;
  const int64_t i = e / r, j = e % r;
  const float v = P32[e];
  if (bf) {
    ((bf16*)Pop)[kp ? kp_index(i, j, s) : e] = f2bf(v);
    ((bf16*)Ptop)[kp ? kp_index(j, i, r) : j * s + i] = f2bf(v);
  } else {
    ((float*)Pop)[e] = v;
    ((float*)Ptop)[j * s + i] = v;
  }
}

}  // namespace

uint32_t gauss_tiles(int64_t s, int32_t w) { return (uint32_t)((s * w + GAUSS_PER_WG - 1) / GAUSS_PER_WG); }
uint32_t gram_tiles(int32_t w) { const int T = (w + 63) / 64; return (uint32_t)(T * (T + 1) / 2); }
uint32_t jacobi_tiles(int32_t wpad) { return (uint32_t)(wpad / JB / 2); }

hipError_t launch_gauss(const RefDev* d, int n, uint32_t total, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_gauss, dim3(total), dim3(256), 0, st, d, n);
  return hipGetLastError();
}
hipError_t launch_gram(const GramProb* g, int n, uint32_t total, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_gram, dim3(total), dim3(256), 0, st, g, n);
  return hipGetLastError();
}
hipError_t launch_jacobi_round(const RefDev* d, int n, uint32_t total, int round, int sweep, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_jacobi_round, dim3(total), dim3(JNT), 0, st, d, n, round, sweep);
  return hipGetLastError();
}
uint32_t transpose_tiles(int64_t rows, int64_t cols) { return (uint32_t)(((rows + 63) / 64) * ((cols + 63) / 64)); }
hipError_t launch_transpose(const TransProb* t, int n, uint32_t total, hipStream_t st) {
  if (!n || !total) return hipSuccess;
  hipLaunchKernelGGL(k_transpose, dim3(total), dim3(256), 0, st, t, n);
  return hipGetLastError();
}
uint32_t split_lo_tiles(int64_t m, int64_t n) { return (uint32_t)(((m + 63) / 64) * ((n + 63) / 64)); }
hipError_t launch_split_lo(const SplitProb* p, int n, uint32_t total, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_split_lo, dim3(total), dim3(256), 0, st, p, n);
  return hipGetLastError();
}
uint32_t r_colmajor_tiles(int32_t w, int32_t wpad) { return (uint32_t)(((w + 31) / 32) * ((wpad + 31) / 32)); }
hipError_t launch_r_colmajor(const RefDev* d, int n, uint32_t total, hipStream_t st) {
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_r_colmajor, dim3(total), dim3(256), 0, st, d, n);
  return hipGetLastError();
}
uint32_t norm_tiles(int32_t wpad) { return (uint32_t)((wpad + NORM_COLS - 1) / NORM_COLS); }
hipError_t launch_finalize_order(const RefDev* d, int n, uint32_t norm_total, hipStream_t st) {
  if (!n) return hipSuccess;
  hipLaunchKernelGGL(k_col_norms, dim3(norm_total), dim3(256), 0, st, d, n);
  hipLaunchKernelGGL(k_finalize_order, dim3(n), dim3(256), 0, st, d);
  return hipGetLastError();
}
hipError_t launch_finalize_out(const RefDev* d, int n, int32_t rmax, hipStream_t st) {
  const int cblocks = (rmax + FO_COLS - 1) / FO_COLS;
  if (!n || !cblocks) return hipSuccess;
  hipLaunchKernelGGL(k_finalize_out, dim3(n * cblocks), dim3(256), 0, st, d, cblocks);
  return hipGetLastError();
}
hipError_t launch_complete_basis(const RefDev* d, int n, hipStream_t st) {
  if (!n) return hipSuccess;
  hipLaunchKernelGGL(k_complete_basis, dim3(n), dim3(256), 0, st, d);
  return hipGetLastError();
}
__global__ __launch_bounds__(256) void k_canonical_projector(float* __restrict__ P32, int64_t s, int64_t r) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < s * r) P32[e] = (e / r == e % r) ? 1.f : 0.f;
}
hipError_t launch_canonical_projector(float* P32, void* Pop, void* Ptop, int64_t s, int64_t r, int operand_bf16,
                                      int kp, hipStream_t st) {
  const int64_t total = s * r;
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_canonical_projector, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st, P32, s, r);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_convert_projector(P32, Pop, Ptop, s, r, operand_bf16, kp, st);
}
hipError_t launch_convert_projector(const float* P32, void* Pop, void* Ptop, int64_t s, int64_t r,
                                    int operand_bf16, int kp, hipStream_t st) {
  const int64_t total = s * r;
  if (!total) return hipSuccess;
  hipLaunchKernelGGL(k_convert_projector, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st, P32, Pop, Ptop,
                     s, r, operand_bf16, kp);
  return hipGetLastError();
}
