// Grouped MFMA GEMM kernels (gfx950, wave64).
//
// Tiles: 128 x 128 per workgroup of 256 threads (4 waves in a 2 x 2 grid, each
// wave owning a 64 x 64 sub-tile made of 2 x 2 MFMA 32x32 blocks).
//   KIND_BF16: v_mfma_f32_32x32x16_bf16, BK = 64, operands staged in LDS as
//              K-contiguous bf16 rows (16-byte fragment reads, rows padded by 16 B
//              so the eight 16-byte reads of a lane octet hit distinct banks).
//   KIND_F32 : v_mfma_f32_32x32x2_f32, BK = 32, LDS layout follows the global
//              contiguity of each operand (no transposition needed, one fp32 per
//              lane per MFMA).
// Direction operands (A_G_ROW / A_G_TRANS) are formed on the fly from the fp32
// gradient and the per-block reciprocal norms, so V is never materialised.
// Pipeline: global loads of tile k+1 are issued into registers before the MFMAs
// of tile k, then written to LDS between two barriers.
#include "gemm.h"

namespace {

constexpr int NT = 256;
constexpr int BF_LD = 64 + 8;     // bf16 LDS row stride (elements)
constexpr int F_LDK = 32 + 1;     // fp32 LDS row stride, K-contiguous layout
constexpr int F_LDT = 128 + 32;   // fp32 LDS row stride, M/N-contiguous layout

__device__ __forceinline__ int find_prob(const GemmProb* probs, int n, uint32_t t) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].tile_start <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Registers holding one prefetched tile slice per thread.
struct Pref {
  float fa[32];
  float sa[8];
  uint4 ua[4];
  float fb[16];
  uint4 ub[4];
};

// ------------------------------------------------------------------ bf16 kind
template <int AM>
__device__ __forceinline__ void bf_load_a(const GemmProb& P, int64_t row0, int64_t k0, int B, Pref& r) {
  const int tid = threadIdx.x;
  if constexpr (AM == A_G_ROW) {
    const float* G = (const float*)P.a;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
      float* d = &r.fa[u * 8];
      if (gr < P.M && gk + 8 <= P.K && (P.vec & 1)) {
        const float4* s = reinterpret_cast<const float4*>(G + gr * P.lda + gk);
        const float4 x0 = s[0], x1 = s[1];
        d[0] = x0.x; d[1] = x0.y; d[2] = x0.z; d[3] = x0.w;
        d[4] = x1.x; d[5] = x1.y; d[6] = x1.z; d[7] = x1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) d[e] = (gr < P.M && gk + e < P.K) ? G[gr * P.lda + gk + e] : 0.f;
      }
      r.sa[u] = (P.inv && gr < P.M && gk < P.K) ? P.inv[gr * P.inv_ld + gk / B] : 1.f;
    }
  } else if constexpr (AM == A_G_TRANS) {
    const float* G = (const float*)P.a;
    const int ig = tid & 31, kc = (tid >> 5) * 8;
    const int64_t gi = row0 + ig * 4;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t gk = k0 + kc + e;
      float* d = &r.fa[e * 4];
      if (gk < P.K && gi + 4 <= P.M && (P.vec & 1)) {
        const float4 x = *reinterpret_cast<const float4*>(G + gk * P.lda + gi);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gi + q < P.M) ? G[gk * P.lda + gi + q] : 0.f;
      }
      r.sa[e] = (P.inv && gk < P.K && gi < P.M) ? P.inv[gk * P.inv_ld + gi / B] : 1.f;
    }
  } else {  // A_KC, bf16 source
    const bf16* A = (const bf16*)P.a;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
      if (gr < P.M && gk + 8 <= P.K && (P.vec & 1)) {
        r.ua[u] = *reinterpret_cast<const uint4*>(A + gr * P.lda + gk);
      } else {
        bf16x8 t;
#pragma unroll
        for (int e = 0; e < 8; ++e) t[e] = (gr < P.M && gk + e < P.K) ? A[gr * P.lda + gk + e] : f2bf(0.f);
        r.ua[u] = *reinterpret_cast<uint4*>(&t);
      }
    }
  }
}

template <int AM>
__device__ __forceinline__ void bf_store_a(const GemmProb& P, int64_t row0, int64_t k0, int B, const Pref& r,
                                           bf16* As) {
  const int tid = threadIdx.x;
  if constexpr (AM == A_G_ROW) {
    const bool per_elem = (P.inv != nullptr) && (B & 7);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int i = idx >> 3, kc = (idx & 7) * 8;
      const int64_t gr = row0 + i, gk = k0 + kc;
      bf16x8 t;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float sc = r.sa[u];
        if (per_elem && gr < P.M && gk + e < P.K) sc = P.inv[gr * P.inv_ld + (gk + e) / B];
        t[e] = f2bf(r.fa[u * 8 + e] * sc);
      }
      *reinterpret_cast<bf16x8*>(As + i * BF_LD + kc) = t;
    }
  } else if constexpr (AM == A_G_TRANS) {
    const bool per_elem = (P.inv != nullptr) && (B & 3);
    const int ig = tid & 31, kc = (tid >> 5) * 8;
    const int64_t gi = row0 + ig * 4;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bf16x8 t;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float sc = r.sa[e];
        const int64_t gk = k0 + kc + e;
        if (per_elem && gk < P.K && gi + q < P.M) sc = P.inv[gk * P.inv_ld + (gi + q) / B];
        t[e] = f2bf(r.fa[e * 4 + q] * sc);
      }
      *reinterpret_cast<bf16x8*>(As + (ig * 4 + q) * BF_LD + kc) = t;
    }
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      *reinterpret_cast<uint4*>(As + (idx >> 3) * BF_LD + (idx & 7) * 8) = r.ua[u];
    }
  }
}

__device__ __forceinline__ void bf_load_b(const GemmProb& P, int64_t col0, int64_t k0, Pref& r) {
  const bf16* Bp = (const bf16*)P.b;
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + NT * u;
    const int64_t gj = col0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
    if (gj < P.N && gk + 8 <= P.K && (P.vec & 2)) {
      r.ub[u] = *reinterpret_cast<const uint4*>(Bp + gj * P.ldb + gk);
    } else {
      bf16x8 t;
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = (gj < P.N && gk + e < P.K) ? Bp[gj * P.ldb + gk + e] : f2bf(0.f);
      r.ub[u] = *reinterpret_cast<uint4*>(&t);
    }
  }
}

__device__ __forceinline__ void bf_store_b(const Pref& r, bf16* Bs) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + NT * u;
    *reinterpret_cast<uint4*>(Bs + (idx >> 3) * BF_LD + (idx & 7) * 8) = r.ub[u];
  }
}

// ------------------------------------------------------------------ fp32 kind
template <int AM>
__device__ __forceinline__ void f_load_a(const GemmProb& P, int64_t row0, int64_t k0, int B, Pref& r) {
  const int tid = threadIdx.x;
  const float* A = (const float*)P.a;
  if constexpr (AM == A_G_TRANS) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int64_t gi = row0 + (idx & 31) * 4, gk = k0 + (idx >> 5);
      float* d = &r.fa[u * 4];
      if (gk < P.K && gi + 4 <= P.M && (P.vec & 1)) {
        const float4 x = *reinterpret_cast<const float4*>(A + gk * P.lda + gi);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gi + q < P.M) ? A[gk * P.lda + gi + q] : 0.f;
      }
      r.sa[u] = (P.inv && gk < P.K && gi < P.M) ? P.inv[gk * P.inv_ld + gi / B] : 1.f;
    }
  } else {  // A_G_ROW or A_KC (fp32)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 4;
      float* d = &r.fa[u * 4];
      if (gr < P.M && gk + 4 <= P.K && (P.vec & 1)) {
        const float4 x = *reinterpret_cast<const float4*>(A + gr * P.lda + gk);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = (gr < P.M && gk + e < P.K) ? A[gr * P.lda + gk + e] : 0.f;
      }
      if constexpr (AM == A_G_ROW)
        r.sa[u] = (P.inv && gr < P.M && gk < P.K) ? P.inv[gr * P.inv_ld + gk / B] : 1.f;
    }
  }
}

template <int AM>
__device__ __forceinline__ void f_store_a(const GemmProb& P, int64_t row0, int64_t k0, int B, const Pref& r,
                                          float* As) {
  const int tid = threadIdx.x;
  if constexpr (AM == A_G_TRANS) {
    const bool per_elem = (P.inv != nullptr) && (B & 3);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int ig = idx & 31, kr = idx >> 5;
      const int64_t gi = row0 + ig * 4, gk = k0 + kr;
      float4 x;
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float sc = r.sa[u];
        if (per_elem && gk < P.K && gi + q < P.M) sc = P.inv[gk * P.inv_ld + (gi + q) / B];
        v[q] = r.fa[u * 4 + q] * sc;
      }
      x.x = v[0]; x.y = v[1]; x.z = v[2]; x.w = v[3];
      *reinterpret_cast<float4*>(As + kr * F_LDT + ig * 4) = x;
    }
  } else {
    const bool per_elem = (AM == A_G_ROW) && (P.inv != nullptr) && (B & 3);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + NT * u;
      const int i = idx >> 3, kq = (idx & 7) * 4;
      const int64_t gr = row0 + i, gk = k0 + kq;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float sc = (AM == A_G_ROW) ? r.sa[u] : 1.f;
        if (per_elem && gr < P.M && gk + e < P.K) sc = P.inv[gr * P.inv_ld + (gk + e) / B];
        As[i * F_LDK + kq + e] = r.fa[u * 4 + e] * sc;
      }
    }
  }
}

template <int BMODE>
__device__ __forceinline__ void f_load_b(const GemmProb& P, int64_t col0, int64_t k0, Pref& r) {
  const int tid = threadIdx.x;
  const float* Bp = (const float*)P.b;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + NT * u;
    float* d = &r.fb[u * 4];
    if constexpr (BMODE == B_NC) {
      const int64_t gj = col0 + (idx & 31) * 4, gk = k0 + (idx >> 5);
      if (gk < P.K && gj + 4 <= P.N && (P.vec & 2)) {
        const float4 x = *reinterpret_cast<const float4*>(Bp + gk * P.ldb + gj);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gj + q < P.N) ? Bp[gk * P.ldb + gj + q] : 0.f;
      }
    } else {
      const int64_t gj = col0 + (idx >> 3), gk = k0 + (idx & 7) * 4;
      if (gj < P.N && gk + 4 <= P.K && (P.vec & 2)) {
        const float4 x = *reinterpret_cast<const float4*>(Bp + gj * P.ldb + gk);
        d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) d[e] = (gj < P.N && gk + e < P.K) ? Bp[gj * P.ldb + gk + e] : 0.f;
      }
    }
  }
}

template <int BMODE>
__device__ __forceinline__ void f_store_b(const Pref& r, float* Bs) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + NT * u;
    if constexpr (BMODE == B_NC) {
      float4 x;
      x.x = r.fb[u * 4 + 0]; x.y = r.fb[u * 4 + 1]; x.z = r.fb[u * 4 + 2]; x.w = r.fb[u * 4 + 3];
      *reinterpret_cast<float4*>(Bs + (idx >> 5) * F_LDT + (idx & 31) * 4) = x;
    } else {
      const int j = idx >> 3, kq = (idx & 7) * 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[j * F_LDK + kq + e] = r.fb[u * 4 + e];
    }
  }
}

// ------------------------------------------------------------------ epilogue
template <int KIND, int EP>
__device__ __forceinline__ void epilogue(const GemmProb& P, const GemmUniform& U, int64_t row0, int64_t col0,
                                         f32x16 (&acc)[2][2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int64_t col = col0 + wn * 64 + ni * 32 + (lane & 31);
      if (col >= P.N) continue;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t row = row0 + wm * 64 + mi * 32 + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
        if (row >= P.M) continue;
        const float v = acc[mi][ni][j];
        if constexpr (EP == EP_STORE) {
          ((float*)P.c)[row * P.ldc + col] = v;
        } else if constexpr (EP == EP_ADAM) {
          const int64_t idx = row * P.ldc + col;
          float e = P.e1[idx], q = P.e2[idx];
          const float out = adam_out(v, e, q, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2);
          P.e1[idx] = e;
          P.e2[idx] = q;
          if constexpr (KIND == KIND_BF16) ((bf16*)P.c)[idx] = f2bf(out);
          else ((float*)P.c)[idx] = out;
        } else {  // EP_UPDATE
          const int64_t idx = row * P.ldc + col;
          const float mag = P.dM ? P.dM[row * P.dM_ld + col / U.B] : 1.f;
          const float u = U.scale * (mag * v);
          if (U.weight_bf16) {
            bf16* W = (bf16*)P.c;
            const float ub = bf2f(f2bf(u));
            W[idx] = f2bf(bf2f(W[idx]) - U.lr * ub);
          } else {
            float* W = (float*)P.c;
            W[idx] = W[idx] - U.lr * u;
          }
        }
      }
    }
}

// ------------------------------------------------------------------ kernels
template <int AM, int EP>
__global__ __launch_bounds__(NT) void k_gemm_bf16(const GemmProb* __restrict__ probs, GemmUniform U) {
  constexpr int BM = 128, BN = 128, BK = 64;
  __shared__ __attribute__((aligned(16))) bf16 As[BM * BF_LD];
  __shared__ __attribute__((aligned(16))) bf16 Bs[BN * BF_LD];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const GemmProb& P = probs[find_prob(probs, U.nprob, t)];
  const uint32_t lt = t - P.tile_start;
  const int64_t row0 = (int64_t)(lt / P.tiles_n) * BM, col0 = (int64_t)(lt % P.tiles_n) * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mi][ni][j] = 0.f;

  Pref r;
  bf_load_a<AM>(P, row0, 0, U.B, r);
  bf_load_b(P, col0, 0, r);
  bf_store_a<AM>(P, row0, 0, U.B, r, As);
  bf_store_b(r, Bs);
  __syncthreads();
  for (int64_t k0 = 0; k0 < P.K; k0 += BK) {
    const bool more = k0 + BK < P.K;
    if (more) {
      bf_load_a<AM>(P, row0, k0 + BK, U.B, r);
      bf_load_b(P, col0, k0 + BK, r);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[2], bv[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        af[mi] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + mi * 32 + (lane & 31)) * BF_LD + kk * 16 + (lane >> 5) * 8);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bv[ni] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + ni * 32 + (lane & 31)) * BF_LD + kk * 16 + (lane >> 5) * 8);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bv[ni], acc[mi][ni], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
      bf_store_a<AM>(P, row0, k0 + BK, U.B, r, As);
      bf_store_b(r, Bs);
    }
    __syncthreads();
  }
  epilogue<KIND_BF16, EP>(P, U, row0, col0, acc);
}

template <int AM, int BMODE, int EP>
__global__ __launch_bounds__(NT) void k_gemm_f32(const GemmProb* __restrict__ probs, GemmUniform U) {
  constexpr int BM = 128, BN = 128, BK = 32;
  constexpr bool AT = (AM == A_G_TRANS);
  constexpr bool BT = (BMODE == B_NC);
  __shared__ __attribute__((aligned(16))) float As[AT ? BK * F_LDT : BM * F_LDK];
  __shared__ __attribute__((aligned(16))) float Bs[BT ? BK * F_LDT : BN * F_LDK];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const GemmProb& P = probs[find_prob(probs, U.nprob, t)];
  const uint32_t lt = t - P.tile_start;
  const int64_t row0 = (int64_t)(lt / P.tiles_n) * BM, col0 = (int64_t)(lt % P.tiles_n) * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mi][ni][j] = 0.f;

  Pref r;
  f_load_a<AM>(P, row0, 0, U.B, r);
  f_load_b<BMODE>(P, col0, 0, r);
  f_store_a<AM>(P, row0, 0, U.B, r, As);
  f_store_b<BMODE>(r, Bs);
  __syncthreads();
  for (int64_t k0 = 0; k0 < P.K; k0 += BK) {
    const bool more = k0 + BK < P.K;
    if (more) {
      f_load_a<AM>(P, row0, k0 + BK, U.B, r);
      f_load_b<BMODE>(P, col0, k0 + BK, r);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 2; ++kk) {
      const int kx = kk * 2 + (lane >> 5);
      float af[2], bv[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int i = wm * 64 + mi * 32 + (lane & 31);
        af[mi] = AT ? As[kx * F_LDT + i] : As[i * F_LDK + kx];
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = wn * 64 + ni * 32 + (lane & 31);
        bv[ni] = BT ? Bs[kx * F_LDT + j] : Bs[j * F_LDK + kx];
      }
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[mi], bv[ni], acc[mi][ni], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
      f_store_a<AM>(P, row0, k0 + BK, U.B, r, As);
      f_store_b<BMODE>(r, Bs);
    }
    __syncthreads();
  }
  epilogue<KIND_F32, EP>(P, U, row0, col0, acc);
}

}  // namespace

uint32_t gemm_tiles_m(int kind, int64_t M) { (void)kind; return (uint32_t)((M + 127) / 128); }
uint32_t gemm_tiles_n(int kind, int64_t N) { (void)kind; return (uint32_t)((N + 127) / 128); }

#define GEMM_BF(AM, EP) \
  if (amode == AM && ep == EP) { hipLaunchKernelGGL((k_gemm_bf16<AM, EP>), grid, dim3(NT), 0, st, probs_dev, u); return hipGetLastError(); }
#define GEMM_F(AM, BMO, EP) \
  if (amode == AM && bmode == BMO && ep == EP) { hipLaunchKernelGGL((k_gemm_f32<AM, BMO, EP>), grid, dim3(NT), 0, st, probs_dev, u); return hipGetLastError(); }

hipError_t launch_gemm(int kind, int amode, int bmode, int ep, const GemmProb* probs_dev, int nprob,
                       uint32_t total_tiles, const GemmUniform& u0, hipStream_t st) {
  if (total_tiles == 0 || nprob == 0) return hipSuccess;
  GemmUniform u = u0;
  u.nprob = nprob;
  const dim3 grid(total_tiles);
  if (kind == KIND_BF16) {
    if (bmode != B_KC) return hipErrorInvalidValue;
    GEMM_BF(A_G_ROW, EP_ADAM)
    GEMM_BF(A_G_TRANS, EP_ADAM)
    GEMM_BF(A_KC, EP_UPDATE)
  } else {
    GEMM_F(A_G_ROW, B_KC, EP_ADAM)
    GEMM_F(A_G_TRANS, B_KC, EP_ADAM)
    GEMM_F(A_KC, B_KC, EP_UPDATE)
    GEMM_F(A_G_ROW, B_NC, EP_STORE)
    GEMM_F(A_G_TRANS, B_NC, EP_STORE)
    GEMM_F(A_KC, B_NC, EP_STORE)
  }
  return hipErrorInvalidValue;
}
