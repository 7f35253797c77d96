// Grouped MFMA GEMM kernels (gfx950, wave64).
//
// Every wave owns a 64 x 64 sub-tile made of 2 x 2 MFMA 32x32 blocks; a
// workgroup stacks WM x WN waves (BM = 64 WM rows, BN = 64 WN columns).
//   KIND_BF16: v_mfma_f32_32x32x16_bf16, BK = 64, 128 x 128 tiles (4 waves).
//              Operands are staged in LDS as K-contiguous bf16 rows (16-byte
//              fragment reads; rows padded by 16 B so the eight 16-byte reads of
//              a lane octet hit distinct banks).
//   KIND_F32 : v_mfma_f32_32x32x2_f32, BK = 32, 128 x 128 tiles (4 waves); the
//              LDS layout follows each operand's global contiguity (no transpose).
// The MFMA is issued as C^T = B A^T, so each lane's accumulators hold four
// consecutive columns of one output row: the epilogues read and write 16-byte
// (fp32) or 8-byte (bf16) vectors.
// Direction operands (A_G_ROW / A_G_TRANS) are formed on the fly from the fp32
// gradient and the per-block reciprocal norms, so V is never materialised.
// Pipeline: two LDS stages, one barrier per tile. bf16 x bf16 operands (the
// back-projection) use two register sets for a prefetch distance of two k-tiles;
// the gradient-sourced operands hold 32 fp32 per thread per tile, so they keep
// one set. Two workgroups per CU overlap one workgroup's epilogue with the
// other's main loop.
#include "gemm.h"

namespace {

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

// ------------------------------------------------------------------ loads
// Fast path: raw buffer loads (V# with the array's byte extent), so rows past
// the end of an operand read as 0 in hardware and the steady-state loop has no
// branches; elements past K inside a row (K tail) or past M/N inside a row
// (transposed layouts) are zeroed with selects when the tile is written to LDS.
// Slow path (row stride not a multiple of the vector width): checked scalar loads.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t mk_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 bld4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}
__device__ __forceinline__ uint4 bld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float bld1(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
__device__ __forceinline__ uint32_t keep2(int nvalid, int e) {   // mask keeping elements e, e+1 if < nvalid
  return (e < nvalid ? 0x0000FFFFu : 0u) | (e + 1 < nvalid ? 0xFFFF0000u : 0u);
}
__device__ __forceinline__ uint4 mask_bf16x8(uint4 v, int nvalid) {   // keep the first nvalid of 8 (branch-free)
  v.x &= keep2(nvalid, 0);
  v.y &= keep2(nvalid, 2);
  v.z &= keep2(nvalid, 4);
  v.w &= keep2(nvalid, 6);
  return v;
}

struct Rs {
  __amdgpu_buffer_rsrc_t a, b, inv;
};
__device__ __forceinline__ Rs make_rs(const GemmProb& P) {
  Rs r;
  r.a = mk_rsrc(P.a, P.a_bytes);
  r.b = mk_rsrc(P.b, P.b_bytes);
  r.inv = mk_rsrc(P.inv, P.inv ? P.inv_bytes : 0u);
  return r;
}

// ------------------------------------------------------------------ bf16 kind
// Tile BM x 64 of A (or BN x 64 of B) = BM*8 chunks of 8 elements.
template <int AM, int BM, int NT, bool FAST>
struct BfA {
  static constexpr int TASKS = (AM == A_G_TRANS) ? (BM / 4) * 8 / NT : BM * 8 / NT;   // per thread
  float f[(AM == A_KC) ? 1 : 32];
  float s[8];
  uint4 u[(AM == A_KC) ? TASKS : 1];

  __device__ __forceinline__ void load(const GemmProb& P, const Rs& R, int64_t row0, int64_t k0, int B) {
    const int tid = threadIdx.x;
    if constexpr (AM == A_G_ROW) {
      static_assert(TASKS == 4, "A_G_ROW expects 4 tasks per thread");
      const float* G = (const float*)P.a;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + NT * u;
        const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
        float* d = &f[u * 8];
        if constexpr (FAST) {
          const uint32_t off = (uint32_t)((gr * P.lda + gk) * 4);
          const float4 x0 = bld4(R.a, off), x1 = bld4(R.a, off + 16);
          d[0] = x0.x; d[1] = x0.y; d[2] = x0.z; d[3] = x0.w;
          d[4] = x1.x; d[5] = x1.y; d[6] = x1.z; d[7] = x1.w;
          s[u] = P.inv ? bld1(R.inv, (uint32_t)((gr * P.inv_ld + gk / B) * 4)) : 1.f;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) d[e] = (gr < P.M && gk + e < P.K) ? G[gr * P.lda + gk + e] : 0.f;
          s[u] = (P.inv && gr < P.M && gk < P.K) ? P.inv[gr * P.inv_ld + gk / B] : 1.f;
        }
      }
    } else if constexpr (AM == A_G_TRANS) {
      static_assert(TASKS == 1, "A_G_TRANS expects 1 task per thread");
      const float* G = (const float*)P.a;
      const int ig = tid % (BM / 4), kc = (tid / (BM / 4)) * 8;
      const int64_t gi = row0 + ig * 4;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t gk = k0 + kc + e;
        float* d = &f[e * 4];
        if constexpr (FAST) {
          const float4 x = bld4(R.a, (uint32_t)((gk * P.lda + gi) * 4));
          d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
          s[e] = P.inv ? bld1(R.inv, (uint32_t)((gk * P.inv_ld + gi / B) * 4)) : 1.f;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gi + q < P.M) ? G[gk * P.lda + gi + q] : 0.f;
          s[e] = (P.inv && gk < P.K && gi < P.M) ? P.inv[gk * P.inv_ld + gi / B] : 1.f;
        }
      }
    } else {
      const bf16* A = (const bf16*)P.a;
#pragma unroll
      for (int u = 0; u < TASKS; ++u) {
        const int idx = tid + NT * u;
        const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
        const bool kpa = P.kp & 1;   // blocked layout: 8-element chunks never straddle a 32-block
        if constexpr (FAST) {
          this->u[u] = bld16(R.a, (uint32_t)((kpa ? kp_index(gr, gk, P.M) : gr * P.lda + gk) * 2));
        } else {
          bf16x8 t;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            t[e] = (gr < P.M && gk + e < P.K) ? A[kpa ? kp_index(gr, gk + e, P.M) : gr * P.lda + gk + e] : f2bf(0.f);
          this->u[u] = *reinterpret_cast<uint4*>(&t);
        }
      }
    }
  }

  __device__ __forceinline__ void store(const GemmProb& P, int64_t row0, int64_t k0, int B, bf16* As) const {
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
          float sc = s[u];
          if (per_elem && gr < P.M && gk + e < P.K) sc = P.inv[gr * P.inv_ld + (gk + e) / B];
          const float v = f[u * 8 + e] * sc;
          t[e] = f2bf((FAST && gk + e >= P.K) ? 0.f : v);
        }
        *reinterpret_cast<bf16x8*>(As + i * BF_LD + kc) = t;
      }
    } else if constexpr (AM == A_G_TRANS) {
      const bool per_elem = (P.inv != nullptr) && (B & 3);
      const int ig = tid % (BM / 4), kc = (tid / (BM / 4)) * 8;
      const int64_t gi = row0 + ig * 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bf16x8 t;
        const bool colok = gi + q < P.M;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float sc = s[e];
          const int64_t gk = k0 + kc + e;
          if (per_elem && gk < P.K && colok) sc = P.inv[gk * P.inv_ld + (gi + q) / B];
          const float v = f[e * 4 + q] * sc;
          t[e] = f2bf((FAST && !colok) ? 0.f : v);
        }
        *reinterpret_cast<bf16x8*>(As + (ig * 4 + q) * BF_LD + kc) = t;
      }
    } else {
#pragma unroll
      for (int u = 0; u < TASKS; ++u) {
        const int idx = tid + NT * u;
        uint4 v = this->u[u];
        if constexpr (FAST) v = mask_bf16x8(v, (int)(P.K - (k0 + (idx & 7) * 8)));
        *reinterpret_cast<uint4*>(As + (idx >> 3) * BF_LD + (idx & 7) * 8) = v;
      }
    }
  }
};

template <int BN, int NT, bool FAST>
struct BfB {
  static constexpr int TASKS = BN * 8 / NT;
  uint4 u[TASKS];
  __device__ __forceinline__ void load(const GemmProb& P, const Rs& R, int64_t col0, int64_t k0) {
    const bf16* Bp = (const bf16*)P.b;
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < TASKS; ++q) {
      const int idx = tid + NT * q;
      const int64_t gj = col0 + (idx >> 3), gk = k0 + (idx & 7) * 8;
      const bool kpb = P.kp & 2;
      if constexpr (FAST) {
        u[q] = bld16(R.b, (uint32_t)((kpb ? kp_index(gj, gk, P.N) : gj * P.ldb + gk) * 2));
      } else {
        bf16x8 t;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = (gj < P.N && gk + e < P.K) ? Bp[kpb ? kp_index(gj, gk + e, P.N) : gj * P.ldb + gk + e] : f2bf(0.f);
        u[q] = *reinterpret_cast<uint4*>(&t);
      }
    }
  }
  __device__ __forceinline__ void store(const GemmProb& P, int64_t k0, bf16* Bs) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < TASKS; ++q) {
      const int idx = tid + NT * q;
      uint4 v = u[q];
      if constexpr (FAST) v = mask_bf16x8(v, (int)(P.K - (k0 + (idx & 7) * 8)));
      *reinterpret_cast<uint4*>(Bs + (idx >> 3) * BF_LD + (idx & 7) * 8) = v;
    }
  }
};

// ------------------------------------------------------------------ fp32 kind (128 x 128, 4 waves)
constexpr int FNT = 256;

template <int AM, bool FAST>
struct FA {
  float f[16];
  float s[4];
  __device__ __forceinline__ void load(const GemmProb& P, const Rs& R, int64_t row0, int64_t k0, int B) {
    const int tid = threadIdx.x;
    const float* A = (const float*)P.a;
    if constexpr (AM == A_G_TRANS) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + FNT * u;
        const int64_t gi = row0 + (idx & 31) * 4, gk = k0 + (idx >> 5);
        float* d = &f[u * 4];
        if constexpr (FAST) {
          const float4 x = bld4(R.a, (uint32_t)((gk * P.lda + gi) * 4));
          d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
          s[u] = P.inv ? bld1(R.inv, (uint32_t)((gk * P.inv_ld + gi / B) * 4)) : 1.f;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gi + q < P.M) ? A[gk * P.lda + gi + q] : 0.f;
          s[u] = (P.inv && gk < P.K && gi < P.M) ? P.inv[gk * P.inv_ld + gi / B] : 1.f;
        }
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + FNT * u;
        const int64_t gr = row0 + (idx >> 3), gk = k0 + (idx & 7) * 4;
        float* d = &f[u * 4];
        if constexpr (FAST) {
          const float4 x = bld4(R.a, (uint32_t)((gr * P.lda + gk) * 4));
          d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
          if constexpr (AM == A_G_ROW) s[u] = P.inv ? bld1(R.inv, (uint32_t)((gr * P.inv_ld + gk / B) * 4)) : 1.f;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) d[e] = (gr < P.M && gk + e < P.K) ? A[gr * P.lda + gk + e] : 0.f;
          if constexpr (AM == A_G_ROW)
            s[u] = (P.inv && gr < P.M && gk < P.K) ? P.inv[gr * P.inv_ld + gk / B] : 1.f;
        }
      }
    }
  }
  __device__ __forceinline__ void store(const GemmProb& P, int64_t row0, int64_t k0, int B, float* As) const {
    const int tid = threadIdx.x;
    if constexpr (AM == A_G_TRANS) {
      const bool per_elem = (P.inv != nullptr) && (B & 3);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + FNT * u;
        const int ig = idx & 31, kr = idx >> 5;
        const int64_t gi = row0 + ig * 4, gk = k0 + kr;
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float sc = s[u];
          if (per_elem && gk < P.K && gi + q < P.M) sc = P.inv[gk * P.inv_ld + (gi + q) / B];
          v[q] = (FAST && gi + q >= P.M) ? 0.f : f[u * 4 + q] * sc;
        }
        *reinterpret_cast<float4*>(As + kr * F_LDT + ig * 4) = make_float4(v[0], v[1], v[2], v[3]);
      }
    } else {
      const bool per_elem = (AM == A_G_ROW) && (P.inv != nullptr) && (B & 3);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = tid + FNT * u;
        const int i = idx >> 3, kq = (idx & 7) * 4;
        const int64_t gr = row0 + i, gk = k0 + kq;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float sc = (AM == A_G_ROW) ? s[u] : 1.f;
          if (per_elem && gr < P.M && gk + e < P.K) sc = P.inv[gr * P.inv_ld + (gk + e) / B];
          As[i * F_LDK + kq + e] = (FAST && gk + e >= P.K) ? 0.f : f[u * 4 + e] * sc;
        }
      }
    }
  }
};

template <int BMODE, bool FAST>
struct FB {
  float f[16];
  __device__ __forceinline__ void load(const GemmProb& P, const Rs& R, int64_t col0, int64_t k0) {
    const int tid = threadIdx.x;
    const float* Bp = (const float*)P.b;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + FNT * u;
      float* d = &f[u * 4];
      if constexpr (BMODE == B_NC) {
        const int64_t gj = col0 + (idx & 31) * 4, gk = k0 + (idx >> 5);
        if constexpr (FAST) {
          const float4 x = bld4(R.b, (uint32_t)((gk * P.ldb + gj) * 4));
          d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) d[q] = (gk < P.K && gj + q < P.N) ? Bp[gk * P.ldb + gj + q] : 0.f;
        }
      } else {
        const int64_t gj = col0 + (idx >> 3), gk = k0 + (idx & 7) * 4;
        if constexpr (FAST) {
          const float4 x = bld4(R.b, (uint32_t)((gj * P.ldb + gk) * 4));
          d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) d[e] = (gj < P.N && gk + e < P.K) ? Bp[gj * P.ldb + gk + e] : 0.f;
        }
      }
    }
  }
  __device__ __forceinline__ void store(const GemmProb& P, int64_t col0, int64_t k0, float* Bs) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + FNT * u;
      if constexpr (BMODE == B_NC) {
        const int64_t gj = col0 + (idx & 31) * 4;
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = (FAST && gj + q >= P.N) ? 0.f : f[u * 4 + q];
        *reinterpret_cast<float4*>(Bs + (idx >> 5) * F_LDT + (idx & 31) * 4) = make_float4(v[0], v[1], v[2], v[3]);
      } else {
        const int j = idx >> 3, kq = (idx & 7) * 4;
        const int64_t gk = k0 + kq;
#pragma unroll
        for (int e = 0; e < 4; ++e) Bs[j * F_LDK + kq + e] = (FAST && gk + e >= P.K) ? 0.f : f[u * 4 + e];
      }
    }
  }
};

// ------------------------------------------------------------------ epilogue
// acc[mi][ni][j] (issued as C^T = B A^T) holds C[row][col] with
//   row = row0 + wm*64 + mi*32 + (lane & 31)
//   col = col0 + wn*64 + ni*32 + 8*(j/4) + 4*(lane/32) + (j%4)
// i.e. four consecutive columns per (mi, ni, g = j/4).
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

template <int KIND, int EP, int WN>
__device__ __forceinline__ void epilogue(const GemmProb& P, const GemmUniform& U, int64_t row0, int64_t col0,
                                         const f32x16 (&acc)[2][2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  double s_gr = 0.0, s_rr = 0.0, s_gg = 0.0;   // EP_ALIGN partial sums
#pragma unroll
  for (int mi = 0; mi < 2; ++mi) {
    const int64_t row = row0 + wm * 64 + mi * 32 + (lane & 31);
    if (row >= P.M) continue;
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t col = col0 + wn * 64 + ni * 32 + 8 * g + 4 * (lane >> 5);
        if (col >= P.N) continue;
        float v[4] = {acc[mi][ni][4 * g + 0], acc[mi][ni][4 * g + 1], acc[mi][ni][4 * g + 2], acc[mi][ni][4 * g + 3]};
        const int64_t idx = row * P.ldc + col;
        // vector access needs the whole group in range and an aligned address (W is caller memory)
        const int esz = (EP == EP_UPDATE) ? (U.weight_bf16 ? 2 : 4) : ((EP == EP_ADAM && KIND == KIND_BF16) ? 2 : 4);
        const bool full = (col + 4 <= P.N) && ((idx & 3) == 0) &&
                          ((((uintptr_t)P.c) & (uintptr_t)(4 * esz - 1)) == 0);
        if constexpr (EP == EP_STORE) {
          float* C = (float*)P.c;
          if (full) *reinterpret_cast<float4*>(C + idx) = make_float4(v[0], v[1], v[2], v[3]);
          else
            for (int q = 0; q < 4; ++q) if (col + q < P.N) C[idx + q] = v[q];
        } else if constexpr (EP == EP_ALIGN) {
          // G_recon = Rep_B(M) * (projected direction); the gradient is read, never written
          const float* Gr = (const float*)P.c;
          const float* ivr = P.inv ? P.inv + row * P.inv_ld : nullptr;
          float gv[4] = {0.f, 0.f, 0.f, 0.f};
          if (full) {
            const float4 x = *reinterpret_cast<const float4*>(Gr + idx);
            gv[0] = x.x; gv[1] = x.y; gv[2] = x.z; gv[3] = x.w;
          } else {
            for (int q = 0; q < 4; ++q) if (col + q < P.N) gv[q] = Gr[idx + q];
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (col + q >= P.N) continue;
            const float mag = ivr ? 1.f / ivr[(col + q) / U.B] - U.decomp_eps : 1.f;
            const double rec = (double)mag * (double)v[q], g = (double)gv[q];
            s_gr += g * rec;
            s_rr += rec * rec;
            s_gg += g * g;
          }
        } else if constexpr (EP == EP_ADAM) {
          if (U.moment_bf16) {   // moments stored in bf16: element by element (fallback shapes only)
            bf16* E1 = reinterpret_cast<bf16*>(P.e1);
            bf16* E2 = reinterpret_cast<bf16*>(P.e2);
            for (int q = 0; q < 4; ++q) {
              if (col + q >= P.N) continue;
              bf16 a = E1[idx + q], b = E2[idx + q];
              const float o = adam_out_bf16(v[q], a, b, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2);
              E1[idx + q] = a;
              E2[idx + q] = b;
              if constexpr (KIND == KIND_BF16) ((bf16*)P.c)[(P.kp & 4) ? kp_index(row, col + q, P.M) : idx + q] = f2bf(o);
              else ((float*)P.c)[idx + q] = o;
            }
            continue;
          }
          float e[4], s2[4], o[4];
          const bool fm = (col + 4 <= P.N) && ((idx & 3) == 0);   // moments are library memory (aligned)
          if (fm) {
            const float4 a = *reinterpret_cast<const float4*>(P.e1 + idx);
            const float4 b = *reinterpret_cast<const float4*>(P.e2 + idx);
            e[0] = a.x; e[1] = a.y; e[2] = a.z; e[3] = a.w;
            s2[0] = b.x; s2[1] = b.y; s2[2] = b.z; s2[3] = b.w;
          } else {
            for (int q = 0; q < 4; ++q) {
              e[q] = (col + q < P.N) ? P.e1[idx + q] : 0.f;
              s2[q] = (col + q < P.N) ? P.e2[idx + q] : 0.f;
            }
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = adam_out(v[q], e[q], s2[q], U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2);
          if (fm) {
            *reinterpret_cast<float4*>(P.e1 + idx) = make_float4(e[0], e[1], e[2], e[3]);
            *reinterpret_cast<float4*>(P.e2 + idx) = make_float4(s2[0], s2[1], s2[2], s2[3]);
            if constexpr (KIND == KIND_BF16) {
              bf16x4 t;
              t[0] = f2bf(o[0]); t[1] = f2bf(o[1]); t[2] = f2bf(o[2]); t[3] = f2bf(o[3]);
              *reinterpret_cast<bf16x4*>((bf16*)P.c + ((P.kp & 4) ? kp_index(row, col, P.M) : idx)) = t;
            } else {
              *reinterpret_cast<float4*>((float*)P.c + idx) = make_float4(o[0], o[1], o[2], o[3]);
            }
          } else {
            for (int q = 0; q < 4; ++q) {
              if (col + q >= P.N) continue;
              P.e1[idx + q] = e[q];
              P.e2[idx + q] = s2[q];
              if constexpr (KIND == KIND_BF16) ((bf16*)P.c)[(P.kp & 4) ? kp_index(row, col + q, P.M) : idx + q] = f2bf(o[q]);
              else ((float*)P.c)[idx + q] = o[q];
            }
          }
        } else {  // EP_UPDATE: W -= lr * scale * dM[row][col/B] * dV
          float mag[4];
          const float* dmr = P.dM ? P.dM + row * P.dM_ld : nullptr;
          if (!dmr) {
            mag[0] = mag[1] = mag[2] = mag[3] = 1.f;
          } else if ((U.B & 3) == 0) {
            mag[0] = mag[1] = mag[2] = mag[3] = dmr[col / U.B];
          } else {
            for (int q = 0; q < 4; ++q) mag[q] = (col + q < P.N) ? dmr[(col + q) / U.B] : 1.f;
          }
          float wv[4] = {0.f, 0.f, 0.f, 0.f};
          if (U.weight_bf16) {
            const bf16* Wr = (const bf16*)P.c;
            if (full) {
              const bf16x4 x = *reinterpret_cast<const bf16x4*>(Wr + idx);
              wv[0] = bf2f(x[0]); wv[1] = bf2f(x[1]); wv[2] = bf2f(x[2]); wv[3] = bf2f(x[3]);
            } else {
              for (int q = 0; q < 4; ++q) if (col + q < P.N) wv[q] = bf2f(Wr[idx + q]);
            }
          } else {
            const float* Wr = (const float*)P.c;
            if (full) {
              const float4 x = *reinterpret_cast<const float4*>(Wr + idx);
              wv[0] = x.x; wv[1] = x.y; wv[2] = x.z; wv[3] = x.w;
            } else {
              for (int q = 0; q < 4; ++q) if (col + q < P.N) wv[q] = Wr[idx + q];
            }
          }
          if (U.weight_bf16) {
            bf16* W = (bf16*)P.c;
            float nw[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) nw[q] = wv[q] - U.lr * bf2f(f2bf(U.scale * (mag[q] * v[q])));
            if (full) {
              bf16x4 t;
              t[0] = f2bf(nw[0]); t[1] = f2bf(nw[1]); t[2] = f2bf(nw[2]); t[3] = f2bf(nw[3]);
              *reinterpret_cast<bf16x4*>(W + idx) = t;
            } else {
              for (int q = 0; q < 4; ++q) if (col + q < P.N) W[idx + q] = f2bf(nw[q]);
            }
          } else {
            float* W = (float*)P.c;
            float nw[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) nw[q] = wv[q] - U.lr * (U.scale * (mag[q] * v[q]));
            if (full) *reinterpret_cast<float4*>(W + idx) = make_float4(nw[0], nw[1], nw[2], nw[3]);
            else
              for (int q = 0; q < 4; ++q) if (col + q < P.N) W[idx + q] = nw[q];
          }
        }
      }
  }
  if constexpr (EP == EP_ALIGN) {   // wave sums (fixed butterfly), one atomic per sum and wave
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      s_gr += __shfl_xor(s_gr, o, 64);
      s_rr += __shfl_xor(s_rr, o, 64);
      s_gg += __shfl_xor(s_gg, o, 64);
    }
    if (lane == 0) {
      atomicAdd(P.red + 0, s_gr);
      atomicAdd(P.red + 1, s_rr);
      atomicAdd(P.red + 2, s_gg);
    }
  }
}

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mi][ni][j] = 0.f;
}

// ------------------------------------------------------------------ kernels
template <int AM, int BWM, int BWN, bool PD2, bool FAST>
__device__ __forceinline__ void mainloop_bf16(const GemmProb& P, const GemmUniform& U, int64_t row0, int64_t col0,
                                              bf16 (*As)[64 * BWM * BF_LD], bf16 (*Bs)[64 * BWN * BF_LD],
                                              f32x16 (&acc)[2][2]) {
  constexpr int BK = 64;
  constexpr int BNT = 64 * BWM * BWN;
  constexpr int BBM = 64 * BWM, BBN = 64 * BWN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / BWN, wn = wave % BWN;
  const Rs R = make_rs(P);
  const int nk = (int)((P.K + BK - 1) / BK);
  auto compute = [&](const bf16* Ac, const bf16* Bc) {
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[2], bv[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        af[mi] = *reinterpret_cast<const bf16x8*>(Ac + (wm * 64 + mi * 32 + (lane & 31)) * BF_LD + kk * 16 + (lane >> 5) * 8);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bv[ni] = *reinterpret_cast<const bf16x8*>(Bc + (wn * 64 + ni * 32 + (lane & 31)) * BF_LD + kk * 16 + (lane >> 5) * 8);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[ni], af[mi], acc[mi][ni], 0, 0, 0);
    }
  };
  if constexpr (PD2) {
    BfA<AM, BBM, BNT, FAST> ra0, ra1;
    BfB<BBN, BNT, FAST> rb0, rb1;
    ra0.load(P, R, row0, 0, U.B);
    rb0.load(P, R, col0, 0);
    if (nk > 1) { ra1.load(P, R, row0, BK, U.B); rb1.load(P, R, col0, BK); }
    ra0.store(P, row0, 0, U.B, As[0]);
    rb0.store(P, 0, Bs[0]);
    __syncthreads();
    if (nk > 2) { ra0.load(P, R, row0, 2 * BK, U.B); rb0.load(P, R, col0, 2 * BK); }
    for (int kt = 0; kt < nk; kt += 2) {
      // even: tile kt in stage 0; register set 1 holds tile kt+1, set 0 holds tile kt+2
      compute(As[0], Bs[0]);
      if (kt + 1 < nk) { ra1.store(P, row0, (int64_t)(kt + 1) * BK, U.B, As[1]); rb1.store(P, (int64_t)(kt + 1) * BK, Bs[1]); }
      __syncthreads();
      if (kt + 3 < nk) { ra1.load(P, R, row0, (int64_t)(kt + 3) * BK, U.B); rb1.load(P, R, col0, (int64_t)(kt + 3) * BK); }
      if (kt + 1 >= nk) break;
      // odd: tile kt+1 in stage 1; set 0 holds tile kt+2, set 1 holds tile kt+3
      compute(As[1], Bs[1]);
      if (kt + 2 < nk) { ra0.store(P, row0, (int64_t)(kt + 2) * BK, U.B, As[0]); rb0.store(P, (int64_t)(kt + 2) * BK, Bs[0]); }
      __syncthreads();
      if (kt + 4 < nk) { ra0.load(P, R, row0, (int64_t)(kt + 4) * BK, U.B); rb0.load(P, R, col0, (int64_t)(kt + 4) * BK); }
    }
  } else {
    BfA<AM, BBM, BNT, FAST> ra;
    BfB<BBN, BNT, FAST> rb;
    ra.load(P, R, row0, 0, U.B);
    rb.load(P, R, col0, 0);
    ra.store(P, row0, 0, U.B, As[0]);
    rb.store(P, 0, Bs[0]);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      const int64_t kn = (int64_t)(kt + 1) * BK;
      if (more) { ra.load(P, R, row0, kn, U.B); rb.load(P, R, col0, kn); }
      compute(As[cur], Bs[cur]);
      if (more) { ra.store(P, row0, kn, U.B, As[cur ^ 1]); rb.store(P, kn, Bs[cur ^ 1]); }
      __syncthreads();
    }
  }
}

template <int AM, int EP, int BWM, int BWN, bool PD2>
__global__ __launch_bounds__(64 * BWM * BWN, 2) void k_gemm_bf16(const GemmProb* __restrict__ probs, GemmUniform U) {
  constexpr int BBM = 64 * BWM, BBN = 64 * BWN;
  __shared__ __attribute__((aligned(16))) bf16 As[2][BBM * BF_LD];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BBN * BF_LD];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const GemmProb& P = probs[find_prob(probs, U.nprob, t)];
  uint32_t tm, tn;
  tile_coords(t - P.tile_start, (uint32_t)((P.M + BBM - 1) / BBM), P.tiles_n, tm, tn);
  const int64_t row0 = (int64_t)tm * BBM, col0 = (int64_t)tn * BBN;
  f32x16 acc[2][2];
  zero_acc(acc);
  if (P.vec & 4) mainloop_bf16<AM, BWM, BWN, PD2, true>(P, U, row0, col0, As, Bs, acc);
  else mainloop_bf16<AM, BWM, BWN, false, false>(P, U, row0, col0, As, Bs, acc);
  epilogue<KIND_BF16, EP, BWN>(P, U, row0, col0, acc);
}

template <int AM, int BMODE, bool FAST>
__device__ __forceinline__ void mainloop_f32(const GemmProb& P, const GemmUniform& U, int64_t row0, int64_t col0,
                                             float (*As)[(AM == A_G_TRANS) ? 32 * F_LDT : 128 * F_LDK],
                                             float (*Bs)[(BMODE == B_NC) ? 32 * F_LDT : 128 * F_LDK],
                                             f32x16 (&acc)[2][2]) {
  constexpr int BK = 32;
  constexpr bool AT = (AM == A_G_TRANS);
  constexpr bool BT = (BMODE == B_NC);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const Rs R = make_rs(P);
  FA<AM, FAST> ra;
  FB<BMODE, FAST> rb;
  // an upper triangular right factor contributes nothing past the tile's last column
  const int64_t kend = (P.tri_b && col0 + 128 < P.K) ? col0 + 128 : P.K;
  const int nk = (int)((kend + BK - 1) / BK);
  auto compute = [&](const float* Ac, const float* Bc) {
#pragma unroll
    for (int kk = 0; kk < BK / 2; ++kk) {
      const int kx = kk * 2 + (lane >> 5);
      float af[2], bv[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int i = wm * 64 + mi * 32 + (lane & 31);
        af[mi] = AT ? Ac[kx * F_LDT + i] : Ac[i * F_LDK + kx];
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int j = wn * 64 + ni * 32 + (lane & 31);
        bv[ni] = BT ? Bc[kx * F_LDT + j] : Bc[j * F_LDK + kx];
      }
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(bv[ni], af[mi], acc[mi][ni], 0, 0, 0);
    }
  };
  ra.load(P, R, row0, 0, U.B);
  rb.load(P, R, col0, 0);
  ra.store(P, row0, 0, U.B, As[0]);
  rb.store(P, col0, 0, Bs[0]);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    const int64_t kn = (int64_t)(kt + 1) * BK;
    if (more) { ra.load(P, R, row0, kn, U.B); rb.load(P, R, col0, kn); }
    compute(As[cur], Bs[cur]);
    if (more) { ra.store(P, row0, kn, U.B, As[cur ^ 1]); rb.store(P, col0, kn, Bs[cur ^ 1]); }
    __syncthreads();
  }
}

template <int AM, int BMODE, int EP>
__global__ __launch_bounds__(FNT, 2) void k_gemm_f32(const GemmProb* __restrict__ probs, GemmUniform U) {
  constexpr int BM = 128, BN = 128, BK = 32;
  constexpr bool AT = (AM == A_G_TRANS);
  constexpr bool BT = (BMODE == B_NC);
  __shared__ __attribute__((aligned(16))) float As[2][AT ? BK * F_LDT : BM * F_LDK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BT ? BK * F_LDT : BN * F_LDK];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const GemmProb& P = probs[find_prob(probs, U.nprob, t)];
  uint32_t tm, tn;
  tile_coords(t - P.tile_start, (uint32_t)((P.M + BM - 1) / BM), P.tiles_n, tm, tn);
  const int64_t row0 = (int64_t)tm * BM, col0 = (int64_t)tn * BN;
  f32x16 acc[2][2];
  zero_acc(acc);
  if (P.vec & 4) mainloop_f32<AM, BMODE, true>(P, U, row0, col0, As, Bs, acc);
  else mainloop_f32<AM, BMODE, false>(P, U, row0, col0, As, Bs, acc);
  epilogue<KIND_F32, EP, 2>(P, U, row0, col0, acc);
}

}  // namespace

uint32_t gemm_tiles_m(int kind, int64_t M) {
  (void)kind;
  return (uint32_t)((M + 127) / 128);
}
uint32_t gemm_tiles_n(int kind, int64_t N) {
  (void)kind;
  return (uint32_t)((N + 127) / 128);
}

#define GEMM_BF(AM, EP)                                                                  \
  if (amode == AM && ep == EP) {                                                       \
    hipLaunchKernelGGL((k_gemm_bf16<AM, EP, 2, 2, AM == A_KC>), grid, dim3(256), 0, st, probs_dev, u); \
    return hipGetLastError();                                                          \
  }
#define GEMM_F(AM, BMO, EP) \
  if (amode == AM && bmode == BMO && ep == EP) { hipLaunchKernelGGL((k_gemm_f32<AM, BMO, EP>), grid, dim3(FNT), 0, st, probs_dev, u); return hipGetLastError(); }

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
    GEMM_F(A_KC, B_KC, EP_STORE)
    GEMM_F(A_KC, B_KC, EP_ALIGN)
    GEMM_F(A_G_ROW, B_NC, EP_STORE)
    GEMM_F(A_G_TRANS, B_NC, EP_STORE)
    GEMM_F(A_KC, B_NC, EP_STORE)
  }
  return hipErrorInvalidValue;
}
