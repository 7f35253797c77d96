// Block-wise magnitude/direction decomposition (Section 3.1, Appendix B.1)
// fused with Optimizer_M (Adam on the block magnitudes, Algorithm 1).
//
// For every row i and block j (columns [jB, min(jB+B, n)) -- the zero padding of
// the last block contributes nothing to the norm):
//   M[i,j]   = ||G[i, block j]||_2
//   inv[i,j] = 1 / (M[i,j] + eps_d)        (V = G * inv is formed on the fly by the GEMMs)
//   dM[i,j]  = Adam(M[i,j])                (when p.adam_m != 0)
//
// Memory-bound: reads G once (4 B/element), writes 4 (inv, dM, two moments)
// and reads 2 fp32 values per block. A block of B <= 256 columns maps onto B/4
// consecutive lanes and is reduced with xor shuffles inside that lane group
// (fixed order, so results are bit-reproducible; the butterfly leaves the same
// sum in every lane of the group). Other block sizes take a generic per-block
// path.
//
// When the step's GEMMs take bf16 operands, the same pass also writes the
// direction tensor V = G * inv in bf16 (2 B/element), oriented so that the
// projection's reduction index runs along its rows (m x n for a RIGHT projection
// V Q, transposed n x m for a LEFT one P^T V) and stored in the blocked K-panel
// layout of the large-tile GEMM (kp_index). The transposed form comes from
// k_decompose_vt, which stages a 32-row x 256-column slab in LDS.
#include "common.h"

namespace {
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
constexpr int DEC_ROWS = 16;   // rows per workgroup (4 waves x 4 rows)

// Sum over aligned groups of gl lanes (gl a power of two <= 64). The first four
// levels use DPP lane permutations (pairs within a quad, then the two quads of an
// 8-lane half-row, then the two halves of a 16-lane row: mirror permutations pair
// lanes whose values are already equal to their group's partial sum), the fifth a
// ds_swizzle xor 16, the sixth a cross-half shuffle. Each level adds two equal
// partial sums in either order, so every lane of a group ends with the same,
// bit-identical total.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float group_sum(float v, int gl) {
  if (gl >= 2) v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
  if (gl >= 4) v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
  if (gl >= 8) v += dpp_f<0x141>(v);   // row_half_mirror
  if (gl >= 16) v += dpp_f<0x140>(v);  // row_mirror
  if (gl >= 32) v += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));   // lane ^ 16
  if (gl >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}

__device__ __forceinline__ void block_out(const MatDev& d, const StepParams& p, int64_t row, int j,
                                          float ss, int adam_m) {
  const float M = sqrtf(ss);
  const int64_t idx = row * d.k + j;
  d.inv[idx] = 1.0f / (M + p.decomp_eps);
  if (adam_m) {
    float e = d.mag1[idx], q = d.mag2[idx];
    const float out = adam_out(M, e, q, p.beta1, p.beta2, p.adam_eps, d.bc1, d.bc2);
    d.mag1[idx] = e;
    d.mag2[idx] = q;
    d.dM[idx] = out;
  }
}

// Phase 1: the block sums of squares of the workgroup's DEC_ROWS rows go to LDS
// (each wave streams one row at a time with UNR 16-byte loads in flight).
// Phase 2: all threads run Optimizer_M over those DEC_ROWS * k blocks, which are
// contiguous in the m x k layout, so the moment/inv/dM traffic is coalesced.
constexpr int DEC_LDS = 8192;   // floats of LDS for block sums (phase 1 -> 2)

__global__ __launch_bounds__(256) void k_decompose(const MatDev* __restrict__ mats, StepParams p, int adam_m) {
  __shared__ float sums[DEC_LDS];
  const uint32_t t = blockIdx.x;
  const int mi = find_mat(mats, p.nmat, t, [](const MatDev& d) { return d.tile_dec; });
  const MatDev d = mats[mi];
  const int64_t row0 = (int64_t)(t - d.tile_dec) * DEC_ROWS;
  const int rows = (int)((d.m - row0 < DEC_ROWS) ? d.m - row0 : DEC_ROWS);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int B = p.B;
  const int64_t n = d.n;
  const int k = d.k;
  const bool staged = (int64_t)rows * k <= DEC_LDS;
  const bool fast = staged && B >= 4 && B <= 256 && (B & (B - 1)) == 0 && (n & 3) == 0 &&
                    ((uintptr_t)d.G & 15) == 0;
  if (!staged) {
    // generic path (very many blocks per row): one block at a time, Optimizer_M inline
    for (int rr = wave; rr < rows; rr += 4) {
      const int64_t row = row0 + rr;
      const float* g = d.G + row * n;
      for (int j = 0; j < k; ++j) {
        const int64_t cs = (int64_t)j * B;
        const int64_t ce = (cs + B < n) ? cs + B : n;
        float ss = 0.f;
        for (int64_t c = cs + lane; c < ce; c += 64) { const float v = g[c]; ss += v * v; }
        ss = wave_sum(ss);
        if (lane == 0) block_out(d, p, row, j, ss, adam_m);
      }
    }
    return;
  }
  if (fast && B <= 128) {
    // Row pairs: the two half-waves take rows 2p and 2p + 1 (blocks of B <= 128 columns
    // stay inside a half-wave), so that each bf16 store of V covers both rows of a
    // 32-column block, i.e. whole 128-byte lines of the blocked layout.
    constexpr int UNR = 8;
    const int gl = B >> 2;   // lanes per block
    const int lgB = __builtin_ctz(B);
    const int hl = lane & 31;
    for (int rp = wave; 2 * rp < rows; rp += 4) {
      const int rr = 2 * rp + (lane >> 5);
      const bool rok = rr < rows;
      const int64_t row = row0 + rr;
      const float* g = d.G + row * n;
      for (int64_t c00 = 0; c00 < n; c00 += 128 * UNR) {
        float4 v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int64_t c = c00 + 128 * u + 4 * hl;
          v[u] = (rok && c < n) ? *reinterpret_cast<const float4*>(g + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int64_t c = c00 + 128 * u + 4 * hl;
          float ss = v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
          ss = group_sum(ss, gl);
          if (rok && c < n) {
            if ((hl & (gl - 1)) == 0) sums[rr * k + (int)(c >> lgB)] = ss;
            if (d.Vb) {
              const float inv = 1.0f / (sqrtf(ss) + p.decomp_eps);
              bf16x4 o;
              o[0] = f2bf(v[u].x * inv); o[1] = f2bf(v[u].y * inv); o[2] = f2bf(v[u].z * inv); o[3] = f2bf(v[u].w * inv);
              *reinterpret_cast<bf16x4*>(d.Vb + kp_index(row, c, d.m)) = o;   // blocked, K = n
            }
          }
        }
      }
    }
  } else
  for (int rr = wave; rr < rows; rr += 4) {
    const int64_t row = row0 + rr;
    const float* g = d.G + row * n;
    if (fast) {
      constexpr int UNR = 8;
      const int gl = B >> 2;   // lanes per block
      const int lgB = __builtin_ctz(B);
      for (int64_t c00 = 0; c00 < n; c00 += 256 * UNR) {
        float4 v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int64_t c = c00 + 256 * u + 4 * lane;
          v[u] = (c < n) ? *reinterpret_cast<const float4*>(g + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const int64_t c = c00 + 256 * u + 4 * lane;
          float ss = v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
          ss = group_sum(ss, gl);
          if ((lane & (gl - 1)) == 0 && c < n) sums[rr * k + (int)(c >> lgB)] = ss;
          if (d.Vb && c < n) {
            const float inv = 1.0f / (sqrtf(ss) + p.decomp_eps);
            bf16x4 o;
            o[0] = f2bf(v[u].x * inv); o[1] = f2bf(v[u].y * inv); o[2] = f2bf(v[u].z * inv); o[3] = f2bf(v[u].w * inv);
            *reinterpret_cast<bf16x4*>(d.Vb + kp_index(row, c, d.m)) = o;   // blocked, K = n
          }
        }
      }
    } else {
      for (int j = 0; j < k; ++j) {
        const int64_t cs = (int64_t)j * B;
        const int64_t ce = (cs + B < n) ? cs + B : n;
        float ss = 0.f;
        for (int64_t c = cs + lane; c < ce; c += 64) { const float v = g[c]; ss += v * v; }
        ss = wave_sum(ss);
        if (lane == 0) sums[rr * k + j] = ss;
      }
    }
  }
  __syncthreads();
  const int total = rows * k;
  for (int e = threadIdx.x; e < total; e += 256) {
    const int rr = e / k, j = e - (e / k) * k;
    block_out(d, p, row0 + rr, j, sums[e], adam_m);
  }
}

// Transposed-V variant (LEFT projections): one workgroup per VT_ROWS (32) rows. For each
// 256-column slab every wave loads VT_RPW of the rows (float4 per lane, all in
// flight), reduces the block sums, writes V in bf16 into an LDS slab
// T[VT_ROWS][256] (row-major, conflict-free 4-byte stores) and records the sums; the
// slab is then written out transposed, VT_ROWS / 8 lanes per output column (16 bytes
// each), i.e. 64-byte (one K panel) segments of Vt. The odd 4-byte pitch of T keeps the
// row groups read by one instruction on distinct banks. Optimizer_M then runs over the
// VT_ROWS x k sums as in k_decompose. 32-row slabs (143 VGPRs, three waves per SIMD)
// measured 1.7 % faster than 64-row ones (231 VGPRs, two). Preconditions (checked by
// the host): B a power of two in [4, 256], n % 4 == 0, m % 32 == 0, k <= DEC_VT_MAX_K,
// G 16-byte aligned.
#ifndef DEC_VT_ROWS
#define DEC_VT_ROWS 32
#endif
constexpr int VT_ROWS = DEC_VT_ROWS, VT_COLS = 256, VT_PITCH = VT_COLS + 2;   // bf16 elements
constexpr int VT_RPW = VT_ROWS / 4;    // rows per wave
constexpr int VT_GRP = VT_ROWS / 8;    // 8-row groups of a column (16-byte output runs)
static_assert(VT_ROWS % 32 == 0, "whole 32-row K panels of the blocked output");

__global__ __launch_bounds__(256) void k_decompose_vt(const MatDev* __restrict__ mats, StepParams p, int adam_m) {
  __shared__ float sums[VT_ROWS * DEC_VT_MAX_K];
  __shared__ __attribute__((aligned(16))) bf16 T[VT_ROWS * VT_PITCH];
  const uint32_t t = blockIdx.x;
  const int mi = find_mat(mats, p.nmat, t, [](const MatDev& d) { return d.tile_dec; });
  const MatDev d = mats[mi];
  const int64_t row0 = (int64_t)(t - d.tile_dec) * VT_ROWS;
  const int rows = (int)((d.m - row0 < VT_ROWS) ? d.m - row0 : VT_ROWS);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int B = p.B, gl = B >> 2, k = d.k, lgB = __builtin_ctz(B);
  const int64_t n = d.n, m = d.m;
  // the slab loop is software-pipelined: the VT_RPW loads of the next slab are issued
  // before the current slab is reduced, transposed and written out
  float4 va[VT_RPW], vb[VT_RPW];
  auto load = [&](int64_t c0, float4 (&v)[VT_RPW]) {
    const int64_t c = c0 + 4 * lane;
#pragma unroll
    for (int i = 0; i < VT_RPW; ++i) {
      const int rr = wave + 4 * i;
      v[i] = (rr < rows && c < n) ? *reinterpret_cast<const float4*>(d.G + (row0 + rr) * n + c)
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto process = [&](int64_t c0, const float4 (&v)[VT_RPW]) {
    const int64_t c = c0 + 4 * lane;
#pragma unroll
    for (int i = 0; i < VT_RPW; ++i) {
      const int rr = wave + 4 * i;
      float ss = v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
      ss = group_sum(ss, gl);
      if (rr < rows && c < n && (lane & (gl - 1)) == 0) sums[rr * k + (int)(c >> lgB)] = ss;
      const float inv = 1.0f / (sqrtf(ss) + p.decomp_eps);
      bf16x2 a, b;
      a[0] = f2bf(v[i].x * inv); a[1] = f2bf(v[i].y * inv);
      b[0] = f2bf(v[i].z * inv); b[1] = f2bf(v[i].w * inv);
      *reinterpret_cast<bf16x2*>(T + rr * VT_PITCH + 4 * lane) = a;
      *reinterpret_cast<bf16x2*>(T + rr * VT_PITCH + 4 * lane + 2) = b;
    }
    __syncthreads();
#pragma unroll 2
    for (int it = 0; it < VT_GRP; ++it) {
      const int q = it * 256 + (int)threadIdx.x;
      const int cl = q / VT_GRP, g = q % VT_GRP;
      const int64_t col = c0 + cl;
      if (col < n && 8 * g < rows) {
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = T[(8 * g + e) * VT_PITCH + cl];
        *reinterpret_cast<bf16x8*>(d.Vb + kp_index(col, row0 + 8 * g, n)) = o;   // blocked V' (n x m), K = m
      }
    }
    __syncthreads();
  };
  load(0, va);
  for (int64_t c0 = 0; c0 < n; c0 += 2 * VT_COLS) {
    if (c0 + VT_COLS < n) load(c0 + VT_COLS, vb);
    process(c0, va);
    if (c0 + VT_COLS >= n) break;
    if (c0 + 2 * VT_COLS < n) load(c0 + 2 * VT_COLS, va);
    process(c0 + VT_COLS, vb);
  }
  const int total = rows * k;
  for (int e = threadIdx.x; e < total; e += 256) {
    const int rr = e / k, j = e - (e / k) * k;
    block_out(d, p, row0 + rr, j, sums[e], adam_m);
  }
}
// A zero gradient gives M = 0, V = 0 and R = P^T V = 0 (Algorithm 1 with G = 0), so the
// step reduces to decaying the moments: Optimizer_M on M = 0 and Optimizer_V on R = 0,
// through the same adam_out as the decomposition and the projection epilogue (bit for
// bit what those kernels produce from an all-zero G). Elements [0, m k) of a matrix are
// its magnitude blocks (only when the decomposition is on), the next L r its direction
// moments; ZG_PER_WG elements per workgroup, consecutive threads on consecutive elements.
constexpr int ZG_PER_WG = 2048;
__global__ __launch_bounds__(256) void k_zero_grad(const MatDev* __restrict__ mats, StepParams p) {
  const uint32_t t = blockIdx.x;
  const MatDev& d = mats[find_mat(mats, p.nmat, t, [](const MatDev& x) { return x.tile_dec; })];
  const int64_t mk = p.decompose ? d.m * d.k : 0;
  const int64_t Lr = (int64_t)d.L * d.r;
  const int64_t e0 = (int64_t)(t - d.tile_dec) * ZG_PER_WG;
  for (int64_t e = e0 + threadIdx.x; e < e0 + ZG_PER_WG && e < mk + Lr; e += 256) {
    if (e < mk) {
      float a = d.mag1[e], q = d.mag2[e];
      const float out = adam_out(0.f, a, q, p.beta1, p.beta2, p.adam_eps, d.bc1, d.bc2);
      d.mag1[e] = a;
      d.mag2[e] = q;
      d.dM[e] = out;
    } else {
      const int64_t x = e - mk;   // (l, j) of the L x r moments, row-major
      float out;
      if (d.mom_bf16) {
        bf16* E1 = reinterpret_cast<bf16*>(d.exp1);
        bf16* E2 = reinterpret_cast<bf16*>(d.exp2);
        bf16 a = E1[x], q = E2[x];
        out = adam_out_bf16(0.f, a, q, p.beta1, p.beta2, p.adam_eps, d.bc1, d.bc2);
        E1[x] = a;
        E2[x] = q;
      } else {
        float a = d.exp1[x], q = d.exp2[x];
        out = adam_out(0.f, a, q, p.beta1, p.beta2, p.adam_eps, d.bc1, d.bc2);
        d.exp1[x] = a;
        d.exp2[x] = q;
      }
      if (d.n_bf16) {
        const int64_t l = x / d.r, j = x % d.r;
        ((bf16*)d.N)[d.n_kp ? kp_index(l, j, d.L) : x] = f2bf(out);
      } else {
        ((float*)d.N)[x] = out;
      }
    }
  }
}
}  // namespace

uint32_t zero_grad_tiles(int64_t mk, int64_t Lr) { return (uint32_t)((mk + Lr + ZG_PER_WG - 1) / ZG_PER_WG); }

hipError_t launch_zero_grad(const MatDev* mats_dev, const StepParams& p, hipStream_t st) {
  if (p.total_dec == 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero_grad, dim3(p.total_dec), dim3(256), 0, st, mats_dev, p);
  return hipGetLastError();
}

int decompose_tiles(int64_t m) { return (int)((m + DEC_ROWS - 1) / DEC_ROWS); }
int decompose_vt_tiles(int64_t m) { return (int)((m + VT_ROWS - 1) / VT_ROWS); }

hipError_t launch_decompose_vt(const MatDev* mats_dev, const StepParams& p, int adam_m, hipStream_t st) {
  if (p.total_dec == 0) return hipSuccess;
  hipLaunchKernelGGL(k_decompose_vt, dim3(p.total_dec), dim3(256), 0, st, mats_dev, p, adam_m);
  return hipGetLastError();
}

hipError_t launch_decompose(const MatDev* mats_dev, const StepParams& p, hipStream_t st) {
  if (p.total_dec == 0) return hipSuccess;
  hipLaunchKernelGGL(k_decompose, dim3(p.total_dec), dim3(256), 0, st, mats_dev, p, 1);
  return hipGetLastError();
}

hipError_t launch_decompose_inv_only(const MatDev* mats_dev, const StepParams& p, hipStream_t st) {
  if (p.total_dec == 0) return hipSuccess;
  hipLaunchKernelGGL(k_decompose, dim3(p.total_dec), dim3(256), 0, st, mats_dev, p, 0);
  return hipGetLastError();
}
