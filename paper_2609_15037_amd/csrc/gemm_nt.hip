// Large-tile bf16 GEMM for the step's projection and back-projection, used when
// both operands are bf16, contiguous along the reduction index and K is a
// multiple of 32:
//
//   C[M x N] = sum_k A[i][k] * B[j][k]     (A: M x K, B: N x K, both row-major)
//
// Default configuration: workgroup tile 256 x 256, sixteen waves (4 along M x 4 along
// N), each wave a 64 x 64 sub-tile of 2 x 2 v_mfma_f32_32x32x16_bf16 blocks (64 fp32
// accumulators per lane), one workgroup per CU. K advances in steps of 32 through a
// ring of LDS stages (32 KB each: four for the step's products, five for the refresh's
// plain-store products) filled by direct global->LDS buffer loads (no register
// staging), the stages ahead of the one being multiplied in flight, one barrier per
// step. Operands may be row-major or in the blocked K-panel layout (kp_index), where
// one K step of the tile's rows is a contiguous run and the DMA loads move whole lines.
// Each 64-byte tile row holds four 16-byte chunks stored at chunk ^ f(row),
// f(row) = ((row >> 1) & 3) ^ ((row >> 3) & 1), so that the 16-byte fragment reads of
// 8- and 16-lane groups hit distinct banks; the lane -> global address map of the DMA
// loads applies the same permutation. Rows past M (N) re-read the last valid row and
// are never stored.
//
// The MFMA is issued as C^T = B A^T: lane l of block (mb, nb), register j holds
//   row = 32 mb + (l & 31), col = 32 nb + 8 (j / 4) + 4 (l / 32) + (j % 4)
// of the wave's sub-tile. The epilogues stage each 32-row slab of the wave's
// accumulators through LDS and then walk it row-contiguously, so that moments,
// N and W move as full 128-byte row segments.
//   EP_ADAM  : Optimizer_V on the projected tile (moments e1/e2, output N bf16);
//              EP_ADAM_B16 the same with the moments stored in bf16 (half the moment traffic).
//   EP_UPDATE: W[i][j] -= lr * bf16(scale * dM[i][j/B] * C[i][j]) (bf16 or fp32 W).
//   EP_STORE / EP_STORE_BF16: C stored as fp32 / bf16 (the refresh's subspace products).
#include "gemm.h"

#ifndef EPDB_ADAM
#define EPDB_ADAM 4
#endif
#ifndef EPA_ROWS
#define EPA_ROWS 4
#endif
#ifndef EPDB_ADAM16
#define EPDB_ADAM16 4
#endif
#ifndef EPDB_UPD
#define EPDB_UPD 1
#endif

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int TBM = 256, TBK = 32;
constexpr int ROWB = TBK * 2;          // bytes per tile row per stage
constexpr int TILEA = TBM * ROWB;      // 16 KB of A per stage

__device__ __forceinline__ int swz(int R) { return ((R >> 1) & 3) ^ ((R >> 3) & 1); }

// s_waitcnt vmcnt(n), n in [0, 15] (larger n waits for 15); expcnt and lgkmcnt are
// left at their maxima (vmcnt occupies bits 3:0 of the immediate)
__device__ __forceinline__ void wait_vm(int n) {
#define WVM(k) case k: __builtin_amdgcn_s_waitcnt(0x0F70 | k); break;
  switch (n) {
    WVM(0) WVM(1) WVM(2) WVM(3) WVM(4) WVM(5) WVM(6) WVM(7)
    WVM(8) WVM(9) WVM(10) WVM(11) WVM(12) WVM(13) WVM(14)
    default: __builtin_amdgcn_s_waitcnt(0x0F7F); break;
  }
#undef WVM
}

// Workgroup barrier for the stage ring: each wave has already waited (vmcnt) for its
// own DMA loads of the stage about to be read, so the barrier needs no fence; the
// empty asm keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int find_prob(const GemmProb* probs, int n, uint32_t t) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].tile_start <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// NWM x NWN waves, each owning a WTM x WTN sub-tile (WTM/32 x WTN/32 MFMA blocks);
// the tile is 256 x (NWN WTN) (NWM WTM = 256); NS LDS stages; OCC workgroups per CU
// (the second launch bound is the minimum number of waves per SIMD).
template <int EP, int NWM, int NWN, int WTN, int NS, int OCC>
__global__ __launch_bounds__(64 * NWM * NWN, (OCC * NWM * NWN + 3) / 4) void k_gemm_nt(const GemmProb* __restrict__ probs, GemmUniform U) {
  constexpr int NW = NWM * NWN, TBN = NWN * WTN, NB = WTN / 32;
  constexpr int WTM = TBM / NWM, MB = WTM / 32;
  static_assert(NWM * WTM == TBM && MB >= 2 && MB <= 4 && NB <= 4, "wave layout");
  constexpr int EPLD = WTN + 4;                      // fp32 row stride of the epilogue staging slab
  constexpr int EPWAVE = 32 * EPLD;                  // floats per wave slab
  constexpr int TILEB = TBN * ROWB, STAGEB = TILEA + TILEB;
  constexpr int SA = 16 / NW, SB = (TBN / 16) / NW;   // 1 KB DMA slots per wave per stage
  constexpr int OPS = SA + SB;                        // DMA instructions per wave per stage
  constexpr int SMEM = NS * STAGEB > NW * EPWAVE * 4 ? NS * STAGEB : NW * EPWAVE * 4;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const uint32_t t = xcd_remap(blockIdx.x, gridDim.x);
  const GemmProb& P = probs[find_prob(probs, U.nprob, t)];
  uint32_t tm, tn;
  // the projection walks two tile rows per group (measured 1.6 % faster than eight on the
  // 7B step; its N is only r / 256 tiles wide), the other products eight
  tile_coords(t - P.tile_start, (uint32_t)((P.M + TBM - 1) / TBM), P.tiles_n, tm, tn,
              (EP == EP_ADAM || EP == EP_ADAM_B16) ? 2u : (uint32_t)GM);
  const int64_t row0 = (int64_t)tm * TBM, col0 = (int64_t)tn * TBN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave % NWM, wn = wave / NWM;

  // ---- DMA address map: wave w fills 1 KB slots [SA w, SA w + SA) of the A tile and
  // [SB w, SB w + SB) of the B tile (16 rows per slot)
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)P.a, (short)0, (int)P.a_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc((void*)P.b, (short)0, (int)P.b_bytes, 0x00020000);
  // K segments (split operands): the refresh's plain-store products only
  constexpr bool SEGS = EP == EP_STORE || EP == EP_STORE_BF16;
  // K steps of one segment; a left factor that is zero above its diagonal ends the K
  // loop of a tile at the tile's last row
  const int nk1 = (SEGS && P.tri_b == 2) ? min((int)(P.K / TBK), (int)((row0 + TBM) / TBK)) : (int)(P.K / TBK);
  static_assert(SA <= 4 && SB <= 4, "DMA slot arrays");
  // blocked operands: one K step of the tile's rows is a contiguous 64-byte-per-row run,
  // the next K step starts rows * 64 bytes further; row-major: the next 64 bytes of each row
  const bool kpa = P.kp & 1, kpb = P.kp & 2;
  const uint32_t sta = kpa ? (uint32_t)P.M * 64u : (uint32_t)(TBK * 2);
  const uint32_t stb = kpb ? (uint32_t)P.N * 64u : (uint32_t)(TBK * 2);
  uint32_t va[4], vb[4];   // (fixed extent: a template-dependent array bound here drops the host launch stub)
#pragma unroll
  for (int j = 0; j < SA; ++j) {
    const int R = 16 * (SA * wave + j) + (lane >> 2);
    const int c = (lane & 3) ^ swz(R);
    const int64_t ga = (row0 + R < P.M) ? row0 + R : P.M - 1;
    va[j] = (uint32_t)((kpa ? ga * 64 : ga * P.lda * 2) + c * 16);
  }
#pragma unroll
  for (int j = 0; j < SB; ++j) {
    const int R = 16 * (SB * wave + j) + (lane >> 2);
    const int c = (lane & 3) ^ swz(R);
    const int64_t gb = (col0 + R < P.N) ? col0 + R : P.N - 1;
    vb[j] = (uint32_t)((kpb ? gb * 64 : gb * P.ldb * 2) + c * 16);
  }
  auto issue = [&](int kt, int slot) {
    char* base = smem + slot * STAGEB;
    if constexpr (!SEGS) {
      const int soa = (int)(kt * sta), sob = (int)(kt * stb);
#pragma unroll
      for (int j = 0; j < SA; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(base + (SA * wave + j) * 1024), 16, va[j], soa, 0, 0);
#pragma unroll
      for (int j = 0; j < SB; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(base + TILEA + (SB * wave + j) * 1024), 16, vb[j], sob, 0, 0);
    } else {
      int seg = 0, kk = kt;   // uniform
      while (kk >= nk1) { kk -= nk1; ++seg; }
      const int soa = (int)(kk * sta), sob = (int)(kk * stb);
      __amdgpu_buffer_rsrc_t rsa = ra, rsb = rb;
      if (seg > 0) {
        rsa = __builtin_amdgcn_make_buffer_rsrc((void*)P.seg_a[seg - 1], (short)0, (int)P.a_bytes, 0x00020000);
        rsb = __builtin_amdgcn_make_buffer_rsrc((void*)P.seg_b[seg - 1], (short)0, (int)P.b_bytes, 0x00020000);
      }
#pragma unroll
      for (int j = 0; j < SA; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_void*)(base + (SA * wave + j) * 1024), 16, va[j], soa, 0, 0);
#pragma unroll
      for (int j = 0; j < SB; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_void*)(base + TILEA + (SB * wave + j) * 1024), 16, vb[j], sob, 0, 0);
    }
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;

  // fragment byte offsets inside a stage (the two K halves of a step differ by chunk 2)
  int offa[4][2], offb[4][2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int c = 2 * ks + (lane >> 5);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int R = WTM * wm + 32 * mb + (lane & 31);
      offa[mb][ks] = R * ROWB + ((c ^ swz(R)) << 4);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int R = WTN * wn + 32 * nb + (lane & 31);
      offb[nb][ks] = TILEA + R * ROWB + ((c ^ swz(R)) << 4);
    }
  }

  // Main loop. Fragments are double-buffered in registers: F0 holds the first K half
  // of the current stage, F1 the second. The stage barrier sits between the two
  // MFMA groups, so that the LDS reads of one half always overlap the MFMAs of the
  // other:
  //   read F1 <- stage kt (2nd half); MFMA(F0)
  //   wait for stage kt+1; barrier; DMA stage kt+NS-1 into the slot of stage kt-1
  //   read F0 <- stage kt+1 (1st half); MFMA(F1)
  // A slot is refilled only after every wave has passed the barrier that follows
  // its last MFMA on that slot's data, and each wave waits (vmcnt) for its own DMA
  // loads of a stage before the barrier that publishes it.
  const int nk = SEGS && P.nseg > 1 ? P.nseg * nk1 : nk1;
  bf16x8 fa0[4], fb0[4], fa1[4], fb1[4];
  auto read_frags = [&](int stage, int ks, bf16x8 (&fa)[4], bf16x8 (&fb)[4]) {
    const char* st = smem + stage * STAGEB;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) fa[mb] = *reinterpret_cast<const bf16x8*>(st + offa[mb][ks]);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) fb[nb] = *reinterpret_cast<const bf16x8*>(st + offb[nb][ks]);
  };
  auto mfma_all = [&](const bf16x8 (&fa)[4], const bf16x8 (&fb)[4]) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[nb], fa[mb], acc[mb][nb], 0, 0, 0);
  };
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nk) issue(s, s);
  wait_vm(OPS * (NS - 2 < nk - 1 ? NS - 2 : nk - 1));   // stages issued after stage 0 may stay in flight
  stage_barrier();
  read_frags(0, 0, fa0, fb0);
  // The last step is peeled so that no fragment read sits behind a branch (the
  // compiler then counts outstanding LDS reads exactly and waits only for the half
  // it uses); sched_barrier(0) keeps the scheduler from interleaving the groups
  // differently: every fragment read is issued before the MFMAs it overlaps.
  int kt = 0;
  for (; kt + 1 < nk; ++kt) {
    read_frags(kt % NS, 1, fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_all(fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    // stage kt+1 was issued in step kt+2-NS; the stages issued in the later steps
    // (kt+3-NS .. kt-1) may stay in flight
    {
      int newer = 0;
      for (int i = kt + 3 - NS; i < kt; ++i)
        if (i + NS - 1 < nk) newer += OPS;
      wait_vm(newer);
    }
    stage_barrier();
    if (kt + NS - 1 < nk) issue(kt + NS - 1, (kt + NS - 1) % NS);
    read_frags((kt + 1) % NS, 0, fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    mfma_all(fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
  }
  read_frags(kt % NS, 1, fa1, fb1);
  mfma_all(fa0, fb0);
  mfma_all(fa1, fb1);
  // Every wave is done with the stages and its DMA writes have landed:
  // LDS becomes the epilogue slabs. Each wave then uses only its own slab, and a wave's
  // LDS accesses complete in program order, so the epilogue needs no further barrier
  // (its global loads stay in flight across slabs).
  wait_vm(0);
  __syncthreads();

  // ---- epilogue, one 32-row slab (block row mb) of the wave's sub-tile at a time.
  // The global operands of the epilogue (moments, or W and the block magnitudes)
  // are loaded before they are needed, many per lane at once, so that their
  // latency is paid once per slab (moments) or once per tile (W) rather than once
  // per row group.
  float* slab = reinterpret_cast<float*>(smem) + wave * EPWAVE;
  const int64_t wrow0 = row0 + WTM * wm, wcol0 = col0 + WTN * wn;
  auto stage_slab = [&](int mb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 32 * nb + 8 * g + 4 * (lane >> 5);
        *reinterpret_cast<float4*>(slab + (lane & 31) * EPLD + c) =
            make_float4(acc[mb][nb][4 * g], acc[mb][nb][4 * g + 1], acc[mb][nb][4 * g + 2], acc[mb][nb][4 * g + 3]);
      }
  };
  if constexpr (EP == EP_STORE || EP == EP_STORE_BF16) {
    // LPR lanes x 4 columns per row, RPP rows per pass, 32 / RPP passes per slab
    constexpr int LPR = WTN / 4, RPP = 64 / LPR, PPS = 32 / RPP;
    const int cc = 4 * (lane % LPR);
    const int64_t col = wcol0 + cc;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      stage_slab(mb);
#pragma unroll
      for (int p = 0; p < PPS; ++p) {
        const int rr = RPP * p + lane / LPR;
        const int64_t row = wrow0 + 32 * mb + rr;
        if (row < P.M && col < P.N) {
          const float4 v = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc);
          const int64_t idx = row * P.ldc + col;
          if constexpr (EP == EP_STORE) {
            *reinterpret_cast<float4*>((float*)P.c + idx) = v;
            if (P.c_parts) {   // v = h + m + l exactly (three 8-bit slices of the 24-bit significand)
              const float x[4] = {v.x, v.y, v.z, v.w};
              bf16x4 ph, pm, pl;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                ph[q] = f2bf(x[q]);
                const float d = x[q] - bf2f(ph[q]);
                pm[q] = f2bf(d);
                pl[q] = f2bf(d - bf2f(pm[q]));
              }
              bf16* pp = (bf16*)P.c_parts + kp_index(row, col, P.M);
              const int64_t plane = P.M * P.N;
              *reinterpret_cast<bf16x4*>(pp) = ph;
              *reinterpret_cast<bf16x4*>(pp + plane) = pm;
              *reinterpret_cast<bf16x4*>(pp + 2 * plane) = pl;
            }
          } else {
            bf16x4 o;
            o[0] = f2bf(v.x); o[1] = f2bf(v.y); o[2] = f2bf(v.z); o[3] = f2bf(v.w);
            const int64_t oi = (P.kp & 4) ? kp_index(row, col, P.M) : idx;
            *reinterpret_cast<bf16x4*>((bf16*)P.c + oi) = o;
            if (P.c_lo) {
              bf16x4 l;
              l[0] = f2bf(v.x - bf2f(o[0])); l[1] = f2bf(v.y - bf2f(o[1]));
              l[2] = f2bf(v.z - bf2f(o[2])); l[3] = f2bf(v.w - bf2f(o[3]));
              *reinterpret_cast<bf16x4*>((bf16*)P.c_lo + oi) = l;
            }
          }
        }
      }
    }
  } else if constexpr (EP == EP_ADAM_B16) {
    // as EP_ADAM below, with bf16 moments (8 bytes per 4-column group instead of 16)
    constexpr int LPR = WTN / 4, RPP = 64 / LPR;
    constexpr int PR = EPA_ROWS, NPC = 32 / PR, HPP = PR / RPP, NPT = MB * NPC, DB = EPDB_ADAM16;
    static_assert(PR % RPP == 0 && 32 % PR == 0 && DB >= 1, "epilogue pieces");
    const int cc = 4 * (lane % LPR);
    const int64_t col = wcol0 + cc;
    const bf16* E1 = reinterpret_cast<const bf16*>(P.e1);
    const bf16* E2 = reinterpret_cast<const bf16*>(P.e2);
    bf16x4 ev[DB][HPP], qv[DB][HPP];
    auto load_piece = [&](int h) {
#pragma unroll
      for (int p = 0; p < HPP; ++p) {
        const int64_t row = wrow0 + PR * h + RPP * p + lane / LPR;
        if (row < P.M && col < P.N) {
          const int64_t idx = row * P.ldc + col;
          // the moments are read and written once per step: non-temporal accesses keep them
          // from displacing the operand panels and the next kernels' data in the caches
          ev[h % DB][p] = __builtin_bit_cast(bf16x4, __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(E1 + idx)));
          qv[h % DB][p] = __builtin_bit_cast(bf16x4, __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(E2 + idx)));
        }
      }
    };
    auto compute_piece = [&](int h) {
#pragma unroll
      for (int p = 0; p < HPP; ++p) {
        const int rr = PR * (h % NPC) + RPP * p + lane / LPR;
        const int64_t row = wrow0 + PR * h + RPP * p + lane / LPR;
        if (row < P.M && col < P.N) {
          const float4 v = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc);
          const float vv[4] = {v.x, v.y, v.z, v.w};
          const int64_t idx = row * P.ldc + col;
          bf16x4 e = ev[h % DB][p], q = qv[h % DB][p], o;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            bf16 ec = e[c], qc = q[c];
            o[c] = f2bf(adam_out_bf16(vv[c], ec, qc, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2));
            e[c] = ec;
            q[c] = qc;
          }
          __builtin_nontemporal_store(__builtin_bit_cast(u32x2, e), reinterpret_cast<u32x2*>(reinterpret_cast<bf16*>(P.e1) + idx));
          __builtin_nontemporal_store(__builtin_bit_cast(u32x2, q), reinterpret_cast<u32x2*>(reinterpret_cast<bf16*>(P.e2) + idx));
          *reinterpret_cast<bf16x4*>((bf16*)P.c + ((P.kp & 4) ? kp_index(row, col, P.M) : idx)) = o;
        }
      }
    };
#pragma unroll
    for (int h = 0; h < DB - 1; ++h)
      if (h < NPT) load_piece(h);
#pragma unroll
    for (int h = 0; h < NPT; ++h) {
      if (h + DB - 1 < NPT) load_piece(h + DB - 1);
      if (h % NPC == 0) stage_slab(h / NPC);
      compute_piece(h);
    }
  } else if constexpr (EP == EP_ADAM) {
    // LPR lanes x 4 columns per row, RPP rows per pass. The moments move in pieces of PR
    // rows through a ring of DB register buffers: while one piece is computed, the loads
    // of the next DB - 1 pieces are in flight.
    constexpr int LPR = WTN / 4, RPP = 64 / LPR;
    constexpr int PR = EPA_ROWS, NPC = 32 / PR, HPP = PR / RPP, NPT = MB * NPC, DB = EPDB_ADAM;
    static_assert(PR % RPP == 0 && 32 % PR == 0 && DB >= 1, "epilogue pieces");
    const int cc = 4 * (lane % LPR);
    const int64_t col = wcol0 + cc;
    float4 ev[DB][HPP], qv[DB][HPP];
    auto load_piece = [&](int h) {   // rows [PR h, PR h + PR) of the wave's sub-tile
#pragma unroll
      for (int p = 0; p < HPP; ++p) {
        const int64_t row = wrow0 + PR * h + RPP * p + lane / LPR;
        if (row < P.M && col < P.N) {
          const int64_t idx = row * P.ldc + col;
          ev[h % DB][p] = *reinterpret_cast<const float4*>(P.e1 + idx);
          qv[h % DB][p] = *reinterpret_cast<const float4*>(P.e2 + idx);
        }
      }
    };
    auto compute_piece = [&](int h) {
#pragma unroll
      for (int p = 0; p < HPP; ++p) {
        const int rr = PR * (h % NPC) + RPP * p + lane / LPR;
        const int64_t row = wrow0 + PR * h + RPP * p + lane / LPR;
        if (row < P.M && col < P.N) {
          const float4 v = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc);
          const int64_t idx = row * P.ldc + col;
          float4 e = ev[h % DB][p], q = qv[h % DB][p];
          bf16x4 o;
          o[0] = f2bf(adam_out(v.x, e.x, q.x, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2));
          o[1] = f2bf(adam_out(v.y, e.y, q.y, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2));
          o[2] = f2bf(adam_out(v.z, e.z, q.z, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2));
          o[3] = f2bf(adam_out(v.w, e.w, q.w, U.beta1, U.beta2, U.adam_eps, P.bc1, P.bc2));
          *reinterpret_cast<float4*>(P.e1 + idx) = e;
          *reinterpret_cast<float4*>(P.e2 + idx) = q;
          *reinterpret_cast<bf16x4*>((bf16*)P.c + ((P.kp & 4) ? kp_index(row, col, P.M) : idx)) = o;
        }
      }
    };
#pragma unroll
    for (int h = 0; h < DB - 1; ++h)
      if (h < NPT) load_piece(h);
#pragma unroll
    for (int h = 0; h < NPT; ++h) {
      if (h + DB - 1 < NPT) load_piece(h + DB - 1);
      if (h % NPC == 0) stage_slab(h / NPC);
      compute_piece(h);
    }
  } else {
    // LPR lanes x 8 columns per row, RPP rows per pass, PPS passes per slab
    constexpr int LPR = WTN / 8, RPP = 64 / LPR, PPS = 32 / RPP;
    const int cc = 8 * (lane % LPR);
    const int64_t col = wcol0 + cc;
    const bool one_mag = (U.B & 7) == 0;   // 8 aligned columns never straddle a block
    if (U.weight_bf16 && one_mag) {
      // W and magnitudes DB slabs ahead (register double buffer with one workgroup per CU)
      constexpr int DB = EPDB_UPD;
      bf16x8 wv[DB][PPS];
      float mg[DB][PPS];
      auto load_w = [&](int mb) {
#pragma unroll
        for (int p = 0; p < PPS; ++p) {
          const int64_t row = wrow0 + 32 * mb + RPP * p + lane / LPR;
          mg[mb % DB][p] = 1.f;
          if (row < P.M && col < P.N) {
            // W is read and written once per step: non-temporal, as the moments above
            wv[mb % DB][p] = __builtin_bit_cast(
                bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>((const bf16*)P.c + row * P.ldc + col)));
            if (P.dM) mg[mb % DB][p] = P.dM[row * P.dM_ld + col / U.B];
          }
        }
      };
      load_w(0);
      if (DB == 2) load_w(1);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        stage_slab(mb);
#pragma unroll
        for (int p = 0; p < PPS; ++p) {
          const int rr = RPP * p + lane / LPR;
          const int64_t row = wrow0 + 32 * mb + rr;
          if (row < P.M && col < P.N) {
            const float4 v0 = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc);
            const float4 v1 = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc + 4);
            const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            const float m = mg[mb % DB][p];
            bf16x8 o;
#pragma unroll
            for (int q = 0; q < 8; ++q) o[q] = f2bf(bf2f(wv[mb % DB][p][q]) - U.lr * bf2f(f2bf(U.scale * (m * v[q]))));
            __builtin_nontemporal_store(__builtin_bit_cast(u32x4, o), reinterpret_cast<u32x4*>((bf16*)P.c + row * P.ldc + col));
          }
        }
        if (mb + DB < MB) load_w(mb + DB);
      }
    } else {
      // general form: fp32 W, or block sizes that split an 8-column group
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        stage_slab(mb);
#pragma unroll 2
        for (int p = 0; p < PPS; ++p) {
          const int rr = RPP * p + lane / LPR;
          const int64_t row = wrow0 + 32 * mb + rr;
          if (row < P.M && col < P.N) {
            const float4 v0 = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc);
            const float4 v1 = *reinterpret_cast<const float4*>(slab + rr * EPLD + cc + 4);
            const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            float mag[8];
            if (P.dM) {
              const float* dmr = P.dM + row * P.dM_ld;
#pragma unroll
              for (int q = 0; q < 8; ++q) mag[q] = dmr[(col + q) / U.B];
            } else {
#pragma unroll
              for (int q = 0; q < 8; ++q) mag[q] = 1.f;
            }
            const int64_t idx = row * P.ldc + col;
            if (U.weight_bf16) {
              bf16* W = (bf16*)P.c + idx;
              const bf16x8 w = *reinterpret_cast<const bf16x8*>(W);
              bf16x8 o;
#pragma unroll
              for (int q = 0; q < 8; ++q) o[q] = f2bf(bf2f(w[q]) - U.lr * bf2f(f2bf(U.scale * (mag[q] * v[q]))));
              *reinterpret_cast<bf16x8*>(W) = o;
            } else {
              float* W = (float*)P.c + idx;
              float4 w0 = *reinterpret_cast<const float4*>(W);
              float4 w1 = *reinterpret_cast<const float4*>(W + 4);
              w0.x -= U.lr * (U.scale * (mag[0] * v[0])); w0.y -= U.lr * (U.scale * (mag[1] * v[1]));
              w0.z -= U.lr * (U.scale * (mag[2] * v[2])); w0.w -= U.lr * (U.scale * (mag[3] * v[3]));
              w1.x -= U.lr * (U.scale * (mag[4] * v[4])); w1.y -= U.lr * (U.scale * (mag[5] * v[5]));
              w1.z -= U.lr * (U.scale * (mag[6] * v[6])); w1.w -= U.lr * (U.scale * (mag[7] * v[7]));
              *reinterpret_cast<float4*>(W) = w0;
              *reinterpret_cast<float4*>(W + 4) = w1;
            }
          }
        }
      }
    }
  }
}

}  // namespace

// Variants (8 layers of the 7B-shaped step, projection / back-projection ms, measured
// with an earlier epilogue that kept the back-projection at four stages and warmed W
// into the cache during the last K steps):
//   1: 256 x 256 tiles, eight waves of 128 x 64, four LDS stages, one workgroup per CU
//      (3.54 / 4.11);
//   2: 256 x 256 tiles, four waves of 128 x 128 (accumulators in AGPRs), four stages
//      (faster main loop, but half the waves to hide the epilogue's memory latency;
//      4.36 / 4.59);
//   3: 256 x 128 tiles, four waves of 128 x 64, three stages, two workgroups per CU
//      (3.86 / 4.36);
//   4: 256 x 128 tiles, eight waves of 64 x 64, three stages, two workgroups per CU
//      (3.61 / 3.89);
//   5: 256 x 256 tiles, sixteen waves of 64 x 64, four stages, one workgroup per CU
//      (3.28 / 3.88) -- the default. Its back-projection (K = r, 16 to 32 steps) ran
//      five stages while the epilogue's W accesses went through the caches (-4 %
//      against four then); with non-temporal W accesses four are faster again (full
//      7B stack: 13.05 -> 12.38 ms). The plain-store products of the projector refresh
//      run five (7B refresh -1.3 %).
// Re-measured with blocked operands and barrier-free epilogues (stand-alone copy of the
// kernel on 8 layers' worth of problems, projection / back-projection ms): variant 5
// 2.64 / 2.95, variant 4 3.04 / 3.11, variant 1 2.87 / 3.52.
// Starting the first round of workgroups at staggered times, so that the epilogues of
// different CUs (or of the two workgroups of a CU) do not coincide, changed nothing
// measurable in any variant.
#ifndef GEMM_NT_VARIANT
#define GEMM_NT_VARIANT 5
#endif
#if GEMM_NT_VARIANT == 1
constexpr int V_NWM = 2, V_NWN = 4, V_WTN = 64, V_NS = 4, V_NSU = 4, V_NSS = 4, V_OCC = 1;
#elif GEMM_NT_VARIANT == 2
constexpr int V_NWM = 2, V_NWN = 2, V_WTN = 128, V_NS = 4, V_NSU = 4, V_NSS = 4, V_OCC = 1;
#elif GEMM_NT_VARIANT == 3
constexpr int V_NWM = 2, V_NWN = 2, V_WTN = 64, V_NS = 3, V_NSU = 3, V_NSS = 3, V_OCC = 2;
#elif GEMM_NT_VARIANT == 4
constexpr int V_NWM = 4, V_NWN = 2, V_WTN = 64, V_NS = 3, V_NSU = 3, V_NSS = 3, V_OCC = 2;
#else
constexpr int V_NWM = 4, V_NWN = 4, V_WTN = 64, V_NS = 4, V_NSU = 4, V_NSS = 5, V_OCC = 1;
#endif
constexpr int GEMM_NT_BN = V_NWN * V_WTN;
uint32_t gemm_nt_tiles_m(int64_t M) { return (uint32_t)((M + TBM - 1) / TBM); }
uint32_t gemm_nt_tiles_n(int64_t N) { return (uint32_t)((N + GEMM_NT_BN - 1) / GEMM_NT_BN); }

bool gemm_nt_eligible(int ep, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc,
                      const void* a, const void* b, const void* c, int weight_bf16) {
  if (M <= 0 || N <= 0 || K <= 0 || K % TBK) return false;
  if (lda % 8 || ldb % 8 || lda < K || ldb < K) return false;
  if (((uintptr_t)a & 15) || ((uintptr_t)b & 15)) return false;
  // byte extents must fit the 32-bit buffer offsets
  if ((M - 1) * lda * 2 + K * 2 > 0x7FFFFFFFLL || (N - 1) * ldb * 2 + K * 2 > 0x7FFFFFFFLL) return false;
  // the epilogue operands are addressed through 32-bit buffer offsets as well
  if (M * ldc * (ep == EP_ADAM ? 4 : 2) > 0x7FFFFFFFLL) return false;
  if (ep == EP_STORE || ep == EP_STORE_BF16) {   // 4-column groups, 16- (8-) byte aligned
    const int esz = ep == EP_STORE ? 4 : 2;
    if (N % 4 || ldc % 4 || ((uintptr_t)c & (4 * esz - 1))) return false;
  } else if (ep == EP_ADAM) {   // moments and N: 4-column groups (library memory, aligned)
    if (N % 4 || ldc % 4) return false;
  } else {                      // W: 8-column groups, 16-byte aligned rows
    const int esz = weight_bf16 ? 2 : 4;
    if (N % 8 || ldc % 8 || ((uintptr_t)c & 15) || (ldc * esz) % 16) return false;
  }
  return true;
}

namespace {
template <int NWM, int NWN, int WTN, int NS, int NSU, int NSS, int OCC>
hipError_t launch_nt(int ep, const GemmProb* probs_dev, uint32_t total_tiles, const GemmUniform& u, hipStream_t st) {
  const dim3 grid(total_tiles), block(64 * NWM * NWN);
  if (ep == EP_ADAM && u.moment_bf16)
    hipLaunchKernelGGL((k_gemm_nt<EP_ADAM_B16, NWM, NWN, WTN, NS, OCC>), grid, block, 0, st, probs_dev, u);
  else if (ep == EP_ADAM) hipLaunchKernelGGL((k_gemm_nt<EP_ADAM, NWM, NWN, WTN, NS, OCC>), grid, block, 0, st, probs_dev, u);
  else if (ep == EP_UPDATE) hipLaunchKernelGGL((k_gemm_nt<EP_UPDATE, NWM, NWN, WTN, NSU, OCC>), grid, block, 0, st, probs_dev, u);
  else if (ep == EP_STORE) hipLaunchKernelGGL((k_gemm_nt<EP_STORE, NWM, NWN, WTN, NSS, OCC>), grid, block, 0, st, probs_dev, u);
  else if (ep == EP_STORE_BF16) hipLaunchKernelGGL((k_gemm_nt<EP_STORE_BF16, NWM, NWN, WTN, NSS, OCC>), grid, block, 0, st, probs_dev, u);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemm_nt(int ep, const GemmProb* probs_dev, int nprob, uint32_t total_tiles, const GemmUniform& u0,
                          hipStream_t st) {
  if (total_tiles == 0 || nprob == 0) return hipSuccess;
  GemmUniform u = u0;
  u.nprob = nprob;
  return launch_nt<V_NWM, V_NWN, V_WTN, V_NS, V_NSU, V_NSS, V_OCC>(ep, probs_dev, total_tiles, u, st);
}
