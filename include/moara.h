/*
 * moara.h -- C ABI of the MI355X (gfx950) MoARa optimizer library.
 *
 * MoARa (module-aware rank allocation, with block-wise magnitude/direction
 * decomposition) is a GaLore-style low-rank optimizer. For every target weight
 * W (m x n, stored out x in, row-major) and every training step it computes,
 * following the training phase of Algorithm 1:
 *
 *   1. Decompose (Section 3.1, Appendix B.1): split each row of the gradient G
 *      into contiguous 1 x B blocks along the columns (the last block is
 *      implicitly zero-padded), M[i,j] = ||block||_2, V = G / (M + eps_d),
 *      eps_d only in the denominator.
 *   2. When t mod T_SVD == 0: P <- TruncatedSVD(V, r) (top-r singular vectors).
 *   3. Project the direction: R = P^T V (LEFT, P is m x r) or R = V Q (RIGHT,
 *      Q is n x r). The projector sits on the smaller side: LEFT when m <= n,
 *      RIGHT when m > n, so the direction state is r x max(m, n) (this is the
 *      layout under which the paper's optimizer-state table, Appendix G,
 *      reproduces).
 *   4. Optimizer_V = Adam on R (beta1, beta2, eps, bias correction; no weight
 *      decay, Appendix D) -> N.
 *   5. Back-project: dV = P N (LEFT) or N Q^T (RIGHT).
 *   6. Optimizer_M = Adam on M with the same hyperparameters -> dM.
 *   7. W <- W - lr * scale * (Rep_B(dM) (.) dV), scale = GaLore scale (0.25 in
 *      Appendix D). With bf16 weights the scaled update is rounded to bf16
 *      (round to nearest even) before it is applied, and the result is rounded
 *      to bf16 (Appendix D).
 *
 * The per-module rank r_tau comes from a rank table, usually produced by the
 * budget-preserving reallocation of Algorithm 1, Phase 3 (moara_allocate_ranks).
 *
 * Conventions for every function:
 *   - Return value: MOARA_OK (0) or a negative moara_status. No exceptions cross
 *     the ABI. moara_last_error() returns a thread-local message for the last
 *     non-OK status of the calling thread.
 *   - Arguments are validated on the host before any HIP call; an invalid
 *     argument never reaches the GPU.
 *   - "Device pointer" means memory on the GPU that the state lives on
 *     (hipMalloc'd, e.g. a torch CUDA tensor's data_ptr()). "Host array" means
 *     ordinary CPU memory read during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     moara_step and moara_refresh_projector only enqueue work on it and return
 *     without synchronising; the caller must keep W and G alive and unmodified
 *     until that work has run.
 *   - A state lives on the HIP device that is current when moara_create_state is
 *     called; every later call that enqueues work on it must be made with that
 *     device current (MOARA_E_STATE otherwise, before anything is enqueued).
 *   - A state is not thread-safe: do not use one state from two threads at once.
 *     It may be used from several streams: every call that enqueues work on a
 *     state first makes its stream wait for the work the previous call on that
 *     state enqueued (an event recorded on the previous call's stream), so the
 *     state's calls run in call order whatever streams they are given. The
 *     caller orders its own buffers (W, G) against the streams it uses.
 */
#ifndef MOARA_H
#define MOARA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct moara_state moara_state; /* opaque; owned by the library */

typedef enum {
  MOARA_OK = 0,
  MOARA_E_ARG = -1,         /* null pointer, bad hyperparameter, bad index */
  MOARA_E_SHAPE = -2,       /* bad matrix shape or buffer size             */
  MOARA_E_RANK = -3,        /* rank outside [1, min(m,n)], bad Phase-3 rule */
  MOARA_E_UNSUPPORTED = -4, /* valid but not implemented (e.g. weight decay != 0) */
  MOARA_E_HIP = -5,         /* a HIP runtime call or kernel launch failed  */
  MOARA_E_OOM = -6,         /* device or pinned host allocation failed      */
  MOARA_E_STATE = -7        /* call not valid in this state (e.g. no projector yet) */
} moara_status;

/* Module types (the set T of Algorithm 1). Index into moara_config.rank_table. */
enum {
  MOARA_Q = 0, MOARA_K = 1, MOARA_V = 2, MOARA_O = 3,
  MOARA_GATE = 4, MOARA_UP = 5, MOARA_DOWN = 6,
  MOARA_EXP_GATE = 7, MOARA_EXP_UP = 8, MOARA_EXP_DOWN = 9,
  MOARA_NUM_MODULES = 10
};

enum { MOARA_SIDE_AUTO = 0, MOARA_SIDE_LEFT = 1, MOARA_SIDE_RIGHT = 2 };
enum { MOARA_F32 = 0, MOARA_BF16 = 1 };

/* Tensor ids for moara_get_tensor / moara_set_tensor. Layouts are the paper's
 * orientation, row-major, fp32 on the host side whatever moment_dtype stores on the
 * device (bf16 moments are widened exactly on get and rounded to nearest-even on set):
 *   MOARA_T_P          : the projector, s x r with s = m (LEFT) or n (RIGHT).
 *   MOARA_T_EXP_AVG    : first moment of Optimizer_V, r x n (LEFT) / m x r (RIGHT).
 *   MOARA_T_EXP_AVG_SQ : second moment of Optimizer_V, same shape.
 *   MOARA_T_MAG_AVG    : first moment of Optimizer_M, m x ceil(n/B).
 *   MOARA_T_MAG_AVG_SQ : second moment of Optimizer_M, m x ceil(n/B).
 *   MOARA_T_STEP       : the matrix's step counter t, one int64.            */
enum {
  MOARA_T_P = 0, MOARA_T_EXP_AVG = 1, MOARA_T_EXP_AVG_SQ = 2,
  MOARA_T_MAG_AVG = 3, MOARA_T_MAG_AVG_SQ = 4, MOARA_T_STEP = 5
};

/* One target weight matrix. rows x cols = m x n in the out x in layout. */
typedef struct {
  int64_t rows;
  int64_t cols;
  int32_t module;        /* MOARA_Q .. MOARA_EXP_DOWN: selects rank_table[module] */
  int32_t rank_override; /* 0: use rank_table[module]; >0: use this rank          */
  int32_t side;          /* MOARA_SIDE_AUTO (m <= n -> LEFT, else RIGHT), LEFT, RIGHT */
  int32_t reserved;      /* must be 0 */
} moara_matrix_desc;

/* Hyperparameters: Algorithm 1's Require line (rank table r_tau, block size B,
 * T_SVD) plus the Adam/GaLore settings of Appendix D. */
typedef struct {
  int32_t rank_table[MOARA_NUM_MODULES]; /* r_tau per module type (>= 1 where used) */
  int32_t block_size;                    /* B >= 1                                 */
  float beta1, beta2;                    /* Adam betas, in [0, 1)                  */
  float adam_eps;                        /* Adam epsilon > 0 (paper: 1e-6)         */
  float decomp_eps;                      /* eps_d >= 0 of the decomposition (1e-12) */
  float scale;                           /* GaLore scale alpha (0.25)              */
  float weight_decay;                    /* must be 0 (the paper uses none)        */
  int32_t refresh_interval;              /* T_SVD >= 0; 0 = refresh only on request */
  int32_t bias_correction;               /* 1 = Adam bias correction (paper), 0 = off */
  int32_t decompose;                     /* 1 = MoARa; 0 = plain GaLore direction (V = G, dM = 1) */
  int32_t weight_dtype;                  /* MOARA_F32 or MOARA_BF16                */
  int32_t grad_dtype;                    /* MOARA_F32 only                         */
  int32_t operand_dtype;                 /* GEMM operands: MOARA_F32 or MOARA_BF16 (fp32 accumulate) */
  int32_t refresh_oversample;            /* p >= 0 extra columns of the subspace iteration; -1 = p = r */
  int32_t refresh_iters;                 /* q >= 1 subspace-iteration sweeps (each applies V and V^T) */
  uint64_t refresh_seed;                 /* seed of the Gaussian start block       */
  int32_t zero_grad_mode;                /* what moara_step does with inactive matrices (active[i] == 0):
                                            0: skip them (no state change, t not advanced);
                                            1: step them with G = 0 (grads[i] is not read; W moves by
                                               the decayed moments, t advances) */
  int32_t moment_dtype;                  /* storage of Optimizer_V's two moments: MOARA_F32, or MOARA_BF16
                                            (the 2-byte direction states of Appendix D / Table 11; each
                                            update is computed in fp32 from the stored values and
                                            rounded to nearest-even on store). Optimizer_M's states
                                            stay fp32 (Appendix D). */
} moara_config;

/* Fill *out with the paper's defaults (Appendix D): B=128, beta=(0.9,0.999),
 * adam_eps=1e-6, decomp_eps=1e-12, scale=0.25, weight_decay=0, T_SVD=200,
 * bias correction on, decomposition on, bf16 weights, fp32 gradients, bf16
 * GEMM operands, p=-1 (p=r), q=20, seed 0, fp32 moments, rank_table all 0 (the caller sets
 * it, e.g. with moara_allocate_ranks). Errors: MOARA_E_ARG if out is NULL. */
int moara_default_config(moara_config* out);

/* Algorithm 1, Phase 3 (the static budget-preserving reallocation of Section 3.2):
 * r_tau = r_base - delta_r for tau in D, r_base + delta_r*|D|/|R| for tau in R,
 * r_base otherwise, for the module types in `types_mask`. Masks are bit sets
 * over module ids (bit i = module i). Entries of out_rank_table for modules not
 * in types_mask are set to 0.
 * Errors: MOARA_E_ARG (null out, empty types_mask, D or R outside types_mask,
 * D and R overlapping, exactly one of D, R empty, r_base < 1, delta_r < 0);
 * MOARA_E_RANK when delta_r*|D| is not a multiple of |R| or a rank falls
 * below 1. On error out_rank_table is left unchanged. */
int moara_allocate_ranks(int32_t r_base, uint32_t types_mask, uint32_t donor_mask,
                         uint32_t receiver_mask, int32_t delta_r,
                         int32_t out_rank_table[MOARA_NUM_MODULES]);

/* Resolve one matrix's rank and projection side from the config (bit-exact
 * host logic used by moara_create_state). out_side receives MOARA_SIDE_LEFT or
 * MOARA_SIDE_RIGHT. Errors: MOARA_E_ARG (nulls, module out of range, bad side),
 * MOARA_E_SHAPE (rows or cols < 1), MOARA_E_RANK (rank < 1 or > min(m, n)). */
int moara_resolve_matrix(const moara_config* cfg, const moara_matrix_desc* desc,
                         int32_t* out_rank, int32_t* out_side);

/* Device bytes a state for these n matrices would hold (persistent state plus
 * the per-step workspace; the refresh workspace is reported separately because
 * it is sized per refresh batch: a refresh works through its matrices in chunks
 * of at most 128 GiB of workspace, so the figure is the smaller of the whole
 * batch's need and that bound plus the average matrix's share). The environment
 * variable MOARA_REFRESH_CHUNK_MIB, when set to a positive integer, replaces the
 * bound (in MiB) for this call and for later refreshes. Errors as
 * moara_create_state's validation. */
int moara_state_bytes(const moara_config* cfg, const moara_matrix_desc* descs, int32_t n,
                      int64_t* out_state_bytes, int64_t* out_refresh_workspace_bytes);

/* Create an optimizer state for n matrices on the current HIP device.
 * descs: host array of n descriptors (copied). Moments start at zero, step
 * counters at 0, no projector is set (the first moara_step with T_SVD > 0, a
 * moara_refresh_projector call or moara_set_tensor(MOARA_T_P) sets it).
 * Allocates all persistent device memory up front; `stream` is used for the
 * initial zero fill, which is complete when this returns.
 * Errors: MOARA_E_ARG/SHAPE/RANK/UNSUPPORTED from validation, MOARA_E_OOM,
 * MOARA_E_HIP. On error *out is NULL and nothing is leaked. */
int moara_create_state(const moara_config* cfg, const moara_matrix_desc* descs, int32_t n,
                       void* stream, moara_state** out);

/* Algorithm 1's TruncatedSVD step (P_tau from V at rank r_tau), run now for the selected
 * matrices from their current gradients: V is formed from G exactly as in the
 * step, and P is computed by fp32 subspace iteration (q sweeps of V and V^T
 * with re-orthonormalisation, p oversampling columns) followed by a
 * Rayleigh-Ritz step, so P holds approximate top-r singular vectors ordered by
 * singular value, each column's largest-magnitude entry made positive.
 * grads: host array of n device pointers to fp32 m x n row-major gradients
 *        (entries of inactive matrices may be NULL).
 * active: host array of n bytes (nonzero = refresh this matrix) or NULL = all.
 * A matrix whose V is exactly zero keeps its previous projector (or gets the
 * first r canonical basis vectors if it had none). Step counters and moments
 * are not touched. Errors: MOARA_E_ARG (null state/grads, null grad of an
 * active matrix), MOARA_E_HIP, MOARA_E_OOM (refresh workspace). */
int moara_refresh_projector(moara_state* st, const void* const* grads, const uint8_t* active,
                            void* stream);

/* One optimizer step (Algorithm 1 training phase) for every active matrix:
 * decompose, refresh if t mod T_SVD == 0 (t = the matrix's count before the
 * step), project, Adam on R and on M, back-project, update W in place; then
 * t <- t + 1. Inactive matrices (active[i] == 0), e.g. MoE experts that
 * received no tokens, are skipped entirely with zero_grad_mode 0: W, the
 * moments, P and t are unchanged. With zero_grad_mode 1 they take the same step
 * with G = 0 instead (M = 0 and V = 0: a refresh that falls due keeps P, or sets
 * the first r canonical basis vectors if there is none; both Adam branches decay
 * their moments; W moves by Rep_B(dM) (.) P N; t advances); grads[i] of such a
 * matrix is not read and may be NULL, weights[i] must be valid.
 * weights: host array of n device pointers to m x n row-major W (weight_dtype).
 * grads:   host array of n device pointers to m x n row-major fp32 G (read only).
 * lr:      learning rate eta for this step (the caller owns the schedule).
 * Errors: MOARA_E_ARG (nulls, non-finite lr), MOARA_E_STATE (a matrix to step
 * has no projector and T_SVD == 0), MOARA_E_HIP. */
int moara_step(moara_state* st, void* const* weights, const void* const* grads,
               const uint8_t* active, float lr, void* stream);

/* moara_step for callers that cannot allocate device memory (allocation-free serving or
 * training loops, harnesses that forbid hipMalloc). It allocates nothing, but it is not
 * made for stream capture: like moara_step it stages each launch's descriptors through
 * the state's pinned host ring (a host-to-device copy on `stream`, and a host wait before
 * a ring slot is reused), so a graph captured from it would not replay correctly.
 * Same arguments, semantics and results as moara_step, bit for bit, but it calls no
 * hipMalloc, hipFree, hipHostMalloc or other device/pinned allocator: the step's
 * descriptors, and when a refresh falls due its descriptors and workspace, live in one
 * fixed array of MOARA_NOALLOC_SCRATCH_BYTES per GPU that the library holds until the
 * process ends (its address on each GPU is looked up once, when a state is created on
 * that GPU). A due refresh runs in chunks that fit the array.
 * Limits, checked before anything is enqueued (nothing changes on error):
 * MOARA_E_UNSUPPORTED when the state's step descriptors take more than the array minus
 * 8 MiB, or when one matrix due for a refresh needs more workspace than the rest of it
 * (e.g. 18944 x 3584 at r = 1024; every Llama-2-7B, Llama-300M and DeepSeek-MoE matrix
 * fits). Such matrices are refreshed with moara_step or moara_refresh_projector, or with
 * refresh_interval = 0 and explicit refreshes outside the allocation-free region.
 * Sharing: every call on one GPU uses that GPU's array, and the array keeps the last
 * call's contents (every region a call reads is written or cleared by it first). Calls on
 * one GPU are ordered on the GPU through an event that each call records and the next
 * one's stream waits on, but calls from two host threads at the same time on one GPU
 * race: serialise them. Per-kernel timing (moara_set_timing) is not recorded. Host
 * bookkeeping uses ordinary heap memory; a refresh chunk's descriptors are copied from
 * it synchronously (the call then waits for that copy). Errors: as moara_step, plus
 * MOARA_E_UNSUPPORTED for the limits above. */
#define MOARA_NOALLOC_SCRATCH_BYTES (1024ull << 20)
int moara_step_noalloc(moara_state* st, void* const* weights, const void* const* grads,
                       const uint8_t* active, float lr, void* stream);

/* Subspace alignment diagnostic of Section 3.2 (Eq. module_alignment; the
 * quantity logged in Algorithm 1, Phases 1-2): for every active matrix,
 *   out_S[i] = cos(G_i, G_recon,i) = <G, G_recon>_F / (||G||_F ||G_recon||_F),
 *   G_recon = Rep_B(M) (elementwise) (P P^T V)  for a LEFT matrix,
 *             Rep_B(M) (elementwise) (V Q Q^T)  for a RIGHT matrix,
 * with M, V the block decomposition of G_i (the state's B and eps_d; with
 * decompose = 0, M = 1 and V = G) and P (Q) the matrix's current fp32 projector.
 * 0 when G or G_recon is zero. The module average S_tau is the caller's mean
 * of these values over logged steps and matrices of one module type.
 * Reads only: weights, moments, projectors and step counters are unchanged.
 * fp32 GEMM operands with fp64 sums (accumulated with atomics, so the last bits
 * may differ between runs).
 * grads:  host array of n device pointers to m x n row-major fp32 G (read only).
 * active: host array of n flags (NULL = all); out_S[i] of an inactive matrix is
 *         left as it was.
 * out_S:  host array of n doubles, written before the call returns (the call
 *         synchronises `stream`).
 * Uses the refresh workspace (4 L r bytes per active matrix). Errors:
 * MOARA_E_ARG (nulls), MOARA_E_STATE (an active matrix has no projector),
 * MOARA_E_OOM (workspace), MOARA_E_HIP. */
int moara_alignment(moara_state* st, const void* const* grads, const uint8_t* active,
                    double* out_S, void* stream);

/* Copy one state tensor of matrix `mat` to host memory (synchronises with the
 * state's work queued so far on `stream`). Layouts and dtypes: see MOARA_T_*
 * (fp32, except MOARA_T_STEP: one int64). bytes must equal the exact size.
 * Errors: MOARA_E_ARG (null, bad index/which), MOARA_E_SHAPE (bytes wrong),
 * MOARA_E_STATE (MOARA_T_P before any projector exists), MOARA_E_HIP. */
int moara_get_tensor(moara_state* st, int32_t mat, int32_t which, void* host_dst, size_t bytes,
                     void* stream);

/* Overwrite one state tensor of matrix `mat` from host memory (same layouts as
 * moara_get_tensor); setting MOARA_T_P also rebuilds the operand copies of the
 * projector and marks it present. Synchronous. Errors as moara_get_tensor. */
int moara_set_tensor(moara_state* st, int32_t mat, int32_t which, const void* host_src, size_t bytes,
                     void* stream);

/* Record of the matrix's last refresh by the library (moara_refresh_projector or a
 * refresh inside moara_step), for callers that check how TruncatedSVD (Algorithm 1)
 * went. The refresh finishes with a Rayleigh-Ritz step whose w x w SVD is computed by
 * one-sided Jacobi sweeps; they stop when every column pair's cosine is below 1e-7 or
 * after a fixed number of sweeps (14).
 *   out_sweeps:    Jacobi sweeps run;
 *   out_converged: 1 if the sweeps met the tolerance, 0 if they stopped at the limit
 *                  (the projector is then still orthonormal, but its directions are
 *                  less accurate);
 *   out_rank:      Ritz directions kept (at most r): those whose Ritz value exceeds 1e-5
 *                  of the largest. When it is below r (V of rank below r), the other
 *                  columns of P are an orthonormal completion (any completion is a top-r
 *                  singular basis of such a V); 0 when V was zero;
 *   out_offdiag:   the largest pair cosine measured in the last sweep.
 * Any output pointer may be NULL. Synchronises `stream`. Errors: MOARA_E_ARG (null
 * state, bad index), MOARA_E_STATE (the library has not refreshed this matrix; a
 * projector set with moara_set_tensor has no record), MOARA_E_HIP. */
int moara_refresh_info(moara_state* st, int32_t mat, int32_t* out_sweeps, int32_t* out_converged,
                       int32_t* out_rank, float* out_offdiag, void* stream);

/* Per-kernel timing for measurement: when enabled, moara_step and
 * moara_refresh_projector bracket each kernel launch with HIP events on the
 * caller's stream and accumulate the elapsed time per kernel id when
 * moara_kernel_stats is called (which synchronises the stream). */
enum {
  MOARA_KERN_DECOMPOSE = 0, /* decompose + Optimizer_M                 */
  MOARA_KERN_PROJECT = 1,   /* projection GEMM + Optimizer_V epilogue  */
  MOARA_KERN_BACKPROJ = 2,  /* back-projection GEMM + update epilogue  */
  MOARA_KERN_REFRESH = 3,   /* whole refresh (all its kernels)         */
  MOARA_KERN_ALIGN = 4,     /* alignment diagnostic GEMMs              */
  MOARA_NUM_KERNELS = 5
};
int moara_set_timing(moara_state* st, int32_t enable);
int moara_kernel_stats(moara_state* st, int32_t kernel, int64_t* out_launches, double* out_total_ms,
                       void* stream);
/* Zero the accumulated per-kernel statistics (synchronises the stream). */
int moara_reset_kernel_stats(moara_state* st, void* stream);

/* Number of matrices in the state and one matrix's resolved layout. */
int moara_matrix_info(const moara_state* st, int32_t mat, int64_t* rows, int64_t* cols,
                      int32_t* rank, int32_t* side, int32_t* n_blocks);

/* Free all device and host memory of the state. NULL is a no-op. Waits for
 * the state's outstanding work first. */
void moara_destroy_state(moara_state* st);

/* Thread-local message describing the last non-OK status on this thread. */
const char* moara_last_error(void);

/* Library version string. */
const char* moara_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MOARA_H */
