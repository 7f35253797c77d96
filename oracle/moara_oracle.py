"""CPU oracle for the MoARa optimizer hot path -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may import
this module. The product path (the HIP library and its Python binding) never
does, and this module imports nothing from the product package.

It is a plain, slow, float64 NumPy transcription of what the paper defines:

* Algorithm 1, training phase: per step and per target weight W,
  Decompose -> (every T_SVD steps) TruncatedSVD -> project -> Optimizer_V ->
  back-project -> Optimizer_M -> recompose and apply.
* Section 3.1 and Appendix B.1: block-wise magnitude/direction decomposition
  along the column (in-feature) axis, right zero padding of the last block,
  epsilon in the denominator only, cropping after recomposition.
* Algorithm 1 Phase 3 (Section 3.2, the static budget-preserving reallocation):
  the integer rank table.
* Appendix D: Adam with beta=(0.9, 0.999), bias correction, zero weight decay,
  GaLore scale 0.25, magnitude branch in fp32, recomposed update cast to bf16.
* Appendix G: optimizer-state memory formulas.
* Section 3.2 (Eq. module_alignment): the subspace alignment diagnostic S(W, t) and
  its module average S_tau (Algorithm 1, Phases 1-2).

Readings taken where the paper is silent or ambiguous are listed in the
repository's design notes; each is also stated at the function that uses it.
Library primitives used as single steps: numpy matmul, numpy.linalg.svd (LAPACK).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Iterable, Optional, Sequence, Tuple

import numpy as np

LEFT, RIGHT = "left", "right"


# ----------------------------------------------------------------------------
# number formats
# ----------------------------------------------------------------------------

def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps the float32 exponent range (normal exponents -126..127) and
    8 significant bits. Computed directly from the binary exponent: the value is
    divided by its bf16 ulp (a power of two, exact), rounded half-to-even by
    numpy.rint, and multiplied back. Results beyond the largest finite bf16
    become +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x) & (x != 0)
    xf = x[fin]
    _, e = np.frexp(xf)                      # xf = f * 2**e, 0.5 <= |f| < 1
    e = np.maximum(e - 1, -126)              # unbiased exponent, clamped into the subnormal range
    ulp = np.ldexp(1.0, e - 7)               # 8 significant bits
    r = np.rint(xf / ulp) * ulp
    maxbf = (2.0 - 2.0 ** -7) * 2.0 ** 127
    r = np.where(np.abs(r) > maxbf, np.copysign(np.inf, r), r)
    out[fin] = r
    return out


def round_f32(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# Phase 3: budget-preserving reallocation (Algorithm 1 setup phase; Section 3.2)
# ----------------------------------------------------------------------------

def allocate_ranks(r_base: int, module_types: Sequence[int], donors: Iterable[int],
                   receivers: Iterable[int], delta_r: int) -> Dict[int, int]:
    """r_tau = r_base - dr for donors, r_base + dr*|D|/|R| for receivers, r_base otherwise.

    The paper uses choices for which the receiver share is an integer ("no
    residual adjustment required"); a non-integer share, an overlap of D and R,
    or a rank below 1 is rejected with ValueError.
    """
    D, R = set(donors), set(receivers)
    if D & R:
        raise ValueError("donor and receiver sets overlap")
    if not D.issubset(module_types) or not R.issubset(module_types):
        raise ValueError("donor/receiver not among module types")
    if r_base < 1 or delta_r < 0:
        raise ValueError("r_base must be >= 1 and delta_r >= 0")
    if (D and not R) or (R and not D):
        raise ValueError("donor and receiver sets must both be empty or both be non-empty")
    out = {}
    gain = 0
    if R:
        if (delta_r * len(D)) % len(R) != 0:
            raise ValueError("receiver share delta_r*|D|/|R| is not an integer")
        gain = delta_r * len(D) // len(R)
    for t in module_types:
        if t in D:
            out[t] = r_base - delta_r
        elif t in R:
            out[t] = r_base + gain
        else:
            out[t] = r_base
        if out[t] < 1:
            raise ValueError("a rank fell below 1")
    return out


# ----------------------------------------------------------------------------
# Appendix G: optimizer-state memory model
# ----------------------------------------------------------------------------

def paper_state_bytes(shapes: Sequence[Tuple[int, int]], ranks: Sequence[int], block_sizes: Sequence[int],
                      b_V: int, b_M: int, decompose: bool) -> int:
    """Sum over target matrices of M_dir = 2 b_V r_W d_W plus, with decomposition,
    2 b_M m_W ceil(n_W / B_W) (Appendix G).

    d_W is the state dimension the projection leaves uncompressed; with the
    projector on the smaller side (state r x max(m, n)) the paper's printed
    state sizes reproduce exactly, so d_W = max(m, n) here.
    """
    tot = 0
    for (m, n), r, B in zip(shapes, ranks, block_sizes):
        tot += 2 * b_V * r * max(m, n)
        if decompose:
            tot += 2 * b_M * m * math.ceil(n / B)
    return tot


# ----------------------------------------------------------------------------
# Section 3.1 / Appendix B.1: block-wise magnitude-direction decomposition
# ----------------------------------------------------------------------------

def flatten(G: np.ndarray) -> np.ndarray:
    """Appendix B.1 (flattened tensors): keep the first axis, flatten all the others into
    the column axis, G_flat = reshape(G, s0, s1 * ... * s_{r-1}) in row-major order."""
    G = np.asarray(G)
    return G.reshape(G.shape[0], -1)


def n_blocks(n: int, B: int) -> int:
    """k = n_pad / B with n_pad the smallest multiple of B that is >= n."""
    return -(-n // B)


def decompose(G: np.ndarray, B: int, eps: float = 1e-12) -> Tuple[np.ndarray, np.ndarray]:
    """M[i, j] = ||G_pad[i, jB:(j+1)B]||_2 and V_pad = G_pad / (m_ij + eps), cropped to n columns.

    The padding columns are zero, so the norm of the last (partial) block is
    the norm over its real columns; cropping V_pad back to n columns gives V.
    """
    G = np.asarray(G, dtype=np.float64)
    m, n = G.shape
    k = n_blocks(n, B)
    Gp = np.zeros((m, k * B))
    Gp[:, :n] = G
    blocks = Gp.reshape(m, k, B)
    M = np.sqrt(np.sum(blocks * blocks, axis=2))
    Vp = blocks / (M[:, :, None] + eps)
    V = Vp.reshape(m, k * B)[:, :n]
    return M, V


def rep_b(M: np.ndarray, B: int, n: int) -> np.ndarray:
    """Rep_B(M): repeat each block value over its B columns, cropped to n columns."""
    return np.repeat(M, B, axis=1)[:, :n]


def recompose(M: np.ndarray, V: np.ndarray, B: int) -> np.ndarray:
    """Rep_B(M) (elementwise) V, i.e. m_ij * v_ij per block (Appendix B.1)."""
    return rep_b(M, B, V.shape[1]) * V


# ----------------------------------------------------------------------------
# TruncatedSVD (Algorithm 1) and its side
# ----------------------------------------------------------------------------

def projection_side(m: int, n: int) -> str:
    """Projector on the smaller side: LEFT (P in R^{m x r}, R = P^T V) when m <= n,
    RIGHT (Q in R^{n x r}, R = V Q) when m > n. With this choice the direction
    state is r x max(m, n), the layout under which the paper's optimizer-state
    table reproduces (Appendix G)."""
    return LEFT if m <= n else RIGHT


def canonical_signs(P: np.ndarray) -> np.ndarray:
    """Flip each column so that its entry of largest magnitude (lowest index on ties) is positive.
    SVD fixes singular vectors only up to sign; this makes the oracle's output unique."""
    P = np.array(P, dtype=np.float64, copy=True)
    idx = np.argmax(np.abs(P), axis=0)
    sgn = np.sign(P[idx, np.arange(P.shape[1])])
    sgn[sgn == 0] = 1.0
    return P * sgn


def truncated_svd(V: np.ndarray, r: int, side: str) -> Optional[np.ndarray]:
    """Top-r singular vectors of V on the projected side (LAPACK SVD in float64).

    LEFT: first r left singular vectors (m x r). RIGHT: first r right singular
    vectors (n x r). Returns None when V is exactly zero (no subspace defined).
    """
    V = np.asarray(V, dtype=np.float64)
    if not np.any(V):
        return None
    U, s, Yt = np.linalg.svd(V, full_matrices=False)
    P = U[:, :r] if side == LEFT else Yt[:r, :].T
    return canonical_signs(P)


def principal_angles(A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Principal angles (radians, ascending) between span(A) and span(B), via the
    singular values of Qa^T Qb; small angles are taken from the sine form
    ||Qb - Qa Qa^T Qb|| for accuracy."""
    Qa = np.linalg.qr(np.asarray(A, dtype=np.float64))[0]
    Qb = np.linalg.qr(np.asarray(B, dtype=np.float64))[0]
    sines = np.linalg.svd(Qb - Qa @ (Qa.T @ Qb), compute_uv=False)
    return np.sort(np.arcsin(np.clip(sines, 0.0, 1.0)))


def max_principal_angle(A: np.ndarray, B: np.ndarray) -> float:
    return float(principal_angles(A, B)[-1])


# ----------------------------------------------------------------------------
# Adam (Optimizer_V and Optimizer_M; Appendix D hyperparameters)
# ----------------------------------------------------------------------------

def adam(x: np.ndarray, exp_avg: np.ndarray, exp_avg_sq: np.ndarray, t: int,
         beta1: float, beta2: float, eps: float, bias_correction: bool = True, store=None):
    """One Adam step on input x at step t (t >= 1), Kingma & Ba form, no weight decay.

    e <- b1 e + (1 - b1) x ;  q <- b2 q + (1 - b2) x^2 ;
    out = (e / (1 - b1^t)) / (sqrt(q / (1 - b2^t)) + eps).
    ``store`` is the number format the two moments are kept in (a rounding function,
    None = exact); the moments are stored first and ``out`` is formed from the stored
    values. Returns (out, e, q).
    """
    e = beta1 * exp_avg + (1.0 - beta1) * x
    q = beta2 * exp_avg_sq + (1.0 - beta2) * x * x
    if store is not None:
        e, q = store(e), store(q)
    if bias_correction:
        c1 = 1.0 - beta1 ** t
        c2 = 1.0 - beta2 ** t
    else:
        c1 = c2 = 1.0
    out = (e / c1) / (np.sqrt(q / c2) + eps)
    return out, e, q


# ----------------------------------------------------------------------------
# One Algorithm 1 training-phase step for one target weight
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class OracleConfig:
    block_size: int
    rank: int
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    decomp_eps: float = 1e-12
    scale: float = 0.25
    refresh_interval: int = 200     # T_SVD; 0 = refresh only when asked
    bias_correction: bool = True
    decompose: bool = True
    weight_dtype: str = "f32"       # "f32" | "bf16"
    operand_dtype: str = "f32"      # "f32" | "bf16": bf16 rounding of V, P and N before the GEMMs
    moment_dtype: str = "f32"       # "f32" | "bf16": storage of Optimizer_V's moments (Appendix G's b_V)
    side: Optional[str] = None      # None = projection_side(m, n)


@dataclasses.dataclass
class OracleState:
    m: int
    n: int
    side: str
    rank: int
    P: Optional[np.ndarray]         # s x r (s = m for LEFT, n for RIGHT)
    exp_avg: np.ndarray             # state in the paper's orientation: r x n (LEFT) or m x r (RIGHT)
    exp_avg_sq: np.ndarray
    mag_avg: np.ndarray             # m x k
    mag_avg_sq: np.ndarray
    t: int = 0


def init_state(m: int, n: int, cfg: OracleConfig) -> OracleState:
    side = cfg.side or projection_side(m, n)
    r = cfg.rank
    if r < 1 or r > min(m, n):
        raise ValueError("rank must be in [1, min(m, n)]")
    shp = (r, n) if side == LEFT else (m, r)
    k = n_blocks(n, cfg.block_size)
    return OracleState(m, n, side, r, None, np.zeros(shp), np.zeros(shp), np.zeros((m, k)), np.zeros((m, k)))


def _operand(x: np.ndarray, cfg: OracleConfig) -> np.ndarray:
    return round_bf16(x) if cfg.operand_dtype == "bf16" else x


def refresh(st: OracleState, V: np.ndarray, cfg: OracleConfig) -> None:
    """P <- TruncatedSVD(V, r). A zero V leaves P as it was; with no previous P the
    first r canonical basis vectors are used (the paper is silent on this case)."""
    P = truncated_svd(V, st.rank, st.side)
    if P is None:
        if st.P is None:
            s = st.m if st.side == LEFT else st.n
            st.P = np.eye(s, st.rank)
        return
    st.P = P


def step(W: np.ndarray, G: np.ndarray, st: OracleState, cfg: OracleConfig, lr: float,
         force_refresh: bool = False) -> np.ndarray:
    """Algorithm 1 training phase for one weight and one step; returns the new W.

    Order: Decompose; refresh when t mod T_SVD == 0 (t = this matrix's step
    count before the step); V~ = P^T V (LEFT) or V Q (RIGHT); Optimizer_V;
    back-projection; Optimizer_M; W <- W - lr * scale * (Rep_B(dM) * dV).

    ``scale`` is GaLore's scale (0.25 in Appendix D; 1 is Algorithm 1 as
    printed). With bf16 weights the recomposed, scaled update is cast to bf16
    first and the subtraction result is rounded to bf16 (Appendix D).

    With moment_dtype "bf16" the direction moments are 2-byte states (b_V = 2 in
    Appendix G's memory formulas; with b_M = 4 they reproduce its optimizer-state
    table exactly): each is rounded to bf16 when stored and N is formed from the
    stored values. The magnitude branch's states stay exact (fp32 in Appendix D).
    """
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    B = cfg.block_size
    if cfg.decompose:
        M, V = decompose(G, B, cfg.decomp_eps)
    else:
        M, V = None, G
    if force_refresh or (cfg.refresh_interval > 0 and st.t % cfg.refresh_interval == 0):
        refresh(st, V, cfg)
    if st.P is None:
        raise RuntimeError("no projector: refresh never ran")
    P = _operand(st.P, cfg)
    Vo = _operand(V, cfg)
    Rt = P.T @ Vo if st.side == LEFT else Vo @ P                      # projected direction
    st.t += 1
    N, st.exp_avg, st.exp_avg_sq = adam(Rt, st.exp_avg, st.exp_avg_sq, st.t,
                                        cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.bias_correction,
                                        store=round_bf16 if cfg.moment_dtype == "bf16" else None)
    No = _operand(N, cfg)
    dV = P @ No if st.side == LEFT else No @ P.T                       # back-projection
    if cfg.decompose:
        dM, st.mag_avg, st.mag_avg_sq = adam(M, st.mag_avg, st.mag_avg_sq, st.t,
                                             cfg.beta1, cfg.beta2, cfg.adam_eps, cfg.bias_correction)
        U = rep_b(dM, B, st.n) * dV
    else:
        U = dV
    U = cfg.scale * U
    if cfg.weight_dtype == "bf16":
        return round_bf16(W - lr * round_bf16(U))
    return W - lr * U


def update_direction(W_old: np.ndarray, W_new: np.ndarray) -> np.ndarray:
    return np.asarray(W_new, dtype=np.float64) - np.asarray(W_old, dtype=np.float64)


# ----------------------------------------------------------------------------
# Subspace alignment diagnostic (Section 3.2, Eq. module_alignment; Algorithm 1,
# Phases 1-2)
# ----------------------------------------------------------------------------

def reconstruct(G: np.ndarray, P: np.ndarray, B: int, eps: float = 1e-12, decompose_on: bool = True,
                side: Optional[str] = None) -> np.ndarray:
    """G_recon = Rep_B(M) (elementwise) (P P^T V): the gradient rebuilt from its block
    magnitudes and the projection of its direction tensor onto the rank-r subspace.

    The paper writes the LEFT form (P in R^{m x r}). Reading: a RIGHT matrix (m > n,
    projector Q in R^{n x r}) uses the same construction on its projected side,
    Rep_B(M) (elementwise) (V Q Q^T). With the decomposition off the reconstruction is
    GaLore's, P P^T G (resp. G Q Q^T).
    """
    G = np.asarray(G, dtype=np.float64)
    P = np.asarray(P, dtype=np.float64)
    m, n = G.shape
    side = side or projection_side(m, n)
    if decompose_on:
        M, V = decompose(G, B, eps)
    else:
        M, V = None, G
    PV = P @ (P.T @ V) if side == LEFT else (V @ P) @ P.T
    return recompose(M, PV, B) if decompose_on else PV


def alignment(G: np.ndarray, P: np.ndarray, B: int, eps: float = 1e-12, decompose_on: bool = True,
              side: Optional[str] = None) -> float:
    """S(W, t) = cos(G, G_recon), the cosine of the two matrices as vectors (Frobenius
    inner product over the product of Frobenius norms). Reading: 0 when G or G_recon
    is the zero matrix (the cosine is undefined there)."""
    G = np.asarray(G, dtype=np.float64)
    R = reconstruct(G, P, B, eps, decompose_on, side)
    den = float(np.linalg.norm(G)) * float(np.linalg.norm(R))
    return float(np.sum(G * R)) / den if den > 0.0 else 0.0


def module_alignment(samples: Iterable[Tuple[int, float]]) -> Dict[int, float]:
    """S_tau = mean of S(W, t) over the logged steps and the matrix instances of module
    type tau: samples are (module type, S) pairs."""
    acc: Dict[int, list] = {}
    for tau, s in samples:
        acc.setdefault(int(tau), []).append(float(s))
    return {tau: float(np.mean(v)) for tau, v in acc.items()}


# ----------------------------------------------------------------------------
# Comparison metric used by the parity tests
# ----------------------------------------------------------------------------

def floored_rel_err(a: np.ndarray, b: np.ndarray) -> float:
    """max_i |a_i - b_i| / (|b_i| + rms(b)); b is the oracle value. 0 for empty or all-zero pairs."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if b.size == 0:
        return 0.0
    rms = math.sqrt(float(np.mean(b * b)))
    den = np.abs(b) + rms
    d = np.abs(a - b)
    if rms == 0.0:
        return float(np.max(d))
    return float(np.max(d / den))
