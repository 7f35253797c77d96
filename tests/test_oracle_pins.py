"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test is chosen so that a plausible slip in the oracle (dropped term, wrong
sign or index, transposed operand, wrong padding) fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

from oracle import moara_oracle as O
from tests.conftest import golden

MODS = ["q", "k", "v", "o", "gate", "up", "down"]


# ---------------------------------------------------------------- bf16 rounding

def test_round_bf16_matches_torch_cast():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(20000) * 10.0 ** g.integers(-40, 38, 20000),
                        [0.0, -0.0, 1.0, -1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 3.0e38, 1e-39, -1e-41]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1.
    assert O.round_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 is halfway between 1+2^-7 and 1+2^-6: even mantissa is 1+2^-6.
    assert O.round_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


# ---------------------------------------------------------------- Phase 3 ranks

def test_final_rank_allocation_row():
    gd = golden("rank_allocations.json")
    types = list(range(7))
    out = O.allocate_ranks(256, types, donors=[0, 1], receivers=[6], delta_r=128)
    assert [out[t] for t in types] == gd["ours_r256"]
    for rb in (256, 512, 1024):
        out = O.allocate_ranks(rb, types, [0, 1], [6], rb // 2)
        assert [out[t] for t in types] == [rb // 2, rb // 2, rb, rb, rb, rb, 2 * rb]
        assert sum(out.values()) == 7 * rb


def test_budget_is_preserved_like_the_random_allocations():
    gd = golden("rank_allocations.json")
    budget = sum(gd["ours_r256"])
    assert budget == 7 * 256
    for row in gd["random_runs"]:
        assert sum(row) == budget
    # the reallocation rule keeps the budget for any integer transfer
    types = list(range(7))
    for D, R, dr in [([0, 1], [6], 64), ([0], [5, 6], 64), ([0, 1, 2, 3], [6], 16), ([2], [4], 200)]:
        out = O.allocate_ranks(256, types, D, R, dr)
        assert sum(out.values()) == budget


def test_non_integer_transfer_rejected():
    with pytest.raises(ValueError):
        O.allocate_ranks(256, list(range(7)), [0, 1, 2], [5, 6], 1)
    with pytest.raises(ValueError):
        O.allocate_ranks(256, list(range(7)), [0, 1], [0], 10)
    with pytest.raises(ValueError):
        O.allocate_ranks(100, list(range(7)), [0, 1], [6], 100)   # donors drop to 0


# ---------------------------------------------------------------- memory model

def _opt_state_mib(sc, vocab, ranks, decompose):
    d, f, L, B = sc["hidden"], sc["intermediate"], sc["layers"], sc["B"]
    shapes = [(d, d), (d, d), (d, d), (d, d), (f, d), (f, d), (d, f)] * L
    rk = [ranks[i % 7] for i in range(7 * L)]
    tgt = O.paper_state_bytes(shapes, rk, [B] * len(shapes), 2, 4, decompose)
    non_target = 2 * 2 * (2 * vocab * d + (2 * L + 1) * d)    # Adam moments of embeddings/head/norms, 2 B each
    return (tgt + non_target) / 2 ** 20


def test_optimizer_state_table_reproduces():
    gd = golden("table11_opt_state.json")
    for name, sc in gd["scales"].items():
        rb = sc["r_base"]
        uni = [rb] * 7
        moa = [rb // 2, rb // 2, rb, rb, rb, rb, 2 * rb]
        got = {
            "baseline": _opt_state_mib(sc, gd["vocab"], uni, False),
            "decomp": _opt_state_mib(sc, gd["vocab"], uni, True),
            "rank": _opt_state_mib(sc, gd["vocab"], moa, False),
            "ours": _opt_state_mib(sc, gd["vocab"], moa, True),
        }
        for k, v in got.items():
            assert round(v, 2) == sc[k], (name, k, v, sc[k])
    sc = gd["scales"]["7B"]
    split = gd["7B_split_MiB"]
    assert round(_opt_state_mib(sc, 32000, [512, 512, 1024, 1024, 1024, 1024, 2048], False)
                 - _opt_state_mib(sc, 32000, [1024] * 7, False)) == split["rank"]
    assert round(_opt_state_mib(sc, 32000, [1024] * 7, True)
                 - _opt_state_mib(sc, 32000, [1024] * 7, False)) == split["decomp"]


def test_memory_model_rejects_transposed_blocking():
    # blocking along rows instead of columns changes the 350M decomposition delta
    gd = golden("table11_opt_state.json")
    sc = gd["scales"]["350M"]
    d, f, L, B = sc["hidden"], sc["intermediate"], sc["layers"], sc["B"]
    shapes_t = [(d, d)] * 4 + [(d, f), (d, f), (f, d)]
    mag_t = sum(2 * 4 * m * math.ceil(n / B) for m, n in shapes_t) * L / 2 ** 20
    assert round(mag_t, 2) != round(sc["decomp"] - sc["baseline"], 2)


# ---------------------------------------------------------------- decomposition

def test_worked_example_decomposition_and_step():
    gd = golden("worked_example.json")
    G = np.array(gd["G"])
    M, V = O.decompose(G, gd["B"], gd["decomp_eps"])
    tol = gd["tolerance"]
    np.testing.assert_allclose(M, gd["M"], atol=tol)
    np.testing.assert_allclose(V, gd["V"], atol=tol)
    s = np.linalg.svd(V, compute_uv=False)
    np.testing.assert_allclose(s, gd["sigma"], atol=tol)
    cfg = O.OracleConfig(block_size=gd["B"], rank=gd["r"], adam_eps=gd["adam_eps"], scale=gd["scale"],
                         beta1=gd["beta1"], beta2=gd["beta2"], decomp_eps=gd["decomp_eps"])
    st = O.init_state(2, 4, cfg)
    assert st.side == gd["side"]
    W = np.zeros((2, 4))
    W1 = O.step(W, G, st, cfg, lr=1.0)
    np.testing.assert_allclose(st.P, gd["P"], atol=tol)
    # the paper's update is W <- W - lr * U
    np.testing.assert_allclose(-W1, gd["U_step1"], atol=tol)
    # same G again: constant-gradient invariance of the Adam step
    W2 = O.step(W1, G, st, cfg, lr=1.0)
    np.testing.assert_allclose(W1 - W2, gd["U_step1"], atol=tol)


def test_partial_block_norm_over_real_columns():
    g = np.random.default_rng(1)
    G = g.standard_normal((5, 11))
    M, V = O.decompose(G, 4)
    assert M.shape == (5, 3)
    np.testing.assert_allclose(M[:, 2], np.linalg.norm(G[:, 8:11], axis=1), rtol=1e-14)
    np.testing.assert_allclose(M[:, 0], np.linalg.norm(G[:, 0:4], axis=1), rtol=1e-14)
    np.testing.assert_allclose(V[:, 9], G[:, 9] / (M[:, 2] + 1e-12), rtol=1e-14)
    assert V.shape == G.shape


def test_block_size_one_gives_sign_and_abs():
    G = np.array([[0.5, -2.0, 0.0, 3.0]])
    M, V = O.decompose(G, 1)
    np.testing.assert_allclose(M, np.abs(G))
    np.testing.assert_allclose(V, np.sign(G), atol=1e-11)


def test_block_at_least_n_is_row_normalisation():
    g = np.random.default_rng(2)
    G = g.standard_normal((4, 7))
    for B in (7, 8, 1024):
        M, V = O.decompose(G, B)
        assert M.shape == (4, 1)
        np.testing.assert_allclose(M[:, 0], np.linalg.norm(G, axis=1), rtol=1e-14)
        np.testing.assert_allclose(np.linalg.norm(V, axis=1), 1.0, rtol=1e-12)


def test_recomposition_identity_and_unit_blocks():
    g = np.random.default_rng(3)
    G = g.standard_normal((6, 20)) * 1e-3
    G[2, 4:8] = 0.0                                  # a zero block
    M, V = O.decompose(G, 4)
    np.testing.assert_allclose(O.recompose(M, V, 4), G * O.rep_b(M / (M + 1e-12), 4, 20), rtol=1e-14, atol=0)
    assert np.all(V[2, 4:8] == 0.0)
    norms = np.sqrt((np.pad(V, ((0, 0), (0, 0))).reshape(6, 5, 4) ** 2).sum(2))
    np.testing.assert_allclose(norms, M / (M + 1e-12), rtol=1e-13)


def test_blockwise_scale_only_moves_magnitude():
    g = np.random.default_rng(4)
    G = g.standard_normal((3, 8))
    M, V = O.decompose(G, 4)
    G2 = G.copy()
    G2[1, 4:8] *= 7.5
    M2, V2 = O.decompose(G2, 4)
    np.testing.assert_allclose(M2[1, 1], 7.5 * M[1, 1], rtol=1e-14)
    np.testing.assert_allclose(V2, V, rtol=1e-12)


def test_proposition1_magnitude_factor_cancels_in_cosine():
    g = np.random.default_rng(5)
    G = g.standard_normal((12, 16))
    B = 4
    M, V = O.decompose(G, B)
    P = O.truncated_svd(V, 3, O.LEFT)
    Vt = P @ (P.T @ V)
    Gt = O.recompose(M, Vt, B)
    for i in range(12):
        for b in range(4):
            sl = slice(b * B, (b + 1) * B)
            c1 = G[i, sl] @ Gt[i, sl] / (np.linalg.norm(G[i, sl]) * np.linalg.norm(Gt[i, sl]))
            c2 = V[i, sl] @ Vt[i, sl] / (np.linalg.norm(V[i, sl]) * np.linalg.norm(Vt[i, sl]))
            assert abs(c1 - c2) < 1e-12


# ---------------------------------------------------------------- truncated SVD

def _jacobi_svd(A, sweeps=30):
    """One-sided (Hestenes) Jacobi SVD, pure Python loops, for tiny matrices."""
    U = np.array(A, dtype=np.float64, copy=True)
    n = U.shape[1]
    Vm = np.eye(n)
    for _ in range(sweeps):
        off = 0.0
        for p in range(n - 1):
            for q in range(p + 1, n):
                a = float(U[:, p] @ U[:, p]); b = float(U[:, q] @ U[:, q]); c = float(U[:, p] @ U[:, q])
                if abs(c) <= 1e-300:
                    continue
                off = max(off, abs(c) / math.sqrt(a * b))
                zeta = (b - a) / (2 * c)
                t = math.copysign(1.0, zeta) / (abs(zeta) + math.sqrt(1 + zeta * zeta))
                cs = 1 / math.sqrt(1 + t * t); sn = cs * t
                up = U[:, p].copy(); U[:, p] = cs * up - sn * U[:, q]; U[:, q] = sn * up + cs * U[:, q]
                vp = Vm[:, p].copy(); Vm[:, p] = cs * vp - sn * Vm[:, q]; Vm[:, q] = sn * vp + cs * Vm[:, q]
        if off < 1e-15:
            break
    s = np.linalg.norm(U, axis=0)
    order = np.argsort(-s)
    return U[:, order] / s[order], s[order], Vm[:, order]


@pytest.mark.parametrize("m,n", [(6, 8), (8, 5), (7, 7)])
def test_truncated_svd_against_hand_written_jacobi(m, n):
    g = np.random.default_rng(m * 10 + n)
    A = g.standard_normal((m, n)) * np.linspace(3.0, 0.2, n)
    Uj, sj, Vj = _jacobi_svd(A if m >= n else A.T)
    if m < n:
        Uj, Vj = Vj, Uj
    sl = np.linalg.svd(A, compute_uv=False)
    np.testing.assert_allclose(sj[:len(sl)], sl, rtol=1e-12)
    r = 3
    side = O.projection_side(m, n)
    P = O.truncated_svd(A, r, side)
    ref = Uj[:, :r] if side == O.LEFT else Vj[:, :r]
    assert O.max_principal_angle(P, ref) < 1e-10


def test_projector_orthonormal_energy_and_full_rank_identity():
    g = np.random.default_rng(7)
    G = g.standard_normal((10, 24))
    _, V = O.decompose(G, 8)
    s = np.linalg.svd(V, compute_uv=False)
    for r in (1, 4, 10):
        P = O.truncated_svd(V, r, O.LEFT)
        np.testing.assert_allclose(P.T @ P, np.eye(r), atol=1e-12)
        np.testing.assert_allclose(np.linalg.norm(P.T @ V) ** 2, np.sum(s[:r] ** 2), rtol=1e-12)   # Eckart-Young
    P = O.truncated_svd(V, 10, O.LEFT)
    np.testing.assert_allclose(P @ P.T, np.eye(10), atol=1e-12)
    M, V = O.decompose(G, 8)
    np.testing.assert_allclose(O.recompose(M, P @ (P.T @ V), 8), G * O.rep_b(M / (M + 1e-12), 8, 24), atol=1e-12)
    # right side: Q spans the top right singular vectors
    Q = O.truncated_svd(V.T, 4, O.RIGHT)
    np.testing.assert_allclose(Q.T @ Q, np.eye(4), atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(V.T @ Q) ** 2, np.sum(s[:4] ** 2), rtol=1e-12)


def test_canonical_signs():
    P = np.array([[0.1, -0.9], [-0.8, 0.2], [0.3, 0.9]])
    C = O.canonical_signs(P)
    np.testing.assert_allclose(C[:, 0], -P[:, 0])      # largest |.| is -0.8 -> flip
    np.testing.assert_allclose(C[:, 1], -P[:, 1])      # tie 0.9: lowest index (-0.9) decides -> flip


def test_principal_angle_helper():
    th = 0.3
    A = np.array([[1.0], [0.0], [0.0]])
    B = np.array([[math.cos(th)], [math.sin(th)], [0.0]])
    assert abs(O.max_principal_angle(A, B) - th) < 1e-14
    assert O.max_principal_angle(A, -A * 3) < 1e-14


# ---------------------------------------------------------------- Adam and the step

def test_identity_projection_without_decomposition_is_torch_adam():
    """decompose=False with P = I (r = m, LEFT) must be exactly torch.optim.Adam."""
    g = np.random.default_rng(8)
    m, n = 4, 6
    cfg = O.OracleConfig(block_size=2, rank=m, decompose=False, refresh_interval=0, scale=1.0,
                         beta1=0.9, beta2=0.999, adam_eps=1e-8)
    st = O.init_state(m, n, cfg)
    st.P = np.eye(m)
    W = g.standard_normal((m, n))
    p = torch.nn.Parameter(torch.from_numpy(W.copy()))
    opt = torch.optim.Adam([p], lr=0.01, betas=(0.9, 0.999), eps=1e-8)
    for t in range(5):
        G = g.standard_normal((m, n))
        W = O.step(W, G, st, cfg, lr=0.01)
        p.grad = torch.from_numpy(G.copy())
        opt.step()
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=0, atol=1e-13)


def test_first_step_closed_forms_and_constant_gradient():
    g = np.random.default_rng(9)
    G = g.standard_normal((8, 12))
    cfg = O.OracleConfig(block_size=4, rank=3, scale=1.0)
    st = O.init_state(8, 12, cfg)
    M, V = O.decompose(G, 4)
    P = O.truncated_svd(V, 3, O.LEFT)
    R = P.T @ V
    W0 = np.zeros((8, 12))
    W1 = O.step(W0, G, st, cfg, lr=1.0)
    N1 = R / (np.abs(R) + cfg.adam_eps)
    dM1 = M / (M + cfg.adam_eps)
    np.testing.assert_allclose(-W1, O.rep_b(dM1, 4, 12) * (P @ N1), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(st.exp_avg, 0.1 * R, rtol=1e-14)
    np.testing.assert_allclose(st.exp_avg_sq, 0.001 * R * R, rtol=1e-14)
    W2 = O.step(W1, G, st, cfg, lr=1.0)
    W3 = O.step(W2, G, st, cfg, lr=1.0)
    np.testing.assert_allclose(W2 - W3, W0 - W1, rtol=1e-9, atol=1e-15)


def test_zero_gradient_zero_moments_is_a_no_op():
    cfg = O.OracleConfig(block_size=4, rank=2, refresh_interval=0)
    st = O.init_state(6, 8, cfg)
    st.P = np.linalg.qr(np.random.default_rng(0).standard_normal((6, 2)))[0]
    W = np.random.default_rng(1).standard_normal((6, 8))
    W1 = O.step(W, np.zeros((6, 8)), st, cfg, lr=0.1)
    np.testing.assert_array_equal(W1, W)


def test_right_side_uses_state_m_by_r():
    g = np.random.default_rng(10)
    m, n = 12, 5
    cfg = O.OracleConfig(block_size=2, rank=2, scale=1.0)
    st = O.init_state(m, n, cfg)
    assert st.side == O.RIGHT and st.exp_avg.shape == (m, 2)
    G = g.standard_normal((m, n))
    W1 = O.step(np.zeros((m, n)), G, st, cfg, lr=1.0)
    M, V = O.decompose(G, 2)
    Q = O.truncated_svd(V, 2, O.RIGHT)
    R = V @ Q
    N1 = R / (np.abs(R) + cfg.adam_eps)
    np.testing.assert_allclose(-W1, O.rep_b(M / (M + 1e-8), 2, n) * (N1 @ Q.T), rtol=1e-12, atol=1e-15)


def test_square_matrix_takes_the_printed_left_form():
    """Algorithm 1 is written in the left form (R = P^T V, dV = P N, P the top-r left
    singular vectors); with m = n neither side keeps a smaller state, and the printed
    form is the one taken. The singular vectors come from the hand-written Jacobi SVD."""
    g = np.random.default_rng(12)
    n, r = 6, 2
    cfg = O.OracleConfig(block_size=2, rank=r, scale=1.0)
    st = O.init_state(n, n, cfg)
    assert st.side == O.LEFT and st.exp_avg.shape == (r, n)
    G = g.standard_normal((n, n)) * np.linspace(3.0, 0.3, n)
    W1 = O.step(np.zeros((n, n)), G, st, cfg, lr=1.0)
    M, V = O.decompose(G, 2)
    Uj, sj, Vj = _jacobi_svd(V)
    assert sj[r - 1] - sj[r] > 1e-3 * sj[0]          # the top-r subspace is separated
    mag = O.rep_b(M / (M + 1e-8), 2, n)
    P = Uj[:, :r]
    R = P.T @ V
    left = mag * (P @ (R / (np.abs(R) + cfg.adam_eps)))
    np.testing.assert_allclose(-W1, left, rtol=1e-10, atol=1e-14)
    Q = Vj[:, :r]                                     # the right form moves W differently here
    Rq = V @ Q
    right = mag * ((Rq / (np.abs(Rq) + cfg.adam_eps)) @ Q.T)
    assert np.max(np.abs(right - left)) > 1e-2


def test_refresh_schedule_and_moment_continuity():
    g = np.random.default_rng(11)
    cfg = O.OracleConfig(block_size=4, rank=2, refresh_interval=3)
    st = O.init_state(6, 8, cfg)
    Ps = []
    for t in range(7):
        O.step(np.zeros((6, 8)), g.standard_normal((6, 8)), st, cfg, lr=0.1)
        Ps.append(st.P.copy())
    # refreshes at t=0,3,6: P constant on [0,2], [3,5]
    assert np.array_equal(Ps[0], Ps[1]) and np.array_equal(Ps[1], Ps[2])
    assert not np.array_equal(Ps[2], Ps[3])
    assert np.array_equal(Ps[3], Ps[5]) and not np.array_equal(Ps[5], Ps[6])
    assert st.t == 7 and np.any(st.exp_avg != 0)


def test_zero_direction_keeps_previous_projector():
    cfg = O.OracleConfig(block_size=4, rank=2, refresh_interval=1)
    st = O.init_state(6, 8, cfg)
    O.step(np.zeros((6, 8)), np.zeros((6, 8)), st, cfg, lr=0.1)
    np.testing.assert_array_equal(st.P, np.eye(6, 2))
    G = np.random.default_rng(0).standard_normal((6, 8))
    O.step(np.zeros((6, 8)), G, st, cfg, lr=0.1)
    P1 = st.P.copy()
    O.step(np.zeros((6, 8)), np.zeros((6, 8)), st, cfg, lr=0.1)
    np.testing.assert_array_equal(st.P, P1)


def test_bf16_weight_path_rounds_update_then_result():
    cfg = O.OracleConfig(block_size=2, rank=1, refresh_interval=0, weight_dtype="bf16", scale=0.25)
    st = O.init_state(1, 2, cfg)
    st.P = np.array([[1.0]])
    W = np.array([[1.0, -1.0]])
    W1 = O.step(W, np.array([[3.0, -4.0]]), st, cfg, lr=2 ** -10)
    # update magnitude 0.25 * 1 * dM(~1) * N(~1) = ~0.25, times lr 2^-10 is below half a bf16 ulp at 1.0
    np.testing.assert_array_equal(W1, W)
    W2 = O.step(W, np.array([[3.0, -4.0]]), st, cfg, lr=2 ** -5)
    assert np.all(O.round_bf16(W2) == W2) and np.all(W2 != W)


def _fx(a):
    from fractions import Fraction
    return np.vectorize(lambda s: float(Fraction(s)), otypes=[np.float64])(np.array(a, dtype=object))


@pytest.mark.parametrize("side", ["left", "right"])
@pytest.mark.parametrize("weights", ["f32", "bf16"])
def test_bf16_operand_step_hand_derived(side, weights):
    """Hand-derived one-step fixture with bf16 GEMM operands (reading 19) and, for bf16
    weights, the cast of the recomposed update before it is applied (Appendix D).
    Where each rounding sits is visible in the result: the moments pin the rounding
    of V and P in the projection; the fp32-weight update pins the rounding of N (and of
    P in the back-projection) to 1e-12; the bf16-weight result differs from the one
    without the inner cast of U in every element chosen for it."""
    gd = golden("bf16_operand_step.json")
    cf, c = gd["config"], gd["cases"][side]
    G = np.array(c["G"], dtype=np.float64)
    m, n = G.shape
    cfg = O.OracleConfig(block_size=cf["block_size"], rank=cf["rank"], beta1=cf["beta1"], beta2=cf["beta2"],
                         adam_eps=cf["adam_eps"], decomp_eps=cf["decomp_eps"], scale=cf["scale"],
                         refresh_interval=1, weight_dtype=weights, operand_dtype="bf16")
    st = O.init_state(m, n, cfg)
    assert st.side == side
    W0 = _fx(c["W0"])
    W1 = O.step(W0, G, st, cfg, lr=cf["lr"])
    # the projector is the exact top singular vector; the step uses its bf16 copy
    np.testing.assert_allclose(O.round_bf16(st.P).ravel(), _fx(c["bf16_P"]), rtol=0, atol=0)
    R = _fx(c["R"]).reshape(st.exp_avg.shape)
    np.testing.assert_allclose(st.exp_avg, (1 - cf["beta1"]) * R, rtol=1e-12, atol=0)
    np.testing.assert_allclose(st.exp_avg_sq, (1 - cf["beta2"]) * R * R, rtol=1e-12, atol=0)
    M = np.array([[float(np.hypot(*G[i, j:j + 2])) for j in range(0, n, 2)] for i in range(m)])
    np.testing.assert_allclose(st.mag_avg, (1 - cf["beta1"]) * M, rtol=1e-12)
    if weights == "f32":
        np.testing.assert_allclose(W1, _fx(c["W1_f32_weights"]), rtol=1e-12, atol=1e-15)
    else:
        ref, other = _fx(c["W1_bf16_weights"]), _fx(c["W1_bf16_weights_without_inner_cast"])
        assert np.count_nonzero(ref != other) >= 6
        np.testing.assert_array_equal(W1, ref)


def test_bf16_direction_moments_two_steps_hand_derived():
    """Two steps with 2-byte direction moments (b_V = 2, Appendix G) and fp32 magnitude
    states (Appendix D). m = 1, so P = [[1]] and R = V exactly; betas 1/2 and 3/4 are
    exact in binary, so every rounding below is a bf16 rounding of a stored moment.

    G1 = [255, 32 | 5, 12] (B = 2): M = (257, 13), V = x1 = (255/257, 32/257, 5/13, 12/13).
    Step 1 stores e = x1/2 and q = x1^2/4 rounded to nearest-even bf16 (8 significant
    bits): 255/514 = 254.007 * 2^-9 -> 127/256; 16/257 = 255.004 * 2^-12 -> 255/4096;
    5/26 = 196.92 * 2^-10 -> 197/1024 (truncation would give 196); 6/13 = 236.31 * 2^-9
    -> 59/128; 65025/264196 = 252.03 * 2^-10 -> 63/256; 256/66049 = 254.02 * 2^-16 ->
    127/32768; 25/676 = 151.48 * 2^-12 -> 151/4096; 36/169 = 218.13 * 2^-10 -> 109/512.
    Step 2 (G2 = [32, 255 | 12, 5]) starts from those stored values; its last e and its
    third q round differently when step 1 is taken unrounded (27/64 and 123/512 here).
    The magnitude states stay exact: e_M = M/2 = (128.5, 6.5), where bf16 would give 128.
    """
    from fractions import Fraction as Fr
    cfg = O.OracleConfig(block_size=2, rank=1, beta1=0.5, beta2=0.75, adam_eps=0.25, decomp_eps=0.0,
                         scale=0.25, refresh_interval=200, moment_dtype="bf16")
    st = O.init_state(1, 4, cfg)
    W0 = np.zeros((1, 4))
    W1 = O.step(W0, np.array([[255.0, 32.0, 5.0, 12.0]]), st, cfg, lr=1.0)
    assert np.array_equal(st.P, [[1.0]])
    e1 = [Fr(127, 256), Fr(255, 4096), Fr(197, 1024), Fr(59, 128)]
    q1 = [Fr(63, 256), Fr(127, 32768), Fr(151, 4096), Fr(109, 512)]
    np.testing.assert_array_equal(st.exp_avg.ravel(), [float(v) for v in e1])
    np.testing.assert_array_equal(st.exp_avg_sq.ravel(), [float(v) for v in q1])
    np.testing.assert_array_equal(st.mag_avg.ravel(), [128.5, 6.5])

    def expect_update(e, q, mag_e, mag_q, t):
        # N and dM from the stored moments at step t; U = scale * Rep_B(dM) * N
        c1, c2 = 1 - 0.5 ** t, 1 - 0.75 ** t
        N = [float(a) / c1 / (math.sqrt(float(b) / c2) + 0.25) for a, b in zip(e, q)]
        dM = [a / c1 / (math.sqrt(b / c2) + 0.25) for a, b in zip(mag_e, mag_q)]
        return np.array([0.25 * dM[j // 2] * N[j] for j in range(4)])

    np.testing.assert_allclose(W0 - W1, [expect_update(e1, q1, [128.5, 6.5], [16512.25, 42.25], 1)],
                               rtol=1e-13, atol=0)
    W2 = O.step(W1, np.array([[32.0, 255.0, 12.0, 5.0]]), st, cfg, lr=1.0)
    e2 = [Fr(159, 512), Fr(135, 256), Fr(143, 256), Fr(27, 64)]
    q2 = [Fr(193, 1024), Fr(255, 1024), Fr(123, 512), Fr(201, 1024)]
    np.testing.assert_array_equal(st.exp_avg.ravel(), [float(v) for v in e2])
    np.testing.assert_array_equal(st.exp_avg_sq.ravel(), [float(v) for v in q2])
    mag_e = [0.5 * 128.5 + 0.5 * 257, 0.5 * 6.5 + 0.5 * 13]
    mag_q = [0.75 * 16512.25 + 0.25 * 257 ** 2, 0.75 * 42.25 + 0.25 * 13 ** 2]
    np.testing.assert_array_equal(st.mag_avg.ravel(), mag_e)
    np.testing.assert_allclose(W1 - W2, [expect_update(e2, q2, mag_e, mag_q, 2)], rtol=1e-13, atol=0)


def test_floored_metric():
    b = np.array([1.0, 0.0, -2.0])
    assert O.floored_rel_err(b, b) == 0.0
    a = b + np.array([0.0, 1e-3, 0.0])
    assert abs(O.floored_rel_err(a, b) - 1e-3 / math.sqrt(5 / 3)) < 1e-15


# ---------------------------------------------------------------- alignment diagnostic (Section 3.2)

def _orth(rng, n, r):
    return np.linalg.qr(rng.standard_normal((n, n)))[0][:, :r]


@pytest.mark.parametrize("shape", [(6, 10), (10, 6)])
def test_alignment_full_rank_projector_is_one(shape):
    # P P^T = I on the projected side: G_recon = Rep_B(M) V = G (up to eps), S = 1
    rng = np.random.default_rng(1)
    G = rng.standard_normal(shape)
    s = min(shape)
    for B in (1, 3, 4, 64):
        assert abs(O.alignment(G, _orth(rng, s, s), B) - 1.0) < 1e-12


@pytest.mark.parametrize("shape", [(6, 10), (10, 6)])
def test_alignment_without_decomposition_is_projected_norm_ratio(shape):
    # cos(G, P P^T G) = ||P^T G|| / ||G|| (LEFT), cos(G, G Q Q^T) = ||G Q|| / ||G|| (RIGHT)
    rng = np.random.default_rng(2)
    G = rng.standard_normal(shape)
    P = _orth(rng, min(shape), 2)
    ref = np.linalg.norm(P.T @ G if shape[0] <= shape[1] else G @ P) / np.linalg.norm(G)
    assert abs(O.alignment(G, P, 4, decompose_on=False) - ref) < 1e-12


def test_alignment_support_inside_and_outside_the_subspace():
    # LEFT 4 x 9: G lives in rows 0-1. V then lives there too (zero blocks stay zero), so
    # P = span(e0, e1) reconstructs G exactly and its complement reconstructs nothing.
    rng = np.random.default_rng(3)
    G = np.zeros((4, 9))
    G[:2] = rng.standard_normal((2, 9))
    I = np.eye(4)
    assert abs(O.alignment(G, I[:, :2], 4) - 1.0) < 1e-12
    assert O.alignment(G, I[:, 2:], 4) == 0.0
    # RIGHT 9 x 4: the same along columns 0-1 (the projector acts on the column side)
    H = np.zeros((9, 4))
    H[:, :2] = rng.standard_normal((9, 2))
    assert abs(O.alignment(H, I[:, :2], 2) - 1.0) < 1e-12
    assert O.alignment(H, I[:, 2:], 2) == 0.0


def test_alignment_block_size_one_keeps_the_projected_columns():
    # B = 1: M = |G|, V = sign(G); RIGHT 3 x 2 with Q = e0 keeps column 0 of V, so
    # G_recon = [G[:, 0], 0] and S = ||G[:, 0]|| / ||G||.
    G = np.array([[3.0, -1.0], [-2.0, 4.0], [0.5, 2.0]])
    S = O.alignment(G, np.array([[1.0], [0.0]]), 1)
    assert abs(S - np.linalg.norm(G[:, 0]) / np.linalg.norm(G)) < 1e-12


def test_alignment_depends_on_the_subspace_only():
    # P -> P O (O orthogonal, including column sign flips) leaves P P^T and S unchanged;
    # a positive scale of G changes neither M's ratios nor V
    rng = np.random.default_rng(4)
    G = rng.standard_normal((8, 13))
    P = _orth(rng, 8, 3)
    S = O.alignment(G, P, 4)
    Orot = np.linalg.qr(rng.standard_normal((3, 3)))[0] @ np.diag([1.0, -1.0, 1.0])
    assert abs(O.alignment(G, P @ Orot, 4) - S) < 1e-12
    assert abs(O.alignment(7.5 * G, P, 4) - S) < 1e-12
    assert 0.0 < S < 1.0


def test_module_alignment_is_the_mean_per_type():
    # three samples of type 0, skewed so that the mean (0.4) is not the median (0.2)
    got = O.module_alignment([(0, 0.2), (3, 1.0), (0, 0.9), (6, -0.5), (0, 0.1)])
    assert got == pytest.approx({0: 0.4, 3: 1.0, 6: -0.5})


def test_flatten_keeps_axis_zero_and_blocks_run_over_the_flattened_columns():
    # a 2 x 3 x 4 tensor is the 2 x 12 matrix of its rows; with B = 4 the blocks of
    # row 0 are its three axis-1 slices (12 contiguous values split in runs of 4)
    G = np.arange(24, dtype=np.float64).reshape(2, 3, 4) - 11.5
    F = O.flatten(G)
    assert F.shape == (2, 12)
    np.testing.assert_array_equal(F[1], G[1].ravel())
    M, _ = O.decompose(F, 4)
    np.testing.assert_allclose(M[0], [np.linalg.norm(G[0, j]) for j in range(3)], rtol=1e-15)
