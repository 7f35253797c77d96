"""Parity of the HIP path (through the C ABI) with the CPU oracle, element by element.

Tolerances: max floored relative error 1e-4 when weights and GEMM operands are
fp32; 2e-2 when bf16 operands or bf16 weights are used (the oracle then applies
the same bf16 roundings of V, P, N and of the update). Projector refreshes are
compared by principal angles (<= 1e-3 rad), since singular vectors are only
defined up to sign and rotation within (near-)degenerate clusters.
"""
import math

import numpy as np
import pytest

import workloads as WL
from oracle import moara_oracle as O
from tests.harness import (TOL_BF16, TOL_F32, TOL_UPDATE_F32, Case, case_from_workload, compare, compare_update,
                           gpu_state, have_gpu, adam_sensitivity, oracle_cfg, oracle_projector, rng, slices_of,
                           to_dev, to_np)

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs an MI355X GPU")]


def _M():
    from paper_2609_15037_amd import moara as M
    return M


def _grad(c: Case, seed, step, i):
    m, n, _ = c.shapes[i]
    return (c.grad_std * rng(seed, 2, step, i).standard_normal((m, n))).astype(np.float32)


def _weights(c: Case, seed):
    return [(c.weight_std * rng(seed, 1, i).standard_normal((m, n))).astype(np.float32)
            for i, (m, n, _) in enumerate(c.shapes)]


def step_parity(c: Case, steps: int, seed: int = 0, grad_fn=None, check_every=False, misalign: bool = False,
                refresh_misaligned: bool = False, max_masked: float = 0.1):
    """Steps on the GPU and in the oracle from the same inputs, from zero moments. The
    projector comes from the oracle's SVD (set into the library). With refresh_misaligned
    the library first refreshes from the first gradients placed at unaligned addresses;
    its projector must lie within 1e-3 rad of the oracle's, which then replaces it.

    At the fp32 bar, elements fed by first-step Adam outputs whose fp32 forward error
    estimate is large (adam_sensitivity) are held to TOL_MASKED instead; at most
    `max_masked` of the elements may be so masked (W and update masks alike). The bf16 bar
    applies to every element. The step-1 sign flips of the projected gradient (exp_avg)
    against the oracle are counted and printed."""
    import torch
    M = _M()
    tol = TOL_F32 if (c.weight_dtype == "f32" and c.operand_dtype == "f32") else TOL_BF16
    n = len(c.shapes)
    grad_fn = grad_fn or (lambda t, i: _grad(c, seed, t, i))
    st = gpu_state(c)
    Wd = [to_dev(w, c.weight_dtype, offset=1 if misalign else 0) for w in _weights(c, seed)]
    W0 = [to_np(w) for w in Wd]
    Wo = [w.copy() for w in W0]
    ocfg = [oracle_cfg(c, i) for i in range(n)]
    ost = [O.init_state(c.shapes[i][0], c.shapes[i][1], ocfg[i]) for i in range(n)]
    report = {}
    masks = [np.zeros(c.shapes[i][:2], dtype=bool) for i in range(n)]     # W check (dN > 0.1)
    masks_u = [np.zeros(c.shapes[i][:2], dtype=bool) for i in range(n)]   # update check (dN > 0.01)
    use_mask = tol == TOL_F32
    for t in range(steps):
        Gs = [grad_fn(t, i) for i in range(n)]
        if t == 0 and refresh_misaligned:
            M.moara_refresh_projector(st, [to_dev(g, "f32", offset=1) for g in Gs])
            torch.cuda.synchronize()
            for i in range(n):
                Pg = M.moara_get_tensor(st, i, M.MOARA_T_P).astype(np.float64)
                np.testing.assert_allclose(Pg.T @ Pg, np.eye(Pg.shape[1]), atol=2e-5)
                ang = O.max_principal_angle(Pg, oracle_projector(Gs[i], c, i))
                assert ang <= 1e-3, f"matrix {i}: refresh from unaligned buffers: principal angle {ang:.2e}"
        if t == 0:
            for i in range(n):
                P = oracle_projector(Gs[i], c, i)
                M.moara_set_tensor(st, i, M.MOARA_T_P, P)
                ost[i].P = P
        Gd = [to_dev(g, "f32", offset=1 if misalign else 0) for g in Gs]
        print(f"[parity] step {t} n={n} B={c.block_size} op={c.operand_dtype} w={c.weight_dtype}", flush=True)
        M.moara_step(st, Wd, Gd, lr=c.lr)
        for i in range(n):
            Wo[i] = O.step(Wo[i], Gs[i], ost[i], ocfg[i], c.lr)
            V = O.decompose(Gs[i], c.block_size)[1] if c.decompose else Gs[i].astype(np.float64)
            dN = adam_sensitivity(V, ost[i].P, ost[i].side, ost[i].exp_avg_sq, ost[i].t, c.beta2, c.adam_eps)
            masks[i] |= slices_of(dN > 0.1, ost[i].side, c.shapes[i][:2])
            masks_u[i] |= slices_of(dN > 0.01, ost[i].side, c.shapes[i][:2])
        torch.cuda.synchronize()
        if t == 0:
            flips = tot = 0
            for i in range(n):
                eg, eo = M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG), ost[i].exp_avg
                nz = eo != 0.0
                flips += int(np.sum(np.sign(eg[nz]) != np.sign(eo[nz])))
                tot += int(nz.sum())
            report["step1_sign_flips"] = flips
            print(f"[parity] step-1 sign flips of the projected gradient: {flips} of {tot}", flush=True)
        if check_every or t == steps - 1:
            for i in range(n):
                Wg = to_np(Wd[i])
                compare(f"W[{i}]", Wg, Wo[i], tol, report, masks[i] if use_mask else None)
                if c.weight_dtype == "f32":
                    compare_update(f"dW[{i}]", Wg - W0[i], Wo[i] - W0[i], max(tol, TOL_UPDATE_F32), report,
                                   masks_u[i] if use_mask else None)
                compare(f"exp_avg[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG), ost[i].exp_avg, tol, report)
                compare(f"exp_avg_sq[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG_SQ), ost[i].exp_avg_sq, tol, report)
                if c.decompose:
                    compare(f"mag_avg[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_MAG_AVG), ost[i].mag_avg, tol, report)
                    compare(f"mag_avg_sq[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_MAG_AVG_SQ), ost[i].mag_avg_sq, tol, report)
                assert M.moara_get_tensor(st, i, M.MOARA_T_STEP) == t + 1
    worst = max(v for k, v in report.items() if not k.endswith("masked_frac") and k != "step1_sign_flips")
    masked = max([v for k, v in report.items() if k.endswith("masked_frac")] or [0.0])
    print(f"[parity] worst floored rel err {worst:.3e} (tol {tol:.0e}); elements masked as "
          f"ill-conditioned {masked:.1e}", flush=True)
    assert masked <= max_masked, f"{masked:.3f} of the elements masked as ill-conditioned (limit {max_masked})"
    return report


# ------------------------------------------------------------------ step parity

def test_layer_d256_fp32_ten_steps():
    c = case_from_workload(WL.WORKLOADS["layer_d256"], operand_dtype="f32")
    step_parity(c, 10, check_every=True, max_masked=0.06)


def test_layer_d256_bf16_operands():
    c = case_from_workload(WL.WORKLOADS["layer_d256"], operand_dtype="bf16")
    rep = step_parity(c, 10)
    # the oracle rounds the same operands to bf16, so the moments agree far below the bar
    assert max(v for k, v in rep.items() if k.startswith("exp_avg")) < 1e-3


def test_llama300m_layers_bf16():
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0, 23])
    c = case_from_workload(wl)
    step_parity(c, 3, grad_fn=lambda t, i: WL.grad_np(wl, i, t))


@pytest.mark.parametrize("name", ["llama32_300m", "qwen25_350m", "deepseek_v2_350m"])
def test_350m_model_family_layers(name):
    # GQA key/value projections (256 x 1024, r = 128 and the full rank 256) and the
    # DeepSeek-V2 MLA projections (q_a, q_b, kv_a, kv_b) at B = 32
    wl = WL.subset(WL.WORKLOADS[name], [0, 23])
    c = case_from_workload(wl)
    step_parity(c, 2, grad_fn=lambda t, i: WL.grad_np(wl, i, t))


def test_llama300m_layer_misaligned_caller_buffers():
    # W and G one element past a 16-byte boundary: no bf16 V workspace this step, the
    # projection and back-projection take the grouped fallback GEMM, which must read and
    # write the blocked projector copies and N
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [3])
    c = case_from_workload(wl)
    step_parity(c, 3, grad_fn=lambda t, i: WL.grad_np(wl, i, t), misalign=True)


def test_llama300m_layer_refresh_from_unaligned_buffers_then_steps():
    # the refresh and the steps read gradients at unaligned addresses (the paths for caller
    # buffers the large-tile kernels cannot take)
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [7])
    c = case_from_workload(wl)
    step_parity(c, 2, grad_fn=lambda t, i: WL.grad_np(wl, i, t), refresh_misaligned=True, misalign=True)


@pytest.mark.parametrize("B", [1, 16, 32, 64, 128, 512, 1024, 48, 20, 256, 1000])   # the block sizes of Fig. 3, then odd ones
def test_ragged_shapes_and_block_sizes(B):
    # several tiles in every dimension plus ragged tails; n % 4 != 0 forces scalar loads
    c = Case(shapes=[(300, 452, WL.Q), (452, 300, WL.GATE), (129, 1000, WL.DOWN), (77, 130, WL.K), (5, 3, WL.V)],
             ranks=[37, 50, 64, 9, 2], block_size=B)
    step_parity(c, 3)


@pytest.mark.parametrize("op", ["f32", "bf16"])
def test_ragged_bf16_weights(op):
    c = Case(shapes=[(300, 452, WL.Q), (452, 300, WL.GATE), (200, 136, WL.UP)], ranks=[40, 33, 136],
             block_size=64, weight_dtype="bf16", operand_dtype=op, weight_std=0.02)
    step_parity(c, 3)


def test_decompose_off_is_galore_direction():
    c = Case(shapes=[(256, 384, WL.Q), (384, 256, WL.UP)], ranks=[32, 48], block_size=64, decompose=False)
    step_parity(c, 4)


# ------------------------------------------------------------------ refresh

def _angles_vs_oracle(c: Case, Gs, P_gpu_list, bar=1e-3):
    worst = 0.0
    for i, G in enumerate(Gs):
        _, V = O.decompose(G, c.block_size)
        side = O.projection_side(*G.shape)
        ref = O.truncated_svd(V, c.ranks[i], side)
        Pg = P_gpu_list[i].astype(np.float64)
        assert Pg.shape == ref.shape
        np.testing.assert_allclose(Pg.T @ Pg, np.eye(Pg.shape[1]), atol=2e-5)
        ang = O.max_principal_angle(Pg, ref)
        worst = max(worst, ang)
        assert ang <= bar, f"matrix {i}: principal angle {ang:.2e} rad"
        # ordering: the Ritz values follow the singular values
        sv = np.linalg.svd(V, compute_uv=False)[: c.ranks[i]]
        X = V if side == O.RIGHT else V.T
        ritz = np.linalg.norm(X @ Pg, axis=0)
        np.testing.assert_allclose(ritz, sv, rtol=1e-3)
    return worst


def test_refresh_layer_d256_principal_angles():
    import torch
    M = _M()
    c = case_from_workload(WL.WORKLOADS["layer_d256"])
    st = gpu_state(c)
    Gs = [_grad(c, 3, 0, i) for i in range(len(c.shapes))]
    print("[refresh] layer_d256", flush=True)
    M.moara_refresh_projector(st, [to_dev(g, "f32") for g in Gs])
    torch.cuda.synchronize()
    Ps = [M.moara_get_tensor(st, i, M.MOARA_T_P) for i in range(len(Gs))]
    worst = _angles_vs_oracle(c, Gs, Ps)
    print(f"[refresh] worst principal angle {worst:.2e}", flush=True)
    for i in range(len(Gs)):   # the Jacobi sweeps met their tolerance and kept all r directions
        info = M.moara_refresh_info(st, i)
        assert info["converged"] and info["rank"] == c.ranks[i] and info["offdiag"] < 1e-7, (i, info)


def test_refresh_lowrank_llama300m_layer():
    import torch
    M = _M()
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0])
    c = case_from_workload(wl)
    st = gpu_state(c)
    Gs = [WL.grad_np(wl, i, 0) for i in range(len(wl.matrices))]
    print("[refresh] llama_300m layer 0", flush=True)
    M.moara_refresh_projector(st, [to_dev(g, "f32") for g in Gs])
    torch.cuda.synchronize()
    Ps = [M.moara_get_tensor(st, i, M.MOARA_T_P) for i in range(len(Gs))]
    worst = _angles_vs_oracle(c, Gs, Ps)
    print(f"[refresh] worst principal angle {worst:.2e}", flush=True)
    for i in range(len(Gs)):
        info = M.moara_refresh_info(st, i)
        assert info["converged"] and info["rank"] == c.ranks[i], (i, info)


def test_refresh_bf16_path_with_fp32_orthonormalisation():
    """A bf16-path matrix whose subspace width is not a multiple of 32 (r = 40, w = 80) keeps
    the early orthonormalisations of its refresh chunk on the fp32 product and the transpose
    (the split bf16 form needs K = w in 32-steps): that path must still match the oracle."""
    import dataclasses
    import torch
    M = _M()
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0])
    rt = list(wl.rank_table)
    rt[WL.Q] = 40
    wl = dataclasses.replace(wl, rank_table=tuple(rt))
    c = case_from_workload(wl)
    st = gpu_state(c)
    Gs = [WL.grad_np(wl, i, 0) for i in range(len(wl.matrices))]
    print("[refresh] llama_300m layer 0, q at r = 40", flush=True)
    M.moara_refresh_projector(st, [to_dev(g, "f32") for g in Gs])
    torch.cuda.synchronize()
    Ps = [M.moara_get_tensor(st, i, M.MOARA_T_P) for i in range(len(Gs))]
    worst = _angles_vs_oracle(c, Gs, Ps)
    print(f"[refresh] worst principal angle {worst:.2e}", flush=True)
    for i in range(len(Gs)):
        info = M.moara_refresh_info(st, i)
        assert info["converged"] and info["rank"] == c.ranks[i], (i, info)


def test_refresh_forced_side_on_the_longer_dimension():
    """A projector forced onto the longer side (LEFT on a 384 x 256 matrix: s = 384 > L = 256)
    is still the top-r left singular subspace of V; such a refresh keeps the fp32
    orthonormalisation (the split one keeps Z2's parts in buffers sized for s <= 4 L / 3).
    Checked next to an automatic-side matrix of the same state against the oracle."""
    import torch
    M = _M()
    B, rk = 32, 32
    shapes = [(384, 256, WL.Q, rk, M.MOARA_SIDE_LEFT), (256, 384, WL.K, rk, M.MOARA_SIDE_AUTO)]
    cfg = M.moara_default_config(block_size=B, refresh_interval=0, weight_dtype=M.MOARA_BF16,
                                 operand_dtype=M.MOARA_BF16, refresh_oversample=rk, refresh_iters=20)
    st = M.moara_create_state(cfg, M.make_descs(shapes))
    rng = np.random.default_rng(7)
    Gs = []
    for (m, n, *_rest) in shapes:   # low rank plus noise, a decaying spectrum
        U = np.linalg.qr(rng.standard_normal((m, 48)))[0]
        Y = np.linalg.qr(rng.standard_normal((n, 48)))[0]
        Gs.append(((U * np.arange(1, 49) ** -1.0) @ Y.T + 1e-3 * rng.standard_normal((m, n))).astype(np.float32))
    print("[refresh] forced LEFT on 384 x 256", flush=True)
    M.moara_refresh_projector(st, [to_dev(g, "f32") for g in Gs])
    torch.cuda.synchronize()
    for i, G in enumerate(Gs):
        Pg = M.moara_get_tensor(st, i, M.MOARA_T_P).astype(np.float64)
        _, V = O.decompose(G, B)
        ref = O.truncated_svd(V, rk, O.LEFT)   # both matrices project on the left
        assert Pg.shape == ref.shape == (G.shape[0], rk)
        np.testing.assert_allclose(Pg.T @ Pg, np.eye(rk), atol=2e-5)
        ang = O.max_principal_angle(Pg, ref)
        print(f"[refresh] matrix {i}: principal angle {ang:.2e}", flush=True)
        assert ang <= 1e-3
        info = M.moara_refresh_info(st, i)
        assert info["converged"] and info["rank"] == rk, (i, info)


def test_refresh_in_several_chunks_is_bit_identical(monkeypatch):
    """A refresh split into chunks (workspace budget below one layer's need) gives the
    same projectors, bit for bit, as one chunk: every matrix is computed on its own."""
    import torch
    M = _M()
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0])
    c = case_from_workload(wl)
    Gs = [to_dev(WL.grad_np(wl, i, 0), "f32") for i in range(len(wl.matrices))]
    out = []
    for budget in (None, "8"):
        if budget:
            monkeypatch.setenv("MOARA_REFRESH_CHUNK_MIB", budget)
        else:
            monkeypatch.delenv("MOARA_REFRESH_CHUNK_MIB", raising=False)
        st = gpu_state(c)
        print(f"[refresh] llama_300m layer 0, chunk budget {budget or 'default'}", flush=True)
        M.moara_refresh_projector(st, Gs)
        torch.cuda.synchronize()
        out.append([M.moara_get_tensor(st, i, M.MOARA_T_P) for i in range(len(Gs))])
    for a, b in zip(*out):
        assert np.array_equal(a, b)


def test_refresh_inside_step_schedule():
    import torch
    M = _M()
    c = Case(shapes=[(96, 160, WL.Q), (160, 96, WL.GATE)], ranks=[16, 24], block_size=32)
    st = gpu_state(c, refresh_interval=2)
    Wd = [to_dev(w, "f32") for w in _weights(c, 0)]
    seen = []
    for t in range(4):
        Gs = [_grad(c, 5, t, i) for i in range(2)]
        M.moara_step(st, Wd, [to_dev(g, "f32") for g in Gs], lr=1e-3)
        torch.cuda.synchronize()
        Ps = [M.moara_get_tensor(st, i, M.MOARA_T_P) for i in range(2)]
        if t in (0, 2):
            _angles_vs_oracle(c, Gs, Ps)
        seen.append(Ps)
    for i in range(2):
        assert np.array_equal(seen[0][i], seen[1][i]) and np.array_equal(seen[2][i], seen[3][i])
        assert not np.array_equal(seen[1][i], seen[2][i])


def _rank_deficient_grad(kind, m, n, rank, seed):
    """Gradients whose direction tensor V has rank `rank` < r. 'rows': only rows 5.. 5+rank
    of G are nonzero (V keeps those rows, any block size); 'lowrank': G = A B^T of that
    rank, used with one block per row so that V = diag(1/M) G keeps the rank."""
    g = rng(seed, 11, m, n, rank)
    G = np.zeros((m, n))
    if kind == "rows":
        G[5:5 + rank] = g.standard_normal((rank, n))
    else:
        G = g.standard_normal((m, rank)) @ g.standard_normal((rank, n))
    return (1e-3 * G).astype(np.float32)


@pytest.mark.parametrize("op", ["f32", "bf16"])
def test_refresh_rank_deficient_direction(op):
    """V of rank below r (Alg. 1 TruncatedSVD of a rank-deficient V): the projector must stay
    orthonormal, its span must contain range(V), and its leading directions (those with
    nonzero singular values) must match the oracle's; the remaining columns complete the
    basis (any orthonormal completion is a top-r singular basis of V)."""
    import torch
    M = _M()
    specs = [("rows", 96, 160, 16, 3, 32, WL.Q), ("rows", 256, 384, 64, 20, 64, WL.K),
             ("lowrank", 160, 96, 24, 10, 96, WL.GATE), ("lowrank", 384, 256, 64, 40, 256, WL.UP)]
    for (kind, m, n, r, rank, B, mod), seed in ((sp, sd) for sp in specs for sd in (0, 1)):
        c = Case(shapes=[(m, n, mod)], ranks=[r], block_size=B, operand_dtype=op)
        st = gpu_state(c)
        G = _rank_deficient_grad(kind, m, n, rank, seed)
        print(f"[refresh] rank-deficient V: {kind} {m}x{n} r={r} rank(V)={rank} B={B} op={op} seed={seed}",
              flush=True)
        M.moara_refresh_projector(st, [to_dev(G, "f32")])
        torch.cuda.synchronize()
        P = M.moara_get_tensor(st, 0, M.MOARA_T_P).astype(np.float64)
        _, V = O.decompose(G, B)
        side = O.projection_side(m, n)
        X = V if side == O.LEFT else V.T            # columns live in the projected space
        orth = float(np.max(np.abs(P.T @ P - np.eye(r))))
        resid = float(np.linalg.norm(X - P @ (P.T @ X)) / np.linalg.norm(X))
        ref = O.truncated_svd(V, rank, side)
        ang = O.max_principal_angle(P[:, :rank], ref)
        print(f"[refresh]   |P^T P - I| {orth:.2e}, |V - P P^T V|/|V| {resid:.2e}, "
              f"leading-{rank} angle {ang:.2e}", flush=True)
        info = M.moara_refresh_info(st, 0)
        print(f"[refresh]   record {info}", flush=True)
        assert orth <= 2e-5
        assert resid <= 1e-4
        assert ang <= 1e-3
        assert info["rank"] == rank


def test_zero_gradient_refresh_keeps_previous_projector():
    import torch
    M = _M()
    c = Case(shapes=[(64, 96, WL.Q)], ranks=[8], block_size=32)
    st = gpu_state(c)
    with pytest.raises(M.MoaraError):
        M.moara_get_tensor(st, 0, M.MOARA_T_P)
    Z = torch.zeros(64, 96, device="cuda")
    M.moara_refresh_projector(st, [Z])
    P0 = M.moara_get_tensor(st, 0, M.MOARA_T_P)
    np.testing.assert_array_equal(P0, np.eye(64, 8, dtype=np.float32))
    G = to_dev(_grad(c, 1, 0, 0), "f32")
    M.moara_refresh_projector(st, [G])
    P1 = M.moara_get_tensor(st, 0, M.MOARA_T_P)
    M.moara_refresh_projector(st, [Z])
    np.testing.assert_array_equal(M.moara_get_tensor(st, 0, M.MOARA_T_P), P1)


# ------------------------------------------------------------------ state handling

def test_inactive_matrices_are_untouched():
    import torch
    M = _M()
    c = Case(shapes=[(128, 192, WL.EXP_GATE), (128, 192, WL.EXP_UP), (192, 128, WL.EXP_DOWN)], ranks=[16] * 3,
             block_size=64)
    st = gpu_state(c, refresh_interval=3)
    Wd = [to_dev(w, "f32") for w in _weights(c, 0)]
    act = np.array([1, 0, 1], dtype=np.uint8)
    before = to_np(Wd[1]).copy()
    for t in range(4):
        Gs = [to_dev(_grad(c, 2, t, i), "f32") for i in range(3)]
        M.moara_step(st, Wd, Gs, lr=1e-3, active=act)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(Wd[1]), before)
    assert M.moara_get_tensor(st, 1, M.MOARA_T_STEP) == 0
    assert M.moara_get_tensor(st, 0, M.MOARA_T_STEP) == 4
    assert not np.any(M.moara_get_tensor(st, 1, M.MOARA_T_EXP_AVG))


@pytest.mark.parametrize("op,wdt,mom", [("f32", "f32", "f32"), ("bf16", "bf16", "f32"), ("bf16", "bf16", "bf16")])
def test_zero_grad_mode_steps_inactive_matrices_with_zero_gradient(op, wdt, mom):
    """zero_grad_mode 1: an inactive matrix takes the step of G = 0 (Algorithm 1 with a zero
    gradient: M = V = 0, both Adam branches decay their moments, W moves by
    Rep_B(dM) (.) P N). Against the oracle's step(W, 0) with the same projector, and bit for
    bit against mode 0 with the zero gradient passed explicitly as an active matrix."""
    import torch
    M = _M()
    c = Case(shapes=[(128, 192, WL.EXP_GATE), (128, 192, WL.EXP_UP), (192, 128, WL.EXP_DOWN)], ranks=[16] * 3,
             block_size=64, operand_dtype=op, weight_dtype=wdt, weight_std=0.02 if wdt == "bf16" else 1e-3,
             moment_dtype=mom)
    tol = TOL_F32 if op == "f32" else TOL_BF16
    n = 3
    masks = [[1, 1, 1], [1, 0, 1], [0, 0, 1], [1, 1, 0], [0, 1, 0]]
    grads = [[_grad(c, 12, t, i) for i in range(n)] for t in range(len(masks))]
    st = gpu_state(c, zero_grad_mode=1)
    ref = gpu_state(c)
    Wd = [to_dev(w, wdt) for w in _weights(c, 0)]
    Wr = [to_dev(w, wdt) for w in _weights(c, 0)]
    Wo = [to_np(w) for w in Wd]
    ocfg = [oracle_cfg(c, i) for i in range(n)]
    ost = [O.init_state(c.shapes[i][0], c.shapes[i][1], ocfg[i]) for i in range(n)]
    for i in range(n):
        P = oracle_projector(grads[0][i], c, i)
        for s_ in (st, ref):
            M.moara_set_tensor(s_, i, M.MOARA_T_P, P)
        ost[i].P = P
    zero = [torch.zeros(c.shapes[i][:2], device="cuda") for i in range(n)]
    for t, mask in enumerate(masks):
        print(f"[zero-grad] step {t} active {mask} op={op} w={wdt} moments={mom}", flush=True)
        act = np.array(mask, dtype=np.uint8)
        M.moara_step(st, Wd, [to_dev(grads[t][i], "f32") if mask[i] else None for i in range(n)], lr=c.lr,
                     active=act)
        M.moara_step(ref, Wr, [to_dev(grads[t][i], "f32") if mask[i] else zero[i] for i in range(n)], lr=c.lr)
        for i in range(n):
            G = grads[t][i] if mask[i] else np.zeros(c.shapes[i][:2])
            Wo[i] = O.step(Wo[i], G, ost[i], ocfg[i], c.lr)
    torch.cuda.synchronize()
    report = {}
    for i in range(n):
        assert M.moara_get_tensor(st, i, M.MOARA_T_STEP) == len(masks)
        assert torch.equal(Wd[i], Wr[i]), f"matrix {i}: zero_grad_mode 1 differs from an explicit zero gradient"
        for k in (M.MOARA_T_EXP_AVG, M.MOARA_T_EXP_AVG_SQ, M.MOARA_T_MAG_AVG, M.MOARA_T_MAG_AVG_SQ):
            assert np.array_equal(M.moara_get_tensor(st, i, k), M.moara_get_tensor(ref, i, k))
        compare(f"W[{i}]", to_np(Wd[i]), Wo[i], tol, report)
        if wdt == "f32":
            compare_update(f"dW[{i}]", to_np(Wd[i]) - _weights(c, 0)[i], Wo[i] - _weights(c, 0)[i],
                           max(tol, TOL_UPDATE_F32), report)
        compare(f"exp_avg[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG), ost[i].exp_avg, tol, report)
        compare(f"exp_avg_sq[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG_SQ), ost[i].exp_avg_sq, tol, report)
        compare(f"mag_avg[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_MAG_AVG), ost[i].mag_avg, tol, report)
        compare(f"mag_avg_sq[{i}]", M.moara_get_tensor(st, i, M.MOARA_T_MAG_AVG_SQ), ost[i].mag_avg_sq, tol, report)
    print(f"[zero-grad] worst floored rel err {max(report.values()):.3e} (tol {tol:.0e})", flush=True)


def test_zero_grad_mode_first_refresh_sets_canonical_projector():
    """A matrix that is inactive on its first step in zero_grad_mode 1 gets the projector of
    a zero V (the first r canonical basis vectors), zero moments stay zero, W does not move
    (N = 0 at t = 1), and t advances; its refresh on a later active step replaces P."""
    import torch
    M = _M()
    c = Case(shapes=[(96, 160, WL.EXP_GATE), (160, 96, WL.EXP_DOWN)], ranks=[8, 12], block_size=32)
    st = gpu_state(c, refresh_interval=2, zero_grad_mode=1)
    Wd = [to_dev(w, "f32") for w in _weights(c, 0)]
    W0 = [w.clone() for w in Wd]
    M.moara_step(st, Wd, [to_dev(_grad(c, 3, 0, 0), "f32"), None], lr=1e-3, active=[1, 0])
    torch.cuda.synchronize()
    assert torch.equal(Wd[1], W0[1])
    np.testing.assert_array_equal(M.moara_get_tensor(st, 1, M.MOARA_T_P), np.eye(96, 12, dtype=np.float32))
    assert M.moara_get_tensor(st, 1, M.MOARA_T_STEP) == 1
    assert not np.any(M.moara_get_tensor(st, 1, M.MOARA_T_EXP_AVG))
    with pytest.raises(M.MoaraError) as e:   # no refresh record: the library did not refresh it
        M.moara_refresh_info(st, 1)
    assert e.value.status == M.MOARA_E_STATE
    G1 = [_grad(c, 3, t, 1) for t in (1, 2)]
    M.moara_step(st, Wd, [to_dev(_grad(c, 3, 1, 0), "f32"), to_dev(G1[0], "f32")], lr=1e-3)
    M.moara_step(st, Wd, [to_dev(_grad(c, 3, 2, 0), "f32"), to_dev(G1[1], "f32")], lr=1e-3)   # t = 2: refresh
    torch.cuda.synchronize()
    _angles_vs_oracle(Case(shapes=[c.shapes[1]], ranks=[12], block_size=32), [G1[1]],
                      [M.moara_get_tensor(st, 1, M.MOARA_T_P)])
    info = M.moara_refresh_info(st, 1)
    assert info["converged"] and info["rank"] == 12 and 1 <= info["sweeps"] <= 14, info


def test_state_used_from_two_streams_keeps_call_order():
    """Steps of one state alternating between two streams give bit for bit the result of
    one stream: each call waits for the work the previous call enqueued."""
    import torch
    M = _M()
    c = Case(shapes=[(256, 384, WL.Q), (384, 256, WL.GATE)], ranks=[32, 48], block_size=64, operand_dtype="bf16",
             weight_dtype="bf16", weight_std=0.02)
    grads = [[to_dev(_grad(c, 13, t, i), "f32") for i in range(2)] for t in range(6)]
    outs = []
    for two in (False, True):
        st = gpu_state(c, refresh_interval=3)
        Wd = [to_dev(w, "bf16") for w in _weights(c, 0)]
        streams = [torch.cuda.Stream(), torch.cuda.Stream()] if two else [torch.cuda.current_stream()]
        torch.cuda.synchronize()
        for t in range(6):
            M.moara_step(st, Wd, grads[t], lr=1e-3, stream=streams[t % len(streams)])
        torch.cuda.synchronize()
        outs.append(([w.clone() for w in Wd], [M.moara_get_tensor(st, i, M.MOARA_T_EXP_AVG) for i in range(2)]))
    for a, b in zip(outs[0][0], outs[1][0]):
        assert torch.equal(a, b)
    for a, b in zip(outs[0][1], outs[1][1]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("mom", ["f32", "bf16"])
def test_checkpoint_roundtrip_is_bit_identical(mom):
    import torch
    M = _M()
    c = Case(shapes=[(160, 224, WL.Q), (224, 160, WL.UP)], ranks=[24, 32], block_size=32, weight_dtype="bf16",
             operand_dtype="bf16", weight_std=0.02, moment_dtype=mom)
    grads = [[to_dev(_grad(c, 9, t, i), "f32") for i in range(2)] for t in range(6)]
    st = gpu_state(c, refresh_interval=4)
    Wa = [to_dev(w, "bf16") for w in _weights(c, 0)]
    for t in range(6):
        M.moara_step(st, Wa, grads[t], lr=1e-3)
    st1 = gpu_state(c, refresh_interval=4)
    Wb = [to_dev(w, "bf16") for w in _weights(c, 0)]
    for t in range(3):
        M.moara_step(st1, Wb, grads[t], lr=1e-3)
    saved = {(i, k): M.moara_get_tensor(st1, i, k) for i in range(2)
             for k in (M.MOARA_T_P, M.MOARA_T_EXP_AVG, M.MOARA_T_EXP_AVG_SQ, M.MOARA_T_MAG_AVG,
                       M.MOARA_T_MAG_AVG_SQ, M.MOARA_T_STEP)}
    M.moara_destroy_state(st1)
    st2 = gpu_state(c, refresh_interval=4)
    for (i, k), v in saved.items():
        M.moara_set_tensor(st2, i, k, v)
    for t in range(3, 6):
        M.moara_step(st2, Wb, grads[t], lr=1e-3)
    torch.cuda.synchronize()
    for i in range(2):
        assert torch.equal(Wa[i], Wb[i])


def test_bf16_moments_are_stored_rounded_to_nearest_even():
    """With bf16 direction moments, moara_set_tensor rounds the fp32 values it is given to
    nearest-even bf16 and moara_get_tensor widens them back exactly, in the paper's
    orientation on both sides (LEFT r x n, RIGHT m x r): equal to the oracle's rounding,
    bit for bit, including ties, subnormals and overflow to infinity."""
    M = _M()
    c = Case(shapes=[(48, 80, WL.Q), (80, 48, WL.UP)], ranks=[8, 8], block_size=16, moment_dtype="bf16")
    st = gpu_state(c)
    special = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 2.0 ** -130, 3.0 * 2.0 ** -134,
                        3.3e38, -3.4e38, 0.0, -0.0, 1e-45], dtype=np.float32)
    for i, (m, n) in enumerate([(48, 80), (80, 48)]):
        shp = (8, n) if m <= n else (m, 8)
        for k, seed in ((M.MOARA_T_EXP_AVG, 1), (M.MOARA_T_EXP_AVG_SQ, 2)):
            v = (rng(seed, i).standard_normal(shp) * 10.0 ** rng(seed, i, 1).uniform(-6, 3, shp)).astype(np.float32)
            v.ravel()[:special.size] = special
            M.moara_set_tensor(st, i, k, v)
            got = M.moara_get_tensor(st, i, k)
            ref = O.round_bf16(v.astype(np.float64))
            assert np.array_equal(got.astype(np.float64), ref), f"matrix {i} tensor {k}"
            assert np.array_equal(np.signbit(got), np.signbit(ref))


def test_runs_are_deterministic():
    import torch
    M = _M()
    c = Case(shapes=[(256, 384, WL.Q), (384, 256, WL.GATE)], ranks=[32, 48], block_size=64)
    outs = []
    for _ in range(2):
        st = gpu_state(c, refresh_interval=2)
        Wd = [to_dev(w, "f32") for w in _weights(c, 0)]
        for t in range(3):
            M.moara_step(st, Wd, [to_dev(_grad(c, 4, t, i), "f32") for i in range(2)], lr=1e-3)
        torch.cuda.synchronize()
        outs.append([w.clone() for w in Wd])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_kernel_timing_counts_each_launch_and_resets():
    """Per-kernel timing (the measurement path): with timing on, every step adds one launch of
    each step kernel with a positive duration, a refresh adds to the refresh entry, a reset
    zeroes them, and with timing off nothing is recorded; results are those of an untimed run."""
    import torch
    M = _M()
    c = Case(shapes=[(256, 384, WL.Q), (384, 256, WL.GATE)], ranks=[32, 48], block_size=64)
    outs = []
    for timed in (True, False):
        st = gpu_state(c, refresh_interval=2)
        M.moara_set_timing(st, timed)
        Wd = [to_dev(w, "f32") for w in _weights(c, 0)]
        for t in range(3):   # refreshes at t = 0 and t = 2
            M.moara_step(st, Wd, [to_dev(_grad(c, 4, t, i), "f32") for i in range(2)], lr=1e-3)
        torch.cuda.synchronize()
        outs.append([w.clone() for w in Wd])
        for kid in (M.MOARA_KERN_DECOMPOSE, M.MOARA_KERN_PROJECT, M.MOARA_KERN_BACKPROJ, M.MOARA_KERN_REFRESH):
            n, ms = M.moara_kernel_stats(st, kid)
            want = (2 if kid == M.MOARA_KERN_REFRESH else 3) if timed else 0
            assert n == want, (kid, n)
            assert (ms > 0.0) == timed, (kid, ms)
        M.moara_reset_kernel_stats(st)
        assert M.moara_kernel_stats(st, M.MOARA_KERN_PROJECT) == (0, 0.0)
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_matrix_info_matches_the_host_resolver():
    """The state's per-matrix layout (moara_matrix_info) equals what moara_resolve_matrix
    gives for the same descriptor: rank (table, override), side (auto, forced) and the
    number of magnitude blocks ceil(n / B)."""
    M = _M()
    cfg = M.moara_default_config(rank_table=[16, 24, 32, 8, 40, 48, 12, 4, 4, 4], block_size=48,
                                 operand_dtype=M.MOARA_F32, weight_dtype=M.MOARA_F32, refresh_interval=0)
    entries = [(96, 200, M.MOARA_Q), (200, 96, M.MOARA_GATE), (128, 128, M.MOARA_K),
               (150, 97, M.MOARA_DOWN, 20), (64, 300, M.MOARA_UP, 0, M.MOARA_SIDE_RIGHT),
               (300, 64, M.MOARA_V, 10, M.MOARA_SIDE_LEFT)]
    descs = M.make_descs(entries)
    st = M.moara_create_state(cfg, descs)
    for i, d in enumerate(descs):
        r, side = M.moara_resolve_matrix(cfg, d)
        assert M.moara_matrix_info(st, i) == (d.rows, d.cols, r, side, -(-d.cols // 48)), i
    assert [M.moara_matrix_info(st, i)[2] for i in range(len(entries))] == [16, 40, 24, 20, 48, 10]
    with pytest.raises(M.MoaraError):
        M.moara_matrix_info(st, len(entries))


def test_step_without_projector_is_rejected_before_launch():
    import torch
    M = _M()
    c = Case(shapes=[(64, 64, WL.Q)], ranks=[8], block_size=32)
    st = gpu_state(c, refresh_interval=0)
    W = to_dev(_weights(c, 0)[0], "f32")
    with pytest.raises(M.MoaraError) as e:
        M.moara_step(st, [W], [to_dev(_grad(c, 0, 0, 0), "f32")], lr=1e-3)
    assert e.value.status == M.MOARA_E_STATE
    with pytest.raises(ValueError):
        M.moara_step(st, [W.t()], [to_dev(_grad(c, 0, 0, 0), "f32")], lr=1e-3)


# ------------------------------------------------------------------ alignment diagnostic (Section 3.2)
# S is a cosine of fp32-GEMM results summed in fp64: it matches the oracle's fp64 value to
# about 1e-6 (K <= 1000 here); the bar is 1e-5, under the fp32 bar of 1e-4.

@pytest.mark.parametrize("decompose,op", [(True, "f32"), (True, "bf16"), (False, "f32")])
def test_alignment_matches_oracle(decompose, op):
    import torch
    M = _M()
    c = Case(shapes=[(300, 452, WL.Q), (452, 300, WL.GATE), (129, 1000, WL.DOWN), (77, 130, WL.K), (5, 3, WL.V)],
             ranks=[37, 50, 64, 9, 2], block_size=48, decompose=decompose, operand_dtype=op)
    st = gpu_state(c)
    Gs = [_grad(c, 6, 0, i) for i in range(len(c.shapes))]
    Gs[4][:] = 0.0   # an all-zero gradient: S = 0 by definition
    Gd = [to_dev(g, "f32") for g in Gs]
    print(f"[alignment] decompose={decompose} operands={op}", flush=True)
    M.moara_refresh_projector(st, Gd)
    steps0 = [M.moara_get_tensor(st, i, M.MOARA_T_STEP) for i in range(len(Gs))]
    # S depends on the projector's span only; both sides take the oracle's (the first r
    # canonical vectors for the all-zero gradient, as after the library's refresh of it)
    Ps = [oracle_projector(G, c, i) if i != 4 else np.eye(3, 2) for i, G in enumerate(Gs)]
    for i, P in enumerate(Ps):
        M.moara_set_tensor(st, i, M.MOARA_T_P, P)
    S = M.moara_alignment(st, Gd)
    for i, G in enumerate(Gs):
        ref = O.alignment(G, Ps[i], c.block_size, decompose_on=decompose)
        assert abs(S[i] - ref) <= 1e-5, (i, S[i], ref)
        assert M.moara_get_tensor(st, i, M.MOARA_T_STEP) == steps0[i]
    assert S[4] == 0.0 and all(0.0 < S[i] < 1.0 for i in range(4))
    # an active mask leaves the other entries alone
    S2 = M.moara_alignment(st, Gd, active=[False, True, False, True, False])
    assert np.isnan(S2[0]) and np.isnan(S2[2]) and np.isnan(S2[4])
    assert abs(S2[1] - S[1]) <= 1e-12 and abs(S2[3] - S[3]) <= 1e-12


def test_alignment_full_rank_projector_is_one_and_needs_a_projector():
    import torch
    M = _M()
    c = Case(shapes=[(64, 96, WL.Q), (96, 40, WL.UP)], ranks=[64, 40], block_size=32)
    st = gpu_state(c)
    Gd = [to_dev(_grad(c, 7, 0, i), "f32") for i in range(2)]
    with pytest.raises(M.MoaraError) as e:
        M.moara_alignment(st, Gd)
    assert e.value.status == M.MOARA_E_STATE
    M.moara_refresh_projector(st, Gd)
    S = M.moara_alignment(st, Gd)
    assert np.all(np.abs(S - 1.0) <= 1e-5), S


def test_profiling_run_gives_the_oracles_module_scores():
    """Phases 1-2 over a short uniform-rank run: at each profiling step the device S of
    every matrix against the oracle's with the same projector and gradient, and the
    aggregated S_tau against the oracle's module average of those values."""
    import torch
    from paper_2609_15037_amd import profiling as PR
    M = _M()
    c = Case(shapes=[(96, 160, WL.Q), (96, 160, WL.K), (160, 96, WL.GATE), (96, 200, WL.DOWN), (96, 160, WL.Q)],
             ranks=[16, 16, 16, 16, 16], block_size=32)
    st = gpu_state(c)
    W = [to_dev(w, c.weight_dtype) for w in _weights(c, 8)]
    prof = PR.AlignmentProfile([sh[2] for sh in c.shapes], stride=2, n_p=6)
    samples, Ps = [], None
    for t in range(1, 8):
        Gs = [_grad(c, 9, t, i) for i in range(len(c.shapes))]
        Gd = [to_dev(g, "f32") for g in Gs]
        if t in (1, 5):   # the T = 4 schedule (counter 0 and 4), with the oracle's projectors
            Ps = [oracle_projector(G, c, i) for i, G in enumerate(Gs)]
            for i, P in enumerate(Ps):
                M.moara_set_tensor(st, i, M.MOARA_T_P, P)
        M.moara_step(st, W, Gd, lr=1e-3)
        torch.cuda.synchronize()
        if prof.due(t):
            S = prof.record(st, Gd, t=t)
            for i, G in enumerate(Gs):
                ref = O.alignment(G, Ps[i], c.block_size)
                assert abs(S[i] - ref) <= 1e-5, (t, i, S[i], ref)
                samples.append((c.shapes[i][2], ref))
    assert prof.steps == [2, 4, 6]
    ref_tau = O.module_alignment(samples)
    got = prof.s_tau()
    assert set(got) == set(ref_tau)
    for tau in ref_tau:
        assert abs(got[tau] - ref_tau[tau]) <= 1e-5, (tau, got[tau], ref_tau[tau])


def test_nd_weights_step_as_their_flattened_matrices():
    """A weight with more than two axes is the matrix of its first axis by all others
    (Appendix B.1): stepping N-d tensors gives bit for bit the result of the 2-D matrices."""
    import torch
    M = _M()
    shapes_nd = [(64, 8, 3, 3), (96, 4, 10)]
    c = Case(shapes=[(*M.flatten_shape(s), WL.Q) for s in shapes_nd], ranks=[16, 12], block_size=16)
    Ws = _weights(c, 3)
    outs = []
    for nd in (False, True):
        st = gpu_state(c, refresh_interval=2)
        Wd = [to_dev(w, "f32") for w in Ws]
        Wv = [w.view(s) for w, s in zip(Wd, shapes_nd)] if nd else Wd
        for t in range(3):
            Gd = [to_dev(_grad(c, 8, t, i), "f32") for i in range(2)]
            Gv = [g.view(s) for g, s in zip(Gd, shapes_nd)] if nd else Gd
            M.moara_step(st, Wv, Gv, lr=1e-3)
        torch.cuda.synchronize()
        outs.append([w.clone() for w in Wd])
    for a, b in zip(*outs):
        assert torch.equal(a, b)
