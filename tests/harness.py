"""Shared helpers of the parity tests: build identical inputs for the HIP path
(through the C ABI binding) and the CPU oracle, and compare them."""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

import workloads as WL
from oracle import moara_oracle as O

TOL_F32 = 1e-4     # all-fp32 path: updated weights and moments, floored relative error
TOL_BF16 = 2e-2    # any bf16 operand or weight
TOL_UPDATE_F32 = 1e-3   # weight update W_t - W_0 in the all-fp32 path (see compare_update)


def have_gpu() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@dataclasses.dataclass
class Case:
    shapes: List[tuple]            # (rows, cols, module)
    ranks: List[int]
    block_size: int
    weight_dtype: str = "f32"
    operand_dtype: str = "f32"
    moment_dtype: str = "f32"      # storage of the direction moments: "f32" or "bf16"
    decompose: bool = True
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    scale: float = 0.25
    lr: float = 1e-3
    weight_std: float = 1e-3
    grad_std: float = 1e-3
    refresh_oversample: int = -1
    refresh_iters: int = 20


def rng(seed, *key):
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([seed, *key])))


def case_from_workload(wl: WL.Workload, operand_dtype: Optional[str] = None) -> Case:
    return Case(shapes=[(m.rows, m.cols, m.module) for m in wl.matrices],
                ranks=[wl.rank_of(m) for m in wl.matrices], block_size=wl.block_size,
                weight_dtype=wl.weight_dtype, operand_dtype=operand_dtype or wl.operand_dtype,
                moment_dtype=wl.moment_dtype,
                adam_eps=wl.adam_eps, beta1=wl.beta1, beta2=wl.beta2, scale=wl.scale, lr=wl.lr,
                weight_std=wl.weight_std, grad_std=wl.grad_std,
                refresh_oversample=wl.refresh_oversample, refresh_iters=wl.refresh_iters)


def oracle_cfg(c: Case, i: int, refresh_interval: int = 0) -> O.OracleConfig:
    return O.OracleConfig(block_size=c.block_size, rank=c.ranks[i], beta1=c.beta1, beta2=c.beta2,
                          adam_eps=c.adam_eps, scale=c.scale, refresh_interval=refresh_interval,
                          decompose=c.decompose, weight_dtype=c.weight_dtype, operand_dtype=c.operand_dtype,
                          moment_dtype=c.moment_dtype)


def gpu_state(c: Case, refresh_interval: int = 0, refresh_iters=None, oversample=None, seed: int = 0, **extra):
    from paper_2609_15037_amd import moara as M
    refresh_iters = c.refresh_iters if refresh_iters is None else refresh_iters
    oversample = c.refresh_oversample if oversample is None else oversample
    cfg = M.moara_default_config(
        block_size=c.block_size, beta1=c.beta1, beta2=c.beta2, adam_eps=c.adam_eps, scale=c.scale,
        refresh_interval=refresh_interval, decompose=1 if c.decompose else 0,
        weight_dtype=M.MOARA_BF16 if c.weight_dtype == "bf16" else M.MOARA_F32,
        operand_dtype=M.MOARA_BF16 if c.operand_dtype == "bf16" else M.MOARA_F32,
        moment_dtype=M.MOARA_BF16 if c.moment_dtype == "bf16" else M.MOARA_F32,
        refresh_iters=refresh_iters, refresh_oversample=oversample, refresh_seed=seed, **extra)
    descs = M.make_descs([(m, n, mod, r) for (m, n, mod), r in zip(c.shapes, c.ranks)])
    return M.moara_create_state(cfg, descs)


def to_dev(a: np.ndarray, dtype: str, offset: int = 0):
    """Device copy of `a` in fp32 or bf16. offset > 0 places it `offset` elements into a
    larger allocation, so that its address is not 16-byte aligned (exercises the library's
    paths for caller buffers the large-tile kernels cannot take)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    if offset:
        flat = torch.zeros(t.numel() + offset, dtype=t.dtype, device=t.device)
        flat[offset:] = t.reshape(-1)
        t = flat[offset:].view(t.shape)
    return t


def to_np(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def oracle_projector(G: np.ndarray, c: Case, i: int) -> np.ndarray:
    """The oracle's top-r projector of G's direction tensor (its truncated SVD), rounded to
    fp32: fed to both sides."""
    _, V = O.decompose(G, c.block_size) if c.decompose else (None, G.astype(np.float64))
    side = O.projection_side(*G.shape)
    return O.round_f32(O.truncated_svd(V, c.ranks[i], side))


def adam_sensitivity(V: np.ndarray, P: np.ndarray, side: str, exp_avg_sq: np.ndarray, t: int,
                     beta2: float, adam_eps: float) -> np.ndarray:
    """Forward error estimate of the Adam output N for fp32 accumulation of R.

    R = P^T V (LEFT) or V P (RIGHT) accumulated in fp32 over K terms has an error
    of about 2 sqrt(K) u32 sum_k |terms| (standard summation bound); N moves by
    about dR / (sqrt(q^) + eps). Computed from the oracle's own float64 values,
    never from the GPU result. Returned in the state orientation (r x n or m x r)."""
    u32 = 2.0 ** -24
    if side == "left":
        K = V.shape[0]
        dR = 2.0 * np.sqrt(K) * u32 * (np.abs(P).T @ np.abs(V))
    else:
        K = V.shape[1]
        dR = 2.0 * np.sqrt(K) * u32 * (np.abs(V) @ np.abs(P))
    qhat = exp_avg_sq / (1.0 - beta2 ** t)
    return dR / (np.sqrt(qhat) + adam_eps)


def slices_of(flags: np.ndarray, side: str, shape) -> np.ndarray:
    """Update elements fed by flagged entries of N: N[j, c] (LEFT) feeds column c of
    the update, N[i, j] (RIGHT) feeds row i."""
    mask = np.zeros(shape, dtype=bool)
    if side == "left":
        mask[:, np.any(flags, axis=0)] = True
    else:
        mask[np.any(flags, axis=1), :] = True
    return mask


def compare_update(name: str, got: np.ndarray, ref: np.ndarray, tol: float, report: dict, mask=None):
    """Weight-update check (stricter than the weight check, whose floor is rms(W)),
    on the elements not fed by ill-conditioned Adam outputs (see adam_sensitivity)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) or 1.0
    err = np.abs(got - ref) / (np.abs(ref) + rms)
    keep = ~mask if mask is not None else np.ones_like(err, dtype=bool)
    e = float(err[keep].max()) if keep.any() else 0.0
    report[name] = max(report.get(name, 0.0), e)
    report[name + ".masked_frac"] = max(report.get(name + ".masked_frac", 0.0), 1.0 - float(keep.mean()))
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert e <= tol, f"{name}: floored relative error {e:.3e} > {tol:.1e} on well-conditioned elements"


TOL_MASKED = 1e-2   # elements fed by ill-conditioned Adam inputs (a full sign flip moves W by ~3e-3)


def compare(name: str, got: np.ndarray, ref: np.ndarray, tol: float, report: dict, mask=None):
    """Floored relative error max_i |a_i - b_i| / (|b_i| + rms(b)) <= tol; elements in
    ``mask`` (fed by Adam outputs whose fp32 forward error estimate exceeds 0.1, see
    adam_sensitivity) are held to TOL_MASKED instead."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    if mask is None or not mask.any():
        e = O.floored_rel_err(got, ref)
        report[name] = max(report.get(name, 0.0), e)
        assert e <= tol, f"{name}: floored relative error {e:.3e} > {tol:.1e}"
        return e
    rms = float(np.sqrt(np.mean(ref * ref))) or 1.0
    err = np.abs(got - ref) / (np.abs(ref) + rms)
    e = float(err[~mask].max()) if (~mask).any() else 0.0
    em = float(err[mask].max())
    report[name] = max(report.get(name, 0.0), e)
    report[name + ".masked_frac"] = max(report.get(name + ".masked_frac", 0.0), float(mask.mean()))
    assert e <= tol, f"{name}: floored relative error {e:.3e} > {tol:.1e} on well-conditioned elements"
    assert em <= TOL_MASKED, f"{name}: {em:.3e} on elements fed by ill-conditioned Adam inputs"
    return e


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bfloat16 values at |x| (8 significant bits; subnormal spacing at the bottom)."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.ldexp(1.0, (np.maximum(e, -126) - 7).astype(int))


def magnitude_steps(st, cfg) -> np.ndarray:
    """The Optimizer_M output dM of the oracle's last step, read back from its moments
    (for reporting how far the magnitude branch moved the update, not for parity)."""
    t = st.t
    return ((st.mag_avg / (1.0 - cfg.beta1 ** t)) /
            (np.sqrt(st.mag_avg_sq / (1.0 - cfg.beta2 ** t)) + cfg.adam_eps))


def seeded_history(c: Case, i: int, R_scale: float, M_scale: np.ndarray, seed: int):
    """Moments of a matrix restored at a late step (as from a checkpoint): per-entry first
    moments around zero (direction) or around the block magnitudes (magnitude), second
    moments spread over a decade and a half; fp32 values, fed to both sides."""
    m, n, _ = c.shapes[i]
    g = rng(seed, 21, i)
    side = O.projection_side(m, n)
    shp = (c.ranks[i], n) if side == O.LEFT else (m, c.ranks[i])
    e1 = R_scale * 0.3 * g.standard_normal(shp)
    e2 = (R_scale ** 2) * 10.0 ** g.uniform(-0.5, 1.0, shp)
    k = M_scale.shape[1]
    a1 = M_scale * 10.0 ** g.uniform(-0.3, 0.3, (m, k))
    a2 = (a1 ** 2) * 10.0 ** g.uniform(0.0, 1.5, (m, k))
    return [O.round_f32(x) for x in (e1, e2, a1, a2)]


# ------------------------------------------------------------------ the library's in-step refresh
# After a refresh, the steps depend on the projector's basis, which is unique only up to
# rotations inside clusters of (nearly) equal singular values. Parity with the oracle is
# therefore taken on a state that receives the oracle's own projector (moara_set_tensor);
# the library's own refresh inside moara_step is checked by principal angle against the
# oracle's SVD, and, library against library, bit for bit against an explicit
# moara_refresh_projector before the step whose projector is read back and set again
# (so that the operand copies the refresh wrote equal those moara_set_tensor derives).

STATE_TENSORS = ("P", "exp_avg", "exp_avg_sq", "mag_avg", "mag_avg_sq")


def explicit_refresh(M, st, Gd, mask):
    """moara_refresh_projector on the matrices in `mask`, then each new projector read back
    and set again through moara_set_tensor."""
    import torch
    if not any(mask):
        return
    M.moara_refresh_projector(st, [g if k else None for g, k in zip(Gd, mask)],
                              active=np.asarray(mask, dtype=np.uint8))
    torch.cuda.synchronize()
    for i, k in enumerate(mask):
        if k:
            M.moara_set_tensor(st, i, M.MOARA_T_P, M.moara_get_tensor(st, i, M.MOARA_T_P))


def assert_same_state(M, sa, sb, Wa, Wb, idx, what=""):
    """W, projector, all four moments and the counter bit-identical in two library states."""
    import torch
    ids = {"P": M.MOARA_T_P, "exp_avg": M.MOARA_T_EXP_AVG, "exp_avg_sq": M.MOARA_T_EXP_AVG_SQ,
           "mag_avg": M.MOARA_T_MAG_AVG, "mag_avg_sq": M.MOARA_T_MAG_AVG_SQ}
    for i in idx:
        assert torch.equal(Wa[i], Wb[i]), f"{what} matrix {i}: W differs"
        ta, tb = M.moara_get_tensor(sa, i, M.MOARA_T_STEP), M.moara_get_tensor(sb, i, M.MOARA_T_STEP)
        assert ta == tb, f"{what} matrix {i}: counter {ta} vs {tb}"
        for name in STATE_TENSORS:
            if name == "P" and ta == 0:
                continue
            a, b = M.moara_get_tensor(sa, i, ids[name]), M.moara_get_tensor(sb, i, ids[name])
            assert np.array_equal(a, b), f"{what} matrix {i}: {name} differs"

