"""moara_step_noalloc (the allocation-free variant of moara_step) against moara_step.

Both entry points run the same kernels on the same descriptors, so the results must
agree bit for bit (stronger than the oracle parity bar, which moara_step itself meets
in the other GPU tests). Two calls in a row share the GPU's scratch array, the second
with a smaller input, so that anything the first call left there would show; the
second state is then stepped again after the first one.
"""
import numpy as np
import pytest

import workloads as WL
from tests.harness import Case, gpu_state, have_gpu, rng, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs an MI355X GPU")]


def _M():
    from paper_2609_15037_amd import moara as M
    return M


def _inputs(c: Case, seed, steps):
    W = [(c.weight_std * rng(seed, 1, i).standard_normal((m, n))).astype(np.float32)
         for i, (m, n, _) in enumerate(c.shapes)]
    G = [[(c.grad_std * rng(seed, 2, t, i).standard_normal((m, n))).astype(np.float32)
          for i, (m, n, _) in enumerate(c.shapes)] for t in range(steps)]
    return W, G


def _pair(c: Case, refresh_interval):
    """Two identical states: one stepped with moara_step, one with moara_step_noalloc."""
    return gpu_state(c, refresh_interval=refresh_interval), gpu_state(c, refresh_interval=refresh_interval)


def _run(M, st, Wd, Gs, lr, noalloc, active=None):
    import torch
    for G in Gs:
        M.moara_step(st, Wd, [to_dev(g, "f32") for g in G], lr=lr, active=active, noalloc=noalloc)
    torch.cuda.synchronize()


def _same(M, sa, sb, Wa, Wb, n):
    import torch
    for i in range(n):
        assert torch.equal(Wa[i], Wb[i]), f"matrix {i}: W differs"
        for k in (M.MOARA_T_P, M.MOARA_T_EXP_AVG, M.MOARA_T_EXP_AVG_SQ, M.MOARA_T_MAG_AVG, M.MOARA_T_MAG_AVG_SQ):
            assert np.array_equal(M.moara_get_tensor(sa, i, k), M.moara_get_tensor(sb, i, k)), (i, k)
        assert M.moara_get_tensor(sa, i, M.MOARA_T_STEP) == M.moara_get_tensor(sb, i, M.MOARA_T_STEP)


def test_step_noalloc_matches_step_on_two_calls_in_a_row():
    M = _M()
    # first call: a larger input (bf16 large-tile path, RIGHT and LEFT, ragged fallback shape), with a
    # refresh at t = 0 and t = 2 (refresh workspace and descriptors in the scratch array)
    big = Case(shapes=[(512, 768, WL.Q), (768, 512, WL.GATE), (300, 452, WL.K), (256, 1024, WL.DOWN)],
               ranks=[64, 96, 40, 128], block_size=64, operand_dtype="bf16", weight_dtype="bf16", weight_std=0.02)
    # second call: a smaller input (fewer, smaller matrices, fp32 path)
    small = Case(shapes=[(96, 160, WL.Q), (160, 96, WL.UP)], ranks=[16, 24], block_size=32)
    states = {}
    for name, c, steps in (("big", big, 3), ("small", small, 3)):
        W, G = _inputs(c, 5 if name == "big" else 6, steps)
        sa, sb = _pair(c, refresh_interval=2)
        Wa = [to_dev(w, c.weight_dtype) for w in W]
        Wb = [to_dev(w, c.weight_dtype) for w in W]
        print(f"[noalloc] {name}: {len(c.shapes)} matrices, {steps} steps (refresh at t = 0, 2)", flush=True)
        _run(M, sa, Wa, G, 1e-3, noalloc=False)
        _run(M, sb, Wb, G, 1e-3, noalloc=True)
        _same(M, sa, sb, Wa, Wb, len(c.shapes))
        states[name] = (c, sa, sb, Wa, Wb)
    # the first state again, after the smaller call left its contents in the scratch array
    c, sa, sb, Wa, Wb = states["big"]
    _, G = _inputs(c, 7, 2)
    print("[noalloc] big again (refresh at t = 4)", flush=True)
    _run(M, sa, Wa, G, 1e-3, noalloc=False)
    _run(M, sb, Wb, G, 1e-3, noalloc=True)
    _same(M, sa, sb, Wa, Wb, len(c.shapes))


def test_step_noalloc_zero_grad_mode_and_inactive_matrices():
    """zero_grad_mode 1 with bf16 direction moments (the zero-gradient kernel's 2-byte path)."""
    M = _M()
    c = Case(shapes=[(128, 192, WL.EXP_GATE), (128, 192, WL.EXP_UP), (192, 128, WL.EXP_DOWN)], ranks=[16] * 3,
             block_size=64, operand_dtype="bf16", weight_dtype="bf16", weight_std=0.02, moment_dtype="bf16")
    W, G = _inputs(c, 8, 4)
    sa = gpu_state(c, refresh_interval=2, zero_grad_mode=1)
    sb = gpu_state(c, refresh_interval=2, zero_grad_mode=1)
    Wa = [to_dev(w, "bf16") for w in W]
    Wb = [to_dev(w, "bf16") for w in W]
    for t, mask in enumerate([[1, 0, 1], [0, 1, 1], [1, 1, 0], [1, 0, 0]]):
        print(f"[noalloc] zero_grad_mode 1, step {t}, active {mask}", flush=True)
        Gd = [to_dev(G[t][i], "f32") if mask[i] else None for i in range(3)]
        M.moara_step(sa, Wa, Gd, lr=1e-3, active=mask)
        M.moara_step(sb, Wb, Gd, lr=1e-3, active=mask, noalloc=True)
    import torch
    torch.cuda.synchronize()
    _same(M, sa, sb, Wa, Wb, 3)


def test_step_noalloc_rejects_a_refresh_larger_than_the_scratch_before_any_work():
    """An 18944 x 3584 matrix at r = 1024 needs about 706 MiB of refresh workspace, more than
    the 512 MiB array: the call fails with MOARA_E_UNSUPPORTED and changes nothing."""
    import torch
    M = _M()
    c = Case(shapes=[(18944, 3584, WL.GATE)], ranks=[1024], block_size=128, operand_dtype="bf16",
             weight_dtype="bf16")
    st = gpu_state(c, refresh_interval=200)
    W = torch.zeros((18944, 3584), dtype=torch.bfloat16, device="cuda")
    G = torch.ones((18944, 3584), dtype=torch.float32, device="cuda")
    print("[noalloc] 18944 x 3584, r = 1024: refresh larger than the scratch", flush=True)
    with pytest.raises(M.MoaraError) as e:
        M.moara_step(st, [W], [G], lr=1e-3, noalloc=True)
    assert e.value.status == M.MOARA_E_UNSUPPORTED
    torch.cuda.synchronize()
    assert M.moara_get_tensor(st, 0, M.MOARA_T_STEP) == 0
    assert not torch.any(W)
    with pytest.raises(M.MoaraError):
        M.moara_get_tensor(st, 0, M.MOARA_T_P)   # no projector was set
