"""The seeded synthetic workloads: shapes and parameter counts of each stack (worked out
by hand from the model dimensions), determinism and keying of the draws, the spectrum of
the low-rank gradient recipe, and the MoE router's active sets."""
import numpy as np

import workloads as WL


def test_stack_shapes_and_parameter_counts():
    wl = WL.WORKLOADS
    # Llama-2-7B: 32 layers of q, k, v, o 4096 x 4096 and gate, up 11008 x 4096, down 4096 x 11008
    assert len(wl["llama2_7b"].matrices) == 224
    assert wl["llama2_7b"].n_params == 32 * (4 * 4096 * 4096 + 3 * 4096 * 11008) == 6_476_005_376
    # Qwen2-7B (GQA): q, o 3584 x 3584, k, v 512 x 3584, ffn 18944
    assert len(wl["qwen2_7b"].matrices) == 196
    assert wl["qwen2_7b"].n_params == 28 * (2 * 3584 ** 2 + 2 * 512 * 3584 + 3 * 18944 * 3584) == 6_525_288_448
    # DeepSeek-MoE: 28 layers of attention (4 matrices) and 64 routed + 2 shared experts (3 each)
    assert len(wl["deepseek_moe"].matrices) == 28 * (4 + 3 * 66) == 5656
    assert len(wl["llama_300m"].matrices) == 24 * 7
    m7 = {(m.module, m.rows, m.cols) for m in wl["llama2_7b"].matrices}
    assert m7 == {(WL.Q, 4096, 4096), (WL.K, 4096, 4096), (WL.V, 4096, 4096), (WL.O, 4096, 4096),
                  (WL.GATE, 11008, 4096), (WL.UP, 11008, 4096), (WL.DOWN, 4096, 11008)}
    for w in wl.values():   # every rank fits its matrix
        for m in w.matrices:
            assert 1 <= w.rank_of(m) <= min(m.rows, m.cols), (w.name, m.name)


def test_draws_are_deterministic_and_keyed():
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0])
    a = WL.grad_np(wl, 0, 3)
    assert a.dtype == np.float32 and a.shape == (1024, 1024)
    assert np.array_equal(a, WL.grad_np(wl, 0, 3))
    assert not np.array_equal(a, WL.grad_np(wl, 0, 4))          # another step
    assert not np.array_equal(a, WL.grad_np(wl, 1, 3))          # another matrix of the same shape
    assert not np.array_equal(a, WL.grad_np(wl, 0, 3, seed=1))  # another seed
    assert np.array_equal(WL.weight_np(wl, 2), WL.weight_np(wl, 2))
    # the low-rank part is fixed per matrix: two steps differ by noise only
    d = WL.grad_np(wl, 0, 3).astype(np.float64) - WL.grad_np(wl, 0, 4)
    assert abs(np.std(d) - np.sqrt(2) * wl.noise_std) < 0.05 * np.sqrt(2) * wl.noise_std


def test_lowrank_recipe_spectrum():
    """G = U diag(i^-p) Y^T + noise: U, Y orthonormal, and by Weyl's inequality every singular
    value of G lies within ||noise||_2 <= noise_std (sqrt(m) + sqrt(n)) (plus a margin) of the
    signal's, so the top singular values follow i^-p and the rest sit at the noise floor."""
    wl = WL.subset(WL.WORKLOADS["llama_300m"], [0])
    i = [k for k, m in enumerate(wl.matrices) if m.module == WL.GATE][0]
    m = wl.matrices[i]
    U, sig, Y = WL.lowrank_factors(wl, i)
    R = wl.lowrank_rank
    np.testing.assert_allclose(U.T @ U, np.eye(R), atol=1e-12)
    np.testing.assert_allclose(Y.T @ Y, np.eye(R), atol=1e-12)
    np.testing.assert_allclose(sig, np.arange(1, R + 1) ** -wl.lowrank_power)
    s = np.linalg.svd(WL.grad_np(wl, i, 0).astype(np.float64), compute_uv=False)
    bound = 1.1 * wl.noise_std * (np.sqrt(m.rows) + np.sqrt(m.cols))
    assert np.max(np.abs(s[:R] - sig)) <= bound
    assert s[R] <= bound


def test_moe_router_activates_six_routed_experts_per_layer():
    wl = WL.WORKLOADS["deepseek_moe"]
    sizes = np.array([m.rows * m.cols for m in wl.matrices])
    sets = []
    for step in range(4):
        act = WL.active_set(wl, step)
        assert all(act[k] for k, m in enumerate(wl.matrices) if not m.routed)   # attention, shared experts
        for layer in range(28):
            experts = {m.expert for k, m in enumerate(wl.matrices) if m.layer == layer and m.routed and act[k]}
            assert len(experts) == 6 and experts <= set(range(64))
            # an expert's three matrices are active together
            assert sum(1 for k, m in enumerate(wl.matrices) if m.layer == layer and m.routed and act[k]) == 18
        # active parameters: per layer 4 * 2048^2 attention + (2 shared + 6 routed) * 3 * 2048 * 1408
        assert int(sizes[act].sum()) == 28 * (4 * 2048 ** 2 + 8 * 3 * 2048 * 1408) == 2_407_530_496
        sets.append(act)
    assert not all(np.array_equal(sets[0], s) for s in sets[1:])
    k = int(np.flatnonzero(~sets[0])[0])   # an inactive routed matrix gets a zero gradient
    assert not np.any(WL.grad_np(wl, k, 0))
