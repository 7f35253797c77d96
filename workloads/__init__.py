"""Seeded synthetic workloads for the MoARa optimizer hot path.

This module only *describes* workloads and *draws* their inputs. It holds none
of the method's arithmetic: no decomposition, projection, Adam or update. Both
the CPU oracle tests and the HIP path's tests/benchmark draw their inputs here,
so that the two sides see identical values.

Shapes follow the model families the paper evaluates (Llama 2 scaling study and
the model-family comparison, Appendix D model table): weights are stored
``out x in`` (the PyTorch ``Linear`` layout), gradients are fp32.

Gradient recipes (all seeded, counter-based Philox keyed by
(seed, workload, layer, module, expert, step, kind)):

* ``iid``     : G ~ N(0, grad_std^2), fresh per step.
* ``lowrank`` : G = U diag(sigma) Y^T + N(0, noise_std^2), with U, Y random
                orthonormal (fixed per matrix) and sigma_i = i^-power; fresh
                noise per step. Stands in for C4 training gradients, which are
                not available.
* MoE routed experts: per (layer, step), ``moe_active`` of ``moe_routed``
  experts are drawn without replacement; the others get an all-zero gradient.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Module-type ids. The order is part of the C ABI (include/moara.h).
Q, K, V, O, GATE, UP, DOWN, EXP_GATE, EXP_UP, EXP_DOWN = range(10)
NUM_MODULES = 10
MODULE_NAMES = ("q", "k", "v", "o", "gate", "up", "down", "exp_gate", "exp_up", "exp_down")

_KIND_IDS = {"weight": 1, "noise": 2, "factor": 3, "route": 4, "iid": 5}


@dataclasses.dataclass(frozen=True)
class MatrixSpec:
    name: str
    module: int
    rows: int
    cols: int
    layer: int
    expert: int = -1          # -1: not an expert; >=0 routed expert id; shared experts use 1000+i
    routed: bool = False      # True for routed MoE experts (may be inactive on a step)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    description: str
    matrices: Tuple[MatrixSpec, ...]
    rank_table: Tuple[int, ...]            # length NUM_MODULES, r_tau per module type
    block_size: int
    weight_dtype: str                      # "f32" | "bf16"
    operand_dtype: str                     # GEMM operand dtype used for this workload's headline run
    moment_dtype: str = "f32"              # storage of the direction moments: "f32" | "bf16" (2-byte
                                           # states, the paper's training setting)
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    scale: float = 0.25
    refresh_interval: int = 200
    steps: int = 10
    weight_std: float = 0.02
    grad_recipe: str = "lowrank"          # "iid" | "lowrank"
    grad_std: float = 1e-3                 # iid recipe
    lowrank_rank: int = 64
    lowrank_power: float = 1.0
    noise_std: float = 1e-4
    moe_routed: int = 0
    moe_active: int = 0
    n_layers: int = 1
    refresh_oversample: int = -1           # subspace-iteration oversampling p (-1: p = r)
    refresh_iters: int = 20                # subspace-iteration sweeps q

    @property
    def n_params(self) -> int:
        return sum(m.rows * m.cols for m in self.matrices)

    def rank_of(self, spec: MatrixSpec) -> int:
        return self.rank_table[spec.module]


def _ranks(**kw) -> Tuple[int, ...]:
    t = [0] * NUM_MODULES
    for k, v in kw.items():
        t[MODULE_NAMES.index(k)] = v
    return tuple(t)


def _dense_layer(layer: int, d: int, ffn: int, kv: Optional[int] = None) -> List[MatrixSpec]:
    kv = d if kv is None else kv
    p = f"layer{layer}."
    return [
        MatrixSpec(p + "q", Q, d, d, layer),
        MatrixSpec(p + "k", K, kv, d, layer),
        MatrixSpec(p + "v", V, kv, d, layer),
        MatrixSpec(p + "o", O, d, d, layer),
        MatrixSpec(p + "gate", GATE, ffn, d, layer),
        MatrixSpec(p + "up", UP, ffn, d, layer),
        MatrixSpec(p + "down", DOWN, d, ffn, layer),
    ]


def _mla_layer(layer: int, d: int, ffn: int, heads: int, q_lora: int, kv_lora: int, nope: int, rope: int,
               vdim: int) -> List[MatrixSpec]:
    """DeepSeek-V2 Multi-head Latent Attention layer plus a dense MLP. Module types (a
    reading: the paper assigns ranks per q/k/v/o type only): the query down/up projections
    are q, the joint key-value down projection (latent plus the shared rope key) is k, the
    key-value up projection is v, the output projection is o."""
    p = f"layer{layer}."
    return [
        MatrixSpec(p + "q_a", Q, q_lora, d, layer),
        MatrixSpec(p + "q_b", Q, heads * (nope + rope), q_lora, layer),
        MatrixSpec(p + "kv_a", K, kv_lora + rope, d, layer),
        MatrixSpec(p + "kv_b", V, heads * (nope + vdim), kv_lora, layer),
        MatrixSpec(p + "o", O, d, heads * vdim, layer),
        MatrixSpec(p + "gate", GATE, ffn, d, layer),
        MatrixSpec(p + "up", UP, ffn, d, layer),
        MatrixSpec(p + "down", DOWN, d, ffn, layer),
    ]


def _moe_layer(layer: int, d: int, eff: int, routed: int, shared: int) -> List[MatrixSpec]:
    p = f"layer{layer}."
    out = [MatrixSpec(p + n, t, d, d, layer) for n, t in (("q", Q), ("k", K), ("v", V), ("o", O))]
    for e in list(range(routed)) + [1000 + i for i in range(shared)]:
        tag = f"expert{e}" if e < 1000 else f"shared{e - 1000}"
        isr = e < 1000
        out += [
            MatrixSpec(f"{p}{tag}.gate", EXP_GATE, eff, d, layer, e, isr),
            MatrixSpec(f"{p}{tag}.up", EXP_UP, eff, d, layer, e, isr),
            MatrixSpec(f"{p}{tag}.down", EXP_DOWN, d, eff, layer, e, isr),
        ]
    return out


def _stack(n_layers: int, fn, *a) -> Tuple[MatrixSpec, ...]:
    out: List[MatrixSpec] = []
    for l in range(n_layers):
        out += fn(l, *a)
    return tuple(out)


def build_workloads() -> dict:
    w = {}
    w["layer_d256"] = Workload(
        name="layer_d256",
        description="single Llama-style layer d=256 ffn=688, fp32 weights, iid N(0,1e-3) gradients",
        matrices=_stack(1, _dense_layer, 256, 688),
        rank_table=_ranks(q=64, k=64, v=64, o=64, gate=32, up=32, down=32),
        block_size=64, weight_dtype="f32", operand_dtype="f32",
        weight_std=1e-3, grad_recipe="iid", grad_std=1e-3, steps=10, n_layers=1,
        refresh_oversample=96, refresh_iters=20)
    w["llama_300m"] = Workload(
        name="llama_300m",
        description="Llama-300M-shaped stack: 24 layers d=1024 ffn=2736, bf16 weights, rank-64 1/i gradients",
        matrices=_stack(24, _dense_layer, 1024, 2736),
        rank_table=_ranks(q=128, k=128, v=256, o=256, gate=192, up=192, down=192),
        block_size=64, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
        lowrank_rank=64, lowrank_power=1.0, noise_std=1e-4, steps=400, n_layers=24)
    w["llama2_7b"] = Workload(
        name="llama2_7b",
        description="Llama-2-7B-shaped stack: 32 layers d=4096 ffn=11008, bf16 weights, rank-256 i^-0.8 gradients",
        matrices=_stack(32, _dense_layer, 4096, 11008),
        rank_table=_ranks(q=512, k=512, v=1024, o=1024, gate=768, up=768, down=768),
        block_size=128, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
        lowrank_rank=256, lowrank_power=0.8, noise_std=1e-4, steps=200, n_layers=32)
    w["qwen2_7b"] = Workload(
        name="qwen2_7b",
        description="Qwen2-7B-shaped GQA stack: 28 layers d=3584, k/v 512x3584, ffn=18944, bf16 weights",
        matrices=_stack(28, _dense_layer, 3584, 18944, 512),
        rank_table=_ranks(q=512, k=128, v=128, o=512, gate=1024, up=1024, down=1024),
        block_size=128, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
        lowrank_rank=256, lowrank_power=0.8, noise_std=1e-4, steps=200, n_layers=28)
    w["deepseek_moe"] = Workload(
        name="deepseek_moe",
        description="DeepSeek-MoE-shaped stack: 28 layers d=2048, 64 routed (6 active) + 2 shared experts of ffn 1408",
        matrices=_stack(28, _moe_layer, 2048, 1408, 64, 2),
        rank_table=_ranks(q=512, k=512, v=512, o=512, exp_gate=128, exp_up=128, exp_down=128),
        block_size=128, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
        lowrank_rank=256, lowrank_power=0.8, noise_std=1e-4, steps=200, n_layers=28,
        moe_routed=64, moe_active=6)
    # model-family comparison at 350M scale (Appendix D model table): d = 1024, 24 layers,
    # 16 query heads of 64; GQA with 4 key-value heads; ranks of the Phase 3 rule at
    # r_base = 256 (D = {q, k}, R = {down}, delta_r = 128); B = 32 as for Llama 2 350M
    r350 = _ranks(q=128, k=128, v=256, o=256, gate=256, up=256, down=512)
    for name, ffn, desc in (("llama32_300m", 2736, "Llama-3.2-300M-shaped GQA stack"),
                            ("qwen25_350m", 2816, "Qwen2.5/Qwen3-350M-shaped GQA stack")):
        w[name] = Workload(
            name=name, description=f"{desc}: 24 layers d=1024, k/v 256x1024 (4 kv heads), ffn={ffn}, bf16 weights",
            matrices=_stack(24, _dense_layer, 1024, ffn, 256), rank_table=r350,
            block_size=32, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
            lowrank_rank=64, lowrank_power=1.0, noise_std=1e-4, steps=200, n_layers=24)
    w["deepseek_v2_350m"] = Workload(
        name="deepseek_v2_350m",
        description="DeepSeek-V2-350M-shaped MLA stack: 24 layers d=1024, q_lora 768, kv_lora 256, "
                    "head dims 64/32/64, 16 heads, dense ffn=2736, bf16 weights",
        matrices=_stack(24, _mla_layer, 1024, 2736, 16, 768, 256, 64, 32, 64), rank_table=r350,
        block_size=32, weight_dtype="bf16", operand_dtype="bf16", moment_dtype="bf16",
        lowrank_rank=64, lowrank_power=1.0, noise_std=1e-4, steps=200, n_layers=24)
    return w


WORKLOADS = build_workloads()


def subset(wl: Workload, layers: Sequence[int]) -> Workload:
    """Same workload restricted to the given layers (shapes, ranks and seeds unchanged)."""
    keep = tuple(m for m in wl.matrices if m.layer in set(layers))
    return dataclasses.replace(wl, matrices=keep)


# ----------------------------------------------------------------------------
# seeded generators
# ----------------------------------------------------------------------------

def _key(seed: int, wl: Workload, spec: Optional[MatrixSpec], step: int, kind: str, extra: int = 0):
    wid = sum((i + 1) * ord(c) for i, c in enumerate(wl.name)) & 0xFFFFFFFF
    if spec is None:
        parts = [seed, wid, 0, 0, 0, step, _KIND_IDS[kind], extra]
    else:
        parts = [seed, wid, spec.layer + 1, spec.module + 1, spec.expert + 2, step, _KIND_IDS[kind], extra]
    return [int(p) & 0xFFFFFFFF for p in parts]


def rng(seed: int, wl: Workload, spec: Optional[MatrixSpec], step: int, kind: str, extra: int = 0) -> np.random.Generator:
    """Counter-based Philox generator keyed by (seed, workload, layer, module, expert, step, kind)."""
    ss = np.random.SeedSequence(_key(seed, wl, spec, step, kind, extra))
    return np.random.Generator(np.random.Philox(ss))


def active_set(wl: Workload, step: int, seed: int = 0) -> np.ndarray:
    """Boolean mask over wl.matrices: which matrices get a nonzero gradient on this step."""
    act = np.ones(len(wl.matrices), dtype=bool)
    if wl.moe_routed == 0:
        return act
    chosen = {}
    for i, m in enumerate(wl.matrices):
        if not m.routed:
            continue
        if m.layer not in chosen:
            g = rng(seed, wl, None, step, "route", extra=m.layer + 1)
            chosen[m.layer] = set(g.choice(wl.moe_routed, size=wl.moe_active, replace=False).tolist())
        act[i] = m.expert in chosen[m.layer]
    return act


def weight_np(wl: Workload, i: int, seed: int = 0) -> np.ndarray:
    """Initial weight of matrix i as float32 (the caller casts to the workload's weight dtype)."""
    m = wl.matrices[i]
    g = rng(seed, wl, m, 0, "weight")
    return (wl.weight_std * g.standard_normal((m.rows, m.cols))).astype(np.float32)


def lowrank_factors(wl: Workload, i: int, seed: int = 0):
    """Fixed per-matrix factors (U, sigma, Y) of the low-rank gradient part, float64."""
    m = wl.matrices[i]
    g = rng(seed, wl, m, 0, "factor")
    R = min(wl.lowrank_rank, m.rows, m.cols)
    U = np.linalg.qr(g.standard_normal((m.rows, R)))[0]
    Y = np.linalg.qr(g.standard_normal((m.cols, R)))[0]
    sig = np.arange(1, R + 1, dtype=np.float64) ** (-wl.lowrank_power)
    return U, sig, Y


def grad_np(wl: Workload, i: int, step: int, seed: int = 0, active: Optional[bool] = None) -> np.ndarray:
    """Gradient of matrix i at a step, float32, drawn on the CPU."""
    m = wl.matrices[i]
    if active is None:
        active = bool(active_set(wl, step, seed)[i])
    if not active:
        return np.zeros((m.rows, m.cols), dtype=np.float32)
    if wl.grad_recipe == "iid":
        g = rng(seed, wl, m, step, "iid")
        return (wl.grad_std * g.standard_normal((m.rows, m.cols))).astype(np.float32)
    U, sig, Y = lowrank_factors(wl, i, seed)
    g = rng(seed, wl, m, step, "noise")
    G = (U * sig) @ Y.T + wl.noise_std * g.standard_normal((m.rows, m.cols))
    return G.astype(np.float32)


def grad_device(wl: Workload, i: int, step: int, out, seed: int = 0, active: Optional[bool] = None):
    """Fill the fp32 device tensor ``out`` (rows x cols) with the gradient of matrix i.

    Same distribution as grad_np; the low-rank factors are the same numpy draws,
    the noise comes from torch's device generator (so values differ from
    grad_np). Used where the CPU would be too slow to synthesise a 7B-sized stack.
    """
    import torch
    m = wl.matrices[i]
    if active is None:
        active = bool(active_set(wl, step, seed)[i])
    if not active:
        out.zero_()
        return out
    gen = torch.Generator(device=out.device)
    gen.manual_seed(int(np.random.SeedSequence(_key(seed, wl, m, step, "noise")).generate_state(1, np.uint64)[0] >> 1))
    if wl.grad_recipe == "iid":
        out.normal_(0.0, wl.grad_std, generator=gen)
        return out
    U, sig, Y = lowrank_factors(wl, i, seed)
    Ud = torch.from_numpy((U * sig).astype(np.float32)).to(out.device)
    Yd = torch.from_numpy(Y.astype(np.float32).T.copy()).to(out.device)
    out.normal_(0.0, wl.noise_std, generator=gen)
    out.addmm_(Ud, Yd)
    return out


def weight_device(wl: Workload, i: int, out, seed: int = 0):
    """Fill the device tensor ``out`` with the initial weight of matrix i (torch device RNG)."""
    import torch
    m = wl.matrices[i]
    gen = torch.Generator(device=out.device)
    gen.manual_seed(int(np.random.SeedSequence(_key(seed, wl, m, 0, "weight")).generate_state(1, np.uint64)[0] >> 1))
    tmp = torch.empty(out.shape, dtype=torch.float32, device=out.device)
    tmp.normal_(0.0, wl.weight_std, generator=gen)
    out.copy_(tmp)
    return out


def gaussian_start_np(s: int, w: int, key: Sequence[int]) -> np.ndarray:
    """Seeded Gaussian s x w start block, float64 (a test helper for subspace methods)."""
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence([int(k) & 0xFFFFFFFF for k in key])))
    return g.standard_normal((s, w))
