"""torch.optim integration of the MoARa library (training-loop use).

MoARa updates the projected weights: the attention q/k/v/o and MLP gate/up/down
matrices of every layer (and MoE experts), each with its module's rank, by the
library's step (`moara_step`: decomposition, projection, Adam on the projected
moments and the magnitudes, back-projection, scaled update, projector refresh
every `refresh_interval` steps). Every other parameter (embeddings, norms, the
output head) takes plain AdamW with the same betas and eps, as in the paper's
training setup (Appendix D: AdamW beta = (0.9, 0.999), eps = 1e-6, zero weight
decay, bias correction, GaLore scale 0.25 and T = 200).

The learning rate of both groups comes from `param_groups`, so torch's LR
schedulers drive it; `warmup_cosine` gives the paper's schedule (10 % linear
warmup, cosine decay to 0.1 of the peak). Gradient clipping (the paper clips at
1.0 for 7B) stays with the training loop (`torch.nn.utils.clip_grad_norm_`),
before `step()`.

    targets, others = moara_targets(model)          # [(param, module id)], [param]
    opt = MoARa(targets, others, lr=1e-2, rank_table=..., block_size=64)
    sched = torch.optim.lr_scheduler.LambdaLR(opt, warmup_cosine(total_steps))
    loss.backward(); opt.step(); sched.step(); opt.zero_grad()

Gradients of the projected weights must be fp32 for the library; for a bf16
model the optimizer copies them into fp32 buffers it owns. The library's
kernels do all the work on the projected weights; this module only marshals.
"""
from __future__ import annotations

import copy
import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import moara as M

# module ids of the usual Llama / Qwen / DeepSeek parameter names (last two name parts);
# MLP projections inside an MoE expert ("...experts.3.gate_proj.weight",
# "...shared_experts.up_proj.weight") take the expert types
_MODULE_OF = {
    "q_proj": M.MOARA_Q, "k_proj": M.MOARA_K, "v_proj": M.MOARA_V, "o_proj": M.MOARA_O,
    "gate_proj": M.MOARA_GATE, "up_proj": M.MOARA_UP, "down_proj": M.MOARA_DOWN,
}
_EXPERT_OF = {M.MOARA_GATE: M.MOARA_EXP_GATE, M.MOARA_UP: M.MOARA_EXP_UP, M.MOARA_DOWN: M.MOARA_EXP_DOWN}


def moara_targets(model: torch.nn.Module) -> Tuple[List[Tuple[torch.nn.Parameter, int]], List[torch.nn.Parameter]]:
    """Split a model's trainable parameters into MoARa targets, (weight, module id) for the
    q/k/v/o/gate/up/down projection weights (`*.q_proj.weight` and so on; expert types for
    MLP projections under a module path containing "expert"), and the rest."""
    targets, others = [], []
    for name, p in model.named_parameters():
        if not p.requires_grad:
            continue
        parts = name.split(".")
        mod = _MODULE_OF.get(parts[-2]) if len(parts) >= 2 and parts[-1] == "weight" and p.dim() >= 2 else None
        if mod is not None and any("expert" in q for q in parts[:-2]):
            mod = _EXPERT_OF.get(mod, mod)
        if mod is None:
            others.append(p)
        else:
            targets.append((p, mod))
    return targets, others


def warmup_cosine(total_steps: int, warmup_frac: float = 0.1, min_ratio: float = 0.1):
    """LR factor for torch.optim.lr_scheduler.LambdaLR: linear warmup over the first
    `warmup_frac` of the steps, then cosine decay from 1 to `min_ratio` (Appendix D)."""
    warm = max(1, int(round(warmup_frac * total_steps)))

    def f(step: int) -> float:
        if step < warm:
            return (step + 1) / warm
        t = min(1.0, (step - warm) / max(1, total_steps - warm))
        return min_ratio + (1.0 - min_ratio) * 0.5 * (1.0 + math.cos(math.pi * t))
    return f


class MoARa(torch.optim.Optimizer):
    """MoARa for the projected weights (C library), AdamW for the other parameters.

    targets: [(weight parameter, module id MOARA_Q .. MOARA_EXP_DOWN)], weights of
             dtype fp32 or bf16 (all the same), at least two axes (flattened by the
             first axis, Appendix B.1).
    others:  the remaining parameters (AdamW).
    rank_table: per-module ranks r_tau (MOARA_NUM_MODULES entries, 0 = unused); see
             moara_allocate_ranks for the Phase 3 rule.
    Other keyword arguments go to moara_default_config (block_size, scale,
    refresh_interval, operand_dtype, refresh_oversample, ...).
    """

    def __init__(self, targets: Sequence[Tuple[torch.nn.Parameter, int]], others: Iterable[torch.nn.Parameter],
                 lr: float = 1e-2, betas=(0.9, 0.999), eps: float = 1e-6, rank_table: Sequence[int] = (),
                 block_size: int = 64, scale: float = 0.25, refresh_interval: int = 200, **config):
        targets = list(targets)
        others = list(others)
        if not targets:
            raise ValueError("MoARa needs at least one target weight")
        wdt = {t.dtype for t, _ in targets}
        if len(wdt) != 1 or next(iter(wdt)) not in (torch.float32, torch.bfloat16):
            raise ValueError(f"target weights must all be fp32 or all bf16, got {wdt}")
        groups = [{"params": [t for t, _ in targets], "moara": True}]
        if others:
            groups.append({"params": others, "moara": False})
        super().__init__(groups, dict(lr=lr, betas=tuple(betas), eps=eps))
        self._modules = [int(m) for _, m in targets]
        self._weight_bf16 = next(iter(wdt)) == torch.bfloat16
        self._cfg = M.moara_default_config(
            rank_table=list(rank_table), block_size=int(block_size), beta1=float(betas[0]),
            beta2=float(betas[1]), adam_eps=float(eps), scale=float(scale), refresh_interval=int(refresh_interval),
            weight_dtype=M.MOARA_BF16 if self._weight_bf16 else M.MOARA_F32, **config)
        self._descs = M.make_descs([(tuple(t.shape), m) for t, m in targets])
        self._st: Optional[M.State] = None
        self._g32: List[Optional[torch.Tensor]] = [None] * len(targets)
        self._adamw = torch.optim.AdamW(others, lr=lr, betas=tuple(betas), eps=eps, weight_decay=0.0) if others else None

    def _device(self):
        """The target weights' GPU as the current device: the library's calls act on the
        current device, and the state lives on the one that was current at its creation."""
        return torch.cuda.device(self.param_groups[0]["params"][0].device)

    @property
    def moara_state(self) -> Optional[M.State]:
        """The library state (created at the first step), e.g. for moara_alignment."""
        return self._st

    def _grads(self) -> List[Optional[torch.Tensor]]:
        """fp32 contiguous gradients of the targets; None where a target has no gradient
        (e.g. a routed expert no token reached this step: it is skipped, its state kept)."""
        out = []
        for i, p in enumerate(self.param_groups[0]["params"]):
            if p.grad is None:
                out.append(None)
                continue
            g = p.grad
            if g.dtype != torch.float32 or not g.is_contiguous():
                if self._g32[i] is None:
                    self._g32[i] = torch.empty(p.shape, dtype=torch.float32, device=p.device)
                self._g32[i].copy_(g)
                g = self._g32[i]
            out.append(g)
        return out

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        tg = self.param_groups[0]
        with self._device():
            if self._st is None:
                self._st = M.moara_create_state(self._cfg, self._descs)
            grads = self._grads()
            active = [g is not None for g in grads]
            if any(active):
                M.moara_step(self._st, list(tg["params"]), grads, lr=float(tg["lr"]),
                             active=None if all(active) else active)
        if self._adamw is not None:
            og = self.param_groups[1]
            for g in self._adamw.param_groups:   # the schedule drives both groups
                g["lr"] = og["lr"]
            self._adamw.step()
        return loss

    def state_dict(self) -> Dict:
        """Library state (projectors, moments, magnitude moments, step counters) as CPU
        tensors, plus the AdamW state of the other parameters and the group settings."""
        lib = None
        if self._st is not None:
            with self._device():
                lib = []
                for i in range(len(self._modules)):
                    d = {"step": int(M.moara_get_tensor(self._st, i, M.MOARA_T_STEP))}
                    for name, which in (("P", M.MOARA_T_P), ("exp_avg", M.MOARA_T_EXP_AVG),
                                        ("exp_avg_sq", M.MOARA_T_EXP_AVG_SQ), ("mag_avg", M.MOARA_T_MAG_AVG),
                                        ("mag_avg_sq", M.MOARA_T_MAG_AVG_SQ)):
                        try:
                            d[name] = torch.from_numpy(np.array(M.moara_get_tensor(self._st, i, which)))
                        except M.MoaraError as e:   # no projector yet: nothing to save for P
                            if which != M.MOARA_T_P or e.status != M.MOARA_E_STATE:
                                raise
                    lib.append(d)
        # the AdamW part is copied: torch's state_dict hands out the live moment tensors, and
        # loading those into another optimizer would alias the two
        return {"moara": lib, "adamw": copy.deepcopy(self._adamw.state_dict()) if self._adamw else None,
                "lr": [g["lr"] for g in self.param_groups]}

    def load_state_dict(self, sd: Dict) -> None:
        for g, lr in zip(self.param_groups, sd["lr"]):
            g["lr"] = lr
        if self._adamw is not None and sd["adamw"] is not None:
            self._adamw.load_state_dict(sd["adamw"])
        if sd["moara"] is None:
            return
        with self._device():
            if self._st is None:
                self._st = M.moara_create_state(self._cfg, self._descs)
            for i, d in enumerate(sd["moara"]):
                for name, which in (("P", M.MOARA_T_P), ("exp_avg", M.MOARA_T_EXP_AVG),
                                    ("exp_avg_sq", M.MOARA_T_EXP_AVG_SQ), ("mag_avg", M.MOARA_T_MAG_AVG),
                                    ("mag_avg_sq", M.MOARA_T_MAG_AVG_SQ)):
                    if name in d:
                        M.moara_set_tensor(self._st, i, which, d[name].numpy())
                M.moara_set_tensor(self._st, i, M.MOARA_T_STEP, np.int64(d["step"]))
