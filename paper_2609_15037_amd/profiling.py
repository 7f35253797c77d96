"""Setup phase of MoARa's rank reallocation (Algorithm 1, Phases 1-3; Section 3.2).

Phase 1 logs the alignment S(W, t) = cos(G_t, G_recon,t) of every projected matrix at
the profiling steps t in {x, 2x, ..., N_p} of a uniform-rank GaLore run; the library
computes S on the device (`moara_alignment`). Phase 2 averages it into the module
scores S_tau = E_{t, W in tau}[S(W, t)] and checks the chosen sets: the receivers must be
the modules of lowest S_tau. The donors cannot be read off S: the paper picks them from
a single-module rank-reduction ablation (high alignment there reflected redundancy, not
robustness), so they are an input here (q and k in the paper's Llama/Qwen runs). Phase 3
turns (r_base, donors, receivers, delta_r) into the per-module rank table
(`moara_allocate_ranks`; delta_r = r_base / 2 by default, as in the paper).

    prof = AlignmentProfile(modules_of_matrices, stride=50, n_p=1000)
    ... each step t of the profiling run (after moara_step, same gradients):
    if prof.due(t): prof.record(state, grads)
    receivers = prof.receivers()                 # lowest S_tau, if clearly separated
    ok, why = prof.validate(donors, receivers)
    ranks = allocate(r_base, types, donors, receivers)
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import moara as M


class AlignmentProfile:
    """Running S_tau over the profiling steps {stride, 2 stride, ..., n_p}.

    modules: the module type of each matrix of the library state, in state order.
    """

    def __init__(self, modules: Sequence[int], stride: int, n_p: int):
        if stride < 1 or n_p < stride:
            raise ValueError("need 1 <= stride <= n_p")
        self.modules = np.asarray([int(m) for m in modules], dtype=np.int64)
        self.stride, self.n_p = int(stride), int(n_p)
        self._sum: Dict[int, float] = {}
        self._cnt: Dict[int, int] = {}
        self.steps: List[int] = []

    def due(self, t: int) -> bool:
        """Whether step t (1-based count of optimizer steps) is a profiling step."""
        return 0 < t <= self.n_p and t % self.stride == 0

    def add(self, s: Sequence[float], t: Optional[int] = None) -> None:
        """Fold one step's per-matrix S values (NaN = matrix not active) into the sums."""
        s = np.asarray(s, dtype=np.float64)
        if s.shape != self.modules.shape:
            raise ValueError(f"expected {self.modules.size} values, got {s.shape}")
        for tau in np.unique(self.modules):
            v = s[(self.modules == tau) & ~np.isnan(s)]
            if v.size:
                self._sum[int(tau)] = self._sum.get(int(tau), 0.0) + float(v.sum())
                self._cnt[int(tau)] = self._cnt.get(int(tau), 0) + int(v.size)
        if t is not None:
            self.steps.append(int(t))

    def record(self, st: M.State, grads, active=None, stream=None, t: Optional[int] = None) -> np.ndarray:
        """S(W, t) of every active matrix with its current projector (device diagnostic),
        folded into the module sums; returns the per-matrix values."""
        s = M.moara_alignment(st, grads, active=active, stream=stream)
        self.add(s, t)
        return s

    def s_tau(self) -> Dict[int, float]:
        """S_tau per module type seen so far."""
        return {tau: self._sum[tau] / self._cnt[tau] for tau in sorted(self._sum)}

    def ranking(self) -> List[Tuple[int, float]]:
        """(module, S_tau) from the lowest score to the highest."""
        return sorted(self.s_tau().items(), key=lambda kv: kv[1])

    def receivers(self, margin: float = 0.05) -> List[int]:
        """The lowest-S_tau module when it sits below every other module by at least
        `margin` (the paper's receiver, mlp.down, is separated by 0.10-0.15); else []."""
        r = self.ranking()
        if len(r) < 2 or r[1][1] - r[0][1] < margin:
            return []
        return [r[0][0]]

    def validate(self, donors: Sequence[int], receivers: Sequence[int]) -> Tuple[bool, str]:
        """Phase 2 check of chosen sets: disjoint, all profiled, and the receivers are
        the |R| modules of lowest S_tau."""
        s = self.s_tau()
        D, R = set(int(x) for x in donors), set(int(x) for x in receivers)
        if D & R:
            return False, "donor and receiver sets overlap"
        missing = (D | R) - set(s)
        if missing:
            return False, f"modules without alignment samples: {sorted(missing)}"
        lowest = {tau for tau, _ in self.ranking()[:len(R)]}
        if R != lowest:
            return False, f"receivers {sorted(R)} are not the {len(R)} lowest-S_tau modules {sorted(lowest)}"
        return True, "ok"


def allocate(r_base: int, types: Sequence[int], donors: Sequence[int], receivers: Sequence[int],
             delta_r: Optional[int] = None) -> List[int]:
    """Phase 3 rank table (MOARA_NUM_MODULES entries): r_base - delta_r for donors,
    r_base + delta_r |D| / |R| for receivers, r_base for the other types in `types`
    (delta_r defaults to r_base / 2)."""
    if delta_r is None:
        delta_r = int(r_base) // 2
    return M.moara_allocate_ranks(int(r_base), types, donors, receivers, int(delta_r))
