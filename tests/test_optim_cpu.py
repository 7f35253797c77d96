"""Host-side parts of the torch.optim integration (no GPU needed)."""
import math

import pytest
import torch

from paper_2609_15037_amd import moara as M
from paper_2609_15037_amd.optim import moara_targets, warmup_cosine


def test_warmup_cosine_schedule_shape():
    # Appendix D: 10 % linear warmup, cosine decay to 0.1 of the peak
    f = warmup_cosine(100)
    assert f(0) == pytest.approx(0.1) and f(9) == pytest.approx(1.0)
    assert f(10) == pytest.approx(1.0)
    assert f(55) == pytest.approx(0.1 + 0.9 * 0.5 * (1 + math.cos(math.pi * 0.5)))
    assert f(100) == pytest.approx(0.1) and f(1000) == pytest.approx(0.1)
    vals = [f(s) for s in range(10, 101)]
    assert all(a >= b for a, b in zip(vals, vals[1:]))


def test_targets_are_the_projection_weights():
    class Attn(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.q_proj = torch.nn.Linear(8, 8, bias=False)
            self.k_proj = torch.nn.Linear(8, 4, bias=False)
            self.o_proj = torch.nn.Linear(8, 8, bias=True)
            self.norm = torch.nn.LayerNorm(8)

    class Net(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.embed = torch.nn.Embedding(10, 8)
            self.attn = Attn()
            self.down_proj = torch.nn.Linear(16, 8, bias=False)

    net = Net()
    t, o = moara_targets(net)
    assert [(p.shape, m) for p, m in t] == [(net.attn.q_proj.weight.shape, M.MOARA_Q),
                                             (net.attn.k_proj.weight.shape, M.MOARA_K),
                                             (net.attn.o_proj.weight.shape, M.MOARA_O),
                                             (net.down_proj.weight.shape, M.MOARA_DOWN)]
    assert len(o) == 4   # embedding, o_proj bias, norm weight and bias


def test_expert_projections_take_the_expert_types():
    class Expert(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.gate_proj = torch.nn.Linear(8, 12, bias=False)
            self.down_proj = torch.nn.Linear(12, 8, bias=False)

    class Moe(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.experts = torch.nn.ModuleList([Expert(), Expert()])
            self.up_proj = torch.nn.Linear(8, 12, bias=False)   # a dense MLP projection

    t, _ = moara_targets(Moe())
    assert [m for _, m in t] == [M.MOARA_EXP_GATE, M.MOARA_EXP_DOWN, M.MOARA_EXP_GATE, M.MOARA_EXP_DOWN,
                                 M.MOARA_UP]
