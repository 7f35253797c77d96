"""The torch.optim integration in a training loop: a small Llama (random init, synthetic
tokens) trained with MoARa on its projection weights and AdamW on the rest."""
import numpy as np
import pytest
import torch

from tests.harness import have_gpu

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs an MI355X GPU")]


def _model(seed=0):
    from transformers import LlamaConfig, LlamaForCausalLM
    torch.manual_seed(seed)
    cfg = LlamaConfig(vocab_size=512, hidden_size=256, intermediate_size=688, num_hidden_layers=2,
                      num_attention_heads=4, num_key_value_heads=4, max_position_embeddings=128)
    return LlamaForCausalLM(cfg).cuda()


def _opt(model, **kw):
    from paper_2609_15037_amd import moara as M
    from paper_2609_15037_amd.optim import MoARa, moara_targets
    targets, others = moara_targets(model)
    ranks = M.moara_allocate_ranks(64, range(7), [M.MOARA_Q, M.MOARA_K], [M.MOARA_DOWN], 32)
    return MoARa(targets, others, lr=kw.pop("lr", 1e-2), rank_table=ranks, block_size=64,
                 refresh_interval=kw.pop("refresh_interval", 20), **kw)


def _batch(seed, step):
    g = torch.Generator().manual_seed(1000 * seed + step)
    return torch.randint(0, 512, (8, 64), generator=g).cuda()


def test_small_llama_trains_with_moara():
    from paper_2609_15037_amd.optim import warmup_cosine
    model = _model()
    opt = _opt(model)
    sched = torch.optim.lr_scheduler.LambdaLR(opt, warmup_cosine(40))
    x = _batch(1, 0)   # one batch, repeated: the loss must fall
    losses = []
    for step in range(40):
        loss = model(input_ids=x, labels=x).loss
        loss.backward()
        torch.nn.utils.clip_grad_norm_(model.parameters(), 1.0)
        opt.step()
        sched.step()
        opt.zero_grad()
        losses.append(float(loss.detach()))
        if step % 10 == 0:
            print(f"[train] step {step} loss {losses[-1]:.4f} lr {sched.get_last_lr()[0]:.2e}", flush=True)
    assert np.isfinite(losses).all()
    assert losses[-1] < 0.8 * losses[0], losses


def test_other_parameters_follow_adamw_and_state_dict_round_trips():
    model = _model(2)
    opt = _opt(model)
    others = opt.param_groups[1]["params"]
    ref = [p.detach().clone().requires_grad_(True) for p in others]
    ref_opt = torch.optim.AdamW(ref, lr=1e-2, betas=(0.9, 0.999), eps=1e-6, weight_decay=0.0)
    for step in range(3):
        x = _batch(2, step)
        model(input_ids=x, labels=x).loss.backward()
        for p, q in zip(others, ref):
            q.grad = p.grad.detach().clone()
        opt.step()
        ref_opt.step()
        opt.zero_grad()
    for p, q in zip(others, ref):
        assert torch.equal(p.detach(), q.detach())
    # checkpoint: a second optimizer loaded from the first continues identically
    model2 = _model(3)
    model2.load_state_dict(model.state_dict())
    opt2 = _opt(model2)
    opt2.load_state_dict(opt.state_dict())
    x = _batch(2, 9)
    model(input_ids=x, labels=x).loss.backward()
    for p1, p2 in zip(model.parameters(), model2.parameters()):   # the same gradients for both
        p2.grad = p1.grad.detach().clone()
    for o in (opt, opt2):
        o.step()
        o.zero_grad()
    for (n1, p1), (n2, p2) in zip(model.named_parameters(), model2.named_parameters()):
        assert torch.equal(p1.detach(), p2.detach()), n1


def test_experts_without_gradient_are_skipped():
    """Routed experts that no token reached have no gradient: their weights, moments and
    step counters stay as they were (the library's skip rule), the others step."""
    from paper_2609_15037_amd import moara as M
    from paper_2609_15037_amd.optim import MoARa, moara_targets

    class Expert(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.up_proj = torch.nn.Linear(64, 96, bias=False)
            self.down_proj = torch.nn.Linear(96, 64, bias=False)

        def forward(self, x):
            return self.down_proj(torch.relu(self.up_proj(x)))

    class Moe(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.experts = torch.nn.ModuleList([Expert() for _ in range(4)])

    torch.manual_seed(4)
    moe = Moe().cuda()
    experts = moe.experts
    targets, others = moara_targets(moe)
    assert [m for _, m in targets[:2]] == [M.MOARA_EXP_UP, M.MOARA_EXP_DOWN]
    ranks = [0] * 10
    ranks[M.MOARA_EXP_UP] = ranks[M.MOARA_EXP_DOWN] = 16
    opt = MoARa(targets, others, lr=1e-2, rank_table=ranks, block_size=32, refresh_interval=10)
    x = torch.randn(32, 64, device="cuda")
    before = [p.detach().clone() for p, _ in targets]
    for _ in range(2):
        loss = experts[0](x).square().mean() + experts[2](x).square().mean()   # experts 1 and 3 unused
        loss.backward()
        opt.step()
        opt.zero_grad()
    for i, (p, _) in enumerate(targets):
        used = i // 2 in (0, 2)
        assert torch.equal(p.detach(), before[i]) != used, i
        assert M.moara_get_tensor(opt.moara_state, i, M.MOARA_T_STEP) == (2 if used else 0)


def test_moara_steps_of_a_bf16_model_match_the_oracle():
    """The optimizer wrapper end to end on a bf16 model: three MoARa.step calls under a
    warmup schedule (the lr is read from param_groups), bf16 gradients copied to fp32 by
    the wrapper. Before the first step every target's projector is set to the oracle's SVD
    of its first gradient through load_state_dict (the library's own refresh is checked
    against the oracle elsewhere). The oracle repeats each step on every target weight from
    the same fp32 gradient values, the same lr and that projector, with the bf16 operand
    and weight roundings; weights agree to the bf16 bar and in bf16 ulps."""
    from oracle import moara_oracle as O
    from paper_2609_15037_amd import moara as M
    from paper_2609_15037_amd.optim import warmup_cosine
    from tests.harness import TOL_BF16, bf16_ulp, compare
    model = _model(5).to(torch.bfloat16)
    opt = _opt(model, refresh_interval=0)
    sched = torch.optim.lr_scheduler.LambdaLR(opt, warmup_cosine(20, warmup_frac=0.2))   # 4 warmup steps
    targets = list(opt.param_groups[0]["params"])
    cfg = opt._cfg
    Wo = [p.detach().float().cpu().numpy().astype(np.float64) for p in targets]
    ocfg, ost = [], []
    for p, mod in zip(targets, opt._modules):
        m, n = M.flatten_shape(p.shape)
        oc = O.OracleConfig(block_size=cfg.block_size, rank=cfg.rank_table[mod], beta1=cfg.beta1, beta2=cfg.beta2,
                            adam_eps=cfg.adam_eps, scale=cfg.scale, refresh_interval=0, weight_dtype="bf16",
                            operand_dtype="bf16")
        ocfg.append(oc)
        ost.append(O.init_state(m, n, oc))
    report, lrs = {}, []
    for step in range(3):
        x = _batch(5, step)
        model(input_ids=x, labels=x).loss.backward()
        grads = [p.grad.detach().float().cpu().numpy().reshape(M.flatten_shape(p.shape)) for p in targets]
        lr = float(opt.param_groups[0]["lr"])
        lrs.append(lr)
        if step == 0:
            for i in range(len(targets)):
                ost[i].P = O.round_f32(O.truncated_svd(O.decompose(grads[i], cfg.block_size)[1], ocfg[i].rank,
                                                       ost[i].side))
            opt.load_state_dict({"moara": [{"step": 0, "P": torch.from_numpy(o.P.astype(np.float32))} for o in ost],
                                 "adamw": None, "lr": [g["lr"] for g in opt.param_groups]})
            sd0 = opt.state_dict()   # a projector set before the first step is saved too
            for o, d in zip(ost, sd0["moara"]):
                assert d["step"] == 0 and np.array_equal(d["P"].numpy(), o.P.astype(np.float32))
        print(f"[wrapper] step {step}, lr {lr:.3e}", flush=True)
        opt.step()
        sched.step()
        opt.zero_grad()
        torch.cuda.synchronize()
        for i in range(len(targets)):
            Wo[i] = O.step(Wo[i], grads[i], ost[i], ocfg[i], lr)
    assert len(set(lrs)) == 3   # the warmup changed the lr every step
    beyond, exact = 0, 1.0
    for i, p in enumerate(targets):
        Wg = p.detach().float().cpu().numpy().astype(np.float64).reshape(Wo[i].shape)
        compare(f"W[{i}]", Wg, Wo[i], TOL_BF16, report)
        d = np.abs(Wg - Wo[i]) / bf16_ulp(np.maximum(np.abs(Wg), np.abs(Wo[i])))
        beyond, exact = beyond + int(np.sum(d > 2)), min(exact, float(np.mean(d == 0)))
        assert M.moara_get_tensor(opt.moara_state, i, M.MOARA_T_STEP) == 3
        np.testing.assert_allclose(M.moara_get_tensor(opt.moara_state, i, M.MOARA_T_EXP_AVG), ost[i].exp_avg,
                                   rtol=0, atol=TOL_BF16 * float(np.sqrt(np.mean(ost[i].exp_avg ** 2))) + 1e-30)
    # first steps from zero moments: where |R| is within fp32 rounding of zero, Adam's
    # first output (about sign(R)) may flip, which moves a few weights by many ulps
    print(f"[wrapper] {len(targets)} targets: worst floored rel err {max(report.values()):.3e}, "
          f"{beyond} weights more than 2 bf16 ulps off, min exact fraction {exact:.4f}", flush=True)
