"""Benchmark of the MoARa optimizer hot path on one MI355X.

One "step" = one Algorithm 1 training-phase optimizer step over every projected
matrix of the stack (decompose + Optimizer_M, projection + Optimizer_V,
back-projection + update), inputs already resident in HBM. The projector refresh
(TruncatedSVD of every matrix) is timed separately and reported as
ms_per_refresh; the refresh interval of 200 steps gives the amortised figure.

Prints ONE JSON line. Default workload: the Llama-2-7B-shaped stack (32 layers,
d=4096, ffn=11008, bf16 weights, fp32 gradients, ranks q/k 512, v/o 1024, mlp
768, B=128), synthetic seeded inputs.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM = 8.0e12          # B/s
PEAK_BF16 = 2.5e15         # dense MFMA flop/s
PEAK_F32 = 157.3e12
PEAK_F64 = 78.6e12


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama2_7b")
    ap.add_argument("--operand", default=None, help="GEMM operand dtype override: bf16 | f32")
    ap.add_argument("--moments", default=None, help="direction-moment storage override: f32 | bf16")
    ap.add_argument("--refresh-reps", type=int, default=3, help="refreshes timed; the median is reported")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-layers", type=int, default=None,
                    help="layers the oracle baseline runs (default: the whole stack up to 0.5 G parameters, else 2)")
    ap.add_argument("--cpu-one-thread", action="store_true",
                    help="also time the oracle baseline with its BLAS limited to one thread")
    ap.add_argument("--layers", type=int, default=None, help="use only the first N layers (profiling runs)")
    ap.add_argument("--refresh-iters", type=int, default=None,
                    help="override the subspace-iteration count (the default is the workload's)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain elementwise copy kernel (y = -x) over this many MiB before the steps: the "
                         "reference dispatch for scaling the FETCH_SIZE / WRITE_SIZE counters of a profiling run")
    return ap.parse_args()


def v_path(wl, m, operand: str) -> bool:
    """Whether the library materialises V in bf16 for this matrix (the large-tile projection
    path): the shape rule of the library's state layout."""
    if operand != "bf16":
        return False
    B = wl.block_size
    if B < 4 or B > 256 or (B & (B - 1)):
        return False
    r = wl.rank_of(m)
    if m.cols % 4 or r % 4:
        return False
    k = -(-m.cols // B)
    if m.rows <= m.cols:
        return k <= 160 and m.rows % 32 == 0
    return k <= 512 and m.cols % 32 == 0


def algorithmic_cost(wl, operand: str, weight_bytes: int, mask=None, moment_bytes: int = 4):
    """Per-step algorithmic bytes and flops per kernel (what each kernel of this split must
    move or compute, given its inputs and outputs), over the matrices in `mask` (all if None)."""
    ob = 2 if operand == "bf16" else 4
    cost = {"decompose": [0, 0], "project": [0, 0], "backproject": [0, 0]}
    for i, m in enumerate(wl.matrices):
        if mask is not None and not mask[i]:
            continue
        r = wl.rank_of(m)
        M, N = m.rows, m.cols
        s, L = (M, N) if M <= N else (N, M)
        k = -(-N // wl.block_size)
        vp = v_path(wl, m, operand)
        # decompose + Optimizer_M: read G; write inv and dM; read+write two magnitude moments;
        # write V in bf16 on the large-tile path
        cost["decompose"][0] += 4 * M * N + 4 * M * k * 6 + (2 * M * N if vp else 0)
        # projection + Optimizer_V: read V (or G and inv), read P, read+write the two direction
        # moments (fp32 or bf16), write N
        cost["project"][0] += ((2 * M * N if vp else 4 * M * N + 4 * M * k) + ob * s * r + 4 * moment_bytes * L * r
                               + ob * L * r)
        cost["project"][1] += 2 * M * N * r
        # back-projection + update: read N and P, read dM, read+write W
        cost["backproject"][0] += ob * L * r + ob * s * r + 4 * M * k + 2 * weight_bytes * M * N
        cost["backproject"][1] += 2 * M * N * r
    return cost


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "llama2_7b_step_pmc_traffic.txt")
TRAFFIC_SOURCES = ["paper_2609_15037_amd/csrc/common.h", "paper_2609_15037_amd/csrc/gemm.h",
                   "paper_2609_15037_amd/csrc/gemm_nt.hip", "paper_2609_15037_amd/csrc/decompose.hip"]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary, if it was taken on this workload with the kernel sources as they are now."""
    import hashlib
    if workload != "llama2_7b" or not os.path.exists(TRAFFIC_FILE):
        return None
    h = hashlib.sha256()
    for src in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    rec, val = None, None
    for line in open(TRAFFIC_FILE):
        parts = line.split()
        if len(parts) == 2 and parts[0] == "sources-sha256":
            rec = parts[1]
        if len(parts) == 3 and parts[0] == "traffic-bytes-per-launch" and parts[1] == kernel:
            val = float(parts[2])
    return val if rec == h.hexdigest() else None


def method_cost(wl, operand_bytes: int, weight_bytes: int, mask=None, moment_bytes: int = 4):
    """What the method itself must move and compute per step, whatever the kernel split:
    read G, read+write W, read+write the two direction moments, read+write the two
    magnitude moments, read P; two GEMMs of 2mnr flops each (matrices in `mask`, all if None)."""
    by, fl = 0, 0
    for i, m in enumerate(wl.matrices):
        if mask is not None and not mask[i]:
            continue
        r = wl.rank_of(m)
        M, N = m.rows, m.cols
        s, L = min(M, N), max(M, N)
        k = -(-N // wl.block_size)
        by += 4 * M * N + 2 * weight_bytes * M * N + 4 * moment_bytes * r * L + 16 * M * k + operand_bytes * s * r
        fl += 4 * M * N * r
    return by, fl


def refresh_cost(wl, p_over: int, q: int, bf16_early: bool):
    """Algorithmic flops of one projector refresh by precision, and its roofline time.

    Per matrix (s = min(m, n), L = max(m, n), w = r + p columns): q iterations of Y = X Z,
    Z2 = X^T Y (4 L s w flops each; the first q - 3 on bf16 MFMA when the operands are bf16,
    taken here for every matrix), q + 1 CholeskyQRs (q of an s x w iterate, one of the
    L x w one): the symmetric fp64 Gram (rows w^2), the fp64 Cholesky and triangular inverse
    (w^3 / 3 each) and the triangular fp32 product Z R^-1 (rows w^2), and the Ritz vectors
    Q B (2 s w r, fp32). The Jacobi sweeps of the Rayleigh-Ritz step are iterative and left
    out, so the bound is below what any implementation of this iteration needs."""
    f16 = f32 = f64 = 0.0
    for m in wl.matrices:
        r = wl.rank_of(m)
        s, L = min(m.rows, m.cols), max(m.rows, m.cols)
        w = min(s, r + (r if p_over < 0 else p_over))
        n16 = max(0, q - 3) if bf16_early else 0
        it = 4.0 * L * s * w
        f16 += n16 * it
        f32 += (q - n16) * it
        rows = q * s + L                           # rows of the q + 1 orthonormalised iterates
        f64 += rows * w * w + (q + 1) * 2.0 * w ** 3 / 3.0
        f32 += rows * w * w + 2.0 * s * w * r
    t = f16 / PEAK_BF16 + f32 / PEAK_F32 + f64 / PEAK_F64
    return {"bf16_flops": f16, "f32_flops": f32, "f64_flops": f64, "roofline_ms": t * 1e3}


def cpu_baseline(wl, layers, one_thread: bool = False, moments: str = "f32"):
    """The oracle (as it stands) on a bounded sample: the first `layers` layers' matrices
    (None: the whole stack if it has at most 0.5 G parameters, else two layers), with their
    projectors already set (steps only), timed on the host cores; optionally again with
    the BLAS limited to one thread. A partial sample also reports the time it extrapolates
    to for the whole stack (per-layer cost times the layer count)."""
    import workloads as WL
    from oracle import moara_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        blas = ",".join(sorted({i.get("internal_api", "?") for i in threadpool_info()}))
    except Exception:
        threads, blas = os.cpu_count(), "?"
    layer_ids = sorted({m.layer for m in wl.matrices})
    if layers is None:
        layers = len(layer_ids) if wl.n_params <= 0.5e9 else 2
    layers = max(1, min(layers, len(layer_ids)))
    sub = WL.subset(wl, layer_ids[:layers])
    if sub.moe_routed > 0:   # MoE: the matrices the router activates on step 0 (attention, shared, 6 routed)
        act = WL.active_set(sub, 0)
        sub = dataclasses.replace(sub, matrices=tuple(m for m, a in zip(sub.matrices, act) if a))
    mats = sub.matrices
    Ws, Gs, sts, cfgs = [], [], [], []
    for i, m in enumerate(mats):
        G = WL.grad_np(sub, i, 0)
        W = WL.weight_np(sub, i).astype(np.float64)
        cfg = O.OracleConfig(block_size=sub.block_size, rank=sub.rank_of(m), adam_eps=sub.adam_eps, scale=sub.scale,
                             refresh_interval=0, weight_dtype=sub.weight_dtype, operand_dtype=sub.operand_dtype,
                             moment_dtype=moments)
        st = O.init_state(m.rows, m.cols, cfg)
        s = min(m.rows, m.cols)
        st.P = np.linalg.qr(np.random.default_rng(i).standard_normal((s, cfg.rank)))[0]
        Ws.append(W); Gs.append(G); sts.append(st); cfgs.append(cfg)
    import copy
    sts1 = copy.deepcopy(sts) if one_thread else None
    W1 = [w.copy() for w in Ws] if one_thread else None
    t0 = time.perf_counter()
    for i in range(len(mats)):
        Ws[i] = O.step(Ws[i], Gs[i], sts[i], cfgs[i], sub.lr)
    dt = time.perf_counter() - t0
    dt1 = None
    if one_thread:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            for i in range(len(mats)):
                W1[i] = O.step(W1[i], Gs[i], sts1[i], cfgs[i], sub.lr)
            dt1 = time.perf_counter() - t0
    params = sum(m.rows * m.cols for m in mats)
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"value": params / dt, "unit": "params/s", "cores": int(min(cores, threads or cores)),
            "kind": "oracle",
            "sample": f"{len(mats)} {'router-active ' if wl.moe_routed else ''}matrices ({layers} layer(s)) of "
                      f"{wl.name}, one optimizer step each with the "
                      f"projector set, float64 NumPy ({blas}, {threads} BLAS threads, {cores} host cores); "
                      f"{params / 1e6:.1f}M params in {dt:.2f}s",
            "seconds": dt,
            "one_thread": None if dt1 is None else {"value": params / dt1, "seconds": dt1},
            "extrapolated_full_stack_s": None if layers == len(layer_ids) else dt * len(layer_ids) / layers}


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "the MoARa library runs on exactly one GPU; --gpus must be 1 "
                                   "(sharding over several GPUs is designed but not implemented)"}))
        return 2
    import torch
    import workloads as WL
    from paper_2609_15037_amd import moara as M

    wl = WL.WORKLOADS[a.workload]
    if a.layers:
        wl = WL.subset(wl, list(range(a.layers)))
    operand = a.operand or wl.operand_dtype
    moments = a.moments or wl.moment_dtype
    ob = 2 if operand == "bf16" else 4
    mob = 2 if moments == "bf16" else 4
    wb = 2 if wl.weight_dtype == "bf16" else 4
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    n = len(wl.matrices)
    log(f"[bench] {wl.name}: {n} matrices, {wl.n_params / 1e9:.3f}G params, operand {operand}, moments {moments}")

    # ---- inputs resident in HBM
    wdt = torch.bfloat16 if wl.weight_dtype == "bf16" else torch.float32
    W, G = [], []
    t0 = time.time()
    for i, m in enumerate(wl.matrices):
        W.append(WL.weight_device(wl, i, torch.empty((m.rows, m.cols), dtype=wdt, device=dev)))
        g = torch.empty((m.rows, m.cols), dtype=torch.float32, device=dev)
        WL.grad_device(wl, i, 0, g, active=True)
        G.append(g)
        if i % 32 == 31:
            log(f"[bench] generated {i + 1}/{n} matrices ({time.time() - t0:.0f}s)")
    torch.cuda.synchronize()

    cfg = M.moara_default_config(
        rank_table=list(wl.rank_table), block_size=wl.block_size, beta1=wl.beta1, beta2=wl.beta2,
        adam_eps=wl.adam_eps, scale=wl.scale, refresh_interval=0,
        weight_dtype=M.MOARA_BF16 if wl.weight_dtype == "bf16" else M.MOARA_F32,
        operand_dtype=M.MOARA_BF16 if operand == "bf16" else M.MOARA_F32,
        moment_dtype=M.MOARA_BF16 if moments == "bf16" else M.MOARA_F32,
        refresh_oversample=wl.refresh_oversample,
        refresh_iters=a.refresh_iters if a.refresh_iters else wl.refresh_iters)
    descs = M.make_descs([(m.rows, m.cols, m.module) for m in wl.matrices])
    stream = torch.cuda.current_stream()
    st = M.moara_create_state(cfg, descs, stream=stream)
    state_bytes, _ = M.moara_state_bytes(cfg, descs)
    log(f"[bench] state {state_bytes / 2**30:.1f} GiB")

    # ---- projector refresh (all matrices), timed with events on the library's stream
    M.moara_set_timing(st, True)
    ref_ms = []
    for rep in range(max(1, a.refresh_reps)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        M.moara_refresh_projector(st, G, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ref_ms.append(e0.elapsed_time(e1))
        log(f"[bench] refresh {rep}: {ref_ms[-1]:.1f} ms")
    M.moara_reset_kernel_stats(st, stream=stream)

    if a.copy_calibration_mib:
        nb = a.copy_calibration_mib << 20
        src = torch.ones(nb // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)   # one elementwise kernel: reads nb bytes, writes nb bytes
        torch.cuda.synchronize()
        log(f"[bench] calibration copy: {nb} bytes read, {nb} bytes written")
        del src, dst

    # ---- steps (MoE batches: per layer and step, moe_active of the moe_routed experts are
    # active, drawn by the workload's router; inactive matrices are skipped)
    lr = wl.lr
    moe = wl.moe_routed > 0
    masks = [WL.active_set(wl, k) if moe else None for k in range(a.warmup + a.steps)]
    act_u8 = [M.moara_active_mask(st, m) if m is not None else None for m in masks]
    sargs = M.StepArgs(st, W, G)   # pointer arrays checked once, outside the timed region
    sizes = np.array([m.rows * m.cols for m in wl.matrices], dtype=np.float64)
    params_timed = sum(float(sizes[masks[a.warmup + k]].sum()) if moe else float(wl.n_params) for k in range(a.steps))
    for k in range(a.warmup):
        M.moara_step(st, W, G, lr, active=act_u8[k], stream=stream, args=sargs)
    torch.cuda.synchronize()
    M.moara_reset_kernel_stats(st, stream=stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_host = time.perf_counter()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps - 1)]   # between steps
    e0.record(stream)
    for k in range(a.steps):
        M.moara_step(st, W, G, lr, active=act_u8[a.warmup + k], stream=stream, args=sargs)
        (ev[k] if k < a.steps - 1 else e1).record(stream)
    torch.cuda.synchronize()
    marks = [e0] + ev + [e1]
    step_ms = [marks[k].elapsed_time(marks[k + 1]) for k in range(a.steps)]
    host_s = time.perf_counter() - t_host
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / a.steps
    log(f"[bench] {a.steps} steps: {ms_step:.3f} ms/step (host clock {host_s / a.steps * 1e3:.3f})")

    kern = {}
    names = {M.MOARA_KERN_DECOMPOSE: "decompose", M.MOARA_KERN_PROJECT: "project",
             M.MOARA_KERN_BACKPROJ: "backproject"}
    for kid, name in names.items():
        nl, ms = M.moara_kernel_stats(st, kid, stream=stream)
        kern[name] = {"launches": nl, "ms_total": ms, "ms_per_step": ms / max(1, a.steps),
                      "ms_per_launch": ms / max(1, nl)}
    if moe:   # per-step average over the timed steps' active sets
        cost = {kk: [0.0, 0.0] for kk in ("decompose", "project", "backproject")}
        for k in range(a.steps):
            ck = algorithmic_cost(wl, operand, wb, masks[a.warmup + k], moment_bytes=mob)
            for kk in cost:
                cost[kk][0] += ck[kk][0] / a.steps
                cost[kk][1] += ck[kk][1] / a.steps
    else:
        cost = algorithmic_cost(wl, operand, wb, moment_bytes=mob)
    peak_mfma = PEAK_BF16 if operand == "bf16" else PEAK_F32
    for name, (bytes_, flops) in cost.items():
        t = kern[name]["ms_per_step"] / 1e3
        kern[name]["alg_bytes_per_step"] = bytes_
        kern[name]["alg_flops_per_step"] = flops
        kern[name]["GBps"] = bytes_ / t / 1e9 if t > 0 else None
        kern[name]["TFLOPs"] = flops / t / 1e12 if t > 0 else None
        kern[name]["hbm_frac"] = bytes_ / t / PEAK_HBM if t > 0 else None
        kern[name]["mfma_frac"] = flops / t / peak_mfma if t > 0 and flops else None
    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    dk = kern[dom]
    t_mem = dk["alg_bytes_per_step"] / PEAK_HBM
    t_mfma = dk["alg_flops_per_step"] / peak_mfma
    launches_per_step = max(1, dk["launches"] // max(1, a.steps))
    if t_mfma > t_mem:
        roof = {"bound": "mfma", "achieved": dk["TFLOPs"], "peak": peak_mfma / 1e12, "unit": "TFLOP/s",
                "frac": dk["mfma_frac"]}
    else:
        roof = {"bound": "hbm", "achieved": dk["GBps"], "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": dk["hbm_frac"]}
    roof.update({"kernel": dom, "launches_per_step": launches_per_step,
                 "alg_bytes_per_launch": dk["alg_bytes_per_step"] / launches_per_step,
                 "alg_flops_per_launch": dk["alg_flops_per_step"] / launches_per_step,
                 "avg_launch_ms": dk["ms_total"] / max(1, dk["launches"]),
                 "traffic": measured_traffic(dom, wl.name) if not a.layers else None})

    # alignment diagnostic (Section 3.2) over every matrix: one untimed call, then one timed
    M.moara_alignment(st, G, stream=stream)
    torch.cuda.synchronize()
    ea0, ea1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ea0.record(stream)
    S = M.moara_alignment(st, G, stream=stream)
    ea1.record(stream)
    torch.cuda.synchronize()
    align_ms = ea0.elapsed_time(ea1)
    align_flops = float(sum(4.0 * m.rows * m.cols * wl.rank_of(m) for m in wl.matrices))
    s_tau = {}
    for m, sv in zip(wl.matrices, S):
        s_tau.setdefault(WL.MODULE_NAMES[m.module], []).append(float(sv))
    log(f"[bench] alignment diagnostic: {align_ms:.1f} ms")

    if moe:
        mb = sum(method_cost(wl, ob, wb, masks[a.warmup + k], mob)[0] for k in range(a.steps)) / a.steps
        mf = sum(method_cost(wl, ob, wb, masks[a.warmup + k], mob)[1] for k in range(a.steps)) / a.steps
    else:
        mb, mf = method_cost(wl, ob, wb, moment_bytes=mob)
    step_roof_ms = max(mb / PEAK_HBM, mf / peak_mfma) * 1e3
    q_used = a.refresh_iters if a.refresh_iters else wl.refresh_iters
    rc = refresh_cost(wl, wl.refresh_oversample, q_used, operand == "bf16")
    ref_med = float(np.median(ref_ms))
    out = {
        "metric": "params updated/sec per optimizer step at Llama-2-7B shapes; ms per projector refresh",
        "value": params_timed / (ms_total / 1e3),
        "unit": "params/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": float(np.median(step_ms)),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": operand, "data": "synthetic",
        "config": {"workload": wl.name, "layers": wl.n_layers, "matrices": n, "params": wl.n_params,
                   "rank_table": list(wl.rank_table[:7] if wl.moe_routed == 0 else wl.rank_table),
                   "block_size": wl.block_size, "weights": wl.weight_dtype, "grads": "f32", "moments": moments,
                   "gemm_operands": operand, "refresh": {"oversample": wl.refresh_oversample,
                                                         "iters": q_used}},
        "ms_per_refresh": ref_med,
        "refresh_ms_all": ref_ms,
        "params_per_step": params_timed / a.steps,
        "refresh_roofline": {"ms": rc["roofline_ms"], "frac": rc["roofline_ms"] / ref_med,
                             "p": "r" if wl.refresh_oversample < 0 else wl.refresh_oversample, "q": q_used,
                             "bf16_tflop": rc["bf16_flops"] / 1e12, "f32_tflop": rc["f32_flops"] / 1e12,
                             "f64_tflop": rc["f64_flops"] / 1e12,
                             "peaks_tflops": {"bf16": PEAK_BF16 / 1e12, "f32": PEAK_F32 / 1e12,
                                              "f64": PEAK_F64 / 1e12},
                             "excludes": "Rayleigh-Ritz Jacobi sweeps (iterative)"},
        "amortized_ms_per_step_T200": ms_step + ref_med / 200.0,
        "step_roofline_ms": step_roof_ms,
        "step_roofline_frac": step_roof_ms / ms_step,
        "kernels": kern,
        "roofline": roof,
        "alignment": {"ms": align_ms, "matrices": n, "alg_flops": align_flops,
                      "tflops": align_flops / (align_ms / 1e3) / 1e12,
                      "frac_fp32_peak": align_flops / (align_ms / 1e3) / PEAK_F32,
                      "S_tau": {k: float(np.mean(v)) for k, v in s_tau.items()}},
        "host_clock_ms_per_step": host_s / a.steps * 1e3,
    }
    # the two performance targets stated for the 7B step, with the live figures (not met so far)
    kp, kb, kd = kern.get("project"), kern.get("backproject"), kern.get("decompose")
    if kp and kb and kd:
        out["targets"] = {
            "projection_gemm_mfma_frac_ge_0.60": {"value": kp["mfma_frac"], "met": kp["mfma_frac"] >= 0.60},
            "fused_update_pass_hbm_frac_ge_0.70": {
                "value": kb["hbm_frac"], "met": kb["hbm_frac"] >= 0.70,
                "note": "weight update fused into the back-projection epilogue: algorithmic bytes / time / 8 TB/s"},
            "decompose_pass_hbm_frac": kd["hbm_frac"],
        }
    if not a.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        cb = cpu_baseline(wl, a.cpu_sample_layers, a.cpu_one_thread, moments)
        out["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample", "one_thread",
                                                  "extrapolated_full_stack_s")}
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    del st
    return 0


if __name__ == "__main__":
    sys.exit(main())
