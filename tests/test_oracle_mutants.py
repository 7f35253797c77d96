"""The oracle's pins catch plausible slips: each case below plants one mistake in a copy
of the oracle's source (on the CPU, in a child process) and requires that the pins in
test_oracle_pins.py then fail. A mistake that no pin notices fails this test.

Each substitution must match the oracle's source exactly once, so a change of the
oracle that removes the line a case plants its mistake in fails here too, and the case
is then rewritten for the new source.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle", "moara_oracle.py")

# (what goes wrong, exact text in the oracle, the mistaken text)
MUTANTS = [
    # Appendix D: the bf16 update cast and the bf16 operands of the GEMMs
    ("bf16 weights: inner cast of the update dropped",
     "return round_bf16(W - lr * round_bf16(U))", "return round_bf16(W - lr * U)"),
    ("bf16 operands: N not rounded", "    No = _operand(N, cfg)", "    No = N"),
    ("bf16 operands: V not rounded", "    Vo = _operand(V, cfg)", "    Vo = V"),
    ("bf16 operands: P not rounded", "    P = _operand(st.P, cfg)", "    P = st.P"),
    ("bf16 direction moments stored exactly",
     'store=round_bf16 if cfg.moment_dtype == "bf16" else None)', "store=None)"),
    # Algorithm 1: recomposition and scale
    ("magnitude branch dropped from the update",
     "U = rep_b(dM, B, st.n) * dV", "U = dV"),
    ("GaLore scale not applied", "U = cfg.scale * U", "U = U"),
    ("Rep_B tiles instead of repeating", "return np.repeat(M, B, axis=1)[:, :n]",
     "return np.tile(M, (1, B))[:, :n]"),
    ("decompose divides by the squared norm", "Vp = blocks / (M[:, :, None] + eps)",
     "Vp = blocks / (M[:, :, None] + eps) ** 2"),
    ("step count never advanced", "    st.t += 1\n    N, st.exp_avg",
     "    N, st.exp_avg"),
    ("left projection transposed", "Rt = P.T @ Vo if st.side == LEFT else Vo @ P",
     "Rt = P.T @ Vo if st.side != LEFT else Vo @ P"),
    ("scheduled refresh skipped",
     "        refresh(st, V, cfg)\n", "        pass\n"),
    # Adam (Appendix D hyper-parameters)
    ("second bias correction one step late", "c2 = 1.0 - beta2 ** t", "c2 = 1.0 - beta2 ** (t + 1)"),
    ("second moment mixes with beta1", "q = beta2 * exp_avg_sq + (1.0 - beta2) * x * x",
     "q = beta2 * exp_avg_sq + (1.0 - beta1) * x * x"),
    ("bias correction outside the square root", "out = (e / c1) / (np.sqrt(q / c2) + eps)",
     "out = (e / c1) / (np.sqrt(q) / c2 + eps)"),
    # projector side and SVD
    ("square matrices projected on the right", "return LEFT if m <= n else RIGHT",
     "return LEFT if m < n else RIGHT"),
    ("right side takes left singular vectors", "P = U[:, :r] if side == LEFT else Yt[:r, :].T",
     "P = U[:, :r] if side == LEFT else Yt[-r:, :].T"),
    ("canonical signs flipped", "sgn[sgn == 0] = 1.0", "sgn[sgn == 0] = 1.0; sgn = -sgn"),
    # Appendix G memory model and Phase 3 ranks
    ("magnitude state counts whole blocks only", "tot += 2 * b_M * m * math.ceil(n / B)",
     "tot += 2 * b_M * m * (n // B)"),
    ("receivers gain delta_r each", "out[t] = r_base + gain", "out[t] = r_base + delta_r"),
    # bf16 rounding
    ("bf16 subnormal range one binade too low", "e = np.maximum(e - 1, -126)",
     "e = np.maximum(e - 1, -127)"),
    ("bf16 keeps nine significant bits", "ulp = np.ldexp(1.0, e - 7)", "ulp = np.ldexp(1.0, e - 8)"),
    ("bf16 ties rounded up", "r = np.rint(xf / ulp) * ulp", "r = np.floor(xf / ulp + 0.5) * ulp"),
    ("bf16 rounding skips negative values", "fin = np.isfinite(x) & (x != 0)",
     "fin = np.isfinite(x) & (x > 0)"),
    # alignment diagnostic (Section 3.2)
    ("right-side reconstruction projects the wrong side",
     "PV = P @ (P.T @ V) if side == LEFT else (V @ P) @ P.T",
     "PV = P @ (P.T @ V) if side == LEFT else V @ (P @ P.T).T[::-1]"),
    ("decomposition-off reconstruction ignores the side",
     "return recompose(M, PV, B) if decompose_on else PV",
     "return recompose(M, PV, B) if decompose_on else P @ (P.T @ V)"),
    ("cosine of absolute values", "return float(np.sum(G * R)) / den if den > 0.0 else 0.0",
     "return float(np.sum(np.abs(G * R))) / den if den > 0.0 else 0.0"),
    ("per-type median instead of mean", "return {tau: float(np.mean(v)) for tau, v in acc.items()}",
     "return {tau: float(np.median(v)) for tau, v in acc.items()}"),
    ("flattening keeps the last axis", "return G.reshape(G.shape[0], -1)", "return G.reshape(-1, G.shape[-1])"),
    ("comparison floor from the tested value", "rms = math.sqrt(float(np.mean(b * b)))",
     "rms = math.sqrt(float(np.mean(a * a)))"),
]

# Child process: load the planted copy as oracle.moara_oracle, then run the pins.
_CHILD = r"""
import sys, types
root, old, new = sys.argv[1], sys.argv[2], sys.argv[3]
sys.path.insert(0, root)
src = open(root + "/oracle/moara_oracle.py").read()
assert src.count(old) == 1, "the planted text must occur exactly once"
import oracle
mod = types.ModuleType("oracle.moara_oracle")
mod.__file__ = "planted_oracle.py"
sys.modules["oracle.moara_oracle"] = mod
oracle.moara_oracle = mod
exec(compile(src.replace(old, new), "planted_oracle.py", "exec"), mod.__dict__)
import pytest
sys.exit(pytest.main(["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", root + "/tests/test_oracle_pins.py"]))
"""


def _run_pins_on(old, new):
    env = dict(os.environ, OMP_NUM_THREADS="1")   # the pins are tiny: one thread per child
    res = subprocess.run([sys.executable, "-c", _CHILD, ROOT, old, new], cwd=ROOT, env=env,
                         capture_output=True, text=True, timeout=300)
    return res.returncode, (res.stdout + res.stderr)[-800:]


@pytest.fixture(scope="module")
def pin_runs():
    """Every planted copy's pin run, six child processes at a time."""
    with ThreadPoolExecutor(max_workers=6) as ex:
        runs = list(ex.map(lambda m: _run_pins_on(m[1], m[2]), MUTANTS))
    return {m[0]: r for m, r in zip(MUTANTS, runs)}


def test_every_planted_text_occurs_once():
    src = open(ORACLE).read()
    for name, old, new in MUTANTS:
        assert src.count(old) == 1, name
        assert old != new, name


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_pins_fail_on_planted_mistake(name, pin_runs):
    code, tail = pin_runs[name]
    assert "the planted text must occur exactly once" not in tail, name
    # pytest exits with 1 when tests ran and some failed; 0 means no pin noticed the mistake
    assert code == 1, f"{name}: pins exit code {code}\n{tail}"
