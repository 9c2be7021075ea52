"""The oracle's pins catch plausible mistakes -- CPU only.

Each case plants one mistake (a flipped comparison, a dropped term, a wrong
index, a transposed operand) in a temporary copy of oracle/orc.c, builds it,
and runs the pin tests against that copy in a child process.  The case
passes when at least one pin fails (or the broken copy crashes)."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "orc.c")

MUTANTS = {
    "fire: > instead of >=": ("int s = (p >= thr);", "int s = (p > thr);"),
    "conv: kernel flipped": (
        "s += (double)wt[((f * Cin + ci) * K + ky) * K + kx];",
        "s += (double)wt[((f * Cin + ci) * K + (K - 1 - ky)) * K + (K - 1 - kx)];"),
    "conv: padding dropped": (
        "for (int ky = 0; ky < K; ++ky)\n                                for (int kx = 0; kx < K; ++kx) {\n"
        "                                    int iy = y * stride + ky - pad, ix = x * stride + kx - pad;",
        "for (int ky = 0; ky < K; ++ky)\n                                for (int kx = 0; kx < K; ++kx) {\n"
        "                                    int iy = y * stride + ky, ix = x * stride + kx;"),
    "conv: stride ignored": ("int iy = y * stride + ky - pad, ix = x * stride + kx - pad;\n"
                             "                                    if (iy < 0",
                             "int iy = y + ky - pad, ix = x + kx - pad;\n"
                             "                                    if (iy < 0"),
    "conv: stride on one axis only": ("int iy = y * stride + ky - pad, ix = x * stride + kx - pad;",
                                      "int iy = y * stride + ky - pad, ix = x + kx - pad;"),
    "conv: output size rounded up": ("return (n + 2 * pad - K) / stride + 1;",
                                     "return (n + 2 * pad - K + stride - 1) / stride + 1;"),
    "stdp: stride ignored": ("int iy = y * stride + ky - pad, ix = x * stride + kx - pad;\n"
                             "                        int pre = 0;",
                             "int iy = y + ky - pad, ix = x + kx - pad;\n"
                             "                        int pre = 0;"),
    "conv_times: prefix off by one step": (
        "run += hist[t];\n                        pot[", "pot["),
    "wave: strict > in Eq.1": ("(uint8_t)(t >= t_first[b * N + i])", "(uint8_t)(t > t_first[b * N + i])"),
    "rank: ceil bins": ("(uint8_t)((rho * (int64_t)T) / n)", "(uint8_t)((rho * (int64_t)T + n - 1) / n)"),
    "rank: ties by descending index": (
        "return (x->idx < y->idx) ? -1 : (x->idx > y->idx);",
        "return (x->idx > y->idx) ? -1 : (x->idx < y->idx);"),
    "rank: zero intensities spike": ("if (I[i] > 0.0f) {", "if (I[i] >= 0.0f) {"),
    "filter: kernel flipped": (
        "s += (double)filt[(c * KF + ky) * KF + kx] *",
        "s += (double)filt[(c * KF + (KF - 1 - ky)) * KF + (KF - 1 - kx)] *"),
    "pool: stride taken from window": ("int iy = yo * R + dy - D, ix = xo * R + dx - D;",
                                       "int iy = yo * P + dy - D, ix = xo * P + dx - D;"),
    "pool: last value instead of max": ("if (v > m) m = v;", "m = v;"),
    "kwta: ties to the higher index": ("(tf[i] == tf[best] && vf[i] > vf[best])",
                                       "(tf[i] == tf[best] && vf[i] >= vf[best])"),
    "kwta: smaller potential wins": ("(tf[i] == tf[best] && vf[i] > vf[best])",
                                     "(tf[i] == tf[best] && vf[i] < vf[best])"),
    "kwta: no feature-wise inhibition": (
        "for (int64_t i = (int64_t)f * H * W; i < (int64_t)(f + 1) * H * W; ++i) inh[i] = 1;", ""),
    "kwta: lateral window one short": ("for (int yy = y - r; yy <= y + r; ++yy)",
                                       "for (int yy = y - r; yy < y + r; ++yy)"),
    "stdp: rates swapped": ("(pre ? (double)a_plus : (double)a_minus)", "(pre ? (double)a_minus : (double)a_plus)"),
    "stdp: stabilizer term dropped": ("((w - (double)lb) * ((double)ub - w))", "(w - (double)lb)"),
    "stdp: pre time read at the last step": ("pre_wave + (b * T + ti) *", "pre_wave + (b * T + T - 1) *"),
    "stdp: punish not negated": ("sgn = (reward[b] > 0) ? 1.0 : -1.0;", "sgn = 1.0;"),
    "decide: wrong class map": ("int d = winners[b * 4 * k] % n_classes;", "int d = winners[b * 4 * k + 1] % n_classes;"),
    "events: silent taps counted": ("c += tin[((b * Cin + ci) * (int64_t)H + iy) * W + ix] < T;",
                                    "c += tin[((b * Cin + ci) * (int64_t)H + iy) * W + ix] <= T;"),
}


def _run_mutant(name, old, new, tmp):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {name}"
    mut = src.replace(old, new, 1)
    path = os.path.join(tmp, f"m{abs(hash(name))}")
    os.makedirs(path, exist_ok=True)
    c, so = os.path.join(path, "orc.c"), os.path.join(path, "liborc.so")
    open(c, "w").write(mut)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-fvisibility=hidden", "-o", so, c, "-lm"], check=True)
    env = dict(os.environ, ORC_LIB=so)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_toys.py"),
                        os.path.join(ROOT, "tests", "test_oracle_props.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode


def test_every_planted_mistake_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max_workers=6) as ex:
            res = list(ex.map(lambda kv: _run_mutant(kv[0], kv[1][0], kv[1][1], tmp), MUTANTS.items()))
    survivors = [n for n, rc in res if rc == 0]
    assert not survivors, f"mistakes not caught by any pin: {survivors}"
