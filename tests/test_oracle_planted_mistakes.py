"""The oracle's pins must catch plausible mistakes: each case below plants one mistake in a
copy of the oracle's source (on the CPU), builds it, and requires the pin suite to fail."""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "bcpnn_oracle.c")

MISTAKES = {
    "trace decay dropped": ("c = (1.0 - lam) * c + lam * (acc[j] * invB);",
                            "c = c + lam * (acc[j] * invB);"),
    "Pj replaced by Pi in the log ratio": ("(clamp_eps(pi, eps) * clamp_eps(pj, eps))",
                                           "(clamp_eps(pi, eps) * clamp_eps(pi, eps))"),
    "argmin ties to the highest index": ("if (a < 0 || v < mi[(int64_t)a * hout + hj]) a = hi;",
                                         "if (a < 0 || v <= mi[(int64_t)a * hout + hj]) a = hi;"),
    "argmax ties to the highest index": ("if (s < 0 || v > mi[(int64_t)s * hout + hj]) s = hi;",
                                         "if (s < 0 || v >= mi[(int64_t)s * hout + hj]) s = hi;"),
    "swap on equal score": ("if (!(mi[(int64_t)s * hout + hj] > mi[(int64_t)a * hout + hj])) break;",
                            "if (!(mi[(int64_t)s * hout + hj] >= mi[(int64_t)a * hout + hj])) break;"),
    "bias left out of the support": ("acc[j] = (double)b[j];", "acc[j] = 0.0;"),
    "softmax gain ignored": ("den += exp(g * ((double)sr[m] - mx));",
                             "den += exp(((double)sr[m] - mx));"),
    "MI stored transposed": ("mi[(int64_t)hi * p->out_hcu + hj] = sum;",
                             "mi[(int64_t)hj * p->in_hcu + hi] = sum;"),
    "Pj trace not divided by B": ("c = (1.0 - lam) * c + lam * (sum * invB);\n        pj[j]",
                                  "c = (1.0 - lam) * c + lam * (sum);\n        pj[j]"),
    "mask read transposed": ("if (mask[hi * p->out_hcu + hj]) v = log_ratio",
                             "if (mask[hj * p->in_hcu + hi]) v = log_ratio"),
    "bias gain ignored": ("b[j] = (float)((double)p->bias_gain * log(clamp_eps(pj[j], eps)));",
                          "b[j] = (float)(log(clamp_eps(pj[j], eps)));"),
    "MI term not weighted by Pij": ("sum += (double)q * log_ratio", "sum += log_ratio"),
    "readout ties to the highest index": ("if (sr[m] > sr[best]) best = m;",
                                          "if (sr[m] >= sr[best]) best = m;"),
    "rounding ties away from even": ("else kept = (fmod(lo, 2.0) == 0.0) ? lo : lo + 1.0;",
                                     "else kept = lo + 1.0;"),
    "activated block not patched": (
        "double v = side ? log_ratio(pij[i * n_out + j], pi[i], pj[j], eps) : 0.0;",
        "double v = 0.0;"),
    "joint trace mixes in a uniform term": ("acc[j] += xi * (double)yr[j];",
                                           "acc[j] += xi * (double)yr[j] * 0.5 + xi * 0.5 / p->out_mcu;"),
}


def _run(name, old, new, tmp):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    base = os.path.join(tmp, "".join(c if c.isalnum() else "_" for c in name))
    with open(base + ".c", "w") as f:
        f.write(src.replace(old, new))
    subprocess.run(["gcc", "-std=c11", "-O1", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    "-I", os.path.join(ROOT, "oracle"), "-o", base + ".so", base + ".c", "-lm"],
                   check=True)
    env = dict(os.environ, BCPNN_ORACLE_LIB=base + ".so", OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True)
    return name, r.returncode


def test_every_planted_mistake_fails_a_pin():
    with tempfile.TemporaryDirectory() as tmp:
        with concurrent.futures.ThreadPoolExecutor(4) as ex:
            res = list(ex.map(lambda kv: _run(kv[0], *kv[1], tmp), MISTAKES.items()))
    missed = [n for n, rc in res if rc == 0]
    assert not missed, f"pins did not catch: {missed}"
