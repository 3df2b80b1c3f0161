"""The oracle's pins catch plausible slips in the oracle (CPU only).

Each case copies the oracle, the workload generator and the oracle pin tests
into a scratch directory, plants one slip in the copy of the oracle (a sign, a
tie direction, a dropped term, a transposed index, a wrong divisor, ...),
rebuilds it there and runs the pin tests against it in a subprocess.  A slip
that every pin lets through fails this test.  The repository's own oracle is
never modified.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PIN_FILES = ["test_oracle_routing.py", "test_oracle_layout.py", "test_oracle_moe.py",
             "test_oracle_adjustment.py"]

# (file under oracle/, text, replacement, what the slip is)
MUTANTS = [
    ("cap_oracle.c", "q = fmaf(q, r, (float)(1.0 / 24.0));", "q = fmaf(q, r, (float)(1.0 / 12.0));",
     "exp: wrong Taylor coefficient"),
    ("cap_oracle.c", "if (!(z >= ORC_EXP_MIN))", "if (!(z >= -80.0f))", "exp: cutoff too high"),
    ("cap_oracle.c", "L[e] > L[best])", "L[e] >= L[best])", "top-k: ties to the higher index"),
    ("cap_oracle.c", "q[s] = orc_exp(L[id[s]] - m);", "q[s] = orc_exp(L[id[s]] - L[id[k - 1]]);",
     "gates: shifted by the wrong logit"),
    ("cap_oracle.c", "if (cum >= target) break;", "if (cum > target) break;", "CAP greedy: > instead of >="),
    ("cap_oracle.c", "(key[j] == key[b] && dev[j] < dev[b])", "(key[j] == key[b] && dev[j] > dev[b])",
     "CAP greedy: ratio ties to the higher device"),
    ("cap_oracle.c", "key[j] = a[j] / 1.0f;", "key[j] = a[j] / c;", "CAP greedy: same-node device costs c"),
    ("cap_oracle.c", "key[j] = INFINITY;", "key[j] = a[j];", "CAP greedy: own device not free"),
    ("cap_oracle.c", "if (kp) S = S + ws[s];", "S = S + ws[s];", "CAP: renormalised by all slots"),
    ("cap_oracle.c", "if (kp) { S = S + ws[s]; m |= (uint64_t)1 << expert_rank[id[s]]; }",
     "S = S + ws[s]; if (kp) { m |= (uint64_t)1 << expert_rank[id[s]]; }",
     "naive pruning: renormalised by the full sum"),
    ("cap_oracle.c", "if (kp) { S = S + ws[s]; m |= (uint64_t)1 << expert_rank[id[s]]; }",
     "if (kp) { S = S + ws[s]; } m |= (uint64_t)1 << expert_rank[id[s]];",
     "naive pruning: mask from every slot"),
    ("cap_oracle.c", "if (cum >= target) { n = s + 1; break; }", "if (cum > target) { n = s + 1; break; }",
     "naive pruning: > instead of >="),
    ("cap_oracle.c", "for (int s = 0; s < R; ++s) acc += send_counts[s * R + d];",
     "for (int s = 0; s < R; ++s) acc += send_counts[d * R + s];", "layout: receive offsets transposed"),
    ("cap_oracle.c", "else if (d != src) ++n_intra;", "else ++n_intra;", "volume: own device counted as sent"),
    ("cap_oracle.c", "(size_t)(send_offsets[src * R + d] + j) * row_bytes",
     "(size_t)(send_offsets[d * R + src] + j) * row_bytes", "send pack: offsets transposed"),
    ("cap_oracle.c", "h[j] = g / (1.0 + exp(-g)) * u;", "h[j] = u / (1.0 + exp(-u)) * g;", "FFN: W1 and W3 swapped"),
    ("cap_oracle.c", "acc[c] += (double)wp[q] * (double)yr[c];", "acc[c] += (double)yr[c];",
     "combine: gate weight dropped"),
    ("cap_oracle.c", "acc[c] = shared ? (double)shared[(size_t)i * d + c] : 0.0;", "acc[c] = 0.0;",
     "combine: shared experts dropped"),
    ("cap_oracle.c", "if (keep[q2]) C[(size_t)i * E + idx[q2]] += 1;",
     "if (keep[q2] && s2 != s) C[(size_t)i * E + idx[q2]] += 1;", "co-activation: diagonal missing"),
    ("cap_oracle.c", "if (!keep[q]) continue;\n            int i = idx[q];", "int i = idx[q];",
     "co-activation: counted on unpruned routing"),
    ("placement.py", "delta < best[2]", "delta <= best[2]", "adjustment: ties to the later candidate"),
    ("placement.py", "N[e] > N[f] and", "N[e] >= N[f] and", "adjustment: equal loads swapped"),
    ("placement.py", "delta += P[f][j] * -a", "delta += P[f][j] * a", "adjustment: sign of the f terms"),
    ("placement.py", "if j == e or j == f:", "if j == e:", "adjustment: pair (e, f) counted as moved"),
    ("placement.py", "er[e], er[f] = lo, hi", "er[e], er[f] = hi, lo", "adjustment: swap not applied"),
    ("placement.py", "el[e], el[f] = expert_local[f], expert_local[e]",
     "el[e], el[f] = expert_local[e], expert_local[f]", "adjustment: local slots not exchanged"),
]


def _run_mutant(case):
    fname, old, new, _ = case
    with tempfile.TemporaryDirectory(prefix="orc_mut_") as tmp:
        shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"),
                        ignore=shutil.ignore_patterns("*.so", "*.so.tmp*", "__pycache__"))
        shutil.copytree(os.path.join(ROOT, "workloads"), os.path.join(tmp, "workloads"),
                        ignore=shutil.ignore_patterns("__pycache__"))
        os.makedirs(os.path.join(tmp, "tests"))
        for f in ["conftest.py", "cases.py", *PIN_FILES]:
            shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(tmp, "tests", f))
        shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tmp, "tests", "golden"))
        path = os.path.join(tmp, "oracle", fname)
        src = open(path).read()
        if src.count(old) != 1:
            return "not applied"
        open(path, "w").write(src.replace(old, new))
        env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1", OMP_NUM_THREADS="2")
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            *[os.path.join("tests", f) for f in PIN_FILES]],
                           cwd=tmp, env=env, capture_output=True, text=True, timeout=600)
        return "killed" if r.returncode != 0 else "survived"


def test_every_planted_slip_fails_a_pin():
    workers = max(1, min(4, (os.cpu_count() or 1) // 2))
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:
        results = list(ex.map(_run_mutant, MUTANTS))
    bad = [(m[3], res) for m, res in zip(MUTANTS, results) if res != "killed"]
    assert not bad, f"slips not caught by the oracle pins: {bad}"


@pytest.mark.parametrize("case", MUTANTS[:1], ids=lambda m: m[3])
def test_unmutated_copy_passes(case):
    """The scratch copy without a slip passes every pin (so a kill above is
    the slip's doing, not the copy's)."""
    fname, old, _, what = case
    assert _run_mutant((fname, old, old, what)) == "survived"
