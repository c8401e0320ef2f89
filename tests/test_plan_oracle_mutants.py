"""The planner oracle's pins catch plausible mistakes (mutation test, CPU).

Each mutant plants one plausible mistake in a copy of
``oracle/plan_oracle.py`` (a wrong synchronisation form, the global batch
for the per-node one, a dropped unit or factor in the time and cost of
Eq. (4), a wrong rounding of the memory bound of Eq. (3), a wrong flip,
normalisation, threshold or return value in Kneedle, a wrong selection key)
and runs the planner oracle's pins (``test_plan_oracle_pins.py``) with the
mutated module standing in for ``oracle.plan_oracle``.  Every mutant must
make at least one pin fail.  The repository's module is never modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "plan_oracle.py")

MUTANTS = [
    # Eq. (2c): synchronisation term
    ("parameter server N - 1", "        return float(nodes)\n", "        return float(nodes - 1)\n"),
    ("ring 1/N", "return 1.0 - 1.0 / nodes", "return 1.0 / nodes"),
    ("ring 2(1 - 1/N)", "return 1.0 - 1.0 / nodes", "return 2.0 * (1.0 - 1.0 / nodes)"),
    # Eq. (2a): compute term on the per-node batch
    ("compute term on a wrong batch", "row.append(float(local_batch))",
     "row.append(float(local_batch) * float(nodes))"),
    ("step time with N for s(N)", "model[\"c_sync\"] * sync_term(nodes, sync)", "model[\"c_sync\"] * nodes"),
    ("rms residual as mean |r|", "math.sqrt(np.mean(r * r))", "np.mean(np.abs(r))"),
    # Eq. (4a), (4b)
    ("per-node batch = global batch", "t = step_time(model, nodes, global_batch / nodes, sync)",
     "t = step_time(model, nodes, global_batch, sync)"),
    ("steps per epoch from the per-node batch", "T = epochs * dataset_size / global_batch * t",
     "T = epochs * dataset_size / (global_batch / nodes) * t"),
    ("cost without N", "C = T / 3600.0 * nodes * price_per_node_hour", "C = T / 3600.0 * price_per_node_hour"),
    ("cost without the hour unit", "C = T / 3600.0 * nodes * price_per_node_hour",
     "C = T * nodes * price_per_node_hour"),
    # Eq. (3)
    ("memory bound rounded up", "math.floor((capacity - m_static) / m_per_sample)",
     "math.ceil((capacity - m_static) / m_per_sample)"),
    ("memory bound without the static part", "math.floor((capacity - m_static) / m_per_sample)",
     "math.floor(capacity / m_per_sample)"),
    # Kneedle
    ("x flipped for the wrong shapes", "flip_x = shape in (\"concave_dec\", \"convex_inc\")",
     "flip_x = shape in (\"convex_dec\", \"convex_inc\")"),
    ("y flipped for the wrong shapes", "flip_y = shape in (\"convex_dec\", \"convex_inc\")",
     "flip_y = shape in (\"concave_dec\", \"convex_inc\")"),
    ("y not normalised by its range", "yn = (y - y.min()) / (y.max() - y.min())", "yn = y / y.max()"),
    ("threshold spacing over n", "step = sensitivity * (xs[-1] - xs[0]) / (n - 1)",
     "step = sensitivity * (xs[-1] - xs[0]) / n"),
    ("threshold without the sensitivity", "step = sensitivity * (xs[-1] - xs[0]) / (n - 1)",
     "step = (xs[-1] - xs[0]) / (n - 1)"),
    ("knee at the point that falls below", "            return order[lmx]", "            return order[j]"),
    ("local maximum strict on both sides", "if j < n - 1 and d[j - 1] < d[j] >= d[j + 1]:",
     "if j < n - 1 and d[j - 1] < d[j] > d[j + 1]:"),
    ("threshold reached counts as a fall", "if threshold is not None and d[j] < threshold:",
     "if threshold is not None and d[j] <= threshold:"),
    ("memory bound not clamped at 0", "return max(0, math.floor((capacity - m_static) / m_per_sample))",
     "return math.floor((capacity - m_static) / m_per_sample)"),
    ("rms residual without the root", "out[\"rms_residual\"] = float(math.sqrt(np.mean(r * r)))",
     "out[\"rms_residual\"] = float(np.mean(r * r))"),
    ("threshold above the maximum", "threshold = d[j] - step", "threshold = d[j] + step"),
    # selection
    ("cost tie to the last candidate", "return min(idx, key=lambda i: (Cs[i], i)), Ts, Cs",
     "return min(idx, key=lambda i: (Cs[i], -i)), Ts, Cs"),
    ("infeasible candidates keep their time", "        Ts.append(T if ok else math.inf)", "        Ts.append(T)"),
    ("time objective ranks by cost", "return min(idx, key=lambda i: (Ts[i], i)), Ts, Cs",
     "return min(idx, key=lambda i: (Cs[i], i)), Ts, Cs"),
    ("feasibility on the global batch", "ok = B / n <= max_local", "ok = B <= max_local"),
    # Not listed: a knee sought on a flat curve (the NaN difference curve has
    # no local maximum either: None both ways); the knee's index into the
    # feasible candidates used without mapping it back (with one cluster
    # size and increasing B the infeasible ones form a suffix, so the two
    # indices agree).
    # Not listed: the knee taken on the cost curve instead of the time curve.
    # The knee objective works on one cluster size, where C = T N p / 3600
    # is a constant multiple of T, so Kneedle (which normalises y) finds the
    # same knee: the mutant is equivalent, not a mistake a pin could see.
]

_RUNNER = r"""
import importlib.util, sys
root, path = sys.argv[1], sys.argv[2]
sys.path.insert(0, root)
import oracle
spec = importlib.util.spec_from_file_location("oracle.plan_oracle", path)
mod = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mod)
sys.modules["oracle.plan_oracle"] = mod
oracle.plan_oracle = mod
import pytest
sys.exit(pytest.main(["-x", "-q", "-p", "no:cacheprovider",
                      root + "/tests/test_plan_oracle_pins.py"]))
"""


def _pins_fail(path):
    r = subprocess.run([sys.executable, "-c", _RUNNER, ROOT, path], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    return r.returncode != 0, r.stdout[-2000:]


def test_mutant_list_applies_to_the_planner_oracle():
    src = open(SRC).read()
    names = [m[0] for m in MUTANTS]
    assert len(set(names)) == len(names)
    for name, old, _ in MUTANTS:
        assert src.count(old) == 1, f"mutant '{name}': its text occurs {src.count(old)} times"


def test_unmutated_planner_oracle_passes_the_pins(tmp_path):
    path = os.path.join(str(tmp_path), "plan_oracle_copy.py")
    with open(path, "w") as f:
        f.write(open(SRC).read())
    failed, out = _pins_fail(path)
    assert not failed, out


def test_every_planner_mutant_fails_a_pin(tmp_path):
    src = open(SRC).read()

    def one(i):
        name, old, new = MUTANTS[i]
        path = os.path.join(str(tmp_path), f"plan_mutant{i}.py")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        return name, _pins_fail(path)[0]

    workers = max(1, min(4, (os.cpu_count() or 2) // 2))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(one, range(len(MUTANTS))))
    survivors = [name for name, failed in results if not failed]
    assert not survivors, f"mutants no pin catches: {survivors}"
