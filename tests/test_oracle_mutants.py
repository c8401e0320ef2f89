"""The oracle's pins catch plausible mistakes (mutation test, CPU only).

Each mutant below plants one plausible mistake in a copy of the float64
oracle's C source (a dropped term, a wrong sign, index or normalisation, a
transposed operand, an off-by-one step, a wrong rule for a special case),
builds it with gcc, and runs the oracle's pins (``test_oracle_pins.py``)
against that build through ``AGS_ORACLE_LIB``.  Every mutant must make at
least one pin fail; a surviving mutant would mean the pins cannot tell that
mistake from the paper's method.  The mutants never touch the repository's
oracle or the GPU library.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ags_oracle.c")

# (name, text to replace, replacement); the text must occur exactly once.
MUTANTS = [
    # step 1: replica mean (Eq. (1c))
    ("mean over K-1", "gbar[j] = s / K;", "gbar[j] = s / (K - 1 > 0 ? K - 1 : 1);"),
    ("mean drops replica 0", "for (int k = 0; k < K; ++k) s += grad_at(c, grads, k, o + j);",
     "for (int k = 1; k < K; ++k) s += grad_at(c, grads, k, o + j);"),
    ("bf16 widened with a wrong shift", "((const uint16_t *)grads)[idx] << 16",
     "((const uint16_t *)grads)[idx] << 15"),
    # step 2: per-layer statistics
    ("W without the square", "W += w[o + j] * w[o + j];", "W += fabs(w[o + j]);"),
    ("G of the first replica", "G += gbar[j] * gbar[j];",
     "G += grad_at(c, grads, 0, o + j) * grad_at(c, grads, 0, o + j);"),
    ("spread with a wrong sign", "double d = grad_at(c, grads, k, o + j) - gbar[j];",
     "double d = grad_at(c, grads, k, o + j) + gbar[j];"),
    ("spread normalised by K-1", "V /= K;", "V /= (K > 1 ? K - 1 : 1);"),
    ("spread not normalised", "V /= K;", ";"),
    ("small batch always replica 0", "double g = grad_at(c, grads, c->small_replica, o + j);",
     "double g = grad_at(c, grads, 0, o + j);"),
    ("RMS small batch not averaged", "            S /= K;\n", "\n"),
    ("noise ratio transposed", "if (G > 0.0) rho = V / G;", "if (V > 0.0) rho = G / V;"),
    ("noise ratio 0/0 infinite", "else rho = (V > 0.0) ? INFINITY : 0.0;", "else rho = INFINITY;"),
    ("noise ratio V/0 zero", "else rho = (V > 0.0) ? INFINITY : 0.0;", "else rho = 0.0;"),
    # step 3: gradient variability (Eq. (5)) and the branch
    ("global norm over scaled layers only", "for (int l = 0; l < L; ++l) G += G_l[l];",
     "for (int l = 0; l < L; ++l) if (layers[l].flags & ORACLE_SCALE) G += G_l[l];"),
    ("Delta divided by the new norm", "delta = fabs((G - Gp) / Gp);", "delta = fabs((G - Gp) / G);"),
    ("Delta without the absolute value", "delta = fabs((G - Gp) / Gp);", "delta = (G - Gp) / Gp;"),
    ("global Delta finite at step 1", "if (t == 1 || !(Gp > 0.0) || !isfinite(Gp) || !isfinite(G))",
     "if (!(Gp > 0.0) || !isfinite(Gp) || !isfinite(G))"),
    ("tie counted as not sensitive", "const int sensitive = !(delta < c->delta);",
     "const int sensitive = !(delta <= c->delta);"),
    ("branch inverted", "const int sensitive = !(delta < c->delta);",
     "const int sensitive = (delta < c->delta);"),
    ("G_prev never updated", "*g_prev = G;", "*g_prev = Gp;"),
    ("layer Delta divided by the new norm", "dl = fabs((G_l[l] - Gpl) / Gpl);",
     "dl = fabs((G_l[l] - Gpl) / G_l[l]);"),
    ("layer and global scope swapped", "out[OUT_SENS] = c->delta_scope ? !(dl < c->delta) : sensitive;",
     "out[OUT_SENS] = c->delta_scope ? sensitive : !(dl < c->delta);"),
    ("layer G_prev never updated", "for (int l = 0; l < L; ++l) g_prev_layers[l] = G_l[l];", ";"),
    # step 3b: per-layer variability
    ("layer Delta finite at step 1", "if (t == 1 || !(Gpl > 0.0) || !isfinite(Gpl) || !isfinite(G_l[l]))",
     "if (!(Gpl > 0.0) || !isfinite(Gpl) || !isfinite(G_l[l]))"),
    ("layer Delta of a non-finite norm not infinite",
     "if (t == 1 || !(Gpl > 0.0) || !isfinite(Gpl) || !isfinite(G_l[l]))",
     "if (t == 1 || !(Gpl > 0.0) || !isfinite(Gpl))"),
    # step 4: coefficients
    ("AGS scale inverted", "a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;",
     "a = (scaled && !out[OUT_SENS]) ? 1.0 / gradscale[l] : 1.0;"),
    ("AGS scales sensitive steps", "a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;",
     "a = (scaled && out[OUT_SENS]) ? gradscale[l] : 1.0;"),
    ("AGS ignores the layer flag", "a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;",
     "a = (!out[OUT_SENS]) ? gradscale[l] : 1.0;"),
    ("AGS drops weight decay", "            a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;\n            b = lam;",
     "            a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;\n            b = 0.0;"),
    ("static scale on sensitive steps", "a = (scaled && !out[OUT_SENS]) ? c->static_scale : 1.0;",
     "a = scaled ? c->static_scale : 1.0;"),
    ("static decay scaled",
     "            a = (scaled && !out[OUT_SENS]) ? c->static_scale : 1.0;\n            b = lam;",
     "            a = (scaled && !out[OUT_SENS]) ? c->static_scale : 1.0;\n            b = a * lam;"),
    ("static scale inverted", "a = (scaled && !out[OUT_SENS]) ? c->static_scale : 1.0;",
     "a = (scaled && !out[OUT_SENS]) ? 1.0 / c->static_scale : 1.0;"),
    ("LARS without the decay term", "c->trust_coef * wn / (gn + lam * wn)", "c->trust_coef * wn / gn"),
    ("LARS ratio transposed", "c->trust_coef * wn / (gn + lam * wn)", "c->trust_coef * gn / (wn + lam * gn)"),
    ("LARS decay not scaled", "            b = a * lam;", "            b = lam;"),
    ("LARS zero-norm fallback 0", "? c->trust_coef * wn / (gn + lam * wn) : 1.0;",
     "? c->trust_coef * wn / (gn + lam * wn) : 0.0;"),
    ("LARS scales unscaled layers", "            if (scaled) {\n                const double wn",
     "            if (1) {\n                const double wn"),
    ("SGD without decay", "double a = 1.0, b = lam;", "double a = 1.0, b = 0.0;"),
    # step 5: wrapped momentum SGD (Eq. (7b), PyTorch semantics)
    ("momentum with dampening", "m[o + j] = c->momentum * m[o + j] + d;",
     "m[o + j] = c->momentum * m[o + j] + (1.0 - c->momentum) * d;"),
    ("weights step on d, not m", "w[o + j] = w[o + j] - c->lr * m[o + j];",
     "w[o + j] = w[o + j] - c->lr * d;"),
    ("decay scaled by the AGS coefficient", "const double d = a * gbar_keep[l][j] + b_l[l] * w[o + j];",
     "const double d = a * (gbar_keep[l][j] + b_l[l] * w[o + j]);"),
    # step 6: UpdateGradScale (Algorithm 1)
    ("refresh ratio transposed", "s = sqrt(S) / (sqrt(Gl) + c->eps);", "s = sqrt(Gl) / (sqrt(S) + c->eps);"),
    ("refresh ratio of squares", "s = sqrt(S) / (sqrt(Gl) + c->eps);", "s = S / (Gl + c->eps);"),
    ("refresh ratio without epsilon", "s = sqrt(S) / (sqrt(Gl) + c->eps);", "s = sqrt(S / Gl);"),
    ("refresh not clipped", "                if (s > smax) s = smax;\n            } else {",
     "            } else {"),
    ("s_max = K", "sqrt((double)K);", "(double)K;"),
    ("zero-norm fallback 0", "            } else {\n                s = 1.0;\n            }",
     "            } else {\n                s = 0.0;\n            }"),
    ("refresh one step late", "(t % c->refresh_every) == 0;", "((t + 1) % c->refresh_every) == 0;"),
    ("refresh of unscaled layers", "if (refresh && (layers[l].flags & ORACLE_SCALE)) {\n            const double S",
     "if (refresh) {\n            const double S"),
    # elementwise AGS (Algorithm 1 read per element)
    ("element ratio transposed", "double s = fabs(gs / (gbar_keep[l][j] + c->eps));",
     "double s = fabs(gbar_keep[l][j] / (gs + c->eps));"),
    ("element RMS without the root", "gs = sqrt(q / K);", "gs = q / K;"),
    ("element RMS over K - 1", "gs = sqrt(q / K);", "gs = sqrt(q / (K > 1 ? K - 1 : 1));"),
    ("element small batch always replica 0", "gs = grad_at(c, grads, c->small_replica, o + j);",
     "gs = grad_at(c, grads, 0, o + j);"),
    ("element eps outside the ratio", "double s = fabs(gs / (gbar_keep[l][j] + c->eps));",
     "double s = fabs(gs / gbar_keep[l][j]) + c->eps;"),
    ("element mean coefficient ignores the decision",
     "sum += (scaled && !sens_l) ? gradscale[o + j] : 1.0;", "sum += scaled ? gradscale[o + j] : 1.0;"),
    ("element scale mean not divided", "            out[OUT_GRADSCALE] = sum / (double)n;\n            continue;",
     "            out[OUT_GRADSCALE] = sum;\n            continue;"),
    ("element 0/0 gives 0", "if (isnan(s)) s = 1.0;", "if (isnan(s)) s = 0.0;"),
    ("element scale ignores the layer flag",
     "const double a = ew ? ((scaled && !sens_l) ? gradscale[o + j] : 1.0) : a_l[l];",
     "const double a = ew ? (!sens_l ? gradscale[o + j] : 1.0) : a_l[l];"),
    ("element scales not clipped", "                    if (s > smax) s = smax;\n", "\n"),
    # bookkeeping
    ("refresh in stats-only calls", "const int refresh = commit && c->mode == ORACLE_AGS && c->refresh_every > 0 &&",
     "const int refresh = c->mode == ORACLE_AGS && c->refresh_every > 0 &&"),
    ("refresh in static and LARS modes",
     "const int refresh = commit && c->mode == ORACLE_AGS && c->refresh_every > 0 &&",
     "const int refresh = commit && c->mode != ORACLE_SGD && c->refresh_every > 0 &&"),
    ("G_prev reported on a first step", "out_global[GOUT_GPREV] = (t == 1) ? 0.0 : Gp;",
     "out_global[GOUT_GPREV] = Gp;"),
    ("state advanced by stats-only calls", "    if (commit) {\n        *g_prev = G;",
     "    if (1) {\n        *g_prev = G;"),
    ("s_max override ignored", "const double smax = (c->s_max > 0.0) ? c->s_max : sqrt((double)K);",
     "const double smax = sqrt((double)K);"),
    ("non-finite statistics not flagged",
     "if (!isfinite(W) || !isfinite(G) || !isfinite(V) || !isfinite(S)) nonfinite = 1;", ";"),
]


def _build(tmp, i, src):
    path = os.path.join(tmp, f"mutant{i}.c")
    lib = os.path.join(tmp, f"libmutant{i}.so")
    with open(path, "w") as f:
        f.write(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
                           "-ffp-contract=off", path, "-o", lib, "-lm"])
    return lib


def _pins_fail(lib):
    env = dict(os.environ, AGS_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode != 0, r.stdout[-2000:]


def test_mutant_list_applies_to_the_oracle():
    src = open(SRC).read()
    names = [m[0] for m in MUTANTS]
    assert len(set(names)) == len(names)
    for name, old, _ in MUTANTS:
        assert src.count(old) == 1, f"mutant '{name}': its text occurs {src.count(old)} times"


def test_unmutated_oracle_passes_the_pins(tmp_path):
    lib = _build(str(tmp_path), 0, open(SRC).read())
    failed, out = _pins_fail(lib)
    assert not failed, out


def test_every_mutant_fails_a_pin(tmp_path):
    src = open(SRC).read()

    def one(i):
        name, old, new = MUTANTS[i]
        lib = _build(str(tmp_path), i + 1, src.replace(old, new))
        return name, _pins_fail(lib)[0]

    workers = max(1, min(4, (os.cpu_count() or 2) // 2))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(one, range(len(MUTANTS))))
    survivors = [name for name, failed in results if not failed]
    assert not survivors, f"mutants no pin catches: {survivors}"
