"""Seeded random configurations against the oracle (marker gpu).

Each case draws a ragged layout (1 to 40 layers of 1 to 150,000 elements,
random scale / decay flags, offsets aligned to 8 or 64), a replica count
from the compiled set and outside it, fp32 or bf16 replicas, a padded or
tight replica stride, and every option of the step that combines with the
others: mode (AGS, SGD, LARS, static), element scales (AGS), the per-layer
Delta scope, carried LARS weight norms, the small-batch replica (0, the
RMS over replicas, or another one), the refresh period and the noise
level.  Five steps run on both sides, the third on gradients doubled (an
exact scaling: Delta is about 3 there and 0.75 after it, so the decisions
run not sensitive, sensitive, sensitive, not sensitive and the correction
pass runs in both directions), with a statistics call between the second
and third steps.  Every statistic is compared on every call and
every element of w and m (and the element scales) after every step.

Delta and Delta_l depend only on the gradient sequence, so a throwaway
oracle run first picks a threshold delta that no Delta (and, with the
per-layer scope, no scaled layer's Delta_l) comes close to: a decision
taken at the threshold itself could go either way.
"""
import math

import numpy as np
import pytest

from paper_2603_18112_amd import layouts, synth
from oracle import OracleAGS
from ags_parity import Pair, log

pytestmark = pytest.mark.gpu

SD = layouts.LAYER_SCALE | layouts.LAYER_DECAY
FLAGS = [0, layouts.LAYER_SCALE, layouts.LAYER_DECAY, SD]
K_CHOICES = [1, 2, 3, 4, 5, 7, 8, 16, 17, 32, 64, 65]
N_CASES = 64
# replica elements per step (K * n_flat) above which a case is redrawn
MAX_REPLICA_ELEMS = 12_000_000
SCALES = [1.0, 1.0, 2.0, 1.0, 1.0]  # gradient factor per step


def draw_case(seed):
    rng = np.random.default_rng(seed)
    K = int(rng.choice(K_CHOICES))
    while True:
        L = int(rng.integers(1, 41))
        kind = rng.random(L)
        sizes = np.where(kind < 0.25, rng.integers(1, 65, L),
                         np.where(kind < 0.8, rng.integers(65, 12_000, L),
                                  rng.integers(12_000, 150_001, L)))
        flags = [FLAGS[int(i)] for i in rng.integers(0, 4, L)]
        pad = int(rng.choice([8, 64]))
        lay = layouts.custom_layout([int(s) for s in sizes], flags, pad=pad, name=f"random{seed}")
        if K * lay.n_flat <= MAX_REPLICA_ELEMS:
            break
    dtype = str(rng.choice(["f32", "bf16"]))
    mode = str(rng.choice(["ags", "sgd", "lars", "static"]))
    hyper = dict(delta_scope=str(rng.choice(["global", "layer"])),
                 refresh_every=int(rng.choice([1, 2, 3])))
    if mode == "ags" and rng.random() < 0.5:
        hyper["elementwise"] = True
    if mode == "lars" and rng.random() < 0.5:
        hyper["reuse_w_norms"] = True
    if mode == "static":
        hyper["static_scale"] = float(rng.choice([0.5, 2.0, 4.0]))
    r = rng.random()
    hyper["small_replica"] = 0 if (r < 0.4 or K == 1) else (-1 if r < 0.7 else int(rng.integers(1, K)))
    stride = lay.n_flat + (0 if rng.random() < 0.5 else 8 * int(rng.integers(1, 600)))
    noise = float(rng.choice([0.1, 0.5, 2.0]))
    return lay, K, dtype, mode, hyper, stride, noise


def doubled(g, dtype):
    """g times 2, exactly: fp32 by multiplication, bf16 by one more in the
    exponent field of every nonzero finite value."""
    if dtype == "f32":
        return g * np.float32(2.0)
    exp = (g >> 7) & 0xFF
    bump = (exp != 0) & (exp < 0xFE)
    return np.where(bump, g + np.uint16(0x80), g).astype(np.uint16)


def pick_delta(lay, K, dtype, grads, layer_scope):
    """A threshold that every Delta (and with the per-layer scope every
    scaled layer's Delta_l) of the sequence clears by at least 1%."""
    table = lay.table()
    o = OracleAGS(table, lay.n_flat, K, np.zeros(lay.n_flat, np.float32), mode="sgd",
                  grad_dtype=dtype)
    deltas = []
    for g in grads:
        layer, glob = o.step(g)
        deltas.append(glob["delta"])
        if layer_scope:
            deltas += [d for d, (_, _, f) in zip(layer["delta"], table) if f & layouts.LAYER_SCALE]
    finite = [d for d in deltas if math.isfinite(d)]
    for cand in (0.5, 0.43, 0.61, 0.37, 0.77, 0.29, 0.93, 1.3, 0.21, 1.9):
        if all(abs(d - cand) > 0.01 * cand for d in finite):
            return cand
    raise AssertionError("no clear threshold for this gradient sequence")


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_configuration_against_oracle(case):
    seed = 7000 + case
    lay, K, dtype, mode, hyper, stride, noise = draw_case(seed)
    desc = (f"case {case}: {len(lay.table())} layers, {lay.n_flat} elements, K={K} {dtype}, "
            f"{mode}, {hyper}, stride {stride}, noise {noise}")
    log(desc)
    sig = synth.layer_sigmas(lay, seed)
    grads = []
    for t, f in enumerate(SCALES):
        g = synth.replica_grads(lay, K, t, seed, noise=noise, dtype=dtype, sigmas=sig, stride=stride)
        grads.append(doubled(g, dtype) if f == 2.0 else g)
    hyper["delta"] = pick_delta(lay, K, dtype, grads, hyper["delta_scope"] == "layer")
    p = Pair(lay, K, dtype=dtype, mode=mode, seed=seed, stride=stride, **hyper)
    try:
        for t, g in enumerate(grads):
            if t == 2:
                p.step(g, commit=False, what=f"{desc} stats call")
            p.step(g, what=f"{desc} step {t + 1}")
            p.check_state(f"{desc} step {t + 1}")
    finally:
        p.close()


@pytest.mark.parametrize("case", range(32))
def test_random_configuration_resume_bitwise(case):
    """Checkpoint and resume on seeded random configurations: a handle
    steps three times (the third on doubled gradients, so its decision is
    sensitive); a second handle over copies of w and m takes the first's
    state, last decision, per-layer state and element scales; then both
    take three more steps (one more doubled) and stay bitwise equal in w,
    m, the element scales, the decisions and every statistic after each.
    The one exception is by design: with element scales the layer means of
    the scales (the coef_a and gradscale records, and the means
    ags_get_state reports) are recomputed on the host in fp64 by
    ags_set_elementwise_scale, while the kernels form them from fp32 tile
    sums; they agree to fp32 rounding until a refresh recomputes them on
    the device."""
    import torch
    from paper_2603_18112_amd import ags
    from ags_parity import to_device
    seed = 8000 + case
    lay, K, dtype, mode, hyper, stride, noise = draw_case(seed)
    desc = f"resume case {case}: {lay.n_flat} elements, K={K} {dtype}, {mode}, {hyper}"
    log(desc)
    sig = synth.layer_sigmas(lay, seed)
    scales = [1.0, 1.0, 2.0, 1.0, 2.0, 1.0]
    grads_np = []
    for t, f in enumerate(scales):
        g = synth.replica_grads(lay, K, t, seed, noise=noise, dtype=dtype, sigmas=sig, stride=stride)
        grads_np.append(doubled(g, dtype) if f == 2.0 else g)
    hyper["delta"] = pick_delta(lay, K, dtype, grads_np, hyper["delta_scope"] == "layer")
    grads = [to_device(g) for g in grads_np]
    table = lay.table()
    w0 = torch.from_numpy(synth.init_weights(lay, seed)).cuda()
    wa, ma = w0.clone(), torch.zeros_like(w0)
    a = ags.AGS(table, wa, ma, K, grad_dtype=dtype, mode=mode, **hyper)
    for g in grads[:3]:
        a.step(g)
    torch.cuda.synchronize()
    ew = bool(hyper.get("elementwise"))
    state, last, layer = a.get_state(), a.get_last_decision(), a.get_layer_state()
    scale = a.get_elementwise_scale() if ew else None
    wb, mb = wa.clone(), ma.clone()
    b = ags.AGS(table, wb, mb, K, grad_dtype=dtype, mode=mode, **hyper)
    b.set_state(None if ew else state[0], state[1], state[2])
    if ew:
        b.set_elementwise_scale(scale)
    b.set_layer_state(layer)
    b.set_last_decision(*last)
    try:
        for t, g in enumerate(grads[3:], start=4):
            a.step(g)
            b.step(g)
            torch.cuda.synchronize()
            assert torch.equal(wa, wb) and torch.equal(ma, mb), f"{desc}: w, m after step {t}"
            sa, sb = a.read_stats(), b.read_stats()
            for f in ags.LAYER_STATS_FIELDS:
                if ew and f in ("coef_a", "gradscale"):
                    np.testing.assert_allclose(sa.layer[f], sb.layer[f], rtol=1e-6, err_msg=f"{desc} {t} {f}")
                else:
                    assert np.array_equal(sa.layer[f], sb.layer[f]), (desc, t, f)
            assert sa.glob == sb.glob, (desc, t)
            ga, gb = a.get_state(), b.get_state()
            assert ga[1:] == gb[1:], (desc, t)
            if ew:
                np.testing.assert_allclose(ga[0], gb[0], rtol=1e-6, err_msg=f"{desc} {t} means")
            else:
                assert np.array_equal(ga[0], gb[0]), (desc, t)
            la, lb = a.get_last_decision(), b.get_last_decision()
            assert la[0] == lb[0] and np.array_equal(la[1], lb[1]), (desc, t)
            if ew:
                assert np.array_equal(a.get_elementwise_scale(), b.get_elementwise_scale()), (desc, t)
    finally:
        a.close()
        b.close()


@pytest.mark.parametrize("case", range(16))
def test_random_configuration_graph_replay_bitwise(case):
    """A step captured into a HIP graph on seeded random configurations:
    the graph, replayed with each step's gradients copied into the captured
    buffer, and eager steps on another handle stay bitwise equal in w, m,
    every statistic and the element scales, through the decision changes
    of doubled gradients (the refresh, the scale buffer in force and the
    sensitive bit are all taken on the device)."""
    import torch
    from paper_2603_18112_amd import ags
    from ags_parity import to_device
    seed = 8500 + case
    lay, K, dtype, mode, hyper, stride, noise = draw_case(seed)
    desc = f"graph case {case}: {lay.n_flat} elements, K={K} {dtype}, {mode}, {hyper}"
    log(desc)
    sig = synth.layer_sigmas(lay, seed)
    grads_np = []
    for t, f in enumerate(SCALES):
        g = synth.replica_grads(lay, K, t, seed, noise=noise, dtype=dtype, sigmas=sig, stride=stride)
        grads_np.append(doubled(g, dtype) if f == 2.0 else g)
    hyper["delta"] = pick_delta(lay, K, dtype, grads_np, hyper["delta_scope"] == "layer")
    grads = [to_device(g) for g in grads_np]
    table = lay.table()
    w0 = torch.from_numpy(synth.init_weights(lay, seed)).cuda()
    we, me = w0.clone(), torch.zeros_like(w0)
    wg, mg = w0.clone(), torch.zeros_like(w0)
    eager = ags.AGS(table, we, me, K, grad_dtype=dtype, mode=mode, **hyper)
    graphed = ags.AGS(table, wg, mg, K, grad_dtype=dtype, mode=mode, **hyper)
    try:
        gbuf = torch.empty_like(grads[0])
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            graphed.step(gbuf)
        torch.cuda.synchronize()
        assert torch.equal(wg, w0), desc
        for t, g in enumerate(grads):
            eager.step(g)
            gbuf.copy_(g)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(we, wg) and torch.equal(me, mg), f"{desc}: replay {t + 1}"
            se, sg = eager.read_stats(), graphed.read_stats()
            for f in ags.LAYER_STATS_FIELDS:
                assert np.array_equal(se.layer[f], sg.layer[f]), (desc, t, f)
            assert se.glob == sg.glob, (desc, t)
            if hyper.get("elementwise"):
                assert np.array_equal(eager.get_elementwise_scale(), graphed.get_elementwise_scale()), (desc, t)
        del graph
    finally:
        eager.close()
        graphed.close()
