"""Per-layer gradient variability (Delta_l decides layer l) on MI355X against
the float64 oracle, through the C-ABI.

Every step compares the statistics (including every layer's Delta_l and the
bit that decided it), every element of w and m, and the per-layer state.
"""
import numpy as np
import pytest

from ags_parity import Pair, log, run_steps, to_device
from paper_2603_18112_amd import ags, layouts, synth

pytestmark = pytest.mark.gpu

SD = layouts.LAYER_SCALE | layouts.LAYER_DECAY
RAGGED = [1, 7, 8, 9, 63, 2047, 2048, 2049, 8191, 8192, 8193, 20003, 5, 64]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ags.load_library()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("mode,kw", [("ags", {}), ("static", {"static_scale": 4.0}),
                                     ("ags", {"elementwise": True})])
def test_tiny_cnn_k4_four_steps(mode, kw):
    lay = layouts.get_layout("tiny_cnn")
    run_steps(lay, 4, 4, mode=mode, delta_scope="layer", label=f"layer-delta tiny {mode}", **kw)


@pytest.mark.parametrize("K,dtype,r", [(3, "f32", 0), (16, "bf16", -1), (5, "bf16", 2)])
def test_ragged_layout(K, dtype, r):
    flags = [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 3
    lay = layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    run_steps(lay, K, 4, dtype=dtype, small_replica=r, delta_scope="layer",
              label=f"layer-delta ragged K={K} {dtype} r={r}")


def test_resnet18_cifar_k8_three_steps():
    lay = layouts.get_layout("resnet18_cifar")
    run_steps(lay, 8, 3, delta_scope="layer", label="layer-delta r18")


def test_resnet50_k16_bf16_three_steps():
    lay = layouts.get_layout("resnet50")
    w = run_steps(lay, 16, 3, dtype="bf16", check_each=False, delta_scope="layer",
                  stride=layouts.replica_stride(lay), label="layer-delta r50")
    log(f"  layer-delta r50 worst param error / tolerance scale: w {w[0]:.2e} m {w[1]:.2e}")


def _rescale(base, table, factors):
    g = base.copy()
    for (o, n, _), c in zip(table, factors):
        g[:, o:o + n] *= np.float32(c)
    return g.astype(np.float32)


@pytest.mark.parametrize("K,dtype,mode,kw", [(4, "f32", "ags", {}), (16, "bf16", "ags", {}),
                                             (3, "bf16", "static", {"static_scale": 3.0}),
                                             (8, "f32", "ags", {"elementwise": True})])
def test_mispredicted_layers_are_corrected(K, dtype, mode, kw):
    """Per-layer factors make some layers sensitive on a step while the
    others are not: even layers x2 on step 2 (Delta_l = 3), odd layers
    x0.25 on step 4 (Delta_l = 0.9375), all unchanged otherwise.  Every layer
    is predicted scaled after the first step, so exactly the sensitive
    scaled layers take the correction pass."""
    lay = layouts.custom_layout(RAGGED, pad=8)
    table = lay.table()
    base = synth.replica_grads(lay, K, 0, 4, dtype="f32")
    L = len(table)
    f1 = [1.0] * L
    f2 = [2.0 if l % 2 == 0 else 1.0 for l in range(L)]
    f4 = [2.0 if l % 2 == 0 else 0.25 for l in range(L)]
    p = Pair(lay, K, dtype=dtype, seed=4, mode=mode, delta_scope="layer", **kw)
    expect = [[1] * L, [1 if l % 2 == 0 else 0 for l in range(L)], [0] * L,
              [0 if l % 2 == 0 else 1 for l in range(L)], [0] * L]
    for t, f in enumerate([f1, f2, f2, f4, f4]):
        g = _rescale(base, table, f)
        if dtype == "bf16":
            g = synth.to_bf16_bits(g)
        s, _ = p.step(g, what=f"layer mispredict step {t + 1}")
        assert list(s.layer["sensitive"]) == expect[t], (t, list(s.layer["sensitive"]))
        p.check_state(f"layer mispredict step {t + 1}")
    p.close()


def test_layer_state_set_from_the_oracle_then_steps():
    lay = layouts.custom_layout([5000, 300, 2049, 77], [SD, 0, layouts.LAYER_SCALE, SD], pad=8)
    p = Pair(lay, 4, delta_scope="layer")
    g0 = synth.replica_grads(lay, 4, 0, 9)
    p.ora.stats(g0)
    st, _ = p.ora.stats(g0)
    # previous norms: each layer's own norm times 0.9, 3, 1.2, 0 (Delta_l =
    # 0.11, 0.67, 0.17, inf on the first step from this state)
    gp = st["g_sq"] * np.array([0.9, 3.0, 1.2, 0.0])
    p.ora.set_state(np.full(4, 1.5), float(gp.sum()), 5)
    p.ora.set_layer_state(gp)
    p.gpu.set_state(np.full(4, 1.5), float(gp.sum()), 5)
    p.gpu.set_layer_state(gp)
    for t in range(3):
        p.step(synth.replica_grads(lay, 4, t, 9), what=f"layer state {t + 1}")
        p.check_state(f"layer state {t + 1}")
    p.close()


def test_checkpoint_resume_bitwise():
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    # step 3 doubles every gradient (every layer sensitive): the resumed run
    # restores the layers' last decisions too
    grads = [to_device(synth.replica_grads(lay, 8, t, 2) * np.float32(2.0 if t >= 2 else 1.0))
             for t in range(8)]
    hyper = dict(delta_scope="layer")
    a = Pair(lay, 8, seed=2, **hyper)
    for g in grads:
        a.gpu.step(g)
    b = Pair(lay, 8, seed=2, **hyper)
    for g in grads[:3]:
        b.gpu.step(g)
    state, lstate = b.gpu.get_state(), b.gpu.get_layer_state()
    last = b.gpu.get_last_decision()
    assert last[1].sum() > 0
    w2, m2 = b.w.clone(), b.m.clone()
    b.close()
    c = ags.AGS(lay.table(), w2, m2, 8, **b.hyper)
    c.set_state(*state)
    c.set_layer_state(lstate)
    assert c.get_last_decision()[1].sum() == 0      # cleared by set_layer_state
    c.set_last_decision(*last)
    for g in grads[3:]:
        c.step(g)
    torch.cuda.synchronize()
    assert torch.equal(a.w, w2) and torch.equal(a.m, m2)
    assert np.array_equal(a.gpu.get_layer_state(), c.get_layer_state())
    a.close()
    c.close()


def test_global_scope_reports_layer_delta_and_global_bit():
    lay = layouts.get_layout("tiny_cnn")
    p = Pair(lay, 4)
    for t in range(3):
        s, (ol, og) = p.step(synth.replica_grads(lay, 4, t, 0), what=f"global scope {t + 1}")
        assert np.all(s.layer["sensitive"] == og["sensitive"])
    p.check_state("global scope")
    p.close()


def test_layer_state_argument_errors():
    lay = layouts.custom_layout([100, 20], pad=8)
    p = Pair(lay, 2)
    for bad in ([-1.0, 0.0], [np.nan, 1.0], [np.inf, 1.0]):
        with pytest.raises(ags.AGSError) as e:
            p.gpu.set_layer_state(bad)
        assert e.value.status == ags.AGS_E_ARG
    assert np.all(p.gpu.get_layer_state() == 0.0)
    # the last decision: bits only, nothing changed on a refusal
    for g, per in ((2, None), (0, [0, 3]), (-1, [0, 0])):
        with pytest.raises(ags.AGSError) as e:
            p.gpu.set_last_decision(g, per)
        assert e.value.status == ags.AGS_E_ARG
    g, per = p.gpu.get_last_decision()
    assert g == 0 and list(per) == [0, 0]
    p.gpu.set_last_decision(1, [1, 0])
    g, per = p.gpu.get_last_decision()
    assert g == 1 and list(per) == [1, 0]
    p.gpu.set_last_decision(0)            # the layers' bits stay
    g, per = p.gpu.get_last_decision()
    assert g == 0 and list(per) == [1, 0]
    p.close()
