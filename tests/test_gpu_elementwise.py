"""Elementwise AGS (Algorithm 1 read per parameter element) on MI355X against
the float64 oracle, through the C-ABI.

Every step compares the statistics (with per-layer means of the applied
coefficients and of the scales), every element of w and m, and every
element scale of every layer.
"""
import numpy as np
import pytest

from ags_parity import Pair, check_scales, log, run_steps, to_device
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


def test_tiny_cnn_k4_four_steps():
    lay = layouts.get_layout("tiny_cnn")
    run_steps(lay, 4, 4, elementwise=True, label="ew tiny")


@pytest.mark.parametrize("K,dtype,r", [(3, "f32", 0), (5, "bf16", 2), (16, "bf16", -1),
                                       (6, "f32", -1), (1, "bf16", 0), (64, "bf16", 0)])
def test_ragged_layout(K, dtype, r):
    flags = [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 3
    lay = layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    run_steps(lay, K, 4, dtype=dtype, small_replica=r, elementwise=True,
              label=f"ew ragged K={K} {dtype} r={r}")


@pytest.mark.parametrize("K,dtype", [(100, "f32"), (1024, "bf16")])
def test_large_k_runtime_replica_loop(K, dtype):
    # The runtime-K replica loop with the fp64 replica sums of the refresh,
    # up to the largest K the C-ABI accepts.
    lay = layouts.custom_layout(RAGGED, pad=8)
    run_steps(lay, K, 2, dtype=dtype, elementwise=True, label=f"ew large K={K} {dtype}")


@pytest.mark.parametrize("n_layers", [1024, 1100])
def test_many_layers(n_layers):
    # Layer means of the refreshed scales over many short layers (the
    # finalize's global part handles several layers per thread).
    rng = np.random.default_rng(n_layers)
    sizes = [int(x) for x in rng.integers(1, 3000, size=n_layers)]
    cyc = [SD, layouts.LAYER_SCALE, 0, layouts.LAYER_DECAY]
    lay = layouts.custom_layout(sizes, [cyc[i % 4] for i in range(n_layers)], pad=8)
    run_steps(lay, 3, 3, elementwise=True, label=f"ew {n_layers} layers")


def test_resnet18_cifar_k8_three_steps():
    lay = layouts.get_layout("resnet18_cifar")
    run_steps(lay, 8, 3, elementwise=True, label="ew r18")


def test_resnet50_k16_bf16_three_steps():
    # The benchmark's elementwise workload: layout, K, dtype and stride.
    lay = layouts.get_layout("resnet50")
    w = run_steps(lay, 16, 3, dtype="bf16", check_each=False, elementwise=True,
                  stride=layouts.replica_stride(lay), label="ew r50")
    log(f"  ew r50 worst param error / tolerance scale: w {w[0]:.2e} m {w[1]:.2e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_streaming_variant_above_the_cache_sized_working_set(dtype):
    # 13.1M elements: w, m and the two scale buffers (16 bytes per element)
    # pass 192 MiB, so the step kernel takes its non-temporal variant; ragged
    # layers and one large one, every flag combination.
    sizes = [13_000_000, 7, 2049, 20003, 63, 77_777, 1]
    flags = [SD, layouts.LAYER_SCALE, 0, layouts.LAYER_DECAY, SD, SD, 0]
    lay = layouts.custom_layout(sizes, flags, pad=8)
    assert 16 * lay.n_flat > 192 << 20
    run_steps(lay, 4, 3, dtype=dtype, elementwise=True, label=f"ew streaming {dtype}")


def test_vgg16_k8_two_steps():
    # The largest layout: streaming accesses, the XCD-aware tile order and
    # fp32 replicas at full size (138M elements, 67,569 tiles).
    lay = layouts.get_layout("vgg16")
    run_steps(lay, 8, 2, check_each=False, elementwise=True, stride=layouts.replica_stride(lay),
              label="ew vgg16")


def test_refresh_every_three_steps():
    # Scales refresh on steps 3 and 6 only: the buffer in force must carry
    # over between refreshes.
    lay = layouts.custom_layout(RAGGED, pad=8)
    run_steps(lay, 4, 7, refresh_every=3, elementwise=True, label="ew refresh 3")


def test_no_refresh_keeps_unit_scales():
    lay = layouts.custom_layout([100, 3000], pad=8)
    p = Pair(lay, 4, elementwise=True, refresh_every=0)
    for t in range(3):
        p.step(synth.replica_grads(lay, 4, t, 0), what=f"no refresh {t + 1}")
        p.check_state(f"no refresh {t + 1}")
    e = p.gpu.get_elementwise_scale()
    assert np.all(e[:100] == 1.0) and np.all(e[104:3104] == 1.0)
    p.close()


@pytest.mark.parametrize("K,dtype,r", [(4, "f32", 0), (16, "bf16", -1), (3, "bf16", 1)])
def test_mispredicted_steps_are_corrected_per_element(K, dtype, r):
    """Gradient scales 1, 1, 2, 2, 0.25, 0.25, 1, 1 make steps 1, 3, 5 and 7
    sensitive; steps 3, 5 and 7 were applied with the element scales and
    take the per-element correction c_j = 1 - gradscale_j."""
    lay = layouts.custom_layout(RAGGED, pad=8)
    base = synth.replica_grads(lay, K, 0, 4, dtype="f32")
    p = Pair(lay, K, dtype=dtype, seed=4, small_replica=r, elementwise=True)
    sens = []
    for t, c in enumerate([1, 1, 2, 2, 0.25, 0.25, 1, 1]):
        g = (base * np.float32(c)).astype(np.float32)
        if dtype == "bf16":
            g = synth.to_bf16_bits(g)
        s, _ = p.step(g, what=f"ew mispredict step {t + 1}")
        sens.append(s.glob["sensitive"])
        p.check_state(f"ew mispredict step {t + 1}")
    assert sens == [1, 0, 1, 0, 1, 0, 1, 0]
    p.close()


def test_degenerate_ratios():
    """eps = 0, K = 2, replica 0 as the small-batch gradient:
    g = (x, -x): gbar = 0, ratio x/0 -> clipped to s_max;
    g = (0, 0): 0/0 -> 1;  g = (0, y): 0 / (y/2) -> 0 (the element is
    frozen on non-sensitive steps); the rest random."""
    lay = layouts.custom_layout([64, 24], [SD, 0], pad=8)
    rng = np.random.default_rng(5)
    g = np.zeros((2, lay.n_flat), np.float32)
    x = rng.standard_normal(16).astype(np.float32)
    g[0, 0:16], g[1, 0:16] = x, -x
    g[1, 32:48] = rng.standard_normal(16).astype(np.float32)
    g[:, 48:64] = rng.standard_normal((2, 16)).astype(np.float32)
    g[:, 64:88] = rng.standard_normal((2, 24)).astype(np.float32)
    p = Pair(lay, 2, eps=0.0, s_max=3.0, elementwise=True)
    s, _ = p.step(g, what="degenerate 1")
    p.check_state("degenerate 1")
    e = p.gpu.get_elementwise_scale()
    assert np.all(e[0:16] == 3.0) and np.all(e[16:32] == 1.0) and np.all(e[32:48] == 0.0)
    assert np.all(e[64:88] == 1.0)            # unscaled layer: never refreshed
    s, _ = p.step(g, what="degenerate 2")     # Delta = 0: scales applied
    assert s.glob["sensitive"] == 0
    p.check_state("degenerate 2")
    p.close()


def test_nonfinite_gradients_give_unit_or_clipped_scales():
    lay = layouts.custom_layout([40], pad=8)
    g = np.ones((3, lay.n_flat), np.float32)
    g[1, 3] = np.inf                      # gbar inf, g_small 1: 1 / inf -> 0
    g[0, 5] = np.inf                      # g_small inf too: inf / inf -> 1
    g[2, 7] = np.nan                      # nan -> 1
    p = Pair(lay, 3, elementwise=True)
    p.gpu.step(to_device(g))
    p.ora.step(g)
    e = p.gpu.get_elementwise_scale()
    ogs = p.ora.get_state()[0]
    check_scales(e, ogs, p.table, "nonfinite")
    assert e[3] == 0.0 and e[5] == e[7] == 1.0
    p.close()


def test_scales_set_from_the_oracle_then_steps():
    """Arbitrary scales (including non-1 values on an unscaled layer, which
    a refresh carries over unchanged) set on both sides, then three steps."""
    flags = [SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY]
    lay = layouts.custom_layout([5000, 300, 2049, 77], flags, pad=8)
    p = Pair(lay, 4, elementwise=True, small_replica=-1)
    rng = np.random.default_rng(9)
    sc = rng.uniform(0.0, 2.0, lay.n_flat).astype(np.float32)
    p.gpu.set_elementwise_scale(sc)
    gs = sc.astype(np.float64)
    p.ora.set_state(gs, 1.0, 3)
    p.gpu.set_state(None, 1.0, 3)
    for t in range(3):
        p.step(synth.replica_grads(lay, 4, t, 9), what=f"set scales {t + 1}")
        p.check_state(f"set scales {t + 1}")
    p.close()


def test_stats_call_does_not_mutate():
    lay = layouts.get_layout("tiny_cnn")
    p = Pair(lay, 4, elementwise=True)
    p.step(synth.replica_grads(lay, 4, 0, 0))
    p.step(synth.replica_grads(lay, 4, 1, 0))
    w, m = p.w.clone(), p.m.clone()
    e = p.gpu.get_elementwise_scale()
    st = p.gpu.get_state()
    p.step(synth.replica_grads(lay, 4, 2, 0), commit=False, what="ew stats only")
    assert p.torch.equal(w, p.w) and p.torch.equal(m, p.m)
    assert np.array_equal(e, p.gpu.get_elementwise_scale())
    st2 = p.gpu.get_state()
    assert np.array_equal(st[0], st2[0]) and st[1:] == st2[1:]
    p.close()


def test_checkpoint_resume_bitwise():
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    # step 3 is sensitive (gradients doubled from it on): the resumed run
    # restores the last decision too
    grads = [to_device(synth.replica_grads(lay, 8, t, 2) * np.float32(2.0 if t >= 2 else 1.0))
             for t in range(8)]
    hyper = dict(elementwise=True, refresh_every=1)
    a = Pair(lay, 8, seed=2, **hyper)
    for g in grads:
        a.gpu.step(g)
    b = Pair(lay, 8, seed=2, **hyper)
    for g in grads[:3]:
        b.gpu.step(g)
    state, last = b.gpu.get_state(), b.gpu.get_last_decision()
    assert last[0] == 1
    scales = b.gpu.get_elementwise_scale()
    w2, m2 = b.w.clone(), b.m.clone()
    b.close()
    c = ags.AGS(lay.table(), w2, m2, 8, **b.hyper)
    c.set_state(None, state[1], state[2])
    c.set_last_decision(*last)
    c.set_elementwise_scale(scales)
    for g in grads[3:]:
        c.step(g)
    torch.cuda.synchronize()
    assert torch.equal(a.w, w2) and torch.equal(a.m, m2)
    assert np.array_equal(a.gpu.get_elementwise_scale(), c.get_elementwise_scale())
    sa, sc = a.gpu.get_state(), c.get_state()
    assert np.array_equal(sa[0], sc[0]) and sa[1:] == sc[1:]
    a.close()
    c.close()


def test_bitwise_determinism():
    lay = layouts.get_layout("resnet18_cifar")
    grads = [to_device(synth.replica_grads(lay, 8, t, 1, dtype="bf16")) for t in range(3)]
    outs = []
    for _ in range(2):
        p = Pair(lay, 8, seed=1, dtype="bf16", elementwise=True, small_replica=-1)
        for g in grads:
            p.gpu.step(g)
        outs.append((p.w.cpu().numpy(), p.m.cpu().numpy(), p.gpu.get_elementwise_scale(),
                     p.gpu.read_stats().layer))
        p.close()
    a, b = outs
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    for f in ags.LAYER_STATS_FIELDS:
        assert np.array_equal(a[3][f], b[3][f]), f


def test_elementwise_scale_argument_errors():
    lay = layouts.custom_layout([100, 20], pad=8)
    p = Pair(lay, 2, elementwise=True)
    n = lay.n_flat
    good = np.ones(n, np.float32)
    for bad in (np.ones(n - 1, np.float32), np.ones(n + 8, np.float32)):
        with pytest.raises(ags.AGSError) as e:
            p.gpu.set_elementwise_scale(bad)
        assert e.value.status == ags.AGS_E_ARG
    for v in (-1.0, np.nan, np.inf):
        x = good.copy()
        x[7] = v
        with pytest.raises(ags.AGSError) as e:
            p.gpu.set_elementwise_scale(x)
        assert e.value.status == ags.AGS_E_ARG
    assert np.all(p.gpu.get_elementwise_scale()[:100] == 1.0)   # nothing changed
    with pytest.raises(ags.AGSError) as e:
        ags.ags_get_elementwise_scale(p.gpu.handle, n + 1)
    assert e.value.status == ags.AGS_E_ARG
    p.close()
    q = Pair(lay, 2)                                            # per-layer handle
    with pytest.raises(ags.AGSError) as e:
        q.gpu.get_elementwise_scale()
    assert e.value.status == ags.AGS_E_STATE
    with pytest.raises(ags.AGSError) as e:
        q.gpu.set_elementwise_scale(good)
    assert e.value.status == ags.AGS_E_STATE
    with pytest.raises(ags.AGSError) as e:
        q.gpu.set_state(None, 0.0, 0)
    assert e.value.status == ags.AGS_E_ARG
    q.close()
