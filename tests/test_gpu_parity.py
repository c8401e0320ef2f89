"""HIP path vs the float64 oracle on MI355X, through the C-ABI.

Workloads: the five CNN-shaped configurations (tiny CNN K=4 fp32 3 steps;
ResNet-18 CIFAR K=8 fp32 1 step; ResNet-50 K=16 bf16 10 steps; VGG-16 K=8
fp32 5 steps; the ResNet-50 K sweep, bf16) plus ragged and degenerate
layouts.  Every step compares all statistics and, after each step, every
element of w and m.
"""
import math

import numpy as np
import pytest

from ags_parity import Pair, check_params, check_stats, log, run_steps, to_device
from oracle import OracleAGS
from paper_2603_18112_amd import ags, layouts, synth

pytestmark = pytest.mark.gpu

SD = layouts.LAYER_SCALE | layouts.LAYER_DECAY


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ags.load_library()   # fails loudly if libags.so is not built
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------ the configs --


@pytest.mark.parametrize("mode", ["ags", "lars", "sgd", "static"])
def test_tiny_cnn_k4_three_steps(mode):
    lay = layouts.get_layout("tiny_cnn")
    run_steps(lay, 4, 3, mode=mode, label=f"tiny {mode}")


def test_resnet18_cifar_k8_one_step():
    lay = layouts.get_layout("resnet18_cifar")
    run_steps(lay, 8, 1, label="r18")


def test_resnet18_cifar_static_scaling_three_steps():
    # Static mapping U(s), s = 4 (one of the paper's s in {2, 4, 8, 16}).
    lay = layouts.get_layout("resnet18_cifar")
    run_steps(lay, 8, 3, mode="static", static_scale=4.0, label="r18 static")


def test_resnet50_k16_bf16_ten_steps():
    # The benchmark's launch configuration: the same layout, K, dtype and
    # replica stride as bench.py's default workload.
    lay = layouts.get_layout("resnet50")
    w = run_steps(lay, 16, 10, dtype="bf16", check_each=False, label="r50",
                  stride=layouts.replica_stride(lay))
    log(f"  r50 worst param error / tolerance scale: w {w[0]:.2e} m {w[1]:.2e}")


def test_vgg16_k8_five_steps():
    lay = layouts.get_layout("vgg16")
    run_steps(lay, 8, 5, check_each=False, label="vgg16")


@pytest.mark.parametrize("K", [1, 2, 4, 8, 32, 64])
def test_resnet50_sweep_parity(K):
    # The batch-size sweep at noise c = 0.5 for its configured 10 steps
    # (K = 16 is the ten-step test above), at the benchmark's stride.
    lay = layouts.get_layout("resnet50")
    run_steps(lay, K, 10, dtype="bf16", check_each=False, label=f"r50 K={K}",
              stride=layouts.replica_stride(lay))


@pytest.mark.parametrize("K,c,steps", [(2, 0.1, 10), (2, 2.0, 10), (64, 0.1, 4), (64, 2.0, 10)])
def test_resnet50_sweep_noise_levels_against_oracle(K, c, steps):
    """The sweep's other noise levels, c = 0.1 and 2.0 (per-replica noise std
    in units of the layer's sigma), against the oracle: every statistic
    (the noise ratio V_l / G_l among them) on every step and every element of
    w and m after every step.  K = 64 with c = 2.0 is the hardest case for
    the compiled replica loop's fp32 sums of g_k - g_0, each of which carries
    replica 0's own deviation (Eq. (1c) averaged in that shifted form)."""
    lay = layouts.get_layout("resnet50")
    w = run_steps(lay, K, steps, dtype="bf16", noise=c, check_each=True,
                  label=f"r50 K={K} c={c}", stride=layouts.replica_stride(lay))
    log(f"  r50 K={K} c={c}: worst param error / tolerance scale: w {w[0]:.2e} m {w[1]:.2e}")


def test_resnet50_sweep_noise_statistic_closed_form():
    """Per-layer noise ratio rho_l = V_l / G_l against its expectation under
    the generator, E[V]/E[G] = c^2 (K-1) / (K + c^2), for every K and c of the
    sweep (a property that holds at any size)."""
    import torch
    lay = layouts.get_layout("resnet50")
    sig = synth.layer_sigmas(lay, 0)
    w = torch.from_numpy(synth.init_weights(lay, 0)).cuda()
    m = torch.zeros_like(w)
    big = lay.numels >= 100_000
    for K in (1, 2, 4, 8, 16, 32, 64):
        h = ags.AGS(lay.table(), w, m, K, grad_dtype="bf16")
        for c in (0.1, 0.5, 2.0):
            g = to_device(synth.replica_grads(lay, K, 0, 0, noise=c, dtype="bf16", sigmas=sig))
            h.stats(g)
            s = h.read_stats()
            rho = s.layer["noise_ratio"]
            expect = c * c * (K - 1) / (K + c * c)
            if K == 1:
                assert np.all(rho == 0.0)
            else:
                n = lay.numels[big].astype(np.float64)
                tol = 8.0 / np.sqrt(n)
                err = np.abs(rho[big] / expect - 1)
                assert np.all(err < tol), (K, c, float(err.max()))
            # 0 < s <= s_max = sqrt(K) for every layer (state after refresh is
            # only formed by a step; the stats record holds the current one)
            assert np.all(s.layer["gradscale"] == 1.0)
            del g
        h.close()
        log(f"  sweep K={K} ok")


# ------------------------------------------------ ragged and edge layouts --


RAGGED = [1, 7, 8, 9, 63, 2047, 2048, 2049, 8191, 8192, 8193, 20003, 5, 64]


@pytest.mark.parametrize("K,dtype,r", [(3, "f32", 0), (5, "bf16", 2), (16, "bf16", -1),
                                       (2, "f32", 1), (6, "f32", -1), (1, "bf16", 0)])
def test_ragged_layout(K, dtype, r):
    flags = [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 3
    lay = layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    run_steps(lay, K, 4, dtype=dtype, small_replica=r, label=f"ragged K={K} {dtype} r={r}")


@pytest.mark.parametrize("K,dtype", [(65, "bf16"), (100, "f32"), (1024, "bf16")])
def test_large_k_runtime_replica_loop(K, dtype):
    # K outside the compiled set {1, 2, 4, 8, 16, 32, 64} takes the
    # runtime-K replica loop; 1024 is the largest K the C-ABI accepts.
    assert ags.AGS_MAX_K == 1024
    lay = layouts.custom_layout(RAGGED, pad=8)
    run_steps(lay, K, 2, dtype=dtype, label=f"large K={K} {dtype}")


def _mixed_sizes(n, seed, hi=5000):
    rng = np.random.default_rng(seed)
    return [int(x) for x in rng.integers(1, hi, size=n)]


@pytest.mark.parametrize("n_layers", [1024, 1300])
def test_many_layers(n_layers):
    # Many short layers of mixed sizes and flags: the finalize's per-layer
    # blocks and its global part over more than one thread per layer.
    sizes = _mixed_sizes(n_layers, n_layers)
    cyc = [SD, layouts.LAYER_SCALE, 0, layouts.LAYER_DECAY]
    flags = [cyc[i % 4] for i in range(n_layers)]
    lay = layouts.custom_layout(sizes, flags, pad=8)
    run_steps(lay, 3, 3, label=f"{n_layers} layers")


def test_one_large_layer_among_many_small_ones():
    sizes = [8] * 500 + [1500 * 2048] + [8] * 500
    lay = layouts.custom_layout(sizes, pad=8)
    run_steps(lay, 2, 3, dtype="bf16", label="large among small")


def test_flat_buffer_beyond_2_31_elements():
    """Element offsets past 2^31: a small layer, a filler of 2^31 + 4104
    elements with zero gradients and uniform weights, and a small layer
    after it (22 GB on the device).  The two small layers are compared
    with the oracle run on them alone: a zero-gradient filler adds nothing
    to ||gbar||^2, so Delta and every decision are the same.  The filler
    follows momentum SGD on weight decay alone, in closed form, checked on
    strided samples; its W is n w^2 and G, V, S are 0 (gradscale 1 by the
    zero-norm rule)."""
    import torch
    fill = (1 << 31) + 4104
    sizes = [1000, fill, 5000]
    lay = layouts.custom_layout(sizes, pad=8)
    table = lay.table()
    (o0, n0, _), (of, nf, _), (o2, n2, _) = table
    assert o2 > (1 << 31)
    K, hyper = 1, dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8)
    rng = np.random.default_rng(31)
    small_w = rng.standard_normal(n0 + n2).astype(np.float32)
    w = torch.full((lay.n_flat,), 0.5, dtype=torch.float32, device="cuda")
    w[o0:o0 + n0] = torch.from_numpy(small_w[:n0]).cuda()
    w[o2:o2 + n2] = torch.from_numpy(small_w[n0:]).cuda()
    m = torch.zeros_like(w)
    h = ags.AGS(table, w, m, K, grad_dtype="bf16", **hyper)
    sub = [(0, n0, SD), (n0, n2, SD)]
    ora = OracleAGS(sub, n0 + n2, K, small_w, grad_dtype="bf16", **hyper)
    g = torch.zeros((1, lay.n_flat), dtype=torch.int16, device="cuda")
    wf, mf = 0.5, 0.0
    lam, mu, eta = hyper["weight_decay"], hyper["momentum"], hyper["lr"]
    for t, c in enumerate([1.0, 1.1, 3.0]):        # the third step is sensitive
        gs = synth.to_bf16_bits((c * rng.standard_normal((1, n0 + n2))).astype(np.float32))
        g[0, o0:o0 + n0] = torch.from_numpy(gs[0, :n0].view(np.int16)).cuda()
        g[0, o2:o2 + n2] = torch.from_numpy(gs[0, n0:].view(np.int16)).cuda()
        h.step(g)
        ol, og = ora.step(gs)
        s = h.read_stats()
        gl = {f: np.asarray(s.layer[f])[[0, 2]] for f in s.layer}
        check_stats(gl, s.glob, ol, og, hyper["delta"], f"beyond 2^31 step {t + 1}")
        # filler: closed form, uniform over the layer
        mf = mu * mf + lam * wf
        wf = wf - eta * mf
        assert s.layer["g_sq"][1] == 0.0 and s.layer["var"][1] == 0.0
        assert s.layer["gsmall_sq"][1] == 0.0 and s.layer["gradscale"][1] == 1.0
        w_prev = wf + eta * mf
        assert abs(s.layer["w_sq"][1] / (nf * w_prev * w_prev) - 1.0) < 1e-4
        idx = torch.arange(of, of + nf, 7919 * 4099, device="cuda", dtype=torch.int64)
        idx = torch.cat([idx, torch.tensor([of + nf - 1], device="cuda")])
        ws, ms = w[idx].double().cpu().numpy(), m[idx].double().cpu().numpy()
        assert np.all(ws == ws[0]) and np.all(ms == ms[0])
        assert abs(ws[0] - wf) <= 1e-5 * abs(wf) and abs(ms[0] - mf) <= 1e-5 * abs(mf)
        torch.cuda.synchronize()
        wk = torch.cat([w[o0:o0 + n0], w[o2:o2 + n2]]).cpu().numpy()
        mk = torch.cat([m[o0:o0 + n0], m[o2:o2 + n2]]).cpu().numpy()
        check_params(wk, ora.w, sub, f"beyond 2^31 step {t + 1} w")
        check_params(mk, ora.m, sub, f"beyond 2^31 step {t + 1} m")
        log(f"  beyond 2^31: step {t + 1} ok (sensitive={og['sensitive']})")
    h.close()
    del w, m, g
    torch.cuda.empty_cache()


def test_stride_larger_than_n_flat():
    lay = layouts.custom_layout([100, 9000, 13], pad=8)
    run_steps(lay, 4, 2, stride=lay.n_flat + 4096 + 8, label="stride")


def test_single_element_layers_and_lars():
    lay = layouts.custom_layout([1] * 40 + [10_000], pad=8)
    run_steps(lay, 4, 3, mode="lars", label="1-elem lars")


@pytest.mark.parametrize("K,dtype", [(8, "f32"), (4, "bf16")])
def test_lars_with_unscaled_layers(K, dtype):
    # Mixed flags: unscaled layers keep a = 1 (plain momentum SGD).  K e_g of
    # 32 bytes keeps the replica mean between the passes, 8 bytes re-reads
    # the replicas in the update pass.
    flags = [SD, layouts.LAYER_DECAY, 0, layouts.LAYER_SCALE] * 4
    lay = layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    run_steps(lay, K, 3, dtype=dtype, mode="lars", label=f"lars mixed flags K={K} {dtype}")


def test_resnet18_cifar_lars_two_steps():
    # 1-D tensors (BN, biases) neither scaled nor decayed.
    lay = layouts.get_layout("resnet18_cifar")
    run_steps(lay, 8, 2, mode="lars", check_each=False, label="r18 lars")


# ------------------------------- LARS with the weight norms carried over --


@pytest.mark.parametrize("name,K,dtype,steps,extra", [
    ("tiny_cnn", 4, "f32", 3, {}),
    ("resnet18_cifar", 8, "f32", 3, {}),
    ("resnet50", 16, "bf16", 3, {}),
    ("ragged", 5, "bf16", 4, {"small_replica": 2}),
    ("ragged", 16, "bf16", 4, {"small_replica": -1}),
    ("ragged", 3, "f32", 4, {})])
def test_lars_carried_weight_norms_match_oracle(name, K, dtype, steps, extra):
    """LARS with reuse_w_norms: from the second step on, W_l comes from the
    sums of w^2 the previous update pass wrote, and every statistic and
    every element of w and m still match the oracle."""
    if name == "ragged":
        flags = [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 3
        lay = layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    else:
        lay = layouts.get_layout(name)
    stride = layouts.replica_stride(lay) if name == "resnet50" else None
    run_steps(lay, K, steps, dtype=dtype, mode="lars", reuse_w_norms=True, stride=stride,
              label=f"{name} lars carried K={K}", **extra)


def test_lars_carried_weight_norms_are_bitwise_those_of_reading_w():
    """The update pass sums the squares of the new w in the statistics
    pass's order, so carrying them gives the bits of reading w: steps and
    interleaved statistics calls with and without reuse_w_norms agree bit for
    bit (w, m, every statistic)."""
    import torch
    lay = layouts.custom_layout(RAGGED, [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 2
                                + [SD] * 4, pad=8)
    grads = [to_device(synth.replica_grads(lay, 16, t, 3, dtype="bf16")) for t in range(5)]
    w0 = synth.init_weights(lay, 3)
    torch.cuda.synchronize()

    def run(reuse):
        w = torch.from_numpy(w0.copy()).cuda()
        h = ags.AGS(lay.table(), w, torch.zeros_like(w), 16, grad_dtype="bf16", mode="lars",
                    reuse_w_norms=reuse)
        recs = []
        for t, g in enumerate(grads):
            h.step(g)
            recs.append(h.read_stats())
            h.stats(grads[(t + 2) % len(grads)])
            recs.append(h.read_stats())
        torch.cuda.synchronize()
        out = (h.w.cpu().numpy(), h.m.cpu().numpy(), recs)
        h.close()
        return out

    a, b = run(False), run(True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    for ra, rb in zip(a[2], b[2]):
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(ra.layer[f], rb.layer[f]), f
        assert ra.glob == rb.glob


def test_lars_weight_norms_dropped_when_the_caller_writes_w():
    """A caller that writes w between steps calls ags_invalidate_weight_norms
    (or restores a state with ags_set_state, which drops them too): the next
    step reads w again and matches the oracle run on the same new w."""
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    p = Pair(lay, 8, mode="lars", reuse_w_norms=True, seed=4)
    sig = synth.layer_sigmas(lay, 4)
    try:
        t = 0

        def one(what):
            nonlocal t
            g = synth.replica_grads(lay, 8, t, 4, sigmas=sig)
            p.step(g, what=what)
            p.check_state(what)
            t += 1

        one("before")
        one("carried")
        # an in-place edit of w by the caller (exact in both precisions)
        p.w.mul_(0.5)
        p.ora.w *= 0.5
        torch.cuda.synchronize()
        p.gpu.invalidate_weight_norms()
        one("after invalidate")
        one("carried again")
        # a checkpoint restore with other weights
        gs, gp, st = p.gpu.get_state()
        p.w.mul_(2.0)
        p.ora.w *= 2.0
        torch.cuda.synchronize()
        p.gpu.set_state(gs, gp, st)
        one("after set_state")
    finally:
        p.close()
    # a handle without carried norms has nothing to drop
    w = torch.from_numpy(synth.init_weights(lay, 0)).cuda()
    h = ags.AGS(lay.table(), w, torch.zeros_like(w), 8, mode="lars")
    with pytest.raises(ags.AGSError) as e:
        h.invalidate_weight_norms()
    assert e.value.status == ags.AGS_E_STATE
    h.close()


def test_identical_replicas_zero_variance_exactly():
    lay = layouts.get_layout("tiny_cnn")
    x = synth.replica_grads(lay, 1, 0, 0)
    for K, dt in ((7, "f32"), (16, "bf16"), (64, "bf16")):
        g = np.tile(x if dt == "f32" else synth.to_bf16_bits(x), (K, 1))
        p = Pair(lay, K, dtype=dt)
        s, _ = p.step(g)
        assert np.all(s.layer["var"] == 0.0) and np.all(s.layer["noise_ratio"] == 0.0)
        p.check_state("identical")
        p.close()


def test_k1_sgd_matches_oracle_and_plain_sgd():
    # K = 1 with scaling off is plain momentum SGD (the oracle is pinned to
    # torch.optim.SGD on the CPU for exactly this case).
    lay = layouts.get_layout("tiny_cnn")
    run_steps(lay, 1, 5, mode="sgd", label="K=1 sgd")
    lay2 = layouts.make_layout("tiny", layouts.tiny_cnn_tensors(), "all")
    t = [(o, n, layouts.LAYER_DECAY) for o, n, _ in lay2.table()]
    lay2.flags[:] = [f for _, _, f in t]
    run_steps(lay2, 1, 5, mode="ags", label="K=1 ags scale off")


def test_forced_spike_takes_unscaled_branch():
    lay = layouts.get_layout("resnet18_cifar")
    g1 = synth.replica_grads(lay, 8, 0, 0)
    p = Pair(lay, 8)
    s, _ = p.step(g1, what="spike 1")
    assert s.glob["sensitive"] == 1
    s, _ = p.step(g1, what="spike 2")          # Delta = 0: scaled
    assert s.glob["sensitive"] == 0 and s.glob["delta"] == 0.0
    scaled = lay.flags & layouts.LAYER_SCALE != 0
    assert np.any(s.layer["coef_a"][scaled] != 1.0)
    s, _ = p.step((g1 * np.float32(2)).astype(np.float32), what="spike 3")  # Delta = 3
    assert s.glob["sensitive"] == 1 and abs(s.glob["delta"] - 3.0) < 1e-6
    assert np.all(s.layer["coef_a"] == 1.0)
    p.check_state("spike")
    p.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_tie_at_the_threshold_is_sensitive(dtype):
    """Delta = delta exactly is sensitive (Algorithm 1 scales only when
    Delta < delta).  Two layers of the same size have the same tiles, so the
    same gradients in both give bitwise equal G_l: a step with the second
    layer zero and then one with it equal to the first doubles G exactly on
    both sides, and Delta = (2G - G) / G = 1 exactly (2G - G is exact).
    With delta = 1 that step is a tie."""
    n, K = 5000, 4
    lay = layouts.custom_layout([n, n], pad=8)
    (o0, _, _), (o1, _, _) = lay.table()
    x = synth.replica_grads(lay, K, 0, 7)[:, o0:o0 + n]
    one = np.zeros((K, lay.n_flat), np.float32)
    one[:, o0:o0 + n] = x
    both = one.copy()
    both[:, o1:o1 + n] = x
    if dtype == "bf16":
        one, both = synth.to_bf16_bits(one), synth.to_bf16_bits(both)
    p = Pair(lay, K, dtype=dtype, delta=1.0)
    expect = [(math.inf, 1), (0.0, 0), (1.0, 1), (0.0, 0)]
    for t, (g, (d, sens)) in enumerate(zip([one, one, both, both], expect)):
        s, (ol, og) = p.step(g, check=False, what=f"tie step {t + 1}")
        assert s.glob["delta"] == d == og["delta"], (t, s.glob["delta"], og["delta"])
        assert s.glob["sensitive"] == sens == og["sensitive"], t
        np.testing.assert_allclose(s.layer["coef_a"], ol["coef_a"], rtol=1e-6)
        p.check_state(f"tie step {t + 1}")
    p.close()


@pytest.mark.parametrize("K,dtype,mode", [(4, "f32", "ags"), (16, "bf16", "ags"),
                                          (3, "bf16", "ags"), (8, "f32", "static")])
def test_mispredicted_steps_are_corrected(K, dtype, mode):
    """AGS steps are applied with the coefficients predicted before the step
    (scaled unless Delta is infinite by definition); a sensitive step then
    takes the correction pass.  Gradient scales 1, 1, 2, 2, 0.25, 0.25, 1, 1
    make steps 1, 3, 5 and 7 sensitive (Delta = inf, 3, 0.9375, 15)."""
    lay = layouts.custom_layout(RAGGED, pad=8)
    base = synth.replica_grads(lay, K, 0, 4, dtype="f32")
    p = Pair(lay, K, dtype=dtype, seed=4, mode=mode, static_scale=3.0)
    sens = []
    for t, c in enumerate([1, 1, 2, 2, 0.25, 0.25, 1, 1]):
        g = (base * np.float32(c)).astype(np.float32)
        if dtype == "bf16":
            g = synth.to_bf16_bits(g)
        s, _ = p.step(g, what=f"mispredict step {t + 1}")
        sens.append(s.glob["sensitive"])
        p.check_state(f"mispredict step {t + 1}")
    assert sens == [1, 0, 1, 0, 1, 0, 1, 0]
    p.close()


def test_zero_and_nonfinite_gradients():
    lay = layouts.custom_layout([300, 17], pad=8)
    p = Pair(lay, 3, w0=np.ones(lay.n_flat, np.float32))
    z = np.zeros((3, lay.n_flat), np.float32)
    s, _ = p.step(z, what="zero 1")
    assert np.all(s.layer["gradscale"] == 1.0)
    s, _ = p.step(z, what="zero 2")
    assert s.glob["sensitive"] == 1 and math.isinf(s.glob["delta"])
    p.check_state("zero")
    bad = np.ones((3, lay.n_flat), np.float32)
    bad[1, 5] = np.inf
    g = to_device(bad)
    p.gpu.stats(g)
    s = p.gpu.read_stats()
    _, og = p.ora.stats(bad)
    assert s.glob["nonfinite"] == 1 == og["nonfinite"] and s.glob["sensitive"] == 1
    p.close()


def test_nonfinite_weight_is_flagged():
    # W_l is not finite while every gradient norm is: the step is flagged
    # although Delta is finite (the oracle's rule; nothing is compared
    # element by element, w holds an infinity).
    lay = layouts.custom_layout([300, 17], pad=8)
    w0 = np.ones(lay.n_flat, np.float32)
    w0[310] = np.inf
    p = Pair(lay, 3, w0=w0)
    g = np.ones((3, lay.n_flat), np.float32)
    for t in range(2):
        p.gpu.step(to_device(g))
        _, og = p.ora.step(g)
        s = p.gpu.read_stats()
        assert s.glob["nonfinite"] == 1 == og["nonfinite"]
        assert s.glob["sensitive"] == og["sensitive"] == (1 if t == 0 else 0)
        # inf on the first step; inf - eta * inf = nan afterwards
        assert not math.isfinite(s.layer["w_sq"][1]) and math.isfinite(s.layer["w_sq"][0])
    p.close()


# ----------------------------------------------------- state and contract --


def test_stats_call_does_not_mutate():
    lay = layouts.get_layout("tiny_cnn")
    p = Pair(lay, 4)
    p.step(synth.replica_grads(lay, 4, 0, 0))
    w, m = p.w.clone(), p.m.clone()
    st = p.gpu.get_state()
    p.step(synth.replica_grads(lay, 4, 1, 0), commit=False, what="stats only")
    assert p.torch.equal(w, p.w) and p.torch.equal(m, p.m)
    st2 = p.gpu.get_state()
    assert np.array_equal(st[0], st2[0]) and st[1:] == st2[1:]
    p.close()


def test_vgg16_capped_launches_against_oracle():
    """Layouts whose w and m outgrow the Infinity Cache (VGG-16: 1.1 GB)
    launch the statistics-only step kernel and the LARS update kernel with
    an LDS pad that caps their blocks per CU.  Here every such launch runs
    against the oracle: LARS steps (the first reads w, the next take the
    carried weight norms), a LARS statistics call between them, and the
    statistics call of an AGS handle; every statistic, and w and m after
    the last step."""
    lay = layouts.get_layout("vgg16")
    K = 8
    sig = synth.layer_sigmas(lay, 0)

    def grads(t):
        return synth.replica_grads(lay, K, t, 0, sigmas=sig)

    p = Pair(lay, K, mode="lars", reuse_w_norms=True)
    try:
        p.step(grads(0), what="vgg16 lars step 1")
        p.step(grads(1), commit=False, what="vgg16 lars stats call")
        p.step(grads(2), what="vgg16 lars step 2")
        p.step(grads(3), what="vgg16 lars step 3")
        p.check_state("vgg16 lars step 3")
    finally:
        p.close()
    log("  vgg16 lars ok")
    p = Pair(lay, K)
    try:
        p.step(grads(0), commit=False, what="vgg16 ags stats call")
        p.step(grads(1), what="vgg16 ags step 1")
        p.step(grads(2), commit=False, what="vgg16 ags stats call after a step")
        p.check_state("vgg16 ags step 1")
    finally:
        p.close()


def test_bitwise_determinism():
    lay = layouts.get_layout("resnet18_cifar")
    grads = [to_device(synth.replica_grads(lay, 8, t, 1)) for t in range(3)]
    outs = []
    for _ in range(2):
        p = Pair(lay, 8, seed=1)
        for g in grads:
            p.gpu.step(g)
        s = p.gpu.read_stats()
        outs.append((p.w.cpu().numpy(), p.m.cpu().numpy(), s.layer, p.gpu.get_state()))
        p.close()
    a, b = outs
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    for f in ags.LAYER_STATS_FIELDS:
        assert np.array_equal(a[2][f], b[2][f]), f
    assert np.array_equal(a[3][0], b[3][0]) and a[3][1:] == b[3][1:]


def test_two_handles_on_two_streams_interleaved():
    """Handles share no device state: two handles stepping in turn on two
    streams, with no synchronisation between their steps, end bitwise where
    each ends alone on the default stream."""
    import torch
    cases = [(layouts.get_layout("tiny_cnn"), 4, "f32", {}),
             (layouts.custom_layout(RAGGED, pad=8), 5, "bf16", {"elementwise": True})]
    grads = [[to_device(synth.replica_grads(lay, K, t, 7, dtype=dt)) for t in range(4)]
             for lay, K, dt, _ in cases]
    torch.cuda.synchronize()

    def run(interleaved):
        hs = []
        for lay, K, dt, extra in cases:
            w = torch.from_numpy(synth.init_weights(lay, 7)).cuda()
            hs.append(ags.AGS(lay.table(), w, torch.zeros_like(w), K, grad_dtype=dt, **extra))
        torch.cuda.synchronize()
        if interleaved:
            streams = [torch.cuda.Stream(), torch.cuda.Stream()]
            for t in range(4):
                for i, h in enumerate(hs):
                    h.step(grads[i][t], streams[i])
        else:
            for i, h in enumerate(hs):
                for t in range(4):
                    h.step(grads[i][t])
        torch.cuda.synchronize()
        out = [(h.w.cpu().numpy(), h.m.cpu().numpy(), h.read_stats().layer, h.get_state()) for h in hs]
        for h in hs:
            h.close()
        return out

    for a, b in zip(run(False), run(True)):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(a[2][f], b[2][f]), f
        assert np.array_equal(a[3][0], b[3][0]) and a[3][1:] == b[3][1:]


def test_one_handle_alternating_streams_is_ordered():
    """Every call of a handle shares its workspace and state, so a call on
    another stream than the handle's last one waits for the work queued
    there: one handle whose steps and statistics calls alternate between
    three streams, with no synchronisation between the calls, ends bitwise
    where the same calls on one stream end (w, m, statistics, state)."""
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    K = 8
    grads = [to_device(synth.replica_grads(lay, K, t, 11)) for t in range(6)]
    w0 = synth.init_weights(lay, 11)
    torch.cuda.synchronize()

    def run(streams):
        w = torch.from_numpy(w0.copy()).cuda()
        h = ags.AGS(lay.table(), w, torch.zeros_like(w), K, grad_dtype="f32")
        torch.cuda.synchronize()
        recs = []
        for t, g in enumerate(grads):
            h.step(g, streams[t % len(streams)])
            h.stats(grads[(t + 1) % len(grads)], streams[(t + 1) % len(streams)])
            if t % 2 == 1:
                # read_stats waits for the handle's last stream only
                recs.append(h.read_stats().layer)
        torch.cuda.synchronize()
        out = (h.w.cpu().numpy(), h.m.cpu().numpy(), recs, h.get_state())
        h.close()
        return out

    a = run([torch.cuda.current_stream()])
    b = run([torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.current_stream()])
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    for ra, rb in zip(a[2], b[2]):
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(ra[f], rb[f]), f
    assert np.array_equal(a[3][0], b[3][0]) and a[3][1:] == b[3][1:]


def _resume_grads(lay, K, n, seed, scale_from):
    # fresh draws; from step scale_from + 1 on the gradients are doubled, so
    # that step is sensitive (Delta = 3) and the next ones are not
    return [to_device(synth.replica_grads(lay, K, t, seed) * np.float32(2.0 if t >= scale_from else 1.0))
            for t in range(n)]


def test_checkpoint_resume_bitwise():
    """Resumed right after a sensitive step: with the last decision restored
    too, the resumed run predicts (and rounds) as the original, bit for bit;
    without it, the next step takes the other rounding path and agrees to
    the parameter tolerance."""
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    grads = _resume_grads(lay, 8, 10, 2, 4)
    a = Pair(lay, 8, seed=2)
    for g in grads:
        a.gpu.step(g)
    b = Pair(lay, 8, seed=2)
    for g in grads[:5]:
        b.gpu.step(g)
    state, last = b.gpu.get_state(), b.gpu.get_last_decision()
    assert last[0] == 1                    # step 5 was sensitive
    w2, m2 = b.w.clone(), b.m.clone()
    w3, m3 = b.w.clone(), b.m.clone()
    b.close()
    c = ags.AGS(lay.table(), w2, m2, 8, **{k: v for k, v in b.hyper.items()})
    c.set_state(*state)
    assert c.get_last_decision()[0] == 0   # cleared by set_state
    c.set_last_decision(*last)
    d = ags.AGS(lay.table(), w3, m3, 8, **{k: v for k, v in b.hyper.items()})
    d.set_state(*state)
    for g in grads[5:]:
        c.step(g)
        d.step(g)
    torch.cuda.synchronize()
    assert torch.equal(a.w, w2) and torch.equal(a.m, m2)
    sa, sc = a.gpu.get_state(), c.get_state()
    assert np.array_equal(sa[0], sc[0]) and sa[1:] == sc[1:]
    assert a.gpu.get_last_decision()[0] == c.get_last_decision()[0] == 0
    table = lay.table()
    check_params(w3.cpu().numpy(), a.w.cpu().numpy().astype(np.float64), table, "resumed without the bit")
    check_params(m3.cpu().numpy(), a.m.cpu().numpy().astype(np.float64), table, "resumed without the bit (m)")
    a.close()
    c.close()
    d.close()


def test_set_lr_and_profiling():
    lay = layouts.get_layout("tiny_cnn")
    p = Pair(lay, 4)
    p.gpu.set_profiling(True)
    for t, lr in enumerate([0.1, 0.05, 0.0]):
        p.gpu.set_lr(lr)
        g = synth.replica_grads(lay, 4, t, 0)
        p.gpu.step(to_device(g))
        p.ora.step(g, lr=lr)
    p.check_state("set_lr")
    ms, n = p.gpu.kernel_times()
    assert n == 3 and np.all(ms > 0)
    p.close()
    # SGD launches no second pass: its interval is empty.
    q = Pair(lay, 4, mode="sgd")
    q.gpu.set_profiling(True)
    for t in range(2):
        g = synth.replica_grads(lay, 4, t, 0)
        q.step(g, what=f"sgd profiled step {t + 1}")
    ms, n = q.gpu.kernel_times()
    assert n == 2 and ms[0] > 0 and ms[1] > 0 and ms[2] == 0
    q.close()


def _hip():
    import ctypes
    import torch  # noqa: F401  (its HIP runtime is the process's runtime)
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    hip.hipFree.argtypes = [ctypes.c_void_p]
    return hip


def _hip_malloc(hip, nbytes):
    import ctypes
    p = ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(p), nbytes) == 0
    return p.value


def test_bad_device_pointers_are_errors_not_faults():
    """Pointers that are not device memory, or allocations smaller than the
    layout needs, are rejected on the host (exact-size hipMalloc buffers:
    the torch caching allocator hides the size of its blocks)."""
    import torch
    hip = _hip()
    MB2 = 2 << 20
    n_flat = MB2 // 4                      # one replica = 2 MiB of fp32
    table = [(0, n_flat, SD)]
    w = _hip_malloc(hip, MB2)
    m = _hip_malloc(hip, MB2)
    g2 = _hip_malloc(hip, 2 * MB2)         # room for 2 replicas, K = 4 needs 4
    half = _hip_malloc(hip, MB2 // 2)
    try:
        cfg = ags.make_config(table, n_flat, 4)
        h = ags.ags_init(cfg, w, m, 0)
        for ptr, stride, status in [(g2, n_flat, ags.AGS_E_ARG),
                                    (g2, n_flat - 8, ags.AGS_E_ARG),
                                    (g2 + 4, n_flat, ags.AGS_E_ALIGN),
                                    (np.zeros((4, n_flat), np.float32).ctypes.data, n_flat, ags.AGS_E_ARG)]:
            with pytest.raises(ags.AGSError) as e:
                ags.ags_step(h, ptr, stride)
            assert e.value.status == status
        with pytest.raises(ags.AGSError) as e:
            ags.ags_step(h, m, n_flat)     # a replica stack on top of m
        assert e.value.status == ags.AGS_E_ARG and "overlap" in str(e.value)
        with pytest.raises(ags.AGSError) as e:
            ags.ags_read_stats(h, 1)       # nothing has run yet
        assert e.value.status == ags.AGS_E_STATE
        ags.ags_destroy(h)
        with pytest.raises(ags.AGSError) as e:
            ags.ags_init(cfg, half, m, 0)  # d_w smaller than n_flat floats
        assert e.value.status == ags.AGS_E_ARG
        host = np.zeros(n_flat, np.float32)
        with pytest.raises(ags.AGSError) as e:
            ags.ags_init(cfg, host.ctypes.data, m, 0)
        assert e.value.status == ags.AGS_E_ARG
    finally:
        torch.cuda.synchronize()
        for p in (w, m, g2, half):
            hip.hipFree(p)


@pytest.mark.parametrize("lay_name,K,dtype,hyper", [
    ("tiny_cnn", 4, "f32", {}), ("resnet18_cifar", 8, "f32", {}),
    ("tiny_cnn", 4, "bf16", {"elementwise": True}),
    ("resnet18_cifar", 8, "f32", {"elementwise": True, "refresh_every": 2}),
    ("tiny_cnn", 4, "f32", {"delta_scope": "layer", "mode": "static"}),
    ("tiny_cnn", 4, "f32", {"mode": "sgd"}),
    ("resnet18_cifar", 8, "bf16", {"mode": "lars"})])
def test_hip_graph_capture_replays_match_eager(lay_name, K, dtype, hyper):
    """One ags_step captured in a HIP graph and replayed with fresh gradients
    copied into the captured buffer between replays (with eager work and a
    synchronisation in between) gives, replay after replay, the same bits as
    eager steps.  The step enqueues kernels only (no memset or copy), and
    every decision that changes from step to step (the sensitive bit, the
    refresh, the element-scale buffer in force) is taken on the device."""
    import torch
    lay = layouts.get_layout(lay_name)
    w0 = torch.from_numpy(synth.init_weights(lay, 5)).cuda()
    grads = [to_device(synth.replica_grads(lay, K, t, 5, dtype=dtype)) for t in range(6)]
    we, me = w0.clone(), torch.zeros_like(w0)
    eager = ags.AGS(lay.table(), we, me, K, grad_dtype=dtype, **hyper)
    wg, mg = w0.clone(), torch.zeros_like(w0)
    graphed = ags.AGS(lay.table(), wg, mg, K, grad_dtype=dtype, **hyper)
    gbuf = torch.empty_like(grads[0])
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    graphed.set_profiling(True)     # a captured step is not timed
    with torch.cuda.graph(graph, stream=s):
        graphed.step(gbuf)
    torch.cuda.synchronize()
    assert graphed.kernel_times()[1] == 0
    graphed.set_profiling(False)
    # capturing does not run the step
    assert torch.equal(wg, w0) and graphed.get_state()[2] == 0
    for t, g in enumerate(grads):
        eager.step(g)
        gbuf.copy_(g)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(we, wg) and torch.equal(me, mg), f"replay {t + 1}"
        se, sg = eager.read_stats(), graphed.read_stats()
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(se.layer[f], sg.layer[f]), (t, f)
        assert se.glob == sg.glob
        if hyper.get("elementwise"):
            assert np.array_equal(eager.get_elementwise_scale(), graphed.get_elementwise_scale())
    eager.close()
    graphed.close()


@pytest.mark.parametrize("lay_name,K,dtype,hyper", [
    ("resnet18_cifar", 8, "f32", {}),
    ("tiny_cnn", 4, "bf16", {"elementwise": True}),
    ("resnet18_cifar", 8, "f32", {"mode": "lars", "reuse_w_norms": True})])
def test_set_lr_reaches_graph_replays(lay_name, K, dtype, hyper):
    """The learning rate lives in the device state: one step captured into a
    HIP graph, replayed under a schedule set with ags_set_lr between the
    replays (warm-up, decay, a zero rate), stays bitwise equal to eager
    steps under the same schedule, and both to the oracle at the last step
    (the update pass of LARS and the correction pass read it too)."""
    import torch
    lay = layouts.get_layout(lay_name)
    schedule = [0.1, 0.05, 0.2, 0.0, 0.08, 0.1]
    grads_np = [synth.replica_grads(lay, K, t, 9, dtype=dtype) * (2 if t == 3 else 1)
                if dtype == "f32" else synth.replica_grads(lay, K, t, 9, dtype=dtype)
                for t in range(len(schedule))]
    grads = [to_device(g) for g in grads_np]
    p = Pair(lay, K, dtype=dtype, seed=9, **hyper)  # "mode" goes to Pair's own argument
    wg, mg = torch.from_numpy(p.w0.copy()).cuda(), torch.zeros_like(p.w)
    graphed = ags.AGS(lay.table(), wg, mg, K, grad_dtype=dtype, mode=hyper.get("mode", "ags"),
                      **p.hyper)
    try:
        gbuf = torch.empty_like(grads[0])
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            graphed.step(gbuf)
        torch.cuda.synchronize()
        for t, (lr, g, g_np) in enumerate(zip(schedule, grads, grads_np)):
            p.gpu.set_lr(lr)
            p.gpu.step(g)
            p.prev_w, p.prev_m = p.ora.w.copy(), p.ora.m.copy()
            p.ora.step(g_np, lr=lr)
            graphed.set_lr(lr)
            gbuf.copy_(g)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(p.w, wg) and torch.equal(p.m, mg), f"lr {lr}, step {t + 1}"
        p.check_state(f"{lay_name} lr schedule")
        del graph
    finally:
        graphed.close()
        p.close()


def test_lars_carried_norms_with_graph_capture():
    """LARS with carried weight norms and HIP graphs: a captured step reads
    w (a replay cannot know whether w still holds what the last update
    wrote), and capturing leaves the handle's own choice alone, since the
    captured step has not run.  (a) A fresh handle captures a step, then
    steps eagerly (which must read w: no update pass has run), replays,
    steps, replays.  (b) A handle steps, captures, replays, has w, m and its
    state (global, last decision, per-layer) restored to an earlier point
    (ags_set_state drops the sums), and replays again.  Both end bitwise where eager steps on the same
    gradients end (the carried sums are bitwise those of reading w)."""
    import torch
    lay = layouts.get_layout("resnet18_cifar")
    K = 8
    hyper = dict(mode="lars", reuse_w_norms=True)
    grads = [to_device(synth.replica_grads(lay, K, t, 6)) for t in range(4)]
    w0 = torch.from_numpy(synth.init_weights(lay, 6)).cuda()

    def handle():
        w, m = w0.clone(), torch.zeros_like(w0)
        return ags.AGS(lay.table(), w, m, K, **hyper), w, m

    ref, wr, mr = handle()
    ref_after = []
    for g in grads:
        ref.step(g)
        torch.cuda.synchronize()
        ref_after.append((wr.clone(), mr.clone(), ref.read_stats()))
    ref.close()

    def same(w, m, h, t, what):
        rw, rm, rs = ref_after[t]
        assert torch.equal(w, rw) and torch.equal(m, rm), f"{what}: w, m after step {t + 1}"
        s = h.read_stats()
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(s.layer[f], rs.layer[f]), (what, t, f)

    def capture(h):
        gbuf = torch.empty_like(grads[0])
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            h.step(gbuf)
        torch.cuda.synchronize()
        return graph, gbuf

    def replay(graph, gbuf, g):
        gbuf.copy_(g)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()

    # (a) capture first, then eager and replayed steps in turn
    h, w, m = handle()
    graph, gbuf = capture(h)
    assert torch.equal(w, w0)
    for t, g in enumerate(grads):
        if t % 2 == 0:
            h.step(g)
            torch.cuda.synchronize()
        else:
            replay(graph, gbuf, g)
        same(w, m, h, t, "capture first")
    h.close()
    del graph

    # (b) step, capture, replay, restore an earlier point, replay again
    h, w, m = handle()
    h.step(grads[0])
    torch.cuda.synchronize()
    w1, m1 = w.clone(), m.clone()
    state1, last1, layer1 = h.get_state(), h.get_last_decision(), h.get_layer_state()
    graph, gbuf = capture(h)
    replay(graph, gbuf, grads[1])
    same(w, m, h, 1, "capture after a step")
    replay(graph, gbuf, grads[2])
    same(w, m, h, 2, "capture after a step")
    w.copy_(w1)
    m.copy_(m1)
    torch.cuda.synchronize()
    h.set_state(*state1)
    h.set_last_decision(*last1)
    h.set_layer_state(layer1)
    replay(graph, gbuf, grads[1])
    same(w, m, h, 1, "replay after a restore")
    h.step(grads[2])
    torch.cuda.synchronize()
    same(w, m, h, 2, "eager step after the replays")
    h.close()


def test_matches_golden_oracle_fixture():
    """The HIP path against the stored oracle output of the tiny CNN layout
    (tests/golden/tiny_cnn_ags_k4.json, written by a script that calls only
    the oracle), at the sampled elements and for every statistic."""
    import json
    import os
    import torch
    from ags_parity import PARAM_RTOL, STAT_RTOL
    with open(os.path.join(os.path.dirname(__file__), "golden", "tiny_cnn_ags_k4.json")) as f:
        gold = json.load(f)
    lay = layouts.get_layout(gold["layout"])
    w = torch.from_numpy(synth.init_weights(lay, gold["seed"])).cuda()
    m = torch.zeros_like(w)
    h = ags.AGS(lay.table(), w, m, gold["K"], **gold["hyper"])
    idx = gold["index"]
    for t, step in enumerate(gold["steps"]):
        h.step(to_device(synth.replica_grads(lay, gold["K"], t, gold["seed"])))
        s = h.read_stats()
        for k, v in step["layer"].items():
            np.testing.assert_allclose(s.layer[k], v, rtol=STAT_RTOL)
        assert s.glob["sensitive"] == step["global"]["sensitive"]
        wv, mv = w.cpu().numpy()[idx], m.cpu().numpy()[idx]
        for got, ref in ((wv, np.array(step["w"])), (mv, np.array(step["m"]))):
            scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref * ref)))
            assert np.all(np.abs(got - ref) <= PARAM_RTOL * scale)
    h.close()
