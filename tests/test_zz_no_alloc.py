"""ags_stats_noalloc, the entry point that allocates no device memory,
against ags_stats on a handle (and both against the oracle), through the
C-ABI.

Its tables live in the library's one scratch array per GPU, which keeps the
last call's contents, so the calls run in a row on shrinking inputs: a
stale tile map, partial or counter from a bigger call would show up as a
difference in a smaller one.
"""
import numpy as np
import pytest

from ags_parity import check_stats, log, to_device
from oracle import OracleAGS
from paper_2603_18112_amd import ags, layouts, synth

pytestmark = pytest.mark.gpu

SD = layouts.LAYER_SCALE | layouts.LAYER_DECAY
RAGGED = [1, 7, 8, 9, 63, 2047, 2048, 2049, 8191, 8192, 8193, 20003, 5, 64]

# Largest first: every call is smaller than the one before it.
CASES = [
    ("resnet50", 16, "bf16", dict(mode="ags")),
    ("resnet18_cifar", 8, "f32", dict(mode="lars")),
    ("ragged", 5, "bf16", dict(mode="ags", elementwise=True, small_replica=-1)),
    ("tiny_cnn", 4, "f32", dict(mode="static", static_scale=4.0, delta_scope="layer")),
]


def _layout(name):
    if name == "ragged":
        flags = [SD, SD, 0, layouts.LAYER_SCALE, layouts.LAYER_DECAY] * 3
        return layouts.custom_layout(RAGGED, flags[:len(RAGGED)], pad=8)
    return layouts.get_layout(name)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ags.load_library()
    yield
    torch.cuda.synchronize()


def test_noalloc_stats_match_ags_stats_call_after_call():
    import torch
    hyper = dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8, s_max=0.0,
                 trust_coef=1e-3, refresh_every=1, small_replica=0)
    stream = torch.cuda.current_stream()
    for seed, (name, K, dt, extra) in enumerate(CASES):
        lay = _layout(name)
        hp = {**hyper, **extra}
        stride = layouts.replica_stride(lay)
        w0 = synth.init_weights(lay, seed)
        g_np = synth.replica_grads(lay, K, 0, seed, dtype=dt, stride=stride)
        w = torch.from_numpy(w0.copy()).cuda()
        m = torch.zeros_like(w)
        g = to_device(g_np)
        torch.cuda.synchronize()
        log(f"  no-alloc {name} K={K} {dt} {extra}")

        cfg = ags.make_config(lay.table(), lay.n_flat, K, grad_dtype=dt, **hp)
        nl, ng = ags.ags_stats_noalloc(cfg, w.data_ptr(), g.data_ptr(), stride,
                                       stream.cuda_stream)

        h = ags.AGS(lay.table(), w, m, K, grad_dtype=dt, **hp)
        h.stats(g)
        s = h.read_stats()
        h.close()
        # the same kernels on the same bytes: the same bits
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(nl[f], s.layer[f]), (name, f)
        assert ng == s.glob, name
        # and the oracle's statistics of a first step
        ora_hyper = {k: v for k, v in hp.items()}
        mode = ora_hyper.pop("mode")
        o = OracleAGS(lay.table(), lay.n_flat, K, w0, mode=mode, grad_dtype=dt, **ora_hyper)
        ol, og = o.stats(g_np)
        check_stats(nl, ng, ol, og, hp["delta"], f"no-alloc {name}")
        assert ng["step"] == 0 and ng["sensitive"] == 1
        # w is only read
        assert torch.equal(w, torch.from_numpy(w0).cuda())
        del g, w, m


def test_noalloc_random_configs_match_ags_stats():
    """Seeded random configurations (the generator of the random parity
    sweep: ragged layouts, K from 2 to 65, fp32 or bf16, every mode, element
    scales, both Delta scopes, every small-batch replica choice, padded
    strides) in no particular order of size: every call bitwise equal to a
    handle's ags_stats on the same bytes, and within tolerance of the
    oracle's statistics of a first step."""
    import torch
    from test_gpu_random_configs import draw_case
    stream = torch.cuda.current_stream()
    for case in range(24):
        seed = 9100 + case
        lay, K, dt, mode, hyper, stride, noise = draw_case(seed)
        hp = dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8, mode=mode,
                  **{k: v for k, v in hyper.items() if k != "reuse_w_norms"})
        w0 = synth.init_weights(lay, seed)
        g_np = synth.replica_grads(lay, K, 0, seed, noise=noise, dtype=dt, stride=stride)
        w = torch.from_numpy(w0.copy()).cuda()
        m = torch.zeros_like(w)
        g = to_device(g_np)
        torch.cuda.synchronize()
        what = f"no-alloc case {case}: {lay.n_flat} elements, K={K} {dt} {hp}"
        log("  " + what)
        cfg = ags.make_config(lay.table(), lay.n_flat, K, grad_dtype=dt, **hp)
        nl, ng = ags.ags_stats_noalloc(cfg, w.data_ptr(), g.data_ptr(), stride, stream.cuda_stream)
        h = ags.AGS(lay.table(), w, m, K, grad_dtype=dt, **hp)
        h.stats(g)
        s = h.read_stats()
        h.close()
        for f in ags.LAYER_STATS_FIELDS:
            assert np.array_equal(nl[f], s.layer[f]), (what, f)
        assert ng == s.glob, what
        ora = {k: v for k, v in hp.items() if k != "mode"}
        o = OracleAGS(lay.table(), lay.n_flat, K, w0, mode=mode, grad_dtype=dt, **ora)
        ol, og = o.stats(g_np)
        check_stats(nl, ng, ol, og, hp["delta"], what,
                    layer_scope=hp.get("delta_scope") == "layer",
                    scaled=[bool(f & layouts.LAYER_SCALE) for _, _, f in lay.table()])
        assert torch.equal(w, torch.from_numpy(w0).cuda()), what
        del g, w, m
