"""Layouts and the seeded input generator (host only)."""
import numpy as np
import pytest
import torch

from paper_2603_18112_amd import layouts, synth


# Parameter counts of the public architectures (He et al. 2016 ResNet-18
# for CIFAR and ResNet-50 for ImageNet; Simonyan & Zisserman 2015 VGG-16).
@pytest.mark.parametrize("name,L,n,n_1d", [
    ("tiny_cnn", 8, 24_234, 4),
    ("resnet18_cifar", 62, 11_173_962, 41),
    ("resnet50", 161, 25_557_032, 107),
    ("vgg16", 32, 138_357_544, 16),
])
def test_layout_counts(name, L, n, n_1d):
    lay = layouts.get_layout(name)
    assert lay.n_layers == L
    assert lay.n_params == n
    assert sum(1 for t in lay.tensors if len(t.shape) == 1) == n_1d
    assert np.all(lay.offsets % layouts.PAD_ELEMS == 0)
    assert np.all(lay.offsets[1:] >= lay.offsets[:-1] + lay.numels[:-1])
    assert lay.n_flat % layouts.PAD_ELEMS == 0
    assert lay.n_flat >= lay.offsets[-1] + lay.numels[-1]


def test_flag_policies():
    tiny = layouts.get_layout("tiny_cnn")
    assert np.all(tiny.flags == layouts.LAYER_SCALE | layouts.LAYER_DECAY)
    r50 = layouts.get_layout("resnet50")
    one_d = np.array([len(t.shape) == 1 for t in r50.tensors])
    assert np.all(r50.flags[one_d] == 0)
    assert np.all(r50.flags[~one_d] == layouts.LAYER_SCALE | layouts.LAYER_DECAY)
    vgg = layouts.get_layout("vgg16")
    fc6 = [i for i, t in enumerate(vgg.tensors) if t.name == "classifier.0.weight"][0]
    assert vgg.numels[fc6] == 102_760_448


def test_bf16_round_to_nearest_even_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100_000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 100_000),
                        np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -1 - 2 ** -8, 0.0, -0.0], np.float32)])
    ours = synth.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    assert ours[-6] == 0x3F80 and ours[-5] == 0x3F80 and ours[-4] == 0x3F82
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(ours),
                                  torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_generator_is_deterministic_and_keyed():
    lay = layouts.get_layout("tiny_cnn")
    a = synth.replica_grads(lay, 4, 0, 0)
    b = synth.replica_grads(lay, 4, 0, 0, threads=1)
    np.testing.assert_array_equal(a, b)
    c = synth.replica_grads(lay, 4, 1, 0)
    assert not np.array_equal(a, c)
    # replica k of a K=4 draw equals replica k of a K=2 draw: streams are keyed
    d = synth.replica_grads(lay, 2, 0, 0)
    np.testing.assert_array_equal(a[:2], d)
    # bf16 draw is the RNE rounding of the fp32 draw
    e = synth.replica_grads(lay, 4, 0, 0, dtype="bf16")
    np.testing.assert_array_equal(e, synth.to_bf16_bits(a))
    # padding is zero
    mask = np.ones(lay.n_flat, bool)
    for o, n, _ in lay.table():
        mask[o:o + n] = False
    assert np.all(a[:, mask] == 0)


def test_generator_statistics_and_init():
    lay = layouts.get_layout("resnet18_cifar")
    sig = synth.layer_sigmas(lay, 0)
    assert np.all((sig >= 1e-4) & (sig <= 1e-1))
    w = synth.init_weights(lay, 0)
    for l, t in enumerate(lay.tensors):
        o, n = int(lay.offsets[l]), int(lay.numels[l])
        x = w[o:o + n].astype(np.float64)
        if t.kind in ("conv", "fc") and n >= 10_000:
            assert abs(x.std() / np.sqrt(2.0 / t.fan_in) - 1) < 6 / np.sqrt(n)
        elif t.kind == "bn_weight":
            assert np.all(x == 1.0)
        elif t.kind == "bn_bias":
            assert np.all(x == 0.0)
        elif t.kind == "bias":
            assert np.all(np.abs(x) <= 1 / np.sqrt(t.fan_in))
    wp = synth.init_weights(lay, 0, perturb_bn=True)
    bn = [l for l, t in enumerate(lay.tensors) if t.kind == "bn_weight"][0]
    o, n = int(lay.offsets[bn]), int(lay.numels[bn])
    assert not np.all(wp[o:o + n] == 1.0)
