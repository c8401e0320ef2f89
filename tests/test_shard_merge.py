"""The sharded design checked on the CPU (no ranks, no collectives).

One GPU here runs the whole step.  Across G GPUs the path would shard as
follows: rank q holds K/G of the
replica gradients; it sums its replicas per element and, per layer, their
squared norms sum_k ||g_k,l||^2 (and ||g_r,l||^2 where it holds the small-batch
replica r); a reduce-scatter leaves rank q the replica sum, hence gbar, on a
contiguous tile-aligned 1/G of the flat buffer, on which it forms the
partials of W_l and G_l; one all-reduce of an [L][4] fp64 vector gives every
rank every layer's W, G, sum of replica norms and S; each rank takes the
same decision from the same numbers, forms V_l = (1/K) sum_k ||g_k,l||^2 - G_l
and updates its shard of w and m.

This test writes those steps out in float64 numpy, emulating the ranks one
after another, and checks them against the float64 oracle's unsharded step:
W, G, S and the updated w, m agree to rounding; V, formed by a difference,
agrees to a bound set by its cancellation, and within the statistics
tolerance (1e-4) even when the per-rank partial sums are accumulated per
tile in fp32 as the GPU kernels do.
"""
import math

import numpy as np
import pytest

from oracle import OracleAGS
from paper_2603_18112_amd import layouts, synth

SD = layouts.LAYER_SCALE | layouts.LAYER_DECAY
TILE = 2048
EPS32 = 2.0 ** -24


def _layout():
    # layers that straddle shard boundaries, tiny and ragged ones, mixed flags
    sizes = [7, 4100, 9000, 1, 20003, 63, 2048, 12001, 300, 5]
    flags = [SD, SD, layouts.LAYER_SCALE, 0, SD, layouts.LAYER_DECAY, SD, SD, 0, SD]
    return layouts.custom_layout(sizes, flags, pad=8)


def _shard_ranges(n_flat, G):
    """Contiguous, tile-aligned element ranges of the flat buffer, one per rank."""
    n_tiles = -(-n_flat // TILE)
    bounds = [min(n_flat, (n_tiles * q // G) * TILE) for q in range(G + 1)]
    bounds[-1] = n_flat
    return [(bounds[q], bounds[q + 1]) for q in range(G)]


def _layer_of(table, n_flat):
    lid = np.full(n_flat, -1)
    for l, (o, n, _) in enumerate(table):
        lid[o:o + n] = l
    return lid


def _sum(x, fp32_tiles):
    """Sum of x: in float64, or (as the kernels do) per 2048-element tile in
    float32 and then the tiles in float64."""
    if not fp32_tiles:
        return float(np.sum(x, dtype=np.float64))
    x = np.asarray(x, dtype=np.float32)
    return float(sum(float(np.sum(x[i:i + TILE], dtype=np.float32)) for i in range(0, x.size, TILE)))


def sharded_stats(table, n_flat, g, w, G, r, fp32_tiles=False):
    """Per-layer W, G, V, S of one step, merged from G ranks."""
    K = g.shape[0]
    assert K % G == 0
    L = len(table)
    lid = _layer_of(table, n_flat)
    kl = K // G
    # per rank: local replica sums per element, local per-layer sums of ||g_k||^2 and S
    local_sum = np.zeros((G, n_flat))
    part = np.zeros((G, L, 4))          # W, G, sum_k ||g_k||^2, S
    for q in range(G):
        ks = range(q * kl, (q + 1) * kl)
        local_sum[q] = np.sum(g[list(ks)], axis=0)
        for l, (o, n, _) in enumerate(table):
            part[q, l, 2] = sum(_sum(g[k, o:o + n] ** 2, fp32_tiles) for k in ks)
            if r in ks:
                part[q, l, 3] = _sum(g[r, o:o + n] ** 2, fp32_tiles)
    # reduce-scatter: rank q receives the replica sum on its shard, in rank order
    gbar = np.zeros(n_flat)
    for q, (a, b) in enumerate(_shard_ranges(n_flat, G)):
        tot = np.zeros(b - a)
        for p in range(G):
            tot = tot + local_sum[p, a:b]
        gbar[a:b] = tot / K
        for l in range(L):
            sel = lid[a:b] == l
            if np.any(sel):
                part[q, l, 0] += _sum(w[a:b][sel] ** 2, fp32_tiles)
                part[q, l, 1] += _sum(gbar[a:b][sel] ** 2, fp32_tiles)
    # all-reduce of the [L][4] vector (rank order)
    merged = np.zeros((L, 4))
    for q in range(G):
        merged += part[q]
    W, Gl, sq, S = merged.T
    V = sq / K - Gl
    return W, Gl, V, S, gbar, sq / K


def _inputs(lay, K, noise, seed=3):
    sig = synth.layer_sigmas(lay, seed)
    g32 = synth.replica_grads(lay, K, 0, seed, noise=noise, sigmas=sig)
    w32 = synth.init_weights(lay, seed)
    return g32, w32


@pytest.mark.parametrize("G,K,r", [(2, 4, 0), (4, 8, 5), (8, 16, 15)])
@pytest.mark.parametrize("noise", [0.1, 0.5, 2.0])
def test_merged_statistics_equal_the_unsharded_ones(G, K, r, noise):
    lay = _layout()
    table = lay.table()
    g32, w32 = _inputs(lay, K, noise)
    g, w = g32.astype(np.float64), w32.astype(np.float64)
    ora = OracleAGS(table, lay.n_flat, K, w32, small_replica=r)
    st, _ = ora.stats(g32)
    W, Gl, V, S, _, msq = sharded_stats(table, lay.n_flat, g, w, G, r)
    np.testing.assert_allclose(W, st["w_sq"], rtol=1e-13)
    np.testing.assert_allclose(Gl, st["g_sq"], rtol=1e-13)
    np.testing.assert_allclose(S, st["gsmall_sq"], rtol=1e-13)
    # V is a difference: its error is relative to the mean replica norm (the
    # two sides sum up to n K terms in different orders)
    err = np.abs(V - st["var"])
    assert np.all(err <= 1e-12 * msq), (err / msq).max()
    nz = st["var"] > 0
    assert np.all(err[nz] / st["var"][nz] < 1e-10)


@pytest.mark.parametrize("G,K", [(2, 8), (8, 16)])
@pytest.mark.parametrize("noise", [0.1, 0.5])
def test_merged_spread_with_fp32_tile_sums_stays_within_the_statistics_tolerance(G, K, noise):
    """With per-tile fp32 sums, V = mean_k ||g_k||^2 - G loses digits when the
    noise is small (rho = V / G down to ~0.01 here): its error is about
    eps32 * (1 + 1/rho) relative, still under the 1e-4 of the statistics."""
    lay = _layout()
    table = lay.table()
    g32, w32 = _inputs(lay, K, noise)
    g = g32.astype(np.float64)
    st, _ = OracleAGS(table, lay.n_flat, K, w32).stats(g32)
    _, Gl, V, _, _, msq = sharded_stats(table, lay.n_flat, g, w32.astype(np.float64), G, 0,
                                        fp32_tiles=True)
    rho = st["var"] / st["g_sq"]
    rel = np.abs(V - st["var"]) / st["var"]
    bound = 64 * EPS32 * (1.0 + 1.0 / rho)
    assert np.all(rel <= bound), (rel / bound).max()
    assert np.all(rel < 1e-4), rel.max()
    if noise == 0.1:
        assert rho.min() < 0.02      # the low-noise case is exercised


@pytest.mark.parametrize("G", [2, 4])
def test_sharded_step_reassembles_the_unsharded_update(G):
    """Every rank decides from the same merged numbers; the shards of w and m
    updated with the coefficients of their layers reassemble the oracle's."""
    lay = _layout()
    table = lay.table()
    K, hyper = 8, dict(lr=0.1, momentum=0.9, weight_decay=5e-4, eps=1e-8, delta=0.5)
    g_steps = [_inputs(lay, K, 0.5, seed=s)[0] for s in (3, 3, 4)]
    g_steps[2] = (g_steps[2] * np.float32(3.0)).astype(np.float32)   # a sensitive step
    w0 = _inputs(lay, K, 0.5)[1]
    ora = OracleAGS(table, lay.n_flat, K, w0, **hyper)
    w, m = w0.astype(np.float64), np.zeros(lay.n_flat)
    gradscale = np.ones(len(table))
    g_prev = 0.0
    lid = _layer_of(table, lay.n_flat)
    flags = np.array([f for _, _, f in table])
    for t, g32 in enumerate(g_steps, start=1):
        ost, oglob = ora.step(g32)
        W, Gl, V, S, gbar, _ = sharded_stats(table, lay.n_flat, g32.astype(np.float64), w, G, 0)
        Gtot = float(np.sum(Gl))
        delta = math.inf if t == 1 or g_prev <= 0 else abs(Gtot - g_prev) / g_prev
        sens = not (delta < hyper["delta"])
        assert sens == bool(oglob["sensitive"])
        scaled = (flags & layouts.LAYER_SCALE) != 0
        a = np.where(scaled & (not sens), gradscale, 1.0)
        b = np.where((flags & layouts.LAYER_DECAY) != 0, hyper["weight_decay"], 0.0)
        np.testing.assert_allclose(a, ost["coef_a"], rtol=1e-13)
        for q, (lo, hi) in enumerate(_shard_ranges(lay.n_flat, G)):
            sl = slice(lo, hi)
            ll = lid[sl]
            inl = ll >= 0
            d = np.where(inl, a[ll] * gbar[sl] + b[ll] * w[sl], 0.0)
            m[sl] = np.where(inl, hyper["momentum"] * m[sl] + d, m[sl])
            w[sl] = np.where(inl, w[sl] - hyper["lr"] * m[sl], w[sl])
        # UpdateGradScale from the merged statistics (refresh every step)
        ok = (S > 0) & (Gl > 0)
        new = np.where(ok, np.sqrt(S) / (np.sqrt(Gl) + hyper["eps"]), 1.0)
        gradscale = np.where(scaled, np.minimum(new, math.sqrt(K)), gradscale)
        np.testing.assert_allclose(gradscale, ost["gradscale"], rtol=1e-12)
        g_prev = Gtot
        for l, (o, n, _) in enumerate(table):
            np.testing.assert_allclose(w[o:o + n], ora.w[o:o + n], rtol=1e-12, atol=1e-15)
            np.testing.assert_allclose(m[o:o + n], ora.m[o:o + n], rtol=1e-12, atol=1e-15)


def test_shards_are_tile_aligned_and_cover_the_buffer():
    lay = _layout()
    for G in (1, 2, 3, 4, 8):
        rs = _shard_ranges(lay.n_flat, G)
        assert rs[0][0] == 0 and rs[-1][1] == lay.n_flat
        for (a, b), (c, _) in zip(rs, rs[1:]):
            assert b == c and a % TILE == 0 and b % TILE == 0
    # some layer straddles a shard boundary for G = 4
    bounds = {b for _, b in _shard_ranges(lay.n_flat, 4)[:-1]}
    assert any(o < x < o + n for o, n, _ in lay.table() for x in bounds)
