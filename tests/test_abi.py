"""libags C-ABI on the host: exports and argument validation (no GPU).

Only calls that fail host-side validation (which runs before any HIP call)
are made here; nothing is launched.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2603_18112_amd import _build, ags, layouts, plan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_build.LIB):
        _build.build()
    return ags.load_library()


def header_functions(name=None):
    names = [name] if name else sorted(os.listdir(os.path.join(ROOT, "include")))
    out = set()
    for h in names:
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        out |= set(re.findall(r"\b(ags_[a-z_]+)\s*\(", text))
    return sorted(out)


def test_header_declares_the_binding_names():
    assert header_functions("ags.h") == sorted(ags.EXPORTS)
    assert header_functions("ags_plan.h") == sorted(plan.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", _build.LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (ags_\w+)$", out, flags=re.M))
    for name in header_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_struct_sizes_match_the_header():
    # Sizes follow from the field lists in include/ags.h on x86-64.
    assert ctypes.sizeof(ags.ags_layer) == 24
    assert ctypes.sizeof(ags.ags_layer_stats) == 9 * 8 + 4 + 4
    assert ctypes.sizeof(plan.ags_plan_sample) == 24
    assert ctypes.sizeof(plan.ags_plan_model) == 4 + 4 + 4 * 8 + 4 + 4
    assert ctypes.sizeof(plan.ags_plan_candidate) == 16
    assert ctypes.sizeof(ags.ags_global_stats) == 40
    # ... static_scale, elementwise, delta_scope, reuse_w_norms and the tail padding
    assert ctypes.sizeof(ags.ags_config) == (4 + 4 + 8 + 8 + 4 + 4 + 4 + 4 + 7 * 8 + 4 + 4 + 8 + 4 + 4
                                             + 4 + 4)


def test_status_strings(lib):
    for s in range(7):
        assert ags.ags_status_string(s).startswith(ags.STATUS_NAMES[s])


def _table():
    return [(0, 100, 3), (104, 16, 0), (120, 9, 1)]


def _ws(layers=None, n_flat=136, K=4, **kw):
    cfg = ags.make_config(_table() if layers is None else layers, n_flat, K, **kw)
    try:
        return ags.AGS_OK, ags.ags_workspace_bytes(cfg)
    except ags.AGSError as e:
        return e.status, str(e)


def test_valid_config_workspace_size(lib):
    st, n = _ws()
    assert st == ags.AGS_OK and n > 0
    # ResNet-50, K = 16 bf16.  AGS and SGD steps update w and m in the
    # statistics pass, so the workspace is only per-tile and per-layer tables.
    lay = layouts.get_layout("resnet50")
    for mode in ("ags", "sgd"):
        cfg = ags.make_config(lay.table(), lay.n_flat, 16, grad_dtype="bf16", mode=mode)
        assert ags.ags_workspace_bytes(cfg) < 2_000_000
    # A LARS step needs its layer norms before the update: it keeps the
    # replica mean (fp32, one per element) between its two passes ...
    cfg = ags.make_config(lay.table(), lay.n_flat, 16, grad_dtype="bf16", mode="lars")
    n = ags.ags_workspace_bytes(cfg)
    assert lay.n_flat * 4 <= n < lay.n_flat * 4 + 2_000_000
    # ... unless re-reading the replicas is as cheap (K = 4 bf16: 8 bytes).
    cfg = ags.make_config(lay.table(), lay.n_flat, 4, grad_dtype="bf16", mode="lars")
    assert ags.ags_workspace_bytes(cfg) < 2_000_000
    # Carried weight norms: one fp32 per tile of 2048 elements.
    cfg2 = ags.make_config(lay.table(), lay.n_flat, 4, grad_dtype="bf16", mode="lars",
                           reuse_w_norms=True)
    assert 12_560 * 4 <= ags.ags_workspace_bytes(cfg2) - ags.ags_workspace_bytes(cfg) < 12_560 * 4 + 512
    # Element scales: two fp32 buffers of n_flat (the scales in force and the
    # refreshed ones) plus a per-tile sum.
    cfg = ags.make_config(lay.table(), lay.n_flat, 16, grad_dtype="bf16", elementwise=True)
    n = ags.ags_workspace_bytes(cfg)
    assert 2 * lay.n_flat * 4 <= n < 2 * lay.n_flat * 4 + 2_000_000


@pytest.mark.parametrize("kw,status", [
    (dict(layers=[]), ags.AGS_E_LAYOUT),
    (dict(layers=[(0, 0, 3)]), ags.AGS_E_LAYOUT),
    (dict(layers=[(-8, 10, 3)]), ags.AGS_E_LAYOUT),
    (dict(layers=[(4, 10, 3)]), ags.AGS_E_ALIGN),
    (dict(layers=[(0, 100, 3), (96, 8, 3)]), ags.AGS_E_LAYOUT),   # overlap
    (dict(layers=[(104, 8, 3), (0, 8, 3)]), ags.AGS_E_LAYOUT),    # out of order
    (dict(layers=[(128, 9, 3)]), ags.AGS_E_LAYOUT),               # past n_flat
    (dict(layers=[(0, 8, 4)]), ags.AGS_E_ARG),                    # unknown flag
    (dict(n_flat=0), ags.AGS_E_LAYOUT),
    (dict(K=0), ags.AGS_E_ARG),
    (dict(K=ags.AGS_MAX_K + 1, small_replica=0), ags.AGS_E_ARG),
    (dict(momentum=1.0), ags.AGS_E_ARG),
    (dict(momentum=-0.1), ags.AGS_E_ARG),
    (dict(lr=float("nan")), ags.AGS_E_ARG),
    (dict(lr=-1.0), ags.AGS_E_ARG),
    (dict(weight_decay=-1e-4), ags.AGS_E_ARG),
    (dict(delta=float("inf")), ags.AGS_E_ARG),
    (dict(eps=-1e-8), ags.AGS_E_ARG),
    (dict(s_max=float("nan")), ags.AGS_E_ARG),
    (dict(mode="lars", trust_coef=0.0), ags.AGS_E_ARG),
    (dict(mode="static", static_scale=0.0), ags.AGS_E_ARG),
    (dict(mode="static", static_scale=float("inf")), ags.AGS_E_ARG),
    (dict(refresh_every=-1), ags.AGS_E_ARG),
    (dict(small_replica=4), ags.AGS_E_ARG),
    (dict(small_replica=-2), ags.AGS_E_ARG),
    (dict(mode="sgd", elementwise=True), ags.AGS_E_ARG),     # element scales: AGS only
    (dict(mode="lars", elementwise=True), ags.AGS_E_ARG),
    (dict(mode="static", elementwise=True), ags.AGS_E_ARG),
    (dict(mode="ags", reuse_w_norms=True), ags.AGS_E_ARG),    # carried weight norms: LARS only
    (dict(mode="sgd", reuse_w_norms=True), ags.AGS_E_ARG),
])
def test_config_validation(lib, kw, status):
    st, msg = _ws(**kw)
    assert st == status, msg
    assert ags.ags_last_error(None)


def test_launch_size_limit(lib):
    # 4e10 elements in one layer: 19.5M tiles of 2048, 5.0e9 work-items in
    # the step kernel launch, more than one launch holds.
    n = 40_000_000_000
    st, msg = _ws(layers=[(0, n, 3)], n_flat=n)
    assert st == ags.AGS_E_LAYOUT and "2^32" in msg
    # 1.6e10 elements fit (7.8M tiles, 2.0e9 work-items)
    st, _ = _ws(layers=[(0, 16_000_000_000, 3)], n_flat=16_000_000_000)
    assert st == ags.AGS_OK


def test_bad_enum_values(lib):
    cfg = ags.make_config(_table(), 136, 4)
    cfg.mode = 7
    with pytest.raises(ags.AGSError) as e:
        ags.ags_workspace_bytes(cfg)
    assert e.value.status == ags.AGS_E_ARG
    cfg = ags.make_config(_table(), 136, 4)
    cfg.grad_dtype = 2
    with pytest.raises(ags.AGSError) as e:
        ags.ags_workspace_bytes(cfg)
    assert e.value.status == ags.AGS_E_ARG


def test_bad_elementwise_and_delta_scope_fields(lib):
    for field, value in (("elementwise", 2), ("elementwise", -1), ("delta_scope", 2),
                         ("delta_scope", -1), ("reuse_w_norms", 2), ("reuse_w_norms", -1)):
        cfg = ags.make_config(_table(), 136, 4, mode="lars")
        setattr(cfg, field, value)
        with pytest.raises(ags.AGSError) as e:
            ags.ags_workspace_bytes(cfg)
        assert e.value.status == ags.AGS_E_ARG, field


def test_init_rejects_null_and_misaligned_pointers_before_any_device_call(lib):
    cfg = ags.make_config(_table(), 136, 4)
    with pytest.raises(ags.AGSError) as e:
        ags.ags_init(cfg, 0, 0x10000)
    assert e.value.status == ags.AGS_E_ARG
    with pytest.raises(ags.AGSError) as e:
        ags.ags_init(cfg, 0x10008, 0x20000)
    assert e.value.status == ags.AGS_E_ALIGN
    h = ctypes.c_void_p(0)
    assert lib.ags_init(ctypes.byref(cfg), 0x10000, 0x20000, None, None) == ags.AGS_E_ARG
    assert h.value is None


def test_init_rejects_overlapping_w_and_m_before_any_device_call(lib):
    cfg = ags.make_config(_table(), 136, 4)        # 544 bytes each
    for w, m in ((0x10000, 0x10000), (0x10000, 0x10000 + 528), (0x10210, 0x10000)):
        with pytest.raises(ags.AGSError) as e:
            ags.ags_init(cfg, w, m)
        assert e.value.status == ags.AGS_E_ARG and "overlap" in str(e.value)


def test_workspace_cap_gives_nomem_before_any_device_call(lib, monkeypatch):
    # The paper's runtime falls back to a smaller batch on out-of-memory; the
    # library reports AGS_E_NOMEM cleanly so a caller can do the same.
    lay = layouts.get_layout("resnet50")
    cfg = ags.make_config(lay.table(), lay.n_flat, 64, grad_dtype="bf16")
    need = ags.ags_workspace_bytes(cfg)
    monkeypatch.setenv("AGS_MAX_WORKSPACE_BYTES", str(need - 1))
    with pytest.raises(ags.AGSError) as e:
        ags.ags_init(cfg, 0x1000000000, 0x2000000000)     # disjoint (fake) w and m
    assert e.value.status == ags.AGS_E_NOMEM
    assert "AGS_MAX_WORKSPACE_BYTES" in str(e.value)


def test_null_handle_calls_are_errors(lib):
    assert lib.ags_step(None, None, 0, None) == ags.AGS_E_ARG
    assert lib.ags_stats(None, None, 0, None) == ags.AGS_E_ARG
    assert lib.ags_read_stats(None, None, None) == ags.AGS_E_ARG
    assert lib.ags_set_lr(None, 0.1) == ags.AGS_E_ARG
    assert lib.ags_set_profiling(None, 1) == ags.AGS_E_ARG
    assert lib.ags_get_elementwise_scale(None, None, 0) == ags.AGS_E_ARG
    assert lib.ags_get_layer_state(None, None) == ags.AGS_E_ARG
    assert lib.ags_set_layer_state(None, None) == ags.AGS_E_ARG
    assert lib.ags_get_last_decision(None, None, None) == ags.AGS_E_ARG
    assert lib.ags_set_last_decision(None, 0, None) == ags.AGS_E_ARG
    assert lib.ags_set_elementwise_scale(None, None, 0) == ags.AGS_E_ARG
    assert lib.ags_invalidate_weight_norms(None) == ags.AGS_E_ARG
    lib.ags_destroy(None)


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(ImportError):
        ags.load_library.__wrapped__(str(tmp_path / "nope.so")) if hasattr(
            ags.load_library, "__wrapped__") else _load_fresh(str(tmp_path / "nope.so"))


def _load_fresh(path):
    saved = ags._lib
    ags._lib = None
    try:
        return ags.load_library(path)
    finally:
        ags._lib = saved


def test_noalloc_stats_rejects_before_any_device_call(lib):
    """ags_stats_noalloc checks its arguments, and that its tables fit the
    library's scratch array, on the host before any HIP call."""
    cfg = ags.make_config(_table(), 136, 4)
    out_l = (ags.ags_layer_stats * 3)()
    out_g = ags.ags_global_stats()
    f = lib.ags_stats_noalloc
    assert f(ctypes.byref(cfg), None, 0x2000000000, 136, out_l, ctypes.byref(out_g), None) == ags.AGS_E_ARG
    assert f(ctypes.byref(cfg), 0x1000000000, 0x2000000000, 136, None, ctypes.byref(out_g),
             None) == ags.AGS_E_ARG
    assert f(ctypes.byref(cfg), 0x1000000004, 0x2000000000, 136, out_l, ctypes.byref(out_g),
             None) == ags.AGS_E_ALIGN
    assert f(ctypes.byref(cfg), 0x1000000000, 0x2000000000, 100, out_l, ctypes.byref(out_g),
             None) == ags.AGS_E_ARG
    assert f(ctypes.byref(cfg), 0x1000000000, 0x1000000000, 136, out_l, ctypes.byref(out_g),
             None) == ags.AGS_E_ARG                        # the replicas overlap w
    # 5e8 parameters: 244k tiles of 2048 at 32 bytes each, more than the 6 MiB
    # array holds
    n = 500_000_000
    big = ags.make_config([(0, n, 3)], n, 1)
    st = f(ctypes.byref(big), 0x1000000000, 0x2000000000, n, out_l, ctypes.byref(out_g), None)
    assert st == ags.AGS_E_NOMEM
    assert "scratch" in ags.ags_last_error(None)
    # VGG-16 (138M parameters, 67,569 tiles) fits
    lay = layouts.get_layout("vgg16")
    ok = ags.make_config(lay.table(), lay.n_flat, 8)
    st = f(ctypes.byref(ok), 0x1000000000, 0x1000000000 + 8 * lay.n_flat, lay.n_flat, out_l,
           ctypes.byref(out_g), None)
    assert st != ags.AGS_E_NOMEM                           # fails later, at the device checks
