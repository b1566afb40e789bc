"""Host-side tests of the C ABI (no GPU needed): the library loads, exports
every entry point ``include/lionmuon.h`` declares, rejects invalid calls
before touching the device, and plans the work of Algorithm 1 as expected."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads
from paper_2605_19811_amd import lionmuon as lm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lionmuon.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lm.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return lm.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lionmuon_\w+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(lm.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert lib.lionmuon_abi_version() == 3


def test_status_strings(lib):
    for code, name in [(0, "LM_OK"), (1, "LM_ERR_INVALID_ARGUMENT"), (2, "LM_ERR_UNSUPPORTED"),
                       (3, "LM_ERR_OUT_OF_MEMORY"), (4, "LM_ERR_WORKSPACE_TOO_SMALL"),
                       (5, "LM_ERR_HIP")]:
        assert lib.lionmuon_status_string(code).decode() == name


def test_config_schedule_fields(lib):
    cfg = lm.config(ns_schedule=[(3.4445, -4.775, 2.0315)] * 3 + [(1.5, -0.5, 0.0)] * 2)
    assert cfg.ns_steps == 5 and cfg.ns_schedule_steps == 5
    assert tuple(cfg.ns_schedule[4]) == (1.5, -0.5, 0.0)
    with pytest.raises(ValueError):
        lm.config(ns_schedule=[(1.0, 0.0)])
    bad = lm.config(ns_schedule=[(1.5, -0.5, 0.0)] * 2)
    bad.ns_schedule[1][2] = float("nan")
    with pytest.raises(lm.LionMuonError):
        lm.lionmuon_workspace_bytes([(8, 8, False)], bad)


def test_config_defaults(lib):
    cfg = lm.lm_config()
    lib.lionmuon_config_default(ctypes.byref(cfg))
    assert cfg.struct_size == ctypes.sizeof(lm.lm_config)
    assert cfg.ns_steps == 5
    assert (cfg.ns_a, cfg.ns_b, cfg.ns_c) == (3.4445, -4.7750, 2.0315)
    assert cfg.ns_eps == 1e-7 and cfg.ns_bf16_min_side == 64 and cfg.reserved == 0
    assert cfg.ns_precision == lm.LM_NS_BF16 and cfg.ns_scale_mode == lm.LM_NS_SCALE_NONE


# --------------------------------------------------------------------------
# plan info: the work one step enqueues
# --------------------------------------------------------------------------
def _specs(wl):
    return [(t.rows, t.cols, t.lion_only) for t in wl.tensors]


def _ns_flops(wl, k=5):
    sym = dense = 0.0
    for t in wl.tensors:
        if t.lion_only or t.rows == 1:
            continue
        s, l = min(t.rows, t.cols), max(t.rows, t.cols)
        # Gram (symmetric, s(s+1)/2 dot products of length l, 2 flops each),
        # A^2 (symmetric, s(s+1)/2 dot products of length s), B X (s*l of length s)
        sym += 2 * (s * (s + 1) // 2) * l + 2 * (s * (s + 1) // 2) * s + 2 * s * s * l
        dense += 2 * s * s * l + 2 * s * s * s + 2 * s * s * l
    return k * sym, k * dense


@pytest.mark.parametrize("name,classes,n_muon,tflops", [
    ("gpt2-124m", 3, 48, 1.088), ("gpt2-355m", 3, 96, 5.156), ("gpt2-720m", 3, 144, 15.104)])
def test_plan_info_muon_step(lib, name, classes, n_muon, tflops):
    wl = workloads.get(name)
    info = lm.lionmuon_plan_info(_specs(wl), t=2, P=2)
    assert info["n_muon"] == n_muon
    assert info["n_shape_classes"] == classes
    assert info["muon_elements"] == wl.matrix_numel
    assert info["n_lion"] == len(wl.tensors) - n_muon
    assert info["lion_elements"] == wl.numel - wl.matrix_numel
    sym, dense = _ns_flops(wl)
    assert info["ns_flops"] == pytest.approx(sym, rel=1e-12)
    assert info["ns_flops_dense"] == pytest.approx(dense, rel=1e-12)
    assert info["ns_flops"] / 1e12 == pytest.approx(tflops, abs=5e-4)
    # workspace: 2 s_pad*l_pad (X ping-pong) + 2 s_pad^2 (A, B) bf16 per matrix
    ws = 0
    for t in wl.tensors:
        if t.lion_only or t.rows == 1:
            continue
        s, l = min(t.rows, t.cols), max(t.rows, t.cols)
        sp, lp = -(-s // 128) * 128, -(-l // 128) * 128
        ws += 2 * (2 * sp * lp + 2 * sp * sp)
    assert ws <= info["workspace_bytes"] < ws + 8 << 20


def test_plan_info_lion_step_and_pure_lion(lib):
    wl = workloads.gpt2_124m()
    for t, P in [(1, 2), (3, 2), (0, 0), (5, 0), (7, 4)]:
        info = lm.lionmuon_plan_info(_specs(wl), t=t, P=P)
        assert info["n_muon"] == 0 and info["n_lion"] == 48
        assert info["lion_bytes"] == 20.0 * wl.numel
        assert info["ns_flops"] == 0.0
    info = lm.lionmuon_plan_info(_specs(wl), t=7, P=1)
    assert info["n_muon"] == 48


def test_plan_info_vectors_and_lion_only_never_muon(lib):
    specs = [(1, 1000, False), (500, 1, False), (64, 64, True), (64, 96, False), (0, 5, False)]
    info = lm.lionmuon_plan_info(specs, t=0, P=1)
    assert info["n_tensors"] == 4            # the empty tensor is skipped
    assert info["n_muon"] == 1 and info["n_lion"] == 3
    # 64 x 96 runs bf16 (short side >= 64): padded to 256; the symmetric stages
    # use 128-tiles (too few 256-tiles), apply one 256-tile
    assert info["gram_tiles"] == 3 and info["poly_tiles"] == 3 and info["apply_tiles"] == 1
    # fp32 (short side below 65): padded to 128; too few 128-tiles to give
    # every CU one, so 64-tiles: 2 x 2 (lower triangle 3), apply 2 x 2
    info = lm.lionmuon_plan_info(specs, t=0, P=1, cfg=lm.config(ns_bf16_min_side=65))
    assert info["gram_tiles"] == 3 and info["poly_tiles"] == 3 and info["apply_tiles"] == 4


def test_plan_info_tiles_span_ragged_shapes(lib):
    specs = [(300, 520, False), (520, 300, False)]
    # fp32: padded to 128 (384 x 640); 12 lower 128-tiles and 30 apply ones
    # would leave most CUs idle, so 64-tiles: s -> 6, l -> 10; lower
    # triangle 21, apply 60, per matrix
    info = lm.lionmuon_plan_info(specs, t=0, P=1, cfg=lm.config(ns_precision="fp32"))
    assert info["n_shape_classes"] == 1
    assert info["gram_tiles"] == 42 and info["poly_tiles"] == 42 and info["apply_tiles"] == 120
    # bf16: padded to 256 (512 x 768); symmetric stages on 128-tiles (4 -> 10
    # lower), apply on 256-tiles (2 x 3)
    info = lm.lionmuon_plan_info(specs, t=0, P=1)
    assert info["gram_tiles"] == 20 and info["poly_tiles"] == 20 and info["apply_tiles"] == 12


# apply: 256-tiles; a last round of at most 128 of them (of 256 CUs) runs as
# sixteen 64-tiles each when those fit one round, else four 128-tiles each:
# 124M 1296 = 5 x 256 + 16 (16 x 16 = 256 64-tiles), 720M 10800 = 42 x 256 + 48
# Gram / polynomial: 256-tiles unless 128-tiles are estimated to finish
# sooner. At 124M the Gram (K = l up to 3072) keeps 256-tiles (288 of them,
# the longest first), the polynomial (K = 768) takes 128-tiles: 288 short
# 256-tiles would leave a second round 12% full.
@pytest.mark.parametrize("name,gram_tiles,poly_tiles,apply_tiles", [
    ("gpt2-124m", 48 * 6, 48 * 21, 1280 + 16 * 16),
    ("gpt2-355m", 96 * 10, 96 * 10, 24 * 48 + 24 * 16 + 48 * 64),   # 4608 = 18 x 256: no tail
    ("gpt2-720m", 144 * 15, 144 * 15, 10752 + 4 * 48)])
def test_plan_tile_choice_for_benchmark_sets(lib, name, gram_tiles, poly_tiles, apply_tiles):
    info = lm.lionmuon_plan_info(_specs(workloads.get(name)), t=0, P=1)
    assert info["gram_tiles"] == gram_tiles and info["poly_tiles"] == poly_tiles
    assert info["apply_tiles"] == apply_tiles


def test_plan_fp32_tile_choice(lib):
    """fp32 products run on 64-tiles when their 128-tiles would not give
    every one of the 256 CUs one, else on 128-tiles."""
    fp32 = lm.config(ns_precision="fp32")
    info = lm.lionmuon_plan_info([(768, 768, False)], t=0, P=1, cfg=fp32)
    assert (info["gram_tiles"], info["poly_tiles"], info["apply_tiles"]) == (78, 78, 144)
    info = lm.lionmuon_plan_info(_specs(workloads.get("gpt2-124m")), t=0, P=1, cfg=fp32)
    assert (info["gram_tiles"], info["poly_tiles"]) == (48 * 21, 48 * 21)
    assert info["apply_tiles"] == 12 * 6 * (18 + 6 + 24 + 24)


def test_workspace_bytes_matches_plan_info(lib):
    specs = _specs(workloads.gpt2_124m())
    ws = lm.lionmuon_workspace_bytes(specs)
    assert ws == lm.lionmuon_plan_info(specs, t=0, P=1)["workspace_bytes"]
    ws32 = lm.lionmuon_workspace_bytes(specs, lm.config(ns_precision="fp32"))
    assert 1.9 * ws < ws32 < 2.1 * ws


def test_plan_info_rejects_bad_arguments(lib):
    with pytest.raises(lm.LionMuonError) as e:
        lm.lionmuon_plan_info([(-1, 5, False)], t=0, P=1)
    assert e.value.status == lm.LM_ERR_INVALID_ARGUMENT
    with pytest.raises(lm.LionMuonError):
        lm.lionmuon_plan_info([(5, 5, False)], t=-1, P=1)
    with pytest.raises(lm.LionMuonError) as e:
        lm.lionmuon_plan_info([(40000, 40000, False)], t=0, P=1)
    assert e.value.status == lm.LM_ERR_UNSUPPORTED


# --------------------------------------------------------------------------
# validation: every error path returns before any device work
# --------------------------------------------------------------------------
class FakeList:
    """Pointer arrays with fake (never dereferenced) device addresses."""

    def __init__(self, shapes, addrs=None):
        n = len(shapes)
        self.n = n
        if addrs is None:
            addrs, a = [], 1 << 32
            for r, c, _ in shapes:
                b = max(r * c * 4, 16)
                addrs.append((a, a + b + 256, a + 2 * (b + 256)))
                a += 3 * (b + 256) + 4096
        self.p = (ctypes.c_void_p * max(n, 1))(*[x[0] for x in addrs])
        self.g = (ctypes.c_void_p * max(n, 1))(*[x[1] for x in addrs])
        self.m = (ctypes.c_void_p * max(n, 1))(*[x[2] for x in addrs])
        self.shapes = lm.shapes_array(shapes)


def _step(lib, fl, t=1, P=2, b1=0.9, b2=0.99, lr=0.01, wd=0.1):
    return lib.lionmuon_step(ctypes.cast(fl.p, ctypes.c_void_p), ctypes.cast(fl.g, ctypes.c_void_p),
                             ctypes.cast(fl.m, ctypes.c_void_p), fl.shapes, fl.n, t, P, b1, b2, lr,
                             wd, None)


def _step_ex(lib, fl, cfg, ws=None, ws_bytes=0, t=0, P=1, v=None):
    return lib.lionmuon_step_ex(ctypes.cast(fl.p, ctypes.c_void_p), ctypes.cast(fl.g, ctypes.c_void_p),
                                ctypes.cast(fl.m, ctypes.c_void_p), v, fl.shapes, fl.n, t, P, 0.9,
                                0.99, 0.1, ctypes.byref(cfg), ws, ws_bytes, None)


INVALID = lm.LM_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("kw", [dict(t=-1), dict(P=-1), dict(b1=1.0), dict(b1=-0.1), dict(b2=1.0),
                                dict(b2=float("nan")), dict(lr=-1e-3), dict(lr=float("inf")),
                                dict(wd=-0.1), dict(wd=float("nan"))])
def test_step_rejects_bad_scalars(lib, kw):
    fl = FakeList([(64, 64, False)])
    assert _step(lib, fl, **kw) == INVALID
    assert lib.lionmuon_last_error().decode() != ""


def test_step_rejects_bad_tensor_lists(lib):
    assert lib.lionmuon_step(None, None, None, None, 3, 1, 2, 0.9, 0.99, 0.01, 0.1, None) == INVALID
    assert lib.lionmuon_step(None, None, None, None, -1, 1, 2, 0.9, 0.99, 0.01, 0.1, None) == INVALID
    fl = FakeList([(64, 64, False), (8, 8, False)])
    fl.g[1] = None
    assert _step(lib, fl) == INVALID
    assert "null" in lib.lionmuon_last_error().decode()
    fl = FakeList([(-4, 64, False)])
    assert _step(lib, fl) == INVALID
    fl = FakeList([(4, 64, False)])
    fl.shapes[0].reserved = 7
    assert _step(lib, fl) == INVALID
    fl = FakeList([(4, 64, False)])
    fl.shapes[0].flags = 2
    assert _step(lib, fl) == INVALID
    fl = FakeList([(4, 64, False)])
    fl.m[0] = fl.p[0] + 2          # misaligned fp32 pointer
    assert _step(lib, fl) == INVALID


def test_step_rejects_overlapping_buffers(lib):
    base = 1 << 33
    # momentum overlaps params of the same tensor
    fl = FakeList([(16, 16, False)], addrs=[(base, base + 4096, base + 512)])
    assert _step(lib, fl) == INVALID
    assert "overlap" in lib.lionmuon_last_error().decode()
    # grads of tensor 1 overlap params of tensor 0
    fl = FakeList([(16, 16, False), (16, 16, False)],
                  addrs=[(base, base + 8192, base + 16384),
                         (base + 32768, base + 512, base + 65536)])
    assert _step(lib, fl) == INVALID
    # two tensors share one momentum buffer
    fl = FakeList([(16, 16, False), (16, 16, False)],
                  addrs=[(base, base + 8192, base + 16384),
                         (base + 32768, base + 40960, base + 16384)])
    assert _step(lib, fl) == INVALID
    # two tensors may share one read-only gradient (no write conflict)... but
    # not with a writable buffer: covered above.


def test_step_ex_rejects_bad_configs_and_workspaces(lib):
    fl = FakeList([(64, 64, False)])

    def cfg(**kw):
        c = lm.lm_config()
        lib.lionmuon_config_default(ctypes.byref(c))
        for k, v in kw.items():
            setattr(c, k, v)
        return c

    for bad in [dict(struct_size=4), dict(ns_steps=0), dict(ns_steps=65), dict(ns_precision=7),
                dict(ns_scale_mode=3), dict(ns_eps=-1.0), dict(ns_a=float("nan")),
                dict(lr_muon=-1.0), dict(lr_lion=float("nan")), dict(ns_bf16_min_side=-1),
                dict(reserved=1), dict(reserved2=1), dict(ns_schedule_steps=4),
                dict(ns_steps=17, ns_schedule_steps=17), dict(adam_beta1=1.0),
                dict(adam_beta2=-0.5), dict(adam_lr=-1.0), dict(adam_eps=float("inf")),
                dict(adam_wd=-0.1)]:
        assert _step_ex(lib, fl, cfg(**bad)) == INVALID, bad
    assert _step_ex(lib, fl, cfg(), ws=1 << 34, ws_bytes=0) == INVALID
    assert _step_ex(lib, fl, cfg(), ws=None, ws_bytes=4096) == INVALID
    assert _step_ex(lib, fl, cfg(), ws=(1 << 34) + 64, ws_bytes=1 << 20) == INVALID


def test_adamw_tensors_need_second_moments(lib):
    fl = FakeList([(1, 64, lm.LM_TENSOR_ADAMW)])
    cfg = lm.config()
    assert _step_ex(lib, fl, cfg) == INVALID                  # no second-moment array
    assert "second-moment" in lib.lionmuon_last_error().decode()
    assert _step(lib, fl) == INVALID                          # lionmuon_step has none
    base = 1 << 35
    v = (ctypes.c_void_p * 1)(fl.p[0] + 64)                   # overlaps params
    assert _step_ex(lib, fl, cfg, v=ctypes.cast(v, ctypes.c_void_p)) == INVALID
    fl2 = FakeList([(1, 64, lm.LM_TENSOR_ADAMW | lm.LM_TENSOR_LION_ONLY)])
    v2 = (ctypes.c_void_p * 1)(base)
    assert _step_ex(lib, fl2, cfg, v=ctypes.cast(v2, ctypes.c_void_p)) == INVALID


def test_plan_info_counts_adamw_tensors(lib):
    specs = [(768, 768, False), (1, 768, lm.LM_TENSOR_ADAMW), (1, 3072, lm.LM_TENSOR_ADAMW),
             (64, 64, lm.LM_TENSOR_ADAMW), (1, 100, False)]
    for t, P in [(0, 1), (1, 2)]:
        info = lm.lionmuon_plan_info(specs, t=t, P=P)
        assert info["n_adamw"] == 3 and info["adamw_elements"] == 768 + 3072 + 4096
        assert info["lion_bytes"] == 20.0 * info["lion_elements"] + 28.0 * info["adamw_elements"]
    assert lm.lionmuon_plan_info(specs, t=0, P=1)["n_muon"] == 1
    assert lm.lionmuon_plan_info(specs, t=1, P=2)["n_lion"] == 2


def test_ns_hook_rejects_bad_arguments(lib):
    base = 1 << 33
    f = lib.lionmuon_ns
    assert f(None, base, 8, 8, 1, None, None, 0, None) == INVALID
    assert f(base, base + 64, 8, 8, 1, None, None, 0, None) == INVALID      # overlap
    assert f(base, base + (1 << 20), -8, 8, 1, None, None, 0, None) == INVALID
    assert f(base, base + (1 << 20), 1, 8, 1, None, None, 0, None) == lm.LM_ERR_UNSUPPORTED
    assert f(base, base + (1 << 20), 8, 8, 0, None, None, 0, None) == lm.LM_OK   # empty batch


def test_empty_calls_are_no_ops(lib):
    fl = FakeList([])
    assert _step(lib, fl) == lm.LM_OK
    fl = FakeList([(0, 64, False), (5, 0, False)])
    fl.p[0] = None                  # empty tensors need no pointers
    # valid but non-empty calls would reach the device; empty ones never do
    assert _step(lib, fl) == lm.LM_OK


# --------------------------------------------------------------------------
# adaptive variant (Appendix G): configuration, plan and validation
# --------------------------------------------------------------------------
def _cfg(lib, **kw):
    c = lm.lm_config()
    lib.lionmuon_config_default(ctypes.byref(c))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_adaptive_config_defaults_and_validation(lib):
    c = _cfg(lib)
    assert c.adaptive_alpha == 0.0 and c.adaptive_power_steps == 5 and c.reserved3 == 0
    fl = FakeList([(64, 64, False)])
    for bad in [dict(adaptive_alpha=-0.01), dict(adaptive_alpha=1.5),
                dict(adaptive_alpha=float("nan")), dict(adaptive_power_steps=-1),
                dict(adaptive_power_steps=65), dict(reserved3=1)]:
        assert _step_ex(lib, fl, _cfg(lib, **bad)) == INVALID, bad


def _step_adaptive(lib, fl, cfg, decisions=None, srank=None):
    return lib.lionmuon_step_adaptive(ctypes.cast(fl.p, ctypes.c_void_p),
                                      ctypes.cast(fl.g, ctypes.c_void_p),
                                      ctypes.cast(fl.m, ctypes.c_void_p), None, fl.shapes, fl.n, 3,
                                      0.9, 0.99, 0.1, ctypes.byref(cfg), None, 0, decisions, srank,
                                      None)


def test_step_adaptive_rejects_bad_arguments(lib):
    fl = FakeList([(64, 64, False), (1, 64, False)])
    assert _step_adaptive(lib, fl, _cfg(lib)) == INVALID            # alpha = 0: not adaptive
    assert "adaptive_alpha" in lib.lionmuon_last_error().decode()
    assert lib.lionmuon_step_adaptive(None, None, None, None, None, 1, 0, 0.9, 0.99, 0.1, None,
                                      None, 0, None, None, None) == INVALID
    cfg = _cfg(lib, adaptive_alpha=0.01)
    base = 1 << 36
    assert _step_adaptive(lib, fl, cfg, decisions=base + 2) == INVALID      # misaligned
    assert _step_adaptive(lib, fl, cfg, srank=base + 4) == INVALID
    assert _step_adaptive(lib, fl, cfg, decisions=base + 8, srank=base) == INVALID  # overlap
    assert "overlap" in lib.lionmuon_last_error().decode()
    assert _step_adaptive(lib, FakeList([(64, 64, False)]), _cfg(lib, adaptive_alpha=0.01,
                                                                  adaptive_power_steps=99)) == INVALID


def test_plan_info_adaptive_step(lib):
    wl = workloads.gpt2_124m()
    specs = _specs(wl)
    k = 4
    cfg = lm.config(adaptive_alpha=0.01, adaptive_power_steps=k)
    info = lm.lionmuon_plan_info(specs, t=1, P=0, cfg=cfg)      # P is ignored
    muon = lm.lionmuon_plan_info(specs, t=0, P=1)
    assert info["n_muon"] == 48 and info["muon_elements"] == wl.matrix_numel
    assert info["n_lion"] == len(wl.tensors) - 48
    assert info["lion_elements"] == wl.numel - wl.matrix_numel
    assert info["ns_flops"] == muon["ns_flops"]                  # every candidate may take Muon
    blocks = part = extra = 0
    for t in wl.tensors:
        if t.lion_only or t.rows == 1:
            continue
        s, l = min(t.rows, t.cols), max(t.rows, t.cols)
        # register paths: blocks of 128 rows (tall) or 256 columns (wide)
        nb = -(-l // (128 if t.rows >= t.cols else 256))
        blocks += nb
        part += nb * s
        # workspace: sized for the generic path's blocks of 32 positions (the
        # most of any path), whatever path the alignment selects
        nbw = -(-l // 32)
        extra += (s + nbw * s + 2 * nbw + -(-s // 64)) * 8
    assert info["srank_bytes"] == 4.0 * wl.matrix_numel * (k + 1) + 16.0 * part * k
    assert muon["srank_bytes"] == 0.0
    ws_extra = info["workspace_bytes"] - muon["workspace_bytes"]
    assert extra <= ws_extra < extra + 256 * (48 + 2)
    assert lm.lionmuon_workspace_bytes(specs, cfg) == info["workspace_bytes"]
    # generic path (rows not a multiple of 4 floats, or a short side beyond the
    # register paths): blocks of 32 positions; register paths: 128 rows (tall)
    # or 256 columns (wide)
    for shape, nb in [((97, 61), 4), ((61, 97), 4), ((3000, 2100), 94), ((1600, 1700), 54),
                      ((1100, 1300), 6), ((1300, 1284), 11), ((700, 900), 4)]:
        one = lm.lionmuon_plan_info([(*shape, False)], t=0, P=0,
                                    cfg=lm.config(adaptive_alpha=0.01, adaptive_power_steps=1))
        assert one["srank_bytes"] == 4.0 * shape[0] * shape[1] * 2 + 16.0 * nb * min(shape), shape
