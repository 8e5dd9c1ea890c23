"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, rejects bad arguments with the documented status before any
launch, and its host mask builder equals the oracle bit for bit."""
import ctypes
import os
import random
import re

import numpy as np
import pytest

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS
from oracle import mask as M

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(lvsa_\w+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert {"lvsa_build_mask", "lvsa_attention", "lvsa_dense_attention",
            "lvsa_build_mask_device"} <= names
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings_and_version():
    lib = L.lib()
    for s in (0, -1, -2, -3, -4, 7):
        assert lib.lvsa_status_str(s)
    assert lib.lvsa_version() >= 100
    p = L.params_default()
    assert (p.budget_frames, p.window, p.tper, p.window_mode, p.rotate, p.tie_high) == \
        (21, 6, 0, L.WINDOW_EXPANDED, 1, 0)


def _oracle_kw(p):
    return dict(C=p.budget_frames, W=p.window, tper=p.tper, mode=p.window_mode,
                rotate=bool(p.rotate), tie_high=bool(p.tie_high))


def _check_frames(T, s, p):
    tper, anchors, lo, hi = L.frame_sets(T, s, p)
    T_per, G, A = M.attended_frames(T, s, **_oracle_kw(p))
    assert tper == T_per
    assert anchors == sorted(G)
    for t in range(T):
        assert set(G) | set(range(lo[t], hi[t] + 1)) == A[t]


def _check_csr(T, P, B, s, p, layer=0):
    csr = L.build_mask(T, P, B, s, p, layer=layer)
    row_ptr, col_idx = csr.arrays()
    want_rp, want_ci = M.build_mask(T, P, B, s, layer=layer, **_oracle_kw(p))
    assert row_ptr.tolist() == want_rp
    assert col_idx.tolist() == want_ci
    assert csr.n_tokens == T * P and csr.block == B
    csr.free()


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_host_builder_matches_oracle_on_workloads(name):
    w = WORKLOADS[name]
    p = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper)
    T_per = M.anchor_period(w.frames, w.budget_frames, w.window, w.tper)
    steps = sorted(set(range(T_per)) | set(w.steps[:3]) | {T_per + 1})
    for s in steps:
        _check_frames(w.frames, s, p)
        _check_csr(w.frames, w.tokens_per_frame, w.block, s, p)


@pytest.mark.parametrize("tie_high", [0, 1])
@pytest.mark.parametrize("mode", [L.WINDOW_BASIC, L.WINDOW_ADAPTIVE, L.WINDOW_EXPANDED])
@pytest.mark.parametrize("rotate", [0, 1])
def test_host_builder_matches_oracle_rules(mode, rotate, tie_high):
    rng = random.Random(1000 * mode + 10 * rotate + tie_high)
    for _ in range(60):
        T = rng.randint(1, 40)
        W = rng.randint(0, 6)
        tper = rng.randint(1, T)
        p = L.Params(window=W, tper=tper, window_mode=mode, rotate=rotate,
                     tie_high=tie_high)
        s = rng.randint(0, 3 * tper)
        _check_frames(T, s, p)
        P = rng.randint(1, 40)
        B = rng.choice([1, 2, 3, 5, 8, 16, 64, 128])
        _check_csr(T, P, B, s, p)


def test_host_builder_derived_period_and_wan_horizons():
    for T in (21, 41, 61, 81, 101, 121):
        p = L.Params()
        for s in (0, 5, 13):
            _check_csr(T, 1560, 128, s, p)


def test_host_builder_layer_independent():
    p = L.Params()
    a = L.build_mask(65, 1590, 128, 7, p, layer=0).arrays()
    for layer in (1, 2, 3):
        b = L.build_mask(65, 1590, 128, 7, p, layer=layer).arrays()
        assert all(np.array_equal(x, y) for x, y in zip(a, b))


def _status(fn, *args):
    return fn(*args)


def test_invalid_mask_arguments():
    lib = L.lib()
    out = ctypes.c_void_p()
    good = L.Params()
    ref = ctypes.byref
    assert lib.lvsa_build_mask(121, 1560, 128, 0, 0, ref(good), ref(out)) == 0
    lib.lvsa_csr_free(out)
    bad_cases = [
        (0, 1560, 128, 0, 0, good),          # T < 1
        (4097, 16, 128, 0, 0, good),         # T > MAX_FRAMES
        (121, 0, 128, 0, 0, good),           # P < 1
        (121, 1560, 0, 0, 0, good),          # B < 1
        (121, 1560, 128, -1, 0, good),       # step < 0
        (121, 1560, 128, 0, -1, good),       # layer < 0
        (121, 1560, 128, 0, 0, L.Params(budget_frames=13, window=6)),  # C <= 2W+1
        (121, 1560, 128, 0, 0, L.Params(window=-1)),
        (121, 1560, 128, 0, 0, L.Params(window_mode=3)),
        (121, 1560, 128, 0, 0, L.Params(rotate=2)),
        (121, 1560, 128, 0, 0, L.Params(tper=-2)),
        (4096, 1 << 20, 128, 0, 0, good),    # N overflows int32
        (4096, 100, 1, 0, 0, good),          # nnz bound overflows int32
    ]
    for T, P, B, s, layer, p in bad_cases:
        out = ctypes.c_void_p(123)
        assert lib.lvsa_build_mask(T, P, B, s, layer, ref(p), ref(out)) == L.EINVAL, \
            (T, P, B, s, layer)
        assert out.value is None
    assert lib.lvsa_build_mask(121, 1560, 128, 0, 0, None, ref(out)) == L.EINVAL
    assert lib.lvsa_build_mask(121, 1560, 128, 0, 0, ref(good), None) == L.EINVAL
    assert lib.lvsa_frame_sets(0, 0, ref(good), None, None, None, None, None) == L.EINVAL
    lib.lvsa_csr_free(None)


def test_device_builder_rejects_before_launch():
    lib = L.lib()
    p = L.Params()
    fake = ctypes.c_void_p(0x1000)
    nb = 1475
    # capacity below nb*nb
    assert lib.lvsa_build_mask_device(121, 1560, 128, 0, 0, ctypes.byref(p), fake, fake,
                                      nb * nb - 1, None) == L.EINVAL
    assert lib.lvsa_build_mask_device(121, 1560, 128, 0, 0, ctypes.byref(p), None, fake,
                                      nb * nb, None) == L.EINVAL
    assert lib.lvsa_build_mask_device(121, 1560, 128, -3, 0, ctypes.byref(p), fake, fake,
                                      nb * nb, None) == L.EINVAL


def test_csr_device_view_requires_upload():
    csr = L.build_mask(4, 256, 64, 0, L.Params(budget_frames=2, window=0, tper=4))
    m = L.BlockMask()
    assert L.lib().lvsa_csr_device_view(csr._h, ctypes.byref(m)) == L.EINVAL


def _t(ptr=0x10000, heads=2, n=1000, d=128, sh=None, st=128):
    sh = n * st if sh is None else sh
    return L._Tensor(ptr, heads, n, d, sh, st)


def test_attention_rejects_before_launch():
    lib = L.lib()
    ref = ctypes.byref
    nb = -(-1000 // 128)
    m = L.BlockMask(1000, 128, nb, 0x2000, 0x3000)
    q, k, v = _t(0x10000), _t(0x20000), _t(0x30000)
    o = _t(0x40000)
    cases = [
        (dict(q=_t(heads=3)), L.EINVAL),                 # head mismatch
        (dict(k=_t(0x20000, n=999)), L.EINVAL),          # token mismatch
        (dict(v=_t(0x30000, d=64)), L.EUNSUPPORTED),     # head_dim
        (dict(q=_t(0x10008)), L.EUNSUPPORTED),           # alignment
        (dict(k=_t(0x20000, st=132)), L.EUNSUPPORTED),   # token stride % 8
        (dict(o=_t(0x10000)), L.EINVAL),                 # out aliases q
        (dict(m=L.BlockMask(1000, 96, 11, 0x2000, 0x3000)), L.EUNSUPPORTED),
        (dict(m=L.BlockMask(1000, 128, nb + 1, 0x2000, 0x3000)), L.EINVAL),
        (dict(m=L.BlockMask(1000, 128, nb, 0, 0x3000)), L.EINVAL),
    ]
    for over, want in cases:
        a = dict(q=q, k=k, v=v, o=o, m=m)
        a.update(over)
        st = lib.lvsa_attention(ref(a["q"]), ref(a["k"]), ref(a["v"]), ref(a["m"]),
                                ref(a["o"]), None)
        assert st == want, over
    assert lib.lvsa_attention(None, ref(k), ref(v), ref(m), ref(o), None) == L.EINVAL
    assert lib.lvsa_dense_attention(ref(q), ref(k), ref(v), 32, ref(o), None) == \
        L.EUNSUPPORTED
    assert lib.lvsa_dense_attention(ref(q), ref(k), ref(_t(0x30000, heads=1)), 128,
                                    ref(o), None) == L.EINVAL
