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
            "lvsa_build_mask_device", "lvsa_csr_info", "lvsa_frame_window"} <= names
    lib = ctypes.CDLL(L.LIB_PATH)
    missing = [n for n in sorted(names) if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings_and_version():
    lib = L.lib()
    for s in (0, -1, -2, -3, -4, 7):
        assert lib.lvsa_status_str(s)
    assert lib.lvsa_version() >= 20000
    p = L.params_default()
    assert (p.budget_frames, p.window, p.tper, p.window_mode, p.rotate, p.tie_high,
            p.extra_anchors) == (21, 6, 0, L.WINDOW_EXPANDED, 1, 0, 0)


def _oracle_kw(p):
    return dict(C=p.budget_frames, W=p.window, tper=p.tper, mode=p.window_mode,
                rotate=bool(p.rotate), tie_high=bool(p.tie_high), extra=p.extra_anchors,
                text=p.text_tokens)


def _check_frames(T, s, p):
    tper, anchors, lo, hi = L.frame_sets(T, s, p)
    kw = _oracle_kw(p)
    kw.pop("text")   # text tokens do not change the frame sets
    T_per, G, A = M.attended_frames(T, s, **kw)
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
    assert csr.n_tokens == T * P + p.text_tokens and csr.block == B
    csr.free()


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_host_builder_matches_oracle_on_workloads(name):
    w = WORKLOADS[name]
    p = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper,
                 text_tokens=w.text_tokens)
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
        # periods beyond T too (Eq. 3 then leaves one anchor, (s mod T_per) mod T)
        tper = rng.randint(1, 3 * T)
        p = L.Params(window=W, tper=tper, window_mode=mode, rotate=rotate,
                     tie_high=tie_high, extra_anchors=rng.choice([0, 0, 1, 2, 5]))
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


@pytest.mark.parametrize("E", [1, 2])
def test_host_builder_extra_anchors_derived_period(E):
    """Dedicated initial anchors with the budget-derived period on the Wan
    and HV horizons (C = 21 and 33, W = 6), against the oracle."""
    for T, C, P in ((21, 21, 1560), (121, 21, 1560), (65, 33, 1590)):
        p = L.Params(budget_frames=C, window=6, extra_anchors=E)
        for s in (0, 7, 10, 17):
            _check_frames(T, s, p)
            _check_csr(T, P, 128, s, p)
    ref = ctypes.byref
    out = ctypes.c_void_p()
    bad = L.Params(budget_frames=14, window=6, extra_anchors=1)   # C = 2W+1+E
    assert L.lib().lvsa_build_mask(121, 1560, 128, 0, 0, ref(bad), ref(out)) == L.EINVAL
    neg = L.Params(extra_anchors=-1)
    assert L.lib().lvsa_build_mask(121, 1560, 128, 0, 0, ref(neg), ref(out)) == L.EINVAL


def test_host_builder_layer_independent():
    p = L.Params()
    a = L.build_mask(65, 1590, 128, 7, p, layer=0).arrays()
    for layer in (1, 2, 3):
        b = L.build_mask(65, 1590, 128, 7, p, layer=layer).arrays()
        assert all(np.array_equal(x, y) for x, y in zip(a, b))


def _status(fn, *args):
    return fn(*args)


@pytest.mark.parametrize("T", [1, 2, 4, 7, 10])
def test_anchor_period_longer_than_the_video(T):
    """T_per > T (an explicit period): Eq. 3 keeps one anchor, (s mod T_per)
    mod T, for every step up to 3 T_per; frame sets and CSR against the
    oracle, and the anchor set against Eq. 3 written out."""
    for tper in (T + 1, 2 * T, 3 * T, 100):
        for s in range(0, 3 * tper + 1, max(1, tper // 7)):
            p = L.Params(window=0, tper=tper)
            _, anchors, _, _ = L.frame_sets(T, s, p)
            assert anchors == [(s % tper) % T], (T, tper, s)
            _check_frames(T, s, p)
            _check_csr(T, 37, 16, s, p)
            pe = L.Params(window=1, tper=tper, window_mode=L.WINDOW_EXPANDED, extra_anchors=1)
            _check_frames(T, s, pe)


def test_csr_info_follows_the_boundary_order():
    """lvsa_csr_info returns (n_q_blocks, n_kv_blocks, nnz, row_ptr, col_idx);
    lvsa_csr_shape the tokens and the block size."""
    T, P, B = 5, 200, 128
    csr = L.build_mask(T, P, B, 1, L.Params(window=1, tper=3, text_tokens=77))
    nq, nk, nnz, rp, ci = csr.info()
    N = T * P + 77
    assert nq == nk == -(-N // B)
    assert csr.shape() == (N, B)
    want_rp, want_ci = M.build_mask(T, P, B, 1, W=1, tper=3, text=77)
    assert nnz == len(want_ci) == want_rp[-1]
    assert [rp[i] for i in range(nq + 1)] == want_rp
    assert [ci[i] for i in range(nnz)] == want_ci


def test_frame_window_call_and_growth_match_alg1():
    """The per-frame call equals the frame sets, and the growth counts equal
    the iterations of Alg. 1 in the oracle, on the Wan and HV horizons and on
    random rules."""
    rng = random.Random(11)
    cases = [(T, L.Params()) for T in (21, 41, 61, 81, 101, 121)]
    cases += [(65, L.Params(budget_frames=33)), (129, L.Params(budget_frames=33))]
    for _ in range(30):
        T = rng.randint(1, 60)
        cases.append((T, L.Params(window=rng.randint(0, 6), tper=rng.randint(1, 2 * T),
                                  tie_high=rng.randint(0, 1),
                                  extra_anchors=rng.choice([0, 1, 3]))))
    for T, p in cases:
        for s in (0, 3, 10, 17):
            tper, anchors, lo, hi, grow = L.frame_sets(T, s, p, growth=True)
            G = set(anchors)
            for t in range(T):
                assert L.frame_window(T, s, t, p) == (lo[t], hi[t], grow[t])
                _, _, iters = M.expanded_window(t, G, p.window, T, bool(p.tie_high))
                assert grow[t] == iters, (T, s, t)
    with pytest.raises(L.LvsaError):
        L.frame_window(21, 0, 21, L.Params())
    # growth is 0 outside the expanded rule
    assert set(L.frame_sets(121, 10, L.Params(window_mode=L.WINDOW_ADAPTIVE),
                            growth=True)[4]) == {0}


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
    assert lib.lvsa_frame_sets(0, 0, ref(good), None, None, None, None, None,
                               None) == L.EINVAL
    lib.lvsa_csr_free(None)


def test_device_builder_rejects_before_launch():
    lib = L.lib()
    p = L.Params()
    fake = ctypes.c_void_p(0x1000)
    nb = 1475
    build = lambda rp, ci, cap, step=0: lib.lvsa_build_mask_device(
        121, 1560, 128, step, 0, ctypes.byref(p), rp, ci, cap, None)
    assert build(fake, fake, nb * nb - 1) == L.EINVAL   # CSR capacity
    assert build(None, fake, nb * nb) == L.EINVAL
    assert build(fake, None, nb * nb) == L.EINVAL
    assert build(fake, fake, nb * nb, step=-3) == L.EINVAL


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
    m = L.BlockMask(1000, 128, nb, nb, 0x2000, 0x3000)
    q, k, v = _t(0x10000), _t(0x20000), _t(0x30000)
    o = _t(0x40000)
    cases = [
        (dict(q=_t(heads=3)), L.EINVAL),                 # head mismatch
        (dict(k=_t(0x20000, n=999)), L.EINVAL),          # token mismatch
        (dict(v=_t(0x30000, d=64)), L.EUNSUPPORTED),     # head_dim
        (dict(q=_t(0x10008)), L.EUNSUPPORTED),           # alignment
        (dict(k=_t(0x20000, st=132)), L.EUNSUPPORTED),   # token stride % 8
        (dict(o=_t(0x10000)), L.EINVAL),                 # out aliases q
        (dict(m=L.BlockMask(1000, 96, 11, 11, 0x2000, 0x3000)), L.EUNSUPPORTED),
        (dict(m=L.BlockMask(1000, 128, nb + 1, nb + 1, 0x2000, 0x3000)), L.EINVAL),
        (dict(m=L.BlockMask(1000, 128, nb, nb - 1, 0x2000, 0x3000)), L.EINVAL),
        (dict(m=L.BlockMask(1000, 128, nb, nb, 0, 0x3000)), L.EINVAL),
        (dict(m=L.BlockMask(1000, 128, nb, nb, 0x2000, 0)), L.EINVAL),
    ]
    # sparse launches merge a pair's two CSR rows in LDS: nb <= 8000
    big_n = 8001 * 128
    big = [_t(a, heads=1, n=big_n) for a in (0x10000, 0x20000, 0x30000, 0x40000)]
    st = lib.lvsa_attention(ref(big[0]), ref(big[1]), ref(big[2]),
                            ref(L.BlockMask(big_n, 128, 8001, 8001, 0x2000, 0x3000)),
                            ref(big[3]), None)
    assert st == L.EUNSUPPORTED
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


# ------------------------------------------------------ token-exact form ---

def decode_entries(row_ptr, col_idx, entry, T, P, B, L=0):
    """Token mask described by the entry words (the token-exact form that
    include/lvsa.h defines), checking each word's fixed fields on the way.
    Segment of a token: its frame, or T for the L text tokens."""
    N = T * P + L
    nb = -(-N // B)
    tm = np.zeros((N, N), dtype=bool)
    tok_frame = np.minimum(np.arange(N) // P, T)
    for qb in range(nb):
        rows = np.arange(qb * B, min((qb + 1) * B, N))
        a = (tok_frame[rows] != tok_frame[qb * B]).astype(np.int64)
        for idx in range(row_ptr[qb], row_ptr[qb + 1]):
            w = int(entry[idx])
            kb = int(col_idx[idx])
            assert w & 0xFFFF == kb and w >> 28 == 0, hex(w)
            kfirst, pat = (w >> 16) & 0xFF, (w >> 24) & 0xF
            cols = np.arange(kb * B, min((kb + 1) * B, N))
            g0 = tok_frame[kb * B]
            b = (tok_frame[cols] != g0).astype(np.int64)
            straddles = tok_frame[min((kb + 1) * B, N) - 1] != g0
            assert kfirst == ((g0 + 1) * P - kb * B if straddles else B), (qb, kb)
            assert np.array_equal(b, (cols - kb * B >= kfirst).astype(np.int64))
            bit = 2 * a[:, None] + b[None, :]
            tm[np.ix_(rows, cols)] = ((pat >> bit) & 1).astype(bool)
    return tm


EXACT_CASES = [  # T, P, B: P >= B, mostly P mod B != 0 and a ragged last block
    (5, 200, 128), (7, 100, 64), (6, 130, 128), (4, 128, 128), (9, 70, 64),
    (3, 255, 128), (12, 96, 64),
]


@pytest.mark.parametrize("T,P,B", EXACT_CASES)
def test_host_entries_decode_to_oracle_token_mask(T, P, B):
    """Bit-exact: the entry words of the host builder describe exactly Eq. 2's
    token mask from the oracle, for every window rule and several steps."""
    for mode, rotate, tie_high in [(2, 1, 0), (2, 1, 1), (1, 1, 0), (0, 0, 0), (2, 0, 0)]:
        for s in (0, 1, 3):
            p = L.Params(budget_frames=0, window=1, tper=3, window_mode=mode,
                         rotate=rotate, tie_high=tie_high)
            csr = L.build_mask(T, P, B, s, p, exact=True)
            blk = L.build_mask(T, P, B, s, p)
            row_ptr, col_idx = csr.arrays()
            assert all(np.array_equal(x, y) for x, y in zip(blk.arrays(), (row_ptr, col_idx)))
            got = decode_entries(row_ptr, col_idx, csr.entries(), T, P, B)
            _, _, A = M.attended_frames(T, s, W=1, tper=3, mode=mode,
                                        rotate=bool(rotate), tie_high=bool(tie_high))
            assert np.array_equal(got, M.token_mask(A, T, P)), (mode, rotate, s)


def test_entries_full_when_block_divides_frame_and_unsupported_below_block():
    p = L.Params(budget_frames=0, window=1, tper=3)
    csr = L.build_mask(6, 256, 128, 2, p, exact=True)
    e = csr.entries()
    assert len(e) == csr.nnz and all(int(w) >> 24 == 0xF for w in e)
    m = L.ExactMask()
    assert L.lib().lvsa_csr_exact_view(csr._h, ctypes.byref(m)) == L.EINVAL  # no upload
    # P < B: no exact form; a block-only handle carries no entry words.
    out = ctypes.c_void_p(123)
    assert L.lib().lvsa_build_exact_mask(6, 100, 128, 0, 0, ctypes.byref(p),
                                         ctypes.byref(out)) == L.EUNSUPPORTED
    assert out.value is None
    blk = L.build_mask(6, 256, 128, 2, p)
    with pytest.raises(L.LvsaError) as ei:
        blk.entries()
    assert ei.value.status == L.EUNSUPPORTED
    assert L.lib().lvsa_csr_exact_view(blk._h, ctypes.byref(m)) == L.EUNSUPPORTED


def test_wan_horizon_entries_decode_on_sampled_rows():
    """Wan 6x shape (P = 1560, B = 128): the entry words of sampled query
    blocks give each query token exactly the keys of its frame set."""
    T, P, B, s = 121, 1560, 128, 10
    csr = L.build_mask(T, P, B, s, L.Params(), exact=True)
    row_ptr, col_idx = csr.arrays()
    entry = csr.entries()
    _, _, A = M.attended_frames(T, s, C=21, W=6)
    N = T * P
    for qb in (0, 12, 13, 700, 1474):
        for i in (qb * B, min(qb * B + B, N) - 1, qb * B + 40):
            got = np.zeros(N, dtype=bool)
            a = int((i // P) != (qb * B) // P)
            for idx in range(row_ptr[qb], row_ptr[qb + 1]):
                w = int(entry[idx])
                kb, kfirst, pat = w & 0xFFFF, (w >> 16) & 0xFF, (w >> 24) & 0xF
                for j in range(kb * B, min((kb + 1) * B, N)):
                    got[j] = (pat >> (2 * a + int(j - kb * B >= kfirst))) & 1
            want = np.array([(j // P) in A[i // P] for j in range(N)])
            assert np.array_equal(got, want), (qb, i)


def test_exact_attention_and_builder_reject_before_launch():
    lib = L.lib()
    ref = ctypes.byref
    p = L.Params()
    fake = ctypes.c_void_p(0x1000)
    nb = 1475
    build = lambda P, rp, e, cap: lib.lvsa_build_exact_mask_device(
        121, P, 128, 0, 0, ref(p), rp, e, cap, None)
    assert build(1560, fake, fake, nb * nb - 1) == L.EINVAL
    assert build(100, fake, fake, 1 << 30) == L.EUNSUPPORTED
    assert build(1560, fake, None, nb * nb) == L.EINVAL
    assert build(1560, None, fake, nb * nb) == L.EINVAL
    n = 1000
    nbk = -(-n // 128)
    q, k, v, o = _t(0x10000), _t(0x20000), _t(0x30000), _t(0x40000)
    em = lambda P, B, nb_, e=0x3000: L.ExactMask(n, B, nb_, P, 0x2000, e)
    cases = [
        (em(100, 128, nbk), L.EUNSUPPORTED),        # P < B
        (em(0, 128, nbk), L.EINVAL),                # P < 1
        (em(200, 128, nbk, e=0), L.EINVAL),         # no entry words
        (em(200, 96, 11), L.EUNSUPPORTED),          # block
    ]
    for m, want in cases:
        assert lib.lvsa_attention_exact(ref(q), ref(k), ref(v), ref(m), ref(o),
                                        None) == want, (m.frame_tokens, m.block)


# ------------------------------------------------------- text tokens ---

TEXT_CASES = [  # T, P, B, L: text after the video, ragged lengths
    (5, 200, 128, 77), (7, 100, 64, 300), (6, 130, 128, 1), (4, 256, 128, 128),
    (3, 255, 128, 513),
]


@pytest.mark.parametrize("T,P,B,Lt", TEXT_CASES)
def test_host_builder_with_text_matches_oracle(T, P, B, Lt):
    """Block CSR bit for bit against the oracle's text block rule, and the
    entry words decode to the oracle's text token mask."""
    for mode, rotate in [(2, 1), (0, 0)]:
        for s in (0, 2):
            p = L.Params(budget_frames=0, window=1, tper=3, window_mode=mode,
                         rotate=rotate, text_tokens=Lt)
            csr = L.build_mask(T, P, B, s, p, exact=True)
            row_ptr, col_idx = csr.arrays()
            kw = dict(W=1, tper=3, mode=mode, rotate=bool(rotate))
            want_rp, want_ci = M.build_mask(T, P, B, s, text=Lt, **kw)
            assert row_ptr.tolist() == want_rp and col_idx.tolist() == want_ci
            assert csr.n_tokens == T * P + Lt
            _, _, A = M.attended_frames(T, s, **kw)
            got = decode_entries(row_ptr, col_idx, csr.entries(), T, P, B, Lt)
            assert np.array_equal(got, M.token_mask_text(A, T, P, Lt)), (mode, s)
            blk = L.build_mask(T, P, B, s, p)
            assert all(np.array_equal(x, y) for x, y in zip(blk.arrays(), (row_ptr, col_idx)))


def test_rebuilds_after_free_match_the_oracle():
    """Freed handles hand their host arrays to later builds: a sequence of
    builds of different sizes and forms, each freed before the next, gives
    every mask bit for bit as a fresh oracle build does (no stale entries from
    a larger earlier mask, no entry words left on a block-only handle)."""
    seq = [  # T, P, B, Lt, exact
        (9, 150, 64, 0, True), (4, 70, 64, 0, False), (12, 96, 64, 40, True),
        (5, 200, 128, 0, False), (5, 200, 128, 0, True), (3, 255, 128, 7, True),
        (9, 150, 64, 0, False),
    ]
    for rep in range(2):
        for i, (T, P, B, Lt, exact) in enumerate(seq):
            s = i + rep
            p = L.Params(budget_frames=0, window=1, tper=3, text_tokens=Lt)
            csr = L.build_mask(T, P, B, s, p, exact=exact)
            row_ptr, col_idx = csr.arrays()
            want_rp, want_ci = M.build_mask(T, P, B, s, W=1, tper=3, text=Lt)
            assert row_ptr.tolist() == want_rp and col_idx.tolist() == want_ci, (rep, i)
            if exact:
                _, _, A = M.attended_frames(T, s, W=1, tper=3)
                got = decode_entries(row_ptr, col_idx, csr.entries(), T, P, B, Lt)
                want = M.token_mask_text(A, T, P, Lt) if Lt else M.token_mask(A, T, P)
                assert np.array_equal(got, want), (rep, i)
            else:
                with pytest.raises(L.LvsaError):
                    csr.entries()
            csr.free()


def test_host_builds_from_threads_match_the_oracle():
    """Builds and frees from four threads at once (ctypes releases the GIL
    around each call) give the oracle's masks: the per-thread working arrays
    and the shared pool of freed arrays do not mix masks."""
    import threading
    cases = [(9, 150, 64, 0), (12, 96, 64, 40), (5, 200, 128, 0), (7, 100, 64, 0)]
    want = {c: M.build_mask(c[0], c[1], c[2], 2, W=1, tper=3, text=c[3]) for c in cases}
    errors = []

    def work(i):
        try:
            for rep in range(30):
                T, P, B, Lt = cases[(i + rep) % len(cases)]
                p = L.Params(budget_frames=0, window=1, tper=3, text_tokens=Lt)
                csr = L.build_mask(T, P, B, 2, p, exact=rep % 2 == 0)
                rp, ci = csr.arrays()
                if (rp.tolist(), ci.tolist()) != tuple(want[(T, P, B, Lt)]):
                    errors.append((i, rep))
                csr.free()
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors[:5]


def test_host_builder_text_on_hv_horizon():
    """HunyuanVideo 1.5 at 2x (65 x 30x53, C = 33) with 512 text tokens."""
    T, P, B, Lt = 65, 1590, 128, 512
    p = L.Params(budget_frames=33, window=6, text_tokens=Lt)
    for s in (0, 10):
        csr = L.build_mask(T, P, B, s, p)
        row_ptr, col_idx = csr.arrays()
        want_rp, want_ci = M.build_mask(T, P, B, s, C=33, W=6, text=Lt)
        assert row_ptr.tolist() == want_rp and col_idx.tolist() == want_ci
    bad = L.Params(text_tokens=-1)
    out = ctypes.c_void_p()
    assert L.lib().lvsa_build_mask(65, 1590, 128, 0, 0, ctypes.byref(bad),
                                   ctypes.byref(out)) == L.EINVAL
