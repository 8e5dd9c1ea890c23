"""Pins for the mask oracle (CPU only).

The oracle is checked against what the LVSA paper fixes, not against itself:
hand-worked examples (tests/golden/), the properties the paper states in
Sec. 2 (budget identity, constant |G^s|, coverage over a period, frame 0 in
Def. 2's G, 2W+1 adaptive frames), and two independent formulations of the
frame -> block rule (token brute force and incidence products).
"""
import itertools
import os

import pytest

from oracle import mask as M

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line


# ---------------------------------------------------------------- golden ---

def test_golden_anchors_eq3():
    n = 0
    for line in _lines("anchors_eq3.txt"):
        lhs, rhs = line.split(":")
        T, T_per, s, rotate = map(int, lhs.split())
        want = sorted(map(int, rhs.split()))
        assert sorted(M.anchors(T, T_per, s, bool(rotate))) == want, line
        n += 1
    assert n >= 10


def test_golden_anchor_period():
    for line in _lines("anchor_period.txt"):
        lhs, rhs = line.split(":")
        T, C, W = map(int, lhs.split())
        T_per, k = map(int, rhs.split())
        assert M.anchor_period(T, C, W) == T_per, line
        assert len(M.anchors(T, T_per, 0)) == k, line


def test_golden_windows():
    n = 0
    for line in _lines("windows.txt"):
        lhs, rhs = line.split(":")
        head, anchors = lhs.split("|")
        mode, T, W, tie_high, t = head.split()
        T, W, tie_high, t = int(T), int(W), bool(int(tie_high)), int(t)
        G = set() if anchors.strip() == "-" else set(map(int, anchors.split(",")))
        l_want, h_want, it_want = map(int, rhs.split())
        if mode == "basic":
            assert M.basic_window(t, W, T) == (l_want, h_want), line
        elif mode == "adaptive":
            assert M.adaptive_window(t, W, T) == (l_want, h_want), line
        else:
            assert M.expanded_window(t, G, W, T, tie_high) == (l_want, h_want, it_want), line
        n += 1
    assert n >= 15


def test_golden_attended_frames_basic_and_adaptive():
    """A(t) through attended_frames for the basic and adaptive windows:
    period, anchors (rotating, fixed, with a dedicated initial anchor) and
    window together."""
    modes = {"basic": M.WINDOW_BASIC, "adaptive": M.WINDOW_ADAPTIVE}
    n = 0
    for line in _lines("attended_frames.txt"):
        lhs, rhs = line.split(":")
        mode, rot, T, C, W, tper, E, s, t = lhs.split()
        T, C, W, tper, E, s, t = map(int, (T, C, W, tper, E, s, t))
        _, _, A = M.attended_frames(T, s, C=C, W=W, tper=tper, mode=modes[mode],
                                    rotate=rot == "1", extra=E)
        assert sorted(A[t]) == [int(x) for x in rhs.split()], line
        n += 1
    assert n >= 15


def test_golden_tiny_mask():
    for line in _lines("tiny_mask.txt"):
        fields = [f.strip() for f in line.split("|")]
        s = int(fields[0])
        A_want = [set(map(int, a.split(","))) for a in fields[1].split(";")]
        _, _, A = M.attended_frames(4, s, C=2, W=0, tper=4)
        assert A == A_want
        rows_want = [None] * 16
        for spec in fields[2:]:
            rng, cols = spec.split(":")
            a, b = map(int, rng.split("-"))
            for qb in range(a, b + 1):
                rows_want[qb] = list(map(int, cols.split()))
        row_ptr, col_idx = M.build_mask(4, 256, 64, s, C=2, W=0, tper=4)
        got = [col_idx[row_ptr[i]:row_ptr[i + 1]] for i in range(16)]
        assert got == rows_want
        assert row_ptr[-1] == 128


def test_golden_straddle_blocks():
    A = [{0}, {1}, {2}]
    want = []
    for line in _lines("straddle_blocks.txt"):
        qb, cols = line.split(":")
        want.append(list(map(int, cols.split())))
    assert M.block_keep_bruteforce(A, 3, 3, 2) == want
    assert M.block_keep(A, 3, 3, 2) == want
    assert M.block_keep_incidence(A, 3, 3, 2) == want


# ------------------------------------------------------------- invariants ---

SMALL = [(T, W, T_per) for T in range(1, 17) for W in range(0, 5)
         for T_per in range(1, T + 1)]


@pytest.mark.parametrize("T", range(1, 17))
def test_anchor_count_coverage_period(T):
    """|G^s| = ceil(T/T_per) for every s; every frame is an anchor within any
    T_per consecutive steps; G^{s+T_per} = G^s; G^0 is Def. 2's G and holds
    frame 0 (Sec. 2, rotation properties; Eq. 3; Def. 2)."""
    for T_per in range(1, T + 1):
        k = M.ceil_div(T, T_per)
        fixed = M.anchors(T, T_per, 0, rotate=False)
        assert M.anchors(T, T_per, 0) == fixed
        assert 0 in fixed
        for s in range(0, 3 * T_per):
            G = M.anchors(T, T_per, s)
            assert len(G) == k
            assert G == M.anchors(T, T_per, s + T_per)
            assert all(0 <= f < T for f in G)
        for s0 in range(0, 2 * T_per):
            cover = set()
            for s in range(s0, s0 + T_per):
                cover |= M.anchors(T, T_per, s)
            assert cover == set(range(T))


def test_adaptive_window_size_and_reflection():
    """Exactly 2W+1 frames containing t when 2W+1 <= T, and the mirror image
    of frame t's window is frame T-1-t's window (Sec. 2, adaptive window)."""
    for T in range(1, 30):
        for W in range(0, 8):
            for t in range(T):
                l, h = M.adaptive_window(t, W, T)
                assert 0 <= l <= t <= h <= T - 1
                if 2 * W + 1 <= T:
                    assert h - l + 1 == 2 * W + 1
                else:
                    assert (l, h) == (0, T - 1)
                lr, hr = M.adaptive_window(T - 1 - t, W, T)
                assert (lr, hr) == (T - 1 - h, T - 1 - l)


def test_basic_window_symmetric():
    """t' in W(t) iff |t - t'| <= W, a symmetric relation (Def. 2)."""
    for T in range(1, 20):
        for W in range(0, 6):
            for t, u in itertools.product(range(T), repeat=2):
                lt, ht = M.basic_window(t, W, T)
                lu, hu = M.basic_window(u, W, T)
                assert (lt <= u <= ht) == (abs(t - u) <= W) == (lu <= t <= hu)


@pytest.mark.parametrize("tie_high", [False, True])
def test_expanded_window_budget_identity(tie_high):
    """|A(t)| = |G| + min(2W+1, T-|G|) for every t (Sec. 2, Fig. 1 caption and
    the paragraph after Alg. 1); the window is contiguous, contains the
    adaptive window and t, and the loop ends within T iterations."""
    for T, W, T_per in SMALL:
        for s in range(0, 2 * T_per):
            G = M.anchors(T, T_per, s)
            for t in range(T):
                l, h, it = M.expanded_window(t, G, W, T, tie_high)
                la, ha = M.adaptive_window(t, W, T)
                assert 0 <= l <= la <= t <= ha <= h <= T - 1
                assert it <= T
                A = set(G) | set(range(l, h + 1))
                assert len(A) == len(G) + min(2 * W + 1, T - len(G))
                nonglobal = sum(1 for f in range(l, h + 1) if f not in G)
                assert nonglobal == min(2 * W + 1, T - len(G))


def test_budget_never_exceeded():
    """With the derived period and T >= C, |A(t)| = |G| + 2W+1 <= C for every t:
    ceil(T / ceil(T/c)) <= c for c = C - (2W+1) (Sec. 2, budget paragraph).
    The paper's wider claim that the shortfall is at most T_per - 1 does not
    hold in general (T = 21, C = 21, W = 3 gives T_per = 2, |A| = 18); it is
    checked only on the paper's own configurations below."""
    for T in range(1, 130):
        for C, W in [(21, 6), (21, 3), (33, 6), (13, 2), (9, 1)]:
            if T < C:
                continue
            T_per, G, A = M.attended_frames(T, 0, C=C, W=W)
            for t in range(T):
                assert len(A[t]) == len(G) + 2 * W + 1 <= C
    T_per, G, A = M.attended_frames(21, 0, C=21, W=3)
    assert (T_per, len(G), len(A[0])) == (2, 11, 18)


def test_paper_configs_budget_and_iterations():
    """On the paper's Wan horizons (T = 21 .. 121, C = 21) with W = 6, every
    frame set is within two frames of C and Alg. 1 runs at most 8 times per
    call (Sec. 2, budget paragraph and the cost remark after Alg. 1)."""
    for T in [21, 41, 61, 81, 101, 121, 62, 83, 104]:
        T_per = M.anchor_period(T, 21, 6)
        for s in range(T_per):
            G = M.anchors(T, T_per, s)
            for t in range(T):
                l, h, it = M.expanded_window(t, G, 6, T)
                assert it <= 8
                A = set(G) | set(range(l, h + 1))
                assert abs(len(A) - 21) <= 2


# -------------------------------------------------------- frame -> block ---

@pytest.mark.parametrize("T,P,B", [(3, 5, 4), (4, 6, 4), (5, 7, 8), (6, 4, 3),
                                   (4, 16, 16), (3, 10, 32), (7, 3, 5)])
def test_block_rule_three_formulations_agree(T, P, B):
    for W, T_per in [(0, 2), (1, 3), (0, T), (2, 1)]:
        for s in range(T_per):
            for mode in (M.WINDOW_BASIC, M.WINDOW_ADAPTIVE, M.WINDOW_EXPANDED):
                _, _, A = M.attended_frames(T, s, W=W, tper=T_per, mode=mode)
                brute = M.block_keep_bruteforce(A, T, P, B)
                assert M.block_keep(A, T, P, B) == brute
                assert M.block_keep_incidence(A, T, P, B) == brute


def test_block_csr_invariants_and_kronecker():
    """Diagonal block kept, columns ascending and unique, nnz = row_ptr[-1];
    when B divides P the CSR is the frame mask expanded by P/B (P9, P10)."""
    for T, W, T_per in [(8, 1, 4), (10, 2, 3), (6, 0, 6), (12, 1, 5)]:
        for s in range(T_per):
            for P, B in [(8, 4), (6, 3), (10, 4), (7, 7)]:
                rp, ci = M.build_mask(T, P, B, s, W=W, tper=T_per)
                nb = M.ceil_div(T * P, B)
                assert len(rp) == nb + 1 and rp[0] == 0 and rp[-1] == len(ci)
                for qb in range(nb):
                    row = ci[rp[qb]:rp[qb + 1]]
                    assert row == sorted(set(row))
                    assert qb in row
                if P % B == 0:
                    _, _, A = M.attended_frames(T, s, W=W, tper=T_per)
                    r = P // B
                    for qb in range(nb):
                        t = qb // r
                        want = [tau * r + j for tau in sorted(A[t]) for j in range(r)]
                        assert ci[rp[qb]:rp[qb + 1]] == want


def test_full_mask_cases():
    """T_per = 1 (every frame an anchor) or 2W+1 >= T gives every block (P11)."""
    for T, P, B, W, T_per in [(4, 256, 64, 1, 4), (5, 6, 4, 0, 1), (3, 9, 4, 3, 3)]:
        for s in range(T_per):
            rp, ci = M.build_mask(T, P, B, s, W=W, tper=T_per)
            nb = M.ceil_div(T * P, B)
            assert ci == list(range(nb)) * nb


def test_layer_has_no_effect():
    a = M.build_mask(21, 1560, 128, 5, layer=0)
    for layer in (1, 3, 29):
        assert M.build_mask(21, 1560, 128, 5, layer=layer) == a


def test_large_config_counts():
    """Block counts of the full-size workloads at step 10, W = 6, from the
    frame-range formulation (pure Python loops) against the incidence form."""
    for T, P, C in [(21, 1560, 21), (65, 1590, 33)]:
        _, _, A = M.attended_frames(T, 10, C=C, W=6)
        assert M.block_keep(A, T, P, 128) == M.block_keep_incidence(A, T, P, 128)
    rp, ci = M.build_mask(121, 1560, 128, 10)
    assert len(rp) - 1 == 1475
    assert all(qb in ci[rp[qb]:rp[qb + 1]] for qb in range(1475))


def test_invalid_budget_rejected():
    with pytest.raises(ValueError):
        M.anchor_period(30, 13, 6)


# ------------------------------------------------------- token level ---

@pytest.mark.parametrize("T,P,s,W,tper", [(4, 3, 0, 0, 4), (5, 7, 2, 1, 2),
                                           (6, 5, 3, 1, 3), (9, 2, 4, 2, 4)])
def test_token_mask_is_eq2_elementwise(T, P, s, W, tper):
    """Eq. 2 at token level: (i, j) kept iff frame(j) in A(frame(i)), checked
    element by element from integer division, and each frame-pair tile of
    the matrix is constant."""
    _, _, A = M.attended_frames(T, s, W=W, tper=tper)
    tm = M.token_mask(A, T, P)
    N = T * P
    assert tm.shape == (N, N)
    for i in range(N):
        for j in range(N):
            assert bool(tm[i, j]) == ((j // P) in A[i // P]), (i, j)
    # Every query token keeps its own frame (t in A(t)), so no row is empty.
    assert tm.any(axis=1).all()
    assert all(tm[i, i] for i in range(N))


@pytest.mark.parametrize("T,P,B", [(5, 7, 4), (6, 5, 3), (4, 6, 4), (7, 3, 2)])
def test_block_rule_is_smallest_cover_of_token_mask(T, P, B):
    """The any-overlap block rule keeps exactly the blocks that hold at least
    one Eq. 2 token pair: a superset of the token mask with no empty block."""
    for s in range(3):
        _, _, A = M.attended_frames(T, s, W=1, tper=3)
        tm = M.token_mask(A, T, P)
        N = T * P
        nb = M.ceil_div(N, B)
        row_ptr, col_idx = M.to_csr(M.block_keep(A, T, P, B))
        for qb in range(nb):
            kept = set(col_idx[row_ptr[qb]:row_ptr[qb + 1]])
            for kb in range(nb):
                tile = tm[qb * B:min((qb + 1) * B, N), kb * B:min((kb + 1) * B, N)]
                assert (kb in kept) == bool(tile.any()), (s, qb, kb)


# ---------------------------------------------------- extra anchors ---

def test_golden_extra_anchors():
    n = 0
    for line in _lines("extra_anchors.txt"):
        kind, rest = line.split(None, 1)
        if kind == "G":
            lhs, tper_s, frames = rest.split(":")
            T, C, W, tper, s, rotate, E = map(int, lhs.split())
            T_per = M.anchor_period(T, C, W, tper, E)
            assert T_per == int(tper_s), line
            assert sorted(M.anchors(T, T_per, s, bool(rotate), E)) == \
                list(map(int, frames.split())), line
        else:
            lhs, frames = rest.split(":")
            T, C, W, tper, s, rotate, E, t = map(int, lhs.split())
            _, _, A = M.attended_frames(T, s, C, W, tper, rotate=bool(rotate), extra=E)
            assert sorted(A[t]) == list(map(int, frames.split())), line
        n += 1
    assert n >= 12


@pytest.mark.parametrize("E", [1, 2, 3])
def test_extra_anchors_invariants(E):
    """Frames 0..E-1 are in every A(t); the Alg. 1 identity |A(t)| = |G| +
    min(2W+1, T-|G|) still holds; E = 0 is the plain rule; with the derived
    period the budget C is never exceeded once T >= C."""
    for T in (9, 21, 40, 121):
        for W in (0, 1, 3, 6):
            C = 2 * W + 1 + E + 3
            for s in range(0, 20, 3):
                for rotate in (True, False):
                    T_per, G, A = M.attended_frames(T, s, C, W, rotate=rotate, extra=E)
                    _, G0, _ = M.attended_frames(T, s, C, W, tper=T_per, rotate=rotate)
                    assert G == G0 | set(range(min(E, T)))
                    for t in range(T):
                        assert set(range(min(E, T))) <= A[t]
                        assert len(A[t]) == len(G) + min(2 * W + 1, T - len(G))
                        if T >= C:
                            assert len(A[t]) <= C
    with pytest.raises(ValueError):
        M.anchor_period(21, 14, 6, extra=1)   # C - (2W+1) - E = 0


# ------------------------------------------------------- text tokens ---

@pytest.mark.parametrize("T,P,L", [(4, 3, 5), (5, 4, 1), (3, 6, 11), (6, 2, 0)])
def test_text_token_mask_elementwise(T, P, L):
    """Text tokens after the video: every pair touching a text token is
    kept, video pairs follow Eq. 2; checked element by element."""
    _, _, A = M.attended_frames(T, 1, W=0, tper=3)
    tm = M.token_mask_text(A, T, P, L)
    V = T * P
    for i in range(V + L):
        for j in range(V + L):
            want = i >= V or j >= V or ((j // P) in A[i // P])
            assert bool(tm[i, j]) == want, (i, j)


@pytest.mark.parametrize("T,P,B,L", [(5, 7, 4, 3), (6, 5, 3, 9), (4, 6, 4, 1),
                                     (7, 3, 2, 6), (5, 8, 8, 8), (4, 9, 4, 0)])
def test_text_block_rule_is_smallest_cover(T, P, B, L):
    """The text block rule keeps exactly the blocks holding at least one kept
    token pair of the text token mask; with L = 0 it is the video rule."""
    for s in range(3):
        _, _, A = M.attended_frames(T, s, W=1, tper=3)
        tm = M.token_mask_text(A, T, P, L)
        N = T * P + L
        nb = M.ceil_div(N, B)
        rows = M.block_keep_text(A, T, P, B, L)
        for qb in range(nb):
            for kb in range(nb):
                tile = tm[qb * B:min((qb + 1) * B, N), kb * B:min((kb + 1) * B, N)]
                assert (kb in rows[qb]) == bool(tile.any()), (s, qb, kb)
        if L == 0:
            assert rows == M.block_keep(A, T, P, B)
