"""CPU model of the position rule by which the attention kernel merges the two
CSR rows of a pair of query blocks into one walk (host logic; the kernel itself
is checked on the GPU by test_gpu_attention.py's caller-CSR tests).

The kernel stages both rows largest key first and places every entry of the
union at: its index in its own row, plus the entries of the other row with a
larger key (found by binary search), minus the keys above it that both rows
hold (its row's entries before it that the other row also holds, counted over
passes of NT entries).  An entry of the second row that the first row also
holds is not written (the first row's entry carries both).  This model applies
the same rule, pass by pass, and must give exactly the union of the two rows
in descending key order, each key once, with its step word.
"""
import bisect
import random

WALK_CAP = 8000
NT = 512


def key(e, exact):
    return e & 0xFFFF if exact else e


def step_word(e0, e1, in0, in1, nb, exact):
    kb = key(e0 if in0 else e1, exact)
    if kb < 0 or kb >= nb:
        return 0xFFFF if exact else 0x3FFFFFFF
    if exact:
        return (((e0 if in0 else e1) & 0xFFFFFF) | (e0 & 0x0F000000 if in0 else 0)
                | (((e1 & 0x0F000000) << 4) if in1 else 0))
    return kb | (1 << 30 if in0 else 0) | (1 << 31 if in1 else 0)


def merge_model(row0, row1, nb, exact):
    """The kernel's rule: returns the walk's words (list)."""
    sa = list(reversed(row0))[:WALK_CAP]
    sb = list(reversed(row1))[:WALK_CAP]
    na, nc = len(sa), len(sb)
    neg_a = [-key(e, exact) for e in sa]      # ascending, for bisect
    neg_b = [-key(e, exact) for e in sb]
    out = [None] * WALK_CAP
    dup_base0 = dup_base1 = 0
    words = 0
    for ps in range((max(na, nc) + NT - 1) // NT):
        span = range(ps * NT, ps * NT + NT)
        d0 = [False] * NT
        d1 = [False] * NT
        above0 = [0] * NT
        above1 = [0] * NT
        p0 = [0] * NT
        for i, t in enumerate(span):
            if t < na:
                x = key(sa[t], exact)
                lo = bisect.bisect_left(neg_b, -x)      # entries of row 1 with a larger key
                above0[i] = lo
                if lo < nc:
                    p0[i] = sb[lo]
                    d0[i] = key(sb[lo], exact) == x
            if t < nc:
                y = key(sb[t], exact)
                lo = bisect.bisect_left(neg_a, -y)
                above1[i] = lo
                d1[i] = lo < na and key(sa[lo], exact) == y
        c0 = c1 = 0
        for i, t in enumerate(span):
            before0, before1 = dup_base0 + c0, dup_base1 + c1
            if t < na:
                r = t + above0[i] - before0
                if 0 <= r < WALK_CAP:
                    out[r] = step_word(sa[t], p0[i], True, d0[i], nb, exact)
            if t < nc and not d1[i]:
                r = t + above1[i] - before1
                if 0 <= r < WALK_CAP:
                    out[r] = step_word(0, sb[t], False, True, nb, exact)
            c0 += d0[i]
            c1 += d1[i]
        dup_base0 += c0
        dup_base1 += c1
        words = na + nc - dup_base1
    n = min(words, WALK_CAP)
    return out[:n]


def union_words(row0, row1, nb, exact):
    """The definition: every key either row holds, largest first, once."""
    h0 = {key(e, exact): e for e in row0}
    h1 = {key(e, exact): e for e in row1}
    words = []
    for kb in sorted(set(h0) | set(h1), reverse=True):
        in0, in1 = kb in h0, kb in h1
        words.append(step_word(h0.get(kb, 0), h1.get(kb, 0), in0, in1, nb, exact))
    return words


def _row(rng, nb, k, exact, lo=0):
    cols = sorted(rng.sample(range(lo, nb), min(k, nb - lo)))
    if not exact:
        return cols
    return [c | rng.randint(0, 255) << 16 | rng.randint(1, 15) << 24 for c in cols]


def test_merge_rule_gives_the_union_on_random_rows():
    rng = random.Random(11)
    for _ in range(400):
        nb = rng.choice([1, 2, 3, 7, 40, 300, 1475, 3000])
        exact = rng.random() < 0.5
        k0 = rng.choice([0, 1, 2, rng.randint(0, nb)])
        k1 = rng.choice([0, 1, rng.randint(0, nb)])
        r0, r1 = _row(rng, nb, k0, exact), _row(rng, nb, k1, exact)
        assert merge_model(r0, r1, nb, exact) == union_words(r0, r1, nb, exact)


def test_merge_rule_edge_rows():
    nb = 8000
    full = list(range(nb))
    for r0, r1 in [
        (full, full),                              # 8000 words over 16 passes
        (full, []), ([], full), ([], []),
        (full[::2], full[1::2]),                   # disjoint, interleaved
        (full[:10], full[-10:]),                   # disjoint, apart
        ([5], [5]), ([0], [nb - 1]),
        (full[:600], full[:600]),                  # identical, past one pass
    ]:
        assert merge_model(r0, r1, nb, False) == union_words(r0, r1, nb, False)


def test_out_of_range_keys_give_words_that_mask_everything():
    """Keys at or past nb (a caller's bad column) become the no-key word and
    are never loaded; the walk stays in bounds."""
    nb = 10
    r0, r1 = [1, 4, 12], [4, 9, 30]
    got = merge_model(r0, r1, nb, False)
    assert got == union_words(r0, r1, nb, False)
    assert got[:2] == [0x3FFFFFFF, 0x3FFFFFFF]
    assert got[2:] == [9 | 1 << 31, 4 | 3 << 30, 1 | 1 << 30]
