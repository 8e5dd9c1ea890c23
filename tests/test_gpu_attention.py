"""GPU parity: block-sparse and dense attention kernels against the fp32
oracle on the same seeded inputs (bf16 in, bf16 out; max-abs 2e-2 and
mean-abs 2e-3)."""
import sys

import numpy as np
import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS, make_qkv, workload_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import (assert_close, compare_rows, oracle_csr,
                            sample_q_blocks)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


def _params(w):
    return L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper,
                    text_tokens=w.text_tokens)


def _run_sparse(w, q, k, v, step, out=None):
    csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, step, _params(w))
    csr.upload()
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    out = L.attention(qd, kd, vd, csr.device_mask(), out=out)
    torch.cuda.synchronize()
    return out, csr


@pytest.mark.parametrize("name", ["tiny", "tiny_full"])
def test_tiny_full_output(name):
    w = WORKLOADS[name]
    q, k, v = workload_qkv(w)
    for step in w.steps:
        _say(f"[tiny] {name} step {step}")
        out, csr = _run_sparse(w, q, k, v, step)
        rp, ci = oracle_csr(w, step)
        ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                    v.float().numpy(), rp, ci, w.block),
                          w.heads, w.n_tokens, 128, w.block)
        err = np.abs(out.float().cpu().numpy() - ref)
        assert_close(float(err.max()), float(err.mean()))
    if name == "tiny_full":
        dense = OA.dense_attention(q.float().numpy(), k.float().numpy(), v.float().numpy())
        err = np.abs(out.float().cpu().numpy() - dense)
        assert_close(float(err.max()), float(err.mean()))


# Mid-size shapes: several tiles, frames that do not align with blocks, a
# ragged last block, both block sizes.
MID = [
    # T, P, B, H, W, T_per
    (6, 200, 128, 2, 1, 3),
    (9, 150, 64, 3, 1, 4),
    (5, 257, 128, 1, 0, 5),
    (12, 96, 64, 2, 2, 4),
    (3, 50, 128, 1, 0, 3),     # N = 150: one full block and one of 22 tokens
]


@pytest.mark.parametrize("T,P,B,H,W,tper", MID)
def test_mid_full_output(T, P, B, H, W, tper):
    _say(f"[mid] T={T} P={P} B={B} H={H} W={W} tper={tper}")
    N = T * P
    q, k, v = make_qkv(H, N, seed=T * 1000 + P)
    p = L.Params(window=W, tper=tper)
    for step in (0, 1):
        csr = L.build_mask(T, P, B, step, p)
        csr.upload()
        out = L.attention(q.cuda(), k.cuda(), v.cuda(), csr.device_mask())
        dense = L.dense_attention(q.cuda(), k.cuda(), v.cuda(), block=B)
        torch.cuda.synchronize()
        rp, ci = M.build_mask(T, P, B, step, W=W, tper=tper)
        ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                    v.float().numpy(), rp, ci, B),
                          H, N, 128, B)
        err = np.abs(out.float().cpu().numpy() - ref)
        assert_close(float(err.max()), float(err.mean()))
        dref = OA.dense_attention(q.float().numpy(), k.float().numpy(), v.float().numpy())
        err = np.abs(dense.float().cpu().numpy() - dref)
        assert_close(float(err.max()), float(err.mean()))


@pytest.mark.parametrize("name", ["wan13_1x", "wan13_6x", "hv15_2x", "wan14_6x"])
def test_full_size_sampled_rows(name):
    """The whole workload in one launch (as the bench runs it), checked on
    sampled query blocks of a few heads."""
    w = WORKLOADS[name]
    _say(f"[full] {name}: generating inputs")
    q, k, v = workload_qkv(w)
    step = 10
    _say(f"[full] {name}: sparse launch step {step}")
    out, csr = _run_sparse(w, q, k, v, step)
    rp, ci = oracle_csr(w, step)
    qbs = sample_q_blocks(rp, w.frames, w.tokens_per_frame, w.block)
    heads = sorted({0, w.heads - 1, w.heads // 2})
    _say(f"[full] {name}: oracle on heads {heads} q-blocks {qbs}")
    assert_close(*compare_rows(out, q, k, v, rp, ci, w.block, heads, qbs))


@pytest.mark.parametrize("name", ["wan13_1x", "hv15_2x", "wan13_6x"])
def test_dense_sampled_rows(name):
    w = WORKLOADS[name]
    heads = 2 if name == "wan13_6x" else w.heads
    _say(f"[dense] {name}: {heads} heads")
    q, k, v = make_qkv(heads, w.n_tokens, value_scale=w.value_scale)
    out = L.dense_attention(q.cuda(), k.cuda(), v.cuda(), block=w.block)
    torch.cuda.synchronize()
    nb = w.n_blocks
    rp = [i * nb for i in range(nb + 1)]
    ci = list(range(nb)) * nb
    qbs = [0, nb // 3, nb - 1]
    assert_close(*compare_rows(out, q, k, v, rp, ci, w.block, [0, heads - 1], qbs))


def test_deterministic_and_canary():
    """Bitwise-equal reruns; rows >= N of a larger output buffer are never
    written; NaN rows past N in the inputs never leak into the result."""
    T, P, B, H = 7, 190, 128, 2
    N = T * P
    _say("[canary] T=7 P=190 B=128 H=2")
    q, k, v = make_qkv(H, N, seed=5)
    pad = 200
    bufs = []
    for x in (q, k, v):
        b = torch.full((H, N + pad, 128), float("nan"), dtype=torch.bfloat16)
        b[:, :N] = x
        bufs.append(b.cuda())
    qd, kd, vd = (b[:, :N] for b in bufs)
    obuf = torch.full((H, N + pad, 128), 7.0, dtype=torch.bfloat16, device="cuda")
    csr = L.build_mask(T, P, B, 3, L.Params(window=1, tper=3))
    csr.upload()
    o1 = L.attention(qd, kd, vd, csr.device_mask(), out=obuf[:, :N])
    torch.cuda.synchronize()
    first = obuf.clone()
    L.attention(qd, kd, vd, csr.device_mask(), out=obuf[:, :N])
    torch.cuda.synchronize()
    assert torch.equal(first, obuf)
    assert bool((obuf[:, N:] == 7.0).all())
    assert bool(torch.isfinite(o1.float()).all())
    d1 = L.dense_attention(qd, kd, vd, block=B)
    d2 = L.dense_attention(qd, kd, vd, block=B)
    torch.cuda.synchronize()
    assert torch.equal(d1, d2)
    assert bool(torch.isfinite(d1.float()).all())


def test_strided_layout_matches_contiguous():
    """[N, H, d] storage (token stride H*d) gives the same bits as [H, N, d]."""
    T, P, B, H = 5, 300, 128, 3
    N = T * P
    _say("[layout] NHD vs HND")
    q, k, v = make_qkv(H, N, seed=9)
    csr = L.build_mask(T, P, B, 2, L.Params(window=1, tper=2))
    csr.upload()
    a = L.attention(q.cuda(), k.cuda(), v.cuda(), csr.device_mask())
    qn, kn, vn = (x.transpose(0, 1).contiguous().cuda().transpose(0, 1) for x in (q, k, v))
    on = torch.empty((N, H, 128), dtype=torch.bfloat16, device="cuda").transpose(0, 1)
    b = L.attention(qn, kn, vn, csr.device_mask(), out=on)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# Degenerate shapes: fewer tokens than one block, a single frame (the mask is
# then full), two frames with one-block rows, and the smallest frames.
EDGE = [
    # T, P, B, H, W, T_per
    (1, 10, 128, 1, 0, 1),      # N = 10 < B: one ragged block
    (1, 200, 64, 2, 0, 1),      # T = 1: every query attends its own frame only
    (2, 40, 128, 1, 0, 2),      # N = 80 < B, two frames in one block
    (3, 1, 64, 1, 0, 3),        # P = 1: frames of a single token
    (5, 64, 64, 1, 0, 5),       # one kept block per row besides the anchor's
]


@pytest.mark.parametrize("T,P,B,H,W,tper", EDGE)
def test_edge_shapes(T, P, B, H, W, tper):
    _say(f"[edge] T={T} P={P} B={B} H={H} W={W} tper={tper}")
    N = T * P
    q, k, v = make_qkv(H, N, seed=N + B)
    p = L.Params(window=W, tper=tper)
    csr = L.build_mask(T, P, B, 0, p)
    csr.upload()
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), csr.device_mask())
    torch.cuda.synchronize()
    rp, ci = M.build_mask(T, P, B, 0, W=W, tper=tper)
    assert csr.arrays()[0].tolist() == rp and csr.arrays()[1].tolist() == ci
    ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                v.float().numpy(), rp, ci, B),
                      H, N, 128, B)
    err = np.abs(out.float().cpu().numpy() - ref)
    assert np.isfinite(out.float().cpu().numpy()).all()
    assert_close(float(err.max()), float(err.mean()))


@pytest.mark.parametrize("scale", [8.0, 30.0])
def test_large_logits_exercise_the_rescale(scale):
    """Q and K scaled up so logits span hundreds of log2 units: the running
    max is raised on most key blocks (the rescale of O and l runs often) and
    the result still matches the fp32 oracle."""
    T, P, B, H = 6, 200, 128, 2
    N = T * P
    _say(f"[large-logits] scale {scale}")
    q, k, v = make_qkv(H, N, seed=int(scale))
    q = (q.float() * scale).to(torch.bfloat16)
    k = (k.float() * scale).to(torch.bfloat16)
    csr = L.build_mask(T, P, B, 1, L.Params(window=1, tper=3))
    csr.upload()
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), csr.device_mask())
    dense = L.dense_attention(q.cuda(), k.cuda(), v.cuda(), block=B)
    torch.cuda.synchronize()
    rp, ci = M.build_mask(T, P, B, 1, W=1, tper=3)
    qf, kf, vf = (x.float().numpy() for x in (q, k, v))
    ref = OA.assemble(OA.block_sparse_attention(qf, kf, vf, rp, ci, B), H, N, 128, B)
    g = out.float().cpu().numpy()
    assert np.isfinite(g).all()
    err = np.abs(g - ref)
    assert_close(float(err.max()), float(err.mean()))
    dref = OA.dense_attention(qf, kf, vf)
    err = np.abs(dense.float().cpu().numpy() - dref)
    assert_close(float(err.max()), float(err.mean()))


@pytest.mark.parametrize("T,P,B,exact", [(9, 150, 64, False), (9, 150, 64, True),
                                         (12, 200, 128, False), (12, 200, 128, True)])
def test_pairs_whose_rows_differ(T, P, B, exact):
    """The kernel walks query blocks in pairs over the union of their key
    lists; where a frame edge falls between the two blocks their rows differ
    and each block's waves must drop the other's extra key blocks.  Shapes
    where that happens in most pairs (narrow windows, P not a multiple of B),
    both forms, against the oracle over every row."""
    H, W, tper = 2, 0, 5
    N = T * P
    p = L.Params(window=W, tper=tper)
    _say(f"[pairs] T={T} P={P} B={B} exact={exact}")
    csr = L.build_mask(T, P, B, 2, p, exact=exact)
    rp, ci = csr.arrays()
    nb = len(rp) - 1
    rows = [set(ci[rp[r]:rp[r + 1]].tolist()) for r in range(nb)] + [set()]
    union = sum(len(rows[2 * q] | rows[2 * q + 1]) for q in range(-(-nb // 2)))
    split = sum(len(rows[2 * q] ^ rows[2 * q + 1]) for q in range(nb // 2))
    assert split > union // 10, (split, union)   # the case is exercised
    q, k, v = make_qkv(H, N, seed=T * 10 + B)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    csr.upload()
    qf, kf, vf = (x.float().numpy() for x in (q, k, v))
    if exact:
        out = L.attention_exact(qd, kd, vd, csr.exact_mask())
        _, _, A = M.attended_frames(T, 2, W=W, tper=tper)
        ref = OA.frame_sparse_attention(qf, kf, vf, A, P)
    else:
        out = L.attention(qd, kd, vd, csr.device_mask())
        ref = OA.assemble(OA.block_sparse_attention(qf, kf, vf, rp.tolist(), ci.tolist(), B),
                          H, N, 128, B)
    torch.cuda.synchronize()
    err = np.abs(out.float().cpu().numpy() - ref)
    assert_close(float(err.max()), float(err.mean()))


def _random_csr(nb, rng, min_len=1, max_len=None):
    """A block CSR that no LVSA rule produces: every row a random sorted set
    of key blocks, its length drawn from min_len .. max_len (nb by default),
    rows independent of each other (so the two rows of a pair differ)."""
    max_len = nb if max_len is None else max_len
    row_ptr, col_idx = [0], []
    for _ in range(nb):
        k = int(rng.integers(min_len, max_len + 1))
        col_idx.extend(sorted(rng.choice(nb, size=k, replace=False).tolist()))
        row_ptr.append(len(col_idx))
    return row_ptr, col_idx


@pytest.mark.parametrize("T,P,B,H,seed", [(6, 200, 128, 2, 1), (9, 150, 64, 2, 2),
                                          (20, 512, 128, 3, 3), (7, 190, 128, 1, 4)])
def test_random_csr_matches_oracle(T, P, B, H, seed):
    """Attention over a caller-built CSR (lvsa_attention reads any block CSR):
    rows of 1 to nb blocks, the two rows of a pair different, a ragged last
    block; every row against the oracle."""
    N = T * P
    nb = -(-N // B)
    rng = np.random.default_rng(seed)
    rp, ci = _random_csr(nb, rng)
    lens = np.diff(rp)
    assert lens.min() >= 1 and lens.max() <= nb
    _say(f"[random-csr] T={T} P={P} B={B} H={H} nb={nb} nnz={len(ci)}")
    q, k, v = make_qkv(H, N, seed=100 + seed)
    rpd = torch.tensor(rp, dtype=torch.int32, device="cuda")
    cid = torch.tensor(ci, dtype=torch.int32, device="cuda")
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), L.csr_mask(rpd, cid, N, B))
    torch.cuda.synchronize()
    ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                v.float().numpy(), rp, ci, B), H, N, 128, B)
    err = np.abs(out.float().cpu().numpy() - ref)
    assert_close(float(err.max()), float(err.mean()))


def test_random_csr_one_block_rows_and_full_rows():
    """Extremes of a caller CSR: every even row keeps one block, every odd row
    keeps all nb, so each pair walks nb blocks of which one is shared."""
    T, P, B, H = 8, 256, 128, 2
    N = T * P
    nb = N // B
    rng = np.random.default_rng(7)
    rp, ci = [0], []
    for r in range(nb):
        cols = [int(rng.integers(0, nb))] if r % 2 == 0 else list(range(nb))
        ci.extend(cols)
        rp.append(len(ci))
    _say("[random-csr] one-block and full rows")
    q, k, v = make_qkv(H, N, seed=71)
    m = L.csr_mask(torch.tensor(rp, dtype=torch.int32, device="cuda"),
                   torch.tensor(ci, dtype=torch.int32, device="cuda"), N, B)
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), m)
    torch.cuda.synchronize()
    ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                v.float().numpy(), rp, ci, B), H, N, 128, B)
    err = np.abs(out.float().cpu().numpy() - ref)
    assert_close(float(err.max()), float(err.mean()))


def test_csr_at_the_block_limit():
    """nb = 8000 key blocks (B = 64), the most the sparse kernels take: rows 0
    and 1 keep every block (their merged walk fills the 8000-word LDS array
    over 16 merge passes), the last pair keeps different blocks in each row,
    the others keep the diagonal and two random blocks; sampled query blocks
    against the oracle."""
    B, H, nb = 64, 1, 8000
    N = nb * B - 19                     # ragged last block
    rng = np.random.default_rng(8000)
    rp, ci = [0], []
    for r in range(nb):
        if r < 2:
            cols = list(range(nb))
        elif r >= nb - 2:
            cols = sorted({r, int(rng.integers(0, nb)), (r * 37) % nb, 5 * (r % 2)})
        else:
            cols = sorted({r, int(rng.integers(0, nb)), int(rng.integers(0, nb))})
        ci.extend(cols)
        rp.append(len(ci))
    _say(f"[csr-limit] N={N} B={B} nb={nb} nnz={len(ci)}")
    g = torch.Generator(device="cpu")
    g.manual_seed(80)
    q, k, v = (torch.randn((H, N, 128), generator=g).to(torch.bfloat16) for _ in range(3))
    m = L.csr_mask(torch.tensor(rp, dtype=torch.int32, device="cuda"),
                   torch.tensor(ci, dtype=torch.int32, device="cuda"), N, B)
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), m)
    torch.cuda.synchronize()
    assert_close(*compare_rows(out, q, k, v, rp, ci, B, [0], [0, 1, 2, 4001, nb - 2, nb - 1]))


def test_empty_rows_give_zeros():
    """A query block whose CSR row is empty gets zeros; its pair partner is
    unaffected."""
    T, P, B, H = 4, 256, 128, 1
    N = T * P
    nb = N // B
    rp, ci = [0], []
    for r in range(nb):
        cols = [] if r in (2, 5, 6) else [r]
        ci.extend(cols)
        rp.append(len(ci))
    q, k, v = make_qkv(H, N, seed=72)
    m = L.csr_mask(torch.tensor(rp, dtype=torch.int32, device="cuda"),
                   torch.tensor(ci, dtype=torch.int32, device="cuda"), N, B)
    out = L.attention(q.cuda(), k.cuda(), v.cuda(), m).float().cpu().numpy()
    torch.cuda.synchronize()
    for r in (2, 5, 6):
        assert (out[:, r * B:(r + 1) * B] == 0).all()
    keep = [r for r in range(nb) if r not in (2, 5, 6)]
    ref = OA.block_sparse_attention(q.float().numpy(), k.float().numpy(), v.float().numpy(),
                                    rp, ci, B, q_blocks=keep)
    worst = max(float(np.abs(out[0, qb * B:(qb + 1) * B] - r).max())
                for (_, qb), r in ref.items())
    assert worst <= 2e-2


@pytest.mark.parametrize("T,P,B,H", [
    (20, 512, 128, 8),    # 40 pairs x 8 heads = 320 tiles: more tiles than CUs
    (6, 200, 64, 1),      # 10 tiles: fewer tiles than CUs
])
def test_shared_mask_on_two_streams(T, P, B, H):
    """One mask (block and token-exact views of one handle) read by launches
    in flight on two streams at once, without serialising them: both outputs
    equal the oracle, and a third launch on the same mask afterwards is still
    correct (launches write nothing into the mask)."""
    N = T * P
    nb = -(-N // B)
    _say(f"[shared-mask] T={T} P={P} B={B} H={H}: {-(-nb // 2) * H} tiles")
    q, k, v = make_qkv(H, N, seed=T * 7 + P)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    q2 = (q.float() * 0.5).to(torch.bfloat16)
    q2d = q2.cuda()
    p = L.Params(budget_frames=7, window=1)
    csr = L.build_mask(T, P, B, 2, p, exact=True)
    csr.upload()
    torch.cuda.synchronize()
    m, me = csr.device_mask(), csr.exact_mask()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [torch.full_like(qd, float("nan")) for _ in range(4)]
    torch.cuda.synchronize()
    for rep in range(3):
        with torch.cuda.stream(streams[0]):
            L.attention(qd, kd, vd, m, out=outs[0], stream=streams[0])
            L.attention_exact(q2d, kd, vd, me, out=outs[2], stream=streams[0])
        with torch.cuda.stream(streams[1]):
            L.attention_exact(qd, kd, vd, me, out=outs[1], stream=streams[1])
            L.attention(q2d, kd, vd, m, out=outs[3], stream=streams[1])
        torch.cuda.synchronize()
        if rep == 0:
            first = [o.clone() for o in outs]
        else:
            for o, f in zip(outs, first):
                assert torch.equal(o, f)
    third = L.attention(qd, kd, vd, m)
    torch.cuda.synchronize()
    assert torch.equal(third, outs[0])
    rpo, cio = M.build_mask(T, P, B, 2, C=7, W=1)
    qf, kf, vf, q2f = (x.float().numpy() for x in (q, k, v, q2))
    _, _, A = M.attended_frames(T, 2, C=7, W=1)
    for qq, ob, oe in ((qf, outs[0], outs[1]), (q2f, outs[3], outs[2])):
        ref = OA.assemble(OA.block_sparse_attention(qq, kf, vf, rpo, cio, B), H, N, 128, B)
        err = np.abs(ob.float().cpu().numpy() - ref)
        assert_close(float(err.max()), float(err.mean()))
        fref = OA.frame_sparse_attention(qq, kf, vf, A, P)
        err = np.abs(oe.float().cpu().numpy() - fref)
        assert_close(float(err.max()), float(err.mean()))


@pytest.mark.parametrize("nb", [8000, 8100])
def test_dense_at_and_past_the_lds_word_array(nb):
    """Dense attention at the walk's LDS word array capacity (nb = 8000 at
    B = 64: the block-mode kernel without a CSR, every word in LDS) and past
    it (nb = 8100: the dense kernel, whose tiles' last steps take computed
    words); sampled rows against Eq. 1."""
    B, H = 64, 1
    N = nb * B - 37                     # ragged last block
    _say(f"[dense-long] N={N} B={B} nb={nb}")
    g = torch.Generator(device="cpu")
    g.manual_seed(nb)
    q, k, v = (torch.randn((H, N, 128), generator=g).to(torch.bfloat16) for _ in range(3))
    out = L.dense_attention(q.cuda(), k.cuda(), v.cuda(), block=B)
    torch.cuda.synchronize()
    rp = [i * nb for i in range(nb + 1)]
    ci = list(range(nb)) * nb
    assert_close(*compare_rows(out, q, k, v, rp, ci, B, [0], [0, 4000, nb - 1]))
