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
    ptr, words, _ = csr.pairs()
    split = sum(1 for w in words.tolist() if (w >> 30) != 3)
    assert split > len(words) // 10, (split, len(words))   # the case is exercised
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


@pytest.mark.parametrize("T,P,B,H", [
    (20, 512, 128, 8),    # 40 pairs x 8 heads = 320 tiles: more tiles than CUs
    (6, 200, 64, 1),      # 10 tiles: fewer tiles than CUs
])
def test_tile_counters_left_zero_and_results_repeat(T, P, B, H):
    """Workgroups take tiles through counters kept after the pair offsets;
    every launch must leave them zero, so back-to-back launches on one mask
    (block and token-exact forms) give identical outputs, matching the
    oracle."""
    N = T * P
    nb = -(-N // B)
    npairs = (nb + 1) // 2
    _say(f"[counters] T={T} P={P} B={B} H={H}: {npairs * H} tiles")
    q, k, v = make_qkv(H, N, seed=T * 7 + P)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    p = L.Params(budget_frames=7, window=1)
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    pp, pw = L.pair_buffers(N, B)
    ppx, pwx = L.pair_buffers(N, B)
    m = L.build_mask_device(T, P, B, 2, rp, ci, params=p, pair_ptr=pp, pair_word=pw)
    me = L.build_exact_mask_device(T, P, B, 2, rp.clone(), ent, params=p, pair_ptr=ppx,
                                   pair_word=pwx)
    outs, outs_x = [], []
    for _ in range(3):
        outs.append(L.attention(qd, kd, vd, m))
        outs_x.append(L.attention_exact(qd, kd, vd, me))
    torch.cuda.synchronize()
    assert bool((pp[npairs + 1:] == 0).all()) and bool((ppx[npairs + 1:] == 0).all())
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    for o in outs_x[1:]:
        assert torch.equal(o, outs_x[0])
    rpo, cio = M.build_mask(T, P, B, 2, C=7, W=1)
    assert_close(*compare_rows(outs[0], q, k, v, rpo, cio, B, range(H), range(nb)))
