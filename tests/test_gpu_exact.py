"""GPU parity of the token-exact form: lvsa_attention_exact against the fp32
oracle of Eq. 2 token for token (frame_sparse_attention / frame_sparse_rows),
and the device builder's entry words against the host builder's, bit for bit.
Shapes have frames that straddle blocks (P mod B != 0) and ragged last blocks.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS, make_qkv, workload_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import MAX_ABS, MEAN_ABS, assert_close

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


# T, P, B, H, W, T_per: P >= B, P mod B != 0 except the last case.
EXACT_MID = [
    (6, 200, 128, 2, 1, 3),
    (9, 150, 64, 2, 1, 4),
    (5, 257, 128, 1, 0, 5),
    (12, 96, 64, 2, 2, 4),
    (7, 130, 128, 1, 1, 3),
    (6, 256, 128, 1, 1, 3),
]


@pytest.mark.parametrize("T,P,B,H,W,tper", EXACT_MID)
def test_exact_full_output_matches_eq2(T, P, B, H, W, tper):
    _say(f"[exact] T={T} P={P} B={B} H={H} W={W} tper={tper}")
    N = T * P
    q, k, v = make_qkv(H, N, seed=T * 1000 + P)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    qf, kf, vf = (x.float().numpy() for x in (q, k, v))
    for step in (0, 1, 2):
        csr = L.build_mask(T, P, B, step, L.Params(window=W, tper=tper), exact=True)
        csr.upload()
        out = L.attention_exact(qd, kd, vd, csr.exact_mask())
        torch.cuda.synchronize()
        _, _, A = M.attended_frames(T, step, W=W, tper=tper)
        ref = OA.frame_sparse_attention(qf, kf, vf, A, P)
        g = out.float().cpu().numpy()
        assert np.isfinite(g).all()
        err = np.abs(g - ref)
        assert_close(float(err.max()), float(err.mean()))


def test_exact_equals_block_mode_when_block_divides_frame():
    """P mod B = 0: every kept block is whole, so the two forms attend the
    same keys with the same scores and probabilities.  They keep the row sums
    differently (fp32 adds of the probabilities in the block form, matrix-core
    sums of their bf16 values in the token-exact form), which moves the
    normalised output by far less than half a bf16 unit: the two agree to one
    unit in the last place of bf16."""
    w = WORKLOADS["tiny"]
    q, k, v = (x.cuda() for x in workload_qkv(w))
    for step in w.steps:
        csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, step,
                           L.Params(budget_frames=w.budget_frames, window=w.window,
                                    tper=w.tper), exact=True)
        csr.upload()
        a = L.attention(q, k, v, csr.device_mask())
        b = L.attention_exact(q, k, v, csr.exact_mask())
        torch.cuda.synchronize()
        af, bf = a.float(), b.float()
        assert bool(((af - bf).abs() <= af.abs() * 2.0 ** -7 + 1e-7).all())
        assert float((af - bf).abs().mean()) < 1e-5


def _sample_rows(w, csr_rp, n_random=6, seed=1):
    """Query tokens on both sides of frame edges inside straddling blocks,
    the first and last token, and seeded random tokens."""
    N, P, B = w.n_tokens, w.tokens_per_frame, w.block
    rows = {0, N - 1}
    for t in (1, w.frames // 2, w.frames - 1):
        edge = t * P
        if edge % B:
            rows |= {edge - 1, edge, (edge // B) * B, min((edge // B + 1) * B, N) - 1}
    rng = np.random.default_rng(seed)
    rows |= {int(x) for x in rng.integers(0, N, size=n_random)}
    return sorted(rows)


@pytest.mark.parametrize("name", ["wan13_6x", "hv15_2x", "wan13_1x"])
def test_exact_full_size_sampled_rows(name):
    """The whole workload in one launch, checked on sampled query tokens of a
    few heads against Eq. 2 row by row."""
    w = WORKLOADS[name]
    _say(f"[exact-full] {name}: generating inputs")
    q, k, v = workload_qkv(w)
    step = 10
    p = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper)
    csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, step, p, exact=True)
    csr.upload()
    _say(f"[exact-full] {name}: launch step {step}")
    out = L.attention_exact(q.cuda(), k.cuda(), v.cuda(), csr.exact_mask())
    torch.cuda.synchronize()
    _, _, A = M.attended_frames(w.frames, step, C=w.budget_frames, W=w.window,
                                tper=w.tper)
    rows = _sample_rows(w, csr.arrays()[0])
    heads = sorted({0, w.heads - 1})
    _say(f"[exact-full] {name}: oracle on heads {heads}, {len(rows)} rows")
    ref = OA.frame_sparse_rows(q.float().numpy(), k.float().numpy(), v.float().numpy(),
                               A, w.tokens_per_frame, heads, rows)
    worst, total, count = 0.0, 0.0, 0
    for h in heads:
        g = out[h, rows].float().cpu().numpy()
        assert np.isfinite(g).all()
        err = np.abs(g - ref[h])
        worst = max(worst, float(err.max()))
        total += float(err.sum())
        count += err.size
    assert_close(worst, total / count)


@pytest.mark.parametrize("name", ["wan13_6x", "hv15_2x", "tiny"])
def test_device_exact_builder_matches_host(name):
    w = WORKLOADS[name]
    T, P, B = w.frames, w.tokens_per_frame, w.block
    nb = w.n_blocks
    p = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper)
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ent = torch.full((nb * nb,), -1, dtype=torch.int32, device="cuda")
    for step in (0, 3, 10):
        _say(f"[exact-builder] {name} step {step}")
        ent.fill_(-1)
        L.build_exact_mask_device(T, P, B, step, rp, ent, p)
        torch.cuda.synchronize()
        csr = L.build_mask(T, P, B, step, p, exact=True)
        hrp, _ = csr.arrays()
        he = csr.entries()
        assert np.array_equal(rp.cpu().numpy(), hrp)
        got = ent[:int(hrp[-1])].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, he)
        assert bool((ent[int(hrp[-1]):] == -1).all())   # nothing written past nnz


def test_exact_with_device_built_mask_and_determinism():
    """Attention over the device-built entry words equals attention over the
    uploaded host words, bit for bit, and reruns are bitwise equal."""
    T, P, B, H = 8, 300, 128, 2
    N = T * P
    q, k, v = (x.cuda() for x in make_qkv(H, N, seed=77))
    p = L.Params(window=1, tper=3)
    nb = -(-N // B)
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    m = L.build_exact_mask_device(T, P, B, 4, rp, ent, p)
    a = L.attention_exact(q, k, v, m)
    csr = L.build_mask(T, P, B, 4, p, exact=True)
    csr.upload()
    b = L.attention_exact(q, k, v, csr.exact_mask())
    c = L.attention_exact(q, k, v, csr.exact_mask())
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(b, c)
    assert MAX_ABS > 0 and MEAN_ABS > 0


def test_exact_strided_layout_matches_contiguous():
    """[N, H, d] storage (token stride H*d) gives the same bits as [H, N, d]
    for the token-exact form too."""
    T, P, B, H = 5, 300, 128, 3
    N = T * P
    q, k, v = make_qkv(H, N, seed=19)
    csr = L.build_mask(T, P, B, 2, L.Params(window=1, tper=2), exact=True)
    csr.upload()
    a = L.attention_exact(q.cuda(), k.cuda(), v.cuda(), csr.exact_mask())
    qn, kn, vn = (x.transpose(0, 1).contiguous().cuda().transpose(0, 1) for x in (q, k, v))
    on = torch.empty((N, H, 128), dtype=torch.bfloat16, device="cuda").transpose(0, 1)
    b = L.attention_exact(qn, kn, vn, csr.exact_mask(), out=on)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
