"""GPU parity with text tokens after the video tokens (a dual-stream model,
whose text-encoder tokens join self-attention): block and token-exact forms
against the oracle, ragged text lengths, the HunyuanVideo 1.5 2x layer with
512 text tokens, and the device builders against the host builders."""
import sys

import numpy as np
import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS, make_qkv, workload_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import assert_close

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


# T, P, B, H, text length: ragged lengths (shorter than, equal to, longer
# than a block), a block-aligned video end and a straddling one.
TEXT_MID = [
    (6, 200, 128, 2, 77),
    (9, 150, 64, 2, 300),
    (5, 256, 128, 1, 128),
    (7, 130, 128, 1, 1),
    (4, 300, 128, 2, 513),
]


def _errs(got, ref):
    g = got.float().cpu().numpy()
    assert np.isfinite(g).all()
    err = np.abs(g - ref)
    return float(err.max()), float(err.mean())


@pytest.mark.parametrize("T,P,B,H,Lt", TEXT_MID)
def test_text_full_output(T, P, B, H, Lt):
    _say(f"[text] T={T} P={P} B={B} H={H} L={Lt}")
    N = T * P + Lt
    q, k, v = make_qkv(H, N, seed=T * 100 + Lt)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    qf, kf, vf = (x.float().numpy() for x in (q, k, v))
    p = L.Params(window=1, tper=3, text_tokens=Lt)
    for step in (0, 1):
        csr = L.build_mask(T, P, B, step, p, exact=True)
        csr.upload()
        blk = L.attention(qd, kd, vd, csr.device_mask())
        ex = L.attention_exact(qd, kd, vd, csr.exact_mask())
        torch.cuda.synchronize()
        rp, ci = M.build_mask(T, P, B, step, W=1, tper=3, text=Lt)
        ref = OA.assemble(OA.block_sparse_attention(qf, kf, vf, rp, ci, B), H, N, 128, B)
        assert_close(*_errs(blk, ref))
        _, _, A = M.attended_frames(T, step, W=1, tper=3)
        rows = list(range(N))
        tref = OA.text_sparse_rows(qf, kf, vf, A, T, P, range(H), rows)
        assert_close(*_errs(ex, np.stack([tref[h] for h in range(H)])))


def test_text_full_size_sampled_rows():
    """HunyuanVideo 1.5 2x layer with 512 text tokens in one launch per form,
    checked on video rows, rows at the video/text boundary and text rows."""
    w = WORKLOADS["hv15_2x_text"]
    T, P, B, Lt = w.frames, w.tokens_per_frame, w.block, w.text_tokens
    V = T * P
    _say("[text-full] generating inputs")
    q, k, v = workload_qkv(w)
    p = L.Params(budget_frames=w.budget_frames, window=w.window, text_tokens=Lt)
    step = 10
    csr = L.build_mask(T, P, B, step, p, exact=True)
    csr.upload()
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    _say("[text-full] launches")
    blk = L.attention(qd, kd, vd, csr.device_mask())
    ex = L.attention_exact(qd, kd, vd, csr.exact_mask())
    torch.cuda.synchronize()
    _, _, A = M.attended_frames(T, step, C=w.budget_frames, W=w.window)
    rows = sorted({0, P - 1, P, V // 2, V - 129, V - 1, V, V + 1, V + Lt // 2,
                   w.n_tokens - 1})
    heads = [0, w.heads - 1]
    qf, kf, vf = (x[heads].float().numpy() for x in (q, k, v))
    _say(f"[text-full] oracle on heads {heads}, {len(rows)} rows")
    tref = OA.text_sparse_rows(qf, kf, vf, A, T, P, range(len(heads)), rows)
    rp, ci = csr.arrays()
    qbs = sorted({r // B for r in rows})
    bref = OA.block_sparse_attention(qf, kf, vf, rp, ci, B, q_blocks=qbs)
    worst_e = worst_b = 0.0
    tot_e = tot_b = 0.0
    cnt = 0
    for hi, h in enumerate(heads):
        g = ex[h, rows].float().cpu().numpy()
        e = np.abs(g - tref[hi])
        worst_e, tot_e = max(worst_e, float(e.max())), tot_e + float(e.sum())
        for r in rows:
            qb = r // B
            gb = blk[h, r].float().cpu().numpy()
            eb = np.abs(gb - bref[(hi, qb)][r - qb * B])
            worst_b, tot_b = max(worst_b, float(eb.max())), tot_b + float(eb.sum())
        cnt += g.size
    assert_close(worst_e, tot_e / cnt)
    assert_close(worst_b, tot_b / cnt)


@pytest.mark.parametrize("Lt", [1, 77, 512, 1000])
def test_text_device_builders_match_host(Lt):
    T, P, B = 65, 1590, 128
    N = T * P + Lt
    nb = -(-N // B)
    p = L.Params(budget_frames=33, window=6, text_tokens=Lt)
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.full((nb * nb,), -1, dtype=torch.int32, device="cuda")
    ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    for step in (0, 10):
        _say(f"[text-builder] L={Lt} step {step}")
        csr = L.build_mask(T, P, B, step, p, exact=True)
        hrp, hci = csr.arrays()
        L.build_mask_device(T, P, B, step, rp, ci, params=p)
        torch.cuda.synchronize()
        assert np.array_equal(rp.cpu().numpy(), hrp)
        assert np.array_equal(ci[:len(hci)].cpu().numpy(), hci)
        assert bool((ci[len(hci):] == -1).all())
        L.build_exact_mask_device(T, P, B, step, rp, ent, params=p)
        torch.cuda.synchronize()
        assert np.array_equal(rp.cpu().numpy(), hrp)
        assert np.array_equal(ent[:len(hci)].cpu().numpy().view(np.uint32), csr.entries())
