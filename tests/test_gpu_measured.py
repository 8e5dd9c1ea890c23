"""GPU parity of every launch the benchmark times, at its full shape: one
launch over all heads, checked against the fp32 oracle on sampled query
blocks (first, last/ragged, first straddling a frame edge, most and fewest
kept blocks, seeded random ones) or sampled rows, of two or three heads
including the last.  One test per workload, so each workload's inputs are
drawn once:

  * at every workload, both dense timings: lvsa_dense_attention and the
    block-sparse kernel with a full mask (a window of T frames keeps every
    block), against Eq. 1;
  * the token-exact form (Eq. 2 token for token) at the Wan-14B 6x shape and
    at the HunyuanVideo 2x shape with the C = 21 budget;
  * the block form at the HunyuanVideo 2x mask with the C = 21 budget.

The other timed launches (the block form at the remaining workloads and
steps, the token-exact form at Wan-1.3B 6x, HunyuanVideo 2x and Wan 1x, both
forms with text tokens, the pattern variants) are checked in
test_gpu_attention.py, test_gpu_exact.py, test_gpu_text.py and
test_gpu_mask.py.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS, workload_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import assert_close, compare_rows, oracle_csr, sample_q_blocks

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()
    yield
    torch.cuda.empty_cache()


def _full_csr(nb):
    return [i * nb for i in range(nb + 1)], list(range(nb)) * nb


def _heads(w):
    return [0, w.heads // 2, w.heads - 1] if w.heads > 16 else [0, w.heads - 1]


def _dense_timings(name, w, q, k, v, qd, kd, vd):
    """lvsa_dense_attention and the full-mask block launch against Eq. 1."""
    nb = w.n_blocks
    frp, fci = _full_csr(nb)
    qbs = sample_q_blocks(frp, w.frames, w.tokens_per_frame, w.block,
                          n_random=1 if w.heads > 16 else 2)
    heads = _heads(w)
    _say(f"[measured] {name}: dense entry point")
    out = L.dense_attention(qd, kd, vd, block=w.block)
    torch.cuda.synchronize()
    _say(f"[measured] {name}: oracle (Eq. 1) on heads {heads} q-blocks {qbs}")
    assert_close(*compare_rows(out, q, k, v, frp, fci, w.block, heads, qbs))
    del out
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    full = L.Params(budget_frames=w.budget_frames, window=w.frames, tper=w.frames,
                    text_tokens=w.text_tokens)
    m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, 10, rp, ci, params=full)
    _say(f"[measured] {name}: full-mask block launch")
    out = L.attention(qd, kd, vd, m)
    torch.cuda.synchronize()
    assert int(rp[-1]) == nb * nb
    assert_close(*compare_rows(out, q, k, v, frp, fci, w.block, heads, qbs))


def _exact_form(name, w, q, k, v, qd, kd, vd):
    """Token-exact attention at step 10 against Eq. 2 on sampled rows (both
    sides of frame edges inside straddling blocks, first and last rows,
    seeded random rows)."""
    p = L.Params(budget_frames=w.budget_frames, window=w.window)
    csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, 10, p, exact=True)
    csr.upload()
    _say(f"[measured] {name}: token-exact launch")
    out = L.attention_exact(qd, kd, vd, csr.exact_mask())
    torch.cuda.synchronize()
    _, _, A = M.attended_frames(w.frames, 10, C=w.budget_frames, W=w.window)
    N, P, B = w.n_tokens, w.tokens_per_frame, w.block
    rows = {0, N - 1}
    for t in (1, 13, w.frames // 2, w.frames - 1):
        edge = t * P
        rows |= {edge - 1, edge, (edge // B) * B, min((edge // B + 1) * B, N) - 1}
    rows |= {int(x) for x in np.random.default_rng(5).integers(0, N, size=6)}
    rows = sorted(rows)
    heads = _heads(w)
    _say(f"[measured] {name}: oracle (Eq. 2) on heads {heads}, {len(rows)} rows")
    ref = OA.frame_sparse_rows(q.float().numpy(), k.float().numpy(), v.float().numpy(),
                               A, P, heads, rows)
    worst, total, count = 0.0, 0.0, 0
    for h in heads:
        g = out[h, rows].float().cpu().numpy()
        assert np.isfinite(g).all()
        err = np.abs(g - ref[h])
        worst = max(worst, float(err.max()))
        total += float(err.sum())
        count += err.size
    assert_close(worst, total / count)


def _block_form(name, w, q, k, v, qd, kd, vd):
    """The block form over the device-built mask of every swept step."""
    p = L.Params(budget_frames=w.budget_frames, window=w.window)
    nb = w.n_blocks
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    for step in w.steps:
        m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, step, rp, ci, params=p)
        _say(f"[measured] {name}: block launch step {step}")
        out = L.attention(qd, kd, vd, m)
        torch.cuda.synchronize()
        orp, oci = oracle_csr(w, step)
        assert rp.cpu().tolist() == orp
        qbs = sample_q_blocks(orp, w.frames, w.tokens_per_frame, w.block)
        assert_close(*compare_rows(out, q, k, v, orp, oci, w.block, _heads(w), qbs))


MEASURED = {
    "wan13_6x": (_dense_timings,),
    "hv15_2x_text": (_dense_timings,),
    "wan14_6x": (_dense_timings, _exact_form),
    "hv15_2x": (_dense_timings,),
    "hv15_2x_c21": (_dense_timings, _exact_form, _block_form),
    "wan13_1x": (_dense_timings,),
}


@pytest.mark.parametrize("name", list(MEASURED))
def test_measured_launches(name):
    w = WORKLOADS[name]
    _say(f"[measured] {name}: generating inputs")
    q, k, v = workload_qkv(w)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    for check in MEASURED[name]:
        check(name, w, q, k, v, qd, kd, vd)
    del qd, kd, vd
    torch.cuda.empty_cache()
