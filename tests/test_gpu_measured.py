"""GPU parity of every launch the benchmark times, at its full shape: one
launch over all heads, checked against the fp32 oracle on sampled query
blocks (first, last/ragged, first straddling a frame edge, most and fewest
kept blocks, seeded random ones) of two or three heads including the last.

  * dense attention (Eq. 1) through the block-sparse kernel with a full mask
    at the Wan-1.3B 6x and HunyuanVideo 2x (+ text) shapes;
  * lvsa_dense_attention at the Wan-14B 6x shape (40 heads), the dense
    baseline of that workload;
  * the block form at the HunyuanVideo 2x mask with the C = 21 budget;
  * the token-exact form (Eq. 2 token for token) at the Wan-14B 6x shape.
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

_INPUTS = {}


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()
    yield
    _INPUTS.clear()
    torch.cuda.empty_cache()


def _inputs(name):
    """(q, k, v) on the host and on the device for workload `name`; one
    workload is kept at a time."""
    if name not in _INPUTS:
        _INPUTS.clear()
        torch.cuda.empty_cache()
        _say(f"[measured] {name}: generating inputs")
        cpu = workload_qkv(WORKLOADS[name])
        _INPUTS[name] = (cpu, tuple(x.cuda() for x in cpu))
    return _INPUTS[name]


def _full_csr(nb):
    return [i * nb for i in range(nb + 1)], list(range(nb)) * nb


@pytest.mark.parametrize("name", ["wan13_6x", "hv15_2x_text"])
def test_full_mask_block_launch(name):
    """Dense attention through the block-sparse kernel (a window of T frames
    keeps every block), the bench's second dense timing, against Eq. 1."""
    w = WORKLOADS[name]
    (q, k, v), (qd, kd, vd) = _inputs(name)
    nb = w.n_blocks
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    full = L.Params(budget_frames=w.budget_frames, window=w.frames, tper=w.frames,
                    text_tokens=w.text_tokens)
    m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, 10, rp, ci, params=full)
    _say(f"[measured] {name}: full-mask block launch")
    out = L.attention(qd, kd, vd, m)
    torch.cuda.synchronize()
    assert int(rp[-1]) == nb * nb
    frp, fci = _full_csr(nb)
    qbs = sample_q_blocks(frp, w.frames, w.tokens_per_frame, w.block)
    heads = [0, w.heads - 1]
    _say(f"[measured] {name}: oracle (Eq. 1) on heads {heads} q-blocks {qbs}")
    assert_close(*compare_rows(out, q, k, v, frp, fci, w.block, heads, qbs))


def test_dense_entry_point_wan14_6x():
    """lvsa_dense_attention over all 40 heads of the Wan-14B 6x layer."""
    w = WORKLOADS["wan14_6x"]
    (q, k, v), (qd, kd, vd) = _inputs("wan14_6x")
    _say("[measured] wan14_6x: dense launch")
    out = L.dense_attention(qd, kd, vd, block=w.block)
    torch.cuda.synchronize()
    nb = w.n_blocks
    frp, fci = _full_csr(nb)
    qbs = sample_q_blocks(frp, w.frames, w.tokens_per_frame, w.block, n_random=1)
    heads = [0, 20, 39]
    _say(f"[measured] wan14_6x: oracle (Eq. 1) on heads {heads} q-blocks {qbs}")
    assert_close(*compare_rows(out, q, k, v, frp, fci, w.block, heads, qbs))


def test_exact_form_wan14_6x():
    """Token-exact attention over all 40 heads of the Wan-14B 6x layer against
    Eq. 2 row by row."""
    w = WORKLOADS["wan14_6x"]
    (q, k, v), (qd, kd, vd) = _inputs("wan14_6x")
    p = L.Params(budget_frames=w.budget_frames, window=w.window)
    csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, 10, p, exact=True)
    csr.upload()
    _say("[measured] wan14_6x: token-exact launch")
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
    heads = [0, 20, 39]
    _say(f"[measured] wan14_6x: oracle (Eq. 2) on heads {heads}, {len(rows)} rows")
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


def test_block_form_hv15_2x_c21():
    """The block form at the HunyuanVideo 2x shape with the C = 21 budget."""
    w = WORKLOADS["hv15_2x_c21"]
    (q, k, v), (qd, kd, vd) = _inputs("hv15_2x_c21")
    p = L.Params(budget_frames=w.budget_frames, window=w.window)
    nb = w.n_blocks
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    for step in w.steps:
        m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, step, rp, ci, params=p)
        _say(f"[measured] hv15_2x_c21: block launch step {step}")
        out = L.attention(qd, kd, vd, m)
        torch.cuda.synchronize()
        orp, oci = oracle_csr(w, step)
        assert rp.cpu().tolist() == orp
        qbs = sample_q_blocks(orp, w.frames, w.tokens_per_frame, w.block)
        heads = [0, w.heads - 1]
        assert_close(*compare_rows(out, q, k, v, orp, oci, w.block, heads, qbs))
