"""The allocation-free entry point (lvsa_attention_noalloc), called through
the C ABI: its output equals lvsa_attention's bit for bit (the same kernels
over the same mask), on two calls in a row, the second with a smaller input,
and both match the fp32 oracle."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import make_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import assert_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


def _noalloc(q, k, v, mask, out):
    tq, tk, tv, to = (L._tensor(x) for x in (q, k, v, out))
    st = L.lib().lvsa_attention_noalloc(ctypes.byref(tq), ctypes.byref(tk), ctypes.byref(tv),
                                        ctypes.byref(mask), ctypes.byref(to),
                                        L._stream_ptr(None))
    assert st == L.OK, L.lib().lvsa_status_str(st)
    return out


def test_noalloc_equals_attention_on_two_calls():
    p = L.Params(budget_frames=7, window=1)
    # (T, P, B, H): the second call is smaller (fewer tiles, fewer tokens)
    for T, P, B, H in ((20, 512, 128, 4), (6, 200, 64, 1)):
        print(f"[noalloc] T={T} P={P} B={B} H={H}", flush=True)
        sys.stdout.flush()
        N = T * P
        q, k, v = make_qkv(H, N, seed=T + P)
        qd, kd, vd = (x.cuda() for x in (q, k, v))
        csr = L.build_mask(T, P, B, 3, p)
        csr.upload()
        mask = csr.device_mask()
        got = _noalloc(qd, kd, vd, mask, torch.full_like(qd, float("nan")))
        want = L.attention(qd, kd, vd, mask)
        torch.cuda.synchronize()
        assert torch.equal(got, want)
        rp, ci = M.build_mask(T, P, B, 3, C=7, W=1)
        ref = OA.assemble(OA.block_sparse_attention(q.float().numpy(), k.float().numpy(),
                                                    v.float().numpy(), rp, ci, B), H, N, 128, B)
        err = np.abs(got.float().cpu().numpy() - ref)
        assert_close(float(err.max()), float(err.mean()))


def test_noalloc_rejects_before_launch():
    lib = L.lib()
    ref = ctypes.byref
    t = L._Tensor(0x10000, 2, 1000, 128, 128000, 128)
    o = L._Tensor(0x40000, 2, 1000, 128, 128000, 128)
    nb = -(-1000 // 128)
    assert lib.lvsa_attention_noalloc(ref(t), ref(t), ref(t),
                                      ref(L.BlockMask(1000, 128, nb, nb, 0, 0x3000)),
                                      ref(o), None) == L.EINVAL
    big = L.BlockMask(8001 * 128, 128, 8001, 8001, 0x2000, 0x3000)
    tb = L._Tensor(0x10000, 1, 8001 * 128, 128, 8001 * 128 * 128, 128)
    ob = L._Tensor(0x40000, 1, 8001 * 128, 128, 8001 * 128 * 128, 128)
    assert lib.lvsa_attention_noalloc(ref(tb), ref(tb), ref(tb), ref(big), ref(ob),
                                      None) == L.EUNSUPPORTED
