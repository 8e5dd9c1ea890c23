"""GPU parity: the device mask builder's CSR equals the oracle's bit for bit,
and attention over it equals attention over the host-built CSR bit for bit."""
import random
import sys

import pytest
import torch

import numpy as np

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import WORKLOADS, make_qkv
from oracle import attention as OA
from oracle import mask as M
from tests.gpu_util import assert_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


def _device_csr(T, P, B, step, p, layer=0):
    nb = -(-(T * P + p.text_tokens) // B)
    rp = torch.full((nb + 1,), -1, dtype=torch.int32, device="cuda")
    ci = torch.full((nb * nb,), -1, dtype=torch.int32, device="cuda")
    L.build_mask_device(T, P, B, step, rp, ci, params=p, layer=layer)
    torch.cuda.synchronize()
    rp = rp.cpu()
    nnz = int(rp[-1])
    return rp.tolist(), ci[:nnz].cpu().tolist(), ci


def _kw(p):
    return dict(C=p.budget_frames, W=p.window, tper=p.tper, mode=p.window_mode,
                rotate=bool(p.rotate), tie_high=bool(p.tie_high), extra=p.extra_anchors,
                text=p.text_tokens)


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_device_builder_matches_oracle_workloads(name):
    w = WORKLOADS[name]
    p = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper,
                 text_tokens=w.text_tokens)
    steps = list(w.steps) if len(w.steps) > 1 else [0, 1, 10, 17]
    print(f"[mask] {name} steps {steps[0]}..{steps[-1]}", flush=True)
    for s in steps:
        for layer in w.layers:
            rp, ci, raw = _device_csr(w.frames, w.tokens_per_frame, w.block, s, p, layer)
            want_rp, want_ci = M.build_mask(w.frames, w.tokens_per_frame, w.block, s,
                                            layer=layer, **_kw(p))
            assert rp == want_rp, (name, s, layer)
            assert ci == want_ci, (name, s, layer)
            # nothing written past nnz
            assert bool((raw[len(ci):] == -1).all())


@pytest.mark.parametrize("mode", [L.WINDOW_BASIC, L.WINDOW_ADAPTIVE, L.WINDOW_EXPANDED])
def test_device_builder_matches_oracle_random(mode):
    rng = random.Random(77 + mode)
    print(f"[mask] random mode {mode}", flush=True)
    for _ in range(40):
        T = rng.randint(1, 60)
        # periods beyond T too (one anchor, (s mod T_per) mod T)
        p = L.Params(window=rng.randint(0, 6), tper=rng.randint(1, 3 * T), window_mode=mode,
                     rotate=rng.randint(0, 1), tie_high=rng.randint(0, 1),
                     extra_anchors=rng.choice([0, 0, 1, 3]))
        P = rng.randint(1, 300)
        B = rng.choice([1, 3, 16, 64, 128])
        if -(-(T * P) // B) > 1500:
            B = 64
        s = rng.randint(0, 3 * p.tper)
        rp, ci, _ = _device_csr(T, P, B, s, p)
        want_rp, want_ci = M.build_mask(T, P, B, s, **_kw(p))
        assert rp == want_rp and ci == want_ci, (T, P, B, s)


def test_device_mask_attention_equals_host_mask_attention():
    T, P, B, H = 9, 333, 128, 2
    print("[mask] device-CSR attention vs host-CSR attention", flush=True)
    q, k, v = (x.cuda() for x in make_qkv(H, T * P, seed=3))
    p = L.Params(budget_frames=7, window=1)
    for s in (0, 1, 2):
        csr = L.build_mask(T, P, B, s, p)
        csr.upload()
        a = L.attention(q, k, v, csr.device_mask())
        nb = -(-(T * P) // B)
        rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
        ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
        m = L.build_mask_device(T, P, B, s, rp, ci, params=p)
        b = L.attention(q, k, v, m)
        torch.cuda.synchronize()
        assert torch.equal(a, b)


# Window rule, anchor rotation and dedicated initial anchors (the pattern
# variants of Sec. 2 and the generalization named after Def. 2).
VARIANTS = [
    (L.WINDOW_BASIC, 1, 0), (L.WINDOW_ADAPTIVE, 1, 0), (L.WINDOW_EXPANDED, 1, 0),
    (L.WINDOW_EXPANDED, 0, 0), (L.WINDOW_BASIC, 0, 0), (L.WINDOW_EXPANDED, 1, 1),
    (L.WINDOW_EXPANDED, 1, 2),
]


@pytest.mark.parametrize("mode,rotate,extra", VARIANTS)
def test_pattern_variant_attention_parity(mode, rotate, extra):
    """Block form against the block oracle and token-exact form against Eq. 2,
    on a straddling shape with a ragged last block, for each pattern variant;
    the device builder equals the oracle for the variant's CSR."""
    T, P, B, H = 10, 200, 128, 2
    N = T * P
    print(f"[pattern] mode {mode} rotate {rotate} extra {extra}", flush=True)
    q, k, v = make_qkv(H, N, seed=40 + mode)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    qf, kf, vf = (x.float().numpy() for x in (q, k, v))
    p = L.Params(window=1, tper=3, window_mode=mode, rotate=rotate, extra_anchors=extra)
    for s in (1, 2):
        kw = _kw(p)
        rp, ci = M.build_mask(T, P, B, s, **kw)
        drp, dci, _ = _device_csr(T, P, B, s, p)
        assert drp == rp and dci == ci
        csr = L.build_mask(T, P, B, s, p, exact=True)
        csr.upload()
        blk = L.attention(qd, kd, vd, csr.device_mask())
        ex = L.attention_exact(qd, kd, vd, csr.exact_mask())
        torch.cuda.synchronize()
        ref = OA.assemble(OA.block_sparse_attention(qf, kf, vf, rp, ci, B), H, N, 128, B)
        err = np.abs(blk.float().cpu().numpy() - ref)
        assert_close(float(err.max()), float(err.mean()))
        _, _, A = M.attended_frames(T, s, W=1, tper=3, mode=mode, rotate=bool(rotate),
                                    extra=extra)
        fref = OA.frame_sparse_attention(qf, kf, vf, A, P)
        err = np.abs(ex.float().cpu().numpy() - fref)
        assert_close(float(err.max()), float(err.mean()))


def test_pattern_variants_full_size_sampled_rows():
    """The five pattern variants the bench times, at the full Wan-1.3B 6x
    shape in one launch each, checked on sampled query blocks of two heads."""
    from paper_2605_31057_amd.inputs import WORKLOADS, workload_qkv
    from tests.gpu_util import compare_rows, sample_q_blocks
    w = WORKLOADS["wan13_6x"]
    print("[pattern-full] generating inputs", flush=True)
    q, k, v = workload_qkv(w, heads=2)
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    for mode, rotate, extra in [(L.WINDOW_EXPANDED, 1, 0), (L.WINDOW_ADAPTIVE, 1, 0),
                                (L.WINDOW_BASIC, 1, 0), (L.WINDOW_EXPANDED, 0, 0),
                                (L.WINDOW_EXPANDED, 1, 1)]:
        print(f"[pattern-full] mode {mode} rotate {rotate} extra {extra}", flush=True)
        p = L.Params(window_mode=mode, rotate=rotate, extra_anchors=extra)
        csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, 10, p)
        csr.upload()
        out = L.attention(qd, kd, vd, csr.device_mask())
        torch.cuda.synchronize()
        rp, ci = M.build_mask(w.frames, w.tokens_per_frame, w.block, 10, **_kw(p))
        assert csr.arrays()[0].tolist() == rp
        qbs = sample_q_blocks(rp, w.frames, w.tokens_per_frame, w.block, n_random=1)
        assert_close(*compare_rows(out, q, k, v, rp, ci, w.block, [0, 1], qbs))
