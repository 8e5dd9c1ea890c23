"""One denoising step of the hot path (device mask build + block-sparse
attention, and the token-exact pair) captured in a HIP graph: every replay,
with eager work and new input values between replays, gives the bits the
eager calls give.  No entry point memsets, and a captured launch keeps its
tile counters (zeroed by a kernel node on every replay), so a step can be
captured and replayed without host work."""
import sys

import pytest
import torch

import paper_2605_31057_amd as L
from paper_2605_31057_amd.inputs import make_qkv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    L.lib()


def test_step_in_hip_graph_replays_match_eager():
    T, P, B, H, step = 9, 333, 128, 2, 4
    N = T * P
    nb = -(-N // B)
    print("[graph] capture mask build + attention", flush=True)
    sys.stdout.flush()
    q, k, v = (x.cuda() for x in make_qkv(H, N, seed=31))
    p = L.Params(budget_frames=7, window=1)
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    out_x = torch.empty_like(q)

    def run(stream):
        m = L.build_mask_device(T, P, B, step, rp, ci, params=p, stream=stream)
        L.attention(q, k, v, m, out=out, stream=stream)
        me = L.build_exact_mask_device(T, P, B, step, rp, ent, params=p, stream=stream)
        L.attention_exact(q, k, v, me, out=out_x, stream=stream)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(side)                      # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(torch.cuda.current_stream())
    torch.cuda.synchronize()

    for rep in range(4):
        # eager work between replays: new query values, poisoned outputs
        q.copy_(make_qkv(H, N, seed=100 + rep)[0].cuda())
        out.fill_(float("nan"))
        out_x.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got, got_x = out.clone(), out_x.clone()
        run(torch.cuda.current_stream())   # eager reference on the same inputs
        torch.cuda.synchronize()
        assert torch.equal(got, out), f"replay {rep}: block form differs from eager"
        assert torch.equal(got_x, out_x), f"replay {rep}: exact form differs from eager"
        assert bool(torch.isfinite(got.float()).all())


def test_concurrent_streams_are_independent():
    """Two steps with different masks and inputs in flight on two streams at
    once give the bits each gives alone (the library keeps no global state)."""
    T, P, B, H = 8, 300, 128, 2
    N = T * P
    nb = -(-N // B)
    print("[streams] two concurrent steps", flush=True)
    ins = [tuple(x.cuda() for x in make_qkv(H, N, seed=s)) for s in (51, 52)]
    params = [L.Params(window=1, tper=3), L.Params(window=0, tper=2, window_mode=L.WINDOW_BASIC)]
    bufs = [(torch.empty(nb + 1, dtype=torch.int32, device="cuda"),
             torch.empty(nb * nb, dtype=torch.int32, device="cuda")) for _ in range(2)]
    outs = [torch.empty_like(ins[0][0]) for _ in range(2)]

    def step(i, stream):
        rp, ci = bufs[i]
        m = L.build_mask_device(T, P, B, 3 + i, rp, ci, params=params[i], stream=stream)
        q, k, v = ins[i]
        L.attention(q, k, v, m, out=outs[i], stream=stream)

    alone = []
    for i in range(2):
        step(i, torch.cuda.current_stream())
        torch.cuda.synchronize()
        alone.append(outs[i].clone())
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for _ in range(3):
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        for s in streams:
            s.wait_stream(torch.cuda.current_stream())
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                step(i, streams[i])
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(outs[i], alone[i]), i
