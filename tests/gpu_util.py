"""Helpers shared by the GPU parity tests: run the library, run the oracle on
the same seeded inputs, compare within the stated tolerances."""
import numpy as np

from oracle import attention as OA
from oracle import mask as M

# bf16 output vs the fp32 oracle (the paper fixes no precision; these are the
# stated acceptance bounds for bf16 attention).
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def oracle_csr(w, step, layer=0):
    return M.build_mask(w.frames, w.tokens_per_frame, w.block, step,
                        C=w.budget_frames, W=w.window, tper=w.tper, layer=layer,
                        text=w.text_tokens)


def sample_q_blocks(row_ptr, T, P, B, n_random=2, seed=0):
    """First, last (ragged when B does not divide N), the first block that
    straddles a frame edge, the rows with most and fewest kept blocks, and a
    few seeded random rows."""
    nb = len(row_ptr) - 1
    N = T * P
    counts = np.diff(np.asarray(row_ptr))
    picks = {0, nb - 1, int(np.argmax(counts)), int(np.argmin(counts))}
    for qb in range(nb):
        if (qb * B) // P != (min((qb + 1) * B, N) - 1) // P:
            picks.add(qb)
            break
    rng = np.random.default_rng(seed)
    picks |= {int(x) for x in rng.integers(0, nb, size=n_random)}
    return sorted(picks)


def compare_rows(out, q, k, v, row_ptr, col_idx, block, heads, q_blocks):
    """Max/mean abs error of out (device bf16 [H,N,d]) against the fp32 oracle
    on the given heads and query blocks.  Returns (max_abs, mean_abs)."""
    worst, total, count = 0.0, 0.0, 0
    for h in heads:
        qh = q[h:h + 1].float().numpy()
        kh = k[h:h + 1].float().numpy()
        vh = v[h:h + 1].float().numpy()
        ref = OA.block_sparse_attention(qh, kh, vh, row_ptr, col_idx, block,
                                        dtype=np.float32, q_blocks=q_blocks)
        for (_, qb), r in ref.items():
            g = out[h, qb * block: qb * block + r.shape[0]].float().cpu().numpy()
            assert np.isfinite(g).all()
            err = np.abs(g - r)
            worst = max(worst, float(err.max()))
            total += float(err.sum())
            count += err.size
    return worst, total / count


def assert_close(max_abs, mean_abs):
    assert max_abs <= MAX_ABS, f"max abs error {max_abs:.3e} > {MAX_ABS}"
    assert mean_abs <= MEAN_ABS, f"mean abs error {mean_abs:.3e} > {MEAN_ABS}"
