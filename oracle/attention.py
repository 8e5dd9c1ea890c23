"""Attention oracle: masked softmax attention written out plainly.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code
with the library under ``paper_2605_31057_amd/`` and imports nothing from it.

What is computed (LVSA paper, Sec. 2):
  * Eq. 1 (dense):  Attn(q_i) = sum_j softmax_j(q_i . k_j / sqrt(d)) v_j over
    all N keys.
  * Eq. 2 (sparse): the same softmax restricted to a key set.
    ``block_sparse_attention`` takes, for every query of query block qb, the
    keys of the kept key blocks of qb (the CSR the mask oracle emits);
    ``frame_sparse_attention`` and ``frame_sparse_rows`` take the keys whose
    frame is in A(frame of the query), which is Eq. 2 token for token.

Plain numpy: one matrix product for the logits, the textbook max-shifted
softmax, one matrix product for the weighted sum.  No blocking, no online
softmax, no fusion.  Inputs are the exact float upcast of the bf16 tensors;
the arithmetic type is float32 by default (float64 for the self-tests).

Parity pins: tests/test_oracle_attention.py (brute-force scalar loops,
closed forms, a library attention routine at full mask, invariants).
"""
import math

import numpy as np


def softmax_rows(s):
    """Row-wise softmax exp(s - max) / sum exp(s - max)."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q, k, v):
    """Eq. 1 for a set of queries against one key set.

    q: [nq, d], k: [nk, d], v: [nk, dv]; returns [nq, dv].
    """
    d = q.shape[-1]
    s = (q @ k.T) / np.asarray(math.sqrt(d), dtype=q.dtype)
    return softmax_rows(s) @ v


def dense_attention(q, k, v, dtype=np.float32):
    """Eq. 1 over every key, all heads.  q, k, v: [H, N, d]."""
    q, k, v = (np.asarray(x, dtype=dtype) for x in (q, k, v))
    return np.stack([attend(q[h], k[h], v[h]) for h in range(q.shape[0])])


def block_keys(kv_blocks, block, n_tokens):
    """Token indices of the listed key blocks, clipped to the N real tokens."""
    idx = [np.arange(kb * block, min((kb + 1) * block, n_tokens))
           for kb in kv_blocks]
    return np.concatenate(idx) if idx else np.zeros(0, dtype=np.int64)


def block_sparse_attention(q, k, v, row_ptr, col_idx, block, dtype=np.float32,
                           heads=None, q_blocks=None):
    """Eq. 2 with the key set of every query block given by a block CSR.

    q, k, v: [H, N, d] (any float type; upcast to ``dtype``).
    row_ptr, col_idx: kept kv-blocks of each query block (ascending).
    heads, q_blocks: optional subsets to evaluate (rows are independent).
    Returns {(h, qb): [rows_of_qb, d]}.
    """
    H, N, _ = q.shape
    heads = range(H) if heads is None else heads
    nqb = len(row_ptr) - 1
    q_blocks = range(nqb) if q_blocks is None else q_blocks
    out = {}
    for h in heads:
        for qb in q_blocks:
            rows = np.arange(qb * block, min((qb + 1) * block, N))
            keys = block_keys(col_idx[row_ptr[qb]:row_ptr[qb + 1]], block, N)
            qh = np.asarray(q[h, rows], dtype=dtype)
            kh = np.asarray(k[h, keys], dtype=dtype)
            vh = np.asarray(v[h, keys], dtype=dtype)
            out[(h, qb)] = attend(qh, kh, vh)
    return out


def frame_sparse_attention(q, k, v, A, P, dtype=np.float32):
    """Eq. 2 token for token: query token i attends to the keys j whose frame
    is in A(frame(i)).  q, k, v: [H, N, d]; A: list of frame sets."""
    H, N, _ = q.shape
    T = N // P
    out = np.zeros(q.shape, dtype=dtype)
    for h in range(H):
        for t in range(T):
            rows = np.arange(t * P, (t + 1) * P)
            keys = np.concatenate([np.arange(tau * P, (tau + 1) * P)
                                   for tau in sorted(A[t])])
            out[h, rows] = attend(np.asarray(q[h, rows], dtype=dtype),
                                  np.asarray(k[h, keys], dtype=dtype),
                                  np.asarray(v[h, keys], dtype=dtype))
    return out


def frame_sparse_rows(q, k, v, A, P, heads, rows, dtype=np.float32):
    """Eq. 2 token for token on selected query rows (rows are independent).

    q, k, v: [H, N, d]; A: list of frame sets; heads, rows: the heads and
    query token indices to evaluate.  Returns {h: [len(rows), d]}.
    """
    out = {}
    for h in heads:
        res = []
        for i in rows:
            keys = np.concatenate([np.arange(tau * P, (tau + 1) * P)
                                   for tau in sorted(A[i // P])])
            res.append(attend(np.asarray(q[h, i:i + 1], dtype=dtype),
                              np.asarray(k[h, keys], dtype=dtype),
                              np.asarray(v[h, keys], dtype=dtype))[0])
        out[h] = np.stack(res)
    return out


def text_sparse_rows(q, k, v, A, T, P, heads, rows, dtype=np.float32):
    """Eq. 2 with text tokens after the T*P video tokens, on selected query
    rows: a video query (i < T*P) takes the keys of the frames in A(frame i)
    plus every text key; a text query takes every key.  q, k, v: [H, N, d]
    with N = T*P + L.  Returns {h: [len(rows), d]}."""
    V = T * P
    N = q.shape[1]
    text_keys = np.arange(V, N)
    out = {}
    for h in heads:
        res = []
        for i in rows:
            if i >= V:
                keys = np.arange(N)
            else:
                keys = np.concatenate([np.arange(tau * P, (tau + 1) * P)
                                       for tau in sorted(A[i // P])] + [text_keys])
            res.append(attend(np.asarray(q[h, i:i + 1], dtype=dtype),
                              np.asarray(k[h, keys], dtype=dtype),
                              np.asarray(v[h, keys], dtype=dtype))[0])
        out[h] = np.stack(res)
    return out


def assemble(blocks, H, N, d, block, dtype=np.float32):
    """Scatter {(h, qb): rows} from block_sparse_attention into [H, N, d]."""
    out = np.zeros((H, N, d), dtype=dtype)
    for (h, qb), val in blocks.items():
        out[h, qb * block: qb * block + val.shape[0]] = val
    return out
