"""LVSA block-sparse video attention for MI355X (gfx950): Python binding.

A thin ctypes layer over ``liblvsa.so`` (C ABI in ``include/lvsa.h``).  It only
marshals arguments: every mask and attention computation runs in the native
library (host C++ builder, HIP kernels).  torch is used for device memory and
streams only.  If the library is missing every call raises; there is no
fallback.

    import paper_2605_31057_amd as lvsa
    p = lvsa.Params(window=6, budget_frames=21)
    csr = lvsa.build_mask(T=121, P=1560, B=128, step=10, params=p)
    csr.upload()
    lvsa.attention(q, k, v, csr.device_mask(), out)      # q,k,v,out: [H,N,128] bf16
    ex = lvsa.build_mask(T=121, P=1560, B=128, step=10, params=p, exact=True)
    ex.upload()
    lvsa.attention_exact(q, k, v, ex.exact_mask(), out)  # Eq. 2 token for token
"""
import ctypes
import os

__all__ = [
    "LvsaError", "Params", "Csr", "BlockMask", "ExactMask", "lib",
    "params_default", "frame_sets", "build_mask", "build_mask_device",
    "build_exact_mask_device", "attention", "attention_exact",
    "dense_attention", "WINDOW_BASIC", "WINDOW_ADAPTIVE", "WINDOW_EXPANDED",
    "MAX_FRAMES", "PAIR_WORK",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblvsa.so")

WINDOW_BASIC, WINDOW_ADAPTIVE, WINDOW_EXPANDED = 0, 1, 2
MAX_FRAMES = 4096
PAIR_WORK = 16   # LVSA_PAIR_WORK: work words after a device pair_ptr's offsets
OK, EINVAL, ENOMEM, EDEVICE, EUNSUPPORTED = 0, -1, -2, -3, -4

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_p = ctypes.c_void_p
_pi32 = ctypes.POINTER(ctypes.c_int32)


class LvsaError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = lib().lvsa_status_str(status).decode()
        super().__init__(f"{where}: {msg} (status {status})")


class Params(ctypes.Structure):
    """lvsa_params: C, W, T_per override, window rule, rotation, tie rule,
    dedicated initial anchors, text tokens after the video tokens."""
    _fields_ = [("budget_frames", _i32), ("window", _i32), ("tper", _i32),
                ("window_mode", _i32), ("rotate", _i32), ("tie_high", _i32),
                ("extra_anchors", _i32), ("text_tokens", _i32)]

    def __init__(self, **kw):
        d = dict(budget_frames=21, window=6, tper=0,
                 window_mode=WINDOW_EXPANDED, rotate=1, tie_high=0,
                 extra_anchors=0, text_tokens=0)
        d.update(kw)
        super().__init__(**{k: int(v) for k, v in d.items()})


class BlockMask(ctypes.Structure):
    """lvsa_block_mask: device-resident block CSR and its pair schedule."""
    _fields_ = [("n_tokens", _i32), ("block", _i32), ("n_blocks", _i32),
                ("row_ptr", _p), ("col_idx", _p), ("pair_ptr", _p), ("pair_word", _p)]


class ExactMask(ctypes.Structure):
    """lvsa_exact_mask: device-resident token-exact form (row_ptr, entry
    words and the token-exact pair schedule)."""
    _fields_ = [("n_tokens", _i32), ("block", _i32), ("n_blocks", _i32),
                ("frame_tokens", _i32), ("row_ptr", _p), ("entry", _p),
                ("pair_ptr", _p), ("pair_word", _p)]


class _Tensor(ctypes.Structure):
    _fields_ = [("data", _p), ("heads", _i32), ("n_tokens", _i32),
                ("head_dim", _i32), ("stride_head", _i64),
                ("stride_token", _i64)]


_LIB = None


def lib():
    """The loaded native library (raises if it was not built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2605_31057_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "lvsa_status_str": (ctypes.c_char_p, [_i32]),
            "lvsa_version": (_i32, []),
            "lvsa_params_default": (None, [ctypes.POINTER(Params)]),
            "lvsa_frame_sets": (_i32, [_i32, _i32, ctypes.POINTER(Params), _pi32,
                                       _pi32, _pi32, _pi32, _pi32]),
            "lvsa_build_mask": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                       ctypes.POINTER(Params), ctypes.POINTER(_p)]),
            "lvsa_csr_info": (_i32, [_p, _pi32, _pi32, _pi32,
                                     ctypes.POINTER(_i64), ctypes.POINTER(_pi32),
                                     ctypes.POINTER(_pi32)]),
            "lvsa_csr_upload": (_i32, [_p, _p]),
            "lvsa_csr_free": (None, [_p]),
            "lvsa_csr_device_view": (_i32, [_p, ctypes.POINTER(BlockMask)]),
            "lvsa_build_mask_device": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                              ctypes.POINTER(Params), _p, _p,
                                              _i64, _p, _p, _i64, _p]),
            "lvsa_csr_pairs": (_i32, [_p, _pi32, ctypes.POINTER(_i64),
                                      ctypes.POINTER(_pi32),
                                      ctypes.POINTER(ctypes.POINTER(ctypes.c_uint32)),
                                      ctypes.POINTER(ctypes.POINTER(ctypes.c_uint32))]),
            "lvsa_build_exact_mask": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                             ctypes.POINTER(Params),
                                             ctypes.POINTER(_p)]),
            "lvsa_csr_entries": (_i32, [_p, _pi32,
                                        ctypes.POINTER(ctypes.POINTER(ctypes.c_uint32))]),
            "lvsa_csr_exact_view": (_i32, [_p, ctypes.POINTER(ExactMask)]),
            "lvsa_build_exact_mask_device": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                                    ctypes.POINTER(Params), _p, _p,
                                                    _i64, _p, _p, _i64, _p]),
            "lvsa_attention_exact": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                                     [ctypes.POINTER(ExactMask),
                                      ctypes.POINTER(_Tensor), _p]),
            "lvsa_attention": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                               [ctypes.POINTER(BlockMask), ctypes.POINTER(_Tensor), _p]),
            "lvsa_dense_attention": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                                     [_i32, ctypes.POINTER(_Tensor), _p]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def _check(status, where):
    if status != OK:
        raise LvsaError(status, where)


def params_default():
    p = Params()
    lib().lvsa_params_default(ctypes.byref(p))
    return p


def frame_sets(T, step, params=None):
    """(T_per, anchors, win_lo, win_hi) for one step (lists of ints)."""
    params = params or Params()
    tper, n = _i32(), _i32()
    anchors = (_i32 * T)()
    lo = (_i32 * T)()
    hi = (_i32 * T)()
    _check(lib().lvsa_frame_sets(T, step, ctypes.byref(params), ctypes.byref(tper),
                                 anchors, ctypes.byref(n), lo, hi), "lvsa_frame_sets")
    return tper.value, list(anchors[:n.value]), list(lo), list(hi)


def _stream_ptr(stream):
    if stream is None:
        import torch
        return _p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return _p(stream)
    return _p(stream.cuda_stream)


class Csr:
    """Host-built block CSR (lvsa_csr handle)."""

    def __init__(self, handle):
        self._h = _p(handle)

    def __del__(self):
        self.free()

    def free(self):
        if getattr(self, "_h", None) and self._h.value and _LIB is not None:
            _LIB.lvsa_csr_free(self._h)
            self._h = _p()

    def info(self):
        n, b, nb, nnz = _i32(), _i32(), _i32(), _i64()
        rp, ci = _pi32(), _pi32()
        _check(lib().lvsa_csr_info(self._h, ctypes.byref(n), ctypes.byref(b),
                                   ctypes.byref(nb), ctypes.byref(nnz),
                                   ctypes.byref(rp), ctypes.byref(ci)), "lvsa_csr_info")
        return n.value, b.value, nb.value, nnz.value, rp, ci

    @property
    def n_tokens(self):
        return self.info()[0]

    @property
    def block(self):
        return self.info()[1]

    @property
    def n_blocks(self):
        return self.info()[2]

    @property
    def nnz(self):
        return self.info()[3]

    def arrays(self):
        """(row_ptr, col_idx) as numpy int32 copies."""
        import numpy as np
        _, _, nb, nnz, rp, ci = self.info()
        row_ptr = np.ctypeslib.as_array(rp, shape=(nb + 1,)).copy()
        col_idx = (np.ctypeslib.as_array(ci, shape=(nnz,)).copy() if nnz
                   else np.zeros(0, dtype=np.int32))
        return row_ptr, col_idx

    def entries(self):
        """Token-exact entry words as a numpy uint32 copy (raises LvsaError
        with EUNSUPPORTED for a handle built without them)."""
        import numpy as np
        nnz = self.nnz
        P = _i32()
        e = ctypes.POINTER(ctypes.c_uint32)()
        _check(lib().lvsa_csr_entries(self._h, ctypes.byref(P), ctypes.byref(e)),
               "lvsa_csr_entries")
        return (np.ctypeslib.as_array(e, shape=(nnz,)).copy() if nnz
                else np.zeros(0, dtype=np.uint32))

    def pairs(self):
        """Pair schedule (pair_ptr, block-form words, token-exact words or
        None) as numpy copies (lvsa_csr_pairs)."""
        import numpy as np
        npairs, nw = _i32(), _i64()
        pp = _pi32()
        pw = ctypes.POINTER(ctypes.c_uint32)()
        pe = ctypes.POINTER(ctypes.c_uint32)()
        _check(lib().lvsa_csr_pairs(self._h, ctypes.byref(npairs), ctypes.byref(nw),
                                    ctypes.byref(pp), ctypes.byref(pw), ctypes.byref(pe)),
               "lvsa_csr_pairs")
        ptr = np.ctypeslib.as_array(pp, shape=(npairs.value + 1,)).copy()
        n = nw.value
        words = (np.ctypeslib.as_array(pw, shape=(n,)).copy() if n
                 else np.zeros(0, dtype=np.uint32))
        exact = None
        if pe:
            exact = (np.ctypeslib.as_array(pe, shape=(n,)).copy() if n
                     else np.zeros(0, dtype=np.uint32))
        return ptr, words, exact

    def upload(self, stream=None):
        _check(lib().lvsa_csr_upload(self._h, _stream_ptr(stream)), "lvsa_csr_upload")
        return self

    def device_mask(self):
        m = BlockMask()
        _check(lib().lvsa_csr_device_view(self._h, ctypes.byref(m)),
               "lvsa_csr_device_view")
        return m

    def exact_mask(self):
        m = ExactMask()
        _check(lib().lvsa_csr_exact_view(self._h, ctypes.byref(m)),
               "lvsa_csr_exact_view")
        return m


def build_mask(T, P, B, step, params=None, layer=0, exact=False):
    """Host LVSA mask builder -> Csr.  ``exact=True`` also builds the
    token-exact entry words (lvsa_build_exact_mask)."""
    params = params or Params()
    h = _p()
    fn, name = ((lib().lvsa_build_exact_mask, "lvsa_build_exact_mask") if exact
                else (lib().lvsa_build_mask, "lvsa_build_mask"))
    _check(fn(T, P, B, step, layer, ctypes.byref(params), ctypes.byref(h)), name)
    return Csr(h.value)


def pair_buffers(n_tokens, block, device=None, stream=None):
    """Device int32 tensors (pair_ptr [ceil(nb/2)+1+PAIR_WORK]: the offsets and
    the attention kernels' work words; pair words [ceil(nb/2)*nb]) sized for a
    device builder's pair schedule, allocated on
    `stream` (a torch stream, a raw stream handle or None for the current
    one) so the caching allocator reuses them only after that stream's work."""
    import torch
    nb = (n_tokens + block - 1) // block
    npairs = (nb + 1) // 2
    dev = device or "cuda"
    if stream is None:
        s = torch.cuda.current_stream()
    elif isinstance(stream, int):
        s = torch.cuda.ExternalStream(stream)
    else:
        s = stream
    with torch.cuda.stream(s):
        return (torch.empty(npairs + 1 + PAIR_WORK, dtype=torch.int32, device=dev),
                torch.empty(max(npairs * nb, 1), dtype=torch.int32, device=dev))


def _check_pair_ptr(pair_ptr, N, B):
    npairs = ((N + B - 1) // B + 1) // 2
    if pair_ptr.numel() < npairs + 1 + PAIR_WORK:
        raise LvsaError(EINVAL, f"pair_ptr holds {pair_ptr.numel()} words, the pair schedule "
                        f"needs ceil(nb/2) + 1 + PAIR_WORK = {npairs + 1 + PAIR_WORK}")


def _mask_with_pairs(mask, tensors):
    mask._keep = tensors   # keep the device buffers alive with the view
    return mask


def build_mask_device(T, P, B, step, row_ptr, col_idx, params=None, layer=0,
                      stream=None, pair_ptr=None, pair_word=None):
    """Device LVSA mask builder into int32 device tensors (the CSR and its
    pair schedule; pair buffers are allocated when not given); returns a
    BlockMask."""
    params = params or Params()
    N = T * P + params.text_tokens
    if pair_ptr is None or pair_word is None:
        pair_ptr, pair_word = pair_buffers(N, B, row_ptr.device, stream)
    _check_pair_ptr(pair_ptr, N, B)
    _check(lib().lvsa_build_mask_device(T, P, B, step, layer, ctypes.byref(params),
                                        _p(row_ptr.data_ptr()), _p(col_idx.data_ptr()),
                                        col_idx.numel(), _p(pair_ptr.data_ptr()),
                                        _p(pair_word.data_ptr()), pair_word.numel(),
                                        _stream_ptr(stream)),
           "lvsa_build_mask_device")
    nb = (N + B - 1) // B
    m = BlockMask(N, B, nb, row_ptr.data_ptr(), col_idx.data_ptr(), pair_ptr.data_ptr(),
                  pair_word.data_ptr())
    return _mask_with_pairs(m, (row_ptr, col_idx, pair_ptr, pair_word))


def build_exact_mask_device(T, P, B, step, row_ptr, entry, params=None, layer=0,
                            stream=None, pair_ptr=None, pair_word=None):
    """Device builder of the token-exact form into device tensors (row_ptr
    int32 [nb+1], entry int32/uint32 [>= nb*nb], and the token-exact pair
    schedule, allocated when not given); returns an ExactMask."""
    params = params or Params()
    N = T * P + params.text_tokens
    if pair_ptr is None or pair_word is None:
        pair_ptr, pair_word = pair_buffers(N, B, row_ptr.device, stream)
    _check_pair_ptr(pair_ptr, N, B)
    _check(lib().lvsa_build_exact_mask_device(
        T, P, B, step, layer, ctypes.byref(params), _p(row_ptr.data_ptr()),
        _p(entry.data_ptr()), entry.numel(), _p(pair_ptr.data_ptr()),
        _p(pair_word.data_ptr()), pair_word.numel(), _stream_ptr(stream)),
        "lvsa_build_exact_mask_device")
    nb = (N + B - 1) // B
    m = ExactMask(N, B, nb, P, row_ptr.data_ptr(), entry.data_ptr(), pair_ptr.data_ptr(),
                  pair_word.data_ptr())
    return _mask_with_pairs(m, (row_ptr, entry, pair_ptr, pair_word))


def _tensor(t):
    if t.dim() != 3:
        raise ValueError("expected a [heads, n_tokens, head_dim] tensor")
    if t.stride(2) != 1:
        raise ValueError("head_dim must be contiguous")
    import torch
    if t.dtype != torch.bfloat16 or not t.is_cuda:
        raise ValueError("expected a bfloat16 device tensor")
    return _Tensor(t.data_ptr(), t.shape[0], t.shape[1], t.shape[2],
                   t.stride(0), t.stride(1))


def attention(q, k, v, mask, out=None, stream=None):
    """Block-sparse attention (lvsa_attention); returns out."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    tq, tk, tv, to = (_tensor(x) for x in (q, k, v, out))
    _check(lib().lvsa_attention(ctypes.byref(tq), ctypes.byref(tk), ctypes.byref(tv),
                                ctypes.byref(mask), ctypes.byref(to),
                                _stream_ptr(stream)), "lvsa_attention")
    return out


def attention_exact(q, k, v, mask, out=None, stream=None):
    """Token-exact attention (lvsa_attention_exact): Eq. 2 token for token."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    tq, tk, tv, to = (_tensor(x) for x in (q, k, v, out))
    _check(lib().lvsa_attention_exact(ctypes.byref(tq), ctypes.byref(tk),
                                      ctypes.byref(tv), ctypes.byref(mask),
                                      ctypes.byref(to), _stream_ptr(stream)),
           "lvsa_attention_exact")
    return out


def dense_attention(q, k, v, block=128, out=None, stream=None):
    """Dense attention of the same kernel design (lvsa_dense_attention)."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    tq, tk, tv, to = (_tensor(x) for x in (q, k, v, out))
    _check(lib().lvsa_dense_attention(ctypes.byref(tq), ctypes.byref(tk),
                                      ctypes.byref(tv), block, ctypes.byref(to),
                                      _stream_ptr(stream)), "lvsa_dense_attention")
    return out
