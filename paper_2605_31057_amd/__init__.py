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
    m = lvsa.csr_mask(row_ptr, col_idx, n_tokens, block)  # any block CSR on the device
    lvsa.attention(q, k, v, m, out)
"""
import ctypes
import os

__all__ = [
    "LvsaError", "Params", "Csr", "BlockMask", "ExactMask", "lib",
    "params_default", "frame_sets", "frame_window", "build_mask", "build_mask_device",
    "build_exact_mask_device", "csr_mask", "attention", "attention_noalloc",
    "attention_exact",
    "dense_attention", "WINDOW_BASIC", "WINDOW_ADAPTIVE", "WINDOW_EXPANDED",
    "MAX_FRAMES",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblvsa.so")

WINDOW_BASIC, WINDOW_ADAPTIVE, WINDOW_EXPANDED = 0, 1, 2
MAX_FRAMES = 4096
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
    """lvsa_block_mask: a block CSR in device memory."""
    _fields_ = [("n_tokens", _i32), ("block", _i32), ("n_q_blocks", _i32),
                ("n_kv_blocks", _i32), ("row_ptr", _p), ("col_idx", _p)]


class ExactMask(ctypes.Structure):
    """lvsa_exact_mask: device-resident token-exact form (row_ptr and entry
    words)."""
    _fields_ = [("n_tokens", _i32), ("block", _i32), ("n_q_blocks", _i32),
                ("frame_tokens", _i32), ("row_ptr", _p), ("entry", _p)]


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
                                       _pi32, _pi32, _pi32, _pi32, _pi32]),
            "lvsa_frame_window": (_i32, [_i32, _i32, ctypes.POINTER(Params), _i32,
                                         _pi32, _pi32, _pi32]),
            "lvsa_build_mask": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                       ctypes.POINTER(Params), ctypes.POINTER(_p)]),
            "lvsa_csr_info": (_i32, [_p, _pi32, _pi32, ctypes.POINTER(_i64),
                                     ctypes.POINTER(_pi32), ctypes.POINTER(_pi32)]),
            "lvsa_csr_shape": (_i32, [_p, _pi32, _pi32]),
            "lvsa_csr_upload": (_i32, [_p, _p]),
            "lvsa_csr_free": (None, [_p]),
            "lvsa_csr_device_view": (_i32, [_p, ctypes.POINTER(BlockMask)]),
            "lvsa_build_mask_device": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                              ctypes.POINTER(Params), _p, _p, _i64, _p]),
            "lvsa_build_exact_mask": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                             ctypes.POINTER(Params),
                                             ctypes.POINTER(_p)]),
            "lvsa_csr_entries": (_i32, [_p, _pi32,
                                        ctypes.POINTER(ctypes.POINTER(ctypes.c_uint32))]),
            "lvsa_csr_exact_view": (_i32, [_p, ctypes.POINTER(ExactMask)]),
            "lvsa_build_exact_mask_device": (_i32, [_i32, _i32, _i32, _i32, _i32,
                                                    ctypes.POINTER(Params), _p, _p,
                                                    _i64, _p]),
            "lvsa_attention_exact": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                                     [ctypes.POINTER(ExactMask),
                                      ctypes.POINTER(_Tensor), _p]),
            "lvsa_attention": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                               [ctypes.POINTER(BlockMask), ctypes.POINTER(_Tensor), _p]),
            "lvsa_attention_noalloc": (_i32, [ctypes.POINTER(_Tensor)] * 3 +
                                       [ctypes.POINTER(BlockMask), ctypes.POINTER(_Tensor),
                                        _p]),
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


def frame_sets(T, step, params=None, growth=False):
    """(T_per, anchors, win_lo, win_hi) for one step (lists of ints), plus the
    Alg. 1 growth steps per frame when ``growth`` is set."""
    params = params or Params()
    tper, n = _i32(), _i32()
    anchors = (_i32 * T)()
    lo = (_i32 * T)()
    hi = (_i32 * T)()
    grow = (_i32 * T)()
    _check(lib().lvsa_frame_sets(T, step, ctypes.byref(params), ctypes.byref(tper),
                                 anchors, ctypes.byref(n), lo, hi, grow), "lvsa_frame_sets")
    res = (tper.value, list(anchors[:n.value]), list(lo), list(hi))
    return res + (list(grow),) if growth else res


def frame_window(T, step, t, params=None):
    """(lo, hi, growth) of query frame t (lvsa_frame_window)."""
    params = params or Params()
    lo, hi, g = _i32(), _i32(), _i32()
    _check(lib().lvsa_frame_window(T, step, ctypes.byref(params), t, ctypes.byref(lo),
                                   ctypes.byref(hi), ctypes.byref(g)), "lvsa_frame_window")
    return lo.value, hi.value, g.value


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
        """(n_q_blocks, n_kv_blocks, nnz, row_ptr, col_idx) as lvsa_csr_info
        returns them (the arrays as ctypes pointers)."""
        nq, nk, nnz = _i32(), _i32(), _i64()
        rp, ci = _pi32(), _pi32()
        _check(lib().lvsa_csr_info(self._h, ctypes.byref(nq), ctypes.byref(nk),
                                   ctypes.byref(nnz), ctypes.byref(rp), ctypes.byref(ci)),
               "lvsa_csr_info")
        return nq.value, nk.value, nnz.value, rp, ci

    def shape(self):
        """(n_tokens, block) of the handle (lvsa_csr_shape)."""
        n, b = _i32(), _i32()
        _check(lib().lvsa_csr_shape(self._h, ctypes.byref(n), ctypes.byref(b)),
               "lvsa_csr_shape")
        return n.value, b.value

    @property
    def n_tokens(self):
        return self.shape()[0]

    @property
    def block(self):
        return self.shape()[1]

    @property
    def n_blocks(self):
        return self.info()[0]

    @property
    def nnz(self):
        return self.info()[2]

    def arrays(self):
        """(row_ptr, col_idx) as numpy int32 copies."""
        import numpy as np
        nb, _, nnz, rp, ci = self.info()
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


def _mask_keep(mask, tensors):
    mask._keep = tensors   # keep the device buffers alive with the view
    return mask


def build_mask_device(T, P, B, step, row_ptr, col_idx, params=None, layer=0,
                      stream=None):
    """Device LVSA mask builder into int32 device tensors row_ptr [nb+1] and
    col_idx [>= nb*nb]; returns a BlockMask over them."""
    params = params or Params()
    _check(lib().lvsa_build_mask_device(T, P, B, step, layer, ctypes.byref(params),
                                        _p(row_ptr.data_ptr()), _p(col_idx.data_ptr()),
                                        col_idx.numel(), _stream_ptr(stream)),
           "lvsa_build_mask_device")
    N = T * P + params.text_tokens
    nb = (N + B - 1) // B
    m = BlockMask(N, B, nb, nb, row_ptr.data_ptr(), col_idx.data_ptr())
    return _mask_keep(m, (row_ptr, col_idx))


def build_exact_mask_device(T, P, B, step, row_ptr, entry, params=None, layer=0,
                            stream=None):
    """Device builder of the token-exact form into device tensors (row_ptr
    int32 [nb+1], entry int32/uint32 [>= nb*nb]); returns an ExactMask."""
    params = params or Params()
    _check(lib().lvsa_build_exact_mask_device(
        T, P, B, step, layer, ctypes.byref(params), _p(row_ptr.data_ptr()),
        _p(entry.data_ptr()), entry.numel(), _stream_ptr(stream)),
        "lvsa_build_exact_mask_device")
    N = T * P + params.text_tokens
    nb = (N + B - 1) // B
    m = ExactMask(N, B, nb, P, row_ptr.data_ptr(), entry.data_ptr())
    return _mask_keep(m, (row_ptr, entry))


def csr_mask(row_ptr, col_idx, n_tokens, block):
    """A BlockMask over a caller-built block CSR in device int32 tensors
    (row_ptr [nb+1], col_idx [nnz], nb = ceil(n_tokens / block))."""
    nb = (n_tokens + block - 1) // block
    if row_ptr.numel() != nb + 1:
        raise LvsaError(EINVAL, f"row_ptr holds {row_ptr.numel()} offsets, the mask has "
                        f"{nb} query blocks")
    m = BlockMask(n_tokens, block, nb, nb, row_ptr.data_ptr(), col_idx.data_ptr())
    return _mask_keep(m, (row_ptr, col_idx))


def exact_csr_mask(row_ptr, entry, n_tokens, block, frame_tokens):
    """An ExactMask over caller-built token-exact entry words in device
    tensors (row_ptr int32 [nb+1], entry int32/uint32 [nnz])."""
    nb = (n_tokens + block - 1) // block
    m = ExactMask(n_tokens, block, nb, frame_tokens, row_ptr.data_ptr(), entry.data_ptr())
    return _mask_keep(m, (row_ptr, entry))


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


def attention_noalloc(q, k, v, mask, out, stream=None):
    """lvsa_attention_noalloc: block-sparse attention that allocates nothing
    (the caller passes `out`); calls overlapping on one device race."""
    tq, tk, tv, to = (_tensor(x) for x in (q, k, v, out))
    _check(lib().lvsa_attention_noalloc(ctypes.byref(tq), ctypes.byref(tk),
                                        ctypes.byref(tv), ctypes.byref(mask),
                                        ctypes.byref(to), _stream_ptr(stream)),
           "lvsa_attention_noalloc")
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
