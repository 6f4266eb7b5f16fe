"""Python binding of librq (the RateQuant hot path on MI355X).

Argument marshalling only: every step of the path runs in the HIP library.
Functions carry the C names; they raise RQError on a non-OK status.  Device
arguments are torch tensors on a HIP device (torch provides device memory
and streams), host arrays are numpy arrays.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librq.so")

RQ_OK, RQ_EINVAL, RQ_EINFEASIBLE, RQ_EUNSUPPORTED, RQ_EDEVICE, RQ_ESMALLWS = (
    0, -1, -2, -3, -4, -5)
RQ_KIVI, RQ_QUAROT, RQ_TURBO, RQ_RTN, RQ_KIVI_RTN = 0, 1, 2, 3, 4
RQ_F16, RQ_BF16, RQ_F32 = 0, 1, 2
RQ_MAX_KV_HEADS = 32

EXPORTS = ("rq_version", "rq_last_error", "rq_cache_sizes", "rq_region_offset",
           "rq_quantize_kv", "rq_decode_workspace", "rq_decode_attention",
           "rq_calibrate_workspace", "rq_calibrate_distortion",
           "rq_fit_distortion", "rq_allocate_bits", "rq_turbo_codebook",
           "rq_sensitivity_workspace", "rq_sensitivity", "rq_cap_weights",
           "rq_fallback_beta", "rq_decode_static_bytes",
           "rq_decode_attention_static", "rq_read_probe", "rq_decode_step")
RQ_TURBO_TABLE_FLOATS = 8 * 2 * 256


class RQError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class RqCache(C.Structure):
    _fields_ = [("family", C.c_int32), ("dtype", C.c_int32),
                ("n_layers", C.c_int32), ("batch", C.c_int32),
                ("n_kv_heads", C.c_int32), ("n_q_heads", C.c_int32),
                ("head_dim", C.c_int32), ("capacity", C.c_int32),
                ("residual", C.c_int32), ("bits", C.POINTER(C.c_int8)),
                ("codes", C.c_void_p), ("meta", C.c_void_p),
                ("resid", C.c_void_p), ("rotation", C.c_void_p),
                ("codebook", C.c_void_p)]


_lib = None


def lib():
    """Load librq.so (built in-tree by build.py).  Raises if it is absent:
    there is no fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2605_06675_amd.build`")
        L = C.CDLL(LIB_PATH)
        i32, u64, vp = C.c_int32, C.c_uint64, C.c_void_p
        pd, pi = C.POINTER(C.c_double), C.POINTER(C.c_int32)
        pu64 = C.POINTER(C.c_uint64)
        pc = C.POINTER(RqCache)
        sig = {
            "rq_version": (i32, []),
            "rq_last_error": (C.c_char_p, []),
            "rq_cache_sizes": (i32, [pc, pu64, pu64, pu64]),
            "rq_region_offset": (i32, [pc, i32, i32, i32, pu64]),
            "rq_quantize_kv": (i32, [pc, i32, i32, vp, vp, i32, vp]),
            "rq_decode_workspace": (i32, [pc, i32, pu64]),
            "rq_decode_attention": (i32, [pc, i32, i32, vp, vp, C.c_float, vp,
                                          u64, vp]),
            "rq_calibrate_workspace": (i32, [i32, i32, i32, pu64]),
            "rq_calibrate_distortion": (i32, [i32, i32, vp, i32, i32, i32, pi,
                                              i32, vp, vp, pd, pd, pd, pd, vp,
                                              u64, vp]),
            "rq_fit_distortion": (i32, [pd, i32, pi, i32, pd, pd, pd]),
            "rq_allocate_bits": (i32, [i32, pd, pd, pd, C.c_double, i32, i32,
                                       pi, pd, pd]),
            "rq_turbo_codebook": (i32, [C.POINTER(C.c_float)]),
            "rq_sensitivity_workspace": (i32, [i32, i32, i32, i32, pu64]),
            "rq_sensitivity": (i32, [i32, vp, i32, i32, i32, pd, vp, u64, vp]),
            "rq_cap_weights": (i32, [i32, pd, C.c_double]),
            "rq_fallback_beta": (i32, [i32, pd, pd, C.c_double]),
            "rq_decode_static_bytes": (u64, []),
            "rq_read_probe": (i32, [vp, u64, vp, i32, vp]),
            "rq_decode_attention_static": (i32, [pc, i32, i32, vp, vp,
                                                 C.c_float, vp]),
            "rq_decode_step": (i32, [pc, i32, i32, vp, vp, vp, vp, C.c_float,
                                     vp, u64, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(status):
    if status != RQ_OK:
        raise RQError(status, lib().rq_last_error().decode())


def _dptr(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.POINTER(np.ctypeslib.as_ctypes_type(dtype)))


def _tptr(t):
    """Device pointer of a contiguous torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("device tensors must be contiguous")
    return C.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


# ----------------------------------------------------------------- host calls
def rq_version():
    return lib().rq_version()


def rq_last_error():
    return lib().rq_last_error().decode()


def rq_fit_distortion(mse, bits):
    mse = np.atleast_2d(np.asarray(mse, dtype=np.float64))
    n_comp, n_bits = mse.shape
    m, mp = _dptr(mse, np.float64)
    b, bp = _dptr(bits, np.int32)
    out = [np.empty(n_comp) for _ in range(3)]
    ptrs = [o.ctypes.data_as(C.POINTER(C.c_double)) for o in out]
    _check(lib().rq_fit_distortion(mp, n_comp, bp, n_bits, *ptrs))
    return tuple(out)


def rq_allocate_bits(w, alpha, beta, avg_bits, bmin, bmax, want_cont=True):
    """Returns (bits int32[n], continuous float64[n] or None, J)."""
    w, wp = _dptr(w, np.float64)
    a, ap = _dptr(alpha, np.float64)
    be, bp = _dptr(beta, np.float64)
    n = w.size
    bits = np.empty(n, dtype=np.int32)
    cont = np.empty(n) if want_cont else None
    J = C.c_double()
    _check(lib().rq_allocate_bits(
        n, wp, ap, bp, float(avg_bits), int(bmin), int(bmax),
        bits.ctypes.data_as(C.POINTER(C.c_int32)),
        cont.ctypes.data_as(C.POINTER(C.c_double)) if want_cont else None,
        C.byref(J)))
    return bits, cont, J.value


def rq_turbo_codebook():
    """The TurboQuant codebook table, float32 [8][2][256]: [b-1][0] the
    thresholds, [b-1][1] the centroids of the b-bit Lloyd-Max quantizer."""
    t = np.empty(RQ_TURBO_TABLE_FLOATS, dtype=np.float32)
    _check(lib().rq_turbo_codebook(t.ctypes.data_as(C.POINTER(C.c_float))))
    return t.reshape(8, 2, 256)


def rq_calibrate_workspace(n_comp, n_tokens, n_bits):
    v = C.c_uint64()
    _check(lib().rq_calibrate_workspace(n_comp, n_tokens, n_bits, C.byref(v)))
    return v.value


def make_cache(family, dtype, n_layers, batch, n_kv_heads, n_q_heads,
               capacity, residual, bits, codes=None, meta=None, resid=None,
               rotation=None, codebook=None):
    """Fill an RqCache descriptor.  bits: int8 [n_layers][n_kv_heads][2];
    rotation, codebook: device tensors (TurboQuant only).  The numpy bit
    table is kept alive on the returned object."""
    bt = np.ascontiguousarray(bits, dtype=np.int8).reshape(-1)
    c = RqCache(family, dtype, n_layers, batch, n_kv_heads, n_q_heads, 128,
                capacity, residual, bt.ctypes.data_as(C.POINTER(C.c_int8)),
                _tptr(codes) if codes is not None else None,
                _tptr(meta) if meta is not None else None,
                _tptr(resid) if resid is not None else None,
                _tptr(rotation) if rotation is not None else None,
                _tptr(codebook) if codebook is not None else None)
    c._bits = bt
    return c


def rq_cache_sizes(cache):
    a, b, c = C.c_uint64(), C.c_uint64(), C.c_uint64()
    _check(lib().rq_cache_sizes(C.byref(cache), C.byref(a), C.byref(b),
                                C.byref(c)))
    return a.value, b.value, c.value


def rq_region_offset(cache, layer, head, kind):
    v = C.c_uint64()
    _check(lib().rq_region_offset(C.byref(cache), layer, head, kind,
                                  C.byref(v)))
    return v.value


def rq_decode_workspace(cache, n_tokens):
    v = C.c_uint64()
    _check(lib().rq_decode_workspace(C.byref(cache), n_tokens, C.byref(v)))
    return v.value


# --------------------------------------------------------------- device calls
def _need_device(t, what, shape, elem):
    """The C side sees raw pointers only: check what it cannot (shape,
    element size, device, contiguity) before a kernel reads or writes the
    buffer."""
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.element_size() != elem:
        raise ValueError(f"{what} has {t.element_size()}-byte elements, expected {elem}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")


def _check_attention_args(cache, q, out):
    import torch
    shape = (cache.batch, cache.n_q_heads, 128)
    _need_device(q, "q", shape, 2)
    _need_device(out, "out", shape, 4)
    if out.dtype != torch.float32 or q.device != out.device:
        raise ValueError("out must be float32 on q's device")


def rq_quantize_kv(cache, layer, n_past, k, v, stream=None):
    """k, v: torch [batch][n_kv_heads][n_new][128] (fp16/bf16, device)."""
    n_new = k.shape[2] if k.dim() == 4 else -1
    shape = (cache.batch, cache.n_kv_heads, n_new, 128)
    _need_device(k, "k", shape, 2)
    _need_device(v, "v", shape, 2)
    _check(lib().rq_quantize_kv(C.byref(cache), layer, n_past, _tptr(k),
                                _tptr(v), n_new, _stream(stream)))


def rq_decode_attention(cache, layer, n_tokens, q, out, ws, scale=None,
                        stream=None):
    """q: torch [batch][n_q_heads][128]; out: fp32 same shape; ws: device
    byte tensor of at least rq_decode_workspace bytes."""
    if scale is None:
        scale = 1.0 / np.sqrt(128.0)
    _check_attention_args(cache, q, out)
    if not ws.is_cuda or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous device tensor")
    _check(lib().rq_decode_attention(
        C.byref(cache), layer, n_tokens, _tptr(q), _tptr(out), float(scale),
        _tptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def rq_decode_step(cache, layer, n_past, k, v, q, out, ws, scale=None,
                   stream=None):
    """Append one token (k, v: [batch][n_kv_heads][1][128]) after n_past and
    attend over n_past + 1 tokens with q in one fused call; out, ws as for
    rq_decode_attention (ws sized for n_past + 1 tokens)."""
    if scale is None:
        scale = 1.0 / np.sqrt(128.0)
    shape = (cache.batch, cache.n_kv_heads, 1, 128)
    _need_device(k, "k", shape, 2)
    _need_device(v, "v", shape, 2)
    _check_attention_args(cache, q, out)
    if not ws.is_cuda or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous device tensor")
    _check(lib().rq_decode_step(
        C.byref(cache), layer, n_past, _tptr(k), _tptr(v), _tptr(q), _tptr(out),
        float(scale), _tptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def rq_decode_attention_static(cache, layer, n_tokens, q, out, scale=None,
                               stream=None):
    """rq_decode_attention with the library's own scratch: allocates
    nothing (for callers that cannot allocate)."""
    if scale is None:
        scale = 1.0 / np.sqrt(128.0)
    _check_attention_args(cache, q, out)
    _check(lib().rq_decode_attention_static(
        C.byref(cache), layer, n_tokens, _tptr(q), _tptr(out), float(scale),
        _stream(stream)))


def rq_read_probe(buf, sink, n_blocks, stream=None):
    """Read the whole device tensor buf once (measurement utility); sink:
    device int32/uint32 tensor of n_blocks elements."""
    _check(lib().rq_read_probe(_tptr(buf), buf.numel() * buf.element_size(),
                               _tptr(sink), int(n_blocks), _stream(stream)))


def rq_calibrate_distortion(family, dtype, x, is_value, bits, ws=None,
                            fit=True, rotation=None, codebook=None,
                            stream=None):
    """x: torch [n_comp][n_tokens][128] (device); rotation (bf16
    [n_comp][128][128]) and codebook (float32 table) on the device for
    TurboQuant.  Returns (mse[n_comp][n_bits], alpha, beta, r2) as numpy
    arrays (None when fit is False)."""
    import torch
    n_comp, T = x.shape[0], x.shape[1]
    b, bp = _dptr(bits, np.int32)
    need = rq_calibrate_workspace(n_comp, T, b.size)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    mse = np.empty((n_comp, b.size))
    outs = [np.empty(n_comp) for _ in range(3)] if fit else [None] * 3
    dp = C.POINTER(C.c_double)
    ptrs = [o.ctypes.data_as(dp) if o is not None else None for o in outs]
    _check(lib().rq_calibrate_distortion(
        family, dtype, _tptr(x), n_comp, T, int(bool(is_value)), bp, b.size,
        _tptr(rotation), _tptr(codebook), mse.ctypes.data_as(dp), *ptrs,
        _tptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return (mse, *outs)


def rq_sensitivity_workspace(gdtype, n_seq, n_comp, n_tokens):
    v = C.c_uint64()
    _check(lib().rq_sensitivity_workspace(gdtype, n_seq, n_comp, n_tokens,
                                          C.byref(v)))
    return v.value


def rq_sensitivity(gdtype, grad, ws=None, stream=None):
    """grad: torch [n_seq][n_comp][n_tokens][128] on the device (float32,
    float16 or bfloat16 as gdtype says).  Returns w float64[n_comp]."""
    import torch
    n_seq, n_comp, T = grad.shape[0], grad.shape[1], grad.shape[2]
    need = rq_sensitivity_workspace(gdtype, n_seq, n_comp, T)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=grad.device)
    w = np.empty(n_comp)
    _check(lib().rq_sensitivity(
        gdtype, _tptr(grad), n_seq, n_comp, T,
        w.ctypes.data_as(C.POINTER(C.c_double)), _tptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return w


def rq_cap_weights(w, factor=5.0):
    """Returns a capped copy of w."""
    w = np.array(w, dtype=np.float64)
    _check(lib().rq_cap_weights(w.size, w.ctypes.data_as(C.POINTER(C.c_double)),
                                float(factor)))
    return w


def rq_fallback_beta(beta, r2, r2_min=0.96):
    """Returns a copy of beta with the fallback applied."""
    beta = np.array(beta, dtype=np.float64)
    r, rp = _dptr(r2, np.float64)
    if r.size != beta.size:
        raise ValueError("beta and r2 differ in length")
    _check(lib().rq_fallback_beta(beta.size,
                                  beta.ctypes.data_as(C.POINTER(C.c_double)),
                                  rp, float(r2_min)))
    return beta


class KVCache:
    """Device buffers (torch) plus the descriptor of one quantized cache."""

    def __init__(self, family, dtype, n_layers, batch, n_kv_heads, n_q_heads,
                 capacity, residual, bits, device="cuda", rotation=None):
        """rotation (TurboQuant only): device tensor of the bf16 rotations
        [n_layers][n_kv_heads][128][128] (y = R x); the codebook table is
        computed by the library and copied to the device here."""
        import torch
        self.desc = make_cache(family, dtype, n_layers, batch, n_kv_heads,
                               n_q_heads, capacity, residual, bits)
        self.rotation = self.codebook = None
        if family == RQ_TURBO:
            if rotation is None:
                raise ValueError("TurboQuant needs the rotations")
            if tuple(rotation.shape) != (n_layers, n_kv_heads, 128, 128) \
                    or rotation.element_size() != 2:
                raise ValueError("rotation must be 16-bit [L][H][128][128]")
            self.rotation = rotation.contiguous()
            self.codebook = torch.from_numpy(
                rq_turbo_codebook().reshape(-1)).to(device)
            self.desc.rotation = self.rotation.data_ptr()
            self.desc.codebook = self.codebook.data_ptr()
        cb, mb, rb = rq_cache_sizes(self.desc)
        self.codes = torch.zeros(max(cb, 1), dtype=torch.uint8, device=device)
        self.meta = torch.zeros(max(mb, 1), dtype=torch.uint8, device=device)
        self.resid = torch.zeros(max(rb, 2) // 2, dtype=torch.int16,
                                 device=device)
        self.desc.codes = self.codes.data_ptr()
        self.desc.meta = self.meta.data_ptr()
        self.desc.resid = self.resid.data_ptr()
        self.n_tokens = [0] * n_layers
        self._ws = None

    def append(self, layer, k, v, stream=None):
        rq_quantize_kv(self.desc, layer, self.n_tokens[layer], k, v, stream)
        self.n_tokens[layer] += k.shape[2]

    def workspace(self, n_tokens, stream=None):
        import torch
        need = rq_decode_workspace(self.desc, n_tokens)
        if self._ws is None or self._ws.numel() < need:
            # zeroed once, on the stream of the call that first uses it (a
            # zeroed counter is always read as stale, whatever the call's
            # number on this workspace)
            s = torch.cuda.current_stream() if stream is None else stream
            with torch.cuda.stream(s):
                self._ws = torch.zeros(need, dtype=torch.uint8,
                                       device=self.codes.device)
        return self._ws

    def attention(self, layer, q, out=None, scale=None, stream=None):
        import torch
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        n = self.n_tokens[layer]
        rq_decode_attention(self.desc, layer, n, q, out,
                            self.workspace(n, stream), scale, stream)
        return out

    def decode_step(self, layer, k, v, q, out=None, scale=None, stream=None):
        """Append one token to `layer` and attend over the cache with q
        (rq_decode_step)."""
        import torch
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        n = self.n_tokens[layer]
        rq_decode_step(self.desc, layer, n, k, v, q, out,
                       self.workspace(n + 1, stream), scale, stream)
        self.n_tokens[layer] = n + 1
        return out

    def attention_static(self, layer, q, out, scale=None, stream=None):
        """Decode attention through rq_decode_attention_static (the
        library's own scratch; no allocation: out is the caller's)."""
        rq_decode_attention_static(self.desc, layer, self.n_tokens[layer], q,
                                   out, scale, stream)
        return out
