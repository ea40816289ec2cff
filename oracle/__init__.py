"""CPU oracle for the SparOA hot path -- TEST INFRASTRUCTURE ONLY.

Only tests/, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does.

Thin ctypes wrapper over ``sparoa_oracle.c`` (plain C, double precision).
Inputs are numpy arrays or CPU torch tensors; floating point tensors are
handed to C as their raw bit patterns and decoded there.

Paper passages followed (SparOA, arXiv 2511.19457):
  * measure()       -- sparsity, Section 3.1 Eq. 1 (zero fraction)
  * conv_intensity(), fc_intensity() -- Section 3.1 Eq. 2, generalised with
                       batch, stride, dilation and groups; FLOP/byte
  * route()         -- Section 2.2 quadrants and the fixed-threshold rule
                       opening Section 3, remapped to GPU kernel paths
  * conv2d(), fc()  -- the operators (Sections 1, 2.1), double precision;
                       with a mask they skip zero blocks (Section 1: skipping
                       zeros leaves the output unchanged)
  * *_executed_blocks() -- work a block-skipping kernel performs
  * maxpool2d()     -- network glue

Parity unpinned: the optimality of the routing thresholds (the paper learns
them with a predictor whose data and weights are not available).
"""
import ctypes
import os

import numpy as np

from .build import LIB, build

F32, F16, BF16 = 0, 1, 2
ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
ROUTE_BLOCK, ROUTE_ELEMENT = 0, 1

_lib = None

_u64p = ctypes.POINTER(ctypes.c_uint64)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_dp = ctypes.POINTER(ctypes.c_double)
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(
            os.path.join(os.path.dirname(LIB), "sparoa_oracle.c")
        ):
            build()
        L = ctypes.CDLL(LIB)
        L.or_decode.restype = ctypes.c_double
        L.or_decode.argtypes = [_vp, ctypes.c_int, _i64]
        L.or_measure.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _i64, _u64p, _u32p, _u64p]
        L.or_sparsity.restype = ctypes.c_double
        L.or_sparsity.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.or_out_dim.restype = _i64
        L.or_out_dim.argtypes = [_i64] * 5
        L.or_conv_intensity.argtypes = [_i64] * 14 + [ctypes.c_int, ctypes.c_int, _u64p, _dp]
        L.or_fc_intensity.argtypes = [_i64] * 3 + [ctypes.c_int, ctypes.c_int, _u64p, _dp]
        L.or_route.argtypes = [ctypes.c_uint64] * 4 + [ctypes.c_double, ctypes.c_int,
                                                        ctypes.c_double, ctypes.c_double, ctypes.c_int]
        L.or_conv2d.argtypes = ([_i64] * 14 + [ctypes.c_int, _vp, _vp, _vp, _vp, ctypes.c_int,
                                               _u32p, _i64, _i64, _dp, _dp, _u64p])
        L.or_conv2d_at.argtypes = ([_i64] * 14 + [ctypes.c_int, _vp, _vp, _vp, _vp, ctypes.c_int,
                                                  ctypes.POINTER(ctypes.c_int64), _i64, _dp, _dp])
        L.or_fc.argtypes = [_i64] * 3 + [ctypes.c_int, _vp, _vp, _vp, _vp, ctypes.c_int, _u32p,
                                         _i64, _i64, _dp, _dp]
        L.or_fc_executed_blocks.argtypes = [_vp, ctypes.c_int, _i64, _i64, _i64, _i64, _u64p]
        L.or_conv_executed_blocks.argtypes = [_vp, ctypes.c_int] + [_i64] * 14 + [_u64p]
        L.or_conv_split_executed_blocks.argtypes = ([_vp, ctypes.c_int] + [_i64] * 14 +
                                                    [ctypes.c_double, _u64p])
        L.or_maxpool2d.argtypes = [_i64] * 7 + [ctypes.c_int, _vp, _dp]
        L.or_set_threads.restype = ctypes.c_int
        L.or_set_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


# --------------------------------------------------------------------------
# Marshalling: raw bits in, numpy out.
# --------------------------------------------------------------------------

def _bits(a, dt=None):
    """Return (contiguous numpy raw-bit array, dtype code) for a tensor."""
    try:
        import torch
        if isinstance(a, torch.Tensor):
            t = a.detach().cpu().contiguous()
            code = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}[t.dtype]
            raw = t.view(torch.int32 if code == F32 else torch.int16).numpy()
            return np.ascontiguousarray(raw.view(np.uint32 if code == F32 else np.uint16)), code
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(a)
    if a.dtype == np.float32:
        return a.view(np.uint32), F32
    if a.dtype == np.float16:
        return a.view(np.uint16), F16
    if a.dtype in (np.uint16, np.uint32):
        if dt is None:
            raise ValueError("raw bit arrays need an explicit dtype code")
        return a, dt
    raise TypeError(f"unsupported array dtype {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_vp)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what}: invalid argument")


def decode(a, dt=None):
    """Decode every element to float64 with the oracle's own decoder."""
    raw, code = _bits(a, dt)
    flat = raw.reshape(-1)
    L = lib()
    return np.array([L.or_decode(_ptr(flat), code, i) for i in range(flat.size)],
                    dtype=np.float64).reshape(raw.shape)


def mask_words(rows, cols, block_rows, block_cols):
    nb = -(-rows // block_rows) * -(-cols // block_cols)
    return (nb + 31) // 32


def measure(x, rows, cols, block_rows=0, block_cols=0, samples=0, dt=None):
    """Eq. 1 statistics.  Returns dict(zeros, numel, zero_blocks, num_blocks,
    mask (uint32 array or None), per_sample (uint64 array or None))."""
    raw, code = _bits(x, dt)
    out = np.zeros(4, dtype=np.uint64)
    mask = None
    if block_rows > 0 and block_cols > 0:
        mask = np.zeros(max(1, mask_words(rows, cols, block_rows, block_cols)), dtype=np.uint32)
    ps = np.zeros(samples, dtype=np.uint64) if samples > 0 else None
    rc = lib().or_measure(_ptr(raw), code, rows, cols, block_rows, block_cols, samples,
                          out.ctypes.data_as(_u64p),
                          None if mask is None else mask.ctypes.data_as(_u32p),
                          None if ps is None else ps.ctypes.data_as(_u64p))
    _check(rc, "measure")
    return dict(zeros=int(out[0]), numel=int(out[1]), zero_blocks=int(out[2]),
                num_blocks=int(out[3]), mask=mask, per_sample=ps)


def sparsity(zeros, numel):
    return lib().or_sparsity(zeros, numel)


def out_dim(n, k, s, p, d):
    return lib().or_out_dim(n, k, s, p, d)


def conv_intensity(n, cin, h, w, cout, kh, kw, sh=1, sw=1, ph=0, pw=0, dh=1, dw=1, groups=1,
                   dt=BF16, has_bias=0):
    res = np.zeros(3, dtype=np.uint64)
    inten = ctypes.c_double()
    rc = lib().or_conv_intensity(n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, dt,
                                 has_bias, res.ctypes.data_as(_u64p), ctypes.byref(inten))
    _check(rc, "conv_intensity")
    return dict(macs=int(res[0]), flops=int(res[1]), bytes=int(res[2]), intensity=inten.value)


def fc_intensity(m, k, n, dt=BF16, has_bias=0):
    res = np.zeros(3, dtype=np.uint64)
    inten = ctypes.c_double()
    rc = lib().or_fc_intensity(m, k, n, dt, has_bias, res.ctypes.data_as(_u64p),
                               ctypes.byref(inten))
    _check(rc, "fc_intensity")
    return dict(macs=int(res[0]), flops=int(res[1]), bytes=int(res[2]), intensity=inten.value)


def route(zeros, numel, zero_blocks, num_blocks, intensity, is_depthwise, sparsity_thr,
          intensity_thr, mode=ROUTE_BLOCK):
    """Path bits (bit0 = skip, bit1 = bandwidth), or -1 for invalid input."""
    return lib().or_route(zeros, numel, zero_blocks, num_blocks, intensity, int(is_depthwise),
                          sparsity_thr, intensity_thr, mode)


def conv2d(x, w, n, cin, h, wd, cout, kh, kw, sh=1, sw=1, ph=0, pw=0, dh=1, dw=1, groups=1,
           bias=None, residual=None, act=ACT_NONE, skip_mask=None, skip_rows=0, skip_cols=0):
    """Direct NHWC convolution, y = act(conv + bias + residual).  Returns
    (y, a, macs) with y, a float64 [n, ho, wo, cout]."""
    xr, code = _bits(x)
    wr, wc = _bits(w)
    assert wc == code
    br = _bits(bias)[0] if bias is not None else None
    rr = _bits(residual)[0] if residual is not None else None
    ho, wo = out_dim(h, kh, sh, ph, dh), out_dim(wd, kw, sw, pw, dw)
    if ho <= 0 or wo <= 0:
        raise ValueError("oracle conv2d: empty output")
    y = np.zeros((n, ho, wo, cout), dtype=np.float64)
    a = np.zeros_like(y)
    macs = ctypes.c_uint64()
    rc = lib().or_conv2d(n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, code,
                         _ptr(xr), _ptr(wr), _ptr(br), _ptr(rr), act,
                         None if skip_mask is None else
                         np.ascontiguousarray(skip_mask, dtype=np.uint32).ctypes.data_as(_u32p),
                         skip_rows, skip_cols, y.ctypes.data_as(_dp), a.ctypes.data_as(_dp),
                         ctypes.byref(macs))
    _check(rc, "conv2d")
    return y, a, macs.value


def conv2d_at(x, w, idx, n, cin, h, wd, cout, kh, kw, sh=1, sw=1, ph=0, pw=0, dh=1, dw=1,
              groups=1, bias=None, residual=None, act=ACT_NONE):
    """The conv definition evaluated at flat NHWC output offsets idx."""
    xr, code = _bits(x)
    wr, _ = _bits(w)
    br = _bits(bias)[0] if bias is not None else None
    rr = _bits(residual)[0] if residual is not None else None
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    y = np.zeros(idx.size, dtype=np.float64)
    a = np.zeros_like(y)
    rc = lib().or_conv2d_at(n, cin, h, wd, cout, kh, kw, sh, sw, ph, pw, dh, dw, groups, code,
                            _ptr(xr), _ptr(wr), _ptr(br), _ptr(rr), act,
                            idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.size,
                            y.ctypes.data_as(_dp), a.ctypes.data_as(_dp))
    _check(rc, "conv2d_at")
    return y, a


def fc(x, w, m, k, n, bias=None, act=ACT_NONE, skip_mask=None, skip_rows=0, skip_cols=0,
       residual=None):
    """y[m][n] = act(bias + x w^T + residual) in double.  w is [n][k].
    Returns (y, a)."""
    xr, code = _bits(x)
    wr, _ = _bits(w)
    br = _bits(bias)[0] if bias is not None else None
    rr = _bits(residual)[0] if residual is not None else None
    y = np.zeros((m, n), dtype=np.float64)
    a = np.zeros_like(y)
    rc = lib().or_fc(m, k, n, code, _ptr(xr), _ptr(wr), _ptr(br), _ptr(rr), act,
                     None if skip_mask is None else
                     np.ascontiguousarray(skip_mask, dtype=np.uint32).ctypes.data_as(_u32p),
                     skip_rows, skip_cols, y.ctypes.data_as(_dp), a.ctypes.data_as(_dp))
    _check(rc, "fc")
    return y, a


def fc_executed_blocks(x, m, k, tile_rows, block_k):
    xr, code = _bits(x)
    out = ctypes.c_uint64()
    _check(lib().or_fc_executed_blocks(_ptr(xr), code, m, k, tile_rows, block_k,
                                       ctypes.byref(out)), "fc_executed_blocks")
    return out.value


def conv_executed_blocks(x, n, cin, h, w, kh, kw, sh, sw, ph, pw, dh, dw, tile_rows, block_c):
    xr, code = _bits(x)
    out = ctypes.c_uint64()
    _check(lib().or_conv_executed_blocks(_ptr(xr), code, n, cin, h, w, kh, kw, sh, sw, ph, pw,
                                         dh, dw, tile_rows, block_c, ctypes.byref(out)),
           "conv_executed_blocks")
    return out.value


def conv_split_executed_blocks(x, n, cin, h, w, kh, kw, sh, sw, ph, pw, dh, dw, tile_rows,
                               block_c, sparsity_thr):
    """Executed triples when each row tile is routed on its own (split execution)."""
    xr, code = _bits(x)
    out = ctypes.c_uint64()
    _check(lib().or_conv_split_executed_blocks(_ptr(xr), code, n, cin, h, w, kh, kw, sh, sw, ph,
                                               pw, dh, dw, tile_rows, block_c, sparsity_thr,
                                               ctypes.byref(out)), "conv_split_executed_blocks")
    return out.value


def set_threads(n=0):
    """Threads of the oracle's OpenMP loops (n <= 0: unchanged); returns the
    count in effect."""
    return lib().or_set_threads(int(n))


def maxpool2d(x, n, c, h, w, k=3, s=2, p=1):
    xr, code = _bits(x)
    ho, wo = out_dim(h, k, s, p, 1), out_dim(w, k, s, p, 1)
    y = np.zeros((n, ho, wo, c), dtype=np.float64)
    _check(lib().or_maxpool2d(n, c, h, w, k, s, p, code, _ptr(xr), y.ctypes.data_as(_dp)),
           "maxpool2d")
    return y
