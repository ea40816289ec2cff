"""ctypes binding of libsparoa.so (argument marshalling only).

Every function carries the name of the C entry point it calls.  Device
tensors come from PyTorch (device memory and streams are PyTorch's); no
computation of the hot path happens here.  If the HIP library is missing the
import fails loudly: there is no fallback.
"""
import ctypes
import os
from dataclasses import dataclass

import torch  # must be imported before the library: both share one HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparoa.so")

F32, F16, BF16 = 0, 1, 2
ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
PATH_DENSE_MFMA, PATH_SKIP_MFMA, PATH_DENSE_BW, PATH_SKIP_BW = 0, 1, 2, 3
ROUTE_BLOCK, ROUTE_ELEMENT = 0, 1
PATH_NAMES = {0: "dense_mfma", 1: "skip_mfma", 2: "dense_bw", 3: "skip_bw"}
COMMIT_WORDS_BYTES = 2048   # SPAROA_COMMIT_WORDS_BYTES

_TORCH_DT = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}

EXPORTS = [
    "sparoa_abi_version", "sparoa_status_string", "sparoa_last_error", "sparoa_mask_words",
    "sparoa_measure_sparsity", "sparoa_measure_sparsity_sync", "sparoa_op_intensity_conv",
    "sparoa_op_intensity_fc", "sparoa_route", "sparoa_conv2d_workspace_size",
    "sparoa_conv2d_skip_block", "sparoa_conv2d_tiling", "sparoa_conv2d", "sparoa_conv2d_dense",
    "sparoa_conv2d_zero_skip", "sparoa_fc_packed_bytes", "sparoa_fc_pack_weights",
    "sparoa_fc_tiling", "sparoa_fc_workspace_size", "sparoa_fc_skip_block", "sparoa_fc",
    "sparoa_fc_dense", "sparoa_fc_zero_skip", "sparoa_maxpool2d", "sparoa_conv2d_routed",
    "sparoa_fc_routed", "sparoa_fc_uses_packed", "sparoa_fc_ops_run",
    "sparoa_fc_measured", "sparoa_conv2d_routed_measured", "sparoa_fc_routed_measured",
    "sparoa_conv2d_split", "sparoa_fc_split", "sparoa_measure_sparsity_preset",
    "sparoa_conv2d_noalloc", "sparoa_conv2d_reads_mask", "sparoa_conv2d_routed_reads_mask",
]


class SparoaError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"sparoa status {status}: {message}")
        self.status = status


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("n", "c_in", "h", "w", "c_out", "kh", "kw", "sh", "sw", "ph", "pw", "dh", "dw",
                 "groups")] + [("dtype", ctypes.c_int), ("has_bias", ctypes.c_int)]


class FcDesc(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int64), ("k", ctypes.c_int64), ("n", ctypes.c_int64),
                ("dtype", ctypes.c_int), ("has_bias", ctypes.c_int)]


class Counts(ctypes.Structure):
    _fields_ = [("zeros", ctypes.c_uint64), ("numel", ctypes.c_uint64),
                ("zero_blocks", ctypes.c_uint64), ("num_blocks", ctypes.c_uint64)]

    def as_dict(self):
        return dict(zeros=self.zeros, numel=self.numel, zero_blocks=self.zero_blocks,
                    num_blocks=self.num_blocks)


class Intensity(ctypes.Structure):
    _fields_ = [("macs", ctypes.c_uint64), ("flops", ctypes.c_uint64),
                ("bytes", ctypes.c_uint64), ("intensity", ctypes.c_double)]

    def as_dict(self):
        return dict(macs=self.macs, flops=self.flops, bytes=self.bytes, intensity=self.intensity)


class Thresholds(ctypes.Structure):
    _fields_ = [("sparsity_thr", ctypes.c_double), ("intensity_thr", ctypes.c_double),
                ("mode", ctypes.c_int)]


class FcOp(ctypes.Structure):
    _fields_ = [("desc", FcDesc), ("x", ctypes.c_void_p), ("w_nk", ctypes.c_void_p),
                ("w_packed", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("residual", ctypes.c_void_p), ("act", ctypes.c_int),
                ("counts", ctypes.c_void_p), ("mask", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t),
                ("path", ctypes.c_void_p), ("thr", Thresholds)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                          "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "sparoa_abi_version": (ctypes.c_uint32, []),
        "sparoa_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "sparoa_last_error": (ctypes.c_char_p, []),
        "sparoa_mask_words": (ctypes.c_int, [i64, i64, i64, i64, P(i64)]),
        "sparoa_measure_sparsity": (ctypes.c_int, [vp, ctypes.c_int, i64, i64, i64, i64, i64, vp,
                                                   vp, vp, vp]),
        "sparoa_measure_sparsity_sync": (ctypes.c_int, [vp, ctypes.c_int, i64, i64, i64, i64, i64,
                                                        vp, vp, vp, P(Counts), vp]),
        "sparoa_op_intensity_conv": (ctypes.c_int, [P(ConvDesc), P(Intensity)]),
        "sparoa_op_intensity_fc": (ctypes.c_int, [P(FcDesc), P(Intensity)]),
        "sparoa_route": (ctypes.c_int, [P(Counts), P(Intensity), ctypes.c_int, P(Thresholds),
                                        P(ctypes.c_int)]),
        "sparoa_conv2d_workspace_size": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, P(sz)]),
        "sparoa_conv2d_skip_block": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, P(i64), P(i64)]),
        "sparoa_conv2d_tiling": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, P(i64), P(i64)]),
        "sparoa_conv2d_reads_mask": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, P(ctypes.c_int)]),
        "sparoa_conv2d_routed_reads_mask": (ctypes.c_int, [P(ConvDesc), P(Thresholds),
                                                           P(ctypes.c_int)]),
        "sparoa_conv2d": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, vp, vp, vp, vp, ctypes.c_int,
                                         vp, vp, vp, sz, vp, vp]),
        "sparoa_conv2d_dense": (ctypes.c_int, [P(ConvDesc), vp, vp, vp, vp, ctypes.c_int, vp, vp,
                                               sz, vp]),
        "sparoa_conv2d_noalloc": (ctypes.c_int, [P(ConvDesc), ctypes.c_int, vp, vp, vp, vp,
                                                 ctypes.c_int, vp, vp, vp, vp]),
        "sparoa_conv2d_zero_skip": (ctypes.c_int, [P(ConvDesc), vp, vp, vp, vp, ctypes.c_int, vp,
                                                   vp, vp, sz, vp, vp]),
        "sparoa_fc_packed_bytes": (ctypes.c_int, [P(FcDesc), P(sz)]),
        "sparoa_fc_pack_weights": (ctypes.c_int, [P(FcDesc), vp, vp, vp]),
        "sparoa_fc_tiling": (ctypes.c_int, [P(FcDesc), ctypes.c_int, P(i64), P(i64)]),
        "sparoa_fc_workspace_size": (ctypes.c_int, [P(FcDesc), ctypes.c_int, P(sz)]),
        "sparoa_fc_skip_block": (ctypes.c_int, [P(FcDesc), ctypes.c_int, P(i64), P(i64)]),
        "sparoa_fc_uses_packed": (ctypes.c_int, [P(FcDesc), ctypes.c_int, P(ctypes.c_int)]),
        "sparoa_fc_ops_run": (ctypes.c_int, [P(FcOp), i64, P(Thresholds), P(vp), vp]),
        "sparoa_fc_measured": (ctypes.c_int, [P(FcDesc), P(Thresholds), vp, vp, vp, vp, vp,
                                              ctypes.c_int, vp, vp, vp, vp, sz, vp, vp]),
        "sparoa_fc": (ctypes.c_int, [P(FcDesc), ctypes.c_int, vp, vp, vp, vp, ctypes.c_int, vp,
                                     vp, vp, sz, vp, vp]),
        "sparoa_fc_dense": (ctypes.c_int, [P(FcDesc), vp, vp, vp, vp, ctypes.c_int, vp, vp, sz,
                                           vp]),
        "sparoa_fc_zero_skip": (ctypes.c_int, [P(FcDesc), vp, vp, vp, vp, ctypes.c_int, vp, vp,
                                               vp, sz, vp, vp]),
        "sparoa_maxpool2d": (ctypes.c_int, [vp, ctypes.c_int, i64, i64, i64, i64, i64, i64, i64,
                                            vp, vp]),
        "sparoa_conv2d_routed": (ctypes.c_int, [P(ConvDesc), P(Thresholds), vp, vp, vp, vp, vp,
                                                ctypes.c_int, vp, vp, vp, sz, vp, vp]),
        "sparoa_fc_routed": (ctypes.c_int, [P(FcDesc), P(Thresholds), vp, vp, vp, vp, vp, vp,
                                            ctypes.c_int, vp, vp, vp, sz, vp, vp]),
        "sparoa_measure_sparsity_preset": (ctypes.c_int, [vp, ctypes.c_int, i64, i64, i64, i64,
                                                          vp, vp, vp, vp]),
        "sparoa_conv2d_split": (ctypes.c_int, [P(ConvDesc), ctypes.c_double, vp, vp, vp, vp, vp,
                                               ctypes.c_int, vp, vp, vp, sz, vp, vp]),
        "sparoa_fc_split": (ctypes.c_int, [P(FcDesc), ctypes.c_double, vp, vp, vp, vp, vp,
                                           ctypes.c_int, vp, vp, vp, sz, vp, vp]),
        "sparoa_conv2d_routed_measured": (ctypes.c_int, [P(ConvDesc), P(Thresholds), vp, vp, vp,
                                                         vp, vp, ctypes.c_int, vp, vp, vp, sz, vp,
                                                         vp, vp, vp, vp]),
        "sparoa_fc_routed_measured": (ctypes.c_int, [P(FcDesc), P(Thresholds), vp, vp, vp, vp, vp,
                                                     vp, ctypes.c_int, vp, vp, vp, sz, vp, vp, vp,
                                                     vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


_L = _load()


def _check(status):
    if status != 0:
        raise SparoaError(status, _L.sparoa_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    return stream if isinstance(stream, int) else stream.cuda_stream


def dtype_code(t):
    return _TORCH_DT[t if isinstance(t, torch.dtype) else t.dtype]


def conv_desc(n, c_in, h, w, c_out, kh, kw, sh=1, sw=1, ph=0, pw=0, dh=1, dw=1, groups=1,
              dtype=BF16, has_bias=0):
    if isinstance(dtype, torch.dtype):
        dtype = dtype_code(dtype)
    return ConvDesc(n, c_in, h, w, c_out, kh, kw, sh, sw, ph, pw, dh, dw, groups, dtype,
                    int(has_bias))


def fc_desc(m, k, n, dtype=BF16, has_bias=0):
    if isinstance(dtype, torch.dtype):
        dtype = dtype_code(dtype)
    return FcDesc(m, k, n, dtype, int(has_bias))


@dataclass
class MeasureBuffers:
    """Device buffers of one measurement: counts (4 x uint64), optional mask
    and per-sample counts."""
    counts: torch.Tensor
    mask: torch.Tensor = None
    per_sample: torch.Tensor = None


# ------------------------------------------------------------------ calls

def sparoa_abi_version():
    return _L.sparoa_abi_version()


def sparoa_status_string(status):
    return _L.sparoa_status_string(status).decode()


def sparoa_last_error():
    return _L.sparoa_last_error().decode()


def sparoa_mask_words(rows, cols, block_rows, block_cols):
    w = ctypes.c_int64()
    _check(_L.sparoa_mask_words(rows, cols, block_rows, block_cols, ctypes.byref(w)))
    return w.value


def sparoa_measure_sparsity(x, rows, cols, block_rows, block_cols, samples, counts, mask=None,
                            per_sample=None, stream=None, dtype=None):
    _check(_L.sparoa_measure_sparsity(
        _ptr(x), dtype_code(x) if dtype is None else dtype, rows, cols, block_rows, block_cols,
        samples, _ptr(counts), _ptr(mask), _ptr(per_sample), _stream(stream)))


def sparoa_measure_sparsity_preset(x, rows, cols, block_rows, block_cols, counts, mask,
                                   stream=None, dtype=None, commit=None):
    """Measurement into counters already set to {0, numel, nb, nb} (see sparoa.h);
    commit: zeroed count-commit words, or None."""
    _check(_L.sparoa_measure_sparsity_preset(
        _ptr(x), dtype_code(x) if dtype is None else dtype, rows, cols, block_rows, block_cols,
        _ptr(counts), _ptr(mask), _ptr(commit), _stream(stream)))


def sparoa_measure_sparsity_sync(x, rows, cols, block_rows, block_cols, samples, counts,
                                 mask=None, per_sample=None, stream=None, dtype=None):
    host = Counts()
    _check(_L.sparoa_measure_sparsity_sync(
        _ptr(x), dtype_code(x) if dtype is None else dtype, rows, cols, block_rows, block_cols,
        samples, _ptr(counts), _ptr(mask), _ptr(per_sample), ctypes.byref(host),
        _stream(stream)))
    return host.as_dict()


def sparoa_op_intensity_conv(desc):
    out = Intensity()
    _check(_L.sparoa_op_intensity_conv(ctypes.byref(desc), ctypes.byref(out)))
    return out.as_dict()


def sparoa_op_intensity_fc(desc):
    out = Intensity()
    _check(_L.sparoa_op_intensity_fc(ctypes.byref(desc), ctypes.byref(out)))
    return out.as_dict()


def sparoa_route(counts, intensity, is_depthwise, sparsity_thr, intensity_thr, mode=ROUTE_BLOCK):
    c = Counts(counts["zeros"], counts["numel"], counts["zero_blocks"], counts["num_blocks"])
    i = Intensity(intensity["macs"], intensity["flops"], intensity["bytes"],
                  intensity["intensity"])
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    out = ctypes.c_int()
    _check(_L.sparoa_route(ctypes.byref(c), ctypes.byref(i), int(is_depthwise), ctypes.byref(t),
                           ctypes.byref(out)))
    return out.value


def _pair(fn, desc, path):
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _check(fn(ctypes.byref(desc), path, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def sparoa_conv2d_workspace_size(desc, path):
    s = ctypes.c_size_t()
    _check(_L.sparoa_conv2d_workspace_size(ctypes.byref(desc), path, ctypes.byref(s)))
    return s.value


def sparoa_conv2d_skip_block(desc, path):
    return _pair(_L.sparoa_conv2d_skip_block, desc, path)


def sparoa_conv2d_reads_mask(desc, path):
    """Whether the kernel serving `path` reads x's bitmap."""
    v = ctypes.c_int()
    _check(_L.sparoa_conv2d_reads_mask(ctypes.byref(desc), path, ctypes.byref(v)))
    return bool(v.value)


def sparoa_conv2d_routed_reads_mask(desc, sparsity_thr, intensity_thr, mode):
    """Whether the routed conv's skip kernel reads x's bitmap (else mask may be None)."""
    v = ctypes.c_int()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_conv2d_routed_reads_mask(ctypes.byref(desc), ctypes.byref(t),
                                              ctypes.byref(v)))
    return bool(v.value)


def sparoa_conv2d_tiling(desc, path):
    return _pair(_L.sparoa_conv2d_tiling, desc, path)


def sparoa_conv2d(desc, path, x, w, bias, residual, act, mask, y, workspace=None,
                  executed=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_conv2d(ctypes.byref(desc), path, _ptr(x), _ptr(w), _ptr(bias),
                            _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes,
                            _ptr(executed), _stream(stream)))


def sparoa_conv2d_noalloc(desc, path, x, w, bias, residual, act, mask, y, executed=None,
                          stream=None):
    """sparoa_conv2d with its split-K scratch in the library's own device array."""
    _check(_L.sparoa_conv2d_noalloc(ctypes.byref(desc), path, _ptr(x), _ptr(w), _ptr(bias),
                                    _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(executed),
                                    _stream(stream)))


def sparoa_conv2d_dense(desc, x, w, bias, residual, act, y, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_conv2d_dense(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias),
                                  _ptr(residual), act, _ptr(y), _ptr(workspace), ws_bytes,
                                  _stream(stream)))


def sparoa_conv2d_zero_skip(desc, x, w, bias, residual, act, mask, y, workspace=None,
                            executed=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_conv2d_zero_skip(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias),
                                      _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(workspace),
                                      ws_bytes, _ptr(executed), _stream(stream)))


def sparoa_fc_packed_bytes(desc):
    s = ctypes.c_size_t()
    _check(_L.sparoa_fc_packed_bytes(ctypes.byref(desc), ctypes.byref(s)))
    return s.value


def sparoa_fc_pack_weights(desc, w_nk, w_packed, stream=None):
    _check(_L.sparoa_fc_pack_weights(ctypes.byref(desc), _ptr(w_nk), _ptr(w_packed),
                                     _stream(stream)))


def sparoa_fc_tiling(desc, path):
    return _pair(_L.sparoa_fc_tiling, desc, path)


def sparoa_fc_workspace_size(desc, path):
    s = ctypes.c_size_t()
    _check(_L.sparoa_fc_workspace_size(ctypes.byref(desc), path, ctypes.byref(s)))
    return s.value


def sparoa_fc_skip_block(desc, path):
    return _pair(_L.sparoa_fc_skip_block, desc, path)


def sparoa_fc(desc, path, x, w, bias, residual, act, mask, y, workspace=None, executed=None,
              stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_fc(ctypes.byref(desc), path, _ptr(x), _ptr(w), _ptr(bias), _ptr(residual),
                        act, _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes, _ptr(executed),
                        _stream(stream)))


def sparoa_fc_dense(desc, x, w, bias, residual, act, y, workspace=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_fc_dense(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias), _ptr(residual),
                              act, _ptr(y), _ptr(workspace), ws_bytes, _stream(stream)))


def sparoa_fc_zero_skip(desc, x, w, bias, residual, act, mask, y, workspace=None, executed=None,
                        stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_fc_zero_skip(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias),
                                  _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(workspace),
                                  ws_bytes, _ptr(executed), _stream(stream)))


def sparoa_maxpool2d(x, n, c, h, w, k, s, p, y, stream=None):
    _check(_L.sparoa_maxpool2d(_ptr(x), dtype_code(x), n, c, h, w, k, s, p, _ptr(y),
                               _stream(stream)))


def sparoa_conv2d_routed(desc, sparsity_thr, intensity_thr, mode, counts, x, w, bias, residual,
                         act, mask, y, workspace=None, path=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_conv2d_routed(ctypes.byref(desc), ctypes.byref(t), _ptr(counts), _ptr(x),
                                   _ptr(w), _ptr(bias), _ptr(residual), act, _ptr(mask), _ptr(y),
                                   _ptr(workspace), ws_bytes, _ptr(path), _stream(stream)))


def sparoa_fc_routed(desc, sparsity_thr, intensity_thr, mode, counts, x, w_nk, w_packed, bias,
                     residual, act, mask, y, workspace=None, path=None, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_fc_routed(ctypes.byref(desc), ctypes.byref(t), _ptr(counts), _ptr(x),
                               _ptr(w_nk), _ptr(w_packed), _ptr(bias), _ptr(residual), act,
                               _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes, _ptr(path),
                               _stream(stream)))


def sparoa_conv2d_routed_measured(desc, sparsity_thr, intensity_thr, mode, counts, x, w, bias,
                                  residual, act, mask, y, y_counts, y_mask, workspace=None,
                                  path=None, y_commit=None, stream=None):
    """sparoa_conv2d_routed that also measures y into y_counts / y_mask
    (y_mask None: counts only; y_commit: zeroed count-commit words, or None)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_conv2d_routed_measured(
        ctypes.byref(desc), ctypes.byref(t), _ptr(counts), _ptr(x), _ptr(w), _ptr(bias),
        _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes, _ptr(path),
        _ptr(y_counts), _ptr(y_mask), _ptr(y_commit), _stream(stream)))


def sparoa_fc_routed_measured(desc, sparsity_thr, intensity_thr, mode, counts, x, w_nk, w_packed,
                              bias, residual, act, mask, y, y_counts, y_mask, workspace=None,
                              path=None, y_commit=None, stream=None):
    """sparoa_fc_routed that also measures y into y_counts / y_mask
    (y_commit: zeroed count-commit words, or None)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_fc_routed_measured(
        ctypes.byref(desc), ctypes.byref(t), _ptr(counts), _ptr(x), _ptr(w_nk), _ptr(w_packed),
        _ptr(bias), _ptr(residual), act, _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes,
        _ptr(path), _ptr(y_counts), _ptr(y_mask), _ptr(y_commit), _stream(stream)))


def sparoa_conv2d_split(desc, sparsity_thr, sample_zeros, x, w, bias, residual, act, mask, y,
                        workspace=None, executed=None, stream=None):
    """One conv split over the skip and dense paths by row tile (see sparoa.h)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_conv2d_split(ctypes.byref(desc), sparsity_thr, _ptr(sample_zeros), _ptr(x),
                                  _ptr(w), _ptr(bias), _ptr(residual), act, _ptr(mask), _ptr(y),
                                  _ptr(workspace), ws_bytes, _ptr(executed), _stream(stream)))


def sparoa_fc_split(desc, sparsity_thr, row_zeros, x, w_nk, bias, residual, act, mask, y,
                    workspace=None, executed=None, stream=None):
    """One FC split over the skip and dense paths by row tile (see sparoa.h)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_L.sparoa_fc_split(ctypes.byref(desc), sparsity_thr, _ptr(row_zeros), _ptr(x),
                              _ptr(w_nk), _ptr(bias), _ptr(residual), act, _ptr(mask), _ptr(y),
                              _ptr(workspace), ws_bytes, _ptr(executed), _stream(stream)))


def sparoa_fc_measured(desc, sparsity_thr, intensity_thr, mode, x, w_nk, w_packed, bias, residual,
                       act, counts, mask, y, workspace=None, path=None, stream=None):
    """Measure -> route -> execute of one FC (see sparoa.h)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(sparsity_thr, intensity_thr, mode)
    _check(_L.sparoa_fc_measured(ctypes.byref(desc), ctypes.byref(t), _ptr(x), _ptr(w_nk),
                                 _ptr(w_packed), _ptr(bias), _ptr(residual), act, _ptr(counts),
                                 _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes, _ptr(path),
                                 _stream(stream)))


def sparoa_fc_uses_packed(desc, path):
    v = ctypes.c_int()
    _check(_L.sparoa_fc_uses_packed(ctypes.byref(desc), path, ctypes.byref(v)))
    return bool(v.value)


def fc_op(desc, x, w_nk, w_packed, bias, residual, act, counts, mask, y, workspace=None,
          path=None, thresholds=None):
    """One entry of a sparoa_fc_ops_run batch (pointers captured now).
    thresholds: (sparsity_thr, intensity_thr, mode) of this op, used when the
    batch call passes no thresholds of its own."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    t = Thresholds(*(thresholds or (0.5, 315.0, ROUTE_BLOCK)))
    return FcOp(desc, _ptr(x), _ptr(w_nk), _ptr(w_packed), _ptr(bias), _ptr(residual), act,
                _ptr(counts), _ptr(mask), _ptr(y), _ptr(workspace), ws_bytes, _ptr(path), t)


def fc_op_array(ops):
    return (FcOp * len(ops))(*ops)


def sparoa_fc_ops_run(op_array, sparsity_thr=None, intensity_thr=None, mode=ROUTE_BLOCK,
                      events=None, stream=None):
    """Runs a batch built by fc_op_array with the given thresholds, or with
    each op's own when sparsity_thr is None.  events: flat list of 2n
    recorded torch.cuda.Event objects (or None)."""
    t = None if sparsity_thr is None else ctypes.byref(Thresholds(sparsity_thr, intensity_thr, mode))
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    _check(_L.sparoa_fc_ops_run(op_array, len(op_array), t, ev, _stream(stream)))