"""Shared helpers of the parity tests (comparison only; no method arithmetic)."""
import numpy as np
import torch

# Tolerances: relative to the abs-product sum |bias| + sum |x w| (+ |residual|)
# per element, and normwise relative to ||y_ref||_2.
RTOL = {torch.float32: 1e-5, torch.float16: 2e-2, torch.bfloat16: 2e-2}
# Outputs are stored in the input dtype: a result in the subnormal range can
# be off by one step of the dtype's subnormal spacing whatever the accuracy
# of the sum (binary16: 2^-24, bfloat16: 2^-133, binary32: 2^-149).
SUBNORMAL_STEP = {torch.float32: 2.0 ** -149, torch.float16: 2.0 ** -24,
                  torch.bfloat16: 2.0 ** -133}


def assert_close(y_gpu, y_ref, a_ref, rtol, what=""):
    yg = y_gpu.detach().float().cpu().numpy().astype(np.float64).reshape(y_ref.shape)
    err = np.abs(yg - y_ref)
    bound = rtol * a_ref + SUBNORMAL_STEP[y_gpu.dtype]
    bad = err > bound
    if bad.any():
        i = int(np.argmax(np.where(bad, err - bound, -np.inf)))
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {err.size} elements out of tolerance; worst at flat "
            f"{i}: gpu {yg.flat[i]!r} ref {y_ref.flat[i]!r} bound {bound.flat[i]!r}")
    nref = float(np.linalg.norm(y_ref))
    nerr = float(np.linalg.norm(yg - y_ref))
    assert nerr <= rtol * nref + 1e-300, f"{what}: normwise error {nerr} vs {rtol} * {nref}"
    return float(err.max()), nerr / max(nref, 1e-300)


def mask_np(mask_t):
    return mask_t.detach().cpu().numpy().view(np.uint32)


def gpu_available():
    return torch.cuda.is_available()
