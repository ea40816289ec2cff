"""Seeded synthetic inputs shared by the oracle checks and the GPU path.

This module holds none of the method's arithmetic: only random draws
(numpy's Philox4x32-10 counter-based generator), rounding to a storage dtype
(torch's round-to-nearest-even casts) and zero patterns.  Both sides of every
parity check read the exact bytes produced here.

Workload recipe (stands in for the paper's ImageNet / COCO inputs and
pretrained weights, which are not available; shapes follow the paper's CNN
and transformer workloads):
  * activations ~ N(0, 1), or ReLU(N(0, 1)) (about half zeros);
  * FC sweep activations: nonzeros |N(0, 1)|, zeros placed i.i.d. with
    probability rho, or as whole 16 x 16 blocks (edge-clipped) with
    probability rho;
  * weights: He normal N(0, 2 / fan_in), or N(0, 1 / fan_in) where a config
    says so.
"""
import numpy as np
import torch

_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def dtype_of(name):
    return _DT[name] if isinstance(name, str) else name


def seed_for(config: int, case: int) -> int:
    """Seed of case `case` of workload `config` (recorded in bench output)."""
    return 0x5EED0000 + config * 100 + case


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(seed))


def _to(a: np.ndarray, dtype) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dtype_of(dtype))


def normal(shape, dtype, seed, std=1.0) -> torch.Tensor:
    """N(0, std^2) rounded to dtype (CPU tensor)."""
    return _to(rng(seed).standard_normal(size=shape) * std, dtype)


def relu_normal(shape, dtype, seed) -> torch.Tensor:
    """max(N(0,1), 0) rounded to dtype: about half exact zeros."""
    a = rng(seed).standard_normal(size=shape)
    return _to(np.where(a > 0, a, 0.0), dtype)


def he_normal(shape, fan_in, dtype, seed, gain=2.0) -> torch.Tensor:
    """N(0, gain / fan_in) rounded to dtype."""
    return normal(shape, dtype, seed, std=float(np.sqrt(gain / fan_in)))


def _fix_nonzeros(t: torch.Tensor, keep_zero: np.ndarray) -> torch.Tensor:
    """Entries meant to be nonzero that rounded to zero become 1.0."""
    z = (t == 0).numpy() & ~keep_zero
    if z.any():
        t = t.clone()
        t[torch.from_numpy(z)] = 1.0
    return t


def sparse_matrix(m, k, rho, pattern, dtype, seed, block=16) -> torch.Tensor:
    """[m, k] activations: |N(0,1)| nonzeros; zeros i.i.d. ("iid") with
    probability rho, or as whole block x block tiles ("block") with
    probability rho per tile (edge tiles clipped)."""
    g = rng(seed)
    vals = np.abs(g.standard_normal(size=(m, k)))
    if pattern == "iid":
        zero = g.random(size=(m, k)) < rho
    elif pattern == "block":
        nbr, nbc = -(-m // block), -(-k // block)
        tile = g.random(size=(nbr, nbc)) < rho
        zero = np.repeat(np.repeat(tile, block, axis=0), block, axis=1)[:m, :k]
    else:
        raise ValueError(pattern)
    t = _to(np.where(zero, 0.0, vals), dtype)
    return _fix_nonzeros(t, zero)


def sparse_nhwc(n, h, w, c, rho, dtype, seed) -> torch.Tensor:
    """NHWC activations with i.i.d. zeros at rate rho, nonzeros |N(0,1)|."""
    g = rng(seed)
    vals = np.abs(g.standard_normal(size=(n, h, w, c)))
    zero = g.random(size=(n, h, w, c)) < rho
    t = _to(np.where(zero, 0.0, vals), dtype)
    return _fix_nonzeros(t, zero)
