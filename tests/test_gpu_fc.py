"""GPU parity of the FC paths (dense MFMA, zero-skip MFMA, bandwidth, skip
bandwidth) against the double-precision oracle, plus the bit-exact work
counts and the skip == dense identity of the MFMA pair."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import RTOL, assert_close

pytestmark = pytest.mark.gpu

DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def run_fc(x, w, bias, act, path, wp=None, residual=None):
    """Measures x at the path's skip granularity, runs the path; returns
    (y, executed, counts, mask)."""
    abi = _abi()
    dev = torch.device("cuda")
    m, k = x.shape
    n = w.shape[0]
    d = abi.fc_desc(m, k, n, x.dtype, has_bias=bias is not None)
    xd = x.to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    br, bc = abi.sparoa_fc_skip_block(d, path)
    mask = torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32, device=dev)
    c = abi.sparoa_measure_sparsity_sync(xd, m, k, br, bc, 0, counts, mask)
    if abi.sparoa_fc_uses_packed(d, path):
        if wp is None:
            wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // x.element_size(), dtype=x.dtype,
                             device=dev)
            abi.sparoa_fc_pack_weights(d, w.to(dev), wp)
        wt = wp
    else:
        wt = w.to(dev)
    ws = torch.zeros(max(16, abi.sparoa_fc_workspace_size(d, path)), dtype=torch.uint8,
                     device=dev)
    y = torch.full((m, n), float("nan"), dtype=x.dtype, device=dev)
    ex = torch.full((1,), -1, dtype=torch.int64, device=dev)
    abi.sparoa_fc(d, path, xd, wt, None if bias is None else bias.to(dev),
                  None if residual is None else residual.to(dev), act,
                  mask if path & 1 else None, y, ws, ex if path & 1 else None)
    torch.cuda.synchronize()
    return y.cpu(), int(ex.item()), c, mask


SHAPES = [(1, 256, 64), (8, 512, 192), (16, 640, 100), (33, 96, 70), (64, 1024, 256),
          (5, 1000, 64), (64, 4096, 128), (65, 256, 64), (96, 520, 130)]


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("path", [0, 1, 2, 3])
def test_fc_paths_vs_oracle(dt, shape, path):
    m, k, n = shape
    seed = SHAPES.index(shape) * 10 + path
    x = synth.sparse_matrix(m, k, 0.7, "iid" if path != 3 else "block", dt, seed)
    w = synth.normal((n, k), dt, seed + 1, std=k ** -0.5)
    b = synth.normal((n,), dt, seed + 2)
    r = synth.normal((m, n), dt, seed + 3)
    y, ex, _, _ = run_fc(x, w, b, 1, path, residual=r)
    yr, ar = oracle.fc(x, w, m, k, n, bias=b, act=oracle.ACT_RELU, residual=r)
    assert_close(y, yr, ar, RTOL[DT[dt]], f"fc {shape} path {path}")
    abi = _abi()
    if path & 1:
        tr, kc = abi.sparoa_fc_tiling(abi.fc_desc(m, k, n, DT[dt]), path)
        assert ex == oracle.fc_executed_blocks(x, m, k, tr, kc)


@pytest.mark.parametrize("shape", [(1, 256, 64), (37, 320, 96), (200, 512, 130)])
def test_fc_fp32_mfma(shape):
    m, k, n = shape
    x = synth.sparse_matrix(m, k, 0.5, "iid", "f32", 500 + m)
    w = synth.normal((n, k), "f32", 501 + m, std=k ** -0.5)
    for path in (0, 1, 2, 3):      # fp32 bandwidth paths run the implicit GEMM
        y, _, _, _ = run_fc(x, w, None, 0, path)
        yr, ar = oracle.fc(x, w, m, k, n)
        assert_close(y, yr, ar, RTOL[torch.float32], f"fc f32 {shape} path {path}")


@pytest.mark.parametrize("m,k,n", [(256, 768, 3072), (300, 3072, 768), (64, 4096, 4096)])
@pytest.mark.parametrize("pattern", ["iid", "block"])
def test_fc_skip_mfma_equals_dense_bitwise(m, k, n, pattern):
    x = synth.sparse_matrix(m, k, 0.95, pattern, "f16", m + k)
    w = synth.normal((n, k), "f16", n, std=k ** -0.5)
    yd, _, _, _ = run_fc(x, w, None, 0, 0)
    ys, ex, _, _ = run_fc(x, w, None, 0, 1)
    assert torch.equal(yd, ys)
    abi = _abi()
    tr, kc = abi.sparoa_fc_tiling(abi.fc_desc(m, k, n, torch.float16), 1)
    assert ex == oracle.fc_executed_blocks(x, m, k, tr, kc)


def test_fc_all_zero_input_gives_bias():
    m, k, n = 8, 512, 128
    x = torch.zeros(m, k, dtype=torch.bfloat16)
    w = synth.normal((n, k), "bf16", 9)
    b = synth.normal((n,), "bf16", 10)
    for path in (1, 3):
        y, ex, c, _ = run_fc(x, w, b, 0, path)
        assert ex == 0 and c["zero_blocks"] == c["num_blocks"]
        assert torch.equal(y, b.reshape(1, n).expand(m, n))


@pytest.mark.parametrize("m", [1, 8, 64])
@pytest.mark.parametrize("rho", [0.0, 0.5, 0.8, 0.95])
@pytest.mark.parametrize("pattern", ["iid", "block"])
def test_fc_sweep_full_size(m, rho, pattern):
    """The FC sweep workload at full size: [m, 4096] x [4096, 4096] bf16."""
    abi = _abi()
    k = n = 4096
    case = [1, 8, 64].index(m) * 8 + [0.0, 0.5, 0.8, 0.95].index(rho) * 2 + \
        ["iid", "block"].index(pattern)
    x = synth.sparse_matrix(m, k, rho, pattern, "bf16", synth.seed_for(2, case))
    w = synth.normal((n, k), "bf16", synth.seed_for(2, 50), std=1 / 64)
    d = abi.fc_desc(m, k, n, abi.BF16)
    inten = abi.sparoa_op_intensity_fc(d)
    path_bw = 2 if inten["intensity"] < 315.0 else 0
    assert path_bw == 2                     # every sweep case is memory-bound
    yr, ar = oracle.fc(x, w, m, k, n)
    for path in (path_bw, path_bw | 1):
        y, ex, c, _ = run_fc(x, w, None, 0, path)
        assert_close(y, yr, ar, RTOL[torch.bfloat16], f"sweep m={m} rho={rho} {pattern} p{path}")
        br, bc = abi.sparoa_fc_skip_block(d, path)
        ref = oracle.measure(x, m, k, br, bc)
        assert (c["zeros"], c["zero_blocks"], c["num_blocks"]) == \
            (ref["zeros"], ref["zero_blocks"], ref["num_blocks"])
        got = abi.sparoa_route(c, inten, 0, 0.5, 315.0)
        assert got == oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"],
                                   ref["num_blocks"], inten["intensity"], 0, 0.5, 315.0)
        if path & 1:
            assert ex == oracle.fc_executed_blocks(x, m, k, m, 1)
