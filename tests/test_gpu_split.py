"""Split execution of one operator over the zero-skip and dense paths (each
row tile of the implicit GEMM routed by the zero fraction of the samples its
rows come from): the executed work must equal the oracle's count under the
same per-tile rule, bit for bit, the output must equal the dense path's bit
for bit, and it must lie within the dtype's tolerance of the oracle's direct
conv / FC element by element."""
import pytest
import torch

import oracle
import synth
from tests._util import RTOL, assert_close

pytestmark = pytest.mark.gpu


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def _mixed_batch(n, h, w, c, dt, seed):
    """Samples of very different sparsity: dense, ReLU-half, block-sparse and
    all-zero samples in turn."""
    xs = []
    for s in range(n):
        kind = s % 4
        if kind == 0:
            xs.append(synth.normal((1, h, w, c), dt, seed + s).abs())
        elif kind == 1:
            xs.append(synth.relu_normal((1, h, w, c), dt, seed + s))
        elif kind == 2:
            xs.append(synth.sparse_matrix(h * w, c, 0.9, "block", dt, seed + s).reshape(1, h, w, c))
        else:
            xs.append(torch.zeros(1, h, w, c, dtype=xs[0].dtype))
    return torch.cat(xs)


CONV_CASES = [
    # n, cin, h, w, cout, k, stride, dtype
    (8, 64, 12, 12, 64, 3, 1, "bf16"),     # 64 x 64 tiles straddling samples, split-K
    (12, 128, 16, 16, 128, 3, 1, "f16"),   # 128 x 64 tiles
    (6, 64, 15, 11, 64, 1, 1, "bf16"),     # 1x1, ragged last tile
    (5, 64, 14, 14, 128, 3, 2, "bf16"),    # stride 2
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv2d_split(case):
    abi = _abi()
    dev = torch.device("cuda")
    n, cin, h, w, cout, k, s, dt = case
    tdt = torch.float16 if dt == "f16" else torch.bfloat16
    p = k // 2
    d = abi.conv_desc(n, cin, h, w, cout, k, k, s, s, p, p, 1, 1, 1, tdt)
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    seed = 1300 + 10 * CONV_CASES.index(case)
    x = _mixed_batch(n, h, w, cin, dt, seed)
    wt = synth.he_normal((cout, k, k, cin), k * k * cin, dt, seed + 7)
    xd, wd = x.to(dev), wt.to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * w, cin, 1, 8), dtype=torch.int32, device=dev)
    zs = torch.zeros(n, dtype=torch.int64, device=dev)
    abi.sparoa_measure_sparsity(xd, n * h * w, cin, 1, 8, n, counts, mask, zs)
    ws = torch.zeros(max(16, max(abi.sparoa_conv2d_workspace_size(d, q) for q in range(4))),
                     dtype=torch.uint8, device=dev)
    y_dense = torch.empty(n, ho, wo, cout, dtype=tdt, device=dev)
    abi.sparoa_conv2d(d, abi.PATH_DENSE_MFMA, xd, wd, None, None, abi.ACT_RELU, None, y_dense, ws)
    yr, ar, _ = oracle.conv2d(x, wt, n, cin, h, w, cout, k, k, s, s, p, p, act=oracle.ACT_RELU)
    rows, kc = abi.sparoa_conv2d_tiling(d, abi.PATH_SKIP_MFMA)
    assert kc == 64
    for thr in (0.0, 0.3, 0.5, 0.9, 2.0):
        y = torch.full_like(y_dense, float("nan"))
        ex = torch.full((1,), -1, dtype=torch.int64, device=dev)
        abi.sparoa_conv2d_split(d, thr, zs, xd, wd, None, None, abi.ACT_RELU, mask, y, ws, ex)
        torch.cuda.synchronize()
        assert_close(y, yr, ar, RTOL[tdt], f"split conv {case} thr {thr} vs oracle")
        assert torch.equal(y, y_dense), f"{case} thr {thr}"
        want = oracle.conv_split_executed_blocks(x, n, cin, h, w, k, k, s, s, p, p, 1, 1, rows,
                                                 64, thr)
        assert int(ex.item()) == want, f"{case} thr {thr}"


@pytest.mark.parametrize("m,k,n", [(300, 512, 256), (64, 4096, 1024)])
def test_fc_split(m, k, n):
    abi = _abi()
    dev = torch.device("cuda")
    d = abi.fc_desc(m, k, n, abi.BF16)
    # rows of varying sparsity: row r has zero fraction about (r % 10) / 10
    x = torch.cat([synth.sparse_matrix(1, k, (r % 10) / 10, "iid", "bf16", 1400 + r)
                   for r in range(m)])
    w = synth.normal((n, k), "bf16", 1500, std=k ** -0.5)
    xd, wd = x.to(dev), w.to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(m, k, 1, 8), dtype=torch.int32, device=dev)
    zs = torch.zeros(m, dtype=torch.int64, device=dev)
    abi.sparoa_measure_sparsity(xd, m, k, 1, 8, m, counts, mask, zs)
    ws = torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, q) for q in range(4))),
                     dtype=torch.uint8, device=dev)
    y_dense = torch.empty(m, n, dtype=torch.bfloat16, device=dev)
    abi.sparoa_fc(d, abi.PATH_DENSE_MFMA, xd, wd, None, None, abi.ACT_NONE, None, y_dense, ws)
    yr, ar = oracle.fc(x, w, m, k, n)
    rows, kc = abi.sparoa_fc_tiling(d, abi.PATH_SKIP_MFMA)
    for thr in (0.0, 0.45, 0.85, 2.0):
        y = torch.full_like(y_dense, float("nan"))
        ex = torch.full((1,), -1, dtype=torch.int64, device=dev)
        abi.sparoa_fc_split(d, thr, zs, xd, wd, None, None, abi.ACT_NONE, mask, y, ws, ex)
        torch.cuda.synchronize()
        assert_close(y, yr, ar, RTOL[torch.bfloat16], f"split fc {m}x{k}x{n} thr {thr} vs oracle")
        assert torch.equal(y, y_dense), f"thr {thr}"
        want = oracle.conv_split_executed_blocks(x.reshape(m, 1, 1, k), m, k, 1, 1, 1, 1, 1, 1,
                                                 0, 0, 1, 1, rows, kc, thr)
        assert int(ex.item()) == want, f"thr {thr}"


def test_split_rejects_unsupported_shapes():
    abi = _abi()
    dev = torch.device("cuda")
    d = abi.conv_desc(1, 32, 8, 8, 64, 3, 3, 1, 1, 1, 1, 1, 1, 1, torch.bfloat16)  # C_in % 64
    t = torch.zeros(4096, dtype=torch.bfloat16, device=dev)
    z = torch.zeros(8, dtype=torch.int64, device=dev)
    with pytest.raises(abi.SparoaError):
        abi.sparoa_conv2d_split(d, 0.5, z, t, t, None, None, abi.ACT_NONE, z, t)
