"""Output measurement fused into the producer (a layer measuring its own
output, the next layer's input): the counts and bitmap must equal the
oracle's measurement of the output bit for bit, and the output must equal
the unfused routed call's bit for bit -- on the fused epilogue, on the fused
split-K reduction, and on the fallbacks (a standalone pass after the layer)."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def _fresh_counts(rows, cols, dev):
    """y_counts as the measured calls expect them on entry: {0, numel, nb, nb}."""
    nb = rows * -(-cols // 8)
    return torch.tensor([0, rows * cols, nb, nb], dtype=torch.int64, device=dev)


def _check_y_measurement(abi, y, rows, cols, y_counts, y_mask, what):
    """y_mask None: a counts-only measurement (the four counts, no bitmap)."""
    ref = oracle.measure(y.cpu(), rows, cols, 1, 8)
    assert y_counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                       ref["num_blocks"]], what
    if y_mask is not None:
        assert np.array_equal(y_mask.cpu().numpy().view(np.uint32), ref["mask"]), what


CONV_CASES = [
    # n, cin, h, w, cout, k, s, dtype; comment: which form runs
    (8, 64, 32, 32, 128, 3, 1, "bf16"),    # fused epilogue, 64 x 64 tiles, no split
    (4, 64, 32, 32, 64, 1, 1, "f16"),      # fused epilogue, 128 x 64 tiles
    (1, 256, 14, 14, 128, 3, 1, "bf16"),   # split-K: fused reduction
    (1, 128, 14, 14, 128, 3, 1, "bf16"),   # too few chunks to split: fused epilogue
    (3, 192, 15, 13, 64, 3, 2, "f16"),     # ragged rows, split-K
    (15, 64, 29, 31, 64, 3, 1, "bf16"),    # ragged rows in the last tile, no split
    (13, 64, 59, 61, 256, 3, 1, "bf16"),   # 128 x 128 tiles, ragged rows (732 tiles)
    (4, 128, 57, 55, 512, 1, 1, "bf16"),   # 128 x 256 tiles (1x1), ragged rows (196 tiles)
    (5, 64, 120, 120, 64, 3, 1, "f16"),    # 128 x 64 tiles (563 tiles)
    (2, 64, 16, 16, 96, 1, 1, "bf16"),     # c_out % 64 != 0: standalone pass
    (2, 3, 40, 40, 64, 7, 2, "bf16"),      # image stem (small-channel kernel): counts fused
    (3, 3, 30, 34, 32, 3, 2, "f16"),       # MobileNetV2-like stem, ragged rows: counts fused
    (2, 32, 16, 16, 64, 3, 1, "bf16"),     # c_in < 48, not a multiple of 64 (first-generation GEMM): standalone
    (4, 96, 14, 14, 576, 1, 1, "f16"),     # c_in % 64 != 0 (partial chunks): fused epilogue
    (2, 160, 7, 7, 960, 1, 1, "f16"),      # partial chunks, 160 = 2 x 64 + 32
    (1, 160, 7, 7, 192, 3, 1, "bf16"),     # partial chunks, split-K: fused reduction
    (1, 160, 7, 7, 96, 3, 1, "bf16"),      # c_out % 64 != 0, split-K: the reduction measures
    (8, 1920, 7, 7, 160, 1, 1, "f16"),     # c_out = 160, split-K: the reduction measures
    (32, 960, 7, 7, 160, 1, 1, "f16"),     # MobileNetV2 project (c_out = 160, no split): standalone
    (3, 72, 17, 15, 128, 3, 1, "bf16"),    # partial chunks per tap of a 3x3 kernel
    (2, 64, 16, 16, 64, 3, 1, "f32"),      # fp32: standalone pass
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_routed_measured(case):
    abi = _abi()
    dev = torch.device("cuda")
    n, cin, h, w, cout, k, s, dt = case
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dt]
    p = k // 2
    d = abi.conv_desc(n, cin, h, w, cout, k, k, s, s, p, p, 1, 1, 1, tdt, has_bias=True)
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    seed = 1100 + CONV_CASES.index(case) * 5
    x = synth.relu_normal((n, h, w, cin), dt, seed).to(dev)
    wt = synth.he_normal((cout, k, k, cin), k * k * cin, dt, seed + 1).to(dev)
    b = synth.normal((cout,), dt, seed + 2).to(dev)
    r = synth.normal((n, ho, wo, cout), dt, seed + 3).to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * w, cin, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x, n * h * w, cin, 1, 8, 0, counts, mask)
    # workspace contents on entry do not matter
    ws = torch.full((max(16, max(abi.sparoa_conv2d_workspace_size(d, q) for q in range(4))),),
                    0xA5, dtype=torch.uint8, device=dev)
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    rows, cols = n * ho * wo, cout
    # the GEMM measures y itself (ticketed commits through `commit`)
    fused = dt != "f32" and (cin % 64 == 0 or (cin % 8 == 0 and cin >= 48)) and cout % 64 == 0
    for s_thr in (0.0, 2.0):       # skip and dense routes
        y = torch.full((n, ho, wo, cout), float("nan"), dtype=tdt, device=dev)
        y_counts = _fresh_counts(rows, cols, dev)
        y_mask = torch.full((abi.sparoa_mask_words(rows, cols, 1, 8),), -1, dtype=torch.int32,
                            device=dev)
        path = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_conv2d_routed_measured(d, s_thr, 0.0, abi.ROUTE_BLOCK, counts, x, wt, b, r,
                                          abi.ACT_RELU, mask, y, y_counts, y_mask, ws, path,
                                          commit)
        y2 = torch.full_like(y, float("nan"))
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_conv2d_routed(d, s_thr, 0.0, abi.ROUTE_BLOCK, counts, x, wt, b, r,
                                 abi.ACT_RELU, mask, y2, ws, p2)
        torch.cuda.synchronize()
        assert int(path.item()) == int(p2.item())
        assert torch.equal(y, y2), f"{case} s_thr {s_thr}"
        _check_y_measurement(abi, y, rows, cols, y_counts, y_mask, f"{case} s_thr {s_thr}")
        # the count-commit words are left zero for the next call
        assert int(commit.count_nonzero().item()) == 0
    if fused:       # no commit words: direct commits, same counts
        y = torch.full((n, ho, wo, cout), float("nan"), dtype=tdt, device=dev)
        y_counts = _fresh_counts(rows, cols, dev)
        y_mask = torch.full((abi.sparoa_mask_words(rows, cols, 1, 8),), -1, dtype=torch.int32,
                            device=dev)
        abi.sparoa_conv2d_routed_measured(d, 0.0, 0.0, abi.ROUTE_BLOCK, counts, x, wt, b, r,
                                          abi.ACT_RELU, mask, y, y_counts, y_mask, ws)
        torch.cuda.synchronize()
        _check_y_measurement(abi, y, rows, cols, y_counts, y_mask, f"{case} direct commits")
    if cout % 8 == 0:   # counts only (no bitmap): fused or standalone, same counts
        for s_thr in (0.0, 2.0):
            y = torch.full((n, ho, wo, cout), float("nan"), dtype=tdt, device=dev)
            y_counts = _fresh_counts(rows, cols, dev)
            abi.sparoa_conv2d_routed_measured(d, s_thr, 0.0, abi.ROUTE_BLOCK, counts, x, wt, b, r,
                                              abi.ACT_RELU, mask, y, y_counts, None, ws, None,
                                              commit)
            y2 = torch.full_like(y, float("nan"))
            abi.sparoa_conv2d_routed(d, s_thr, 0.0, abi.ROUTE_BLOCK, counts, x, wt, b, r,
                                     abi.ACT_RELU, mask, y2, ws)
            torch.cuda.synchronize()
            assert torch.equal(y, y2), f"{case} counts only s_thr {s_thr}"
            _check_y_measurement(abi, y, rows, cols, y_counts, None,
                                 f"{case} counts only s_thr {s_thr}")
            assert int(commit.count_nonzero().item()) == 0


DW_CASES = [
    # n, c, h, w, stride, dtype: MobileNetV2 depthwise shapes and ragged ones;
    # the 16-bit 3x3 cases measure in the kernel, fp32 in a standalone pass
    (2, 144, 56, 56, 1, "f16"),    # 18 channel vectors per pixel
    (2, 96, 112, 112, 2, "bf16"),  # stride 2
    (3, 384, 14, 14, 1, "bf16"),
    (3, 576, 14, 14, 2, "f16"),    # stride 2, Wo 7
    (2, 24, 13, 15, 1, "bf16"),    # odd Wo, 3 channel vectors per pixel
    (2, 960, 7, 7, 1, "bf16"),     # 120 vectors per pixel
    (1, 8, 5, 3, 1, "f16"),        # fewer items than one wave
    (2, 32, 9, 9, 1, "f32"),       # fp32: standalone pass
]


@pytest.mark.parametrize("case", DW_CASES)
def test_depthwise_routed_measured(case):
    """The depthwise kernel measuring its own output: counts and bitmap equal
    the oracle's measurement, y equals the unmeasured call's bit for bit and
    the oracle's conv within tolerance; with and without commit words.  The
    bias drives whole 8-channel groups below zero so zero blocks occur."""
    from tests._util import RTOL, assert_close
    abi = _abi()
    dev = torch.device("cuda")
    n, c, h, w, s, dt = case
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dt]
    d = abi.conv_desc(n, c, h, w, c, 3, 3, s, s, 1, 1, 1, 1, c, tdt, has_bias=True)
    ho, wo = (h + 2 - 3) // s + 1, (w + 2 - 3) // s + 1
    seed = 1500 + DW_CASES.index(case) * 5
    x = synth.relu_normal((n, h, w, c), dt, seed)
    wt = synth.he_normal((c, 3, 3, 1), 9, dt, seed + 1)
    b = synth.normal((c,), dt, seed + 2).float()
    b[(torch.arange(c) // 8) % 3 == 0] = -20.0
    b = b.to(tdt)
    r = synth.normal((n, ho, wo, c), dt, seed + 3)
    xd, wd, bd, rd = x.to(dev), wt.to(dev), b.to(dev), r.to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * w, c, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(xd, n * h * w, c, 1, 8, 0, counts, mask)
    ws = torch.zeros(16, dtype=torch.uint8, device=dev)
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    rows = n * ho * wo
    y2 = torch.full((n, ho, wo, c), float("nan"), dtype=tdt, device=dev)
    abi.sparoa_conv2d_routed(d, 0.5, 0.0, abi.ROUTE_BLOCK, counts, xd, wd, bd, rd,
                             abi.ACT_RELU, mask, y2, ws)
    torch.cuda.synchronize()
    yr, ar, _ = oracle.conv2d(x, wt, n, c, h, w, c, 3, 3, s, s, 1, 1, 1, 1, c, bias=b,
                              residual=r, act=abi.ACT_RELU)
    assert_close(y2.cpu(), yr, ar, RTOL[tdt], f"depthwise {case}")
    for words in (commit, None):
        for rep in range(2):
            y = torch.full_like(y2, float("nan"))
            y_counts = _fresh_counts(rows, c, dev)
            y_mask = torch.full((abi.sparoa_mask_words(rows, c, 1, 8),), -1, dtype=torch.int32,
                                device=dev)
            abi.sparoa_conv2d_routed_measured(d, 0.5, 0.0, abi.ROUTE_BLOCK, counts, xd, wd, bd, rd,
                                              abi.ACT_RELU, mask, y, y_counts, y_mask, ws, None,
                                              words)
            torch.cuda.synchronize()
            what = f"{case} commit words {words is not None} rep {rep}"
            assert torch.equal(y, y2), what
            _check_y_measurement(abi, y, rows, c, y_counts, y_mask, what)
            assert int(commit.count_nonzero().item()) == 0
    if c % 8 == 0:   # counts only: the plain kernel counting per lane (fp32: standalone)
        for words in (commit, None):
            y = torch.full_like(y2, float("nan"))
            y_counts = _fresh_counts(rows, c, dev)
            abi.sparoa_conv2d_routed_measured(d, 0.5, 0.0, abi.ROUTE_BLOCK, counts, xd, wd, bd, rd,
                                              abi.ACT_RELU, mask, y, y_counts, None, ws, None,
                                              words)
            torch.cuda.synchronize()
            what = f"{case} counts only, commit words {words is not None}"
            assert torch.equal(y, y2), what
            _check_y_measurement(abi, y, rows, c, y_counts, None, what)
            assert int(commit.count_nonzero().item()) == 0


FC_CASES = [
    # m, k, n, dtype, intensity threshold (0: MFMA family)
    (256, 768, 3072, "f16", 0.0),     # fused epilogue
    (2048, 768, 3072, "f16", 0.0),    # fused epilogue, 128 x 128 tiles
    (64, 4096, 4096, "bf16", 0.0),    # split-K: fused reduction
    (100, 512, 256, "bf16", 0.0),     # ragged rows, split-K
    (8, 1024, 512, "bf16", 315.0),    # weight-streaming FC: standalone pass
]


@pytest.mark.parametrize("case", FC_CASES)
def test_fc_routed_measured(case):
    abi = _abi()
    dev = torch.device("cuda")
    m, k, n, dt, c_thr = case
    tdt = torch.float16 if dt == "f16" else torch.bfloat16
    d = abi.fc_desc(m, k, n, abi.F16 if dt == "f16" else abi.BF16)
    seed = 1200 + FC_CASES.index(case) * 5
    x = synth.sparse_matrix(m, k, 0.5, "block", dt, seed).to(dev)
    w = synth.normal((n, k), dt, seed + 1, std=k ** -0.5).to(dev)
    wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=tdt, device=dev)
    abi.sparoa_fc_pack_weights(d, w, wp)
    fam = abi.PATH_SKIP_BW if abi.sparoa_op_intensity_fc(d)["intensity"] < c_thr \
        else abi.PATH_SKIP_MFMA
    br, bc = abi.sparoa_fc_skip_block(d, fam)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x, m, k, br, bc, 0, counts, mask)
    ws = torch.full((max(16, max(abi.sparoa_fc_workspace_size(d, q) for q in range(4))),),
                    0x5A, dtype=torch.uint8, device=dev)
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    y = torch.full((m, n), float("nan"), dtype=tdt, device=dev)
    y_counts = _fresh_counts(m, n, dev)
    y_mask = torch.full((abi.sparoa_mask_words(m, n, 1, 8),), -1, dtype=torch.int32, device=dev)
    abi.sparoa_fc_routed_measured(d, 0.5, c_thr, abi.ROUTE_BLOCK, counts, x, w, wp, None, None,
                                  abi.ACT_RELU, mask, y, y_counts, y_mask, ws, None, commit)
    y2 = torch.full_like(y, float("nan"))
    abi.sparoa_fc_routed(d, 0.5, c_thr, abi.ROUTE_BLOCK, counts, x, w, wp, None, None,
                         abi.ACT_RELU, mask, y2, ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    _check_y_measurement(abi, y, m, n, y_counts, y_mask, str(case))
    assert int(commit.count_nonzero().item()) == 0     # commit words left zero
    if c_thr == 0.0 and n % 64 == 0:   # fused, no commit words: direct commits
        y_counts = _fresh_counts(m, n, dev)
        abi.sparoa_fc_routed_measured(d, 0.5, c_thr, abi.ROUTE_BLOCK, counts, x, w, wp, None,
                                      None, abi.ACT_RELU, mask, y, y_counts, y_mask, ws)
        torch.cuda.synchronize()
        _check_y_measurement(abi, y, m, n, y_counts, y_mask, f"{case} direct commits")
    if n % 8 == 0:   # counts only (no bitmap)
        y_counts = _fresh_counts(m, n, dev)
        y = torch.full_like(y2, float("nan"))
        abi.sparoa_fc_routed_measured(d, 0.5, c_thr, abi.ROUTE_BLOCK, counts, x, w, wp, None,
                                      None, abi.ACT_RELU, mask, y, y_counts, None, ws, None,
                                      commit)
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
        _check_y_measurement(abi, y, m, n, y_counts, None, f"{case} counts only")
        assert int(commit.count_nonzero().item()) == 0


POINTWISE_NO_MASK = [
    # n, cin, h, w, cout, dtype: 1x1 convs the pointwise kernel serves on the BW path
    # (with 64 output channels or more: from 32768 pixels)
    (42, 64, 28, 28, 96, "f16"),
    (2, 32, 56, 56, 144, "bf16"),
]


@pytest.mark.parametrize("case", POINTWISE_NO_MASK)
def test_pointwise_consumer_without_bitmap(case):
    """A routed 1x1 conv on the pointwise kernel routes on x's counts and
    tests x itself: it takes no bitmap, and its output equals the call's
    with one, on the skip and the dense route."""
    abi = _abi()
    dev = torch.device("cuda")
    n, cin, h, w, cout, dt = case
    tdt = torch.float16 if dt == "f16" else torch.bfloat16
    d = abi.conv_desc(n, cin, h, w, cout, 1, 1, 1, 1, 0, 0, 1, 1, 1, tdt)
    c_thr = abi.sparoa_op_intensity_conv(d)["intensity"] * 2   # the BW family
    assert not abi.sparoa_conv2d_routed_reads_mask(d, 0.5, c_thr, abi.ROUTE_BLOCK)
    seed = 1600 + POINTWISE_NO_MASK.index(case) * 3
    x = synth.sparse_matrix(n * h * w, cin, 0.6, "block", dt, seed).reshape(n, h, w, cin).to(dev)
    wt = synth.he_normal((cout, 1, 1, cin), cin, dt, seed + 1).to(dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(n * h * w, cin, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x, n * h * w, cin, 1, 8, 0, counts, mask)
    ws = torch.zeros(16, dtype=torch.uint8, device=dev)
    for s_thr in (0.0, 2.0):
        y = torch.full((n, h, w, cout), float("nan"), dtype=tdt, device=dev)
        y2 = torch.full_like(y, float("nan"))
        p1 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_conv2d_routed(d, s_thr, c_thr, abi.ROUTE_BLOCK, counts, x, wt, None, None,
                                 abi.ACT_RELU, None, y, ws, p1)
        abi.sparoa_conv2d_routed(d, s_thr, c_thr, abi.ROUTE_BLOCK, counts, x, wt, None, None,
                                 abi.ACT_RELU, mask, y2, ws, p2)
        torch.cuda.synchronize()
        assert int(p1.item()) == int(p2.item()) == (abi.PATH_SKIP_BW if s_thr == 0.0
                                                    else abi.PATH_DENSE_BW)
        assert torch.equal(y, y2), f"{case} s_thr {s_thr}"
        yr, ar, _ = oracle.conv2d(x.cpu(), wt.cpu(), n, cin, h, w, cout, 1, 1, act=abi.ACT_RELU)
        from tests._util import RTOL, assert_close
        assert_close(y.cpu(), yr, ar, RTOL[tdt], f"{case} s_thr {s_thr}")


def test_shared_workspace_split_k_then_fused():
    """One workspace serves a split-K layer (its partial sums fill the
    workspace) and then a layer whose epilogue measures its output with
    ticketed commits: the second layer's counts and bitmap still equal the
    oracle's measurement of its output (the commit words are an argument of
    their own, never workspace bytes)."""
    abi = _abi()
    dev = torch.device("cuda")
    d1 = abi.fc_desc(64, 4096, 4096, abi.BF16)        # split-K
    d2 = abi.conv_desc(8, 64, 32, 32, 128, 3, 3, 1, 1, 1, 1, 1, 1, 1, torch.bfloat16)
    assert abi.sparoa_fc_workspace_size(d1, abi.PATH_SKIP_MFMA) > 0
    ws = torch.full((max(abi.sparoa_fc_workspace_size(d1, abi.PATH_SKIP_MFMA),
                         abi.sparoa_conv2d_workspace_size(d2, abi.PATH_SKIP_MFMA), 16),),
                    0xFF, dtype=torch.uint8, device=dev)
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    x1 = synth.sparse_matrix(64, 4096, 0.5, "block", "bf16", 1290).to(dev)
    w1 = synth.normal((4096, 4096), "bf16", 1291, std=1 / 64).to(dev)
    c1 = torch.zeros(4, dtype=torch.int64, device=dev)
    m1 = torch.zeros(abi.sparoa_mask_words(64, 4096, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x1, 64, 4096, 1, 8, 0, c1, m1)
    y1 = torch.empty(64, 4096, dtype=torch.bfloat16, device=dev)
    y1_counts = _fresh_counts(64, 4096, dev)
    y1_mask = torch.zeros(abi.sparoa_mask_words(64, 4096, 1, 8), dtype=torch.int32, device=dev)
    x2 = synth.relu_normal((8, 32, 32, 64), "bf16", 1292).to(dev)
    w2 = synth.he_normal((128, 3, 3, 64), 576, "bf16", 1293).to(dev)
    c2 = torch.zeros(4, dtype=torch.int64, device=dev)
    m2 = torch.zeros(abi.sparoa_mask_words(8 * 32 * 32, 64, 1, 8), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x2, 8 * 32 * 32, 64, 1, 8, 0, c2, m2)
    y2 = torch.empty(8, 32, 32, 128, dtype=torch.bfloat16, device=dev)
    for rep in range(2):
        y1_counts.copy_(_fresh_counts(64, 4096, dev))
        y2_counts = _fresh_counts(8 * 32 * 32, 128, dev)
        y2_mask = torch.full((abi.sparoa_mask_words(8 * 32 * 32, 128, 1, 8),), -1,
                             dtype=torch.int32, device=dev)
        abi.sparoa_fc_routed_measured(d1, 0.5, 0.0, abi.ROUTE_BLOCK, c1, x1, w1, None, None, None,
                                      abi.ACT_RELU, m1, y1, y1_counts, y1_mask, ws, None, commit)
        abi.sparoa_conv2d_routed_measured(d2, 0.5, 0.0, abi.ROUTE_BLOCK, c2, x2, w2, None, None,
                                          abi.ACT_RELU, m2, y2, y2_counts, y2_mask, ws, None,
                                          commit)
        torch.cuda.synchronize()
        _check_y_measurement(abi, y1, 64, 4096, y1_counts, y1_mask, f"split-K layer, rep {rep}")
        _check_y_measurement(abi, y2, 8 * 32 * 32, 128, y2_counts, y2_mask,
                             f"fused layer after it, rep {rep}")
        assert int(commit.count_nonzero().item()) == 0


def test_measured_calls_reject_missing_outputs():
    abi = _abi()
    dev = torch.device("cuda")
    d = abi.fc_desc(64, 256, 128, abi.BF16)
    t = torch.zeros(64, 256, dtype=torch.bfloat16, device=dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(64, dtype=torch.int32, device=dev)
    y = torch.empty(64, 128, dtype=torch.bfloat16, device=dev)
    with pytest.raises(abi.SparoaError):
        abi.sparoa_fc_routed_measured(d, 0.5, 0.0, abi.ROUTE_BLOCK, counts, t, t, None, None, None,
                                      abi.ACT_NONE, mask, y, None, mask)
