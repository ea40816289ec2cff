"""Device-side routing: the path a kernel takes from the counts in device
memory must equal sparoa_route's (and the oracle's) on the same counts, and
its output must equal the fixed-path output bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.gpu


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def _measure(abi, x, rows, cols, br, bc):
    dev = x.device
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(rows, cols, br, bc), dtype=torch.int32, device=dev)
    abi.sparoa_measure_sparsity(x, rows, cols, br, bc, 0, counts, mask)
    return counts, mask


FC_CASES = [(1, 4096, 1024, "iid", 0.9), (8, 2048, 512, "block", 0.8), (64, 1024, 256, "block", 0.9),
            (16, 512, 80, "iid", 0.3), (256, 768, 512, "block", 0.95), (300, 512, 200, "iid", 0.5)]


@pytest.mark.parametrize("case", FC_CASES)
@pytest.mark.parametrize("thr_kind", ["below", "tie", "above"])
def test_fc_routed_matches_host_route_and_fixed_path(case, thr_kind):
    abi = _abi()
    m, k, n, pattern, rho = case
    dev = torch.device("cuda")
    x = synth.sparse_matrix(m, k, rho, pattern, "bf16", FC_CASES.index(case))
    w = synth.normal((n, k), "bf16", 99, std=k ** -0.5)
    d = abi.fc_desc(m, k, n, abi.BF16)
    inten = abi.sparoa_op_intensity_fc(d)
    fam = abi.PATH_SKIP_BW if inten["intensity"] < 315.0 else abi.PATH_SKIP_MFMA
    br, bc = abi.sparoa_fc_skip_block(d, fam)
    ref = oracle.measure(x, m, k, br, bc)
    rho_b = ref["zero_blocks"] / ref["num_blocks"]
    s_thr = {"below": rho_b / 2, "tie": rho_b, "above": min(1.0, rho_b + 0.01)}[thr_kind]
    if thr_kind == "above" and rho_b >= 1.0:
        pytest.skip("nothing above a fully sparse input")
    want = oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"],
                        inten["intensity"], 0, s_thr, 315.0)
    xd, wd = x.to(dev), w.to(dev)
    wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=torch.bfloat16, device=dev)
    abi.sparoa_fc_pack_weights(d, wd, wp)
    ws = torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                     dtype=torch.uint8, device=dev)
    counts, mask = _measure(abi, xd, m, k, br, bc)
    y = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device=dev)
    path = torch.full((1,), -1, dtype=torch.int32, device=dev)
    abi.sparoa_fc_routed(d, s_thr, 315.0, abi.ROUTE_BLOCK, counts, xd, wd, wp, None, None,
                         abi.ACT_RELU, mask, y, ws, path)
    torch.cuda.synchronize()
    assert int(path.item()) == want
    host = abi.sparoa_route(dict(zip(("zeros", "numel", "zero_blocks", "num_blocks"),
                                     counts.cpu().tolist())), inten, 0, s_thr, 315.0)
    assert host == want
    y2 = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device=dev)
    abi.sparoa_fc(d, want, xd, wp if abi.sparoa_fc_uses_packed(d, want) else wd, None, None,
                  abi.ACT_RELU,
                  mask if want & 1 else None, y2, ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


CONV_CASES = [(2, 64, 14, 14, 64, 3, 3, 1, 1, 1, 1, 1), (1, 32, 20, 20, 192, 1, 1, 1, 1, 0, 0, 1),
              (2, 96, 12, 12, 96, 3, 3, 2, 2, 1, 1, 96),
              (2, 3, 30, 30, 64, 7, 7, 2, 2, 3, 3, 1)]    # 3-channel stem (direct kernel)


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("rho", [0.2, 0.999])
def test_conv_routed_matches_host_route_and_fixed_path(case, rho):
    abi = _abi()
    n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, g = case
    dev = torch.device("cuda")
    d = abi.conv_desc(n, cin, h, w, cout, kh, kw, sh, sw, ph, pw, 1, 1, g, abi.F16)
    x = synth.sparse_nhwc(n, h, w, cin, rho, "f16", int(rho * 100) + cin)
    wt = synth.he_normal((cout, kh, kw, cin // g), kh * kw * cin // g, "f16", 7)
    inten = abi.sparoa_op_intensity_conv(d)
    dwise = g > 1
    fam = abi.PATH_SKIP_BW if (dwise or inten["intensity"] < 315.0) else abi.PATH_SKIP_MFMA
    br, bc = abi.sparoa_conv2d_skip_block(d, fam)
    ref = oracle.measure(x, n * h * w, cin, br, bc)
    s_thr = 0.5
    want = oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"],
                        inten["intensity"], int(dwise), s_thr, 315.0)
    xd, wd = x.to(dev), wt.to(dev)
    counts, mask = _measure(abi, xd, n * h * w, cin, br, bc)
    ws = torch.zeros(max(16, max(abi.sparoa_conv2d_workspace_size(d, p) for p in range(4))),
                     dtype=torch.uint8, device=dev)
    ho = (h + 2 * ph - kh) // sh + 1
    wo = (w + 2 * pw - kw) // sw + 1
    y = torch.full((n, ho, wo, cout), float("nan"), dtype=torch.float16, device=dev)
    path = torch.full((1,), -1, dtype=torch.int32, device=dev)
    abi.sparoa_conv2d_routed(d, s_thr, 315.0, abi.ROUTE_BLOCK, counts, xd, wd, None, None,
                             abi.ACT_RELU, mask, y, ws, path)
    torch.cuda.synchronize()
    assert int(path.item()) == want
    y2 = torch.full_like(y, float("nan"))
    abi.sparoa_conv2d(d, want, xd, wd, None, None, abi.ACT_RELU, mask if want & 1 else None, y2,
                      ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


MEASURED_CASES = [(1, 4096, 512, "iid", 0.9), (8, 2048, 256, "block", 0.8),
                  (16, 1024, 100, "iid", 0.97), (33, 520, 64, "block", 0.9),
                  (64, 1024, 128, "block", 0.95), (5, 300, 48, "iid", 0.9),
                  (96, 512, 256, "block", 0.9), (4, 4096, 4096, "iid", 0.0)]


@pytest.mark.parametrize("case", MEASURED_CASES)
@pytest.mark.parametrize("mode,thr_kind", [("block", "below"), ("block", "tie"),
                                           ("block", "above"), ("element", "tie")])
def test_fc_measured_equals_measure_then_routed(case, mode, thr_kind):
    """sparoa_fc_measured (the FC kernel measuring its own input where it
    can) gives the oracle's counts, bitmap and route bit for bit, and the
    output of the fixed path it chose."""
    abi = _abi()
    m, k, n, pattern, rho = case
    dev = torch.device("cuda")
    dt = "f16" if m % 2 else "bf16"
    tdt = torch.float16 if dt == "f16" else torch.bfloat16
    x = synth.sparse_matrix(m, k, rho, pattern, dt, 700 + MEASURED_CASES.index(case))
    w = synth.normal((n, k), dt, 98, std=k ** -0.5)
    d = abi.fc_desc(m, k, n, abi.F16 if dt == "f16" else abi.BF16)
    inten = abi.sparoa_op_intensity_fc(d)
    fam = abi.PATH_SKIP_BW if inten["intensity"] < 315.0 else abi.PATH_SKIP_MFMA
    br, bc = abi.sparoa_fc_skip_block(d, fam)
    ref = oracle.measure(x, m, k, br, bc)
    mcode = abi.ROUTE_BLOCK if mode == "block" else abi.ROUTE_ELEMENT
    r = (ref["zero_blocks"] / ref["num_blocks"]) if mode == "block" else ref["zeros"] / ref["numel"]
    s_thr = {"below": r / 2, "tie": r, "above": min(1.0, r + 0.01)}[thr_kind]
    want = oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"],
                        inten["intensity"], 0, s_thr, 315.0, mcode)
    xd, wd = x.to(dev), w.to(dev)
    wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=tdt, device=dev)
    abi.sparoa_fc_pack_weights(d, wd, wp)
    ws = torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                     dtype=torch.uint8, device=dev)
    counts = torch.full((4,), -1, dtype=torch.int64, device=dev)
    mask = torch.full((abi.sparoa_mask_words(m, k, br, bc),), -1, dtype=torch.int32, device=dev)
    y = torch.full((m, n), float("nan"), dtype=tdt, device=dev)
    path = torch.full((1,), -1, dtype=torch.int32, device=dev)
    abi.sparoa_fc_measured(d, s_thr, 315.0, mcode, xd, wd, wp, None, None, abi.ACT_RELU, counts,
                           mask, y, ws, path)
    torch.cuda.synchronize()
    assert counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                     ref["num_blocks"]]
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), ref["mask"])
    assert int(path.item()) == want
    y2 = torch.full_like(y, float("nan"))
    wf = wp if abi.sparoa_fc_uses_packed(d, want) else wd
    abi.sparoa_fc(d, want, xd, wf, None, None, abi.ACT_RELU, mask if want & 1 else None, y2, ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


@pytest.mark.parametrize("m,k,n", [(96, 512, 256), (200, 16384, 64)])
def test_fc_measured_gemm_family_consecutive_calls(m, k, n):
    """GEMM-family FC (measurement launch, then the routed GEMM): the
    oracle's counts, bitmap and route on consecutive calls that share one
    workspace and one set of count/bitmap buffers -- over several measuring
    work-groups (m=96) and past their grid cap, with lanes looping (m=200)."""
    abi = _abi()
    dev = torch.device("cuda")
    d = abi.fc_desc(m, k, n, abi.BF16)
    br, bc = abi.sparoa_fc_skip_block(d, abi.PATH_SKIP_MFMA)
    w = synth.normal((n, k), "bf16", 5, std=k ** -0.5).to(dev)
    ws = torch.zeros(max(abi.sparoa_fc_workspace_size(d, p) for p in range(4)), dtype=torch.uint8,
                     device=dev)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32, device=dev)
    y = torch.empty(m, n, dtype=torch.bfloat16, device=dev)
    path = torch.zeros(1, dtype=torch.int32, device=dev)
    for call, (rho, pattern) in enumerate([(0.7, "block"), (0.3, "iid"), (0.95, "block")]):
        x = synth.sparse_matrix(m, k, rho, pattern, "bf16", 900 + call)
        ref = oracle.measure(x, m, k, br, bc)
        abi.sparoa_fc_measured(d, 0.5, 0.0, abi.ROUTE_BLOCK, x.to(dev), w, None, None, None,
                               abi.ACT_NONE, counts, mask, y, ws, path)
        torch.cuda.synchronize()
        assert counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                         ref["num_blocks"]], f"call {call}"
        assert np.array_equal(mask.cpu().numpy().view(np.uint32), ref["mask"]), f"call {call}"
        assert int(path.item()) == (1 if ref["zero_blocks"] / ref["num_blocks"] >= 0.5 else 0)


def test_fc_measured_without_split_k_needs_no_workspace():
    """An FC whose GEMM has no split-K runs the whole path with a token
    workspace, and measures exactly."""
    abi = _abi()
    dev = torch.device("cuda")
    m, k, n = 4096, 256, 512
    d = abi.fc_desc(m, k, n, abi.BF16)
    br, bc = abi.sparoa_fc_skip_block(d, abi.PATH_SKIP_MFMA)
    x = synth.sparse_matrix(m, k, 0.6, "block", "bf16", 950)
    w = synth.normal((n, k), "bf16", 951, std=k ** -0.5)
    ref = oracle.measure(x, m, k, br, bc)
    ws = torch.zeros(64, dtype=torch.uint8, device=dev)
    counts = torch.full((4,), -1, dtype=torch.int64, device=dev)
    mask = torch.full((abi.sparoa_mask_words(m, k, br, bc),), -1, dtype=torch.int32, device=dev)
    y = torch.empty(m, n, dtype=torch.bfloat16, device=dev)
    abi.sparoa_fc_measured(d, 0.5, 0.0, abi.ROUTE_BLOCK, x.to(dev), w.to(dev), None, None, None,
                           abi.ACT_NONE, counts, mask, y, ws, None)
    torch.cuda.synchronize()
    assert counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                     ref["num_blocks"]]
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), ref["mask"])


def test_fc_ops_run_equals_per_op_routed_calls():
    """The native batch executor runs measure + routed FC per op: paths and
    outputs equal the per-op calls, counts equal the oracle's."""
    abi = _abi()
    dev = torch.device("cuda")
    specs = [(1, 2048, 512, "iid", 0.95), (8, 1024, 256, "block", 0.9), (64, 512, 128, "iid", 0.5),
             (200, 512, 256, "block", 0.9), (16, 300, 70, "iid", 0.0)]
    ops, bufs = [], []
    for i, (m, k, n, pat, rho) in enumerate(specs):
        d = abi.fc_desc(m, k, n, abi.F16)
        x = synth.sparse_matrix(m, k, rho, pat, "f16", 300 + i).to(dev)
        w = synth.normal((n, k), "f16", 400 + i, std=k ** -0.5).to(dev)
        wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=torch.float16, device=dev)
        abi.sparoa_fc_pack_weights(d, w, wp)
        inten = abi.sparoa_op_intensity_fc(d)
        fam = abi.PATH_SKIP_BW if inten["intensity"] < 315.0 else abi.PATH_SKIP_MFMA
        br, bc = abi.sparoa_fc_skip_block(d, fam)
        b = dict(d=d, x=x, w=w, wp=wp, br=br, bc=bc,
                 counts=torch.zeros(4, dtype=torch.int64, device=dev),
                 mask=torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32,
                                  device=dev),
                 y=torch.full((m, n), float("nan"), dtype=torch.float16, device=dev),
                 ws=torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                                dtype=torch.uint8, device=dev),
                 path=torch.full((1,), -1, dtype=torch.int32, device=dev))
        bufs.append(b)
        ops.append(abi.fc_op(d, x, w, wp, None, None, abi.ACT_RELU, b["counts"], b["mask"], b["y"],
                             b["ws"], b["path"]))
    arr = abi.fc_op_array(ops)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * len(ops))]
    for e in evs:
        e.record()
    abi.sparoa_fc_ops_run(arr, 0.5, 315.0, abi.ROUTE_BLOCK, events=evs)
    torch.cuda.synchronize()
    for i, b in enumerate(bufs):
        m, k = b["x"].shape
        ref = oracle.measure(b["x"].cpu(), m, k, b["br"], b["bc"])
        c = b["counts"].cpu().tolist()
        assert c == [ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"]]
        assert np.array_equal(b["mask"].cpu().numpy().view(np.uint32), ref["mask"])
        y2 = torch.full_like(b["y"], float("nan"))
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_fc_routed(b["d"], 0.5, 315.0, abi.ROUTE_BLOCK, b["counts"], b["x"], b["w"],
                             b["wp"], None, None, abi.ACT_RELU, b["mask"], y2, b["ws"], p2)
        torch.cuda.synchronize()
        assert int(p2.item()) == int(b["path"].item())
        assert torch.equal(y2, b["y"])
        assert evs[2 * i].elapsed_time(evs[2 * i + 1]) > 0


def _batch_op(abi, dev, d, x, seed, thr=None, residual=None):
    m, k, n = d.m, d.k, d.n
    tdt = torch.float16 if d.dtype == abi.F16 else torch.bfloat16
    w = synth.normal((n, k), "f16" if d.dtype == abi.F16 else "bf16", seed, std=k ** -0.5).to(dev)
    wp = torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=tdt, device=dev)
    abi.sparoa_fc_pack_weights(d, w, wp)
    fam = abi.PATH_SKIP_BW if abi.sparoa_op_intensity_fc(d)["intensity"] < (thr or (0.5, 315.0))[1] \
        else abi.PATH_SKIP_MFMA
    br, bc = abi.sparoa_fc_skip_block(d, fam)
    return dict(d=d, x=x, w=w, wp=wp, br=br, bc=bc, res=residual,
                thr=thr or (0.5, 315.0),
                counts=torch.zeros(4, dtype=torch.int64, device=dev),
                mask=torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32, device=dev),
                y=torch.full((m, n), float("nan"), dtype=tdt, device=dev),
                ws=torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                               dtype=torch.uint8, device=dev),
                path=torch.full((1,), -1, dtype=torch.int32, device=dev))


def test_fc_ops_run_batched_equals_op_by_op():
    """The batched executor (grouped measurements and split-K reductions,
    here 20 GEMM-family ops in two dtypes next to streaming ops, so groups
    fill and spill over 16) gives every op the counts, bitmap, path and
    output bits of op-by-op sparoa_fc_measured calls; a chained pair (an
    op's output is the next op's input) is detected and run in order."""
    abi = _abi()
    dev = torch.device("cuda")
    bufs = []
    for i in range(24):
        if i % 6 == 0:      # streaming, self-measuring
            m, k, n, dt = 8, 1024, 256, abi.BF16
        else:               # GEMM family (m > 64), split-K
            m, k, n, dt = 96 + 8 * (i % 3), 1024, 128, (abi.F16 if i % 2 else abi.BF16)
        d = abi.fc_desc(m, k, n, dt)
        x = synth.sparse_matrix(m, k, 0.3 + 0.02 * i, "block" if i % 4 else "iid",
                                "f16" if dt == abi.F16 else "bf16", 600 + i).to(dev)
        # intensity threshold 0 puts the m > 64 ops on the MFMA family
        bufs.append(_batch_op(abi, dev, d, x, 700 + i,
                              thr=(0.25 + 0.02 * i, 315.0 if i % 6 == 0 else 0.0)))
    ops = [abi.fc_op(b["d"], b["x"], b["w"], b["wp"], None, b["res"], abi.ACT_RELU, b["counts"],
                     b["mask"], b["y"], b["ws"], b["path"], (b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK))
           for b in bufs]
    abi.sparoa_fc_ops_run(abi.fc_op_array(ops))
    torch.cuda.synchronize()
    for i, b in enumerate(bufs):
        c2 = torch.zeros_like(b["counts"])
        k2 = torch.zeros_like(b["mask"])
        y2 = torch.full_like(b["y"], float("nan"))
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_fc_measured(b["d"], b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK, b["x"], b["w"],
                               b["wp"], None, b["res"], abi.ACT_RELU, c2, k2, y2, b["ws"], p2)
        torch.cuda.synchronize()
        assert torch.equal(c2, b["counts"]), f"op {i}"
        assert torch.equal(k2, b["mask"]), f"op {i}"
        assert int(p2.item()) == int(b["path"].item()), f"op {i}"
        assert torch.equal(y2, b["y"]), f"op {i}"
    # a chain: op 1 reads op 0's output (same shape in and out)
    d = abi.fc_desc(128, 256, 256, abi.BF16)
    x0 = synth.sparse_matrix(128, 256, 0.5, "block", "bf16", 620).to(dev)
    b0 = _batch_op(abi, dev, d, x0, 720)
    b1 = _batch_op(abi, dev, d, b0["y"], 721)
    ops = [abi.fc_op(b["d"], b["x"], b["w"], b["wp"], None, None, abi.ACT_RELU, b["counts"],
                     b["mask"], b["y"], b["ws"], b["path"]) for b in (b0, b1)]
    abi.sparoa_fc_ops_run(abi.fc_op_array(ops), 0.5, 315.0, abi.ROUTE_BLOCK)
    torch.cuda.synchronize()
    y_chain = b1["y"].clone()
    ref = oracle.measure(b0["y"].cpu(), 128, 256, b1["br"], b1["bc"])
    assert b1["counts"].cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                           ref["num_blocks"]]
    y2 = torch.full_like(y_chain, float("nan"))
    abi.sparoa_fc_measured(d, 0.5, 315.0, abi.ROUTE_BLOCK, b0["y"], b1["w"], b1["wp"], None, None,
                           abi.ACT_RELU, b1["counts"], b1["mask"], y2, b1["ws"], b1["path"])
    torch.cuda.synchronize()
    assert torch.equal(y2, y_chain)


def test_fc_ops_run_shared_scratch_runs_in_order():
    """Ops that share their counts, mask and split-K workspace (valid one op
    after another) are detected and run in order: each output equals a
    private op-by-op call's, and the shared counts hold the last op's."""
    abi = _abi()
    dev = torch.device("cuda")
    d = abi.fc_desc(64, 4096, 1024, abi.BF16)
    thr = (0.5, 0.0, abi.ROUTE_BLOCK)              # MFMA family: split-K partials
    assert abi.sparoa_fc_workspace_size(d, abi.PATH_SKIP_MFMA) > 0
    shared = _batch_op(abi, dev, d, synth.sparse_matrix(64, 4096, 0.3, "block", "bf16", 640).to(dev),
                       740, thr=thr[:2])
    bufs = []
    for i in range(3):
        x = synth.sparse_matrix(64, 4096, 0.2 + 0.3 * i, "block", "bf16", 641 + i).to(dev)
        bufs.append(_batch_op(abi, dev, d, x, 741 + i, thr=thr[:2]))
    ops = [abi.fc_op(b["d"], b["x"], b["w"], b["wp"], None, None, abi.ACT_RELU, shared["counts"],
                     shared["mask"], b["y"], shared["ws"], b["path"], thr) for b in bufs]
    abi.sparoa_fc_ops_run(abi.fc_op_array(ops))
    torch.cuda.synchronize()
    for i, b in enumerate(bufs):
        c2 = torch.zeros_like(b["counts"])
        y2 = torch.full_like(b["y"], float("nan"))
        abi.sparoa_fc_measured(b["d"], thr[0], thr[1], abi.ROUTE_BLOCK, b["x"], b["w"], b["wp"],
                               None, None, abi.ACT_RELU, c2, b["mask"], y2, b["ws"])
        torch.cuda.synchronize()
        assert torch.equal(y2, b["y"]), f"op {i}"
        if i == len(bufs) - 1:
            assert torch.equal(c2, shared["counts"])


def test_fc_ops_run_grouped_streaming_equals_op_by_op():
    """Self-measuring streaming FCs run as grouped launches (one per dtype,
    at most 16 ops each): 22 ops in 3 launches, m from 1 to 64 (ragged, up to
    four 16-row tiles), bias and residual on some, skip and dense routes --
    counts, bitmap, path and output bits equal op-by-op calls; counts equal
    the oracle's."""
    abi = _abi()
    dev = torch.device("cuda")
    specs = []
    for i in range(18):                 # one key (bf16, one row tile): groups of 16 + 2
        specs.append((1 + (i % 3) * 7, 1024 + 256 * (i % 2), 64 + 16 * (i % 5), abi.BF16))
    specs += [(20, 512, 96, abi.BF16), (33, 768, 128, abi.F16), (64, 1024, 160, abi.F16),
              (5, 2048, 48, abi.F16)]
    bufs = []
    for i, (m, k, n, dt) in enumerate(specs):
        d = abi.fc_desc(m, k, n, dt, has_bias=(i % 4 == 1))
        sd = "f16" if dt == abi.F16 else "bf16"
        x = synth.sparse_matrix(m, k, (0.0, 0.5, 0.8, 0.95)[i % 4], "block" if i % 2 else "iid",
                                sd, 800 + i).to(dev)
        res = synth.normal((m, n), sd, 850 + i).to(dev) if i % 3 == 2 else None
        b = _batch_op(abi, dev, d, x, 900 + i, thr=(0.1 + 0.05 * i, 315.0), residual=res)
        b["bias"] = synth.normal((n,), sd, 950 + i).to(dev) if d.has_bias else None
        bufs.append(b)
    ops = [abi.fc_op(b["d"], b["x"], b["w"], b["wp"], b["bias"], b["res"], abi.ACT_RELU,
                     b["counts"], b["mask"], b["y"], b["ws"], b["path"],
                     (b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK)) for b in bufs]
    abi.sparoa_fc_ops_run(abi.fc_op_array(ops))
    torch.cuda.synchronize()
    seen = set()
    for i, b in enumerate(bufs):
        m, k = b["x"].shape
        ref = oracle.measure(b["x"].cpu(), m, k, b["br"], b["bc"])
        assert b["counts"].cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                              ref["num_blocks"]], f"op {i}"
        assert np.array_equal(b["mask"].cpu().numpy().view(np.uint32), ref["mask"]), f"op {i}"
        c2 = torch.zeros_like(b["counts"])
        k2 = torch.zeros_like(b["mask"])
        y2 = torch.full_like(b["y"], float("nan"))
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_fc_measured(b["d"], b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK, b["x"], b["w"],
                               b["wp"], b["bias"], b["res"], abi.ACT_RELU, c2, k2, y2, b["ws"], p2)
        torch.cuda.synchronize()
        assert int(p2.item()) == int(b["path"].item()), f"op {i}"
        assert torch.equal(y2, b["y"]), f"op {i}"
        seen.add(int(p2.item()))
    assert seen == {abi.PATH_DENSE_BW, abi.PATH_SKIP_BW}


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_fc_ops_run_grouped_streaming_edge_cases(dt):
    """One grouped streaming launch over ten FCs with m <= 16: K up to 4096
    (full slices) and ragged (a partial last slice), N from one panel to 32
    and ragged, an all-zero input (skip route, every slice list empty), a
    dense input routed to the skip path (threshold 0: lists of every
    column), bias and residual on some -- counts, bitmap, path and output
    bits equal op-by-op calls and the oracle's measurement."""
    abi = _abi()
    dev = torch.device("cuda")
    tdt = abi.F16 if dt == "f16" else abi.BF16
    specs = [  # m, k, n, rho, pattern, sparsity threshold
        (1, 4096, 512, 0.0, "iid", 0.8), (8, 4096, 512, 0.95, "block", 0.8),
        (1, 4096, 16, 0.95, "iid", 0.8), (16, 4096, 100, 0.5, "iid", 0.8),
        (3, 2048, 256, 1.0, "iid", 0.8), (8, 4096, 64, 0.3, "iid", 0.0),
        (15, 1000, 200, 0.8, "block", 0.6), (8, 4096, 512, 0.8, "block", 0.8),
        (1, 64, 48, 0.5, "iid", 0.4), (12, 4096, 512, 0.0, "block", 0.9),
    ]
    bufs = []
    for i, (m, k, n, rho, pat, st) in enumerate(specs):
        d = abi.fc_desc(m, k, n, tdt, has_bias=(i % 3 == 1))
        x = synth.sparse_matrix(m, k, rho, pat, dt, 1200 + i).to(dev)
        res = synth.normal((m, n), dt, 1250 + i).to(dev) if i % 4 == 3 else None
        b = _batch_op(abi, dev, d, x, 1300 + i, thr=(st, 315.0), residual=res)
        b["bias"] = synth.normal((n,), dt, 1350 + i).to(dev) if d.has_bias else None
        bufs.append(b)
    ops = [abi.fc_op(b["d"], b["x"], b["w"], b["wp"], b["bias"], b["res"], abi.ACT_NONE,
                     b["counts"], b["mask"], b["y"], b["ws"], b["path"],
                     (b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK)) for b in bufs]
    abi.sparoa_fc_ops_run(abi.fc_op_array(ops))
    torch.cuda.synchronize()
    seen = set()
    for i, b in enumerate(bufs):
        m, k = b["x"].shape
        ref = oracle.measure(b["x"].cpu(), m, k, b["br"], b["bc"])
        assert b["counts"].cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                              ref["num_blocks"]], f"op {i}"
        assert np.array_equal(b["mask"].cpu().numpy().view(np.uint32), ref["mask"]), f"op {i}"
        c2 = torch.zeros_like(b["counts"])
        k2 = torch.zeros_like(b["mask"])
        y2 = torch.full_like(b["y"], float("nan"))
        p2 = torch.full((1,), -1, dtype=torch.int32, device=dev)
        abi.sparoa_fc_measured(b["d"], b["thr"][0], b["thr"][1], abi.ROUTE_BLOCK, b["x"], b["w"],
                               b["wp"], b["bias"], b["res"], abi.ACT_NONE, c2, k2, y2, b["ws"], p2)
        torch.cuda.synchronize()
        assert int(p2.item()) == int(b["path"].item()), f"op {i}"
        assert torch.equal(y2, b["y"]), f"op {i}"
        seen.add(int(p2.item()))
    assert seen == {abi.PATH_DENSE_BW, abi.PATH_SKIP_BW}


def test_fc_ops_run_in_a_hip_graph_equals_eager():
    """The executor captured in a HIP graph: every replay (with eager work and
    synchronisations in between) gives the eager run's counts, paths and
    outputs."""
    abi = _abi()
    dev = torch.device("cuda")
    ops, bufs = [], []
    for i, (m, rho, pat) in enumerate([(1, 0.95, "iid"), (8, 0.9, "block"), (64, 0.9, "block"),
                                       (8, 0.0, "iid"), (96, 0.9, "block")]):
        k, n = 2048, 512
        d = abi.fc_desc(m, k, n, abi.BF16)
        inten = abi.sparoa_op_intensity_fc(d)
        fam = abi.PATH_SKIP_BW if inten["intensity"] < 315.0 else abi.PATH_SKIP_MFMA
        br, bc = abi.sparoa_fc_skip_block(d, fam)
        b = dict(x=synth.sparse_matrix(m, k, rho, pat, "bf16", 500 + i).to(dev),
                 w=synth.normal((n, k), "bf16", 600 + i, std=k ** -0.5).to(dev),
                 wp=torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=torch.bfloat16,
                                device=dev),
                 counts=torch.zeros(4, dtype=torch.int64, device=dev),
                 mask=torch.zeros(abi.sparoa_mask_words(m, k, br, bc), dtype=torch.int32,
                                  device=dev),
                 y=torch.zeros(m, n, dtype=torch.bfloat16, device=dev),
                 ws=torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                                dtype=torch.uint8, device=dev),
                 path=torch.zeros(1, dtype=torch.int32, device=dev))
        abi.sparoa_fc_pack_weights(d, b["w"], b["wp"])
        bufs.append(b)          # keeps every buffer alive while the op structs point at it
        ops.append(abi.fc_op(d, b["x"], b["w"], b["wp"], None, None, abi.ACT_NONE, b["counts"],
                             b["mask"], b["y"], b["ws"], b["path"]))
    arr = abi.fc_op_array(ops)
    abi.sparoa_fc_ops_run(arr, 0.5, 315.0)
    torch.cuda.synchronize()
    ref = [(b["y"].clone(), int(b["path"].item()), b["counts"].clone(), b["mask"].clone())
           for b in bufs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            abi.sparoa_fc_ops_run(arr, 0.5, 315.0)
    torch.cuda.synchronize()
    scratch = torch.ones(1 << 20, device=dev)
    for rep in range(3):
        for b in bufs:                      # eager work between replays
            b["y"].zero_()
            b["path"].fill_(-1)
            b["counts"].fill_(-1)
            b["mask"].fill_(-1)
        scratch.mul_(2.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for b, (y, p, c, mk) in zip(bufs, ref):
            assert torch.equal(b["y"], y), rep
            assert int(b["path"].item()) == p, rep
            assert torch.equal(b["counts"], c) and torch.equal(b["mask"], mk), rep


def test_fc_ops_run_uses_each_ops_own_thresholds():
    """With no batch thresholds, every op routes with its own (sparsity,
    intensity) pair: the path equals the host rule on that op's counts, and
    an intensity threshold at the op's own intensity sends it to the MFMA
    family (measured at that family's granularity)."""
    abi = _abi()
    dev = torch.device("cuda")
    ops, bufs = [], []
    specs = [(8, 0.9, "block", (0.5, 315.0)), (8, 0.9, "block", (0.99, 315.0)),
             (64, 0.9, "block", (0.5, None)), (1, 0.95, "iid", (0.2, 315.0))]
    for i, (m, rho, pat, (s_thr, c_thr)) in enumerate(specs):
        k, n = 1024, 256
        d = abi.fc_desc(m, k, n, abi.BF16)
        inten = abi.sparoa_op_intensity_fc(d)
        c_thr = inten["intensity"] if c_thr is None else c_thr
        words = max(abi.sparoa_mask_words(m, k, *abi.sparoa_fc_skip_block(d, f))
                    for f in (abi.PATH_SKIP_BW, abi.PATH_SKIP_MFMA))
        b = dict(d=d, x=synth.sparse_matrix(m, k, rho, pat, "bf16", 800 + i).to(dev),
                 w=synth.normal((n, k), "bf16", 810 + i, std=k ** -0.5).to(dev),
                 wp=torch.empty(abi.sparoa_fc_packed_bytes(d) // 2, dtype=torch.bfloat16,
                                device=dev),
                 counts=torch.zeros(4, dtype=torch.int64, device=dev),
                 mask=torch.zeros(words, dtype=torch.int32, device=dev),
                 y=torch.zeros(m, n, dtype=torch.bfloat16, device=dev),
                 ws=torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                                dtype=torch.uint8, device=dev),
                 path=torch.full((1,), -1, dtype=torch.int32, device=dev), thr=(s_thr, c_thr),
                 inten=inten)
        abi.sparoa_fc_pack_weights(d, b["w"], b["wp"])
        bufs.append(b)
        ops.append(abi.fc_op(d, b["x"], b["w"], b["wp"], None, None, abi.ACT_NONE, b["counts"],
                             b["mask"], b["y"], b["ws"], b["path"],
                             (s_thr, c_thr, abi.ROUTE_BLOCK)))
    arr = abi.fc_op_array(ops)
    abi.sparoa_fc_ops_run(arr)
    torch.cuda.synchronize()
    for b in bufs:
        m, k = b["x"].shape
        fam = abi.PATH_SKIP_BW if b["inten"]["intensity"] < b["thr"][1] else abi.PATH_SKIP_MFMA
        ref = oracle.measure(b["x"].cpu(), m, k, *abi.sparoa_fc_skip_block(b["d"], fam))
        assert b["counts"].cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                              ref["num_blocks"]]
        want = oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"],
                            b["inten"]["intensity"], 0, b["thr"][0], b["thr"][1])
        assert int(b["path"].item()) == want
    assert int(bufs[2]["path"].item()) & 2 == 0          # m = 64 sent to the MFMA family
    assert int(bufs[0]["path"].item()) != int(bufs[1]["path"].item())
