"""Per-layer parity of the measure -> route -> execute driver over the
network-shaped stacks.  Each layer is checked on the GPU's own input bytes
(a value that is exactly zero after an activation depends on sub-ulp
rounding upstream, so the chain is not compared end to end): sparsity counts
and routing decisions bit-exact, outputs on sampled elements within the
dtype's tolerance element by element and normwise over the sample.  At full
size the sample is every output of sample 0 (of the first sequence for the
FFN) plus 4096 seeded elements of the rest."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import RTOL, SUBNORMAL_STEP

pytestmark = pytest.mark.gpu


def _sample_idx(L, total, n_samples, rng, whole_first):
    """Flat output offsets to check: n_samples seeded ones, the first and the
    last, and with whole_first every output of the first sample (conv: the
    first image; FC: the first sequence of 128 tokens)."""
    parts = [rng.integers(0, total, size=n_samples), [0, total - 1]]
    if whole_first:
        s = L.shape
        first = (total // s["n"]) if L.kind == "conv" else min(128, s["m"]) * s["n"]
        parts.append(np.arange(first))
    return np.unique(np.concatenate(parts))


def _check_layer(eng, i, rec, n_samples, rng, whole_first=False):
    from paper_2511_19457_amd import abi
    L, st = eng.layers[i], eng.st[i]
    x = eng.acts[L.src].cpu()
    y = eng.acts[i + 1].cpu()
    s = L.shape
    if L.kind == "maxpool":
        ref = oracle.maxpool2d(x, s["n"], s["c"], s["h"], s["w"], s["k"], s["s"], s["p"])
        assert np.array_equal(y.float().numpy().astype(np.float64), ref), L.name
        return
    ref = oracle.measure(x.reshape(st["rows"], st["cols"]), st["rows"], st["cols"], st["br"],
                         st["bc"])
    c = rec.counts
    assert (c["zeros"], c["numel"], c["zero_blocks"], c["num_blocks"]) == \
        (ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"]), L.name
    assert np.array_equal(st["mask"].cpu().numpy().view(np.uint32), ref["mask"]), L.name
    path = oracle.route(ref["zeros"], ref["numel"], ref["zero_blocks"], ref["num_blocks"],
                        rec.intensity, int(L.depthwise), eng.s_thr, eng.c_thr, eng.mode)
    assert rec.path == path, L.name
    w = st["w"].cpu()
    r = eng.acts[L.res].cpu() if L.res is not None else None
    total = y.numel()
    idx = _sample_idx(L, total, n_samples, rng, whole_first)
    if L.kind == "conv":
        yr, ar = oracle.conv2d_at(x, w, idx, s["n"], s["cin"], s["h"], s["w"], s["cout"],
                                  s["kh"], s["kw"], s["sh"], s["sw"], s["ph"], s["pw"], 1, 1,
                                  s["groups"], residual=r, act=L.act)
    else:   # an FC is the 1x1 convolution over m pixels
        yr, ar = oracle.conv2d_at(x, w.reshape(s["n"], 1, 1, s["k"]), idx, s["m"], s["k"], 1, 1,
                                  s["n"], 1, 1, residual=r, act=L.act)
    yg = y.reshape(-1)[idx].float().numpy().astype(np.float64)
    bound = RTOL[y.dtype] * ar + SUBNORMAL_STEP[y.dtype]
    err = np.abs(yg - yr)
    assert np.all(err <= bound), (L.name, float(np.max(err - bound)))
    # normwise backstop over the checked elements
    nref = float(np.linalg.norm(yr))
    assert float(np.linalg.norm(yg - yr)) <= RTOL[y.dtype] * nref + 1e-300, L.name


def _run_stack(layers, dtype, seed, n_samples, thr=0.5, whole_first=False):
    from paper_2511_19457_amd.driver import Engine
    from paper_2511_19457_amd.stacks import input_shape
    eng = Engine(layers, dtype, "cuda", seed=seed, sparsity_thr=thr)
    x = synth.normal(input_shape(layers), dtype, seed).cuda()
    _, recs, _ = eng.run(x)
    rng = np.random.default_rng(seed)
    for i, rec in enumerate(recs):
        _check_layer(eng, i, rec, n_samples, rng, whole_first)
    return eng, recs


def test_resnet50_batch1_bf16():
    from paper_2511_19457_amd.stacks import resnet50
    L = resnet50(1)
    assert sum(l.kind == "conv" for l in L) == 53
    _, recs = _run_stack(L, torch.bfloat16, synth.seed_for(3, 1), 512)
    # ReLU between layers gives natural activation sparsity
    assert np.mean([r.rho_e for r in recs if r.kind == "conv"][1:]) > 0.2


def test_mobilenet_v2_batch2_fp16():
    from paper_2511_19457_amd.stacks import mobilenet_v2
    L = mobilenet_v2(2)
    assert sum(l.kind == "conv" for l in L) == 52 and sum(l.depthwise for l in L) == 17
    _, recs = _run_stack(L, torch.float16, synth.seed_for(4, 2), 512)
    assert all(r.path & 2 for r, l in zip(recs, L) if l.depthwise)


def test_ffn_two_blocks_fp16():
    from paper_2511_19457_amd.stacks import ffn
    _, recs = _run_stack(ffn(2048, 768, 3072, 2), torch.float16, synth.seed_for(5, 1), 512)
    assert all(not (r.path & 2) for r in recs)      # I = 472.6 > 315: MFMA paths
    assert recs[1].rho_e > 0.4                      # FC2 input is ReLU-sparse


@pytest.mark.parametrize("stack,batch", [("resnet50", 8), ("resnet50", 32),
                                         ("mobilenet_v2", 32), ("ffn", 0)])
def test_stack_full_size(stack, batch):
    """The stack configurations at full size: every layer's counts and route
    bit-exact; per layer, every output of the first sample plus 4096 seeded
    outputs within tolerance."""
    from paper_2511_19457_amd import stacks
    if stack == "resnet50":
        layers, dt, seed = stacks.resnet50(batch), torch.bfloat16, synth.seed_for(3, batch)
    elif stack == "mobilenet_v2":
        layers, dt, seed = stacks.mobilenet_v2(batch), torch.float16, synth.seed_for(4, batch)
    else:
        layers, dt, seed = stacks.ffn(), torch.float16, synth.seed_for(5, 12)
    _run_stack(layers, dt, seed, 4096, whole_first=True)


@pytest.mark.parametrize("stack", ["resnet50", "mobilenet_v2", "ffn"])
def test_device_routing_equals_host_routing(stack):
    """Device-side routing takes the same path as the host route on every
    layer and produces bit-identical activations."""
    from paper_2511_19457_amd import stacks
    from paper_2511_19457_amd.driver import Engine
    from paper_2511_19457_amd.stacks import input_shape
    if stack == "resnet50":
        layers, dt = stacks.resnet50(1), torch.bfloat16
    elif stack == "mobilenet_v2":
        layers, dt = stacks.mobilenet_v2(2), torch.float16
    else:
        layers, dt = stacks.ffn(2048, 768, 3072, 2), torch.float16
    for thr in (0.05, 0.5):
        eng = Engine(layers, dt, "cuda", seed=11, sparsity_thr=thr)
        x = synth.normal(input_shape(layers), dt, 12).cuda()
        y_host, rec_host, _ = eng.run(x)
        y_host = y_host.clone()
        acts_host = [a.clone() for a in eng.acts[1:]]
        masks_host = [st["mask"].clone() if "mask" in st else None for st in eng.st]
        y_dev, rec_dev, _ = eng.run(x, routed=True)
        assert [r.path for r in rec_dev] == [r.path for r in rec_host]
        for a, b in zip(acts_host, eng.acts[1:]):
            assert torch.equal(a, b)
        assert torch.equal(y_host, y_dev)
        # the producers' fused measurements equal the consumers' own passes
        for i, (rh, rd) in enumerate(zip(rec_host, rec_dev)):
            if masks_host[i] is None:
                continue
            assert rd.counts == rh.counts, (stack, thr, i)
            used = eng.st[i]["used"][1]
            if used is None:   # counts-only measurement: this consumer reads no bitmap
                assert not eng._reads_mask(i), (stack, thr, i)
            else:
                assert torch.equal(used, masks_host[i]), (stack, thr, i)
        assert eng.tmeas, "some layer measures its output in its epilogue"
