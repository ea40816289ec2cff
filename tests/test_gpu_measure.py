"""GPU parity of the sparsity measurement kernel (Eq. 1) against the oracle:
zero counts, block bitmaps, zero-block counts and per-sample counts must be
bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests._util import mask_np

pytestmark = pytest.mark.gpu

DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _abi():
    from paper_2511_19457_amd import abi
    return abi


def _measure(x_cpu, rows, cols, br, bc, samples):
    abi = _abi()
    dev = torch.device("cuda")
    x = x_cpu.to(dev)
    counts = torch.full((4,), -1, dtype=torch.int64, device=dev)
    mask = None
    if br > 0:
        mask = torch.full((abi.sparoa_mask_words(rows, cols, br, bc),), -1, dtype=torch.int32,
                          device=dev)
    ps = torch.full((samples,), -1, dtype=torch.int64, device=dev) if samples > 0 else None
    c = abi.sparoa_measure_sparsity_sync(x, rows, cols, br, bc, samples, counts, mask, ps)
    return c, mask, ps


def _check(x_cpu, rows, cols, br, bc, samples):
    c, mask, ps = _measure(x_cpu, rows, cols, br, bc, samples)
    ref = oracle.measure(x_cpu, rows, cols, br, bc, samples)
    assert c["zeros"] == ref["zeros"] and c["numel"] == ref["numel"]
    assert c["zero_blocks"] == ref["zero_blocks"] and c["num_blocks"] == ref["num_blocks"]
    if br > 0:
        assert np.array_equal(mask_np(mask), ref["mask"])
    if samples > 0:
        assert np.array_equal(ps.cpu().numpy().view(np.uint64), ref["per_sample"])
    return c


CASES = [
    # rows, cols, block_rows, block_cols, samples
    (1, 4096, 1, 1, 0), (8, 4096, 8, 1, 0), (64, 4096, 64, 1, 0), (64, 4096, 16, 16, 0),
    (37, 1000, 16, 16, 0), (3136, 64, 1, 8, 0), (4 * 49, 256, 1, 8, 4), (100, 24, 1, 8, 4),
    (50, 3, 1, 8, 5), (7, 13, 2, 3, 0), (33, 96, 3, 2, 0), (1000, 40, 7, 4, 0),
    (256, 512, 16, 32, 2), (5, 8, 100, 100, 0), (300, 128, 0, 0, 3),
    # rows narrower than 16 bytes, one block per row (one bit per row)
    (1001, 3, 1, 8, 0), (777, 1, 1, 4, 0), (3000, 7, 1, 8, 0), (4099, 3, 1, 3, 0),
    (2100001, 3, 1, 8, 0),
    # 1 x 8 blocks of fewer than 4096 vectors (one work-group; fp32: two vectors per block)
    (37, 64, 1, 8, 0),
]


@pytest.mark.parametrize("dt", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("rho", [0.0, 0.6, 0.99])
def test_measure_parity(dt, case, rho):
    rows, cols, br, bc, samples = case
    seed = CASES.index(case) * 10 + int(rho * 3)
    x = synth.sparse_matrix(rows, cols, rho, "iid", dt, seed)
    _check(x, rows, cols, br, bc, samples)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_measure_block_pattern_and_all_zero(dt):
    x = synth.sparse_matrix(64, 4096, 0.8, "block", dt, 77)
    _check(x, 64, 4096, 16, 16, 0)
    z = torch.zeros(64, 4096, dtype=DT[dt])
    c = _check(z, 64, 4096, 16, 16, 0)
    assert c["zeros"] == c["numel"] and c["zero_blocks"] == c["num_blocks"]


def test_measure_special_values():
    for dt, bits in ((torch.float16, [0x0000, 0x8000, 0x0001, 0x8001, 0x7E00, 0x7C00, 0x3C00, 0]),
                     (torch.bfloat16, [0x0000, 0x8000, 0x0001, 0x8001, 0x7FC0, 0x7F80, 0x3F80, 0])):
        x = torch.tensor(bits * 4, dtype=torch.int32).to(torch.int16).view(dt).reshape(4, 8)
        c = _check(x, 4, 8, 1, 1, 0)
        assert c["zeros"] == 12
    xf = torch.tensor([0.0, -0.0, 1e-45, -1e-45, float("nan"), float("inf"), 1.0, 0.0] * 2)
    c = _check(xf.reshape(2, 8), 2, 8, 1, 4, 2)
    assert c["zeros"] == 6


def test_measure_reuses_buffers_and_reinitialises():
    x1 = synth.sparse_matrix(64, 4096, 0.9, "iid", "bf16", 5)
    x2 = synth.sparse_matrix(64, 4096, 0.1, "iid", "bf16", 6)
    abi = _abi()
    dev = torch.device("cuda")
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(64, 4096, 64, 1), dtype=torch.int32, device=dev)
    for x in (x1, x2, x1):
        c = abi.sparoa_measure_sparsity_sync(x.to(dev), 64, 4096, 64, 1, 0, counts, mask)
        ref = oracle.measure(x, 64, 4096, 64, 1)
        assert c["zeros"] == ref["zeros"] and c["zero_blocks"] == ref["zero_blocks"]
        assert np.array_equal(mask_np(mask), ref["mask"])


@pytest.mark.parametrize("shape,dt,blk", [
    ((32, 56, 56, 256), "bf16", (1, 8)),       # ResNet-50 stage-2 activation, batch 32
    ((32, 112, 112, 96), "f16", (1, 8)),       # MobileNetV2 largest depthwise input
    ((2048, 3072), "f16", (1, 8)),             # FFN second-FC input
    ((32, 224, 224, 3), "bf16", (1, 8)),       # ResNet-50 stem input (3 channels)
])
def test_measure_full_size(shape, dt, blk):
    x = synth.relu_normal(shape, dt, seed=synth.seed_for(3, 90))
    rows = int(np.prod(shape[:-1]))
    cols = shape[-1]
    samples = shape[0] if len(shape) == 4 else 0
    _check(x, rows, cols, blk[0], blk[1], samples)


@pytest.mark.parametrize("rows,cols,br,bc,dt", [
    (3136, 64, 1, 8, "bf16"),         # 1 x one 16-byte vector: one launch
    (100352, 96, 1, 8, "f16"),        # same, grid-stride over many work-groups
    (262144, 64, 1, 8, "bf16"),       # 33.5 MB: 256 work-groups, two passes each
    (40, 2048, 1, 4, "f32"),          # fp32 vector
    (40, 2048, 1, 8, "f32"),          # fp32 blocks of 8: two vectors per lane
    (3136, 64, 1, 8, "f32"),
    (8, 4096, 8, 1, "bf16"),          # whole-column strips
    (37, 100, 2, 4, "bf16"),          # other blocks: initialises everything itself
    (1001, 3, 1, 8, "bf16"),          # rows narrower than 16 bytes, one bit per row
    (1001, 3, 1, 8, "f32"),
])
def test_measure_preset_counters(rows, cols, br, bc, dt):
    """sparoa_measure_sparsity_preset: with counters preset to
    {0, numel, nb, nb} it gives the oracle's counts and bitmap; block shapes
    that need their bitmap cleared ignore the preset (garbage in, exact out)."""
    abi = _abi()
    dev = torch.device("cuda")
    x = synth.sparse_matrix(rows, cols, 0.7, "block", dt, rows + cols)
    ref = oracle.measure(x, rows, cols, br, bc)
    nb = -(-rows // br) * -(-cols // bc)
    esz = torch.tensor([], dtype=DT[dt]).element_size()
    owns_words = (br == 1 and bc * esz == 16) or (bc == 1 and br >= rows) or \
        (br == 1 and bc >= cols and cols * esz < 16) or \
        (br == 1 and bc == 8 and esz == 4 and cols % 8 == 0)
    preset = [0, rows * cols, nb, nb] if owns_words else [7, 7, 7, 7]
    commit = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
    # twice without and twice with commit words: each call starts from the
    # preset again, and the commit words are left zero for the next call
    for use_commit in (False, False, True, True):
        counts = torch.tensor(preset, dtype=torch.int64, device=dev)
        mask = torch.full((abi.sparoa_mask_words(rows, cols, br, bc),), -1, dtype=torch.int32,
                          device=dev)
        abi.sparoa_measure_sparsity_preset(x.to(dev), rows, cols, br, bc, counts, mask,
                                           commit=commit if use_commit else None)
        torch.cuda.synchronize()
        assert counts.cpu().tolist() == [ref["zeros"], ref["numel"], ref["zero_blocks"],
                                         ref["num_blocks"]], use_commit
        assert np.array_equal(mask_np(mask), ref["mask"])
        assert int(commit.count_nonzero().item()) == 0
