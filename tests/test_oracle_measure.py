"""Pins of the oracle's decoder and sparsity statistics (Eq. 1) against
library routines, exhaustive enumeration and hand-written expected values."""
import numpy as np
import pytest
import torch

import oracle
import synth


def test_decode_f16_exhaustive_vs_numpy():
    bits = np.arange(65536, dtype=np.uint16)
    got = oracle.decode(bits, oracle.F16)
    ref = bits.view(np.float16).astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def test_decode_bf16_exhaustive_vs_torch():
    bits = np.arange(65536, dtype=np.uint16)
    got = oracle.decode(bits, oracle.BF16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def test_decode_f32_vs_numpy():
    g = np.random.default_rng(1)
    bits = g.integers(0, 2**32, size=20000, dtype=np.uint64).astype(np.uint32)
    special = np.array([0, 0x80000000, 1, 0x007FFFFF, 0x00800000, 0x7F800000, 0xFF800000,
                        0x7FC00000, 0x3F800000], dtype=np.uint32)
    bits = np.concatenate([bits, special])
    got = oracle.decode(bits, oracle.F32)
    ref = bits.view(np.float32).astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def test_hand_example_counts_and_bitmap():
    # 4 x 6 matrix, blocks 2 x 3 -> 2 x 2 blocks; indices 0..3 row-major.
    x = np.array([[0, 0, 0, 1, 0, 0],
                  [0, 0, 0, 0, 0, 0],
                  [0, 2, 0, 0, 0, 0],
                  [0, 0, 0, 0, 0, 0]], dtype=np.float32)
    r = oracle.measure(x, 4, 6, 2, 3)
    assert r["zeros"] == 22 and r["numel"] == 24
    # block 0 (rows 0-1, cols 0-2): zero; block 1 (rows 0-1, cols 3-5): 1.0;
    # block 2 (rows 2-3, cols 0-2): 2.0; block 3: zero.  Bits 1 and 2 set.
    assert r["num_blocks"] == 4 and r["zero_blocks"] == 2
    assert r["mask"].tolist() == [0b0110]


def test_hand_example_clipped_blocks():
    # 3 x 5 matrix with 2 x 2 blocks: 2 x 3 blocks, the last row and column clipped.
    x = np.zeros((3, 5), dtype=np.float32)
    x[2, 4] = -3.0          # block (1, 2) -> index 5
    x[0, 1] = 0.5           # block (0, 0) -> index 0
    r = oracle.measure(x, 3, 5, 2, 2)
    assert r["num_blocks"] == 6 and r["zero_blocks"] == 4
    assert r["mask"].tolist() == [(1 << 0) | (1 << 5)]
    assert r["zeros"] == 13


def test_signed_zero_subnormal_nan_inf_f16_bf16():
    # raw bit patterns: +0, -0, smallest subnormal, -smallest subnormal, NaN, +Inf, 1.0
    f16 = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x7E00, 0x7C00, 0x3C00], dtype=np.uint16)
    bf16 = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x7FC0, 0x7F80, 0x3F80], dtype=np.uint16)
    for bits, code in ((f16, oracle.F16), (bf16, oracle.BF16)):
        r = oracle.measure(bits, 1, 7, 1, 1, dt=code)
        assert r["zeros"] == 2
        assert r["mask"].tolist() == [0b1111100]


def test_signed_zero_subnormal_f32():
    x = np.array([0.0, -0.0, 1e-45, -1e-45, np.nan, np.inf, -np.inf, 1.0], dtype=np.float32)
    r = oracle.measure(x, 2, 4, 1, 1)
    assert r["zeros"] == 2
    assert r["mask"].tolist() == [0b11111100]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_zero_count_vs_numpy_count_nonzero(dt):
    x = synth.relu_normal((3, 17, 29), dt, seed=7)
    r = oracle.measure(x, 3 * 17, 29)
    ref = x.numel() - int(np.count_nonzero(x.to(torch.float32).numpy()))
    assert r["zeros"] == ref and r["numel"] == x.numel()


@pytest.mark.parametrize("rows,cols,br,bc", [(64, 96, 16, 16), (37, 50, 16, 16), (8, 4096, 8, 1),
                                             (100, 64, 1, 32), (5, 7, 3, 2), (64, 64, 64, 64)])
def test_bitmap_vs_numpy_block_reduction(rows, cols, br, bc):
    x = synth.sparse_matrix(rows, cols, 0.9, "iid", "bf16", seed=rows * 1000 + cols)
    r = oracle.measure(x, rows, cols, br, bc)
    nbr, nbc = -(-rows // br), -(-cols // bc)
    v = np.zeros((nbr * br, nbc * bc), dtype=bool)
    v[:rows, :cols] = x.to(torch.float32).numpy() != 0
    nz = v.reshape(nbr, br, nbc, bc).any(axis=(1, 3)).reshape(-1)
    bits = np.unpackbits(r["mask"].view(np.uint8), bitorder="little")[: nz.size].astype(bool)
    assert np.array_equal(bits, nz)
    assert r["zero_blocks"] == int((~nz).sum()) and r["num_blocks"] == nz.size
    # bits past the last block stay clear
    assert not np.unpackbits(r["mask"].view(np.uint8), bitorder="little")[nz.size:].any()


def test_all_zero_and_no_zero():
    z = torch.zeros(33, 40, dtype=torch.float16)
    r = oracle.measure(z, 33, 40, 16, 16)
    assert r["zeros"] == r["numel"] == 1320
    assert r["zero_blocks"] == r["num_blocks"] == 9
    assert oracle.sparsity(r["zeros"], r["numel"]) == 1.0
    o = torch.ones(33, 40, dtype=torch.float16)
    r = oracle.measure(o, 33, 40, 16, 16)
    assert r["zeros"] == 0 and r["zero_blocks"] == 0
    assert oracle.sparsity(0, r["numel"]) == 0.0


def test_per_sample_counts_vs_numpy():
    x = synth.relu_normal((4, 5, 6, 8), "f16", seed=3)
    r = oracle.measure(x, 4 * 5 * 6, 8, samples=4)
    ref = [(x[i] == 0).sum().item() for i in range(4)]
    assert r["per_sample"].tolist() == ref
    assert sum(ref) == r["zeros"]


def test_sparsity_is_one_division():
    # rho evaluated as z / n, correctly rounded (not 1 - c/n)
    assert oracle.sparsity(1, 3) == 1.0 / 3.0
    assert oracle.sparsity(2, 4) == 0.5


def test_relu_normal_statistics_config1():
    # ReLU(N(0,1)) at [1, 64, 56, 56]: zeros ~ Binomial(n, 1/2); 5 sigma band.
    x = synth.relu_normal((1, 56, 56, 64), "f32", seed=synth.seed_for(1, 0))
    r = oracle.measure(x, 56 * 56, 64)
    n = r["numel"]
    assert n == 200704
    assert abs(r["zeros"] - n / 2) < 5 * np.sqrt(n) / 2


def test_invalid_arguments():
    with pytest.raises(ValueError):
        oracle.measure(np.zeros(4, np.float32), 0, 4)
    with pytest.raises(ValueError):
        oracle.measure(np.zeros(6, np.float32), 3, 2, samples=2)  # 3 rows % 2 samples
