"""Pin the oracle's bf16 rounding against torch's own conversion (CPU)."""
import numpy as np
import torch

from oracle import bf16


def _torch_bits(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(x32).to(torch.bfloat16)
    return (t.view(torch.int16).numpy().astype(np.int32) & 0xFFFF).astype(np.uint16)


def test_random_values_match_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32),
        (rng.standard_normal(100000) * 1e-3).astype(np.float32),
        (rng.standard_normal(100000) * 1e30).astype(np.float32),
        rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32).view(np.float32),
    ])
    x = x[~np.isnan(x)]
    assert np.array_equal(bf16.from_f32(x), _torch_bits(x))


def test_ties_and_edges_match_torch():
    patterns = np.array([
        0x3F808000,  # exact tie, even below -> stays
        0x3F818000,  # exact tie, odd below -> rounds up
        0x3F808001, 0x3F807FFF,
        0x7F7FFFFF,  # max finite -> rounds to inf
        0x7F800000, 0xFF800000,  # infinities
        0x00000001, 0x00008000, 0x00018000, 0x807FFFFF,  # subnormals
        0x80000000, 0x00000000,  # signed zeros
    ], dtype=np.uint32)
    x = patterns.view(np.float32)
    assert np.array_equal(bf16.from_f32(x), _torch_bits(x))


def test_nan_stays_nan():
    x = np.array([0x7FC00000, 0x7F800001, 0xFFC01234], dtype=np.uint32).view(np.float32)
    back = bf16.to_f64(bf16.from_f32(x))
    assert np.isnan(back).all()


def test_widen_is_exact_against_torch():
    bits = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    t = torch.from_numpy(bits.astype(np.int32).astype(np.int16)).view(torch.bfloat16)
    want = t.to(torch.float64).numpy()
    got = bf16.to_f64(bits)
    ok = np.isnan(want)
    assert np.array_equal(np.isnan(got), ok)
    assert np.array_equal(got[~ok], want[~ok])
