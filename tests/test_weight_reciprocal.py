"""The I420 row kernel forms each output row's luma weight rem / den (the
fractional part of the half-pixel source coordinate, 0 < rem < den <= 2^24)
as the fp32 rounding of the fp64 product rem * RN64(1 / den) instead of an
fp32 division. The argument (kernel comment): the product is within 2^-52
of the quotient, and no such quotient comes within 2^-49 of a midpoint
between fp32 values. Checked here against IEEE fp32 division: exhaustively
for every denominator up to 2^13, and on seeded samples up to 2^24."""
import numpy as np


def _same(den: np.ndarray, rem: np.ndarray) -> bool:
    div = rem.astype(np.float32) / den.astype(np.float32)
    prod = (rem.astype(np.float64) * (1.0 / den.astype(np.float64))).astype(np.float32)
    return bool(np.array_equal(div.view(np.uint32), prod.view(np.uint32)))


def test_every_weight_up_to_8192():
    for lo in range(2, 8193, 256):
        dens = np.arange(lo, min(lo + 256, 8193), dtype=np.int64)
        den = np.repeat(dens, dens - 1)
        start = np.cumsum(dens - 1) - (dens - 1)
        rem = np.arange(den.size, dtype=np.int64) - np.repeat(start, dens - 1) + 1
        assert _same(den, rem), (lo, lo + 256)


def test_sampled_weights_up_to_2_pow_24():
    rng = np.random.default_rng(24)
    den = rng.integers(8193, 2**24 + 1, size=2_000_000, dtype=np.int64)
    rem = 1 + (rng.integers(0, 2**62, size=den.size, dtype=np.int64) % (den - 1))
    assert _same(den, rem)
    # quotients next to powers of two and halves, where fp32 spacing changes
    den = rng.integers(2**20, 2**24 + 1, size=200_000, dtype=np.int64)
    for frac in (0.5, 0.25, 0.75, 2.0**-10):
        for d in (-1, 0, 1):
            rem = np.clip(np.floor(den * frac).astype(np.int64) + d, 1, den - 1)
            assert _same(den, rem), frac
