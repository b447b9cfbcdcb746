"""The fp8 QK path's reading of a bf16 query (CPU, no GPU needed).

The attend kernel runs QK^T of the fp8 caches on the fp8 matrix pipe: each
head's query row is scaled by a power of two that puts its largest |q| in
[128, 256), and every scaled value x becomes two E4M3 codes, hi = rne(x) and
lo = rne(16 (x - hi)), applied as hi + lo / 16 (the lo MFMA carries block
scale 2^-4).  These tests pin that arithmetic against a plain E4M3 table
(OCP E4M3: bias 7, 3 mantissa bits, largest finite 448, no infinities), over
every bf16 value of the range: the split is exact for |x| >= 2^-6 and off by
at most 2^-14 below, and neither code overflows.  The kernel's use of it is
checked end to end by the fp8 parity tests on the GPU.
"""
import numpy as np


def e4m3_table():
    """All finite non-negative E4M3 values with their codes, ascending."""
    vals, codes = [], []
    for c in range(0x7F):  # 0x7F is NaN
        e, m = (c >> 3) & 15, c & 7
        v = m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
        vals.append(v)
        codes.append(c)
    return np.array(vals), np.array(codes)


def rne_e4m3(x):
    """Round to the nearest E4M3 value, ties to the even code (|x| <= 448)."""
    vals, codes = e4m3_table()
    a = np.abs(x)
    assert np.all(a <= 448.0)
    hi = np.clip(np.searchsorted(vals, a), 1, len(vals) - 1)
    lo = hi - 1
    dl, dh = a - vals[lo], vals[hi] - a
    pick = np.where(dl < dh, lo, np.where(dh < dl, hi, np.where(codes[lo] % 2 == 0, lo, hi)))
    return np.sign(x) * vals[pick]


def all_bf16_below(limit):
    """Every finite bf16 value with |x| < limit."""
    bits = np.arange(0, 0x7F80, dtype=np.uint32)  # below the exponent field of infinity
    pos = (bits << 16).view(np.float32).astype(np.float64)
    pos = pos[pos < limit]
    return np.concatenate([pos, -pos])


def split(x):
    hi = rne_e4m3(x)
    lo = rne_e4m3(16.0 * (x - hi))
    return hi, lo


def test_rne_table_matches_known_codes():
    assert rne_e4m3(np.array([1.0625, 1.1875, 448.0, 2.0 ** -9, 2.0 ** -10, 3 * 2.0 ** -10])).tolist() == \
        [1.0, 1.25, 448.0, 2.0 ** -9, 0.0, 2.0 ** -8]


def test_split_is_exact_above_2_to_minus_6_and_bounded_below():
    x = all_bf16_below(256.0)
    hi, lo = split(x)
    assert np.all(np.abs(hi) <= 448) and np.all(np.abs(lo) <= 448)
    err = np.abs(hi + lo / 16.0 - x)
    big = np.abs(x) >= 2.0 ** -6
    assert big.sum() == 2 * 14 * 128  # every bf16 value with 2^-6 <= |x| < 2^8
    assert np.all(err[big] == 0.0)
    assert np.max(err[~big]) <= 2.0 ** -14


def test_row_scale_puts_the_largest_value_in_128_256():
    rng = np.random.Generator(np.random.PCG64(5))
    for mag in (1e-30, 1e-3, 1.0, 37.0, 1e20):
        q = rng.standard_normal(576) * mag
        q = (q.astype(np.float32).view(np.uint32) & 0xFFFF0000).view(np.float32).astype(np.float64)  # bf16
        e = int(np.floor(np.log2(np.abs(q).max())))
        x = q * 2.0 ** (7 - e)
        assert 128.0 <= np.abs(x).max() < 256.0
        hi, lo = split(x)
        err = np.abs((hi + lo / 16.0) * 2.0 ** (e - 7) - q)
        assert err.max() <= 2.0 ** -14 * 2.0 ** (e - 7)
