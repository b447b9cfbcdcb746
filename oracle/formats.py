"""Decoders of the two cache formats, written from their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* bf16: the upper 16 bits of an IEEE-754 binary32 -- 1 sign bit, 8 exponent
  bits (bias 127), 7 fraction bits.  The activations are BF16 (App. C,
  "B200 fixed-layout sweeps").
* OCP E4M3 ("fn" variant): 1 sign, 4 exponent bits (bias 7), 3 mantissa bits;
  exponent field 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; there are no
  infinities and the largest finite magnitude is 448.  The B200 runs keep the
  KV cache in FP8 E4M3 (App. C).

Both decoders are exact in float64.
"""
import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits).astype(np.int64)
    sign = np.where((b >> 15) & 1, -1.0, 1.0)
    exp = (b >> 7) & 0xFF
    frac = (b & 0x7F).astype(np.float64)
    normal = np.ldexp(1.0 + frac / 128.0, (exp - 127).astype(np.int32))
    subnormal = np.ldexp(frac / 128.0, -126)
    special = np.where(frac == 0, np.inf, np.nan)
    mag = np.where(exp == 0, subnormal, np.where(exp == 0xFF, special, normal))
    return sign * mag


def e4m3_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits).astype(np.int64)
    sign = np.where((b >> 7) & 1, -1.0, 1.0)
    exp = (b >> 3) & 0xF
    man = (b & 0x7).astype(np.float64)
    normal = np.ldexp(1.0 + man / 8.0, (exp - 7).astype(np.int32))
    subnormal = np.ldexp(man / 8.0, -6)
    mag = np.where(exp == 0, subnormal, normal)
    mag = np.where((exp == 0xF) & (man == 7), np.nan, mag)
    return sign * mag
