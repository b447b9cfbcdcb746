"""Decoders of the cache formats, written from their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* bf16: the upper 16 bits of an IEEE-754 binary32 -- 1 sign bit, 8 exponent
  bits (bias 127), 7 fraction bits.  The activations are BF16 (App. C,
  "B200 fixed-layout sweeps").
* OCP E4M3 ("fn" variant): 1 sign, 4 exponent bits (bias 7), 3 mantissa bits;
  exponent field 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; there are no
  infinities and the largest finite magnitude is 448.  The B200 runs keep the
  KV cache in FP8 E4M3 (App. C).

* Latent-row format (the DeepSeek-V3.2 cache row of App. B, "Theoretical
  Scenarios for DCU and H200", residency assumptions: FP8 latent with its
  scales and BF16 RoPE; the indexer state that completes the paper's 788
  bytes per token and layer is a separate pool that attention never reads).
  The paper fixes neither the split nor the scale granularity; the reading
  taken here is 656 bytes per token:
      bytes [0, 512)    E4M3 codes of the 512 latent columns
      bytes [512, 528)  four little-endian IEEE binary32 scales, scale t
                        covering latent columns [128 t, 128 t + 128)
      bytes [528, 656)  the 64 RoPE columns as little-endian bf16
  decoded as K[d] = e4m3(code[d]) * scale[d // 128] for d < 512 and
  K[512 + r] = bf16(rope[r]).  (Scales are powers of two in the workloads;
  the decoder does not depend on it.)

All decoders are exact in float64.
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


DS_ROW_BYTES = 656


def ds_rows_to_f64(rows: np.ndarray) -> np.ndarray:
    """Latent-format rows (uint8 [n, 656]) -> float64 [n, 576]."""
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.uint8).reshape(-1, DS_ROW_BYTES))
    codes = e4m3_bits_to_f64(r[:, :512])
    scales = r[:, 512:528].copy().view('<f4').astype(np.float64)          # [n, 4]
    rope_bits = r[:, 528:656].copy().view('<u2')                          # [n, 64]
    latent = codes * np.repeat(scales, 128, axis=1)
    return np.concatenate([latent, bf16_bits_to_f64(rope_bits)], axis=1)
