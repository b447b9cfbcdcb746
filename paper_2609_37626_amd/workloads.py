"""Seeded synthetic inputs for owner-local paged MLA decode attention.

This module draws the batches that both the HIP path and the fp64 reference
consume.  It holds no attention arithmetic: it only draws lengths, latent rows
and queries, rounds them to the storage formats, and lays the pages out behind
a block table.

Workload shape (Sec. 3 "DOP: Computation", App. B "Per-Step Cost Model"):
an owner holds the ``N_r = B*q`` current query rows of its requests for all
``H`` heads, ``[N_r, H, d_q]`` with ``d_q = d_c + d_r = 576``, and each
request's latent history of ``s`` tokens (``s`` includes the current chunk,
``1 <= q <= s``).  The cache row of one token is ``d_c + d_r`` elements
(Sec. 2 "Footprint"), stored here as ``[latent 512 | rope 64]``.  The paper
measures only synthetic length sweeps (App. C), so every input is drawn.

Recipe, one PCG64 stream per configuration, drawn in this order:
  1. ``seq_lens``: uniform integers in ``[lo, hi]`` (both ends included), or
     ``clip(rint(lognormal(8, 1.5)), 64, 131072)`` for the ragged mix;
  2. the KV pool, ``standard_normal((num_pages, 64, 576), float32)``,
     ``num_pages = sum(ceil(s_b / 64))`` with no slack;
  3. the queries, ``standard_normal((B*q, H, 576), float32)``;
  4. ``perm = permutation(num_pages)``; request ``b``'s k-th page is
     physical page ``perm[offset_b + k]``;
  5. fp8 latent-row cache only: ``integers(-3, 0, (num_pages, 64, 4))``
     (both ends included), an exponent per 128-column latent tile of each
     row; the tile is multiplied by 2 to that power before encoding.
Values are rounded to bf16 (round to nearest even) or, for the fp8 cache,
encoded per token as OCP E4M3 ("fn": bias 7, max 448, no infinities) with one
fp32 scale per token, ``scale = max|row| / 448``, or, for the fp8 latent-row
cache, packed into 656-byte rows: each 128-column tile of the latent encoded
as E4M3 with its own scale, the smallest power of two not below
``max|tile| / 448`` (so that no code saturates), and the RoPE part rounded
to bf16.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

PAGE = 64
DIM_QK = 576      # d_c + d_r
DIM_V = 512       # d_c
SOFTMAX_SCALE = np.float32(1.0 / np.sqrt(192.0))   # 1/sqrt(d_n + d_r), d_n=128, d_r=64

KV_BF16 = 0
KV_FP8_E4M3 = 1
KV_FP8_LATENT = 2     # 656-byte rows: E4M3 latent, 4 fp32 tile scales, bf16 RoPE
LATENT_ROW_BYTES = 656

INT32_MAX = np.iinfo(np.int32).max


@dataclasses.dataclass(frozen=True)
class ConfigSpec:
    name: str
    B: int
    H: int
    q_chunk: int
    lengths: tuple            # ("uniform", lo, hi) or ("lognormal", mu, sigma, lo, hi)
    kv_dtype: int
    seed: int


# The five workloads: the shift from many short to few long requests, a
# ragged mix, and a causal query chunk over an fp8 cache.
CONFIGS = {
    1: ConfigSpec("tiny B=4 H=16 q=1 s~U[128,512]", 4, 16, 1, ("uniform", 128, 512), KV_BF16, 0),
    2: ConfigSpec("many-short B=256 H=128 q=1 s~U[1024,4096]", 256, 128, 1,
                  ("uniform", 1024, 4096), KV_BF16, 1),
    3: ConfigSpec("few-long B=4 H=128 q=1 s~U[65536,131072]", 4, 128, 1,
                  ("uniform", 65536, 131072), KV_BF16, 2),
    4: ConfigSpec("ragged B=64 H=128 q=1 s~LN(8,1.5) in [64,131072]", 64, 128, 1,
                  ("lognormal", 8.0, 1.5, 64, 131072), KV_BF16, 3),
    5: ConfigSpec("chunk8-fp8 B=16 H=128 q=8 s~U[8192,32768] e4m3", 16, 128, 8,
                  ("uniform", 8192, 32768), KV_FP8_E4M3, 4),
}


@dataclasses.dataclass
class Batch:
    """Host arrays of one batch; bit patterns, not values, for 16/8-bit data."""
    q: np.ndarray             # uint16 [B*q_chunk, H, 576]  (bf16 bits)
    kv: np.ndarray            # uint16 [num_pages, 64, 576] (bf16), uint8 (e4m3) or uint8 [num_pages, 64, 656] (latent rows)
    kv_scales: Optional[np.ndarray]   # float32 [num_pages, 64] for e4m3, else None
    block_table: np.ndarray   # int32 [B, max_pages]
    seq_lens: np.ndarray      # int32 [B]
    q_chunk: int
    H: int
    kv_dtype: int
    softmax_scale: np.float32

    @property
    def B(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.kv.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 with round-to-nearest-even; returns uint16 bits.

    bf16 keeps the upper 16 bits of an IEEE binary32; adding 0x7FFF plus the
    lowest kept bit before truncation rounds to nearest, ties to even.  Inputs
    are finite draws far below the overflow threshold.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _e4m3_positive_table() -> np.ndarray:
    """Values of the finite non-negative OCP E4M3 codes 0x00..0x7E, ascending."""
    vals = np.empty(127, dtype=np.float64)
    for code in range(127):
        e, m = code >> 3, code & 7
        vals[code] = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


_E4M3_POS = _e4m3_positive_table()


def f32_to_e4m3_bits(x: np.ndarray) -> np.ndarray:
    """Encode to OCP E4M3 (fn) with round-to-nearest-even, saturating at 448."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 448.0)
    hi = np.searchsorted(_E4M3_POS, a, side="left").clip(0, 126)
    lo = (hi - 1).clip(0, 126)
    d_hi = np.abs(_E4M3_POS[hi] - a)
    d_lo = np.abs(a - _E4M3_POS[lo])
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(pick_lo, lo, hi).astype(np.uint8)
    sign = np.where(np.signbit(x), np.uint8(0x80), np.uint8(0))
    return (code | sign).astype(np.uint8)


def encode_e4m3_per_token(rows: np.ndarray):
    """Quantise ``[..., 576]`` float32 rows: one fp32 scale per row."""
    amax = np.max(np.abs(rows), axis=-1).astype(np.float32)
    scale = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    codes = f32_to_e4m3_bits(rows / scale[..., None])
    return codes, scale


def encode_fp8_latent_rows(rows: np.ndarray) -> np.ndarray:
    """Pack ``[..., 576]`` float32 rows into 656-byte latent rows (uint8):
    bytes [0, 512) E4M3 codes of the latent, [512, 528) four little-endian
    fp32 tile scales (tile t = latent columns [128t, 128t + 128)), [528, 656)
    the 64 RoPE values as little-endian bf16."""
    lead = rows.shape[:-1]
    tiles = rows[..., :DIM_V].reshape(*lead, 4, 128)
    amax = np.max(np.abs(tiles), axis=-1).astype(np.float64)
    expo = np.ceil(np.log2(np.where(amax > 0, amax / 448.0, 1.0)))
    scale = np.ldexp(1.0, expo.astype(np.int32)).astype(np.float32)       # [..., 4], powers of two
    codes = f32_to_e4m3_bits(tiles / scale[..., None]).reshape(*lead, DIM_V)
    out = np.empty((*lead, LATENT_ROW_BYTES), dtype=np.uint8)
    out[..., :512] = codes
    out[..., 512:528] = np.ascontiguousarray(scale.astype('<f4')).view(np.uint8).reshape(*lead, 16)
    rope = f32_to_bf16_bits(rows[..., DIM_V:]).astype('<u2')
    out[..., 528:] = np.ascontiguousarray(rope).view(np.uint8).reshape(*lead, 128)
    return out


def draw_lengths(rng: np.random.Generator, spec: ConfigSpec) -> np.ndarray:
    kind = spec.lengths[0]
    if kind == "uniform":
        _, lo, hi = spec.lengths
        s = rng.integers(lo, hi, size=spec.B, endpoint=True)
    elif kind == "lognormal":
        _, mu, sigma, lo, hi = spec.lengths
        s = np.clip(np.rint(rng.lognormal(mu, sigma, size=spec.B)), lo, hi)
    else:
        raise ValueError(kind)
    return s.astype(np.int32)


def build_batch(rng: np.random.Generator, seq_lens, H: int, q_chunk: int,
                kv_dtype: int = KV_BF16, unused_slot: int = -1,
                extra_pages: int = 0, latent_exp=(-3, 0)) -> Batch:
    """Draw pool and queries for given lengths, following the recipe above.

    ``extra_pages`` appends never-referenced pages to the pool (their rows are
    drawn too); ``unused_slot`` fills block-table slots past each history;
    ``latent_exp`` is the range (ends included) of the latent-row tile
    exponents u of step 5.
    """
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    B = int(seq_lens.shape[0])
    if np.any(seq_lens < q_chunk):
        raise ValueError("every history must hold at least the query chunk")
    pages_per = (seq_lens.astype(np.int64) + PAGE - 1) // PAGE
    used_pages = int(pages_per.sum())
    num_pages = used_pages + int(extra_pages)
    max_pages = max(1, int(pages_per.max()) if B else 1)

    pool = rng.standard_normal((num_pages, PAGE, DIM_QK), dtype=np.float32)
    queries = rng.standard_normal((B * q_chunk, H, DIM_QK), dtype=np.float32)
    perm = rng.permutation(num_pages)

    if kv_dtype == KV_BF16:
        kv = f32_to_bf16_bits(pool)
        scales = None
    elif kv_dtype == KV_FP8_E4M3:
        kv, scales = encode_e4m3_per_token(pool)
    elif kv_dtype == KV_FP8_LATENT:
        # 5. (this format only) every 128-column latent tile of every row is
        # multiplied by 2^u, u uniform in [-3, 0] (latent_exp), so that tile
        # scales differ within a row and across rows while values stay at the
        # N(0,1) scale
        u = rng.integers(latent_exp[0], latent_exp[1], size=(num_pages, PAGE, 4), endpoint=True)
        pool[..., :DIM_V] *= np.repeat(np.ldexp(np.float32(1.0), u).astype(np.float32), 128, axis=-1)
        kv = np.concatenate([encode_fp8_latent_rows(pool[i:i + 256]) for i in range(0, num_pages, 256)]) \
            if num_pages else np.zeros((0, PAGE, LATENT_ROW_BYTES), np.uint8)
        scales = None
    else:
        raise ValueError(kv_dtype)
    del pool

    block_table = np.full((B, max_pages), unused_slot, dtype=np.int32)
    off = 0
    for b in range(B):
        n = int(pages_per[b])
        block_table[b, :n] = perm[off:off + n]
        off += n
    return Batch(q=f32_to_bf16_bits(queries), kv=kv, kv_scales=scales,
                 block_table=block_table, seq_lens=seq_lens, q_chunk=q_chunk,
                 H=H, kv_dtype=kv_dtype, softmax_scale=SOFTMAX_SCALE)


def make_config(cfg: int, seed: Optional[int] = None, unused_slot: int = -1,
                kv_dtype: Optional[int] = None) -> Batch:
    """Batch of workload ``cfg`` (1..5); seed defaults to ``cfg - 1``;
    ``kv_dtype`` overrides the workload's cache format (same lengths)."""
    spec = CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(spec.seed if seed is None else seed))
    seq_lens = draw_lengths(rng, spec)
    return build_batch(rng, seq_lens, spec.H, spec.q_chunk, spec.kv_dtype if kv_dtype is None else kv_dtype,
                       unused_slot)


KV_LABELS = {KV_BF16: "bf16", KV_FP8_E4M3: "fp8-e4m3+fp32 scale",
             KV_FP8_LATENT: "fp8-e4m3 latent, fp32 tile scales, bf16 rope (656 B rows)"}


def make_custom(seq_lens, H: int, q_chunk: int = 1, kv_dtype: int = KV_BF16,
                seed: int = 0, unused_slot: int = -1, extra_pages: int = 0, latent_exp=(-3, 0)) -> Batch:
    """Batch with explicit lengths (parity cases, edge cases)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return build_batch(rng, seq_lens, H, q_chunk, kv_dtype, unused_slot, extra_pages, latent_exp)


def poison_unused_rows(batch: Batch) -> Batch:
    """Fill every pool row that no history reaches with NaN (bf16 0x7FC0 /
    e4m3 0x7F, scale NaN; latent rows: NaN codes, scales and RoPE).  Results
    must not change."""
    kv = batch.kv.copy()
    scales = None if batch.kv_scales is None else batch.kv_scales.copy()
    used = np.zeros((batch.num_pages, PAGE), dtype=bool)
    for b in range(batch.B):
        s = int(batch.seq_lens[b])
        j = np.arange(s)
        used[batch.block_table[b, j // PAGE], j % PAGE] = True
    if batch.kv_dtype == KV_FP8_LATENT:
        nan_row = np.full(LATENT_ROW_BYTES, 0x7F, dtype=np.uint8)              # E4M3 NaN codes
        nan_row[512:528] = np.full(4, np.nan, dtype='<f4').view(np.uint8)      # NaN scales
        nan_row[528:] = np.full(64, 0x7FC0, dtype='<u2').view(np.uint8)        # bf16 NaN
        kv[~used] = nan_row
    else:
        kv[~used] = np.uint16(0x7FC0) if batch.kv_dtype == KV_BF16 else np.uint8(0x7F)
    if scales is not None:
        scales[~used] = np.float32(np.nan)
    return dataclasses.replace(batch, kv=kv, kv_scales=scales)


def workload_bytes_flops(batch: Batch):
    """Algorithmic bytes and flops of one step (what the method must move or
    compute): each token's cache row once (V is the same bytes as K), plus the
    queries, outputs, LSE, block table and lengths; flops 2*H*(576+512) per
    visible (query row, key)."""
    s = batch.seq_lens.astype(np.int64)
    q = batch.q_chunk
    row_bytes = {KV_BF16: DIM_QK * 2, KV_FP8_E4M3: DIM_QK + 4, KV_FP8_LATENT: LATENT_ROW_BYTES}[batch.kv_dtype]
    N = batch.B * q
    kv_bytes = int(s.sum()) * row_bytes
    other = (N * batch.H * DIM_QK * 2 + N * batch.H * DIM_V * 2 + N * batch.H * 4
             + int(((s + PAGE - 1) // PAGE).sum()) * 4 + batch.B * 4)
    visible = int(sum(int(sb) * q - q * (q - 1) // 2 for sb in s))
    flops = 2 * batch.H * (DIM_QK + DIM_V) * visible
    return kv_bytes, kv_bytes + other, flops
