"""The seeded input generator (CPU only)."""
import numpy as np
import pytest
import torch

from paper_2609_37626_amd import workloads as W


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    rng = np.random.Generator(np.random.PCG64(0))
    x = rng.standard_normal(200_000, dtype=np.float32) * np.float32(3.0)
    # exact ties: low 16 bits = 0x8000 with both parities of the kept bit
    u = rng.integers(0x3F000000, 0x40800000, size=4096, dtype=np.uint32)
    ties = ((u & np.uint32(0xFFFF0000)) | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    mine = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


def test_e4m3_encoding_matches_torch_float8_e4m3fn_in_range():
    rng = np.random.Generator(np.random.PCG64(1))
    x = rng.uniform(-448, 448, size=100_000).astype(np.float32)
    small = rng.uniform(-0.02, 0.02, size=20_000).astype(np.float32)   # subnormal range
    codes = np.arange(127, dtype=np.uint8)
    vals = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)                 # exact ties
    x = np.concatenate([x, small, mids, -mids, np.float32([0.0, -0.0, 448.0, -448.0])])
    mine = W.f32_to_e4m3_bits(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(mine, ref)


def test_e4m3_encoding_saturates():
    assert W.f32_to_e4m3_bits(np.float32([1e6, -1e6, 449.0])).tolist() == [0x7E, 0xFE, 0x7E]


def test_per_token_scale_maps_row_max_to_448():
    rng = np.random.Generator(np.random.PCG64(2))
    rows = rng.standard_normal((50, 576), dtype=np.float32)
    codes, scale = W.encode_e4m3_per_token(rows)
    amax_code = np.max(codes & 0x7F, axis=-1)
    assert np.all(amax_code == 0x7E)
    assert scale.dtype == np.float32


@pytest.mark.parametrize("cfg,total,pages,lo,hi", [
    (1, 1383, 24, 231, 455),
    (2, 661514, 10465, 1041, 4091),
    (3, 360906, 5640, 72699, 120428),
    (4, 539528, 8461, 64, 131072),
    (5, 375232, 5872, 10178, 32185),
])
def test_realised_lengths_of_the_five_workloads(cfg, total, pages, lo, hi):
    spec = W.CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(spec.seed))
    s = W.draw_lengths(rng, spec).astype(np.int64)
    assert (s.sum(), ((s + 63) // 64).sum(), s.min(), s.max()) == (total, pages, lo, hi)


def test_block_table_is_a_permutation_of_the_pool():
    b = W.make_custom([1, 64, 65, 300], H=16, q_chunk=1, seed=3)
    used = b.block_table[b.block_table >= 0]
    assert sorted(used.tolist()) == list(range(b.num_pages))
    for r, s in enumerate(b.seq_lens):
        n = (int(s) + 63) // 64
        assert np.all(b.block_table[r, n:] == -1)


def test_poison_marks_only_rows_no_history_reaches():
    b = W.make_custom([5, 70], H=16, q_chunk=1, seed=4, extra_pages=2)
    p = W.poison_unused_rows(b)
    changed = np.any(p.kv != b.kv, axis=-1)
    assert changed.sum() == b.num_pages * 64 - int(b.seq_lens.sum())


def test_chunk_longer_than_history_is_rejected():
    with pytest.raises(ValueError):
        W.make_custom([3], H=16, q_chunk=4)


def test_workload_accounting_cfg2():
    spec = W.CONFIGS[2]
    rng = np.random.Generator(np.random.PCG64(spec.seed))
    s = W.draw_lengths(rng, spec)
    # accounting only needs lengths; build a tiny stand-in batch with the same lengths
    class _B:
        seq_lens = s
        q_chunk = 1
        H = 128
        kv_dtype = W.KV_BF16
        B = 256
    kv, total, flops = W.workload_bytes_flops(_B)
    assert kv == 661514 * 1152
    assert flops == 2 * 128 * 1088 * 661514
    assert 833e6 < total < 834e6


def test_latent_rows_recipe():
    # 656-byte rows: every tile scale is the smallest power of two not below
    # max|tile| / 448 (so max|tile| / scale lies in (224, 448], and its E4M3
    # code in [224, 448]: the codes are 32 apart there), codes are
    # finite, the RoPE bytes are the bf16 rounding of the drawn values, and
    # the other draws of the stream are those of the bf16 cache
    b = W.make_custom([70, 130, 64], H=16, q_chunk=2, kv_dtype=W.KV_FP8_LATENT, seed=9)
    assert b.kv.shape == (b.num_pages, 64, 656) and b.kv.dtype == np.uint8
    rows = b.kv.reshape(-1, 656)
    scales = rows[:, 512:528].copy().view('<f4')
    m, e = np.frexp(scales)
    assert np.all(m == 0.5)                                    # powers of two
    codes = torch.from_numpy(rows[:, :512].copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.all(np.isfinite(codes))
    amax = np.abs(codes.reshape(-1, 4, 128)).max(axis=-1)
    assert np.all((amax >= 224) & (amax <= 448))
    assert len(np.unique(scales)) >= 3                         # tile scales differ
    ref = W.make_custom([70, 130, 64], H=16, q_chunk=2, kv_dtype=W.KV_BF16, seed=9)
    assert np.array_equal(b.q, ref.q) and np.array_equal(b.block_table, ref.block_table)
    assert np.array_equal(rows[:, 528:].copy().view('<u2'), ref.kv.reshape(-1, 576)[:, 512:])
