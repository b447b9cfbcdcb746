"""GPU parity of the fp8 latent-row cache (SPLASH_KV_FP8_LATENT).

A 656-byte row holds the 512 E4M3 latent codes, four fp32 tile scales (one
per 128 latent columns) and the 64 RoPE values in bf16 (App. B, theoretical
scenarios for DCU and H200, residency assumptions; the split and the scale
granularity are this library's reading).  The oracle decodes the rows in
float64; the kernel converts each latent tile with its scale for QK^T and
scales each wave's P by its tile's key scales for PV.  The tolerances are
the fp8 bar: outputs max-abs 3e-2, LSE 1e-3.
"""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W
from paper_2609_37626_amd.device import to_device
from tests.test_gpu_parity import assert_parity, gpu_attend, run_oracle
from tests.test_gpu_shards import check_merged, check_shards, page_cuts, run_shards

pytestmark = pytest.mark.gpu

LAT = W.KV_FP8_LATENT


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


CASES = {
    # tails of every length class, a page-exact history, the longest here
    "ragged_q1_H128": lambda: W.make_custom([1, 31, 32, 33, 63, 64, 65, 700, 2222, 5000], H=128, kv_dtype=LAT,
                                            seed=61),
    "chunk8_H128": lambda: W.make_custom([900, 1700, 2500], H=128, q_chunk=8, kv_dtype=LAT, seed=62),
    "heads112_q1": lambda: W.make_custom([33, 640, 1999], H=112, kv_dtype=LAT, seed=63),
    "heads16_q3": lambda: W.make_custom([50, 130, 3], H=16, q_chunk=3, kv_dtype=LAT, seed=64),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_latent_parity_against_oracle(name):
    batch = CASES[name]()
    print(f"{name}: lens {batch.seq_lens.tolist()} H={batch.H} q={batch.q_chunk}", flush=True)
    out, lse = gpu_attend(batch)
    assert_parity(batch, out, lse, label=name)


@pytest.mark.parametrize("split_pages", [1, 3])
def test_latent_forced_splits(split_pages):
    batch = W.make_custom([3000, 77, 1500], H=128, kv_dtype=LAT, seed=65)
    out, lse = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=split_pages)
    assert_parity(batch, out, lse, label=f"latent split {split_pages}")


def test_latent_poisoned_unused_rows_change_nothing():
    clean = W.make_custom([63, 100, 129], H=128, q_chunk=2, kv_dtype=LAT, seed=66, extra_pages=2)
    poisoned = W.poison_unused_rows(clean)
    o1, l1 = gpu_attend(clean)
    o2, l2 = gpu_attend(poisoned)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    assert_parity(clean, o1, l1, label="latent poison")


def test_each_output_tile_takes_its_own_scale():
    # every latent code 1.0 and tile scales 1/2, 2, 8, 1/8 in every row: the
    # weights sum to one, so output columns [128t, 128t+128) equal scale t
    batch = W.make_custom([300, 5, 64], H=128, kv_dtype=LAT, seed=67)
    kv = batch.kv.copy()
    kv[..., :512] = 0x38
    kv[..., 512:528] = np.array([0.5, 2.0, 8.0, 0.125], dtype='<f4').view(np.uint8)
    out, _ = gpu_attend(dataclasses.replace(batch, kv=kv))
    o = out.float().cpu().numpy()
    for t, sc in enumerate([0.5, 2.0, 8.0, 0.125]):
        assert np.abs(o[..., 128 * t:128 * (t + 1)] - sc).max() <= 1e-2 * sc, t


def test_latent_shards_merge_to_the_whole():
    lens = np.random.Generator(np.random.PCG64(68)).integers(1, 3000, size=8, endpoint=True)
    batch = W.make_custom(np.concatenate([lens, [1, 64, 65]]), H=128, kv_dtype=LAT, seed=68)
    cuts = page_cuts(batch.seq_lens, 3, np.random.default_rng(68), empty_every=4)
    part_out, part_lse, out, lse = run_shards(batch, cuts)
    check_shards(batch, cuts, part_out, part_lse, "latent T=3")
    check_merged(batch, out, lse, "latent T=3")


def test_latent_debug_gather_is_bit_exact():
    batch = W.make_custom([129, 7, 64], H=16, kv_dtype=LAT, seed=69)
    db = to_device(batch)
    total = int(batch.seq_lens.sum())
    dense = torch.zeros((total, W.LATENT_ROW_BYTES), dtype=torch.uint8, device="cuda")
    B.splash_mla_debug_gather(db.kv, db.block_table, db.seq_lens, db.desc(), dense)
    torch.cuda.synchronize()
    flat = batch.kv.reshape(batch.num_pages * 64, -1)
    rows = [flat[int(batch.block_table[b, j // 64]) * 64 + j % 64]
            for b, s in enumerate(batch.seq_lens) for j in range(int(s))]
    assert np.array_equal(dense.cpu().numpy(), np.stack(rows))



def test_debug_check_rejects_scales_that_are_not_powers_of_two():
    batch = W.make_custom([130, 64], H=16, kv_dtype=LAT, seed=71)
    out_ref, lse_ref = gpu_attend(batch)
    out_dbg, lse_dbg = gpu_attend(batch, flags=B.FLAG_DEBUG_CHECK)   # valid data passes, same result
    assert torch.equal(out_ref.view(torch.int16), out_dbg.view(torch.int16)) and torch.equal(lse_ref, lse_dbg)
    p0, p1 = int(batch.block_table[0, 2]), int(batch.block_table[1, 0])
    # (the weights take a scale as an exponent step, so the format also caps
    # scales at 2^63)
    for page, row, value in [(p0, 1, 3.0), (p1, 63, -0.5), (p0, 0, 0.0), (p0, 1, np.inf), (p1, 2, 2.0 ** 64)]:
        kv = batch.kv.copy()
        kv[page, row, 512 + 4:512 + 8] = np.array([value], dtype='<f4').view(np.uint8)   # tile 1
        with pytest.raises(B.SplashError):
            gpu_attend(dataclasses.replace(batch, kv=kv), flags=B.FLAG_DEBUG_CHECK)
    kv = batch.kv.copy()
    kv[p1, 2, 512 + 4:512 + 8] = np.array([2.0 ** 63], dtype='<f4').view(np.uint8)    # the largest allowed
    gpu_attend(dataclasses.replace(batch, kv=kv), flags=B.FLAG_DEBUG_CHECK)
    # a row past the end of history 0 (130 keys: page 2 holds keys 128, 129)
    # is never reached, so its scales may hold anything
    kv = batch.kv.copy()
    kv[p0, 5, 512:528] = np.full(4, 3.0, dtype='<f4').view(np.uint8)
    gpu_attend(dataclasses.replace(batch, kv=kv), flags=B.FLAG_DEBUG_CHECK)


def test_latent_history_longer_than_one_unit():
    # 70,000 keys = 1,094 pages: more than one unit may hold, so the history
    # is split and its partials combined
    batch = W.make_custom([70000, 3000], H=32, kv_dtype=LAT, seed=72)
    out, lse = gpu_attend(batch)
    assert_parity(batch, out, lse, label="latent 70000 keys")


@pytest.mark.parametrize("k,q_chunk", [(64, 1), (700, 1), (3000, 1), (300, 8)])
def test_latent_topk_against_oracle(k, q_chunk):
    # top-k rows over latent rows: the sparse attention of the paper's
    # backend over the DeepSeek-V3.2-style cache (k = 3000 splits a list
    # over units)
    from tests.test_gpu_topk import check, lists, run_topk
    lens = np.random.Generator(np.random.PCG64(73 + k)).integers(q_chunk, 4000, size=6, endpoint=True)
    batch = W.make_custom(lens, H=128, q_chunk=q_chunk, kv_dtype=LAT, seed=73)
    idx, cnt = lists(batch, k, np.random.default_rng(k), empty_rows=(1,), recent=8)
    out, lse = run_topk(batch, idx, cnt)
    check(batch, idx, cnt, out, lse, f"latent top-k k={k} q={q_chunk}")


def test_topk_debug_check_rejects_listed_scales_that_are_not_powers_of_two():
    # DEBUG_CHECK of the top-k entry checks the tile scales of every listed
    # row; a row nobody lists may hold anything
    from tests.test_gpu_topk import run_topk
    batch = W.make_custom([300, 200], H=16, kv_dtype=LAT, seed=74)
    N = batch.B
    idx = np.full((N, 4), -1, dtype=np.int32)
    idx[0, :3] = [5, 130, 299]
    idx[1, :2] = [0, 199]
    cnt = np.array([3, 2], dtype=np.int32)
    out_ref, lse_ref = run_topk(batch, idx, cnt)
    out_dbg, lse_dbg = run_topk(batch, idx, cnt, flags=B.FLAG_DEBUG_CHECK)   # valid data passes, same result
    assert torch.equal(out_ref.view(torch.int16), out_dbg.view(torch.int16)) and torch.equal(lse_ref, lse_dbg)

    def row_of(b, pos):
        return int(batch.block_table[b, pos // 64]), pos % 64

    for (b, pos), value in [((0, 130), 3.0), ((1, 199), -0.5), ((0, 5), 0.0), ((1, 0), np.inf), ((0, 299), 2.0 ** 64)]:
        page, r = row_of(b, pos)
        kv = batch.kv.copy()
        kv[page, r, 512 + 8:512 + 12] = np.array([value], dtype='<f4').view(np.uint8)   # tile 2
        with pytest.raises(B.SplashError):
            run_topk(dataclasses.replace(batch, kv=kv), idx, cnt, flags=B.FLAG_DEBUG_CHECK)
    page, r = row_of(0, 6)   # position 6 of history 0 is not listed
    kv = batch.kv.copy()
    kv[page, r, 512:528] = np.full(4, 3.0, dtype='<f4').view(np.uint8)
    run_topk(dataclasses.replace(batch, kv=kv), idx, cnt, flags=B.FLAG_DEBUG_CHECK)


def test_latent_tile_exponents_up_to_three():
    """Tile exponents u in [-3, 3] (scales 2^-10 ... 2^-3): latent values up to
    8 times the N(0,1) scale, outputs up to tens.  Checked against a bar
    relative to the magnitude: |out - ref| <= 3e-2 + 2^-7 |ref| (the fp8
    absolute bar, plus the bf16 rounding of the output and of the weights,
    each 2^-9 relative), |lse - ref| <= 1e-3 + 1e-5 |ref|."""
    batch = W.make_custom([300, 1700, 65], H=64, q_chunk=2, kv_dtype=LAT, seed=75, latent_exp=(-3, 3))
    out, lse = gpu_attend(batch)
    ref_o, ref_l = run_oracle(batch)
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
    excess_o = np.abs(o - ref_o) - (3e-2 + 2.0 ** -7 * np.abs(ref_o))
    excess_l = np.abs(l - ref_l) - (1e-3 + 1e-5 * np.abs(ref_l))
    print(f"wide exponents: |ref out| max {np.abs(ref_o).max():.2f}; out max-abs {np.abs(o - ref_o).max():.3e}; "
          f"worst excess over the bar {excess_o.max():.3e}; lse max-abs {np.abs(l - ref_l).max():.3e}", flush=True)
    assert excess_o.max() <= 0 and excess_l.max() <= 0
