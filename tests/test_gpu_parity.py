"""GPU parity: libsplash_attn through its C-ABI against the fp64 oracle.

Tolerances (the parity bar): outputs max-abs 1e-2 for bf16 caches and 3e-2
for the fp8 cache, LSE max-abs 1e-3; page resolution and run-to-run results
bit-exact.
"""
import dataclasses
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W
from paper_2609_37626_amd.device import to_device

pytestmark = pytest.mark.gpu

OUT_TOL = {W.KV_BF16: 1e-2, W.KV_FP8_E4M3: 3e-2, W.KV_FP8_LATENT: 3e-2}
LSE_TOL = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def run_oracle(batch, **kw):
    return oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens, batch.q_chunk,
                                batch.softmax_scale, kv_dtype=batch.kv_dtype, kv_scales=batch.kv_scales, **kw)


def gpu_attend(batch, flags=0, split_pages=0, max_partials=0):
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    ws = db.workspace(max_partials)
    B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse,
                        db.desc(flags, split_pages), ws)
    torch.cuda.synchronize()
    return out, lse


def assert_parity(batch, out, lse, ref_out=None, ref_lse=None, label=""):
    if ref_out is None:
        ref_out, ref_lse = run_oracle(batch)
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l)), label
    err_o = np.abs(o - ref_out).max()
    err_l = np.abs(l - ref_lse).max()
    print(f"{label}: out max-abs {err_o:.3e}  lse max-abs {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[batch.kv_dtype], (label, err_o)
    assert err_l <= LSE_TOL, (label, err_l)


def lognormal_lengths(seed, n, lo, hi):
    rng = np.random.Generator(np.random.PCG64(seed))
    return np.clip(np.rint(rng.lognormal(8.0, 1.5, size=n)), lo, hi).astype(np.int32)


CASES = {
    "tiny_cfg1": lambda: W.make_config(1),
    "many_short_B6_H128": lambda: W.make_custom(
        np.random.Generator(np.random.PCG64(11)).integers(1024, 4096, size=6, endpoint=True), H=128, seed=11),
    "ragged_lognormal_B12_with_edges": lambda: W.make_custom(
        np.concatenate([lognormal_lengths(12, 9, 1, 6000), [1, 64, 65]]), H=128, seed=12),
    "chunk8_fp8_B3": lambda: W.make_custom([900, 1700, 2500], H=128, q_chunk=8, kv_dtype=W.KV_FP8_E4M3,
                                           seed=13),
    "chunk4_bf16_B3": lambda: W.make_custom([4, 129, 1000], H=128, q_chunk=4, seed=14),
    "heads48_q2": lambda: W.make_custom([70, 300, 2], H=48, q_chunk=2, seed=15),
    "heads16_single_tokens": lambda: W.make_custom([1, 1, 1], H=16, seed=16),
    "heads112_fp8_q1": lambda: W.make_custom([33, 640, 1999], H=112, kv_dtype=W.KV_FP8_E4M3, seed=17),
    # batches whose plan is a fold (each worker runs its own units; the
    # longest histories hand their tails to the workers with the shortest
    # or to idle ones; ragged last pages)
    "fold_many_short_B250": lambda: W.make_custom(
        np.random.Generator(np.random.PCG64(31)).integers(64, 900, size=250, endpoint=True), H=128, seed=31),
    "fold_chunk8_fp8_B20": lambda: W.make_custom(
        np.random.Generator(np.random.PCG64(32)).integers(300, 1500, size=20, endpoint=True), H=128, q_chunk=8,
        kv_dtype=W.KV_FP8_E4M3, seed=32),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_parity_against_oracle(name):
    batch = CASES[name]()
    print(f"case {name}: B={batch.B} H={batch.H} q={batch.q_chunk} lens={batch.seq_lens.tolist()[:12]}", flush=True)
    if name.startswith("fold_"):
        seq = np.asarray(batch.seq_lens, np.int32)
        d = B.make_desc(batch.B, batch.H, int(-(-seq.max() // 64)), 1 << 20)
        assert B.splash_mla_plan_host(seq, batch.q_chunk, d, B.device_workers(), 0)[2]["fold"]
    out, lse = gpu_attend(batch)
    assert_parity(batch, out, lse, label=name)


@pytest.mark.parametrize("split_pages", [1, 3, 7])
def test_forced_splits_and_combine(split_pages):
    batch = W.make_custom([9000, 13001, 65], H=128, seed=21)
    ref = run_oracle(batch)
    out, lse = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=split_pages)
    assert_parity(batch, out, lse, *ref, label=f"forced split {split_pages}")


def scale_bf16_bits(bits, k):
    """Multiply bf16 values (bit patterns) by 2^k exactly: k added to the
    exponent field of every nonzero value (all normal here, none overflows)."""
    b = bits.astype(np.int32)
    nz = (b & 0x7FFF) != 0
    assert np.all(((b[nz] >> 7) & 0xFF) + k > 0) and np.all(((b[nz] >> 7) & 0xFF) + k < 255)
    return np.where(nz, b + (k << 7), b).astype(np.uint16)


@pytest.mark.parametrize("split_pages", [3, 40])
def test_split_partials_beyond_fp16_range(split_pages):
    """Split partials are kept in fp16 with a power-of-two scale per (slot,
    head, 128 columns).  With the cache times 2^17 and the query times 2^-17
    the scores are unchanged and every output is exactly 2^17 times the
    unscaled one, up to |out| ~ 2^19, far past fp16's 65504: the scaled run
    divided by 2^17 must meet the bar against the unscaled oracle (an
    unscaled fp16 partial would be infinite)."""
    base = W.make_custom([9000, 13001, 65], H=128, seed=21)
    ref_out, ref_lse = run_oracle(base)
    batch = dataclasses.replace(base, q=scale_bf16_bits(base.q, -17), kv=scale_bf16_bits(base.kv, 17))
    out, lse = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=split_pages)
    assert float(out.float().abs().max()) > 65504.0
    assert_parity(base, out.float() * 2.0 ** -17, lse, ref_out, ref_lse, label=f"fp16 range, split {split_pages}")


def test_many_split_rows_with_several_parts_each():
    """The step's merge takes each (split tile, head) on one wave when there
    are at least 8,192 of them with at most 16 parts each, in several
    batches of four parts: 9 requests x 8 chunk rows = 72 split tiles, x 128
    heads = 9,216 rows, 5 or 6 parts per tile."""
    batch = W.make_custom([610, 640, 700, 655, 620, 690, 600, 680, 645], H=128, q_chunk=8, seed=24)
    out, lse = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=2)
    assert_parity(batch, out, lse, label="merge by wave, 5-6 parts")


def test_fp8_query_heads_of_very_different_magnitude():
    """The fp8 caches run QK on the fp8 matrix pipe with each head's query
    row scaled by its own power of two (its largest value into [128, 256))
    and split in two E4M3 terms.  Heads scaled by 2^-12 .. 2^3 (exact bf16
    exponent steps) must each meet the bar against the oracle on the same
    scaled query, per-token cache and latent rows alike."""
    for kv_dtype in (W.KV_FP8_E4M3, W.KV_FP8_LATENT):
        batch = W.make_custom([700, 1500], H=128, q_chunk=2, kv_dtype=kv_dtype, seed=25)
        q = batch.q.copy()
        for hh in range(batch.H):
            q[:, hh] = scale_bf16_bits(q[:, hh], hh % 16 - 12)
        case = dataclasses.replace(batch, q=q)
        out, lse = gpu_attend(case)
        ref_out, ref_lse = run_oracle(case)
        assert_parity(case, out, lse, ref_out, ref_lse, label=f"fp8 query scales 2^-12..2^3, kv {kv_dtype}")
        # SPLASH_FLAG_EXACT_QK: K converted to bf16, products summed in fp32
        out_x, lse_x = gpu_attend(case, flags=B.FLAG_EXACT_QK)
        assert_parity(case, out_x, lse_x, ref_out, ref_lse, label=f"  exact QK, kv {kv_dtype}")
        assert np.abs(lse_x.cpu().numpy() - ref_lse).max() <= 5e-5


def test_forced_splits_fp8_chunk():
    batch = W.make_custom([700, 2000], H=128, q_chunk=8, kv_dtype=W.KV_FP8_E4M3, seed=22)
    out, lse = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=4)
    assert_parity(batch, out, lse, label="fp8 chunk forced split")


def test_auto_split_single_long_request():
    batch = W.make_custom([20000], H=128, seed=23)
    out, lse = gpu_attend(batch)
    assert_parity(batch, out, lse, label="single long auto split")


def test_small_partial_capacity_still_correct():
    batch = W.make_custom([9000, 13001], H=128, seed=24)
    out, lse = gpu_attend(batch, max_partials=3)
    assert_parity(batch, out, lse, label="3 partial slots")


def test_poisoned_unused_rows_and_slots_change_nothing():
    clean = W.make_custom([63, 65, 200, 1], H=128, seed=25, extra_pages=3)
    poisoned = W.poison_unused_rows(W.make_custom([63, 65, 200, 1], H=128, seed=25, extra_pages=3,
                                                  unused_slot=W.INT32_MAX))
    o1, l1 = gpu_attend(clean)
    o2, l2 = gpu_attend(poisoned)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    assert_parity(clean, o1, l1, label="poison")


def test_poisoned_fp8_unused_rows():
    clean = W.make_custom([63, 100], H=128, q_chunk=2, kv_dtype=W.KV_FP8_E4M3, seed=26, extra_pages=2)
    poisoned = W.poison_unused_rows(clean)
    o1, l1 = gpu_attend(clean)
    o2, l2 = gpu_attend(poisoned)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)


def test_run_to_run_and_page_permutation_bit_identical():
    batch = W.make_custom([3000, 77, 1500], H=128, seed=27, extra_pages=4)
    o1, l1 = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=5)
    o2, l2 = gpu_attend(batch, flags=B.FLAG_FORCE_SPLIT, split_pages=5)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    rng = np.random.Generator(np.random.PCG64(99))
    perm = rng.permutation(batch.num_pages)
    kv2 = np.empty_like(batch.kv)
    kv2[perm] = batch.kv
    bt2 = np.where(batch.block_table >= 0, perm[batch.block_table.clip(0)], -1).astype(np.int32)
    import dataclasses
    moved = dataclasses.replace(batch, kv=kv2, block_table=bt2)
    o3, l3 = gpu_attend(moved, flags=B.FLAG_FORCE_SPLIT, split_pages=5)
    assert torch.equal(o1.view(torch.int16), o3.view(torch.int16)) and torch.equal(l1, l3)


@pytest.mark.parametrize("target", [0, 31, 32, 63, 64, 100, 191])
def test_dominant_logit_returns_that_latent_bit_exactly(target):
    """q_rope = k_rope = 8 on one token: its weight rounds to exactly 1 in fp32,
    so the output is that token's latent, bit for bit, wherever its page sits."""
    batch = W.make_custom([192], H=16, seed=28)
    s = 192
    q = W.f32_to_bf16_bits(np.zeros((1, 16, 576), np.float32))
    q[..., 512:] = W.f32_to_bf16_bits(np.float32(8.0))
    kv = batch.kv.copy()
    phys = lambda j: (int(batch.block_table[0, j // 64]), j % 64)
    for j in range(s):
        kv[phys(j)][512:] = 0
    kv[phys(target)][512:] = W.f32_to_bf16_bits(np.float32(8.0))
    import dataclasses
    case = dataclasses.replace(batch, q=q, kv=kv)
    out, _ = gpu_attend(case)
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got[0, 0], kv[phys(target)][:512])
    assert np.array_equal(got[0, 15], kv[phys(target)][:512])


def test_unit_values_give_unit_output():
    batch = W.make_custom([300, 5], H=32, seed=29)
    kv = batch.kv.copy()
    kv[..., :512] = W.f32_to_bf16_bits(np.float32(1.0))
    import dataclasses
    out, _ = gpu_attend(dataclasses.replace(batch, kv=kv))
    assert np.abs(out.float().cpu().numpy() - 1.0).max() <= 1e-2


def test_debug_gather_is_bit_exact():
    for dtype, batch in [(W.KV_BF16, W.make_custom([1, 64, 65, 300], H=16, seed=30, unused_slot=W.INT32_MAX)),
                         (W.KV_FP8_E4M3, W.make_custom([129, 7], H=16, kv_dtype=W.KV_FP8_E4M3, seed=31))]:
        db = to_device(batch)
        total = int(batch.seq_lens.sum())
        row_bytes = 1152 if dtype == W.KV_BF16 else 576
        dense = torch.zeros((total, row_bytes), dtype=torch.uint8, device="cuda")
        B.splash_mla_debug_gather(db.kv, db.block_table, db.seq_lens, db.desc(), dense)
        torch.cuda.synchronize()
        flat = batch.kv.reshape(batch.num_pages * 64, -1)
        rows = []
        for b, s in enumerate(batch.seq_lens):
            j = np.arange(int(s))
            rows.append(flat[batch.block_table[b, j // 64].astype(np.int64) * 64 + j % 64])
        want = np.concatenate(rows).view(np.uint8).reshape(total, row_bytes)
        assert np.array_equal(dense.cpu().numpy(), want)


def _plan_lengths(case):
    if case.startswith("cfg"):
        spec = W.CONFIGS[int(case[3:])]
        rng = np.random.Generator(np.random.PCG64(spec.seed))
        return W.draw_lengths(rng, spec), spec.q_chunk, spec.H
    lens = {
        # one history long enough that the geometric candidates (index >= 64)
        # are distinct sizes and can win
        "one_long": [262144],
        "long_and_short": [200000, 64, 65, 3000, 1],
        "equal_lengths": [4096] * 40,
    }.get(case)
    if case == "over_8192_tiles":
        # 2,100 requests of 4-row chunks: 8,400 tiles, more than the planner
        # caches in LDS (the uncached path, units in tile order)
        lens = np.random.Generator(np.random.PCG64(41)).integers(4, 400, size=2100, endpoint=True)
        return lens.astype(np.int32), 4, 16
    return np.asarray(lens, dtype=np.int32), 1, 128


@pytest.mark.parametrize("case", ["cfg2", "cfg3", "cfg4", "cfg5", "one_long", "long_and_short", "equal_lengths",
                                  "over_8192_tiles"])
def test_device_plan_matches_host_plan(case):
    seq, q_chunk, H = _plan_lengths(case)
    Bn = len(seq)
    d = B.make_desc(Bn, H, int(-(-seq.max() // 64)), int((-(-seq // 64)).sum()))
    ws = torch.zeros(B.workspace_size(Bn, q_chunk, H, 0), dtype=torch.uint8, device="cuda")
    B.splash_mla_plan(torch.from_numpy(seq).cuda(), q_chunk, d, ws)
    torch.cuda.synchronize()
    units, indptr, stats = B.splash_mla_plan_host(seq, q_chunk, d, B.device_workers(), 0)
    offs, _ = B.workspace_offsets(Bn, q_chunk, H, 0)
    raw = ws.cpu().numpy()
    G = B.device_workers()
    hdr = raw[offs[0]:offs[0] + 4 * (64 + G + 1)].view(np.int32)
    print(f"plan {case}: chunk {stats['chunk_pages']} units {stats['units']} partials {stats['partials']} "
          f"fold {stats['fold']}", flush=True)
    assert hdr[1] == stats["units"] and hdr[2] == stats["partials"] and hdr[3] == stats["chunk_pages"]
    assert hdr[8] == stats["max_parts"] and hdr[9] == (G if stats["fold"] else 0)
    dev_units = raw[offs[1]:offs[1] + 16 * stats["units"]].view(np.int32).reshape(-1, 4)
    if stats["fold"]:
        # the same cap, units and worker runs; histories of equal length may
        # sit at each other's ranks (the device orders ties with atomics), so
        # each worker's run is compared by its unit lengths and the split
        # pieces by their pages
        assert hdr[10] == stats["cap"]
        canon = lambda u: u[np.lexsort(u.T[::-1])]
        assert np.array_equal(canon(dev_units), canon(units))
        ws = stats["worker_start"]
        assert np.array_equal(hdr[64:64 + G + 1], ws)
        runs = lambda u: [sorted((u[a:b, 2] - u[a:b, 1]).tolist()) for a, b in zip(ws[:-1], ws[1:])]
        assert runs(dev_units) == runs(units)
    elif stats["units"] > G and Bn * q_chunk <= 8192:
        # the same units (the device leaves the order of equal-length units
        # open), and both queues hand out the longest units first; with query
        # chunks, whole requests (each request's units side by side, the
        # requests ordered by their longest unit, ties in any order)
        canon = lambda u: u[np.lexsort(u.T[::-1])]
        assert np.array_equal(canon(dev_units), canon(units))
        for u in (dev_units, units):
            ln = u[:, 2] - u[:, 1]
            if q_chunk == 1:
                assert np.all(ln[:-1] >= ln[1:])
                continue
            req = u[:, 0] // q_chunk
            starts = np.flatnonzero(np.r_[True, req[1:] != req[:-1]])
            assert len(starts) == len(np.unique(req)), "a request's units are not contiguous"
            keys = [ln[a:b].max() for a, b in zip(starts, np.r_[starts[1:], len(u)])]
            assert all(k0 >= k1 for k0, k1 in zip(keys[:-1], keys[1:]))
    elif stats["units"] > G:
        # more tiles than the planner caches in LDS: the units in tile order
        assert np.array_equal(dev_units, units)
        assert np.all(np.diff(units[:, 0]) >= 0)
    else:
        # at most one unit per worker: tile order
        assert np.array_equal(dev_units, units)
    T = Bn * q_chunk
    dev_indptr = raw[offs[2]:offs[2] + 4 * (T + 1)].view(np.int32)
    assert np.array_equal(dev_indptr, indptr)


def test_plan_once_run_many():
    batch = W.make_custom([5000, 300, 64], H=128, seed=32)
    db = to_device(batch)
    ws = db.workspace()
    d = db.desc()
    B.splash_mla_plan(db.seq_lens, 1, d, ws)
    outs = []
    for _ in range(3):
        out, lse = db.alloc_outputs()
        B.splash_mla_run(db.q, db.kv, db.block_table, db.seq_lens, 1, out, lse, d, ws)
        outs.append((out, lse))
    torch.cuda.synchronize()
    for out, lse in outs[1:]:
        assert torch.equal(out.view(torch.int16), outs[0][0].view(torch.int16)) and torch.equal(lse, outs[0][1])
    assert_parity(batch, *outs[0], label="plan once, run three times")


def test_standalone_combine_matches_oracle_merge():
    batch = W.make_custom([500, 240], H=16, q_chunk=2, seed=33)
    cuts = {0: [0, 100, 101, 500], 1: [0, 240, 240]}        # includes an empty part
    parts_o, parts_l, indptr = [], [], [0]
    for b in range(batch.B):
        for lo, hi in zip(cuts[b][:-1], cuts[b][1:]):
            kr = np.zeros((batch.B, 2), np.int64)
            kr[b] = (lo, hi)
            o, l = run_oracle(batch, requests=[b], key_ranges=kr)
            parts_o.append(np.nan_to_num(o[b * 2:(b + 1) * 2]))
            parts_l.append(l[b * 2:(b + 1) * 2])
        indptr.append(indptr[-1] + len(cuts[b]) - 1)
    partials = torch.tensor(np.stack(parts_o), dtype=torch.float32, device="cuda")
    plse = torch.tensor(np.stack(parts_l), dtype=torch.float32, device="cuda")
    ip = torch.tensor(indptr, dtype=torch.int32, device="cuda")
    out = torch.empty((batch.B * 2, 16, 512), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((batch.B * 2, 16), dtype=torch.float32, device="cuda")
    B.splash_mla_combine(partials, plse, ip, batch.B, 2, 16, out, lse)
    torch.cuda.synchronize()
    assert_parity(batch, out, lse, label="standalone combine")


def test_idle_owner_on_gpu():
    d = B.make_desc(0, 128, 1, 1)
    ws = torch.zeros(1024, dtype=torch.uint8, device="cuda")
    B.splash_mla_attend(None, None, None, None, 1, None, None, d, ws)


def test_debug_check_rejects_bad_device_data():
    batch = W.make_custom([100, 300], H=16, seed=34)
    bad = batch.block_table.copy()
    bad[1, 2] = batch.num_pages + 5                          # outside the pool
    import dataclasses
    db = to_device(dataclasses.replace(batch, block_table=bad))
    out, lse = db.alloc_outputs()
    with pytest.raises(B.SplashError) as e:
        B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, 1, out, lse,
                            db.desc(flags=B.FLAG_DEBUG_CHECK), db.workspace())
    assert e.value.status == B.SPLASH_ERR_INVALID_ARGUMENT
    good = to_device(batch)
    out, lse = good.attend(flags=B.FLAG_DEBUG_CHECK)
    torch.cuda.synchronize()
    assert_parity(batch, out, lse, label="debug check passes good data")


def test_more_than_8192_tiles():
    """8,400 tiles (2,100 requests x 4 chunk rows): the planner's uncached
    path and the snake-dealt unit queue, against the oracle on sampled rows of
    every kind (first, middle, last request; every chunk row; three heads)."""
    lens, q_chunk, H = _plan_lengths("over_8192_tiles")
    batch = W.make_custom(lens, H=H, q_chunk=q_chunk, seed=42)
    out, lse = gpu_attend(batch)
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
    reqs = sorted({0, 1, 777, 1049, 1500, 2098, 2099, int(np.argmax(lens)), int(np.argmin(lens))})
    samples = [(b, i, h) for b in reqs for i in range(q_chunk) for h in (0, 7, 15)]
    ref_o, ref_l = oracle.mla_attention_sampled(batch.q, batch.kv, batch.block_table, batch.seq_lens, q_chunk,
                                                batch.softmax_scale, samples)
    got_o = np.stack([o[b * q_chunk + i, h] for b, i, h in samples])
    got_l = np.array([l[b * q_chunk + i, h] for b, i, h in samples])
    err_o, err_l = np.abs(got_o - ref_o).max(), np.abs(got_l - ref_l).max()
    print(f"8400 tiles, {len(samples)} sampled rows: out max-abs {err_o:.3e}  lse max-abs {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[W.KV_BF16] and err_l <= LSE_TOL
