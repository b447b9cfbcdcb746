"""GPU parity of position shards (splash_mla_attend_shard + splash_mla_combine).

A shard holds the keys [key_begin[b], key_end[b]) of each request's history
(App. E, position-sharded CP).  Each shard's partial result is checked against
the oracle restricted to those keys, and the merge of all shards against the
oracle over the whole history.  Tolerances are the parity bar's (outputs
max-abs 1e-2 for bf16 caches, 3e-2 for fp8; LSE 1e-3); rows with no key in a
shard must come back as exactly out = 0, lse = -inf.
"""
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


def page_cuts(seq_lens, num_shards, rng, empty_every=0):
    """[B, num_shards + 1] shard boundaries: 0, page-aligned interior cuts
    (some shards empty when two cuts coincide), seq_len."""
    cuts = []
    for k, s in enumerate(seq_lens):
        pages = -(-int(s) // 64)
        inner = np.sort(rng.integers(0, pages + 1, size=num_shards - 1)) * 64
        if empty_every and k % empty_every == 0:
            inner[:] = inner[0]                      # all but two shards empty
        inner = np.minimum(inner, int(s))
        cuts.append(np.concatenate([[0], inner, [int(s)]]))
    return np.asarray(cuts, dtype=np.int32)


def run_shards(batch, cuts, bt=None, flags=0):
    db = to_device(batch)
    if bt is not None:
        db.block_table = torch.from_numpy(bt).cuda()
    T = cuts.shape[1] - 1
    N = batch.B * batch.q_chunk
    part_out = torch.full((batch.B * T * batch.q_chunk, batch.H, 512), float("nan"), device="cuda")
    part_lse = torch.full((batch.B * T * batch.q_chunk, batch.H), float("nan"), device="cuda")
    ws = db.workspace()
    for k in range(T):
        kb = torch.from_numpy(np.ascontiguousarray(cuts[:, k])).cuda()
        ke = torch.from_numpy(np.ascontiguousarray(cuts[:, k + 1])).cuda()
        B.splash_mla_attend_shard(db.q, db.kv, db.block_table, db.seq_lens, batch.q_chunk, kb, ke, T, k,
                                  part_out, part_lse, db.desc(flags), ws)
    out, lse = db.alloc_outputs()
    indptr = torch.arange(0, (batch.B + 1) * T, T, dtype=torch.int32, device="cuda")
    B.splash_mla_combine(part_out, part_lse, indptr, batch.B, batch.q_chunk, batch.H, out, lse)
    torch.cuda.synchronize()
    assert out.shape[0] == N
    return part_out, part_lse, out, lse


def oracle_of(batch, key_ranges=None):
    return oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens, batch.q_chunk,
                                batch.softmax_scale, kv_dtype=batch.kv_dtype, kv_scales=batch.kv_scales,
                                key_ranges=key_ranges)


def check_shards(batch, cuts, part_out, part_lse, label):
    T = cuts.shape[1] - 1
    q, H = batch.q_chunk, batch.H
    po = part_out.cpu().numpy().reshape(batch.B, T, q, H, 512)
    pl = part_lse.cpu().numpy().reshape(batch.B, T, q, H)
    for k in range(T):
        ref_o, ref_l = oracle_of(batch, np.stack([cuts[:, k], cuts[:, k + 1]], axis=1))
        ref_o = ref_o.reshape(batch.B, q, H, 512)
        ref_l = ref_l.reshape(batch.B, q, H)
        o, l = po[:, k], pl[:, k]
        empty = ~np.isfinite(ref_l)
        assert np.array_equal(np.isneginf(l), empty), label
        assert np.all(o[empty] == 0.0), label
        if np.any(~empty):
            err_o = np.abs(o[~empty] - ref_o[~empty]).max()
            err_l = np.abs(l[~empty] - ref_l[~empty]).max()
            print(f"{label} shard {k}: {int((~empty).sum())} rows, out max-abs {err_o:.3e} lse {err_l:.3e}",
                  flush=True)
            assert err_o <= OUT_TOL[batch.kv_dtype] and err_l <= LSE_TOL, (label, k, err_o, err_l)


def check_merged(batch, out, lse, label):
    ref_o, ref_l = oracle_of(batch)
    err_o = np.abs(out.float().cpu().numpy() - ref_o).max()
    err_l = np.abs(lse.cpu().numpy() - ref_l).max()
    print(f"{label} merged: out max-abs {err_o:.3e}  lse {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[batch.kv_dtype] and err_l <= LSE_TOL, (label, err_o, err_l)


def test_shards_of_ragged_histories_merge_to_the_whole():
    lens = np.random.Generator(np.random.PCG64(41)).integers(1, 3000, size=10, endpoint=True)
    batch = W.make_custom(np.concatenate([lens, [1, 64, 65]]), H=128, seed=41)
    cuts = page_cuts(batch.seq_lens, 3, np.random.default_rng(41), empty_every=4)
    print(f"lens {batch.seq_lens.tolist()}", flush=True)
    part_out, part_lse, out, lse = run_shards(batch, cuts)
    check_shards(batch, cuts, part_out, part_lse, "ragged T=3")
    check_merged(batch, out, lse, "ragged T=3")


def test_shards_of_a_chunk_with_fp8_cache():
    # q_chunk = 8: the rows of a chunk see different prefixes, so the last
    # shard of every request is cut by the causal mask row by row
    batch = W.make_custom([700, 1500, 2222], H=128, q_chunk=8, kv_dtype=W.KV_FP8_E4M3, seed=42)
    cuts = page_cuts(batch.seq_lens, 4, np.random.default_rng(42))
    cuts[:, -2] = (cuts[:, -1] - 8) // 64 * 64          # the last shard starts just before the chunk
    cuts[:, 1:-1] = np.minimum.accumulate(cuts[:, 1:-1][:, ::-1], axis=1)[:, ::-1]
    part_out, part_lse, out, lse = run_shards(batch, cuts)
    check_shards(batch, cuts, part_out, part_lse, "chunk8 fp8 T=4")
    check_merged(batch, out, lse, "chunk8 fp8 T=4")


def test_long_histories_in_many_shards():
    # the CP use: a few long histories, each cut into 8 position shards whose
    # pieces the planner splits further (partials inside a shard, then the
    # shard's own combine)
    batch = W.make_custom([40000, 23001], H=64, seed=43)
    s = batch.seq_lens.astype(np.int64)
    cuts = np.stack([np.minimum(s, (s * k // 8) // 64 * 64) for k in range(8)] + [s], axis=1).astype(np.int32)
    part_out, part_lse, out, lse = run_shards(batch, cuts)
    check_shards(batch, cuts, part_out, part_lse, "long T=8")
    check_merged(batch, out, lse, "long T=8")


def test_shard_end_inside_a_page():
    # a shard may end anywhere (its start is a page boundary)
    batch = W.make_custom([1000, 777, 130], H=32, seed=44)
    cuts = np.array([[128, 555], [64, 700], [0, 65]], dtype=np.int32)
    part_out, part_lse, _, _ = run_shards(batch, cuts)
    check_shards(batch, cuts, part_out, part_lse, "end inside a page")


def test_pages_outside_the_shard_are_never_read():
    batch = W.make_custom([900, 2100, 64], H=128, seed=45)
    cuts = page_cuts(batch.seq_lens, 3, np.random.default_rng(45))
    ref = run_shards(batch, cuts)
    T = cuts.shape[1] - 1
    po_ref = ref[0].cpu().numpy().reshape(batch.B, T, -1)
    pl_ref = ref[1].cpu().numpy().reshape(batch.B, T, -1)
    for k in range(T):
        # poison every block-table entry outside shard k, run shard k alone
        bt = np.full_like(batch.block_table, np.iinfo(np.int32).max)
        for b in range(batch.B):
            lo, hi = cuts[b, k] // 64, -(-cuts[b, k + 1] // 64)
            bt[b, lo:hi] = batch.block_table[b, lo:hi]
        db = to_device(batch)
        db.block_table = torch.from_numpy(bt).cuda()
        part_out = torch.zeros((batch.B * T, batch.H, 512), device="cuda")
        part_lse = torch.zeros((batch.B * T, batch.H), device="cuda")
        kb = torch.from_numpy(np.ascontiguousarray(cuts[:, k])).cuda()
        ke = torch.from_numpy(np.ascontiguousarray(cuts[:, k + 1])).cuda()
        B.splash_mla_attend_shard(db.q, db.kv, db.block_table, db.seq_lens, 1, kb, ke, T, k, part_out, part_lse,
                                  db.desc(), db.workspace())
        torch.cuda.synchronize()
        po = part_out.cpu().numpy().reshape(batch.B, T, -1)
        pl = part_lse.cpu().numpy().reshape(batch.B, T, -1)
        assert np.array_equal(po[:, k], po_ref[:, k]) and np.array_equal(pl[:, k], pl_ref[:, k])


def test_debug_check_rejects_bad_key_ranges():
    batch = W.make_custom([300, 400], H=16, seed=46)
    db = to_device(batch)
    part_out = torch.zeros((batch.B, batch.H, 512), device="cuda")
    part_lse = torch.zeros((batch.B, batch.H), device="cuda")
    for kb, ke in [([32, 0], [300, 400]), ([0, 128], [300, 64]), ([-64, 0], [300, 400])]:
        with pytest.raises(B.SplashError):
            B.splash_mla_attend_shard(db.q, db.kv, db.block_table, db.seq_lens, 1,
                                      torch.tensor(kb, dtype=torch.int32, device="cuda"),
                                      torch.tensor(ke, dtype=torch.int32, device="cuda"), 1, 0, part_out, part_lse,
                                      db.desc(B.FLAG_DEBUG_CHECK), db.workspace())
