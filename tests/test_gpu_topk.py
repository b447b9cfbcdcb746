"""GPU parity of the top-k (sparse) variant (splash_mla_attend_topk) against
the oracle's top-k definition, at the parity bar's tolerances (outputs
max-abs 1e-2 bf16 / 3e-2 fp8, LSE 1e-3).  Rows with an empty list must come
back as exactly out = 0, lse = -inf."""
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


def lists(batch, k, rng, empty_rows=(), recent=0):
    """Per row: up to k distinct visible positions (the `recent` last ones
    always, the rest a random subset), shuffled; -1 padding."""
    N = batch.B * batch.q_chunk
    idx = np.full((N, k), -1, dtype=np.int32)
    cnt = np.zeros(N, dtype=np.int32)
    for n in range(N):
        if n in empty_rows:
            continue
        b, i = divmod(n, batch.q_chunk)
        vis = int(batch.seq_lens[b]) - batch.q_chunk + i + 1
        c = min(k, vis)
        keep = np.arange(max(0, vis - recent), vis)
        rest = rng.permutation(max(0, vis - recent))[:max(0, c - len(keep))]
        sel = rng.permutation(np.concatenate([keep, rest]))[:c]
        idx[n, :len(sel)] = sel
        cnt[n] = len(sel)
    return idx, cnt


def run_topk(batch, idx, cnt, flags=0, split_pages=0):
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    B.splash_mla_attend_topk(db.q, db.kv, db.block_table, db.seq_lens, batch.q_chunk,
                             torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), out, lse,
                             db.desc(flags, split_pages), db.workspace())
    torch.cuda.synchronize()
    return out, lse


def check(batch, idx, cnt, out, lse, label):
    ref_o, ref_l = oracle.mla_attention_topk(batch.q, batch.kv, batch.block_table, batch.seq_lens, batch.q_chunk,
                                             batch.softmax_scale, idx, cnt, kv_dtype=batch.kv_dtype,
                                             kv_scales=batch.kv_scales)
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    empty = cnt == 0
    assert np.all(o[empty] == 0.0) and np.all(np.isneginf(l[empty])), label
    err_o = np.abs(o[~empty] - ref_o[~empty]).max()
    err_l = np.abs(l[~empty] - ref_l[~empty]).max()
    print(f"{label}: out max-abs {err_o:.3e}  lse {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[batch.kv_dtype] and err_l <= LSE_TOL, (label, err_o, err_l)


@pytest.mark.parametrize("k", [1, 31, 64, 100, 512, 2048, 3000])
def test_topk_ragged_bf16(k):
    lens = np.random.Generator(np.random.PCG64(50 + k)).integers(1, 4000, size=12, endpoint=True)
    batch = W.make_custom(lens, H=128, seed=50)
    idx, cnt = lists(batch, k, np.random.default_rng(k), empty_rows=(3,), recent=16)
    print(f"k={k} counts {cnt.tolist()}", flush=True)
    out, lse = run_topk(batch, idx, cnt)
    check(batch, idx, cnt, out, lse, f"bf16 k={k}")


def test_topk_chunk8_fp8():
    batch = W.make_custom([900, 2500, 5000], H=128, q_chunk=8, kv_dtype=W.KV_FP8_E4M3, seed=51)
    idx, cnt = lists(batch, 1500, np.random.default_rng(51), recent=64)
    out, lse = run_topk(batch, idx, cnt)
    check(batch, idx, cnt, out, lse, "fp8 q=8 k=1500")


def test_topk_forced_small_units_and_heads64():
    batch = W.make_custom([3000, 1200], H=64, seed=52)
    idx, cnt = lists(batch, 700, np.random.default_rng(52))
    out, lse = run_topk(batch, idx, cnt, flags=B.FLAG_FORCE_SPLIT, split_pages=2)
    check(batch, idx, cnt, out, lse, "forced 2-group units")


def test_topk_pages_not_listed_are_never_read():
    # poison every block-table entry whose page holds no listed position
    batch = W.make_custom([2000, 3000], H=128, seed=53)
    idx, cnt = lists(batch, 300, np.random.default_rng(53))
    ref = run_topk(batch, idx, cnt)
    bt = np.full_like(batch.block_table, np.iinfo(np.int32).max)
    for n in range(len(cnt)):
        pages = np.unique(idx[n, :cnt[n]] // 64)
        bt[n, pages] = batch.block_table[n, pages]
    db = to_device(batch)
    db.block_table = torch.from_numpy(bt).cuda()
    out, lse = db.alloc_outputs()
    B.splash_mla_attend_topk(db.q, db.kv, db.block_table, db.seq_lens, 1, torch.from_numpy(idx).cuda(),
                             torch.from_numpy(cnt).cuda(), out, lse, db.desc(), db.workspace())
    torch.cuda.synchronize()
    assert torch.equal(out, ref[0]) and torch.equal(lse, ref[1])


def test_topk_debug_check_rejects_bad_lists():
    batch = W.make_custom([300, 400], H=16, seed=54)
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    good = np.array([[0, 5, 299], [1, 2, 399]], dtype=np.int32)
    for idx, cnt in [(good.copy(), [3, 4]), (np.array([[0, 5, 300], [1, 2, 3]], np.int32), [3, 3]),
                     (np.array([[0, -2, 3], [1, 2, 3]], np.int32), [3, 3])]:
        with pytest.raises(B.SplashError):
            B.splash_mla_attend_topk(db.q, db.kv, db.block_table, db.seq_lens, 1, torch.from_numpy(idx).cuda(),
                                     torch.tensor(cnt, dtype=torch.int32, device="cuda"), out, lse,
                                     db.desc(B.FLAG_DEBUG_CHECK), db.workspace())
