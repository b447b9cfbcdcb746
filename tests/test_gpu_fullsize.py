"""GPU parity at the benchmark workloads' full sizes.

Each of the four benchmark workloads (many short, few long, ragged, chunk +
fp8) runs through splash_mla_attend exactly as the benchmark launches it
(device planner, persistent attend kernel, combine).  The fp64 oracle then
evaluates sampled output rows one at a time from the definition: the longest
and the shortest history, histories that were split across units, and random
others, at the first, a middle and the last head, and (for the chunked
workload) the first and last rows of the chunk.  Tolerances are those of the
small parity cases.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W
from paper_2609_37626_amd.device import to_device

pytestmark = pytest.mark.gpu

OUT_TOL = {W.KV_BF16: 1e-2, W.KV_FP8_E4M3: 3e-2}
LSE_TOL = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def pick_samples(batch, rng, n_requests=12):
    seq = batch.seq_lens
    order = np.argsort(seq, kind="stable")
    chosen = [int(order[-1]), int(order[0])]
    others = rng.choice(batch.B, size=min(batch.B, n_requests), replace=False)
    for b in others:
        if int(b) not in chosen:
            chosen.append(int(b))
    rows = sorted({0, batch.q_chunk - 1, batch.q_chunk // 2})
    heads = sorted({0, batch.H // 2, batch.H - 1})
    return [(b, i, h) for b in sorted(chosen) for i in rows for h in heads]


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_full_size_workload_sampled_rows(cfg):
    batch = W.make_config(cfg)
    print(f"config {cfg}: {W.CONFIGS[cfg].name}, sum s = {int(batch.seq_lens.sum())}", flush=True)
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc()
    B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, desc, ws)
    torch.cuda.synchronize()
    offs, _ = B.workspace_offsets(batch.B, batch.q_chunk, batch.H, 0)
    hdr = ws[offs[0]:offs[0] + 32].cpu().numpy().view(np.int32)
    print(f"  plan: {int(hdr[1])} units, {int(hdr[2])} partials, {int(hdr[6])} split tiles", flush=True)
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
    samples = pick_samples(batch, np.random.Generator(np.random.PCG64(100 + cfg)))
    ref_o, ref_l = oracle.mla_attention_sampled(batch.q, batch.kv, batch.block_table, batch.seq_lens,
                                                batch.q_chunk, batch.softmax_scale, samples,
                                                kv_dtype=batch.kv_dtype, kv_scales=batch.kv_scales)
    got_o = np.stack([o[b * batch.q_chunk + i, h] for b, i, h in samples])
    got_l = np.array([l[b * batch.q_chunk + i, h] for b, i, h in samples])
    err_o = np.abs(got_o - ref_o).max()
    err_l = np.abs(got_l - ref_l).max()
    print(f"  {len(samples)} sampled rows: out max-abs {err_o:.3e}  lse max-abs {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[batch.kv_dtype]
    assert err_l <= LSE_TOL


def test_single_history_of_524288_tokens():
    """One request of 524,288 keys (8,192 pages: twice the paper's 256K
    evaluation context, App. C), decode, 128 heads: the history is cut into
    many units and their partials combined.  Sampled heads against the
    oracle evaluated from the definition."""
    batch = W.make_custom([524288], H=128, seed=91)
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, 1, out, lse, db.desc(), ws)
    torch.cuda.synchronize()
    offs, _ = B.workspace_offsets(1, 1, 128, 0)
    hdr = ws[offs[0]:offs[0] + 32].cpu().numpy().view(np.int32)
    print(f"  plan: {int(hdr[1])} units, {int(hdr[2])} partials", flush=True)
    assert int(hdr[2]) > 8   # more than a unit may hold: split
    o = out.float().cpu().numpy()
    l = lse.cpu().numpy()
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(l))
    samples = [(0, 0, h) for h in (0, 1, 31, 64, 100, 127)]
    ref_o, ref_l = oracle.mla_attention_sampled(batch.q, batch.kv, batch.block_table, batch.seq_lens, 1,
                                                batch.softmax_scale, samples)
    got_o = np.stack([o[0, h] for _, _, h in samples])
    got_l = np.array([l[0, h] for _, _, h in samples])
    err_o, err_l = np.abs(got_o - ref_o).max(), np.abs(got_l - ref_l).max()
    print(f"  524288 keys, {len(samples)} heads: out max-abs {err_o:.3e}  lse max-abs {err_l:.3e}", flush=True)
    assert err_o <= OUT_TOL[W.KV_BF16] and err_l <= LSE_TOL
