"""Graph capture of the step's calls (Sec. 4.1, "3. Handoff": graphs are
captured once at startup; App. E: captured graphs bind buffer addresses).

splash_mla_attend (plan, attend, combine) and the plan-once pair
splash_mla_plan + splash_mla_run only enqueue kernels on the caller's stream:
no allocation, no host synchronisation, no memset.  A captured graph is
replayed with new contents written into the same buffers (queries, cache
pages, block table, lengths); every replay is compared bit for bit with an
eager call on the same contents, with eager work and synchronisations in
between, and with the fp64 oracle at the parity bar.
"""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W
from paper_2609_37626_amd.device import to_device
from tests.test_gpu_parity import assert_parity, run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def new_contents(base: W.Batch, seed: int, keep_lengths: bool) -> W.Batch:
    """Fresh queries and cache rows, the pool's pages permuted in the block
    table, and (unless keep_lengths) shorter or equal lengths: everything
    fits the buffers of `base`."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if base.kv_dtype == W.KV_BF16:
        kv = W.f32_to_bf16_bits(rng.standard_normal(base.kv.shape, dtype=np.float32))
        scales = None
    else:
        flat = rng.standard_normal((base.kv.shape[0] * base.kv.shape[1], 576), dtype=np.float32)
        codes, sc = W.encode_e4m3_per_token(flat)
        kv = codes.reshape(base.kv.shape)
        scales = sc.reshape(base.kv_scales.shape).astype(np.float32)
    q = W.f32_to_bf16_bits(rng.standard_normal(base.q.shape, dtype=np.float32))
    perm = rng.permutation(base.kv.shape[0]).astype(np.int32)
    bt = np.where(base.block_table >= 0, perm[np.maximum(base.block_table, 0)], base.block_table).astype(np.int32)
    lens = base.seq_lens.copy()
    if not keep_lengths:
        lens = np.maximum(base.q_chunk, rng.integers(1, base.seq_lens, endpoint=True)).astype(np.int32)
    return dataclasses.replace(base, q=q, kv=kv, kv_scales=scales, block_table=bt, seq_lens=lens)


def write_into(db, batch: W.Batch) -> None:
    """Copy a host batch into the existing device buffers (same addresses)."""
    src = to_device(batch)
    for name in ("q", "kv", "block_table", "seq_lens"):
        getattr(db, name).copy_(getattr(src, name))
    if db.kv_scales is not None:
        db.kv_scales.copy_(src.kv_scales)


def bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy().view(np.int32)


CASES = {
    # splits and a combine in every replay (lengths change, so does the plan)
    "bf16_q1_B5": lambda: W.make_custom([3000, 9000, 65, 1, 4500], H=128, seed=71),
    "fp8_q4_B3": lambda: W.make_custom([700, 2600, 9], H=128, q_chunk=4, kv_dtype=W.KV_FP8_E4M3, seed=72),
    # one tile per worker or fewer: a fold plan in the first replays
    "bf16_fold_B40": lambda: W.make_custom(
        np.random.Generator(np.random.PCG64(73)).integers(100, 2500, size=40, endpoint=True), H=128, seed=73),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_captured_attend_replays_new_contents(name):
    base = CASES[name]()
    db = to_device(base)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc()
    side = torch.cuda.Stream()

    def call():
        B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, desc, ws)

    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()  # warm-up outside the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        call()
    torch.cuda.synchronize()

    for rep, seed in enumerate([101, 102, 103, 104]):
        batch = new_contents(base, seed, keep_lengths=(rep == 0))
        write_into(db, batch)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        g_out, g_lse = bits(out), bits(lse)
        out.fill_(0)
        lse.fill_(0)
        call()  # eager, same contents and buffers
        torch.cuda.synchronize()
        assert np.array_equal(g_out, bits(out)) and np.array_equal(g_lse, bits(lse)), (name, rep)
        assert_parity(batch, out, lse, label=f"{name} replay {rep}")


def test_captured_plan_once_run_replays():
    """The plan is made once (eagerly) for fixed lengths; splash_mla_run is
    captured and replayed over new queries and cache contents."""
    base = W.make_custom([5000, 700, 12000, 64], H=128, seed=74)
    db = to_device(base)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc()
    B.splash_mla_plan(db.seq_lens, db.q_chunk, desc, ws)
    side = torch.cuda.Stream()

    def run():
        B.splash_mla_run(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, desc, ws)

    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        run()
    torch.cuda.synchronize()
    for rep, seed in enumerate([111, 112, 113]):
        batch = new_contents(base, seed, keep_lengths=True)
        write_into(db, batch)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        g_out, g_lse = bits(out), bits(lse)
        run()
        torch.cuda.synchronize()
        assert np.array_equal(g_out, bits(out)) and np.array_equal(g_lse, bits(lse)), rep
        assert_parity(batch, out, lse, label=f"plan once, run replay {rep}")
