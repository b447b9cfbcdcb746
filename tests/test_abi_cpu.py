"""The C-ABI library without a GPU: it loads, exports every declared entry
point, rejects bad arguments with the documented status before touching the
device, and its host planner produces valid plans."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch  # noqa: F401  (torch's HIP runtime must be loaded before the library)

from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "splash_attn.h")

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="library not built")


def declared_functions(header=None):
    text = open(header or HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(splash_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["splash_mla_attend", "splash_mla_combine", "splash_mla_plan", "splash_mla_run",
                     "splash_mla_workspace_size", "splash_mla_debug_gather", "splash_status_string"]:
        assert required in names


def test_binding_flag_values_match_the_header():
    text = open(HEADER).read()
    values = {m.group(1): int(m.group(2)) for m in re.finditer(r"#define SPLASH_FLAG_(\w+)\s+(\d+)u", text)}
    assert values == {"DEBUG_CHECK": B.FLAG_DEBUG_CHECK, "FORCE_SPLIT": B.FLAG_FORCE_SPLIT,
                      "EXACT_QK": B.FLAG_EXACT_QK}


def test_library_loads_and_exports_every_declared_symbol():
    raw = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(raw, n)]
    assert not missing, missing
    assert B.version().startswith("libsplash_attn")


def test_calib_library_exports_every_declared_symbol():
    from paper_2609_37626_amd import calib
    header = os.path.join(os.path.dirname(HEADER), "splash_calib.h")
    raw = ctypes.CDLL(calib.LIB_PATH)
    names = declared_functions(header)
    assert "splash_calib_stream_read" in names and "splash_calib_mfma_loop" in names
    missing = [n for n in names if not hasattr(raw, n)]
    assert not missing, missing


FAKE = 1 << 20  # 16-byte aligned non-null address that is never dereferenced


def call_attend(desc, q=FAKE, kv=FAKE, bt=FAKE, seq=FAKE, q_chunk=1, out=FAKE, lse=FAKE, ws=FAKE,
                ws_bytes=1 << 30):
    L = B.lib()
    return L.splash_mla_attend(q, kv, bt, seq, q_chunk, out, lse,
                               None if desc is None else ctypes.byref(desc), ws, ws_bytes, None)


def good_desc(**kw):
    d = B.make_desc(4, 16, 8, 24)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("mutate,status", [
    (dict(dim_qk=512), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(dim_v=576), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(page_size=32), B.SPLASH_ERR_UNSUPPORTED),
    (dict(num_heads=8), B.SPLASH_ERR_UNSUPPORTED),
    (dict(num_heads=24), B.SPLASH_ERR_UNSUPPORTED),
    (dict(num_heads=144), B.SPLASH_ERR_UNSUPPORTED),
    (dict(kv_dtype=7), B.SPLASH_ERR_UNSUPPORTED),
    (dict(kv_dtype=B.KV_FP8_E4M3), B.SPLASH_ERR_INVALID_ARGUMENT),   # no scales
    (dict(softmax_scale=float("nan")), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(softmax_scale=0.0), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(max_pages_per_seq=0), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(flags=B.FLAG_FORCE_SPLIT, split_pages=0), B.SPLASH_ERR_INVALID_ARGUMENT),
    (dict(batch=-1), B.SPLASH_ERR_INVALID_ARGUMENT),
])
def test_bad_descriptor_is_rejected(mutate, status):
    assert call_attend(good_desc(**mutate)) == status
    assert B.lib().splash_last_error()


def test_null_descriptor_and_bad_chunk():
    assert call_attend(None) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_attend(good_desc(), q_chunk=0) == B.SPLASH_ERR_INVALID_ARGUMENT


def test_null_and_misaligned_tensors():
    assert call_attend(good_desc(), q=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_attend(good_desc(), out=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_attend(good_desc(), q=FAKE + 8) == B.SPLASH_ERR_MISALIGNED
    assert call_attend(good_desc(), kv=FAKE + 2) == B.SPLASH_ERR_MISALIGNED
    assert call_attend(good_desc(), ws=FAKE + 4) == B.SPLASH_ERR_MISALIGNED


def test_workspace_too_small():
    need = B.workspace_size(4, 1, 16, 1)
    assert need > 0
    base = B.lib().splash_mla_workspace_offsets(4, 1, 16, 0, None)
    assert base > need
    assert call_attend(good_desc(), ws_bytes=64) == B.SPLASH_ERR_WORKSPACE_TOO_SMALL
    # histories longer than one unit's 1024-page cap need room for partials
    d = good_desc(max_pages_per_seq=2048)
    small = B.workspace_size(4, 1, 16, 1)
    assert call_attend(d, ws_bytes=small) == B.SPLASH_ERR_WORKSPACE_TOO_SMALL


def test_idle_owner_is_a_noop_even_with_null_pointers():
    d = good_desc(batch=0)
    assert call_attend(d, q=0, kv=0, bt=0, seq=0, out=0, lse=0, ws=0, ws_bytes=0) == B.SPLASH_OK
    L = B.lib()
    assert L.splash_mla_combine(None, None, None, 0, 1, 16, None, None, None) == B.SPLASH_OK


def test_latent_row_cache_is_accepted_without_scales():
    # the latent-row cache carries its scales in the rows: no kv_scales; an
    # idle owner returns OK through the dense and the top-k entry points
    assert call_attend(good_desc(kv_dtype=B.KV_FP8_LATENT, batch=0), q=0, kv=0, bt=0, seq=0, out=0, lse=0,
                       ws=0, ws_bytes=0) == B.SPLASH_OK
    d = good_desc(kv_dtype=B.KV_FP8_LATENT, batch=0)
    assert B.lib().splash_mla_attend_topk(0, 0, 0, 0, 1, 0, 0, 64, 0, 0, ctypes.byref(d), 0, 0, None) == B.SPLASH_OK


def call_shard(desc, kb=FAKE, ke=FAKE, num_shards=2, shard=0, part_out=FAKE, part_lse=FAKE, ws_bytes=1 << 30):
    L = B.lib()
    return L.splash_mla_attend_shard(FAKE, FAKE, FAKE, FAKE, 1, kb, ke, num_shards, shard, part_out, part_lse,
                                     ctypes.byref(desc), FAKE, ws_bytes, None)


def test_shard_arguments_are_checked_before_the_device():
    assert call_shard(good_desc(), kb=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), ke=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), part_lse=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), shard=2) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), shard=-1) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), num_shards=0, shard=0) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert call_shard(good_desc(), part_out=FAKE + 4) == B.SPLASH_ERR_MISALIGNED
    assert call_shard(good_desc(flags=B.FLAG_FORCE_SPLIT, split_pages=2)) == B.SPLASH_ERR_UNSUPPORTED
    # a partial slot per query row: 4 rows need 4 slots
    assert call_shard(good_desc(), ws_bytes=B.workspace_size(4, 1, 16, 3)) == B.SPLASH_ERR_WORKSPACE_TOO_SMALL
    assert b"partial slot" in B.lib().splash_last_error()
    assert call_shard(good_desc(batch=0), kb=0, ke=0, part_out=0, part_lse=0) == B.SPLASH_OK


def test_dop_regroup_arguments_are_checked_before_the_device():
    L = B.lib()
    assert L.splash_dop_pack_q(None, None, None, 0, 16, None, None) == B.SPLASH_OK          # an idle rank
    assert L.splash_dop_unpack_q(None, 8, 0, 16, None, None) == B.SPLASH_OK                # an idle owner
    assert L.splash_dop_pack_q(FAKE, FAKE, FAKE, -1, 16, FAKE, None) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert L.splash_dop_pack_q(FAKE, FAKE, FAKE, 4, 0, FAKE, None) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert L.splash_dop_pack_q(FAKE, None, FAKE, 4, 16, FAKE, None) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert L.splash_dop_pack_q(FAKE, FAKE + 8, FAKE, 4, 16, FAKE, None) == B.SPLASH_ERR_MISALIGNED
    assert L.splash_dop_unpack_q(FAKE, 0, 4, 16, FAKE, None) == B.SPLASH_ERR_INVALID_ARGUMENT
    assert L.splash_dop_pack_out(FAKE, 8, 1 << 20, 128, FAKE, None) == B.SPLASH_ERR_UNSUPPORTED
    assert L.splash_dop_unpack_out(FAKE, FAKE, 4, 16, FAKE + 2, None) == B.SPLASH_ERR_MISALIGNED


def test_status_strings():
    L = B.lib()
    for st in [0, -1, -2, -3, -4, -5]:
        assert L.splash_status_string(st)


def test_workspace_layout_is_aligned_and_ordered():
    offs, total = B.workspace_offsets(256, 1, 128, 0)
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
    assert total == B.workspace_size(256, 1, 128, 0)
    assert total >= offs[5] + 1024 * 128 * 512 * 4


# ----------------------------------------------------------- host planner ---

def _lengths(cfg):
    spec = W.CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(spec.seed))
    return W.draw_lengths(rng, spec), spec


def check_plan(seq_lens, q_chunk, units, indptr, stats, max_partials):
    T = len(seq_lens) * q_chunk
    covered = {}
    slots = []
    for t, p0, p1, slot in units:
        assert 0 <= p0 < p1 and p1 - p0 <= 1024
        covered.setdefault(int(t), []).append((int(p0), int(p1), int(slot)))
        if slot >= 0:
            slots.append(int(slot))
    for t in range(T):
        b, i = divmod(t, q_chunk)
        pages = -(-(int(seq_lens[b]) - q_chunk + i + 1) // 64)
        segs = sorted(covered[t])
        assert segs[0][0] == 0 and segs[-1][1] == pages
        assert all(a[1] == c[0] for a, c in zip(segs, segs[1:]))   # contiguous, no overlap
        if len(segs) == 1:
            assert segs[0][2] == -1 and indptr[t + 1] == indptr[t]
        else:
            assert sorted(s[2] for s in segs) == list(range(indptr[t], indptr[t + 1]))
    assert len(slots) == len(set(slots)) == stats["partials"] <= max_partials
    assert stats["units"] == len(units)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_host_plan_covers_every_page_once(cfg):
    seq, spec = _lengths(cfg)
    max_pages = int(-(-seq.max() // 64))
    d = B.make_desc(spec.B, spec.H, max_pages, int((-(-seq // 64)).sum()), spec.kv_dtype,
                    kv_scales=None)
    if spec.kv_dtype:
        d.kv_scales = FAKE
    units, indptr, stats = B.splash_mla_plan_host(seq, spec.q_chunk, d, 256, 0)
    check_plan(seq, spec.q_chunk, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)
    if stats["fold"]:
        check_fold(seq, spec.q_chunk, units, stats, 256)
    again = B.splash_mla_plan_host(seq, spec.q_chunk, d, 256, 0)
    assert np.array_equal(units, again[0]) and np.array_equal(indptr, again[1])


def test_host_plan_splits_few_long_and_balances():
    seq, spec = _lengths(3)
    d = B.make_desc(4, 128, 1882, 5640)
    units, _, stats = B.splash_mla_plan_host(seq, 1, d, 256, 0)
    assert stats["units"] >= 128                    # the four histories spread over the workers
    sizes = units[:, 2] - units[:, 1]
    assert sizes.max() <= 1.3 * stats["total_pages"] / 256 + 1


UNIT_X16 = 96   # the planner's fixed cost of a unit, pages * 16


def worker_loads(units, stats):
    ws = stats["worker_start"]
    w = 16 * (units[:, 2] - units[:, 1]).astype(np.int64) + UNIT_X16
    return np.array([w[ws[g]:ws[g + 1]].sum() for g in range(len(ws) - 1)])


def fold_makespan(pages, cap, G):
    """The busiest worker of a fold with this cap, from its definition: ranks
    by pages (longest first), the j-th longest tile above the cap hands its
    tail to worker G-1-j."""
    q = sorted(pages, reverse=True) + [0] * (G - len(pages))
    loads = [16 * x + UNIT_X16 if x > 0 else 0 for x in q]
    for j in range(G):
        if q[j] <= cap:
            break
        loads[j] = 16 * cap + UNIT_X16
        loads[G - 1 - j] += 16 * (q[j] - cap) + UNIT_X16
    return max(loads)


def check_fold(seq_lens, q_chunk, units, stats, G):
    ws = stats["worker_start"]
    assert stats["fold"] and stats["chunk_pages"] == 0 and len(ws) == G + 1
    assert ws[0] == 0 and ws[-1] == stats["units"] and np.all(np.diff(ws) >= 0)
    # a worker runs at most its own tile and one tail; split tiles have two
    # parts: the head [0, cap) and the tail [cap, P)
    assert np.diff(ws).max() <= 2 and stats["max_parts"] <= 2
    split = units[units[:, 3] >= 0]
    assert np.all((split[:, 1] == 0) & (split[:, 2] == stats["cap"]) | (split[:, 1] == stats["cap"]))
    pages = [-(-(int(seq_lens[t // q_chunk]) - q_chunk + t % q_chunk + 1) // 64) for t in range(len(seq_lens) * q_chunk)]
    loads = worker_loads(units, stats)
    assert loads.max() == fold_makespan(pages, stats["cap"], G)
    return loads


def test_host_plan_folds_many_short_requests():
    # one short history per worker, 16-64 pages: one unit each would leave
    # the busiest worker with 64 pages while the mean is 41, so the longest
    # histories keep a head of `cap` pages and hand their tails to the
    # workers with the shortest ones
    seq, spec = _lengths(2)
    d = B.make_desc(256, 128, 64, int((-(-seq // 64)).sum()))
    units, indptr, stats = B.splash_mla_plan_host(seq, 1, d, 256, 0)
    check_plan(seq, 1, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)
    loads = check_fold(seq, 1, units, stats, 256)
    assert loads.max() < 0.8 * (16 * 64 + UNIT_X16)
    assert stats["partials"] < 256


def test_host_plan_equal_tiles_stay_whole():
    # equal histories, one per worker: nothing to balance, no partials
    seq = np.full(256, 640, np.int32)
    d = B.make_desc(256, 128, 10, 2560)
    units, indptr, stats = B.splash_mla_plan_host(seq, 1, d, 256, 0)
    check_plan(seq, 1, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)
    assert stats["partials"] == 0 and stats["units"] == 256


def test_host_plan_fold_random_shapes():
    # Random batches of at most one tile per worker: whenever the fold plan is
    # taken it covers every page once, keeps runs of at most two units, and
    # its busiest worker is the definition's makespan, no worse than one unit
    # per tile.
    rng = np.random.default_rng(7)
    seen = 0
    for trial in range(300):
        G = int(rng.integers(2, 300))
        qc = int(rng.choice([1, 1, 2, 4]))
        Bn = max(1, int(rng.integers(1, G + 1)) // qc)
        seq = rng.integers(qc, 64 * 200, size=Bn).astype(np.int32)
        d = B.make_desc(Bn, 128, int(-(-seq.max() // 64)), int((-(-seq // 64)).sum()) + 1)
        units, indptr, stats = B.splash_mla_plan_host(seq, qc, d, G, 0)
        check_plan(seq, qc, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)
        if not stats["fold"]:
            continue
        seen += 1
        loads = check_fold(seq, qc, units, stats, G)
        pages = [-(-(int(seq[t // qc]) - qc + t % qc + 1) // 64) for t in range(Bn * qc)]
        assert loads.max() <= 16 * max(pages) + UNIT_X16
    assert seen > 50


def test_host_plan_respects_partial_capacity_and_forced_split():
    seq, spec = _lengths(3)
    d = B.make_desc(4, 128, 1882, 5640)
    units, _, stats = B.splash_mla_plan_host(seq, 1, d, 256, 16)
    assert stats["partials"] <= 16
    d.flags, d.split_pages = B.FLAG_FORCE_SPLIT, 100
    units, indptr, stats = B.splash_mla_plan_host(seq, 1, d, 256, 0)
    assert stats["chunk_pages"] == 100
    check_plan(seq, 1, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)


def test_host_plan_single_short_request_is_one_unit():
    d = B.make_desc(1, 16, 1, 1)
    units, indptr, stats = B.splash_mla_plan_host(np.array([1], np.int32), 1, d, 256, 0)
    assert units.tolist() == [[0, 0, 1, -1]] and indptr.tolist() == [0, 0]


@pytest.mark.parametrize("cfg,split", [(2, 0), (4, 0), (5, 0), (4, 20), (5, 64), (2, 64)])
def test_host_plan_queue_order(cfg, split):
    # A fold plan lists units worker by worker (each worker runs its own).  A
    # plan of one unit size puts its units in a queue the persistent workers
    # draw from: with more units than workers the longest go first (ties in
    # tile order), which packs them like a longest-processing-time-first
    # schedule; with at most one unit per worker every unit starts at once
    # and the queue stays in tile order.  A forced unit size always makes the
    # second kind.
    seq, spec = _lengths(cfg)
    d = B.make_desc(spec.B, spec.H, int(-(-seq.max() // 64)), int((-(-seq // 64)).sum()), spec.kv_dtype)
    if spec.kv_dtype:
        d.kv_scales = FAKE
    if split:
        d.flags, d.split_pages = B.FLAG_FORCE_SPLIT, split
    units, indptr, stats = B.splash_mla_plan_host(seq, spec.q_chunk, d, 256, 0)
    key = units[:, 0].astype(np.int64) * (1 << 32) + units[:, 1]
    ln = units[:, 2] - units[:, 1]
    assert stats["fold"] == (cfg == 2 and split == 0)
    if stats["fold"]:
        check_fold(seq, spec.q_chunk, units, stats, 256)
    elif stats["units"] > 256 and spec.q_chunk == 1:
        assert np.all(ln[:-1] >= ln[1:])
        same = ln[:-1] == ln[1:]
        assert np.all(key[:-1][same] < key[1:][same])
    elif stats["units"] > 256:
        # query chunks: whole requests, longest unit first (ties in request
        # order), each request's units unit index major so that the rows of
        # one page range sit side by side
        req = units[:, 0] // spec.q_chunk
        starts = np.flatnonzero(np.r_[True, req[1:] != req[:-1]])
        assert len(starts) == len(np.unique(req))
        ends = np.r_[starts[1:], len(units)]
        keys = np.array([ln[a:b].max() for a, b in zip(starts, ends)])
        assert np.all(keys[:-1] >= keys[1:])
        assert np.all(req[starts][:-1][keys[:-1] == keys[1:]] < req[starts][1:][keys[:-1] == keys[1:]])
        for a, b in zip(starts, ends):
            blk = units[a:b]
            for i in range(1, len(blk)):
                if blk[i, 0] == blk[i - 1, 0]:
                    continue
                # a new row: its unit starts where the previous row's unit of
                # the same index would (same unit index, next row)
                assert blk[i, 0] > blk[i - 1, 0] or blk[i, 1] >= blk[i - 1, 1]
    else:
        assert np.all(key[:-1] < key[1:])
    check_plan(seq, spec.q_chunk, units, indptr, stats, B.DEFAULT_MAX_PARTIALS)


def test_noalloc_refusals_happen_on_the_host():
    """splash_mla_attend_noalloc refuses a batch whose minimum workspace
    exceeds its scratch, and DEBUG_CHECK, before any HIP call; an empty
    batch is a no-op."""
    L = B.lib()

    def call(desc):
        return L.splash_mla_attend_noalloc(FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, ctypes.byref(desc), None)

    # 600 histories of up to 2000 pages force 1200 partials of 256 KB each
    assert call(B.make_desc(600, 128, 2000, 1 << 20)) == B.SPLASH_ERR_WORKSPACE_TOO_SMALL
    assert "scratch holds" in L.splash_last_error().decode()
    assert call(B.make_desc(4, 16, 8, 24, flags=B.FLAG_DEBUG_CHECK)) == B.SPLASH_ERR_UNSUPPORTED
    assert call(B.make_desc(0, 16, 8, 24)) == B.SPLASH_OK
    assert B.NOALLOC_SCRATCH_BYTES == 128 << 20
