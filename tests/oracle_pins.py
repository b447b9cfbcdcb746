"""Checks that pin the fp64 oracle to facts that do not come from it.

Each ``pin_*`` function returns the largest deviation it finds (0.0 when the
oracle agrees exactly); the tests assert on it, and the mutation tests use the
same functions to show that a plausible mistake in the oracle fails a pin.
Nothing here imports the HIP path.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
from paper_2609_37626_amd import workloads as W


def dense_to_paged(dense_keys, rng, extra_pages=3):
    """Scatter per-request dense histories ``[s_b, 576]`` (bf16 bits) into a
    randomly permuted 64-row page pool; written independently of the oracle's
    block-table walk.  Unused rows are NaN."""
    pages_per = [(k.shape[0] + 63) // 64 for k in dense_keys]
    num_pages = sum(pages_per) + extra_pages
    perm = rng.permutation(num_pages)
    pool = np.full((num_pages, 64, 576), 0x7FC0, dtype=np.uint16)
    table = np.full((len(dense_keys), max(pages_per)), -1, dtype=np.int32)
    nxt = 0
    for b, keys in enumerate(dense_keys):
        for lp in range(pages_per[b]):
            phys = int(perm[nxt])
            nxt += 1
            table[b, lp] = phys
            rows = keys[lp * 64:(lp + 1) * 64]
            pool[phys, :rows.shape[0]] = rows
    return pool, table


def brute_force(dense_keys, q_bits, q_chunk, sigma):
    """Pure-Python loops over dense, un-paged histories: softmax of sigma*<q,k>
    over the causal prefix, value = first 512 entries of the key row."""
    out, lse = [], []
    H = q_bits.shape[1]
    for b, keys_bits in enumerate(dense_keys):
        keys = [[float(v) for v in row] for row in
                (keys_bits.astype(np.uint32) << 16).view(np.float32)]
        s = len(keys)
        for i in range(q_chunk):
            qrow = (q_bits[b * q_chunk + i].astype(np.uint32) << 16).view(np.float32)
            orow, lrow = [], []
            for h in range(H):
                qv = [float(v) for v in qrow[h]]
                z = [sigma * math.fsum(a * c for a, c in zip(qv, keys[j]))
                     for j in range(s - q_chunk + i + 1)]
                m = max(z)
                tot = math.fsum(math.exp(v - m) for v in z)
                lv = m + math.log(tot)
                w = [math.exp(v - lv) for v in z]
                orow.append([math.fsum(w[j] * keys[j][d] for j in range(len(z)))
                             for d in range(512)])
                lrow.append(lv)
            out.append(orow)
            lse.append(lrow)
    return np.array(out), np.array(lse)


def random_dense_case(seed, B, H, q_chunk, s_max=130):
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(q_chunk, s_max, size=B, endpoint=True)
    dense = [W.f32_to_bf16_bits(rng.standard_normal((int(s), 576), dtype=np.float32))
             for s in lens]
    q_bits = W.f32_to_bf16_bits(rng.standard_normal((B * q_chunk, H, 576), dtype=np.float32))
    pool, table = dense_to_paged(dense, rng)
    return dense, q_bits, pool, table, lens.astype(np.int32)


def pin_brute_force(seed=0, B=3, H=2, q_chunk=3, s_max=130):
    dense, q_bits, pool, table, lens = random_dense_case(seed, B, H, q_chunk, s_max)
    sigma = float(W.SOFTMAX_SCALE)
    ref_out, ref_lse = brute_force(dense, q_bits, q_chunk, sigma)
    out, lse = oracle.mla_attention(q_bits, pool, table, lens, q_chunk, W.SOFTMAX_SCALE)
    return max(np.abs(out - ref_out).max(), np.abs(lse - ref_lse).max())


def pin_sdpa(seed=1, B=3, H=4, q_chunk=4, s_max=300):
    """torch's float64 scaled-dot-product attention on the dense histories,
    with an explicit causal mask: row i sees keys 0..s-q+i."""
    dense, q_bits, pool, table, lens = random_dense_case(seed, B, H, q_chunk, s_max)
    out, _ = oracle.mla_attention(q_bits, pool, table, lens, q_chunk, W.SOFTMAX_SCALE)
    worst = 0.0
    for b, keys_bits in enumerate(dense):
        s = keys_bits.shape[0]
        k = torch.from_numpy((keys_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        qb = q_bits[b * q_chunk:(b + 1) * q_chunk]
        qt = torch.from_numpy((qb.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        qt = qt.permute(1, 0, 2).unsqueeze(0)                    # [1, H, q, 576]
        kt = k.unsqueeze(0).unsqueeze(0).expand(1, H, s, 576)
        vt = k[:, :512].unsqueeze(0).unsqueeze(0).expand(1, H, s, 512)
        rows = torch.arange(q_chunk).unsqueeze(1)
        cols = torch.arange(s).unsqueeze(0)
        mask = cols <= (s - q_chunk + rows)
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=mask, scale=float(W.SOFTMAX_SCALE))
        ref = ref[0].permute(1, 0, 2).numpy()                    # [q, H, 512]
        worst = max(worst, np.abs(out[b * q_chunk:(b + 1) * q_chunk] - ref).max())
    return worst


def _single_request(keys_f32, q_f32, q_chunk=1, sigma=W.SOFTMAX_SCALE, seed=5):
    rng = np.random.Generator(np.random.PCG64(seed))
    kb = W.f32_to_bf16_bits(keys_f32)
    qb = W.f32_to_bf16_bits(q_f32)
    pool, table = dense_to_paged([kb], rng)
    lens = np.array([kb.shape[0]], dtype=np.int32)
    return oracle.mla_attention(qb, pool, table, lens, q_chunk, sigma), kb, qb


def pin_single_key():
    """s = 1: the softmax weight is exactly 1, out = V_0, lse = z_0."""
    rng = np.random.Generator(np.random.PCG64(11))
    keys = rng.standard_normal((1, 576), dtype=np.float32)
    q = rng.standard_normal((1, 3, 576), dtype=np.float32)
    (out, lse), kb, qb = _single_request(keys, q)
    k = (kb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[0]
    qq = (qb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[0]
    z0 = float(np.float32(W.SOFTMAX_SCALE)) * (qq @ k)
    return max(np.abs(out[0] - k[None, :512]).max(), np.abs(lse[0] - z0).max())


def pin_zero_query():
    """Q = 0: all logits equal, lse = ln(p+1), out = mean of the visible V."""
    rng = np.random.Generator(np.random.PCG64(12))
    s, q_chunk = 150, 3
    keys = rng.standard_normal((s, 576), dtype=np.float32)
    q = np.zeros((q_chunk, 2, 576), dtype=np.float32)
    (out, lse), kb, _ = _single_request(keys, q, q_chunk)
    k = (kb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    worst = 0.0
    for i in range(q_chunk):
        p = s - q_chunk + i
        worst = max(worst, np.abs(lse[i] - math.log(p + 1)).max(),
                    np.abs(out[i] - k[:p + 1, :512].mean(axis=0)[None]).max())
    return worst


def pin_shared_rope_distinct_latents():
    """q_nope = 0 and one k_rope for all tokens: equal logits over distinct
    latents, so out = mean of the latents and lse = z + ln(s)."""
    rng = np.random.Generator(np.random.PCG64(13))
    s = 97
    keys = rng.standard_normal((s, 576), dtype=np.float32)
    keys[:, 512:] = rng.standard_normal(64, dtype=np.float32)[None]
    q = rng.standard_normal((1, 2, 576), dtype=np.float32)
    q[:, :, :512] = 0
    (out, lse), kb, qb = _single_request(keys, q)
    k = (kb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    qq = (qb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[0]
    z = float(np.float32(W.SOFTMAX_SCALE)) * (qq[:, 512:] @ k[0, 512:])
    return max(np.abs(out[0] - k[:, :512].mean(axis=0)[None]).max(),
               np.abs(lse[0] - (z + math.log(s))).max())


def pin_one_hot(target=70):
    """A dominant logit on one token: out equals that token's latent."""
    rng = np.random.Generator(np.random.PCG64(14))
    s = 130
    keys = rng.standard_normal((s, 576), dtype=np.float32)
    keys[:, 512:] = 0
    keys[target, 512:] = 8.0
    q = np.zeros((1, 1, 576), dtype=np.float32)
    q[:, :, 512:] = 8.0
    (out, _), kb, _ = _single_request(keys, q)
    k = (kb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.abs(out[0, 0] - k[target, :512]).max()


def pin_probs_sum_to_one(seed=2):
    dense, q_bits, pool, table, lens = random_dense_case(seed, 2, 3, 2)
    _, _, probs = oracle.mla_attention(q_bits, pool, table, lens, 2, W.SOFTMAX_SCALE,
                                       return_probs=True)
    return max(np.abs(P.sum(axis=-1) - 1.0).max() for P in probs.values())


def pin_page_permutation(seed=3):
    """Relabelling physical pages (pool and table together) changes nothing,
    bit for bit."""
    batch = W.make_custom([200, 64, 129], H=4, q_chunk=2, seed=seed, extra_pages=5)
    out, lse = oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens,
                                    2, batch.softmax_scale)
    rng = np.random.Generator(np.random.PCG64(seed + 100))
    perm = rng.permutation(batch.num_pages)
    pool2 = np.empty_like(batch.kv)
    pool2[perm] = batch.kv
    table2 = np.where(batch.block_table >= 0, perm[batch.block_table.clip(0)], -1).astype(np.int32)
    out2, lse2 = oracle.mla_attention(batch.q, pool2, table2, batch.seq_lens, 2, batch.softmax_scale)
    same = np.array_equal(out, out2) and np.array_equal(lse, lse2)
    return 0.0 if same else float("inf")


def pin_chunk_rows_are_decodes(seed=4):
    """Row i of a q-chunk equals a q=1 step over the first s-q+i+1 tokens."""
    q_chunk = 4
    batch = W.make_custom([150, 77], H=3, q_chunk=q_chunk, seed=seed)
    out, lse = oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens,
                                    q_chunk, batch.softmax_scale)
    worst = 0.0
    for b in range(batch.B):
        for i in range(q_chunk):
            n = b * q_chunk + i
            s1 = int(batch.seq_lens[b]) - q_chunk + i + 1
            o1, l1 = oracle.mla_attention(batch.q[n:n + 1], batch.kv, batch.block_table[b:b + 1],
                                          np.array([s1], np.int32), 1, batch.softmax_scale)
            worst = max(worst, np.abs(o1[0] - out[n]).max(), np.abs(l1[0] - lse[n]).max())
    return worst


def pin_head_and_request_partition(seed=6):
    """Heads and requests are independent: computing any subset alone gives
    the same rows (an owner may hold any subset of requests; a head shard
    sees the same history)."""
    batch = W.make_custom([90, 200, 33], H=6, q_chunk=1, seed=seed)
    args = (batch.q, batch.kv, batch.block_table, batch.seq_lens, 1, batch.softmax_scale)
    out, lse = oracle.mla_attention(*args)
    o2, l2 = oracle.mla_attention(*args, requests=[2, 0], heads=[1, 4, 5])
    idx = np.ix_([0, 2], [1, 4, 5])
    return max(np.abs(o2[idx] - out[idx]).max(), np.abs(l2[idx] - lse[idx]).max())


def pin_merge_identity(seed=7, cuts=(0, 37, 64, 65, 190, 300)):
    """Attention over [0,s) equals the merge of attention over a partition of
    [0,s) into ranges (empty ranges included)."""
    q_chunk = 2
    batch = W.make_custom([300], H=3, q_chunk=q_chunk, seed=seed)
    args = (batch.q, batch.kv, batch.block_table, batch.seq_lens, q_chunk, batch.softmax_scale)
    full_o, full_l = oracle.mla_attention(*args)
    parts_o, parts_l = [], []
    bounds = list(cuts) + [300, 300]
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        o, l = oracle.mla_attention(*args, key_ranges=np.array([[lo, hi]]))
        parts_o.append(o)
        parts_l.append(l)
    mo, ml = oracle.merge_partials(np.stack(parts_o), np.stack(parts_l))
    return max(np.abs(mo - full_o).max(), np.abs(ml - full_l).max())


def pin_worked_example(path):
    vals = {}
    for line in open(path):
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = line.split()
            vals[k] = float(v)
    keys = np.zeros((2, 576), dtype=np.float32)
    keys[0, 1] = 0.5
    keys[1, 0] = 0.5
    keys[1, 512] = 1.0
    q = np.zeros((1, 1, 576), dtype=np.float32)
    q[0, 0, 0] = 2.0
    q[0, 0, 512] = 1.0
    (out, lse), _, _ = _single_request(keys, q, sigma=np.float32(1.0))
    expect = np.zeros(512)
    expect[0], expect[1] = vals["out0"], vals["out1"]
    return max(abs(lse[0, 0] - vals["lse"]), np.abs(out[0, 0] - expect).max())


def pin_fp8_dequant(seed=8):
    """fp8 cache: attention equals attention over the exactly dequantised rows
    given as a bf16-free float64 dense history (SDPA cross-check)."""
    batch = W.make_custom([70, 130], H=2, q_chunk=2, kv_dtype=W.KV_FP8_E4M3, seed=seed)
    out, _ = oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens, 2,
                                  batch.softmax_scale, kv_dtype=1, kv_scales=batch.kv_scales)
    tbl = torch.from_numpy(batch.kv.reshape(-1, 576).copy()).view(torch.float8_e4m3fn).to(torch.float64)
    sc = torch.from_numpy(batch.kv_scales.reshape(-1).astype(np.float64))
    worst = 0.0
    for b in range(batch.B):
        s = int(batch.seq_lens[b])
        rows = [int(batch.block_table[b, j // 64]) * 64 + j % 64 for j in range(s)]
        k = tbl[rows] * sc[rows].unsqueeze(1)
        qb = batch.q[b * 2:(b + 1) * 2]
        qt = torch.from_numpy((qb.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        qt = qt.permute(1, 0, 2).unsqueeze(0)
        kt = k.unsqueeze(0).unsqueeze(0).expand(1, 2, s, 576)
        vt = k[:, :512].unsqueeze(0).unsqueeze(0).expand(1, 2, s, 512)
        mask = torch.arange(s).unsqueeze(0) <= (s - 2 + torch.arange(2).unsqueeze(1))
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=mask, scale=float(batch.softmax_scale))[0].permute(1, 0, 2).numpy()
        worst = max(worst, np.abs(out[b * 2:(b + 1) * 2] - ref).max())
    return worst


def pin_latent_rows(seed=13):
    """fp8 latent-row cache: attention equals torch's float64 SDPA over rows
    decoded with torch's own dtypes (float8_e4m3fn codes times the tile's
    float32 scale, bfloat16 RoPE), none of the oracle's decoders involved."""
    batch = W.make_custom([70, 130], H=2, q_chunk=2, kv_dtype=W.KV_FP8_LATENT, seed=seed)
    out, lse = oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens, 2,
                                    batch.softmax_scale, kv_dtype=2)
    raw = torch.from_numpy(batch.kv.reshape(-1, 656).copy())
    codes = raw[:, :512].contiguous().view(torch.float8_e4m3fn).to(torch.float64)
    scales = raw[:, 512:528].contiguous().view(torch.float32).to(torch.float64)       # [rows, 4]
    rope = raw[:, 528:].contiguous().view(torch.bfloat16).to(torch.float64)           # [rows, 64]
    tbl = torch.cat([codes * scales.repeat_interleave(128, dim=1), rope], dim=1)
    worst = 0.0
    for b in range(batch.B):
        s = int(batch.seq_lens[b])
        rows = [int(batch.block_table[b, j // 64]) * 64 + j % 64 for j in range(s)]
        k = tbl[rows]
        qb = batch.q[b * 2:(b + 1) * 2]
        qt = torch.from_numpy((qb.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        qt = qt.permute(1, 0, 2).unsqueeze(0)
        kt = k.unsqueeze(0).unsqueeze(0).expand(1, 2, s, 576)
        vt = k[:, :512].unsqueeze(0).unsqueeze(0).expand(1, 2, s, 512)
        mask = torch.arange(s).unsqueeze(0) <= (s - 2 + torch.arange(2).unsqueeze(1))
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=mask, scale=float(batch.softmax_scale))[0].permute(1, 0, 2).numpy()
        worst = max(worst, np.abs(out[b * 2:(b + 1) * 2] - ref).max())
    return worst


def latent_worked_row():
    """One 656-byte latent row built by hand and its decoded values worked out
    by hand: latent tile t has scale 2, 1/4, 8, 1/64; RoPE is bf16.
    E4M3 codes used: 0x38 = +1.0 (exponent 7 = bias, mantissa 0), 0xB8 = -1.0,
    0x3C = 1.5 (mantissa 4/8), 0x01 = 2^-9 (subnormal 1/8 * 2^-6), 0x7E = 448
    (1.75 * 2^8), 0x00 = 0.  bf16 0x3F80 = 1.0, 0xC040 = -3.0."""
    row = np.zeros(656, dtype=np.uint8)
    row[0], row[1], row[130], row[300], row[511] = 0x38, 0xB8, 0x3C, 0x01, 0x7E
    row[512:528] = np.array([2.0, 0.25, 8.0, 1.0 / 64.0], dtype='<f4').view(np.uint8)
    row[528:530] = [0x80, 0x3F]        # rope[0] = 0x3F80, little-endian
    row[654:656] = [0x40, 0xC0]        # rope[63] = 0xC040
    expect = np.zeros(576)
    expect[0], expect[1] = 2.0, -2.0          # tile 0, scale 2
    expect[130] = 1.5 * 0.25                  # tile 1
    expect[300] = 2.0 ** -9 * 8.0             # tile 2
    expect[511] = 448.0 / 64.0                # tile 3
    expect[512], expect[575] = 1.0, -3.0
    return row, expect


def pin_latent_worked_row():
    row, expect = latent_worked_row()
    return float(np.abs(oracle.ds_rows_to_f64(row[None, :])[0] - expect).max())


def topk_lists(lens, q_chunk, rng, frac=0.4):
    """Distinct visible positions for every row (a random subset, shuffled),
    padded with -1 to a common length; returns idx [N, k] and count [N]."""
    rows = []
    for b, s in enumerate(lens):
        for i in range(q_chunk):
            vis = int(s) - q_chunk + i + 1
            c = max(1, int(round(frac * vis)))
            rows.append(rng.permutation(vis)[:c])
    k = max(len(r) for r in rows)
    idx = np.full((len(rows), k), -1, dtype=np.int32)
    for n, r in enumerate(rows):
        idx[n, :len(r)] = r
    return idx, np.array([len(r) for r in rows], dtype=np.int32)


def pin_topk_sdpa(seed=11, B=3, H=4, q_chunk=3, s_max=300):
    """Top-k rows against torch's float64 scaled-dot-product attention on the
    dense histories with a mask that keeps exactly each row's listed
    positions."""
    dense, q_bits, pool, table, lens = random_dense_case(seed, B, H, q_chunk, s_max)
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    idx, cnt = topk_lists(lens, q_chunk, rng)
    out, lse = oracle.mla_attention_topk(q_bits, pool, table, lens, q_chunk, W.SOFTMAX_SCALE, idx, cnt)
    worst = 0.0
    for b, keys_bits in enumerate(dense):
        s = keys_bits.shape[0]
        k = torch.from_numpy((keys_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
        for i in range(q_chunk):
            n = b * q_chunk + i
            qt = torch.from_numpy((q_bits[n].astype(np.uint32) << 16).view(np.float32).astype(np.float64))
            mask = torch.zeros(s, dtype=torch.bool)
            mask[torch.from_numpy(idx[n, :cnt[n]].astype(np.int64))] = True
            ref = torch.nn.functional.scaled_dot_product_attention(
                qt.unsqueeze(1), k.unsqueeze(0).expand(H, s, 576), k[:, :512].unsqueeze(0).expand(H, s, 512),
                attn_mask=mask.unsqueeze(0).unsqueeze(0).expand(H, 1, s), scale=float(W.SOFTMAX_SCALE))
            worst = max(worst, np.abs(out[n] - ref[:, 0].numpy()).max())
    return worst


def pin_topk_all_positions(seed=12, B=2, H=2, q_chunk=2, s_max=120):
    """Listing every visible position (in shuffled order) is dense attention:
    equal to the pure-Python brute force."""
    dense, q_bits, pool, table, lens = random_dense_case(seed, B, H, q_chunk, s_max)
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    idx, cnt = topk_lists(lens, q_chunk, rng, frac=1.0)
    out, lse = oracle.mla_attention_topk(q_bits, pool, table, lens, q_chunk, W.SOFTMAX_SCALE, idx, cnt)
    ref_out, ref_lse = brute_force(dense, q_bits, q_chunk, float(W.SOFTMAX_SCALE))
    return max(np.abs(out - ref_out).max(), np.abs(lse - ref_lse).max())
