"""Owner-local absorbed-MLA attention over a paged latent cache, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition followed (Sec. 3 "DOP: Computation"; Sec. 3 "Cost"; App. B;
Sec. 4.1 "Handoff"), for request b with history length s_b (which includes
the current chunk of q rows, 1 <= q <= s_b), chunk row i in [0, q), head h,
and output row n = b*q + i:

  position        p = s_b - q + i
  visible keys    j = 0 .. p                      (complete causal prefix)
  physical row    phys(b, j) = block_table[b, j // 64] * 64 + j % 64
  key row         K_j = decode(pool row phys(b, j))            (576 wide)
                  (fp8 cache: K_j = e4m3(code) * scale[phys(b, j)];
                  latent-row cache: each 128-column latent tile has its
                  own scale and the RoPE part is bf16, see formats)
  value row       V_j = K_j[0:512]                  (the latent; d_z = d_c)
  logit           z_j = sigma * <Q[n, h, :], K_j>   (sigma: the fp32 scale)
  log-sum-exp     lse = M + ln sum_j exp(z_j - M),  M = max_j z_j
  output          out[n, h, :] = sum_j exp(z_j - lse) * V_j

The latent row has no head axis, so one gathered K serves every head.
"""
from __future__ import annotations

import numpy as np

from .formats import bf16_bits_to_f64, ds_rows_to_f64, e4m3_bits_to_f64

PAGE = 64
DIM_V = 512


def gather_history(kv, kv_scales, block_table, b, n_keys, kv_dtype):
    """Rows 0..n_keys-1 of request b's history, decoded to float64 [n_keys, 576].

    Walks the block table: token j lives in logical page j // 64 at offset
    j % 64; the table maps the logical page to a physical page of the pool.
    """
    j = np.arange(n_keys, dtype=np.int64)
    pages = block_table[b, j // PAGE].astype(np.int64)
    phys = pages * PAGE + j % PAGE
    flat = kv.reshape(-1, kv.shape[-1])
    rows = flat[phys]
    if kv_dtype == 0:
        return bf16_bits_to_f64(rows)
    if kv_dtype == 2:
        return ds_rows_to_f64(rows)
    vals = e4m3_bits_to_f64(rows)
    scales = kv_scales.reshape(-1).astype(np.float64)[phys]
    return vals * scales[:, None]


def attention_rows(Q, K, sigma, key_hi, key_lo=None, return_probs=False):
    """Softmax attention of query rows over one request's gathered keys.

    Q: [R, H, 576] float64; K: [n, 576] float64; row r sees keys
    key_lo[r] <= j < key_hi[r] (key_lo defaults to 0).  A row that sees no
    key gets lse = -inf and out = 0 (its weight in a merge is zero).
    Returns out [R, H, 512], lse [R, H] (and P [R, H, n] if asked).
    """
    R, H, _ = Q.shape
    n = K.shape[0]
    if key_lo is None:
        key_lo = np.zeros(R, dtype=np.int64)
    Z = sigma * (Q.reshape(R * H, -1) @ K.T).reshape(R, H, n)
    j = np.arange(n)
    visible = (j[None, :] >= np.asarray(key_lo)[:, None]) & (j[None, :] < np.asarray(key_hi)[:, None])
    Z = np.where(visible[:, None, :], Z, -np.inf)
    M = Z.max(axis=2, initial=-np.inf)
    empty = ~np.isfinite(M)
    M_safe = np.where(empty, 0.0, M)
    E = np.exp(Z - M_safe[:, :, None])
    lse = np.where(empty, -np.inf, M_safe + np.log(np.where(empty, 1.0, E.sum(axis=2))))
    P = np.where(empty[:, :, None], 0.0, np.exp(Z - np.where(empty, 0.0, lse)[:, :, None]))
    out = (P.reshape(R * H, n) @ K[:, :DIM_V]).reshape(R, H, DIM_V)
    if return_probs:
        return out, lse, P
    return out, lse


def _sigma(softmax_scale):
    return float(np.float32(softmax_scale))


def mla_attention(q, kv, block_table, seq_lens, q_chunk, softmax_scale,
                  kv_dtype=0, kv_scales=None, requests=None, heads=None,
                  key_ranges=None, return_probs=False):
    """Reference result for a whole batch (or a subset of requests / heads).

    q: uint16 bf16 bits [B*q_chunk, H, 576]; kv: uint16 [num_pages, 64, 576]
    (bf16) or uint8 (e4m3) with kv_scales float32 [num_pages, 64], or
    (kv_dtype 2) uint8 latent-format rows [num_pages, 64, 656].
    ``key_ranges``: optional int array [B, 2]; restricts request b to keys
    [lo, hi) intersected with each row's causal prefix (a partial result over
    a slice of the history, as one split or one position shard computes).
    Returns float64 out [B*q, H, 512] and lse [B*q, H]; rows and heads that
    were not evaluated hold NaN.  With return_probs, also a dict b -> P.
    """
    B = int(len(seq_lens))
    H = q.shape[1]
    sigma = _sigma(softmax_scale)
    heads = np.arange(H) if heads is None else np.asarray(heads)
    requests = range(B) if requests is None else requests
    out = np.full((B * q_chunk, H, DIM_V), np.nan)
    lse = np.full((B * q_chunk, H), np.nan)
    probs = {}
    for b in requests:
        s = int(seq_lens[b])
        K = gather_history(kv, kv_scales, block_table, b, s, kv_dtype)
        rows = slice(b * q_chunk, (b + 1) * q_chunk)
        Q = bf16_bits_to_f64(q[rows][:, heads, :])
        hi = s - q_chunk + np.arange(q_chunk) + 1
        lo = np.zeros(q_chunk, dtype=np.int64)
        if key_ranges is not None:
            lo = np.maximum(lo, int(key_ranges[b][0]))
            hi = np.minimum(hi, int(key_ranges[b][1]))
        res = attention_rows(Q, K, sigma, hi, lo, return_probs)
        idx = np.ix_(np.arange(rows.start, rows.stop), heads)
        out[idx] = res[0]
        lse[idx] = res[1]
        if return_probs:
            probs[b] = res[2]
    if return_probs:
        return out, lse, probs
    return out, lse


def mla_attention_sampled(q, kv, block_table, seq_lens, q_chunk, softmax_scale,
                          samples, kv_dtype=0, kv_scales=None):
    """Reference values for a list of (request b, chunk row i, head h) triples.

    Each sample is evaluated on its own from the definition, so full-size
    batches can be checked one output row at a time.  Returns out [S, 512],
    lse [S].
    """
    sigma = _sigma(softmax_scale)
    outs = np.empty((len(samples), DIM_V))
    lses = np.empty(len(samples))
    cache = {}
    for k, (b, i, h) in enumerate(samples):
        s = int(seq_lens[b])
        if b not in cache:
            cache.clear()
            cache[b] = gather_history(kv, kv_scales, block_table, b, s, kv_dtype)
        K = cache[b]
        n = b * q_chunk + i
        Q = bf16_bits_to_f64(q[n, h][None, None, :])
        o, l = attention_rows(Q, K, sigma, np.array([s - q_chunk + i + 1]))
        outs[k] = o[0, 0]
        lses[k] = l[0, 0]
    return outs, lses


def gather_positions(kv, kv_scales, block_table, b, positions, kv_dtype):
    """Rows of request b's history at the given token positions, decoded to
    float64 [len(positions), 576] (the same block-table walk as
    gather_history, for an arbitrary list of positions)."""
    j = np.asarray(positions, dtype=np.int64)
    phys = block_table[b, j // PAGE].astype(np.int64) * PAGE + j % PAGE
    rows = kv.reshape(-1, kv.shape[-1])[phys]
    if kv_dtype == 0:
        return bf16_bits_to_f64(rows)
    if kv_dtype == 2:
        return ds_rows_to_f64(rows)
    return e4m3_bits_to_f64(rows) * kv_scales.reshape(-1).astype(np.float64)[phys][:, None]


def mla_attention_topk(q, kv, block_table, seq_lens, q_chunk, softmax_scale, topk_idx, topk_count,
                       kv_dtype=0, kv_scales=None):
    """Top-k (sparse) attention: row n = b*q_chunk + i attends only the token
    positions topk_idx[n, :topk_count[n]] of request b's history (each within
    its causal prefix), with the same logits, values and log-sum-exp as the
    dense definition.  Every listed position is one key (a position listed
    twice would count twice); a row with an empty list gets out = 0, lse =
    -inf.  Returns float64 out [B*q, H, 512] and lse [B*q, H]."""
    H = q.shape[1]
    sigma = _sigma(softmax_scale)
    N = int(len(seq_lens)) * q_chunk
    out = np.zeros((N, H, DIM_V))
    lse = np.full((N, H), -np.inf)
    for n in range(N):
        b = n // q_chunk
        c = int(topk_count[n])
        K = gather_positions(kv, kv_scales, block_table, b, topk_idx[n, :c], kv_dtype)
        Q = bf16_bits_to_f64(q[n:n + 1])
        o, l = attention_rows(Q, K, sigma, np.array([c]))
        out[n], lse[n] = o[0], l[0]
    return out, lse


def merge_partials(parts_out, parts_lse):
    """Merge attention over disjoint key sets into attention over their union.

    parts_out: [S, ..., 512] normalised partial outputs; parts_lse: [S, ...].
    With L = ln sum_s exp(lse_s), out = sum_s exp(lse_s - L) * out_s.  Parts
    with lse = -inf (no visible key) weigh zero; if every part is empty the
    merge is empty too (lse = -inf, out = 0).  This is the merge a
    position-sharded history needs (App. E, position-sharded CP).
    """
    parts_out = np.asarray(parts_out, dtype=np.float64)
    parts_lse = np.asarray(parts_lse, dtype=np.float64)
    M = parts_lse.max(axis=0)
    empty = ~np.isfinite(M)
    M_safe = np.where(empty, 0.0, M)
    w = np.exp(parts_lse - M_safe[None])
    tot = w.sum(axis=0)
    L = np.where(empty, -np.inf, M_safe + np.log(np.where(empty, 1.0, tot)))
    wn = np.where(empty[None], 0.0, np.exp(parts_lse - np.where(empty, 0.0, L)[None]))
    out = (wn[..., None] * parts_out).sum(axis=0)
    return out, L
