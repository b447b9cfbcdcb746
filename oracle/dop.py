"""DOP regrouping of query and output rows, written out from its definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3 "DOP: Computation": with sharded projections, rank t of T holds all N
current query rows for its H/T heads, [N, H/T, d_q] (global row, local head).
Attention at an owner needs its own N_o rows for all H heads, [N_o, H, d_q]
(owner row, all heads).  A variable-size all-to-all converts between the
two before attention, and a reverse one returns [N_o, H, d_z] to the ranks'
[N, H/T, d_z] afterwards.  The transfer keeps row identity, head order and
positions, packs the no-position and rotary query parts together, and uses
per-owner row counts as split sizes (App. E, DOP transfer).  Each exchange
moves the blocks between different ranks; Sec. 3 "Cost" gives their total,
V_DOP = (1 - 1/T) N H (d_q + d_z) b.

Here rank t's heads are [t H/T, (t+1) H/T) and the rows an owner receives
are its rows in ascending global order ("row_order": all rows grouped by
owner, ascending within an owner).  The all-to-all itself is plain block
copying: send block o of rank t becomes receive block t of owner o.
"""
from __future__ import annotations

import numpy as np


def row_order(owner_of_row, num_owners):
    """Rows grouped by owner (ascending within an owner) and the owners'
    offsets into that order: owner o's rows are order[off[o]:off[o+1]]."""
    owner_of_row = np.asarray(owner_of_row)
    order = np.concatenate([np.flatnonzero(owner_of_row == o) for o in range(num_owners)]).astype(np.int64)
    counts = np.array([np.count_nonzero(owner_of_row == o) for o in range(num_owners)], dtype=np.int64)
    return order, np.concatenate([[0], np.cumsum(counts)])


def pack_q(q_nope, q_rope, order):
    """Sender side, one rank: send row k = q_nope[order[k]] followed by
    q_rope[order[k]] (no-position part, then rotary part), every local head."""
    return np.concatenate([q_nope[order], q_rope[order]], axis=-1)


def exchange(send, splits):
    """The all-to-all: send[s] holds, for every receiver r in turn, the rows
    of its split splits[s][r].  Receiver r gets the blocks of senders 0, 1,
    ... in turn.  Returns the receive buffers and the bytes that crossed
    between different ranks (sender s != receiver r)."""
    recv, moved = [], 0
    num = len(send)
    offs = [np.concatenate([[0], np.cumsum(splits[s])]) for s in range(num)]
    for r in range(num):
        parts = []
        for s in range(num):
            blk = send[s][offs[s][r]:offs[s][r + 1]]
            parts.append(blk)
            if s != r:
                moved += blk.nbytes
        recv.append(np.concatenate(parts, axis=0))
    return recv, moved


def unpack_q(recv, num_ranks, n_rows):
    """Owner side: recv [T * n_rows, H/T, 576] (rank t's block first) ->
    [n_rows, H, 576] with head t H/T + h = rank t's local head h."""
    blocks = np.asarray(recv).reshape(num_ranks, n_rows, *np.asarray(recv).shape[1:])
    return np.concatenate(list(blocks), axis=1)


def pack_out(out_owner, num_ranks):
    """Owner side of the reverse exchange: [n_rows, H, 512] -> send blocks
    for ranks t = 0..T-1, block t = heads [t H/T, (t+1) H/T)."""
    hl = out_owner.shape[1] // num_ranks
    return np.concatenate([out_owner[:, t * hl:(t + 1) * hl] for t in range(num_ranks)], axis=0)


def unpack_out(recv, order):
    """Sender side of the reverse exchange: recv rows in owner-grouped order
    -> global row order, out[order[k]] = recv[k]."""
    out = np.empty_like(recv)
    out[np.asarray(order)] = recv
    return out
