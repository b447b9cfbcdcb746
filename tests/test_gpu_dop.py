"""GPU parity of the DOP regroup kernels (bit-exact: pure data movement).

T ranks and their owners are emulated on one GPU: every rank packs its head
slice of all N rows by owner (splash_dop_pack_q), the all-to-all is a plain
block copy here, every owner assembles its rows with all heads
(splash_dop_unpack_q); after attention the owner splits its output by rank
(splash_dop_pack_out) and every rank puts its rows back in global order
(splash_dop_unpack_out).  Each kernel's output is compared with the oracle's
definition of that step, and the round trip with the full tensors.
"""
import numpy as np
import pytest
import torch

from oracle import dop
from paper_2609_37626_amd import binding as B

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def host(t):
    return t.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("N,H,T,seed", [(256, 128, 8, 1), (37, 64, 4, 2), (5, 16, 16, 3), (1, 128, 8, 4),
                                        (1024, 128, 8, 5)])
def test_dop_regroup_matches_definition(N, H, T, seed):
    rng = np.random.default_rng(seed)
    hl = H // T
    q = rng.integers(0, 1 << 16, size=(N, H, 576), dtype=np.uint16)
    out_full = rng.integers(0, 1 << 16, size=(N, H, 512), dtype=np.uint16)
    owner = rng.integers(0, T, size=N)
    if T > 2:
        owner[owner == T - 1] = 0                      # an owner with no rows
    order, off = dop.row_order(owner, T)
    counts = np.diff(off)
    print(f"N={N} H={H} T={T} rows per owner {counts.tolist()}", flush=True)
    order_d = torch.from_numpy(order.astype(np.int32)).cuda()
    # forward
    sends = []
    for t in range(T):
        nope, rope = q[:, t * hl:(t + 1) * hl, :512], q[:, t * hl:(t + 1) * hl, 512:]
        send = torch.empty((N, hl, 576), dtype=torch.int16, device="cuda")
        B.splash_dop_pack_q(bits(nope), bits(rope), order_d, send)
        torch.cuda.synchronize()
        assert np.array_equal(host(send), dop.pack_q(nope, rope, order))
        sends.append(send)
    for o in range(T):
        recv = torch.cat([s[off[o]:off[o + 1]] for s in sends]).contiguous()     # the all-to-all
        q_owner = torch.empty((counts[o], H, 576), dtype=torch.int16, device="cuda")
        B.splash_dop_unpack_q(recv, T, q_owner)
        torch.cuda.synchronize()
        rows = np.flatnonzero(owner == o)
        assert np.array_equal(host(q_owner), q[rows])
        assert np.array_equal(host(q_owner), dop.unpack_q(host(recv), T, len(rows)))
    # reverse
    sends_r = []
    for o in range(T):
        rows = np.flatnonzero(owner == o)
        send = torch.empty((T * len(rows), hl, 512), dtype=torch.int16, device="cuda")
        B.splash_dop_pack_out(bits(out_full[rows]), T, send)
        torch.cuda.synchronize()
        assert np.array_equal(host(send), dop.pack_out(out_full[rows], T))
        sends_r.append(send.view(T, len(rows), hl, 512))
    for t in range(T):
        recv = torch.cat([s[t] for s in sends_r]).contiguous()                   # the reverse all-to-all
        out = torch.empty((N, hl, 512), dtype=torch.int16, device="cuda")
        B.splash_dop_unpack_out(recv, order_d, out)
        torch.cuda.synchronize()
        assert np.array_equal(host(out), out_full[:, t * hl:(t + 1) * hl])
