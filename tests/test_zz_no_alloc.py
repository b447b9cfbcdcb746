"""splash_mla_attend_noalloc: the step on the library's own device scratch
(no allocation by the call), checked against splash_mla_attend and the fp64
oracle at the parity bar, on two calls in a row (the second with a smaller
input, so it runs over the first call's leftovers), and its refusals."""
import numpy as np
import pytest
import torch

from paper_2609_37626_amd import binding as B
from paper_2609_37626_amd import workloads as W
from paper_2609_37626_amd.device import to_device
from tests.test_gpu_parity import LSE_TOL, OUT_TOL, assert_parity, gpu_attend

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def noalloc_attend(batch):
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    B.splash_mla_attend_noalloc(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, db.desc())
    torch.cuda.synchronize()
    return out, lse


def test_noalloc_matches_attend_on_two_calls_second_smaller():
    first = W.make_custom([4096, 300, 9000, 65, 1, 2500, 1800, 7000], H=128, seed=81)
    second = W.make_custom([700, 33], H=64, q_chunk=2, seed=82)
    for label, batch in [("first (larger)", first), ("second (smaller)", second)]:
        out, lse = noalloc_attend(batch)
        ref_out, ref_lse = gpu_attend(batch)
        d_o = float((out.float() - ref_out.float()).abs().max())
        d_l = float((lse - ref_lse).abs().max())
        print(f"{label}: vs splash_mla_attend out {d_o:.2e} lse {d_l:.2e}", flush=True)
        assert d_o <= OUT_TOL[batch.kv_dtype] and d_l <= LSE_TOL, (label, d_o, d_l)
        assert_parity(batch, out, lse, label=f"noalloc {label}")


def test_noalloc_fp8_chunk():
    batch = W.make_custom([900, 2000, 8], H=128, q_chunk=8, kv_dtype=W.KV_FP8_E4M3, seed=83)
    out, lse = noalloc_attend(batch)
    assert_parity(batch, out, lse, label="noalloc fp8 chunk")


def test_noalloc_refuses_what_it_cannot_hold():
    small = W.make_custom([100], H=128, seed=84)
    db = to_device(small)
    out, lse = db.alloc_outputs()
    # 600 histories of up to 2000 pages force 1200 partials of 256 KB: far
    # more than the scratch; refused on the host before any launch
    big = B.make_desc(600, 128, 2000, int(db.kv.shape[0]))
    with pytest.raises(B.SplashError) as e:
        B.splash_mla_attend_noalloc(db.q, db.kv, db.block_table, db.seq_lens, 1, out, lse, big)
    assert e.value.status == B.SPLASH_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(B.SplashError) as e:
        B.splash_mla_attend_noalloc(db.q, db.kv, db.block_table, db.seq_lens, 1, out, lse,
                                    db.desc(flags=B.FLAG_DEBUG_CHECK))
    assert e.value.status == B.SPLASH_ERR_UNSUPPORTED
