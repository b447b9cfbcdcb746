"""Thin ctypes binding of libsplash_attn (include/splash_attn.h).

Argument marshalling only: every step of the attention path runs in the
library's gfx950 kernels.  Tensors are torch tensors on the GPU; their device
pointers and the current HIP stream are handed to the C entry points of the
same names.  A missing library raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsplash_attn.so")

SPLASH_OK = 0
SPLASH_ERR_INVALID_ARGUMENT = -1
SPLASH_ERR_UNSUPPORTED = -2
SPLASH_ERR_MISALIGNED = -3
SPLASH_ERR_WORKSPACE_TOO_SMALL = -4
SPLASH_ERR_HIP = -5

KV_BF16 = 0
KV_FP8_E4M3 = 1
KV_FP8_LATENT = 2   # 656-byte rows: E4M3 latent, 4 fp32 tile scales, bf16 RoPE
FLAG_DEBUG_CHECK = 1
FLAG_FORCE_SPLIT = 2
FLAG_EXACT_QK = 4
DEFAULT_MAX_PARTIALS = 1024


class SplashError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class MlaDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_heads", ctypes.c_int32),
        ("dim_qk", ctypes.c_int32),
        ("dim_v", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("kv_scales", ctypes.c_void_p),
        ("softmax_scale", ctypes.c_float),
        ("flags", ctypes.c_uint32),
        ("split_pages", ctypes.c_int32),
    ]


_lib = None

_VP = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t
_PD = ctypes.POINTER(MlaDesc)
_PI32 = ctypes.POINTER(ctypes.c_int32)

_SIGNATURES = {
    "splash_mla_workspace_size": (_SZ, [_I32, _I32, _I32, _I32]),
    "splash_mla_workspace_offsets": (_SZ, [_I32, _I32, _I32, _I32, ctypes.POINTER(_SZ)]),
    "splash_mla_attend": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _PD, _VP, _SZ, _VP]),
    "splash_mla_attend_noalloc": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _PD, _VP]),
    "splash_mla_plan": (ctypes.c_int, [_VP, _I32, _PD, _VP, _SZ, _VP]),
    "splash_mla_run": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _PD, _VP, _SZ, _VP]),
    "splash_mla_attend_units": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _PD, _VP, _SZ, _VP]),
    "splash_mla_combine_splits": (ctypes.c_int, [_I32, _VP, _VP, _PD, _VP, _SZ, _VP]),
    "splash_mla_combine": (ctypes.c_int, [_VP, _VP, _VP, _I32, _I32, _I32, _VP, _VP, _VP]),
    "splash_mla_attend_topk": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _I32, _VP, _VP, _PD, _VP, _SZ,
                                              _VP]),
    "splash_dop_pack_q": (ctypes.c_int, [_VP, _VP, _VP, _I32, _I32, _VP, _VP]),
    "splash_dop_unpack_q": (ctypes.c_int, [_VP, _I32, _I32, _I32, _VP, _VP]),
    "splash_dop_pack_out": (ctypes.c_int, [_VP, _I32, _I32, _I32, _VP, _VP]),
    "splash_dop_unpack_out": (ctypes.c_int, [_VP, _VP, _I32, _I32, _VP, _VP]),
    "splash_mla_attend_shard": (ctypes.c_int, [_VP, _VP, _VP, _VP, _I32, _VP, _VP, _I32, _I32, _VP, _VP, _PD, _VP,
                                               _SZ, _VP]),
    "splash_mla_debug_gather": (ctypes.c_int, [_VP, _VP, _VP, _PD, _VP, _VP]),
    "splash_mla_plan_host": (ctypes.c_int, [_PI32, _I32, _PD, _I32, _I32, _PI32, _I32, _PI32, _PI32, _PI32]),
    "splash_mla_max_units": (_I32, [_I32, _I32, _I32]),
    "splash_device_workers": (_I32, []),
    "splash_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "splash_last_error": (ctypes.c_char_p, []),
    "splash_version": (ctypes.c_char_p, []),
}


def _hip_runtimes_mapped():
    try:
        with open("/proc/self/maps") as f:
            return sorted({l.split()[-1] for l in f if "libamdhip64" in l})
    except OSError:
        return []


def lib():
    """Load libsplash_attn.so (built in-tree); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_37626_amd.build`")
    import torch  # noqa: F401  (load torch's HIP runtime first so the library binds to it)
    handle = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes are mapped into this process: {runtimes}")
    _lib = handle
    return _lib


def _check(status: int) -> None:
    if status != SPLASH_OK:
        L = lib()
        raise SplashError(status, f"{L.splash_status_string(status).decode()}: {L.splash_last_error().decode()}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    import torch
    return torch.cuda.current_stream().cuda_stream


def make_desc(batch: int, num_heads: int, max_pages_per_seq: int, num_pages: int,
              kv_dtype: int = KV_BF16, kv_scales=None, softmax_scale: float = 1.0 / 192 ** 0.5,
              flags: int = 0, split_pages: int = 0) -> MlaDesc:
    d = MlaDesc()
    d.batch = batch
    d.num_heads = num_heads
    d.dim_qk = 576
    d.dim_v = 512
    d.page_size = 64
    d.max_pages_per_seq = max_pages_per_seq
    d.num_pages = num_pages
    d.kv_dtype = kv_dtype
    d.kv_scales = _ptr(kv_scales)
    d.softmax_scale = float(np.float32(softmax_scale))
    d.flags = flags
    d.split_pages = split_pages
    return d


def workspace_size(batch: int, q_chunk: int, num_heads: int, max_partials: int = 0) -> int:
    return int(lib().splash_mla_workspace_size(batch, q_chunk, num_heads, max_partials))


def workspace_offsets(batch: int, q_chunk: int, num_heads: int, max_partials: int = 0):
    offs = (_SZ * 6)()
    total = lib().splash_mla_workspace_offsets(batch, q_chunk, num_heads, max_partials, offs)
    return list(offs), int(total)


def device_workers() -> int:
    return int(lib().splash_device_workers())


def splash_mla_attend(q, kv_pages, block_table, seq_lens, q_chunk: int, out, lse, desc: MlaDesc,
                      workspace, stream=None) -> None:
    _check(lib().splash_mla_attend(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                   _ptr(out), _ptr(lse), ctypes.byref(desc), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_attend_noalloc(q, kv_pages, block_table, seq_lens, q_chunk: int, out, lse, desc: MlaDesc,
                              stream=None) -> None:
    """splash_mla_attend on the library's own workspace (no allocation)."""
    _check(lib().splash_mla_attend_noalloc(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                           _ptr(out), _ptr(lse), ctypes.byref(desc), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 128 << 20  # SPLASH_NOALLOC_SCRATCH_BYTES


def splash_mla_plan(seq_lens, q_chunk: int, desc: MlaDesc, workspace, stream=None) -> None:
    _check(lib().splash_mla_plan(_ptr(seq_lens), q_chunk, ctypes.byref(desc), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_run(q, kv_pages, block_table, seq_lens, q_chunk: int, out, lse, desc: MlaDesc,
                   workspace, stream=None) -> None:
    _check(lib().splash_mla_run(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                _ptr(out), _ptr(lse), ctypes.byref(desc), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_attend_units(q, kv_pages, block_table, seq_lens, q_chunk: int, out, lse, desc: MlaDesc,
                            workspace, stream=None) -> None:
    _check(lib().splash_mla_attend_units(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                         _ptr(out), _ptr(lse), ctypes.byref(desc), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_combine_splits(q_chunk: int, out, lse, desc: MlaDesc, workspace, stream=None) -> None:
    _check(lib().splash_mla_combine_splits(q_chunk, _ptr(out), _ptr(lse), ctypes.byref(desc), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_attend_shard(q, kv_pages, block_table, seq_lens, q_chunk: int, key_begin, key_end,
                            num_shards: int, shard: int, part_out, part_lse, desc: MlaDesc, workspace,
                            stream=None) -> None:
    _check(lib().splash_mla_attend_shard(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                         _ptr(key_begin), _ptr(key_end), num_shards, shard, _ptr(part_out),
                                         _ptr(part_lse), ctypes.byref(desc), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_mla_attend_topk(q, kv_pages, block_table, seq_lens, q_chunk: int, topk_idx, topk_count, out, lse,
                           desc: MlaDesc, workspace, stream=None) -> None:
    """Row n attends the positions topk_idx[n, :topk_count[n]] of its request's history."""
    _check(lib().splash_mla_attend_topk(_ptr(q), _ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), q_chunk,
                                        _ptr(topk_idx), _ptr(topk_count), int(topk_idx.shape[1]), _ptr(out), _ptr(lse),
                                        ctypes.byref(desc), _ptr(workspace),
                                        workspace.numel() * workspace.element_size(), _stream(stream)))


def splash_dop_pack_q(q_nope, q_rope, row_order, send, stream=None) -> None:
    """Rank side: send[k] = q_nope[row_order[k]] | q_rope[row_order[k]] (all local heads)."""
    n, hl = int(q_nope.shape[0]), int(q_nope.shape[1])
    _check(lib().splash_dop_pack_q(_ptr(q_nope), _ptr(q_rope), _ptr(row_order), n, hl, _ptr(send), _stream(stream)))


def splash_dop_unpack_q(recv, num_ranks: int, q_owner, stream=None) -> None:
    """Owner side: recv [T, n, H/T, 576] -> q_owner [n, H, 576]."""
    n, H = int(q_owner.shape[0]), int(q_owner.shape[1])
    _check(lib().splash_dop_unpack_q(_ptr(recv), num_ranks, n, H // num_ranks, _ptr(q_owner), _stream(stream)))


def splash_dop_pack_out(out_owner, num_ranks: int, send, stream=None) -> None:
    """Owner side: out_owner [n, H, 512] -> send [T, n, H/T, 512]."""
    n, H = int(out_owner.shape[0]), int(out_owner.shape[1])
    _check(lib().splash_dop_pack_out(_ptr(out_owner), num_ranks, n, H // num_ranks, _ptr(send), _stream(stream)))


def splash_dop_unpack_out(recv, row_order, out, stream=None) -> None:
    """Rank side: out[row_order[k]] = recv[k] (all local heads)."""
    n, hl = int(out.shape[0]), int(out.shape[1])
    _check(lib().splash_dop_unpack_out(_ptr(recv), _ptr(row_order), n, hl, _ptr(out), _stream(stream)))


def splash_mla_combine(partials, partial_lse, split_indptr, batch: int, q_chunk: int, num_heads: int,
                       out, out_lse=None, stream=None) -> None:
    _check(lib().splash_mla_combine(_ptr(partials), _ptr(partial_lse), _ptr(split_indptr), batch, q_chunk,
                                    num_heads, _ptr(out), _ptr(out_lse), _stream(stream)))


def splash_mla_debug_gather(kv_pages, block_table, seq_lens, desc: MlaDesc, dense_out, stream=None) -> None:
    _check(lib().splash_mla_debug_gather(_ptr(kv_pages), _ptr(block_table), _ptr(seq_lens), ctypes.byref(desc),
                                         _ptr(dense_out), _stream(stream)))


def splash_mla_plan_host(seq_lens: np.ndarray, q_chunk: int, desc: MlaDesc, num_workers: int,
                         max_partials: int = 0):
    """Host mirror of the planner: returns (units [U,4], indptr [T+1], stats dict).

    stats["fold"] tells a fold plan (each worker runs its own units) from a
    plan of one unit size (workers draw units from a queue); for a fold plan
    stats["cap"] is the pages a long tile keeps and stats["worker_start"]
    the first unit of each of the num_workers workers and the end
    (num_workers + 1 entries), else None.
    """
    L = lib()
    seq = np.ascontiguousarray(seq_lens, dtype=np.int32)
    T = int(seq.shape[0]) * q_chunk
    max_units = int(L.splash_mla_max_units(int(seq.shape[0]), q_chunk, max_partials))
    units = np.zeros((max(max_units, 1), 4), dtype=np.int32)
    indptr = np.zeros(T + 1, dtype=np.int32)
    stats = np.zeros(7, dtype=np.int32)
    wstart = np.zeros(num_workers + 1, dtype=np.int32)
    as_p = lambda a: a.ctypes.data_as(_PI32)
    _check(L.splash_mla_plan_host(as_p(seq), q_chunk, ctypes.byref(desc), num_workers, max_partials,
                                  as_p(units), max_units, as_p(indptr), as_p(stats), as_p(wstart)))
    n = int(stats[0])
    fold = int(stats[4]) > 0
    return units[:n].copy(), indptr, {"units": n, "partials": int(stats[1]), "chunk_pages": int(stats[2]),
                                      "total_pages": int(stats[3]), "fold": fold, "cap": int(stats[5]),
                                      "max_parts": int(stats[6]), "worker_start": wstart if fold else None}


def version() -> str:
    return lib().splash_version().decode()
