"""Move a host batch to the GPU and call the library on it (marshalling only)."""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

from . import binding as B
from .workloads import Batch, KV_FP8_E4M3, KV_FP8_LATENT


@dataclasses.dataclass
class DeviceBatch:
    q: torch.Tensor            # bf16 [N, H, 576]
    kv: torch.Tensor           # bf16 or uint8 [num_pages, 64, 576]
    kv_scales: Optional[torch.Tensor]
    block_table: torch.Tensor  # int32 [B, max_pages]
    seq_lens: torch.Tensor     # int32 [B]
    q_chunk: int
    H: int
    kv_dtype: int
    softmax_scale: float

    @property
    def B(self) -> int:
        return int(self.seq_lens.shape[0])

    def desc(self, flags: int = 0, split_pages: int = 0) -> B.MlaDesc:
        return B.make_desc(self.B, self.H, int(self.block_table.shape[1]), int(self.kv.shape[0]),
                           self.kv_dtype, self.kv_scales, self.softmax_scale, flags, split_pages)

    def alloc_outputs(self):
        N = self.B * self.q_chunk
        out = torch.empty((N, self.H, 512), dtype=torch.bfloat16, device=self.q.device)
        lse = torch.empty((N, self.H), dtype=torch.float32, device=self.q.device)
        return out, lse

    def workspace(self, max_partials: int = 0) -> torch.Tensor:
        nbytes = B.workspace_size(self.B, self.q_chunk, self.H, max_partials)
        return torch.empty(nbytes, dtype=torch.uint8, device=self.q.device)

    def attend(self, out=None, lse=None, workspace=None, flags: int = 0, split_pages: int = 0, stream=None):
        if out is None:
            out, lse = self.alloc_outputs()
        if workspace is None:
            workspace = self.workspace()
        B.splash_mla_attend(self.q, self.kv, self.block_table, self.seq_lens, self.q_chunk, out, lse,
                            self.desc(flags, split_pages), workspace, stream)
        return out, lse


def to_device(batch: Batch, device: str = "cuda") -> DeviceBatch:
    q = torch.from_numpy(batch.q.view(np.int16)).to(device).view(torch.bfloat16)
    if batch.kv_dtype == KV_FP8_E4M3:
        kv = torch.from_numpy(batch.kv).to(device)
        scales = torch.from_numpy(batch.kv_scales).to(device)
    elif batch.kv_dtype == KV_FP8_LATENT:
        kv = torch.from_numpy(batch.kv).to(device)
        scales = None
    else:
        kv = torch.from_numpy(batch.kv.view(np.int16)).to(device).view(torch.bfloat16)
        scales = None
    return DeviceBatch(q=q, kv=kv, kv_scales=scales,
                       block_table=torch.from_numpy(batch.block_table).to(device),
                       seq_lens=torch.from_numpy(batch.seq_lens).to(device),
                       q_chunk=batch.q_chunk, H=batch.H, kv_dtype=batch.kv_dtype,
                       softmax_scale=float(batch.softmax_scale))


def bf16_to_float(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy()
