"""Move a synthetic workload into device memory (PyTorch allocations only).

Storage is copied bit for bit: bf16 patterns become ``torch.bfloat16``
tensors, fp8 codes ``torch.uint8``, fp32 stays ``torch.float32``.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .workload import Workload


def _dev_store(a: np.ndarray, dtype: str, device) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    if dtype == "fp8":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


@dataclass
class DeviceInputs:
    wl: Workload
    q: torch.Tensor
    k_cache: torch.Tensor
    v_cache: torch.Tensor
    k_scale: Optional[torch.Tensor]
    v_scale: Optional[torch.Tensor]
    block_tables: torch.Tensor
    seq_lens: torch.Tensor

    @property
    def shape(self):
        return self.wl.shape


def to_device(wl: Workload, device="cuda:0") -> DeviceInputs:
    sh = wl.shape
    return DeviceInputs(
        wl=wl,
        q=_dev_store(wl.q, sh.q_dtype, device),
        k_cache=_dev_store(wl.k_cache, sh.kv_dtype, device),
        v_cache=_dev_store(wl.v_cache, sh.kv_dtype, device),
        k_scale=None if wl.k_scale is None else torch.from_numpy(wl.k_scale).to(device),
        v_scale=None if wl.v_scale is None else torch.from_numpy(wl.v_scale).to(device),
        block_tables=torch.from_numpy(np.ascontiguousarray(wl.block_tables)).to(device),
        seq_lens=torch.from_numpy(np.ascontiguousarray(wl.seq_lens)).to(device),
    )
