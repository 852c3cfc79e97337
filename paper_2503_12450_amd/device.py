"""Device placement of the seeded inputs (torch is used for memory only)."""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .workload import MATRIX_NAMES


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def to_device(a: np.ndarray, dtype: str, device="cuda"):
    """float32 host values (already exact in `dtype`) -> device tensor."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device=device).to(torch_dtype(dtype)).contiguous()


def upload_blocks(blocks: Sequence[Dict[str, np.ndarray]], dtype: str, device="cuda") -> List[Dict[str, object]]:
    """Matrices in the storage dtype, LayerNorm parameters and biases fp32."""
    out = []
    for blk in blocks:
        out.append({k: to_device(v, dtype if k in MATRIX_NAMES else "f32", device) for k, v in blk.items()})
    return out
