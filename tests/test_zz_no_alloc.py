"""mar_head_sample_noalloc (the diffusion head's entry point for callers that
cannot allocate device memory) against mar_head_sample: the same kernels on
the library's static scratch array instead of the handle's workspace, so
the results must be identical, bit for bit.  Two calls in a row, the second
on fewer tokens (the array keeps the first call's contents), a call on more
tokens than the handle's own max_rows, and a call past the array's size."""
import numpy as np
import pytest
import torch

from paper_2503_12450_amd import binding as B
from paper_2503_12450_amd.device import to_device, upload_head
from paper_2503_12450_amd.workload import HEADS, HeadDims, head_weights, normal_rows

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(hd, R, y_rows, seed):
    g = np.random.Generator(np.random.Philox(seed))
    y = to_device(normal_rows((2, y_rows, hd.cond_dim), seed=seed + 1, std=2.0), "f32")
    rc = torch.from_numpy(g.permutation(y_rows)[:R].astype(np.int32)).to(DEV)
    ru = torch.from_numpy(g.permutation(y_rows)[:R].astype(np.int32)).to(DEV)
    x0 = to_device(normal_rows((R, hd.token_dim), seed=seed + 2), "f32")
    xi = to_device(normal_rows((hd.steps, R, hd.token_dim), seed=seed + 3), "f32")
    return y[0].contiguous(), y[1].contiguous(), rc, ru, x0, xi


def _outs(hd, R):
    return (torch.empty((R, hd.token_dim), device=DEV),
            torch.empty((hd.steps + 1, R, hd.token_dim), device=DEV),
            torch.empty((hd.steps, R, hd.token_dim), device=DEV))


def _both(head_ref, head_na, hd, R, y_rows, seed, scale):
    args = _inputs(hd, R, y_rows, seed)
    ref, got = _outs(hd, R), _outs(hd, R)
    print(f"[no-alloc] {R} tokens, width {hd.width}, depth {hd.depth}, seed {seed}", flush=True)
    head_ref.sample(*args, scale, *ref)
    head_na.sample(*args, scale, *got, noalloc=True)
    torch.cuda.synchronize()
    for a, b in zip(got, ref):
        assert torch.equal(a, b)


def test_noalloc_matches_workspace_entry_point_twice():
    hd = HeadDims(width=192, depth=2, cond_dim=128, token_dim=16, steps=8, train_steps=80, freq_dim=64,
                  max_rows=64)
    W = upload_head(head_weights(hd, seed=8), hd.dtype)
    head = B.MarHead(hd, W)
    _both(head, head, hd, 50, 120, seed=30, scale=3.0)
    _both(head, head, hd, 17, 120, seed=40, scale=3.0)   # fewer tokens: stale rows left in the array


def test_noalloc_is_not_bounded_by_the_handles_rows():
    from dataclasses import replace
    hd = replace(HEADS["mar-l"], max_rows=200, steps=20, train_steps=200)
    W = upload_head(head_weights(hd, seed=9), hd.dtype)
    big = B.MarHead(hd, W)
    small = B.MarHead(replace(hd, max_rows=8), W)
    _both(big, small, hd, 200, 1000, seed=50, scale=4.0)
    _both(big, small, hd, 64, 1000, seed=60, scale=4.0)


def test_noalloc_refuses_rows_past_the_array():
    from dataclasses import replace
    hd = replace(HEADS["mar-l"], max_rows=8, steps=4, train_steps=40)
    head = B.MarHead(hd, upload_head(head_weights(hd, seed=9), hd.dtype))
    R = 388   # 387 tokens fit 64 MiB at this shape
    args = _inputs(hd, R, 400, seed=70)
    out = _outs(hd, R)
    sentinel = torch.full_like(out[0], 7.0)
    out[0].copy_(sentinel)
    with pytest.raises(B.MarError) as e:
        head.sample(*args, 2.0, *out, noalloc=True)
    assert e.value.status == B.MAR_E_SHAPE
    torch.cuda.synchronize()
    assert torch.equal(out[0], sentinel)
