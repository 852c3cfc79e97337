"""The diffusion head on the GPU against its oracle (oracle/diffusion_head.py),
through the C ABI of include/mar_head.h.

Teacher forcing along the whole sampler trajectory: for every sampling step
the oracle evaluates the network (both guidance branches, Eq. 7) on the
latent the GPU held before that step, and
* the GPU's guided noise prediction must match the oracle's within the bf16
  bar of the method's statement, max-abs 2e-2 / rel 1e-2 per branch,
  carried through the guidance mix: |d eps| <= (|1 - s| + |s|) (2e-2 +
  1e-2 max(|eps_c|, |eps_u|)) elementwise;
* the GPU's next latent must equal the oracle's DDPM step taken from the
  GPU's own latent and noise prediction within fp32 resolution (the step is
  a few fp32 operations on O(1) values).
The per-step checks keep errors from compounding over 100 steps; the final
latents are then the trajectory's last entry.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import diffusion_head as DH
from paper_2503_12450_amd import binding as B
from paper_2503_12450_amd.device import to_device, upload_head
from paper_2503_12450_amd.workload import HEADS, HeadDims, head_weights, normal_rows

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run(hd, R, y_rows, scale, seed=0, bad_index=False):
    W = head_weights(hd, seed=seed)
    yc = normal_rows((y_rows, hd.cond_dim), seed=seed + 11, std=2.0)
    yu = normal_rows((y_rows, hd.cond_dim), seed=seed + 12, std=2.0)
    g = np.random.Generator(np.random.Philox(seed + 13))
    rc = g.permutation(y_rows)[:R].astype(np.int32)
    ru = g.permutation(y_rows)[:R].astype(np.int32)
    if bad_index:
        rc[1], ru[2] = y_rows + 5, -3     # outside the rows: read as zeros
    x0 = normal_rows((R, hd.token_dim), seed=seed + 14)
    xi = normal_rows((hd.steps, R, hd.token_dim), seed=seed + 15)
    print(f"[head] width {hd.width} depth {hd.depth} cond {hd.cond_dim} steps {hd.steps}: {R} tokens, "
          f"scale {scale}", flush=True)
    head = B.MarHead(hd, upload_head(W, hd.dtype))
    dyc, dyu = to_device(yc, "f32"), to_device(yu, "f32")
    drc = torch.from_numpy(rc).to(DEV)
    dru = torch.from_numpy(ru).to(DEV)
    dx0, dxi = to_device(x0, "f32"), to_device(xi, "f32")
    x_out = torch.empty((R, hd.token_dim), dtype=torch.float32, device=DEV)
    traj = torch.empty((hd.steps + 1, R, hd.token_dim), dtype=torch.float32, device=DEV)
    eps = torch.empty((hd.steps, R, hd.token_dim), dtype=torch.float32, device=DEV)
    head.sample(dyc, dyu, drc, dru, dx0, dxi, scale, x_out, traj, eps)
    torch.cuda.synchronize()
    zc = np.where((rc >= 0)[:, None] & (rc < y_rows)[:, None], yc[np.clip(rc, 0, y_rows - 1)], 0.0)
    zu = np.where((ru >= 0)[:, None] & (ru < y_rows)[:, None], yu[np.clip(ru, 0, y_rows - 1)], 0.0)
    # the head conditions on the transformer rows as it stores them (bf16)
    from oracle import storage_round
    zc, zu = storage_round(zc, hd.dtype), storage_round(zu, hd.dtype)
    return W, zc, zu, x0, xi, x_out.cpu().numpy(), traj.cpu().numpy(), eps.cpu().numpy()


def _teacher_forced(hd, W, zc, zu, xi, scale, traj, eps, rows=None):
    sched = DH.ddpm_schedule(hd)
    e = DH.time_embeddings(hd, W)
    rows = np.arange(traj.shape[1]) if rows is None else np.asarray(rows)
    worst, worst_x = 0.0, 0.0
    for j in range(hd.steps):
        i = hd.steps - 1 - j
        x = traj[j][rows].astype(np.float64)
        ec = DH.head_eps(x, e[i], zc[rows], W, hd)
        eu = DH.head_eps(x, e[i], zu[rows], W, hd)
        want = DH.guided_eps(ec, eu, scale)
        bar = (abs(1 - scale) + abs(scale)) * (2e-2 + 1e-2 * np.maximum(np.abs(ec), np.abs(eu)))
        d = np.abs(eps[j][rows] - want)
        worst = max(worst, float((d / bar).max()))
        assert np.all(d <= bar), f"sampling step {i}: eps off by {d.max():.3e}"
        nx = DH.ddpm_step(x, eps[j][rows].astype(np.float64), i, sched, xi[i][rows])
        dx = np.abs(traj[j + 1][rows] - nx)
        worst_x = max(worst_x, float(dx.max()))
        np.testing.assert_allclose(traj[j + 1][rows], nx, rtol=2e-6, atol=2e-6,
                                   err_msg=f"sampling step {i}: DDPM update")
    print(f"  worst eps deviation {worst:.3f} of the bar; worst latent step deviation {worst_x:.2e}", flush=True)


@pytest.mark.parametrize("width,cond", [(192, 128), (256, 512)])
@pytest.mark.parametrize("scale", [1.0, 4.0])
def test_head_small_ragged_rows(scale, width, cond):
    """Two widths, 37 tokens = 74 rows that end mid-tile, one token
    conditioned on an index past the rows (read as a zero row)."""
    hd = HeadDims(width=width, depth=2, cond_dim=cond, token_dim=16, steps=12, train_steps=120, freq_dim=64,
                  max_rows=64)
    W, zc, zu, x0, xi, x_out, traj, eps = _run(hd, 37, 90, scale, bad_index=True)
    np.testing.assert_array_equal(traj[0], x0)
    np.testing.assert_array_equal(traj[-1], x_out)
    _teacher_forced(hd, W, zc, zu, xi, scale, traj, eps)


def test_head_mar_l_size_sampled_tokens():
    """The MAR-L head (width 1280, 8 blocks, 100 steps) on 448 tokens, the
    most a 64-image decoding step of the 64-step cosine schedule decodes;
    the oracle follows 6 sampled tokens through all 100 steps."""
    hd = replace(HEADS["mar-l"], max_rows=512)
    W, zc, zu, x0, xi, x_out, traj, eps = _run(hd, 448, 128 * 320, 4.0, seed=3)
    assert np.all(np.isfinite(x_out))
    _teacher_forced(hd, W, zc, zu, xi, 4.0, traj, eps, rows=[0, 1, 100, 255, 446, 447])


def test_head_rows_are_independent():
    """A token's latent depends only on its own rows, noise and the weights:
    sampling a subset gives the same bits for those tokens."""
    hd = HeadDims(width=128, depth=2, cond_dim=64, token_dim=16, steps=6, train_steps=60, freq_dim=64,
                  max_rows=64)
    W = head_weights(hd, seed=5)
    y = to_device(normal_rows((50, hd.cond_dim), seed=21), "f32")
    idx = torch.arange(40, dtype=torch.int32, device=DEV)
    x0 = to_device(normal_rows((40, hd.token_dim), seed=22), "f32")
    xi = to_device(normal_rows((hd.steps, 40, hd.token_dim), seed=23), "f32")
    head = B.MarHead(hd, upload_head(W, hd.dtype))
    full = torch.empty((40, hd.token_dim), device=DEV)
    head.sample(y, y, idx, idx, x0, xi, 3.0, full)
    part = torch.empty((10, hd.token_dim), device=DEV)
    head.sample(y, y, idx[5:15].contiguous(), idx[5:15].contiguous(), x0[5:15].contiguous(),
                xi[:, 5:15].contiguous(), 3.0, part)
    torch.cuda.synchronize()
    assert torch.equal(part, full[5:15])


@pytest.mark.parametrize("model", ["mar-b", "mar-h"])
def test_head_other_model_widths(model):
    """The MAR-B (width 1024, 6 blocks) and MAR-H (width 1536, 12 blocks)
    heads, whose row kernels have their own width-specialised forms, on 9
    tokens over 10 sampling steps of the respaced 1000-step schedule."""
    hd = replace(HEADS[model], steps=10, max_rows=16)
    W, zc, zu, x0, xi, x_out, traj, eps = _run(hd, 9, 40, 4.0, seed=7)
    np.testing.assert_array_equal(traj[-1], x_out)
    _teacher_forced(hd, W, zc, zu, xi, 4.0, traj, eps)


def test_head_one_token_and_no_tokens():
    """One token samples like any other (teacher-forced); zero tokens is a
    no-op that leaves the output untouched."""
    hd = HeadDims(width=128, depth=2, cond_dim=64, token_dim=16, steps=8, train_steps=80, freq_dim=64,
                  max_rows=4)
    W, zc, zu, x0, xi, x_out, traj, eps = _run(hd, 1, 3, 2.0, seed=9)
    _teacher_forced(hd, W, zc, zu, xi, 2.0, traj, eps)
    head = B.MarHead(hd, upload_head(W, hd.dtype))
    y = to_device(normal_rows((3, hd.cond_dim), seed=31), "f32")
    none = torch.empty(0, dtype=torch.int32, device=DEV)
    x0e = torch.empty((0, hd.token_dim), device=DEV)
    xie = torch.empty((hd.steps, 0, hd.token_dim), device=DEV)
    out = torch.full((1, hd.token_dim), 7.0, device=DEV)
    head.sample(y, y, none, none, x0e, xie, 2.0, out)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
