"""Plain fp64 CPU oracle of MAR's per-token diffusion head with classifier-free
guidance fed by the condition cache.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the tests,
the smoke check and the benchmark's CPU-baseline leg use it, and it imports
nothing from the product.

What the paper fixes.  MAR models the distribution of each token with
diffusion (Sec. 2): for every token decoded at a decoding step a small
denoising network, conditioned on the transformer's output row z of that
token, turns Gaussian noise into the token's latent over 100 diffusion steps
of the standard DDPM setting (Sec. 4.1).  Classifier-free guidance mixes a
conditional and an unconditional prediction (Eq. 7); with the condition
cache the unconditional transformer rows of a reuse step are the cached
residual added to the conditional rows (Eq. 10), and they feed the head's
unconditional branch.  Its cost does not depend on the number of decoding
steps: it is the constant term of Table 1's baseline FLOPs.

Readings (the paper gives neither the network nor the sampler):

* Network eps(x, i, z): a residual MLP of `depth` blocks and width w with
  adaptive-LayerNorm conditioning.
      c   = z W_z^T + b_z                         (once per decoding step)
      e_i = W_t2 silu(W_t1 phi(t_i) + b_t1) + b_t2   (sinusoidal phi of the
                                                    training timestep t_i)
      s   = silu(c + e_i)
      m   = s W_ada^T + b_ada    -> per block k: shift_k, scale_k, gate_k;
                                    final: shift_f, scale_f
      h   = x W_in^T + b_in
      block k:  u = ln(h) (1 + scale_k) + shift_k
                h = h + gate_k * (silu(u W1_k^T + b1_k) W2_k^T + b2_k)
      eps = (ln(h) (1 + scale_f) + shift_f) W_out^T + b_out
  with ln a LayerNorm without gain and shift.  Width and depth per model
  are read off Table 1: with them the head's FLOPs over one image
  reproduce the table's step-independent constant within a few percent.
* Sampler: DDPM ancestral sampling (Ho et al. 2020, Algorithm 2) on the
  linear schedule of that paper (beta from 1e-4 to 0.02 over 1000 training
  steps), respaced to 100 evenly spaced timesteps t_i = floor(i * 1000 /
  100) (Nichol & Dhariwal 2021, respacing): alpha_bar_i = prod over the
  training steps up to t_i, beta_i = 1 - alpha_bar_i / alpha_bar_(i-1);
      x_(i-1) = (x_i - beta_i / sqrt(1 - alpha_bar_i) eps) / sqrt(1 - beta_i)
                + sigma_i xi_i,
      sigma_i^2 = beta_i (1 - alpha_bar_(i-1)) / (1 - alpha_bar_i),
  sigma_0 = 0, from x_(steps-1) = the initial noise.  The Gaussian draws
  xi_i are inputs (drawn by the caller).
* Guidance: per token and per diffusion step, eps = eps_u + s (eps_c -
  eps_u) (Eq. 7 is garbled in the text; this is its usual form); the two
  evaluations of a token share x.  Temperature 1, constant s.
"""
from __future__ import annotations

import math
from typing import Dict

import numpy as np

from .mar_oracle import linear

__all__ = ["silu", "plain_layer_norm", "timestep_features", "ddpm_schedule", "time_embeddings",
           "head_eps", "guided_eps", "ddpm_step", "sample", "head_flops_per_eval"]


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def silu(x) -> np.ndarray:
    """x * sigmoid(x)."""
    x = _f64(x)
    return x / (1.0 + np.exp(-x))


def plain_layer_norm(x, eps: float) -> np.ndarray:
    """Row LayerNorm without gain and shift (biased variance)."""
    x = _f64(x)
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps)


def timestep_features(t, freq_dim: int) -> np.ndarray:
    """Sinusoidal features of integer timesteps: [cos(t f_k) ..., sin(t f_k)
    ...] with f_k = 10000^(-k / half), k = 0..half-1."""
    t = _f64(np.atleast_1d(t))
    half = freq_dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    a = t[:, None] * f[None, :]
    return np.concatenate([np.cos(a), np.sin(a)], axis=1)


def ddpm_schedule(hd) -> Dict[str, np.ndarray]:
    """Per sampling step i = 0..steps-1 (run from steps-1 down to 0): the
    training timestep t_i, alpha_bar_i, beta_i, the step's coefficients
    a_i = 1 / sqrt(1 - beta_i), b_i = beta_i / sqrt(1 - alpha_bar_i), and
    sigma_i (0 at i = 0)."""
    betas = np.linspace(hd.beta_start, hd.beta_end, hd.train_steps, dtype=np.float64)
    abar_all = np.cumprod(1.0 - betas)
    t = (np.arange(hd.steps) * hd.train_steps) // hd.steps
    abar = abar_all[t]
    abar_prev = np.concatenate([[1.0], abar[:-1]])
    beta = 1.0 - abar / abar_prev
    sigma = np.sqrt(beta * (1.0 - abar_prev) / (1.0 - abar))
    sigma[0] = 0.0
    return {"t": t, "abar": abar, "beta": beta, "a": 1.0 / np.sqrt(1.0 - beta),
            "b": beta / np.sqrt(1.0 - abar), "sigma": sigma}


def time_embeddings(hd, W) -> np.ndarray:
    """e_i for every sampling step i: [steps, w]."""
    phi = timestep_features(ddpm_schedule(hd)["t"], hd.freq_dim)
    return linear(silu(linear(phi, W["t1_w"], W["t1_b"])), W["t2_w"], W["t2_b"])


def head_eps(x, e_i, z, W, hd) -> np.ndarray:
    """Noise prediction of the head for rows x [R, token_dim] conditioned on
    z [R, cond_dim] at the diffusion step whose time embedding is e_i [w]."""
    w = hd.width
    c = linear(z, W["z_w"], W["z_b"])
    s = silu(c + _f64(e_i)[None, :])
    m = linear(s, W["ada_w"], W["ada_b"])
    h = linear(x, W["in_w"], W["in_b"])
    for k in range(hd.depth):
        shift, scale, gate = (m[:, (3 * k + j) * w:(3 * k + j + 1) * w] for j in range(3))
        u = plain_layer_norm(h, hd.ln_eps) * (1.0 + scale) + shift
        u = linear(silu(linear(u, W["fc1_w"][k], W["fc1_b"][k])), W["fc2_w"][k], W["fc2_b"][k])
        h = h + gate * u
    shift_f = m[:, 3 * hd.depth * w:(3 * hd.depth + 1) * w]
    scale_f = m[:, (3 * hd.depth + 1) * w:(3 * hd.depth + 2) * w]
    u = plain_layer_norm(h, hd.ln_eps) * (1.0 + scale_f) + shift_f
    return linear(u, W["out_w"], W["out_b"])


def guided_eps(eps_c, eps_u, scale: float) -> np.ndarray:
    """Eq. (7) read as eps_u + s (eps_c - eps_u)."""
    eps_c, eps_u = _f64(eps_c), _f64(eps_u)
    return eps_u + scale * (eps_c - eps_u)


def ddpm_step(x, eps, i: int, sched, xi) -> np.ndarray:
    """One ancestral step from sampling step i to i-1 (Ho et al. 2020,
    Algorithm 2, with the respaced coefficients)."""
    x, eps = _f64(x), _f64(eps)
    mean = sched["a"][i] * (x - sched["b"][i] * eps)
    return mean + sched["sigma"][i] * _f64(xi)


def sample(z_cond, z_uncond, x_init, xi, scale: float, W, hd, trajectory: bool = False):
    """Run the head's sampler for rows of tokens: z_cond, z_uncond
    [R, cond_dim] (the conditional and the unconditional transformer rows
    of each token, the latter from the condition cache on reuse steps),
    x_init [R, token_dim], xi [steps, R, token_dim] (xi[0] is unused).
    Returns x after the last step, or every x from the initial one down
    (trajectory [steps + 1, R, token_dim], entry j = x before step
    steps-1-j)."""
    sched = ddpm_schedule(hd)
    e = time_embeddings(hd, W)
    x = _f64(x_init)
    traj = [x]
    for i in range(hd.steps - 1, -1, -1):
        eps = guided_eps(head_eps(x, e[i], z_cond, W, hd), head_eps(x, e[i], z_uncond, W, hd), scale)
        x = ddpm_step(x, eps, i, sched, xi[i])
        traj.append(x)
    return np.stack(traj) if trajectory else x


def head_flops_per_eval(hd) -> float:
    """Multiply-adds x 2 of one evaluation of the network for one row, in the
    convention of Table 1 (every product of the network counted per
    evaluation: input, modulation, the blocks' two products, output).  The
    conditioning product and the time embedding are computed once per
    decoding step (per run) here and are left out."""
    w, T = hd.width, hd.token_dim
    macs = T * w + hd.n_mod * w * w + 2 * hd.depth * w * w + w * T
    return 2.0 * macs
