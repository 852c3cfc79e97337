"""The whole cached step through the C ABI, against the CPU oracle.

Inputs are seeded (weights, this step's input, the previous step's input of
the cache fill).  The oracle runs the same steps in fp64 with a feature
cache; the GPU keeps key/value caches.  Selected indices are compared bit
for bit; block outputs within the storage dtype's tolerance.

Where the selection is decided by similarity computed from values that the
two sides round differently (bf16 products upstream), the inputs are built
so that the decision is well conditioned: the previous step differs from
this one on N rows per slot by O(1) noise, so the N least similar rows are
far from the rest.  The given-rows mode checks the cached blocks on an
arbitrary selection with no such construction.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2503_12450_amd import binding as B
from paper_2503_12450_amd.device import to_device, upload_blocks
from paper_2503_12450_amd.workload import (WORKLOADS, MarDims, all_block_weights, block_weights,
                                           normal_rows, perturbed, random_index_sets, to_storage)

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = {"f32": dict(atol=1e-4, rtol=1e-5), "bf16": dict(atol=2e-2, rtol=1e-2)}


def _host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _make(dims, std=0.02):
    W = [block_weights(dims, l, seed=0, std=std) for l in range(dims.n_layers)]
    cache = B.MarCache(dims, upload_blocks(W, dims.dtype))
    return W, cache


def _gap_inputs(dims, n_slots, n, seed=1):
    """x, and a previous-step input that differs from x on n rows per slot."""
    x = normal_rows((n_slots, dims.seq_len, dims.d_model), seed=seed, dtype=dims.dtype)
    rows = random_index_sets(n_slots, dims.seq_len, n, seed=seed + 10)
    prev = x.copy()
    noise = normal_rows(x.shape, seed=seed + 20)
    for b in range(n_slots):
        prev[b, rows[b]] = to_storage(x[b, rows[b]] + noise[b, rows[b]], dims.dtype)
    return x, prev, rows


def _step(cache, x, mode, n=0, slot0=0, given=None):
    xd = to_device(x, cache.dims.dtype)
    y = torch.empty((x.shape[0], cache.dims.seq_len, cache.dims.d_model), dtype=torch.float32, device=DEV)
    sel = None
    ranked = mode in (B.MAR_TOKEN_CACHED, B.MAR_TOKEN_CACHED_MOST_SIMILAR)
    if ranked:
        sel = torch.full((x.shape[0], max(n, 1)), -1, dtype=torch.int32, device=DEV)
    elif mode == B.MAR_TOKEN_GIVEN:
        sel = given
    cache.step(xd, mode, n, slot0=slot0, y=y, sel_idx=sel)
    torch.cuda.synchronize()
    idx = sel[:, :n].cpu().numpy() if ranked else None
    return y, idx


SMALL = {
    "f32-block-P0": MarDims(1, 768, 12, 3072, 320, 2, 0, "f32"),
    "bf16-stack-P2": MarDims(4, 256, 4, 1024, 100, 4, 2, "bf16"),
    "bf16-dh80-P1": MarDims(3, 320, 4, 1280, 70, 2, 1, "bf16"),
    "bf16-P0": MarDims(2, 128, 2, 512, 65, 2, 0, "bf16"),
    "f32-stack-P1": MarDims(3, 128, 2, 256, 40, 2, 1, "f32"),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_full_then_cached_matches_oracle(name):
    dims = SMALL[name]
    n = max(1, dims.seq_len // 4)
    W, cache = _make(dims)
    x, prev, changed = _gap_inputs(dims, dims.max_slots, n)
    orc = O.MarOracle(dims, W)
    y0, _ = _step(cache, prev, B.MAR_FULL)
    np.testing.assert_allclose(_host(y0), orc.full(prev), **TOL[dims.dtype])
    y1, idx = _step(cache, x, B.MAR_TOKEN_CACHED, n)
    yo, idxo, so = orc.cached(x, n)
    np.testing.assert_array_equal(idx, idxo)
    np.testing.assert_array_equal(idx, np.sort(changed, axis=1))
    np.testing.assert_allclose(_host(y1), yo, **TOL[dims.dtype])
    # the output cache holds the same rows
    np.testing.assert_array_equal(_host(cache.output()[: dims.max_slots]), _host(y1))


def test_config1_noise_selection_matches_oracle():
    """The single fp32 block with the previous step = this step + N(0, 0.05^2)
    on every row (no built-in gap): fp32 values and fp64 scores decide the
    same 80 rows on both sides unless the oracle's threshold gap is below
    what fp32 rounding of the value rows can move."""
    w = WORKLOADS["block-f32"]
    dims, n = w.dims, w.n_recompute
    W, cache = _make(dims)
    x = normal_rows((2, dims.seq_len, dims.d_model), seed=1)
    prev = perturbed(x, seed=2, std=0.05, dtype="f32")
    orc = O.MarOracle(dims, W)
    _step(cache, prev, B.MAR_FULL)
    orc.full(prev)
    y, idx = _step(cache, x, B.MAR_TOKEN_CACHED, n)
    yo, idxo, so = orc.cached(x, n)
    for b in range(2):
        srt = np.sort(so[b])
        gap = srt[n] - srt[n - 1]
        if gap > 1e-9:
            np.testing.assert_array_equal(idx[b], idxo[b])
        else:  # near tie: any valid choice at the threshold
            thr = srt[n - 1]
            assert np.all(so[b][idx[b]] <= thr + 1e-9)
    if np.array_equal(idx, idxo):
        np.testing.assert_allclose(_host(y), yo, **TOL["f32"])


@pytest.mark.parametrize("name", ["f32-block-P0", "bf16-P0"])
def test_most_similar_rule_matches_oracle(name):
    """Table 3's opposite ranking (the n most similar rows computed).  With
    no always-computed block the value rows depend on each token's own input
    only, so the construction is exact: n rows per slot change by small
    noise and all others by large noise, and the n most similar rows are the
    small-noise ones on both sides."""
    dims = SMALL[name]
    n = max(1, dims.seq_len // 5)
    W, cache = _make(dims)
    slots = dims.max_slots
    x = normal_rows((slots, dims.seq_len, dims.d_model), seed=5, dtype=dims.dtype)
    near = random_index_sets(slots, dims.seq_len, n, seed=6)
    small = normal_rows(x.shape, seed=7, std=0.2)
    large = normal_rows(x.shape, seed=8, std=3.0)
    prev = x + large
    for b in range(slots):
        prev[b, near[b]] = x[b, near[b]] + small[b, near[b]]
    prev = to_storage(prev, dims.dtype)
    orc = O.MarOracle(dims, W)
    _step(cache, prev, B.MAR_FULL)
    orc.full(prev)
    y, idx = _step(cache, x, B.MAR_TOKEN_CACHED_MOST_SIMILAR, n)
    yo, idxo, so = orc.cached(x, n, rule="most")
    np.testing.assert_array_equal(idxo, np.sort(near, axis=1))  # the construction is well conditioned
    np.testing.assert_array_equal(idx, idxo)
    np.testing.assert_allclose(_host(y), yo, **TOL[dims.dtype])


@pytest.mark.parametrize("name", ["bf16-stack-P2", "f32-stack-P1", "bf16-P0", "f32-block-P0", "bf16-dh80-P1"])
@pytest.mark.parametrize("option", ["features", "fresh_kv", "both"])
def test_method_options_match_oracle(name, option):
    """Sec. 4.4 alternatives: scoring the features instead of the value rows,
    and recomputing every row's keys/values at block P.  Two cached steps
    after a fill (the second scores against the first's reference)."""
    from dataclasses import replace
    dims = replace(SMALL[name], score_source="features" if option in ("features", "both") else "values",
                   fresh_kv=option in ("fresh_kv", "both"))
    n = max(1, dims.seq_len // 4)
    W, cache = _make(dims)
    x, prev, changed = _gap_inputs(dims, dims.max_slots, n)
    x2, _, changed2 = _gap_inputs(dims, dims.max_slots, n, seed=31)
    # the second step differs from the first on its own n rows
    for b in range(dims.max_slots):
        keep = np.setdiff1d(np.arange(dims.seq_len), changed2[b])
        x2[b, keep] = x[b, keep]
    orc = O.MarOracle(dims, W)
    _step(cache, prev, B.MAR_FULL)
    orc.full(prev)
    for xs, ch in ((x, changed), (x2, changed2)):
        y, idx = _step(cache, xs, B.MAR_TOKEN_CACHED, n)
        yo, idxo, _ = orc.cached(xs, n)
        np.testing.assert_array_equal(idxo, np.sort(ch, axis=1))  # well conditioned
        np.testing.assert_array_equal(idx, idxo)
        np.testing.assert_allclose(_host(y), yo, **TOL[dims.dtype])


@pytest.mark.parametrize("compute", ["decoded", "undecoded"])
def test_token_type_rule_through_given_rows(compute):
    """Table 3's token-type strategies: the host rule picks the rows from the
    sampler's decoded mask, the step computes them as given rows."""
    from paper_2503_12450_amd import selection as SEL
    dims = SMALL["bf16-stack-P2"]
    n = dims.seq_len // 4
    W, cache = _make(dims)
    x, prev, _ = _gap_inputs(dims, dims.max_slots, n)
    decoded = np.random.default_rng(9).random((dims.max_slots, dims.seq_len)) < 0.3
    rows = SEL.observation_rows(decoded, n, compute)
    orc = O.MarOracle(dims, W)
    _step(cache, prev, B.MAR_FULL)
    orc.full(prev)
    y, _ = _step(cache, x, B.MAR_TOKEN_GIVEN, n, given=rows)
    yo, _, _ = orc.cached(x, n, given=rows)
    np.testing.assert_allclose(_host(y), yo, **TOL[dims.dtype])


@pytest.mark.parametrize("name", ["bf16-stack-P2", "f32-stack-P1", "bf16-P0"])
def test_given_rows_match_oracle(name):
    dims = SMALL[name]
    n = dims.seq_len // 3
    W, cache = _make(dims)
    x = normal_rows((dims.max_slots, dims.seq_len, dims.d_model), seed=3, dtype=dims.dtype)
    prev = perturbed(x, seed=4, std=0.5, dtype=dims.dtype)
    given = random_index_sets(dims.max_slots, dims.seq_len, n, seed=5)
    orc = O.MarOracle(dims, W)
    _step(cache, prev, B.MAR_FULL)
    orc.full(prev)
    y, _ = _step(cache, x, B.MAR_TOKEN_GIVEN, n, given=given)
    yo, _, _ = orc.cached(x, n, given=given)
    np.testing.assert_allclose(_host(y), yo, **TOL[dims.dtype])
    # a second cached step keeps using the updated caches
    x2 = perturbed(x, seed=6, std=0.5, dtype=dims.dtype)
    given2 = random_index_sets(dims.max_slots, dims.seq_len, n, seed=7)
    y2, _ = _step(cache, x2, B.MAR_TOKEN_GIVEN, n, given=given2)
    yo2, _, _ = orc.cached(x2, n, given=given2)
    np.testing.assert_allclose(_host(y2), yo2, **TOL[dims.dtype])


# --------------------------------------------------------------------------
# Invariants the GPU path must satisfy bit for bit
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["bf16-stack-P2", "f32-block-P0", "bf16-dh80-P1"])
def test_unchanged_input_reuse_is_bitwise_full(name):
    dims = SMALL[name]
    W, cache = _make(dims)
    x = normal_rows((dims.max_slots, dims.seq_len, dims.d_model), seed=8, dtype=dims.dtype)
    y_full, _ = _step(cache, x, B.MAR_FULL)
    for n in (0, 1, dims.seq_len // 2, dims.seq_len):
        y, idx = _step(cache, x, B.MAR_TOKEN_CACHED, n)
        assert torch.equal(y, y_full), n
        np.testing.assert_array_equal(idx, np.tile(np.arange(n), (dims.max_slots, 1)))


@pytest.mark.parametrize("name", ["bf16-stack-P2", "bf16-P0"])
def test_full_recompute_ratio_is_bitwise_full(name):
    dims = SMALL[name]
    W, cache = _make(dims)
    _, cache2 = _make(dims)
    x = normal_rows((dims.max_slots, dims.seq_len, dims.d_model), seed=9, dtype=dims.dtype)
    prev = perturbed(x, seed=10, std=0.5, dtype=dims.dtype)
    _step(cache, prev, B.MAR_FULL)
    y, idx = _step(cache, x, B.MAR_TOKEN_CACHED, dims.seq_len)
    y_ref, _ = _step(cache2, x, B.MAR_FULL)
    assert torch.equal(y, y_ref)


OPTIONS = {"values": {}, "features": dict(score_source="features"), "fresh_kv": dict(fresh_kv=True),
           "both": dict(score_source="features", fresh_kv=True)}
RANKED = {"least": B.MAR_TOKEN_CACHED, "most": B.MAR_TOKEN_CACHED_MOST_SIMILAR}


@pytest.mark.parametrize("name", ["bf16-stack-P2", "f32-block-P0", "bf16-P0", "bf16-dh80-P1"])
@pytest.mark.parametrize("option", list(OPTIONS))
@pytest.mark.parametrize("rule", list(RANKED))
def test_invariants_hold_for_every_rule_and_option(name, option, rule):
    """With an unchanged input every score is exactly 1 under both sources,
    so both rankings break the tie by index and compute rows 0..n-1, and the
    step equals the full step bit for bit for any n; computing every row
    equals the full step too (fresh keys/values included: the key/value
    product visits k in the same order); n = 0 returns the output cache."""
    from dataclasses import replace
    dims = replace(SMALL[name], **OPTIONS[option])
    mode = RANKED[rule]
    W, cache = _make(dims)
    _, cache2 = _make(dims)
    x = normal_rows((dims.max_slots, dims.seq_len, dims.d_model), seed=12, dtype=dims.dtype)
    y_full, _ = _step(cache, x, B.MAR_FULL)
    for n in (0, 1, dims.seq_len // 3, dims.seq_len):
        y, idx = _step(cache, x, mode, n)
        assert torch.equal(y, y_full), n
        np.testing.assert_array_equal(idx, np.tile(np.arange(n), (dims.max_slots, 1)))
    x2 = perturbed(x, seed=13, std=0.5, dtype=dims.dtype)
    y_all, _ = _step(cache, x2, mode, dims.seq_len)
    y_ref, _ = _step(cache2, x2, B.MAR_FULL)
    assert torch.equal(y_all, y_ref)
    y0, idx0 = _step(cache, x, mode, 0)
    assert torch.equal(y0, y_all) and idx0.shape == (dims.max_slots, 0)


def test_zero_recompute_returns_cache_and_updates_reference():
    dims = SMALL["bf16-stack-P2"]
    W, cache = _make(dims)
    x, prev, _ = _gap_inputs(dims, dims.max_slots, 10)
    y_prev, _ = _step(cache, prev, B.MAR_FULL)
    y0, _ = _step(cache, x, B.MAR_TOKEN_CACHED, 0)
    assert torch.equal(y0, y_prev)
    # the reference now holds this step's value rows: the same x scores 1
    # everywhere, so the first rows win the ties
    _, idx = _step(cache, x, B.MAR_TOKEN_CACHED, 10)
    np.testing.assert_array_equal(idx, np.tile(np.arange(10), (dims.max_slots, 1)))


def test_slot_ranges_are_isolated_and_deterministic():
    dims = MarDims(3, 256, 4, 1024, 80, 6, 1, "bf16")
    W, cache = _make(dims)
    _, cache2 = _make(dims)
    x, prev, _ = _gap_inputs(dims, 6, 12)
    for c in (cache, cache2):
        _step(c, prev, B.MAR_FULL)
    before = cache.output().clone()
    # advance only slots [0, 3) (the conditional pathway of a reuse step)
    ya, idxa = _step(cache, x[:3], B.MAR_TOKEN_CACHED, 12, slot0=0)
    after = cache.output()
    assert torch.equal(after[3:], before[3:])
    # the same call on a second handle gives the same bits
    yb, idxb = _step(cache2, x[:3], B.MAR_TOKEN_CACHED, 12, slot0=0)
    assert torch.equal(ya, yb)
    np.testing.assert_array_equal(idxa, idxb)
    # slots [3, 6) still hold the state of the fill: advancing them now
    # equals advancing them on a handle where slots [0, 3) never moved
    _, cache3 = _make(dims)
    _step(cache3, prev, B.MAR_FULL)
    yc, idxc = _step(cache, x[3:], B.MAR_TOKEN_CACHED, 12, slot0=3)
    yd, idxd = _step(cache3, x[3:], B.MAR_TOKEN_CACHED, 12, slot0=3)
    assert torch.equal(yc, yd)
    np.testing.assert_array_equal(idxc, idxd)


# --------------------------------------------------------------------------
# Condition cache (Eq. 10) and guidance (Eq. 7)
# --------------------------------------------------------------------------

def test_cfg_store_reuse_matches_oracle():
    dims = SMALL["f32-block-P0"]
    _, cache = _make(dims)
    S, D = dims.seq_len, dims.d_model
    c = normal_rows((1, S, D), seed=81)
    u = normal_rows((1, S, D), seed=82)
    c2 = perturbed(c, seed=83, std=0.1, dtype="f32")
    orc = O.MarOracle(dims, [block_weights(dims, 0)])
    g = torch.empty((1, S, D), device=DEV)
    uo = torch.empty((1, S, D), device=DEV)
    with pytest.raises(B.MarError) as e:
        cache.cfg_combine(B.MAR_CFG_REUSE, to_device(c2, "f32"), None, 4.0, g)
    assert e.value.status == B.MAR_E_STATE
    cache.cfg_combine(B.MAR_CFG_STORE, to_device(c, "f32"), to_device(u, "f32"), 4.0, g, uo)
    torch.cuda.synchronize()
    go, _ = orc.cfg("store", c, u, 4.0)
    np.testing.assert_allclose(_host(g), go, atol=1e-5, rtol=1e-6)
    np.testing.assert_array_equal(_host(uo), u)
    cache.cfg_combine(B.MAR_CFG_REUSE, to_device(c2, "f32"), None, 4.0, g, uo)
    torch.cuda.synchronize()
    go2, uh = orc.cfg("reuse", c2, None, 4.0)
    np.testing.assert_allclose(_host(uo), uh, atol=1e-6, rtol=1e-6)
    np.testing.assert_allclose(_host(g), go2, atol=1e-5, rtol=1e-6)
    # scale 0 returns the unconditional output exactly, scale 1 the conditional
    cache.cfg_combine(B.MAR_CFG_STORE, to_device(c, "f32"), to_device(u, "f32"), 0.0, g)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(g), u)


# --------------------------------------------------------------------------
# Host-side errors: nothing is enqueued
# --------------------------------------------------------------------------

def test_errors_leave_state_untouched():
    dims = SMALL["bf16-stack-P2"]
    W, cache = _make(dims)
    x, prev, _ = _gap_inputs(dims, dims.max_slots, 5)
    xd = to_device(x, "bf16")
    with pytest.raises(B.MarError) as e:
        cache.step(xd, B.MAR_TOKEN_CACHED, 5)
    assert e.value.status == B.MAR_E_STATE
    _step(cache, prev, B.MAR_FULL)
    torch.cuda.synchronize()
    before = cache.output().clone()
    bad = [
        dict(mode=7), dict(n_recompute=-1), dict(n_recompute=dims.seq_len + 1),
        dict(slot0=3), dict(slot0=-1),
    ]
    for kw in bad:
        args = dict(mode=B.MAR_TOKEN_CACHED, n_recompute=5, slot0=0)
        args.update(kw)
        with pytest.raises(B.MarError) as e:
            cache.step(xd, args["mode"], args["n_recompute"], slot0=args["slot0"])
        assert e.value.status == B.MAR_E_ARG, kw
    for given in (np.array([[3, 2, 5, 7, 9]] * 4), np.array([[0, 1, 2, 3, 100]] * 4),
                  np.array([[1, 1, 2, 3, 4]] * 4)):
        with pytest.raises(B.MarError) as e:
            cache.step(xd, B.MAR_TOKEN_GIVEN, 5, sel_idx=given)
        assert e.value.status == B.MAR_E_ARG
    torch.cuda.synchronize()
    assert torch.equal(cache.output(), before)
    mis = xd.view(torch.uint8)[..., 1:]  # data pointer one byte off
    with pytest.raises(B.MarError) as e:
        cache.step(mis, B.MAR_FULL)
    assert e.value.status == B.MAR_E_ARG


# --------------------------------------------------------------------------
# Graph capture: a step is a fixed sequence of launches on the caller's
# stream with no allocation, so serving loops can capture it once
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mode", [B.MAR_TOKEN_CACHED, B.MAR_TOKEN_CACHED_MOST_SIMILAR])
def test_captured_step_replays_like_eager_steps(mode):
    """A cached step captured in a HIP graph, replayed three times with eager
    work and synchronisation in between, gives bit for bit what three eager
    calls give on a twin handle (each replay rescored against the reference
    the previous one left)."""
    dims = SMALL["bf16-stack-P2"]
    n = dims.seq_len // 4
    W, eager = _make(dims)
    _, graphed = _make(dims)
    x, prev, _ = _gap_inputs(dims, dims.max_slots, n)
    xd = to_device(x, dims.dtype)
    pd = to_device(prev, dims.dtype)
    shape = (dims.max_slots, dims.seq_len, dims.d_model)
    want = []
    eager.step(pd, B.MAR_FULL)
    for _ in range(3):
        y = torch.empty(shape, dtype=torch.float32, device=DEV)
        sel = torch.empty((dims.max_slots, n), dtype=torch.int32, device=DEV)
        eager.step(xd, mode, n, y=y, sel_idx=sel)
        want.append((y, sel))
    torch.cuda.synchronize()

    graphed.step(pd, B.MAR_FULL)
    y_g = torch.empty(shape, dtype=torch.float32, device=DEV)
    sel_g = torch.empty((dims.max_slots, n), dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.step(xd, mode, n, y=y_g, sel_idx=sel_g)
    for k in range(3):
        y_g.fill_(-7.0)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(sel_g, want[k][1]), k
        assert torch.equal(y_g, want[k][0]), k


def test_profiler_counts_the_class_launches_and_their_work():
    """A session around one full step times exactly the class's launches
    (fc1: one per block) and sums their algorithmic FLOPs (2 M F D each);
    stopping without a session is a state error."""
    dims = SMALL["bf16-stack-P2"]
    W, cache = _make(dims)
    x = normal_rows((dims.max_slots, dims.seq_len, dims.d_model), seed=14, dtype=dims.dtype)
    with pytest.raises(B.MarError) as e:
        cache.profile_stop()
    assert e.value.status == B.MAR_E_STATE
    cache.profile_start("fc1")
    _step(cache, x, B.MAR_FULL)
    ms, launches, flops, nbytes = cache.profile_stop()
    M = dims.max_slots * dims.seq_len
    assert launches == dims.n_layers
    assert flops == pytest.approx(dims.n_layers * 2.0 * M * dims.d_mlp * dims.d_model, rel=1e-12)
    assert ms > 0.0 and nbytes > 0.0
    # a class that the step does not launch on this path times nothing
    cache.profile_start("select")
    _step(cache, x, B.MAR_FULL)
    assert cache.profile_stop()[1] == 0
