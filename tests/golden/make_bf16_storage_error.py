"""Writes bf16_storage_error.json: how far bfloat16 storage alone moves each
full-size parity check away from the fp64 oracle.

    python tests/golden/make_bf16_storage_error.py [workload ...]

For every bf16 workload of the full-size parity plan it follows the sampled
slots (the first and the last) through the same steps as
tests/test_gpu_fullsize.py -- one full step, the plan's cached steps, and
for two-pathway workloads a conditional-only step of slot 0 -- twice: with
the fp64 oracle (oracle.MarOracle) and with the same oracle rounding every
tensor where the GPU path stores it (oracle.storage_emulation).  For each
check it records the emulation's maximum deviation from the oracle and the
number of elements beyond the elementwise bar 2e-2 + 1e-2 |oracle|.

Only oracle/ computes here; the inputs come from the seeded generators.
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import MarOracle  # noqa: E402
from oracle.storage_emulation import StorageEmulation  # noqa: E402
from paper_2503_12450_amd.workload import (FULLSIZE_COND_SEED, FULLSIZE_PLANS, FULLSIZE_STEP_SEED,  # noqa: E402
                                           WORKLOADS, all_block_weights, changed_rows, normal_rows,
                                           to_storage)

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "bf16_storage_error.json")
ATOL, RTOL = 2e-2, 1e-2


def _figures(emu, ref):
    err = np.abs(emu - ref)
    return {"max_err": float(err.max()),
            "beyond": int((err > ATOL + RTOL * np.abs(ref)).sum()),
            "size": int(ref.size),
            "max_abs": float(np.abs(ref).max())}


def workload_figures(name):
    wl = WORKLOADS[name]
    d = wl.dims
    W = all_block_weights(d)
    slots = d.max_slots
    sample = sorted({0, slots - 1})
    orc, emu = MarOracle(d, W), StorageEmulation(d, W)
    out = {}
    x = normal_rows((slots, d.seq_len, d.d_model), seed=1, dtype=d.dtype)
    for b in sample:
        out[f"full step, slot {b}"] = _figures(emu.full_slot(b, x[b]), orc.full_slot(b, x[b]))
    plan = FULLSIZE_PLANS[name]
    for k, n in enumerate(plan):
        nxt, rows = changed_rows(x, n, seed=FULLSIZE_STEP_SEED + 10 * k)
        nxt = to_storage(nxt, d.dtype)
        for b in sample:
            yo, io, _ = orc.cached_slot(b, nxt[b], n)
            ye, ie, _ = emu.cached_slot(b, nxt[b], n)
            if not (np.array_equal(io, ie) and np.array_equal(io, np.sort(rows[b]))):
                raise AssertionError(f"{name}: selection of slot {b} differs at cached step {k}")
            out[f"cached step {k} (N={n}), slot {b}"] = _figures(ye, yo)
        x = nxt
    if slots >= 2 and slots % 2 == 0 and wl.images:
        half = slots // 2
        n = plan[-1]
        nxt, _ = changed_rows(x[:half], n, seed=FULLSIZE_COND_SEED)
        nxt = to_storage(nxt, d.dtype)
        yo, io, _ = orc.cached_slot(0, nxt[0], n)
        ye, ie, _ = emu.cached_slot(0, nxt[0], n)
        if not np.array_equal(io, ie):
            raise AssertionError(f"{name}: selection of the conditional-only step differs")
        out["conditional-only step, slot 0"] = _figures(ye, yo)
    return out


def main(names):
    data = {}
    if os.path.exists(OUT):
        data = json.load(open(OUT))
    data["_about"] = ("bf16 storage rounding alone (oracle.storage_emulation) against the fp64 oracle, "
                      "per check of tests/test_gpu_fullsize.py; written by "
                      "tests/golden/make_bf16_storage_error.py; bar 2e-2 + 1e-2 |oracle|")
    for name in names:
        t0 = time.time()
        data[name] = workload_figures(name)
        worst = max(v["max_err"] for v in data[name].values())
        print(f"{name}: {len(data[name])} checks, worst max err {worst:.4f} ({time.time() - t0:.0f} s)",
              flush=True)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)
            f.write("\n")


if __name__ == "__main__":
    default = [n for n in FULLSIZE_PLANS if WORKLOADS[n].dims.dtype == "bf16"]
    main(sys.argv[1:] or default)
