"""Comparison rules for GPU-vs-oracle parity.

Logits: row-wise relative error  max_v |g_v - o_v| / max_v |o_v|  <= tol
(tol = 1e-4 for fp32 models, 2e-2 for bf16 models).

Tokens (greedy head decoding): the GPU's token must equal the oracle's argmax
except where the oracle's top-2 gap is below tol * max_v |o_v| (a near-tie,
where two logits within tolerance can swap).  Near-ties are counted and
reported; so are gaps below 2 * tol * s_r.
"""
from __future__ import annotations

import numpy as np

import oracle as O

TOL = {0: 1e-4, 1: 2e-2}  # by dtype (0 fp32, 1 bf16)


def compare_head(gpu_logits: np.ndarray, orc_logits: np.ndarray, gpu_tokens, tol: float,
                 where: str = "") -> dict:
    g = np.asarray(gpu_logits, np.float64)
    o = np.asarray(orc_logits, np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    s = np.abs(o).max(axis=1)
    rel = np.abs(g - o).max(axis=1) / s
    assert np.all(rel <= tol), f"{where}: logit rel err {rel.max():.3e} > {tol}"
    top = np.sort(o, axis=1)
    gap = top[:, -1] - top[:, -2]
    near = gap < tol * s
    near2 = gap < 2 * tol * s
    want = O.argmax(o)
    got = np.asarray(gpu_tokens).reshape(-1)
    bad = (got != want) & ~near
    assert not bad.any(), (f"{where}: token mismatch at rows {np.nonzero(bad)[0].tolist()} "
                           f"gpu={got[bad].tolist()} oracle={want[bad].tolist()}")
    return dict(rows=len(s), max_rel=float(rel.max()), near=int(near.sum()),
                near2=int(near2.sum()), mismatch_near=int(((got != want) & near).sum()))


def merge(stats: list) -> dict:
    out = dict(rows=0, max_rel=0.0, near=0, near2=0, mismatch_near=0)
    for s in stats:
        out["rows"] += s["rows"]
        out["max_rel"] = max(out["max_rel"], s["max_rel"])
        for k in ("near", "near2", "mismatch_near"):
            out[k] += s[k]
    return out


# Merged statistics of every parity configuration run in this session, by
# name: the near-tie counts the tolerance rule exempts are part of the result
# (tests/conftest.py prints them after the run and writes them to the JSON
# file named by KF_PARITY_STATS, when set).
RECORDED: dict = {}


def report(name: str, stats: dict) -> dict:
    """Print and record the merged statistics of one parity configuration."""
    RECORDED[name] = dict(stats)
    print(f"{name}: {stats}", flush=True)
    return stats
