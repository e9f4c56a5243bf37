"""GPU parity of the training-mask attention (Appendix C.2: SingleForward M_S
and DoubleForward M_D) through kf_training_attention, against the oracle's
plain masked attention (fp64) on the same bfloat16 inputs.

Tolerance: the kernel takes bf16 inputs exactly, forms scores and the softmax
in fp32, rounds the probabilities to bf16 for the P.V product (relative error
<= 2^-9 per term, so <= 2^-9 * max|v| on the weighted mean) and the output to
bf16 (<= 2^-9 |o|).  With |v| <= ~5 for these N(0, 1) draws that is < 1.2e-2;
the test asks |gpu - oracle| <= 1.2e-2 + 2^-8 |oracle|.
"""
import sys

import numpy as np
import pytest

import kf_synth as S
import oracle as O

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ATOL, RTOL = 1.2e-2, 2.0 ** -8
KIND = {0: "single", 1: "double"}


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bd():
    from paper_2606_10820_amd import binding as Bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return Bd


def _run(Bd, mask, q, k_, v, N, k, scale):
    dev = torch.device("cuda:0")
    tq, tk, tv = (torch.from_numpy(a).to(dev).to(torch.bfloat16).contiguous() for a in (q, k_, v))
    out = Bd.training_attention(mask, tq, tk, tv, N, k, scale)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


def _check(got, ref, where):
    err = np.abs(got - ref)
    bound = ATOL + RTOL * np.abs(ref)
    worst = float((err / bound).max())
    _log(f"{where}: max |err| {err.max():.3e}, worst err/bound {worst:.3f}")
    assert np.isfinite(got).all(), where
    assert worst <= 1.0, where


# (mask, B, H, N, k, d_head, std): ragged row counts (not multiples of the
# 64-row workgroup), k = 1 (one token per group), odd k = 5 (the kernel's
# division of row indices by k), N = 1, every d_head, and peaked softmax rows
# (std 2: scores ~ N(0, 16))
CASES = [
    (0, 2, 3, 37, 3, 64, 1.0),
    (1, 2, 3, 37, 3, 64, 1.0),
    (0, 1, 2, 50, 1, 32, 1.0),
    (1, 1, 2, 50, 1, 32, 1.0),
    (0, 1, 2, 64, 4, 128, 1.0),
    (1, 1, 2, 64, 4, 128, 1.0),
    (0, 2, 2, 1, 4, 64, 1.0),
    (1, 2, 2, 1, 4, 64, 1.0),
    (0, 1, 3, 129, 2, 64, 2.0),
    (1, 1, 3, 129, 2, 64, 2.0),
    (0, 1, 1, 200, 4, 64, 1.0),
    (1, 1, 1, 200, 4, 64, 1.0),
    (0, 1, 2, 70, 5, 64, 1.0),
    (1, 1, 2, 70, 5, 64, 1.0),
    (0, 1, 2, 90, 1, 64, 1.0),
    (1, 1, 2, 90, 1, 64, 1.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s_B%d_H%d_N%d_k%d_dh%d_s%g" % (
    KIND[c[0]], *c[1:]))
def test_training_attention_parity(case):
    Bd = _bd()
    mask, B, H, N, k, dh, std = case
    rows, keys = Bd.training_attention_shapes(mask, N, k)
    _log(f"case {case}: rows {rows} keys {keys}")
    q, k_, v = S.attention_batch(11 + N, B, H, rows, keys, dh, std)
    scale = dh ** -0.5
    got = _run(Bd, mask, q, k_, v, N, k, scale)
    ref = O.masked_attention(q, k_, v, O.training_mask(KIND[mask], N, k), scale)
    _check(got, ref, f"{KIND[mask]} N={N} k={k} dh={dh}")


def test_empty_problem_launches_nothing():
    Bd = _bd()
    L = Bd.lib()
    s = torch.cuda.current_stream().cuda_stream
    for mask in (0, 1):
        assert L.kf_training_attention(s, mask, 0, 12, 8, 4, 64, None, None, None, None, 0.125) == 0
        assert L.kf_training_attention(s, mask, 2, 12, 0, 4, 64, None, None, None, None, 0.125) == 0


@pytest.mark.parametrize("mask", [0, 1], ids=["single", "double"])
def test_owt_training_shape_sampled(mask):
    """One GPU's share of an OWT training batch (512 sequences over 8 GPUs):
    B = 64, H = 12, N = 1024 context tokens, k = 4, d_head = 64, the launch the
    benchmark times.  Sampled (sequence, head) slices and rows are checked
    against the oracle: first and last rows, rows on both sides of each
    64-row workgroup edge near the region boundaries, and random rows."""
    Bd = _bd()
    B, H, N, k, dh = 64, 12, 1024, 4, 64
    rows, keys = Bd.training_attention_shapes(mask, N, k)
    dev = torch.device("cuda:0")
    _log(f"owt {KIND[mask]}: filling inputs [{B}][{H}][{rows}/{keys}][{dh}]")
    tq = torch.empty((B, H, rows, dh), dtype=torch.bfloat16, device=dev)
    tk = torch.empty((B, H, keys, dh), dtype=torch.bfloat16, device=dev)
    tv = torch.empty((B, H, keys, dh), dtype=torch.bfloat16, device=dev)
    seed = 5
    for b in range(B):
        for h in range(H):
            q, k_, v = S.attention_inputs(seed, b, h, rows, keys, dh)
            tq[b, h].copy_(torch.from_numpy(q))
            tk[b, h].copy_(torch.from_numpy(k_))
            tv[b, h].copy_(torch.from_numpy(v))
    scale = dh ** -0.5
    _log("launch")
    out = Bd.training_attention(mask, tq, tk, tv, N, k, scale)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all().item()
    full_mask = O.training_mask(KIND[mask], N, k)
    rng = np.random.default_rng(7)
    edges = [0, rows - 1, N - 1, N, N * k - 1, N * k, rows // 2]
    sel = sorted({min(max(r + d, 0), rows - 1) for r in edges for d in (-1, 0, 1)}
                 | set(rng.integers(0, rows, 24).tolist()))
    for b, h in [(0, 0), (B - 1, H - 1), (37, 5)]:
        q, k_, v = S.attention_inputs(seed, b, h, rows, keys, dh)
        ref = O.masked_attention(q[None, None, sel], k_[None, None], v[None, None],
                                 full_mask[sel], scale)[0, 0]
        got = out[b, h, sel].float().cpu().numpy()
        _check(got, ref, f"owt {KIND[mask]} b={b} h={h} ({len(sel)} rows)")
