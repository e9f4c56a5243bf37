"""Pins for the CPU oracle: what the paper and the mathematics fix, independent
of the oracle's own code.

Each test names the passage it checks.  A plausible slip in the oracle (a
dropped bias, a transposed weight, a wrong mask offset, a position off by one,
a cache that keeps noise K/V, a >= instead of > in the inverse CDF) fails at
least one of them.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import kf_synth as S
import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")

# a small model for brute force: 2 layers, d=64, 4 heads, MLP 128, V=96, n_ctx=64
SMALL = S.ModelConfig(2, 64, 4, 128, 96, 64, S.DTYPE_FP32)


def _blob(cfg, seed=0, affine=True):
    return S.pack_blob(cfg, S.make_weights(cfg, seed=seed, random_affine=affine))


@pytest.fixture(scope="module")
def small():
    blob = _blob(SMALL)
    return blob, O.Model(blob)


@pytest.fixture(scope="module")
def toy():
    w = S.WORKLOADS["toy"]
    blob = _blob(w["cfg"], affine=True)
    return blob, O.Model(blob)


# ------------------------------------------------------------------ Philox

def test_oracle_philox_kat():
    """Salmon et al. SC'11 known-answer vectors (tests/golden)."""
    for line in open(os.path.join(GOLD, "philox4x32_10_kat.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        assert list(O.philox4x32_10(w[:4], w[4:6])) == w[6:10]


# --------------------------------------------------------- inverse CDF

def _frac(s):
    return Fraction(s)


def _appB():
    cond, regions, mass = {}, [], {}
    for line in open(os.path.join(GOLD, "appB_pushforward_example.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = line.split()
        if w[0] == "cond":
            cond[w[1]] = [_frac(x) for x in w[2:5]]
        elif w[0] == "region":
            regions.append(([_frac(x) for x in w[1:5]], (w[5], w[6])))
        elif w[0] == "mass":
            mass[(w[1], w[2])] = _frac(w[3])
    return cond, regions, mass


NAMES = "ABC"


def _gstar(cond, z1, z2):
    q1 = [float(x) for x in cond["sos"]]
    a = NAMES[O.icdf(q1, z1)]
    b = NAMES[O.icdf([float(x) for x in cond[a]], z2)]
    return a, b


def test_appendix_b_regions():
    """Appendix B example: the unrolled inverse-CDF map partitions [0,1)^2 into
    the three printed regions; interior points and the boundary points
    z1 = 1/3, z2 = 1/2 (which belong to the right-hand interval)."""
    cond, regions, _ = _appB()
    rng = np.random.default_rng(0)
    for (z1lo, z1hi, z2lo, z2hi), want in regions:
        for _ in range(200):
            z1 = float(z1lo) + (float(z1hi) - float(z1lo)) * rng.random()
            z2 = float(z2lo) + (float(z2hi) - float(z2lo)) * rng.random()
            assert _gstar(cond, z1, z2) == want
        # the lower corner belongs to the region (half-open intervals)
        assert _gstar(cond, float(z1lo), float(z2lo)) == want
    assert _gstar(cond, 1 / 3, 0.0) == ("B", "A")
    assert _gstar(cond, 1 / 3, 0.5) == ("B", "C")
    assert _gstar(cond, 0.0, 0.0) == ("A", "B")   # never the zero-probability A after A


def _measure(q, v):
    """Lebesgue measure of {z in [0,1): icdf(q, z) == v}, found by bisection on
    the black-box map (the map is monotone non-decreasing in z)."""
    def first_at_least(target):
        lo, hi = 0.0, 1.0
        if O.icdf(q, 0.0) >= target:
            return 0.0
        for _ in range(80):
            mid = 0.5 * (lo + hi)
            if O.icdf(q, mid) >= target:
                hi = mid
            else:
                lo = mid
        return hi
    a = first_at_least(v)
    b = first_at_least(v + 1) if v + 1 < len(q) else 1.0
    return max(0.0, b - a)


def test_appendix_b_masses():
    """Each region has mass 1/3 (Appendix B)."""
    cond, _, mass = _appB()
    q1 = [float(x) for x in cond["sos"]]
    for (a, b), m in mass.items():
        ma = _measure(q1, NAMES.index(a))
        mb = _measure([float(x) for x in cond[a]], NAMES.index(b))
        assert abs(ma * mb - float(m)) < 1e-12


def test_icdf_pushes_uniform_to_q():
    """Standard result stated in Appendix B: with z ~ U(0,1), the inverse-CDF
    map samples q.  Checked on random q including zero-probability tokens."""
    rng = np.random.default_rng(1)
    for trial in range(20):
        V = int(rng.integers(2, 9))
        q = rng.random(V)
        q[rng.random(V) < 0.3] = 0.0
        if q.sum() == 0:
            q[0] = 1.0
        q = q / q.sum()
        for v in range(V):
            assert abs(_measure(list(q), v) - q[v]) < 1e-12


def test_gstar_reproduces_ar_joint():
    """Eq. (correctness): the sequential inverse-CDF map reproduces the AR
    joint p(v1..vk) = prod_j q(v_j | prefix).  A context-dependent random table
    model, V = 3, k = 3; the measure of each output block is computed from the
    black-box map and compared with the chain rule."""
    rng = np.random.default_rng(2)
    V, k = 3, 3
    table = {}

    def cond(prefix):
        if prefix not in table:
            q = rng.random(V) + 0.05
            table[prefix] = q / q.sum()
        return table[prefix]

    total = 0.0
    for seq in np.ndindex(*(V,) * k):
        meas, chain = 1.0, 1.0
        for j in range(k):
            q = cond(tuple(seq[:j]))
            meas *= _measure(list(q), seq[j])
            chain *= q[seq[j]]
        assert abs(meas - chain) < 1e-12
        total += meas
    assert abs(total - 1.0) < 1e-12


# ------------------------------------------------------------- mask counts

def _counts():
    nnz, nfe, params = [], [], []
    for line in open(os.path.join(GOLD, "paper_counts.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = line.split()
        if w[0] == "nnz":
            nnz.append(tuple(int(x) for x in w[1:5]))
        elif w[0] == "nfe":
            nfe.append((w[1], int(w[2]), int(w[3])))
        elif w[0] == "params":
            params.append((w[1], int(w[2]), int(w[3]), int(w[4])))
    return nnz, nfe, params


def test_mask_nnz_closed_forms():
    """Appendix C.2 cost analysis: the mask builders used by the brute force
    have exactly |M_S| and |M_D| non-zeros."""
    nnz, _, _ = _counts()
    for N, k, ms, md in nnz:
        M, _, _ = O.single_forward_layout(N, k)
        assert int(M.sum()) == ms == O.nnz_single(N, k)
        MD, _ = O.double_forward_layout(N, k)
        f2 = slice(N + N * k, N + 2 * N * k)
        assert int(MD[f2].sum()) == md == O.nnz_double(N, k)
    for N in range(1, 9):
        for k in range(1, 5):
            M, _, _ = O.single_forward_layout(N, k)
            assert int(M.sum()) == O.nnz_single(N, k)
            MD, _ = O.double_forward_layout(N, k)
            assert int(MD[N + N * k:].sum()) == O.nnz_double(N, k)
            # F1 rows of M_D are the noise rows of M_S (same staircase + block-causal)
            assert int(MD[N:N + N * k].sum()) == int(M[N:].sum())


def test_table4_backbone_size():
    """Table 4: ~124 M (OWT) / ~108 M (LM1B) parameters.  The counts match only
    with the head tied to the token table; checked on the blob layout without
    the noise encoder (the paper lists it separately)."""
    _, _, params = _counts()
    for name, V, T, pm in params:
        cfg = S.ModelConfig(12, 768, 12, 3072, V, T, S.DTYPE_BF16)
        noise = 4 * 768 * 768 * 2 + 4 * 768 + 768
        got = (S.n_params(cfg) - noise) / 1e6
        assert abs(got - pm) / pm < 0.01, (name, got)


# -------------------------------------------------------------- components

def test_components_textbook():
    d = 16
    rng = np.random.default_rng(3)
    g, b = rng.normal(size=d), rng.normal(size=d)
    # LayerNorm of a constant vector is the shift beta
    np.testing.assert_allclose(O.layernorm(np.full(d, 3.25), g, b), b, atol=0, rtol=0)
    # LayerNorm output has zero mean / unit variance before the affine map
    x = rng.normal(size=d) * 5 + 2
    y = O.layernorm(x, np.ones(d), np.zeros(d))
    assert abs(y.mean()) < 1e-12 and abs((y ** 2).mean() - 1) < 1e-5
    # GELU
    assert O.gelu(0.0) == 0.0
    assert abs(O.gelu(12.0) - 12.0) < 1e-12 and abs(O.gelu(-12.0)) < 1e-12
    for x in np.linspace(-6, 6, 241):
        exact = 0.5 * x * (1 + math.erf(x / math.sqrt(2)))
        assert abs(O.gelu(x) - exact) < 1e-3   # tanh form vs erf form
    # sinusoid(0) = [1..1, 0..0]; each (cos, sin) pair on the unit circle
    e = O.sinusoid(0.0, 64)
    np.testing.assert_array_equal(e, np.r_[np.ones(32), np.zeros(32)])
    e = O.sinusoid(0.7316, 64)
    np.testing.assert_allclose(e[:32] ** 2 + e[32:] ** 2, 1.0, atol=1e-14)
    assert abs(e[0] - math.cos(731.6)) < 1e-12          # frequency 1 at i = 0
    assert abs(e[31] - math.cos(731.6 * 10000 ** (-31 / 32))) < 1e-12
    # attention: one key returns its value; equal scores average the values
    q = rng.normal(size=8)
    K, Vv = rng.normal(size=(1, 8)), rng.normal(size=(1, 8))
    o, s = O.attend(q, K, Vv)
    np.testing.assert_allclose(o, Vv[0], rtol=0, atol=1e-15)
    K, Vv = rng.normal(size=(5, 8)), rng.normal(size=(5, 8))
    o, s = O.attend(np.zeros(8), K, Vv)
    np.testing.assert_allclose(o, Vv.mean(0), atol=1e-15)
    assert abs(s - 1) < 1e-15
    # softmax weights: scaled dot products, 1/sqrt(dh)
    K = np.eye(8)[:2] * 4.0
    Vv = np.array([[1.0] * 8, [0.0] * 8])
    q = np.eye(8)[0]
    o, _ = O.attend(q, K, Vv)
    w = 1 / (1 + math.exp(-4.0 / math.sqrt(8)))
    assert abs(o[0] - w) < 1e-14
    # bf16 round-to-nearest-even
    assert O.round_bf16(1.0 + 2 ** -8) == 1.0
    assert O.round_bf16(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6
    assert O.round_bf16(1.0 + 2 ** -8 + 2 ** -20) == 1.0 + 2 ** -7
    # greedy decoding: ties to the lowest id
    assert list(O.argmax(np.array([[0.0, 2.0, 2.0, 1.0]]))) == [1]


def test_zero_head_weights_all_tie(small):
    """A zero token table gives all-zero logits and token 0 everywhere."""
    w = S.make_weights(SMALL, seed=4, random_affine=True)
    w["tok_emb"][:] = 0.0
    m = O.Model(S.pack_blob(SMALL, w))
    s, logits, toks = O.prefill(m, [1, 2, 3], [0.1, 0.6])
    assert np.all(logits == 0) and list(toks) == [0, 0]


# ------------------------------------------------- (a) k = 1 and prefixes

def test_prefix_consistency(small):
    """Fully causal design (Sec. 3.3): the j-th output depends only on the
    context and z_1..z_j, so outputs 1..j of a k-block equal a j-block's."""
    _, m = small
    prompt = [5, 17, 3, 90, 44, 2]
    u = [0.13, 0.77, 0.41, 0.93]
    s4, l4, t4 = O.prefill(m, prompt, u)
    for j in (1, 2, 3):
        sj, lj, tj = O.prefill(m, prompt, u[:j])
        np.testing.assert_array_equal(lj, l4[:j])
    # decode-step prefixes
    base = m.seq(); base.step(prompt, [0.5], commit=True)
    a = m.seq(); a.step(prompt, [0.5], commit=True)
    l4, _ = base.step([7, 8, 9, 10], [0.2, 0.5, 0.8, 0.3], commit=False)
    for j in (1, 2, 3):
        lj, _ = a.step([7, 8, 9, 10], [0.2, 0.5, 0.8, 0.3][:j], commit=False)
        np.testing.assert_array_equal(lj, l4[:j])


def test_k1_commits_like_ar(small):
    """(a) k = 1: each step commits one position, and the cache equals the one
    an ordinary causal KV-cached AR decode builds from the same tokens."""
    _, m = small
    prompt = [4, 8, 15, 16, 23, 42]
    kf, ar = m.seq(), m.seq()
    lk, _ = kf.step(prompt, [0.31], commit=True)
    ar.step(prompt, [], commit=True)
    pending = list(O.argmax(lk))
    rng = np.random.default_rng(5)
    for step in range(8):
        lk, _ = kf.step(pending, [float(rng.random())], commit=True)
        ar.step(pending, [], commit=True)
        assert kf.C == ar.C == len(prompt) + step + 1
        pending = list(O.argmax(lk))
    for l in range(m.n_layer):
        for which in (0, 1):
            np.testing.assert_array_equal(kf.kv(l, which), ar.kv(l, which))


def _dense_ar_logits(cfg, W, seq):
    n = len(seq)
    M = np.tril(np.ones((n, n), bool))
    return O.dense_forward(cfg, W, [("tok", t) for t in seq], list(range(n)), M)[-1]


def test_ar_mode_is_sequential_icdf(small):
    """(a) AR mode equals the closed-form map G* (Eq. sequential-icdf) built
    from the dense no-cache forward pass and a numpy inverse CDF."""
    blob, m = small
    cfg, W = O.parse_blob(blob)
    prompt = np.array([[3, 1, 4, 1, 5]], np.int32)
    seed = 11
    got = O.generate_ar(m, prompt, 10, seed)[0]
    seq = list(prompt[0])
    for p in range(5, 15):
        lg = _dense_ar_logits(cfg, W, seq)
        q = np.exp(lg - lg.max()); q /= q.sum()
        F = np.cumsum(q)
        z = O.noise_u(seed, 0, p)
        assert np.min(np.abs(F - z)) > 1e-9
        want = int(np.argmax(F > z))
        assert got[p - 5] == want
        seq.append(want)


# ------------------------------------------- (b) incremental == recompute

def test_incremental_equals_full_recompute(toy):
    """(b) Appendix C.1: the cached decode equals a no-cache forward over
    [prompt, emitted tokens, k noise rows] -- bitwise in the oracle, since
    every row's arithmetic is the same in both modes."""
    _, m = toy
    w = S.WORKLOADS["toy"]
    prompt = S.prompts_uniform(1, 1, 16, 1024)[0]
    k, seed = 4, 2
    s = m.seq()
    history = list(prompt)
    pending = list(prompt)
    p = 16
    for step in range(6):
        u = [O.noise_u(seed, 0, p + j) for j in range(k)]
        lg, _ = s.step(pending, u, commit=True)
        full = O.full_recompute(m, history, u)
        np.testing.assert_array_equal(lg, full)
        toks = list(O.argmax(lg))
        history += toks
        pending = toks
        p += k


# ------------------------------------------------------------ (c) causality

def test_causality_noise(small):
    """(c) Perturbing z_j leaves outputs before j unchanged (Sec. 3.3)."""
    _, m = small
    prompt = [9, 8, 7, 6]
    u = [0.1, 0.2, 0.3, 0.4]
    _, base, _ = O.prefill(m, prompt, u)
    for j in range(4):
        v = list(u); v[j] = 0.9
        _, pert, _ = O.prefill(m, prompt, v)
        np.testing.assert_array_equal(pert[:j], base[:j])
        assert np.max(np.abs(pert[j] - base[j])) > 0


def test_causality_prompt(small):
    """(c) Perturbing the prompt token at position p leaves earlier rows and
    their committed K/V unchanged."""
    _, m = small
    prompt = [9, 8, 7, 6, 5, 4]
    a, b = m.seq(), m.seq()
    _, _, ha = a.step(prompt, [0.5, 0.25], commit=True, want_hidden=True)
    pert = list(prompt); pert[3] = 60
    _, _, hb = b.step(pert, [0.5, 0.25], commit=True, want_hidden=True)
    np.testing.assert_array_equal(ha[:3], hb[:3])
    assert np.max(np.abs(ha[3] - hb[3])) > 0
    for l in range(m.n_layer):
        np.testing.assert_array_equal(a.kv(l, 0)[:3], b.kv(l, 0)[:3])
        np.testing.assert_array_equal(a.kv(l, 1)[:3], b.kv(l, 1)[:3])


def test_noise_kv_discarded(small):
    """(c) Appendix C.1 cache rule: noise K/V are dropped, so a different noise
    block at step s (with the same emitted tokens fed back) leaves step s+1
    unchanged."""
    _, m = small
    prompt = [1, 2, 3, 4, 5]
    a, b = m.seq(), m.seq()
    a.step(prompt, [0.1, 0.2, 0.3], commit=True)
    b.step(prompt, [0.9, 0.8, 0.7], commit=True)
    forced = [11, 12, 13]
    la, _ = a.step(forced, [0.5, 0.6, 0.7], commit=True)
    lb, _ = b.step(forced, [0.5, 0.6, 0.7], commit=True)
    np.testing.assert_array_equal(la, lb)
    assert a.C == b.C == 8


# ------------------------------------------------------- (d) softmax sums

def test_softmax_rows_sum_to_one(toy):
    _, m = toy
    s = m.seq()
    lg, dev = s.step(list(range(16)), [0.1, 0.2, 0.3, 0.4], commit=True)
    assert dev < 1e-12
    lg, dev = s.step([1, 2, 3, 4], [0.5, 0.6, 0.7, 0.8], commit=True)
    assert dev < 1e-12
    q = O.softmax(lg[0])
    assert abs(q.sum() - 1) < 1e-12 and (q >= 0).all()


# ---------------------------------------------------- (e) dense brute force

def _check_single_forward(blob, m, N, k, rng, tol=1e-10):
    cfg, W = O.parse_blob(blob)
    x = [int(t) for t in rng.integers(0, cfg["V"], N)]
    z = rng.random((N, k))
    M, pos, grp = O.single_forward_layout(N, k)
    rows = [("tok", t) for t in x] + [("noise", float(z[t, j])) for t in range(N) for j in range(k)]
    dense = O.dense_forward(cfg, W, rows, pos, M)
    outs = {}
    for t in range(1, N + 1):
        s, lg, toks = O.prefill(m, x[:t], z[t - 1])
        ref = dense[N + (t - 1) * k:N + t * k]
        scale = np.abs(ref).max()
        assert np.max(np.abs(lg - ref)) <= tol * scale, (t, np.max(np.abs(lg - ref)) / scale)
        outs[t] = (s, list(toks))
    return cfg, W, x, outs


def test_single_forward_brute_force(small):
    """(e) SingleForward (Appendix C.2): one dense-masked pass over N context
    tokens and N*k noise tokens equals, group by group, the oracle's prefill of
    x_1..x_t with that group's noise."""
    blob, m = small
    _check_single_forward(blob, m, N=6, k=3, rng=np.random.default_rng(6))


def test_double_forward_brute_force(small):
    """(e) DoubleForward (Appendix C.2): the Future-2 outputs of the fused
    two-round mask equal the oracle's decode step that feeds the first round's
    tokens as real rows after a prefill of x_1..x_t."""
    blob, m = small
    N, k = 5, 3
    rng = np.random.default_rng(7)
    cfg, W, x, outs = _check_single_forward(blob, m, N, k, rng)
    z2 = rng.random((N, k))
    MD, pos = O.double_forward_layout(N, k)
    rows = [("tok", t) for t in x]
    rows += [("tok", outs[t][1][j]) for t in range(1, N + 1) for j in range(k)]
    rows += [("noise", float(z2[t - 1, j])) for t in range(1, N + 1) for j in range(k)]
    dense = O.dense_forward(cfg, W, rows, pos, MD)
    for t in range(1, N + 1):
        s, _ = outs[t]
        lg, _ = O.decode(s, outs[t][1], z2[t - 1])
        ref = dense[N + N * k + (t - 1) * k:N + N * k + t * k]
        assert np.max(np.abs(lg - ref)) <= 1e-10 * np.abs(ref).max()


def test_brute_force_bf16_weights():
    """(e) with a bf16 model: both the C oracle and the numpy brute force round
    2-D tensors to bf16; a mismatch in that rule shows here."""
    cfg = S.ModelConfig(2, 64, 4, 128, 96, 64, S.DTYPE_BF16)
    blob = _blob(cfg, seed=9)
    _check_single_forward(blob, O.Model(blob), N=4, k=2, rng=np.random.default_rng(8))


def test_toy_config_brute_force(toy):
    """(e) on the 2-layer toy configuration itself (d=128, 4 heads, V=1024)."""
    blob, m = toy
    _check_single_forward(blob, m, N=4, k=4, rng=np.random.default_rng(10))


# --------------------------------------------------------------- NFE

def test_nfe_counts(small):
    """Table 3: NFE = new tokens / k with the prefill as the first pass."""
    _, nfe, _ = _counts()
    for _, k, want in nfe:
        assert 960 // k == want
    _, m = small
    prompt = np.array([[1, 2, 3]], np.int32)
    for k in (1, 2, 4):
        toks, passes = O.generate(m, prompt, 8, k, seed=3)
        assert passes == 8 // k and toks.shape == (1, 8)


def test_generate_matches_manual_steps(small):
    """The generation driver feeds each block's argmax back as the next real
    rows and draws u by absolute position (noise stream 2)."""
    _, m = small
    prompt = np.array([[5, 6, 7, 8]], np.int32)
    toks, _ = O.generate(m, prompt, 6, 3, seed=21)
    s, lg, t = O.prefill(m, prompt[0], [O.noise_u(21, 0, 4 + j) for j in range(3)])
    lg2, t2 = O.decode(s, t, [O.noise_u(21, 0, 7 + j) for j in range(3)])
    assert list(toks[0]) == list(t) + list(t2)


def test_generate_batched_equals_generate(toy):
    """The batched driver (one orc_step_batch call per block, OpenMP over
    sequences), which the CPU baseline times, emits exactly the tokens of
    generate() on the toy workload, in both instantiations."""
    blob, m = toy
    w = S.WORKLOADS["toy"]
    prompt = S.prompts_uniform(1, w["B"], w["N"], w["cfg"].vocab)
    for model in (m, O.Model(blob, "f32")):
        want, passes = O.generate(model, prompt, w["L"], w["k"], seed=9)
        got = O.generate_batched(model, prompt, w["L"], w["k"], seed=9)
        assert passes == w["L"] // w["k"]
        assert np.array_equal(got, want)


def test_step_independent_of_thread_count(toy):
    """The row loops of a step run over OpenMP threads; each row is computed in
    the same order whatever the thread count, so logits and the committed
    cache are identical bit for bit with one thread and with several."""
    import ctypes
    _, m = toy
    gomp = ctypes.CDLL("libgomp.so.1")
    res = []
    try:
        for n in (1, 5):
            gomp.omp_set_num_threads(n)
            s = m.seq()
            la, _ = s.step(list(range(37)), [0.25, 0.5, 0.75], commit=True)
            lb, _ = s.step([3, 1, 4], [0.1, 0.9, 0.2], commit=True)
            res.append((la, lb, s.kv(1, 0), s.kv(0, 1)))
    finally:
        gomp.omp_set_num_threads(os.cpu_count() or 1)
    for x, y in zip(*res):
        assert np.array_equal(x, y)


def test_f32_instantiation_close(toy):
    """The fp32 instantiation (CPU timing) computes the same function."""
    blob, m = toy
    m32 = O.Model(blob, "f32")
    a, b = m.seq(), m32.seq()
    la, _ = a.step(list(range(20)), [0.3, 0.6], commit=True)
    lb, _ = b.step(list(range(20)), [0.3, 0.6], commit=True)
    assert np.max(np.abs(la - lb)) < 1e-4 * np.abs(la).max()


def test_bad_arguments_rejected(small):
    _, m = small
    s = m.seq()
    with pytest.raises(ValueError):
        s.step([1000], [0.5])          # token outside the vocabulary
    with pytest.raises(ValueError):
        s.step([], [])                 # nothing to run
    with pytest.raises(ValueError):
        s.step(list(range(60)), [0.1] * 5)   # past n_ctx
    assert s.C == 0


# ----------------------------------------------------- temperature encoder
# Sec. 3.3 "Temperature-controlled generation" and Appendix C.2 "Temperature
# control at inference": the noise encoder also receives tau.  Reading: tau
# goes through the same sinusoid and its own Linear(d, d), GELU, Linear(d, d),
# and the result is added to every noise row of the sequence.

SMALL_T = S.ModelConfig(2, 64, 4, 128, 96, 64, S.DTYPE_FP32, temperature=True)


@pytest.fixture(scope="module")
def small_t():
    blob = _blob(SMALL_T)
    return blob, O.Model(blob)


def _encoder_count():
    for line in open(os.path.join(GOLD, "paper_counts.txt")):
        w = line.split()
        if w and w[0] == "encoder":
            return int(w[1]), float(w[2])
    raise AssertionError("no encoder line")


def test_temperature_encoder_size():
    """Model table (Appendix D): the noise encoder, with the noise and
    temperature embeddings, has ~5.9 M parameters at d = 768.  The reading
    (noise MLP d -> 4d -> d plus a temperature MLP d -> d -> d) gives
    10 d^2 + 7 d = 5.90 M; feeding [sin(u), sin(tau)] to one MLP would give
    7.1 M and a temperature embedding without its own MLP 4.7 M."""
    d, pm = _encoder_count()
    cfg = S.ModelConfig(12, d, 12, 4 * d, 30522, 128, S.DTYPE_BF16, temperature=True)
    enc = sum(int(np.prod(s)) for n, s in S.tensor_table(cfg) if n.startswith(("noise_", "temp_")))
    assert enc == 10 * d * d + 7 * d
    assert abs(enc / 1e6 - pm) / pm < 0.01, enc


def test_temperature_required_for_noise_rows(small_t):
    """A temperature-conditioned model needs each sequence's tau before it can
    embed noise rows; AR steps (no noise rows) do not."""
    _, m = small_t
    s = m.seq()
    with pytest.raises(ValueError):
        s.step([1, 2, 3], [0.5, 0.25])
    s.step([1, 2, 3], [])  # AR step: fine
    with pytest.raises(ValueError):
        O.Model(_blob(SMALL)).seq().set_temperature(0.5)


def test_temperature_zero_encoder_is_unconditioned():
    """With the temperature MLP's output layer zero, every tau leaves the model
    exactly the unconditioned one."""
    W = S.make_weights(SMALL_T, seed=0, random_affine=True)
    W["temp_w2"][:] = 0.0
    W["temp_b2"][:] = 0.0
    mt = O.Model(S.pack_blob(SMALL_T, W))
    mu = O.Model(S.pack_blob(SMALL, {k: v for k, v in W.items() if not k.startswith("temp_")}))
    x, u = [5, 9, 1, 40], [0.3, 0.7, 0.05]
    lu, _ = mu.seq().step(x, u)
    for tau in (0.01, 0.5, 1.0):
        s = mt.seq()
        s.set_temperature(tau)
        lt, _ = s.step(x, u)
        assert np.array_equal(lt, lu)


def test_temperature_is_a_per_sequence_noise_bias(small_t):
    """The temperature enters only as a vector added to the sequence's noise
    rows: an unconditioned model whose noise-MLP output bias absorbs that vector
    gives the same outputs, prefill and decode, while real rows (and so the
    committed cache) are untouched."""
    blob, m = small_t
    cfg, Wp = O.parse_blob(blob)
    d, tau = cfg["d"], 0.42
    h = d // 2
    a = 1000.0 * tau * 10000.0 ** (-np.arange(h) / h)
    e = np.concatenate([np.cos(a), np.sin(a)])
    z = Wp["tw1"] @ e + Wp["tb1"]
    z = 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))
    temb = Wp["tw2"] @ z + Wp["tb2"]
    # the unconditioned model with the folded bias, through the fp64 numpy
    # forward (a blob would round the folded bias to fp32)
    W = S.make_weights(SMALL_T, seed=0, random_affine=True)
    cfg_u, Wu_p = O.parse_blob(S.pack_blob(SMALL, {k: v for k, v in W.items() if not k.startswith("temp_")}))
    Wu_p["nb2"] = Wp["nb2"] + temb
    x, uu = [3, 17, 8, 60, 2], [0.11, 0.83, 0.5]
    s = m.seq()
    s.set_temperature(tau)
    lt, _ = s.step(x, uu)
    n = len(x) + len(uu)
    mask = np.tril(np.ones((n, n), bool))
    rows = [("tok", t) for t in x] + [("noise", q) for q in uu]
    ref = O.dense_forward(cfg_u, Wu_p, rows, list(range(n)), mask)[len(x):]
    assert np.max(np.abs(lt - ref)) <= 1e-10 * np.abs(ref).max()


def test_temperature_brute_force(small_t):
    """(e) with temperature: the numpy dense SingleForward of a
    temperature-conditioned model equals the oracle's prefills group by group,
    and different tau give different outputs."""
    blob, m = small_t
    cfg, W = O.parse_blob(blob)
    rng = np.random.default_rng(11)
    N, k, tau = 5, 3, 0.3
    x = [int(t) for t in rng.integers(0, cfg["V"], N)]
    zz = rng.random((N, k))
    M, pos, _ = O.single_forward_layout(N, k)
    rows = [("tok", t) for t in x] + [("noise", float(zz[t, j])) for t in range(N) for j in range(k)]
    dense = O.dense_forward(cfg, W, rows, pos, M, tau=tau)
    for t in range(1, N + 1):
        s = m.seq()
        s.set_temperature(tau)
        lg, _ = s.step(x[:t], zz[t - 1])
        ref = dense[N + (t - 1) * k:N + t * k]
        assert np.max(np.abs(lg - ref)) <= 1e-10 * np.abs(ref).max(), t
    s = m.seq()
    s.set_temperature(0.9)
    lg9, _ = s.step(x, zz[N - 1])
    assert np.max(np.abs(lg9 - dense[N + (N - 1) * k:])) > 1e-3 * np.abs(lg9).max()


# ------------------------------------------- training-mask attention (C.2)

def test_masked_attention_definition():
    """The plain masked attention: a row with one visible key returns that
    key's value; equal scores average the visible values; each row agrees with
    the C oracle's own single-query attention over the visible keys."""
    rng = np.random.default_rng(21)
    B, H, nq, nk, dh = 1, 2, 6, 9, 8
    Q, K, V = rng.standard_normal((B, H, nq, dh)), rng.standard_normal((B, H, nk, dh)), rng.standard_normal((B, H, nk, dh))
    mask = rng.random((nq, nk)) < 0.5
    mask[:, 0] = True
    mask[0] = False
    mask[0, 3] = True
    Om = O.masked_attention(Q, K, V, mask, 0.37)
    assert np.allclose(Om[:, :, 0], V[:, :, 3], rtol=0, atol=1e-15)
    Oq = O.masked_attention(np.zeros_like(Q), K, V, mask, 1.0)
    for r in range(nq):
        assert np.allclose(Oq[0, 0, r], V[0, 0, mask[r]].mean(axis=0), atol=1e-14)
    for h in range(H):  # the C oracle's attend scales by 1/sqrt(dh) itself
        for r in range(nq):
            idx = np.flatnonzero(mask[r])
            o, _ = O.attend(Q[0, h, r] * 0.37 * math.sqrt(dh), K[0, h, idx], V[0, h, idx])
            assert np.allclose(Om[0, h, r], o, atol=1e-12)


def test_training_masks_nnz():
    """The masks the training attention uses have the Appendix C.2 sizes:
    |M_S| over all rows, and the Future-2 rows of M_D."""
    for N, k in [(5, 3), (7, 1), (4, 4), (9, 2)]:
        assert int(O.training_mask("single", N, k).sum()) == O.nnz_single(N, k)
        Md = O.training_mask("double", N, k)
        assert Md.shape == (2 * N * k, N + 2 * N * k)
        assert int(Md[N * k:].sum()) == O.nnz_double(N, k)


# ------------------------------------ Stage-1 distillation targets (C.2)

def test_tempered_icdf_closed_form():
    """softmax(l / tau) of l = (0, ln 2, ln 3) is (1, 2, 3)^(1/tau) normalised;
    the strict inverse CDF picks the first index whose CDF exceeds u."""
    l = np.array([0.0, math.log(2.0), math.log(3.0)])
    for tau in (0.5, 1.0, 2.0):
        w = np.array([1.0, 2.0, 3.0]) ** (1.0 / tau)
        F = np.cumsum(w) / w.sum()
        for u in (0.0, 0.5 * F[0], F[0] - 1e-9, F[0] + 1e-9, 0.5 * (F[0] + F[1]),
                  F[1] - 1e-9, F[1] + 1e-9, 0.999999):
            expect = int(np.argmax(F > u))
            assert O.tempered_icdf(l, tau, u) == expect, (tau, u)
    # tau = 1 is the untempered sampler; tau = 0.5 squares the odds
    assert O.tempered_icdf(l, 0.5, 1.0 / 14 + 1e-9) == 1
    assert O.tempered_icdf(l, 0.5, 5.0 / 14 + 1e-9) == 2


def test_tempered_icdf_limits():
    """Low temperature is greedy decoding; very high temperature is uniform,
    so the map becomes floor(u V)."""
    rng = np.random.default_rng(3)
    l = rng.normal(size=50)
    V = l.size
    for u in np.linspace(0.0, 0.999, 37):
        assert O.tempered_icdf(l, 1e-3, float(u)) == int(np.argmax(l))
        if abs(u * V - round(u * V)) > 1e-3:
            assert O.tempered_icdf(l, 1e9, float(u)) == int(math.floor(u * V))


def test_teacher_targets_brute_force(small):
    """The teacher's logits at every position equal the independent numpy
    dense causal forward over the prefix, and each target is the tempered
    inverse CDF of them (rows with u near a CDF boundary are skipped)."""
    blob, m = small
    cfg, W = O.parse_blob(blob)
    rng = np.random.default_rng(11)
    B, N = 2, 7
    tokens = rng.integers(0, SMALL.vocab, (B, N)).astype(np.int32)
    tau = [0.7, 1.6]
    u = rng.random((B, N))
    tg, lg = O.teacher_targets(m, tokens, tau, u)
    for b in range(B):
        n = N
        M = np.tril(np.ones((n, n), bool))
        dense = O.dense_forward(cfg, W, [("tok", t) for t in tokens[b]], list(range(n)), M)
        np.testing.assert_allclose(lg[b], dense, rtol=0, atol=1e-9)
        for p in range(N):
            z = dense[p] / tau[b]
            q = np.exp(z - z.max())
            F = np.cumsum(q / q.sum())
            if np.min(np.abs(F - u[b, p])) > 1e-9:
                assert tg[b, p] == int(np.argmax(F > u[b, p]))


# ------------------------------------ Stage-2 self-forcing targets (C.2)

def test_selfforcing_targets_equal_decode_steps(small):
    """The teacher rollout's round-1 group t equals a K-Forcing prefill over
    the first t+1 context tokens with noise z1[t] (C oracle, cached steps),
    and its round-2 group t equals the decode step that follows with x1[t]
    as the real rows and z2[t] as the noise: the DoubleForward window is one
    decode step (Appendix C.2), here across every group of a sequence."""
    blob, m = small
    cfg, W = O.parse_blob(blob)
    rng = np.random.default_rng(13)
    B, N, k = 2, 5, 3
    tokens = rng.integers(0, SMALL.vocab, (B, N)).astype(np.int32)
    z1 = rng.random((B, N, k))
    z2 = rng.random((B, N, k))
    x1, x2, l1, l2 = O.selfforcing_targets(cfg, W, tokens, k, z1, z2)
    for b in range(B):
        for t in range(N):
            s, lg, toks = O.prefill(m, list(tokens[b, :t + 1]), list(z1[b, t]))
            np.testing.assert_allclose(l1[b, t * k:(t + 1) * k], lg, rtol=0, atol=1e-9)
            assert list(toks) == list(x1[b, t])
            lg2, toks2 = O.decode(s, list(x1[b, t]), list(z2[b, t]))
            np.testing.assert_allclose(l2[b, t * k:(t + 1) * k], lg2, rtol=0, atol=1e-9)
            assert list(toks2) == list(x2[b, t])


def test_selfforcing_teacher_forcing_changes_only_round_two(small):
    """Forcing other Future-1 tokens leaves round 1 alone and changes the
    Future-2 logits of exactly the groups whose Future-1 tokens changed."""
    blob, m = small
    cfg, W = O.parse_blob(blob)
    rng = np.random.default_rng(14)
    B, N, k = 1, 4, 2
    tokens = rng.integers(0, SMALL.vocab, (B, N)).astype(np.int32)
    z1, z2 = rng.random((B, N, k)), rng.random((B, N, k))
    x1, x2, l1, l2 = O.selfforcing_targets(cfg, W, tokens, k, z1, z2)
    forced = x1.copy()
    forced[0, 2, 1] = (forced[0, 2, 1] + 1) % SMALL.vocab
    f1, f2, g1, g2 = O.selfforcing_targets(cfg, W, tokens, k, z1, z2, x1_forced=forced)
    np.testing.assert_array_equal(f1, x1)
    np.testing.assert_allclose(g1, l1, rtol=0, atol=0)
    for t in range(N):
        same = np.allclose(g2[0, t * k:(t + 1) * k], l2[0, t * k:(t + 1) * k], rtol=0, atol=1e-12)
        assert same == (t != 2), t


# ------------------------- the paper's backbone: RMSNorm + rotary positions

def test_rmsnorm_closed_form():
    """RMSNorm of (3, 4) with gain (1, 2): mean square 12.5."""
    r = 1.0 / math.sqrt(12.5 + 1e-5)
    np.testing.assert_allclose(O.rmsnorm([3.0, 4.0], [1.0, 2.0]), [3 * r, 8 * r], rtol=1e-15)
    # scale invariance: RMSNorm(c x) = RMSNorm(x) up to the epsilon
    x = np.random.default_rng(0).normal(size=32)
    np.testing.assert_allclose(O.rmsnorm(1e3 * x, np.ones(32)), O.rmsnorm(x, np.ones(32)),
                               rtol=1e-5)


def test_rope_closed_form_and_relative_positions():
    """RoFormer's rotary map: pair 0 turns by p radians, pair i by
    p * 10000^(-2i/64); position 0 is the identity; norms are kept; and the
    score of a query at m and a key at n depends on n - m only."""
    H, dh = 2, 64
    e0 = np.zeros(H * dh)
    e0[0] = 1.0
    for p in (0, 1, 7, 100):
        y = O.rope(e0, H, dh, p)
        assert abs(y[0] - math.cos(p)) < 1e-14 and abs(y[1] - math.sin(p)) < 1e-14
    e = np.zeros(H * dh)
    e[dh + 10] = 1.0  # head 1, pair 5
    y = O.rope(e, H, dh, 3)
    a = 3 * 10000.0 ** (-10.0 / 64)
    assert abs(y[dh + 10] - math.cos(a)) < 1e-14 and abs(y[dh + 11] - math.sin(a)) < 1e-14
    rng = np.random.default_rng(1)
    q, k = rng.normal(size=H * dh), rng.normal(size=H * dh)
    np.testing.assert_allclose(O.rope(q, H, dh, 0), q, rtol=0, atol=0)
    np.testing.assert_allclose(np.linalg.norm(O.rope(q, H, dh, 37)), np.linalg.norm(q), rtol=1e-14)
    for m, n, sft in ((3, 9, 5), (20, 2, 11)):
        for h in range(H):
            sl = slice(h * dh, (h + 1) * dh)
            a = O.rope(q, H, dh, m)[sl] @ O.rope(k, H, dh, n)[sl]
            b = O.rope(q, H, dh, m + sft)[sl] @ O.rope(k, H, dh, n + sft)[sl]
            assert abs(a - b) < 1e-12 * (1 + abs(a))
    # d_rot = 64 < d_head = 128: dimensions 64.. are left alone
    x = rng.normal(size=128)
    np.testing.assert_allclose(O.rope(x, 1, 128, 9)[64:], x[64:], rtol=0, atol=0)


def test_rms_rope_backbone_brute_force():
    """(e) for the paper's backbone: the C oracle's cached steps (prefill and
    decode with noise rows, RMSNorm, rotary q/k at each row's position) equal
    the independent numpy dense SingleForward / DoubleForward passes."""
    cfg = S.ModelConfig(2, 64, 4, 128, 96, 64, S.DTYPE_FP32, rms_rope=True)
    blob = _blob(cfg, seed=12)
    m = O.Model(blob)
    N, k = 5, 2
    rng = np.random.default_rng(15)
    c, W, x, outs = _check_single_forward(blob, m, N, k, rng)
    assert c["rms_rope"]
    z2 = rng.random((N, k))
    MD, pos = O.double_forward_layout(N, k)
    rows = [("tok", t) for t in x]
    rows += [("tok", outs[t][1][j]) for t in range(1, N + 1) for j in range(k)]
    rows += [("noise", float(z2[t - 1, j])) for t in range(1, N + 1) for j in range(k)]
    dense = O.dense_forward(c, W, rows, pos, MD)
    for t in range(1, N + 1):
        s, _ = outs[t]
        lg, _ = O.decode(s, outs[t][1], z2[t - 1])
        ref = dense[N + N * k + (t - 1) * k:N + N * k + t * k]
        assert np.max(np.abs(lg - ref)) <= 1e-10 * np.abs(ref).max()
