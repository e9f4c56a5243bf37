"""GPU parity of continuous batching over the paged KV cache (KF_FLAG_SERVING).

Sequences are independent (each computes the decode of Appendix C.1 on its
own), so every served sequence is checked against the oracle's sequence run
alone, teacher-forced on the GPU's own tokens (rules of tests.parity_util),
while other sequences are admitted, stepped in changing orders and released
around it.  The paged cache is exercised by sequences that cross 128-position
page boundaries, by pages that return to the pool and are handed to a new
sequence, and by a pool too small for a step (KF_ENOMEM, nothing changes).
A served batch in any slot order must also equal the lock-step path bit for
bit: the rows of a step do not interact."""
import sys

import numpy as np
import pytest

import kf_synth as S
import oracle as O
from tests.parity_util import TOL, compare_head, merge, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOY = S.WORKLOADS["toy"]["cfg"]


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _bd():
    from paper_2606_10820_amd import binding as Bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return Bd


def _ctx(cfg, blob, max_batch, max_k, max_prompt, kv_pages=0, serving=True, extra=0):
    Bd = _bd()
    flags = Bd.KF_FLAG_DEBUG_LOGITS | extra | (Bd.KF_FLAG_SERVING if serving else 0)
    c = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                       cfg.dtype, max_batch, max_k, max_prompt, flags, kv_pages)
    kf = Bd.KForcing(c)
    kf.load_weights(blob)
    return kf


class Served:
    """Drives a serving context and an oracle sequence per live slot."""

    def __init__(self, kf, model, tol, rng, taus=None):
        self.kf, self.model, self.tol, self.rng = kf, model, tol, rng
        self.taus = taus  # per-slot temperature of a temperature-conditioned model
        self.seq, self.pending, self.C = {}, {}, {}
        self.stats = []

    def _check(self, slots, k, u, out):
        torch.cuda.synchronize()
        gl = self.kf.debug_logits(len(slots) * k).cpu().numpy().reshape(len(slots), k, -1)
        toks = out.cpu().numpy()
        for r, q in enumerate(slots):
            ol, _ = self.seq[q].step(self.pending[q], u[r].astype(np.float64), commit=True)
            self.stats.append(compare_head(gl[r], ol, toks[r], self.tol, where=f"slot {q}"))
            self.C[q] += len(self.pending[q])
            self.pending[q] = list(toks[r])
            assert self.kf.serve_state(q)[:2] == (self.C[q], k), q

    def admit(self, slots, N, k, vocab):
        prompts = self.rng.integers(0, vocab, (len(slots), N)).astype(np.int32)
        u = self.rng.random((len(slots), k)).astype(np.float32)
        out = self.kf.serve_admit(slots, prompts, k, u)
        for r, q in enumerate(slots):
            self.seq[q] = self.model.seq()
            if self.taus is not None:
                self.seq[q].set_temperature(float(self.taus[q]))
            self.pending[q] = list(prompts[r])
            self.C[q] = 0
        self._check(slots, k, u, out)

    def step(self, slots, k):
        u = self.rng.random((len(slots), k)).astype(np.float32)
        out = self.kf.serve_step(slots, u)
        self._check(slots, k, u, out)

    def release(self, slots):
        self.kf.serve_release(slots)
        for q in slots:
            del self.seq[q], self.pending[q], self.C[q]


TOY512 = S.ModelConfig(2, 128, 4, 512, 1024, 512, S.DTYPE_FP32)


def test_serving_churn_toy_fp32():
    """fp32 toy model (context 512), 6 slots, a pool of 9 pages of 128
    positions: admissions of different prompt lengths, steps over changing
    slot orders, releases and re-admissions into freed slots and pages;
    sequences run past position 128 (into their second page)."""
    Bd = _bd()
    blob = S.pack_blob(TOY512, S.make_weights(TOY512, seed=0, random_affine=True))
    kf = _ctx(TOY512, blob, 6, 4, 96, kv_pages=9)
    sv = Served(kf, O.Model(blob), TOL[0], np.random.default_rng(11))
    V = TOY512.vocab
    sv.admit([0, 2], 60, 4, V)
    sv.step([0, 2], 4)
    sv.step([2, 0], 4)
    sv.admit([5], 7, 4, V)
    sv.step([0, 2, 5], 4)
    sv.release([2])
    sv.step([5, 0], 4)
    sv.admit([2, 4], 80, 4, V)         # slot 2 again: fresh sequence on reused pages
    for it in range(14):
        order = [0, 2, 4, 5]
        sv.rng.shuffle(order)
        sv.step(order, 4)
    assert sv.C[0] > 128 and sv.C[2] > 128  # both reach their second page
    free, total = kf.serve_pages()
    used = sum(kf.serve_state(q)[2] for q in range(6))
    assert total == 9 and free + used == 9
    sv.release([0])
    sv.admit([1], 96, 2, V)            # a different window: steps alone
    sv.step([1], 2)
    sv.step([2, 4, 5], 4)
    _log(f"serving churn: {merge(sv.stats)}; C = {sv.C}; pages free {kf.serve_pages()[0]}")
    assert kf.device_errors() == 0


def test_serving_pool_exhaustion_changes_nothing():
    Bd = _bd()
    cfg = S.ModelConfig(2, 128, 4, 512, 1024, 256, S.DTYPE_FP32)
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=1, random_affine=True))
    kf = _ctx(cfg, blob, 4, 4, 128, kv_pages=3)
    sv = Served(kf, O.Model(blob), TOL[0], np.random.default_rng(12))
    sv.admit([0], 122, 4, cfg.vocab)  # positions 0..125: one page
    sv.admit([1], 30, 4, cfg.vocab)   # one page
    sv.admit([3], 4, 4, cfg.vocab)    # one page: the pool is full
    assert kf.serve_pages() == (0, 3)
    before = [kf.serve_state(q) for q in range(4)]
    with pytest.raises(Bd.KfError) as e:
        sv.kf.serve_step([1, 0], np.full((2, 4), 0.5, np.float32))  # slot 0 needs a page
    assert e.value.code == Bd.KF_ENOMEM
    with pytest.raises(Bd.KfError) as e:
        sv.kf.serve_admit([2], np.zeros((1, 4), np.int32), 4, np.full((1, 4), 0.5, np.float32))
    assert e.value.code == Bd.KF_ENOMEM
    assert [kf.serve_state(q) for q in range(4)] == before
    with pytest.raises(Bd.KfError) as e:
        sv.kf.serve_admit([1], np.zeros((1, 4), np.int32), 4, np.full((1, 4), 0.5, np.float32))
    assert e.value.code == Bd.KF_ESTATE  # slot in use
    sv.step([1], 4)                    # slot 1 stays within its page
    sv.release([3])
    sv.step([0, 1], 4)                 # slot 0 takes the freed page
    assert kf.serve_state(0)[2] == 2 and kf.serve_pages() == (0, 3)
    _log(f"pool exhaustion: {merge(sv.stats)}")


@pytest.mark.parametrize("dtype", [S.DTYPE_FP32, S.DTYPE_BF16], ids=["fp32", "bf16"])
def test_serving_equals_lockstep_bitwise(dtype):
    """The same four sequences served in slots [3, 1, 0, 2] and run lock-step
    (prefill + 3 decode blocks, positions past 128: two pages) give identical
    tokens and logits."""
    cfg = S.ModelConfig(2, 128, 4, 512, 1024, 256, dtype)
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=2, random_affine=True))
    B, N, k = 4, 118, 4
    prompt = S.prompts_uniform(7, B, N, cfg.vocab)
    us = [S.noise_block(8, B, N + 4 * i, k) for i in range(4)]
    ls = _ctx(cfg, blob, B, k, N, serving=False)
    lt, ll = [], []
    for i, u in enumerate(us):
        out = ls.prefill(prompt, k, u) if i == 0 else ls.decode_block(u)
        torch.cuda.synchronize()
        lt.append(out.cpu().numpy())
        ll.append(ls.debug_logits(B * k).cpu().numpy().reshape(B, k, -1))
    sv = _ctx(cfg, blob, B, k, N)
    slots = [3, 1, 0, 2]
    rows = np.array(slots)  # served row r (slot slots[r]) holds lock-step sequence slots[r]
    for i, u in enumerate(us):
        out = (sv.serve_admit(slots, prompt[rows], k, u[rows]) if i == 0
               else sv.serve_step(slots, u[rows]))
        torch.cuda.synchronize()
        st = out.cpu().numpy()
        sl = sv.debug_logits(B * k).cpu().numpy().reshape(B, k, -1)
        np.testing.assert_array_equal(st, lt[i][rows])
        np.testing.assert_array_equal(sl, ll[i][rows])
    assert all(sv.serve_state(q)[0] == N + 3 * k for q in range(B))


def test_serving_temperature_per_slot():
    """Temperature model: each slot's noise rows carry the tau of its slot."""
    cfg = S.ModelConfig(2, 128, 4, 512, 1024, 128, S.DTYPE_FP32, temperature=True)
    Bd = _bd()
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=3, random_affine=True))
    kf = _ctx(cfg, blob, 4, 4, 16, extra=Bd.KF_FLAG_TEMPERATURE)
    taus = np.array([0.2, 0.5, 0.9, 1.3], np.float32)
    kf.set_temperature(taus)
    sv = Served(kf, O.Model(blob), TOL[0], np.random.default_rng(13), taus=taus)
    sv.admit([3, 1], 9, 4, cfg.vocab)
    sv.step([1, 3], 4)
    sv.admit([0], 5, 4, cfg.vocab)
    sv.step([3, 0, 1], 4)
    _log(f"serving temperature: {merge(sv.stats)}")


def test_serving_lm1b_bf16():
    """LM1B-shaped bf16 model (MFMA attention with key splits): 8 slots, two
    admission waves, sequences to position 68 of the 128-position context."""
    cfg = S.WORKLOADS["lm1b"]["cfg"]
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=0))
    kf = _ctx(cfg, blob, 8, 4, 16)
    sv = Served(kf, O.Model(blob), TOL[1], np.random.default_rng(14))
    sv.admit([6, 1, 4], 16, 4, cfg.vocab)
    for _ in range(4):
        sv.step([1, 4, 6], 4)
    sv.admit([0, 7], 12, 4, cfg.vocab)
    for it in range(9):
        order = [0, 1, 4, 6, 7]
        sv.rng.shuffle(order)
        sv.step(order, 4)
    report("serving lm1b bf16", merge(sv.stats))


def test_serving_bf16_dh128_pages():
    """bf16 model with d_head 128 (MFMA attention at its widest head, value
    blocks of 128 rows): sequences cross a page boundary (position 128) while
    slots are stepped in changing orders."""
    cfg = S.ModelConfig(2, 256, 2, 512, 1024, 256, S.DTYPE_BF16)
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=8, random_affine=True))
    kf = _ctx(cfg, blob, 4, 4, 120)
    sv = Served(kf, O.Model(blob), TOL[1], np.random.default_rng(15))
    sv.admit([2, 0], 110, 4, cfg.vocab)
    sv.admit([3], 9, 4, cfg.vocab)
    for it in range(6):
        sv.step([0, 2] if it % 2 else [2, 0], 4)
    assert sv.C[0] > 128 and sv.C[2] > 128
    sv.step([3], 4)
    report("serving bf16 d_head 128", merge(sv.stats))


def test_serving_graph_replay_matches_direct():
    """On a real stream, served steps replay one captured graph per (sequences,
    pending count, k); tokens and logits equal the direct launches through a
    churn of admissions, steps in changing orders and releases."""
    from paper_2606_10820_amd import binding as Bd
    cfg = S.ModelConfig(2, 128, 4, 512, 1024, 256, S.DTYPE_BF16)
    blob = S.pack_blob(cfg, S.make_weights(cfg, seed=7, random_affine=True))
    stream = torch.cuda.Stream()
    res = {}
    with torch.cuda.stream(stream):
        for graphs in (False, True):
            c = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab,
                               cfg.n_ctx, cfg.dtype, 6, 4, 40,
                               Bd.KF_FLAG_DEBUG_LOGITS | Bd.KF_FLAG_SERVING)
            kf = Bd.KForcing(c, stream=stream)
            kf.load_weights(blob)
            kf.set_graphs(graphs)
            rng = np.random.default_rng(3)
            outs = []

            def step(slots, k):
                u = rng.random((len(slots), k)).astype(np.float32)
                outs.append(kf.serve_step(slots, u).cpu().numpy())
                outs.append(kf.debug_logits(len(slots) * k).cpu().numpy())

            kf.serve_admit([0, 3], rng.integers(0, cfg.vocab, (2, 30)).astype(np.int32), 4,
                           rng.random((2, 4)).astype(np.float32))
            for it in range(5):
                step([0, 3] if it % 2 else [3, 0], 4)
            kf.serve_admit([5], rng.integers(0, cfg.vocab, (1, 12)).astype(np.int32), 4,
                           rng.random((1, 4)).astype(np.float32))
            for it in range(4):
                step([5, 0, 3], 4)
            kf.serve_release([0])
            for it in range(3):
                step([3, 5], 4)
            stream.synchronize()
            res[graphs] = outs
    assert len(res[False]) == len(res[True])
    for a, b in zip(res[False], res[True]):
        np.testing.assert_array_equal(a, b)
