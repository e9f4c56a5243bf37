"""bf16 decode parity at full context (Appendix C.1: every decode block attends
over the whole cached history, so the benchmark workloads with a 1024-position
context run their attention over up to 1016 cached keys plus the block).

Two models:

* a cheap model at the real head shape (2 layers, d = 256, 4 heads of
  d_head 64, MLP 1024, vocabulary 8192, context 1024, bf16), decoded from a
  128-token prompt at k = 4 until the context is full (223 decode blocks,
  C = 128 .. 1016), teacher-forced and compared with the oracle after EVERY
  block.  The batch sizes pick the three decode-attention launch shapes of
  d_head 64:
    - B = 1: 4 query blocks, so the key range is split 8 ways (a merge kernel
      combines the parts); at C ~ 1000 each split spans 128 keys, one 32-key
      tile for each of the four wavefronts;
    - B = 16: 64 query blocks, one eight-wavefront workgroup each with no
      split; at C ~ 1000 each wavefront walks 4 tiles, so both halves of the
      load/compute ping-pong run;
    - B = 64: 256 query blocks, four wavefronts each with no split; 8 tiles per
      wavefront at C ~ 1000.
* the OpenWebText-shaped model (12 layers, d = 768, 12 heads, vocabulary
  50257, context 1024) through a full kf_generate run of the benchmark sweep
  (prompt 128, 896 new tokens, device noise, graph-replayed blocks) at
  batches 1 and 16; the oracle rebuilds the last block's context (C = 1016)
  from the GPU's own token history and compares the last block of sequences
  0 and B - 1.
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import kf_synth as S
import oracle as O
from tests.parity_util import TOL, compare_head, merge, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

CHEAP = S.ModelConfig(2, 256, 4, 1024, 8192, 1024, S.DTYPE_BF16)
OWT = S.WORKLOADS["owt"]["cfg"]
_CACHE = {}


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _blob(cfg):
    key = (cfg, "blob")
    if key not in _CACHE:
        _CACHE[key] = S.pack_blob(cfg, S.make_weights(cfg, seed=0, random_affine=True))
    return _CACHE[key]


def _model(cfg):
    key = (cfg, "model")
    if key not in _CACHE:
        _CACHE[key] = O.Model(_blob(cfg))
    return _CACHE[key]


def _ctx(cfg, max_batch, max_k, max_prompt):
    from paper_2606_10820_amd import binding as Bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                       cfg.dtype, max_batch, max_k, max_prompt, Bd.KF_FLAG_DEBUG_LOGITS)
    kf = Bd.KForcing(c)
    kf.load_weights(_blob(cfg))
    return kf


@pytest.mark.parametrize("B", [1, 16, 64])
def test_cheap_model_decodes_to_full_context(B):
    """Prefill of 128 prompt tokens, then k = 4 blocks until C = 1016 (the last
    block that fits 1024 positions); every block of sequences 0 and B - 1 is
    compared with the oracle fed the GPU's own emitted tokens."""
    cfg, N, k, seed = CHEAP, 128, 4, 11
    kf = _ctx(cfg, B, k, N)
    model = _model(cfg)
    prompt = S.prompts_zipf(1, B, N, cfg.vocab)
    rows = sorted({0, B - 1})
    seqs = {b: model.seq() for b in rows}
    pending = {b: list(prompt[b]) for b in rows}
    stats, late = [], []
    p, si = N, 0
    _log(f"cheap model B={B}: prefill N={N}, decode to C={cfg.n_ctx - 2 * k}")
    while True:
        C = p - k if si else 0
        if si and C + 2 * k > cfg.n_ctx:
            break
        u = S.noise_block(seed, B, p, k)
        out = kf.prefill(prompt, k, u) if si == 0 else kf.decode_block(u)
        torch.cuda.synchronize()
        gl = kf.debug_logits(B * k).cpu().numpy().reshape(B, k, -1)
        toks = out.cpu().numpy()
        with ThreadPoolExecutor(len(rows)) as ex:
            ols = list(ex.map(lambda b: seqs[b].step(pending[b], u[b].astype(np.float64),
                                                     commit=True)[0], rows))
        for b, ol in zip(rows, ols):
            st = compare_head(gl[b], ol, toks[b], TOL[1], where=f"B={B} block {si} (C={C}) seq {b}")
            stats.append(st)
            if C >= 896:
                late.append(st)
            pending[b] = list(toks[b])
        p += k
        si += 1
    Cf, pend, Bs = kf.get_state()
    assert (Cf, pend, Bs) == (cfg.n_ctx - k, k, B)
    assert seqs[rows[0]].C == Cf
    report(f"cheap bf16 B={B}, C=128..1016 every block", merge(stats))
    report(f"cheap bf16 B={B}, blocks at C>=896", merge(late))


@pytest.mark.parametrize("B", [1, 16])
def test_owt_generate_last_block_full_context(B):
    """The sweep's generate (prompt 128, 896 new tokens, k = 4) on the
    OWT-shaped model; the last block runs at C = 1016 over 8 KV pages."""
    w = S.WORKLOADS["owt"]
    N, L, k, seed = w["N"], w["L"], 4, 2
    kf = _ctx(OWT, B, k, N)
    prompt = S.prompts_zipf(1, B, N, OWT.vocab)
    _log(f"owt generate B={B}: N={N}, L={L}")
    out = kf.generate(prompt, L, k, seed).cpu().numpy()
    gl = kf.debug_logits(B * k).cpu().numpy().reshape(B, k, -1)
    assert kf.get_state() == (N + L - k, k, B)
    model = _model(OWT)

    def last_block(b):
        hist = list(prompt[b]) + list(out[b, :L - 2 * k])
        pend = list(out[b, L - 2 * k:L - k])
        s = model.seq()
        s.step(hist, [], commit=True)  # the context of the last block: C = N + L - 2k
        u = [O.noise_u(seed, b, N + L - k + j) for j in range(k)]
        return s.step(pend, u, commit=True)[0]

    rows = sorted({0, B - 1})
    with ThreadPoolExecutor(len(rows)) as ex:
        ols = list(ex.map(last_block, rows))
    stats = [compare_head(gl[b], ol, out[b, L - k:], TOL[1], where=f"owt B={B} last block seq {b}")
             for b, ol in zip(rows, ols)]
    report(f"owt bf16 B={B} generate, last block (C={N + L - 2 * k})", merge(stats))
