"""GPU parity of temperature-controlled generation (Sec. 3.3; Appendix C.2,
temperature control at inference): each sequence's tau conditions its noise
rows through the temperature encoder.  Teacher-forced against the oracle,
with a different tau per sequence."""
import sys

import numpy as np
import pytest

import kf_synth as S
import oracle as O
from tests.parity_util import TOL, compare_head, merge, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _ctx(cfg, blob, max_batch, max_k, max_prompt):
    from paper_2606_10820_amd import binding as Bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                       cfg.dtype, max_batch, max_k, max_prompt,
                       Bd.KF_FLAG_DEBUG_LOGITS | Bd.KF_FLAG_TEMPERATURE)
    kf = Bd.KForcing(c)
    kf.load_weights(blob)
    return kf


def _teacher_forced(kf, model, prompt, taus, ks, seed, tol, rows):
    B, N = prompt.shape
    kf.set_temperature(np.asarray(taus, np.float32))
    seqs = {}
    for b in rows:
        seqs[b] = model.seq()
        seqs[b].set_temperature(float(np.float32(taus[b])))
    pending = {b: list(prompt[b]) for b in rows}
    stats, p = [], N
    for si, k in enumerate(ks):
        u = S.noise_block(seed, B, p, k)
        out = kf.prefill(prompt, k, u) if si == 0 else kf.decode_block(u)
        torch.cuda.synchronize()
        gl = kf.debug_logits(B * k).cpu().numpy().reshape(B, k, -1)
        toks = out.cpu().numpy()
        for b in rows:
            ol, _ = seqs[b].step(pending[b], u[b].astype(np.float64), commit=True)
            stats.append(compare_head(gl[b], ol, toks[b], tol, where=f"step {si} seq {b}"))
            pending[b] = list(toks[b])
        p += k
    return merge(stats)


TOY_T = S.ModelConfig(2, 128, 4, 512, 1024, 128, S.DTYPE_FP32, temperature=True)
LM1B_T = S.ModelConfig(12, 768, 12, 3072, 30522, 128, S.DTYPE_BF16, temperature=True)


def test_toy_temperature_parity():
    """fp32 toy model with a temperature encoder, batch 4, tau in [0.05, 1]."""
    blob = S.pack_blob(TOY_T, S.make_weights(TOY_T, seed=0, random_affine=True))
    kf = _ctx(TOY_T, blob, 4, 4, 16)
    prompt = S.prompts_uniform(1, 4, 16, TOY_T.vocab)
    st = _teacher_forced(kf, O.Model(blob), prompt, [0.05, 0.3, 0.7, 1.0], [4, 4, 2],
                         seed=9, tol=TOL[0], rows=range(4))
    report("toy fp32 temperature", st)


def test_temperature_required_and_changeable():
    """Noise-row steps refuse to run until every sequence's tau is set; AR steps
    do not need it; a new tau takes effect at the next step."""
    from paper_2606_10820_amd import binding as Bd
    blob = S.pack_blob(TOY_T, S.make_weights(TOY_T, seed=1, random_affine=True))
    kf = _ctx(TOY_T, blob, 4, 4, 16)
    prompt = S.prompts_uniform(2, 4, 16, TOY_T.vocab)
    u = S.noise_block(3, 4, 16, 4)
    with pytest.raises(Bd.KfError):
        kf.prefill(prompt, 4, u)
    kf.set_temperature(np.full(2, 0.5, np.float32))
    with pytest.raises(Bd.KfError):
        kf.prefill(prompt, 4, u)  # only 2 of 4 sequences have a temperature
    kf.prefill_ar(prompt, np.full(4, 0.5, np.float32))  # no noise rows: allowed
    kf.set_temperature(np.full(4, 0.5, np.float32))
    a = kf.prefill(prompt, 4, u).cpu().numpy()
    kf.set_temperature(np.full(4, 0.5, np.float32))
    b = kf.prefill(prompt, 4, u).cpu().numpy()
    assert np.array_equal(a, b)
    torch.cuda.synchronize()
    la = kf.debug_logits(16).cpu().numpy()
    kf.set_temperature(np.full(4, 0.9, np.float32))
    kf.prefill(prompt, 4, u)
    torch.cuda.synchronize()
    lb = kf.debug_logits(16).cpu().numpy()
    assert np.abs(la - lb).max() > 1e-4 * np.abs(la).max()


@pytest.mark.parametrize("B", [8, 2])
def test_lm1b_shape_temperature_bf16(B):
    """LM1B-shaped bf16 model with a temperature encoder: prompt 16, prefill and
    one decode block, the first and last sequence; at batch 2 the decode block
    (16 body rows, 8 noise rows) runs the skinny GEMMs, the temperature
    embedding added in the second noise GEMM's epilogue."""
    blob = S.pack_blob(LM1B_T, S.make_weights(LM1B_T, seed=0, random_affine=True))
    kf = _ctx(LM1B_T, blob, B, 4, 16)
    prompt = S.prompts_zipf(1, B, 16, LM1B_T.vocab)
    taus = np.linspace(0.01, 1.0, B)
    st = _teacher_forced(kf, O.Model(blob), prompt, taus, [4, 4], seed=5, tol=TOL[1],
                         rows=[0, B - 1])
    report(f"lm1b bf16 temperature B={B}", st)


def test_toy_temperature_generate():
    """kf_generate of a temperature-conditioned model: the noise rows of every
    pass come from the noise encoder computed ahead for the whole generate, the
    temperature embedding added by the embedding kernel.  Tokens against the
    oracle on the GPU's own history (near-ties exempt), and equal to the
    explicit prefill / decode-block sequence with the same noise, whose noise
    rows go through the per-step encoder."""
    blob = S.pack_blob(TOY_T, S.make_weights(TOY_T, seed=2, random_affine=True))
    model = O.Model(blob)
    B, N, L, k, seed = 4, 16, 48, 4, 31
    taus = np.asarray([0.05, 0.3, 0.7, 1.0], np.float32)
    kf = _ctx(TOY_T, blob, B, k, N)
    kf.set_temperature(taus)
    prompt = S.prompts_uniform(3, B, N, TOY_T.vocab)
    out = kf.generate(prompt, L, k, seed).cpu().numpy()
    near_total = 0
    for b in range(B):
        s = model.seq()
        s.set_temperature(float(taus[b]))
        pending = list(prompt[b])
        for p in range(N, N + L, k):
            u = [O.noise_u(seed, b, p + j) for j in range(k)]
            ol, _ = s.step(pending, u, commit=True)
            toks = out[b, p - N:p - N + k]
            top = np.sort(ol, axis=1)
            near = (top[:, -1] - top[:, -2]) < TOL[0] * np.abs(ol).max(axis=1)
            assert np.all((toks == O.argmax(ol)) | near), (b, p)
            near_total += int(near.sum())
            pending = list(toks)
    _log(f"temperature generate: near-ties {near_total} of {B * L}")
    kf2 = _ctx(TOY_T, blob, B, k, N)
    kf2.set_temperature(taus)
    t = [kf2.prefill(prompt, k, kf2.fill_noise(seed, B, N, k)).cpu().numpy()]
    for p in range(N + k, N + L, k):
        t.append(kf2.decode_block(kf2.fill_noise(seed, B, p, k)).cpu().numpy())
    np.testing.assert_array_equal(np.concatenate(t, axis=1), out)
