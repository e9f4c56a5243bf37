"""GPU parity of the rotary RMSNorm backbone (Appendix D, model table:
RMSNorm pre-norm and rotary positions in place of LayerNorm and a learned
position table) on every path: prefill and decode blocks, kf_generate, the AR
baseline, the Stage-1 and the Stage-2 targets.  The comparison rules are the
LayerNorm model's (tests.parity_util); every check is teacher-forced.

Head sizes: d_head 32 (every pair rotated), 64 (the LM1B shape) and 128
(only the first 64 dimensions rotated)."""
import sys

import numpy as np
import pytest

import kf_synth as S
import oracle as O
from tests.parity_util import TOL, compare_head, merge, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

RT32 = S.ModelConfig(2, 128, 4, 512, 1024, 128, S.DTYPE_FP32, rms_rope=True)
RT128 = S.ModelConfig(2, 256, 2, 512, 1024, 128, S.DTYPE_FP32, rms_rope=True)
LM1B_R = S.ModelConfig(12, 768, 12, 3072, 30522, 128, S.DTYPE_BF16, rms_rope=True)


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _ctx(cfg, blob, max_batch, max_k, max_prompt, extra=0):
    from paper_2606_10820_amd import binding as Bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = Bd.make_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.n_ctx,
                       cfg.dtype, max_batch, max_k, max_prompt,
                       Bd.KF_FLAG_DEBUG_LOGITS | Bd.KF_FLAG_RMS_ROPE | extra)
    kf = Bd.KForcing(c)
    kf.load_weights(blob)
    return kf


def _blob(cfg, seed):
    return S.pack_blob(cfg, S.make_weights(cfg, seed=seed, random_affine=True))


def _teacher_forced(kf, model, prompt, ks, seed, tol, rows):
    B, N = prompt.shape
    seqs = {b: model.seq() for b in rows}
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


@pytest.mark.parametrize("cfg", [RT32, RT128], ids=["dh32", "dh128"])
def test_rms_rope_prefill_decode(cfg):
    """fp32, batch 3, prompt 13, ragged k per block; positions reach 13 + 4 + 3 + 1 + 4 + 2."""
    blob = _blob(cfg, 0)
    kf = _ctx(cfg, blob, 3, 4, 13)
    prompt = S.prompts_uniform(3, 3, 13, cfg.vocab)
    _log(f"rms/rope dh={cfg.d_head} prefill + decode")
    st = _teacher_forced(kf, O.Model(blob), prompt, [4, 3, 1, 4, 2], seed=12, tol=TOL[0],
                         rows=range(3))
    report(f"rms/rope d_head {cfg.d_head}", st)
    assert kf.device_errors() == 0


def test_rms_rope_unused_tensors_ignored():
    """The position table and the norm shifts of a rotary RMSNorm blob are not
    read: random values there give the same tokens and logits as zeros."""
    w = S.make_weights(RT32, seed=1, random_affine=True)
    blob0 = S.pack_blob(RT32, w)
    rng = np.random.default_rng(0)
    for name in list(w):
        base = name.split(".")[-1]
        if name == "pos_emb" or (base.startswith("ln") and base.endswith("_b")):
            w[name] = rng.normal(0, 0.5, w[name].shape).astype(np.float32)
    blob1 = S.pack_blob(RT32, w)
    assert not np.array_equal(blob0, blob1)
    prompt = S.prompts_uniform(4, 2, 9, RT32.vocab)
    res = []
    for blob in (blob0, blob1):
        kf = _ctx(RT32, blob, 2, 4, 9)
        a = kf.prefill(prompt, 4, S.noise_block(2, 2, 9, 4)).cpu().numpy()
        b = kf.decode_block(S.noise_block(2, 2, 13, 4)).cpu().numpy()
        torch.cuda.synchronize()
        res.append((a, b, kf.debug_logits(8).cpu().numpy()))
    for x, y in zip(*res):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("B", [8, 2])
def test_lm1b_shape_rms_rope_bf16(B):
    """LM1B-shaped bf16 rotary model (d_head 64): prompt 16, prefill and two
    decode blocks; batch 8 (sequences 0, 3 and 7) and batch 2, whose 16-row
    decode blocks run the skinny GEMMs (RMS statistics, rotary QKV epilogue)."""
    blob = _blob(LM1B_R, 0)
    kf = _ctx(LM1B_R, blob, B, 4, 16)
    prompt = S.prompts_zipf(2, B, 16, LM1B_R.vocab)
    st = _teacher_forced(kf, O.Model(blob), prompt, [4, 4, 4], seed=6, tol=TOL[1],
                         rows=sorted({0, B // 2 - 1, B - 1}))
    report(f"lm1b rms/rope bf16 B={B}", st)


def test_rms_rope_generate():
    """kf_generate (device Philox noise) against the oracle on the GPU's own
    token history; positions up to 16 + 64."""
    blob = _blob(RT32, 2)
    model = O.Model(blob)
    B, N, L, k, seed = 3, 16, 64, 4, 78
    kf = _ctx(RT32, blob, B, k, N)
    prompt = S.prompts_uniform(5, B, N, RT32.vocab)
    out = kf.generate(prompt, L, k, seed).cpu().numpy()
    near_total = 0
    for b in range(B):
        s = model.seq()
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
    _log(f"rms/rope generate: near-ties {near_total} of {B * L}")


def test_rms_rope_ar_decoding():
    """AR baseline on the rotary model: logits within tolerance of the oracle,
    inverse-CDF decisions equal on the GPU's own logits (1e-5 boundary margin)."""
    blob = _blob(RT32, 3)
    model = O.Model(blob)
    B, N = 3, 10
    kf = _ctx(RT32, blob, B, 4, N)
    prompt = S.prompts_uniform(9, B, N, RT32.vocab)
    seqs = [model.seq() for _ in range(B)]
    pending = [list(prompt[b]) for b in range(B)]
    close = 0
    for step in range(10):
        u = S.noise_block(6, B, N + step, 1)[:, 0]
        out = kf.prefill_ar(prompt, u) if step == 0 else kf.decode_ar(u)
        torch.cuda.synchronize()
        gl = kf.debug_logits(B).cpu().numpy()
        toks = out.cpu().numpy()
        for b in range(B):
            ol, _ = seqs[b].step(pending[b], [], commit=True)
            assert np.abs(gl[b] - ol[0]).max() <= TOL[0] * np.abs(ol[0]).max(), (step, b)
            want = O.icdf(O.softmax(gl[b].astype(np.float64)), float(u[b]))
            if O.cdf_margin(gl[b].astype(np.float64), float(u[b])) < 1e-5:
                close += 1
            else:
                assert toks[b] == want, (step, b)
            pending[b] = [int(toks[b])]
    _log(f"rms/rope AR: {close} decisions within 1e-5 of a CDF boundary")


def test_rms_rope_teacher_targets():
    """Stage-1 targets on the rotary model (fp32, d_head 128)."""
    from tests import test_gpu_teacher as T
    blob = _blob(RT128, 4)
    B, N = 3, 20
    tau = [0.6, 1.0, 1.7]
    tokens, u = T._inputs(RT128, B, N, 25)
    kf = T._ctx(RT128, blob, B, N)
    tg = T._run(kf, tokens, tau, u)
    gl = kf.debug_logits(B * N).cpu().numpy().astype(np.float64)
    otg, olg = O.teacher_targets(O.Model(blob), tokens, tau, u)
    rel = T._check_logits(gl, olg.reshape(B * N, -1), TOL[0], "rms/rope teacher")
    ex = T._check_gpu_logits(gl, tg.reshape(-1), np.repeat(tau, N), u.reshape(-1),
                             "rms/rope teacher")
    _log(f"rms/rope teacher: max logit rel err {rel:.2e}; near-boundary rows {ex}")
    assert kf.device_errors() == 0


def test_rms_rope_teacher_targets_bf16():
    """Stage-1 targets on a bf16 rotary model (d_head 128): the teacher pass of
    a 16-bit model attends through the block kernel of the training masks."""
    from tests import test_gpu_teacher as T
    cfg = S.ModelConfig(2, 256, 2, 512, 1024, 128, S.DTYPE_BF16, rms_rope=True)
    blob = _blob(cfg, 6)
    B, N = 3, 70
    tau = [float(np.float32(t)) for t in (0.7, 1.0, 1.6)]
    tokens, u = T._inputs(cfg, B, N, 26)
    kf = T._ctx(cfg, blob, B, N)
    tg = T._run(kf, tokens, tau, u)
    gl = kf.debug_logits(B * N).cpu().numpy().astype(np.float64)
    otg, olg = O.teacher_targets(O.Model(blob), tokens, tau, u)
    rel = T._check_logits(gl, olg.reshape(B * N, -1), TOL[1], "rms/rope bf16 teacher")
    ex = T._check_gpu_logits(gl, tg.reshape(-1), np.repeat(tau, N), u.reshape(-1),
                             "rms/rope bf16 teacher")
    _log(f"rms/rope bf16 teacher: max logit rel err {rel:.2e}; near-boundary rows {ex}")
    assert kf.device_errors() == 0


@pytest.mark.parametrize("cfg", [
    S.ModelConfig(2, 128, 4, 512, 1024, 128, S.DTYPE_BF16, rms_rope=True),
    S.ModelConfig(2, 256, 2, 512, 1024, 128, S.DTYPE_BF16, rms_rope=True),
], ids=["dh32", "dh128"])
def test_rms_rope_rollout(cfg):
    """Stage-2 targets on the rotary model (bf16): both rounds' rows sit at
    their own positions (context i, F1 t+1+j, F2 t+1+k+j)."""
    from tests import test_gpu_rollout as R
    blob = _blob(cfg, 5)
    R._run_case(cfg, blob, 2, 9, 3, 37)
    R._run_case(cfg, blob, 2, 5, 1, 38)
