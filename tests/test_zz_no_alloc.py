"""kf_decode_block_noalloc against kf_decode_block: the same decode blocks with
the step's partial results (attention key-split states, split-K parts, head
argmax partials) in the library's device scratch instead of the state
buffer's workspace.  Two calls in a row, the second with a smaller input
(k = 4, then k = 2), on a model whose steps use all three kinds of partial
results; a second context then reuses the same scratch at another batch size.
The kernels are the same, so tokens and logits must be identical bit for
bit; the tokens are also held to the oracle's (teacher-forced) at the bf16
tolerance."""
import numpy as np
import pytest

import kf_synth as S
import oracle as O
from tests.parity_util import TOL, compare_head

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# 2 layers, d 256, 4 heads of d_head 64, MLP 2048, vocabulary 8192, context 256,
# bf16.  At batch 4 a k = 4 block has 32 body rows: tiled GEMMs, MLP-down
# (K = 2048) split 16 ways into the split-K parts, decode attention over 16
# query blocks split 2 ways, 16 head rows x 64 tiles of argmax partials.
CFG = S.ModelConfig(2, 256, 4, 2048, 8192, 256, S.DTYPE_BF16)


@pytest.fixture(scope="module")
def model():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    blob = S.pack_blob(CFG, S.make_weights(CFG, seed=0, random_affine=True))
    return blob, O.Model(blob)


def _ctx(blob, B):
    from paper_2606_10820_amd import binding as Bd
    c = Bd.make_config(CFG.n_layer, CFG.d_model, CFG.n_head, CFG.d_mlp, CFG.vocab, CFG.n_ctx,
                       CFG.dtype, B, 4, 64, Bd.KF_FLAG_DEBUG_LOGITS)
    kf = Bd.KForcing(c)
    kf.load_weights(blob)
    return kf


@pytest.mark.parametrize("B", [4, 2])
def test_noalloc_decode_matches_decode_block(model, B):
    blob, m = model
    N = 48
    prompt = S.prompts_zipf(1, B, N, CFG.vocab)
    ref, nal = _ctx(blob, B), _ctx(blob, B)
    u0 = S.noise_block(3, B, N, 4)
    t_ref = ref.prefill(prompt, 4, u0).cpu().numpy()
    t_nal = nal.prefill(prompt, 4, u0).cpu().numpy()
    assert np.array_equal(t_ref, t_nal)
    seqs = [m.seq() for _ in (0, B - 1)]
    pend = [list(prompt[0]), list(prompt[B - 1])]
    for b_i, s in enumerate(seqs):
        s.step(pend[b_i], u0[(0, B - 1)[b_i]].astype(np.float64), commit=True)
        pend[b_i] = list(t_ref[(0, B - 1)[b_i]])
    p = N + 4
    for k in (4, 2):  # the second call has the smaller input
        u = S.noise_block(3, B, p, k)
        o_ref = ref.decode_block(u)
        torch.cuda.synchronize()
        l_ref = ref.debug_logits(B * k).cpu().numpy()
        o_nal = nal.decode_block_noalloc(u)
        torch.cuda.synchronize()
        l_nal = nal.debug_logits(B * k).cpu().numpy()
        assert np.array_equal(o_ref.cpu().numpy(), o_nal.cpu().numpy()), f"tokens differ at k={k}"
        assert np.array_equal(l_ref, l_nal), f"logits differ at k={k}"
        assert ref.get_state() == nal.get_state()
        toks = o_nal.cpu().numpy()
        gl = l_nal.reshape(B, k, -1)
        for b_i, b in enumerate((0, B - 1)):
            ol, _ = seqs[b_i].step(pend[b_i], u[b].astype(np.float64), commit=True)
            compare_head(gl[b], ol, toks[b], TOL[1], where=f"noalloc B={B} k={k} seq {b}")
            pend[b_i] = list(toks[b])
        p += k
    print(f"noalloc B={B}: identical to kf_decode_block at k = 4 and 2", flush=True)
