"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/kforcing.h, and rejects bad arguments before touching a
device (each rejection leaves the context's state unchanged)."""
import ctypes
import dataclasses
import os
import re
import subprocess

import numpy as np
import pytest

import kf_synth as S
from paper_2606_10820_amd import binding as Bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kforcing.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kf_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    return Bd.lib()


def _cfg(**kw):
    base = dict(n_layer=2, d_model=128, n_head=4, d_mlp=512, vocab=1024, n_ctx=128,
                dtype=Bd.KF_FP32, max_batch=8, max_k=4, max_prompt=32, flags=0)
    base.update(kw)
    return Bd.make_config(**base)


def _ctx(L, cfg):
    h = ctypes.c_void_p()
    assert L.kf_create(ctypes.byref(cfg), None, ctypes.byref(h)) == Bd.KF_OK
    return h


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert len(names) >= 19
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", Bd.lib_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (kf_[a-z_]+)$", out, flags=re.M))
    assert set(names) <= exported, set(names) - exported


def test_noalloc_decode_rejects_oversized_head(L):
    """kf_decode_block_noalloc holds at most KF_NOALLOC_HEAD_ENTRIES head
    partials (B * k * ceil(V / 128)) in its device scratch: a larger step is
    rejected with a message naming the limit, before any state check."""
    cfg = _cfg(d_model=64, n_head=1, d_mlp=64, vocab=1 << 20, max_batch=64, max_k=4)
    h = _ctx(L, cfg)
    fake = ctypes.c_void_p(0x10000)
    assert L.kf_decode_block_noalloc(h, 33, 4, fake, fake) == Bd.KF_EINVAL  # 132 * 8192 > 2^20
    assert b"KF_NOALLOC_HEAD_ENTRIES" in L.kf_last_error(h)
    assert L.kf_decode_block_noalloc(h, 32, 4, fake, fake) == Bd.KF_ESTATE  # 128 * 8192 fits
    L.kf_destroy(h)


def test_strerror(L):
    assert L.kf_strerror(Bd.KF_OK) == b"ok"
    assert L.kf_strerror(Bd.KF_ECTX) == b"context length exceeded"
    assert L.kf_strerror(-99) == b"unknown error"


@pytest.mark.parametrize("bad", [
    dict(n_layer=0), dict(d_model=100), dict(n_head=3), dict(d_model=256, n_head=1),
    dict(d_mlp=100), dict(vocab=1), dict(n_ctx=100), dict(dtype=7), dict(max_batch=0), dict(max_k=0),
    dict(max_k=1000), dict(max_prompt=0), dict(flags=64),
    dict(kv_pages=-1), dict(kv_pages=8),  # a page pool needs KF_FLAG_SERVING
    dict(max_batch=65535, max_prompt=128, d_mlp=4096),
    # the teacher rollout's DoubleForward rows (2 * max_batch * max_prompt * max_k) count too
    dict(flags=8, max_batch=4096, max_prompt=128),
])
def test_bad_config_rejected(L, bad):
    cfg = _cfg(**bad)
    h = ctypes.c_void_p()
    assert L.kf_create(ctypes.byref(cfg), None, ctypes.byref(h)) == Bd.KF_EINVAL
    assert L.kf_state_bytes(ctypes.byref(cfg)) == 0


def test_state_bytes_covers_kv_cache(L):
    cfg = _cfg()
    n = L.kf_state_bytes(ctypes.byref(cfg))
    kv = 8 * 2 * 2 * 128 * 128 * 4
    weights = S.n_params(S.WORKLOADS["toy"]["cfg"]) * 4
    assert n > kv + weights
    big = _cfg(dtype=Bd.KF_BF16, flags=Bd.KF_FLAG_DEBUG_LOGITS)
    assert L.kf_state_bytes(ctypes.byref(big)) > L.kf_state_bytes(ctypes.byref(_cfg(dtype=Bd.KF_BF16)))
    # the rotary backbone keeps a cos/sin table of n_ctx x 32 float2 beside the weights
    rr = _cfg(flags=Bd.KF_FLAG_RMS_ROPE)
    assert L.kf_state_bytes(ctypes.byref(rr)) >= n + 128 * 32 * 8


def test_state_machine_without_device(L):
    cfg = _cfg()
    h = _ctx(L, cfg)
    P = ctypes.c_void_p
    fake = P(0x10000)  # never dereferenced: every call below fails validation first
    # nothing bound yet
    assert L.kf_prefill(h, 2, 4, fake, 2, fake, fake) == Bd.KF_ESTATE
    assert L.kf_decode_block(h, 2, 2, fake, fake) == Bd.KF_ESTATE
    # argument checks come before state checks
    assert L.kf_prefill(h, 0, 4, fake, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 9, 4, fake, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 2, 4, fake, 0, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 2, 4, fake, 5, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 2, 33, fake, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 2, 4, None, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_prefill(h, 2, 4, fake, 2, None, fake) == Bd.KF_EINVAL
    assert L.kf_generate(h, 2, 4, fake, 6, 4, 0, fake) == Bd.KF_EINVAL   # L % k
    assert L.kf_generate(h, 2, 4, fake, -4, 4, 0, fake) == Bd.KF_EINVAL
    assert L.kf_generate(h, 2, 32, fake, 100, 4, 0, fake) == Bd.KF_ECTX  # N + L > n_ctx
    assert L.kf_prefill_ar(h, 2, 0, fake, fake, fake) == Bd.KF_EINVAL
    assert L.kf_generate_ar(h, 2, 4, fake, -1, 0, fake) == Bd.KF_EINVAL
    assert L.kf_decode_block(h, 2, 0, fake, fake) == Bd.KF_EINVAL
    assert L.kf_decode_block_noalloc(h, 2, 2, fake, fake) == Bd.KF_ESTATE
    assert L.kf_decode_block_noalloc(h, 2, 0, fake, fake) == Bd.KF_EINVAL
    assert L.kf_decode_block_noalloc(h, 2, 2, None, fake) == Bd.KF_EINVAL
    assert L.kf_fill_noise(h, 0, 0, 0, 4, fake) == Bd.KF_EINVAL
    # binding: alignment and size
    need = L.kf_state_bytes(ctypes.byref(cfg))
    assert L.kf_bind_state(h, P(0x10010), need) == Bd.KF_EINVAL
    assert L.kf_bind_state(h, fake, need - 1) == Bd.KF_ENOMEM
    assert L.kf_bind_state(h, fake, need) == Bd.KF_OK
    assert b"" == L.kf_last_error(h) or True
    # bound but no weights
    assert L.kf_prefill(h, 2, 4, fake, 2, fake, fake) == Bd.KF_ESTATE
    assert b"weights" in L.kf_last_error(h)
    assert L.kf_debug_logits(h, fake, 10) == Bd.KF_ESTATE
    # weight blob checks happen on the host before any copy
    blob = S.pack_blob(S.WORKLOADS["toy"]["cfg"], S.make_weights(S.WORKLOADS["toy"]["cfg"]))
    ptr = P(blob.ctypes.data)
    assert L.kf_load_weights(h, ptr, blob.nbytes - 4, 0) == Bd.KF_EINVAL
    bad = blob.copy()
    bad[:16].view(np.int32)[0] = 0
    assert L.kf_load_weights(h, P(bad.ctypes.data), bad.nbytes, 0) == Bd.KF_EINVAL
    assert b"header" in L.kf_last_error(h)
    bad = blob.copy()
    bad[:16].view(np.int32)[8] = 1  # dtype mismatch with the config
    assert L.kf_load_weights(h, P(bad.ctypes.data), bad.nbytes, 0) == Bd.KF_EINVAL
    assert L.kf_load_weights(h, ptr, blob.nbytes, 2) == Bd.KF_EINVAL
    C, p, B = ctypes.c_int(-1), ctypes.c_int(-1), ctypes.c_int(-1)
    assert L.kf_get_state(h, ctypes.byref(C), ctypes.byref(p), ctypes.byref(B)) == Bd.KF_OK
    assert (C.value, p.value, B.value) == (0, 0, 0)
    L.kf_destroy(h)


def test_temperature_entry_point_checks(L):
    P = ctypes.c_void_p
    fake = P(0x10000)  # never dereferenced: every call below fails validation first
    plain = _ctx(L, _cfg())
    assert L.kf_set_temperature(plain, fake, 2) == Bd.KF_ESTATE  # no temperature encoder
    L.kf_destroy(plain)
    cfg = _cfg(flags=Bd.KF_FLAG_TEMPERATURE)
    assert L.kf_state_bytes(ctypes.byref(cfg)) > L.kf_state_bytes(ctypes.byref(_cfg()))
    h = _ctx(L, cfg)
    assert L.kf_set_temperature(h, None, 2) == Bd.KF_EINVAL
    assert L.kf_set_temperature(h, fake, 0) == Bd.KF_EINVAL
    assert L.kf_set_temperature(h, fake, 9) == Bd.KF_EINVAL
    assert L.kf_set_temperature(h, fake, 2) == Bd.KF_ESTATE  # no state buffer yet
    need = L.kf_state_bytes(ctypes.byref(cfg))
    assert L.kf_bind_state(h, fake, need) == Bd.KF_OK
    assert L.kf_set_temperature(h, fake, 2) == Bd.KF_ESTATE  # no weights yet
    # blobs with and without the encoder are told apart before any copy
    toy = S.WORKLOADS["toy"]["cfg"]
    plain_blob = S.pack_blob(toy, S.make_weights(toy))
    assert L.kf_load_weights(h, P(plain_blob.ctypes.data), plain_blob.nbytes, 0) == Bd.KF_EINVAL
    toy_t = dataclasses.replace(toy, temperature=True)
    t_blob = S.pack_blob(toy_t, S.make_weights(toy_t))
    bad = t_blob.copy()
    bad[:16].view(np.int32)[9] = 0
    assert L.kf_load_weights(h, P(bad.ctypes.data), bad.nbytes, 0) == Bd.KF_EINVAL
    assert b"header word 9" in L.kf_last_error(h)
    L.kf_destroy(h)


def test_training_attention_argument_checks(L):
    P = ctypes.c_void_p
    a = P(0x10000)  # 16-byte aligned, never dereferenced: each call fails validation first
    ok = dict(mask=0, B=2, H=3, N=8, k=4, dh=64)

    def call(**kw):
        x = dict(ok, **kw)
        ptrs = kw.get("ptrs", (a, a, a, a))
        return L.kf_training_attention(None, x["mask"], x["B"], x["H"], x["N"], x["k"], x["dh"],
                                       *ptrs, kw.get("scale", 0.125))

    assert call(mask=2) == Bd.KF_EINVAL
    assert call(mask=-1) == Bd.KF_EINVAL
    assert call(k=0) == Bd.KF_EINVAL
    assert call(B=-1) == Bd.KF_EINVAL
    assert call(N=-3) == Bd.KF_EINVAL
    for dh in (0, 16, 48, 96, 256):
        assert call(dh=dh) == Bd.KF_EINVAL
    assert call(scale=float("inf")) == Bd.KF_EINVAL
    assert call(scale=float("nan")) == Bd.KF_EINVAL
    assert call(ptrs=(a, None, a, a)) == Bd.KF_EINVAL
    assert call(ptrs=(a, a, P(0x10008), a)) == Bd.KF_EINVAL  # misaligned
    # per-head keys * d_head must stay below 2^31: N + 2Nk = 2^25 + ... keys at d_head 64
    assert call(mask=1, N=1 << 22, k=4) == Bd.KF_EINVAL
    # empty problems succeed without touching the (null) pointers or a device
    for mask in (0, 1):
        assert call(mask=mask, B=0, ptrs=(None,) * 4) == Bd.KF_OK
        assert call(mask=mask, N=0, ptrs=(None,) * 4) == Bd.KF_OK
        assert call(mask=mask, H=0, ptrs=(None,) * 4) == Bd.KF_OK


def test_training_attention_shapes():
    import oracle as O
    assert Bd.training_attention_shapes(Bd.KF_MASK_SINGLE, 5, 3) == (20, 20)
    assert Bd.training_attention_shapes(Bd.KF_MASK_DOUBLE, 5, 3) == (30, 35)
    for N, k in [(1, 1), (5, 3), (17, 4), (9, 8)]:
        for mask, kind in ((Bd.KF_MASK_SINGLE, "single"), (Bd.KF_MASK_DOUBLE, "double")):
            M = O.training_mask(kind, N, k)
            assert M.shape == Bd.training_attention_shapes(mask, N, k)
            assert Bd.training_attention_entries(mask, N, k) == int(M.sum())


def test_teacher_targets_argument_checks(L):
    P = ctypes.c_void_p
    fake = P(0x10000)  # never dereferenced: every call below fails validation first
    plain = _ctx(L, _cfg())
    assert L.kf_teacher_targets(plain, 1, 4, fake, fake, fake, fake) == Bd.KF_ESTATE  # no state
    L.kf_destroy(plain)
    cfg = _cfg(flags=Bd.KF_FLAG_TEACHER)
    assert L.kf_state_bytes(ctypes.byref(cfg)) > L.kf_state_bytes(ctypes.byref(_cfg()))
    h = _ctx(L, cfg)
    assert L.kf_teacher_targets(h, 1, 4, fake, fake, fake, fake) == Bd.KF_ESTATE  # no state buffer
    assert L.kf_bind_state(h, fake, L.kf_state_bytes(ctypes.byref(cfg))) == Bd.KF_OK
    assert L.kf_teacher_targets(h, 1, 4, fake, fake, fake, fake) == Bd.KF_ESTATE  # no weights
    L.kf_destroy(h)
    # argument ranges are checked after the state: a context without KF_FLAG_TEACHER
    # and with weights would say ESTATE; with the flag, bad sizes say EINVAL
    assert L.kf_teacher_targets(None, 1, 4, fake, fake, fake, fake) == Bd.KF_EINVAL


def test_selfforcing_argument_checks(L):
    P = ctypes.c_void_p
    fake = P(0x10000)  # never dereferenced: every call below fails validation first
    plain = _ctx(L, _cfg())
    assert L.kf_selfforcing_targets(plain, 1, 4, 2, fake, fake, fake, fake, fake) == Bd.KF_ESTATE
    L.kf_destroy(plain)
    cfg = _cfg(flags=Bd.KF_FLAG_ROLLOUT)
    assert L.kf_state_bytes(ctypes.byref(cfg)) > L.kf_state_bytes(ctypes.byref(_cfg()))
    h = _ctx(L, cfg)
    assert L.kf_selfforcing_targets(h, 1, 4, 2, fake, fake, fake, fake, fake) == Bd.KF_ESTATE
    L.kf_destroy(h)
    assert L.kf_selfforcing_targets(None, 1, 4, 2, fake, fake, fake, fake, fake) == Bd.KF_EINVAL


def test_serving_state_bytes_and_checks(L):
    """The KV pool of a serving context is kv_pages pages of 64 positions x
    n_layer x 2 x d_model elements; serving calls check their arguments before
    touching any device memory."""
    dense = _cfg(flags=Bd.KF_FLAG_SERVING, n_ctx=256)
    small = _cfg(flags=Bd.KF_FLAG_SERVING, n_ctx=256, kv_pages=5)
    page = Bd.KF_PAGE * 2 * 2 * 128 * 4  # positions x layers x (K, V) x d_model x fp32
    nd, ns = L.kf_state_bytes(ctypes.byref(dense)), L.kf_state_bytes(ctypes.byref(small))
    assert nd - ns >= (8 * 2 - 5) * page - 4096
    assert nd - ns <= (8 * 2 - 5) * page + 4096
    h = _ctx(L, small)
    P = ctypes.c_void_p
    fake = P(0x10000)
    one = (ctypes.c_int32 * 1)(3)
    two = (ctypes.c_int32 * 2)(1, 1)
    bad = (ctypes.c_int32 * 1)(8)
    # argument checks come first (no state bound yet)
    assert L.kf_serve_admit(h, 0, one, 4, fake, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_serve_admit(h, 2, two, 4, fake, 2, fake, fake) == Bd.KF_EINVAL  # repeated slot
    assert L.kf_serve_admit(h, 1, bad, 4, fake, 2, fake, fake) == Bd.KF_EINVAL  # slot >= max_batch
    assert L.kf_serve_admit(h, 1, None, 4, fake, 2, fake, fake) == Bd.KF_EINVAL
    assert L.kf_serve_admit(h, 1, one, 33, fake, 2, fake, fake) == Bd.KF_EINVAL  # N > max_prompt
    assert L.kf_serve_admit(h, 1, one, 4, fake, 5, fake, fake) == Bd.KF_EINVAL   # k > max_k
    assert L.kf_serve_admit(h, 1, one, 4, fake, 2, None, fake) == Bd.KF_EINVAL
    assert L.kf_serve_step(h, 1, one, 0, fake, fake) == Bd.KF_EINVAL
    assert L.kf_serve_admit(h, 1, one, 4, fake, 2, fake, fake) == Bd.KF_ESTATE   # nothing bound
    assert L.kf_serve_release(h, 1, one) == Bd.KF_ESTATE
    C, pend, pg = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    assert L.kf_serve_state(h, 3, ctypes.byref(C), ctypes.byref(pend), ctypes.byref(pg)) == Bd.KF_OK
    assert (C.value, pend.value, pg.value) == (-1, 0, 0)
    assert L.kf_serve_state(h, 8, None, None, None) == Bd.KF_EINVAL
    fr, tot = ctypes.c_int(), ctypes.c_int()
    assert L.kf_serve_pages(h, ctypes.byref(fr), ctypes.byref(tot)) == Bd.KF_OK
    assert (fr.value, tot.value) == (5, 5)
    L.kf_destroy(h)
    # a context without the flag refuses the serving calls
    h = _ctx(L, _cfg())
    assert L.kf_serve_admit(h, 1, one, 4, fake, 2, fake, fake) == Bd.KF_ESTATE
    assert L.kf_serve_step(h, 1, one, 2, fake, fake) == Bd.KF_ESTATE
    L.kf_destroy(h)


def test_null_context(L):
    assert L.kf_prefill(None, 1, 1, None, 1, None, None) == Bd.KF_EINVAL
    assert L.kf_create(None, None, None) == Bd.KF_EINVAL
    assert L.kf_last_error(None) == b"null context"
    L.kf_destroy(None)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(Bd, "_LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(Bd, "_lib", None)
    with pytest.raises(ImportError):
        Bd.lib()
