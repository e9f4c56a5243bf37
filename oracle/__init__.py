"""CPU oracle for the K-Forcing batched joint next-k-token decode.

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the cpu_baseline leg of bench.py, never by the product library.  It shares no
code with the HIP path; the only module both sides use is kf_synth (seeded
inputs, no arithmetic of the method).

Pieces:
  * kf_oracle.c  -- the loop-nest forward pass (fp64 parity instantiation and
    an fp32 instantiation for CPU timing), greedy head decoding and the
    inverse-CDF map;
  * this module  -- ctypes wrapper, the algorithm driver (prefill, decode
    blocks, generation, full recompute, AR decoding), the oracle's own
    Philox4x32-10 for the noise of a generation run, and an independent numpy
    dense-mask forward pass used as a brute-force pin (SingleForward /
    DoubleForward masks of Appendix C.2);
  * the Stage-1 distillation targets of the AR teacher (temperature-scaled
    inverse CDF at every position), the Stage-2 self-forcing targets (two
    dense-mask passes of a K-Forcing teacher) and plain masked attention
    under the training masks.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "kf_oracle.c")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile both instantiations of kf_oracle.c into liboracle.so (gcc)."""
    tmp = os.path.join(_HERE, "_build")
    os.makedirs(tmp, exist_ok=True)
    objs = []
    for real, sfx in (("double", "_f64"), ("float", "_f32")):
        obj = os.path.join(tmp, f"kf_oracle{sfx}.o")
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-std=c99", "-Wall", f"-DREAL={real}",
               f"-DSFX={sfx}", "-c", SRC_PATH, "-o", obj]
        subprocess.run(cmd, check=True, capture_output=not verbose)
        objs.append(obj)
    out_tmp = LIB_PATH + ".tmp"
    subprocess.run(["gcc", "-shared", "-fopenmp", "-o", out_tmp] + objs + ["-lm"],
                   check=True, capture_output=not verbose)
    os.replace(out_tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        for sfx in ("_f64", "_f32"):
            f = getattr(L, "orc_model_new" + sfx); f.restype = P; f.argtypes = [P, ctypes.c_long]
            f = getattr(L, "orc_model_free" + sfx); f.restype = None; f.argtypes = [P]
            f = getattr(L, "orc_seq_new" + sfx); f.restype = P; f.argtypes = [P]
            f = getattr(L, "orc_seq_free" + sfx); f.restype = None; f.argtypes = [P]
            f = getattr(L, "orc_seq_len" + sfx); f.restype = ctypes.c_int; f.argtypes = [P]
            f = getattr(L, "orc_seq_copy" + sfx); f.restype = ctypes.c_int; f.argtypes = [P, P]
            f = getattr(L, "orc_seq_set_temperature" + sfx); f.restype = ctypes.c_int
            f.argtypes = [P, ctypes.c_double]
            f = getattr(L, "orc_seq_kv" + sfx); f.restype = None
            f.argtypes = [P, ctypes.c_int, ctypes.c_int, dp]
            f = getattr(L, "orc_step" + sfx); f.restype = ctypes.c_int
            f.argtypes = [P, ctypes.c_int, ip, ctypes.c_int, dp, ctypes.c_int, dp, dp, dp]
            f = getattr(L, "orc_step_batch" + sfx); f.restype = ctypes.c_int
            f.argtypes = [ctypes.POINTER(P), ctypes.c_int, ctypes.c_int, ip, ctypes.c_int, dp,
                          ctypes.c_int, dp]
            f = getattr(L, "orc_argmax" + sfx); f.restype = ctypes.c_int; f.argtypes = [dp, ctypes.c_int]
            f = getattr(L, "orc_icdf" + sfx); f.restype = ctypes.c_int
            f.argtypes = [dp, ctypes.c_int, ctypes.c_double]
            f = getattr(L, "orc_softmax" + sfx); f.restype = ctypes.c_double
            f.argtypes = [dp, ctypes.c_int, dp]
            f = getattr(L, "orc_gelu" + sfx); f.restype = ctypes.c_double; f.argtypes = [ctypes.c_double]
            f = getattr(L, "orc_layernorm" + sfx); f.restype = None
            f.argtypes = [dp, dp, dp, ctypes.c_int, dp]
            f = getattr(L, "orc_rmsnorm" + sfx); f.restype = None
            f.argtypes = [dp, dp, ctypes.c_int, dp]
            f = getattr(L, "orc_rope" + sfx); f.restype = None
            f.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int]
            f = getattr(L, "orc_sinusoid" + sfx); f.restype = None
            f.argtypes = [ctypes.c_double, ctypes.c_int, dp]
            f = getattr(L, "orc_attend" + sfx); f.restype = ctypes.c_double
            f.argtypes = [dp, dp, dp, ctypes.c_int, ctypes.c_int, dp]
            f = getattr(L, "orc_round_bf16" + sfx); f.restype = ctypes.c_float
            f.argtypes = [ctypes.c_float]
        _lib = L
    return _lib


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f(name: str, prec: str):
    return getattr(lib(), f"{name}_{prec}")


# ---------------------------------------------------------------------------
# Model and sequence handles
# ---------------------------------------------------------------------------
class Model:
    """Weights parsed from a kf_synth blob (fp32 words; header in the first 16)."""

    def __init__(self, blob: np.ndarray, prec: str = "f64"):
        assert prec in ("f64", "f32")
        self.prec = prec
        self._blob = np.ascontiguousarray(blob, dtype=np.float32)
        hdr = self._blob[:16].view(np.int32)
        self.n_layer, self.d, self.H, self.f, self.V, self.T, self.dtype = (int(x) for x in hdr[2:9])
        self.h = _f("orc_model_new", prec)(self._blob.ctypes.data, self._blob.size)
        if not self.h:
            raise ValueError("oracle: malformed weight blob")

    def __del__(self):
        if getattr(self, "h", None):
            _f("orc_model_free", self.prec)(self.h)
            self.h = None

    def seq(self) -> "Seq":
        return Seq(self)


class Seq:
    """One sequence's committed KV cache (context only)."""

    def __init__(self, model: Model):
        self.model = model
        self.h = _f("orc_seq_new", model.prec)(model.h)

    def __del__(self):
        if getattr(self, "h", None):
            _f("orc_seq_free", self.model.prec)(self.h)
            self.h = None

    @property
    def C(self) -> int:
        return _f("orc_seq_len", self.model.prec)(self.h)

    def copy(self) -> "Seq":
        """A new sequence holding this one's committed context."""
        s = Seq(self.model)
        if _f("orc_seq_copy", self.model.prec)(s.h, self.h) < 0:
            raise ValueError("oracle: sequence copy across models")
        return s

    def set_temperature(self, tau: float) -> None:
        """Temperature conditioning of this sequence's later noise rows."""
        if _f("orc_seq_set_temperature", self.model.prec)(self.h, float(tau)) < 0:
            raise ValueError("oracle: the model has no temperature encoder")

    def kv(self, layer: int, which: int) -> np.ndarray:
        out = np.zeros((self.C, self.model.d), np.float64)
        _f("orc_seq_kv", self.model.prec)(self.h, layer, which, _dp(out))
        return out

    def step(self, toks: Sequence[int], u: Sequence[float], commit: bool = True,
             want_hidden: bool = False):
        """nr real rows then k noise rows; returns (logits [nh, V], softmax_dev[, hidden])."""
        toks = np.ascontiguousarray(np.asarray(toks, np.int32).reshape(-1))
        u = np.ascontiguousarray(np.asarray(u, np.float64).reshape(-1))
        nr, k = toks.size, u.size
        nh = k if k > 0 else 1
        logits = np.zeros((nh, self.model.V), np.float64)
        hidden = np.zeros((nr + k, self.model.d), np.float64) if want_hidden else None
        dev = np.zeros(1, np.float64)
        rc = _f("orc_step", self.model.prec)(
            self.h, nr, _ip(toks), k, _dp(u), int(commit), _dp(logits),
            _dp(hidden) if want_hidden else None, _dp(dev))
        if rc < 0:
            raise ValueError(f"oracle step rejected (nr={nr}, k={k}, C={self.C})")
        if want_hidden:
            return logits, float(dev[0]), hidden
        return logits, float(dev[0])


def argmax(logits: np.ndarray) -> np.ndarray:
    """Greedy head decoding per row: argmax, exact ties to the lowest id."""
    lg = np.ascontiguousarray(np.atleast_2d(logits), np.float64)
    f = _f("orc_argmax", "f64")
    return np.array([f(_dp(np.ascontiguousarray(r)), lg.shape[1]) for r in lg], np.int32)


def softmax(logits: np.ndarray) -> np.ndarray:
    lg = np.ascontiguousarray(logits, np.float64)
    q = np.zeros_like(lg)
    _f("orc_softmax", "f64")(_dp(lg), lg.size, _dp(q))
    return q


def icdf(q: Sequence[float], z: float) -> int:
    """Inverse-CDF map with the strict-inequality convention of Appendix B."""
    q = np.ascontiguousarray(np.asarray(q, np.float64))
    return int(_f("orc_icdf", "f64")(_dp(q), q.size, float(z)))


def rmsnorm(x, g, prec: str = "f64") -> np.ndarray:
    x = np.ascontiguousarray(x, np.float64)
    g = np.ascontiguousarray(g, np.float64)
    y = np.zeros_like(x)
    _f("orc_rmsnorm", prec)(_dp(x), _dp(g), x.size, _dp(y))
    return y


def rope(x, H: int, dh: int, p: int, prec: str = "f64") -> np.ndarray:
    """The oracle's rotary map of one row x [H*dh] at position p."""
    y = np.ascontiguousarray(np.array(x, np.float64))
    _f("orc_rope", prec)(_dp(y), H, dh, int(p))
    return y


def gelu(x: float, prec: str = "f64") -> float:
    return float(_f("orc_gelu", prec)(float(x)))


def layernorm(x, g, b, prec: str = "f64") -> np.ndarray:
    x = np.ascontiguousarray(x, np.float64); g = np.ascontiguousarray(g, np.float64)
    b = np.ascontiguousarray(b, np.float64)
    y = np.zeros_like(x)
    _f("orc_layernorm", prec)(_dp(x), _dp(g), _dp(b), x.size, _dp(y))
    return y


def sinusoid(u: float, d: int, prec: str = "f64") -> np.ndarray:
    e = np.zeros(d, np.float64)
    _f("orc_sinusoid", prec)(float(u), d, _dp(e))
    return e


def attend(q, K, V, prec: str = "f64") -> Tuple[np.ndarray, float]:
    q = np.ascontiguousarray(q, np.float64); K = np.ascontiguousarray(K, np.float64)
    V = np.ascontiguousarray(V, np.float64)
    o = np.zeros(q.size, np.float64)
    s = _f("orc_attend", prec)(_dp(q), _dp(K), _dp(V), K.shape[0], q.size, _dp(o))
    return o, float(s)


def round_bf16(x: float) -> float:
    return float(_f("orc_round_bf16", "f64")(float(x)))


# ---------------------------------------------------------------------------
# The oracle's own Philox4x32-10 (Salmon et al., SC'11), for generation runs
# ---------------------------------------------------------------------------

def philox4x32_10(ctr: Sequence[int], key: Sequence[int]) -> Tuple[int, int, int, int]:
    c = [int(x) & 0xFFFFFFFF for x in ctr]
    k0, k1 = int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF
    for rnd in range(10):
        if rnd:
            k0 = (k0 + 0x9E3779B9) & 0xFFFFFFFF
            k1 = (k1 + 0xBB67AE85) & 0xFFFFFFFF
        p0 = 0xD2511F53 * c[0]
        p1 = 0xCD9E8D57 * c[2]
        c = [((p1 >> 32) ^ c[1] ^ k0) & 0xFFFFFFFF, p1 & 0xFFFFFFFF,
             ((p0 >> 32) ^ c[3] ^ k1) & 0xFFFFFFFF, p0 & 0xFFFFFFFF]
    return c[0], c[1], c[2], c[3]


def noise_u(seed: int, b: int, p: int) -> float:
    """u for sequence b and absolute emitted position p (noise stream 2)."""
    seed &= 0xFFFFFFFFFFFFFFFF
    w0 = philox4x32_10((p, b, 2, 0), (seed & 0xFFFFFFFF, seed >> 32))[0]
    return (w0 >> 8) * (1.0 / 16777216.0)


# ---------------------------------------------------------------------------
# The algorithm (Appendix C.1) driven over the per-sequence core
# ---------------------------------------------------------------------------

def prefill(model: Model, prompt: Sequence[int], u: Sequence[float]):
    """First step: prompt rows plus k noise rows; commits the prompt (C = N)."""
    s = model.seq()
    logits, dev = s.step(prompt, u, commit=True)
    return s, logits, argmax(logits)


def decode(seq: Seq, pending: Sequence[int], u: Sequence[float]):
    """Later steps: the previously emitted tokens plus fresh noise rows."""
    logits, dev = seq.step(pending, u, commit=True)
    return logits, argmax(logits)


def full_recompute(model: Model, history: Sequence[int], u: Sequence[float]):
    """No cache: one causal pass over [prompt, emitted tokens, k noise rows]."""
    s = model.seq()
    logits, _ = s.step(history, u, commit=False)
    return logits


def generate(model: Model, prompt: np.ndarray, L: int, k: int, seed: int,
             rows: Optional[Sequence[int]] = None):
    """K-Forcing generation of L new tokens per sequence (L % k == 0).

    Returns (tokens [len(rows), L], number of forward passes per sequence)."""
    prompt = np.asarray(prompt, np.int32)
    B, N = prompt.shape
    rows = list(range(B)) if rows is None else list(rows)
    out = np.zeros((len(rows), L), np.int32)
    passes = 0
    for ri, b in enumerate(rows):
        passes = 0
        s = model.seq()
        pending = list(prompt[b])
        p = N
        while p < N + L:
            u = [noise_u(seed, b, p + j) for j in range(k)]
            logits, _ = s.step(pending, u, commit=True)
            toks = argmax(logits)
            out[ri, p - N:p - N + k] = toks
            pending = list(toks)
            p += k
            passes += 1
    return out, passes


def ar_step(seq: Seq, pending: Sequence[int], u: float):
    """AR decoding: feed the pending real rows, sample the next token by inverse CDF."""
    logits, _ = seq.step(pending, [], commit=True)
    q = softmax(logits[0])
    return logits[0], icdf(q, u)


def generate_ar(model: Model, prompt: np.ndarray, L: int, seed: int,
                rows: Optional[Sequence[int]] = None):
    prompt = np.asarray(prompt, np.int32)
    B, N = prompt.shape
    rows = list(range(B)) if rows is None else list(rows)
    out = np.zeros((len(rows), L), np.int32)
    for ri, b in enumerate(rows):
        s = model.seq()
        pending = list(prompt[b])
        for p in range(N, N + L):
            _, tok = ar_step(s, pending, noise_u(seed, b, p))
            out[ri, p - N] = tok
            pending = [tok]
    return out


def tempered_icdf(logits: np.ndarray, tau: float, u: float) -> int:
    """The teacher's sampler of forward distillation (Appendix C.2, Stage-1
    algorithm): the inverse-CDF map (strict convention) of softmax(logits / tau)
    at u."""
    return icdf(softmax(np.asarray(logits, np.float64) / float(tau)), u)


def teacher_targets(model: Model, tokens: np.ndarray, tau: Sequence[float], u: np.ndarray,
                    rows: Optional[Sequence[int]] = None):
    """Stage-1 distillation targets (Appendix C.2, forward distillation, the
    teacher's lines): an AR causal pass over each sequence's tokens; at
    position p the target is tempered_icdf of the next-token logits at
    u[b][p] with the sequence's temperature tau[b].

    Returns (targets [len(rows), N], logits [len(rows), N, V])."""
    tokens = np.asarray(tokens, np.int32)
    u = np.asarray(u, np.float64)
    B, N = tokens.shape
    rows = list(range(B)) if rows is None else list(rows)
    out = np.zeros((len(rows), N), np.int32)
    lg = np.zeros((len(rows), N, model.V), np.float64)
    for ri, b in enumerate(rows):
        s = model.seq()
        for p in range(N):
            logits, _ = s.step([int(tokens[b, p])], [], commit=True)
            lg[ri, p] = logits[0]
            out[ri, p] = tempered_icdf(logits[0], float(tau[b]), float(u[b, p]))
    return out, lg


def tempered_margin(logits: np.ndarray, tau: float, u: float) -> float:
    """Distance from u to the nearest CDF boundary of softmax(logits / tau)."""
    return cdf_margin(np.asarray(logits, np.float64) / float(tau), u)


def cdf_margin(logits: np.ndarray, u: float) -> float:
    """Distance from u to the nearest CDF boundary of the inverse-CDF decision."""
    q = softmax(logits)
    F = np.cumsum(q)
    return float(np.min(np.abs(np.concatenate([[0.0], F]) - u)))


# ---------------------------------------------------------------------------
# Independent numpy brute force: dense attention masks over whole sequences
# ---------------------------------------------------------------------------

def _bf16_np(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return u.view(np.float32)


def parse_blob(blob: np.ndarray) -> Tuple[dict, dict]:
    """Weights as fp64 numpy arrays (2-D tensors rounded to bf16 for bf16 models)."""
    blob = np.asarray(blob, np.float32)
    hdr = blob[:16].view(np.int32)
    L, d, H, f, V, T, dt = (int(x) for x in hdr[2:9])
    temp = bool(int(hdr[9]) & 1)
    rope = bool(int(hdr[9]) & 2)
    shapes = [("tok", (V, d)), ("pos", (T, d)), ("nw1", (4 * d, d)), ("nb1", (4 * d,)),
              ("nw2", (d, 4 * d)), ("nb2", (d,))]
    for l in range(L):
        shapes += [(f"{l}.ln1_g", (d,)), (f"{l}.ln1_b", (d,)), (f"{l}.wqkv", (3 * d, d)),
                   (f"{l}.bqkv", (3 * d,)), (f"{l}.wo", (d, d)), (f"{l}.bo", (d,)),
                   (f"{l}.ln2_g", (d,)), (f"{l}.ln2_b", (d,)), (f"{l}.w1", (f, d)),
                   (f"{l}.b1", (f,)), (f"{l}.w2", (d, f)), (f"{l}.b2", (d,))]
    shapes += [("lnf_g", (d,)), ("lnf_b", (d,))]
    if temp:
        shapes += [("tw1", (d, d)), ("tb1", (d,)), ("tw2", (d, d)), ("tb2", (d,))]
    W = {}
    off = 16
    for name, shp in shapes:
        n = int(np.prod(shp))
        a = blob[off:off + n]
        if len(shp) == 2 and dt == 1:
            a = _bf16_np(a)
        W[name] = a.astype(np.float64).reshape(shp)
        off += n
    assert off == blob.size
    return dict(L=L, d=d, H=H, f=f, V=V, T=T, temperature=temp, rms_rope=rope), W


def _np_ln(x, g, b):
    mu = x.mean(-1, keepdims=True)
    var = ((x - mu) ** 2).mean(-1, keepdims=True)
    return (x - mu) / np.sqrt(var + 1e-5) * g + b


def _np_rms(x, g):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + 1e-5) * g


def _np_rope(x, positions, H, dh):
    """RoFormer rotary map on rows x [n][H*dh] at the given positions: in each
    head, pairs (2i, 2i+1), i < d_rot/2, d_rot = min(64, dh), turned by
    p * 10000^(-2i/d_rot)."""
    x = np.array(x, np.float64)
    dr = min(64, dh)
    i = np.arange(dr // 2)
    ang = np.asarray(positions, np.float64)[:, None] * 10000.0 ** (-2.0 * i / dr)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    for h in range(H):
        x0 = x[:, h * dh + 2 * i].copy()
        x1 = x[:, h * dh + 2 * i + 1].copy()
        x[:, h * dh + 2 * i] = x0 * c - x1 * s
        x[:, h * dh + 2 * i + 1] = x0 * s + x1 * c
    return x


def _np_gelu(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def _np_sinusoid(u, d):
    h = d // 2
    w = 10000.0 ** (-np.arange(h) / h)
    a = 1000.0 * np.asarray(u, np.float64)[:, None] * w[None, :]
    return np.concatenate([np.cos(a), np.sin(a)], axis=1)


def dense_forward(cfg: dict, W: dict, rows: List[Tuple[str, float]], positions: Sequence[int],
                  mask: np.ndarray, tau: float = None) -> np.ndarray:
    """Whole-sequence forward with an explicit boolean mask[q, key]; returns logits per row.

    rows[i] is ("tok", id) or ("noise", u); tau (temperature models) conditions
    every noise row with W_t2 GELU(W_t1 sin(tau) + b_t1) + b_t2."""
    d, H = cfg["d"], cfg["H"]
    dh = d // H
    n = len(rows)
    X = np.zeros((n, d))
    pos = np.asarray(positions)
    tok_idx = [i for i, r in enumerate(rows) if r[0] == "tok"]
    noi_idx = [i for i, r in enumerate(rows) if r[0] == "noise"]
    if tok_idx:
        X[tok_idx] = W["tok"][[int(rows[i][1]) for i in tok_idx]]
    if noi_idx:
        E = _np_sinusoid([rows[i][1] for i in noi_idx], d)
        Hn = _np_gelu(E @ W["nw1"].T + W["nb1"])
        X[noi_idx] = Hn @ W["nw2"].T + W["nb2"]
        if cfg.get("temperature"):
            Et = _np_sinusoid([tau], d)[0]
            X[noi_idx] += _np_gelu(Et @ W["tw1"].T + W["tb1"]) @ W["tw2"].T + W["tb2"]
    rope = cfg.get("rms_rope", False)
    nrm = (lambda x, g, b: _np_rms(x, g)) if rope else _np_ln
    if not rope:
        X = X + W["pos"][pos]
    neg = np.where(mask, 0.0, -np.inf)
    for l in range(cfg["L"]):
        A = nrm(X, W[f"{l}.ln1_g"], W[f"{l}.ln1_b"])
        QKV = A @ W[f"{l}.wqkv"].T + W[f"{l}.bqkv"]
        Q, K, Vv = QKV[:, :d], QKV[:, d:2 * d], QKV[:, 2 * d:]
        if rope:
            Q, K = _np_rope(Q, pos, H, dh), _np_rope(K, pos, H, dh)
        O = np.zeros((n, d))
        for h in range(H):
            sl = slice(h * dh, (h + 1) * dh)
            S = Q[:, sl] @ K[:, sl].T / np.sqrt(dh) + neg
            S = S - S.max(axis=1, keepdims=True)
            P = np.exp(S)
            P = P / P.sum(axis=1, keepdims=True)
            O[:, sl] = P @ Vv[:, sl]
        X = X + O @ W[f"{l}.wo"].T + W[f"{l}.bo"]
        A = nrm(X, W[f"{l}.ln2_g"], W[f"{l}.ln2_b"])
        X = X + _np_gelu(A @ W[f"{l}.w1"].T + W[f"{l}.b1"]) @ W[f"{l}.w2"].T + W[f"{l}.b2"]
    return nrm(X, W["lnf_g"], W["lnf_b"]) @ W["tok"].T


def single_forward_layout(N: int, k: int):
    """SingleForward (Appendix C.2): N context tokens then N groups of k noise tokens.

    Returns (mask [(N+Nk)^2], positions, group index per row (-1 for context)).
    Context->context causal; group t (t = 1..N) sees x_1..x_t (staircase) and
    its own group causally (block-diagonal causal).  Noise j of group t sits at
    0-based position t + j, the position of the token it emits."""
    n = N + N * k
    M = np.zeros((n, n), bool)
    pos = np.zeros(n, np.int64)
    grp = -np.ones(n, np.int64)
    for i in range(N):
        M[i, :i + 1] = True
        pos[i] = i
    for t in range(1, N + 1):
        for j in range(k):
            r = N + (t - 1) * k + j
            M[r, :t] = True
            M[r, N + (t - 1) * k:r + 1] = True
            pos[r] = t + j
            grp[r] = t
    return M, pos, grp


def double_forward_layout(N: int, k: int):
    """DoubleForward (Appendix C.2): context, Future-1 (N groups of k tokens),
    Future-2 (N groups of k noise tokens).  Square mask over all N + 2Nk rows.

    F1 rows follow SingleForward; F2 group t sees x_1..x_t, all k F1 tokens of
    its window, and its own F2 group causally.  F1 token j of group t sits at
    position t + j, F2 token j at t + k + j."""
    n = N + 2 * N * k
    M = np.zeros((n, n), bool)
    pos = np.zeros(n, np.int64)
    for i in range(N):
        M[i, :i + 1] = True
        pos[i] = i
    for t in range(1, N + 1):
        f1 = N + (t - 1) * k
        f2 = N + N * k + (t - 1) * k
        for j in range(k):
            M[f1 + j, :t] = True
            M[f1 + j, f1:f1 + j + 1] = True
            pos[f1 + j] = t + j
            M[f2 + j, :t] = True
            M[f2 + j, f1:f1 + k] = True
            M[f2 + j, f2:f2 + j + 1] = True
            pos[f2 + j] = t + k + j
    return M, pos


def nnz_single(N: int, k: int) -> int:
    """|M_S| closed form (Appendix C.2, theoretical training cost)."""
    return N * (N + 1) // 2 + k * N * (N + 1) // 2 + N * k * (k + 1) // 2


def nnz_double(N: int, k: int) -> int:
    """|M_D| closed form over the Future-2 queries (Appendix C.2)."""
    return k * N * (N + 1) // 2 + N * k * k + N * k * (k + 1) // 2


def decode_batched(seqs: Sequence[Seq], pending: np.ndarray, k: int, u: np.ndarray) -> np.ndarray:
    """One decode block over several sequences at once (one orc_step_batch
    call, OpenMP over sequences): pending [B][nr] real rows, u [B][k] noise;
    commits the real rows and returns the argmax tokens [B][k]."""
    B = len(seqs)
    model = seqs[0].model
    arr = (ctypes.c_void_p * B)(*[s.h for s in seqs])
    toks = np.ascontiguousarray(pending, np.int32).reshape(B, -1)
    u = np.ascontiguousarray(u, np.float64).reshape(B, k)
    logits = np.zeros((B, k, model.V), np.float64)
    rc = _f("orc_step_batch", model.prec)(arr, B, toks.shape[1], _ip(toks), k, _dp(u), 1,
                                         _dp(logits))
    if rc < 0:
        raise ValueError("oracle batched step rejected")
    return np.stack([argmax(logits[b]) for b in range(B)])


def generate_batched(model: Model, prompt: np.ndarray, L: int, k: int, seed: int) -> np.ndarray:
    """generate() over all rows at once, one orc_step_batch call per block
    (OpenMP over sequences in the C core).  Same result as generate()."""
    prompt = np.ascontiguousarray(prompt, np.int32)
    B, N = prompt.shape
    seqs = [model.seq() for _ in range(B)]
    arr = (ctypes.c_void_p * B)(*[s.h for s in seqs])
    out = np.zeros((B, L), np.int32)
    pending = prompt
    f = _f("orc_step_batch", model.prec)
    for p in range(N, N + L, k):
        u = np.array([[noise_u(seed, b, p + j) for j in range(k)] for b in range(B)], np.float64)
        logits = np.zeros((B, k, model.V), np.float64)
        toks = np.ascontiguousarray(pending, np.int32)
        rc = f(arr, B, toks.shape[1], _ip(toks), k, _dp(u), 1, _dp(logits))
        if rc < 0:
            raise ValueError("oracle batched step rejected")
        pending = np.stack([argmax(logits[b]) for b in range(B)])
        out[:, p - N:p - N + k] = pending
    return out


def masked_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, mask: np.ndarray,
                     scale: float) -> np.ndarray:
    """Attention with an explicit boolean mask, the plain definition in fp64:
    per (batch, head), O = softmax(scale * Q K^T over the visible keys) V.
    Q [B][H][nq][dh], K and V [B][H][nk][dh], mask [nq][nk]; every query row
    must see at least one key."""
    Q, K, V = (np.asarray(a, np.float64) for a in (Q, K, V))
    assert mask.shape == (Q.shape[2], K.shape[2]) and mask.any(axis=1).all()
    S = np.einsum("bhqd,bhkd->bhqk", Q, K) * scale
    S = np.where(mask[None, None], S, -np.inf)
    S = S - S.max(axis=-1, keepdims=True)
    P = np.exp(S)
    P /= P.sum(axis=-1, keepdims=True)
    return np.einsum("bhqk,bhkd->bhqd", P, V)


def selfforcing_targets(cfg: dict, W: dict, tokens: np.ndarray, k: int, z1: np.ndarray,
                        z2: np.ndarray, tau: Optional[Sequence[float]] = None,
                        x1_forced: Optional[np.ndarray] = None):
    """Stage-2 self-forcing targets (Appendix C.2, self-forcing distillation,
    the teacher's lines) with the dense masks.  Per sequence b:
      round 1: SingleForward over [context | noise z1[b]]; x1 = argmax of
               each noise row (group t, token j);
      round 2: DoubleForward over [context | Future-1 tokens | Future-2 noise
               z2[b]]; x2 = argmax of each Future-2 row.
    Future-1 carries x1, or x1_forced[b] when given (teacher forcing).
    Returns x1, x2 [B][N][k] and the logits of both rounds' noise rows
    [B][N*k][V]."""
    tokens = np.asarray(tokens)
    B, N = tokens.shape
    z1 = np.asarray(z1, np.float64).reshape(B, N * k)
    z2 = np.asarray(z2, np.float64).reshape(B, N * k)
    MS, posS, _ = single_forward_layout(N, k)
    MD, posD = double_forward_layout(N, k)
    x1 = np.zeros((B, N * k), np.int32)
    x2 = np.zeros((B, N * k), np.int32)
    l1 = np.zeros((B, N * k, cfg["V"]))
    l2 = np.zeros((B, N * k, cfg["V"]))
    for b in range(B):
        tb = None if tau is None else float(tau[b])
        ctx = [("tok", int(t)) for t in tokens[b]]
        rows = ctx + [("noise", float(z)) for z in z1[b]]
        l1[b] = dense_forward(cfg, W, rows, posS, MS, tau=tb)[N:]
        x1[b] = argmax(l1[b])
        f1 = x1[b] if x1_forced is None else np.asarray(x1_forced[b]).reshape(-1)
        rows = ctx + [("tok", int(t)) for t in f1] + [("noise", float(z)) for z in z2[b]]
        l2[b] = dense_forward(cfg, W, rows, posD, MD, tau=tb)[N + N * k:]
        x2[b] = argmax(l2[b])
    return x1.reshape(B, N, k), x2.reshape(B, N, k), l1, l2


def training_mask(kind: str, N: int, k: int) -> np.ndarray:
    """Query x key mask of the training attention calls (Appendix C.2):
    "single" = M_S over all N + Nk tokens; "double" = M_D, the Future-1 and
    Future-2 query rows over the N + 2Nk context, Future-1, Future-2 keys."""
    if kind == "single":
        return single_forward_layout(N, k)[0]
    if kind == "double":
        return double_forward_layout(N, k)[0][N:]
    raise ValueError(kind)
