"""Seeded synthetic inputs for the K-Forcing decode path.

This module holds no arithmetic of the method itself. It only draws the
inputs that both the HIP path and the CPU oracle consume:

* model weights  (Gaussian N(0, std) via Box-Muller, optionally random affine
  parameters for tests),
* prompt token ids (uniform over the vocabulary, or truncated Zipf(s)),
* noise blocks u in [0, 1) handed to an explicit decode call,
* query/key/value tensors of the training-mask attention (bfloat16 values).

Every random word comes from the counter-based generator Philox4x32-10
(Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC'11), written here from that paper's definition: ten rounds of two 32x32->64
bit multiplies with the constants 0xD2511F53 / 0xCD9E8D57 and a Weyl key
schedule 0x9E3779B9 / 0xBB67AE85.  Counters and streams:

    key      = (seed & 0xffffffff, seed >> 32)
    weights  : counter = (call index, tensor index, 0, 0)
    prompts  : counter = (position i, sequence b, 1, 0)
    noise    : counter = (absolute emitted position p, sequence b, 2, 0)
    u        = (word0 >> 8) * 2**-24            (24-bit uniform in [0, 1))

The noise rule lets k = 1, 2, 4 and the autoregressive baseline consume the
same u for the same emitted position.

Attention inputs are many (up to ~10^9 values at a training batch), so they
come from numpy's PCG64 instead, seeded with (seed, 3, b, h) per sequence and
head, so that any one (b, h) slice can be drawn again on its own.
"""
from __future__ import annotations

import dataclasses
import json
import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Philox4x32-10
# ---------------------------------------------------------------------------
_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = 0x9E3779B9
_W1 = 0xBB67AE85
_MASK = np.uint64(0xFFFFFFFF)

STREAM_WEIGHTS = 0
STREAM_PROMPTS = 1
STREAM_NOISE = 2


def philox4x32_10(c0, c1, c2, c3, key: Tuple[int, int]):
    """Vectorised Philox4x32-10 on uint32 counter arrays; returns 4 uint32 arrays."""
    c0 = np.asarray(c0, dtype=np.uint64) & _MASK
    c1 = np.asarray(c1, dtype=np.uint64) & _MASK
    c2 = np.asarray(c2, dtype=np.uint64) & _MASK
    c3 = np.asarray(c3, dtype=np.uint64) & _MASK
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    k0, k1 = int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _W0) & 0xFFFFFFFF
            k1 = (k1 + _W1) & 0xFFFFFFFF
        p0 = _M0 * c0
        p1 = _M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1,
                          hi0 ^ c3 ^ np.uint64(k1), lo0)
    return (c0.astype(np.uint32), c1.astype(np.uint32),
            c2.astype(np.uint32), c3.astype(np.uint32))


def seed_key(seed: int) -> Tuple[int, int]:
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & 0xFFFFFFFF, seed >> 32


def word_to_unit(w: np.ndarray) -> np.ndarray:
    """24-bit uniform in [0, 1): (w >> 8) * 2^-24, exact in float32."""
    return ((np.asarray(w, dtype=np.uint32) >> np.uint32(8)).astype(np.float64)
            * (1.0 / 16777216.0))


# ---------------------------------------------------------------------------
# Draws
# ---------------------------------------------------------------------------

def normal(seed: int, tensor_index: int, n: int, std: float) -> np.ndarray:
    """n draws of N(0, std^2) as float32 (Box-Muller on Philox words)."""
    calls = (n + 3) // 4
    idx = np.arange(calls, dtype=np.uint64)
    w0, w1, w2, w3 = philox4x32_10(idx, np.uint64(tensor_index), 0, 0, seed_key(seed))
    out = np.empty((calls, 4), dtype=np.float64)
    for col, (wa, wb) in enumerate(((w0, w1), (w2, w3))):
        u1 = ((wa >> np.uint32(8)).astype(np.float64) + 1.0) * (1.0 / 16777216.0)  # (0, 1]
        u2 = (wb >> np.uint32(8)).astype(np.float64) * (1.0 / 16777216.0)         # [0, 1)
        r = np.sqrt(-2.0 * np.log(u1))
        out[:, 2 * col] = r * np.cos(2.0 * math.pi * u2)
        out[:, 2 * col + 1] = r * np.sin(2.0 * math.pi * u2)
    return (out.reshape(-1)[:n] * std).astype(np.float32)


def noise_block(seed: int, B: int, p0: int, k: int) -> np.ndarray:
    """u[b, j] for emitted positions p0 .. p0+k-1 (float32, exact 24-bit values)."""
    p = np.arange(p0, p0 + k, dtype=np.uint64)[None, :]
    b = np.arange(B, dtype=np.uint64)[:, None]
    w0, _, _, _ = philox4x32_10(p, b, STREAM_NOISE, 0, seed_key(seed))
    return word_to_unit(w0).astype(np.float32)


def prompts_uniform(seed: int, B: int, N: int, V: int) -> np.ndarray:
    i = np.arange(N, dtype=np.uint64)[None, :]
    b = np.arange(B, dtype=np.uint64)[:, None]
    w0, _, _, _ = philox4x32_10(i, b, STREAM_PROMPTS, 0, seed_key(seed))
    return (word_to_unit(w0) * V).astype(np.int64).clip(0, V - 1).astype(np.int32)


def prompts_zipf(seed: int, B: int, N: int, V: int, s: float = 1.1) -> np.ndarray:
    """Truncated Zipf over ranks 1..V, P(r) ~ r^-s, token id = r - 1 (inverse CDF)."""
    ranks = np.arange(1, V + 1, dtype=np.float64)
    cdf = np.cumsum(ranks ** (-s))
    cdf /= cdf[-1]
    i = np.arange(N, dtype=np.uint64)[None, :]
    b = np.arange(B, dtype=np.uint64)[:, None]
    w0, _, _, _ = philox4x32_10(i, b, STREAM_PROMPTS, 0, seed_key(seed))
    u = word_to_unit(w0)
    ids = np.searchsorted(cdf, u, side="right")
    return ids.clip(0, V - 1).astype(np.int32)


# ---------------------------------------------------------------------------
# Model configuration and the flat weight blob
# ---------------------------------------------------------------------------
DTYPE_FP32 = 0
DTYPE_BF16 = 1
BLOB_MAGIC = 0x4B465731          # "KFW1"
BLOB_VERSION = 1
HEADER_INTS = 16


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    n_layer: int
    d_model: int
    n_head: int
    d_mlp: int
    vocab: int
    n_ctx: int
    dtype: int  # DTYPE_FP32 or DTYPE_BF16
    temperature: bool = False  # temperature-conditioned noise encoder
    rms_rope: bool = False     # RMSNorm + rotary positions (no learned positions)

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_head


def tensor_table(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical order and shapes of the blob's tensors.

    Matrices are stored [out_features][in_features]; the token table doubles as
    the (tied) output head.  2-D tensors are "matrices" and are held in the
    compute dtype by a consumer; 1-D tensors (biases, norm gains) stay fp32.
    """
    d, f, V, T = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.n_ctx
    t: List[Tuple[str, Tuple[int, ...]]] = [
        ("tok_emb", (V, d)),
        ("pos_emb", (T, d)),
        ("noise_w1", (4 * d, d)),
        ("noise_b1", (4 * d,)),
        ("noise_w2", (d, 4 * d)),
        ("noise_b2", (d,)),
    ]
    for l in range(cfg.n_layer):
        t += [
            (f"l{l}.ln1_g", (d,)), (f"l{l}.ln1_b", (d,)),
            (f"l{l}.w_qkv", (3 * d, d)), (f"l{l}.b_qkv", (3 * d,)),
            (f"l{l}.w_o", (d, d)), (f"l{l}.b_o", (d,)),
            (f"l{l}.ln2_g", (d,)), (f"l{l}.ln2_b", (d,)),
            (f"l{l}.w_1", (f, d)), (f"l{l}.b_1", (f,)),
            (f"l{l}.w_2", (d, f)), (f"l{l}.b_2", (d,)),
        ]
    t += [("lnf_g", (d,)), ("lnf_b", (d,))]
    if cfg.temperature:  # tau sinusoid -> Linear(d, d) -> GELU -> Linear(d, d)
        t += [("temp_w1", (d, d)), ("temp_b1", (d,)), ("temp_w2", (d, d)), ("temp_b2", (d,))]
    return t


def n_params(cfg: ModelConfig) -> int:
    return int(sum(int(np.prod(s)) for _, s in tensor_table(cfg)))


BLOB_FLAG_TEMPERATURE = 1  # header word 9: the temperature encoder's tensors follow lnf_b
BLOB_FLAG_RMS_ROPE = 2     # header word 9: RMSNorm + rotary positions (pos and norm shifts unused)


def header(cfg: ModelConfig) -> np.ndarray:
    h = np.zeros(HEADER_INTS, dtype=np.int32)
    h[:10] = [BLOB_MAGIC, BLOB_VERSION, cfg.n_layer, cfg.d_model, cfg.n_head,
              cfg.d_mlp, cfg.vocab, cfg.n_ctx, cfg.dtype,
              (BLOB_FLAG_TEMPERATURE if cfg.temperature else 0)
              | (BLOB_FLAG_RMS_ROPE if cfg.rms_rope else 0)]
    return h


def make_weights(cfg: ModelConfig, seed: int = 0, std: float = 0.02,
                 random_affine: bool = False) -> Dict[str, np.ndarray]:
    """Seeded weights.  Default: every matrix ~ N(0, std^2), biases 0, gains 1.

    random_affine=True also randomises biases (N(0, std^2)) and norm gains
    (1 + N(0, 0.1^2)) and shifts (N(0, std^2)) so that tests see every term.
    """
    out: Dict[str, np.ndarray] = {}
    for ti, (name, shape) in enumerate(tensor_table(cfg)):
        n = int(np.prod(shape))
        base = name.split(".")[-1]
        if cfg.rms_rope and (name == "pos_emb" or (base.endswith("_b") and base.startswith("ln"))):
            arr = np.zeros(n, np.float32)  # a rotary RMSNorm model has neither
        elif len(shape) == 2:
            arr = normal(seed, ti, n, std)
        elif base.endswith("_g"):
            arr = (np.ones(n, np.float32) if not random_affine
                   else (1.0 + normal(seed, ti, n, 0.1)).astype(np.float32))
        else:
            arr = (np.zeros(n, np.float32) if not random_affine
                   else normal(seed, ti, n, std))
        out[name] = arr.reshape(shape)
    return out


def pack_blob(cfg: ModelConfig, weights: Dict[str, np.ndarray]) -> np.ndarray:
    """Flat blob: 16 int32 header words followed by every tensor as fp32, in order."""
    parts = [header(cfg).view(np.float32)]
    for name, shape in tensor_table(cfg):
        arr = np.ascontiguousarray(weights[name], dtype=np.float32)
        assert arr.shape == tuple(shape), (name, arr.shape, shape)
        parts.append(arr.reshape(-1))
    return np.concatenate(parts)


# ---------------------------------------------------------------------------
# Named workloads (shapes of the paper's LM1B / OpenWebText runs)
# ---------------------------------------------------------------------------
WORKLOADS = {
    # 2-layer toy, fp32, uniform prompts
    "toy": dict(cfg=ModelConfig(2, 128, 4, 512, 1024, 128, DTYPE_FP32),
                B=4, N=16, k=4, L=64, prompts="uniform"),
    # GPT-2-small-shaped LM1B stand-in
    "lm1b": dict(cfg=ModelConfig(12, 768, 12, 3072, 30522, 128, DTYPE_BF16),
                 B=64, N=16, k=4, L=112, prompts="zipf"),
    # GPT-2-small-shaped OpenWebText stand-in
    "owt": dict(cfg=ModelConfig(12, 768, 12, 3072, 50257, 1024, DTYPE_BF16),
                B=32, N=128, k=4, L=896, prompts="zipf"),
    # 24-layer backbone
    "large": dict(cfg=ModelConfig(24, 1024, 16, 4096, 50257, 1024, DTYPE_BF16),
                  B=256, N=256, k=4, L=768, prompts="zipf"),
}


def make_prompts(kind: str, seed: int, B: int, N: int, V: int) -> np.ndarray:
    if kind == "uniform":
        return prompts_uniform(seed, B, N, V)
    if kind == "zipf":
        return prompts_zipf(seed, B, N, V)
    raise ValueError(kind)


def describe(cfg: ModelConfig) -> str:
    return json.dumps(dataclasses.asdict(cfg))


# ---------------------------------------------------------------------------
# Attention inputs of the training masks
# ---------------------------------------------------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16 (ties to even), as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def attention_inputs(seed: int, b: int, h: int, rows: int, keys: int, dh: int,
                     std: float = 1.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Q [rows][dh], K [keys][dh], V [keys][dh] of sequence b, head h:
    N(0, std^2) draws (PCG64 seeded with (seed, 3, b, h)) rounded to bfloat16."""
    g = np.random.default_rng([seed, STREAM_NOISE + 1, b, h])
    q = g.standard_normal((rows, dh), dtype=np.float32) * np.float32(std)
    k = g.standard_normal((keys, dh), dtype=np.float32) * np.float32(std)
    v = g.standard_normal((keys, dh), dtype=np.float32)
    return round_bf16(q), round_bf16(k), round_bf16(v)


def attention_batch(seed: int, B: int, H: int, rows: int, keys: int, dh: int,
                    std: float = 1.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """attention_inputs stacked to [B][H][rows or keys][dh]."""
    q = np.empty((B, H, rows, dh), np.float32)
    k = np.empty((B, H, keys, dh), np.float32)
    v = np.empty((B, H, keys, dh), np.float32)
    for b in range(B):
        for h in range(H):
            q[b, h], k[b, h], v[b, h] = attention_inputs(seed, b, h, rows, keys, dh, std)
    return q, k, v
