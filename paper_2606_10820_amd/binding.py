"""ctypes binding of libkforcing.so (include/kforcing.h).

`lib()` returns the loaded library with typed signatures for every kf_*
entry point (same names as the C ABI).  `KForcing` wraps one context: it
allocates the state buffer with torch on a CUDA (HIP) device, passes device
pointers and the current stream, and turns error codes into KfError.  No
computation happens here.  If the shared library is missing the import of
`lib()` fails loudly: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libkforcing.so")

KF_OK, KF_EINVAL, KF_ESTATE, KF_ECTX, KF_ENOMEM, KF_EHIP = 0, -1, -2, -3, -4, -5
KF_FP32, KF_BF16 = 0, 1
KF_FLAG_DEBUG_LOGITS = 1
KF_FLAG_TEMPERATURE = 2
KF_FLAG_TEACHER = 4
KF_FLAG_ROLLOUT = 8
KF_FLAG_RMS_ROPE = 16
KF_FLAG_SERVING = 32
KF_PAGE = 128  # positions per KV page
KF_MASK_SINGLE, KF_MASK_DOUBLE = 0, 1
KF_KC_NAMES = ["embed", "noise", "norm", "qkv", "attn", "oproj", "mlp_up", "mlp_down", "head",
               "select"]
KF_TIMING_ALL = (1 << len(KF_KC_NAMES)) - 1

_lib = None


class KfConfig(ctypes.Structure):
    _fields_ = [
        ("n_layer", ctypes.c_int), ("d_model", ctypes.c_int), ("n_head", ctypes.c_int),
        ("d_mlp", ctypes.c_int), ("vocab", ctypes.c_int), ("n_ctx", ctypes.c_int),
        ("dtype", ctypes.c_int), ("max_batch", ctypes.c_int), ("max_k", ctypes.c_int),
        ("max_prompt", ctypes.c_int), ("flags", ctypes.c_uint), ("kv_pages", ctypes.c_int),
    ]


class KfError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"kforcing error {code}: {msg}")
        self.code = code


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libkforcing.so and declare every entry point of include/kforcing.h."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2606_10820_amd.build` (there is no CPU fallback)")
    L = ctypes.CDLL(_LIB_PATH)
    P, I, U64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_uint64, ctypes.c_size_t
    CP = ctypes.POINTER(KfConfig)
    IP = ctypes.POINTER(ctypes.c_int)
    sigs = {
        "kf_create": (I, [CP, P, ctypes.POINTER(P)]),
        "kf_state_bytes": (SZ, [CP]),
        "kf_bind_state": (I, [P, P, SZ]),
        "kf_load_weights": (I, [P, P, SZ, I]),
        "kf_prefill": (I, [P, I, I, P, I, P, P]),
        "kf_decode_block": (I, [P, I, I, P, P]),
        "kf_decode_block_noalloc": (I, [P, I, I, P, P]),
        "kf_generate": (I, [P, I, I, P, I, I, U64, P]),
        "kf_prefill_ar": (I, [P, I, I, P, P, P]),
        "kf_decode_ar": (I, [P, I, P, P]),
        "kf_generate_ar": (I, [P, I, I, P, I, U64, P]),
        "kf_debug_logits": (I, [P, P, SZ]),
        "kf_fill_noise": (I, [P, U64, I, I, I, P]),
        "kf_set_temperature": (I, [P, P, I]),
        "kf_teacher_targets": (I, [P, I, I, P, P, P, P]),
        "kf_selfforcing_targets": (I, [P, I, I, I, P, P, P, P, P]),
        "kf_get_state": (I, [P, IP, IP, IP]),
        "kf_device_errors": (I, [P, IP]),
        "kf_set_graphs": (I, [P, I]),
        "kf_set_timing": (I, [P, I]),
        "kf_kernel_time": (I, [P, I, ctypes.POINTER(ctypes.c_double), IP]),
        "kf_destroy": (None, [P]),
        "kf_last_error": (ctypes.c_char_p, [P]),
        "kf_strerror": (ctypes.c_char_p, [I]),
        "kf_training_attention": (I, [P, I, I, I, I, I, I, P, P, P, P, ctypes.c_float]),
        "kf_serve_admit": (I, [P, I, P, I, P, I, P, P]),
        "kf_serve_step": (I, [P, I, P, I, P, P]),
        "kf_serve_release": (I, [P, I, P]),
        "kf_serve_state": (I, [P, I, IP, IP, IP]),
        "kf_serve_pages": (I, [P, IP, IP]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def make_config(n_layer, d_model, n_head, d_mlp, vocab, n_ctx, dtype, max_batch, max_k,
                max_prompt, flags=0, kv_pages=0) -> KfConfig:
    return KfConfig(n_layer, d_model, n_head, d_mlp, vocab, n_ctx, dtype, max_batch, max_k,
                    max_prompt, flags, kv_pages)


class KForcing:
    """One library context with its device state buffer (allocated by torch)."""

    def __init__(self, cfg: KfConfig, device: str = "cuda:0", stream=None):
        import torch
        self.torch = torch
        self.L = lib()
        self.cfg = cfg
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        h = ctypes.c_void_p()
        rc = self.L.kf_create(ctypes.byref(cfg), ctypes.c_void_p(self.stream.cuda_stream),
                              ctypes.byref(h))
        if rc != KF_OK:
            raise KfError(rc, "kf_create rejected the configuration")
        self.h = h
        nbytes = self.L.kf_state_bytes(ctypes.byref(cfg))
        self.state = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.state.data_ptr()
        aligned = (base + 255) // 256 * 256
        self._check(self.L.kf_bind_state(self.h, ctypes.c_void_p(aligned), nbytes))

    # -- plumbing -------------------------------------------------------
    def _check(self, rc: int):
        if rc != KF_OK:
            raise KfError(rc, self.L.kf_last_error(self.h).decode())

    @staticmethod
    def _p(t) -> ctypes.c_void_p:
        return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)

    def _i32(self, x):
        return self.torch.as_tensor(x, dtype=self.torch.int32, device=self.device).contiguous()

    def _f32(self, x):
        return self.torch.as_tensor(x, dtype=self.torch.float32, device=self.device).contiguous()

    def close(self):
        if getattr(self, "h", None):
            self.L.kf_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- entry points ----------------------------------------------------
    def load_weights(self, blob, on_device: bool = True):
        """blob: numpy float32 array (header + tensors), copied as given."""
        import numpy as np
        arr = np.ascontiguousarray(blob, dtype=np.float32)
        if on_device:
            t = self.torch.from_numpy(arr).to(self.device)
            self._check(self.L.kf_load_weights(self.h, self._p(t), arr.nbytes, 1))
            self.torch.cuda.synchronize(self.device)
        else:
            self._check(self.L.kf_load_weights(self.h, ctypes.c_void_p(arr.ctypes.data),
                                               arr.nbytes, 0))

    def prefill(self, prompt, k: int, noise, out=None):
        prompt = self._i32(prompt)
        noise = self._f32(noise)
        B, N = prompt.shape
        if out is None:
            out = self.torch.empty((B, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_prefill(self.h, B, N, self._p(prompt), k, self._p(noise),
                                      self._p(out)))
        return out

    def decode_block(self, noise, out=None):
        noise = self._f32(noise)
        B, k = noise.shape
        if out is None:
            out = self.torch.empty((B, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_decode_block(self.h, B, k, self._p(noise), self._p(out)))
        return out

    def decode_block_noalloc(self, noise, out=None):
        """kf_decode_block with the step's partial results in the library's
        device scratch (no allocation inside the call)."""
        noise = self._f32(noise)
        B, k = noise.shape
        if out is None:
            out = self.torch.empty((B, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_decode_block_noalloc(self.h, B, k, self._p(noise), self._p(out)))
        return out

    def generate(self, prompt, L: int, k: int, seed: int, out=None):
        prompt = self._i32(prompt)
        B, N = prompt.shape
        if out is None:
            out = self.torch.empty((B, L), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_generate(self.h, B, N, self._p(prompt), L, k, seed, self._p(out)))
        return out

    def prefill_ar(self, prompt, u, out=None):
        prompt = self._i32(prompt)
        u = self._f32(u)
        B, N = prompt.shape
        if out is None:
            out = self.torch.empty((B,), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_prefill_ar(self.h, B, N, self._p(prompt), self._p(u), self._p(out)))
        return out

    def decode_ar(self, u, out=None):
        u = self._f32(u)
        B = u.shape[0]
        if out is None:
            out = self.torch.empty((B,), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_decode_ar(self.h, B, self._p(u), self._p(out)))
        return out

    def generate_ar(self, prompt, L: int, seed: int, out=None):
        prompt = self._i32(prompt)
        B, N = prompt.shape
        if out is None:
            out = self.torch.empty((B, L), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_generate_ar(self.h, B, N, self._p(prompt), L, seed, self._p(out)))
        return out

    def debug_logits(self, rows: int):
        out = self.torch.empty((rows, self.cfg.vocab), dtype=self.torch.float32,
                               device=self.device)
        self._check(self.L.kf_debug_logits(self.h, self._p(out), out.numel()))
        return out

    def set_temperature(self, tau):
        """Per-sequence temperatures tau [B] (temperature-conditioned models)."""
        t = self._f32(tau).reshape(-1)
        self._check(self.L.kf_set_temperature(self.h, self._p(t), int(t.numel())))
        self.torch.cuda.synchronize(self.device)  # t is read during the call's kernels

    def teacher_targets(self, tokens, tau, u, out=None):
        """Stage-1 teacher targets: tokens [B][N] int32, tau [B], u [B][N]
        (device tensors or array-likes); returns targets [B][N] int32."""
        tk = self._i32(tokens)
        B, N = tk.shape
        t = self._f32(tau).reshape(-1)
        uu = self._f32(u).reshape(B, N)
        if out is None:
            out = self.torch.empty((B, N), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_teacher_targets(self.h, B, N, self._p(tk), self._p(t), self._p(uu),
                                              self._p(out)))
        self.torch.cuda.synchronize(self.device)  # the inputs may be temporaries
        return out

    def selfforcing_targets(self, tokens, k: int, z1, z2):
        """Stage-2 teacher rollout: tokens [B][N], z1/z2 [B][N][k]; returns (x1, x2),
        each int32 [B][N][k]."""
        tk = self._i32(tokens)
        B, N = tk.shape
        a = self._f32(z1).reshape(B, N, k)
        b = self._f32(z2).reshape(B, N, k)
        x1 = self.torch.empty((B, N, k), dtype=self.torch.int32, device=self.device)
        x2 = self.torch.empty((B, N, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_selfforcing_targets(self.h, B, N, k, self._p(tk), self._p(a),
                                                  self._p(b), self._p(x1), self._p(x2)))
        self.torch.cuda.synchronize(self.device)  # the inputs may be temporaries
        return x1, x2

    # -- continuous batching (KF_FLAG_SERVING) ---------------------------
    @staticmethod
    def _slots(slots):
        import numpy as np
        arr = np.ascontiguousarray(slots, dtype=np.int32)
        return arr, ctypes.c_void_p(arr.ctypes.data)

    def serve_admit(self, slots, prompts, k: int, noise, out=None):
        """Start len(slots) sequences: prompts [n][N], noise [n][k] -> out [n][k]."""
        arr, sp = self._slots(slots)
        prompts = self._i32(prompts).reshape(len(arr), -1)
        noise = self._f32(noise)
        n, N = prompts.shape
        if out is None:
            out = self.torch.empty((n, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_serve_admit(self.h, n, sp, N, self._p(prompts), k, self._p(noise),
                                          self._p(out)))
        return out

    def serve_step(self, slots, noise, out=None):
        """One decode block for the listed slots: noise [n][k] -> out [n][k]."""
        arr, sp = self._slots(slots)
        noise = self._f32(noise)
        n, k = noise.shape
        if out is None:
            out = self.torch.empty((n, k), dtype=self.torch.int32, device=self.device)
        self._check(self.L.kf_serve_step(self.h, n, sp, k, self._p(noise), self._p(out)))
        return out

    def serve_release(self, slots):
        arr, sp = self._slots(slots)
        self._check(self.L.kf_serve_release(self.h, len(arr), sp))

    def serve_state(self, slot: int):
        C, p, g = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        self._check(self.L.kf_serve_state(self.h, slot, ctypes.byref(C), ctypes.byref(p),
                                          ctypes.byref(g)))
        return C.value, p.value, g.value

    def serve_pages(self):
        f, t = ctypes.c_int(), ctypes.c_int()
        self._check(self.L.kf_serve_pages(self.h, ctypes.byref(f), ctypes.byref(t)))
        return f.value, t.value

    def fill_noise(self, seed: int, B: int, p0: int, n: int):
        out = self.torch.empty((B, n), dtype=self.torch.float32, device=self.device)
        self._check(self.L.kf_fill_noise(self.h, seed, B, p0, n, self._p(out)))
        return out

    def get_state(self):
        C, p, B = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        self._check(self.L.kf_get_state(self.h, ctypes.byref(C), ctypes.byref(p), ctypes.byref(B)))
        return C.value, p.value, B.value

    def device_errors(self) -> int:
        f = ctypes.c_int()
        self._check(self.L.kf_device_errors(self.h, ctypes.byref(f)))
        return f.value

    def set_graphs(self, enable: bool):
        self._check(self.L.kf_set_graphs(self.h, int(enable)))

    def set_timing(self, class_mask: int = KF_TIMING_ALL):
        """Bracket launches of the selected kernel classes (bit mask) with HIP events."""
        self._check(self.L.kf_set_timing(self.h, int(class_mask)))

    def kernel_time(self, cls: int):
        ms, n = ctypes.c_double(), ctypes.c_int()
        self._check(self.L.kf_kernel_time(self.h, cls, ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value


def training_attention_shapes(mask: int, N: int, k: int):
    """(query rows, keys) of one sequence under a training mask."""
    if mask == KF_MASK_SINGLE:
        return N + N * k, N + N * k
    return 2 * N * k, N + 2 * N * k


def training_attention_entries(mask: int, N: int, k: int) -> int:
    """Visible (query, key) pairs of one sequence under a training mask: the
    algorithmic work (4 * d_head flops each) of kf_training_attention."""
    ctx = N * (N + 1) // 2                      # context rows, causal
    noise = k * N * (N + 1) // 2 + N * k * (k + 1) // 2   # staircase + in-group causal
    if mask == KF_MASK_SINGLE:
        return ctx + noise
    # Future-1 rows as the noise rows above; Future-2 rows add all k Future-1 keys
    return 2 * noise + N * k * k


def training_attention(mask: int, q, k_, v, N: int, k: int, scale: Optional[float] = None,
                       out=None, stream=None):
    """Attention of the training masks (kf_training_attention).

    q [B][H][rows][dh], k_/v [B][H][keys][dh]: contiguous bf16 device tensors.
    Returns out (allocated like q when None).  The call is asynchronous on
    `stream` (default: torch's current stream)."""
    import torch
    B, H, rows, dh = q.shape
    if (rows, k_.shape[2]) != training_attention_shapes(mask, N, k):
        raise ValueError("q/k rows do not match the mask's layout")
    for t in (q, k_, v):
        if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("q, k, v must be contiguous bf16 device tensors")
    if k_.shape != v.shape or k_.shape[:2] != (B, H) or k_.shape[3] != dh:
        raise ValueError("k and v must be [B][H][keys][dh] like q")
    if out is None:
        out = torch.empty_like(q)
    if scale is None:
        scale = dh ** -0.5
    s = stream if stream is not None else torch.cuda.current_stream(q.device)
    rc = lib().kf_training_attention(
        ctypes.c_void_p(s.cuda_stream), mask, B, H, N, k, dh, ctypes.c_void_p(q.data_ptr()),
        ctypes.c_void_p(k_.data_ptr()), ctypes.c_void_p(v.data_ptr()),
        ctypes.c_void_p(out.data_ptr()), float(scale))
    if rc != KF_OK:
        raise KfError(rc, lib().kf_strerror(rc).decode())
    return out
