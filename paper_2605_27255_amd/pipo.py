"""ctypes binding of ``libpipo.so`` (argument marshalling only).

Every step of the PIPO path runs in the HIP library; this module only passes
device pointers of torch CUDA tensors and the current HIP stream through the
C ABI declared in ``include/pipo.h``.  It raises if the library is missing:
there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libpipo.so")

PIPO_OK, PIPO_EINVAL, PIPO_ENOMEM, PIPO_EHIP, PIPO_ECAPACITY, PIPO_ESTATE = 0, -1, -2, -3, -4, -5
EXPORTED = ("pipo_init_weights", "pipo_prefill", "pipo_prefill_ragged", "pipo_decode_step", "pipo_decode_step_noalloc",
            "pipo_regular_prefill", "pipo_regular_prefill_ragged", "pipo_regular_step", "pipo_free",
            "pipo_last_error", "pipo_read_weight", "pipo_profile_enable", "pipo_profile_read",
            "pipo_opd_teacher_rows", "pipo_opd_targets", "pipo_opd_targets_bf16",
            "pipo_calibrate_stream", "pipo_calibrate_mfma")
#: kernel classes of the profiling counters (PIPO_K_* in include/pipo.h)
KERNEL_CLASSES = ("gemv_layer", "gemv_lmhead", "gemv_small", "attn_decode", "sample", "gate",
                  "prefill_gemm", "prefill_attn", "prefill_misc")


class PipoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"pipo error {code}: {msg}")
        self.code = code


class PipoConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("pad_id", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_latent", ctypes.c_int32),
                ("prefill_chunk", ctypes.c_int32), ("gain_mode", ctypes.c_int32), ("heads", ctypes.c_int32)]


class PipoSampling(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("temperature", ctypes.c_float), ("top_p", ctypes.c_float),
                ("seeds", ctypes.POINTER(ctypes.c_uint64)), ("top_k", ctypes.c_int32),
                ("rep_penalty", ctypes.c_float)]


class PipoPair(ctypes.Structure):
    _fields_ = [("tok_b", ctypes.c_int32), ("tok_d", ctypes.c_int32), ("conf", ctypes.c_float),
                ("accept", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built library (raises FileNotFoundError if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is missing: build it with paper_2605_27255_amd/build.py")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.pipo_init_weights.argtypes = [ctypes.POINTER(PipoConfig), ctypes.c_uint64, vp, ctypes.POINTER(vp)]
    lib.pipo_prefill.argtypes = [vp, i32, vp, i32, ctypes.POINTER(PipoSampling), vp, vp, vp, vp]
    lib.pipo_decode_step.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.pipo_decode_step_noalloc.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.pipo_regular_prefill.argtypes = [vp, i32, vp, i32, ctypes.POINTER(PipoSampling), vp, vp, vp]
    lib.pipo_prefill_ragged.argtypes = [vp, i32, vp, i32, ctypes.POINTER(i32), ctypes.POINTER(PipoSampling),
                                        vp, vp, vp, vp]
    lib.pipo_regular_prefill_ragged.argtypes = [vp, i32, vp, i32, ctypes.POINTER(i32), ctypes.POINTER(PipoSampling),
                                                vp, vp, vp]
    lib.pipo_regular_step.argtypes = [vp, vp, vp, vp, vp]
    lib.pipo_free.argtypes = [vp]
    lib.pipo_last_error.argtypes = [vp]
    lib.pipo_last_error.restype = ctypes.c_char_p
    lib.pipo_read_weight.argtypes = [vp, ctypes.c_char_p, i64, i64, vp]
    lib.pipo_profile_enable.argtypes = [vp, ctypes.c_int]
    lib.pipo_profile_read.argtypes = [vp, ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]
    lib.pipo_opd_teacher_rows.argtypes = [vp, i32, i32, vp, vp]
    lib.pipo_opd_targets.argtypes = [i32, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    lib.pipo_opd_targets_bf16.argtypes = [i32, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    lib.pipo_calibrate_stream.argtypes = [vp, i64, i64, i32, ctypes.POINTER(ctypes.c_double), vp]
    lib.pipo_calibrate_mfma.argtypes = [vp, i32, i32, i32, ctypes.POINTER(ctypes.c_double), vp]
    for fn in ("pipo_init_weights", "pipo_prefill", "pipo_prefill_ragged", "pipo_decode_step",
               "pipo_decode_step_noalloc", "pipo_regular_prefill",
               "pipo_regular_prefill_ragged", "pipo_regular_step", "pipo_free", "pipo_read_weight",
               "pipo_profile_enable", "pipo_profile_read", "pipo_opd_teacher_rows", "pipo_opd_targets",
               "pipo_opd_targets_bf16", "pipo_calibrate_stream", "pipo_calibrate_mfma"):
        getattr(lib, fn).restype = ctypes.c_int
    _lib = lib
    return lib


def make_config(model, max_batch: int, max_latent: int, prefill_chunk: int = 4096) -> PipoConfig:
    """A PipoConfig from any object with the model-shape attributes."""
    return PipoConfig(model.n_layers, model.hidden, model.n_q_heads, model.n_kv_heads, model.head_dim,
                      model.ffn, model.vocab, float(model.rope_base), float(model.rms_eps), -1,
                      max_batch, max_latent, prefill_chunk, int(getattr(model, "gain_mode", 0)),
                      int(getattr(model, "heads", 0)))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class PipoModel:
    """One PIPO context on the current CUDA (HIP) device."""

    def __init__(self, model, seed: int = 0, max_batch: int = 1, max_latent: int = 4096,
                 prefill_chunk: int = 4096):
        import torch
        self.torch = torch
        self.lib = load_library()
        self.model = model
        self.cfg = make_config(model, max_batch, max_latent, prefill_chunk)
        self.ctx = ctypes.c_void_p()
        rc = self.lib.pipo_init_weights(ctypes.byref(self.cfg), ctypes.c_uint64(seed), self._stream(),
                                        ctypes.byref(self.ctx))
        if rc != PIPO_OK:
            raise PipoError(rc, self.lib.pipo_last_error(None).decode())
        self.batch = 0

    def _stream(self):
        return ctypes.c_void_p(self.torch.cuda.current_stream().cuda_stream)

    def _check(self, rc):
        if rc != PIPO_OK:
            raise PipoError(rc, self.lib.pipo_last_error(self.ctx).decode())

    def _outputs(self, B, logits):
        t = self.torch
        out = t.empty((B, 4), dtype=t.int32, device="cuda")
        lb = t.empty((B, self.model.vocab), dtype=t.float32, device="cuda") if logits else None
        ld = t.empty((B, self.model.vocab), dtype=t.float32, device="cuda") if logits else None
        return out, lb, ld

    @staticmethod
    def _sampling(tau, temperature, top_p, seeds, top_k=0, rep_penalty=1.0):
        seed_arr = None
        if seeds is not None:
            seed_arr = (ctypes.c_uint64 * len(seeds))(*[int(s) for s in seeds])
        smp = PipoSampling(tau, temperature, top_p,
                           ctypes.cast(seed_arr, ctypes.POINTER(ctypes.c_uint64)) if seed_arr else None,
                           int(top_k), float(rep_penalty))
        return smp, seed_arr

    def _tokens(self, tokens):
        t = self.torch
        assert tokens.dtype == t.int32 and tokens.is_cuda and tokens.dim() == 2 and tokens.is_contiguous()
        return tokens.shape

    @staticmethod
    def _lens(lens, B):
        arr = (ctypes.c_int32 * B)(*[int(v) for v in lens])
        return arr

    def prefill(self, tokens, tau: float, temperature: float = 0.0, top_p: float = 1.0, seeds=None,
                logits: bool = False, top_k: int = 0, rep_penalty: float = 1.0, lens=None):
        """tokens: int32 CUDA tensor [B, n]; lens: optional per-sequence prompt
        lengths (a ragged batch, each the first lens[i] tokens of row i).
        Returns (pairs [B,4] int32, logits_b, logits_d)."""
        B, n = self._tokens(tokens)
        smp, _keep = self._sampling(tau, temperature, top_p, seeds, top_k, rep_penalty)
        out, lb, ld = self._outputs(B, logits)
        if lens is None:
            self._check(self.lib.pipo_prefill(self.ctx, B, _ptr(tokens), n, ctypes.byref(smp), _ptr(out),
                                              _ptr(lb), _ptr(ld), self._stream()))
        else:
            self._check(self.lib.pipo_prefill_ragged(self.ctx, B, _ptr(tokens), n, self._lens(lens, B),
                                                     ctypes.byref(smp), _ptr(out), _ptr(lb), _ptr(ld),
                                                     self._stream()))
        self.batch = B
        self._keep = tokens
        return out, lb, ld

    def decode_step(self, in_pairs=None, logits: bool = False):
        """One pair step; in_pairs: optional int32 CUDA tensor [B, 2] (teacher forcing)."""
        out, lb, ld = self._outputs(self.batch, logits)
        self._check(self.lib.pipo_decode_step(self.ctx, _ptr(in_pairs), _ptr(out), _ptr(lb), _ptr(ld),
                                              self._stream()))
        return out, lb, ld

    def decode_step_noalloc(self, out, in_pairs=None, logits_b=None, logits_d=None):
        """pipo_decode_step_noalloc into caller-provided tensors: the library
        allocates nothing and builds no graph (scratch in its static array)."""
        self._check(self.lib.pipo_decode_step_noalloc(self.ctx, _ptr(in_pairs), _ptr(out), _ptr(logits_b),
                                                      _ptr(logits_d), self._stream()))

    def decode_into(self, out, in_pairs=None, logits_b=None, logits_d=None):
        """decode_step writing into caller-provided tensors (no allocation)."""
        self._check(self.lib.pipo_decode_step(self.ctx, _ptr(in_pairs), _ptr(out), _ptr(logits_b),
                                              _ptr(logits_d), self._stream()))

    def regular_prefill(self, tokens, temperature: float = 0.0, top_p: float = 1.0, seeds=None,
                        logits: bool = False, top_k: int = 0, rep_penalty: float = 1.0, lens=None):
        """Regular decoding's prefill over the n prompt tokens (lens: ragged
        batch, as in prefill).  Returns (tok [B] int32, logits)."""
        t = self.torch
        B, n = self._tokens(tokens)
        smp, _keep = self._sampling(0.0, temperature, top_p, seeds, top_k, rep_penalty)
        tok = t.empty(B, dtype=t.int32, device="cuda")
        lg = t.empty((B, self.model.vocab), dtype=t.float32, device="cuda") if logits else None
        if lens is None:
            self._check(self.lib.pipo_regular_prefill(self.ctx, B, _ptr(tokens), n, ctypes.byref(smp), _ptr(tok),
                                                      _ptr(lg), self._stream()))
        else:
            self._check(self.lib.pipo_regular_prefill_ragged(self.ctx, B, _ptr(tokens), n, self._lens(lens, B),
                                                             ctypes.byref(smp), _ptr(tok), _ptr(lg),
                                                             self._stream()))
        self.batch = B
        self._keep = tokens
        return tok, lg

    def regular_step(self, in_tok=None, logits: bool = False):
        """One regular decoding step; in_tok: optional int32 CUDA tensor [B] (teacher forcing)."""
        t = self.torch
        tok = t.empty(self.batch, dtype=t.int32, device="cuda")
        lg = t.empty((self.batch, self.model.vocab), dtype=t.float32, device="cuda") if logits else None
        self._check(self.lib.pipo_regular_step(self.ctx, _ptr(in_tok), _ptr(tok), _ptr(lg), self._stream()))
        return tok, lg

    def regular_into(self, tok, in_tok=None, logits=None):
        """regular_step writing into caller-provided tensors (no allocation)."""
        self._check(self.lib.pipo_regular_step(self.ctx, _ptr(in_tok), _ptr(tok), _ptr(logits), self._stream()))

    def read_weight(self, name: str, start: int, count: int):
        import numpy as np
        buf = np.empty(count, dtype=np.uint16)
        self._check(self.lib.pipo_read_weight(self.ctx, name.encode(), start, count,
                                              buf.ctypes.data_as(ctypes.c_void_p)))
        return buf

    def profile(self, on: bool):
        """Per-kernel-class HIP-event timing (eager launches while on)."""
        self._check(self.lib.pipo_profile_enable(self.ctx, 1 if on else 0))

    def profile_read(self) -> dict:
        """{class: (total_ms, launches)} since profiling was turned on."""
        res = {}
        for k, name in enumerate(KERNEL_CLASSES):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            self._check(self.lib.pipo_profile_read(self.ctx, k, ctypes.byref(ms), ctypes.byref(n)))
            res[name] = (ms.value, n.value)
        return res

    def close(self):
        if self.ctx:
            self.lib.pipo_free(self.ctx)
            self.ctx = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def unpack_pairs(out):
    """[B,4] int32 tensor -> (tok_b, tok_d, conf, accept) numpy arrays."""
    import numpy as np
    a = out.cpu().numpy()
    return a[:, 0].copy(), a[:, 1].copy(), a[:, 2].copy().view(np.float32), a[:, 3].copy()


def _opd_check(lib, rc):
    if rc != PIPO_OK:
        raise PipoError(rc, "pipo_opd_*: invalid arguments or launch failure")


def opd_teacher_rows(tokens, pad_id: int):
    """PAD-compaction teacher rows of a trajectory (int32 CUDA tensor [T])."""
    import torch
    lib = load_library()
    assert tokens.dtype == torch.int32 and tokens.is_cuda and tokens.dim() == 1 and tokens.is_contiguous()
    rows = torch.empty_like(tokens)
    _opd_check(lib, lib.pipo_opd_teacher_rows(_ptr(tokens), tokens.numel(), int(pad_id), _ptr(rows),
                                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)))
    return rows


def opd_targets(logits_s, logits_t, labels, rows=None, sums: bool = True):
    """Sampled reverse-KL terms and confidence targets of the OPD loss.
    logits_s: float32 or bfloat16 CUDA [T, V]; logits_t: the same dtype, [Tt, V]; labels:
    int32 CUDA [T] (negative: not scored); rows: int32 CUDA [T] teacher rows
    (None: row t).  Returns (kl [T], alpha [T], sums [4] float64 or None)."""
    import torch
    lib = load_library()
    for x in (logits_s, logits_t):
        assert x.dtype in (torch.float32, torch.bfloat16) and x.is_cuda and x.dim() == 2 and x.is_contiguous()
    assert logits_s.dtype == logits_t.dtype
    fn = lib.pipo_opd_targets if logits_s.dtype == torch.float32 else lib.pipo_opd_targets_bf16
    T, V = logits_s.shape
    kl = torch.empty(T, dtype=torch.float32, device="cuda")
    alpha = torch.empty(T, dtype=torch.float32, device="cuda")
    sm = torch.empty(4, dtype=torch.float64, device="cuda") if sums else None
    _opd_check(lib, fn(T, V, _ptr(logits_s), _ptr(logits_t), logits_t.shape[0], _ptr(rows),
                                         _ptr(labels), _ptr(kl), _ptr(alpha), _ptr(sm),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)))
    return kl, alpha, sm


def calibrate_stream(buf, nbytes: int, reps: int = 20) -> float:
    """Mean microseconds per launch of the weight-stream pattern reading
    ``nbytes`` of the CUDA tensor ``buf``, a different window each launch
    (measurement only)."""
    import torch
    lib = load_library()
    total = buf.numel() * buf.element_size()
    assert buf.is_cuda and buf.is_contiguous() and nbytes <= total
    us = ctypes.c_double()
    rc = lib.pipo_calibrate_stream(_ptr(buf), int(total), int(nbytes), int(reps), ctypes.byref(us),
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    if rc != PIPO_OK:
        raise PipoError(rc, "pipo_calibrate_stream failed")
    return us.value


def calibrate_mfma(operands, waves_per_simd: int, iters: int = 4096, reps: int = 5) -> float:
    """bf16 16x16x32 MFMA issue rate in TFLOP/s with register operands taken
    from the CUDA tensor ``operands`` (at least 8 KB; measurement only)."""
    import torch
    lib = load_library()
    assert operands.is_cuda and operands.is_contiguous() and operands.numel() * operands.element_size() >= 8192
    tf = ctypes.c_double()
    rc = lib.pipo_calibrate_mfma(_ptr(operands), int(waves_per_simd), int(iters), int(reps), ctypes.byref(tf),
                                 ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    if rc != PIPO_OK:
        raise PipoError(rc, "pipo_calibrate_mfma failed")
    return tf.value
