"""Counter-based synthetic inputs ("R-spec").

Every random quantity of the benchmark workloads is a pure function of a seed
and an element index, so the host (this module) and the device (the HIP
library's initialiser) can produce bit-identical values independently.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), used as a stateless hash ``sm(x)``: the value
the published generator returns when its state is ``x`` before the increment.

* ``key(seed, tid) = sm(seed ^ sm(tid))``.
* Weight element ``i`` of tensor ``tid``: ``r1 = sm(key + 2i)``,
  ``r2 = sm(key + 2i + 1)``; the four 24-bit fields ``r>>40`` and
  ``(r>>16) & 0xFFFFFF`` of both words are summed to ``S``; then
  ``w = float32(int32(S - 2**25)) * C`` with ``C = float32(0.02*sqrt(3)/2**24)``
  (both float32 operations round to nearest even).  ``S`` is an Irwin-Hall(4)
  sum of 24-bit uniforms, so ``w`` has mean 0, standard deviation 0.02,
  excess kurtosis -0.3 and support within +-2*0.02*sqrt(3) = +-0.0693: a
  stand-in for the N(0, 0.02^2) initialisation.
* Prompt token ``j`` of sequence ``b``:
  ``((sm(key(1, 2**32 + b) + j) >> 32) * (V - 1)) >> 32``, uniform in
  ``[0, V-2]``, so the reserved PAD id ``V-1`` never occurs in a prompt.
* Sampler draw for sequence seed ``sd``, step ``s`` and slot ``k``
  (0 backbone token, 1 draft token):
  ``(sm(key(sd, 2**33) + 2s + k) >> 40) * 2**-24`` in ``[0, 1)``.
* bf16 storage: round-to-nearest-even of the float32 bit pattern.
"""
from __future__ import annotations

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_MIX1 = np.uint64(0xBF58476D1CE4E5B9)
_MIX2 = np.uint64(0x94D049BB133111EB)
_MASK64 = (1 << 64) - 1

#: float32 scale turning the centred Irwin-Hall(4) integer into sd 0.02.
WEIGHT_SCALE = np.float32(0.02 * np.sqrt(3.0) / 2.0 ** 24)
assert WEIGHT_SCALE.view(np.uint32) == 0x310DE3BD

#: Tensor ids of the model-level tensors.  Per-layer tensors use layer_tid().
TENSOR_IDS = {
    "embed": 0,      # E [V, H], also the (tied) LM head
    "w_comp": 1,     # W_c [H, 2H]
    "b_comp": 2,     # b_c [H]
    "w_fc": 3,       # MTP projection [H, 2H]
    "w_conf": 4,     # confidence head [2H]
    "g_final": 5,    # final RMSNorm gain [H]
    "g_mtp_h": 6,    # MTP RMSNorm gain on h_b [H]
    "g_mtp_e": 7,    # MTP RMSNorm gain on the token embedding [H]
    "g_mtp_o": 8,    # MTP output RMSNorm gain [H]
    "g_conf": 9,     # confidence RMSNorm gain [2H]
    "comp_w1": 10,   # MLP compressor W1 [H, 2H]
    "comp_w2": 11,   # MLP compressor W2 [H, H]
    "conf_w1": 12,   # confidence MLP W1 [H, 2H]
    "conf_w2": 13,   # confidence MLP W2 [H]
}
_LAYER_SLOTS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "wgate": 4, "wup": 5,
                "wdown": 6, "g_attn": 7, "g_ffn": 8}


def layer_tid(layer: int, name: str) -> int:
    return 100 + 10 * layer + _LAYER_SLOTS[name]


def mtp_tid(name: str) -> int:
    """Tensor id of the MTP head's decoder layer (the same slots as a layer)."""
    return 90 + _LAYER_SLOTS[name]


def tensor_id(name: str) -> int:
    """Tensor id of a tensor named as in ``model_tensor_shapes``."""
    if name.startswith("mtp."):
        return mtp_tid(name[4:])
    if "." in name:
        return layer_tid(int(name.split(".")[0][1:]), name.split(".")[1])
    return TENSOR_IDS[name]


def splitmix64(x):
    """Stateless SplitMix64 output for state(s) ``x`` (uint64 array or int)."""
    scalar = not isinstance(x, np.ndarray)
    z = np.asarray(x, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z = z + _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _MIX1
        z = (z ^ (z >> np.uint64(27))) * _MIX2
        z = z ^ (z >> np.uint64(31))
    return int(z) if scalar else z


def key(seed: int, tid: int) -> int:
    return splitmix64((int(seed) & _MASK64) ^ splitmix64(int(tid) & _MASK64))


def _fields24(r):
    return (r >> np.uint64(40)) + ((r >> np.uint64(16)) & np.uint64(0xFFFFFF))


def _fast_lib():
    """The OpenMP build of the same recipe (synth/rspec_fast.c), if compiled."""
    global _FAST
    if _FAST is None:
        import ctypes
        import os
        so = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_rspec_fast.so")
        _FAST = False
        if os.path.exists(so):
            lib = ctypes.CDLL(so)
            lib.rspec_fill.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                       ctypes.c_int64, ctypes.c_void_p, ctypes.c_int]
            lib.rspec_fill64.argtypes = lib.rspec_fill.argtypes
            _FAST = lib
    return _FAST


_FAST = None


def weight_values(seed: int, tid: int, start: int, count: int, fast: bool = True,
                  bf16: bool = False) -> np.ndarray:
    """float32 values of elements ``[start, start+count)`` of tensor ``tid``
    (rounded to bf16 when ``bf16``)."""
    lib = _fast_lib() if fast else False
    if lib:
        out = np.empty(count, dtype=np.float32)
        lib.rspec_fill(seed & _MASK64, tid & _MASK64, start, count, out.ctypes.data, 1 if bf16 else 0)
        return out
    if bf16:
        return bf16_round(weight_values(seed, tid, start, count, fast=False))
    k = np.uint64(key(seed, tid))
    idx = np.arange(start, start + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        base = k + np.uint64(2) * idx
        s = _fields24(splitmix64(base)) + _fields24(splitmix64(base + np.uint64(1)))
    centred = (s.astype(np.int64) - (1 << 25)).astype(np.int32)
    return centred.astype(np.float32) * WEIGHT_SCALE


def weight_tensor(seed: int, tid: int, shape, chunk: int = 1 << 26, bf16: bool = False,
                  dtype=np.float32) -> np.ndarray:
    """A whole tensor in logical row-major ``[out][in]`` order (float32 values,
    stored as ``dtype``)."""
    n = int(np.prod(shape))
    lib = _fast_lib()
    if lib and dtype == np.float64:
        out = np.empty(n, dtype=np.float64)
        lib.rspec_fill64(seed & _MASK64, tid & _MASK64, 0, n, out.ctypes.data, 1 if bf16 else 0)
        return out.reshape(shape)
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, chunk):
        c = min(chunk, n - s)
        out[s:s + c] = weight_values(seed, tid, s, c, bf16=bf16)
    return out.reshape(shape).astype(dtype, copy=False)


def gain_values(seed: int, tid: int, n: int, gain_mode: int) -> np.ndarray:
    """RMSNorm gains: exactly 1 (mode 0), or 1 + 10*w (mode 1, sd 0.2)."""
    if gain_mode == 0:
        return np.ones(n, dtype=np.float32)
    return np.float32(1.0) + np.float32(10.0) * weight_values(seed, tid, 0, n)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bf16 patterns of float32 ``x``, round to nearest even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return rounded.astype(np.uint16)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 ``x`` rounded to the nearest bf16 value (returned as float32)."""
    return (bf16_bits(x).astype(np.uint32) << np.uint32(16)).view(np.float32)


def prompt_tokens(batch: int, n: int, vocab: int, seed: int = 1) -> np.ndarray:
    """int32 ``[batch, n]`` prompt ids, uniform in ``[0, vocab-2]``."""
    out = np.empty((batch, n), dtype=np.int32)
    j = np.arange(n, dtype=np.uint64)
    for b in range(batch):
        k = np.uint64(key(seed, (1 << 32) + b))
        with np.errstate(over="ignore"):
            r = splitmix64(k + j) >> np.uint64(32)
            out[b] = ((r * np.uint64(vocab - 1)) >> np.uint64(32)).astype(np.int32)
    return out


def uniform_draw(seq_seed: int, step: int, slot: int) -> float:
    """The sampler's uniform in [0, 1) for (sequence seed, step, slot)."""
    k = key(seq_seed, 1 << 33)
    r = splitmix64((k + 2 * step + slot) & _MASK64)
    return (r >> 40) * 2.0 ** -24
