"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This module is the only code both sides use.  It holds no arithmetic of the
decoder: it names the workloads (shapes, dtypes, LoRA settings, load orders),
draws every tensor from a counter-based generator (Philox4x32-10 with the
Box-Muller transform, in ``synth.c``) and stores the draws in the requested
type.  Random-init OPT-shaped models have no released values, so the recipe
follows the paper's model family (OPT decoders, LoRA on attention projections)
with the usual random-init scales:

* every weight matrix and bias ~ N(0, 0.02) (std), stored ``[out, in]``;
* LayerNorm gamma = 1 + N(0, 0.02), beta ~ N(0, 0.02);
* LoRA A ~ N(0, 1/r) (std), shape ``[r, d_in]``; B ~ N(0, 0.02), ``[d_out, r]``;
* prompt tokens uniform in [2, V), no BOS, no padding.

Streams are keyed by (config seed, stream id); see ``weight_stream``,
``lora_stream`` and ``TOKEN_STREAM``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

KIND_CODE = {"f32": 0, "f16": 1, "bf16": 2}


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b

            _b.build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.synth_normal.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                     ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_int, ctypes.c_void_p]
        lib.synth_normal.restype = None
        lib.synth_uniform_int.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
        lib.synth_uniform_int.restype = None
        lib.synth_const.argtypes = [ctypes.c_uint64, ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
        lib.synth_const.restype = None
        lib.synth_philox4x32.argtypes = [ctypes.POINTER(ctypes.c_uint32),
                                         ctypes.POINTER(ctypes.c_uint32), ctypes.c_int,
                                         ctypes.POINTER(ctypes.c_uint32)]
        lib.synth_philox4x32.restype = None
        lib.synth_f32_to_f16.argtypes = [ctypes.c_float]
        lib.synth_f32_to_f16.restype = ctypes.c_uint16
        lib.synth_f32_to_bf16.argtypes = [ctypes.c_float]
        lib.synth_f32_to_bf16.restype = ctypes.c_uint16
        _lib = lib
    return _lib


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------

TARGETS = ("q", "k", "v", "o")
LAYER_TENSORS = ("ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo",
                 "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")
GLOBAL_TENSORS = ("embed", "pos", "lnf_g", "lnf_b")


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: model shape, storage type, LoRA setup and prompt."""

    name: str
    seed: int
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int
    max_pos: int
    dtype: str  # GPU storage type: "bf16" or "f16"
    batch: int
    seq_len: int
    lora_targets: Tuple[str, ...] = ("q", "v")
    lora_rank: int = 16
    lora_alpha: float = 32.0
    n_adapters: int = 1
    # adapter index used by each sequence (-1 = base model only); None -> all 0
    adapter_of_seq: Optional[Tuple[int, ...]] = None
    # order in which the layers are streamed; None -> natural order
    layer_order: Optional[Tuple[int, ...]] = None
    # "f32": the oracle uses the float draws and the GPU their rounding to dtype;
    # "storage": the stored dtype values are the model on both sides
    oracle_weights: str = "storage"
    # LoRA B drawn as zeros (adapter that must leave the base model unchanged)
    lora_zero_b: bool = False
    ln_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def n_tokens(self) -> int:
        return self.batch * self.seq_len

    @property
    def lora_scale(self) -> float:
        return self.lora_alpha / self.lora_rank

    def adapters(self) -> Tuple[int, ...]:
        if self.adapter_of_seq is not None:
            return tuple(self.adapter_of_seq)
        return tuple(0 for _ in range(self.batch)) if self.n_adapters > 0 else tuple(
            -1 for _ in range(self.batch))

    def order(self) -> Tuple[int, ...]:
        if self.layer_order is not None:
            return tuple(self.layer_order)
        return tuple(range(self.n_layers))

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    # -- byte and FLOP counts (algorithmic, see the design notes) ------------
    def layer_params(self) -> int:
        d, f = self.d_model, self.d_ffn
        return 4 * d * d + 2 * d * f + f + 9 * d

    def global_params(self) -> int:
        return self.vocab * self.d_model + self.max_pos * self.d_model + 2 * self.d_model

    def storage_bytes(self) -> int:
        return 2 * (self.n_layers * self.layer_params() + self.global_params())

    def lora_bytes(self) -> int:
        return (2 * self.n_adapters * self.n_layers * len(self.lora_targets)
                * 2 * self.lora_rank * self.d_model)

    def prefill_flops(self) -> dict:
        """Algorithmic FLOPs of one prefill (multiply-add = 2)."""
        d, f, L, B, T = self.d_model, self.d_ffn, self.n_layers, self.batch, self.seq_len
        n = B * T
        used = [a for a in self.adapters() if a >= 0]
        n_lora_rows = sum(T for a in self.adapters() if a >= 0)
        gemm = 2 * n * (4 * d * d + 2 * d * f) * L
        attn = 2 * B * d * T * (T + 1) * L
        lora = 4 * n_lora_rows * self.lora_rank * d * len(self.lora_targets) * L if used else 0
        lm = 2 * B * d * self.vocab
        return {"gemm": gemm, "attn": attn, "lora": lora, "lm_head": lm,
                "total": gemm + attn + lora + lm}


WORKLOADS = {
    "tiny": Workload(name="tiny", seed=1, n_layers=2, d_model=256, n_heads=4, d_ffn=1024,
                     vocab=2048, max_pos=128, dtype="bf16", batch=1, seq_len=32,
                     lora_targets=("q", "v"), lora_rank=8, lora_alpha=16.0, n_adapters=1,
                     oracle_weights="f32"),
    "opt-1.3b": Workload(name="opt-1.3b", seed=2, n_layers=24, d_model=2048, n_heads=32,
                         d_ffn=8192, vocab=50272, max_pos=2048, dtype="f16", batch=1,
                         seq_len=512, lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0,
                         n_adapters=1),
    "opt-6.7b": Workload(name="opt-6.7b", seed=3, n_layers=32, d_model=4096, n_heads=32,
                         d_ffn=16384, vocab=50272, max_pos=2048, dtype="f16", batch=4,
                         seq_len=1024, lora_targets=("q", "k", "v", "o"), lora_rank=16,
                         lora_alpha=32.0, n_adapters=4, adapter_of_seq=(0, 1, 2, 3)),
    "opt-13b": Workload(name="opt-13b", seed=4, n_layers=40, d_model=5120, n_heads=40,
                        d_ffn=20480, vocab=50272, max_pos=2048, dtype="f16", batch=1,
                        seq_len=2048, lora_targets=("q", "k", "v", "o"), lora_rank=32,
                        lora_alpha=64.0, n_adapters=1,
                        layer_order=tuple(list(range(20, 40)) + list(range(0, 20)))),
    "opt-66b": Workload(name="opt-66b", seed=5, n_layers=64, d_model=9216, n_heads=72,
                        d_ffn=36864, vocab=50272, max_pos=2048, dtype="f16", batch=2,
                        seq_len=2048, lora_targets=("q", "v"), lora_rank=16, lora_alpha=32.0,
                        n_adapters=1),
}


# ----------------------------------------------------------------------------
# stream ids
# ----------------------------------------------------------------------------

TOKEN_STREAM = 3 << 48


def weight_stream(layer: int, name: str) -> int:
    """Stream of a base tensor; layer -1 names the global tensors."""
    if layer < 0:
        tid = GLOBAL_TENSORS.index(name)
        return (1 << 48) | tid
    tid = LAYER_TENSORS.index(name)
    return (1 << 48) | ((layer + 1) << 8) | tid


def lora_stream(adapter: int, layer: int, target: str, which: str) -> int:
    t = TARGETS.index(target)
    return (2 << 48) | (adapter << 32) | ((layer + 1) << 8) | (t << 1) | (1 if which == "B" else 0)


def tensor_shape(w: Workload, layer: int, name: str) -> Tuple[int, ...]:
    d, f = w.d_model, w.d_ffn
    if layer < 0:
        return {"embed": (w.vocab, d), "pos": (w.max_pos, d), "lnf_g": (d,), "lnf_b": (d,)}[name]
    return {"ln1_g": (d,), "ln1_b": (d,), "wq": (d, d), "bq": (d,), "wk": (d, d), "bk": (d,),
            "wv": (d, d), "bv": (d,), "wo": (d, d), "bo": (d,), "ln2_g": (d,), "ln2_b": (d,),
            "w1": (f, d), "b1": (f,), "w2": (d, f), "b2": (d,)}[name]


def tensor_dist(name: str) -> Tuple[float, float]:
    """(mean, std) of a base tensor."""
    if name.endswith("_g"):
        return 1.0, 0.02
    return 0.0, 0.02


def _np_kind(kind: str):
    return np.float32 if kind == "f32" else np.uint16


def fill_normal(seed: int, stream: int, n: int, mean: float, std: float, kind: str,
                ptr: int, offset: int = 0) -> None:
    """Write n draws of (seed, stream) starting at element offset into raw memory."""
    _load().synth_normal(seed, stream, offset, n, mean, std, KIND_CODE[kind], ptr)


def normal(seed: int, stream: int, shape, mean: float, std: float, kind: str) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=_np_kind(kind))
    if n:
        fill_normal(seed, stream, n, mean, std, kind, out.ctypes.data)
    return out.reshape(shape)


def fill_const(n: int, value: float, kind: str, ptr: int) -> None:
    _load().synth_const(n, value, KIND_CODE[kind], ptr)


def base_tensor(w: Workload, layer: int, name: str, kind: str) -> np.ndarray:
    mean, std = tensor_dist(name)
    return normal(w.seed, weight_stream(layer, name), tensor_shape(w, layer, name), mean, std, kind)


def fill_base_tensor(w: Workload, layer: int, name: str, kind: str, ptr: int) -> None:
    mean, std = tensor_dist(name)
    n = int(np.prod(tensor_shape(w, layer, name)))
    fill_normal(w.seed, weight_stream(layer, name), n, mean, std, kind, ptr)


def lora_shape(w: Workload, which: str) -> Tuple[int, int]:
    r, d = w.lora_rank, w.d_model
    return (r, d) if which == "A" else (d, r)


def lora_dist(w: Workload, which: str) -> Tuple[float, float]:
    return (0.0, 1.0 / w.lora_rank) if which == "A" else (0.0, 0.02)


def lora_tensor(w: Workload, adapter: int, layer: int, target: str, which: str,
                kind: str) -> np.ndarray:
    shape = lora_shape(w, which)
    if which == "B" and w.lora_zero_b:
        out = np.empty(int(np.prod(shape)), dtype=_np_kind(kind))
        fill_const(out.size, 0.0, kind, out.ctypes.data)
        return out.reshape(shape)
    mean, std = lora_dist(w, which)
    return normal(w.seed, lora_stream(adapter, layer, target, which), shape, mean, std, kind)


def fill_lora_tensor(w: Workload, adapter: int, layer: int, target: str, which: str, kind: str,
                     ptr: int) -> None:
    n = int(np.prod(lora_shape(w, which)))
    if which == "B" and w.lora_zero_b:
        fill_const(n, 0.0, kind, ptr)
        return
    mean, std = lora_dist(w, which)
    fill_normal(w.seed, lora_stream(adapter, layer, target, which), n, mean, std, kind, ptr)


def tokens(w: Workload, stream: int = TOKEN_STREAM) -> np.ndarray:
    n = w.batch * w.seq_len
    out = np.empty(n, dtype=np.int32)
    if n:
        _load().synth_uniform_int(w.seed, stream, n, 2, w.vocab, out.ctypes.data)
    return out.reshape(w.batch, w.seq_len)


def philox4x32(ctr, key, rounds: int = 10):
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    _load().synth_philox4x32(c, k, rounds, o)
    return tuple(o)


def f32_to_f16_bits(x: float) -> int:
    return int(_load().synth_f32_to_f16(x))


def f32_to_bf16_bits(x: float) -> int:
    return int(_load().synth_f32_to_bf16(x))
