"""Thin ctypes binding of libpipeboost.so (argument marshalling only).

Every step of the prefill runs inside the HIP library.  PyTorch is used only
to allocate the device arena and the two streams.  There is no fallback: if
the library is missing, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# PIPEBOOST_LIB selects another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("PIPEBOOST_LIB") or os.path.join(HERE, "lib", "libpipeboost.so")

PB_OK, PB_EINVAL, PB_ENOTPINNED, PB_ENOMEM, PB_EHIP, PB_ESTATE = 0, -1, -2, -3, -4, -5
PB_BF16, PB_F16 = 0, 1
LORA_BITS = {"q": 1, "k": 2, "v": 4, "o": 8}
TARGET_INDEX = {"q": 0, "k": 1, "v": 2, "o": 3}
LAYER_TENSOR_ID = {n: i for i, n in enumerate(
    ("ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "ln2_g", "ln2_b",
     "w1", "b1", "w2", "b2"))}
GLOBAL_TENSOR_ID = {"embed": 0, "pos": 1, "lnf_g": 2, "lnf_b": 3}
KERNEL_KINDS = ("embed", "layernorm", "lora_shrink", "gemm_qkv", "attention", "gemm_o",
                "gemm_fc1", "gemm_fc2", "lm_head", "argmax")


class PbError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("pipeboost error %d: %s" % (code, msg))
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("max_pos", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("max_adapters", ctypes.c_int32), ("max_rank", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float),
                ("max_new_tokens", ctypes.c_int32), ("merge_shadow", ctypes.c_int32)]


_SIGS = {
    "pb_layer_bytes": (ctypes.c_size_t, [ctypes.POINTER(Config)]),
    "pb_globals_bytes": (ctypes.c_size_t, [ctypes.POINTER(Config)]),
    "pb_layer_tensor": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.c_int32,
                                       ctypes.POINTER(ctypes.c_size_t),
                                       ctypes.POINTER(ctypes.c_size_t)]),
    "pb_globals_tensor": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.c_int32,
                                         ctypes.POINTER(ctypes.c_size_t),
                                         ctypes.POINTER(ctypes.c_size_t)]),
    "pb_lora_layer_bytes": (ctypes.c_size_t, [ctypes.POINTER(Config), ctypes.c_int32,
                                              ctypes.c_uint32]),
    "pb_lora_tensor": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.c_int32, ctypes.c_uint32,
                                      ctypes.c_int32, ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_size_t),
                                      ctypes.POINTER(ctypes.c_size_t)]),
    "pb_arena_bytes": (ctypes.c_size_t, [ctypes.POINTER(Config)]),
    "pb_host_alloc": (ctypes.c_int, [ctypes.c_size_t, ctypes.POINTER(ctypes.c_void_p)]),
    "pb_host_free": (ctypes.c_int, [ctypes.c_void_p]),
    "pb_host_numa_node": (ctypes.c_int, [ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
    "pb_set_host_numa_node": (ctypes.c_int, [ctypes.c_int32]),
    "pb_model_create": (ctypes.c_int, [ctypes.POINTER(Config), ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_void_p)]),
    "pb_stream_layers": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                        ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p),
                                        ctypes.c_void_p]),
    "pb_attach_lora": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_float, ctypes.c_uint32,
                                      ctypes.POINTER(ctypes.c_void_p)]),
    "pb_rebuild_kv": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                     ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_float)]),
    "pb_invalidate_kv": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint8), ctypes.c_int32]),
    "pb_merge_lora": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "pb_prefill_stage": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                        ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_float)]),
    "pb_unmerge_lora": (ctypes.c_int, [ctypes.c_void_p]),
    "pb_sched_create": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p)]),
    "pb_sched_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "pb_sched_submit": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32]),
    "pb_sched_next": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                     ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_int32)]),
    "pb_sched_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64),
                                      ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)]),
    "pb_plan_loading": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_uint8),
                                       ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                       ctypes.POINTER(ctypes.c_int32)]),
    "pb_decode_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                      ctypes.POINTER(ctypes.c_float)]),
    "pb_prefill_first_token": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                              ctypes.c_int32, ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_int32),
                                              ctypes.POINTER(ctypes.c_int32),
                                              ctypes.POINTER(ctypes.c_float)]),
    "pb_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "pb_last_error": (ctypes.c_char_p, []),
    "pb_set_chunk_bytes": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t]),
    "pb_last_load_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_double)]),
    "pb_set_kernel_timing": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "pb_set_graph_replay": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "pb_get_kernel_timing": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_int64)]),
    "pb_reset_kernel_timing": (ctypes.c_int, [ctypes.c_void_p]),
    "pb_poison_weights": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "pb_set_stream_delay_us": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "pb_op_gemm": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                  ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "pb_op_gemm_lora": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_uint32, ctypes.c_float, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_size_t, ctypes.c_void_p]),
    "pb_op_gemm_noalloc": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                          ctypes.c_void_p]),
    "pb_op_attention": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_void_p]),
    "pb_op_layernorm": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                       ctypes.c_int32, ctypes.c_int32, ctypes.c_float,
                                       ctypes.c_void_p]),
}

_lib = None


def lib():
    """Load libpipeboost.so (built by ``paper_2503_17707_amd.build``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libpipeboost.so is not built (%s); run __graft_entry__.build()"
                               % LIB_PATH)
        # One HIP runtime per process: torch ships its own libamdhip64.so.7 with
        # the same soname, so it must be loaded first and the library then binds
        # to it (the streams torch creates are only valid in that runtime).
        import torch  # noqa: F401

        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(rc: int) -> None:
    if rc != PB_OK:
        raise PbError(rc, lib().pb_last_error().decode())


def make_config(w, max_tokens: Optional[int] = None, max_batch: Optional[int] = None,
                max_adapters: Optional[int] = None, max_rank: Optional[int] = None,
                max_new_tokens: int = 0, merge_shadow: bool = False) -> Config:
    """pb_config of a synth.Workload (capacities default to the workload's own sizes;
    max_new_tokens > 0 adds a KV cache for decode steps; merge_shadow keeps the
    unmerged attention weights for adapter switching)."""
    return Config(n_layers=w.n_layers, d_model=w.d_model, n_heads=w.n_heads, d_ffn=w.d_ffn,
                  vocab=w.vocab, max_pos=w.max_pos,
                  max_tokens=max_tokens or w.batch * w.seq_len,
                  max_batch=max_batch or w.batch,
                  max_adapters=w.n_adapters if max_adapters is None else max_adapters,
                  max_rank=max_rank or w.lora_rank,
                  dtype=PB_BF16 if w.dtype == "bf16" else PB_F16, ln_eps=w.ln_eps,
                  max_new_tokens=max_new_tokens, merge_shadow=1 if merge_shadow else 0)


def layer_tensor(cfg: Config, name: str):
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    check(lib().pb_layer_tensor(ctypes.byref(cfg), LAYER_TENSOR_ID[name], ctypes.byref(off),
                                ctypes.byref(n)))
    return off.value, n.value


def globals_tensor(cfg: Config, name: str):
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    check(lib().pb_globals_tensor(ctypes.byref(cfg), GLOBAL_TENSOR_ID[name], ctypes.byref(off),
                                  ctypes.byref(n)))
    return off.value, n.value


def lora_tensor(cfg: Config, rank: int, mask: int, target: str, which: str):
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    check(lib().pb_lora_tensor(ctypes.byref(cfg), rank, mask, TARGET_INDEX[target],
                               0 if which == "A" else 1, ctypes.byref(off), ctypes.byref(n)))
    return off.value, n.value


class Pinned:
    """A pinned host buffer from pb_host_alloc, freed with pb_host_free."""

    def __init__(self, nbytes: int):
        p = ctypes.c_void_p()
        check(lib().pb_host_alloc(nbytes, ctypes.byref(p)))
        self.ptr = p.value
        self.nbytes = nbytes

    def view(self, dtype=np.uint8) -> np.ndarray:
        buf = (ctypes.c_uint8 * self.nbytes).from_address(self.ptr)
        return np.frombuffer(buf, dtype=np.uint8).view(dtype)

    def free(self):
        if self.ptr:
            lib().pb_host_free(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def gpu_numa_node(device: int = 0) -> int:
    """NUMA node of the GPU (pb_host_numa_node), -1 if the system reports none."""
    n = ctypes.c_int32(-1)
    check(lib().pb_host_numa_node(device, ctypes.byref(n)))
    return n.value


def _mbind(ptr: int, nbytes: int, node: int) -> bool:
    """Prefer one NUMA node for a page-aligned, not yet touched range (mbind,
    MPOL_PREFERRED), so its pages come from that node whichever thread first
    writes them (from another node only if that one is full)."""
    if node < 0 or nbytes <= 0:
        return False
    libc = ctypes.CDLL(None, use_errno=True)
    bits = 8 * ctypes.sizeof(ctypes.c_ulong)
    mask = (ctypes.c_ulong * (1024 // bits))()
    mask[node // bits] = 1 << (node % bits)
    length = (nbytes + 4095) // 4096 * 4096
    SYS_mbind = 237  # x86_64
    return libc.syscall(SYS_mbind, ctypes.c_void_p(ptr), ctypes.c_ulong(length), 1, mask,
                        ctypes.c_ulong(1024), 0) == 0


class Pageable:
    """A page-aligned ordinary (pageable) host buffer with the interface of
    Pinned; with a NUMA node its pages are bound there before first touch."""

    def __init__(self, nbytes: int, node: int = -1):
        self._buf = np.empty(nbytes + 2 * 4096, np.uint8)
        off = (-self._buf.ctypes.data) % 4096
        self._arr = self._buf[off:off + nbytes]
        self.ptr = self._arr.ctypes.data
        self.nbytes = nbytes
        self.bound = _mbind(self.ptr, nbytes, node)

    def view(self, dtype=np.uint8) -> np.ndarray:
        return self._arr.view(dtype)

    def free(self):
        self._buf = self._arr = None
        self.ptr = None


# Host memory the layer blobs may pin (the rest stay pageable and the loader
# stages them through its own pinned ring): hosts can cap locked memory well
# below their RAM.  PIPEBOOST_PIN_BUDGET_GB overrides.
DEFAULT_PIN_BUDGET = int(float(os.environ.get("PIPEBOOST_PIN_BUDGET_GB", "48")) * (1 << 30))


class HostWeights:
    """Host blobs of a workload in the library's device layout, drawn by synth:
    the globals and LoRA blobs pinned, layer blobs pinned while they fit in
    pin_budget bytes (in layer-id order) and pageable after that.  With
    numa (default: on unless PIPEBOOST_NUMA=0) every blob sits on the GPU's
    NUMA node."""

    def __init__(self, w, cfg: Config, pin_budget: Optional[int] = None, numa: Optional[bool] = None):
        import synth

        self.w, self.cfg = w, cfg
        budget = DEFAULT_PIN_BUDGET if pin_budget is None else pin_budget
        L = lib()
        if numa is None:
            numa = os.environ.get("PIPEBOOST_NUMA", "1") != "0"
        self.numa_node = gpu_numa_node() if numa else -1
        check(L.pb_set_host_numa_node(self.numa_node))
        kind = w.dtype
        self.layer_bytes = L.pb_layer_bytes(ctypes.byref(cfg))
        self.globals_bytes = L.pb_globals_bytes(ctypes.byref(cfg))
        if not self.layer_bytes or not self.globals_bytes:
            raise PbError(PB_EINVAL, "invalid config for %s" % w.name)
        self.globals = Pinned(self.globals_bytes)
        self.globals.view()[:] = 0
        for name in synth.GLOBAL_TENSORS:
            off, _ = globals_tensor(cfg, name)
            synth.fill_base_tensor(w, -1, name, kind, self.globals.ptr + 2 * off)
        self.layers: List[Pinned] = []
        self.pinned_layers = 0
        for layer in range(w.n_layers):
            if (layer + 1) * self.layer_bytes <= budget:
                blob = Pinned(self.layer_bytes)
                self.pinned_layers += 1
            else:
                blob = Pageable(self.layer_bytes, self.numa_node)
            self._zero_padding(blob, cfg)
            for name in synth.LAYER_TENSORS:
                off, _ = layer_tensor(cfg, name)
                synth.fill_base_tensor(w, layer, name, kind, blob.ptr + 2 * off)
            self.layers.append(blob)
        self.loras: Dict[int, List[Pinned]] = {}

    def _zero_padding(self, blob: Pinned, cfg: Config):
        # every byte of the blob is written by a tensor except the alignment
        # gaps between them: zero only those (the tensors' own fills touch the
        # rest first, from all of the generator's threads)
        import synth

        spans = sorted(layer_tensor(cfg, n) for n in synth.LAYER_TENSORS)
        pos = 0
        for off, n in spans:
            if 2 * off > pos:
                ctypes.memset(blob.ptr + pos, 0, 2 * off - pos)
            pos = max(pos, 2 * (off + n))
        if blob.nbytes > pos:
            ctypes.memset(blob.ptr + pos, 0, blob.nbytes - pos)

    def lora_mask(self) -> int:
        m = 0
        for t in self.w.lora_targets:
            m |= LORA_BITS[t]
        return m

    def add_lora(self, adapter: int) -> List[Pinned]:
        import synth

        w, cfg = self.w, self.cfg
        mask = self.lora_mask()
        nbytes = lib().pb_lora_layer_bytes(ctypes.byref(cfg), w.lora_rank, mask)
        if not nbytes:
            raise PbError(PB_EINVAL, "invalid LoRA shape")
        blobs = []
        for layer in range(w.n_layers):
            blob = Pinned(nbytes)
            for t in w.lora_targets:
                for which in ("A", "B"):
                    off, _ = lora_tensor(cfg, w.lora_rank, mask, t, which)
                    synth.fill_lora_tensor(w, adapter, layer, t, which, w.dtype,
                                           blob.ptr + 2 * off)
            blobs.append(blob)
        self.loras[adapter] = blobs
        return blobs

    def free(self):
        self.globals.free()
        for b in self.layers:
            b.free()
        for bl in self.loras.values():
            for b in bl:
                b.free()


class Model:
    """A pb_model over a torch-allocated arena and two torch streams."""

    def __init__(self, cfg: Config, device: str = "cuda:0"):
        import torch

        self.cfg = cfg
        L = lib()
        self.arena_bytes = L.pb_arena_bytes(ctypes.byref(cfg))
        if not self.arena_bytes:
            raise PbError(PB_EINVAL, "invalid config")
        self.device = torch.device(device)
        self.arena = torch.empty(self.arena_bytes + 256, dtype=torch.uint8, device=self.device)
        base = self.arena.data_ptr()
        self.base = (base + 255) // 256 * 256
        self.copy_stream = torch.cuda.Stream(device=self.device)
        self.compute_stream = torch.cuda.Stream(device=self.device)
        torch.cuda.synchronize(self.device)
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            check(L.pb_model_create(ctypes.byref(cfg), ctypes.c_void_p(self.base),
                                    self.arena_bytes, ctypes.c_void_p(self.copy_stream.cuda_stream),
                                    ctypes.c_void_p(self.compute_stream.cuda_stream),
                                    ctypes.byref(h)))
        self.h = h

    def stream_layers(self, hw: HostWeights, order: Optional[Sequence[int]] = None):
        n = self.cfg.n_layers
        order = list(range(n)) if order is None else list(order)
        arr = (ctypes.c_int32 * len(order))(*order)
        ptrs = (ctypes.c_void_p * n)(*[b.ptr for b in hw.layers])
        check(lib().pb_stream_layers(self.h, arr, len(order), ptrs, ctypes.c_void_p(hw.globals.ptr)))

    def attach_lora(self, slot: int, blobs: List[Pinned], rank: int, alpha: float, mask: int):
        ptrs = (ctypes.c_void_p * len(blobs))(*[b.ptr for b in blobs])
        check(lib().pb_attach_lora(self.h, slot, rank, alpha, mask, ptrs))

    def prefill(self, tokens: np.ndarray, adapter_of_seq: Optional[Sequence[int]] = None,
                want_logits: bool = True):
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        B, T = tokens.shape
        out_tok = np.empty(B, dtype=np.int32)
        logits = np.empty((B, self.cfg.vocab), dtype=np.float32) if want_logits else None
        ad = None
        if adapter_of_seq is not None:
            ad_arr = np.ascontiguousarray(adapter_of_seq, dtype=np.int32)
            ad = ad_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        check(lib().pb_prefill_first_token(
            self.h, tokens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), B, T, ad,
            out_tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            logits.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if want_logits else None))
        return out_tok, logits

    def prefill_stage(self, tokens: np.ndarray, adapter_of_seq: Optional[Sequence[int]], layer_begin: int,
                      layer_end: int, hidden_in=None, hidden_out=None, want_logits: bool = True):
        """Layers [layer_begin, layer_end) of a prefill (pb_prefill_stage).  hidden_in /
        hidden_out: device fp32 tensors of [B*T, d_model] (or None at the ends).
        Returns (tokens, logits) from the last stage, None from the others."""
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        B, T = tokens.shape
        last = layer_end == self.cfg.n_layers
        out_tok = np.empty(B, dtype=np.int32) if last else None
        logits = np.empty((B, self.cfg.vocab), dtype=np.float32) if (last and want_logits) else None
        ad = None
        if adapter_of_seq is not None:
            ad_arr = np.ascontiguousarray(adapter_of_seq, dtype=np.int32)
            ad = ad_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        check(lib().pb_prefill_stage(
            self.h, tokens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), B, T, ad, layer_begin, layer_end,
            ctypes.c_void_p(hidden_in.data_ptr()) if hidden_in is not None else None,
            ctypes.c_void_p(hidden_out.data_ptr()) if hidden_out is not None else None,
            out_tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if last else None,
            logits.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if logits is not None else None))
        return (out_tok, logits) if last else None

    def decode(self, tokens: np.ndarray, adapter_of_seq: Optional[Sequence[int]] = None,
               want_logits: bool = True):
        """One decode step: tokens [B] (the newest token of each sequence)."""
        tokens = np.ascontiguousarray(tokens, dtype=np.int32).reshape(-1)
        B = tokens.shape[0]
        out_tok = np.empty(B, dtype=np.int32)
        logits = np.empty((B, self.cfg.vocab), dtype=np.float32) if want_logits else None
        ad = None
        if adapter_of_seq is not None:
            ad_arr = np.ascontiguousarray(adapter_of_seq, dtype=np.int32)
            ad = ad_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        check(lib().pb_decode_step(
            self.h, tokens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), B, ad,
            out_tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            logits.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if want_logits else None))
        return out_tok, logits

    def rebuild_kv(self, tokens: np.ndarray, layer_has_kv: Sequence[bool],
                   adapter_of_seq: Optional[Sequence[int]] = None, want_logits: bool = True):
        """KV-cache rebuild over tokens [B, T]; returns the next token of each sequence."""
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        B, T = tokens.shape
        has = np.ascontiguousarray([1 if h else 0 for h in layer_has_kv], dtype=np.uint8)
        out_tok = np.empty(B, dtype=np.int32)
        logits = np.empty((B, self.cfg.vocab), dtype=np.float32) if want_logits else None
        ad = None
        if adapter_of_seq is not None:
            ad_arr = np.ascontiguousarray(adapter_of_seq, dtype=np.int32)
            ad = ad_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        check(lib().pb_rebuild_kv(
            self.h, tokens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), B, T, ad,
            has.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
            out_tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            logits.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if want_logits else None))
        return out_tok, logits

    def merge_lora(self, slot: int):
        check(lib().pb_merge_lora(self.h, slot))

    def unmerge_lora(self):
        check(lib().pb_unmerge_lora(self.h))

    def invalidate_kv(self, layer_lost: Sequence[bool], value: int = 0xFF):
        lost = np.ascontiguousarray([1 if x else 0 for x in layer_lost], dtype=np.uint8)
        check(lib().pb_invalidate_kv(self.h, lost.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), value))

    def poison(self, value: int = 0xFF):
        check(lib().pb_poison_weights(self.h, value))

    def set_chunk_bytes(self, n: int):
        check(lib().pb_set_chunk_bytes(self.h, n))

    def set_stream_delay_us(self, us: int):
        check(lib().pb_set_stream_delay_us(self.h, us))

    def load_stats(self):
        b, ms = ctypes.c_double(), ctypes.c_double()
        check(lib().pb_last_load_stats(self.h, ctypes.byref(b), ctypes.byref(ms)))
        return b.value, ms.value

    def set_graph_replay(self, on: bool):
        """Record settled forward shapes as HIP graphs and replay them (default on)."""
        check(lib().pb_set_graph_replay(self.h, 1 if on else 0))

    def set_timing(self, on: bool):
        check(lib().pb_set_kernel_timing(self.h, 1 if on else 0))

    def reset_timing(self):
        check(lib().pb_reset_kernel_timing(self.h))

    def timing(self) -> Dict[str, tuple]:
        out = {}
        for i, k in enumerate(KERNEL_KINDS):
            ms, n = ctypes.c_double(), ctypes.c_int64()
            check(lib().pb_get_kernel_timing(self.h, i, ctypes.byref(ms), ctypes.byref(n)))
            out[k] = (ms.value, n.value)
        return out

    def destroy(self):
        if self.h:
            lib().pb_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def setup(w, device: str = "cuda:0", hw: Optional[HostWeights] = None, **cap):
    """Create the host blobs (layer blobs pinned up to the budget) and a model."""
    cfg = make_config(w, **cap)
    hw = hw or HostWeights(w, cfg)
    m = Model(cfg, device)
    return hw, m


def attach_all(m: Model, hw: HostWeights):
    """Attach adapter a of the workload into slot a, for every adapter it uses."""
    w = hw.w
    used = sorted({a for a in w.adapters() if a >= 0})
    for a in used:
        blobs = hw.loras.get(a) or hw.add_lora(a)
        m.attach_lora(a, blobs, w.lora_rank, w.lora_alpha, hw.lora_mask())


class Scheduler:
    """Epoch-based adapter switching (pb_sched_*): per-adapter request queues;
    epoch_batches = 0 is the eager, arrival-order baseline."""

    def __init__(self, n_adapters: int, epoch_batches: int):
        h = ctypes.c_void_p()
        check(lib().pb_sched_create(n_adapters, epoch_batches, ctypes.byref(h)))
        self.h = h

    def submit(self, request_id: int, adapter: int):
        check(lib().pb_sched_submit(self.h, request_id, adapter))

    def next(self, max_batch: int):
        """(request ids, adapter, switched), or None when every queue is empty."""
        ids = (ctypes.c_int64 * max_batch)()
        n, a, sw = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        check(lib().pb_sched_next(self.h, max_batch, ids, ctypes.byref(n), ctypes.byref(a), ctypes.byref(sw)))
        if n.value == 0:
            return None
        return list(ids[:n.value]), a.value, bool(sw.value)

    def stats(self):
        """(pending, switches, active adapter; -2 before the first batch)."""
        p, sw, a = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
        check(lib().pb_sched_stats(self.h, ctypes.byref(p), ctypes.byref(sw), ctypes.byref(a)))
        return p.value, sw.value, a.value

    def close(self):
        if self.h:
            check(lib().pb_sched_destroy(self.h))
            self.h = None


def plan_loading(n_layers: int, alive: Sequence[bool]):
    """Per-GPU layer orders and owned blocks (pb_plan_loading): returns
    (orders [n_gpus][n_layers] with -1 rows for failed GPUs, [(first, len)] per GPU)."""
    G = len(alive)
    al = np.ascontiguousarray([1 if a else 0 for a in alive], dtype=np.uint8)
    order = np.empty((G, n_layers), dtype=np.int32)
    first = np.empty(G, dtype=np.int32)
    ln = np.empty(G, dtype=np.int32)
    p32 = ctypes.POINTER(ctypes.c_int32)
    check(lib().pb_plan_loading(n_layers, G, al.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                order.ctypes.data_as(p32), first.ctypes.data_as(p32), ln.ctypes.data_as(p32)))
    return order, list(zip(first.tolist(), ln.tolist()))


# ---- kernel-level entry points (include/pipeboost_ops.h) --------------------
# Arguments are torch tensors on the GPU; the call is enqueued on `stream`
# (a torch.cuda.Stream, default: the current stream).

def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    return ctypes.c_void_p((stream or torch.cuda.current_stream()).cuda_stream)


def op_gemm(dtype: int, epi: int, X, W, bias, C=None, R=None, qscale: float = 1.0,
            qcols: int = 0, workspace=None, stream=None):
    M, K = X.shape
    N = W.shape[0]
    check(lib().pb_op_gemm(dtype, epi, _ptr(X), _ptr(W), _ptr(bias), _ptr(C), _ptr(R), M, N, K,
                           qscale, qcols, _ptr(workspace),
                           0 if workspace is None else workspace.numel() * workspace.element_size(),
                           _stream(stream)))


def op_gemm_lora(dtype: int, epi: int, X, W, bias, Z, zs: int, W2, group: int, group_mask: int,
                 C=None, R=None, qscale: float = 1.0, qcols: int = 0, workspace=None, stream=None):
    """pb_op_gemm_lora: Z [M, ldz] scaled shrinks (group g's block at column g * zs), W2 [N, K2]."""
    M, K = X.shape
    N = W.shape[0]
    K2 = W2.shape[1]
    check(lib().pb_op_gemm_lora(dtype, epi, _ptr(X), _ptr(W), _ptr(bias), _ptr(C), _ptr(R), M, N, K,
                                _ptr(Z), Z.shape[1], zs, _ptr(W2), K2, group, group_mask, qscale, qcols,
                                _ptr(workspace),
                                0 if workspace is None else workspace.numel() * workspace.element_size(),
                                _stream(stream)))


def op_gemm_noalloc(dtype: int, epi: int, X, W, bias, C=None, R=None, qscale: float = 1.0,
                    qcols: int = 0, stream=None):
    """pb_op_gemm_noalloc: pb_op_gemm with the library's own split-K scratch."""
    M, K = X.shape
    N = W.shape[0]
    check(lib().pb_op_gemm_noalloc(dtype, epi, _ptr(X), _ptr(W), _ptr(bias), _ptr(C), _ptr(R), M, N,
                                   K, qscale, qcols, _stream(stream)))


def op_attention(dtype: int, qkv, out, B: int, T: int, H: int, hd: int, stream=None):
    check(lib().pb_op_attention(dtype, _ptr(qkv), _ptr(out), B, T, H, hd, _stream(stream)))


def op_layernorm(dtype: int, x, g, b, out, eps: float = 1e-5, stream=None):
    rows, d = x.shape
    import torch

    check(lib().pb_op_layernorm(dtype, _ptr(x), _ptr(g), _ptr(b), _ptr(out),
                                1 if out.dtype == torch.float32 else 0, rows, d, eps,
                                _stream(stream)))
