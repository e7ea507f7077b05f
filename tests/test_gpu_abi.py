"""Error convention of the C ABI on a live device: every misuse returns its
documented code, leaves a message, and the model stays usable."""
import ctypes

import numpy as np
import pytest

import synth
from gpu_common import log

pytestmark = pytest.mark.gpu

W = synth.Workload(name="abi", seed=41, n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=300,
                   max_pos=16, dtype="f16", batch=2, seq_len=8, lora_targets=("q", "v"),
                   lora_rank=4, lora_alpha=8.0, n_adapters=1)


def test_error_codes():
    from paper_2503_17707_amd import binding as pb

    L = pb.lib()
    log("case abi errors")
    hw, m = pb.setup(W)
    try:
        toks = synth.tokens(W)
        # prefill before any streaming
        with pytest.raises(pb.PbError) as e:
            m.prefill(toks)
        assert e.value.code == pb.PB_ESTATE
        # repeated, out of range, empty or too many layer ids
        for bad in ([0, 0], [1, 2], [], [0, 1, 0]):
            arr = (ctypes.c_int32 * len(bad))(*bad)
            ptrs = (ctypes.c_void_p * 2)(*[b.ptr for b in hw.layers])
            rc = L.pb_stream_layers(m.h, arr, len(bad), ptrs, ctypes.c_void_p(hw.globals.ptr))
            assert rc == pb.PB_EINVAL, bad
            assert L.pb_last_error()
        # a NULL layer blob
        arr = (ctypes.c_int32 * 2)(0, 1)
        ptrs = (ctypes.c_void_p * 2)(None, hw.layers[1].ptr)
        assert L.pb_stream_layers(m.h, arr, 2, ptrs, ctypes.c_void_p(hw.globals.ptr)) == pb.PB_EINVAL
        # a subset of the layers (a pipeline stage's share) streams, but a full
        # prefill needs the layer it lacks
        m.stream_layers(hw, [0])
        with pytest.raises(pb.PbError) as e:
            m.prefill(toks)
        assert e.value.code == pb.PB_ESTATE
        # a valid stream, then argument errors of the prefill
        m.stream_layers(hw)
        with pytest.raises(pb.PbError) as e:
            m.prefill(np.zeros((3, 8), np.int32))  # B > max_batch
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:
            m.prefill(np.zeros((1, 17), np.int32))  # T > max_pos
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:
            m.prefill(np.full((1, 4), 300, np.int32))  # token outside the vocabulary
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:
            m.prefill(toks, [0, 0])  # slot 0 never attached
        assert e.value.code == pb.PB_ESTATE
        with pytest.raises(pb.PbError) as e:
            m.prefill(toks, [1, 0])  # slot outside [-1, max_adapters)
        assert e.value.code == pb.PB_EINVAL
        # LoRA attach errors
        blobs = hw.add_lora(0)
        with pytest.raises(pb.PbError) as e:
            m.attach_lora(1, blobs, 4, 8.0, 5)  # slot >= max_adapters
        assert e.value.code == pb.PB_EINVAL
        with pytest.raises(pb.PbError) as e:
            m.attach_lora(0, blobs, 5, 8.0, 5)  # rank > max_rank
        assert e.value.code == pb.PB_EINVAL
        # LoRA blobs must be pinned
        pageable = [pb.Pageable(b.nbytes) for b in blobs]
        with pytest.raises(pb.PbError) as e:
            m.attach_lora(0, pageable, 4, 8.0, 5)
        assert e.value.code == pb.PB_ENOTPINNED
        # the model still works after every refusal
        m.attach_lora(0, blobs, 4, 8.0, 5)
        tok, logits = m.prefill(toks, [0, -1])
        assert np.all(np.isfinite(logits)) and tok.shape == (2,)
    finally:
        m.destroy()
        hw.free()


def test_create_refuses_small_arena_and_equal_streams():
    import torch

    from paper_2503_17707_amd import binding as pb

    L = pb.lib()
    cfg = pb.make_config(W)
    need = L.pb_arena_bytes(ctypes.byref(cfg))
    buf = torch.empty(need + 512, dtype=torch.uint8, device="cuda:0")
    base = (buf.data_ptr() + 255) // 256 * 256
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    h = ctypes.c_void_p()
    assert L.pb_model_create(ctypes.byref(cfg), ctypes.c_void_p(base), need - 256,
                             ctypes.c_void_p(s1.cuda_stream), ctypes.c_void_p(s2.cuda_stream),
                             ctypes.byref(h)) == pb.PB_ENOMEM
    assert L.pb_model_create(ctypes.byref(cfg), ctypes.c_void_p(base), need,
                             ctypes.c_void_p(s1.cuda_stream), ctypes.c_void_p(s1.cuda_stream),
                             ctypes.byref(h)) == pb.PB_EINVAL
    assert L.pb_model_create(ctypes.byref(cfg), ctypes.c_void_p(base + 8), need,
                             ctypes.c_void_p(s1.cuda_stream), ctypes.c_void_p(s2.cuda_stream),
                             ctypes.byref(h)) == pb.PB_EINVAL
    assert L.pb_model_create(ctypes.byref(cfg), ctypes.c_void_p(base), need,
                             ctypes.c_void_p(s1.cuda_stream), ctypes.c_void_p(s2.cuda_stream),
                             ctypes.byref(h)) == pb.PB_OK
    assert L.pb_destroy(h) == pb.PB_OK
