"""Kernel-level parity through include/pipeboost_ops.h: each kernel against the
CPU oracle's component functions (float64), on seeded inputs that span
several tiles, ragged edges and both storage types."""
import numpy as np
import pytest

import oracle
import synth
from gpu_common import log

pytestmark = pytest.mark.gpu


def _dev(bits_or_f32, kind):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(bits_or_f32))
    if kind == "f16":
        t = t.view(torch.float16)
    elif kind == "bf16":
        t = t.view(torch.bfloat16)
    return t.cuda()


def _host_f64(t, kind):
    import torch

    a = t.detach().cpu()
    if kind in ("f16", "bf16"):
        a = a.view(torch.int16).numpy().view(np.uint16)
        return oracle.widen(a, kind)
    return a.numpy().astype(np.float64)


def _draw(seed, stream, shape, std, kind, mean=0.0):
    return synth.normal(seed, stream, shape, mean, std, kind)


DT = {"bf16": 0, "f16": 1}


@pytest.mark.parametrize("kind", ["f16", "bf16"])
@pytest.mark.parametrize("M,N,K", [(37, 192, 128), (300, 384, 576), (512, 1024, 2048),
                                   (1030, 768, 512), (1, 64, 64),
                                   # at most 8 rows: the weight-streaming path, K ragged
                                   # against its 1024-column steps
                                   (1, 2048, 2048), (3, 576, 1600), (8, 128, 8192),
                                   # 256 x 256 tiles: many tiles with a ragged M, and few
                                   # tiles over a long K (split along K)
                                   (4000, 4096, 512), (2048, 2048, 8192),
                                   # 384 tiles of 256: one whole round, the 128 tail tiles
                                   # split in two (ragged last round)
                                   (2048, 12288, 4096)])
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_gemm_epilogues(kind, M, N, K, epi):
    import torch

    log("gemm", kind, M, N, K, epi)
    from paper_2503_17707_amd import binding as pb

    X = _draw(71, 1, (M, K), 1.0, kind)
    W = _draw(71, 2, (N, K), 0.02, kind)
    b = _draw(71, 3, (N,), 0.02, kind)
    Xd, Wd, bd = _dev(X, kind), _dev(W, kind), _dev(b, kind)
    ref = oracle.widen(X, kind) @ oracle.widen(W, kind).T + oracle.widen(b, kind)
    ws = torch.empty(max(16 << 20, min(256 << 20, 16 * M * N)), dtype=torch.uint8, device="cuda")
    if epi == 2:
        R0 = synth.normal(71, 4, (M, N), 0.0, 1.0, "f32")
        R = torch.from_numpy(R0.copy()).cuda()
        pb.op_gemm(DT[kind], 2, Xd, Wd, bd, R=R, workspace=ws)
        torch.cuda.synchronize()
        got = R.cpu().numpy().astype(np.float64)
        ref = ref + R0
        tol = 1e-5 * np.abs(ref).max() + 2e-5 * np.sqrt(K)
    else:
        C = torch.empty((M, N), dtype=Xd.dtype, device="cuda")
        qcols = N // 3
        qs = 0.125
        pb.op_gemm(DT[kind], epi, Xd, Wd, bd, C=C, qscale=qs, qcols=qcols, workspace=ws)
        torch.cuda.synchronize()
        got = _host_f64(C, kind)
        if epi == 0:
            ref[:, :qcols] *= qs
        else:
            ref = np.maximum(ref, 0.0)
        ulp = 2.0 ** -8 if kind == "bf16" else 2.0 ** -11
        tol = ulp * np.abs(ref) + 1e-4
    err = np.abs(got - ref)
    assert np.all(err <= tol), "max err %.3e" % err.max()


@pytest.mark.parametrize("kind,hd,B,T,H", [("f16", 64, 2, 200, 3), ("bf16", 64, 1, 37, 2),
                                           ("f16", 128, 1, 130, 2), ("bf16", 128, 2, 64, 1),
                                           ("f16", 128, 1, 1100, 4), ("f16", 64, 1, 1, 2),
                                           ("bf16", 64, 1, 530, 2), ("f16", 64, 2, 129, 2),
                                           # long prompts (8-wave blocks): 32 and 16 queries per
                                           # wave, (sequence, head) pairs a multiple of 8, ragged T
                                           ("f16", 128, 4, 1024, 32), ("bf16", 128, 1, 2000, 40)])
def test_attention(kind, hd, B, T, H):
    import torch

    log("attention", kind, hd, B, T, H)
    from paper_2503_17707_amd import binding as pb

    d = H * hd
    qkv = _draw(72, 1, (B * T, 3 * d), 1.0, kind)
    qd = _dev(qkv, kind)
    out = torch.empty((B * T, d), dtype=qd.dtype, device="cuda")
    pb.op_attention(DT[kind], qd, out, B, T, H, hd)
    torch.cuda.synchronize()
    got = _host_f64(out, kind)
    q64 = oracle.widen(qkv, kind)
    ref = np.concatenate([oracle.causal_self_attention(q64[b * T:(b + 1) * T, :d],
                                                       q64[b * T:(b + 1) * T, d:2 * d],
                                                       q64[b * T:(b + 1) * T, 2 * d:], H)
                          for b in range(B)])
    # probabilities enter the MFMA rounded to the storage type
    ulp = 2.0 ** -8 if kind == "bf16" else 2.0 ** -11
    err = np.abs(got - ref)
    assert err.max() <= 4 * ulp * np.abs(ref).max() + 1e-3, "max err %.3e" % err.max()


@pytest.mark.parametrize("kind,rows,d", [("f16", 5, 2048), ("bf16", 33, 256), ("f16", 2, 9216),
                                         ("f16", 3, 16384)])
def test_layernorm(kind, rows, d):
    import torch

    log("layernorm", kind, rows, d)
    from paper_2503_17707_amd import binding as pb

    x = synth.normal(73, 1, (rows, d), 0.3, 2.0, "f32")
    g = _draw(73, 2, (d,), 0.02, kind, mean=1.0)
    b = _draw(73, 3, (d,), 0.02, kind)
    xd = torch.from_numpy(x).cuda()
    gd, bd = _dev(g, kind), _dev(b, kind)
    out16 = torch.empty((rows, d), dtype=gd.dtype, device="cuda")
    out32 = torch.empty((rows, d), dtype=torch.float32, device="cuda")
    pb.op_layernorm(DT[kind], xd, gd, bd, out16)
    pb.op_layernorm(DT[kind], xd, gd, bd, out32)
    torch.cuda.synchronize()
    ref = oracle.layer_norm(x.astype(np.float64), oracle.widen(g, kind), oracle.widen(b, kind), 1e-5)
    ulp = 2.0 ** -8 if kind == "bf16" else 2.0 ** -11
    assert np.all(np.abs(_host_f64(out16, kind) - ref) <= ulp * np.abs(ref) + 1e-5)
    assert np.max(np.abs(out32.cpu().numpy() - ref)) < 1e-4
