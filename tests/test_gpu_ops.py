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


@pytest.mark.parametrize("kind", ["f16", "bf16"])
@pytest.mark.parametrize("M,group,K", [(300, 256, 512), (4000, 1024, 512)])
@pytest.mark.parametrize("epi", [0, 2])
def test_gemm_lora_expand(kind, M, group, K, epi):
    """The LoRA expand as extra K tiles (pb_op_gemm_lora): three output groups
    (q, k, v), the expand on groups 0 and 2 only, rows cycling through adapter
    slots 0, 1 and none; against the plain product with the same operands and
    against the oracle's unmerged LoRA delta."""
    import torch

    log("gemm lora", kind, M, group, K, epi)
    from paper_2503_17707_amd import binding as pb

    r, n_slots, K2 = 16, 2, 64  # slot columns [16 slot, 16 slot + 16), 32 .. 63 zero
    N, mask, scale = 3 * group, 0b101, 2.0
    X = _draw(81, 1, (M, K), 1.0, kind)
    W = _draw(81, 2, (N, K), 0.02, kind)
    b = _draw(81, 3, (N,), 0.02, kind)
    A = [[_draw(81, 10 + 3 * a + g, (r, K), 1.0 / r, kind) for g in range(3)] for a in range(n_slots)]
    Bm = [[_draw(81, 20 + 3 * a + g, (group, r), 0.02, kind) for g in range(3)] for a in range(n_slots)]
    slot = np.array([(0, 1, -1)[m % 3] for m in range(M)])
    x64 = oracle.widen(X, kind)
    # the scaled shrink of each row's adapter in its slot's columns of every group block
    Zf = np.zeros((M, 3 * K2))
    W2f = np.zeros((N, K2))
    for a in range(n_slots):
        rows = slot == a
        for g in range(3):
            Zf[rows, g * K2 + r * a: g * K2 + r * (a + 1)] = scale * (x64[rows] @ oracle.widen(A[a][g], kind).T)
            W2f[g * group:(g + 1) * group, r * a: r * (a + 1)] = oracle.widen(Bm[a][g], kind)
    dt = torch.float16 if kind == "f16" else torch.bfloat16
    Zd = torch.from_numpy(Zf).to(dt).cuda()
    W2d = torch.from_numpy(W2f).to(dt).cuda()
    z64 = Zd.double().cpu().numpy()  # the shrink as the kernel reads it (rounded to the storage type)
    Xd, Wd, bd = _dev(X, kind), _dev(W, kind), _dev(b, kind)
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    base = x64 @ oracle.widen(W, kind).T + oracle.widen(b, kind)
    delta_k = np.zeros((M, N))  # what the K2 tiles add, from the operands as given
    delta_o = np.zeros((M, N))  # the oracle's unmerged LoRA delta
    for g in range(3):
        if not (mask >> g) & 1:
            continue
        cols = slice(g * group, (g + 1) * group)
        delta_k[:, cols] = z64[:, g * K2:(g + 1) * K2] @ W2f[cols].T
        for a in range(n_slots):
            rows = slot == a
            delta_o[rows, cols] = oracle.lora_delta(x64[rows], oracle.widen(A[a][g], kind),
                                                    oracle.widen(Bm[a][g], kind), scale)
    # the expand is the LoRA delta up to the shrink's rounding to the storage type
    ulp = 2.0 ** -8 if kind == "bf16" else 2.0 ** -11
    assert np.max(np.abs(delta_k - delta_o)) <= 2 * ulp * np.max(np.abs(delta_o))
    ref = base + delta_k
    if epi == 2:
        R0 = synth.normal(81, 4, (M, N), 0.0, 1.0, "f32")
        R = torch.from_numpy(R0.copy()).cuda()
        pb.op_gemm_lora(DT[kind], 2, Xd, Wd, bd, Zd, K2, W2d, group, mask, R=R, workspace=ws)
        torch.cuda.synchronize()
        got = R.cpu().numpy().astype(np.float64)
        ref = ref + R0
        tol = 1e-5 * np.abs(ref).max() + 2e-5 * np.sqrt(K + K2)
    else:
        C = torch.empty((M, N), dtype=dt, device="cuda")
        pb.op_gemm_lora(DT[kind], 0, Xd, Wd, bd, Zd, K2, W2d, group, mask, C=C, qscale=0.125,
                        qcols=group, workspace=ws)
        torch.cuda.synchronize()
        got = _host_f64(C, kind)
        ref[:, :group] *= 0.125
        tol = ulp * np.abs(ref) + 1e-4
    err = np.abs(got - ref)
    assert np.all(err <= tol), "max err %.3e" % err.max()
    # k (mask bit clear) got no expand: equal to the plain product there
    kcols = slice(group, 2 * group)
    assert np.max(np.abs(delta_k[:, kcols])) == 0.0


def test_gemm_lora_rejects_bad_operands():
    import torch
    from paper_2503_17707_amd import binding as pb

    X = torch.zeros(8, 64, dtype=torch.float16, device="cuda")
    W = torch.zeros(512, 64, dtype=torch.float16, device="cuda")
    b = torch.zeros(512, dtype=torch.float16, device="cuda")
    C = torch.zeros(8, 512, dtype=torch.float16, device="cuda")
    Z = torch.zeros(8, 64, dtype=torch.float16, device="cuda")
    W2 = torch.zeros(512, 64, dtype=torch.float16, device="cuda")
    for group, zs in ((128, 0), (256, 64)):  # group not a multiple of 256; blocks past Z's row
        with pytest.raises(pb.PbError) as e:
            pb.op_gemm_lora(1, 1, X, W, b, Z, zs, W2, group, 0b11, C=C)
        assert e.value.code == pb.PB_EINVAL


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
