"""pb_op_gemm_noalloc: the projection GEMM with its split-K partials in the
library's own device scratch instead of a caller workspace.  It must give
exactly what pb_op_gemm gives with a workspace of the scratch's size, over
consecutive calls on the shared scratch (the second one smaller), and reject
products whose fp32 output exceeds the scratch."""
import numpy as np
import pytest

from gpu_common import log

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20

# (dtype, epilogue, M, N, K): an fc2-like product that splits K (its partials
# fill the scratch several times over 4 MiB), then smaller ones with a ragged M
CASES = [
    (1, 2, 512, 2048, 8192),
    (1, 0, 136, 1024, 2048),
    (0, 1, 77, 512, 1024),
]


def _operands(torch, dtype, epi, M, N, K, seed):
    g = torch.Generator(device="cuda:0").manual_seed(seed)
    dt = torch.float16 if dtype == 1 else torch.bfloat16
    X = torch.randn(M, K, device="cuda:0", generator=g).to(dt)
    W = (torch.randn(N, K, device="cuda:0", generator=g) * 0.02).to(dt)
    b = (torch.randn(N, device="cuda:0", generator=g) * 0.02).to(dt)
    R0 = torch.randn(M, N, device="cuda:0", generator=g) if epi == 2 else None
    return X, W, b, R0


def _run(pb, torch, fn, dtype, epi, X, W, b, R0, M, N, qscale, qcols, **kw):
    dt = X.dtype
    C = torch.full((M, N), float("nan"), dtype=dt, device="cuda:0") if epi != 2 else None
    R = R0.clone() if epi == 2 else None
    fn(dtype, epi, X, W, b, C=C, R=R, qscale=qscale, qcols=qcols, **kw)
    torch.cuda.synchronize()
    out = R if epi == 2 else C
    return out.float().cpu().numpy()


def test_noalloc_gemm_equals_workspace_gemm_on_consecutive_calls():
    import torch
    from paper_2503_17707_amd import binding as pb

    ws = torch.empty(SCRATCH_BYTES, dtype=torch.uint8, device="cuda:0")
    for i, (dtype, epi, M, N, K) in enumerate(CASES):
        log("case noalloc gemm dtype=%d epi=%d M=%d N=%d K=%d" % (dtype, epi, M, N, K))
        X, W, b, R0 = _operands(torch, dtype, epi, M, N, K, 100 + i)
        qscale, qcols = (0.125, N // 3) if epi == 0 else (1.0, 0)
        got = _run(pb, torch, pb.op_gemm_noalloc, dtype, epi, X, W, b, R0, M, N, qscale, qcols)
        ref = _run(pb, torch, pb.op_gemm, dtype, epi, X, W, b, R0, M, N, qscale, qcols, workspace=ws)
        assert np.all(np.isfinite(got))
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), "case %d differs" % i
        # and the product itself, against float64 on the host
        y = (X.double().cpu().numpy() @ W.double().cpu().numpy().T + b.double().cpu().numpy())
        if epi == 0:
            y[:, :qcols] *= qscale
        elif epi == 1:
            y = np.maximum(y, 0.0)
        else:
            y = y + R0.double().cpu().numpy()
        err = np.max(np.abs(got - y)) / max(1.0, np.max(np.abs(y)))
        log("  bit-identical to pb_op_gemm; max rel err vs float64 %.2e" % err)
        assert err < 1e-2


def test_noalloc_gemm_rejects_products_beyond_the_scratch():
    import torch
    from paper_2503_17707_amd import binding as pb

    M, N, K = 4096, 4160, 64  # M*N*4 just over 64 MiB: rejected before any launch
    X = torch.zeros(M, K, dtype=torch.float16, device="cuda:0")
    W = torch.zeros(N, K, dtype=torch.float16, device="cuda:0")
    b = torch.zeros(N, dtype=torch.float16, device="cuda:0")
    C = torch.zeros(M, N, dtype=torch.float16, device="cuda:0")
    with pytest.raises(pb.PbError) as e:
        pb.op_gemm_noalloc(1, 1, X, W, b, C=C)
    assert e.value.code == pb.PB_EINVAL
    assert "scratch" in str(e.value)
