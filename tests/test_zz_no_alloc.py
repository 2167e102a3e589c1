"""The allocation-free layer, orbit_qlinear_noalloc, through the C ABI: the K-split's partial sums go
to the library's own scratch array instead of a caller workspace, so the result must be the bits of
orbit_qlinear_ws given a workspace of the size it asks for.  Two calls in a row, the second on a
smaller layer with the first call's partial sums still in the scratch array; both also against the
fp64 oracle contraction on the same codes (the per-element and relative Frobenius bars)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import check_gemm, gemm_scale, qlinear_oracle_bf16

pytestmark = pytest.mark.gpu

DEV = "cuda"
SCRATCH_BYTES = 32 << 20


def _operands(M, N, K, ba, bw, seed):
    xc = workloads.random_codes(M, K, ba, seed)
    wc = workloads.random_codes(N, K, bw, seed + 1)
    xs = workloads.random_norms(M, seed, 0)
    wr = workloads.random_norms(N, seed, 1).to(torch.bfloat16)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    dev = (torch.from_numpy(oracle.pack_codes(oracle.to_labels(xc.numpy(), ba), ba)).to(DEV), xs.to(DEV),
           torch.from_numpy(oracle.pack_codes(oracle.to_labels(wc.numpy(), bw), bw)).to(DEV), wr.to(DEV))
    return (xc, xs, wc, wr), (cba, cbw), dev


def _oracle_check(name, Y, host, ba, bw, K):
    xc, xs, wc, wr = host
    args = (xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
    la = oracle.bf16_round(oracle.lloydmax_codebook(ba, K).levels)
    lw = oracle.bf16_round(oracle.lloydmax_codebook(bw, K).levels)
    check_gemm(name, Y.cpu().numpy().astype(np.float64), qlinear_oracle_bf16(*args),
               gemm_scale(args[0], args[1], la, args[3], args[4], lw), K)


def test_two_calls_in_a_row_match_the_workspace_layer():
    # c1's layer (256 x 3072 -> 3072, split over K), then a smaller split layer
    for M, N, K, ba, bw, seed in ((256, 3072, 3072, 4, 4, 1), (40, 700, 1024, 4, 3, 2)):
        host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, ba, bw, seed)
        n = oq.orbit_qlinear_workspace_size(M, N, K)
        assert 0 < n <= SCRATCH_BYTES
        ws = torch.full((n // 4,), float("nan"), dtype=torch.float32, device=DEV)
        Y_ws = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
        out = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
        Y = oq.orbit_qlinear_noalloc(cba, xp, xs, cbw, wp, wr, out=out)
        torch.cuda.synchronize()
        assert Y.data_ptr() == out.data_ptr()
        assert torch.equal(Y, Y_ws), f"M={M} N={N} K={K}: differs from orbit_qlinear_ws"
        _oracle_check(f"noalloc M={M} N={N} K={K} W{bw}A{ba}", Y, host, ba, bw, K)


def test_fused_epilogue_and_unsplit_layers():
    # bias + GELU + bf16 output on a split layer; a layer that fills the device (no split, no
    # scratch) gives orbit_qlinear_ex's bits
    M, N, K = 200, 390, 2048
    _, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, 4, 4, 11)
    bias = (torch.randn(N, device=DEV) * 0.1).to(torch.bfloat16)
    n = oq.orbit_qlinear_workspace_size(M, N, K)
    assert 0 < n <= SCRATCH_BYTES
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    a = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws, bias=bias, gelu=True, out_dtype=torch.bfloat16)
    b = oq.orbit_qlinear_noalloc(cba, xp, xs, cbw, wp, wr, bias=bias, gelu=True, out_dtype=torch.bfloat16)
    Mb, Nb, Kb = 4133, 8061, 192
    assert oq.orbit_qlinear_workspace_size(Mb, Nb, Kb) == 0
    _, (cba2, cbw2), (xp2, xs2, wp2, wr2) = _operands(Mb, Nb, Kb, 4, 3, 12)
    c = oq.orbit_qlinear_ex(cba2, xp2, xs2, cbw2, wp2, wr2)
    d = oq.orbit_qlinear_noalloc(cba2, xp2, xs2, cbw2, wp2, wr2)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(c, d)


def test_layer_beyond_the_scratch_limit_is_refused():
    # a small grid with a long contraction splits into more partial sums than the scratch holds
    K = 8192
    shapes = [(256, 12288), (200, 12288), (300, 8192), (128, 24576)]
    big = [(M, N) for M, N in shapes if oq.orbit_qlinear_workspace_size(M, N, K) > SCRATCH_BYTES]
    assert big, "no test shape needs more than the scratch limit"
    M, N = big[0]
    cb = oq.lloydmax_codebook(4, K)
    xp = torch.zeros((M, K // 2), dtype=torch.uint8, device=DEV)
    xs = torch.ones(M, device=DEV)
    wp = torch.zeros((N, K // 2), dtype=torch.uint8, device=DEV)
    wr = torch.ones(N, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(oq.OrbitError) as err:
        oq.orbit_qlinear_noalloc(cb, xp, xs, cb, wp, wr)
    assert err.value.status == oq.ORBIT_EUNSUPPORTED
    assert "scratch limit" in str(err.value)
