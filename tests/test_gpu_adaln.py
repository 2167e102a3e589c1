"""GPU parity of the INT4 round-to-nearest (group 64) AdaLN layer against the fp64 oracle: the
offline pass's codes and FP16 scales bit for bit (both sides form the same IEEE quotients), and
the layer's output within the relative Frobenius bar of the oracle's fp64 contraction on the
same codes and scales."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import GEMM_REL_F, log_stats, rel_frobenius, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _weights(N, K, seed, scale=0.02):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn((N, K), generator=g, device=DEV) * scale).to(torch.bfloat16)


def _check_pass(name, W):
    q, s = oq.adaln_int4_quantize_weights(W)
    torch.cuda.synchronize()
    oqq, osc = oracle.rtn_int4_quantize(to_f64(W))
    want_q = oracle.pack_rtn_int4(oqq)
    got_q = q.cpu().numpy()
    got_s = s.cpu().numpy().view(np.uint16)
    want_s = osc.astype(np.float16).view(np.uint16)
    bad_q, bad_s = int(np.sum(got_q != want_q)), int(np.sum(got_s != want_s))
    log_stats(name, N=W.shape[0], K=W.shape[1], code_byte_mismatches=bad_q, scale_mismatches=bad_s)
    assert bad_q == 0 and bad_s == 0
    return q, s, oqq, osc


@pytest.mark.parametrize("N,K", [(1, 64), (37, 128), (300, 3072), (129, 5120), (64, 16384)])
def test_weight_pass_bit_exact(N, K):
    _check_pass(f"adaln pass N={N} K={K}", _weights(N, K, seed=N + K))


def test_weight_pass_special_groups():
    K = 256
    W = torch.zeros((6, K), dtype=torch.float32)
    W[1, :8] = torch.tensor([3.5, -1.75, 0.25, 1.25, 0.75, -3.5, 0.0, 1.0])   # ties at 0.5 steps
    W[2] = torch.arange(K, dtype=torch.float32) % 15 - 7                      # on the grid, scale 1
    W[3] = 1e6                                                                # scale saturates
    W[4, 64:128] = 1e-7                                                       # scale underflows to 0
    W[5] = torch.linspace(-3, 3, K)
    _check_pass("adaln pass special groups", W.to(torch.bfloat16).to(DEV))


def test_weight_pass_strided_rows():
    base = _weights(50, 3072 + 64, seed=3)
    _check_pass("adaln pass strided", base[:, 32:32 + 3072])


@pytest.mark.parametrize("M", [1, 2, 3, 5])
@pytest.mark.parametrize("N,K", [(1, 64), (31, 128), (33, 3072), (1000, 3072), (257, 5120), (70, 16384)])
@pytest.mark.parametrize("bias", [False, True])
def test_linear(M, N, K, bias):
    W = _weights(N, K, seed=M + N + K)
    q, s, oqq, osc = _check_pass(f"adaln pass N={N} K={K}", W)
    X = workloads.adaln_tokens(M, K, seed=M + K, device=DEV)
    b = (torch.randn(N, generator=torch.Generator().manual_seed(N)) * 0.1).to(torch.bfloat16) if bias else None
    Y = oq.adaln_int4_linear(X, q, s, bias=b.to(DEV) if bias else None)
    torch.cuda.synchronize()
    ref = oracle.rtn_int4_linear(to_f64(X), oqq, osc, bias=b.double().numpy() if bias else None)
    err = rel_frobenius(Y.double().cpu().numpy(), ref)
    log_stats(f"adaln linear M={M} N={N} K={K} bias={bias}", rel_f=err)
    assert err <= GEMM_REL_F


def test_linear_strided_input_and_padded_output():
    M, N, K = 3, 100, 3072
    W = _weights(N, K, seed=11)
    q, s, oqq, osc = _check_pass("adaln pass", W)
    X = workloads.adaln_tokens(M, K + 64, seed=5, device=DEV)[:, 64:]
    out = torch.full((M, N + 3), float("nan"), device=DEV)[:, :N]
    Y = oq.adaln_int4_linear(X, q, s, out=out)
    torch.cuda.synchronize()
    ref = oracle.rtn_int4_linear(to_f64(X), oqq, osc)
    assert rel_frobenius(Y.double().cpu().numpy(), ref) <= GEMM_REL_F
    assert not torch.isnan(out).any()


@pytest.mark.parametrize("N", [18432, 9216])
def test_flux_shaped_projection(N):
    # the benchmark's layer shapes: one conditioning token, 3072 -> 6 x 3072 and 3 x 3072
    W = workloads.adaln_weights(N, 0, device=DEV)
    q, s, oqq, osc = _check_pass(f"adaln pass flux N={N}", W)
    X = workloads.adaln_tokens(1, device=DEV)
    Y = oq.adaln_int4_linear(X, q, s)
    torch.cuda.synchronize()
    ref = oracle.rtn_int4_linear(to_f64(X), oqq, osc)
    err = rel_frobenius(Y.double().cpu().numpy(), ref)
    dense = to_f64(X) @ to_f64(W).T
    log_stats(f"adaln linear flux N={N}", rel_f=err, rel_f_vs_bf16_weights=rel_frobenius(Y.double().cpu().numpy(), dense))
    assert err <= GEMM_REL_F


def test_empty_is_noop():
    q = torch.zeros((0, 32), dtype=torch.uint8, device=DEV)
    s = torch.zeros((0, 1), dtype=torch.float16, device=DEV)
    X = torch.zeros((2, 64), dtype=torch.bfloat16, device=DEV)
    assert oq.adaln_int4_linear(X, q, s).shape == (2, 0)
    assert oq.adaln_int4_linear(X[:0], torch.zeros((4, 32), dtype=torch.uint8, device=DEV),
                                torch.zeros((4, 1), dtype=torch.float16, device=DEV)).shape == (0, 4)
