"""GPU parity of the K-split quantized layer (orbit_qlinear_ws with a caller workspace) against
the fp64 oracle contraction, and against the unsplit layer on the same codes.  The split only
regroups the fp32 sum over K, so the oracle bar of the unsplit kernel applies unchanged, and
the two layers agree to fp32 accumulation error.  Codes and norms come from the seeded
generator, never from the HIP path."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import GEMM_REL_F, check_gemm, gemm_scale, log_stats, qlinear_oracle_bf16, rel_frobenius

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _operands(M, N, K, ba, bw, seed):
    xc = workloads.random_codes(M, K, ba, seed)
    wc = workloads.random_codes(N, K, bw, seed + 1)
    xs = workloads.random_norms(M, seed, 0)
    wr = workloads.random_norms(N, seed, 1).to(torch.bfloat16)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    dev = (torch.from_numpy(oracle.pack_codes(oracle.to_labels(xc.numpy(), ba), ba)).to(DEV), xs.to(DEV),
           torch.from_numpy(oracle.pack_codes(oracle.to_labels(wc.numpy(), bw), bw)).to(DEV), wr.to(DEV))
    return (xc, xs, wc, wr), (cba, cbw), dev


def _scale(xc, xs, ba, wc, wr, bw, K):
    """Per-element unit s_n r'_i ||a_n|| ||b_i|| on the oracle's bf16 levels."""
    la = oracle.bf16_round(oracle.lloydmax_codebook(ba, K).levels)
    lw = oracle.bf16_round(oracle.lloydmax_codebook(bw, K).levels)
    return gemm_scale(xc, xs, la, wc, wr, lw)


def _workspace(M, N, K, fill=float("nan")):
    n = oq.orbit_qlinear_workspace_size(M, N, K)
    # stale contents must not matter: every partial sum is written before it is read
    return n, torch.full((max(n, 4) // 4,), fill, dtype=torch.float32, device=DEV)


def _splits(M, N, K, n):
    assert n % (M * N * 4) == 0
    return n // (M * N * 4)


# Ragged M and N, one token, c1's layer (256 x 3072 x 3072).  On 256 compute units the split
# lengths (K-steps per split, then the last split's: 5/4, 10/8, 6/6, 5/3, 4/4, 8/1, 7/1, 5/2 and
# 6/3) cover each remainder of the kernel's 6-set code ring, with and without a full round.
@pytest.mark.parametrize("M,N,K", [(300, 130, 1216), (256, 3072, 3072), (129, 257, 13824), (1, 3072, 3072),
                                   (64, 1000, 4096), (200, 1000, 7232), (200, 1000, 6336), (1, 96, 1088),
                                   (200, 1000, 5184)])
@pytest.mark.parametrize("ba,bw", [(4, 4), (4, 3), (2, 2), (3, 4), (6, 4), (6, 2)])
def test_split_matches_oracle_and_unsplit(M, N, K, ba, bw):
    host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, ba, bw, seed=M + N + K + ba)
    n, ws = _workspace(M, N, K)
    S = _splits(M, N, K, n)
    assert 2 <= S <= K // 256
    Y = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
    Y0 = oq.orbit_qlinear(cba, xp, xs, cbw, wp, wr)
    torch.cuda.synchronize()
    Y, Y0 = Y.cpu().numpy().astype(np.float64), Y0.cpu().numpy().astype(np.float64)
    xc, xsh, wc, wrh = host
    args = (xc.numpy(), xsh.double().numpy(), ba, wc.numpy(), wrh.double().numpy(), bw, K)
    ref = qlinear_oracle_bf16(*args)
    err0, d = rel_frobenius(Y0, ref), rel_frobenius(Y, Y0)
    check_gemm(f"split M={M} N={N} K={K} W{bw}A{ba} splits={S}", Y, ref, _scale(*args), K, rel_f_unsplit=err0,
               vs_unsplit=d)
    assert d <= 1e-5


# Grids of a large tile per compute unit or more whose last round of large tiles would be mostly
# empty: the large kernel takes the rows of its full rounds and the 128x128 kernel the rest (37
# and 517 rows on 256 compute units), split over K with the workspace.  Sampled rows from both
# parts against the oracle, every output against the unsplit layer.
@pytest.mark.parametrize("M,N,K", [(4133, 8061, 1024), (8197, 4099, 4096)])
def test_split_tail_of_large_grid(M, N, K):
    ba, bw = 4, 3
    host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, ba, bw, seed=M + K)
    n, ws = _workspace(M, N, K)
    assert 0 < n < M * N * 4            # partial sums for the tail rows only
    Y = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
    Y0 = oq.orbit_qlinear(cba, xp, xs, cbw, wp, wr)
    torch.cuda.synchronize()
    Y, Y0 = Y.cpu().numpy().astype(np.float64), Y0.cpu().numpy().astype(np.float64)
    rows = np.unique(np.concatenate([np.random.default_rng(K).choice(M, 48, replace=False),
                                     np.arange(M - 16, M)]))
    xc, xsh, wc, wrh = host
    args = (xc.numpy()[rows], xsh.double().numpy()[rows], ba, wc.numpy(), wrh.double().numpy(), bw, K)
    d = rel_frobenius(Y, Y0)
    check_gemm(f"split tail M={M} N={N} K={K} workspace={n}", Y[rows], qlinear_oracle_bf16(*args), _scale(*args), K,
               vs_unsplit=d)
    assert d <= 1e-5


# every bit-width pair the GEMM implements, on c1's layer and a ragged one
@pytest.mark.parametrize("M,N,K", [(256, 3072, 3072), (33, 200, 2048)])
@pytest.mark.parametrize("ba,bw", [(3, 3), (3, 2), (2, 3), (2, 4), (4, 2), (6, 3)])
def test_split_remaining_bit_pairs(M, N, K, ba, bw):
    host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, ba, bw, seed=2 * M + N + ba * 8 + bw)
    n, ws = _workspace(M, N, K)
    assert _splits(M, N, K, n) >= 2
    Y = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
    torch.cuda.synchronize()
    xc, xsh, wc, wrh = host
    args = (xc.numpy(), xsh.double().numpy(), ba, wc.numpy(), wrh.double().numpy(), bw, K)
    check_gemm(f"split bits M={M} N={N} K={K} W{bw}A{ba}", Y.cpu().numpy().astype(np.float64),
               qlinear_oracle_bf16(*args), _scale(*args), K)


@pytest.mark.parametrize("bias,gelu,bf16", [(True, False, False), (False, True, False), (False, False, True),
                                            (True, True, True)])
@pytest.mark.parametrize("pad", [0, 1])
@pytest.mark.parametrize("N", [390, 392])   # 392 with pad 0: the partial sums and Y through LDS
def test_split_fused_epilogue(bias, gelu, bf16, pad, N):
    M, K, ba, bw = 200, 2048, 4, 4
    host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, ba, bw, seed=11)
    n, ws = _workspace(M, N, K)
    assert _splits(M, N, K, n) >= 2
    g = torch.Generator()
    g.manual_seed(N)
    b = torch.randn(N, generator=g).to(torch.bfloat16) if bias else None
    dt = torch.bfloat16 if bf16 else torch.float32
    out = torch.full((M, N + pad), float("nan"), dtype=dt, device=DEV)[:, :N]
    Y = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws, bias=b.to(DEV) if bias else None, gelu=gelu,
                            out_dtype=dt, out=out)
    torch.cuda.synchronize()
    Yn = Y.float().cpu().numpy().astype(np.float64)
    xc, xsh, wc, wrh = host
    base = qlinear_oracle_bf16(xc.numpy(), xsh.double().numpy(), ba, wc.numpy(), wrh.double().numpy(), bw, K)
    bd = b.double().numpy() if bias else None
    ref = oracle.layer_epilogue(base, bias=bd, gelu=gelu)
    if bf16:
        # one bf16 ulp of the fp64 layer plus an absolute slack of 1e-5 of the largest output,
        # and mostly exactly its rounding (as for the unsplit layer)
        rb = oracle.layer_epilogue(base, bias=bd, gelu=gelu, out_bf16=True)
        ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(ref), 1e-30))[1] - 8)
        assert not (np.abs(Yn - ref) > ulp + 1e-5 * np.max(np.abs(ref))).any()
        assert np.mean(Yn == rb) > 0.999
        ref = rb
    else:
        # fp32 outputs: the per-element bar through GELU's slope (below 1.13) plus the epilogue's
        # own roundings
        scale = _scale(xc.numpy(), xsh.double().numpy(), ba, wc.numpy(), wrh.double().numpy(), bw, K)
        pre = np.abs(base) + (np.abs(bd)[None, :] if bias else 0.0)
        check_gemm(f"split epilogue fp32 bias={bias} gelu={gelu} pad={pad}", Yn, ref, 1.13 * scale if gelu else scale,
                   K, slack=1e-6 * pre)
    err = rel_frobenius(Yn, ref)
    log_stats(f"split epilogue bias={bias} gelu={gelu} bf16={bf16} pad={pad}", rel_f=err)
    assert err <= GEMM_REL_F
    if pad:
        assert torch.isnan(out.float()).sum() == 0


def test_split_is_deterministic_and_ignores_stale_workspace():
    M, N, K = 256, 3072, 3072
    _, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, 4, 4, seed=5)
    n, ws = _workspace(M, N, K)
    Y1 = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
    ws.fill_(1e30)
    Y2 = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2)


def test_workspace_reused_across_shapes():
    # one workspace for two layers in a row on the stream, the second smaller
    big, small = (256, 3072, 3072), (40, 700, 1024)
    n = max(oq.orbit_qlinear_workspace_size(*big), oq.orbit_qlinear_workspace_size(*small))
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    outs = []
    for (M, N, K), seed in ((big, 1), (small, 2)):
        host, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, 4, 3, seed=seed)
        outs.append((host, K, oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, ws)))
    torch.cuda.synchronize()
    for (xc, xsh, wc, wrh), K, Y in outs:
        args = (xc.numpy(), xsh.double().numpy(), 4, wc.numpy(), wrh.double().numpy(), 3, K)
        check_gemm(f"split workspace reuse K={K}", Y.cpu().numpy().astype(np.float64), qlinear_oracle_bf16(*args),
                   _scale(*args), K)


def test_small_or_missing_workspace_runs_unsplit():
    # too small a workspace (or a layer that does not split) gives orbit_qlinear_ex's bits
    M, N, K = 256, 3072, 3072
    _, (cba, cbw), (xp, xs, wp, wr) = _operands(M, N, K, 4, 4, seed=3)
    n = oq.orbit_qlinear_workspace_size(M, N, K)
    short = torch.empty(n - 4, dtype=torch.uint8, device=DEV)
    Y0 = oq.orbit_qlinear_ex(cba, xp, xs, cbw, wp, wr)
    Y1 = oq.orbit_qlinear_ws(cba, xp, xs, cbw, wp, wr, short)
    # a layer that fills the device (no split): zero bytes asked, the same bits as the unsplit call
    Mb, Nb, Kb = 4133, 8061, 192
    assert oq.orbit_qlinear_workspace_size(Mb, Nb, Kb) == 0
    _, (cba2, cbw2), (xp2, xs2, wp2, wr2) = _operands(Mb, Nb, Kb, 4, 3, seed=4)
    Yb0 = oq.orbit_qlinear(cba2, xp2, xs2, cbw2, wp2, wr2)
    Yb1 = oq.orbit_qlinear_ws(cba2, xp2, xs2, cbw2, wp2, wr2, torch.empty(1 << 20, dtype=torch.uint8, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(Y0, Y1)
    assert torch.equal(Yb0, Yb1)


def test_workspace_size_rules():
    # too short a contraction (under 8 K-steps) never splits; a small grid with a long one does
    assert oq.orbit_qlinear_workspace_size(256, 3072, 448) == 0
    assert oq.orbit_qlinear_workspace_size(0, 3072, 3072) == 0
    n = oq.orbit_qlinear_workspace_size(1, 128, 65536)
    assert _splits(1, 128, 65536, n) >= 2


def test_schedule_matches_the_workspace_size():
    # the schedule query names the rows each kernel runs and the split count; the workspace size
    # follows from it (splits x rows on the 128 x 128 kernel x N x 4 bytes when it splits)
    cases = [(256, 3072, 3072), (workloads.C4_M, 5120, 13824), (workloads.C4_M, 13824, 5120), (4133, 8061, 192),
             (1, 3072, 3072)]
    for M, N, K in cases:
        rows, splits = oq.orbit_qlinear_schedule(M, N, K)
        assert 0 <= rows <= M and splits >= 1
        want = splits * (M - rows) * N * 4 if splits > 1 else 0
        assert oq.orbit_qlinear_workspace_size(M, N, K) == want
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        # on 256 compute units: c1 all on the small kernel, five splits; c4's up-projection all on
        # the large one; its down-projection 32768 rows (ten full rounds) large, 504 split three ways
        assert oq.orbit_qlinear_schedule(256, 3072, 3072) == (0, 5)
        assert oq.orbit_qlinear_schedule(workloads.C4_M, 13824, 5120) == (workloads.C4_M, 1)
        assert oq.orbit_qlinear_schedule(workloads.C4_M, 5120, 13824) == (32768, 3)
