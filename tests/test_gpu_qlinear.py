"""GPU parity of the LUT-decode GEMM against the fp64 oracle contraction with identical codes
and identical (bf16-rounded) levels: relative Frobenius error <= 2e-3 (fp32 accumulation
leaves ~1e-6).  Codes and norms come from the seeded generator or from the oracle, never
from the HIP path."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import (GEMM_REL_F, check_gemm, gemm_scale, log_stats, near_tie_flip_bound, qlinear_oracle_bf16,
                            rel_frobenius, to_f64)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _inputs(M, N, K, ba, bw, seed):
    xc = workloads.random_codes(M, K, ba, seed)
    wc = workloads.random_codes(N, K, bw, seed + 1)
    xs = workloads.random_norms(M, seed, 0)
    wr = workloads.random_norms(N, seed, 1).to(torch.bfloat16)
    return xc, xs, wc, wr


def _scale(xc, xs, ba, wc, wr, bw, K):
    """Per-element unit s_n r'_i ||a_n|| ||b_i|| on the oracle's bf16 levels."""
    la = oracle.bf16_round(oracle.lloydmax_codebook(ba, K).levels)
    lw = oracle.bf16_round(oracle.lloydmax_codebook(bw, K).levels)
    return gemm_scale(xc, xs, la, wc, wr, lw)


def _gpu(xc, xs, wc, wr, ba, bw, K):
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    xp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(xc.numpy(), ba), ba)).to(DEV)
    wp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(wc.numpy(), bw), bw)).to(DEV)
    Y = oq.orbit_qlinear(cba, xp, xs.to(DEV), cbw, wp, wr.to(DEV))
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


# the 128 x 128 kernel keeps the codes of 5 K-steps in flight in 6 register sets: step counts 1, 2,
# 3, 4, 5, 7, 8, 9, 48, 216 cover no full round of that ring, whole rounds and each remainder
@pytest.mark.parametrize("M,N,K", [(1, 128, 64), (257, 384, 256), (300, 130, 512), (64, 3072, 3072),
                                   (129, 257, 13824), (5, 1, 128), (70, 96, 320), (33, 200, 448),
                                   (40, 200, 192), (40, 200, 576)])
@pytest.mark.parametrize("ba,bw", [(4, 4), (4, 3), (4, 2), (3, 3), (2, 2), (3, 4), (2, 4), (6, 4), (6, 3), (6, 2)])
def test_random_codes(M, N, K, ba, bw):
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=M + N + K)
    Y = _gpu(xc, xs, wc, wr, ba, bw, K)
    args = (xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
    check_gemm(f"gemm random M={M} N={N} K={K} W{bw}A{ba}", Y, qlinear_oracle_bf16(*args), _scale(*args), K)


# shapes with at least one 256x256 tile per compute unit (256) run the large-tile kernel; these
# cover its ragged edges in M and N, a single K-step, an odd number of K-steps and a grid of
# under two tiles per compute unit (289).  On 256 compute units the first four leave a last round
# that is mostly empty, so the large kernel takes the rows of its full rounds and the 128x128
# kernel the rest (shifted operands and output, ragged in M and N); 3900 x 8000 fills exactly two
# rounds (16 x 32 tiles) and runs the large kernel alone, ragged in both.
# K-step counts 1, 2, 3, 4, 5, 16 cover the large kernel's three-set code ring: no full round, whole
# rounds, and each length of the remainder
@pytest.mark.parametrize("M,N,K", [(4133, 8061, 64), (4133, 8061, 128), (4133, 8061, 192), (4133, 8061, 256),
                                   (8197, 4099, 1024), (4133, 4099, 320), (3900, 8000, 192)])
@pytest.mark.parametrize("ba,bw", [(4, 4), (4, 3), (2, 2), (3, 4), (6, 4), (6, 2)])
def test_random_codes_large_tiles(M, N, K, ba, bw):
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=M + N + K)
    Y = _gpu(xc, xs, wc, wr, ba, bw, K)
    args = (xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
    ref = qlinear_oracle_bf16(*args)
    worst_row = float(np.max(np.linalg.norm(Y - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-300)))
    check_gemm(f"gemm large-tile M={M} N={N} K={K} W{bw}A{ba}", Y, ref, _scale(*args), K, worst_row_rel=worst_row)
    assert worst_row <= GEMM_REL_F


# the fused layer epilogue (bias, GELU, bf16 output) on both kernels, with vector and element-wise
# stores (ldy a multiple of 4 or not); with N and ldy multiples of 4 the outputs go through the
# kernels' LDS turn-around
@pytest.mark.parametrize("M,N,K", [(300, 130, 512), (4133, 8061, 192), (300, 132, 512), (4133, 8064, 192)])
@pytest.mark.parametrize("bias,gelu,bf16", [(True, False, False), (False, True, False), (False, False, True),
                                            (True, True, True)])
@pytest.mark.parametrize("pad", [0, 1])
def test_fused_epilogue(M, N, K, bias, gelu, bf16, pad):
    ba, bw = 4, 4 if M < 1000 else 3
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=M + N + K + 7)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    xp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(xc.numpy(), ba), ba)).to(DEV)
    wp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(wc.numpy(), bw), bw)).to(DEV)
    g = torch.Generator()
    g.manual_seed(N)
    b = torch.randn(N, generator=g).to(torch.bfloat16) if bias else None
    dt = torch.bfloat16 if bf16 else torch.float32
    out = torch.full((M, N + pad), float("nan"), dtype=dt, device=DEV)[:, :N]
    Y = oq.orbit_qlinear_ex(cba, xp, xs.to(DEV), cbw, wp, wr.to(DEV), bias=b.to(DEV) if bias else None,
                            gelu=gelu, out_dtype=dt, out=out)
    torch.cuda.synchronize()
    Yn = Y.float().cpu().numpy().astype(np.float64)
    base = qlinear_oracle_bf16(xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
    ref = oracle.layer_epilogue(base, bias=b.double().numpy() if bias else None, gelu=gelu)
    err = rel_frobenius(Yn, ref)
    stats = {"rel_f": err}
    if not bf16:
        # fp32 outputs: the contraction's per-element bar, carried through GELU (slope below 1.13),
        # plus the epilogue's own roundings (the rescale, the bias add, the erfc form's 1.2e-7)
        scale = _scale(xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
        pre = np.abs(base) + (np.abs(b.double().numpy())[None, :] if bias else 0.0)
        check_gemm(f"fused epilogue fp32 M={M} N={N} K={K} bias={bias} gelu={gelu} pad={pad}", Yn, ref,
                   1.13 * scale if gelu else scale, K, slack=1e-6 * pre)
    if bf16:
        # every bf16 output is the rounding of a value within the fp32 accumulation error of the
        # fp64 result: at most one bf16 ulp from it, plus an absolute slack of 1e-5 of the
        # largest output for values that cancel to almost nothing; mostly exactly the rounding
        rb = oracle.layer_epilogue(base, bias=b.double().numpy() if bias else None, gelu=gelu, out_bf16=True)
        ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(ref), 1e-30))[1] - 8)
        far = np.abs(Yn - ref) > ulp + 1e-5 * np.max(np.abs(ref))
        stats.update(equal_to_rounding=float(np.mean(Yn == rb)), beyond=int(far.sum()),
                     rel_f_vs_rounded=rel_frobenius(Yn, rb))
        assert not far.any()
        assert np.mean(Yn == rb) > 0.999
        # bf16 output alone carries ~1.7e-3 of rounding (8 significant bits); the bar applies to
        # the kernel's difference from the correctly rounded layer
        err = rel_frobenius(Yn, rb)
    log_stats(f"fused epilogue M={M} N={N} K={K} bias={bias} gelu={gelu} bf16={bf16} pad={pad}", **stats)
    assert err <= GEMM_REL_F
    if pad:
        assert torch.isnan(out.float()).sum() == 0      # every valid element written


def test_constant_codes_closed_form():
    M, N, K = 70, 200, 1024
    cba, cbw = oq.lloydmax_codebook(4, K), oq.lloydmax_codebook(3, K)
    xc = torch.full((M, K), 13, dtype=torch.int64)
    wc = torch.full((N, K), 2, dtype=torch.int64)
    xs = workloads.random_norms(M, 3, 0)
    wr = workloads.random_norms(N, 3, 1).to(torch.bfloat16)
    Y = _gpu(xc, xs, wc, wr, 4, 3, K)
    la = (cba.lut_bf16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    lw = (cbw.lut_bf16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    want = xs.double().numpy()[:, None] * wr.double().numpy()[None, :] * K * la[13] * lw[2]
    assert np.max(np.abs(Y - want) / np.abs(want)) < 1e-5


def test_c4_up_shape_sampled_rows():
    # the video-DiT up-projection at full size in the benchmark's launch configuration
    M, N, K = workloads.C4_M, 13824, 5120
    g = torch.Generator(device=DEV)
    g.manual_seed(4)
    xc = torch.randint(0, 16, (M, K), generator=g, device=DEV, dtype=torch.int64)
    wc = torch.randint(0, 16, (N, K), generator=g, device=DEV, dtype=torch.int64)
    xs = workloads.random_norms(M, 4, 0, device=DEV)
    wr = workloads.random_norms(N, 4, 1, device=DEV).to(torch.bfloat16)
    # store on the device with plain torch ops (sign-magnitude labels of the level indices in
    # LSB-first nibbles), outside the HIP path
    xl, wl = (torch.where(c >= 8, c - 8, 15 - c) for c in (xc, wc))
    xp = (xl[:, 0::2] | (xl[:, 1::2] << 4)).to(torch.uint8)
    wp = (wl[:, 0::2] | (wl[:, 1::2] << 4)).to(torch.uint8)
    cb = oq.lloydmax_codebook(4, K)
    Y = oq.orbit_qlinear(cb, xp, xs, cb, wp, wr)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(46).choice(M, 256, replace=False))
    rows[-1] = M - 1
    ridx = torch.as_tensor(rows, device=DEV)
    ref = qlinear_oracle_bf16(xc[ridx].cpu().numpy(), xs[ridx].double().cpu().numpy(), 4,
                              wc.cpu().numpy(), wr.double().cpu().numpy(), 4, K)
    la = oracle.bf16_round(oracle.lloydmax_codebook(4, K).levels)
    scale = gemm_scale(xc[ridx].cpu().numpy(), xs[ridx].double().cpu().numpy(), la, wc.cpu().numpy(),
                       wr.double().cpu().numpy(), la)
    check_gemm("gemm c4 up sampled", Y[ridx].double().cpu().numpy(), ref, scale, K, rows=len(rows))


@pytest.mark.parametrize("bw,ba", [(4, 4), (3, 4), (2, 4), (3, 3), (4, 6)])
def test_end_to_end_c1(bw, ba):
    """GPU quantize (acts + weights) -> GPU GEMM against the oracle pipeline on the same bf16
    inputs.  Codes may differ only at near-ties, so the outputs must agree to within the bound on
    what flipping every near-tie code could change (computed from the oracle alone) plus fp32
    accumulation; the layer error against X W^T sits in the sqrt(D_w + D_a) band."""
    X, W = workloads.c1_inputs(device=DEV)
    K = X.shape[1]
    plan = oq.rpbh_plan(K, 128, 0)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    wcodes, wnorm = oq.quantize_weights_offline(plan, cbw, W)
    xcodes, xnorm = oq.rpbh_quantize_act(plan, cba, X)
    Y = oq.orbit_qlinear(cba, xcodes, xnorm, cbw, wcodes, wnorm)
    torch.cuda.synchronize()
    Xd, Wd = to_f64(X), to_f64(W)
    oplan = oracle.rpbh_plan(K, 128, 0)
    oca, ocw = oracle.lloydmax_codebook(ba, K), oracle.lloydmax_codebook(bw, K)
    cx, s, Ux = oracle.quantize_act(Xd, oplan, oca)
    cw, r, Uw = oracle.quantize_weights(Wd, oplan, ocw)
    la, lw = oracle.bf16_round(oca.levels), oracle.bf16_round(ocw.levels)
    ref_q = oracle.qlinear(cx, s, la, cw, r, lw)
    dense = oracle.qlinear_dense_reference(Xd, Wd)
    Yn = Y.cpu().numpy().astype(np.float64)
    bound = near_tie_flip_bound(cx, s, Ux, la, oca.thresholds, cw, r, Uw, lw, ocw.thresholds)
    diff = float(np.linalg.norm(Yn - ref_q))
    e_pipe = rel_frobenius(Yn, ref_q)
    e_dense = rel_frobenius(Yn, dense)
    log_stats(f"end-to-end c1 W{bw}A{ba}", rel_f_vs_oracle_pipeline=e_pipe, rel_f_vs_dense=e_dense,
              near_tie_bound_rel=bound / float(np.linalg.norm(ref_q)))
    assert diff <= bound + GEMM_REL_F * float(np.linalg.norm(ref_q))
    band = {(4, 4): (0.11, 0.19), (3, 4): (0.17, 0.26), (2, 4): (0.31, 0.42), (3, 3): (0.22, 0.32),
            (4, 6): (0.08, 0.13)}[(bw, ba)]
    assert band[0] < e_dense < band[1]


def test_binding_rejects_bad_operands():
    # operands whose sizes do not match the codebooks are refused before any launch
    K = 256
    cb4, cb3, cb_other = oq.lloydmax_codebook(4, K), oq.lloydmax_codebook(3, K), oq.lloydmax_codebook(4, 512)
    xc = torch.zeros((8, K // 2), dtype=torch.uint8, device=DEV)
    xn = torch.ones(8, device=DEV)
    wc = torch.zeros((16, K // 2), dtype=torch.uint8, device=DEV)
    wn = torch.ones(16, dtype=torch.bfloat16, device=DEV)
    cases = [
        lambda: oq.orbit_qlinear(cb4, xc[:, :100], xn, cb4, wc, wn),            # too few code bytes
        lambda: oq.orbit_qlinear(cb4, xc, xn, cb3, wc, wn),                     # 3-bit rows are 96 bytes
        lambda: oq.orbit_qlinear(cb4, xc, xn.double(), cb4, wc, wn),            # norm dtype
        lambda: oq.orbit_qlinear(cb4, xc, xn[:7], cb4, wc, wn),                 # norm count
        lambda: oq.orbit_qlinear(cb4, xc, xn, cb4, wc, wn.float()),             # r' must be bf16
        lambda: oq.orbit_qlinear(cb4, xc, xn, cb_other, wc, wn),                # codebooks for another d
        lambda: oq.orbit_qlinear(cb4, xc, xn, cb4, wc, wn, out=torch.empty((8, 15), device=DEV)),
        lambda: oq.orbit_qlinear_ex(cb4, xc, xn, cb4, wc, wn, bias=torch.zeros(15, dtype=torch.bfloat16,
                                                                                  device=DEV)),
        lambda: oq.rpbh_quantize_act(oq.rpbh_plan(K, 128, 0), cb4, torch.zeros((8, K), dtype=torch.bfloat16,
                                     device=DEV), codes=torch.empty((8, K // 4), dtype=torch.uint8, device=DEV)),
    ]
    for i, call in enumerate(cases):
        with pytest.raises(ValueError):
            call()
    torch.cuda.synchronize()


@pytest.mark.parametrize("ba,bw", [(4, 4), (2, 3)])
def test_long_contraction(ba, bw):
    # K = 65536 (1024 K-steps of fp32 accumulation) on the 128 x 128 kernel, all outputs
    M, N, K = 300, 260, 65536
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=K + ba)
    Y = _gpu(xc, xs, wc, wr, ba, bw, K)
    args = (xc.numpy(), xs.double().numpy(), ba, wc.numpy(), wr.double().numpy(), bw, K)
    check_gemm(f"gemm long K={K} W{bw}A{ba}", Y, qlinear_oracle_bf16(*args), _scale(*args), K)


def test_long_contraction_large_tiles_sampled_rows():
    # K = 16384 (256 K-steps) on the 256 x 256 kernel (289 tiles, ragged), 64 sampled rows x all N
    M, N, K, ba, bw = 4133, 4099, 16384, 4, 4
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=7)
    Y = _gpu(xc, xs, wc, wr, ba, bw, K)
    rows = np.sort(np.random.default_rng(9).choice(M, 64, replace=False))
    rows[-1] = M - 1
    args = (xc.numpy()[rows], xs.double().numpy()[rows], ba, wc.numpy(), wr.double().numpy(), bw, K)
    check_gemm(f"gemm long large-tile K={K}", Y[rows], qlinear_oracle_bf16(*args), _scale(*args), K, rows=len(rows))


def test_empty_operands_are_noops():
    K = 256
    cb = oq.lloydmax_codebook(4, K)
    xc = torch.zeros((0, K // 2), dtype=torch.uint8, device=DEV)
    xn = torch.zeros((0,), device=DEV)
    wc = torch.zeros((16, K // 2), dtype=torch.uint8, device=DEV)
    wn = torch.ones(16, dtype=torch.bfloat16, device=DEV)
    assert oq.orbit_qlinear(cb, xc, xn, cb, wc, wn).shape == (0, 16)
    xc1, xn1 = torch.zeros((8, K // 2), dtype=torch.uint8, device=DEV), torch.ones(8, device=DEV)
    Y = oq.orbit_qlinear_ex(cb, xc1, xn1, cb, wc[:0], wn[:0], gelu=True, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert Y.shape == (8, 0)


# The two store paths of both GEMM kernels hold the same values: with N and ldy multiples of 4 the
# outputs are turned around in LDS before the stores, otherwise each lane stores its runs of four
# columns directly.  Each output is the same arithmetic either way, so a layer written into rows of
# N + 4 and into rows of N + 1 must agree bit for bit (large tiles, the 128 x 128 rows of a
# partial last round, and a small grid; fp32 and the fused bias + GELU + bf16 epilogue).
@pytest.mark.parametrize("M,N,K", [(4133, 8064, 192), (300, 132, 512)])
@pytest.mark.parametrize("fused", [False, True])
def test_store_paths_agree(M, N, K, fused):
    ba, bw = 4, 4
    xc, xs, wc, wr = _inputs(M, N, K, ba, bw, seed=M + 3 * N + K)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    xp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(xc.numpy(), ba), ba)).to(DEV)
    wp = torch.from_numpy(oracle.pack_codes(oracle.to_labels(wc.numpy(), bw), bw)).to(DEV)
    g = torch.Generator()
    g.manual_seed(N + 1)
    b = torch.randn(N, generator=g).to(torch.bfloat16).to(DEV) if fused else None
    dt = torch.bfloat16 if fused else torch.float32
    outs = []
    for pad in (4, 1):
        out = torch.full((M, N + pad), float("nan"), dtype=dt, device=DEV)[:, :N]
        oq.orbit_qlinear_ex(cba, xp, xs.to(DEV), cbw, wp, wr.to(DEV), bias=b, gelu=fused, out_dtype=dt, out=out)
        outs.append(out)
    torch.cuda.synchronize()
    assert not torch.isnan(outs[0].float()).any() and not torch.isnan(outs[1].float()).any()
    assert torch.equal(outs[0].view(torch.int16) if fused else outs[0].view(torch.int32),
                       outs[1].view(torch.int16) if fused else outs[1].view(torch.int32))
