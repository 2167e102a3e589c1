"""Full-size parity of the whole GPU pipeline (offline weight pass -> activation quantizer ->
LUT GEMM) on every linear of the five DiT-shaped workloads, in the launch configuration the
benchmark uses.  The oracle quantizes a sample of activation rows and weight rows (the last of
each included) and contracts them in fp64; on that sample the GPU's codes must equal the oracle's
off near-ties, its norms must match, the GEMM on the GPU's own codes must be within the relative
Frobenius bar of the fp64 contraction with identical codes and levels, and the pipeline output
must be within the near-tie flip bound of the oracle pipeline's."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import (GEMM_REL_F, assert_codes, check_gemm, code_stats, gemm_scale, log_stats,
                            near_tie_flip_bound, to_f64)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _sample(n, count, seed):
    idx = np.sort(np.random.default_rng(seed).choice(n, min(count, n), replace=False))
    idx[-1] = n - 1
    return idx


def _check_codes(name, gpu_codes, bits, K, oc, U, thresholds):
    gc = oracle.from_labels(oracle.unpack_codes(gpu_codes, bits, K), bits)
    stats = code_stats(gc, oc, U, thresholds)
    assert_codes(name, stats)
    return gc, stats


def pipeline_check(name, X, W, bw, ba, seed, rows=128, cols=256, plan_seed=0):
    M, K = X.shape
    N = W.shape[0]
    plan = oq.rpbh_plan(K, 128, plan_seed)
    cba, cbw = oq.lloydmax_codebook(ba, K), oq.lloydmax_codebook(bw, K)
    wcodes, wnorm = oq.quantize_weights_offline(plan, cbw, W)
    xcodes, xnorm = oq.rpbh_quantize_act(plan, cba, X)
    Y = oq.orbit_qlinear(cba, xcodes, xnorm, cbw, wcodes, wnorm)
    torch.cuda.synchronize()

    R, C = _sample(M, rows, seed), _sample(N, cols, seed + 1)
    Rt, Ct = torch.as_tensor(R, device=DEV), torch.as_tensor(C, device=DEV)
    oplan = oracle.rpbh_plan(K, 128, plan_seed)
    oca, ocw = oracle.lloydmax_codebook(ba, K), oracle.lloydmax_codebook(bw, K)
    cx, s, Ux = oracle.quantize_act(to_f64(X[Rt]), oplan, oca)
    cw, r, Uw = oracle.quantize_weights(to_f64(W[Ct]), oplan, ocw)

    gx, st_x = _check_codes(name + " act", xcodes[Rt].cpu().numpy(), ba, K, cx, Ux, oca.thresholds)
    gw, st_w = _check_codes(name + " weights", wcodes[Ct].cpu().numpy(), bw, K, cw, Uw, ocw.thresholds)
    gs = xnorm[Rt].cpu().numpy().astype(np.float64)
    gr = wnorm[Ct].float().cpu().numpy().astype(np.float64)
    s_err = float(np.max(np.abs(gs - s) / np.maximum(s, 1e-30)))
    r_ulps = float(np.max(np.abs(gr - r) / np.ldexp(1.0, np.frexp(np.maximum(r, 1e-30))[1] - 8)))
    assert s_err <= 1e-5 and r_ulps <= 1.0

    la, lw = oracle.bf16_round(oca.levels), oracle.bf16_round(ocw.levels)
    Ys = Y[Rt][:, Ct].double().cpu().numpy()
    # the GEMM alone: identical codes, levels and norms
    gstats = check_gemm(name + " gemm", Ys, oracle.qlinear(gx, gs, la, gw, gr, lw), gemm_scale(gx, gs, la, gw, gr, lw),
                        K)
    # the whole pipeline against the oracle's own pipeline
    ref_q = oracle.qlinear(cx, s, la, cw, r, lw)
    bound = near_tie_flip_bound(cx, s, Ux, la, oca.thresholds, cw, r, Uw, lw, ocw.thresholds)
    diff = float(np.linalg.norm(Ys - ref_q))
    log_stats(name, M=M, N=N, K=K, bw=bw, ba=ba, rows=len(R), cols=len(C),
              near_ties_act=st_x["near_ties"], near_tie_mismatches_act=st_x["near_tie_mismatches"],
              near_ties_w=st_w["near_ties"], near_tie_mismatches_w=st_w["near_tie_mismatches"],
              s_rel_err=s_err, r_err_bf16_ulps=r_ulps, gemm_rel_f=gstats["rel_f"],
              gemm_worst_elem_over_bar=gstats["worst_elem_over_bar"],
              pipeline_rel_f=diff / float(np.linalg.norm(ref_q)),
              near_tie_bound_rel=bound / float(np.linalg.norm(ref_q)))
    assert diff <= bound + GEMM_REL_F * float(np.linalg.norm(ref_q))


@pytest.mark.parametrize("step", [0, 27])
@pytest.mark.parametrize("bw", [4, 3])
def test_c2_image_mlp(bw, step):
    # up 3072 -> 12288 on the timestep's activations, then down 12288 -> 3072 on the GELU of the
    # dense up-projection; both guidance branches are in the 9216 rows
    Wu, Wd = workloads.c2_weights(device=DEV)
    Xu = workloads.c2_up_acts(step, device=DEV)
    pipeline_check(f"c2 up W{bw}A4 step {step}", Xu, Wu, bw, 4, seed=20 + step)
    del Xu
    Xd = workloads.c2_down_acts(step, device=DEV)
    pipeline_check(f"c2 down W{bw}A4 step {step}", Xd, Wd, bw, 4, seed=40 + step)


@pytest.mark.parametrize("bw,ba", [(2, 4), (3, 3)])
def test_c3_image_attention(bw, ba):
    Xq, Xo, Wq, Wo = workloads.c3_inputs(device=DEV)
    pipeline_check(f"c3 qkv W{bw}A{ba}", Xq, Wq, bw, ba, seed=31)
    pipeline_check(f"c3 out W{bw}A{ba}", Xo, Wo, bw, ba, seed=32)


@pytest.mark.parametrize("layer", ["up", "down"])
def test_c4_video_mlp(layer):
    fr, tpf, txt = workloads.C4.extra["frames"], workloads.C4.extra["tokens_per_frame"], workloads.C4.extra["text_tokens"]
    K, N, stream = (5120, 13824, 0) if layer == "up" else (13824, 5120, 1)
    X = workloads.video_acts(fr * tpf, txt, K, 4, fr, workloads.C4.data_seed, stream, device=DEV)
    W = workloads.gaussian_weights(N, K, 0.015, workloads.C4.data_seed, stream, device=DEV)
    pipeline_check(f"c4 {layer} W4A4", X, W, 4, 4, seed=50 + stream)


@pytest.mark.parametrize("block", [0, 39])
def test_c5_video_trunk_block(block):
    acts = workloads.c5_acts(device=DEV)
    for layer, lin in enumerate(workloads.C5.linears):
        W = workloads.c5_weight(block, layer, device=DEV)
        pipeline_check(f"c5 block {block} {lin.name} W4A4", acts[lin.K], W, 4, 4, seed=60 + 4 * block + layer)
        del W
