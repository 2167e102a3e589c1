"""Helpers for the GPU parity tests: run the HIP path through the C ABI, run the oracle on the
same inputs, and compare.  Statistics of each comparison (near-ties, mismatches, errors) are
appended to $ORBIT_PARITY_LOG when that variable names a file."""

import json
import os
import sys

import numpy as np
import torch

import oracle
import paper_2607_02461_amd as oq

TIE_BAND = 1e-5      # |u - tau| at or below this is a near-tie: counted, not a failure
GEMM_REL_F = 2e-3    # relative Frobenius bar for the GEMM against fp64 with identical codes/levels


def log_stats(name, **stats):
    line = json.dumps({"case": name, **stats})
    print(line, flush=True)
    path = os.environ.get("ORBIT_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(line + "\n")


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def quantize_gpu(X: torch.Tensor, bits: int, seed: int = 0, weights: bool = False, eps: float = 1e-10,
                 plan=None, h: int = 128):
    K = X.shape[1]
    plan = plan or oq.rpbh_plan(K, h, seed)
    cb = oq.lloydmax_codebook(bits, K)
    if weights:
        codes, norms = oq.quantize_weights_offline(plan, cb, X, eps)
    else:
        codes, norms = oq.rpbh_quantize_act(plan, cb, X, eps)
    torch.cuda.synchronize()
    return codes, norms


def compare_quantizer(name, X: torch.Tensor, bits: int, seed: int = 0, weights: bool = False,
                      eps: float = 1e-10, rows=None, oplan=None, plan=None, h: int = 128):
    """Quantize all rows of X on the GPU (block size h); compare `rows` (default all) with the
    oracle."""
    M, K = X.shape
    codes, norms = quantize_gpu(X, bits, seed, weights, eps, plan=plan, h=h)
    sel = np.arange(M) if rows is None else np.asarray(rows)
    Xs = to_f64(X[torch.as_tensor(sel, device=X.device)]) if rows is not None else to_f64(X)
    oplan = oplan or oracle.rpbh_plan(K, h, seed)
    ocb = oracle.lloydmax_codebook(bits, K)
    if weights:
        oc, on, U = oracle.quantize_weights(Xs, oplan, ocb, eps)
    else:
        oc, on, U = oracle.quantize_act(Xs, oplan, ocb, eps)
    gcodes = codes.cpu().numpy()[sel]
    gc = oracle.unpack_codes(gcodes, bits, K)
    near = oracle.near_tie_mask(U, ocb.thresholds, TIE_BAND)
    mism = gc != oc
    bad = int(np.sum(mism & ~near))
    if weights:
        gn = norms.float().cpu().numpy().astype(np.float64)[sel]
        ulp = np.ldexp(1.0, np.frexp(np.maximum(on, 1e-30))[1] - 8)
        norm_err = float(np.max(np.abs(gn - on) / ulp)) if len(on) else 0.0   # in bf16 ulps
        norm_ok = norm_err <= 1.0
    else:
        gn = norms.cpu().numpy().astype(np.float64)[sel]
        norm_err = float(np.max(np.abs(gn - on) / np.maximum(on, 1e-30))) if len(on) else 0.0
        norm_ok = norm_err <= 1e-5 or bool(np.all(np.abs(gn - on) <= 1e-30))
    log_stats(name, M=M, K=K, h=oplan.h, bits=bits, weights=weights, rows_checked=len(sel), elements=int(gc.size),
              near_ties=int(near.sum()), near_tie_frac=float(near.mean()) if near.size else 0.0,
              near_tie_mismatches=int(np.sum(mism & near)), mismatches_off_tie=bad,
              norm_err=norm_err)
    assert bad == 0, f"{name}: {bad} code mismatches farther than {TIE_BAND} from a threshold"
    assert norm_ok, f"{name}: norm error {norm_err}"
    return codes, norms


def qlinear_oracle_fp16(xc, xs, cba_bits, wc, wr, cbw_bits, K):
    """The oracle contraction with the fp16 images of the oracle's own codebooks."""
    la = oracle.fp16_round(oracle.lloydmax_codebook(cba_bits, K).levels)
    lw = oracle.fp16_round(oracle.lloydmax_codebook(cbw_bits, K).levels)
    return oracle.qlinear(xc, xs, la, wc, wr, lw)


def rel_frobenius(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def near_tie_flip_bound(cx, s, Ux, la, tha, cw, r, Uw, lw, thw, band=TIE_BAND):
    """Frobenius bound on how far the quantized layer can move when every coordinate within
    `band` of a threshold takes the neighbouring code instead (the oracle's own codes, levels
    and norms only).  Flipping weight code (i, k) by one level changes column i by
    r_i * dL * (s_n La[cx[n, k]])_n; flipping activation code (n, k) changes row n by
    s_n * dL * (r_i Lw[cw[i, k]])_i.  The triangle inequality over flips gives the bound."""
    la, lw = np.asarray(la), np.asarray(lw)

    def step(U, th, codes, levels):
        # level difference to the neighbour across the nearest threshold, 0 off near-ties
        near = oracle.near_tie_mask(U, th, band)
        idx = np.searchsorted(th, U)                        # threshold index at or above u
        lo = np.clip(idx - 1, 0, len(th) - 1)
        hi = np.clip(idx, 0, len(th) - 1)
        j = np.where(np.abs(U - th[lo]) <= np.abs(U - th[hi]), lo, hi)   # nearest threshold
        d = np.abs(levels[j + 1] - levels[j])
        return np.where(near, d, 0.0)

    dw = step(Uw, thw, cw, lw)                              # [N, K]
    da = step(Ux, tha, cx, la)                              # [M, K]
    A = s[:, None] * la[cx]                                 # [M, K]
    B = r[:, None] * lw[cw]                                 # [N, K]
    col = r * (dw @ np.linalg.norm(A, axis=0))              # per output column i
    row = s * (da @ np.linalg.norm(B, axis=0))              # per output row n
    return float(np.sqrt(np.sum(col ** 2)) + np.sqrt(np.sum(row ** 2)))
