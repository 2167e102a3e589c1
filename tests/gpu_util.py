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
# Per-element bar of the contraction: |Y[n,i] - ref[n,i]| <= ELEM_TOL * s_n r'_i ||a_n|| ||b_i||, with
# a_n = L_a[x_code[n]] and b_i = L_w[w_code[i]] (bf16 levels).  The bf16 products are exact in fp32;
# what remains is the fp32 sum of K of them (plus split partials and a few epilogue roundings).  The
# probabilistic bound on a sum of n terms (Higham and Mary, SIAM J. Sci. Comput. 2019),
# lambda sqrt(n) u sum|a_k b_k| with u = 2^-24 and lambda = 10, is below 8e-5 ||a|| ||b|| (Cauchy-Schwarz)
# for n up to 16384 + 64, so 1e-4 holds with margin for every K these tests use up to 16384; the
# K = 65536 cases take the same formula at their n (1.5e-4).  A wrong tile, a dropped K-step or a
# misplaced row fails it at once: such errors are of the order of the outputs themselves,
# ~||a|| ||b|| / sqrt(K).
ELEM_TOL = 1e-4


def elem_tol(K: int) -> float:
    """The per-element bar for a contraction of length K (see ELEM_TOL)."""
    n = K + 64
    return max(ELEM_TOL, 10.0 * np.sqrt(n) * 2.0 ** -24)


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
    gc = oracle.from_labels(oracle.unpack_codes(gcodes, bits, K), bits)
    cstats = code_stats(gc, oc, U, ocb.thresholds)
    if weights:
        gn = norms.float().cpu().numpy().astype(np.float64)[sel]
        ulp = np.ldexp(1.0, np.frexp(np.maximum(on, 1e-30))[1] - 8)
        norm_err = float(np.max(np.abs(gn - on) / ulp)) if len(on) else 0.0   # in bf16 ulps
        norm_ok = norm_err <= 1.0
    else:
        gn = norms.cpu().numpy().astype(np.float64)[sel]
        norm_err = float(np.max(np.abs(gn - on) / np.maximum(on, 1e-30))) if len(on) else 0.0
        norm_ok = norm_err <= 1e-5 or bool(np.all(np.abs(gn - on) <= 1e-30))
    log_stats(name, M=M, K=K, h=oplan.h, bits=bits, weights=weights, rows_checked=len(sel), **cstats,
              norm_err=norm_err)
    assert_codes(name, cstats)
    assert norm_ok, f"{name}: norm error {norm_err}"
    return codes, norms


def code_stats(gc, oc, U, thresholds, band=TIE_BAND) -> dict:
    """Counts of a comparison of the HIP path's codes `gc` with the oracle's `oc` (both unpacked).

    Off near-ties the codes must be equal.  Within `band` of a threshold tau_j the nearest-centroid
    map of Eq. (3) ties between codes j and j+1 at tau_j itself, so either is correct there and
    nothing else is: a near-tie code outside that pair is invalid."""
    near = oracle.near_tie_mask(U, thresholds, band)
    mism = gc != oc
    j = oracle.nearest_threshold(U, thresholds)
    pair = (gc == j) | (gc == j + 1)
    return dict(elements=int(gc.size), near_ties=int(near.sum()),
                near_tie_frac=float(near.mean()) if near.size else 0.0,
                near_tie_mismatches=int(np.sum(mism & near)),
                near_tie_invalid=int(np.sum(mism & near & ~pair)),
                mismatches_off_tie=int(np.sum(mism & ~near)))


def assert_codes(name, stats):
    assert stats["mismatches_off_tie"] == 0, \
        f"{name}: {stats['mismatches_off_tie']} code mismatches farther than {TIE_BAND} from a threshold"
    assert stats["near_tie_invalid"] == 0, \
        f"{name}: {stats['near_tie_invalid']} near-tie codes neither the oracle's nor its neighbour across the threshold"


def qlinear_oracle_bf16(xc, xs, cba_bits, wc, wr, cbw_bits, K):
    """The oracle contraction with the bf16 images of the oracle's own codebooks."""
    la = oracle.bf16_round(oracle.lloydmax_codebook(cba_bits, K).levels)
    lw = oracle.bf16_round(oracle.lloydmax_codebook(cbw_bits, K).levels)
    return oracle.qlinear(xc, xs, la, wc, wr, lw)


def rel_frobenius(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def gemm_scale(xc, s, la, wc, r, lw) -> np.ndarray:
    """s_n r'_i ||L_a[x_code[n]]|| ||L_w[w_code[i]]||: the Cauchy-Schwarz bound on |Y[n,i]|, the
    unit of the per-element bar."""
    la, lw = np.asarray(la, dtype=np.float64), np.asarray(lw, dtype=np.float64)
    na = np.linalg.norm(la[np.asarray(xc)], axis=1)
    nb = np.linalg.norm(lw[np.asarray(wc)], axis=1)
    return (np.asarray(s, dtype=np.float64) * na)[:, None] * (np.asarray(r, dtype=np.float64) * nb)[None, :]


def check_gemm(name, Y, ref, scale, K, slack=0.0, **extra) -> dict:
    """fp32 layer output `Y` against the fp64 oracle `ref` on identical codes, levels and norms:
    relative Frobenius error <= GEMM_REL_F, and every element within elem_tol(K) * scale (+ slack,
    an epilogue's own allowance).  Returns and logs the figures."""
    Y = np.asarray(Y, dtype=np.float64)
    err = rel_frobenius(Y, ref)
    tol = elem_tol(K)
    excess = np.abs(Y - ref) - (tol * scale + slack)
    worst = float(np.max(np.abs(Y - ref) / np.maximum(tol * scale + slack, 1e-300))) if Y.size else 0.0
    stats = dict(rel_f=err, worst_elem_over_bar=worst, elems_beyond_bar=int(np.sum(excess > 0)), **extra)
    log_stats(name, **stats)
    assert err <= GEMM_REL_F, f"{name}: relative Frobenius error {err}"
    assert stats["elems_beyond_bar"] == 0, f"{name}: {stats['elems_beyond_bar']} outputs beyond the per-element bar"
    return stats


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
