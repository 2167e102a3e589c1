"""INT4 round-to-nearest weight-only layer of the AdaLN modulation projections
(test infrastructure only).

The experimental setup (Sec. 5) keeps the adaptive-layer-norm modulation projections at INT4
weight round-to-nearest; the supplementary material fixes the group size at 64 and the
activations at BF16, and says why these layers are not rotated (their dynamic scale-and-shift
cannot be folded into neighbouring weights, and their input is a single conditioning token per
step).  Sec. 6.2 ablates their bit-width.

Readings taken where the paper is silent (it does not spell out the rounding grid):
  * symmetric scaling per group of 64 consecutive inputs of a weight row;
  * the group's scale is the FP16 rounding (to nearest even, saturating at the largest finite
    FP16) of the FP32 quotient absmax / 7, and a group whose scale rounds to 0 has codes 0;
  * q = clamp(RNE(w / scale), -8, 7), the quotient formed in FP32 with the stored FP16 scale
    (the scale a dequantizer reads back, so q is the nearest integer multiple of the scale that
    is actually stored; FP32 holds every BF16 weight exactly and the quotient needs only one
    IEEE rounding before the integer rounding, so the definition is exact bit for bit;
    |w / scale| <= 7 up to the scale's rounding, so the clamp only guards);
  * storage: q + 8 (offset binary, 0..15) as LSB-first nibbles, element 2j in the low nibble
    of byte j; scales as FP16 [N][K/64].
The dequantized weight is q * scale and the layer is Y = X W_deq^T (+ bias) with BF16 X, here
in fp64.
"""

import numpy as np

GROUP = 64
FP16_MAX = 65504.0


def rtn_int4_quantize(W):
    """W [N, K] (BF16 values, K a multiple of 64) -> (q int8 [N, K], scale fp64 [N, K/64])."""
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    if K % GROUP:
        raise ValueError("K must be a multiple of the group size 64")
    Wg = W.reshape(N, K // GROUP, GROUP).astype(np.float32)            # exact: BF16 values
    absmax = np.max(np.abs(Wg), axis=2)
    scale32 = np.minimum(absmax / np.float32(7.0), np.float32(FP16_MAX))  # IEEE fp32 quotient
    scale = scale32.astype(np.float16)                                  # RNE to fp16
    s32 = scale.astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        quot = Wg / s32[:, :, None]                                     # IEEE fp32 quotient
        q = np.where(s32[:, :, None] > 0, np.clip(np.rint(quot), -8, 7), 0)
    return q.astype(np.int8).reshape(N, K), scale.astype(np.float64)


def rtn_int4_dequantize(q, scale):
    """q * scale, group by group (fp64)."""
    q = np.asarray(q, dtype=np.float64)
    return q * np.repeat(np.asarray(scale, dtype=np.float64), GROUP, axis=1)


def pack_rtn_int4(q):
    """int8 codes in [-8, 7] [N, K] -> uint8 [N, K/2]: q + 8 per nibble, element 2j low."""
    u = (np.asarray(q, dtype=np.int16) + 8).astype(np.uint8)
    return (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)


def unpack_rtn_int4(packed, K):
    p = np.asarray(packed, dtype=np.uint8)
    u = np.empty((p.shape[0], K), dtype=np.int16)
    u[:, 0::2] = p & 0xF
    u[:, 1::2] = p >> 4
    return (u - 8).astype(np.int8)


def rtn_int4_linear(X, q, scale, bias=None):
    """Y = X (q * scale)^T (+ bias) in fp64: the AdaLN modulation projection on its INT4 weights."""
    Y = np.asarray(X, dtype=np.float64) @ rtn_int4_dequantize(q, scale).T
    if bias is not None:
        Y = Y + np.asarray(bias, dtype=np.float64)[None, :]
    return Y
