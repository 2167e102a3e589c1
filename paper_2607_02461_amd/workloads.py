"""Seeded synthetic inputs shaped like the paper's DiT workloads.

This module holds no part of the quantization method: it only draws random
activations and weights, rounds them to BF16, and names the shapes of the
benchmark workloads.  It is the one module read both by the CPU oracle's
tests and by the HIP path's tests and benchmark.

Shapes follow the paper's models: an image DiT at 1024^2 has attention width
d = 3072 and feed-forward width 12288 with 4096 image + 512 text tokens
(Sec. 4.5, Fig. 3 caption); a video DiT at 480x832 with 81 frames has a
21x30x52 latent patch grid and hidden width 5120 (Suppl. B generation settings).
The activation laws (Student-t, outlier channels, per-token log-normal scale,
mean drift across timesteps and frames) stand in for real activations, which
this repository does not have.

All draws use torch generators (CPU or GPU) seeded per (workload, tensor), in
fp32, then rounded to BF16 (round-to-nearest-even by torch's conversion).
Tensors are returned as torch.bfloat16 on the requested device.
"""

from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import torch


@dataclass(frozen=True)
class Linear:
    """One quantized linear: M tokens x K inputs -> N outputs at (b_w, b_a) bits."""
    name: str
    M: int
    K: int
    N: int
    bw: int
    ba: int
    h: int = 128


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    linears: Tuple[Linear, ...]
    data_seed: int
    plan_seed: int = 0
    repeat: int = 1          # e.g. transformer blocks sharing the shapes
    extra: Dict = field(default_factory=dict)


# --- the five workloads -----------------------------------------------------------------------
C1 = Workload(
    "c1_single_w4a4",
    "single quantized linear W4A4, 256 tokens, 3072 -> 3072, 5% outlier channels x20",
    (Linear("proj", 256, 3072, 3072, 4, 4),), data_seed=1)

C2_M = 2 * (4096 + 512)
C2 = Workload(
    "c2_image_mlp",
    "image-DiT MLP pair, 2 guidance branches x (4096 image + 512 text) tokens, 3072 -> 12288 -> 3072,"
    " Student-t(3) activations with per-channel drift over 28 timesteps",
    (Linear("up_w4a4", C2_M, 3072, 12288, 4, 4), Linear("down_w4a4", C2_M, 12288, 3072, 4, 4),
     Linear("up_w3a4", C2_M, 3072, 12288, 3, 4), Linear("down_w3a4", C2_M, 12288, 3072, 3, 4)),
    data_seed=2, extra={"timesteps": 28, "branches": 2, "text_tokens": 512})

C3_M = 2 * 4608
C3 = Workload(
    "c3_image_attn",
    "image-DiT attention projections, 9216 tokens, fused QKV 3072 -> 9216 and out 3072 -> 3072,"
    " 2% outlier channels x50, per-token log-normal scale, 1% outlier weight rows x10",
    (Linear("qkv_w2a4", C3_M, 3072, 9216, 2, 4), Linear("out_w2a4", C3_M, 3072, 3072, 2, 4),
     Linear("qkv_w3a3", C3_M, 3072, 9216, 3, 3), Linear("out_w3a3", C3_M, 3072, 3072, 3, 3)),
    data_seed=3)

C4_M = 21 * 30 * 52 + 512
C4 = Workload(
    "c4_video_mlp_w4a4",
    "video-DiT MLP W4A4, 32760 latent-patch tokens (21x30x52) + 512 text tokens,"
    " 5120 -> 13824 -> 5120, Student-t(4) activations with per-frame mean shift",
    (Linear("up", C4_M, 5120, 13824, 4, 4), Linear("down", C4_M, 13824, 5120, 4, 4)),
    data_seed=4, extra={"frames": 21, "tokens_per_frame": 30 * 52, "text_tokens": 512})

C5_M = 21 * 30 * 52
C5 = Workload(
    "c5_video_trunk_w4a4",
    "video-DiT trunk sweep W4A4, 40 blocks x {QKV 5120->15360, out 5120->5120,"
    " FFN 5120->13824->5120} at 32760 tokens, plus the offline weight pass",
    (Linear("qkv", C5_M, 5120, 15360, 4, 4), Linear("out", C5_M, 5120, 5120, 4, 4),
     Linear("ffn_up", C5_M, 5120, 13824, 4, 4), Linear("ffn_down", C5_M, 13824, 5120, 4, 4)),
    data_seed=5, repeat=40, extra={"frames": 21, "tokens_per_frame": 30 * 52})

WORKLOADS = {w.name: w for w in (C1, C2, C3, C4, C5)}

# The adjacent layer type: the AdaLN modulation projections of the image DiT (FLUX-shaped,
# hidden 3072), kept at INT4 weight round-to-nearest with BF16 activations.  Each of the 19
# double-stream blocks has two (image and text stream) of 3072 -> 6 x 3072; each of the 38
# single-stream blocks one of 3072 -> 3 x 3072: 3.2e9 weights, the share of the model the paper
# gives for these layers.  The input is one conditioning token per step.
ADALN_K = 3072
ADALN_LAYERS = ((18432, 2 * 19), (9216, 38))   # (N, count)
ADALN_SEED = 6


def adaln_weights(N: int, index: int, device="cpu") -> torch.Tensor:
    """Weights of AdaLN projection `index` with N outputs: N(0, 0.02^2), BF16."""
    return gaussian_weights(N, ADALN_K, 0.02, ADALN_SEED, index, device=device)


def adaln_tokens(M: int, K: int = ADALN_K, seed: int = ADALN_SEED, device="cpu") -> torch.Tensor:
    """Conditioning tokens: SiLU of N(0, 1) draws (the modulation MLP's input activation), BF16."""
    g = _gen(seed, 701, M, device=device)
    return to_bf16(torch.nn.functional.silu(_randn((M, K), g, device)))


# --- helpers ----------------------------------------------------------------------------------
def _gen(seed: int, *stream: int, device="cpu") -> torch.Generator:
    """A torch generator for (seed, stream ids); distinct ids give unrelated streams."""
    g = torch.Generator(device=device)
    key = seed
    for s in stream:
        key = (key * 1_000_003 + s + 1) % (2 ** 62)
    g.manual_seed(key)
    return g


def _randn(shape, g, device) -> torch.Tensor:
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def student_t(shape, nu: int, g, device) -> torch.Tensor:
    """Student-t with integer nu: Z / sqrt(chi2_nu / nu), chi2 as a sum of nu squared normals."""
    z = _randn(shape, g, device)
    chi2 = torch.zeros(shape, device=device, dtype=torch.float32)
    for _ in range(nu):
        e = _randn(shape, g, device)
        chi2 += e * e
    return z * torch.sqrt(nu / chi2)


def to_bf16(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.bfloat16)


def choose_channels(K: int, count: int, g, device) -> torch.Tensor:
    """`count` distinct channel indices out of K (seeded)."""
    return torch.randperm(K, generator=g, device=device)[:count]


# --- generic laws -------------------------------------------------------------------------------
def gaussian_weights(N: int, K: int, std: float, seed: int, stream: int, device="cpu",
                     outlier_rows_frac: float = 0.0, outlier_scale: float = 1.0) -> torch.Tensor:
    g = _gen(seed, 101, stream, device=device)
    W = _randn((N, K), g, device) * std
    if outlier_rows_frac > 0:
        rows = choose_channels(N, int(round(outlier_rows_frac * N)), g, device)
        W[rows] *= outlier_scale
    return to_bf16(W)


def gaussian_outlier_acts(M: int, K: int, seed: int, stream: int, frac: float, scale: float,
                          device="cpu", lognormal_token_scale: bool = False) -> torch.Tensor:
    g = _gen(seed, 202, stream, device=device)
    X = _randn((M, K), g, device)
    ch = choose_channels(K, int(round(frac * K)), g, device)
    X[:, ch] *= scale
    if lognormal_token_scale:
        X *= torch.exp(_randn((M, 1), g, device))
    return to_bf16(X)


# --- per-workload inputs ------------------------------------------------------------------------
def c1_inputs(device="cpu"):
    """(X [256,3072], W [3072,3072]) for the single W4A4 linear."""
    lin = C1.linears[0]
    X = gaussian_outlier_acts(lin.M, lin.K, C1.data_seed, 0, frac=0.05, scale=20.0, device=device)
    W = gaussian_weights(lin.N, lin.K, 0.02, C1.data_seed, 0, device=device)
    return X, W


def c2_up_acts(step: int, device="cpu", rows: slice = None) -> torch.Tensor:
    """Up-projection input at denoising step `step` (0..27): Student-t(3) plus a per-branch
    channel drift interpolated between two endpoints; text tokens add a per-branch offset."""
    K, T = 3072, C2.extra["timesteps"]
    img, txt = 4096, C2.extra["text_tokens"]
    parts = []
    for branch in range(C2.extra["branches"]):
        ge = _gen(C2.data_seed, 301, branch, device=device)
        a, b, c = _randn((K,), ge, device), _randn((K,), ge, device), _randn((K,), ge, device)
        lam = step / (T - 1)
        mu = (1 - lam) * a + lam * b
        g = _gen(C2.data_seed, 302, branch, step, device=device)
        Xi = student_t((img, K), 3, g, device) + mu
        Xt = student_t((txt, K), 3, g, device) + mu + c
        parts += [Xi, Xt]
    X = torch.cat(parts, 0)
    if rows is not None:
        X = X[rows]
    return to_bf16(X)


def c2_weights(device="cpu"):
    up = gaussian_weights(12288, 3072, 0.02, C2.data_seed, 1, device=device)
    down = gaussian_weights(3072, 12288, 0.02, C2.data_seed, 2, device=device)
    return up, down


def c2_down_acts(step: int, device="cpu") -> torch.Tensor:
    """Down-projection input at denoising step `step`: GELU (exact erf) of the unquantized
    up-projection X_up W_up^T in fp32, rounded to BF16 (the dense layer stands in for the real
    model's hidden activations)."""
    Xu = c2_up_acts(step, device=device).float()
    Wu, _ = c2_weights(device=device)
    H = Xu @ Wu.float().t().contiguous()
    return to_bf16(torch.nn.functional.gelu(H))


def c3_inputs(device="cpu"):
    """(X_qkv, X_out, W_qkv, W_out) for the attention projections."""
    M, K = C3_M, 3072
    Xq = gaussian_outlier_acts(M, K, C3.data_seed, 0, frac=0.02, scale=50.0, device=device,
                               lognormal_token_scale=True)
    Xo = gaussian_outlier_acts(M, K, C3.data_seed, 1, frac=0.02, scale=50.0, device=device,
                               lognormal_token_scale=True)
    Wq = gaussian_weights(9216, K, 0.02, C3.data_seed, 0, device=device, outlier_rows_frac=0.01,
                          outlier_scale=10.0)
    Wo = gaussian_weights(3072, K, 0.02, C3.data_seed, 1, device=device, outlier_rows_frac=0.01,
                          outlier_scale=10.0)
    return Xq, Xo, Wq, Wo


def video_acts(M_img: int, text: int, K: int, nu: int, frames: int, seed: int, stream: int,
               device="cpu", chunk_rows: int = 4096) -> torch.Tensor:
    """Student-t(nu) tokens; frame f of `frames` owns a contiguous run of image rows and adds
    mu_f = (1 - f/(frames-1)) a + f/(frames-1) b; text rows (appended last) are unshifted.
    Generated in row chunks so that large inputs never hold an fp32 copy of the whole tensor."""
    ge = _gen(seed, 401, stream, device=device)
    a, b = _randn((K,), ge, device), _randn((K,), ge, device)
    per = M_img // frames
    out = torch.empty((M_img + text, K), dtype=torch.bfloat16, device=device)
    for r0 in range(0, M_img + text, chunk_rows):
        r1 = min(M_img + text, r0 + chunk_rows)
        g = _gen(seed, 402, stream, r0, device=device)
        X = student_t((r1 - r0, K), nu, g, device)
        idx = torch.arange(r0, r1, device=device)
        f = torch.clamp(idx // per, max=frames - 1).to(torch.float32)
        lam = (f / max(frames - 1, 1))[:, None]
        shift = (1 - lam) * a[None, :] + lam * b[None, :]
        X += torch.where((idx < M_img)[:, None], shift, torch.zeros_like(shift))
        out[r0:r1] = to_bf16(X)
    return out


def c4_inputs(device="cpu"):
    """(X_up [33272,5120], X_down [33272,13824], W_up [13824,5120], W_down [5120,13824])."""
    fr, tpf, txt = C4.extra["frames"], C4.extra["tokens_per_frame"], C4.extra["text_tokens"]
    Xu = video_acts(fr * tpf, txt, 5120, 4, fr, C4.data_seed, 0, device=device)
    Xd = video_acts(fr * tpf, txt, 13824, 4, fr, C4.data_seed, 1, device=device)
    Wu = gaussian_weights(13824, 5120, 0.015, C4.data_seed, 0, device=device)
    Wd = gaussian_weights(5120, 13824, 0.015, C4.data_seed, 1, device=device)
    return Xu, Xd, Wu, Wd


def c5_acts(device="cpu"):
    """One activation draw per input width, reused by every block: {5120: X, 13824: X}."""
    fr, tpf = C5.extra["frames"], C5.extra["tokens_per_frame"]
    return {K: video_acts(fr * tpf, 0, K, 4, fr, C5.data_seed, i, device=device)
            for i, K in enumerate((5120, 13824))}


def c5_weight(block: int, layer: int, device="cpu") -> torch.Tensor:
    lin = C5.linears[layer]
    return gaussian_weights(lin.N, lin.K, 0.015, C5.data_seed, 1000 + 10 * block + layer, device=device)


def random_codes(M: int, K: int, bits: int, seed: int, device="cpu") -> torch.Tensor:
    """Uniform random codes in [0, 2^bits) as int64 [M, K] (GEMM-only test inputs)."""
    g = _gen(seed, 501, bits, device=device)
    return torch.randint(0, 1 << bits, (M, K), generator=g, device=device, dtype=torch.int64)


def random_norms(n: int, seed: int, stream: int, device="cpu", lo: float = 0.25, hi: float = 4.0):
    """Positive per-row magnitudes, log-uniform in [lo, hi] (fp32)."""
    g = _gen(seed, 601, stream, device=device)
    u = torch.rand((n,), generator=g, device=device, dtype=torch.float32)
    return torch.exp(torch.log(torch.tensor(lo)) + u * (torch.log(torch.tensor(hi)) - torch.log(torch.tensor(lo))))
