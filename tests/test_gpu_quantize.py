"""GPU parity of the fused RPBH quantizer (activations and the offline weight pass) against
the fp64 oracle: codes bit-exact wherever the normalized rotated value lies more than 1e-5
from a decision threshold (near-ties are counted and logged), fp32 norms within 1e-5
relative, BF16 weight norms within one BF16 ulp."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02461_amd as oq
from paper_2607_02461_amd import workloads
from tests.gpu_util import compare_quantizer, quantize_gpu, log_stats, to_f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _randn_bf16(M, K, seed, scale=1.0):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn((M, K), generator=g, device=DEV) * scale).to(torch.bfloat16)


@pytest.mark.parametrize("K,M", [(128, 1), (384, 3), (1024, 64), (3072, 257), (128, 1000), (16384, 5),
                                 (5120, 130), (13824, 3)])
@pytest.mark.parametrize("bits", [2, 3, 4, 6])
@pytest.mark.parametrize("weights", [False, True])
def test_small_shapes(K, M, bits, weights):
    X = _randn_bf16(M, K, seed=K * 7 + M)
    compare_quantizer(f"small K={K} M={M}", X, bits, seed=K % 5, weights=weights)


# a workgroup holds fewer rows than it could when that leaves compute units idle: ceil(M / 256)
# rows on 256 compute units, up to 128 / (K / 128).  These row counts step through 1..5 rows per
# group at K = 3072 (5 at most) and 9 and 20 at K = 256 (64 at most), with ragged last groups.
@pytest.mark.parametrize("K,M", [(3072, 255), (3072, 257), (3072, 513), (3072, 769), (3072, 1281),
                                 (256, 2049), (256, 5000)])
@pytest.mark.parametrize("weights", [False, True])
def test_rows_per_group_from_row_count(K, M, weights):
    X = _randn_bf16(M, K, seed=K + 3 * M)
    compare_quantizer(f"rows per group K={K} M={M}", X, 4, seed=1, weights=weights)


# block sizes above 128: the paper's rule (largest power of two dividing d) for the workload
# dimensions, every size up to 4096 alone, and ragged row counts spanning several groups
@pytest.mark.parametrize("K,h,M", [(256, 256, 77), (512, 512, 33), (1024, 1024, 129), (2048, 2048, 17),
                                   (4096, 4096, 9), (3072, 1024, 257), (5120, 1024, 130), (12288, 4096, 7),
                                   (13824, 512, 5), (8192, 4096, 6), (16384, 4096, 3), (6144, 2048, 11),
                                   (1536, 512, 40), (2560, 256, 50)])
@pytest.mark.parametrize("weights", [False, True])
def test_block_sizes(K, h, M, weights):
    X = _randn_bf16(M, K, seed=K + h + M, scale=0.5)
    for bits in (4,) if weights else (2, 3, 4):
        compare_quantizer(f"block h={h} K={K} M={M}", X, bits, seed=K % 3, weights=weights, h=h)


def test_paper_block_rule_c1():
    # h = 0 selects the paper's rule: 1024 for d = 3072
    X, W = workloads.c1_inputs(device=DEV)
    plan = oq.rpbh_plan(3072, 0, 0)
    assert plan.h == 1024
    compare_quantizer("c1 act paper h", X, 4, seed=0, plan=plan, h=1024)
    compare_quantizer("c1 weights paper h", W, 4, seed=0, weights=True, plan=plan, h=1024)


def test_block_size_outlier_channels():
    # outlier channels spread by the permutation across a 4096-block
    Xq, _, _, _ = workloads.c3_inputs(device=DEV)
    X = torch.cat([Xq[:64], Xq[:64], Xq[:64], Xq[:64]], dim=1).contiguous()  # K = 12288
    compare_quantizer("c3-like act h=4096", X, 4, seed=1, h=4096)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("bits", [2, 3, 4, 6])
def test_c1_activations_full(seed, bits):
    X, _ = workloads.c1_inputs(device=DEV)
    compare_quantizer(f"c1 act seed={seed}", X, bits, seed=seed)


def test_c1_weights_full():
    _, W = workloads.c1_inputs(device=DEV)
    compare_quantizer("c1 weights", W, 4, seed=0, weights=True)


def test_c2_activations_every_timestep():
    # the image MLP's up-projection input: every row at timestep 0, 256 sampled rows (the last
    # included) at each of the other 27 steps, all with the one fixed codebook
    T = workloads.C2.extra["timesteps"]
    for step in range(T):
        X = workloads.c2_up_acts(step, device=DEV)
        rows = None
        if step > 0:
            rows = np.sort(np.random.default_rng(70 + step).choice(X.shape[0], 256, replace=False))
            rows[-1] = X.shape[0] - 1
        compare_quantizer(f"c2 up act step {step}", X, 4, seed=0, rows=rows)


@pytest.mark.parametrize("bits", [3, 4])
def test_c3_activations_full(bits):
    Xq, _, _, _ = workloads.c3_inputs(device=DEV)
    compare_quantizer(f"c3 qkv act A{bits}", Xq, bits, seed=0)


def test_c3_weights_outlier_rows():
    _, _, Wq, _ = workloads.c3_inputs(device=DEV)
    compare_quantizer("c3 qkv weights W2", Wq, 2, seed=0, weights=True)


def test_c4_down_sampled_rows():
    # the full video-DiT down-projection input in the launch configuration the benchmark times
    fr, tpf, txt = 21, 30 * 52, 512
    X = workloads.video_acts(fr * tpf, txt, 13824, 4, fr, workloads.C4.data_seed, 1, device=DEV)
    rows = np.sort(np.random.default_rng(44).choice(X.shape[0], 4096, replace=False))
    rows[-1] = X.shape[0] - 1                     # include the ragged tail
    compare_quantizer("c4 down act sampled", X, 4, seed=0, rows=rows)
    # and with the paper's block-size rule (512 for d = 13824)
    compare_quantizer("c4 down act sampled, h=512", X, 4, seed=0, rows=rows, h=512)


def test_c4_up_a6_sampled_rows():
    # the video recipe's 6-bit activations (W4A6) on the full up-projection input
    fr, tpf, txt = 21, 30 * 52, 512
    X = workloads.video_acts(fr * tpf, txt, 5120, 4, fr, workloads.C4.data_seed, 0, device=DEV)
    rows = np.sort(np.random.default_rng(48).choice(X.shape[0], 2048, replace=False))
    rows[-1] = X.shape[0] - 1
    compare_quantizer("c4 up act sampled A6", X, 6, seed=0, rows=rows)
    compare_quantizer("c4 up act sampled A6, h=1024", X, 6, seed=0, rows=rows, h=1024)


def test_c4_up_paper_block_rule_sampled_rows():
    fr, tpf, txt = 21, 30 * 52, 512
    X = workloads.video_acts(fr * tpf, txt, 5120, 4, fr, workloads.C4.data_seed, 0, device=DEV)
    rows = np.sort(np.random.default_rng(47).choice(X.shape[0], 4096, replace=False))
    rows[-1] = X.shape[0] - 1
    compare_quantizer("c4 up act sampled, h=1024", X, 4, seed=0, rows=rows, h=1024)


def test_c4_up_weights_sampled_rows():
    W = workloads.gaussian_weights(13824, 5120, 0.015, workloads.C4.data_seed, 0, device=DEV)
    rows = np.sort(np.random.default_rng(45).choice(W.shape[0], 2048, replace=False))
    compare_quantizer("c4 up weights sampled", W, 4, seed=0, weights=True, rows=rows)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_zero_rows(bits):
    X = _randn_bf16(9, 256, seed=3)
    X[2] = 0
    X[7] = 0
    codes, norms = quantize_gpu(X, bits)
    labels = oracle.unpack_codes(codes.cpu().numpy(), bits, 256)
    gc = oracle.from_labels(labels, bits)
    assert norms[2].item() == 0.0 and norms[7].item() == 0.0
    # u = 0 sits on the middle threshold: the upper level, index 2^(b-1), stored as label 0
    assert np.all(gc[2] == 1 << (bits - 1)) and np.all(gc[7] == 1 << (bits - 1))
    assert np.all(labels[2] == 0) and np.all(labels[7] == 0)
    cw, nw = quantize_gpu(X, bits, weights=True)
    assert nw[2].item() == 0.0


@pytest.mark.parametrize("bits", [2, 4])
def test_power_of_two_scaling_is_exact(bits):
    # codes depend only on the direction; the norm scales exactly (eps = 0 so nothing is added)
    X = _randn_bf16(33, 3072, seed=5)
    c0, n0 = quantize_gpu(X, bits, eps=0.0)
    for k in (-6, 5):
        ck, nk = quantize_gpu((X.float() * 2.0 ** k).to(torch.bfloat16), bits, eps=0.0)
        assert torch.equal(ck, c0)
        assert torch.equal(nk, n0 * 2.0 ** k)


def test_deterministic():
    X = _randn_bf16(300, 5120, seed=9)
    a = quantize_gpu(X, 4)
    b = quantize_gpu(X, 4)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_plan_from_caller_arrays():
    K = 3072
    g = torch.Generator()
    g.manual_seed(77)
    perm = torch.randperm(K, generator=g).numpy()
    sign = np.where(torch.rand(K, generator=g).numpy() < 0.5, -1, 1)
    plan = oq.rpbh_plan_from_arrays(K, 128, perm, sign)
    oplan = oracle.Plan(d=K, h=128, perm=perm.astype(np.int64), sign=sign.astype(np.float64))
    X, _ = workloads.c1_inputs(device=DEV)
    compare_quantizer("c1 act caller plan", X, 4, plan=plan, oplan=oplan)


@pytest.mark.parametrize("K,h", [(3072, 128), (3072, 1024), (4096, 4096)])
def test_rotation_classes_without_permutation(K, h):
    # Block-RHT (RPBH without the permutation) and, for h = K = 4096, Full RHT (the rotation
    # classes of the paper's ablation, Table 4)
    signs = oq.rpbh_plan(K, h, 0).arrays()[1]
    ident = np.arange(K)
    plan = oq.rpbh_plan_from_arrays(K, h, ident, signs)
    oplan = oracle.Plan(d=K, h=h, perm=ident.astype(np.int64), sign=signs.astype(np.float64))
    X = _randn_bf16(129, K, seed=K + h)
    X[:, 5:37] = X[:, 5:37] * 30          # clustered outlier channels
    for bits in (2, 4):
        compare_quantizer(f"rotation class identity-pi K={K} h={h}", X, bits, plan=plan, oplan=oplan)


def _identity_plans(K, h, seed=0):
    signs = oq.rpbh_plan(K, h, seed).arrays()[1]
    ident = np.arange(K)
    return (oq.rpbh_plan_from_arrays(K, h, ident, signs),
            oracle.Plan(d=K, h=h, perm=ident.astype(np.int64), sign=signs.astype(np.float64)))


# An identity permutation takes the kernel's direct-load path (each lane reads its 32 consecutive
# elements straight from HBM, no LDS staging): every block size, bit width and norm type, with
# ragged row counts.
@pytest.mark.parametrize("K,h,M", [(128, 128, 3), (1024, 128, 131), (2560, 256, 50), (1536, 512, 40),
                                   (5120, 1024, 30), (6144, 2048, 11), (8192, 4096, 6), (16384, 4096, 3),
                                   (13824, 512, 5), (16384, 128, 2)])
@pytest.mark.parametrize("weights", [False, True])
def test_identity_permutation_direct_loads(K, h, M, weights):
    plan, oplan = _identity_plans(K, h, seed=K % 7)
    X = _randn_bf16(M, K, seed=K + 3 * h + M)
    for bits in (4,) if weights else (2, 3, 4, 6):
        compare_quantizer(f"identity-pi K={K} h={h} M={M}", X, bits, weights=weights, plan=plan, oplan=oplan)


def test_identity_permutation_many_group_iterations():
    # enough row groups (64 rows each at K = 256) that every persistent workgroup runs several
    # iterations, alternating its two buffers of block partials; every row checked
    K, M = 256, 100003
    plan, oplan = _identity_plans(K, 128, seed=3)
    X = _randn_bf16(M, K, seed=17)
    compare_quantizer("identity-pi many iterations", X, 4, plan=plan, oplan=oplan)
    plan2, oplan2 = _identity_plans(K, 256, seed=4)
    compare_quantizer("identity-pi many iterations h=256", X, 3, weights=True, plan=plan2, oplan=oplan2)


def test_identity_permutation_strided_rows():
    base = _randn_bf16(41, 3072 + 64, seed=12)
    X = base[:, 32:32 + 3072]            # ldx = 3136, rows start 64 bytes in
    plan, oplan = _identity_plans(3072, 1024, seed=2)
    compare_quantizer("identity-pi strided rows", X, 4, plan=plan, oplan=oplan)


def test_c4_up_block_rht_sampled_rows():
    # Block-RHT on the full up-projection input, in the launch configuration the benchmark's
    # rotation-class comparison times (h = 128 and the paper's rule, h = 1024)
    fr, tpf, txt = 21, 30 * 52, 512
    X = workloads.video_acts(fr * tpf, txt, 5120, 4, fr, workloads.C4.data_seed, 0, device=DEV)
    rows = np.sort(np.random.default_rng(49).choice(X.shape[0], 2048, replace=False))
    rows[-1] = X.shape[0] - 1
    for h in (128, 1024):
        plan, oplan = _identity_plans(5120, h, seed=0)
        compare_quantizer(f"c4 up act sampled, Block-RHT h={h}", X, 4, rows=rows, plan=plan, oplan=oplan)


def test_strided_rows():
    base = _randn_bf16(40, 3072 + 64, seed=11)
    X = base[:, 32:32 + 3072]            # ldx = 3136, rows start 64 bytes in
    assert X.stride(0) == 3136
    compare_quantizer("strided rows", X, 4, seed=1)


def test_zero_row_count_is_noop():
    X = torch.empty((0, 256), dtype=torch.bfloat16, device=DEV)
    codes, norms = quantize_gpu(X, 4)
    assert codes.shape == (0, 128) and norms.shape == (0,)


@pytest.mark.parametrize("bits", [2, 3, 4, 6])
def test_sign_symmetry(bits):
    # the codebook is antisymmetric and RPBH linear: code(-x) = 2^b - 1 - code(x) off near-ties,
    # the same norm
    X = _randn_bf16(65, 3072, seed=21)
    c_pos, n_pos = quantize_gpu(X, bits)
    c_neg, n_neg = quantize_gpu(-X, bits)
    lp = oracle.unpack_codes(c_pos.cpu().numpy(), bits, 3072)
    ln = oracle.unpack_codes(c_neg.cpu().numpy(), bits, 3072)
    gp, gn = oracle.from_labels(lp, bits), oracle.from_labels(ln, bits)
    ocb = oracle.lloydmax_codebook(bits, 3072)
    _, _, U = oracle.quantize_act(to_f64(X), oracle.rpbh_plan(3072, 128, 0), ocb)
    near = oracle.near_tie_mask(U, ocb.thresholds, 1e-5)
    bad = int(np.sum((gn != (1 << bits) - 1 - gp) & ~near))
    # in the stored labels the mirror flips the sign bit only
    bad += int(np.sum((ln != (lp ^ (1 << (bits - 1)))) & ~near))
    log_stats(f"sign symmetry b={bits}", near_ties=int(near.sum()), mismatches_off_tie=bad)
    assert bad == 0
    assert torch.equal(n_pos, n_neg)


def test_zero_row_gives_zero_output_row():
    K, N = 1024, 300
    X = _randn_bf16(5, K, seed=31)
    X[3] = 0
    W = _randn_bf16(N, K, seed=32, scale=0.02)
    plan = oq.rpbh_plan(K, 128, 0)
    cb = oq.lloydmax_codebook(4, K)
    wc, wn = oq.quantize_weights_offline(plan, cb, W)
    xc, xn = oq.rpbh_quantize_act(plan, cb, X)
    Y = oq.orbit_qlinear(cb, xc, xn, cb, wc, wn)
    torch.cuda.synchronize()
    assert torch.all(Y[3] == 0) and torch.all(Y[[0, 1, 2, 4]].abs().sum(dim=1) > 0)


@pytest.mark.parametrize("h", [128, 1024])
@pytest.mark.parametrize("weights", [False, True])
def test_extreme_coordinates(h, weights):
    # Rows whose rotated image is (up to bf16 rounding of the input) a single coordinate of
    # magnitude ||x||: the normalized coordinate reaches +-1 and the encoder looks up the last
    # cells at both ends of its table, while every other coordinate sits at the middle
    # threshold's cell.  Built with the oracle's inverse RPBH, at magnitudes from 2^-60 to 2^60,
    # plus the same rows with small noise added.
    K, seed = 3072, 5
    op = oracle.rpbh_plan(K, h, seed)
    idx = [0, 1, 127, 128, 1023, 1024, 2047, 3071]
    E = np.zeros((2 * len(idx), K))
    for r, i in enumerate(idx):
        E[2 * r, i], E[2 * r + 1, i] = 1.0, -1.0
    base = oracle.rpbh_inverse(E, op)
    rows = [base * 2.0 ** s for s in (-60, -10, 0, 10, 60)]
    noisy = base + 1e-3 * np.random.default_rng(3).standard_normal(base.shape)
    X = torch.from_numpy(np.concatenate(rows + [noisy]).astype(np.float32)).to(torch.bfloat16).to(DEV)
    for bits in (4,) if weights else (2, 3, 4, 6):
        compare_quantizer(f"extreme coordinates h={h}", X, bits, seed=seed, weights=weights, h=h, oplan=op)
