"""The C-ABI library on the CPU: it loads, exports every declared symbol, its host-side
plan and codebook match the oracle, and device calls reject bad arguments before any
launch (no GPU work is started by these tests)."""

import ctypes
import os
import re

import numpy as np
import torch
import pytest

import oracle
import paper_2607_02461_amd as oq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "orbitquant.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(\w+)\s*\(", src, flags=re.M)) - {"if"})


def test_library_loads_and_exports_every_declared_symbol():
    lib = oq.lib()
    names = declared_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(oq.SIGNATURES), "binding signatures must cover the header exactly"
    assert lib.orbit_version().decode().startswith("orbitquant")


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("d", [16, 64, 3072, 5120, 12288, 13824])
def test_codebook_matches_oracle(bits, d):
    cb = oq.lloydmax_codebook(bits, d)
    ref = oracle.lloydmax_codebook(bits, d)
    assert cb.bits == bits and cb.d == d
    assert np.max(np.abs(cb.levels - ref.levels) / np.abs(ref.levels)) < 1e-12
    assert np.max(np.abs(cb.thresholds - ref.thresholds)) < 1e-12 * np.max(np.abs(ref.levels))
    # exact antisymmetry, middle threshold exactly zero
    assert np.array_equal(cb.levels, -cb.levels[::-1])
    assert cb.thresholds[(1 << bits) // 2 - 1] == 0.0
    # the bf16 image equals the oracle's levels rounded once to 8 significant bits, ties to even
    want = oracle.bf16_bits(oracle.bf16_round(ref.levels))
    assert np.array_equal(cb.lut_bf16, want)


def test_codebook_d3_uniform_and_large_d():
    cb = oq.lloydmax_codebook(3, 3)
    assert np.max(np.abs(cb.levels - (-1 + (2 * np.arange(8) + 1) / 8))) < 1e-13
    big = oq.lloydmax_codebook(2, 10 ** 6)
    assert np.max(np.abs(big.levels[2:] * 1000 - [0.4528, 1.510])) < 6e-4


@pytest.mark.parametrize("seed", [0, 1, 2, 12345, 2 ** 63 + 7])
@pytest.mark.parametrize("d,h", [(3072, 128), (5120, 128), (13824, 128), (24, 8), (1920, 0)])
def test_plan_matches_oracle(seed, d, h):
    p = oq.rpbh_plan(d, h, seed)
    perm, sign = p.arrays()
    hh = h if h else (d & -d)
    ref = oracle.rpbh_plan(d, hh, seed)
    assert p.d == d and p.h == hh
    assert np.array_equal(perm, ref.perm)
    assert np.array_equal(sign.astype(np.float64), ref.sign)


def test_plan_block_size_rule():
    # Sec. 4.4: h is the largest power of two dividing d
    for d, h in ((3072, 1024), (5120, 1024), (12288, 4096), (13824, 512), (1920, 128)):
        assert oq.rpbh_plan(d, 0, 0).h == h


def test_plan_from_arrays_roundtrip_and_validation():
    perm = np.random.default_rng(0).permutation(256).astype(np.int32)
    sign = np.where(np.random.default_rng(1).random(256) < 0.5, -1, 1).astype(np.int8)
    p = oq.rpbh_plan_from_arrays(256, 128, perm, sign)
    got_perm, got_sign = p.arrays()
    assert np.array_equal(got_perm, perm) and np.array_equal(got_sign, sign)
    bad = perm.copy()
    bad[3] = bad[4]
    with pytest.raises(oq.OrbitError) as e:
        oq.rpbh_plan_from_arrays(256, 128, bad, sign)
    assert e.value.status == oq.ORBIT_EINVAL
    bad_sign = sign.copy()
    bad_sign[0] = 0
    with pytest.raises(oq.OrbitError):
        oq.rpbh_plan_from_arrays(256, 128, perm, bad_sign)


@pytest.mark.parametrize("d,h", [(100, 3), (96, 64), (0, 1), (-5, 1)])
def test_plan_rejects_bad_arguments(d, h):
    with pytest.raises(oq.OrbitError) as e:
        oq.rpbh_plan(d, h, 0)
    assert e.value.status == oq.ORBIT_EINVAL


@pytest.mark.parametrize("bits,d", [(0, 64), (7, 64), (2, 2), (3, 0)])
def test_codebook_rejects_bad_arguments(bits, d):
    with pytest.raises(oq.OrbitError) as e:
        oq.lloydmax_codebook(bits, d)
    assert e.value.status == oq.ORBIT_EINVAL


def _status(fn, *args):
    st = fn(*args)
    return st, oq.lib().orbit_last_error().decode()


def test_device_calls_validate_before_launch():
    lib = oq.lib()
    p = oq.rpbh_plan(256, 128, 0)
    p_h64 = oq.rpbh_plan(256, 64, 0)
    cb4 = oq.lloydmax_codebook(4, 256)
    cb1 = oq.lloydmax_codebook(1, 256)
    cb_other = oq.lloydmax_codebook(4, 512)
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: every case fails validation first
    # K mismatch
    st, msg = _status(lib.rpbh_quantize_act, p.handle, cb_other.handle, fake, 4, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL and "K=" in msg
    # unsupported block size and bit-width
    st, _ = _status(lib.rpbh_quantize_act, p_h64.handle, cb4.handle, fake, 4, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EUNSUPPORTED
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb1.handle, fake, 4, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EUNSUPPORTED
    p_h8k, cb_8k = oq.rpbh_plan(8192, 8192, 0), oq.lloydmax_codebook(4, 8192)   # above the 4096 limit
    st, msg = _status(lib.rpbh_quantize_act, p_h8k.handle, cb_8k.handle, fake, 4, 8192, 8192, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EUNSUPPORTED and "h=8192" in msg
    # bad stride, negative rows, bad eps, null pointers, misalignment
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb4.handle, fake, 4, 256, 100, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb4.handle, fake, -1, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb4.handle, fake, 4, 256, 256, float("nan"), fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb4.handle, null, 4, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.quantize_weights_offline, p.handle, cb4.handle, ctypes.c_void_p((1 << 20) + 2), 4, 256,
                    256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.rpbh_quantize_act, None, cb4.handle, fake, 4, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EINVAL
    # zero rows is a successful no-op (no device touched)
    st, _ = _status(lib.rpbh_quantize_act, p.handle, cb4.handle, null, 0, 256, 256, 1e-10, null, null, null)
    assert st == oq.ORBIT_OK
    st, _ = _status(lib.quantize_weights_offline, p.handle, cb4.handle, null, 0, 256, 256, 1e-10, null, null, null)
    assert st == oq.ORBIT_OK
    # qlinear
    st, _ = _status(lib.orbit_qlinear, cb4.handle, fake, fake, 4, cb_other.handle, fake, fake, 4, 256, fake, 4, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.orbit_qlinear, cb4.handle, fake, fake, 4, cb4.handle, fake, fake, 8, 256, fake, 4, null)
    assert st == oq.ORBIT_EINVAL   # ldy < N
    st, _ = _status(lib.orbit_qlinear, cb1.handle, fake, fake, 4, cb4.handle, fake, fake, 4, 256, fake, 4, null)
    assert st == oq.ORBIT_EUNSUPPORTED
    st, _ = _status(lib.orbit_qlinear, cb4.handle, null, null, 0, cb4.handle, null, null, 4, 256, null, 4, null)
    assert st == oq.ORBIT_OK
    st, _ = _status(lib.orbit_qlinear, cb4.handle, null, null, 4, cb4.handle, null, null, 0, 256, null, 0, null)
    assert st == oq.ORBIT_OK
    assert lib.orbit_last_error().decode() == ""


def test_qlinear_workspace_calls_validate_before_launch():
    lib = oq.lib()
    cb4, cb_other = oq.lloydmax_codebook(4, 256), oq.lloydmax_codebook(4, 512)
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    n = ctypes.c_size_t(7)
    # the size query: argument errors before any device is asked; an empty layer needs nothing
    st, _ = _status(lib.orbit_qlinear_workspace_size, 4, 4, 256, None)
    assert st == oq.ORBIT_EINVAL
    for M, N, K in ((-1, 4, 256), (4, -1, 256), (4, 4, 0), (4, 4, 100), (4, 4, (1 << 30) + 64)):
        st, _ = _status(lib.orbit_qlinear_workspace_size, M, N, K, ctypes.byref(n))
        assert st == oq.ORBIT_EINVAL and n.value == 0
    for M, N in ((0, 3072), (256, 0)):
        n.value = 7
        st, _ = _status(lib.orbit_qlinear_workspace_size, M, N, 3072, ctypes.byref(n))
        assert st == oq.ORBIT_OK and n.value == 0
    if not torch.cuda.is_available():
        # a real layer asks the device for its compute units: without one, ORBIT_EHIP and 0 bytes
        n.value = 7
        st, msg = _status(lib.orbit_qlinear_workspace_size, 256, 3072, 3072, ctypes.byref(n))
        assert st == oq.ORBIT_EHIP and n.value == 0 and msg
    # the layer with a workspace validates as orbit_qlinear_ex does
    ws = ctypes.c_size_t(1 << 20)
    st, _ = _status(lib.orbit_qlinear_ws, cb4.handle, fake, fake, 4, cb_other.handle, fake, fake, 4, 256, null,
                    0, 0, fake, 4, fake, ws, null)
    assert st == oq.ORBIT_EINVAL
    st, _ = _status(lib.orbit_qlinear_ws, cb4.handle, fake, fake, 4, cb4.handle, fake, fake, 4, 256, null,
                    2, 0, fake, 4, fake, ws, null)
    assert st == oq.ORBIT_EINVAL   # unknown act
    st, _ = _status(lib.orbit_qlinear_ws, cb4.handle, null, null, 0, cb4.handle, null, null, 4, 256, null,
                    0, 0, null, 4, null, ctypes.c_size_t(0), null)
    assert st == oq.ORBIT_OK
    assert lib.orbit_last_error().decode() == ""


def test_device_calls_reject_grids_beyond_32_bits():
    lib = oq.lib()
    p = oq.rpbh_plan(256, 128, 0)
    cb = oq.lloydmax_codebook(4, 256)
    null, fake = ctypes.c_void_p(0), ctypes.c_void_p(1 << 20)
    st, msg = _status(lib.rpbh_quantize_act, p.handle, cb.handle, fake, 1 << 31, 256, 256, 1e-10, fake, fake, null)
    assert st == oq.ORBIT_EUNSUPPORTED and "M=" in msg
    st, msg = _status(lib.orbit_qlinear, cb.handle, fake, fake, 1 << 32, cb.handle, fake, fake, 16, 256, fake, 16, null)
    assert st == oq.ORBIT_EUNSUPPORTED
    st, msg = _status(lib.orbit_qlinear, cb.handle, fake, fake, 1 << 30, cb.handle, fake, fake, 1 << 30, 256, fake,
                      1 << 30, null)
    assert st == oq.ORBIT_EUNSUPPORTED and "grid" in msg


def test_binding_rejects_host_tensors():
    # the wrappers hand raw pointers to device kernels: tensors that are not on a GPU never get there
    import torch
    plan, cb = oq.rpbh_plan(256, 128, 0), oq.lloydmax_codebook(4, 256)
    X = torch.zeros((4, 256), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        oq.rpbh_quantize_act(plan, cb, X)
    with pytest.raises(ValueError):
        oq.quantize_weights_offline(plan, cb, X)
    xc, xn = torch.zeros((4, 128), dtype=torch.uint8), torch.ones(4)
    wc, wn = torch.zeros((8, 128), dtype=torch.uint8), torch.ones(8, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        oq.orbit_qlinear(cb, xc, xn, cb, wc, wn)
    with pytest.raises(ValueError):
        oq.orbit_qlinear_ex(cb, xc, xn, cb, wc, wn, gelu=True)


def test_binding_tensor_contract():
    # the shape/dtype/layout checks every operand passes before a launch
    import torch
    dev = torch.device("cpu")
    t = torch.zeros((4, 128), dtype=torch.uint8)
    oq._expect(t, "t", torch.uint8, (4, 128), dev)
    for bad in (t.to(torch.int16), t[:, :64], torch.zeros((128, 4), dtype=torch.uint8).t(),
                torch.zeros((4, 129), dtype=torch.uint8), torch.zeros((5, 128), dtype=torch.uint8)):
        with pytest.raises(ValueError):
            oq._expect(bad, "t", torch.uint8, (4, 128), dev)
    oq._check_out(torch.zeros((4, 10)), 4, 10, torch.float32, dev)
    oq._check_out(torch.zeros((4, 12))[:, :10], 4, 10, torch.float32, dev)   # padded rows
    for bad in (torch.zeros((10, 4)).t(), torch.zeros((4, 11)), torch.zeros((4, 10), dtype=torch.bfloat16),
                torch.zeros((40,)).as_strided((4, 10), (5, 1))):              # overlapping rows
        with pytest.raises(ValueError):
            oq._check_out(bad, 4, 10, torch.float32, dev)


def test_adaln_calls_validate_before_launch():
    lib = oq.lib()
    null, fake = ctypes.c_void_p(0), ctypes.c_void_p(1 << 20)
    cases = [
        (lib.adaln_int4_quantize_weights, (fake, 4, 100, 104, fake, fake, null), oq.ORBIT_EINVAL),   # K % 64
        (lib.adaln_int4_quantize_weights, (fake, 4, 128, 100, fake, fake, null), oq.ORBIT_EINVAL),   # ldw < K
        (lib.adaln_int4_quantize_weights, (fake, -1, 128, 128, fake, fake, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_quantize_weights, (null, 4, 128, 128, fake, fake, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_quantize_weights, (ctypes.c_void_p((1 << 20) + 8), 4, 128, 128, fake, fake, null),
         oq.ORBIT_EINVAL),                                                                            # misaligned W
        (lib.adaln_int4_linear, (fake, 2, 128, fake, fake, 16, 96, null, fake, 16, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_linear, (fake, 2, 120, fake, fake, 16, 128, null, fake, 16, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_linear, (fake, 2, 128, fake, fake, 16, 128, null, fake, 8, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_linear, (fake, 2, 128, null, fake, 16, 128, null, fake, 16, null), oq.ORBIT_EINVAL),
        (lib.adaln_int4_linear, (fake, 1 << 20, 128, fake, fake, 16, 128, null, fake, 16, null),
         oq.ORBIT_EUNSUPPORTED),
        (lib.adaln_int4_linear, (fake, 2, 32768, fake, fake, 16, 32768, null, fake, 16, null),
         oq.ORBIT_EUNSUPPORTED),                                                                      # K > 16384
        (lib.adaln_int4_quantize_weights, (fake, 1 << 30, 1 << 20, 1 << 20, fake, fake, null),
         oq.ORBIT_EUNSUPPORTED),                                                                      # grid > 2^31
    ]
    for fn, args, want in cases:
        st, msg = _status(fn, *args)
        assert st == want, (fn.__name__, args, st, msg)
    # empty calls succeed without touching the device
    assert _status(lib.adaln_int4_linear, null, 0, 128, null, null, 16, 128, null, null, 16, null)[0] == oq.ORBIT_OK
    assert _status(lib.adaln_int4_quantize_weights, null, 0, 128, 128, null, null, null)[0] == oq.ORBIT_OK


def test_quantizer_rejects_row_gaps_of_2_23_elements():
    # the staging offsets use 24-bit products of the byte gap between rows: ld - K must stay
    # below 2^23 elements, for activations and weights alike (checked before any device work)
    lib = oq.lib()
    p = oq.rpbh_plan(256, 128, 0)
    cb = oq.lloydmax_codebook(4, 256)
    null, fake = ctypes.c_void_p(0), ctypes.c_void_p(1 << 20)
    st, msg = _status(lib.rpbh_quantize_act, p.handle, cb.handle, fake, 4, 256, 256 + (1 << 23), 1e-10, fake, fake,
                      null)
    assert st == oq.ORBIT_EUNSUPPORTED and "stride" in msg
    st, msg = _status(lib.quantize_weights_offline, p.handle, cb.handle, fake, 4, 256, 256 + (1 << 23), 1e-10, fake,
                      fake, null)
    assert st == oq.ORBIT_EUNSUPPORTED and "stride" in msg


def test_qlinear_schedule_validates_and_needs_a_device():
    lib = oq.lib()
    rows, splits = ctypes.c_int64(5), ctypes.c_int32(5)
    st, _ = _status(lib.orbit_qlinear_schedule, 4, 4, 256, None, ctypes.byref(splits))
    assert st == oq.ORBIT_EINVAL
    for M, N, K in ((-1, 4, 256), (4, -1, 256), (4, 4, 0), (4, 4, 100)):
        st, _ = _status(lib.orbit_qlinear_schedule, M, N, K, ctypes.byref(rows), ctypes.byref(splits))
        assert st == oq.ORBIT_EINVAL and rows.value == 0 and splits.value == 1
    st, _ = _status(lib.orbit_qlinear_schedule, 0, 3072, 3072, ctypes.byref(rows), ctypes.byref(splits))
    assert st == oq.ORBIT_OK and rows.value == 0 and splits.value == 1
    if not torch.cuda.is_available():
        st, msg = _status(lib.orbit_qlinear_schedule, 256, 3072, 3072, ctypes.byref(rows), ctypes.byref(splits))
        assert st == oq.ORBIT_EHIP and msg
