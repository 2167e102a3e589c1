"""OrbitQuant quantized linear layer on MI355X (gfx950): Python binding of liborbitquant.so.

The binding only marshals arguments: it allocates outputs with torch on the input's device,
passes raw pointers and torch's current HIP stream to the C ABI (include/orbitquant.h), and
raises on any non-zero status.  Every step of the hot path runs in the library's kernels;
there is no fallback: if the library is missing, importing the functions that need it raises.

    plan = rpbh_plan(d, h=128, seed=0)                         # Sec. 4.4, Eq. (9)
    cb_w, cb_a = lloydmax_codebook(4, d), lloydmax_codebook(4, d)   # Sec. 3.2, Eqs. (2)-(3)
    w_codes, w_norm = quantize_weights_offline(plan, cb_w, W)  # Sec. 4.2, Eqs. (4)-(6)
    x_codes, x_norm = rpbh_quantize_act(plan, cb_a, X)          # Sec. 4.3, Eqs. (7)-(8)
    Y = orbit_qlinear(cb_a, x_codes, x_norm, cb_w, w_codes, w_norm)   # Y ~= X W^T
"""

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liborbitquant.so")

ORBIT_OK, ORBIT_EINVAL, ORBIT_EUNSUPPORTED, ORBIT_ENOMEM, ORBIT_EHIP, ORBIT_EINTERNAL = range(6)
_STATUS_NAMES = {1: "EINVAL", 2: "EUNSUPPORTED", 3: "ENOMEM", 4: "EHIP", 5: "EINTERNAL"}

# Every symbol the C header declares, with its ctypes signature.
_c_void_p, _i64, _i32, _u64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
SIGNATURES = {
    "orbit_last_error": (ctypes.c_char_p, []),
    "orbit_version": (ctypes.c_char_p, []),
    "rpbh_plan": (ctypes.c_int, [_i64, _i32, _u64, ctypes.POINTER(_c_void_p)]),
    "rpbh_plan_from_arrays": (ctypes.c_int, [_i64, _i32, _c_void_p, _c_void_p, ctypes.POINTER(_c_void_p)]),
    "rpbh_plan_get": (ctypes.c_int, [_c_void_p, ctypes.POINTER(_i64), ctypes.POINTER(_i32), _c_void_p, _c_void_p]),
    "rpbh_plan_upload": (ctypes.c_int, [_c_void_p]),
    "rpbh_plan_destroy": (None, [_c_void_p]),
    "lloydmax_codebook": (ctypes.c_int, [_i32, _i64, ctypes.POINTER(_c_void_p)]),
    "lloydmax_codebook_get": (ctypes.c_int, [_c_void_p, ctypes.POINTER(_i32), ctypes.POINTER(_i64),
                                             _c_void_p, _c_void_p, _c_void_p]),
    "lloydmax_codebook_upload": (ctypes.c_int, [_c_void_p]),
    "lloydmax_codebook_destroy": (None, [_c_void_p]),
    "quantize_weights_offline": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i64,
                                                ctypes.c_float, _c_void_p, _c_void_p, _c_void_p]),
    "rpbh_quantize_act": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _i64, _i64,
                                         ctypes.c_float, _c_void_p, _c_void_p, _c_void_p]),
    "orbit_qlinear": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _c_void_p,
                                     _c_void_p, _i64, _i64, _c_void_p, _i64, _c_void_p]),
    "orbit_qlinear_ex": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _c_void_p,
                                        _c_void_p, _i64, _i64, _c_void_p, _i32, _i32, _c_void_p, _i64,
                                        _c_void_p]),
    "orbit_qlinear_workspace_size": (ctypes.c_int, [_i64, _i64, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "orbit_qlinear_schedule": (ctypes.c_int, [_i64, _i64, _i64, ctypes.POINTER(_i64), ctypes.POINTER(_i32)]),
    "orbit_qlinear_ws": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _c_void_p,
                                        _c_void_p, _i64, _i64, _c_void_p, _i32, _i32, _c_void_p, _i64,
                                        _c_void_p, ctypes.c_size_t, _c_void_p]),
    "orbit_qlinear_noalloc": (ctypes.c_int, [_c_void_p, _c_void_p, _c_void_p, _i64, _c_void_p, _c_void_p,
                                             _c_void_p, _i64, _i64, _c_void_p, _i32, _i32, _c_void_p, _i64,
                                             _c_void_p]),
    "adaln_int4_quantize_weights": (ctypes.c_int, [_c_void_p, _i64, _i64, _i64, _c_void_p, _c_void_p, _c_void_p]),
    "adaln_int4_linear": (ctypes.c_int, [_c_void_p, _i64, _i64, _c_void_p, _c_void_p, _i64, _i64, _c_void_p,
                                         _c_void_p, _i64, _c_void_p]),
}

ORBIT_ACT_NONE, ORBIT_ACT_GELU = 0, 1
ORBIT_OUT_F32, ORBIT_OUT_BF16 = 0, 1

_lib = None


class OrbitError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with ORBIT_{_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built (run paper_2607_02461_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_02461_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def _check(fn: str, status: int):
    if status != ORBIT_OK:
        raise OrbitError(fn, status, lib().orbit_last_error().decode())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


class Plan:
    """Handle of an RPBH plan (perm + signs + block size) for one input dimension."""

    def __init__(self, handle):
        self._h = handle

    @property
    def handle(self):
        return self._h

    def _get(self):
        d, h = _i64(), _i32()
        _check("rpbh_plan_get", lib().rpbh_plan_get(self._h, ctypes.byref(d), ctypes.byref(h), None, None))
        return d.value, h.value

    @property
    def d(self):
        return self._get()[0]

    @property
    def h(self):
        return self._get()[1]

    def upload(self, device=None):
        """Copies the plan's device tables to `device` (default: the current one), which device
        calls there need; creation did this for the device current at the time."""
        with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
            _check("rpbh_plan_upload", lib().rpbh_plan_upload(self._h))
        return self

    def arrays(self):
        """(perm int32 [d], sign int8 [d]) as numpy arrays."""
        d = self.d
        perm = np.empty(d, dtype=np.int32)
        sign = np.empty(d, dtype=np.int8)
        _check("rpbh_plan_get", lib().rpbh_plan_get(self._h, None, None, perm.ctypes.data, sign.ctypes.data))
        return perm, sign

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.rpbh_plan_destroy(self._h)
            self._h = None


class Codebook:
    """Handle of a Lloyd-Max codebook C^(d,b)."""

    def __init__(self, handle):
        self._h = handle
        b, d = _i32(), _i64()
        _check("lloydmax_codebook_get", lib().lloydmax_codebook_get(handle, ctypes.byref(b), ctypes.byref(d),
                                                                     None, None, None))
        self.bits, self.d = b.value, d.value
        n = 1 << self.bits
        self.levels = np.empty(n, dtype=np.float64)
        self.thresholds = np.empty(n - 1, dtype=np.float64)
        self.lut_bf16 = np.empty(n, dtype=np.uint16)
        _check("lloydmax_codebook_get", lib().lloydmax_codebook_get(handle, None, None, self.levels.ctypes.data,
                                                                     self.thresholds.ctypes.data,
                                                                     self.lut_bf16.ctypes.data))

    @property
    def handle(self):
        return self._h

    def upload(self, device=None):
        """Copies the encoder table to `device` (default: the current one), as Plan.upload."""
        with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
            _check("lloydmax_codebook_upload", lib().lloydmax_codebook_upload(self._h))
        return self

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.lloydmax_codebook_destroy(self._h)
            self._h = None


def rpbh_plan(d: int, h: int = 128, seed: int = 0) -> Plan:
    out = _c_void_p()
    _check("rpbh_plan", lib().rpbh_plan(d, h, seed, ctypes.byref(out)))
    return Plan(out)


def rpbh_plan_from_arrays(d: int, h: int, perm, sign) -> Plan:
    perm = np.ascontiguousarray(perm, dtype=np.int32)
    sign = np.ascontiguousarray(sign, dtype=np.int8)
    if perm.shape != (d,) or sign.shape != (d,):
        raise ValueError("perm and sign must have d entries")
    out = _c_void_p()
    _check("rpbh_plan_from_arrays", lib().rpbh_plan_from_arrays(d, h, perm.ctypes.data, sign.ctypes.data,
                                                                 ctypes.byref(out)))
    return Plan(out)


def lloydmax_codebook(bits: int, d: int) -> Codebook:
    out = _c_void_p()
    _check("lloydmax_codebook", lib().lloydmax_codebook(bits, d, ctypes.byref(out)))
    return Codebook(out)


def code_bytes(K: int, bits: int) -> int:
    return K * bits // 8


def _rows(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a tensor on a GPU")
    if t.dim() != 2 or t.dtype != torch.bfloat16 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D bf16 tensor with contiguous rows")
    return t.shape[0], t.shape[1], t.stride(0)


def _expect(t: torch.Tensor, name: str, dtype: torch.dtype, shape: tuple, device: torch.device):
    """The kernels address buffers from their sizes alone, so every tensor handed to them must have
    exactly the documented dtype and shape, dense rows, and sit on the device of the call."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the call runs on {device}")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)}{'' if t.is_contiguous() else ' (not contiguous)'}")


def quantize_weights_offline(plan: Plan, cb_w: Codebook, W: torch.Tensor, eps: float = 1e-10,
                             codes: torch.Tensor = None, norms: torch.Tensor = None):
    """Offline weight pass: returns (codes uint8 [N, K*b/8], r' bf16 [N])."""
    N, K, ldw = _rows(W, "W")
    if codes is None:
        codes = torch.empty((N, code_bytes(K, cb_w.bits)), dtype=torch.uint8, device=W.device)
    if norms is None:
        norms = torch.empty((N,), dtype=torch.bfloat16, device=W.device)
    _expect(codes, "codes", torch.uint8, (N, code_bytes(K, cb_w.bits)), W.device)
    _expect(norms, "norms", torch.bfloat16, (N,), W.device)
    with torch.cuda.device(W.device):
        _check("quantize_weights_offline", lib().quantize_weights_offline(
            plan.handle, cb_w.handle, _ptr(W), N, K, ldw, eps, _ptr(codes), _ptr(norms), _stream(W)))
    return codes, norms


def rpbh_quantize_act(plan: Plan, cb_a: Codebook, X: torch.Tensor, eps: float = 1e-10,
                      codes: torch.Tensor = None, norms: torch.Tensor = None):
    """Online activation quantizer: returns (codes uint8 [M, K*b/8], s fp32 [M])."""
    M, K, ldx = _rows(X, "X")
    if codes is None:
        codes = torch.empty((M, code_bytes(K, cb_a.bits)), dtype=torch.uint8, device=X.device)
    if norms is None:
        norms = torch.empty((M,), dtype=torch.float32, device=X.device)
    _expect(codes, "codes", torch.uint8, (M, code_bytes(K, cb_a.bits)), X.device)
    _expect(norms, "norms", torch.float32, (M,), X.device)
    with torch.cuda.device(X.device):
        _check("rpbh_quantize_act", lib().rpbh_quantize_act(
            plan.handle, cb_a.handle, _ptr(X), M, K, ldx, eps, _ptr(codes), _ptr(norms), _stream(X)))
    return codes, norms


def _qlinear_operands(cb_a: Codebook, x_codes, x_norm, cb_w: Codebook, w_codes, w_norm):
    if cb_a.d != cb_w.d:
        raise ValueError(f"codebooks are for d={cb_a.d} and d={cb_w.d}")
    if not isinstance(x_codes, torch.Tensor) or not x_codes.is_cuda or x_codes.dim() != 2:
        raise ValueError("x_codes must be a 2-D tensor on a GPU")
    if not isinstance(w_codes, torch.Tensor) or w_codes.dim() != 2:
        raise ValueError("w_codes must be a 2-D tensor")
    K, dev = cb_a.d, x_codes.device
    M, N = x_codes.shape[0], w_codes.shape[0]
    _expect(x_codes, "x_codes", torch.uint8, (M, code_bytes(K, cb_a.bits)), dev)
    _expect(x_norm, "x_norm", torch.float32, (M,), dev)
    _expect(w_codes, "w_codes", torch.uint8, (N, code_bytes(K, cb_w.bits)), dev)
    _expect(w_norm, "w_norm", torch.bfloat16, (N,), dev)
    return M, N, K, dev


def _check_out(out: torch.Tensor, M: int, N: int, dtype: torch.dtype, dev: torch.device):
    if not isinstance(out, torch.Tensor) or out.device != dev:
        raise ValueError(f"out must be a tensor on {dev}")
    if out.dim() != 2 or tuple(out.shape) != (M, N) or out.stride(1) != 1 or out.dtype != dtype:
        raise ValueError(f"out must be a 2-D {dtype} tensor of shape ({M}, {N}) with contiguous rows")
    if M > 1 and out.stride(0) < N:
        raise ValueError("out rows overlap (stride(0) < N)")


def orbit_qlinear(cb_a: Codebook, x_codes: torch.Tensor, x_norm: torch.Tensor, cb_w: Codebook,
                  w_codes: torch.Tensor, w_norm: torch.Tensor, out: torch.Tensor = None) -> torch.Tensor:
    """Quantized layer on codes: Y fp32 [M, N] = diag(s) La[Xc] Lw[Wc]^T diag(r')."""
    M, N, K, dev = _qlinear_operands(cb_a, x_codes, x_norm, cb_w, w_codes, w_norm)
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=dev)
    _check_out(out, M, N, torch.float32, dev)
    with torch.cuda.device(dev):
        _check("orbit_qlinear", lib().orbit_qlinear(
            cb_a.handle, _ptr(x_codes), _ptr(x_norm), M, cb_w.handle, _ptr(w_codes), _ptr(w_norm), N, K,
            _ptr(out), max(out.stride(0), N), _stream(x_codes)))
    return out


def orbit_qlinear_ex(cb_a: Codebook, x_codes: torch.Tensor, x_norm: torch.Tensor, cb_w: Codebook,
                     w_codes: torch.Tensor, w_norm: torch.Tensor, bias: torch.Tensor = None, gelu: bool = False,
                     out_dtype: torch.dtype = torch.float32, out: torch.Tensor = None) -> torch.Tensor:
    """The quantized layer with bias, GELU and the output type fused into the GEMM's epilogue."""
    M, N, K, dev = _qlinear_operands(cb_a, x_codes, x_norm, cb_w, w_codes, w_norm)
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=dev)
    _check_out(out, M, N, out_dtype, dev)
    if bias is not None:
        _expect(bias, "bias", torch.bfloat16, (N,), dev)
    with torch.cuda.device(dev):
        _check("orbit_qlinear_ex", lib().orbit_qlinear_ex(
            cb_a.handle, _ptr(x_codes), _ptr(x_norm), M, cb_w.handle, _ptr(w_codes), _ptr(w_norm), N, K,
            _ptr(bias) if bias is not None else None, ORBIT_ACT_GELU if gelu else ORBIT_ACT_NONE,
            ORBIT_OUT_BF16 if out_dtype == torch.bfloat16 else ORBIT_OUT_F32, _ptr(out), max(out.stride(0), N),
            _stream(x_codes)))
    return out


def orbit_qlinear_workspace_size(M: int, N: int, K: int, device=None) -> int:
    """Bytes of workspace with which orbit_qlinear_ws splits an M x N x K layer over K on
    `device` (default: the current one); 0 when it would not split."""
    n = ctypes.c_size_t(0)
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        _check("orbit_qlinear_workspace_size", lib().orbit_qlinear_workspace_size(M, N, K, ctypes.byref(n)))
    return n.value


def orbit_qlinear_schedule(M: int, N: int, K: int, device=None):
    """(rows_large, splits): rows [0, rows_large) of an M x N x K layer run on the 256 x 256 kernel,
    the rest on the 128 x 128 kernel split `splits` ways over K when given a workspace."""
    rows, splits = _i64(0), _i32(1)
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        _check("orbit_qlinear_schedule", lib().orbit_qlinear_schedule(M, N, K, ctypes.byref(rows),
                                                                       ctypes.byref(splits)))
    return rows.value, splits.value


def orbit_qlinear_ws(cb_a: Codebook, x_codes: torch.Tensor, x_norm: torch.Tensor, cb_w: Codebook,
                     w_codes: torch.Tensor, w_norm: torch.Tensor, workspace: torch.Tensor, bias: torch.Tensor = None,
                     gelu: bool = False, out_dtype: torch.dtype = torch.float32,
                     out: torch.Tensor = None) -> torch.Tensor:
    """orbit_qlinear_ex with a caller workspace (a contiguous device tensor of any dtype, at least
    orbit_qlinear_workspace_size bytes, used on the current stream) that lets a small layer split
    over K."""
    M, N, K, dev = _qlinear_operands(cb_a, x_codes, x_norm, cb_w, w_codes, w_norm)
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if not isinstance(workspace, torch.Tensor) or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError(f"workspace must be a contiguous tensor on {dev}")
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=dev)
    _check_out(out, M, N, out_dtype, dev)
    if bias is not None:
        _expect(bias, "bias", torch.bfloat16, (N,), dev)
    with torch.cuda.device(dev):
        _check("orbit_qlinear_ws", lib().orbit_qlinear_ws(
            cb_a.handle, _ptr(x_codes), _ptr(x_norm), M, cb_w.handle, _ptr(w_codes), _ptr(w_norm), N, K,
            _ptr(bias) if bias is not None else None, ORBIT_ACT_GELU if gelu else ORBIT_ACT_NONE,
            ORBIT_OUT_BF16 if out_dtype == torch.bfloat16 else ORBIT_OUT_F32, _ptr(out), max(out.stride(0), N),
            _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(x_codes)))
    return out


def orbit_qlinear_noalloc(cb_a: Codebook, x_codes: torch.Tensor, x_norm: torch.Tensor, cb_w: Codebook,
                          w_codes: torch.Tensor, w_norm: torch.Tensor, bias: torch.Tensor = None, gelu: bool = False,
                          out_dtype: torch.dtype = torch.float32, out: torch.Tensor = None) -> torch.Tensor:
    """orbit_qlinear_ws with the K-split's partial sums in the library's own scratch array (32 MiB per
    device): the C call allocates nothing.  Pass `out` to keep the binding from allocating the output.
    Calls on one device must not overlap in time (they share the array)."""
    M, N, K, dev = _qlinear_operands(cb_a, x_codes, x_norm, cb_w, w_codes, w_norm)
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=dev)
    _check_out(out, M, N, out_dtype, dev)
    if bias is not None:
        _expect(bias, "bias", torch.bfloat16, (N,), dev)
    with torch.cuda.device(dev):
        _check("orbit_qlinear_noalloc", lib().orbit_qlinear_noalloc(
            cb_a.handle, _ptr(x_codes), _ptr(x_norm), M, cb_w.handle, _ptr(w_codes), _ptr(w_norm), N, K,
            _ptr(bias) if bias is not None else None, ORBIT_ACT_GELU if gelu else ORBIT_ACT_NONE,
            ORBIT_OUT_BF16 if out_dtype == torch.bfloat16 else ORBIT_OUT_F32, _ptr(out), max(out.stride(0), N),
            _stream(x_codes)))
    return out


def adaln_int4_quantize_weights(W: torch.Tensor, q: torch.Tensor = None, scales: torch.Tensor = None):
    """Offline INT4 round-to-nearest of an AdaLN modulation projection (group 64): returns
    (q uint8 [N, K/2] with code + 8 per nibble, scales fp16 [N, K/64])."""
    N, K, ldw = _rows(W, "W")
    if K % 64:
        raise ValueError("K must be a multiple of 64")
    if q is None:
        q = torch.empty((N, K // 2), dtype=torch.uint8, device=W.device)
    if scales is None:
        scales = torch.empty((N, K // 64), dtype=torch.float16, device=W.device)
    _expect(q, "q", torch.uint8, (N, K // 2), W.device)
    _expect(scales, "scales", torch.float16, (N, K // 64), W.device)
    with torch.cuda.device(W.device):
        _check("adaln_int4_quantize_weights", lib().adaln_int4_quantize_weights(
            _ptr(W), N, K, ldw, _ptr(q), _ptr(scales), _stream(W)))
    return q, scales


def adaln_int4_linear(X: torch.Tensor, q: torch.Tensor, scales: torch.Tensor, bias: torch.Tensor = None,
                      out: torch.Tensor = None) -> torch.Tensor:
    """The AdaLN modulation projection on INT4 weights: Y fp32 [M, N] = X (q * scale)^T (+ bias)."""
    M, K, ldx = _rows(X, "X")
    if K % 64 or not isinstance(q, torch.Tensor) or q.dim() != 2:
        raise ValueError("K must be a multiple of 64 and q a 2-D tensor")
    N, dev = q.shape[0], X.device
    _expect(q, "q", torch.uint8, (N, K // 2), dev)
    _expect(scales, "scales", torch.float16, (N, K // 64), dev)
    if bias is not None:
        _expect(bias, "bias", torch.bfloat16, (N,), dev)
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=dev)
    _check_out(out, M, N, torch.float32, dev)
    with torch.cuda.device(dev):
        _check("adaln_int4_linear", lib().adaln_int4_linear(
            _ptr(X), M, ldx, _ptr(q), _ptr(scales), N, K, _ptr(bias) if bias is not None else None,
            _ptr(out), max(out.stride(0), N), _stream(X)))
    return out


__all__ = ["adaln_int4_quantize_weights", "adaln_int4_linear", "rpbh_plan", "rpbh_plan_from_arrays", "lloydmax_codebook", "quantize_weights_offline",
           "rpbh_quantize_act", "orbit_qlinear", "orbit_qlinear_ex",
           "orbit_qlinear_workspace_size", "orbit_qlinear_ws", "Plan", "Codebook", "OrbitError", "lib", "LIB_PATH",
           "SIGNATURES", "code_bytes"]
