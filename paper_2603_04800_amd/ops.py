"""ctypes binding of libmasq.so (the C ABI declared in include/masq.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  torch is used for device memory, pointers and the current stream.
If the library has not been built this module raises ImportError at import
time; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

from . import _libpath

_LIB_PATH = _libpath.LIB
if not os.path.exists(_LIB_PATH):
    raise ImportError(
        f"{_LIB_PATH} is missing: build the HIP library first "
        "(python -m paper_2603_04800_amd.build)")
_lib = ctypes.CDLL(_LIB_PATH)

F32, BF16 = 0, 1
STATUS = {0: "MASQ_OK", 1: "MASQ_ERR_NULL", 2: "MASQ_ERR_SHAPE", 3: "MASQ_ERR_DTYPE",
          4: "MASQ_ERR_ALIGN", 5: "MASQ_ERR_WORKSPACE", 6: "MASQ_ERR_HIP",
          7: "MASQ_ERR_UNSUPPORTED", 8: "MASQ_ERR_SCRATCH"}

_p, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t

_FUSED_ARGS = [_p, _i32, _p, _p, _p, _p, _p, _p, _i32, _i64, _i64, _i64, _i32, _i32, _p, _i32,
               _p, _sz, _p]
_SIGS = {
    "masq_abi_version": ([], ctypes.c_int),
    "masq_status_str": ([_i32], ctypes.c_char_p),
    "masq_smooth_quant": ([_p, _i32, _p, _p, _i64, _i64, _i32, _p, _p, _p], ctypes.c_int),
    "masq_w8a8_gemm": ([_p, _p, _p, _p, _i64, _i64, _i64, _p, _p, _i32, _p], ctypes.c_int),
    "masq_lowrank_comp": ([_p, _i32, _p, _p, _p, _p, _i32, _i64, _i64, _i64, _i32, _i32, _p,
                           _i32, _p], ctypes.c_int),
    "masq_linear_fused": (_FUSED_ARGS, ctypes.c_int),
    "masq_linear_stage1": (_FUSED_ARGS, ctypes.c_int),
    "masq_linear_stage2": (_FUSED_ARGS, ctypes.c_int),
    "masq_linear_fused_workspace_bytes": ([_i64, _i64, _i64, _i32, _i32], ctypes.c_size_t),
    "masq_linear_fused_noalloc": (_FUSED_ARGS[:16] + [_p], ctypes.c_int),
    "masq_mas_only_linear": ([_p, _i32, _p, _p, _p, _p, _i64, _i64, _i64, _i32, _p, _i32, _p, _sz,
                              _p], ctypes.c_int),
    "masq_mas_only_workspace_bytes": ([_i64, _i64, _i64, _i32], ctypes.c_size_t),
    "masq_w4a8_gemm": ([_p, _p, _p, _p, _i64, _i64, _i64, _p, _p, _i32, _p], ctypes.c_int),
    "masq_linear_fused_w4a8": (_FUSED_ARGS, ctypes.c_int),
    "masq_linear_stage1_w4a8": (_FUSED_ARGS, ctypes.c_int),
    "masq_linear_stage2_w4a8": (_FUSED_ARGS, ctypes.c_int),
    "masq_channel_range": ([_p, _i32, _p, _i64, _i64, _i32, _p, _p], ctypes.c_int),
    "masq_smoothing_factors": ([_p, _p, _i64, _i64, _i32, _p, _p, _p], ctypes.c_int),
    "masq_quantize_weight": ([_p, _p, _i64, _i64, _i32, _p, _p, _p], ctypes.c_int),
    "masq_gather_smoothed": ([_p, _i32, _i64, _i64, _p, _i64, _p, _p, _p], ctypes.c_int),
    "masq_weight_difference": ([_p, _p, _p, _p, _i64, _i64, _p, _p], ctypes.c_int),
    "masq_dgemm": ([_i64, _i64, _i64, _p, _i64, _i64, _p, _i64, _i64, ctypes.c_double, _p, _i64,
                    _p], ctypes.c_int),
    "masq_cholesky": ([_i64, _p, _i64, ctypes.c_double, _p, _p, _p], ctypes.c_int),
    "masq_trsm_right": ([_i64, _i64, _p, _i64, _i32, _p, _i64, _p], ctypes.c_int),
    "masq_jacobi_svd": ([_i64, _i64, _p, _p, _p, _p, _p, _i32, _i32, _p, _p], ctypes.c_int),
    "masq_dequantize_rows": ([_p, _p, _i64, _i64, _p, _p], ctypes.c_int),
    "masq_mae_partials": ([_i64], _i64),
    "masq_mae_sign": ([_p, _p, _i64, _p, _p, _p], ctypes.c_int),
    "masq_mas_gradient": ([_p, _p, _p, _p, _p, _i64, _i64, _i64, _p, _p, _p], ctypes.c_int),
    "masq_mae_loss": ([_p, _i64, _p, _p], ctypes.c_int),
    "masq_adam_log_step": ([_p, _p, _p, _p, _p, _p, _i64, ctypes.c_double, ctypes.c_double,
                            ctypes.c_double, ctypes.c_double, ctypes.c_double, _i64, _p],
                           ctypes.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res

EXPORTED = tuple(_SIGS)


class MasqError(RuntimeError):
    def __init__(self, fn: str, code: int):
        msg = _lib.masq_status_str(code).decode()
        super().__init__(f"{fn}: {msg}")
        self.code = code


def _check(fn: str, code: int):
    if code != 0:
        raise MasqError(fn, code)


def raw():
    """The ctypes library handle (for tests of the C ABI itself)."""
    return _lib


def abi_version() -> int:
    return _lib.masq_abi_version()


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, dtype, name):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")


def smooth_quant(x, modality, inv_smooth, q=None, x_scale=None, stream=None):
    """Per-token smoothing + int8 quantisation -> (q int8 [T][K], x_scale f32 [T])."""
    T, K = x.shape
    _need(modality, torch.int32, "modality")
    _need(inv_smooth, torch.float32, "inv_smooth")
    if q is None:
        q = torch.empty((T, K), dtype=torch.int8, device=x.device)
    if x_scale is None:
        x_scale = torch.empty((T,), dtype=torch.float32, device=x.device)
    _check("masq_smooth_quant", _lib.masq_smooth_quant(
        _ptr(x), _dt(x), _ptr(modality), _ptr(inv_smooth), T, K, inv_smooth.shape[0],
        _ptr(q), _ptr(x_scale), _stream(stream)))
    return q, x_scale


def w8a8_gemm(q, x_scale, wq, w_scale, want_acc=True, out_dtype=torch.float32, stream=None):
    """Shared-weight int8 product -> (acc int32 [T][N] or None, y [T][N] or None)."""
    T, K = q.shape
    N = wq.shape[0]
    acc = torch.empty((T, N), dtype=torch.int32, device=q.device) if want_acc else None
    y = torch.empty((T, N), dtype=out_dtype, device=q.device) if out_dtype is not None else None
    _check("masq_w8a8_gemm", _lib.masq_w8a8_gemm(
        _ptr(q), _ptr(x_scale), _ptr(wq), _ptr(w_scale), T, K, N, _ptr(acc), _ptr(y),
        _dt(y) if y is not None else F32, _stream(stream)))
    return acc, y


def w4a8_gemm(q, x_scale, wq4, w_scale, want_acc=True, out_dtype=torch.float32, stream=None):
    """The same product with the 4-bit shared weight packed two codes per byte
    (uint8 [N][K / 2], layout of :mod:`paper_2603_04800_amd.int4`)."""
    T, K = q.shape
    N = wq4.shape[0]
    _need(wq4, torch.uint8, "wq4")
    if wq4.shape[1] * 2 != K:
        raise ValueError(f"wq4 holds {2 * wq4.shape[1]} codes a row, q has {K} columns")
    acc = torch.empty((T, N), dtype=torch.int32, device=q.device) if want_acc else None
    y = torch.empty((T, N), dtype=out_dtype, device=q.device) if out_dtype is not None else None
    _check("masq_w4a8_gemm", _lib.masq_w4a8_gemm(
        _ptr(q), _ptr(x_scale), _ptr(wq4), _ptr(w_scale), T, K, N, _ptr(acc), _ptr(y),
        _dt(y) if y is not None else F32, _stream(stream)))
    return acc, y


def lowrank_comp(x, modality, inv_smooth, l_down, r_up, y, stream=None):
    """In place: y[t] += (x_t S_m^-1 L1^m) L2^m on non-text rows; returns y."""
    T, K = x.shape
    N = y.shape[1]
    n_mod = inv_smooth.shape[0]
    rank = l_down.shape[1] if l_down is not None and l_down.dim() == 3 else 0
    lr_dt = _dt(l_down) if l_down is not None else F32
    _check("masq_lowrank_comp", _lib.masq_lowrank_comp(
        _ptr(x), _dt(x), _ptr(modality), _ptr(inv_smooth), _ptr(l_down), _ptr(r_up), lr_dt,
        T, K, N, rank, n_mod, _ptr(y), _dt(y), _stream(stream)))
    return y


def channel_range(x, modality, n_mod, stream=None):
    """Per-modality channel ranges R^m [n_mod][K] f32 (calibration, Sec. 4.1)."""
    T, K = x.shape
    _need(modality, torch.int32, "modality")
    out = torch.empty((n_mod, K), dtype=torch.float32, device=x.device)
    _check("masq_channel_range", _lib.masq_channel_range(
        _ptr(x), _dt(x), _ptr(modality), T, K, n_mod, _ptr(out), _stream(stream)))
    return out


def smoothing_factors(range_, w, stream=None):
    """MAS factors from the ranges and the float weight W [K][N] (paper layout):
    (s [n_mod][K], inv_s [n_mod][K]) f32 (Sec. 4.2)."""
    n_mod, K = range_.shape
    _need(range_, torch.float32, "range")
    _need(w, torch.float32, "w")
    s = torch.empty_like(range_)
    inv = torch.empty_like(range_)
    _check("masq_smoothing_factors", _lib.masq_smoothing_factors(
        _ptr(range_), _ptr(w), K, w.shape[1], n_mod, _ptr(s), _ptr(inv), _stream(stream)))
    return s, inv


def quantize_weight(w, smooth_text, bits=8, stream=None):
    """Q(S_t W) per output channel: (codes int8 [N][K], steps f32 [N]) (Sec. 4.3)."""
    K, N = w.shape
    _need(w, torch.float32, "w")
    _need(smooth_text, torch.float32, "smooth_text")
    wq = torch.empty((N, K), dtype=torch.int8, device=w.device)
    scale = torch.empty((N,), dtype=torch.float32, device=w.device)
    _check("masq_quantize_weight", _lib.masq_quantize_weight(
        _ptr(w), _ptr(smooth_text), K, N, bits, _ptr(wq), _ptr(scale), _stream(stream)))
    return wq, scale


def gather_smoothed(x, rows, smooth, stream=None):
    """Smoothed calibration rows of one modality, fp64 [n][K]:
    x[rows[i]] / smooth (Sec. 4.3)."""
    T, K = x.shape
    _need(rows, torch.int32, "rows")
    _need(smooth, torch.float32, "smooth")
    z = torch.empty((rows.shape[0], K), dtype=torch.float64, device=x.device)
    _check("masq_gather_smoothed", _lib.masq_gather_smoothed(
        _ptr(x), _dt(x), T, K, _ptr(rows), rows.shape[0], _ptr(smooth), _ptr(z),
        _stream(stream)))
    return z


def weight_difference(w, smooth, wq, w_scale, stream=None):
    """dW = S_m W - Q(S_t W), fp64 [K][N] (Sec. 4.3), from the float weight
    W [K][N], S_m's diagonal and the shared weight's codes [N][K] and steps."""
    K, N = w.shape
    _need(w, torch.float32, "w")
    _need(smooth, torch.float32, "smooth")
    _need(wq, torch.int8, "wq")
    _need(w_scale, torch.float32, "w_scale")
    dw = torch.empty((K, N), dtype=torch.float64, device=w.device)
    _check("masq_weight_difference", _lib.masq_weight_difference(
        _ptr(w), _ptr(smooth), _ptr(wq), _ptr(w_scale), K, N, _ptr(dw), _stream(stream)))
    return dw


def _view_ptr(t):
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    return ctypes.c_void_p(t.data_ptr())


def dgemm(a, b, c=None, beta=0.0, stream=None):
    """C = A B (+ beta C) in fp64.  a [m][k] and b [k][n] are 2-D fp64 device
    tensors of any strides (a transpose view costs nothing); c, if given,
    is a contiguous [m][n] fp64 tensor, updated in place."""
    _need(a, torch.float64, "a")
    _need(b, torch.float64, "b")
    m, k = a.shape
    k2, n = b.shape
    if k != k2:
        raise ValueError(f"inner sizes differ: {k} and {k2}")
    if c is None:
        if beta != 0.0:
            raise ValueError("beta needs c")
        c = torch.empty((m, n), dtype=torch.float64, device=a.device)
    _need(c, torch.float64, "c")
    if tuple(c.shape) != (m, n):
        raise ValueError(f"c must be [{m}][{n}]")
    if c.numel() and any(t.numel() and t.untyped_storage().data_ptr() ==
                         c.untyped_storage().data_ptr() for t in (a, b)):
        raise ValueError("c must not share memory with a or b")
    _check("masq_dgemm", _lib.masq_dgemm(
        m, n, k, _view_ptr(a), a.stride(0), a.stride(1), _view_ptr(b), b.stride(0), b.stride(1),
        float(beta), _ptr(c), n, _stream(stream)))
    return c


def _square_f64(a, name):
    _need(a, torch.float64, name)
    if a.dim() != 2 or a.shape[0] != a.shape[1]:
        raise ValueError(f"{name} must be a square matrix")


def cholesky(a, ridge=0.0, info=None, trace=None, stream=None):
    """In place: a := L with L L^T = a + (ridge tr(a) / n) I, L lower (the
    upper triangle zeroed).  Returns (info, trace): device int32 [1] (0, or
    k + 1 when the leading minor of order k + 1 is not positive) and fp64 [1]
    (tr(a) before the shift); pass views to have them written elsewhere."""
    _square_f64(a, "a")
    n = a.shape[0]
    if info is None:
        info = torch.zeros((1,), dtype=torch.int32, device=a.device)
    if trace is None:
        trace = torch.zeros((1,), dtype=torch.float64, device=a.device)
    _check("masq_cholesky", _lib.masq_cholesky(n, _ptr(a), n, float(ridge), _view_ptr(info),
                                               _view_ptr(trace), _stream(stream)))
    return info, trace


def trsm_right(l, y, trans, stream=None):
    """In place on y [m][n]: X with X L^T = Y (trans) or X L = Y, for the
    lower-triangular L [n][n] of cholesky()."""
    _square_f64(l, "l")
    _need(y, torch.float64, "y")
    m, n = y.shape
    if l.shape[0] != n:
        raise ValueError(f"l must be [{n}][{n}]")
    _check("masq_trsm_right", _lib.masq_trsm_right(m, n, _ptr(l), n, 1 if trans else 0, _ptr(y), n,
                                                   _stream(stream)))
    return y


def jacobi_svd(cols, flags=0, max_sweeps=60, stream=None):
    """SVD of the m x n matrix whose columns are the rows of cols [n][m]
    (overwritten): (sigma [n] decreasing, u [n][m], v [n][n], sweeps) with
    the matrix = sum_j sigma_j u_j v_j^T; u_j is scaled by sigma_j with flag
    bit 0, v_j with bit 1."""
    _need(cols, torch.float64, "cols")
    n, m = cols.shape
    dev = cols.device
    vw = torch.empty((n, n), dtype=torch.float64, device=dev)
    sigma = torch.empty((n,), dtype=torch.float64, device=dev)
    u = torch.empty((n, m), dtype=torch.float64, device=dev)
    v = torch.empty((n, n), dtype=torch.float64, device=dev)
    sweeps = torch.empty((1,), dtype=torch.int32, device=dev)
    _check("masq_jacobi_svd", _lib.masq_jacobi_svd(m, n, _ptr(cols), _ptr(vw), _ptr(sigma),
                                                   _ptr(u), _ptr(v), flags, max_sweeps,
                                                   _ptr(sweeps), _stream(stream)))
    return sigma, u, v, sweeps


def dequantize_rows(codes, scale, stream=None):
    """codes [R][C] int8 times scale [R] f32, as fp64 [R][C] (exact)."""
    _need(codes, torch.int8, "codes")
    _need(scale, torch.float32, "scale")
    R, C = codes.shape
    out = torch.empty((R, C), dtype=torch.float64, device=codes.device)
    _check("masq_dequantize_rows", _lib.masq_dequantize_rows(
        _ptr(codes), _ptr(scale), R, C, _ptr(out), _stream(stream)))
    return out


def mae_sign(y, ref, loss=None, stream=None):
    """(G = sign(y - ref) / count, mean |y - ref|) for fp64 tensors of one
    shape; the mean is a device fp64 scalar (written to loss, a [1] view,
    when given), summed from fixed-order block sums (masq_mae_loss)."""
    _need(y, torch.float64, "y")
    _need(ref, torch.float64, "ref")
    if y.shape != ref.shape:
        raise ValueError("y and ref differ in shape")
    n = y.numel()
    g = torch.empty_like(y)
    part = torch.empty((max(int(_lib.masq_mae_partials(n)), 1),), dtype=torch.float64,
                       device=y.device)
    if loss is None:
        loss = torch.empty((1,), dtype=torch.float64, device=y.device)
    _need(loss, torch.float64, "loss")
    _check("masq_mae_sign", _lib.masq_mae_sign(_ptr(y), _ptr(ref), n, _ptr(g), _ptr(part),
                                               _stream(stream)))
    _check("masq_mae_loss", _lib.masq_mae_loss(_ptr(part), n, _view_ptr(loss), _stream(stream)))
    return g, loss


def adam_log_step(theta, m1, m2, grad, smooth, inv_smooth, step, lam=1.0, lr=1e-2, b1=0.9,
                  b2=0.999, eps=1e-8, stream=None):
    """One Adam step on theta = ln s in place (masq_adam_log_step): theta,
    m1, m2 fp64 [K]; smooth, inv_smooth f32 [K] (the factors the step's
    forward pass used; replaced by the next ones); grad fp64 [K] (dL/ds).
    step = 0 initialises theta, m1, m2 from smooth."""
    for t, name in ((theta, "theta"), (m1, "m1"), (m2, "m2")):
        _need(t, torch.float64, name)
    _need(smooth, torch.float32, "smooth")
    _need(inv_smooth, torch.float32, "inv_smooth")
    if step > 0:
        _need(grad, torch.float64, "grad")
    _check("masq_adam_log_step", _lib.masq_adam_log_step(
        _ptr(theta), _ptr(m1), _ptr(m2), _ptr(grad) if step > 0 else None, _ptr(smooth),
        _ptr(inv_smooth), theta.numel(), float(lam), float(lr), float(b1), float(b2), float(eps),
        int(step), _stream(stream)))


def mas_gradient(x, a, w, b, smooth, stream=None):
    """dL/ds [K] fp64 of the MAS objective from the batch's rows x [T][K],
    A [T][K], W [K][N], B [K][N] (fp64) and the factors s [K] f32."""
    T, K = x.shape
    N = w.shape[1]
    for t, name in ((x, "x"), (a, "a"), (w, "w"), (b, "b")):
        _need(t, torch.float64, name)
    _need(smooth, torch.float32, "smooth")
    colpart = torch.empty((K,), dtype=torch.float64, device=w.device)
    grad = torch.empty((K,), dtype=torch.float64, device=w.device)
    _check("masq_mas_gradient", _lib.masq_mas_gradient(
        _ptr(x), _ptr(a), _ptr(w), _ptr(b), _ptr(smooth), T, K, N, _ptr(colpart), _ptr(grad),
        _stream(stream)))
    return grad


def workspace_bytes(T, K, N, rank, n_mod) -> int:
    return int(_lib.masq_linear_fused_workspace_bytes(T, K, N, rank, n_mod))


class Linear:
    """One modality-aware quantized linear with device-resident artifacts.

    Holds inv_smooth [M][K] f32, wq [N][K] int8 (or, for the 4-bit shared
    weight, uint8 [N][K / 2] packed codes), w_scale [N] f32 and the low-rank
    factors l_down [M-1][r][K], r_up [M-1][N][r] (f32 or bf16)."""

    def __init__(self, inv_smooth, wq, w_scale, l_down=None, r_up=None):
        self.inv_smooth, self.wq, self.w_scale = inv_smooth, wq, w_scale
        self.l_down, self.r_up = l_down, r_up
        self.n_mod = inv_smooth.shape[0]
        self.w4 = wq.dtype == torch.uint8
        self.c_out, self.c_in = wq.shape[0], inv_smooth.shape[1]
        if wq.shape[1] * (2 if self.w4 else 1) != self.c_in:
            raise ValueError("wq does not match inv_smooth's width")
        self.rank = l_down.shape[1] if l_down is not None and l_down.dim() == 3 else 0
        self._ws = None

    @classmethod
    def from_arrays(cls, art: dict, device="cuda"):
        """Move calibration arrays (NumPy, C-ABI layouts) to the device."""
        lr = torch.bfloat16 if art.get("lr_dtype", "bf16") == "bf16" else torch.float32

        def dev(a, dtype):
            return torch.as_tensor(a).to(device=device, dtype=dtype).contiguous()

        if int(art.get("weight_bits", 8)) == 4:
            from . import int4
            wq = dev(int4.pack(art["wq"]), torch.uint8)
        else:
            wq = dev(art["wq"], torch.int8)
        return cls(dev(art["inv_smooth"], torch.float32), wq,
                   dev(art["w_scale"], torch.float32), dev(art["l_down"], lr),
                   dev(art["r_up"], lr))

    def workspace(self, T, device):
        need = workspace_bytes(T, self.c_in, self.c_out, self.rank, self.n_mod)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
        return self._ws

    def _call(self, fn, x, modality, out, workspace, stream):
        T = x.shape[0]
        ws = workspace if workspace is not None else self.workspace(T, x.device)
        lr_dt = _dt(self.l_down) if self.l_down is not None else F32
        if self.w4:
            fn += "_w4a8"
        _check(fn, getattr(_lib, fn)(
            _ptr(x), _dt(x), _ptr(modality), _ptr(self.inv_smooth), _ptr(self.wq),
            _ptr(self.w_scale), _ptr(self.l_down), _ptr(self.r_up), lr_dt, T, self.c_in,
            self.c_out, self.rank, self.n_mod, _ptr(out), _dt(out), _ptr(ws), ws.numel(),
            _stream(stream)))
        return out

    def __call__(self, x, modality, out=None, out_dtype=None, workspace=None, stream=None):
        if out is None:
            out = torch.empty((x.shape[0], self.c_out), device=x.device,
                              dtype=out_dtype or x.dtype)
        return self._call("masq_linear_fused", x, modality, out, workspace, stream)

    def noalloc(self, x, modality, out, stream=None):
        """The layer through masq_linear_fused_noalloc: no workspace, the
        library's static scratch instead (int8 shared weight only)."""
        if self.w4:
            raise ValueError("the allocation-free entry point takes the int8 shared weight")
        lr_dt = _dt(self.l_down) if self.l_down is not None else F32
        _check("masq_linear_fused_noalloc", _lib.masq_linear_fused_noalloc(
            _ptr(x), _dt(x), _ptr(modality), _ptr(self.inv_smooth), _ptr(self.wq),
            _ptr(self.w_scale), _ptr(self.l_down), _ptr(self.r_up), lr_dt, x.shape[0],
            self.c_in, self.c_out, self.rank, self.n_mod, _ptr(out), _dt(out), _stream(stream)))
        return out

    def stage1(self, x, modality, out, workspace=None, stream=None):
        return self._call("masq_linear_stage1", x, modality, out, workspace, stream)

    def stage2(self, x, modality, out, workspace=None, stream=None):
        return self._call("masq_linear_stage2", x, modality, out, workspace, stream)

    def bind(self, x, modality, out, workspace=None, stream=None):
        """The layer's calls on fixed buffers with their arguments checked and
        converted once, for tight loops: returns an object whose stage1(),
        stage2() and __call__() each make one C call."""
        return BoundLinear(self, x, modality, out, workspace, stream)


class BoundLinear:
    """Pre-marshalled masq_linear_fused / _stage1 / _stage2 calls (see
    :meth:`Linear.bind`); keeps its tensors alive."""

    def __init__(self, lin, x, modality, out, workspace=None, stream=None):
        T = x.shape[0]
        ws = workspace if workspace is not None else lin.workspace(T, x.device)
        if ws.numel() < workspace_bytes(T, lin.c_in, lin.c_out, lin.rank, lin.n_mod):
            raise ValueError("workspace too small")
        lr_dt = _dt(lin.l_down) if lin.l_down is not None else F32
        self._args = (_ptr(x), _dt(x), _ptr(modality), _ptr(lin.inv_smooth), _ptr(lin.wq),
                      _ptr(lin.w_scale), _ptr(lin.l_down), _ptr(lin.r_up), lr_dt, T, lin.c_in,
                      lin.c_out, lin.rank, lin.n_mod, _ptr(out), _dt(out), _ptr(ws), ws.numel(),
                      _stream(stream))
        sfx = "_w4a8" if lin.w4 else ""
        self._names = tuple(n + sfx for n in ("masq_linear_fused", "masq_linear_stage1",
                                              "masq_linear_stage2"))
        self._fns = tuple(getattr(_lib, n) for n in self._names)
        self._keep = (lin, x, modality, out, ws)

    def __call__(self):
        code = self._fns[0](*self._args)
        if code:
            raise MasqError(self._names[0], code)

    def stage1(self):
        code = self._fns[1](*self._args)
        if code:
            raise MasqError(self._names[1], code)

    def stage2(self):
        code = self._fns[2](*self._args)
        if code:
            raise MasqError(self._names[2], code)


class MasOnlyLinear:
    """The MAS-only comparator (Sec. 4.2 without the shared weight): every
    modality has its own int8 weight Q(S_m W), no compensation, through
    masq_mas_only_linear (rows grouped by modality on the device; any
    layout of modalities).

    Holds inv_smooth [M][K] f32, wq [M][N][K] int8, w_scale [M][N] f32."""

    def __init__(self, inv_smooth, wq, w_scale):
        if wq.dim() != 3 or wq.dtype != torch.int8:
            raise ValueError("wq must be int8 [M][N][K]")
        self.inv_smooth, self.wq, self.w_scale = inv_smooth, wq, w_scale
        self.n_mod, self.c_out, self.c_in = wq.shape
        self.rank = 0
        self.w4 = False
        self._ws = None

    @classmethod
    def from_arrays(cls, art: dict, device="cuda"):
        def dev(a, dtype):
            return torch.as_tensor(a).to(device=device, dtype=dtype).contiguous()
        return cls(dev(art["inv_smooth"], torch.float32), dev(art["wq"], torch.int8),
                   dev(art["w_scale"], torch.float32))

    def workspace(self, T, device):
        need = int(_lib.masq_mas_only_workspace_bytes(T, self.c_in, self.c_out, self.n_mod))
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
        return self._ws

    def bind(self, x, modality, out, workspace=None, stream=None):
        return BoundMasOnly(self, x, modality, out, workspace, stream)

    def __call__(self, x, modality, out=None, out_dtype=None, workspace=None, stream=None):
        if out is None:
            out = torch.empty((x.shape[0], self.c_out), device=x.device,
                              dtype=out_dtype or x.dtype)
        self.bind(x, modality, out, workspace, stream)()
        return out


class BoundMasOnly:
    """A pre-marshalled masq_mas_only_linear call on fixed buffers; stage1()
    is a no-op and stage2() the whole call, so that it times like a layer."""

    def __init__(self, lin, x, modality, out, workspace=None, stream=None):
        T = x.shape[0]
        ws = workspace if workspace is not None else lin.workspace(T, x.device)
        need = int(_lib.masq_mas_only_workspace_bytes(T, lin.c_in, lin.c_out, lin.n_mod))
        if ws.numel() < need:
            raise ValueError("workspace too small")
        _need(modality, torch.int32, "modality")
        self._args = (_ptr(x), _dt(x), _ptr(modality), _ptr(lin.inv_smooth), _ptr(lin.wq),
                      _ptr(lin.w_scale), T, lin.c_in, lin.c_out, lin.n_mod, _ptr(out), _dt(out),
                      _ptr(ws), ws.numel(), _stream(stream))
        self._keep = (lin, x, modality, out, ws)

    def __call__(self):
        _check("masq_mas_only_linear", _lib.masq_mas_only_linear(*self._args))

    def stage1(self):
        pass

    def stage2(self):
        self()


def linear_fused(x, modality, inv_smooth, wq, w_scale, l_down=None, r_up=None,
                 out_dtype=None, stream=None):
    """Functional form of :class:`Linear` (allocates its workspace per call)."""
    return Linear(inv_smooth, wq, w_scale, l_down, r_up)(x, modality, out_dtype=out_dtype,
                                                         stream=stream)
