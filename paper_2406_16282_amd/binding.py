"""Thin ctypes binding of liblmbp (include/lmbp.h).

Argument marshalling only: tensors are checked for device, dtype, size and
contiguity, their device pointers and the current HIP stream are passed to the C
ABI, and a non-OK status raises ``LmbpError``. Every step of the computation runs
in the library's HIP kernels. There is no fallback: if liblmbp.so has not been
built, the first call raises.
"""

import contextlib
import ctypes
import math
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblmbp.so")

FP32, BF16 = 0, 1
OK, EINVAL, EDTYPE, EOVERLAP, EHIP = 0, 1, 2, 3, 4

ACT_OPS = ("regelu2_fwd", "regelu2_bwd", "resilu2_fwd", "resilu2_bwd")
NORM_OPS = ("msln_fwd", "msln_bwd", "msrms_fwd", "msrms_bwd")
GLU_OPS = ("reswiglu2_fwd", "reswiglu2_bwd")
STEP_OPS = ("stepact_fwd", "stepact_bwd")
LINEAR_OPS = ("linear_act_fwd", "linear_swiglu_fwd", "msrms_linear_act_fwd", "msrms_linear_swiglu_fwd")
ACT_GELU, ACT_SILU = 0, 1


class LmbpError(RuntimeError):
    def __init__(self, op, status, message):
        super().__init__(f"{op}: status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """Load liblmbp.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`"
            " (the HIP kernels are the only implementation)")
    L = ctypes.CDLL(LIB_PATH)
    i32, i64, f32, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    L.lmbp_codes_bytes.argtypes = [i64]
    L.lmbp_codes_bytes.restype = ctypes.c_size_t
    L.lmbp_strerror.argtypes = [i32]
    L.lmbp_strerror.restype = ctypes.c_char_p
    L.lmbp_last_hip_error.argtypes = []
    L.lmbp_last_hip_error.restype = i32
    for name in ACT_OPS:
        fn = getattr(L, name)
        fn.argtypes = [i32, i64, vp, vp, vp, vp]
        fn.restype = i32
    for name in ("msln_fwd", "msrms_fwd"):
        fn = getattr(L, name)
        fn.argtypes = [i32, i64, i64, f32, vp, vp, vp, vp]
        fn.restype = i32
    for name in ("msln_bwd", "msrms_bwd"):
        fn = getattr(L, name)
        fn.argtypes = [i32, i64, i64, vp, vp, vp, vp, vp]
        fn.restype = i32
    L.reswiglu2_fwd.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp]
    L.reswiglu2_fwd.restype = i32
    L.reswiglu2_bwd.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp, vp]
    L.reswiglu2_bwd.restype = i32
    dp = ctypes.POINTER(ctypes.c_double)
    L.lmbp_stepact_codes_bytes.argtypes = [i32, i64]
    L.lmbp_stepact_codes_bytes.restype = ctypes.c_size_t
    L.stepact_fwd.argtypes = [i32, i32, dp, i32, i64, vp, vp, vp, vp]
    L.stepact_fwd.restype = i32
    L.stepact_bwd.argtypes = [i32, dp, i32, i64, vp, vp, vp, vp]
    L.stepact_bwd.restype = i32
    L.linear_act_fwd.argtypes = [i32, i32, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
    L.linear_act_fwd.restype = i32
    L.linear_swiglu_fwd.argtypes = [i32, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.linear_swiglu_fwd.restype = i32
    L.msrms_linear_act_fwd.argtypes = [i32, i32, i64, i64, i64, f32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.msrms_linear_act_fwd.restype = i32
    L.msrms_linear_swiglu_fwd.argtypes = [i32, i64, i64, i64, f32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.msrms_linear_swiglu_fwd.restype = i32
    L.lmbp_copy.argtypes = [vp, vp, i64, vp]
    L.lmbp_copy.restype = i32
    _lib = L
    return L


def strerror(status):
    return lib().lmbp_strerror(int(status)).decode()


def codes_bytes(n):
    return int(lib().lmbp_codes_bytes(int(n)))


def codes_words(n):
    return codes_bytes(n) // 4


def _check(op, status):
    if status != OK:
        msg = strerror(status)
        if status == EHIP:
            msg += f" (hipError {lib().lmbp_last_hip_error()})"
        raise LmbpError(op, status, msg)


def _dtype_code(t):
    if t.dtype == torch.float32:
        return FP32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}; expected float32 or bfloat16")


def _dev(t, what):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{what} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t


def _on(t, ref, what):
    """``t`` must be a GPU tensor on the same device as ``ref``."""
    _dev(t, what)
    if t.device != ref.device:
        raise ValueError(f"{what} must be on {ref.device}, not {t.device}")
    return t


# torch's own accessor of the current stream's raw handle (a few hundred ns, against ~2 us
# for building a torch.cuda.Stream object); the public call is the fallback.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(t, stream):
    """The HIP stream to launch on: the tensors' current stream by default, else a
    torch.cuda.Stream of the same device or a raw stream handle."""
    if stream is None:
        if _raw_stream is not None:
            return ctypes.c_void_p(_raw_stream(t.device.index))
        return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        if stream.device != t.device:
            raise ValueError(f"stream is on {stream.device}, the tensors on {t.device}")
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _device_of(t):
    """Launches go to the tensors' GPU: a no-op context when it is already the current
    device (the common case; switching costs ~1.5 us per call)."""
    if torch.cuda.current_device() == t.device.index:
        return contextlib.nullcontext()
    return torch.cuda.device(t.device)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _like(t, out, what):
    if out is None:
        return torch.empty_like(t)
    _dev(out, what)
    if out.dtype != t.dtype or out.numel() != t.numel() or out.device != t.device:
        raise ValueError(f"{what} must match the input's dtype, size and device")
    return out


def _codes_out(n, device, codes):
    words = codes_words(n)
    if codes is None:
        return torch.empty(words, dtype=torch.int32, device=device)
    _dev(codes, "codes")
    if codes.dtype != torch.int32 or codes.numel() < words or codes.device != device:
        raise ValueError(f"codes must be an int32 GPU tensor of at least {words} words")
    return codes


def _act_fwd(op, x, y, codes, stream):
    _dev(x, "x")
    dt = _dtype_code(x)
    y = _like(x, y, "y")
    codes = _codes_out(x.numel(), x.device, codes)
    with _device_of(x):   # launches go to the tensors' GPU
        _check(op, getattr(lib(), op)(dt, x.numel(), _ptr(x), _ptr(y), _ptr(codes), _stream(x, stream)))
    return y, codes


def _act_bwd(op, dy, codes, dx, stream):
    _dev(dy, "dy")
    dt = _dtype_code(dy)
    _on(codes, dy, "codes")
    if codes.dtype != torch.int32 or codes.numel() < codes_words(dy.numel()):
        raise ValueError("codes must be the int32 buffer written by the forward")
    dx = _like(dy, dx, "dx")
    with _device_of(dy):   # launches go to the tensors' GPU
        _check(op, getattr(lib(), op)(dt, dy.numel(), _ptr(dy), _ptr(codes), _ptr(dx), _stream(dy, stream)))
    return dx


def regelu2_fwd(x, y=None, codes=None, stream=None):
    """ReGELU2 forward: returns (GELU(x), packed 2-bit codes as int32 words)."""
    return _act_fwd("regelu2_fwd", x, y, codes, stream)


def regelu2_bwd(dy, codes, dx=None, stream=None):
    """ReGELU2 backward: dx = dy * step derivative selected by the codes."""
    return _act_bwd("regelu2_bwd", dy, codes, dx, stream)


def resilu2_fwd(x, y=None, codes=None, stream=None):
    """ReSiLU2 forward: returns (SiLU(x), packed 2-bit codes as int32 words)."""
    return _act_fwd("resilu2_fwd", x, y, codes, stream)


def resilu2_bwd(dy, codes, dx=None, stream=None):
    """ReSiLU2 backward: dx = dy * step derivative selected by the codes."""
    return _act_bwd("resilu2_bwd", dy, codes, dx, stream)


def _same(t, ref, what):
    _dev(t, what)
    if t.dtype != ref.dtype or t.numel() != ref.numel() or t.device != ref.device:
        raise ValueError(f"{what} must match {ref.dtype} x {ref.numel()} on {ref.device}")
    return t


def reswiglu2_fwd(g, u, h=None, s=None, codes=None, stream=None):
    """ReSiLU2 in a SwiGLU product: returns (h = SiLU(g) * u, s = SiLU(g), codes of g)."""
    _dev(g, "g")
    dt = _dtype_code(g)
    _same(u, g, "u")
    h = _like(g, h, "h")
    s = _like(g, s, "s")
    codes = _codes_out(g.numel(), g.device, codes)
    with _device_of(g):   # launches go to the tensors' GPU
        _check("reswiglu2_fwd", lib().reswiglu2_fwd(dt, g.numel(), _ptr(g), _ptr(u), _ptr(h), _ptr(s),
                                                    _ptr(codes), _stream(g, stream)))
    return h, s, codes


def reswiglu2_bwd(dh, u, s, codes, dg=None, du=None, stream=None):
    """Backward of reswiglu2_fwd: returns (dg = dh * u * slope[code], du = dh * s)."""
    _dev(dh, "dh")
    dt = _dtype_code(dh)
    _same(u, dh, "u")
    _same(s, dh, "s")
    _on(codes, dh, "codes")
    if codes.dtype != torch.int32 or codes.numel() < codes_words(dh.numel()):
        raise ValueError("codes must be the int32 buffer written by the forward")
    dg = _like(dh, dg, "dg")
    du = _like(dh, du, "du")
    with _device_of(dh):   # launches go to the tensors' GPU
        _check("reswiglu2_bwd", lib().reswiglu2_bwd(dt, dh.numel(), _ptr(dh), _ptr(u), _ptr(s), _ptr(codes),
                                                    _ptr(dg), _ptr(du), _stream(dh, stream)))
    return dg, du


def _doubles(values, count, what):
    vals = [float(v) for v in values]
    if len(vals) != count:
        raise ValueError(f"{what} needs {count} values, got {len(vals)}")
    return (ctypes.c_double * count)(*vals)


def stepact_fwd(x, act, thresholds, bits, y=None, codes=None, stream=None):
    """k-bit family member: returns (act(x), k-bit codes). ``act`` is "gelu" or "silu";
    ``thresholds`` are the 2^k - 1 increasing biases of the ReLU combination."""
    _dev(x, "x")
    dt = _dtype_code(x)
    if act not in ("gelu", "silu"):
        raise ValueError("act must be 'gelu' or 'silu'")
    if bits not in (1, 2, 3, 4):
        raise ValueError("bits must be 1, 2, 3 or 4")
    a = ACT_GELU if act == "gelu" else ACT_SILU
    tab = _doubles(thresholds, (1 << bits) - 1, "thresholds")
    y = _like(x, y, "y")
    words = int(lib().lmbp_stepact_codes_bytes(bits, x.numel())) // 4
    if codes is None:
        codes = torch.empty(words, dtype=torch.int32, device=x.device)
    elif _on(codes, x, "codes").dtype != torch.int32 or codes.numel() < words:
        raise ValueError(f"codes must be an int32 GPU tensor of at least {words} words")
    with _device_of(x):   # launches go to the tensors' GPU
        _check("stepact_fwd", lib().stepact_fwd(a, bits, tab, dt, x.numel(), _ptr(x), _ptr(y), _ptr(codes),
                                                _stream(x, stream)))
    return y, codes


def stepact_bwd(dy, codes, levels, bits, dx=None, stream=None):
    """Backward of stepact_fwd: dx = dy * levels[code] (2^k levels)."""
    _dev(dy, "dy")
    dt = _dtype_code(dy)
    _on(codes, dy, "codes")
    if bits not in (1, 2, 3, 4):
        raise ValueError("bits must be 1, 2, 3 or 4")
    words = int(lib().lmbp_stepact_codes_bytes(bits, dy.numel())) // 4
    if codes.dtype != torch.int32 or codes.numel() < words:
        raise ValueError("codes must be the int32 buffer written by the forward")
    tab = _doubles(levels, 1 << bits, "levels")
    dx = _like(dy, dx, "dx")
    with _device_of(dy):   # launches go to the tensors' GPU
        _check("stepact_bwd", lib().stepact_bwd(bits, tab, dt, dy.numel(), _ptr(dy), _ptr(codes), _ptr(dx),
                                                _stream(dy, stream)))
    return dx


def _rows_cols(t):
    if t.dim() == 0:
        raise ValueError("norm input needs at least one dimension")
    cols = t.shape[-1]
    rows = t.numel() // cols if cols else 0
    return rows, cols


def _norm_fwd(op, x, eps, z, rstd, stream):
    _dev(x, "x")
    dt = _dtype_code(x)
    rows, cols = _rows_cols(x)
    z = _like(x, z, "z")
    if rstd is None:
        rstd = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device)
    else:
        _on(rstd, x, "rstd")
        if rstd.dtype != torch.float32 or rstd.numel() != rows:
            raise ValueError("rstd must be float32 with one value per row")
    with _device_of(x):   # launches go to the tensors' GPU
        _check(op, getattr(lib(), op)(dt, rows, cols, float(eps), _ptr(x), _ptr(z), _ptr(rstd),
                                      _stream(x, stream)))
    return z, rstd


def _norm_bwd(op, dz, z, rstd, dx, stream):
    _dev(dz, "dz")
    _on(z, dz, "z")
    _on(rstd, dz, "rstd")
    dt = _dtype_code(dz)
    if z.dtype != dz.dtype or z.shape != dz.shape:
        raise ValueError("z must match dz in dtype and shape")
    rows, cols = _rows_cols(dz)
    if rstd.dtype != torch.float32 or rstd.numel() != rows:
        raise ValueError("rstd must be float32 with one value per row")
    dx = _like(dz, dx, "dx")
    with _device_of(dz):   # launches go to the tensors' GPU
        _check(op, getattr(lib(), op)(dt, rows, cols, _ptr(dz), _ptr(z), _ptr(rstd), _ptr(dx),
                                      _stream(dz, stream)))
    return dx


def msln_fwd(x, eps, z=None, rstd=None, stream=None):
    """MS-LN forward over the last dimension: returns (z, rstd)."""
    return _norm_fwd("msln_fwd", x, eps, z, rstd, stream)


def msln_bwd(dz, z, rstd, dx=None, stream=None):
    """MS-LN backward from the saved output z and rstd."""
    return _norm_bwd("msln_bwd", dz, z, rstd, dx, stream)


def msrms_fwd(x, eps, z=None, rstd=None, stream=None):
    """MS-RMSNorm forward over the last dimension: returns (z, rstd)."""
    return _norm_fwd("msrms_fwd", x, eps, z, rstd, stream)


def msrms_bwd(dz, z, rstd, dx=None, stream=None):
    """MS-RMSNorm backward from the saved output z and rstd."""
    return _norm_bwd("msrms_bwd", dz, z, rstd, dx, stream)


def copy_bytes(src, dst, stream=None):
    """Measurement utility: 16-byte vector copy of src into dst (same byte size)."""
    _dev(src, "src")
    _on(dst, src, "dst")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must have the same byte size")
    with _device_of(src):   # launches go to the tensors' GPU
        _check("lmbp_copy", lib().lmbp_copy(_ptr(src), _ptr(dst), nbytes, _stream(src, stream)))
    return dst


def linear_act_fwd(x, w, bias=None, act="gelu", y=None, codes=None, z=None, store_z=False,
                   stream=None):
    """Fused linear layer + ReGELU2 / ReSiLU2 forward (bf16): z = bf16(x W^T + b),
    y = act(z), codes of z. x is [..., k], w is [n, k] (nn.Linear weight), bias [n] or
    None. Returns (y, codes) or, with store_z (or a z tensor given), (y, codes, z)."""
    if act not in ("gelu", "silu"):
        raise ValueError("act must be 'gelu' or 'silu'")
    _dev(x, "x")
    _on(w, x, "w")
    if x.dtype != torch.bfloat16 or w.dtype != torch.bfloat16:
        raise TypeError("linear_act_fwd takes bfloat16 x and w")
    if w.dim() != 2 or x.shape[-1] != w.shape[1]:
        raise ValueError("x must be [..., k] and w [n, k]")
    n, k = w.shape
    m = math.prod(x.shape[:-1])
    out_shape = (*x.shape[:-1], n)
    if bias is not None:
        _on(bias, x, "bias")
        if bias.dtype != torch.bfloat16 or bias.numel() != n:
            raise ValueError("bias must be a bfloat16 tensor of n elements")
    if y is None:
        y = torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
    else:
        _on(y, x, "y")
        if y.dtype != torch.bfloat16 or y.numel() != m * n:
            raise ValueError("y must be a bfloat16 tensor of m * n elements")
    if z is None and store_z:
        z = torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
    elif z is not None:
        _on(z, x, "z")
        if z.dtype != torch.bfloat16 or z.numel() != m * n:
            raise ValueError("z must be a bfloat16 tensor of m * n elements")
    codes = _codes_out(m * n, x.device, codes)
    L = lib()
    with _device_of(x):   # launches go to the tensors' GPU
        _check("linear_act_fwd", L.linear_act_fwd(ACT_GELU if act == "gelu" else ACT_SILU, BF16, m, n, k,
                                                  _ptr(x), _ptr(w),
                                                  _ptr(bias) if bias is not None else None,
                                                  _ptr(y), _ptr(codes),
                                                  _ptr(z) if z is not None else None, _stream(x, stream)))
    return (y, codes, z) if z is not None else (y, codes)


def linear_swiglu_fwd(x, w_gate, w_up, h=None, s=None, u=None, codes=None, g=None, store_g=False,
                      stream=None):
    """Fused LLaMA MLP input side (bf16): g = bf16(x Wg^T), u = bf16(x Wu^T),
    h = SiLU(g) * u, s = SiLU(g), codes of g. Returns (h, s, u, codes) or, with store_g
    (or a g tensor given), (h, s, u, codes, g)."""
    for t, nm in ((x, "x"), (w_gate, "w_gate"), (w_up, "w_up")):
        _on(t, x, nm)
        if t.dtype != torch.bfloat16:
            raise TypeError("linear_swiglu_fwd takes bfloat16 tensors")
    if w_gate.dim() != 2 or w_gate.shape != w_up.shape or x.shape[-1] != w_gate.shape[1]:
        raise ValueError("x must be [..., k], w_gate and w_up [n, k]")
    n, k = w_gate.shape
    m = math.prod(x.shape[:-1])
    out_shape = (*x.shape[:-1], n)

    def out(t, name):
        if t is None:
            return torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
        _on(t, x, name)
        if t.dtype != torch.bfloat16 or t.numel() != m * n:
            raise ValueError(f"{name} must be a bfloat16 tensor of m * n elements")
        return t

    h, s, u = out(h, "h"), out(s, "s"), out(u, "u")
    if g is not None or store_g:
        g = out(g, "g")
    codes = _codes_out(m * n, x.device, codes)
    with _device_of(x):   # launches go to the tensors' GPU
        _check("linear_swiglu_fwd", lib().linear_swiglu_fwd(
            BF16, m, n, k, _ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(h), _ptr(s), _ptr(u), _ptr(codes),
            _ptr(g) if g is not None else None, _stream(x, stream)))
    return (h, s, u, codes, g) if g is not None else (h, s, u, codes)


def _norm_outs(x, m, k, z, rstd):
    if z is None:
        z = torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    else:
        _on(z, x, "z")
        if z.dtype != torch.bfloat16 or z.numel() != m * k:
            raise ValueError("z must be a bfloat16 tensor of m * k elements")
    if rstd is None:
        rstd = torch.empty(m, dtype=torch.float32, device=x.device)
    else:
        _on(rstd, x, "rstd")
        if rstd.dtype != torch.float32 or rstd.numel() != m:
            raise ValueError("rstd must be a float32 tensor of m elements")
    return z, rstd


def msrms_linear_act_fwd(x, w, eps, bias=None, act="silu", y=None, codes=None, z=None, rstd=None,
                         pre=None, store_pre=False, stream=None):
    """MS-RMSNorm + fused linear layer + ReGELU2 / ReSiLU2 forward (bf16): rstd and
    z = bf16(x rstd) as msrms_fwd, y = act(bf16(rstd (x W^T) + b)) and its codes.
    Returns (y, codes, z, rstd) or, with store_pre (or a pre tensor given),
    (y, codes, z, rstd, pre) with pre the rounded pre-activation."""
    if act not in ("gelu", "silu"):
        raise ValueError("act must be 'gelu' or 'silu'")
    _dev(x, "x")
    _on(w, x, "w")
    if x.dtype != torch.bfloat16 or w.dtype != torch.bfloat16:
        raise TypeError("msrms_linear_act_fwd takes bfloat16 x and w")
    if w.dim() != 2 or x.shape[-1] != w.shape[1]:
        raise ValueError("x must be [..., k] and w [n, k]")
    n, k = w.shape
    m = math.prod(x.shape[:-1])
    out_shape = (*x.shape[:-1], n)
    if bias is not None:
        _on(bias, x, "bias")
        if bias.dtype != torch.bfloat16 or bias.numel() != n:
            raise ValueError("bias must be a bfloat16 tensor of n elements")
    if y is None:
        y = torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
    else:
        _on(y, x, "y")
        if y.dtype != torch.bfloat16 or y.numel() != m * n:
            raise ValueError("y must be a bfloat16 tensor of m * n elements")
    z, rstd = _norm_outs(x, m, k, z, rstd)
    if pre is None and store_pre:
        pre = torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
    elif pre is not None:
        _on(pre, x, "pre")
        if pre.dtype != torch.bfloat16 or pre.numel() != m * n:
            raise ValueError("pre must be a bfloat16 tensor of m * n elements")
    codes = _codes_out(m * n, x.device, codes)
    with _device_of(x):   # launches go to the tensors' GPU
        _check("msrms_linear_act_fwd", lib().msrms_linear_act_fwd(
            ACT_GELU if act == "gelu" else ACT_SILU, BF16, m, n, k, float(eps), _ptr(x), _ptr(w),
            _ptr(bias) if bias is not None else None, _ptr(y), _ptr(codes),
            _ptr(pre) if pre is not None else None, _ptr(z), _ptr(rstd), _stream(x, stream)))
    return (y, codes, z, rstd, pre) if pre is not None else (y, codes, z, rstd)


def msrms_linear_swiglu_fwd(x, w_gate, w_up, eps, h=None, s=None, u=None, codes=None, z=None, rstd=None,
                            g=None, store_g=False, stream=None):
    """MS-RMSNorm + the fused LLaMA MLP input side (bf16): rstd and z = bf16(x rstd) as
    msrms_fwd; g, u = bf16(rstd (x W^T)); h = SiLU(g) u, s = SiLU(g), codes of g.
    Returns (h, s, u, codes, z, rstd) or, with store_g (or a g tensor given),
    (h, s, u, codes, z, rstd, g)."""
    for t, nm in ((x, "x"), (w_gate, "w_gate"), (w_up, "w_up")):
        _on(t, x, nm)
        if t.dtype != torch.bfloat16:
            raise TypeError("msrms_linear_swiglu_fwd takes bfloat16 tensors")
    if w_gate.dim() != 2 or w_gate.shape != w_up.shape or x.shape[-1] != w_gate.shape[1]:
        raise ValueError("x must be [..., k], w_gate and w_up [n, k]")
    n, k = w_gate.shape
    m = math.prod(x.shape[:-1])
    out_shape = (*x.shape[:-1], n)

    def out(t, name):
        if t is None:
            return torch.empty(out_shape, dtype=torch.bfloat16, device=x.device)
        _on(t, x, name)
        if t.dtype != torch.bfloat16 or t.numel() != m * n:
            raise ValueError(f"{name} must be a bfloat16 tensor of m * n elements")
        return t

    h, s, u = out(h, "h"), out(s, "s"), out(u, "u")
    if g is not None or store_g:
        g = out(g, "g")
    z, rstd = _norm_outs(x, m, k, z, rstd)
    codes = _codes_out(m * n, x.device, codes)
    with _device_of(x):   # launches go to the tensors' GPU
        _check("msrms_linear_swiglu_fwd", lib().msrms_linear_swiglu_fwd(
            BF16, m, n, k, float(eps), _ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(h), _ptr(s), _ptr(u),
            _ptr(codes), _ptr(g) if g is not None else None, _ptr(z), _ptr(rstd), _stream(x, stream)))
    return (h, s, u, codes, z, rstd, g) if g is not None else (h, s, u, codes, z, rstd)
