"""Thin ctypes binding of librotate_attn.so (argument marshalling only).

Every step of the path runs in the HIP kernels of the library; this module
only turns torch tensors into device pointers, fills ``ra_params`` and raises
on a non-zero status.  If the library is not built the import of the first
call fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librotate_attn.so")

ROT_NONE, ROT_INTERLEAVED, ROT_HALF, ROT_HADAMARD = 0, 1, 2, 3
PQ_RANGE15, PQ_SYM7 = 0, 1
VROT_NONE, VROT_HADAMARD = 0, 1
SMOOTH_K, SMOOTH_V, SMOOTH_Q = 1, 2, 4
BF16, FP16, FP32 = 0, 1, 2
CODES_INT4, CODES_E2M3 = 0, 1
PATH_INT4, PATH_FP16 = 0, 1


class RAError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where} failed with status {status}: {message}")
        self.status = status


class Params(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("N", ctypes.c_int32), ("D", ctypes.c_int32),
        ("grid", ctypes.c_int32 * 3), ("rope_split", ctypes.c_int32 * 3), ("rope_theta", ctypes.c_float),
        ("rotation", ctypes.c_int32), ("rot_blocks", ctypes.POINTER(ctypes.c_double)),
        ("p_quant", ctypes.c_int32), ("smooth", ctypes.c_int32),
        ("q_group", ctypes.c_int32), ("k_group", ctypes.c_int32), ("v_group", ctypes.c_int32),
        ("kv_block", ctypes.c_int32), ("sm_scale", ctypes.c_float),
        ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32), ("code_format", ctypes.c_int32),
        ("v_rotation", ctypes.c_int32), ("l_quant", ctypes.c_int32),
    ]


class Layout(ctypes.Structure):
    _fields_ = [("n_pad", ctypes.c_int64), ("qk_code_bytes", ctypes.c_int64), ("q_scale_count", ctypes.c_int64),
                ("k_scale_count", ctypes.c_int64), ("v_code_bytes", ctypes.c_int64),
                ("v_scale_count", ctypes.c_int64), ("mu_count", ctypes.c_int64), ("k_bias_count", ctypes.c_int64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        # torch (which provides the device memory and streams) brings its own HIP
        # runtime under the same soname; loading it first makes the library bind
        # to that one instead of starting a second runtime in the process
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        PP = ctypes.POINTER(Params)
        sig = {
            "rotate_attn_layout": [PP, ctypes.POINTER(Layout)],
            "rotate_attn_workspace_size": [PP, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)],
            "rotate_attn_quantize_qk": [PP, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_quantize_v": [PP, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_quantize_qkv": [PP, P, P, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_attn_int4": [PP, P, P, P, P, P, P, P, P, P, P],
            "rotate_attn_attn_int4_debug": [PP, P, P, P, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32, P, P, P, P],
            "rotate_attn_fwd_int4": [PP, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_prepare_fp16": [PP, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_attn_fp16": [PP, P, ctypes.c_size_t, P, P],
            "rotate_attn_fwd_fp16": [PP, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_fwd": [PP, ctypes.c_int, P, P, P, P, P, ctypes.c_size_t, P],
            "rotate_attn_fwd_int4_noalloc": [PP, P, P, P, P, P],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.rotate_attn_error_string.argtypes = [ctypes.c_int]
        L.rotate_attn_error_string.restype = ctypes.c_char_p
        L.rotate_attn_last_error.argtypes = []
        L.rotate_attn_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != 0:
        raise RAError(status, where, lib().rotate_attn_last_error().decode())


def make_params(B, H, grid, split=(44, 42, 42), theta=10000.0, *, rotation=ROT_INTERLEAVED, rot_blocks=None,
                p_quant=PQ_RANGE15, smooth=SMOOTH_K | SMOOTH_V, q_group=128, k_group=128, v_group=128,
                kv_block=128, sm_scale=0.0, in_dtype=BF16, out_dtype=BF16, code_format=CODES_E2M3, D=128,
                v_rotation=VROT_NONE, l_quant=0) -> Params:
    p = Params()
    p.B, p.H, p.D = B, H, D
    p.N = int(grid[0] * grid[1] * grid[2])
    p.grid[:] = [int(g) for g in grid]
    p.rope_split[:] = [int(s) for s in split]
    p.rope_theta = float(theta)
    p.rotation = rotation
    if rot_blocks is not None:
        arr = np.ascontiguousarray(rot_blocks, dtype=np.float64).reshape(D // 2, 2, 2)
        p._rot_keep = arr  # keep alive with the struct
        p.rot_blocks = arr.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    p.p_quant, p.smooth = p_quant, smooth
    p.q_group, p.k_group, p.v_group, p.kv_block = q_group, k_group, v_group, kv_block
    p.sm_scale = float(sm_scale)
    p.in_dtype, p.out_dtype = in_dtype, out_dtype
    p.code_format = code_format
    p.v_rotation = v_rotation
    p.l_quant = int(l_quant)
    return p


def layout(p: Params) -> dict:
    out = Layout()
    _check(lib().rotate_attn_layout(ctypes.byref(p), ctypes.byref(out)), "rotate_attn_layout")
    return {f: getattr(out, f) for f, _ in Layout._fields_}


def workspace_size(p: Params, path: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().rotate_attn_workspace_size(ctypes.byref(p), path, ctypes.byref(n)), "rotate_attn_workspace_size")
    return n.value


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _need(t, nbytes, name, optional=False):
    """The library takes raw pointers: check here that a tensor is a contiguous
    device tensor holding at least the bytes the call will touch."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, the call needs {nbytes}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")


def _io_bytes(p):
    n = int(p.B) * int(p.H) * int(p.N) * int(p.D)
    return 2 * n, n * (4 if p.out_dtype == FP32 else 2)


def _check_codes(p, L, q_codes=None, q_scale=None, k_codes=None, k_scale=None, v_codes=None, v_scale=None,
                 mu=(), k_bias=None, need_bias=False):
    for t, nb, name in ((q_codes, L["qk_code_bytes"], "q_codes"), (k_codes, L["qk_code_bytes"], "k_codes"),
                        (q_scale, 4 * L["q_scale_count"], "q_scale"), (k_scale, 4 * L["k_scale_count"], "k_scale"),
                        (v_codes, L["v_code_bytes"], "v_codes"), (v_scale, 4 * L["v_scale_count"], "v_scale")):
        if nb and t is not False:
            _need(t, nb, name)
    for t, name in mu:
        _need(t, 4 * L["mu_count"], name, optional=True)
    if need_bias or k_bias is not None:
        _need(k_bias, 4 * L["k_bias_count"], "k_bias", optional=not need_bias)


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def quantize_qk(p, q, k, q_codes, q_scale, k_codes, k_scale, mu_k, ws, stream=None, mu_q=None, k_bias=None):
    L = layout(p)
    nin, _ = _io_bytes(p)
    _need(q, nin, "q")
    _need(k, nin, "k")
    _check_codes(p, L, q_codes=q_codes, q_scale=q_scale, k_codes=k_codes, k_scale=k_scale, v_codes=False,
                 v_scale=False, mu=((mu_k, "mu_k"), (mu_q, "mu_q")), k_bias=k_bias,
                 need_bias=bool(p.smooth & SMOOTH_Q))
    _need(ws, workspace_size(p, PATH_INT4), "workspace")
    _check(lib().rotate_attn_quantize_qk(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(q_codes), _ptr(q_scale),
                                         _ptr(k_codes), _ptr(k_scale), _ptr(mu_k), _ptr(mu_q), _ptr(k_bias),
                                         _ptr(ws), _nbytes(ws), _stream(stream)), "rotate_attn_quantize_qk")


def quantize_v(p, v, v_codes, v_scale, mu_v, ws, stream=None):
    L = layout(p)
    _need(v, _io_bytes(p)[0], "v")
    _check_codes(p, L, q_codes=False, q_scale=False, k_codes=False, k_scale=False, v_codes=v_codes, v_scale=v_scale,
                 mu=((mu_v, "mu_v"),))
    _need(ws, workspace_size(p, PATH_INT4), "workspace")
    _check(lib().rotate_attn_quantize_v(ctypes.byref(p), _ptr(v), _ptr(v_codes), _ptr(v_scale), _ptr(mu_v),
                                        _ptr(ws), _nbytes(ws), _stream(stream)), "rotate_attn_quantize_v")


def quantize_qkv(p, q, k, v, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, ws, stream=None, mu_k=None,
                 mu_q=None, mu_v=None, k_bias=None):
    """quantize_qk and quantize_v in one call."""
    L = layout(p)
    nin, _ = _io_bytes(p)
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, nin, name)
    _check_codes(p, L, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale,
                 mu=((mu_k, "mu_k"), (mu_q, "mu_q"), (mu_v, "mu_v")), k_bias=k_bias,
                 need_bias=bool(p.smooth & SMOOTH_Q))
    _need(ws, workspace_size(p, PATH_INT4), "workspace")
    _check(lib().rotate_attn_quantize_qkv(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(q_codes), _ptr(q_scale),
                                          _ptr(k_codes), _ptr(k_scale), _ptr(v_codes), _ptr(v_scale), _ptr(mu_k),
                                          _ptr(mu_q), _ptr(mu_v), _ptr(k_bias), _ptr(ws), _nbytes(ws),
                                          _stream(stream)), "rotate_attn_quantize_qkv")


def attn_int4(p, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu_v, o, stream=None, k_bias=None):
    L = layout(p)
    _check_codes(p, L, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu=((mu_v, "mu_v"),), k_bias=k_bias,
                 need_bias=bool(p.smooth & SMOOTH_Q))
    _need(o, _io_bytes(p)[1], "o")
    _check(lib().rotate_attn_attn_int4(ctypes.byref(p), _ptr(q_codes), _ptr(q_scale), _ptr(k_codes), _ptr(k_scale),
                                       _ptr(v_codes), _ptr(v_scale), _ptr(mu_v), _ptr(k_bias), _ptr(o),
                                       _stream(stream)), "rotate_attn_attn_int4")


def attn_int4_debug(p, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu_v, o, bh, row0, rows,
                    s_out=None, u_out=None, m_out=None, stream=None, k_bias=None):
    L = layout(p)
    _check_codes(p, L, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu=((mu_v, "mu_v"),), k_bias=k_bias,
                 need_bias=bool(p.smooth & SMOOTH_Q))
    _need(o, _io_bytes(p)[1], "o")
    nb = -(-int(p.N) // int(p.kv_block))
    _need(s_out, 4 * rows * int(p.N), "s_out", optional=True)
    _need(u_out, rows * int(p.N), "u_out", optional=True)
    _need(m_out, 4 * rows * nb, "m_out", optional=True)
    _check(lib().rotate_attn_attn_int4_debug(ctypes.byref(p), _ptr(q_codes), _ptr(q_scale), _ptr(k_codes),
                                             _ptr(k_scale), _ptr(v_codes), _ptr(v_scale), _ptr(mu_v),
                                             _ptr(k_bias), _ptr(o),
                                             bh, row0, rows, _ptr(s_out), _ptr(u_out), _ptr(m_out),
                                             _stream(stream)), "rotate_attn_attn_int4_debug")


def _check_fwd(p, q, k, v, o, ws, path):
    nin, nout = _io_bytes(p)
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, nin, name)
    _need(o, nout, "o")
    _need(ws, workspace_size(p, path), "workspace")


def fwd_int4(p, q, k, v, o, ws, stream=None):
    _check_fwd(p, q, k, v, o, ws, PATH_INT4)
    _check(lib().rotate_attn_fwd_int4(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(ws), _nbytes(ws),
                                      _stream(stream)), "rotate_attn_fwd_int4")


NOALLOC_SCRATCH_BYTES = 128 << 20


def fwd_int4_noalloc(p, q, k, v, o, stream=None):
    """The INT4 forward on the library's static per-GPU scratch (no workspace,
    nothing allocated); calls that overlap on one GPU race."""
    nin, nout = _io_bytes(p)
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, nin, name)
    _need(o, nout, "o")
    _check(lib().rotate_attn_fwd_int4_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _stream(stream)),
           "rotate_attn_fwd_int4_noalloc")


def prepare_fp16(p, q, k, v, ws, stream=None):
    nin, _ = _io_bytes(p)
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, nin, name)
    _need(ws, workspace_size(p, PATH_FP16), "workspace")
    _check(lib().rotate_attn_prepare_fp16(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(ws), _nbytes(ws),
                                          _stream(stream)), "rotate_attn_prepare_fp16")


def attn_fp16(p, ws, o, stream=None):
    _need(ws, workspace_size(p, PATH_FP16), "workspace")
    _need(o, _io_bytes(p)[1], "o")
    _check(lib().rotate_attn_attn_fp16(ctypes.byref(p), _ptr(ws), _nbytes(ws), _ptr(o), _stream(stream)),
           "rotate_attn_attn_fp16")


def fwd_fp16(p, q, k, v, o, ws, stream=None):
    _check_fwd(p, q, k, v, o, ws, PATH_FP16)
    _check(lib().rotate_attn_fwd_fp16(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(ws), _nbytes(ws),
                                      _stream(stream)), "rotate_attn_fwd_fp16")


def fwd(p, fallback, q, k, v, o, ws, stream=None):
    _check_fwd(p, q, k, v, o, ws, PATH_FP16 if fallback else PATH_INT4)
    _check(lib().rotate_attn_fwd(ctypes.byref(p), int(bool(fallback)), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(ws),
                                 _nbytes(ws), _stream(stream)), "rotate_attn_fwd")


# ---------------------------------------------------------------- helpers --

def alloc_int4(p: Params, device="cuda"):
    """Caller-side buffers for the quantize / attention entry points."""
    import torch
    L = layout(p)
    return dict(
        q_codes=torch.zeros(L["qk_code_bytes"], dtype=torch.uint8, device=device),
        k_codes=torch.zeros(L["qk_code_bytes"], dtype=torch.uint8, device=device),
        v_codes=torch.zeros(L["v_code_bytes"], dtype=torch.uint8, device=device),
        q_scale=torch.zeros(L["q_scale_count"], dtype=torch.float32, device=device),
        k_scale=torch.zeros(L["k_scale_count"], dtype=torch.float32, device=device),
        v_scale=torch.zeros(L["v_scale_count"], dtype=torch.float32, device=device),
        mu_k=torch.zeros(L["mu_count"], dtype=torch.float32, device=device),
        mu_v=torch.zeros(L["mu_count"], dtype=torch.float32, device=device),
        mu_q=torch.zeros(L["mu_count"], dtype=torch.float32, device=device),
        k_bias=torch.zeros(L["k_bias_count"], dtype=torch.float32, device=device),
    )


def workspace(p: Params, path: int, device="cuda"):
    import torch
    return torch.empty(max(workspace_size(p, path), 256), dtype=torch.uint8, device=device)


def to_device_bits(x_bits: np.ndarray, device="cuda"):
    """uint16 bit patterns -> int16 device tensor holding the same bits."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(device)
