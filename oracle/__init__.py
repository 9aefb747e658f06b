"""CPU oracle of the RotateAttention INT4 attention path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It wraps ``ra_oracle.c`` (plain C, built
with gcc) through ctypes and composes the per-head routines into the whole
forward pass of the paper's method:

* Sec. 3 / Sec. 4.1.2 / Sec. 4.1.3: 3D RoPE followed by the interleaved
  (merged) or half rotation of Q and K, or by the full D x D Hadamard
  rotation (the "Full" baseline of Sec. 5.3, matrix of Sec. 4.3),
* Sec. 4: smoothing (K and V means; Q mean with its per-key score bias),
* Sec. 5.1: per-token / per-block INT4 quantization of Q and K, per-group V,
* Sec. 4.2: blockwise online softmax with the Range-optimized P quantizer.

It shares no code with the GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ra_oracle.c")
_LIB = os.path.join(_HERE, "libra_oracle.so")

ROT_NONE, ROT_INTERLEAVED, ROT_HALF, ROT_HADAMARD = 0, 1, 2, 3
PQ_RANGE15, PQ_SYM7, PQ_NONE = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile ``ra_oracle.c`` into ``libra_oracle.so`` next to it."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", "-Wall", "-Werror", "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _RopeCfg(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("D", ctypes.c_int), ("T", ctypes.c_int), ("Hg", ctypes.c_int),
                ("W", ctypes.c_int), ("split", ctypes.c_int * 3), ("theta", ctypes.c_double),
                ("rotation", ctypes.c_int), ("rot", ctypes.POINTER(ctypes.c_double)), ("in_fp16", ctypes.c_int)]


class _AttnCfg(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int), ("D", ctypes.c_int), ("q_group", ctypes.c_int),
                ("k_group", ctypes.c_int), ("v_group", ctypes.c_int), ("kv_block", ctypes.c_int),
                ("p_quant", ctypes.c_int), ("sm_scale", ctypes.c_double), ("l_quant", ctypes.c_int)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        L.ora_rope_block.argtypes = [ctypes.POINTER(_RopeCfg), ctypes.c_int, ctypes.c_int, P]
        L.ora_rope_rot_f32.argtypes = [ctypes.POINTER(_RopeCfg), P, P]
        L.ora_rope_rot_f64.argtypes = [ctypes.POINTER(_RopeCfg), P, P]
        L.ora_hadamard_f32.argtypes = [P, ctypes.c_int]
        L.ora_hadamard_f64.argtypes = [P, ctypes.c_int]
        L.ora_mean_fixed.argtypes = [P, ctypes.c_int, ctypes.c_int, P]
        L.ora_center.argtypes = [P, P, ctypes.c_int, ctypes.c_int, P]
        L.ora_quant_tokens.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P]
        L.ora_quant_v.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P]
        L.ora_key_bias.argtypes = [P, P, ctypes.c_int, ctypes.c_int, P]
        L.ora_attn_int4.argtypes = [ctypes.POINTER(_AttnCfg), P, P, P, P, P, P, P, P, ctypes.c_int, ctypes.c_int,
                                    P, P, P, P, P, P]
        L.ora_attn_ref_f64.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_int,
                                       ctypes.c_int, P]
        L.ora_attn_bf16.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                    ctypes.c_int, ctypes.c_int, P]
        L.ora_attn_fb16.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_int, P]
        L.ora_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.ora_f16_to_f32.restype = ctypes.c_float
        L.ora_f32_to_f16.argtypes = [ctypes.c_float]
        L.ora_f32_to_f16.restype = ctypes.c_uint16
        L.ora_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.ora_bf16_to_f32.restype = ctypes.c_float
        L.ora_f32_to_bf16.argtypes = [ctypes.c_float]
        L.ora_f32_to_bf16.restype = ctypes.c_uint16
        L.ora_exp2_f32.argtypes = [ctypes.c_float]
        L.ora_exp2_f32.restype = ctypes.c_float
        L.ora_pcode.argtypes = [ctypes.c_float, ctypes.c_int]
        L.ora_pcode.restype = ctypes.c_int
        L.ora_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


@dataclass
class Geometry:
    """3D RoPE geometry of one head (Sec. 3)."""

    T: int
    Hg: int
    W: int
    split: tuple = (44, 42, 42)
    theta: float = 10000.0
    D: int = 128

    @property
    def N(self) -> int:
        return self.T * self.Hg * self.W


def _rope_cfg(geo: Geometry, rotation: int, rot, fp16: bool = False):
    c = _RopeCfg()
    c.N, c.D, c.T, c.Hg, c.W = geo.N, geo.D, geo.T, geo.Hg, geo.W
    c.in_fp16 = int(bool(fp16))
    c.split[:] = list(geo.split)
    c.theta = float(geo.theta)
    c.rotation = int(rotation)
    keep = None
    if rot is not None:
        keep = np.ascontiguousarray(rot, dtype=np.float64).reshape(geo.D // 2, 2, 2)
        c.rot = keep.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    return c, keep


def rope_block(geo: Geometry, n: int, p: int, rotation: int = ROT_NONE, rot=None) -> np.ndarray:
    c, _keep = _rope_cfg(geo, rotation, rot)
    G = np.zeros(4, np.float64)
    lib().ora_rope_block(ctypes.byref(c), n, p, _p(G))
    return G.reshape(2, 2)


def rope_rot_f32(geo: Geometry, x_bf16: np.ndarray, rotation: int, rot=None, fp16: bool = False) -> np.ndarray:
    """16-bit bits [N][D] (uint16; bf16, or fp16 with ``fp16``) -> fp32 [N][D]
    (the single-precision sequence)."""
    x = np.ascontiguousarray(x_bf16, dtype=np.uint16)
    assert x.shape == (geo.N, geo.D)
    c, _keep = _rope_cfg(geo, rotation, rot, fp16)
    y = np.empty((geo.N, geo.D), np.float32)
    lib().ora_rope_rot_f32(ctypes.byref(c), _p(x), _p(y))
    return y


def rope_rot_f64(geo: Geometry, x_bf16: np.ndarray, rotation: int, rot=None, fp16: bool = False) -> np.ndarray:
    x = np.ascontiguousarray(x_bf16, dtype=np.uint16)
    assert x.shape == (geo.N, geo.D)
    c, _keep = _rope_cfg(geo, rotation, rot, fp16)
    y = np.empty((geo.N, geo.D), np.float64)
    lib().ora_rope_rot_f64(ctypes.byref(c), _p(x), _p(y))
    return y


def hadamard_f32(y: np.ndarray) -> np.ndarray:
    """Rows of y (binary32) times the orthonormal Sylvester-Hadamard matrix,
    the binary32 butterfly sequence of ``ora_hadamard_f32``."""
    out = np.array(y, dtype=np.float32, order="C", copy=True)
    D = out.shape[-1]
    for row in out.reshape(-1, D):
        lib().ora_hadamard_f32(_p(row), D)
    return out


def hadamard_f64(y: np.ndarray) -> np.ndarray:
    out = np.array(y, dtype=np.float64, order="C", copy=True)
    D = out.shape[-1]
    for row in out.reshape(-1, D):
        lib().ora_hadamard_f64(_p(row), D)
    return out


def mean_fixed(y: np.ndarray) -> np.ndarray:
    y = np.ascontiguousarray(y, dtype=np.float32)
    mu = np.empty(y.shape[1], np.float32)
    lib().ora_mean_fixed(_p(y), y.shape[0], y.shape[1], _p(mu))
    return mu


def center(y: np.ndarray, mu: np.ndarray) -> np.ndarray:
    y = np.ascontiguousarray(y, dtype=np.float32)
    mu = np.ascontiguousarray(mu, dtype=np.float32)
    z = np.empty_like(y)
    lib().ora_center(_p(y), _p(mu), y.shape[0], y.shape[1], _p(z))
    return z


def quant_tokens(z: np.ndarray, g: int):
    z = np.ascontiguousarray(z, dtype=np.float32)
    N, D = z.shape
    codes = np.empty((N, D), np.int8)
    scales = np.empty((N + g - 1) // g, np.float32)
    lib().ora_quant_tokens(_p(z), N, D, g, _p(codes), _p(scales))
    return codes, scales


def quant_v(z: np.ndarray, g: int):
    z = np.ascontiguousarray(z, dtype=np.float32)
    N, D = z.shape
    codes = np.empty((N, D), np.int8)
    scales = np.empty(((N + g - 1) // g, D), np.float32)
    lib().ora_quant_v(_p(z), N, D, g, _p(codes), _p(scales))
    return codes, scales


def key_bias(mu_q: np.ndarray, zk: np.ndarray) -> np.ndarray:
    """Per-key score bias of Q smoothing, b_j = mu_Q . zk_j (binary32, pairwise)."""
    mu_q = np.ascontiguousarray(mu_q, dtype=np.float32)
    zk = np.ascontiguousarray(zk, dtype=np.float32)
    b = np.empty(zk.shape[0], np.float32)
    lib().ora_key_bias(_p(mu_q), _p(zk), zk.shape[0], zk.shape[1], _p(b))
    return b


def attn_int4(qc, qs, kc, ks, vc, vs, mu_v=None, *, q_group, k_group, v_group, kv_block,
              p_quant=PQ_RANGE15, sm_scale=0.0, rows=None, dumps=False, bias=None, l_quant=False):
    """Blockwise INT4 attention for one head; returns O (fp64) and optional dumps.
    ``bias``: per-key score bias of Q smoothing, or None."""
    qc = np.ascontiguousarray(qc, dtype=np.int8)
    kc = np.ascontiguousarray(kc, dtype=np.int8)
    vc = np.ascontiguousarray(vc, dtype=np.int8)
    qs = np.ascontiguousarray(qs, dtype=np.float32)
    ks = np.ascontiguousarray(ks, dtype=np.float32)
    vs = np.ascontiguousarray(vs, dtype=np.float32)
    mu = None if mu_v is None else np.ascontiguousarray(mu_v, dtype=np.float32)
    bias = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    N, D = kc.shape
    row0, nrows = (0, N) if rows is None else rows
    a = _AttnCfg()
    a.N, a.D, a.q_group, a.k_group, a.v_group, a.kv_block = N, D, q_group, k_group, v_group, kv_block
    a.p_quant, a.sm_scale, a.l_quant = p_quant, sm_scale, int(bool(l_quant))
    O = np.empty((nrows, D), np.float64)
    nb = (N + kv_block - 1) // kv_block
    S = u = x = m = l = None
    if dumps:
        S = np.empty((nrows, N), np.int32)
        u = np.empty((nrows, N), np.uint8)
        x = np.empty((nrows, N), np.float32)
        m = np.empty((nrows, nb), np.float32)
        l = np.empty(nrows, np.float64)
    lib().ora_attn_int4(ctypes.byref(a), _p(qc), _p(qs), _p(kc), _p(ks), _p(vc), _p(vs), _p(mu), _p(bias),
                        row0, nrows,
                        _p(O), _p(S), _p(u), _p(x), _p(m), _p(l))
    if dumps:
        return O, dict(S=S, u=u, x=x, m=m, l=l)
    return O


def attn_ref_f64(q, k, v, sm_scale=0.0, rows=None) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    N, D = k.shape
    row0, nrows = (0, q.shape[0]) if rows is None else rows
    O = np.empty((nrows, D), np.float64)
    lib().ora_attn_ref_f64(_p(q), _p(k), _p(v), N, D, sm_scale, row0, nrows, _p(O))
    return O


def attn_fb16(qb, kb, vb, kv_block=64, sm_scale=0.0, rows=None, fp16=False) -> np.ndarray:
    """The 16-bit fallback attention (``ora_attn_fb16``) on 16-bit bits: bf16,
    or fp16 with ``fp16``."""
    qb = np.ascontiguousarray(qb, dtype=np.uint16)
    kb = np.ascontiguousarray(kb, dtype=np.uint16)
    vb = np.ascontiguousarray(vb, dtype=np.uint16)
    N, D = kb.shape
    row0, nrows = (0, qb.shape[0]) if rows is None else rows
    O = np.empty((nrows, D), np.float64)
    lib().ora_attn_fb16(_p(qb), _p(kb), _p(vb), N, D, kv_block, sm_scale, int(bool(fp16)), row0, nrows, _p(O))
    return O


def attn_bf16(qb, kb, vb, kv_block=128, sm_scale=0.0, rows=None) -> np.ndarray:
    return attn_fb16(qb, kb, vb, kv_block=kv_block, sm_scale=sm_scale, rows=rows, fp16=False)


def f16_to_f32(b: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(b, dtype=np.uint16).view(np.float16).astype(np.float32)


def f32_to_f16(f) -> np.ndarray:
    """Round-to-nearest-even binary32 -> binary16 bits through the C helper."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    L = lib()
    return np.array([L.ora_f32_to_f16(float(v)) for v in f.ravel()], np.uint16).reshape(f.shape)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(f) -> np.ndarray:
    """Round-to-nearest-even binary32 -> bf16 bits, element by element through the C helper."""
    f = np.ascontiguousarray(f, dtype=np.float32)
    L = lib()
    return np.array([L.ora_f32_to_bf16(float(v)) for v in f.ravel()], np.uint16).reshape(f.shape)


@dataclass
class Int4Config:
    """Parameters of the INT4 path for the whole-head pipeline."""

    rotation: int = ROT_INTERLEAVED
    rot: object = None
    p_quant: int = PQ_RANGE15
    l_quant: bool = False      # normaliser from the quantized P (ablation) instead of the exact P
    smooth_k: bool = True
    smooth_v: bool = True
    smooth_q: bool = False
    v_hadamard: bool = False   # online V Hadamard: V H before quantization, O H^T after
    q_group: int = 128
    k_group: int = 128
    v_group: int = 128
    kv_block: int = 128
    sm_scale: float = 0.0


def quantize_qk_head(geo: Geometry, cfg: Int4Config, q_bf16, k_bf16):
    """Sec. 3-4.1 + Sec. 5.1 for one head: RoPE+rotation, K (and Q) smoothing,
    INT4 codes; with Q smoothing also the per-key score bias mu_Q . K_j."""
    yq = rope_rot_f32(geo, q_bf16, cfg.rotation, cfg.rot)
    yk = rope_rot_f32(geo, k_bf16, cfg.rotation, cfg.rot)
    if cfg.smooth_k:
        mu_k = mean_fixed(yk)
        zk = center(yk, mu_k)
    else:
        mu_k = np.zeros(geo.D, np.float32)
        zk = yk
    bias = None
    if cfg.smooth_q:
        mu_q = mean_fixed(yq)
        zq = center(yq, mu_q)
        bias = key_bias(mu_q, zk)
    else:
        mu_q = np.zeros(geo.D, np.float32)
        zq = yq
    qc, qs = quant_tokens(zq, cfg.q_group)
    kc, ks = quant_tokens(zk, cfg.k_group)
    return dict(q_codes=qc, q_scale=qs, k_codes=kc, k_scale=ks, mu_k=mu_k, mu_q=mu_q, k_bias=bias)


def quantize_v_head(cfg: Int4Config, v_bf16):
    """Sec. 4.3 + Sec. 5.1 for one head: V (rotated by H online if asked, the
    binary32 transform of Q/K's full rotation), V smoothing, per-group codes."""
    v = bf16_to_f32(v_bf16)
    if cfg.v_hadamard:
        v = hadamard_f32(v)
    if cfg.smooth_v:
        mu_v = mean_fixed(v)
        zv = center(v, mu_v)
    else:
        mu_v = np.zeros(v.shape[1], np.float32)
        zv = v
    vc, vs = quant_v(zv, cfg.v_group)
    return dict(v_codes=vc, v_scale=vs, mu_v=mu_v)


def fwd_int4_head(geo: Geometry, cfg: Int4Config, q_bf16, k_bf16, v_bf16, rows=None, dumps=False):
    """The whole INT4 forward for one head: returns (O fp64, intermediates)."""
    qk = quantize_qk_head(geo, cfg, q_bf16, k_bf16)
    vv = quantize_v_head(cfg, v_bf16)
    res = attn_int4(qk["q_codes"], qk["q_scale"], qk["k_codes"], qk["k_scale"], vv["v_codes"], vv["v_scale"],
                    vv["mu_v"] if cfg.smooth_v else None, q_group=cfg.q_group, k_group=cfg.k_group,
                    v_group=cfg.v_group, kv_block=cfg.kv_block, p_quant=cfg.p_quant, sm_scale=cfg.sm_scale,
                    l_quant=cfg.l_quant,
                    rows=rows, dumps=dumps, bias=qk["k_bias"])
    inter = dict(qk, **vv)
    if dumps:
        O, d = res
        inter.update(d)
    else:
        O = res
    if cfg.v_hadamard:
        # O' = P (V H) is the output in the rotated basis; O = O' H^T = O' H
        O = hadamard_f64(O)
    return O, inter


def rope_bf16_head(geo: Geometry, x_bf16) -> np.ndarray:
    """Fallback producer: plain 3D RoPE (no rotation), rounded to bf16 bits."""
    y = rope_rot_f32(geo, x_bf16, ROT_NONE)
    u = y.view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def rope_f16_head(geo: Geometry, x_f16) -> np.ndarray:
    """Fallback producer on binary16 inputs: plain 3D RoPE in binary32, rounded
    to binary16 bits (numpy's conversion rounds to nearest even)."""
    y = rope_rot_f32(geo, x_f16, ROT_NONE, fp16=True)
    return y.astype(np.float16).view(np.uint16)


def fwd_fp16_head(geo: Geometry, q_bits, k_bits, v_bits, kv_block=64, sm_scale=0.0, rows=None, fp16=False):
    """Whole fallback forward of one head on 16-bit input bits (bf16, or fp16
    with ``fp16``): RoPE rounded to the 16-bit type, then ``attn_fb16``."""
    rope = rope_f16_head if fp16 else rope_bf16_head
    qb = rope(geo, q_bits)
    kb = rope(geo, k_bits)
    return attn_fb16(qb, kb, v_bits, kv_block=kv_block, sm_scale=sm_scale, rows=rows, fp16=fp16)


def ref_head(geo: Geometry, q_bf16, k_bf16, v_bf16, sm_scale=0.0, rows=None) -> np.ndarray:
    """Unquantized fp64 attention with plain 3D RoPE: the fidelity reference."""
    q = rope_rot_f64(geo, q_bf16, ROT_NONE)
    k = rope_rot_f64(geo, k_bf16, ROT_NONE)
    v = bf16_to_f32(v_bf16).astype(np.float64)
    return attn_ref_f64(q, k, v, sm_scale=sm_scale, rows=rows)


def threads() -> int:
    return lib().ora_threads()
