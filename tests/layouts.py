"""Unpackers of the packed INT4 layouts documented in include/rotate_attn.h
(test-side readers of the library's output format)."""
import numpy as np


def _nib(b: np.ndarray):
    lo = (b & 0x0F).astype(np.int8)
    hi = (b >> 4).astype(np.int8)
    lo = np.where(lo >= 8, lo - 16, lo).astype(np.int8)
    hi = np.where(hi >= 8, hi - 16, hi).astype(np.int8)
    return lo, hi


def unpack_qk(codes: np.ndarray, BH: int, Npad: int, N: int) -> np.ndarray:
    """[BH*Npad*64] bytes -> int8 codes [BH][N][128].
    byte ((c*8 + j/8)*32 + r)*8 + j%8 holds channels 2j (low) and 2j+1 (high) of token 32c+r."""
    b = np.asarray(codes, np.uint8).reshape(BH, Npad // 32, 8, 32, 8)
    b = b.transpose(0, 1, 3, 2, 4).reshape(BH, Npad, 64)
    lo, hi = _nib(b)
    out = np.empty((BH, Npad, 128), np.int8)
    out[:, :, 0::2] = lo
    out[:, :, 1::2] = hi
    return out[:, :N]


def v_key_of_nibble() -> np.ndarray:
    """key (0..31 inside a chunk) held by half h, nibble np: 16(np/8) + 8(np%2) + 4h + (np%8)/2."""
    k = np.empty((2, 16), np.int64)
    for h in range(2):
        for np_ in range(16):
            k[h, np_] = 16 * (np_ // 8) + 8 * (np_ % 2) + 4 * h + (np_ % 8) // 2
    return k


def unpack_v(codes: np.ndarray, BH: int, Npad: int, N: int) -> np.ndarray:
    """[BH*Npad*64] bytes -> int8 codes [BH][N][128] (see the V layout in the header)."""
    b = np.asarray(codes, np.uint8).reshape(BH, Npad // 32, 2, 128, 8)
    lo, hi = _nib(b)
    nib = np.empty((BH, Npad // 32, 2, 128, 16), np.int8)
    nib[..., 0::2] = lo
    nib[..., 1::2] = hi
    keys = v_key_of_nibble()
    out = np.empty((BH, Npad // 32, 32, 128), np.int8)
    for h in range(2):
        for np_ in range(16):
            out[:, :, keys[h, np_], :] = nib[:, :, h, :, np_]
    return out.reshape(BH, Npad, 128)[:, :N]


def _e2m3_value(f: np.ndarray) -> np.ndarray:
    """6-bit E2M3 field -> float (sign bit 5, exponent bits 4-3 with bias 1, mantissa bits 2-0)."""
    f = f.astype(np.int64)
    sign = np.where(f & 0x20, -1.0, 1.0)
    e = (f >> 3) & 3
    m = f & 7
    mag = np.where(e == 0, m / 8.0, (1.0 + m / 8.0) * np.exp2(e - 1.0))
    return sign * mag


def _fields(recs: np.ndarray) -> np.ndarray:
    """[..., 24] bytes -> [..., 32] 6-bit fields (field f at bits 6f.. of the little-endian record)."""
    bits = np.unpackbits(recs.astype(np.uint8), axis=-1, bitorder="little")
    bits = bits.reshape(*recs.shape[:-1], 32, 6).astype(np.int64)
    return (bits * (1 << np.arange(6))).sum(-1)


def _as_codes(vals: np.ndarray) -> np.ndarray:
    assert np.all(vals == np.round(vals)), "E2M3 field is not an integer code"
    return vals.astype(np.int8)


def unpack_qk_e2m3(codes: np.ndarray, BH: int, Npad: int, N: int) -> np.ndarray:
    """E2M3 container -> int8 codes [BH][N][128].
    record ((c*2 + ch/64)*2 + (ch/32)%2)*32 + r, field ch%32, token 32c + r."""
    r = np.asarray(codes, np.uint8).reshape(BH, Npad // 32, 2, 2, 32, 24)
    v = _e2m3_value(_fields(r))                      # [BH, c, kc, h, r, f]
    v = v.transpose(0, 1, 4, 2, 3, 5).reshape(BH, Npad, 128)
    return _as_codes(v)[:, :N]


def v_key_of_field() -> np.ndarray:
    """key (0..63 inside a 64-token group) of half h, field e: 32(e%2) + 8(e/8) + 4h + (e/2)%4."""
    k = np.empty((2, 32), np.int64)
    for h in range(2):
        for e in range(32):
            k[h, e] = 32 * (e % 2) + 8 * (e // 8) + 4 * h + (e // 2) % 4
    return k


def unpack_v_e2m3(codes: np.ndarray, BH: int, Npad: int, N: int) -> np.ndarray:
    """E2M3 V container -> int8 codes [BH][N][128]."""
    r = np.asarray(codes, np.uint8).reshape(BH, Npad // 64, 4, 2, 32, 24)
    v = _e2m3_value(_fields(r))                      # [BH, g, mt, h, chl, e]
    keys = v_key_of_field()
    out = np.empty((BH, Npad // 64, 64, 128))
    for h in range(2):
        for e in range(32):
            out[:, :, keys[h, e], :] = v[:, :, :, h, :, e].reshape(BH, Npad // 64, 128)
    return _as_codes(out.reshape(BH, Npad, 128))[:, :N]
