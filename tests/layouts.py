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
