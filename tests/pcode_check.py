"""P-code comparison shared by the GPU parity tests.

The INT4 kernels form the scaled probability pscale * P (pscale = 15 for the
Range-optimized mapping of Sec. 4.2.1, 7 for SYM7) with the hardware
exponential and, in the FP6 kernel, as 2^fma(S, c, -(m - log2 pscale)); the
oracle takes exp2 in binary64 rounded once to binary32 and multiplies by the
scale.  The code u = rint(pscale * P) can therefore differ, by one, only where
pscale * P lies within a small band around a rounding boundary k + 1/2:
  2^-18 (v_exp_f32 is within 1 ulp, the oracle's exp2 is rounded once:
         pscale * P differs by < 15 * 1.5 * 2^-23 < 2^-18),
plus pscale * P * ln 2 * |e|, e being the binary32 rounding error of
m - log2(pscale) for the score's block, plus the rounding of the exponent
argument itself (2^-21 relative on |x| <= 5 wherever a code can be nonzero).
Codes outside the band must be equal; the band's mismatches are counted.
"""
import math

import numpy as np

TIE_BAND = 2.0 ** -18


def tie_band(val, m, scale, kv, n):
    """Per-score half-width of the band around a rounding boundary of scale*P."""
    m64 = m.astype(np.float64)
    mq = m.astype(np.float32) - np.float32(math.log2(scale))
    err = np.nan_to_num(np.abs(mq.astype(np.float64) - (m64 - math.log2(scale))), nan=0.0)
    err_key = np.repeat(err, kv, axis=1)[:, :n]
    return TIE_BAND + val * math.log(2.0) * (err_key + 2.0 ** -21)


def compare(u_gpu, d, p_quant, kv, n, label=""):
    """Asserts that the GPU's P codes equal the oracle's outside the band and
    differ by at most one inside it; returns (mismatches, in-band scores,
    scores) and prints one '[ties]' line."""
    ug = np.asarray(u_gpu).astype(np.int64)
    uo = d["u"].astype(np.int64)
    diff = ug != uo
    scale = 7.0 if p_quant == 1 else 15.0
    val = scale * np.exp2(d["x"].astype(np.float64))
    near = np.abs(val - np.floor(val) - 0.5) <= tie_band(val, d["m"], scale, kv, n)
    assert np.all(np.abs(ug - uo) <= 1), f"{label}: a P code differs by more than one"
    assert np.all(near[diff]), f"{label}: {int((diff & ~near).sum())} P-code mismatches outside the tie band"
    res = (int(diff.sum()), int(near.sum()), int(diff.size))
    print(f"[ties] {label}: {res[0]} mismatches / {res[1]} in band / {res[2]} scores "
          f"(rate {res[0] / max(res[2], 1):.3e})", flush=True)
    return res
