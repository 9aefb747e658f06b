"""The learnable-rotation calibration (Sec. 4.1.4), CPU only.

Checked against the oracle (the tool shares no code with it): the tool's
RoPE, half permutation and O(2) blocks put a calibration token in the same
basis as the kernels' producers (so learned blocks mean the same thing to
the library), its fake quantiser rounds to the oracle's INT4 codes and
scales, and the optimisation does what the objective asks on a case with a
known answer: with outliers on one channel of several pairs and the blocks
started without mixing, the angles go to an equal mix (|a| = pi/4) and the
objective falls to that of the paper's H_2 blocks.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")


def _cal():
    from paper_2607_02584_amd import calibrate as cal
    return cal


def _rand_bits(rng, shape, scale=1.0):
    from paper_2607_02584_amd.datagen import f32_to_bf16_bits
    return f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def _orth_blocks(rng, n=64):
    R = np.empty((n, 2, 2))
    for i in range(n):
        a = rng.uniform(0, 2 * np.pi)
        c, s = math.cos(a), math.sin(a)
        R[i] = [[c, s], [-s, c]] if i % 2 == 0 else [[c, s], [s, -c]]
    return R


def test_blocks_are_o2_and_default_is_h2():
    cal = _cal()
    a = torch.linspace(-3, 3, 64, dtype=torch.float64)
    for kinds in (torch.ones(64, dtype=torch.int64), torch.zeros(64, dtype=torch.int64)):
        R = cal.blocks_from_angles(a, kinds).numpy()
        np.testing.assert_allclose(R @ R.transpose(0, 2, 1), np.tile(np.eye(2), (64, 1, 1)), atol=1e-15)
        det = np.linalg.det(R)
        np.testing.assert_allclose(det, -1.0 if kinds[0] == 1 else 1.0, atol=1e-15)
    R = cal.blocks_from_angles(torch.full((64,), math.pi / 4, dtype=torch.float64), torch.ones(64, dtype=torch.int64))
    h2 = np.array([[1, 1], [1, -1]]) / math.sqrt(2)
    np.testing.assert_allclose(R.numpy(), np.tile(h2, (64, 1, 1)), atol=1e-15)


@pytest.mark.parametrize("mode,rot", [("interleaved", 1), ("half", 2)])
def test_tool_basis_matches_the_oracle_producer(ora, mode, rot):
    """RoPE (+ half permutation) + blocks in the tool == the oracle's RoPE+rotation
    (fp64) with the same blocks, for the 44/42/42 and 16/56/56 geometries."""
    cal = _cal()
    rng = np.random.default_rng(51)
    for split, theta in (((44, 42, 42), 1e4), ((16, 56, 56), 256.0)):
        geo = ora.Geometry(3, 4, 5, split=split, theta=theta)
        x = _rand_bits(rng, (geo.N, 128), 2.0)
        R = _orth_blocks(rng)
        ref = ora.rope_rot_f64(geo, x, rot, R)
        xf = torch.from_numpy(ora.bf16_to_f32(x).astype(np.float64))
        cos, sin = cal.rope_tables((3, 4, 5), split, theta, "cpu")
        y = cal.apply_rope(xf, cos.double(), sin.double())
        if mode == "half":
            y = y[:, cal.half_permutation(split)]
        z = cal.apply_blocks(y, torch.from_numpy(R)).numpy()
        # the tool's tables are binary32 cos/sin: agreement to their rounding
        assert np.abs(z - ref).max() <= 1e-6 * np.abs(ref).max()


@pytest.mark.parametrize("g", [1, 128])
def test_fake_quantiser_rounds_to_the_oracle_codes(ora, g):
    cal = _cal()
    rng = np.random.default_rng(52)
    z = (rng.standard_normal((512, 128)) * rng.uniform(0.1, 30, 128)).astype(np.float32)
    z[7] = 0.0
    codes, scales = cal.int4_codes(torch.from_numpy(z), g)
    oc, os_ = ora.quant_tokens(z, g)
    assert np.array_equal(codes.numpy(), oc)
    assert np.array_equal(scales.numpy().ravel().view(np.uint32), os_.view(np.uint32))
    fq = cal.fake_quant(torch.from_numpy(z), g).numpy()
    expect = oc.astype(np.float32) * np.repeat(os_, g)[:512, None]
    np.testing.assert_allclose(fq, expect, rtol=2e-7, atol=0)


def test_calibration_finds_the_equal_mix():
    cal = _cal()
    rng = np.random.default_rng(3)
    N = 512
    Q = rng.standard_normal((N, 128)).astype(np.float32)
    K = rng.standard_normal((N, 128)).astype(np.float32)
    for X in (Q, K):
        X[:, 0:16:2] *= 6.0          # one channel of pairs 0..7 (t segment, position 0: no RoPE turn)
    kw = dict(mode="interleaved", steps=100, rows=512, cols=512, device="cpu", lr=0.05)
    bad = cal.calibrate_rotation(Q, K, (1, 1, N), (44, 42, 42), 1e4, init=np.zeros(64), **kw)
    h2 = cal.calibrate_rotation(Q, K, (1, 1, N), (44, 42, 42), 1e4, steps=0,
                                **{k: v for k, v in kw.items() if k != "steps"})
    assert bad.final < 0.75 * bad.initial
    assert bad.final <= 1.05 * h2.initial
    assert np.all(np.abs(np.abs(bad.angles[:8]) - math.pi / 4) < 0.15)
    assert len(bad.history) == 100 and h2.final == h2.initial
