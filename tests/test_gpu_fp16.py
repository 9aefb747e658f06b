"""GPU parity of the BF16/FP16 fallback attention against the CPU oracle."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

O_TOL = 2e-3


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _ra():
    from paper_2607_02584_amd import rotate_attn as ra
    ra.lib()
    return ra


def _f32_to_f16_bits(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def _kv(p):
    return int(p.kv_block)


SMALL = {
    "ragged": dict(T=3, Hg=7, W=11, H=2, seed=21),
    "b2n15": dict(T=1, Hg=3, W=5, H=2, seed=23, B=2),   # batch 2, less than one key block
    "n1": dict(T=1, Hg=1, W=1, H=1, seed=24),           # a single token: O is its V row
}


@pytest.mark.parametrize("wname,dtype,kv", [("c1", "bf16", 64), ("ragged", "bf16", 64), ("c1", "fp16", 64),
                                            ("b2n15", "bf16", 64), ("n1", "bf16", 64), ("c1", "bf16", 128),
                                            ("ragged", "fp16", 128), ("b2n15", "fp16", 64)])
def test_fp16_fallback_parity(ora, wname, dtype, kv):
    """The fallback against the oracle's 16-bit attention with the same block
    size (P rounded to the input type at its block's running maximum, Sec. 4.2
    blockwise softmax; FP16 attention of Sec. 5.1)."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    if wname == "c1":
        w = dg.WORKLOADS["c1"]
    else:
        g = dict(SMALL[wname])
        w = dg.small_workload(wname, g.pop("T"), g.pop("Hg"), g.pop("W"), **g)
    print(f"[fp16 parity] {wname} {dtype} kv_block={kv} N={w.N}", flush=True)
    fp16 = dtype == "fp16"
    q, k, v = dg.make_inputs(w)
    if fp16:
        # binary16 inputs: the generator's values rounded to fp16
        q, k, v = (_f32_to_f16_bits(dg.bf16_bits_to_f32(x)) for x in (q, k, v))
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=0, in_dtype=ra.FP16 if fp16
                       else ra.BF16, out_dtype=ra.FP32, kv_block=kv)
    ws = ra.workspace(p, ra.PATH_FP16)
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    o = torch.empty((w.B * w.H, w.N, 128), dtype=torch.float32, device="cuda")
    ra.fwd_fp16(p, qd, kd, vd, o, ws)
    o2 = torch.empty_like(o)
    ra.fwd(p, True, qd, kd, vd, o2, ws)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)
    geo = ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)
    for bh in range(w.B * w.H):
        b, hh = divmod(bh, w.H)
        O_ref = ora.fwd_fp16_head(geo, q[b, hh], k[b, hh], v[b, hh], kv_block=kv, fp16=fp16)
        og = o[bh].cpu().numpy()
        err = np.abs(og - O_ref).max() / np.abs(O_ref).max()
        print(f"  head {bh}: O rel err {err:.3e}", flush=True)
        assert err <= O_TOL


# sequence lengths around whole numbers of 64- and 128-key blocks (the kernel
# takes a block's scores during the previous block, so the first and the last
# blocks take their own paths)
BOUNDARY_GRIDS = {64: (1, 8, 8), 128: (2, 8, 8), 129: (3, 43, 1), 192: (3, 8, 8), 256: (4, 8, 8),
                  257: (1, 1, 257), 384: (6, 8, 8), 385: (5, 7, 11)}


@pytest.mark.parametrize("n", list(BOUNDARY_GRIDS))
@pytest.mark.parametrize("kv", [64, 128])
def test_fallback_block_count_boundaries(ora, n, kv):
    """The fallback at every block count from one to six, full and partial last blocks."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    T, Hg, W = BOUNDARY_GRIDS[n]
    w = dg.small_workload(f"n{n}", T, Hg, W, H=1, seed=60 + n)
    assert w.N == n
    q, k, v = dg.make_inputs(w)
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=0, out_dtype=ra.FP32, kv_block=kv)
    ws = ra.workspace(p, ra.PATH_FP16)
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    o = torch.empty((1, n, 128), dtype=torch.float32, device="cuda")
    ra.fwd_fp16(p, qd, kd, vd, o, ws)
    torch.cuda.synchronize()
    geo = ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)
    O_ref = ora.fwd_fp16_head(geo, q[0, 0], k[0, 0], v[0, 0], kv_block=kv)
    err = np.abs(o[0].cpu().numpy() - O_ref).max() / np.abs(O_ref).max()
    print(f"[fallback boundary] N={n} kv_block={kv}: O rel err {err:.3e}", flush=True)
    assert err <= O_TOL


def test_fallback_c2_full_size_sampled_rows(ora):
    """The 32760-token layer in the launch configuration the benchmark times
    (12 heads, bf16 inputs, 64-key blocks), fp32 output: sampled query rows of two
    heads against the fallback oracle within 2e-3."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c2"]
    print("[fp16 c2 sampled] generating inputs", flush=True)
    q, k, v = dg.make_inputs(w)
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=0, out_dtype=ra.FP32, kv_block=64)
    ws = ra.workspace(p, ra.PATH_FP16)
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    o = torch.empty((w.B * w.H, w.N, 128), dtype=torch.float32, device="cuda")
    ra.fwd_fp16(p, qd, kd, vd, o, ws)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    geo = ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)
    rng = np.random.default_rng(33)
    for hh in (0, int(rng.integers(1, w.H))):
        for r0 in (0, int(rng.integers(1, w.N // 64 - 1)) * 64 + 5, w.N - 29):
            nr = 29
            O_ref = ora.fwd_fp16_head(geo, q[0, hh], k[0, hh], v[0, hh], kv_block=_kv(p), rows=(r0, nr))
            og = o[hh, r0:r0 + nr].cpu().numpy()
            err = np.abs(og - O_ref).max() / np.abs(O_ref).max()
            print(f"  head {hh} rows {r0}+{nr}: O rel err {err:.3e}", flush=True)
            assert err <= O_TOL
