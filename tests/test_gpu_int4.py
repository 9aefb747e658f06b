"""GPU parity of the INT4 path against the CPU oracle, through the C ABI.

Bars (from the method's definition): INT4 codes, scales and smoothing means
bit-exact; int32 S tiles bit-exact; running maxima bit-exact; P codes equal
except where 15*2^x lies near a rounding boundary: within 2^-18 (the kernel's
exponential is the hardware one, within 1 ulp; the oracle's is exp2 rounded to binary32)
plus, for the FP6 kernel, which forms 15 P as 2^fma(S, c, -(m - log2 15)),
the effect of the binary32 rounding of m - log2 15 on 15 P; O within
max|O_gpu - O_oracle| / max|O_oracle| <= 2e-3 on binary32 output.
"""
import numpy as np
import pytest

import pcode_check
from layouts import unpack_qk, unpack_qk_e2m3, unpack_v, unpack_v_e2m3

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


def _inputs(w):
    from paper_2607_02584_amd import datagen as dg
    return dg.make_inputs(w)


def _geo(ora, w):
    return ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)


def _cfg(ora, rotation, qg, kg, vg, kv, pq=0, smooth=3, vrot=0, lq=0):
    return ora.Int4Config(rotation=rotation, p_quant=pq, smooth_k=bool(smooth & 1), smooth_v=bool(smooth & 2),
                          smooth_q=bool(smooth & 4), q_group=qg, k_group=kg, v_group=vg, kv_block=kv,
                          v_hadamard=bool(vrot), l_quant=bool(lq))


def _params(ra, w, rotation, qg, kg, vg, kv, pq=0, smooth=3, out=2, fmt=1, vrot=0, lq=0):
    return ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=rotation, p_quant=pq,
                          smooth=smooth, q_group=qg, k_group=kg, v_group=vg, kv_block=kv, out_dtype=out,
                          code_format=fmt, v_rotation=vrot, l_quant=lq)


FORMATS = {"int4": 0, "e2m3": 1}


def _run_quant(torch, ra, p, q, k, v):
    bufs = ra.alloc_int4(p)
    ws = ra.workspace(p, ra.PATH_INT4)
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    ra.quantize_qk(p, qd, kd, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["mu_k"], ws,
                   mu_q=bufs["mu_q"], k_bias=bufs["k_bias"])
    ra.quantize_v(p, vd, bufs["v_codes"], bufs["v_scale"], bufs["mu_v"], ws)
    torch.cuda.synchronize()
    return bufs, (qd, kd, vd), ws


def _host(bufs):
    return {k: v.cpu().numpy() for k, v in bufs.items()}


CASES = [
    # rotation, q_group, k_group, v_group, kv_block, p_quant, smooth
    (1, 128, 128, 128, 128, 0, 3),
    (2, 1, 1, 128, 128, 0, 3),
    (0, 16, 32, 64, 64, 0, 3),
    (1, 1, 64, 10 ** 6, 64, 1, 3),
    (2, 128, 128, 256, 128, 0, 0),
    (3, 1, 128, 128, 128, 0, 3),
    (1, 1, 1, 128, 128, 0, 7),       # Q smoothing with the per-key bias, per-token Q/K (the paper's setting)
    (2, 128, 64, 10 ** 6, 64, 1, 5),  # Q and K smoothing, no V smoothing, kv_block 64, SYM7
    # rotation, q_group, k_group, v_group, kv_block, p_quant, smooth, online V Hadamard
    (1, 128, 128, 128, 128, 0, 3, 1),
    (3, 1, 1, 256, 64, 0, 7, 1),
    # ... and the normaliser from the quantized P
    (1, 128, 128, 128, 128, 0, 3, 0, 1),
    (2, 1, 1, 128, 64, 1, 7, 1, 1),
    # K scales per 16 keys (per block of 16 tokens for Q too)
    (1, 16, 16, 128, 128, 0, 3),
]


def _small_ragged(name="ragged"):
    from paper_2607_02584_amd import datagen as dg
    if name == "b2n15":
        # batch 2, 15 tokens: less than one 32-key chunk, every block partial
        return dg.small_workload("b2n15", 1, 3, 5, H=2, seed=23, B=2)
    if name == "n1":
        # one token: the softmax row is a single 1, O is the dequantized V row (+ mean)
        return dg.small_workload("n1", 1, 1, 1, H=1, seed=24)
    if name == "ragged300":
        # N = 300: the padded length 384 is not a whole number of 256-query workgroups
        return dg.small_workload("ragged300", 3, 10, 10, H=2, seed=22)
    return dg.small_workload("ragged", 3, 7, 11, H=2, seed=21)          # N = 231


def _workloads():
    from paper_2607_02584_amd import datagen as dg
    return [dg.WORKLOADS["c1"], _small_ragged()]


@pytest.mark.parametrize("fmt", ["e2m3", "int4"])
@pytest.mark.parametrize("wname", ["c1", "ragged", "ragged300", "b2n15", "n1"])
@pytest.mark.parametrize("case", CASES)
def test_int4_codes_scores_and_output(ora, wname, case, fmt):
    """Producer codes/scales/means bit-exact; S, m bit-exact; P codes up to ties; O <= 2e-3."""
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c1"] if wname == "c1" else _small_ragged(wname)
    _check_case(ora, w, wname, case, fmt)


# sequence lengths around whole numbers of 64- and 128-key blocks: one, two,
# three and four blocks, each full and with a partial last block (the kernels
# compute a block's scores during the previous block, so the first and last
# blocks take their own paths)
BOUNDARY_GRIDS = {64: (1, 8, 8), 128: (2, 8, 8), 129: (3, 43, 1), 192: (3, 8, 8), 256: (4, 8, 8),
                  257: (1, 1, 257), 384: (6, 8, 8), 385: (5, 7, 11), 512: (8, 8, 8)}


@pytest.mark.parametrize("fmt", ["e2m3", "int4"])
@pytest.mark.parametrize("n", list(BOUNDARY_GRIDS))
@pytest.mark.parametrize("kv", [64, 128])
def test_block_count_boundaries(ora, n, kv, fmt):
    """The same bars at every block count from one to four, full and partial last blocks."""
    from paper_2607_02584_amd import datagen as dg
    T, Hg, W = BOUNDARY_GRIDS[n]
    w = dg.small_workload(f"n{n}", T, Hg, W, H=1, seed=40 + n)
    assert w.N == n
    _check_case(ora, w, f"n{n}", (1, 128, 128, 128, kv, 0, 3), fmt)


# RoPE splits whose axis boundaries (in pairs: D_t/2 and (D_t + D_h)/2) fall
# at a multiple of 16 pairs (the first pair of a thread's 16), at the first
# and last pairs, and in the middle of a thread's range; the geometries keep
# the tile's table rows in LDS, except the two 130- and 160-wide ones, whose
# 128 W rows of 21 or 24 pairs (more than 40 KB) the producer reads from the
# tables in place
SPLIT_CASES = {
    "t16": ((32, 48, 48), (3, 7, 11)),       # boundaries 16, 40
    "t32h16": ((64, 32, 32), (3, 7, 11)),    # boundaries 32, 48
    "t1h1": ((2, 2, 124), (2, 3, 40)),       # boundaries 1, 2
    "t62h1": ((124, 2, 2), (3, 7, 11)),      # boundaries 62, 63
    "inplace": ((44, 42, 42), (1, 2, 160)),  # boundaries 22, 43, tables read in place
    "inplace_t16": ((32, 48, 48), (1, 3, 130)),
}


@pytest.mark.parametrize("fmt", ["e2m3", "int4"])
@pytest.mark.parametrize("rot", [1, 2])
@pytest.mark.parametrize("sname", list(SPLIT_CASES))
def test_rope_split_axis_boundaries(ora, sname, rot, fmt):
    """Producer codes and the whole forward at RoPE splits that put the axis
    boundaries at every kind of place within a thread's 16 pairs, with the
    table rows staged in LDS and read in place."""
    from paper_2607_02584_amd import datagen as dg
    split, (T, Hg, W) = SPLIT_CASES[sname]
    w = dg.small_workload(f"split_{sname}", T, Hg, W, H=1, split=split, seed=60)
    _check_case(ora, w, f"split_{sname}", (rot, 128, 128, 128, 128, 0, 3), fmt)


def _check_case(ora, w, wname, case, fmt):
    torch, ra = _torch(), _ra()
    rot, qg, kg, vg, kv, pq, sm, *rest = case
    vrot = rest[0] if rest else 0
    lq = rest[1] if len(rest) > 1 else 0
    vg = min(vg, 10 ** 6)
    print(f"[int4 parity] {wname} N={w.N} case={case} container={fmt}", flush=True)
    q, k, v = _inputs(w)
    p = _params(ra, w, rot, qg, kg, vg, kv, pq, sm, fmt=FORMATS[fmt], vrot=vrot, lq=lq)
    bufs, _, _ = _run_quant(torch, ra, p, q, k, v)
    Np = ra.layout(p)["n_pad"]
    BH, N = w.B * w.H, w.N
    h = _host(bufs)
    uqk, uv = (unpack_qk_e2m3, unpack_v_e2m3) if fmt == "e2m3" else (unpack_qk, unpack_v)
    qc = uqk(h["q_codes"], BH, Np, N)
    kc = uqk(h["k_codes"], BH, Np, N)
    vc = uv(h["v_codes"], BH, Np, N)
    nvg = -(-N // vg)
    geo = _geo(ora, w)
    cfg = _cfg(ora, rot, qg, kg, vg, kv, pq, sm, vrot, lq)
    o_gpu = torch.empty((BH, N, 128), dtype=torch.float32, device="cuda")
    nb = -(-N // kv)
    for bh in range(BH):
        b, hh = divmod(bh, w.H)
        ref = ora.quantize_qk_head(geo, cfg, q[b, hh], k[b, hh])
        refv = ora.quantize_v_head(cfg, v[b, hh])
        assert np.array_equal(qc[bh], ref["q_codes"])
        assert np.array_equal(kc[bh], ref["k_codes"])
        assert np.array_equal(vc[bh], refv["v_codes"])
        qs = h["q_scale"].reshape(BH, -1)[bh]
        ks = h["k_scale"].reshape(BH, -1)[bh]
        assert np.array_equal(qs[:len(ref["q_scale"])].view(np.uint32), ref["q_scale"].view(np.uint32))
        assert not qs[len(ref["q_scale"]):].any()
        assert np.array_equal(ks[:len(ref["k_scale"])].view(np.uint32), ref["k_scale"].view(np.uint32))
        vs = h["v_scale"].reshape(BH, nvg, 128)[bh]
        assert np.array_equal(vs.view(np.uint32), refv["v_scale"].view(np.uint32))
        assert np.array_equal(h["mu_k"].reshape(BH, 128)[bh].view(np.uint32), ref["mu_k"].view(np.uint32))
        assert np.array_equal(h["mu_v"].reshape(BH, 128)[bh].view(np.uint32), refv["mu_v"].view(np.uint32))
        assert np.array_equal(h["mu_q"].reshape(BH, 128)[bh].view(np.uint32), ref["mu_q"].view(np.uint32))
        if sm & 4:
            kb = h["k_bias"].reshape(BH, Np)[bh]
            assert np.array_equal(kb[:N].view(np.uint32), ref["k_bias"].view(np.uint32)), "key bias mismatch"
            assert not kb[N:].any()

    s_d = torch.zeros((N, N), dtype=torch.int32, device="cuda")
    u_d = torch.zeros((N, N), dtype=torch.uint8, device="cuda")
    m_d = torch.zeros((N, nb), dtype=torch.float32, device="cuda")
    o_plain = torch.empty_like(o_gpu)
    mu_v = bufs["mu_v"] if sm & 2 else None
    kbias = bufs["k_bias"] if sm & 4 else None
    ra.attn_int4(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["v_codes"],
                 bufs["v_scale"], mu_v, o_plain, k_bias=kbias)
    for bh in range(BH):
        b, hh = divmod(bh, w.H)
        ra.attn_int4_debug(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["v_codes"],
                           bufs["v_scale"], mu_v, o_gpu, bh, 0, N, s_d, u_d, m_d, k_bias=kbias)
        torch.cuda.synchronize()
        O_ref, d = ora.fwd_int4_head(geo, cfg, q[b, hh], k[b, hh], v[b, hh], dumps=True)
        S = s_d.cpu().numpy()
        assert np.array_equal(S, d["S"]), "int32 S tile mismatch"
        mg = m_d.cpu().numpy()
        assert np.all(mg == d["m"]), "running max mismatch"
        pcode_check.compare(u_d.cpu().numpy(), d, pq, kv, N, label=f"{wname} {fmt} case={case} bh={bh}")
        og = o_gpu[bh].cpu().numpy().astype(np.float64)
        err = np.abs(og - O_ref).max() / np.abs(O_ref).max()
        print(f"  bh={bh} O rel err={err:.3e}", flush=True)
        assert err <= O_TOL
    # the debug build of the kernel computes exactly what the plain one does
    assert torch.equal(o_plain, o_gpu)


@pytest.mark.parametrize("rot", [1, 2])
def test_learned_rotation_blocks(ora, rot):
    """Blocks from the Sec. 4.1.4 calibration (run on the GPU in PyTorch) drive the
    producer: codes and scales bit-exact against the oracle with the same blocks,
    O within 2e-3."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import calibrate as cal
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c1"]
    q, k, v = _inputs(w)
    mode = "interleaved" if rot == 1 else "half"
    print(f"[learned rotation] c1 {mode}: calibrating", flush=True)
    res = cal.calibrate_rotation(q[0], k[0], (w.T, w.Hg, w.W), w.split, w.theta, mode=mode, q_group=1, k_group=1,
                                 steps=30, rows=512, cols=1024, device="cuda")
    assert res.final <= res.initial
    R = res.blocks
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=rot, rot_blocks=R, q_group=1,
                       k_group=1, v_group=128, kv_block=128, out_dtype=ra.FP32)
    bufs, (qd, kd, vd), ws = _run_quant(torch, ra, p, q, k, v)
    Np = ra.layout(p)["n_pad"]
    BH, N = w.B * w.H, w.N
    h = _host(bufs)
    qc = unpack_qk_e2m3(h["q_codes"], BH, Np, N)
    kc = unpack_qk_e2m3(h["k_codes"], BH, Np, N)
    o = torch.empty((BH, N, 128), dtype=torch.float32, device="cuda")
    ra.fwd_int4(p, qd, kd, vd, o, ws)
    torch.cuda.synchronize()
    cfg = ora.Int4Config(rotation=rot, rot=R, q_group=1, k_group=1, v_group=128, kv_block=128)
    geo = _geo(ora, w)
    for bh in range(BH):
        ref = ora.quantize_qk_head(geo, cfg, q[0, bh], k[0, bh])
        assert np.array_equal(qc[bh], ref["q_codes"]) and np.array_equal(kc[bh], ref["k_codes"])
        assert np.array_equal(h["q_scale"].reshape(BH, -1)[bh][:N].view(np.uint32), ref["q_scale"].view(np.uint32))
        O_ref, _ = ora.fwd_int4_head(geo, cfg, q[0, bh], k[0, bh], v[0, bh])
        err = np.abs(o[bh].cpu().numpy().astype(np.float64) - O_ref).max() / np.abs(O_ref).max()
        assert err <= O_TOL


@pytest.mark.parametrize("fmt", ["e2m3", "int4"])
def test_fwd_int4_matches_stepwise_and_oracle(ora, fmt):
    """The fused entry point equals the three-call sequence bit for bit and the
    oracle within 2e-3; repeated calls give identical bytes."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c1"]
    q, k, v = _inputs(w)
    p = _params(ra, w, 1, 128, 128, 128, 128, fmt=FORMATS[fmt])
    bufs, (qd, kd, vd), _ = _run_quant(torch, ra, p, q, k, v)
    o1 = torch.empty((w.H, w.N, 128), dtype=torch.float32, device="cuda")
    ra.attn_int4(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["v_codes"],
                 bufs["v_scale"], bufs["mu_v"], o1)
    ws = ra.workspace(p, ra.PATH_INT4)
    o2 = torch.empty_like(o1)
    o3 = torch.empty_like(o1)
    ra.fwd_int4(p, qd, kd, vd, o2, ws)
    ra.fwd(p, False, qd, kd, vd, o3, ws)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(o2, o3)
    geo = _geo(ora, w)
    cfg = _cfg(ora, 1, 128, 128, 128, 128)
    for hh in range(w.H):
        O_ref, _ = ora.fwd_int4_head(geo, cfg, q[0, hh], k[0, hh], v[0, hh])
        err = np.abs(o2[hh].cpu().numpy() - O_ref).max() / np.abs(O_ref).max()
        assert err <= O_TOL


@pytest.mark.parametrize("out", [0, 1])
def test_int4_16bit_output_rounds_fp32_result(ora, out):
    """bf16/fp16 output is the binary32 result rounded to nearest."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c1"]
    q, k, v = _inputs(w)
    p32 = _params(ra, w, 1, 128, 128, 128, 128, out=2)
    p16 = _params(ra, w, 1, 128, 128, 128, 128, out=out)
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    ws = ra.workspace(p32, ra.PATH_INT4)
    o32 = torch.empty((w.H, w.N, 128), dtype=torch.float32, device="cuda")
    o16 = torch.empty((w.H, w.N, 128), dtype=torch.bfloat16 if out == 0 else torch.float16, device="cuda")
    ra.fwd_int4(p32, qd, kd, vd, o32, ws)
    ra.fwd_int4(p16, qd, kd, vd, o16, ws)
    torch.cuda.synchronize()
    assert torch.equal(o32.to(o16.dtype), o16)


C2_VARIANTS = {
    # container, rotation, q_group, k_group, smoothing, online V Hadamard, l from quantized P, v_group (0 = N)
    "e2m3": ("e2m3", 1, 128, 128, 3, 0, 0, 128),
    "int4": ("int4", 1, 128, 128, 3, 0, 0, 128),
    "e2m3-hadamard-qsmooth-pertoken-vhad": ("e2m3", 3, 1, 1, 7, 1, 0, 128),
    "e2m3-half-lquant": ("e2m3", 2, 128, 128, 3, 0, 1, 128),
    # the variants the benchmark times, each in its own kernel instantiation
    "per_token_qk": ("e2m3", 1, 1, 1, 3, 0, 0, 128),
    "q_smoothing": ("e2m3", 1, 128, 128, 7, 0, 0, 128),
    "full_hadamard": ("e2m3", 3, 128, 128, 3, 0, 0, 128),
    "per_channel_v": ("e2m3", 1, 128, 128, 3, 0, 0, 0),
    "k_group16": ("e2m3", 1, 16, 16, 3, 0, 0, 128),
}


@pytest.mark.parametrize("variant", list(C2_VARIANTS))
def test_c2_full_size_sampled_rows(ora, variant):
    """Headline 32760-token shape (12 heads) in the benchmark's launch
    configuration (and variants of the method at the same size): sampled query
    rows of two heads against the oracle -- S and the running maxima bit for
    bit, P codes outside the tie band bit for bit (band mismatches counted), O
    within 2e-3."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c2"]
    fmt, rot, qg, kg, sm, vrot, lq, vg = C2_VARIANTS[variant]
    vg = vg or w.N
    print(f"[c2 sampled] {variant}: generating inputs", flush=True)
    q, k, v = _inputs(w)
    p = _params(ra, w, rot, qg, kg, vg, 128, smooth=sm, fmt=FORMATS[fmt], vrot=vrot, lq=lq)
    bufs, (qd, kd, vd), ws = _run_quant(torch, ra, p, q, k, v)
    kbias = bufs["k_bias"] if sm & 4 else None
    BH, N = w.B * w.H, w.N
    o = torch.empty((BH, N, 128), dtype=torch.float32, device="cuda")
    ra.fwd_int4(p, qd, kd, vd, o, ws)
    torch.cuda.synchronize()
    geo = _geo(ora, w)
    cfg = _cfg(ora, rot, qg, kg, vg, 128, smooth=sm, vrot=vrot, lq=lq)
    rng = np.random.default_rng(2)
    nb = -(-N // 128)
    ties = [0, 0, 0]
    for bh in (0, 7):
        rows0 = [0, int(rng.integers(1, N // 128 - 1)) * 128, N - 40]
        for r0 in rows0:
            nr = 40
            s_d = torch.zeros((nr, N), dtype=torch.int32, device="cuda")
            u_d = torch.zeros((nr, N), dtype=torch.uint8, device="cuda")
            m_d = torch.zeros((nr, nb), dtype=torch.float32, device="cuda")
            od = torch.empty_like(o)
            ra.attn_int4_debug(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"],
                               bufs["v_codes"], bufs["v_scale"], bufs["mu_v"], od, bh, r0, nr, s_d, u_d, m_d,
                               k_bias=kbias)
            torch.cuda.synchronize()
            O_ref, d = ora.fwd_int4_head(geo, cfg, q[0, bh], k[0, bh], v[0, bh], rows=(r0, nr), dumps=True)
            assert np.array_equal(s_d.cpu().numpy(), d["S"])
            assert np.all(m_d.cpu().numpy() == d["m"])
            t = pcode_check.compare(u_d.cpu().numpy(), d, 0, 128, N, label=f"c2 {variant} bh={bh} rows {r0}+{nr}")
            ties = [a + b for a, b in zip(ties, t)]
            og = o[bh, r0:r0 + nr].cpu().numpy()
            err = np.abs(og - O_ref).max() / np.abs(O_ref).max()
            print(f"  bh={bh} rows {r0}+{nr}: O rel err {err:.3e}", flush=True)
            assert err <= O_TOL
    print(f"[ties-total] c2 {variant}: {ties[0]} mismatches / {ties[1]} in band / {ties[2]} scores", flush=True)
    # properties at full size: finite output, determinism
    o2 = torch.empty_like(o)
    ra.fwd_int4(p, qd, kd, vd, o2, ws)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all() and torch.equal(o, o2)


@pytest.mark.parametrize("wname,case", [("c1", (1, 128, 128, 128, 128, 0, 3, 0)), ("c1", (3, 1, 1, 256, 64, 0, 7, 1)),
                                        ("ragged300", (2, 128, 64, 128, 64, 1, 7, 1)), ("c2", (1, 128, 128, 128, 128, 0, 3, 0))])
def test_quantize_qkv_equals_the_two_producers(ora, wname, case):
    """The combined producer call writes exactly the bytes of quantize_qk
    followed by quantize_v, every time."""
    torch, ra = _torch(), _ra()
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS[wname] if wname in ("c1", "c2") else _small_ragged(wname)
    rot, qg, kg, vg, kv, pq, sm, vrot = case
    print(f"[qkv] {wname} case={case}", flush=True)
    q, k, v = _inputs(w)
    p = _params(ra, w, rot, qg, kg, vg, kv, pq, sm, vrot=vrot)
    ref, (qd, kd, vd), ws = _run_quant(torch, ra, p, q, k, v)
    for rep in range(3):
        b = ra.alloc_int4(p)
        ra.quantize_qkv(p, qd, kd, vd, b["q_codes"], b["q_scale"], b["k_codes"], b["k_scale"], b["v_codes"],
                        b["v_scale"], ws, mu_k=b["mu_k"], mu_q=b["mu_q"], mu_v=b["mu_v"], k_bias=b["k_bias"])
        torch.cuda.synchronize()
        for name in ("q_codes", "q_scale", "k_codes", "k_scale", "v_codes", "v_scale", "mu_k", "mu_q", "mu_v"):
            assert torch.equal(b[name], ref[name]), (name, rep)
        if sm & 4:
            assert torch.equal(b["k_bias"], ref["k_bias"])
