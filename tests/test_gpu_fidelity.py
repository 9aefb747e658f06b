"""Fidelity of the INT4 path and the BF16 fallback to unquantized attention.

Reference: fp64 softmax attention of the 3D-RoPE'd inputs (the oracle's
ref_head).  Reported as cosine similarity and relative L2 (||O - R|| / ||R||)
over sampled query rows of the 1024-token case (all rows) and of the
32760-token layer (two heads, three row blocks each), for the INT4 path with
each rotation (none, merged interleaved, half, full Hadamard), the SYM7 P mapping (the
"without range-optimized P" ablation of the paper's Table 1), the paper's
per-token Q/K scales, Q smoothing with its per-key bias, no smoothing at all,
the online V Hadamard, the normaliser from the quantized P, per-channel V
scales, and the BF16 fallback.

The paper gives no per-layer attention accuracy to compare with (its Table 1
is video-level), so these numbers are reported, not pinned ("parity
unpinned"): the asserts are sanity floors only.  Qualitative expectations from the paper (Sec. 5.4):
rotation helps on RoPE-structured outliers, the range-optimized P mapping
beats the symmetric 7-level one.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

VARIANTS = [
    # name, rotation, p_quant, q/k group, smoothing flags[, online V rotation[, l from quantized P]]
    ("int4 none", 0, 0, 128, 3),
    ("int4 interleaved", 1, 0, 128, 3),
    ("int4 half", 2, 0, 128, 3),
    ("int4 full hadamard", 3, 0, 128, 3),
    ("int4 interleaved SYM7", 1, 1, 128, 3),
    ("int4 interleaved per-token", 1, 0, 1, 3),
    ("int4 interleaved Q smoothing", 1, 0, 128, 7),
    ("int4 interleaved no smoothing", 1, 0, 128, 0),
    ("int4 interleaved online V had.", 1, 0, 128, 3, 1),
    ("int4 interleaved l = sum P^", 1, 0, 128, 3, 0, 1),
    ("int4 interleaved per-channel V", 1, 0, 128, 3, 0, 0, "N"),
]


def _metrics(o, r):
    o = o.astype(np.float64).ravel()
    r = r.astype(np.float64).ravel()
    cos = float(np.dot(o, r) / (np.linalg.norm(o) * np.linalg.norm(r)))
    rl2 = float(np.linalg.norm(o - r) / np.linalg.norm(r))
    return cos, rl2


@pytest.mark.parametrize("wname", ["c1", "c2"])
def test_fidelity_to_fp64_attention(ora, wname):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_02584_amd import datagen as dg
    from paper_2607_02584_amd import rotate_attn as ra
    ra.lib()
    w = dg.WORKLOADS[wname]
    print(f"[fidelity] {wname} N={w.N} H={w.H}: generating inputs", flush=True)
    q, k, v = dg.make_inputs(w)
    geo = ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)
    BH, N = w.B * w.H, w.N
    if wname == "c1":
        samples = [(h, 0, N) for h in range(w.H)]
    else:
        rng = np.random.default_rng(7)
        samples = [(h, int(rng.integers(0, N // 128)) * 128, 128) for h in (0, 7) for _ in range(3)]
    refs = [ora.ref_head(geo, q[0, h], k[0, h], v[0, h], rows=(r0, nr)) for h, r0, nr in samples]
    qd, kd, vd = (ra.to_device_bits(x) for x in (q, k, v))
    results = {}
    for name, rot, pq, g, sm, *vr in VARIANTS:
        p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=rot, p_quant=pq, q_group=g,
                           k_group=g, v_group=128, kv_block=128, smooth=sm, out_dtype=ra.FP32,
                           code_format=ra.CODES_E2M3, v_rotation=vr[0] if vr else 0,
                           l_quant=vr[1] if len(vr) > 1 else 0)
        if len(vr) > 2:   # one V scale per channel over all tokens
            p.v_group = w.N
        ws = ra.workspace(p, ra.PATH_INT4)
        o = torch.empty((BH, N, 128), dtype=torch.float32, device="cuda")
        ra.fwd_int4(p, qd, kd, vd, o, ws)
        torch.cuda.synchronize()
        results[name] = o.cpu().numpy()
        del o, ws
    pf = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_NONE, out_dtype=ra.FP32,
                       kv_block=64)
    wsf = ra.workspace(pf, ra.PATH_FP16)
    of = torch.empty((BH, N, 128), dtype=torch.float32, device="cuda")
    ra.fwd_fp16(pf, qd, kd, vd, of, wsf)
    torch.cuda.synchronize()
    results["bf16 fallback"] = of.cpu().numpy()
    print(f"[fidelity] {wname}: {len(samples)} row blocks, {sum(s[2] for s in samples)} query rows", flush=True)
    table = {}
    for name, out in results.items():
        og = np.concatenate([out[h, r0:r0 + nr] for h, r0, nr in samples])
        rg = np.concatenate(refs)
        cos, rl2 = _metrics(og, rg)
        table[name] = (cos, rl2)
        print(f"  {name:28s} cosine {cos:.6f}   rel L2 {rl2:.4e}", flush=True)
    # sanity floors only: these workloads put x10..x30 outliers on a few
    # channel pairs of Q and K, so the logits span hundreds and the INT4
    # per-block scales leave the ordinary channels with few levels
    assert table["bf16 fallback"][0] > 0.99
    for name, *_ in VARIANTS:
        assert table[name][0] > 0.5, name
