"""Benchmark of the INT4 RotateAttention forward on one MI355X.

One step = the whole INT4 hot path over one batch: Q/K producer (3D RoPE +
merged interleaved rotation + K smoothing + per-block INT4 quantization), V
producer (smoothing + per-group INT4), and the INT4 attention kernel, on the
32760-token video-DiT layer (B=1, H=12, grid 21x30x52, d=128), inputs resident
in HBM.  value = effective TOPS = 4*B*H*N^2*d / step time.

Also measured in the same run: the attention kernel alone (HIP events around
its launch inside every timed step), the BF16 fallback (producer + kernel),
and the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0   # MI355X dense int8 matrix-core peak (published)
FP6_PEAK_TOPS = 10100.0   # MI355X dense fp6/fp4 matrix-core peak (published)
BF16_PEAK_TFLOPS = 2500.0
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--skip-fallback", action="store_true")
    ap.add_argument("--container", choices=["e2m3", "int4"], default="e2m3",
                    help="INT4 code container: e2m3 (FP6 matrix core) or int4 nibbles (int8 matrix core)")
    ap.add_argument("--schedule", action="store_true",
                    help="instead of the headline: the mixed-precision schedule (40 calls x 10 steps at the "
                         "32760-token shape, fallback for the first 2 steps and a seeded 15%% of blocks)")
    ap.add_argument("--profile-run", action="store_true",
                    help="untimed: one INT4 step and one fallback step, then a plain copy of COPY_BYTES through "
                         "an elementwise kernel (the calibration for HBM byte counters); for rocprofv3 --pmc")
    return ap.parse_args()


COPY_BYTES = 512 << 20   # calibration copy: larger than the 256 MB last-level cache
KERNEL_SRC = os.path.join(ROOT, "paper_2607_02584_amd", "csrc", "ra_attn_e2m3.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_e2m3_c2_traffic.json")


def source_digest(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(container, wname):
    """HBM bytes per launch of the attention kernel from the committed counter
    summary, or None when it is missing, covers another workload, or the
    kernel source changed since."""
    if container != "e2m3" or not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != source_digest(KERNEL_SRC):
        return None
    if t.get("workload", "").split(":")[0] != wname:
        return None
    return t.get("hbm_bytes_per_launch")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def host_info():
    """The host the CPU baseline ran on: CPU model, logical CPUs, CPUs this process may use."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = None
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def sclk_reader(torch, dev):
    """A function returning the GPU's current shader clock in MHz, read from
    the amdgpu driver's DPM table of this device (the level marked '*'), or
    None where the table is not readable."""
    import re
    props = torch.cuda.get_device_properties(dev)
    path = (f"/sys/bus/pci/devices/{props.pci_domain_id:04x}:{props.pci_bus_id:02x}:"
            f"{props.pci_device_id:02x}.0/pp_dpm_sclk")

    def read():
        try:
            with open(path) as f:
                for ln in f:
                    if ln.rstrip().endswith("*"):
                        m = re.search(r"(\d+)\s*[Mm][Hh]z", ln)
                        return int(m.group(1)) if m else None
        except OSError:
            return None
        return None
    return read


def producer_bytes(w, container, q_group=128, k_group=128, v_group=128):
    """Algorithmic bytes of the Q/K/V producer call: each bf16 input read
    once, each code buffer, scale array and mean written once; and the bytes
    the two-pass smoothing actually reads (K and V once more for their channel
    means, which must be known before any of their codes)."""
    BH, N = w.B * w.H, w.N
    Npad = -(-N // 128) * 128
    rec = 96 if container == "e2m3" else 64
    inp = 3 * BH * N * 128 * 2
    codes = 3 * BH * Npad * rec
    scales = BH * (Npad // q_group + Npad // k_group) * 4 + BH * (-(-N // v_group)) * 128 * 4
    means = 2 * BH * 128 * 4
    algo = inp + codes + scales + means
    return algo, algo + 2 * BH * N * 128 * 2


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1 (heads are independent, "
                                   "so the path would shard by head with no communication)"}))
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2607_02584_amd import datagen as dg
    from paper_2607_02584_amd import rotate_attn as ra

    assert torch.cuda.is_available(), "bench needs a GPU"
    dev = torch.device("cuda:0")
    if args.schedule:
        return schedule(args, torch, dg, ra, dev)
    w = dg.WORKLOADS[args.workload]
    BH, N = w.B * w.H, w.N
    log(f"workload {w.name}: {w.desc}; generating inputs")
    if args.profile_run:
        args.warmup, args.steps = 0, 0
    q, k, v = dg.make_inputs(w)
    qd, kd, vd = (ra.to_device_bits(x, dev) for x in (q, k, v))
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_INTERLEAVED,
                       q_group=128, k_group=128, v_group=128, kv_block=128, out_dtype=ra.BF16,
                       code_format=ra.CODES_E2M3 if args.container == "e2m3" else ra.CODES_INT4)
    bufs = ra.alloc_int4(p, dev)
    ws = ra.workspace(p, ra.PATH_INT4, dev)
    o = torch.empty((BH, N, 128), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[2].record(stream)
        # the Q, K and V producers in one call
        ra.quantize_qkv(p, qd, kd, vd, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"],
                        bufs["v_codes"], bufs["v_scale"], ws, mu_k=bufs["mu_k"], mu_v=bufs["mu_v"])
        if ev is not None:
            ev[0].record(stream)
        ra.attn_int4(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["v_codes"],
                     bufs["v_scale"], bufs["mu_v"], o)
        if ev is not None:
            ev[1].record(stream)

    if args.profile_run:
        step()
        pf = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_NONE, out_dtype=ra.BF16,
                           kv_block=64)
        wsf = ra.workspace(pf, ra.PATH_FP16)
        ra.fwd_fp16(pf, qd, kd, vd, torch.empty_like(o), wsf)
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)   # elementwise: reads COPY_BYTES, writes COPY_BYTES
        torch.cuda.synchronize()
        log(f"profile run done (copy kernel moved {COPY_BYTES} bytes each way)")
        return
    wev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(max(args.warmup, 1))]
    for i in range(args.warmup):
        step(wev[i])
    torch.cuda.synchronize()
    est_ms = wev[args.warmup - 1][0].elapsed_time(wev[args.warmup - 1][1]) if args.warmup > 0 else 5.0
    # The shader clock while the attention kernel runs back to back for about
    # one second, sampled in the second half.  This runs before the timed
    # steps: the first launches of a cold GPU ramp the clock up (the first ten
    # or so run up to 15 % slower), and the fallback below is timed after it,
    # so both paths are timed at the settled clock.
    read_sclk = sclk_reader(torch, dev)
    clk = []
    n_launch = max(40, int(1000.0 / max(est_ms, 0.1)))
    for _ in range(n_launch):
        ra.attn_int4(p, bufs["q_codes"], bufs["q_scale"], bufs["k_codes"], bufs["k_scale"], bufs["v_codes"],
                     bufs["v_scale"], bufs["mu_v"], o)
    time.sleep(0.4 * n_launch * est_ms * 1e-3)
    for _ in range(12):
        time.sleep(0.02)
        clk.append(read_sclk())
    torch.cuda.synchronize()
    clk = [c for c in clk if c is not None]
    log(f"warmup done; timing {args.steps} steps")
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(args.steps):
        step(evs[i])
    t1.record(stream)
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    attn_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in evs]))
    prod_ms = float(np.mean([c.elapsed_time(a) for a, _, c in evs]))
    p_algo, p_reads = producer_bytes(w, args.container)
    prod = {"ms": round(prod_ms, 4), "algorithmic_bytes": p_algo, "gbps": round(p_algo / (prod_ms * 1e-3) / 1e9, 1),
            "peak_gbps": HBM_PEAK_GBS, "frac": round(p_algo / (prod_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "bytes_moved_two_pass": p_reads,
            "gbps_two_pass": round(p_reads / (prod_ms * 1e-3) / 1e9, 1),
            "what": "quantize_qkv: table copy, channel sums of K and V, Q/K/V codes and scales (HIP events on "
                    "the launch stream, mean over the timed steps)"}
    log(f"producers {prod_ms * 1e3:.1f} us: {prod['gbps']} GB/s algorithmic ({prod['frac']:.3f} of HBM peak), "
        f"{prod['gbps_two_pass']} GB/s of bytes moved")
    gpu = {"name": torch.cuda.get_device_properties(dev).name, "arch": torch.cuda.get_device_properties(dev).gcnArchName,
           "compute_units": torch.cuda.get_device_properties(dev).multi_processor_count,
           "sclk_mhz_under_load": {"median": float(np.median(clk)), "min": min(clk), "max": max(clk),
                                   "samples": len(clk)} if clk else None,
           "sclk_source": f"amdgpu DPM table of this device (pp_dpm_sclk, current level), sampled every 20 ms "
                          f"in the second half of {n_launch} back-to-back attention launches"}
    log(f"gpu: {gpu['name']} {gpu['arch']} {gpu['compute_units']} CUs, shader clock under load "
        f"{gpu['sclk_mhz_under_load']}")
    ops = w.ops()
    tops = ops / (ms_step * 1e-3) / 1e12
    attn_tops = ops / (attn_ms * 1e-3) / 1e12
    log(f"int4 step {ms_step:.3f} ms ({tops:.1f} TOPS); attention kernel {attn_ms:.3f} ms ({attn_tops:.1f} TOPS)")

    extra = {}
    fb_kernel_ms = None
    if not args.skip_fallback:
        pf = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_NONE, out_dtype=ra.BF16,
                           kv_block=64)
        wsf = ra.workspace(pf, ra.PATH_FP16, dev)
        of = torch.empty_like(o)
        for _ in range(2):
            ra.fwd_fp16(pf, qd, kd, vd, of, wsf)
        torch.cuda.synchronize()
        nrep = max(3, args.steps // 2)
        e = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nrep)]
        a0 = torch.cuda.Event(enable_timing=True)
        a1 = torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        for i in range(nrep):
            ra.prepare_fp16(pf, qd, kd, vd, wsf)
            e[i][0].record(stream)
            ra.attn_fp16(pf, wsf, of)
            e[i][1].record(stream)
        a1.record(stream)
        torch.cuda.synchronize()
        f_step = a0.elapsed_time(a1) / nrep
        f_attn = float(np.mean([x.elapsed_time(y) for x, y in e]))
        fb_kernel_ms = f_attn
        # the shader clock under the fallback kernel (untimed, about 0.6 s of
        # back-to-back launches, sampled in the second half): the matrix-core
        # heavy kernel may run at another clock than the INT4 kernel
        nfb = max(20, int(600.0 / f_attn))
        for _ in range(nfb):
            ra.attn_fp16(pf, wsf, of)
        time.sleep(0.4 * nfb * f_attn * 1e-3)
        fclk = []
        for _ in range(8):
            time.sleep(0.02)
            fclk.append(read_sclk())
        torch.cuda.synchronize()
        fclk = [c for c in fclk if c is not None]
        extra = {
            "bf16_fallback": {"op_ms": round(f_step, 4), "kernel_ms": round(f_attn, 4),
                              "kernel_tflops": round(ops / (f_attn * 1e-3) / 1e12, 1),
                              "kernel_frac_of_bf16_peak": round(ops / (f_attn * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                              "sclk_mhz_under_load": {"median": float(np.median(fclk)), "min": min(fclk),
                                                      "max": max(fclk), "samples": len(fclk)} if fclk else None},
            "speedup_vs_bf16": {"kernel": round(f_attn / attn_ms, 3), "op": round(f_step / ms_step, 3)},
        }
        log(f"bf16 fallback op {f_step:.3f} ms, kernel {f_attn:.3f} ms; speedup kernel {f_attn / attn_ms:.2f}x; "
            f"shader clock under the fallback {extra['bf16_fallback']['sclk_mhz_under_load']}")

    # context only: PyTorch's own scaled_dot_product_attention on the same shape,
    # bf16, restricted to its flash / memory-efficient backends (never the math path)
    sdpa = None
    if not args.skip_fallback:
        try:
            from torch.nn.attention import SDPBackend, sdpa_kernel
            qt, kt, vt = (torch.randn(w.B, w.H, N, 128, device=dev, dtype=torch.bfloat16) for _ in range(3))
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)
                torch.cuda.synchronize()
                es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(5)]
                for e0, e1 in es:
                    e0.record(stream)
                    torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)
                    e1.record(stream)
                torch.cuda.synchronize()
            sms = float(np.median([e0.elapsed_time(e1) for e0, e1 in es]))
            sdpa = {"kernel": "torch.nn.functional.scaled_dot_product_attention (flash/efficient backend), bf16",
                    "ms": round(sms, 4), "tflops": round(ops / (sms * 1e-3) / 1e12, 1)}
            log(f"torch SDPA (context): {sms:.3f} ms")
            del qt, kt, vt
        except Exception as exc:   # context only: a missing backend is reported, not fatal
            sdpa = {"unavailable": f"{type(exc).__name__}: {str(exc)[:120]}"}

    # variants of the method on the same inputs: the paper's own Q/K granularity
    # (per token, Sec. 5.1), Q smoothing with the per-key bias (Sec. 4), the full
    # Hadamard rotation (the Sec. 5.3 baseline), per-channel V scales, and the
    # int8-matrix-core kernel over nibble-packed codes
    variants = None
    if args.container == "e2m3" and not args.skip_fallback:
        variants = {}
        specs = {
            "per_token_qk": dict(rotation=ra.ROT_INTERLEAVED, q_group=1, k_group=1, smooth=ra.SMOOTH_K | ra.SMOOTH_V),
            "q_smoothing": dict(rotation=ra.ROT_INTERLEAVED, q_group=128, k_group=128,
                                smooth=ra.SMOOTH_K | ra.SMOOTH_V | ra.SMOOTH_Q),
            "full_hadamard": dict(rotation=ra.ROT_HADAMARD, q_group=128, k_group=128,
                                  smooth=ra.SMOOTH_K | ra.SMOOTH_V),
            # one V scale per channel over all tokens
            "per_channel_v": dict(rotation=ra.ROT_INTERLEAVED, q_group=128, k_group=128,
                                  smooth=ra.SMOOTH_K | ra.SMOOTH_V, v_group=N),
            # the headline configuration with the codes packed two per byte and
            # multiplied on the int8 matrix core (int32 accumulation), reported
            # beside the FP6-operand kernel
            "int8_nibble_container": dict(rotation=ra.ROT_INTERLEAVED, q_group=128, k_group=128,
                                          smooth=ra.SMOOTH_K | ra.SMOOTH_V, code_format=ra.CODES_INT4),
        }
        for name, kw in specs.items():
            kw = dict({"v_group": 128, "code_format": ra.CODES_E2M3}, **kw)
            pt = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, kv_block=128,
                                out_dtype=ra.BF16, **kw)
            bt = ra.alloc_int4(pt, dev)
            wst = ra.workspace(pt, ra.PATH_INT4, dev)
            ot = torch.empty_like(o)
            kb = bt["k_bias"] if kw["smooth"] & ra.SMOOTH_Q else None
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))

            def tstep():
                e0.record(stream)
                ra.quantize_qkv(pt, qd, kd, vd, bt["q_codes"], bt["q_scale"], bt["k_codes"], bt["k_scale"],
                                bt["v_codes"], bt["v_scale"], wst, mu_k=bt["mu_k"], mu_v=bt["mu_v"], k_bias=kb)
                e1.record(stream)
                ra.attn_int4(pt, bt["q_codes"], bt["q_scale"], bt["k_codes"], bt["k_scale"], bt["v_codes"],
                             bt["v_scale"], bt["mu_v"], ot, k_bias=kb)
                e2.record(stream)
            tstep()
            torch.cuda.synchronize()
            ka, pa = [], []
            for _ in range(5):
                tstep()
                torch.cuda.synchronize()
                ka.append(e1.elapsed_time(e2))
                pa.append(e0.elapsed_time(e1))
            kms = float(np.median(ka))
            variants[name] = {"kernel_ms": round(kms, 4), "kernel_tops": round(ops / (kms * 1e-3) / 1e12, 1),
                              "producer_ms": round(float(np.median(pa)), 4)}
            if kw["code_format"] == ra.CODES_INT4:
                variants[name]["kernel_frac_of_int8_peak"] = round(ops / (kms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4)
                if fb_kernel_ms:
                    variants[name]["speedup_vs_bf16_kernel"] = round(fb_kernel_ms / kms, 3)
            log(f"variant {name}: attention kernel {kms:.3f} ms, producers {variants[name]['producer_ms']} ms")
            del bt, wst, ot

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, q, k, v, args.cpu_seconds)

    line = {
        "metric": f"effective attention TOPS (4*B*H*N^2*d / time), INT4 RotateAttention forward, {N}-token DiT shape",
        "value": round(tops, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.B} H={w.H} grid {w.T}x{w.Hg}x{w.W} (N={N}) d=128 split "
                               f"{'/'.join(map(str, w.split))} theta={w.theta:g}, interleaved rotation, "
                               f"Q/K/V groups 128, kv_block 128, RANGE15 P, bf16 in/out, "
                               f"{args.container} code container",
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "k_attn_e2m3" if args.container == "e2m3" else "k_attn_int4",
                     "operand_type": "fp6 e2m3 (exact INT4 codes)" if args.container == "e2m3" else "int8",
                     "achieved": round(attn_tops, 2),
                     "peak": FP6_PEAK_TOPS if args.container == "e2m3" else INT8_PEAK_TOPS, "unit": "TOPS",
                     "frac": round(attn_tops / (FP6_PEAK_TOPS if args.container == "e2m3" else INT8_PEAK_TOPS), 4),
                     "frac_of_int8_peak": round(attn_tops / INT8_PEAK_TOPS, 4),
                     "traffic": measured_traffic(args.container, w.name)},
        "cpu_baseline": cpu,
        "producers": prod,
        "gpu": gpu,
        "host": host_info(),
    }
    line.update(extra)
    if variants is not None:
        line["variants"] = variants
    if sdpa is not None:
        line["torch_sdpa_context"] = sdpa
    print(json.dumps(line), flush=True)


def schedule(args, torch, dg, ra, dev):
    """Mixed-precision schedule at the 32760-token shape: rotate_attn_fwd picks
    the fallback or the INT4 path per call; three input sets rotate so the
    last-level cache cannot hold the inputs from one call to the next."""
    import numpy as np
    w = dg.WORKLOADS["c2"]
    mask = dg.schedule_mask()
    sets = []
    for i in range(dg.SCHEDULE["input_sets"]):
        wi = dg.Workload(w.name, w.B, w.H, w.T, w.Hg, w.W, split=w.split, theta=w.theta, seed=w.seed + 10 * i,
                         dist=w.dist)
        sets.append(tuple(ra.to_device_bits(x, dev) for x in dg.make_inputs(wi)))
    p = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_INTERLEAVED, out_dtype=ra.BF16)
    pf = ra.make_params(w.B, w.H, (w.T, w.Hg, w.W), w.split, w.theta, rotation=ra.ROT_NONE, out_dtype=ra.BF16,
                           kv_block=64)
    ws = ra.workspace(p, ra.PATH_INT4, dev)
    wsf = ra.workspace(pf, ra.PATH_FP16, dev)
    o = torch.empty((w.B * w.H, w.N, 128), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    calls = [(s, b, bool(mask[s, b])) for s in range(mask.shape[0]) for b in range(mask.shape[1])]

    def run(i, fb, ev=None):
        qd, kd, vd = sets[i % len(sets)]
        if ev is not None:
            ev[0].record(stream)
        ra.fwd(pf if fb else p, fb, qd, kd, vd, o, wsf if fb else ws)
        if ev is not None:
            ev[1].record(stream)
    for i in range(6):
        run(i, i % 2 == 0)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in calls]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i, (_, _, fb) in enumerate(calls):
        run(i, fb, evs[i])
    t1.record(stream)
    torch.cuda.synchronize()
    total = t0.elapsed_time(t1)
    per = np.array([a.elapsed_time(b) for a, b in evs])
    fbm = np.array([c[2] for c in calls])
    ops = w.ops() * len(calls)
    line = {"metric": "mixed-precision schedule: 400 attention calls (40 blocks x 10 steps) at the 32760-token shape",
            "value": round(total, 2), "unit": "ms", "higher_is_better": False, "n_gpus": 1, "calls": len(calls),
            "int4_calls": int((~fbm).sum()), "fallback_calls": int(fbm.sum()),
            "int4_ms_total": round(float(per[~fbm].sum()), 2), "fallback_ms_total": round(float(per[fbm].sum()), 2),
            "int4_ms_per_call": round(float(per[~fbm].mean()), 4),
            "fallback_ms_per_call": round(float(per[fbm].mean()), 4),
            "effective_tops": round(ops / (total * 1e-3) / 1e12, 1),
            "all_fallback_estimate_ms": round(float(per[fbm].mean()) * len(calls), 1),
            "speedup_vs_all_fallback": round(float(per[fbm].mean()) * len(calls) / total, 3),
            "dtype": "int4+bf16", "data": "synthetic (3 rotating input sets)",
            "config": {"workload": "c5: c2 shape, fallback for steps 0-1 and a seeded 6 of 40 blocks"}}
    print(json.dumps(line), flush=True)


def cpu_baseline(w, q, k, v, seconds):
    """The oracle (plain C, every host thread) on a bounded sample of the same
    workload: head after head, the head's producer pass, then its query rows
    in blocks of 256 against all N keys, until about `seconds` have passed.
    TOPS = 4 * rows * N * d / wall time (producer time included)."""
    import oracle as ora
    geo = ora.Geometry(w.T, w.Hg, w.W, w.split, w.theta)
    cfg = ora.Int4Config()
    t = time.perf_counter()
    rows, heads, t_prod = 0, 0, 0.0
    for h in range(w.H):
        if time.perf_counter() - t >= seconds:
            break
        tp = time.perf_counter()
        qk = ora.quantize_qk_head(geo, cfg, q[0, h], k[0, h])
        vv = ora.quantize_v_head(cfg, v[0, h])
        t_prod += time.perf_counter() - tp
        heads += 1
        r = 0
        while r < w.N and time.perf_counter() - t < seconds:
            nr = min(256, w.N - r)
            ora.attn_int4(qk["q_codes"], qk["q_scale"], qk["k_codes"], qk["k_scale"], vv["v_codes"], vv["v_scale"],
                          vv["mu_v"], q_group=128, k_group=128, v_group=128, kv_block=128, rows=(r, nr))
            r += nr
        rows += r
    el = time.perf_counter() - t
    val = 4.0 * rows * w.N * 128 / el / 1e12
    # the whole workload at the sampled rates: every head's producer pass plus
    # all N query rows of every head (an extrapolation, not a measurement)
    per_prod = t_prod / heads
    per_row = (el - t_prod) / rows
    full_s = w.B * w.H * (per_prod + w.N * per_row)
    log(f"cpu oracle: {rows} query rows over {heads} head(s) in {el:.1f} s on {ora.threads()} threads")
    # the 1024-token case in full (both heads, every row), for scale
    from paper_2607_02584_amd import datagen as dg
    w1 = dg.WORKLOADS["c1"]
    q1, k1, v1 = dg.make_inputs(w1)
    geo1 = ora.Geometry(w1.T, w1.Hg, w1.W, w1.split, w1.theta)
    t1 = time.perf_counter()
    for h in range(w1.H):
        ora.fwd_int4_head(geo1, cfg, q1[0, h], k1[0, h], v1[0, h])
    e1 = time.perf_counter() - t1
    log(f"cpu oracle: the 1024-token case in full in {e1:.2f} s")
    return {"value": round(val, 5), "unit": "TOPS", "cores": ora.threads(), "kind": "oracle",
            "sample": f"{heads} head(s) of {w.name}: each head's producer pass over all {w.N} tokens, then "
                      f"{rows} query rows in all against all {w.N} keys ({el:.1f} s wall)",
            "c1_full": {"seconds": round(e1, 3), "tops": round(w1.ops() / e1 / 1e12, 5),
                        "what": "B=1 H=2 N=1024, producers and every query row"},
            "full_workload_extrapolated": {"seconds": round(full_s, 1), "tops": round(w.ops() / full_s / 1e12, 5),
                                           "producer_s_per_head": round(per_prod, 3),
                                           "us_per_query_row": round(per_row * 1e6, 2),
                                           "label": f"extrapolation, not a measurement: {w.B * w.H} heads x "
                                                    f"(producer pass + {w.N} rows) at the sampled rates"}}


if __name__ == "__main__":
    main()
