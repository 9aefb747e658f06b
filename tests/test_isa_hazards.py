"""Static check of the FP6 attention kernel's machine code (CPU only).

The FP6 packing conversion v_cvt_scalef32_2xpk16_fp6_f32 reads 32 source
registers, and on gfx950 a vector instruction issued right behind it may
overwrite those registers before they are read: the compiler does not hold
such writes back, and the result is silently wrong P codes (seen on the device
as wrong output rows).  The kernel keeps the sources live past the PV
products; this test compiles it to gfx950 assembly and checks that in every
instantiation no instruction within the next MIN_DISTANCE instructions writes
a source register of a packing conversion.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_02584_amd", "csrc", "ra_attn_e2m3.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
MIN_DISTANCE = 16
_STORES = ("ds_write", "global_store", "buffer_store", "v_cmp", "s_")


def _regs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _kernels(asm):
    kern, body = None, []
    for ln in asm.splitlines():
        m = re.match(r"^(_Z\S+):", ln)
        if m:
            if kern:
                yield kern, body
            kern, body = m.group(1), []
        elif kern and re.match(r"^\s+[a-z]", ln) and not ln.strip().startswith(";"):
            body.append(ln.strip())
    if kern:
        yield kern, body


def _violations(body):
    out = []
    for i, ins in enumerate(body):
        if not ins.startswith("v_cvt_scalef32_2xpk16"):
            continue
        ops = [o.strip() for o in ins.split(None, 1)[1].split(",")]
        src = _regs(ops[1]) | _regs(ops[2])
        for d in range(1, MIN_DISTANCE + 1):
            if i + d >= len(body):
                break
            nxt = body[i + d]
            if nxt.startswith(_STORES):
                continue
            parts = nxt.split(None, 1)
            if len(parts) == 2 and _regs(parts[1].split(",")[0].strip()) & src:
                out.append((d, nxt))
    return out


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not available")
def test_fp6_pack_sources_not_overwritten_early():
    with tempfile.TemporaryDirectory() as td:
        out = os.path.join(td, "k.s")
        cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-ffp-contract=off", "-Xclang",
               "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
               "--cuda-device-only", "-S", "-x", "hip", SRC, "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(out) as f:
            asm = f.read()
    n_conv, bad = 0, {}
    for kern, body in _kernels(asm):
        n_conv += sum(1 for b in body if b.startswith("v_cvt_scalef32_2xpk16"))
        v = _violations(body)
        if v:
            bad[kern] = v[:3]
    assert n_conv > 0, "no packing conversion found: the scan is not looking at the kernel"
    assert not bad, f"packing-conversion sources overwritten within {MIN_DISTANCE} instructions: {bad}"
