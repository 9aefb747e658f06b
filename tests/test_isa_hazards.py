"""Static check of the machine code of the kernels that use the FP6 packing
conversion: the FP6 attention kernel (P codes) and the Q/K producer (E2M3
Q/K codes), CPU only.

The FP6 packing conversion v_cvt_scalef32_2xpk16_fp6_f32 (32 binary32 source
registers in two 16-register tuples, 6 result registers) has two properties on
gfx950 that the compiler does not model; both were measured on the device
with fixed-register probes:

1. It writes its result before it has read all of its sources: a result tuple
   that overlaps the end of a source corrupts the last codes (seen as whole
   output rows going wrong when the compiler placed the result over registers
   14 and 15 of the second source).
2. It reads the first register of each source one cycle early: a v_exp_f32
   result written by the instruction right before it is missed.

Both issue the conversion from inline assembly with an early-clobber result
and a leading wait state.  This test compiles them to gfx950 assembly and
checks every instantiation: no conversion's result overlaps a
source, and no v_exp_f32 right before a conversion writes the first register
of one of its sources.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_02584_amd", "csrc")
SOURCES = [os.path.join(CSRC, "ra_attn_e2m3.hip"), os.path.join(CSRC, "ra_attn_e2m3_debug.hip"),
           os.path.join(CSRC, "ra_producer.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CONV = "v_cvt_scalef32_2xpk16_fp6_f32"


def _tuples(ins):
    return [(int(a), int(b)) for a, b in re.findall(r"v\[(\d+):(\d+)\]", ins)]


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
        if not ins.startswith(CONV):
            continue
        dst, s0, s1 = _tuples(ins)[:3]
        for src in (s0, s1):
            if max(dst[0], src[0]) <= min(dst[1], src[1]):
                out.append(("result overlaps a source", ins))
        prev = body[i - 1] if i else ""
        m = re.match(r"v_exp_f32(?:_e32|_e64)?\s+v(\d+)", prev)
        if m and int(m.group(1)) in (s0[0], s1[0]):
            out.append(("exp result read with no wait state", prev + " ; " + ins))
    return out


_ASM_CACHE = []


def _asm():
    """gfx950 assembly of the translation units (attention, debug attention, producers), compiled in parallel
    once per test session."""
    if not _ASM_CACHE:
        _ASM_CACHE.append(_compile())
    return _ASM_CACHE[0]


def _compile():
    with tempfile.TemporaryDirectory() as td:
        procs = []
        for i, src in enumerate(SOURCES):
            out = os.path.join(td, f"k{i}.s")
            cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-ffp-contract=off", "-Xclang",
                   "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
                   "--cuda-device-only", "-S", "-x", "hip", src, "-o", out]
            procs.append((subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True), out))
        text = []
        for pr, out in procs:
            _, err = pr.communicate()
            assert pr.returncode == 0, err[-2000:]
            with open(out) as f:
                text.append(f.read())
        return "\n".join(text)


def test_violation_scan_detects_both_patterns():
    """The scan itself flags the two patterns (hand-written instruction lists)."""
    overlap = [CONV + " v[96:101], v[66:81], v[82:97], s27"]
    early = ["v_exp_f32_e32 v66, v66", CONV + " v[140:145], v[66:81], v[82:97], s27"]
    clean = ["v_exp_f32_e32 v67, v67", "s_nop 0", CONV + " v[140:145], v[66:81], v[82:97], s27"]
    assert _violations(overlap) and _violations(early) and not _violations(clean)


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not available")
def test_fp6_pack_register_hazards():
    asm = _asm()
    n_conv, bad = 0, {}
    for kern, body in _kernels(asm):
        n_conv += sum(1 for b in body if b.startswith(CONV))
        v = _violations(body)
        if v:
            bad[kern] = v[:3]
    assert n_conv > 0, "no packing conversion found: the scan is not looking at the kernels"
    producers = [k for k, body in _kernels(asm) if "k_pass" in k and any(b.startswith(CONV) for b in body)]
    assert producers, "the Q/K producer's E2M3 packing was not found"
    assert not bad, f"packing-conversion register hazards: {bad}"


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not available")
def test_no_kernel_uses_scratch():
    """No production kernel of these units keeps anything in per-lane private
    memory: a small array indexed with a run-time value (or a by-value argument
    indexed that way) lands there and costs a round trip to memory per access.
    Exempt: the debug instantiations of the attention kernel (they dump S, P
    codes and maxima for the parity tests and spill freely)."""
    asm = _asm()
    names = re.findall(r"\.amdhsa_kernel\s+(\S+)", asm)
    sizes = [int(z) for z in re.findall(r"\.amdhsa_private_segment_fixed_size\s+(\d+)", asm)]
    assert names and len(names) == len(sizes), "kernel descriptors not found"
    bad = []
    for n, z in zip(names, sizes):
        m = re.search(r"k_attn_e2m3ILi\d+ELb([01])ELb([01])ELb([01])ELb([01])ELb([01])E", n)
        if m and m.group(3) == "1":
            continue                      # debug dump instantiation
        if z > 0:
            bad.append((n, z))
    assert any("k_pass" in n for n in names) and any("k_attn_e2m3" in n for n in names)
    assert not bad, f"kernels with a private segment: {bad}"
