"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rotate_attn.h")


def _ra():
    from paper_2607_02584_amd import rotate_attn as ra
    if not os.path.exists(ra.LIB_PATH):
        pytest.skip("library not built")
    return ra


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(rotate_attn_\w+)\(", text, re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ["rotate_attn_quantize_qk", "rotate_attn_fwd_int4", "rotate_attn_fwd_fp16", "rotate_attn_quantize_v",
              "rotate_attn_attn_int4", "rotate_attn_fwd", "rotate_attn_workspace_size"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    ra = _ra()
    L = ctypes.CDLL(ra.LIB_PATH)
    for n in declared_functions():
        assert hasattr(L, n), n


def _base(ra, **kw):
    return ra.make_params(1, 2, (4, 16, 16), **kw)


@pytest.mark.parametrize("field,value,status", [
    ("D", 64, -2),
    ("N", 1000, -1),           # T*Hg*W != N
    ("B", 0, -1),
    ("rope_split", (44, 42, 40), -1),
    ("rope_split", (43, 43, 42), -1),
    ("rope_theta", 0.0, -1),
    ("rotation", 4, -1),
    ("p_quant", 5, -1),
    ("smooth", 8, -1),
    ("v_rotation", 2, -1),
    ("l_quant", 2, -1),
    ("q_group", 3, -2),
    ("k_group", 8, -2),
    ("kv_block", 32, -2),
    ("v_group", 96, -2),       # not a multiple of kv_block and < N
    ("in_dtype", 2, -1),
    ("out_dtype", 7, -1),
    ("code_format", 2, -1),
    ("sm_scale", -1.0, -1),
])
def test_validation_rejects(field, value, status):
    ra = _ra()
    p = _base(ra)
    if field == "rope_split":
        p.rope_split[:] = list(value)
    else:
        setattr(p, field, value)
    with pytest.raises(ra.RAError) as e:
        ra.layout(p)
    assert e.value.status == status


def test_validation_accepts_defaults_and_reports_sizes():
    ra = _ra()
    p = _base(ra)
    L = ra.layout(p)
    assert L["n_pad"] == 1024 and L["qk_code_bytes"] == 2 * 1024 * 96 and L["v_scale_count"] == 2 * 8 * 128
    L4 = ra.layout(ra.make_params(1, 2, (4, 16, 16), code_format=ra.CODES_INT4))
    assert L4["qk_code_bytes"] == 2 * 1024 * 64 and L4["v_code_bytes"] == 2 * 1024 * 64
    assert ra.workspace_size(p, ra.PATH_INT4) > 3 * L["qk_code_bytes"]
    assert ra.workspace_size(p, ra.PATH_FP16) >= 3 * 2 * 1024 * 128 * 2
    p2 = ra.make_params(1, 1, (3, 7, 11), v_group=10 ** 6)
    assert ra.layout(p2)["n_pad"] == 256 and ra.layout(p2)["v_scale_count"] == 128


def test_groups_and_blocks_the_contract_lists_are_accepted():
    """k_group 16 (per block of 16 keys) and kv_block 128 for both paths are
    valid requests; their workspaces include the RoPE tables."""
    ra = _ra()
    for kg in (1, 16, 32, 64, 128):
        assert ra.layout(_base(ra, k_group=kg))["k_scale_count"] == 2 * 1024 // kg
    for kv in (64, 128):
        p = _base(ra, kv_block=kv, v_group=128)
        tables = (4 * 22 + 16 * 21 + 16 * 21 + 64) * 16
        assert ra.workspace_size(p, ra.PATH_FP16) >= 3 * 2 * 1024 * 128 * 2 + tables
        assert ra.workspace_size(p, ra.PATH_INT4) >= 3 * 2 * 1024 * 96 + tables


def test_rotation_blocks_must_be_orthogonal():
    """Sec. 4.1 needs R R^T = I: a scaled or sheared block is rejected before any
    HIP call; O(2) blocks (rotations and reflections) are accepted."""
    import math
    ra = _ra()
    c, s = math.cos(0.3), math.sin(0.3)
    R = [[[c, s], [-s, c]] if i % 2 else [[c, s], [s, -c]] for i in range(64)]
    for rot in (ra.ROT_INTERLEAVED, ra.ROT_HALF):
        ra.layout(_base(ra, rotation=rot, rot_blocks=R))
        bad = [list(map(list, b)) for b in R]
        bad[17] = [[1.01 * c, s], [-s, c]]
        with pytest.raises(ra.RAError) as e:
            ra.layout(_base(ra, rotation=rot, rot_blocks=bad))
        assert e.value.status == -1 and "orthogonal" in str(e.value)
        shear = [list(map(list, b)) for b in R]
        shear[63] = [[1.0, 0.5], [0.0, 1.0]]
        with pytest.raises(ra.RAError):
            ra.layout(_base(ra, rotation=rot, rot_blocks=shear))
    # the blocks are unused (and unchecked) for the other rotations
    ra.layout(_base(ra, rotation=ra.ROT_NONE, rot_blocks=[[[2.0, 0.0], [0.0, 2.0]]] * 64))


def test_null_pointers_and_workspace_errors_before_gpu():
    ra = _ra()
    L = ra.lib()
    p = _base(ra)
    P = ctypes.c_void_p
    # NULL tensors -> RA_ERR_INVALID; no GPU call happens on this path
    st = L.rotate_attn_fwd_int4(ctypes.byref(p), None, None, None, None, None, 0, None)
    assert st == -1 and b"NULL" in L.rotate_attn_last_error()
    fake = P(0x1000)
    st = L.rotate_attn_fwd_int4(ctypes.byref(p), fake, fake, fake, fake, None, 0, None)
    assert st == -3
    st = L.rotate_attn_fwd_int4(ctypes.byref(p), fake, fake, fake, fake, P(0x1001), 1 << 30, None)
    assert st == -3  # misaligned
    st = L.rotate_attn_fwd_fp16(ctypes.byref(p), fake, fake, fake, fake, P(0x1000), 16, None)
    assert st == -3  # too small
    st = L.rotate_attn_attn_int4_debug(ctypes.byref(p), fake, fake, fake, fake, fake, fake, None, None, fake, 5, 0,
                                       1, None, None, None, None)
    assert st == -1  # bh out of range
    # Q smoothing needs the per-key bias buffer on both sides
    pq = _base(ra, smooth=ra.SMOOTH_K | ra.SMOOTH_V | ra.SMOOTH_Q)
    st = L.rotate_attn_quantize_qk(ctypes.byref(pq), fake, fake, fake, fake, fake, fake, None, None, None, fake,
                                   1 << 30, None)
    assert st == -1 and b"k_bias" in L.rotate_attn_last_error()
    st = L.rotate_attn_attn_int4(ctypes.byref(pq), fake, fake, fake, fake, fake, fake, None, None, fake, None)
    assert st == -1 and b"k_bias" in L.rotate_attn_last_error()
    assert ra.layout(pq)["k_bias_count"] == 2 * 1024
    assert ra.workspace_size(pq, ra.PATH_INT4) >= ra.workspace_size(p, ra.PATH_INT4) + 2 * 1024 * 4
    assert L.rotate_attn_error_string(-4) == b"HIP runtime error"
    assert L.rotate_attn_fwd_int4(None, fake, fake, fake, fake, fake, 1 << 30, None) == -1
    # inputs and code buffers are moved in 16-byte pieces: an 8-byte aligned one is refused
    half = P(0x1008)
    for args in ((half, fake, fake), (fake, half, fake), (fake, fake, half)):
        st = L.rotate_attn_fwd_int4(ctypes.byref(p), *args, fake, fake, 1 << 30, None)
        assert st == -1 and b"16-byte aligned" in L.rotate_attn_last_error()
    st = L.rotate_attn_quantize_qk(ctypes.byref(p), fake, fake, half, fake, fake, fake, None, None, None, fake,
                                   1 << 30, None)
    assert st == -1 and b"16-byte aligned" in L.rotate_attn_last_error()
    st = L.rotate_attn_quantize_v(ctypes.byref(p), fake, half, fake, None, fake, 1 << 30, None)
    assert st == -1 and b"16-byte aligned" in L.rotate_attn_last_error()


def test_binding_checks_tensors_before_the_library():
    """The ctypes binding refuses host tensors, non-contiguous tensors and
    buffers smaller than the call touches (the C ABI cannot see sizes)."""
    ra = _ra()
    torch = pytest.importorskip("torch")
    p = _base(ra)
    x = torch.zeros(2, 1024, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        ra.fwd_int4(p, x, x, x, x, x)
    with pytest.raises(ValueError, match="required"):
        ra._need(None, 16, "q")
    t = torch.zeros(4, 4)
    with pytest.raises(ValueError, match="contiguous"):
        ra._need(t.t(), 16, "q")
    with pytest.raises(ValueError, match="needs 128"):
        ra._need(t, 128, "q")
    # fp32 output needs 4 bytes per element of [B][H][N][D]
    assert ra._io_bytes(ra.make_params(1, 2, (4, 16, 16), out_dtype=ra.FP32)) == (2 * 262144, 4 * 262144)
