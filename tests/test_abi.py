"""The C ABI on the CPU: the library loads without a GPU, exports every entry point the
header declares, and rejects bad arguments on the host, before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2508_06024_amd import ec2moe as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ec2moe.h")

OK, INVALID, UNSUPPORTED, TOO_FEW, WS_SMALL = 0, 1, 2, 3, 4


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:ec2moe_status|const char\s*\*)\s*(ec2moe_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_expected_calls():
    names = declared_functions()
    for n in ("ec2moe_group_gate", "ec2moe_moe_forward", "ec2moe_lowrank_encode", "ec2moe_lowrank_decode",
              "ec2moe_permute", "ec2moe_combine", "ec2moe_expert_ffn"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(E.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(declared_functions()) == sorted(E.EXPORTS)


def test_status_strings():
    assert E.status_string(0) == "ok"
    assert "candidate" in E.status_string(3)
    assert E.status_string(99) == "unknown status"


def _desc(**kw):
    base = dict(n_tokens=64, n_experts=8, n_groups=2, d_model=128, ffn_hidden=256, top_k=2, dtype=E.BF16,
                renormalize=True)
    base.update(kw)
    return E.moe_desc(**base)


def _ws_size(desc):
    n = ctypes.c_size_t(0)
    st = E._lib.ec2moe_moe_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("kw,status", [
    (dict(n_groups=3), OK),                 # K need not divide M after the gate
    (dict(n_groups=9), INVALID),            # K > M
    (dict(top_k=9), INVALID),               # k > M
    (dict(n_tokens=-1), INVALID),
    (dict(d_model=0), INVALID),
    (dict(dtype=7), INVALID),
    (dict(d_model=96), UNSUPPORTED),        # not a multiple of 128
    (dict(ffn_hidden=200), UNSUPPORTED),
    (dict(n_experts=512, n_groups=8), UNSUPPORTED),
    (dict(top_k=17, n_experts=32, n_groups=4), UNSUPPORTED),
    (dict(), OK),
])
def test_descriptor_validation(kw, status):
    st, n = _ws_size(_desc(**kw))
    assert st == status, E.last_error()
    if status == OK:
        assert n > 0
    else:
        assert E.last_error()


def test_descriptor_flags():
    d = _desc(activation="relu")
    assert d.flags == E.GATE_RENORMALIZE | E.EXPERT_RELU
    assert _ws_size(d)[0] == OK
    d.flags = 4  # no such flag
    assert _ws_size(d)[0] == INVALID and "flags" in E.last_error()
    with pytest.raises(ValueError):
        _desc(activation="gelu")


def _gate_ex(desc, words, top_groups=0, sizes=None, ptr=1 << 20):
    arr = E.mask_array(words)
    p = ctypes.c_void_p(ptr)
    opts = E.gate_opts(top_groups, sizes)
    return E._lib.ec2moe_group_gate_ex(ctypes.byref(desc), ctypes.byref(opts), arr, p, p, None, p, None, p, p,
                                       None, None)


def test_gate_options_validation():
    d0 = _desc(n_tokens=0, n_experts=12, n_groups=5)  # K does not divide M: fine with sizes
    assert _gate_ex(d0, [0xFFF], sizes=[2, 3, 1, 4, 2]) == OK
    assert _gate_ex(d0, [0xFFF], sizes=[2, 3, 1, 4, 3]) == INVALID and "exceed" in E.last_error()
    assert _gate_ex(d0, [0xFFF], sizes=[2, 3, 1, 4, 1]) == INVALID and "sum" in E.last_error()
    assert _gate_ex(d0, [0xFFF], sizes=[2, 3, 0, 5, 2]) == INVALID
    assert _gate_ex(d0, [0xFFF]) == INVALID  # equal groups need K | M
    d1 = _desc(n_tokens=0)
    assert _gate_ex(d1, [0xFF], top_groups=-1) == INVALID
    assert _gate_ex(d1, [0xFF], top_groups=1) == OK
    assert E._lib.ec2moe_group_gate_ex(ctypes.byref(d1), None, E.mask_array([0xFF]), None, None, None, None,
                                       None, None, None, None, None) == OK


def _gate_ws_size(desc):
    n = ctypes.c_size_t(0)
    st = E._lib.ec2moe_gate_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    return st, n.value


def test_gate_workspace_size():
    """Small batches (under 64 tiles of 16 tokens) with d >= 2048 get d split over up to 32
    workgroups per tile, about 256 workgroups in all; the partials are float32
    [tile][split][16 * padded row blocks][16]."""
    dec = dict(n_tokens=32, n_experts=64, n_groups=8, d_model=4096, top_k=8)
    assert _gate_ws_size(_desc(**dec)) == (OK, 2 * 32 * 80 * 16 * 4)
    assert _gate_ws_size(_desc(**dict(dec, dtype=E.F32))) == (OK, 2 * 32 * 80 * 16 * 4)
    assert _gate_ws_size(_desc(**dict(dec, n_tokens=33))) == (OK, 3 * 32 * 80 * 16 * 4)
    assert _gate_ws_size(_desc(**dict(dec, n_tokens=160))) == (OK, 10 * 16 * 80 * 16 * 4)  # 10 tiles: 16 splits
    assert _gate_ws_size(_desc(**dict(dec, n_tokens=1024))) == (OK, 0)   # 64 tiles: unsplit
    assert _gate_ws_size(_desc(**dict(dec, n_tokens=0))) == (OK, 0)
    assert _gate_ws_size(_desc(n_tokens=64, d_model=1024)) == (OK, 0)   # narrow gates run unsplit
    # 320 gate rows pad to 20 blocks of 16; 2048 = 16 splits of 128
    assert _gate_ws_size(_desc(n_tokens=53, n_experts=256, n_groups=64, d_model=2048, top_k=16)) == \
        (OK, 4 * 16 * 320 * 16 * 4)


def test_gate_workspace_validation():
    desc = _desc(n_tokens=32, n_experts=64, n_groups=8, d_model=4096, top_k=8)
    need = _gate_ws_size(desc)[1]
    arr = E.mask_array([(1 << 64) - 1])
    p = ctypes.c_void_p(1 << 20)
    call = lambda opts: E._lib.ec2moe_group_gate_ex(ctypes.byref(desc), ctypes.byref(opts), arr, p, p, None, p,
                                                    None, p, p, None, None)
    assert call(E.GateOpts(0, None, 1 << 20, need - 1)) == WS_SMALL and "gate workspace" in E.last_error()
    assert call(E.GateOpts(0, None, (1 << 20) + 8, need)) == INVALID and "aligned" in E.last_error()


def test_workspace_size_grows_with_tokens():
    _, a = _ws_size(_desc(n_tokens=64))
    _, b = _ws_size(_desc(n_tokens=4096))
    assert b > a
    _, z = _ws_size(_desc(n_tokens=0))
    assert 0 < z < a


def _gate(desc, words, ptr=1 << 20):
    arr = E.mask_array(words)
    p = ctypes.c_void_p(ptr)
    return E._lib.ec2moe_group_gate(ctypes.byref(desc), arr, p, p, None, p, None, p, p, None, None)


def test_plain_gate_needs_equal_groups():
    assert _gate(_desc(n_groups=3), [0xFF]) == INVALID and "divide" in E.last_error()


def test_gate_rejects_too_few_candidates_before_launch():
    assert _gate(_desc(top_k=2), [0b1]) == TOO_FEW
    assert "candidate" in E.last_error()


def test_gate_rejects_mask_bits_beyond_experts():
    assert _gate(_desc(), [0x1FF]) == INVALID


def test_gate_rejects_null_and_misaligned_pointers():
    words = [0xFF]
    d = _desc()
    arr = E.mask_array(words)
    assert E._lib.ec2moe_group_gate(ctypes.byref(d), arr, None, None, None, None, None, None, None, None,
                                    None) == INVALID
    assert _gate(d, words, ptr=(1 << 20) + 4) == INVALID
    assert "aligned" in E.last_error()


def test_gate_with_no_tokens_is_a_no_op():
    assert _gate(_desc(n_tokens=0), [0xFF]) == OK


def test_moe_forward_rejects_small_workspace():
    d = _desc()
    _, need = _ws_size(d)
    p = ctypes.c_void_p(1 << 20)
    st = E._lib.ec2moe_moe_forward(ctypes.byref(d), p, p, p, p, p, p, p, need - 1, None)
    assert st == WS_SMALL
    st = E._lib.ec2moe_moe_forward(ctypes.byref(d), p, p, p, p, p, p, None, need, None)
    assert st == INVALID


def test_permute_requires_x_and_x_perm_together():
    d = _desc()
    _, need = _ws_size(d)
    p = ctypes.c_void_p(1 << 20)
    st = E._lib.ec2moe_permute(ctypes.byref(d), p, p, p, p, p, None, p, need, None)
    assert st == INVALID


def test_codec_validation():
    def size(**kw):
        base = dict(h=64, w=128, r_h=16, r_w=16, dtype=E.F32, n_slices=1)
        base.update(kw)
        desc = E.codec_desc(**base)
        n = ctypes.c_size_t(0)
        return E._lib.ec2moe_lowrank_workspace_size(ctypes.byref(desc), ctypes.byref(n)), n.value

    assert size()[0] == OK and size()[1] > 0
    assert size(r_h=80)[0] == INVALID      # r_h > h
    assert size(r_w=24)[0] == UNSUPPORTED  # not a multiple of 16
    assert size(w=96)[0] == UNSUPPORTED
    assert size(r_w=512, w=1024)[0] == UNSUPPORTED


def test_profile_collect_without_records():
    assert E.profile_collect() == {}


# ----------------------------------------------------------------------------- descriptor layout

# The descriptors' field order is the interface contract: T, d, M, K, k, H, dtype, flags for
# the MoE layer and c, h, w, r_h, r_w, dtype for the codec, every field 4 bytes.
MOE_FIELDS = ["n_tokens", "d_model", "n_experts", "n_groups", "top_k", "ffn_hidden", "dtype", "flags"]
CODEC_FIELDS = ["n_slices", "h", "w", "r_h", "r_w", "dtype"]


def _c_offsets(tmp_path):
    """offsetof / sizeof of every descriptor field as a C compiler lays out the header."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ec2moe.h"', 'int main(void) {']
    for s, fields in (("ec2moe_moe_desc", MOE_FIELDS), ("ec2moe_codec_desc", CODEC_FIELDS)):
        for f in fields:
            lines.append(f'printf("{s} {f} %zu %zu\\n", offsetof({s}, {f}), sizeof((({s}*)0)->{f}));')
        lines.append(f'printf("{s} sizeof %zu 0\\n", sizeof({s}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "offsets.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "offsets"
    subprocess.run([cc, "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe)], check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    res = {}
    for ln in out.splitlines():
        s, f, off, size = ln.split()
        res[(s, f)] = (int(off), int(size))
    return res


def test_descriptor_layout_matches_the_contract(tmp_path):
    c = _c_offsets(tmp_path)
    for s, fields, py in (("ec2moe_moe_desc", MOE_FIELDS, E.MoeDesc), ("ec2moe_codec_desc", CODEC_FIELDS, E.CodecDesc)):
        for i, f in enumerate(fields):
            assert c[(s, f)] == (4 * i, 4), (s, f, c[(s, f)])
            assert getattr(py, f).offset == 4 * i and getattr(py, f).size == 4, (s, f)
        assert c[(s, "sizeof")][0] == 4 * len(fields) == ctypes.sizeof(py)
        assert [n for n, _ in py._fields_] == fields
    # a descriptor built by the binding carries each shape in its own field
    d = E.moe_desc(n_tokens=11, n_experts=12, n_groups=3, d_model=256, ffn_hidden=384, top_k=2, dtype=E.BF16)
    raw = bytes(d)
    vals = [int.from_bytes(raw[4 * i:4 * i + 4], "little") for i in range(8)]
    assert vals == [11, 256, 12, 3, 2, 384, E.BF16, E.GATE_RENORMALIZE]


def test_permute_noalloc_rejects_inputs_beyond_its_array():
    """ceil(T*k / 1024) * n_experts count words must fit the library's 262144-word array; the
    error comes from the host before any launch (no device pointer is touched)."""
    p = ctypes.c_void_p(1 << 20)
    over = _desc(n_tokens=1048577, top_k=1, n_experts=256, n_groups=16)
    assert E._lib.ec2moe_permute_noalloc(ctypes.byref(over), p, None, p, p, p, None, None) == UNSUPPORTED
    assert "count words" in E.last_error()
    assert E._lib.ec2moe_permute_noalloc(ctypes.byref(_desc()), p, p, p, p, p, None, None) == INVALID  # x without x_perm
    assert E._lib.ec2moe_permute_noalloc(ctypes.byref(_desc()), p, None, None, p, p, None, None) == INVALID
