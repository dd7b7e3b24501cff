"""The C-ABI library loads on a machine without a GPU, exports every entry
point that include/moddit.h declares, and rejects bad arguments on the host
before touching the device."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moddit.h")
LIB = os.path.join(ROOT, "paper_2601_11641_amd", "libmoddit.so")


@pytest.fixture(scope="module")
def M():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    import paper_2601_11641_amd as m
    return m


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mod_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for core in ("mod_collect_stats", "mod_predict_block_mask", "mod_block_sparse_attn_fwd"):
        assert core in names


def test_library_exports_every_declared_symbol(M):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (mod_[a-z_]+)\b", out))
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    assert set(M.EXPORTED) == set(declared_functions())


def test_block_and_coefficient_counts(M):
    s = M.make_shape(1, 24, 118800, 128, 128, 3600)
    assert M.mod_num_blocks(s) == 929 and M.mod_num_coeffs(s) == 3 * 929 - 1 + 33
    s = M.make_shape(1, 40, 75600, 128, 128, 3600)
    assert M.mod_num_blocks(s) == 591 and M.mod_num_coeffs(s) == 3 * 591 - 1 + 21
    assert M.mod_num_blocks(None) == 0
    assert M.mod_num_coeffs(M.make_shape(1, 1, 100, 64, 64, 30)) == 0
    # a text segment: the masks count every block, the model the video ones
    s = M.make_shape(1, 24, 118800 + 256, 128, 128, 3600, text_tokens=256)
    assert M.mod_num_blocks(s) == 931 and M.mod_num_coeffs(s) == 3 * 929 - 1 + 33
    assert M.num_video_blocks(s) == 929
    s = M.make_shape(1, 2, 1000 + 100, 64, 64, 250, text_tokens=100)
    assert M.mod_num_blocks(s) == 18 and M.mod_num_coeffs(s) == 3 * 16 - 1 + 4
    assert M.mod_num_coeffs(M.make_shape(1, 2, 1024, 64, 64, 256, text_tokens=1024)) == 0


@pytest.mark.parametrize("shape,status", [
    ((1, 2, 1024, 96, 64, 256), 2),      # d unsupported
    ((1, 2, 1024, 64, 32, 256), 2),      # block unsupported
    ((1, 2, 1024, 64, 64, 1000), 2),     # not whole frames
    ((1, 2, 1024, 64, 64, 1024), 2),     # a single frame
    ((0, 2, 1024, 64, 64, 256), 1),      # empty batch
    ((1, 2, 1024, 64, 64, 0), 1),        # frame_tokens missing
    ((1, 1, 128 * 4097, 64, 128, 128), 2),  # n above the limit
    ((1, 2, 1024 + 64, 64, 64, 256, 64 + 1), 2),   # video not whole frames
    ((1, 2, 512 + 64, 64, 64, 256, 64 + 256), 2),  # a single video frame
    ((1, 2, 1024, 64, 64, 256, -1), 1),            # negative text_tokens
    ((1, 2, 1024, 64, 64, 256, 1024), 1),          # no video tokens
])
def test_create_rejects_bad_shapes_on_host(M, shape, status):
    with pytest.raises(M.ModError) as e:
        M.mod_stats_create(M.make_shape(*shape), M.make_params())
    assert e.value.status == status
    assert M.mod_last_error()


def test_create_rejects_bad_params(M):
    with pytest.raises(M.ModError) as e:
        M.mod_stats_create(M.make_shape(1, 2, 1024, 64, 64, 256), M.make_params(anchor_rule=3))
    assert e.value.status == M.MOD_ERR_INVALID_ARG


def test_attention_rejects_null_pointers_on_host(M):
    lib = M.raw_lib()
    s = M.make_shape(1, 2, 1024, 64, 64, 256)
    import ctypes
    st = lib.mod_block_sparse_attn_fwd(ctypes.byref(s), None, None, None, None, None, 0.0, None,
                                       None, None, 0, None)
    assert st == M.MOD_ERR_INVALID_ARG
    st = lib.mod_block_sparse_attn_fwd(None, 1, 1, 1, 1, 1, 0.0, 1, None, None, 0, None)
    assert st == M.MOD_ERR_INVALID_ARG
    assert M.mod_status_string(st) == "MOD_ERR_INVALID_ARG"


def test_workspace_size(M):
    """The attention workspace holds the work plan (one int per (head, pair of
    query blocks) plus per-head tables) and, for walks longer than one
    64-step chunk, up to 1024 partial-result slots of 8 * block * (d + 1)
    bytes for the split-KV path; the plan alone is the minimum.  0 for an
    invalid shape."""
    hy = M.make_shape(1, 24, 118800, 128, 128, 3600)
    plan = M.mod_attn_plan_bytes(hy)
    assert plan >= 4 * 24 * 465 and plan % 256 == 0 and plan < 64 * 1024
    ws = M.mod_attn_workspace_bytes(hy)
    slot = 8 * 128 * 129
    assert 1024 * slot + plan <= ws <= 1024 * (slot + 64) + plan
    tiny = M.make_shape(1, 2, 1024, 64, 64, 256)           # n = 16: never split
    assert M.mod_attn_workspace_bytes(tiny) == M.mod_attn_plan_bytes(tiny)
    for bad in (M.make_shape(1, 2, 1024, 96, 64, 256), None):
        assert M.mod_attn_workspace_bytes(bad) == 0 and M.mod_attn_plan_bytes(bad) == 0


def test_struct_layouts_match_the_header(M, tmp_path):
    """The ctypes mirrors of the ABI structs have the header's layout
    (sizes and field offsets from a C program compiled against it)."""
    import ctypes
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "moddit.h"\n'
        'int main(void) {\n'
        '  printf("%zu %zu %zu %zu %zu\\n", sizeof(mod_budget), offsetof(mod_budget, mode),\n'
        '         offsetof(mod_budget, density), offsetof(mod_budget, mass), offsetof(mod_budget, patterns));\n'
        '  printf("%zu %zu %zu\\n", sizeof(mod_shape), offsetof(mod_shape, frame_tokens),\n'
        '         offsetof(mod_shape, text_tokens));\n'
        '  printf("%zu %zu %zu\\n", sizeof(mod_params), offsetof(mod_params, anchor_rule),\n'
        '         offsetof(mod_params, eta));\n'
        '  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()
    got = [int(x) for x in out]
    want = [ctypes.sizeof(M.mod_budget), M.mod_budget.mode.offset, M.mod_budget.density.offset,
            M.mod_budget.mass.offset, M.mod_budget.patterns.offset,
            ctypes.sizeof(M.mod_shape), M.mod_shape.frame_tokens.offset, M.mod_shape.text_tokens.offset,
            ctypes.sizeof(M.mod_params), M.mod_params.anchor_rule.offset, M.mod_params.eta.offset]
    assert got == want
