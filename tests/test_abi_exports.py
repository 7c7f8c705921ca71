"""The C-ABI library loads and exports every symbol include/gnnav.h declares.

No compute call is made, so this runs without a GPU.
"""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gnnav.h")
LIB = os.path.join(ROOT, "paper_2404_09544_amd", "libgnnav.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gnnav_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ["gnnav_build_csr", "gnnav_build_cache", "gnnav_sample", "gnnav_gather",
                 "gnnav_sage_forward"]:
        assert must in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(LIB), "build first: python paper_2404_09544_amd/build.py"
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_export():
    import paper_2404_09544_amd as g
    assert sorted(g.EXPORTS) == declared_functions()
    assert g.abi_version() == 1
    assert g._lib.gnnav_last_error() == b""


def test_combine_kernel_choice():
    """Host-only query of the combine kernel a launch takes: few rows run the
    skinny kernel, larger fp32 the split-bf16 kernel, larger bf16 the ring."""
    import paper_2404_09544_amd as g
    assert g.combine_kernel(1024, 41, "f32") == "skinny"      # 16 64x64 tiles
    assert g.combine_kernel(10176, 64, "f32") == "skinny"     # 159 64x64 tiles
    assert g.combine_kernel(10177, 47, "f32") == "split"      # 160 tiles
    assert g.combine_kernel(20902, 256, "f32") == "split"
    assert g.combine_kernel(106857, 256, "bf16") == "ring"
    assert g.combine_kernel(100, 3000, "bf16") == "skinny"
    for bad in [(0, 5, "f32"), (5, 0, "f32")]:
        try:
            g.combine_kernel(*bad)
        except g.GnnavError:
            continue
        raise AssertionError(f"{bad} accepted")


def test_stream_create_argument_checks():
    """gnnav_stream_create rejects a bad share before touching the device,
    and leaves *out unwritten when it fails."""
    import paper_2404_09544_amd as g
    lib = g._lib
    out = ctypes.c_void_p(12345)
    for part, parts in [(0, 0), (0, 9), (-1, 2), (2, 2), (3, 1)]:
        assert lib.gnnav_stream_create(part, parts, ctypes.byref(out)) == 1, (part, parts)
        assert out.value == 12345
        assert b"outside" in lib.gnnav_last_error()
    assert lib.gnnav_stream_create(0, 2, None) == 1
    assert lib.gnnav_stream_destroy(None) == 0
