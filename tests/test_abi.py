"""CPU checks of the C ABI: the library loads, exports every function that
include/rs3.h declares, and rejects malformed arguments on the host before
any HIP call (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "rs3.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:rs3_status|void|const char\s*\*)\s*(rs3_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22526_amd as p
    return p.lib()


def test_library_exports_header(lib):
    names = _declared()
    assert len(names) >= 19
    missing = [n for n in names if not hasattr(lib, n)]
    assert missing == []
    import paper_2608_22526_amd as p
    assert sorted(p.exported_symbols()) == names


def test_status_strings(lib):
    for code in range(5):
        assert lib.rs3_status_str(code)
    assert lib.rs3_status_str(0) == b"ok"


def test_host_validation_before_device(lib):
    import paper_2608_22526_amd as p
    g = p.Grid(64, 64, 1)
    bad = p.Grid(0, 64, 1)
    huge = p.Grid(256, 256, 1)
    sz = ctypes.c_size_t()
    assert lib.rs3_select_workspace_size(ctypes.byref(g), 1, 0, ctypes.byref(sz)) == p.RS3_OK
    assert sz.value >= 64 * 64 * 8   # fp64 energies plus per-block ranges
    assert lib.rs3_select_workspace_size(ctypes.byref(bad), 1, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    assert lib.rs3_select_workspace_size(ctypes.byref(huge), 1, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    assert lib.rs3_select_workspace_size(ctypes.byref(g), 0, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    assert lib.rs3_select_workspace_size(ctypes.byref(g), p.RS3_MAX_OBJ + 1, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    # null handles and pointers
    assert lib.rs3_select_queries(None, 1, None, None, None, 0, 256, 1, None, None, None, 0, None, None, None,
                                  None) == p.RS3_E_INVALID
    assert lib.rs3_readout(None, ctypes.byref(g), 1, None, 0, None, None, None, 0, 0, 0, None, 0, 0, None, 0,
                           None) == p.RS3_E_INVALID
    assert lib.rs3_commit(None, 1, ctypes.byref(g), None, None, 0, None, 0, 0, 0, 4096, None, None) == p.RS3_E_INVALID
    assert lib.rs3_layer_set_rope(None, 4, 4, None) == p.RS3_E_INVALID
    assert lib.rs3_layer_set_rope_axial(None, 4, 4, 10000.0) == p.RS3_E_INVALID
    out = ctypes.c_void_p()
    assert lib.rs3_track_create(0, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_bank_create(None, 100, 4, 1, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_readout_workspace_size(None, 1, 10, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    # layer shape rules: d_h must be 32/64/128/256 for bf16, d_kv a multiple of 16
    w = (ctypes.c_uint16 * (256 * 256))()
    assert lib.rs3_layer_create(256, 3, 64, p.RS3_BF16, 0, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_layer_create(256, 1, 60, p.RS3_BF16, 0, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_layer_create(256, 1, 64, 7, 0, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    # absorbed attention needs one head, and a bf16 width in {64, 128, 256}
    assert lib.rs3_layer_create(256, 8, 64, p.RS3_BF16, 1, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_layer_create(256, 1, 32, p.RS3_BF16, 1, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_layer_create(256, 1, 64, p.RS3_BF16, 2, w, w, w, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_profile_enable(1, 0) == p.RS3_E_INVALID


def test_frame_io_layout_matches_header(tmp_path):
    """The binding's rs3_frame_io mirror has the header's size and field
    offsets (compiled here with the host C compiler)."""
    import shutil
    import subprocess
    from paper_2608_22526_amd._binding import FrameIO
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    names = [n for n, _ in FrameIO._fields_]
    src = tmp_path / "layout.c"
    src.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"rs3.h\"\nint main(void) {\n"
                   "  printf(\"%zu\", sizeof(rs3_frame_io));\n"
                   + "".join("  printf(\" %%zu\", offsetof(rs3_frame_io, %s));\n" % n for n in names)
                   + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.check_call([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    got = [int(v) for v in subprocess.check_output([str(exe)]).split()]
    assert got == [ctypes.sizeof(FrameIO)] + [getattr(FrameIO, n).offset for n in names]


def test_stack_host_validation(lib):
    """rs3_stack_create / rs3_stack_readout reject bad shapes and pointers on
    the host, before any device call."""
    import paper_2608_22526_amd as p
    from paper_2608_22526_amd._binding import StackWeights
    out = ctypes.c_void_p()
    buf = (ctypes.c_uint16 * (256 * 2048))()
    w = (StackWeights * 2)()
    for i in range(2):
        for name, _ in StackWeights._fields_:
            setattr(w[i], name, ctypes.addressof(buf))
    bad = [(0, 256, 1, 64, 2048, p.RS3_BF16), (17, 256, 1, 64, 2048, p.RS3_BF16),   # layer count
           (2, 128, 1, 64, 2048, p.RS3_BF16), (2, 256, 3, 64, 2048, p.RS3_BF16),    # d_model, heads
           (2, 256, 16, 64, 2048, p.RS3_BF16), (2, 256, 1, 32, 2048, p.RS3_BF16),   # head width 16, d_kv
           (2, 256, 1, 64, 2000, p.RS3_BF16), (2, 256, 1, 64, 8448, p.RS3_BF16),    # F
           (2, 256, 1, 64, 2048, p.RS3_F32)]
    for args in bad:
        assert lib.rs3_stack_create(*args, w, ctypes.byref(out)) == p.RS3_E_INVALID, args
    w[1].W2 = None
    assert lib.rs3_stack_create(2, 256, 1, 64, 2048, p.RS3_BF16, w, ctypes.byref(out)) == p.RS3_E_INVALID
    assert lib.rs3_stack_create(2, 256, 1, 64, 2048, p.RS3_BF16, None, ctypes.byref(out)) == p.RS3_E_INVALID
    g = p.Grid(64, 64, 1)
    sz = ctypes.c_size_t()
    assert lib.rs3_stack_workspace_size(None, 10, 0, ctypes.byref(sz)) == p.RS3_E_INVALID
    assert lib.rs3_stack_readout(None, ctypes.byref(g), None, None, None, None, 0, 0, None, 0, None, 0,
                                 None) == p.RS3_E_INVALID


def test_stack_weights_layout_matches_header(tmp_path):
    import shutil
    import subprocess
    from paper_2608_22526_amd._binding import StackWeights
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    names = [n for n, _ in StackWeights._fields_]
    src = tmp_path / "layout.c"
    src.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"rs3.h\"\nint main(void) {\n"
                   "  printf(\"%zu\", sizeof(rs3_stack_weights));\n"
                   + "".join("  printf(\" %%zu\", offsetof(rs3_stack_weights, %s));\n" % n for n in names)
                   + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.check_call([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    got = [int(v) for v in subprocess.check_output([str(exe)]).split()]
    assert got == [ctypes.sizeof(StackWeights)] + [getattr(StackWeights, n).offset for n in names]
