"""The C ABI without a GPU: the library loads, exports every entry point
declared in include/*.h, and rejects bad arguments before touching a
device."""

import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        for m in re.finditer(r"^[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M):
            if not m.group(0).lstrip().startswith(("typedef", "#")):
                names.append(m.group(1))
    return sorted(set(names))


@pytest.fixture(scope="module")
def L():
    from paper_1801_03855_amd import build as b
    if not os.path.exists(b.LIBRARY):
        b.build()
    import paper_1801_03855_amd as tc
    return tc.lib()


def test_header_declares_the_entry_points():
    names = _declared_functions()
    for required in ("tc_group_create", "tc_pack", "tc_unpack", "tc_reduce", "easgd_step",
                     "tc_reduce_ex", "easgd_step_ex", "tc_last_error"):
        assert required in names, required


def test_every_declared_symbol_is_exported(L):
    for name in _declared_functions():
        assert hasattr(L, name), f"{name} declared in include/ but not exported"


def test_version_and_empty_error(L):
    assert L.tc_version() == 100
    assert L.tc_last_error() == b""


def test_group_create_rejects_bad_sizes(L):
    assert not L.tc_group_create(None, 0)
    assert b"n must be" in L.tc_last_error()
    arr = (ctypes.c_int64 * 3)(4, -2, 5)
    assert not L.tc_group_create(arr, 3)
    assert b"negative" in L.tc_last_error()
    big = (ctypes.c_int64 * 2)(1 << 62, 1 << 62)
    assert not L.tc_group_create(big, 2)
    assert b"too large" in L.tc_last_error()


def test_null_handles_are_rejected(L):
    import paper_1801_03855_amd as tc
    arr = (ctypes.c_void_p * 1)()
    assert L.tc_reduce(None, 2, arr, None, 0, None) == tc.TC_EINVAL
    assert L.tc_reduce_ex(None, 2, arr, 0, None, 0, None) == tc.TC_EINVAL
    assert L.easgd_step(None, 2, arr, arr, None, 0.1, 0.5, None) == tc.TC_EINVAL
    assert L.easgd_step_ex(None, 2, arr, arr, 1, None, 0.1, 0.5, None) == tc.TC_EINVAL
    assert L.reduce_easgd_step(None, 2, arr, arr, 0, None, None, 1, 0.1, 0.5, None) == tc.TC_EINVAL
    assert L.reduce_easgd_step_tensor(None, 2, None, None, 0, None, None, 1, 0.1, 0.5, None) == tc.TC_EINVAL
    assert L.tc_pack(None, arr, None) == tc.TC_EINVAL
    assert L.tc_unpack(None, arr, None) == tc.TC_EINVAL
    assert not L.tc_tensorlist_create(None, 1, arr, 0)
    assert L.tc_group_numel(None) == -1
    assert L.tc_group_ntensors(None) == -1
    assert L.tc_group_offsets(None, None) == tc.TC_EINVAL
    L.tc_group_destroy(None)
    L.tc_tensorlist_destroy(None)


def test_product_path_never_touches_the_oracle():
    """Neither the package nor the C sources import, load or call the oracle."""
    pat = re.compile(r"(import\s+oracle|from\s+oracle|libtc_oracle|oracle_[a-z]+\s*\(|tc_oracle)")
    paths = glob.glob(os.path.join(ROOT, "paper_1801_03855_amd", "**", "*.*"), recursive=True)
    paths += glob.glob(os.path.join(ROOT, "include", "*.h"))
    for path in paths:
        if path.endswith((".py", ".hip", ".h", ".cpp")):
            assert not pat.search(open(path).read()), path
