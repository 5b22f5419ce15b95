"""The C-ABI library on a machine without a GPU: it loads, it exports every
symbol the header declares, and host-side argument checks return the same
status codes as the oracle (no compute call is made)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1706_01307_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    text = open(os.path.join(ROOT, "include", "spconv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spconv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    names = _declared_symbols()
    assert len(names) == 21, names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib.SIGNATURES)


def test_status_strings():
    lib = _lib.load()
    for code in (0, -1, -2, -3, -4, -5, -6, -7):
        s = lib.spconv_status_string(code).decode()
        assert s and s != "unknown status"
    assert lib.spconv_status_string(-99).decode() == "unknown status"


def _build_status(kind, D, N, size, f, s):
    lib = _lib.load()
    size = np.asarray(size, np.int32)
    f = np.asarray(f, np.int32)
    s = np.asarray(s, np.int32)
    h = ctypes.c_void_p()
    # coords pointer: a non-null dummy; every case below fails before any
    # device access
    dummy = ctypes.c_void_p(16) if N else None
    return lib.spconv_build_rulebook(kind, D, dummy, N, size.ctypes.data, f.ctypes.data,
                                     s.ctypes.data, 0, None, ctypes.byref(h)), h.value


@pytest.mark.parametrize("kind,size,f,s", [
    (0, [1, 4, 4], [1, 2, 2], [1, 1, 1]),      # even VSC filter
    (0, [1, 4, 4], [1, 3, 3], [1, 2, 2]),      # VSC with a stride
    (1, [1, 4, 4], [3, 3, 3], [1, 2, 2]),      # filter on the sample axis
    (1, [1, 4, 4], [1, 2, 2], [2, 2, 2]),      # stride on the sample axis
    (1, [1, 4, 4], [1, 0, 2], [1, 2, 2]),      # zero filter
    (1, [1, 4, 4], [1, 2, 2], [1, 0, 2]),      # zero stride
    (1, [1, 4, 70000], [1, 2, 2], [1, 2, 2]),  # extent beyond 65535
    (0, [0, 4, 4], [1, 3, 3], [1, 1, 1]),      # empty extent
])
def test_host_argument_errors_match_oracle(kind, size, f, s):
    st, h = _build_status(kind, len(size), 1, size, f, s)
    assert st == _lib.EINVAL and h is None
    coords = np.zeros((1, len(size)), np.int32)
    assert oracle.status_of_build(kind, coords, size, f, s) == oracle.EINVAL


def test_other_host_errors():
    assert _build_status(2, 3, 1, [1, 4, 4], [1, 3, 3], [1, 1, 1])[0] == _lib.EINVAL  # kind
    assert _build_status(0, 5, 1, [1] * 5, [1] * 5, [1] * 5)[0] == _lib.EINVAL       # D
    assert _build_status(0, 3, -1, [1, 4, 4], [1, 3, 3], [1, 1, 1])[0] == _lib.EINVAL
    # more offsets than the library supports (K > 1024)
    assert _build_status(0, 4, 1, [1, 99, 99, 99], [1, 11, 11, 11], [1, 1, 1, 1])[0] == _lib.EINVAL
    lib = _lib.load()
    # NULL handle / kind mismatch on the forward side
    assert lib.spconv_vsc_forward(None, 0, None, None, None, 0, None, 1, 1, None) == _lib.EINVAL
    assert lib.spconv_rulebook_status(None) == _lib.EINVAL
    assert lib.spconv_rulebook_query(None, None, None, None, None, None) == _lib.EINVAL
    lib.spconv_rulebook_destroy(None)


def test_new_entry_points_reject_bad_arguments_on_the_host():
    """Pooling, DC and gradient entry points: NULL books and bad flags fail
    before any device work."""
    lib = _lib.load()
    E = _lib.EINVAL
    assert lib.spconv_pool_forward(None, 0, 0, None, None, 4, None) == E
    assert lib.spconv_dc_forward(None, 0, None, None, None, 0, None, 1, 1, None) == E
    assert lib.spconv_forward_fused(None, 0, None, None, None, None, None, 0, 0, None, 1, 1,
                                    None) == E
    assert lib.spconv_backward_data(None, 0, 0, None, None, 0, None, 1, 1, None) == E
    nbytes = ctypes.c_size_t()
    assert lib.spconv_backward_weight_workspace(None, 0, 1, 1, ctypes.byref(nbytes)) == E
    assert lib.spconv_backward_weight(None, 0, 0, None, None, None, None, 1, 1, None, 0,
                                      None) == E
    assert lib.spconv_backward_weight_noalloc(None, 0, 0, None, None, None, None, 1, 1,
                                              None) == E
    # the transposed book exists for SC only; unknown flag bits are rejected
    size = np.asarray([1, 4, 4], np.int32)
    f = np.asarray([1, 3, 3], np.int32)
    s = np.asarray([1, 1, 1], np.int32)
    h = ctypes.c_void_p()
    for kind, flags in ((0, _lib.BUILD_TRANSPOSE), (1, 4), (0, 8)):
        st = lib.spconv_build_rulebook(kind, 3, ctypes.c_void_p(16), 1, size.ctypes.data,
                                       f.ctypes.data, s.ctypes.data, flags, None,
                                       ctypes.byref(h))
        assert st == E and h.value is None


def test_set_allocator_needs_both_functions():
    lib = _lib.load()
    alloc = _lib.ALLOC_FN(lambda n, s, c: 0)
    release = _lib.RELEASE_FN(lambda p, s, c: None)
    assert lib.spconv_set_allocator(alloc, _lib.RELEASE_FN(), None) == _lib.EINVAL
    assert lib.spconv_set_allocator(_lib.ALLOC_FN(), release, None) == _lib.EINVAL
    assert lib.spconv_set_allocator(_lib.ALLOC_FN(), _lib.RELEASE_FN(), None) == _lib.OK


def test_chained_build_and_bounds_reject_null():
    lib = _lib.load()
    h = ctypes.c_void_p()
    f = np.asarray([1, 3, 3], np.int32)
    s = np.asarray([1, 1, 1], np.int32)
    assert lib.spconv_build_rulebook_on(None, 0, f.ctypes.data, s.ctypes.data, 0, None,
                                        ctypes.byref(h)) == _lib.EINVAL
    assert h.value is None
    assert lib.spconv_rulebook_bounds(None, None, None) == _lib.EINVAL


def test_block_cache_entry_points_without_a_device():
    lib = _lib.load()
    n = ctypes.c_int64(-1)
    assert lib.spconv_release_cached_memory(ctypes.byref(n)) == _lib.OK
    assert n.value == 0
    assert lib.spconv_release_cached_memory(None) == _lib.OK
    assert lib.spconv_memory_stats(-1, None, None) in (_lib.EINVAL, _lib.EHIP)


def test_product_path_does_not_load_the_oracle():
    """The package never imports the oracle (which is test infrastructure)."""
    import subprocess
    import sys
    code = ("import sys; import paper_1706_01307_amd as spc; from paper_1706_01307_amd import "
            "_lib, inputs; _lib.load(); print('oracle' in sys.modules)")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=120)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "False"
    pkg = os.path.join(ROOT, "paper_1706_01307_amd")
    for dirpath, _, files in os.walk(pkg):
        for name in files:
            if name.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, name)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), name
                assert "oracle.h" not in text and "oracle.cpp" not in text, name


def test_missing_library_fails_loudly(tmp_path):
    """Without the built library every entry point raises: no fallback."""
    import subprocess
    import sys
    code = ("import paper_1706_01307_amd._lib as L; L.LIB_PATH = %r; L._lib = None\n"
            "import paper_1706_01307_amd as spc\n"
            "try:\n    spc.release_cached_memory()\nexcept ImportError as e:\n"
            "    print('raised', 'missing' in str(e))\n" % str(tmp_path / "libspconv.so"))
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                         timeout=120)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "raised True"
