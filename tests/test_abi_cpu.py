"""Host-side checks of the C-ABI library (CPU only): it loads, exports every
entry point the header declares, and rejects bad arguments before any HIP
call is made (so these run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("lmzipf.h", "lmzipf_test.h")]
LIB = os.path.join(ROOT, "paper_1810_10045_amd", "liblmzipf.so")


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lm_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_1810_10045_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_include_holds_only_these_headers():
    """Every header under include/ is one the symbol checks read."""
    found = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert found == sorted(os.path.basename(h) for h in HEADERS)


def test_test_hook_is_not_in_the_training_header():
    text = open(HEADERS[0]).read()
    assert "lm_test_" not in text


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("lm_unique", "lm_segsum", "lm_segsum_rows", "lm_segsum_sgd", "lm_segsum_adam",
              "lm_fill_values",
              "lm_sparse_apply",
              "lm_map_ids", "lm_unique_workspace_bytes", "lm_segsum_workspace_bytes",
              "lm_status_string"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), f"{n} declared in include/ but not exported"


def test_binding_names_match_the_header():
    src = open(os.path.join(ROOT, "paper_1810_10045_amd", "lmzipf.py")).read()
    for n in declared_functions():
        assert f'"{n}"' in src, n
    for n in ("unique", "segsum", "segsum_rows", "segsum_sgd", "segsum_adam", "map_ids",
              "fill_values",
              "sparse_apply", "fill_values_f16",
              "sparse_apply_f16", "sample_ids"):
        assert re.search(rf"^def {n}\(", src, re.M), n


def test_status_strings(lib):
    lib.lm_status_string.restype = ctypes.c_char_p
    for code in (0, 1, 3, 4, 5, 99):
        assert lib.lm_status_string(code)
    assert lib.lm_abi_version() == 106


def test_workspace_queries(lib):
    lib.lm_unique_workspace_bytes.restype = ctypes.c_size_t
    lib.lm_unique_workspace_bytes.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int64]
    lib.lm_segsum_workspace_bytes.restype = ctypes.c_size_t
    lib.lm_segsum_workspace_bytes.argtypes = [ctypes.c_int64, ctypes.c_int64]
    assert lib.lm_unique_workspace_bytes(65536, 0, 800000) >= 8192 + 65536 * 16
    assert lib.lm_unique_workspace_bytes(65536, 1, 800000) > lib.lm_unique_workspace_bytes(65536, 0, 800000)
    assert lib.lm_unique_workspace_bytes(-1, 0, 10) == 0
    assert lib.lm_unique_workspace_bytes(10, 7, 10) == 0
    assert lib.lm_unique_workspace_bytes(1 << 30, 0, 10) == 0
    assert lib.lm_segsum_workspace_bytes(65536, 1024) >= 8192
    assert lib.lm_segsum_workspace_bytes(-1, 4) == 0


def _v(x=0x1000):
    return ctypes.c_void_p(x)


def test_argument_errors_return_before_any_launch(lib):
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.lm_unique.argtypes = [P, I32, I64, I64, P, P, P, P, P, P, P, P, SZ, P]
    # unknown id dtype, negative K, V < 1, K too large, NULL workspace, misaligned workspace
    assert lib.lm_unique(_v(), 7, 10, 10, *([_v()] * 7), _v(), 1 << 20, None) == 5
    assert lib.lm_unique(_v(), 0, -1, 10, *([_v()] * 7), _v(), 1 << 20, None) == 1
    assert lib.lm_unique(_v(), 0, 10, 0, *([_v()] * 7), _v(), 1 << 20, None) == 1
    assert lib.lm_unique(_v(), 0, 1 << 30, 10, *([_v()] * 7), _v(), 1 << 40, None) == 5
    assert lib.lm_unique(_v(), 0, 10, 10, *([_v()] * 7), None, 1 << 20, None) == 1
    assert lib.lm_unique(_v(), 0, 10, 10, *([_v()] * 7), _v(0x1010), 1 << 20, None) == 1
    assert lib.lm_unique(_v(), 0, 10, 10, *([_v()] * 7), _v(), 16, None) == 3
    lib.lm_segsum.argtypes = [P, I32, I64, I64, I64, P, P, P, P, I64, P, I64, P, P, SZ, P]
    assert lib.lm_segsum(_v(), 2, 10, 4, 4, _v(), _v(), _v(), _v(), 10, _v(), 4, _v(), _v(), 1 << 20, None) == 5
    assert lib.lm_segsum(_v(), 0, 10, 4, 3, _v(), _v(), _v(), _v(), 10, _v(), 4, _v(), _v(), 1 << 20, None) == 1
    assert lib.lm_segsum(_v(), 0, 10, 4, 4, _v(), _v(), _v(), _v(), 10, _v(), 2, _v(), _v(), 1 << 20, None) == 1
    assert lib.lm_segsum(None, 0, 10, 4, 4, _v(), _v(), _v(), _v(), 10, _v(), 4, _v(), _v(), 1 << 20, None) == 1
    assert lib.lm_segsum(_v(), 0, 10, 4, 4, _v(), _v(), _v(), _v(), 10, _v(), 4, _v(), _v(), 8, None) == 3
    lib.lm_segsum_rows.argtypes = [P, I32, I64, I64, I64, P, P, P, P, P, I32, I64, P, I64, I64,
                                   P, P, SZ, P]

    def rows(gtype=0, idtype=0, rows_cap=10, row_ids=_v(), out_rows=100, ld_out=4, ws=_v(),
             ws_bytes=1 << 20):
        return lib.lm_segsum_rows(_v(), gtype, 10, 4, 4, _v(), _v(), _v(), _v(), row_ids, idtype,
                                  rows_cap, _v(), out_rows, ld_out, _v(), ws, ws_bytes, None)
    # unknown gradient or id dtype, an output of 2^31 rows, ld_out < D, NULL or
    # negative row ids, a misaligned or short workspace
    assert rows(gtype=2) == 5 and rows(idtype=7) == 5 and rows(out_rows=1 << 31) == 5
    assert rows(ld_out=3) == 1 and rows(row_ids=None) == 1 and rows(rows_cap=-1) == 1
    assert rows(ws=_v(0x1010)) == 1 and rows(ws_bytes=8) == 3
    lib.lm_segsum_sgd.argtypes = [P, I32, I64, I64, I64, P, P, P, P, P, I32, I64, P, I64, I64,
                                  ctypes.c_float, P, P, SZ, P]

    def sgd(gtype=0, idtype=0, rows_cap=10, row_ids=_v(), V=100, ld_table=4, table=_v(), ws=_v(),
            ws_bytes=1 << 20):
        return lib.lm_segsum_sgd(_v(), gtype, 10, 4, 4, _v(), _v(), _v(), _v(), row_ids, idtype,
                                 rows_cap, table, V, ld_table, 0.1, _v(), ws, ws_bytes, None)
    # the same argument errors, and a NULL table or a negative row count
    assert sgd(gtype=2) == 5 and sgd(idtype=7) == 5 and sgd(V=1 << 31) == 5
    assert sgd(ld_table=3) == 1 and sgd(row_ids=None) == 1 and sgd(rows_cap=-1) == 1
    assert sgd(table=None) == 1 and sgd(V=-1) == 1
    assert sgd(ws=_v(0x1010)) == 1 and sgd(ws_bytes=8) == 3
    F = ctypes.c_float
    lib.lm_segsum_adam.argtypes = [P, I32, I64, I64, I64, P, P, P, P, P, I32, I64, P, I64, I64,
                                   F, F, F, F, F, I64, P, P, P, P, SZ, P]

    def adam(gtype=0, V=100, ld_table=4, b1=0.9, b2=0.999, step=1, m=_v(), v=_v(), ws=_v(),
             ws_bytes=1 << 20):
        return lib.lm_segsum_adam(_v(), gtype, 10, 4, 4, _v(), _v(), _v(), _v(), _v(), 0, 10,
                                  _v(), V, ld_table, 1e-3, b1, b2, 1e-8, 0.0, step, m, v, _v(),
                                  ws, ws_bytes, None)
    # a bad dtype, step 0, a beta of 1 or below 0, NULL moments, ld < D, a
    # short workspace
    assert adam(gtype=2) == 5 and adam(step=0) == 1 and adam(b1=1.0) == 1 and adam(b2=-0.5) == 1
    assert adam(m=None) == 1 and adam(v=None) == 1 and adam(ld_table=3) == 1
    assert adam(V=1 << 31) == 5 and adam(ws_bytes=8) == 3
    lib.lm_fill_values.argtypes = [P, I64, P, P, I64, P, P, I32, I64, P, I64, I64, I32, P, P]
    assert lib.lm_fill_values(_v(), 4, _v(), _v(), 10, _v(), _v(), 0, 4, _v(), 10, 4, 9, _v(), None) == 5
    assert lib.lm_fill_values(_v(), 4, _v(), _v(), 10, None, None, 0, 4, _v(), 10, 4, 0, _v(), None) == 1
    assert lib.lm_fill_values(_v(), 2, _v(), _v(), 10, _v(), _v(), 0, 4, _v(), 10, 4, 0, _v(), None) == 1
    lib.lm_sparse_apply.argtypes = [P, I64, I64, I64, P, I32, P, I64, P, I64, I32] + \
        [ctypes.c_float] * 5 + [I64, P, P, P, P]
    assert lib.lm_sparse_apply(_v(), 10, 4, 4, _v(), 0, _v(), 5, _v(), 4, 3, 0.1, 0.9, 0.999, 1e-8, 0.0, 1,
                               None, None, _v(), None) == 5
    assert lib.lm_sparse_apply(_v(), 10, 4, 4, _v(), 0, _v(), 5, _v(), 4, 1, 0.1, 0.9, 0.999, 1e-8, 0.0, 0,
                               _v(), _v(), _v(), None) == 1
    assert lib.lm_sparse_apply(_v(), 10, 4, 4, _v(), 0, _v(), 5, _v(), 4, 1, 0.1, 0.9, 0.999, 1e-8, 0.0, 1,
                               None, None, _v(), None) == 1
    assert lib.lm_sparse_apply(_v(), 10, 4, 4, _v(), 0, _v(), 5, _v(), 4, 1, 0.1, 1.5, 0.999, 1e-8, 0.0, 1,
                               _v(), _v(), _v(), None) == 1
    F = ctypes.c_float
    lib.lm_fill_values_f16.argtypes = [P, I64, P, P, I64, P, P, I32, I64, P, I64, I64, I32, F, P, P]
    # SCATTER_ADD into a binary16 payload, a zero or non-finite scale, ld_dst < D
    assert lib.lm_fill_values_f16(_v(), 8, _v(), _v(), 10, _v(), _v(), 0, 8, _v(), 10, 8, 2, 256.0, _v(), None) == 5
    assert lib.lm_fill_values_f16(_v(), 8, _v(), _v(), 10, _v(), _v(), 0, 8, _v(), 10, 8, 0, 0.0, _v(), None) == 1
    assert lib.lm_fill_values_f16(_v(), 8, _v(), _v(), 10, _v(), _v(), 0, 8, _v(), 10, 8, 0, float("inf"), _v(), None) == 1
    assert lib.lm_fill_values_f16(_v(), 8, _v(), _v(), 10, _v(), _v(), 0, 8, _v(), 10, 4, 0, 256.0, _v(), None) == 1
    lib.lm_sparse_apply_f16.argtypes = [P, I64, I64, I64, P, I32, P, I64, P, I64, F, I32] + \
        [F] * 5 + [I64, P, P, P, P]
    assert lib.lm_sparse_apply_f16(_v(), 10, 8, 8, _v(), 0, _v(), 5, _v(), 8, float("nan"), 0, 0.1, 0.9,
                                   0.999, 1e-8, 0.0, 1, None, None, _v(), None) == 1
    assert lib.lm_sparse_apply_f16(_v(), 10, 8, 8, _v(), 0, _v(), 5, _v(), 8, 1 / 256, 4, 0.1, 0.9,
                                   0.999, 1e-8, 0.0, 1, None, None, _v(), None) == 5
    assert lib.lm_sparse_apply_f16(_v(), 10, 8, 8, _v(), 0, _v(), 5, _v(), 8, 1 / 256, 1, 0.1, 0.9,
                                   0.999, 1e-8, 0.0, 1, None, None, _v(), None) == 1
    lib.lm_sample_ids.argtypes = [P, I64, I64, P, I32, P]
    assert lib.lm_sample_ids(_v(), 10, 0, _v(), 0, None) == 1          # V < 1
    assert lib.lm_sample_ids(_v(), 10, 1 << 32, _v(), 0, None) == 1    # int32 ids, V > 2^31
    assert lib.lm_sample_ids(None, 10, 100, _v(), 0, None) == 1
    assert lib.lm_sample_ids(_v(), 10, 100, _v(), 4, None) == 5
    lib.lm_map_ids.argtypes = [P, P, I64, P, P, I64, I32, P, P, P]
    assert lib.lm_map_ids(_v(), _v(), 4, _v(), _v(), 4, 3, _v(), _v(), None) == 5
    assert lib.lm_map_ids(None, _v(), 4, _v(), _v(), 4, 0, _v(), _v(), None) == 1
    assert lib.lm_map_ids(_v(), _v(), 4, _v(), _v(), -1, 0, _v(), _v(), None) == 1
