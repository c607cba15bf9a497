"""C-ABI checks that need no GPU: the library loads, exports every function
include/neuroute.h declares, its struct layout matches the Python binding,
and host-side argument validation rejects bad calls before touching HIP."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2608_15438_amd import neuroute as NR

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "neuroute.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(NR.SO_PATH):
        from paper_2608_15438_amd import build_lib
        build_lib.build()
    return NR.lib()


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(nr_[a-z_]+)\s*\(", txt)))


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert set(names) == set(NR.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", NR.SO_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (nr_[a-z_]+)\b", out))
    assert set(names) <= exported
    for n in names:
        assert hasattr(L, n)


def test_struct_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r'''
#include <stddef.h>
#include <stdio.h>
#include "neuroute.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu\n", sizeof(nr_index_desc),
         offsetof(nr_index_desc, rows), offsetof(nr_index_desc, n_clusters),
         offsetof(nr_index_desc, head_bytes), sizeof(nr_params), offsetof(nr_params, refine_mode),
         offsetof(nr_params, shared_seed_rows), offsetof(nr_params, m_x), offsetof(nr_params, m_y));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    exp = [C.sizeof(NR.nr_index_desc), NR.nr_index_desc.rows.offset,
           NR.nr_index_desc.n_clusters.offset, NR.nr_index_desc.head_bytes.offset,
           C.sizeof(NR.nr_params), NR.nr_params.refine_mode.offset,
           NR.nr_params.shared_seed_rows.offset, NR.nr_params.m_x.offset, NR.nr_params.m_y.offset]
    assert got == exp


def test_status_strings(L):
    assert L.nr_status_string(0) == b"ok"
    assert L.nr_status_string(5) == b"corrupt index"


def _desc(**kw):
    d = NR.nr_index_desc()
    d.n, d.d, d.dtype, d.b, d.n_layers = 100, 32, NR.NR_F32, 8, 1
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("field,value,status", [
    ("n", 0, NR.NR_EINVAL),
    ("d", 0, NR.NR_EINVAL),
    ("dtype", 7, NR.NR_EINVAL),
    ("b", 31, NR.NR_EUNSUPPORTED),
    ("n_layers", 0, NR.NR_EUNSUPPORTED),
    ("d", 3, NR.NR_EUNSUPPORTED),        # 12-byte rows: not a multiple of 16
])
def test_upload_rejects_bad_description(L, field, value, status):
    d = _desc(**{field: value})
    h = C.c_void_p()
    assert L.nr_index_upload(C.byref(d), C.byref(h), None) == status
    assert not h.value
    assert L.nr_last_error()


def test_null_arguments(L):
    h = C.c_void_p()
    assert L.nr_index_upload(None, C.byref(h), None) == NR.NR_EINVAL
    d = _desc()
    assert L.nr_index_upload(C.byref(d), C.byref(h), None) == NR.NR_EINVAL   # no widths/weights
    p = NR.Params().c()
    assert L.nr_search(None, None, 1, 10, 4, C.byref(p), None, None, None) == NR.NR_EINVAL
    assert L.nr_route_capacity(None, 4, C.byref(p)) == 0
    assert L.nr_index_free(None) == NR.NR_OK


def test_counter_enums_match_header():
    txt = open(HEADER).read()
    assert int(re.search(r"#define NR_STAGES (\d+)", txt).group(1)) == NR.NR_STAGES == len(NR.STAGES)
    work = dict((m.group(1).lower(), int(m.group(2)))
                for m in re.finditer(r"NR_WORK_([A-Z_]+) = (\d+)", txt))
    assert int(re.search(r"\bNR_WORK = (\d+)", txt).group(1)) == len(NR.WORK)
    assert [work[n] for n in NR.WORK] == list(range(len(NR.WORK)))
