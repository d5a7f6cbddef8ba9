"""The code-object reader that ties the committed HBM counter record to the
machine code of the kernel it was taken on (CPU only: reads the built
library's gfx950 code objects)."""
import json
import os

import pytest

from paper_2609_06498_amd import codeobj, library_path

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    p = library_path()
    if not os.path.exists(p):
        pytest.skip("libdflow.so not built")
    return p


def test_every_source_has_a_gfx950_code_object(lib):
    cos = list(codeobj.code_objects(lib))
    assert len(cos) == 4                       # gemm, attention, elementwise, sampling
    assert all(co[:4] == b"\x7fELF" for co in cos)


def test_kernels_have_code_and_descriptors(lib):
    for needle in ("gemm_kernel", "gemm_tile_kernel", "attn_kernel", "accept_kernel", "draw_kernel"):
        syms = codeobj.kernel_symbols(lib, needle)
        assert syms, needle
    for co in codeobj.code_objects(lib):
        s = codeobj.symbols(co)
        for name, code in s.items():
            if name + ".kd" in s:
                assert len(s[name + ".kd"]) == 64 and len(code) % 4 == 0 and len(code) > 0


def test_digest_is_deterministic_and_kernel_specific(lib):
    a, b = codeobj.kernel_symbols(lib, "gemm_kernel")[:2]
    assert codeobj.kernel_code_digest(lib, a) == codeobj.kernel_code_digest(lib, a)
    assert codeobj.kernel_code_digest(lib, a) != codeobj.kernel_code_digest(lib, b)
    with pytest.raises(KeyError):
        codeobj.kernel_code_digest(lib, "no_such_kernel")


def test_counter_record_names_a_kernel_of_the_library(lib):
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as fh:
        rec = json.load(fh)
    assert rec["symbol"] in codeobj.kernel_symbols(lib, "gemm_kernel")
    assert len(rec["code_sha256"]) == 64
    assert rec["fetch_bytes"] > 0 and rec["write_bytes"] > 0
