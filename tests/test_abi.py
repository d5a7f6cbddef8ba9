"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/dflow.h, and host-side validation reports errors before
any device work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dflow.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(?:int|size_t|const char\*)\s+(\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_06498_amd.runtime import library_path, load_library
    if not os.path.exists(library_path()):
        pytest.skip("libdflow.so not built")
    return load_library()


def test_header_declares_round_calls():
    names = _declared()
    for n in ("dflow_verify_block", "dflow_accept_and_carry", "dflow_draft_block", "kv_commit"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for n in _declared():
        assert hasattr(lib, n), n


def test_binding_covers_header():
    from paper_2609_06498_amd.runtime import EXPORTS
    assert sorted(EXPORTS) == _declared()


def test_validation_errors_without_device(lib):
    from paper_2609_06498_amd.runtime import Dims
    d = Dims()
    d.dtype = 7
    assert lib.dflow_workspace_bytes(ctypes.byref(d)) == 0
    assert "dtype" in lib.dflow_last_error().decode()
    d.dtype = 1
    d.d, d.n_layers, d.n_heads, d.n_kv_heads, d.head_dim = 512, 2, 8, 2, 96
    assert lib.dflow_workspace_bytes(ctypes.byref(d)) == 0
    assert "head_dim" in lib.dflow_last_error().decode()
    assert lib.dflow_pack_linear(None, 1, None, 16, 32, 0, None, None) == -1
    assert lib.dflow_pack_linear(None, 1, ctypes.c_void_p(16), 16, 48, 0, None, ctypes.c_void_p(16)) == -2
    assert lib.dflow_create(None, None, None, None, 0, None, None, None) == -1
    assert lib.dflow_move_slot(None, None, 0, 1) == -1
    assert lib.dflow_qkv_parts(None) == -1
    assert lib.dflow_attention_split(None, None, None) == -1
    assert lib.dflow_sample_draft(None, None, 1, None, None, None, None, None, None) == -1
    assert lib.dflow_accept_sampled(None, None, 1, None, None, None, None, None, None, None, None, None, None) == -1
    assert lib.dflow_trajectory_targets(None, None, 1, None, 8, 8, None, None) == -1
    assert lib.dflow_draft_loss(None, None, 1, None, None, 8, 8, None, 7.0, None) == -1
    assert lib.dflow_packed_bytes(1, 32, 64) == 32 * 64 * 2
    assert lib.dflow_packed_bytes(0, 32, 64) == 32 * 64 * 4


def _dims_8b():
    from paper_2609_06498_amd.runtime import Dims
    d = Dims()
    d.dtype, d.d, d.n_layers, d.n_heads, d.n_kv_heads, d.head_dim = 1, 4096, 36, 32, 8, 128
    d.ffn, d.vocab, d.n_draft_layers, d.n_capture = 12288, 151936, 5, 5
    for i, l in enumerate((0, 8, 17, 26, 35)):
        d.capture_layers[i] = l
    d.relay_hidden, d.block, d.max_batch, d.max_rows = 4096, 16, 1, 128
    d.max_pages, d.num_pages, d.carry_window = 100, 100, 0
    d.rope_theta, d.rms_eps, d.ln_eps = 1e6, 1e-6, 1e-5
    return d


def test_workspace_bytes_for_8b_shape(lib):
    d = _dims_8b()
    n = lib.dflow_workspace_bytes(ctypes.byref(d))
    assert 0 < n < 1 << 30, (n, lib.dflow_last_error())


def test_create_checks_the_callers_workspace_and_status(lib):
    """dflow_create takes the workspace and the status word from the caller and
    rejects a missing, misaligned or short workspace before any device call."""
    from paper_2609_06498_amd.runtime import Cache, Weights
    d = _dims_8b()
    need = lib.dflow_workspace_bytes(ctypes.byref(d))
    W, C, ctx = Weights(), Cache(), ctypes.c_void_p()
    fake = ctypes.c_void_p(1 << 20)        # never dereferenced: every check below fails first
    args = lambda ws, nb, st: (ctypes.byref(d), ctypes.byref(W), ctypes.byref(C), ws, nb, st, None, ctypes.byref(ctx))
    assert lib.dflow_create(*args(None, need, fake)) == -1
    assert lib.dflow_create(*args(fake, need, None)) == -1
    assert lib.dflow_create(*args(ctypes.c_void_p((1 << 20) + 16), need, fake)) == -1
    assert "aligned" in lib.dflow_last_error().decode()
    assert lib.dflow_create(*args(fake, need - 256, fake)) == -4
    assert "workspace" in lib.dflow_last_error().decode()
    assert ctx.value is None


def test_library_allocates_no_device_memory():
    """Every device buffer is the caller's: no allocation or free call in the
    library sources."""
    csrc = os.path.join(ROOT, "paper_2609_06498_amd", "csrc")
    bad = re.compile(r"\bhip(Malloc\w*|Free\w*|ExtMalloc\w*|HostMalloc|MallocManaged)\s*\(")
    for f in sorted(os.listdir(csrc)):
        src = open(os.path.join(csrc, f)).read()
        assert not bad.search(src), f"{f}: {bad.search(src).group(0)}"
