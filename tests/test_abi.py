"""The C ABI: the library loads, exports every symbol the header declares (and
nothing else), and its host-side validation answers without a GPU."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scanweaver.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sw_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2606_00601_amd as pkg
    return pkg.lib()


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("sw_affine_scan", "sw_affine_scan_i32", "sw_selective_scan_fwd",
              "sw_selective_scan_fwd_bf16", "sw_set_stream", "sw_status_string",
              "sw_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in _declared():
        assert hasattr(lib, n), n


def test_library_exports_nothing_else():
    from paper_2606_00601_amd._lib import LIB_PATH
    out = subprocess.run(["nm", "-D", "--defined-only", LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    syms = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert syms == set(_declared())


def test_call_extension_mirrors_the_header():
    import paper_2606_00601_amd as pkg
    f = pkg.fast()
    for n in _declared():
        assert callable(getattr(f, n)), n
    from paper_2606_00601_amd import build
    assert os.path.exists(build.swcall_path())


def test_call_extension_answers_like_ctypes(lib):
    import paper_2606_00601_amd as pkg
    f = pkg.fast()
    cases = [("sw_affine_scan", (None, None, None, None, -1, 2, 3)),
             ("sw_affine_scan_noalloc", (None, None, None, None, 1, 2, -3)),
             ("sw_selective_scan_fwd", (*([None] * 8), 1, 1, 65, 4)),
             ("sw_selective_scan_fwd_ex", (*([None] * 11), 1, 1, 16, 4, 7, 0, 0)),
             ("sw_selective_scan_bwd", (*([None] * 22), 1, 1, 16, 4, 0, 0, 8)),
             ("sw_affine_scan_schedule", (None, None, None, None, 1, 1, 1, 9))]
    for name, args in cases:
        want = getattr(lib, name)(*args)
        want_msg = lib.sw_last_error()
        got = getattr(f, name)(*args)
        assert got == want and got != 0, name
        assert f.sw_last_error() == want_msg, name
    assert f.sw_version() == lib.sw_version()
    assert f.sw_status_string(2) == lib.sw_status_string(2)
    # one library underneath: the stream set through one view is the other's
    f.sw_set_stream(0x1234)
    assert lib.sw_get_stream() == 0x1234 and f.sw_get_stream() == 0x1234
    lib.sw_set_stream(None)
    assert f.sw_get_stream() is None
    with pytest.raises(TypeError):
        f.sw_affine_scan(None, None, None, None, 1, 1)  # one argument short
    with pytest.raises(TypeError):
        f.sw_affine_scan(1.5, None, None, None, 1, 1, 1)  # not an address
    with pytest.raises(OverflowError):
        f.sw_affine_scan_schedule(None, None, None, None, 1, 1, 1, 2 ** 40)


def test_binding_signatures_match_header():
    from paper_2606_00601_amd._lib import SIGNATURES
    assert set(SIGNATURES) == set(_declared())


def test_validation_without_gpu(lib):
    # negative sizes: invalid argument, before any HIP call
    assert lib.sw_affine_scan(None, None, None, None, -1, 2, 3) == 1
    assert "negative" in lib.sw_last_error().decode()
    assert lib.sw_affine_scan_i32(None, None, None, None, 1, -2, 3) == 1
    assert lib.sw_affine_scan_noalloc(None, None, None, None, 1, 2, -3) == 1
    assert lib.sw_selective_scan_fwd(*([None] * 8), 1, 1, -1, 4) == 1
    # N outside [1, 64]: unsupported
    assert lib.sw_selective_scan_fwd(*([None] * 8), 1, 1, 65, 4) == 2
    assert lib.sw_selective_scan_fwd_bf16(*([None] * 8), 1, 1, 0, 4) == 2
    # empty outputs: nothing to do, pointers not inspected
    assert lib.sw_affine_scan(None, None, None, None, 0, 5, 7) == 0
    assert lib.sw_affine_scan(None, None, None, None, 3, 5, 0) == 0
    assert lib.sw_selective_scan_fwd(*([None] * 8), 2, 0, 16, 9) == 0
    # overflowing sizes are refused
    big = 1 << 40
    assert lib.sw_affine_scan(None, None, None, None, big, big, 4) == 2
    # schedules: unknown ones are refused; the Blelloch one validates like the default
    assert lib.sw_affine_scan_schedule(None, None, None, None, 1, 1, 4, 7) == 1
    assert "schedule" in lib.sw_last_error().decode()
    assert lib.sw_affine_scan_schedule(None, None, None, None, -1, 1, 4, 1) == 1
    assert lib.sw_affine_scan_schedule_i32(None, None, None, None, 0, 1, 4, 1) == 0
    # the projection form: negative sizes, then empty shapes are a no-op
    assert lib.sw_affine_scan_proj(*([None] * 7), -1, 1, 1) == 1
    assert lib.sw_affine_scan_proj_i32(*([None] * 7), 1, 1, -1) == 1
    assert lib.sw_affine_scan_proj(*([None] * 7), 0, 4, 9) == 0
    assert lib.sw_affine_scan_proj_i32(*([None] * 7), big, big, 4) == 2
    # the extended fused entry point: unknown dtypes and flags are refused
    # before anything else; otherwise it validates like the plain one
    ex = lib.sw_selective_scan_fwd_ex
    assert ex(*([None] * 11), 1, 1, 16, 4, 2, 0, 0) == 1
    assert "dtype" in lib.sw_last_error().decode()
    assert ex(*([None] * 11), 1, 1, 16, 4, 0, 5, 0) == 1
    assert ex(*([None] * 11), 1, 1, 16, 4, 0, 0, 2) == 1
    assert "flags" in lib.sw_last_error().decode()
    assert ex(*([None] * 11), 1, 1, 65, 4, 1, 1, 1) == 2
    assert ex(*([None] * 11), 2, 0, 16, 9, 1, 1, 1) == 0


def test_status_strings(lib):
    assert lib.sw_status_string(0) == b"SW_OK"
    assert lib.sw_status_string(1) == b"SW_ERR_INVALID_ARG"
    assert lib.sw_status_string(2) == b"SW_ERR_UNSUPPORTED"
    assert lib.sw_status_string(3) == b"SW_ERR_HIP"
    assert lib.sw_status_string(4) == b"SW_ERR_ALLOC"
    assert lib.sw_status_string(99) == b"SW_ERR_UNKNOWN"


def test_stream_is_per_thread(lib):
    import threading
    lib.sw_set_stream(ctypes.c_void_p(0x1234))
    seen = []
    t = threading.Thread(target=lambda: seen.append(lib.sw_get_stream()))
    t.start()
    t.join()
    assert lib.sw_get_stream() == 0x1234
    assert seen == [None]
    lib.sw_set_stream(None)


def test_binding_rejects_cpu_tensors():
    torch = pytest.importorskip("torch")
    import paper_2606_00601_amd as pkg
    a = torch.zeros((1, 2, 3))
    with pytest.raises(ValueError):
        pkg.affine_scan(a, a)


def test_bwd_s_pre_requires_z(lib):
    # a pre-gate output without a gate is an invalid argument, before any HIP call
    args = [None] * 22 + [1, 1, 16, 8, 0, 0, 0]
    args[12] = 0x1000  # s_pre
    assert lib.sw_selective_scan_bwd(*args) == 1
    assert "s_pre requires z" in lib.sw_last_error().decode()


def test_abi_version(lib):
    # 0.2.0: sw_selective_scan_fwd_train and sw_selective_scan_bwd take s_pre
    assert lib.sw_version() == 200
