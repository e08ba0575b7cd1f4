"""C-ABI checks that need no GPU: the library loads, exports every function
include/fsched.h declares, its structs have the declared layout, and argument
errors are reported before any device work."""
import ctypes
import os
import re

import pytest

import paper_2608_02244_amd as fs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fsched.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fsched_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert set(names) >= {"fsched_simulate", "fsched_cost_decompose", "fsched_bruteforce_opt"}
    L = fs.lib()
    for name in names:
        assert hasattr(L, name), f"{name} declared in fsched.h but not exported"
    assert set(fs.EXPORTS) == set(names)


def test_abi_version_and_strerror():
    L = fs.lib()
    assert L.fsched_abi_version() == 1
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert L.fsched_strerror(code)
    assert L.fsched_strerror(12345) == b"unknown error code"


def test_struct_layout():
    assert ctypes.sizeof(fs.Params) == 40
    offs = {f: getattr(fs.Params, f).offset for f, _ in fs.Params._fields_}
    assert offs == {"B": 0, "alpha": 4, "M_kv": 8, "policy": 16, "flags": 20, "cost_c": 24,
                    "cost_tau": 32}
    assert fs.METRICS_DTYPE.itemsize == fs.METRICS_BYTES == 104
    assert fs.METRICS_DTYPE.fields["max_active"][1] == 100


DUMMY = ctypes.c_void_p(0x1000)  # never dereferenced: every case fails before device work


def call_sim(p, n_inst=1, n_jobs=4, ptr=DUMMY):
    return fs.lib().fsched_simulate(ctypes.byref(p) if p is not None else None, n_inst, n_jobs,
                                    ptr, ptr, ptr, ptr, None, None, None)


@pytest.mark.parametrize("field,value", [("B", -1), ("alpha", -1), ("M_kv", -5),
                                         ("policy", 7), ("policy", -1), ("flags", 2),
                                         ("flags", 1 << 9), ("cost_c", -1), ("cost_tau", -2)])
def test_bad_params_rejected(field, value):
    p = fs.make_params("isjl", 2, 1, device=True)
    setattr(p, field, value)
    assert call_sim(p) == fs.EINVAL


def test_bad_sizes_and_pointers():
    p = fs.make_params("fcfs", 2, 1, device=True)
    assert call_sim(None) == fs.EINVAL
    assert call_sim(p, n_jobs=0) == fs.EINVAL
    assert call_sim(p, n_inst=-1) == fs.EINVAL
    assert call_sim(p, ptr=None) == fs.EINVAL
    assert call_sim(p, n_inst=0) == fs.OK  # nothing to do


def test_kernel_limits_rejected_before_launch():
    p = fs.make_params("isjl", 0, 4, device=True)
    assert call_sim(p, n_jobs=4097) == fs.ETOOLARGE
    p = fs.make_params("fcfs", 0, 4, device=True)
    assert call_sim(p, n_jobs=2000) == fs.ETOOLARGE  # B unlimited -> 2000 workers > 1024
    p = fs.make_params("fcfs", 1025, 4, device=True)
    assert call_sim(p, n_jobs=2000) == fs.ETOOLARGE


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(fs, "LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(fs, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        fs.lib()


def call_noalloc(p, n_inst=1, n_jobs=4, ptr=DUMMY):
    return fs.lib().fsched_simulate_noalloc(ctypes.byref(p) if p is not None else None, n_inst,
                                            n_jobs, ptr, ptr, ptr, ptr, None, None, None)


def test_noalloc_argument_errors_before_device_work():
    """The no-allocation call refuses host mode (it would have to stage), checks
    arguments like fsched_simulate, and refuses a shape whose scratch exceeds its
    fixed buffer with FSCHED_ESCRATCH, all before touching the device."""
    assert call_noalloc(fs.make_params("isjl", 2, 1, device=False)) == fs.EINVAL
    assert call_noalloc(None) == fs.EINVAL
    p = fs.make_params("isjl", 512, 128, device=True)
    assert call_noalloc(p, n_jobs=0) == fs.EINVAL
    assert call_noalloc(p, n_inst=0) == fs.OK
    assert call_noalloc(p, ptr=None) == fs.EINVAL
    assert call_noalloc(p, n_jobs=4097) == fs.ETOOLARGE
    # 65,536 x 2,000 jobs: a 256 MiB rank table against the 64 MiB buffer
    assert call_noalloc(p, n_inst=65536, n_jobs=2000) == fs.ESCRATCH
    # 8 slots per lane at a finite alpha: the plan links in HBM add 8 KiB to the
    # 4 KiB rank row, so 5,462 instances of 2,000 jobs no longer fit
    assert call_noalloc(p, n_inst=5462, n_jobs=2000) == fs.ESCRATCH
    assert call_noalloc(fs.make_params("fcfs", 512, 128, device=True), n_inst=65536,
                        n_jobs=2000, ptr=None) == fs.EINVAL
