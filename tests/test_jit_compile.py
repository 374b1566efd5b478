"""The per-graph specialised kernels compile (hipRTC cross-compiles for
gfx950 without a GPU): the sources the library generates for the workloads
and for a comparison pair, with the library's own options and headers, and
no private (scratch) memory in the resulting kernels."""

import ctypes
import os
import re
import subprocess
import tempfile

import pytest

import hostemu
from paper_2609_19611_amd import workloads as W

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2609_19611_amd", "csrc")
HIPRTC = "/opt/rocm/lib/libhiprtc.so"
READELF = "/opt/rocm/llvm/bin/llvm-readelf"

pytestmark = pytest.mark.skipif(not os.path.exists(HIPRTC), reason="hipRTC not installed")


def _rtc():
    L = ctypes.CDLL(HIPRTC)
    P = ctypes.c_void_p
    L.hiprtcCreateProgram.argtypes = [ctypes.POINTER(P), ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_char_p)]
    L.hiprtcCompileProgram.argtypes = [P, ctypes.c_int, ctypes.POINTER(ctypes.c_char_p)]
    L.hiprtcGetCodeSize.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    L.hiprtcGetCode.argtypes = [P, ctypes.c_char_p]
    L.hiprtcGetProgramLogSize.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    L.hiprtcGetProgramLog.argtypes = [P, ctypes.c_char_p]
    L.hiprtcDestroyProgram.argtypes = [ctypes.POINTER(P)]
    return L


def _compile(src):
    L = _rtc()
    names = ["program.h", "core.h", "kernels_dev.h", "dag_program.h", "dag_core.h", "dag_dev.h"]
    texts = [open(os.path.join(CSRC, n), "rb").read() for n in names]
    hdr = (ctypes.c_char_p * len(names))(*texts)
    nm = (ctypes.c_char_p * len(names))(*[n.encode() for n in names])
    prog = ctypes.c_void_p()
    assert L.hiprtcCreateProgram(ctypes.byref(prog), src.encode(), b"dg_plan.hip", len(names), hdr, nm) == 0
    buf = ctypes.create_string_buffer(4096)
    hostemu.lib().dgh_jit_options(buf, 4096)
    opts = buf.value.decode().split()
    arr = (ctypes.c_char_p * len(opts))(*[o.encode() for o in opts])
    rc = L.hiprtcCompileProgram(prog, len(opts), arr)
    n = ctypes.c_size_t()
    L.hiprtcGetProgramLogSize(prog, ctypes.byref(n))
    log = ctypes.create_string_buffer(max(1, n.value))
    L.hiprtcGetProgramLog(prog, log)
    assert rc == 0, log.value.decode()[-2000:]
    L.hiprtcGetCodeSize(prog, ctypes.byref(n))
    code = ctypes.create_string_buffer(n.value)
    L.hiprtcGetCode(prog, code)
    L.hiprtcDestroyProgram(ctypes.byref(prog))
    return code.raw


def _kernel_notes(code):
    """(name, private segment bytes) of every kernel in a code object."""
    with tempfile.NamedTemporaryFile(suffix=".co") as f:
        f.write(code)
        f.flush()
        out = subprocess.run([READELF, "--notes", f.name], capture_output=True, text=True).stdout
    names = re.findall(r"^\s+\.name:\s+(\S+)", out, re.M)
    priv = [int(x) for x in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", out)]
    return list(zip(names, priv))


def _source(fn, *args):
    buf = ctypes.create_string_buffer(1 << 24)
    n = fn(*args, buf, 1 << 24)
    assert n > 0, hostemu.lib().dgh_error().decode()
    return buf.value.decode()


@pytest.mark.parametrize("name,block", [("c1", 64), ("c3", 256), ("c4", 256)])
def test_enumeration_kernels_compile(name, block):
    t = W.CONFIGS[name]["text"]().encode()
    src = _source(hostemu.lib().dgh_jit_source, t, len(t), block)
    code = _compile(src)
    notes = _kernel_notes(code)
    assert {n for n, _ in notes} >= {"dg_sizes", "dg_fill", "dg_enumerate"}
    if os.path.exists(READELF):
        assert all(p == 0 for _, p in notes), notes


@pytest.mark.parametrize("name,block", [("c1", 64), ("c4", 256)])
def test_wide_enumeration_kernel_compiles(name, block):
    t = W.CONFIGS[name]["text"]().encode()
    src = _source(hostemu.lib().dgh_jit_wide_source, t, len(t), block)
    notes = _kernel_notes(_compile(src))
    assert [n for n, _ in notes] == ["dg_enumerate_wide"]
    assert all(p == 0 for _, p in notes), notes


def test_comparison_kernel_compiles():
    a = W.c5_reference_text(n=2, c=4, hw=6, co=3).encode()
    b = W.c5_variant_text(fault=W.c5_faults()[0], n=2, c=4, hw=6, co=3).encode()
    src = _source(hostemu.lib().dgh_jit_compare_source, a, len(a), b, len(b), 64)
    notes = _kernel_notes(_compile(src))
    assert [n for n, _ in notes] == ["dg_compare"]
    assert all(p == 0 for _, p in notes), notes


@pytest.mark.parametrize("name,block", [("c3", 256), ("c5", 64)])
def test_dag_kernels_compile(name, block):
    """The specialised DAG kernels of a workload compile, carry only the
    ways of taking a group that its program uses, and use no scratch."""
    t = W.CONFIGS[name]["text"]().encode()
    src = _source(hostemu.lib().dgh_jit_dag_source, t, len(t), block)
    assert "#define DG_DAG_BOX 0" in src and "#define DG_DAG_NOPS" in src
    notes = _kernel_notes(_compile(src))
    assert sorted(n for n, _ in notes) == ["dg_dag_fill", "dg_dag_onepass", "dg_dag_sizes"]
    assert all(p == 0 for _, p in notes), notes


HELPER = os.path.join(os.path.dirname(CSRC), "lib", "dirigo_jitc")


@pytest.mark.skipif(not os.path.exists(HELPER), reason="compile helper not built")
def test_compile_helper_builds_the_specialised_kernels():
    """The compile helper the library spawns: a status byte 0 and the code
    object of a workload's enumeration source on stdout (a kernel named
    dg_enumerate, no scratch memory); status 1 and the compiler's log for
    a source that does not compile; and it needs no HIP runtime."""
    L = hostemu.lib()
    t = W.CONFIGS["c4"]["text"]().encode()
    buf = ctypes.create_string_buffer(1 << 24)
    k = L.dgh_jit_source(t, len(t), 256, buf, len(buf))
    assert k > 0
    r = subprocess.run([HELPER], input=buf.value, capture_output=True, timeout=300)
    assert r.returncode == 0 and r.stdout[:1] == b"\x00"
    with tempfile.NamedTemporaryFile(suffix=".co") as f:
        f.write(r.stdout[1:])
        f.flush()
        notes = subprocess.run([READELF, "--notes", f.name], capture_output=True, text=True).stdout
    assert "dg_enumerate" in notes
    assert all(int(v) == 0 for v in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", notes))
    bad = subprocess.run([HELPER], input=b"this is not a kernel", capture_output=True, timeout=300)
    assert bad.returncode == 1 and bad.stdout[:1] == b"\x01" and len(bad.stdout) > 1
    libs = subprocess.run(["ldd", HELPER], capture_output=True, text=True).stdout
    assert "libhiprtc" in libs and "libamdhip64" not in libs


def test_dag_specialisation_range():
    """By default the specialised DAG kernels run calls of at least 2^26
    edges (static bound): the conv2d pair check's 1,048,576 DAGs, the GEMM
    + GroupNorm workload's 65,536 and the conv-transpose + softmax
    workload's 8,192 are in that range; the 4,096 small DAGs of the conv2d
    + pool workload are not."""
    def bound(name):
        return hostemu.dag_bounds(W.CONFIGS[name]["text"](), 64)[1]
    n = {name: len(W.config_locations(name)) for name in ("c2", "c4", "c5")}
    n["c3"] = 8192
    for name in ("c3", "c4", "c5"):
        assert n[name] * bound(name) >= 1 << 26, name
    assert n["c2"] * bound("c2") < 1 << 26
