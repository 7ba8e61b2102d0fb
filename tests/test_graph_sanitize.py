"""The graph index builder (csrc/graph.cpp with the status helpers of
csrc/status.cpp) compiled for the host alone with g++ under
AddressSanitizer and UndefinedBehaviorSanitizer, driven by
tests/native/graph_host_check.cpp: bit-exact indexes against the oracle's
construction, the documented status codes for invalid input, and
RGNN_ENOMEM without leaks when any single host allocation of a graph
creation fails (the leak checker runs at the harness's exit)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2301_06284_amd", "csrc")
HARNESS = os.path.join(ROOT, "tests", "native", "graph_host_check.cpp")
OUT = os.path.join(ROOT, "_build", "sanitize")
EXE = os.path.join(OUT, "graph_host_check")
KINDS = ["dst_rowptr", "in_src", "in_rel", "in_eid", "seg_ptr", "seg_rel", "dst_segptr", "uniq_src",
         "uniq_rel_ptr", "edge2uniq", "ntype_perm", "ntype_ptr", "out_ptr", "out_pos"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


@pytest.fixture(scope="module")
def exe():
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    os.makedirs(OUT, exist_ok=True)
    srcs = [os.path.join(CSRC, "graph.cpp"), os.path.join(CSRC, "status.cpp"), HARNESS]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"),
           "-I" + CSRC, "-o", EXE] + srcs
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return EXE


def write_graph(path, g, csr=False, flags=0):
    N, E = g["N"], g["E"]
    with open(path, "wb") as f:
        np.array([N, E], np.int64).tofile(f)
        np.array([g["T"], g["R"], int(csr), flags], np.int32).tofile(f)
        if csr:
            order = np.argsort(g["dst"], kind="stable")
            rowptr = np.zeros(N + 1, np.int64)
            np.cumsum(np.bincount(g["dst"], minlength=N), out=rowptr[1:])
            rowptr.tofile(f)
            np.asarray(g["src"], np.int32)[order].tofile(f)
            np.asarray(g["rel"], np.int32)[order].tofile(f)
        else:
            for k in ("src", "dst", "rel"):
                np.asarray(g[k], np.int32).tofile(f)
        np.asarray(g["ntype"], np.int32).tofile(f)


def read_index(path):
    raw = open(path, "rb").read()
    head = np.frombuffer(raw[:32], np.int64)
    out, off = {}, 32
    for k in KINDS:
        n = int(np.frombuffer(raw[off:off + 8], np.int64)[0])
        off += 8
        out[k] = np.frombuffer(raw[off:off + 4 * n], np.int32)
        off += 4 * n
    return head, out


def run(exe, *args):
    r = subprocess.run([exe, *args], capture_output=True, text=True, env=ENV, timeout=300)
    return r.returncode, r.stdout + r.stderr


@pytest.mark.parametrize("kind", ["random", "hub", "srchub", "dups", "isolated", "empty", "complete"])
@pytest.mark.parametrize("csr", [False, True])
def test_index_under_sanitizers(exe, tmp_path, kind, csr):
    g = workloads.tiny_graph(11, N=90, E=700, R=5, T=3, kind=kind)
    inp, outp = str(tmp_path / "g.bin"), str(tmp_path / "ix.bin")
    write_graph(inp, g, csr=csr)
    rc, log = run(exe, "index", inp, outp)
    assert rc == 0, log
    head, got = read_index(outp)
    if csr:   # CSR edge ids are the CSR positions
        order = np.argsort(g["dst"], kind="stable")
        g = dict(g, src=g["src"][order], dst=g["dst"][order], rel=g["rel"][order])
    ix = oracle.graph_index(g)
    for k in KINDS:
        np.testing.assert_array_equal(got[k], ix[k], err_msg=k)
    assert head[0] == ix["U_src"] and head[1] == ix["U_dst"]


def test_index_workload1_under_sanitizers(exe, tmp_path):
    g = workloads.make_graph(1)
    inp, outp = str(tmp_path / "g.bin"), str(tmp_path / "ix.bin")
    write_graph(inp, g)
    rc, log = run(exe, "index", inp, outp)
    assert rc == 0, log
    _, got = read_index(outp)
    ix = oracle.graph_index(g)
    for k in KINDS:
        np.testing.assert_array_equal(got[k], ix[k], err_msg=k)


def test_error_codes_under_sanitizers(exe):
    rc, log = run(exe, "errors")
    assert rc == 0 and "FAIL" not in log, log
    assert log.count("ok ") >= 25, log


@pytest.mark.parametrize("kind,csr", [("hub", False), ("dups", True)])
def test_allocation_failure_enomem_no_leak(exe, tmp_path, kind, csr):
    """Every host allocation of a graph creation is failed in turn: each
    returns RGNN_ENOMEM with no graph, and the leak checker finds nothing."""
    g = workloads.tiny_graph(12, N=60, E=400, R=4, T=2, kind=kind)
    inp = str(tmp_path / "g.bin")
    write_graph(inp, g, csr=csr)
    rc, log = run(exe, "nomem", inp)
    assert rc == 0, log
    assert "each failure returned RGNN_ENOMEM" in log, log
    assert "LeakSanitizer" not in log and "runtime error" not in log, log
