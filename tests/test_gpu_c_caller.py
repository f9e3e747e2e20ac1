"""A C program that uses only the C ABI and the HIP runtime (no Python, no torch in its
process) fills tables on the device, plans (the planner's choice, then each strategy
forced), looks up a batch with empty bags and two out-of-range indices, plain and with
per-lookup weights, and writes everything to a file; the oracle checks each output.
The program also times back-to-back emb_lookup calls from native code."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import workloads as W
from gpu_helpers import TOL, log
from oracle import pool as OP

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INC = os.path.join(ROOT, "include")
PKG = os.path.join(ROOT, "paper_2507_01676_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")]


def _read(path):
    buf = open(path, "rb").read()
    pos = 0

    def take(dtype, n):
        nonlocal pos
        a = np.frombuffer(buf, dtype=dtype, count=n, offset=pos)
        pos += a.nbytes
        return a

    T, B, E, dtype, mode, n_plans, _, _ = take(np.int32, 8).tolist()
    nnz = int(take(np.int64, 1)[0])
    d = dict(T=T, B=B, E=E, dtype="f16" if dtype else "f32", mode=mode, rows=take(np.int64, T).tolist(),
             pooling=["mean" if p else "sum" for p in take(np.int32, T)], offsets=take(np.int64, T * B + 1),
             indices=take(np.int64, nnz), psw=take(np.float32, nnz), plans=[])
    for _ in range(n_plans):
        force, n_bad = take(np.int32, 2).tolist()
        d["plans"].append((force, n_bad, take(np.float32, B * T * E).reshape(B, T, E)))
    d["weighted"] = (int(take(np.int32, 1)[0]), take(np.float32, B * T * E).reshape(B, T, E))
    assert pos == len(buf)
    return d


@pytest.fixture(scope="module")
def exe(tmp_path_factory):
    path = tmp_path_factory.mktemp("c") / "lookup_from_c"
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", INC,
                        "-I", os.path.join(ROCM, "include"), os.path.join(ROOT, "tests", "c", "lookup_from_c.c"),
                        "-L", PKG, "-lembx", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                        f"-Wl,-rpath,{PKG}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", str(path)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return path


@pytest.mark.parametrize("dtype,mode", [(0, W.VAL_UNIFORM), (1, W.VAL_UNIFORM), (0, W.VAL_INTEGER)])
def test_c_caller_lookups_match_the_oracle(exe, tmp_path, dtype, mode):
    log(f"C caller: dtype {dtype}, value mode {mode}")
    out = tmp_path / "out.bin"
    r = subprocess.run([str(exe), str(out), str(dtype), str(mode)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    log("  " + r.stdout.strip())
    d = _read(out)
    us = float(r.stdout.split()[1])
    assert 0 < us < 1000
    host = [W.materialize_table(t, m, d["E"], d["dtype"], seed=11 + t, lo=-1.0, hi=1.0, mode=mode)
            for t, m in enumerate(d["rows"])]
    empty = OP.empty_bag_mask(d["offsets"], d["T"], d["B"])
    assert empty.any()

    def check(got, psw, what):
        ref, mag, bad = OP.pool_reference(host, d["indices"], d["offsets"], d["B"], pooling=d["pooling"], psw=psw)
        assert bad == 2
        assert np.all(got[empty] == 0) and not np.any(np.signbit(got[empty])), f"{what}: empty bags must be +0.0"
        if mode == W.VAL_INTEGER and psw is None:   # weighted sums of integers round
            diff = np.argwhere(got != ref)
            assert diff.size == 0, f"{what}: {diff.shape[0]} elements differ, first {diff[:3].tolist()}"
        else:
            err = OP.pooled_error(got, ref, mag)
            assert err <= TOL[d["dtype"]], f"{what}: pooled error {err:.3e}"

    assert [p[0] for p in d["plans"]] == [-1, 0, 1, 2, 3, 4]
    for force, n_bad, got in d["plans"]:
        assert n_bad == 2, (force, n_bad)
        check(got, None, f"strategy {force}")
    n_bad, got = d["weighted"]
    assert n_bad == 2
    check(got, d["psw"], "weighted")
