"""Host-side sanitizer runs (CPU only): the oracle and the library's host
scheduler built with AddressSanitizer and UndefinedBehaviorSanitizer.

- The oracle (oracle/psw_oracle.c) with a C driver (tests/native/
  oracle_driver.c) that runs whole training loops (orc_train, the resume
  form orc_train_from, orc_loss_and_grad) on small ResNet-20, LeNet-5 and
  VGG-16-with-dropout problems, fp32 and bf16 products, plain and Nesterov
  momentum; any out-of-bounds access, leak or undefined operation aborts the
  driver, and its results must equal the regular build's bit for bit.
- The scheduler's host code (paper_1912_12675_amd/csrc/api.hip, compiled
  with the sanitizers on its host pass only) with a C++ driver (tests/
  native/plan_driver.cpp) that creates the five configurations' networks,
  queries their sizes, writes their dry-run plans and exercises the argument
  checks; its plans must equal the regular library's.  No device is used.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

from paper_1912_12675_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")


@pytest.fixture(scope="module")
def oracle_driver(tmp_path_factory):
    d = tmp_path_factory.mktemp("asan_oracle")
    exe = str(d / "oracle_driver")
    subprocess.check_call(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           os.path.join(ROOT, "oracle", "psw_oracle.c"), os.path.join(NATIVE, "oracle_driver.c"),
                           "-o", exe, "-lm"])
    return exe


ORACLE_CASES = [
    ("resnet20_fp32", lambda: synth.resnet20_workload(batch=2), 4, False),
    ("resnet20_bf16", lambda: synth.resnet20_workload(batch=2, bf16=True), 4, False),
    ("lenet5_nesterov", lambda: synth.lenet5_workload(batch=4), 2, True),
    ("vgg16_dropout", lambda: synth.vgg16_workload(batch=1, n_pipelined=1, dropout=0.3), 2, False),
]


@pytest.mark.parametrize("name,factory,T,nesterov", ORACLE_CASES, ids=[c[0] for c in ORACLE_CASES])
def test_oracle_under_sanitizers(oracle, oracle_driver, tmp_path, name, factory, T, nesterov):
    wl = factory()
    N = wl.batch
    ops = np.ascontiguousarray(wl.ops, dtype=np.int32)
    se = np.ascontiguousarray(wl.stage_end, dtype=np.int32)
    p0 = synth.init_params(wl).astype(np.float64)
    xs, ys = synth.batches(wl, T, N)
    st = wl.staleness(T).astype(np.int32)
    lr = wl.lr_table(T)
    inp = tmp_path / "in.bin"
    with open(inp, "wb") as f:
        f.write(np.array([len(ops), N, *wl.in_shape, len(se), T, int(wl.bf16), int(nesterov)], np.int32).tobytes())
        f.write(ops.tobytes())
        f.write(se.tobytes())
        f.write(np.array([p0.size], np.int64).tobytes())
        f.write(p0.tobytes())
        f.write(np.ascontiguousarray(xs, np.float32).tobytes())
        f.write(np.ascontiguousarray(ys, np.int32).tobytes())
        f.write(st.tobytes())
        f.write(np.ascontiguousarray(lr, np.float64).tobytes())
    out = tmp_path / "out.bin"
    r = subprocess.run([oracle_driver, str(inp), str(out)], env=SAN_ENV, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, f"{name}: driver exit {r.returncode}\n{r.stderr[-3000:]}"
    got = np.fromfile(out, dtype=np.float64)
    n = p0.size
    params, losses = got[:n], got[n:n + T]
    params2, losses2 = got[n + T:2 * n + T], got[2 * n + T:2 * n + 2 * T]
    loss0, g0 = got[2 * n + 2 * T], got[2 * n + 2 * T + 1:]
    ref = oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, st, lr, 0.9, 1e-4, nesterov, bf16=wl.bf16,
                       dropout_seed=77)
    np.testing.assert_array_equal(params, ref["params"])
    np.testing.assert_array_equal(losses, ref["losses"])
    np.testing.assert_array_equal(params2, ref["params"])  # resumed at T/2: the same result
    np.testing.assert_array_equal(losses2, ref["losses"])
    l_ref, g_ref = oracle.loss_and_grad(wl.ops, wl.in_shape, wl.stage_end, p0, xs[0], ys[0], bf16=wl.bf16,
                                        dropout_seed=77, step=0)
    assert loss0 == l_ref
    np.testing.assert_array_equal(g0, g_ref)


@pytest.fixture(scope="module")
def plan_driver(tmp_path_factory):
    """The scheduler's host code with ASan + UBSan (host pass only), linked
    with the library's other objects as the regular build compiles them."""
    from paper_1912_12675_amd import build as B

    d = tmp_path_factory.mktemp("asan_plan")
    objs = [os.path.join(B.BUILD, f.replace(".hip", ".o")) for f in B.SOURCES if f != "api.hip"]
    if not all(os.path.exists(o) for o in objs):
        B.build()
    api = str(d / "api_asan.o")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([B.HIPCC, *B.FLAGS, "-g", *san, "-c", os.path.join(B.CSRC, "api.hip"), "-o", api],
                   check=True, capture_output=True)
    # the driver is plain C++ (no device code): ROCm's clang, the compiler of the library's host code
    drv = str(d / "plan_driver.o")
    clang = os.path.join(os.path.dirname(os.path.realpath(B.HIPCC)), "..", "lib", "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang++"
    subprocess.run([clang, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-c", os.path.join(NATIVE, "plan_driver.cpp"), "-o", drv],
                   check=True, capture_output=True)
    exe = str(d / "plan_driver")
    subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", *san, drv, api, *objs, "-o", exe], check=True,
                   capture_output=True)
    return exe


def test_scheduler_under_sanitizers(plan_driver, tmp_path):
    from paper_1912_12675_amd import psw

    T = 12
    wls = [synth.lenet5_workload(), synth.alexnet_workload(batch=4), synth.resnet20_workload(),
           synth.resnet20_workload(bf16=True), synth.vgg16_workload(batch=8, dropout=0.4), synth.resnet110_workload(),
           synth.resnet_two_partition_workload(56, batch=8, n_pipelined=4)]
    inp = tmp_path / "nets.bin"
    with open(inp, "wb") as f:
        f.write(np.array([len(wls)], np.int32).tobytes())
        for wl in wls:
            st = wl.staleness(T).astype(np.int32)
            rd = np.array(wl.ring_depth(T), np.int32)
            f.write(np.array([len(wl.ops), wl.batch, *wl.in_shape, wl.n_stages, int(wl.bf16), T], np.int32).tobytes())
            f.write(np.ascontiguousarray(wl.ops, np.int32).tobytes())
            f.write(np.ascontiguousarray(wl.stage_end, np.int32).tobytes())
            f.write(rd.tobytes())
            f.write(st.tobytes())
    env = dict(SAN_ENV, LSAN_OPTIONS="suppressions=" + os.path.join(NATIVE, "lsan_runtime.supp"))
    r = subprocess.run([plan_driver, str(inp)], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, f"driver exit {r.returncode}\n{r.stderr[-3000:]}"
    lines = r.stdout.splitlines()
    it = iter(lines)
    for wl in wls:
        st = wl.staleness(T)
        sizes = next(it).split()
        assert sizes[0] == "sizes"
        for t in range(T):
            got = [int(v) for v in next(it).split()[1:]]
            assert got[0] == t
            ref = psw.net_plan_only(wl.ops, wl.batch, wl.in_shape, wl.stage_end, wl.ring_depth(T), t, st[t],
                                    bf16=wl.bf16)
            assert got[1] == len(ref)
            assert [tuple(got[2 + 4 * i:6 + 4 * i]) for i in range(len(ref))] == [tuple(p) for p in ref]
        assert next(it) == "checks ok"
