"""AddressSanitizer + UndefinedBehaviorSanitizer builds of the host code (CPU).

The CPU oracle (oracle/akvref.c) and the library's host layer (plan,
layout offsets, argument and size checks, export, fault injection; the
kernels' device code is built normally, the sanitizers instrument the host
side only) are rebuilt with -fsanitize=address,undefined into a temporary
directory, and a child Python process with the sanitizer runtime preloaded
runs the oracle on small problems and the host entry points on valid,
invalid and undersized arguments.  Any sanitizer report ends the child with
an error.  No GPU.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_02901_amd", "csrc")
LLVM = "/opt/rocm/llvm/bin"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]

CHILD = textwrap.dedent(r'''
    import ctypes, sys
    import numpy as np
    sys.path.insert(0, ROOT)
    from oracle import akvref as R
    from paper_2608_02901_amd import _native as N
    R._lib = ctypes.CDLL(ORACLE)
    R._declare(R._lib)
    N.LIB_PATH = HOSTLIB
    N._lib = None
    L = N.lib()

    # oracle: a small compression pass (selection, assignment, utilities,
    # budget, codec), reconstruction and attention
    rng = np.random.default_rng(0)
    bf = lambda x: np.asarray(x, np.float32).astype(np.float64)
    H, Hq, S, D, W = 2, 4, 160, 32, 8
    K, V, Q = bf(rng.standard_normal((H, S, D))), bf(rng.standard_normal((H, S, D))), bf(rng.standard_normal((Hq, W, D)))
    for mode in (R.SCALE_ABSMAX_OUTER, R.SCALE_RMS):
        enc = R.encode(K, V, Q, W=W, k=24, bf16=False, budget=0.1, G=8, scale_mode=mode)
        Kh = R.reconstruct(K, enc, "K", 8, 0)
        Vh = R.reconstruct(V, enc, "V", 8, 0)
        R.attention(Kh, Vh, rng.standard_normal((Hq, D)))
    R.encode(K, V, Q, W=W, k=S, bf16=True, G=D)
    R.encode(K, V, Q, W=W, k=W, bf16=True, G=D, budget_mode=R.BUDGET_THETA, budget=0.3)
    assert R.theta_budget(32768, 8, 128, 32, 256, 128, 0.05) == 91056

    # host layer: plans over a grid of configurations, invalid ones included
    ok = bad = 0
    for H_ in (1, 8):
        for g in (1, 3, 4, 8):
            for S_ in ([33], [4096], [1000, 70000], [40 + 7 * i for i in range(64)], [1 << 22]):
                for kw in (dict(anchor_frac=0.02), dict(anchor_count=64, anchor_frac=0.0),
                           dict(anchor_count=16384, anchor_frac=0.0, budget_mode=N.BUDGET_THETA, budget=0.05)):
                    cfg = N.Config.make(num_kv_heads=H_, num_q_heads=H_ * g, dtype=N.BF16, max_append=4, **kw)
                    try:
                        p = N.Plan(cfg, S_)
                        ok += 1
                    except N.AnchorKVError:
                        bad += 1
                        continue
                    host = np.zeros(p.cache_bytes, np.uint8)
                    try:
                        N.export(p, host, 0)
                    except N.AnchorKVError as e:
                        assert e.status == N.ERR_CORRUPT_CACHE
                    assert L.anchorkv_encode(p.handle, 1, 1, 0, 1, 0, None, 0, 1, 0, 1, 0, None) == N.ERR_BUFFER_TOO_SMALL
    assert ok > 20 and bad > 5, (ok, bad)
    # the fault-injection path (stops at the first kernel, before any launch)
    import os
    os.environ["ANCHORKV_FAULT_INJECT"] = "k_init"
    p = N.Plan(N.Config.make(num_kv_heads=8, num_q_heads=32, anchor_frac=0.02, dtype=N.BF16), [4096])
    kv, qo = 8 * 4096 * 128 * 2, 32 * 32 * 128 * 2
    st = L.anchorkv_encode(p.handle, 8, 8, kv, 8, qo, None, 0, 8, p.cache_bytes, 8, p.encode_ws_bytes, None)
    assert st == N.ERR_HIP and b"k_init" in L.anchorkv_last_error()
    print("sanitized child ok", ok, bad)
''')


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    if r.returncode != 0:
        raise AssertionError(f"{' '.join(cmd[:3])} ... failed ({r.returncode}):\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}")
    return r


@pytest.mark.skipif(not os.path.exists(os.path.join(LLVM, "clang")), reason="ROCm clang not present")
def test_oracle_and_host_layer_under_asan_ubsan(tmp_path):
    oracle = str(tmp_path / "libakvref_san.so")
    _run([os.path.join(LLVM, "clang"), "-O1", "-g", "-ffp-contract=off", "-fPIC", "-shared", *SAN, "-o", oracle,
          os.path.join(ROOT, "oracle", "akvref.c"), "-lm"])
    # host layer: every source of the library, the sanitizers on the host side
    # only (each -fsanitize= right after -Xarch_host); device code as usual
    from paper_2608_02901_amd import build as B
    host_san = [x for f in SAN for x in ("-Xarch_host", f)]
    import concurrent.futures as cf

    def compile_one(src):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        _run([HIPCC, *B.FLAGS, *B.EXTRA.get(src, []), *host_san, "-g", "-x", "hip", "-c", os.path.join(CSRC, src),
              "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(compile_one, B.SOURCES))
    hostlib = str(tmp_path / "libanchorkv_san.so")
    _run([os.path.join(LLVM, "clang++"), "-shared", *SAN, "-o", hostlib, *objs, "-L/opt/rocm/lib", "-lamdhip64",
          "-Wl,-rpath,/opt/rocm/lib"])
    rt = _run([os.path.join(LLVM, "clang"), "-print-file-name=libclang_rt.asan-x86_64.so"]).stdout.strip()
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = f"ROOT = {ROOT!r}\nORACLE = {oracle!r}\nHOSTLIB = {hostlib!r}\n" + CHILD
    r = _run([sys.executable, "-c", code], env=env, timeout=600)
    assert "sanitized child ok" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-3000:]
    # the harness reports a planted heap overflow (so a clean run means something)
    bug = tmp_path / "bug.c"
    bug.write_text("#include <stdlib.h>\nint oob(int n){int*a=(int*)malloc(4*n);int s=a[n];free(a);return s;}\n")
    buglib = str(tmp_path / "libbug.so")
    _run([os.path.join(LLVM, "clang"), "-O0", "-g", "-fPIC", "-shared", *SAN, "-o", buglib, str(bug)])
    r = subprocess.run([sys.executable, "-c", f"import ctypes; ctypes.CDLL({buglib!r}).oob(8)"], env=env,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr
