"""The host C code under AddressSanitizer and UndefinedBehaviorSanitizer:
the fp64 oracle and the host input generator are rebuilt with
-fsanitize=address,undefined (errors fatal) and driven, in a child Python
process that preloads the ASan runtime, through every oracle entry point
on the tiny and wide configurations, an expert-parallel share, the dense
form, the stacked residual and the small attention block.  The child must exit cleanly and produce the
same bits as the regular builds."""
import hashlib
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]

# Runs in the child (and, for the reference digest, in this process).
DRIVER = r'''
import hashlib, sys
import numpy as np
import moe_inputs as mi
import oracle


def run():
    h = hashlib.sha256()
    tiny = mi.WORKLOADS["tiny"]
    for wl in (tiny, tiny.with_(T=40, E=24, k=6)):
        x = wl.x()
        G = [wl.gate(e) for e in range(wl.E)]
        U = [wl.up(e) for e in range(wl.E)]
        D = [wl.down(e) for e in range(wl.E)]
        lg = oracle.router_logits(x, wl.router())
        idx, w = oracle.route_from_logits(lg, wl.k)
        full = oracle.layer(x, wl.router(), wl.bias(), G, U, D, wl.k)
        share = oracle.layer(x, wl.router(), wl.bias(), G, U, D, wl.k, e_begin=2, n_local=2)
        dense = oracle.layer_dense(x, idx, w, G, U, D)
        y2 = oracle.residual_add(x, full["y"])
        for a in (x, lg, idx, w, full["y64"], full["y"], share["y64"], dense, y2):
            h.update(np.ascontiguousarray(a).tobytes())
    # the attention block: T new tokens after a cached prefix
    aw = mi.ATTN_WORKLOADS["attn_tiny"]
    k0, v0 = aw.cache_prefix()
    kc = np.zeros((aw.max_seq, aw.n_kv, aw.hd), np.uint16)
    vc = np.zeros_like(kc)
    kc[:aw.pos0], vc[:aw.pos0] = k0, v0
    r = oracle.attention_block(aw.x(), aw.gamma(), aw.wqkv(), aw.wo(), kc, vc, aw.pos0,
                               aw.n_heads, aw.n_kv, aw.eps, aw.theta)
    for key in ("h", "qkv64", "q", "attn", "o64", "y64", "y"):
        h.update(np.ascontiguousarray(r[key]).tobytes())
    h.update(kc.tobytes())
    return h.hexdigest()


if __name__ == "__main__":
    print(run())
'''


def _build_sanitized(tmp):
    ora = os.path.join(tmp, "libmoe_oracle_san.so")
    gen = os.path.join(tmp, "libmoe_inputs_host_san.so")
    subprocess.run(["gcc", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC",
                    "-shared", *SAN, "-o", ora, os.path.join(ROOT, "oracle", "moe_oracle.c"),
                    os.path.join(ROOT, "oracle", "attn_oracle.c"), "-lm"],
                   check=True)
    subprocess.run(["gcc", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", *SAN,
                    "-o", gen, os.path.join(ROOT, "moe_inputs", "gen_host.c")], check=True)
    return ora, gen


def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's ASan runtime is not installed")
    ora, gen = _build_sanitized(str(tmp_path))
    driver = tmp_path / "driver.py"
    driver.write_text(DRIVER)
    child = ("import sys; sys.path[:0] = [%r, %r]\n" % (ROOT, str(tmp_path)) +
             "import oracle, oracle.build as ob, moe_inputs as mi\n"
             "ob.build = lambda force=False: %r\n" % ora +
             "mi._HOST_LIB = %r\n" % gen +
             "import driver; print(oracle.lib()._name); print(driver.run())\n")
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.stdout.strip().splitlines()[-2] == ora      # the sanitized oracle ran
    # the same bits as the regular builds
    sys.path.insert(0, str(tmp_path))
    try:
        import driver as ref
        assert r.stdout.strip().splitlines()[-1] == ref.run()
    finally:
        sys.path.remove(str(tmp_path))
        sys.modules.pop("driver", None)


def test_the_harness_catches_an_out_of_bounds_read(tmp_path):
    """Control: the same flags, runtime and child setup on a function that
    reads one element past its buffer must end the child with an ASan
    report."""
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's ASan runtime is not installed")
    src = tmp_path / "oob.c"
    src.write_text("#include <stdlib.h>\n"
                   "unsigned oob(int n) { unsigned* p = calloc(n, sizeof(unsigned)); unsigned s = 0;\n"
                   "  for (int i = 0; i <= n; ++i) s += p[i];\n"
                   "  free(p); return s; }\n")
    lib = tmp_path / "liboob.so"
    subprocess.run(["gcc", "-fPIC", "-shared", *SAN, "-o", str(lib), str(src)], check=True)
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([sys.executable, "-c", "import ctypes; ctypes.CDLL(%r).oob(8)" % str(lib)],
                       capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr
