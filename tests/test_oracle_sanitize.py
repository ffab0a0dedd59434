"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (host build only).

`oracle/cr_oracle.c` is compiled a second time with ``-fsanitize=address,undefined
-fno-sanitize-recover=all`` and loaded into a child interpreter (the sanitizer runtimes
preloaded, ``CR_ORACLE_LIB`` pointing at the sanitized library). The child runs every
oracle entry point over small streams -- counting, admission, LPT and hash placement (all
ablation variants), static and live dispatch, the replay with carried state, and the
thread fan-out -- and prints a digest of each result. Any out-of-bounds access, use after
free or undefined operation aborts the child; the digests must equal those of the plain
build in this process."""
import hashlib
import json
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "cr_oracle.c")

# The child and this process run the same script; only the library differs.
SCRIPT = r"""
import hashlib, json, sys
import numpy as np
sys.path.insert(0, sys.argv[1])
from oracle import pipeline as opipe
from paper_2608_19677_amd import workload as wl

def digest(v, path="", out=None):
    out = {} if out is None else out
    if isinstance(v, dict):
        for k in sorted(v, key=repr):
            digest(v[k], f"{path}.{k}", out)
    elif isinstance(v, (list, tuple)):
        for i, x in enumerate(v):
            digest(x, f"{path}[{i}]", out)
    elif isinstance(v, np.ndarray):
        out[path] = hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest()
    else:
        out[path] = repr(v)
    return out

res = {}
a = wl.small_random(3, num_keys=400, n=30_000, R=30, Ws=[16, 40], J=3, hot=2, hot_share=0.3)
res["static"] = digest(opipe.run(a))
res["threads"] = digest(opipe.run(a, threads=3))
res["live"] = digest(opipe.run(a, dispatch="live"))
b = wl.small_random(5, num_keys=3000, n=40_000, R=100, Ws=[8, 70], J=2, hot=3, hot_share=0.4, qs=[(1, 1), (4, 5)])
first = opipe.run(b)
res["wide"] = digest(first)
res["carried"] = digest(opipe.run(b, lru=first["lru"], counts_prev=first["counts"][-1]))
c = wl.small_random(9, num_keys=500, n=20_000, R=16, Ws=[32], J=2, hot=8, hot_share=0.5)
c.candidates = [wl.Candidate(32, 2, 5, v, 7) for v in ("flat", "affinity", "replicated", "full")]
res["variants"] = digest(opipe.run(c))
d = wl.small_random(2, num_keys=1, n=5_000, R=1, Ws=[3], J=1)
res["one_key"] = digest(opipe.run(d))
print("DIGESTS " + json.dumps(res, sort_keys=True))
"""


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.fixture(scope="module")
def san_lib(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("sanitizer runtimes not available")
    out = str(tmp_path_factory.mktemp("san") / "libcr_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                           "-fPIC", "-shared", SRC, "-o", out])
    return out, asan, ubsan


def _digests(env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    p = subprocess.run([sys.executable, "-c", SCRIPT, ROOT], capture_output=True, text=True, env=env, timeout=600)
    assert p.returncode == 0, f"exit {p.returncode}\n{p.stderr[-4000:]}"
    line = [x for x in p.stdout.splitlines() if x.startswith("DIGESTS ")]
    assert line, p.stdout[-2000:] + p.stderr[-2000:]
    return json.loads(line[0][len("DIGESTS "):])


def test_oracle_clean_under_asan_and_ubsan(san_lib):
    lib, asan, ubsan = san_lib
    san = _digests({"CR_ORACLE_LIB": lib, "LD_PRELOAD": f"{asan}:{ubsan}",
                    "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                    "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    plain = _digests({})
    assert san.keys() == plain.keys()
    for k in plain:
        assert san[k] == plain[k], k
