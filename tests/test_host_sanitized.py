"""The KV-store table and the prefix-key hash built with AddressSanitizer and
UndefinedBehaviorSanitizer (host code only, g++), driven by random operations
that are replayed on the Python FIFO model and checked against the xxhash
package; failed host allocations are injected and must leave the table as it
was.  No GPU."""
import os
import shutil
import subprocess

import numpy as np
import pytest
import xxhash

from oracle.cache_table import FifoTable

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
CSRC = os.path.join(ROOT, "paper_2606_07571_amd", "csrc")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("asan") / "table_check")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", f"-I{CSRC}",
           os.path.join(NATIVE, "table_check_main.cpp"), os.path.join(CSRC, "xxh64.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip(f"sanitizer build unavailable: {r.stderr[-400:]}")
    return exe


def _run(exe, lines):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:exitcode=24")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                       env=env, timeout=120)
    assert r.returncode == 0, f"sanitizer run failed ({r.returncode}):\n{r.stderr[-3000:]}"
    assert "runtime error" not in r.stderr, r.stderr[-3000:]
    return r.stdout.splitlines()


@pytest.mark.parametrize("cap", [1, 3, 8])
def test_table_under_sanitizers_matches_model(checker, cap):
    rng = np.random.default_rng(100 + cap)
    keys = [int(x) for x in rng.integers(0, 2**64 - 1, size=20, dtype=np.uint64)]
    ref = FifoTable(cap)
    cmds, expect = [f"C {cap}"], ["ok"]
    for step in range(3000):
        k = keys[rng.integers(len(keys))]
        op = rng.integers(4)
        if op == 0:
            cmds.append(f"I {k} {step}")
            try:
                e = ref.insert(k, step)
                expect.append(f"{1 if e is not None else 0} {e if e is not None else 0}")
            except KeyError:
                expect.append("-1 0")
        elif op == 1:
            cmds.append(f"E {k}")
            expect.append("1" if ref.invalidate(k) else "0")
        elif op == 2:
            cmds.append(f"L {k}")
            meta = ref.lookup(k)
            expect.append(str(-1 if meta is None else meta))
        else:
            cmds.append("K")
            order = ref.order()
            expect.append(" ".join([str(len(order))] + [str(x) for x in order]))
    got = _run(checker, cmds)
    assert got == expect


def test_failed_allocation_leaves_table_unchanged(checker):
    """Every allocation of an insert fails in turn (the first, the second, ...):
    each failed insert reports the failure, evicts nothing and leaves keys,
    FIFO order and entries as they were; the next insert succeeds."""
    cap = 3
    ref = FifoTable(cap)
    cmds, expect = [f"C {cap}"], ["ok"]
    nxt = 1
    for round_ in range(12):
        for n_ok in range(4):
            k = 1000 + nxt
            cmds += [f"F {n_ok}", f"I {k} {nxt}", "F -1", "K"]
            order = ref.order()
            # with n_ok allocations allowed the insert may or may not need more;
            # the driver reports -2 (failed, unchanged) or success
            expect += ["ok", None, "ok", None]
            nxt += 1
        k = 5000 + round_
        cmds += [f"I {k} {round_}", "K"]
        expect += [None, None]
    got = _run(checker, cmds)
    assert len(got) == len(expect)
    # replay: a failed insert (-2) must not change the keys; a successful one
    # must match the model
    i = 0
    ref = FifoTable(cap)
    failures = 0
    for c in cmds:
        line = got[i]
        i += 1
        if c.startswith("I "):
            _, k, m = c.split()
            r, ev = line.split()
            if r == "-2":
                failures += 1
                assert ev == "0"
            else:
                e = ref.insert(int(k), int(m))
                assert int(r) == (1 if e is not None else 0)
                assert int(ev) == (e if e is not None else 0)
        elif c == "K":
            order = ref.order()
            assert line == " ".join([str(len(order))] + [str(x) for x in order])
    assert failures >= 12, "no allocation failure was injected"


def test_xxh64_under_sanitizers(checker):
    rng = np.random.default_rng(7)
    cmds, expect = [], []
    for n in list(range(0, 72)) + [255, 1000, 4099]:
        data = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        for seed in (0, 2**64 - 1, 12345):
            cmds.append(f"H {seed} {data.hex() if n else '-'}")
            expect.append(str(xxhash.xxh64_intdigest(data, seed=seed)))
    assert _run(checker, cmds) == expect
