"""The host half of libdlfp built with AddressSanitizer and UndefinedBehaviorSanitizer.

The metadata builder and the Eq. 2 controller (plain C++, no HIP calls) are
compiled with the host compiler, sanitizers on and recovery off, into
tests/native/host_driver.cpp, which runs them on seeded random iterations
(every supported g, 1 to 8 KV heads, automatic and forced split policies,
capacity probing, malformed inputs) and prints inputs and outputs.  Any
out-of-bounds access, use after free, leak or undefined operation aborts the
driver; every output must also equal the oracle twins: slot mapping and query
offsets bit-exact, the work list and append records valid (every visible pair
covered once), controller caps equal to Eq. 2 step for step.
"""
import json
import os
import shutil
import subprocess

import pytest

from oracle import controller as oc
from oracle import meta as om

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CASES = 12


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    out = str(tmp_path_factory.mktemp("native") / "host_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", f"-I{ROOT}/include", f"-I{ROOT}/paper_2609_38386_amd/csrc",
           os.path.join(ROOT, "tests", "native", "host_driver.cpp"),
           os.path.join(ROOT, "paper_2609_38386_amd", "csrc", "dlfp_host.cpp"), "-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return out


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_host_code_under_sanitizers_matches_the_twins(driver, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([driver, str(seed), str(CASES)], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    lines = [json.loads(x) for x in r.stdout.splitlines()]
    kinds = {}
    for c in lines:
        kinds[c["kind"]] = kinds.get(c["kind"], 0) + 1
        if c["kind"] == "meta":
            _check_meta(c)
        elif c["kind"] == "errors":
            assert c["q_len_zero"] == -1 and c["bad_tuning"] == -1 and c["null_q_len"] == -1
            assert c["block_out_of_pool"] == -2 and c["head_dim_64"] == -5
        else:
            _check_controller(c)
    assert kinds == {"meta": CASES, "errors": CASES, "controller": CASES}


def _check_meta(c):
    import numpy as np
    n = len(c["q_len"])
    bt = np.asarray(c["bt"], dtype=np.int64).reshape(n, c["max_blocks"])
    if c["probe_status"] == -2:      # more split groups than counters: refused outright
        assert c["status"] == -2
        return
    assert c["probe_status"] == -3   # no capacity given: the counts come back
    assert c["status"] == 0, c["status"]
    cu_q, q_pos0, slots = om.varlen_meta(c["q_len"], c["kv_len"], bt)
    assert c["cu_q"] == cu_q and c["q_pos0"] == q_pos0 and c["slots"] == slots
    work = np.asarray(c["work"], dtype=np.int64).reshape(-1, om.WORK_INTS)
    units = work[:c["num_units"]]
    om.check_work_list(units, c["num_prefill"], c["q_len"], c["kv_len"], c["hq"], c["hkv"],
                       c["num_groups"], c["workspace_bytes"])
    om.check_append_records(work[c["num_units"]:], units, c["num_prefill"], c["q_len"],
                            c["kv_len"], c["hkv"], c["num_waiting"])


def _check_controller(c):
    assert c["status"] == 0
    ctrl = oc.Controller(c["target"], c["c_initial"], c["c_min"], c["c_max"], 128)
    for nd, guarded, obs, st, nxt in c["steps"]:
        assert st == 0
        assert nxt == ctrl.step(nd, bool(guarded), obs)
    assert c["negative_observation"] == -1
