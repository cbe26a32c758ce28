"""The checked build (lib/libpgsr_checked.so, compiled with PGSR_CHECKED):
block ids that device metadata written outside the library puts out of range
make every pool call that reads them return PGSR_ERANGE, on each path that
reads a table or the free stack (three bf16 prefill kernels, decode, crop,
restore + replay in one call, fork), without any access outside the pool; an
intact replay gives the same bits as the default build.

The corrupting cases run in a child process against the checked library only
(tests/checked_build_probe.py refuses any other build)."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHECKED = os.path.join(ROOT, "paper_2609_04875_amd", "lib", "libpgsr_checked.so")

pytestmark = pytest.mark.gpu


def test_checked_build_reports_out_of_range_block_ids(tmp_path):
    import checked_build_probe as probe   # the episode and pool recipe only
    from paper_2609_04875_amd import _native as N
    assert os.path.exists(CHECKED), "build the checked library with __graft_entry__.build()"
    assert not N.LIB_PATH.endswith("libpgsr_checked.so"), "this process must hold the default build"

    # the intact replay on the default build, in this process
    ep = probe.episode()
    pool = probe.fresh_pool(ep)
    q, k, v, o = probe.suffix(ep)
    assert pool.replay(0, [0], [probe.S], q, k, v, o, probe.SCALE) == 0
    torch.cuda.synchronize()
    want = o.view(torch.int16).cpu().numpy()
    pool.close()

    out = tmp_path / "o_checked.npy"
    env = dict(os.environ, PGSR_LIB=CHECKED)
    print("checked build probe: child process", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "checked_build_probe.py"),
                        "--save", str(out)], env=env, capture_output=True, text=True, timeout=240)
    print(r.stderr[-2000:], flush=True)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    res = json.loads(r.stdout.strip().splitlines()[-1])

    assert res["intact"] == N.OK and res["after"] == N.OK
    assert np.array_equal(np.load(out), want), "checked build differs from the default build"
    assert res["after_equal"], "a call after an error differs from the first intact call"
    for case in ("prefill_auto", "prefill_pipelined", "prefill_four_wave", "decode", "crop",
                 "restore_replay", "fork"):
        assert res[case] == N.ERANGE, (case, res[case])
    assert "block id outside" in res["prefill_auto_msg"]
