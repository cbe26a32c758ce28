"""Drives the checked build (lib/libpgsr_checked.so) for test_gpu_checked.py.

Run as a child process with PGSR_LIB naming the checked library; main()
refuses to run against any other build, because the cases below write block ids
outside the pool into device metadata, which only the checked build turns
into an error (the default build would use them as addresses).

Output: one JSON line with the status of every case, and (``--save PATH``)
the bits of the intact replay's output, which the parent compares with the
default build's.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import workloads as W  # noqa: E402
from paper_2609_04875_amd import BF16, KVPool, workspace_bytes  # noqa: E402
from paper_2609_04875_amd import _native as N  # noqa: E402

GEOM = W.AttnGeometry(32, 8, 128)
P, S, T = 300, 100, 420        # kept prefix, replayed suffix, contaminated run
SCALE = 128 ** -0.5


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def episode():
    return W.draw_episode(np.random.default_rng(77), GEOM, "bf16", P, S, T)


def fresh_pool(ep, ws=False):
    """A pool holding the contaminated run of seq 0, cropped to P (blocks 0..18 kept)."""
    pool = KVPool(1, 32, 8, 128, n_blocks=96, max_seqs=4, max_blocks_per_seq=40, dtype=BF16,
                  workspace_bytes=workspace_bytes(32, 128, 64) if ws else 0)
    cq, ck, cv = (dev(ep.contaminated(x)) for x in ("q", "k", "v"))
    assert pool.replay(0, [0], [T], cq, ck, cv, torch.empty_like(cq), SCALE) == 0
    assert pool.crop([0], [P]) == 0
    torch.cuda.synchronize()
    return pool


def suffix(ep):
    q, k, v = (dev(getattr(ep, x)[P:]) for x in ("q", "k", "v"))
    return q, k, v, torch.empty_like(q)


def corrupt(pool, seq, entry):
    pool.block_tables[seq, entry] = pool.n_blocks + 1000   # outside [0, n_blocks)
    torch.cuda.synchronize()


def main():
    if not N.LIB_PATH.endswith("libpgsr_checked.so"):
        sys.exit("checked_build_probe.py runs only with PGSR_LIB naming libpgsr_checked.so")
    ap = argparse.ArgumentParser()
    ap.add_argument("--save", required=True)
    args = ap.parse_args()
    torch.cuda.set_device(0)
    ep = episode()
    res = {}

    log("case: intact replay (checked build)")
    pool = fresh_pool(ep)
    q, k, v, o = suffix(ep)
    res["intact"] = pool.replay(0, [0], [S], q, k, v, o, SCALE)
    torch.cuda.synchronize()
    np.save(args.save, o.view(torch.int16).cpu().numpy())
    pool.close()

    # a kept prefix entry (block 3 of seq 0) corrupted: only the attention
    # kernels read it, through each prefill kernel in turn
    for kind in ("auto", "pipelined", "four_wave"):
        log(f"case: corrupted prefix entry, {kind} prefill kernel")
        pool = fresh_pool(ep)
        pool.set_prefill_kernel(kind)
        corrupt(pool, 0, 3)
        q, k, v, o = suffix(ep)
        res[f"prefill_{kind}"] = pool.replay(0, [0], [S], q, k, v, o, SCALE)
        res[f"prefill_{kind}_msg"] = N.lib.pgsr_last_error().decode()
        pool.close()

    log("case: corrupted prefix entry, decode (one token, split keys)")
    pool = fresh_pool(ep, ws=True)
    corrupt(pool, 0, 5)
    q, k, v, o = (t[:1] for t in suffix(ep))
    res["decode"] = pool.replay(0, [0], [1], q.contiguous(), k.contiguous(), v.contiguous(),
                                o.contiguous(), SCALE)
    pool.close()

    log("case: corrupted entry released by a crop")
    pool = fresh_pool(ep)
    corrupt(pool, 0, 17)
    res["crop"] = pool.crop([0], [100])
    pool.close()

    log("case: corrupted entry released by restore + replay in one call")
    pool = fresh_pool(ep)
    corrupt(pool, 0, 16)
    q, k, v, o = suffix(ep)
    q2, k2, v2, o2 = (t[: S // 2].contiguous() for t in (q, k, v, o))
    res["restore_replay"] = pool.restore_replay(0, [0], [240], [S // 2], q2, k2, v2, o2, SCALE)
    pool.close()

    log("case: corrupted entry of a fork source")
    pool = fresh_pool(ep)
    corrupt(pool, 0, 2)
    res["fork"] = pool.fork([0], [1])
    pool.close()

    log("case: intact replay after an error (flag cleared)")
    pool = fresh_pool(ep)
    q, k, v, o = suffix(ep)
    res["after"] = pool.replay(0, [0], [S], q, k, v, o, SCALE)
    torch.cuda.synchronize()
    res["after_equal"] = bool(np.array_equal(o.view(torch.int16).cpu().numpy(), np.load(args.save)))
    pool.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
