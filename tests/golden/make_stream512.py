#!/usr/bin/env python3
"""Write stream512.json beside this script: the fp64 oracle's run of
Algorithm 1 over the 512-step streaming workload (16 sequences, starting
prefix 1024, W=32, Hq/Hkv=32/8, D=128, V=151936, the window starting as all
masks, greedy fill, T=0.1, tau=0.9, lambda=0.01, seed 0).

It calls only the oracle and the seeded input generator.  The selection
does not depend on attention (the logits are inputs), so no attention is run
here; the GPU test checks attention at sampled steps against the oracle
itself, rebuilding the oracle's cache from the per-step commit counts stored
here.  Sequences are independent, so each runs in its own process.

Stored per sequence: the commit count of every step, the number of
committed tokens, sha256 of the committed token stream and of the slot
stream (int32 little-endian), the first 64 committed tokens, the final
window and prefix length, and the window and prefix length before each of
the snapshot steps.

Usage: python tests/golden/make_stream512.py [--procs 8]
"""
import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import wedlm_oracle as O  # noqa: E402
from paper_2512_22737_amd import workloads as WL  # noqa: E402

SEED = 0
SNAPSHOTS = (0, 1, 100, 255, 511)   # window state before these steps


def _sha(a) -> str:
    return hashlib.sha256(np.asarray(a, dtype="<i4").tobytes()).hexdigest()


def run_sequence(b: int) -> dict:
    wl = WL.WORKLOADS["stream512"]
    c0 = WL.prefix_lengths(wl, SEED)
    win0 = WL.initial_window(wl, SEED)
    bt, _ = WL.block_table(wl, c0, SEED)
    pool = WL.logit_pool(wl, SEED)
    params = {}

    def row(t, _b, i):
        if t not in params:
            params.clear()
            params[t] = WL.logit_row_params(wl, SEED, t)
        idx, shift, spiked, tok = params[t]
        r = b * wl.W + i
        x = np.roll(pool[idx[r]], shift[r])
        if spiked[r]:
            x[tok[r]] += np.float32(wl.spike)
        return x

    win = win0[b:b + 1].copy()
    c = c0[b:b + 1].copy()
    n_hist, toks, slots, snaps = [], [], [], {}
    bounds = list(SNAPSHOTS) + [wl.steps]
    for s0, s1 in zip(bounds[:-1], bounds[1:]):
        snaps[s0] = {"win": [int(x) for x in win[0]], "c": int(c[0])}
        if s1 == s0:
            continue
        r = O.stream(win, c, s1 - s0, lambda t: {}, wl.Hq, wl.Hkv, wl.theta,
                     wl.tau, wl.lam, wl.temp, bt[b:b + 1],
                     logits_row=lambda t, bb, i, s0=s0: row(s0 + t, bb, i))
        n_hist += [int(x) for x in r["n"][:, 0]]
        toks += r["tokens"][0]
        slots += r["slots"][0]
        win, c = r["win"], r["c"]
    return {"n": n_hist, "n_tokens": len(toks), "tokens_sha256": _sha(toks),
            "slots_sha256": _sha(slots), "tokens_head": toks[:64],
            "final_win": [int(x) for x in win[0]], "final_c": int(c[0]),
            "snapshots": {str(k): v for k, v in snaps.items()}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--procs", type=int, default=8)
    args = ap.parse_args()
    wl = WL.WORKLOADS["stream512"]
    t0 = time.time()
    with ProcessPoolExecutor(max_workers=args.procs) as ex:
        seqs = list(ex.map(run_sequence, range(wl.B)))
    out = {
        "what": ("oracle token stream of the 512-step streaming workload "
                 "(Algorithm 1 with Eq. (11) selection; readings D1-D14)"),
        "workload": "stream512", "seed": SEED, "steps": wl.steps,
        "B": wl.B, "W": wl.W, "tau": wl.tau, "lambda": wl.lam,
        "temperature": wl.temp, "snapshots": list(SNAPSHOTS),
        "p_cache": O.p_cache(np.array([s["n"] for s in seqs]).T, wl.W),
        "sequences": seqs,
    }
    path = os.path.join(HERE, "stream512.json")
    with open(path, "w") as f:
        json.dump(out, f, separators=(",", ":"))
        f.write("\n")
    print(f"wrote {path} in {time.time() - t0:.0f} s; p_cache "
          f"{out['p_cache']:.4f}; tokens per sequence "
          f"{[s['n_tokens'] for s in seqs]}")


if __name__ == "__main__":
    main()
