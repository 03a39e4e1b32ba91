"""Writes the full-size oracle fixtures ``fullsize_<workload>.npz`` (test data).

For the 32768-token layers ``q8b`` and ``stress`` (seed 0 of
``synth.make_layer``), every page's window deletion effect on every query
head, before and after the commit, in float64 from the oracle's closed form
of Eq. (6) (``oracle.page_effects(method="closed")``, itself pinned to the
brute-force definition by the CPU tests):

    R_pre [n], R_head_pre [n, Hq]   prefix cache [0, S_pre), window Q^-
    R_post [n], R_head_post [n, Hq] whole cache, window Q^+

plus SHA-256 digests of the inputs the values were computed from, so that a
change of the synthetic generator shows up as a clear error instead of a
parity failure.  Only ``oracle/`` and ``synth/`` are used.

    python tests/golden/make_fullsize.py [q8b] [stress]

Runtime on 8 cores: about 10 minutes per workload (one process per
(pass, query head)).
"""
from __future__ import annotations

import hashlib
import os
import sys
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

SEED = 0


def input_digest(L) -> str:
    h = hashlib.sha256()
    for a in (L.k, L.v, L.q_pre, L.q_post, L.pos, L.qpos_pre, L.qpos_post,
              np.asarray(L.pages, dtype=np.int64)):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def _one(args):
    name, which, h = args
    from threadpoolctl import threadpool_limits
    import oracle as O
    from synth import WORKLOADS, make_layer
    with threadpool_limits(1):
        L = make_layer(WORKLOADS[name], seed=SEED)
        if which == "pre":
            S = L.layout.s_pre
            _, Rh = O.page_effects(L.k[:, :S], L.v[:, :S], L.pos[:S], L.q_pre, L.qpos_pre, L.pages,
                                   method="closed", heads=[h])
        else:
            _, Rh = O.page_effects(L.k, L.v, L.pos, L.q_post, L.qpos_post, L.pages, method="closed",
                                   heads=[h])
    return which, h, Rh[:, h]


def make(name: str, workers: int = 8) -> str:
    from synth import WORKLOADS, make_layer
    L = make_layer(WORKLOADS[name], seed=SEED)
    Hq, n = L.w.n_q_heads, len(L.pages)
    out = {"R_head_pre": np.full((n, Hq), np.nan), "R_head_post": np.full((n, Hq), np.nan)}
    jobs = [(name, which, h) for which in ("pre", "post") for h in range(Hq)]
    with ProcessPoolExecutor(max_workers=workers) as ex:
        for which, h, col in ex.map(_one, jobs):
            out[f"R_head_{which}"][:, h] = col
            print(f"{name} {which} head {h} done", flush=True)
    path = os.path.join(HERE, f"fullsize_{name}.npz")
    np.savez_compressed(path, R_pre=out["R_head_pre"].max(axis=1), R_post=out["R_head_post"].max(axis=1),
                        R_head_pre=out["R_head_pre"], R_head_post=out["R_head_post"],
                        digest=np.array(input_digest(L)), seed=np.array(SEED))
    return path


if __name__ == "__main__":
    for nm in (sys.argv[1:] or ["q8b", "stress"]):
        print(make(nm), flush=True)
