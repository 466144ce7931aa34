"""Write the full-batch fp64 oracle scores of the scoring workloads.

    python -m tests.golden.make_golden [workload ...]

For each named scoring workload this draws the seeded inputs and weights
(paper_2604_12891_amd.workload, which holds no model arithmetic), scores
every program with the fp64 oracle (oracle.model.score, in chunks of
programs: programs are independent) and writes
tests/golden/<workload>.npz with

  scores   float64 [B]   the oracle's score of every program
  sha256   str           digest of the weights, features and lengths scored
                         (the GPU tests recompute it, so a changed generator
                         fails loudly instead of comparing other inputs)

Nothing here calls the HIP library: every stored value is the oracle's.
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import model as om  # noqa: E402
from paper_2604_12891_amd import workload as wl  # noqa: E402

# configs 2-4 of the scoring path: the headline round, the large bf16 pool
# and the long sequences
DEFAULT = ["score_B4096_L25_d256_f32", "score_B65536_L25_d256_bf16", "score_B8192_L256_d256_f32"]


def digest(blob: np.ndarray, X: np.ndarray, lengths: np.ndarray) -> str:
    h = hashlib.sha256()
    for a in (blob, X, lengths):
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode() + str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()


def oracle_cfg(m: wl.ModelShape) -> dict:
    return dict(F=m.F, d_model=m.d_model, d_inner=m.d_inner, d_state=m.d_state, d_conv=m.d_conv,
                dt_rank=m.dt_rank, n_layers=m.n_layers, head_hidden=m.head_hidden,
                final_norm=m.final_norm, norm_eps=m.norm_eps, enc_hidden=tuple(m.enc_hidden),
                dec_hidden2=m.dec_hidden2)


def path(name: str) -> str:
    return os.path.join(HERE, name + ".npz")


_job = {}


def _score_chunk(i: int) -> tuple:
    j = _job
    sl = slice(i, i + j["chunk"])
    return i, om.score(j["blob"], j["X"][sl], j["lengths"][sl], j["cfg"])


def make(name: str, chunk: int = 128, jobs: int = 1) -> None:
    """Score the whole batch; `jobs` worker processes (forked, sharing the
    inputs) each take chunks of programs."""
    w = wl.WORKLOADS[name]
    blob, X, lengths = wl.make_workload(name)
    _job.update(blob=blob, X=X, lengths=lengths, cfg=oracle_cfg(w.model), chunk=chunk)
    out = np.full(w.B, np.nan, dtype=np.float64)
    t0 = time.time()
    starts = list(range(0, w.B, chunk))
    if jobs > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(jobs) as pool:
            for n, (i, s) in enumerate(pool.imap_unordered(_score_chunk, starts)):
                out[i:i + chunk] = s
                if n % 32 == 0:
                    print(f"{name}: {(n + 1) * chunk}/{w.B} programs, {time.time() - t0:.0f} s", flush=True)
    else:
        for n, i in enumerate(starts):
            out[i:i + chunk] = _score_chunk(i)[1]
            if n % 32 == 0:
                print(f"{name}: {(n + 1) * chunk}/{w.B} programs, {time.time() - t0:.0f} s", flush=True)
    assert np.all(np.isfinite(out))
    np.savez(path(name), scores=out, sha256=np.array(digest(blob, X, lengths)))
    print(f"{name}: wrote {path(name)} in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("workloads", nargs="*", default=DEFAULT)
    ap.add_argument("--jobs", type=int, default=1, help="worker processes (set OPENBLAS_NUM_THREADS to match)")
    a = ap.parse_args()
    for n in a.workloads:
        make(n, jobs=a.jobs)
