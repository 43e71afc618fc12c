"""Write the native action-chunk fixtures of the mid and large workloads.

Calls only the float64 oracle (`oracle/`) and the seeded input generators
(`synth/`); nothing here touches the HIP library.  For each workload it runs
the native replan of the joint runtime (Sec. 3.4 with no retained state: K
Euler steps from the seeded initial noise under the first observation, the
step counts of Table app-schedules) and stores, in float64:

  action_per_step  [K, B, Na, A]  action rows of x after every Euler step
                                  (the last entry is the action chunk)
  video_rows       [B, n, Cv]     final video latent at the token indices
  video_index      [n]            below (a fixed spread over the sequence)
  sigmas           [K + 1]        the schedule as the device sees it
                                  (float32 values, widened)

Usage (8 cores: about half an hour for mid, two hours for large):

  MALLOC_ARENA_MAX=1 MALLOC_MMAP_MAX_=0 MALLOC_TRIM_THRESHOLD_=68719476736 \
      python tests/golden/make_chunk_goldens.py mid large

The malloc settings keep freed arrays in one heap, so that the per-head
T x T score arrays reuse memory instead of being faulted in anew for every
head (slow on hosts where a first touch of fresh memory is expensive).
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import dit as OD, method as OM  # noqa: E402
from synth import get_workload, make_weights, make_initial_noise, make_observations  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def fixture_path(name: str) -> str:
    return os.path.join(HERE, f"native_chunk_{name}.npz")


def video_index(spec, n: int = 64) -> np.ndarray:
    """n video token indices spread over [0, Nv), first and last included."""
    return np.unique(np.linspace(0, spec.Nv - 1, n).round().astype(np.int64))


def make(name: str) -> None:
    spec = get_workload(name)
    t0 = time.time()
    W = make_weights(spec)
    x0 = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    sig = OM.flow_schedule(spec.K).astype(np.float32).astype(np.float64)
    print(f"{name}: inputs ready in {time.time() - t0:.0f} s", flush=True)
    x = OD.as64(x0)
    per_step = []
    for k in range(spec.K):
        t1 = time.time()
        x, _, _ = OM.denoise(W, spec, x, cond, sig, k, k + 1, None, OM.LayerState())
        per_step.append(OM.action_chunk(spec, x))
        print(f"{name}: step {k + 1}/{spec.K} in {time.time() - t1:.0f} s", flush=True)
    vi = video_index(spec)
    xv, _ = OD.split_trajectory(spec, x)
    np.savez(fixture_path(name), action_per_step=np.stack(per_step), video_rows=xv[:, vi],
             video_index=vi, sigmas=sig, workload=np.array(name), seed=np.array(spec.seed))
    print(f"{name}: wrote {fixture_path(name)} after {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    OD.ATTENTION_THREADS = os.cpu_count() or 1
    for n in sys.argv[1:] or ["mid", "large"]:
        make(n)
