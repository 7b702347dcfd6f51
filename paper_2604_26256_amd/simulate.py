"""Control-plane simulator of a rollout cluster (CPU only).

Compares the synchronous batch barrier with multi-version streaming (Sec. 3.2)
driven by the library's native orchestrator planners (Sec. 3.3), on synthetic
long-tailed response lengths, and reports the inter-node bubble the paper
measures (App. C.3: the share of decode time spent waiting for the longest
trajectory of a step), slot utilisation and token throughput.

Model (kept small on purpose):
* D DP groups with S request slots each; every running request emits one
  token per TPOT tau (Eq. (1): tau is about constant for a rollout engine).
  Time advances in ticks of `chunk` tokens.
* Synchronous: each step dispatches RBS = TBS prompts, waits until all are
  done, then trains for `train_s` while the cluster idles.
* Multi-version: RBS > TBS prompts per version; the trainer starts as soon as
  TBS trajectories are collected (overlapping rollout) and, when done,
  promotes a new version.  At each promotion the planners re-partition the
  groups over the versions by workload (requests migrate with their KV, at no
  cost here) and supplement prompts: the latest version up to its RBS, legacy
  versions only into idle slots.  A version with work may not fall more than
  K - 1 versions behind the latest (the sliding window): the trainer waits for
  it.

    python -m paper_2604_26256_amd.simulate --steps 8
"""
from __future__ import annotations

import argparse
import dataclasses
import json

import numpy as np


@dataclasses.dataclass
class Config:
    groups: int = 16
    slots: int = 32
    rbs: int = 512
    tbs: int = 256
    staleness: int = 3
    tau_s: float = 0.02
    train_s: float = 30.0
    chunk: int = 64
    median: float = 1024.0
    sigma: float = 1.2
    lo: int = 16
    hi: int = 32768
    seed: int = 0


def _lengths(cfg: Config, rng, n):
    x = np.rint(np.exp(rng.normal(np.log(cfg.median), cfg.sigma, n)))
    return np.clip(x, cfg.lo, cfg.hi).astype(np.int64)


def bubble(lengths) -> float:
    """Inter-node bubble of one step: 1 - mean / max response length."""
    lengths = np.asarray(lengths, np.float64)
    return float(1.0 - lengths.mean() / lengths.max()) if lengths.size else 0.0


def simulate_sync(cfg: Config, steps: int) -> dict:
    rng = np.random.default_rng(cfg.seed)
    cap = cfg.groups * cfg.slots
    t, busy_slot_s, tokens, bubbles = 0.0, 0.0, 0, []
    for _ in range(steps):
        rem = _lengths(cfg, rng, cfg.tbs)
        bubbles.append(bubble(rem))
        queue = list(range(len(rem)))
        running: list = []
        while queue or running:
            while queue and len(running) < cap:
                running.append(queue.pop())
            adv = cfg.chunk
            dt = adv * cfg.tau_s
            busy_slot_s += len(running) * dt
            for r in running:
                done = min(adv, rem[r])
                tokens += int(done)
                rem[r] -= done
            running = [r for r in running if rem[r] > 0]
            t += dt
        t += cfg.train_s                                   # the cluster idles while training
    return {"mode": "synchronous", "time_s": t, "tokens": tokens,
            "tokens_per_s": tokens / t, "utilisation": busy_slot_s / (t * cap),
            "bubble_mean": float(np.mean(bubbles))}


def simulate_multiversion(cfg: Config, steps: int, plan_partition=None,
                          plan_supplement=None) -> dict:
    if plan_partition is None or plan_supplement is None:
        from . import dora
        plan_partition, plan_supplement = dora.plan_partition, dora.plan_supplement
    if cfg.rbs < cfg.tbs:
        raise ValueError("multi-version streaming over-provisions: rbs >= tbs")
    rng = np.random.default_rng(cfg.seed)
    cap = cfg.groups * cfg.slots
    versions = [0]                           # maintained versions, oldest first
    rem: dict = {0: []}                      # remaining tokens of running requests
    queue: dict = {0: []}                    # lengths of dispatched, not yet running
    owed = {0: cfg.rbs}                      # prompts the version's batch still needs
    groups = {0: cfg.groups}
    collected, trained, t, busy_slot_s, tokens = 0, 0, 0.0, 0.0, 0
    train_end = None
    max_lag = 0

    def rebalance():
        work = [len(rem[v]) + len(queue[v]) for v in versions]
        g = plan_partition(work, cfg.groups)
        for v, x in zip(versions, g):
            groups[v] = x
        active = [len(rem[v]) + len(queue[v]) for v in versions]  # queued hold slots too
        inject = plan_supplement([groups[v] for v in versions], active, cfg.slots,
                                 owed[versions[-1]])
        for v, k in zip(versions, inject):
            if k:
                queue[v].extend(_lengths(cfg, rng, k).tolist())
                if v == versions[-1]:
                    owed[v] -= k

    rebalance()
    while trained < steps:
        # admit queued requests into each version's slots
        for v in versions:
            room = groups[v] * cfg.slots - len(rem[v])
            while room > 0 and queue[v]:
                rem[v].append(queue[v].pop())
                room -= 1
        dt = cfg.chunk * cfg.tau_s
        running = sum(len(rem[v]) for v in versions)
        busy_slot_s += min(running, cap) * dt
        for v in versions:
            left = []
            for r in rem[v]:
                done = min(cfg.chunk, r)
                tokens += int(done)
                if r > done:
                    left.append(r - done)
                else:
                    collected += 1
            rem[v] = left
        t += dt
        if train_end is None and collected >= cfg.tbs:
            collected -= cfg.tbs
            train_end = t + cfg.train_s                    # training overlaps rollout
        if train_end is not None and t >= train_end:
            busy = [v for v in versions if rem[v] or queue[v]]
            if busy and versions[-1] + 1 - busy[0] > cfg.staleness - 1:
                continue                                   # window full: wait for stragglers
            trained += 1
            train_end = None
            new = versions[-1] + 1
            versions = [v for v in versions if rem[v] or queue[v]] + [new]
            rem[new], queue[new], owed[new] = [], [], cfg.rbs
            max_lag = max(max_lag, new - versions[0])
            rebalance()
        elif running == 0 and all(not queue[v] for v in versions):
            rebalance()                                    # idle slots: supplement again
    return {"mode": "multi-version", "time_s": t, "tokens": tokens,
            "tokens_per_s": tokens / t, "utilisation": busy_slot_s / (t * cap),
            "max_version_lag": max_lag}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    for f in dataclasses.fields(Config):
        ap.add_argument("--" + f.name.replace("_", "-"), type=type(f.default), default=f.default)
    ap.add_argument("--steps", type=int, default=6)
    a = ap.parse_args()
    cfg = Config(**{f.name: getattr(a, f.name) for f in dataclasses.fields(Config)})
    s = simulate_sync(cfg, a.steps)
    m = simulate_multiversion(cfg, a.steps)
    print(json.dumps({"config": dataclasses.asdict(cfg), "steps": a.steps, "synchronous": s,
                      "multi_version": m,
                      "speedup": s["time_s"] / m["time_s"]}, indent=1))


if __name__ == "__main__":
    main()
