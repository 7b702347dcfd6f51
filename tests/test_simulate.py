"""Control-plane simulator (CPU): its bubble statistic is the paper's, it
conserves work, it runs identically on the native planners and the oracle's,
keeps versions inside the staleness window, and shows the long-tail bubble
that multi-version streaming removes."""
import dataclasses

import numpy as np
import pytest

import workloads as wl
from oracle import plan as oplan
from paper_2604_26256_amd import simulate as sim

SMALL = sim.Config(groups=4, slots=16, rbs=96, tbs=64, staleness=3, tau_s=0.02, train_s=5.0,
                   chunk=64, median=512.0, sigma=1.2, lo=16, hi=16384, seed=3)


def test_bubble_matches_the_generator_statistic_and_the_paper_case():
    rng = np.random.default_rng(0)
    for _ in range(50):
        lens = rng.integers(1, 30000, int(rng.integers(1, 300)))
        assert sim.bubble(lens) == pytest.approx(wl.bubble(lens), abs=1e-12)
    # App. C.3: max response 30,720 tokens vs mean 3,536 gives 88.5%
    lens = [30720.0] + [(3536.0 * 100 - 30720.0) / 99] * 99     # max 30,720, mean 3,536
    assert sim.bubble(lens) == pytest.approx(0.885, abs=1e-3)


def test_sync_conserves_tokens():
    steps = 3
    r = sim.simulate_sync(SMALL, steps)
    rng = np.random.default_rng(SMALL.seed)
    want = sum(int(sim._lengths(SMALL, rng, SMALL.tbs).sum()) for _ in range(steps))
    assert r["tokens"] == want
    assert 0 < r["utilisation"] < 1


def test_multiversion_native_and_oracle_planners_agree():
    a = sim.simulate_multiversion(SMALL, 4)
    b = sim.simulate_multiversion(SMALL, 4, plan_partition=oplan.partition,
                                  plan_supplement=oplan.supplement)
    assert a == b


@pytest.mark.parametrize("K", [1, 2, 3])
def test_multiversion_respects_the_staleness_window(K):
    cfg = dataclasses.replace(SMALL, staleness=K)
    r = sim.simulate_multiversion(cfg, 5)
    assert r["max_version_lag"] <= K - 1


def test_long_tail_bubble_is_recovered():
    steps = 5
    s = sim.simulate_sync(SMALL, steps)
    m = sim.simulate_multiversion(SMALL, steps)
    assert s["bubble_mean"] > 0.5                  # long-tailed: most slot time waits
    assert m["utilisation"] > s["utilisation"]
    assert m["time_s"] < s["time_s"]               # steps finish sooner
