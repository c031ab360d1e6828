"""I/O-aware dynamic verification width (paper Sec. 4.2) through the C ABI,
on the CPU, against synthetic rounds whose costs follow the controller's
stated model: history transfer constant in q, verification compute and
draft time linear in q, committed tokens from the geometric acceptance
model.  The controller must pick the width that minimises round time per
committed token, found here by brute force."""
from __future__ import annotations

import os
import random

import pytest

from paper_2609_33184_amd import build_lib
from paper_2609_33184_amd import specstream as ss

WIDTHS = [1, 2, 3, 4, 5, 6, 7, 8]


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ss.lib_path()):
        build_lib.build(verbose=False)
    return ss.load()


class Env:
    """Round costs of a Cohort at width q (q candidate rows = q - 1 drafts)."""

    def __init__(self, transfer, compute0, compute1, draft1, correct, accept):
        self.transfer, self.c0, self.c1, self.d1, self.corr, self.a = transfer, compute0, compute1, draft1, correct, accept

    def parts(self, q):
        return self.transfer, self.c0 + self.c1 * q, self.d1 * (q - 1), self.corr

    def expected_committed(self, q):
        return sum(self.a ** i for i in range(q))

    def cost(self, q):
        t, c, d, k = self.parts(q)
        return (max(t, c) + d + k) / self.expected_committed(q)

    def best(self):
        return min(WIDTHS, key=self.cost)

    def sample_committed(self, q, rng):
        n = 1
        while n < q and rng.random() < self.a:
            n += 1
        return n


ENVS = [
    Env(0.038, 0.0004, 0.00002, 0.002, 0.0005, 0.8),    # transfer-bound, good drafts: wide
    Env(0.038, 0.0004, 0.00002, 0.020, 0.0005, 0.5),    # expensive drafts, weak acceptance: narrow
    Env(0.0004, 0.0003, 0.0003, 0.0002, 0.0001, 0.7),   # history in HBM, compute grows with q
    Env(0.010, 0.0004, 0.0020, 0.001, 0.0005, 0.9),     # compute overtakes transfer at wide q
]


@pytest.mark.parametrize("env", ENVS, ids=[f"env{i}" for i in range(len(ENVS))])
def test_controller_finds_the_best_width(lib, env):
    c = ss.ss_width_create(WIDTHS, switch_threshold=0.0, min_samples=1, decay=1.0)
    try:
        for _ in range(3 * len(WIDTHS)):
            q = ss.ss_width_select(c)
            ss.ss_width_observe(c, q, *env.parts(q), env.expected_committed(q))
        assert ss.ss_width_select(c) == env.best()
        for q in WIDTHS:
            assert ss.ss_width_estimate(c, q) == pytest.approx(env.cost(q), rel=1e-6)
    finally:
        ss.ss_width_destroy(c)


def test_sampling_phase_visits_every_width_in_order(lib):
    c = ss.ss_width_create(WIDTHS, min_samples=2)
    env = ENVS[0]
    seen = []
    try:
        for _ in range(2 * len(WIDTHS)):
            q = ss.ss_width_select(c)
            seen.append(q)
            ss.ss_width_observe(c, q, *env.parts(q), env.expected_committed(q))
        assert seen == [q for q in WIDTHS for _ in range(2)]
    finally:
        ss.ss_width_destroy(c)


def test_estimates_for_unmeasured_widths_follow_the_model(lib):
    """With widths 2, 3 and 4 measured (exact model costs), the estimates for
    the unmeasured widths reproduce the environment's costs: the linear fits
    and the fitted acceptance recover the generating parameters."""
    env = Env(0.038, 0.0004, 0.00002, 0.002, 0.0005, 0.8)
    c = ss.ss_width_create([2, 3, 4, 6, 8], min_samples=1)
    try:
        for q in (2, 3, 4):
            assert ss.ss_width_select(c) == q
            ss.ss_width_observe(c, q, *env.parts(q), env.expected_committed(q))
        for q in (6, 8):
            assert ss.ss_width_estimate(c, q) == pytest.approx(env.cost(q), rel=2e-3)
    finally:
        ss.ss_width_destroy(c)


def test_noisy_rounds_settle_near_the_optimum(lib):
    rng = random.Random(5)
    for env in ENVS:
        c = ss.ss_width_create(WIDTHS, switch_threshold=0.03, min_samples=3, decay=0.05)
        try:
            picks = []
            for _ in range(600):
                q = ss.ss_width_select(c)
                picks.append(q)
                ss.ss_width_observe(c, q, *env.parts(q), env.sample_committed(q, rng))
            final = picks[-100:]
            worst = max(env.cost(q) for q in set(final))
            assert worst <= env.cost(env.best()) * 1.08, (final[-5:], env.best())
        finally:
            ss.ss_width_destroy(c)


def test_switching_threshold_keeps_the_current_width(lib):
    """Width 4 is current; width 5's latest record becomes 1.5% cheaper per
    committed token: with a 5% threshold the controller stays, without a
    threshold it moves."""
    env = Env(0.038, 0.0004, 0.00002, 0.002, 0.0005, 0.8)
    t, cp, d, k = env.parts(4)
    u4 = env.expected_committed(4)
    for thr, moves in ((0.05, False), (0.0, True)):
        c = ss.ss_width_create([4, 5], switch_threshold=thr, min_samples=1, decay=1.0)
        try:
            assert ss.ss_width_select(c) == 4
            ss.ss_width_observe(c, 4, t, cp, d, k, u4)
            assert ss.ss_width_select(c) == 5
            ss.ss_width_observe(c, 5, t, cp, d, k, u4 * 0.5)      # width 5 looks poor at first
            assert ss.ss_width_select(c) == 4
            for _ in range(40):                                    # then is re-measured as slightly better
                ss.ss_width_observe(c, 5, t, cp, d, k, u4 * 1.015)
                ss.ss_width_observe(c, 4, t, cp, d, k, u4)
            assert ss.ss_width_estimate(c, 5) < ss.ss_width_estimate(c, 4) < ss.ss_width_estimate(c, 5) * 1.05
            assert (ss.ss_width_select(c) == 5) == moves
        finally:
            ss.ss_width_destroy(c)


def test_width_argument_errors(lib):
    for widths in ([], [0, 2], [2, 2], [3, 1], [9]):
        with pytest.raises(ss.SpecStreamError):
            ss.ss_width_create(widths)
    with pytest.raises(ss.SpecStreamError):
        ss.ss_width_create([2, 4], decay=0.0)
    c = ss.ss_width_create([2, 4])
    try:
        with pytest.raises(ss.SpecStreamError):
            ss.ss_width_observe(c, 3, 0.1, 0.1, 0.1, 0.1, 1.0)
        with pytest.raises(ss.SpecStreamError):
            ss.ss_width_observe(c, 2, -0.1, 0.1, 0.1, 0.1, 1.0)
        assert ss.ss_width_estimate(c, 3) == -1
    finally:
        ss.ss_width_destroy(c)
