"""The library's trajectory counts (cllm_trace_count: host code, no device) against the oracle's
independent implementation, on hand-built trajectories and on trajectories the oracle records."""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import binding, workload
from paper_2403_00835_amd.configs import (BLOCK_SHRINK, BLOCK_SLIDE, GUESS_STREAM, GUESS_STREAM_REINJECT,
                                          GUESS_UNIFORM, TINY)
from tests.test_oracle_trajectory import CHANGED, STATIONARY, Y


def _same(traj, tokens, n, block_policy):
    o = oracle.trajectory_counts(traj, tokens, n, block_policy)
    c = binding.trace_count(traj, tokens, n, block_policy)
    for k in ("iterations", "stationary", "windows"):
        assert c[k] == o[k], k
    for k in ("fast_forward_mean", "stationary_per_window"):
        assert c[k] == pytest.approx(o[k]), k
    return c


def test_fixtures():
    assert _same(STATIONARY, Y, 4, BLOCK_SHRINK)["stationary"] == 1
    assert _same(CHANGED, Y, 4, BLOCK_SHRINK)["stationary"] == 0
    assert _same(STATIONARY[1:], Y, 4, BLOCK_SHRINK)["stationary"] == 1


def test_record_layout_roundtrip():
    raw = binding.dicts_to_records(STATIONARY)
    assert raw.shape == (3, binding.TRACE_STRIDE)
    back = binding.records_to_dicts(raw)
    for a, b in zip(back, STATIONARY):
        assert {k: a[k] for k in ("L", "e", "b0", "m", "a")} == {k: b[k] for k in ("L", "e", "b0", "m", "a")}
        np.testing.assert_array_equal(a["z"], b["z"])
        np.testing.assert_array_equal(a["pred"], b["pred"])


def test_inconsistent_records_rejected():
    bad = [dict(r) for r in STATIONARY]
    bad[2] = dict(bad[2], a=3)  # a > m
    with pytest.raises(binding.CllmError):
        binding.trace_count(bad, Y, 4, BLOCK_SHRINK)
    with pytest.raises(binding.CllmError):
        binding.trace_count(STATIONARY, Y[:3], 4, BLOCK_SHRINK)  # accepts past the tokens
    with pytest.raises(binding.CllmError):
        binding.trace_count(STATIONARY, Y, 4, 2)  # unknown policy


@pytest.fixture(scope="module")
def tiny():
    return oracle.load_model(TINY, seed=0)


@pytest.mark.parametrize("policy,block_policy,p", [(GUESS_UNIFORM, BLOCK_SHRINK, 0.0), (GUESS_STREAM, BLOCK_SHRINK, 0.2),
                                                   (GUESS_STREAM, BLOCK_SHRINK, 0.6), (GUESS_STREAM_REINJECT, BLOCK_SHRINK, 0.3),
                                                   (GUESS_STREAM, BLOCK_SLIDE, 0.3), (GUESS_STREAM_REINJECT, BLOCK_SLIDE, 0.5)])
def test_recorded_trajectories(tiny, policy, block_policy, p):
    prompt = workload.make_prompt(TINY, 16, seed=6)
    ar = tiny.ar_decode(prompt, 64)
    for n in (4, 8, 13):
        spec = oracle.GuessSpec(policy, block_policy, None if policy == GUESS_UNIFORM else ar, p=p, seed=n)
        out, st = tiny.jacobi_decode(prompt, n, 64, spec, trace=True)
        _same(st["trajectory"], out, n, block_policy)


def test_synthetic_trajectories_with_stationary_tokens():
    # Random trajectories built to hold stationary tokens: one block of n, the state is the
    # final tokens with random wrong ones; predictions right except at random positions.
    rng = np.random.default_rng(0)
    for _ in range(200):
        n = int(rng.integers(2, 12))
        y = rng.integers(0, 50, n + 1).astype(np.int32)
        traj, e = [], 0
        while e < n:
            m = n - e
            z = y[e:n].copy()
            wrong = rng.random(m) < 0.4
            wrong[0] = False
            z[wrong] = 99
            pred = y[e + 1:n + 1].copy()
            pred[rng.random(m) < 0.3] = 98
            r = {"L": 100 + e, "e": e, "b0": 0, "m": m, "z": z, "pred": pred}
            r["a"] = oracle.accept_len(z, pred)
            if not 1 <= r["a"] <= m:
                break
            traj.append(r)
            e += r["a"]
        _same(traj, y[:e], n, BLOCK_SHRINK)
