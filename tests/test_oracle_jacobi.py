"""Pins of the oracle's Jacobi decoding against what the paper fixes (Section 3.1):
the fixed point equals greedy AR output for any initial guess; every iteration fixes at
least one token, so a block of m tokens converges in at most m iterations (k <= n); the stop
test y(k) = y(k-1); plus the special cases of exact and fully corrupted guesses and the
closed-form mean acceptance of independently corrupted guesses.
"""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import (BLOCK_SHRINK, BLOCK_SLIDE, GUESS_STREAM, GUESS_STREAM_REINJECT,
                                          GUESS_UNIFORM, ModelConfig, TINY)


@pytest.fixture(scope="module")
def model():
    return oracle.load_model(TINY)


@pytest.fixture(scope="module")
def bf16_model():
    cfg = ModelConfig(n_layers=2, d_model=64, n_heads=4, head_dim=16, ffn_dim=172, vocab=256, dtype="bf16")
    return oracle.load_model(cfg)


def _check_trajectory(stats, n, max_new):
    sm, sa = stats["step_m"], stats["step_a"]
    assert (sa >= 1).all() and (sa <= sm).all()
    assert int(sa.sum()) == max_new == stats["tokens"]
    assert stats["steps"] <= max_new


@pytest.mark.parametrize("policy", [GUESS_UNIFORM, GUESS_STREAM, GUESS_STREAM_REINJECT])
@pytest.mark.parametrize("block_policy", [BLOCK_SHRINK, BLOCK_SLIDE])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_jacobi_equals_greedy_ar(model, policy, block_policy, seed):
    prompt = workload.make_prompt(TINY, 16, seed=seed + 10)
    ar = model.ar_decode(prompt, 40)
    for n in (1, 3, 8, 13):
        spec = oracle.GuessSpec(policy, block_policy, ar, p=0.35, seed=seed)
        out, st = model.jacobi_decode(prompt, n, 40, spec)
        np.testing.assert_array_equal(out, ar)
        _check_trajectory(st, n, 40)


def test_jacobi_equals_ar_with_bf16_rounding(bf16_model):
    prompt = workload.make_prompt(bf16_model.cfg, 12, seed=3)
    ar = bf16_model.ar_decode(prompt, 30)
    spec = oracle.GuessSpec(GUESS_STREAM_REINJECT, BLOCK_SHRINK, ar, p=0.3, seed=5)
    out, st = bf16_model.jacobi_decode(prompt, 8, 30, spec)
    np.testing.assert_array_equal(out, ar)


def test_block_converges_within_its_length(model):
    # Shrink policy: each block of m tokens takes at most m iterations (k <= n).
    prompt = workload.make_prompt(TINY, 16, seed=4)
    spec = oracle.GuessSpec(GUESS_UNIFORM, BLOCK_SHRINK, None, seed=7)
    n, max_new = 8, 37
    out, st = model.jacobi_decode(prompt, n, max_new, spec)
    sm, sa = st["step_m"], st["step_a"]
    # split the trajectory into blocks: a block starts when m equals its full size
    steps_in_block, first_m, blocks = 0, None, []
    left = 0
    for m, a in zip(sm, sa):
        if left == 0:
            first_m, steps_in_block, left = m, 0, m
        assert m == left  # shrink: the state is exactly the unfixed rest of the block
        steps_in_block += 1
        left -= a
        if left == 0:
            blocks.append((first_m, steps_in_block))
    assert left == 0 and len(blocks) == st["blocks"] == -(-max_new // n)
    for size, k in blocks:
        assert k <= size


def test_fixed_point_brute_force(model):
    # Each emitted token solves f(y_i, y_<i, x) = 0: a fresh full forward over (x, y_<i)
    # (no cache) has its argmax at y_i.
    prompt = workload.make_prompt(TINY, 16, seed=5)
    spec = oracle.GuessSpec(GUESS_UNIFORM, BLOCK_SHRINK, None, seed=1)
    out, _ = model.jacobi_decode(prompt, 8, 24, spec)
    seq = np.concatenate([prompt, out]).astype(np.int32)
    lg = model.forward_full(seq)
    for i in range(24):
        assert oracle.argmax(lg[len(prompt) - 1 + i]) == out[i]


def test_exact_guesses_converge_in_one_iteration_per_block(model):
    prompt = workload.make_prompt(TINY, 16, seed=6)
    ar = model.ar_decode(prompt, 35)
    for n in (4, 8, 16):
        spec = oracle.GuessSpec(GUESS_STREAM, BLOCK_SHRINK, ar, p=0.0, seed=0)
        out, st = model.jacobi_decode(prompt, n, 35, spec)
        np.testing.assert_array_equal(out, ar)
        assert st["steps"] == -(-35 // n)
        assert (st["step_a"] == st["step_m"]).all()


def test_fully_corrupted_reinjected_guesses_accept_one(model):
    prompt = workload.make_prompt(TINY, 16, seed=7)
    ar = model.ar_decode(prompt, 20)
    spec = oracle.GuessSpec(GUESS_STREAM_REINJECT, BLOCK_SLIDE, ar, p=1.0, seed=3)
    out, st = model.jacobi_decode(prompt, 8, 20, spec)
    np.testing.assert_array_equal(out, ar)
    assert st["steps"] == 20 and (st["step_a"] == 1).all()


def test_mean_acceptance_matches_closed_form(model):
    # Re-drawn guesses are right independently with probability 1-p, so at a full window
    # a = 1 + leading run, E[a] = 1 + (1-p)(1-(1-p)^(m-1))/p.
    prompt = workload.make_prompt(TINY, 16, seed=8)
    max_new, n, p = 600, 8, 0.3
    ar = model.ar_decode(prompt, max_new)
    spec = oracle.GuessSpec(GUESS_STREAM_REINJECT, BLOCK_SLIDE, ar, p=p, seed=11)
    out, st = model.jacobi_decode(prompt, n, max_new, spec)
    np.testing.assert_array_equal(out, ar)
    a = st["step_a"][st["step_m"] == n].astype(np.float64)
    expect = 1 + (1 - p) * (1 - (1 - p) ** (n - 1)) / p
    se = a.std(ddof=1) / np.sqrt(a.size)
    assert abs(a.mean() - expect) < 4 * se, (a.mean(), expect, se)


def test_guess_provider_corruption():
    V = 256
    stream = np.arange(300, dtype=np.int32) % V
    s0 = oracle.GuessSpec(GUESS_STREAM, 0, stream, p=0.0, seed=2)
    s1 = oracle.GuessSpec(GUESS_STREAM, 0, stream, p=1.0, seed=2)
    s3 = oracle.GuessSpec(GUESS_STREAM, 0, stream, p=0.3, seed=2)
    g0 = [oracle.guess(s0, 0, t, 0, V) for t in range(300)]
    g1 = [oracle.guess(s1, 0, t, 0, V) for t in range(300)]
    g3 = np.array([oracle.guess(s3, 0, t, d, V) for t in range(300) for d in range(20)])
    assert g0 == list(stream)
    assert all(a != b and 0 <= a < V for a, b in zip(g1, stream))
    frac = (g3 != np.repeat(stream, 20)).mean()
    assert abs(frac - 0.3) < 0.03


def test_uniform_guesses_cover_vocab():
    V = 64
    s = oracle.GuessSpec(GUESS_UNIFORM, 0, None, seed=9)
    g = np.array([oracle.guess(s, 1, t, d, V) for t in range(200) for d in range(32)])
    assert g.min() >= 0 and g.max() < V
    cnt = np.bincount(g, minlength=V)
    exp = g.size / V
    chi2 = ((cnt - exp) ** 2 / exp).sum()
    assert chi2 < 120  # 63 degrees of freedom; p ~ 1e-5 tail
