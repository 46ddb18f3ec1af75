"""Pins of the oracle's row operations against closed forms, invariants, special cases that
reduce to a library routine, and brute force on tiny inputs. No test retypes the oracle's
formula: each checks a property the mathematics fixes.
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---- SplitMix64 (counter-based draws of the guess provider) -------------------------------

def test_splitmix64_published_sequence():
    vals = [int(l, 16) for l in open(os.path.join(GOLDEN, "splitmix64_seed0.txt")) if l.startswith("0x")]
    gamma = 0x9E3779B97F4A7C15
    for k, v in enumerate(vals):
        assert oracle.mix((k * gamma) % (1 << 64)) == v


def test_workload_generator_uses_same_mixer():
    from paper_2403_00835_amd import workload
    # bits(seed, stream, i) = mix(mix(mix(seed) ^ stream) ^ i)
    for seed, stream, i in [(0, 0, 0), (3, 7, 11), (2**63 + 5, 1001, 123456789)]:
        key = oracle.mix(oracle.mix(seed) ^ stream)
        assert workload.bits(seed, stream, i) == oracle.mix(key ^ i)


# ---- bf16 rounding ------------------------------------------------------------------------

def test_bf16_matches_torch_rne_on_fp32_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 3,
                        rng.standard_normal(2000).astype(np.float32) * 1e-30,
                        rng.standard_normal(2000).astype(np.float32) * 1e30])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.bf16(float(v)) for v in x])
    np.testing.assert_array_equal(got, ref)


def test_bf16_ties_to_even_and_exact_values():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7: ties go to the even significand (1.0).
    assert oracle.bf16(1.0 + 2.0 ** -8) == 1.0
    # 1 + 3 * 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: the even one is 1 + 2^-6.
    assert oracle.bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    # a hair above the halfway point rounds up
    assert oracle.bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    for v in [0.0, -0.0, 1.0, -2.5, 0.015625, 3.0 * 2.0 ** 100, 2.0 ** -133]:
        assert oracle.bf16(v) == v
    assert math.isinf(oracle.bf16(1e39))


# ---- matrix product -----------------------------------------------------------------------

def test_linear_exact_on_small_integers():
    rng = np.random.default_rng(1)
    a = rng.integers(-8, 9, size=(5, 37)).astype(np.float64)
    W = rng.integers(-8, 9, size=(23, 37)).astype(np.float32)
    ref = a.astype(np.int64) @ W.astype(np.int64).T
    np.testing.assert_array_equal(oracle.linear(a, W), ref.astype(np.float64))


def test_linear_orientation_non_square():
    # y = a . W^T: row o of W produces output feature o.
    a = np.zeros((1, 4))
    a[0, 2] = 1.0
    W = np.arange(12, dtype=np.float32).reshape(3, 4)
    np.testing.assert_array_equal(oracle.linear(a, W)[0], W[:, 2])


# ---- RMSNorm ------------------------------------------------------------------------------

def test_rmsnorm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(96) * 7
    g = np.ones(96, dtype=np.float32)
    y = oracle.rmsnorm(x, g, 0.0)
    assert abs(np.sqrt(np.mean(y * y)) - 1.0) < 1e-14
    np.testing.assert_allclose(oracle.rmsnorm(x * 1e-3, g, 0.0), y, rtol=1e-13, atol=0)


def test_rmsnorm_epsilon_closed_form():
    # rms(out) = sqrt(ms / (ms + eps)) with gain 1.
    x = np.full(10, 1e-3)
    eps = 1e-6
    y = oracle.rmsnorm(x, np.ones(10, dtype=np.float32), eps)
    ms = 1e-6
    assert abs(np.sqrt(np.mean(y * y)) - math.sqrt(ms / (ms + eps))) < 1e-14


def test_rmsnorm_gain_is_elementwise():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(8)
    g = rng.standard_normal(8).astype(np.float32)
    y1 = oracle.rmsnorm(x, np.ones(8, dtype=np.float32), 1e-6)
    yg = oracle.rmsnorm(x, g, 1e-6)
    np.testing.assert_allclose(yg, y1 * g.astype(np.float64), rtol=1e-15)


# ---- RoPE ---------------------------------------------------------------------------------

def test_rope_identity_at_zero_and_pairing():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(16)
    np.testing.assert_array_equal(oracle.rope(x, 0), x)
    # rotate-half pairing: e_0 only mixes with e_{hd/2}
    e0 = np.zeros(16)
    e0[0] = 1.0
    r = oracle.rope(e0, 1)
    nz = set(np.nonzero(np.abs(r) > 1e-15)[0].tolist())
    assert nz == {0, 8}
    # frequency of pair 0 is 1 rad per position: (1, 0) -> (cos 1, sin 1)
    assert abs(r[0] - math.cos(1.0)) < 1e-15 and abs(r[8] - math.sin(1.0)) < 1e-15


def test_rope_last_pair_frequency():
    hd, base, t = 16, 10000.0, 37
    e = np.zeros(hd)
    e[hd // 2 - 1] = 1.0
    r = oracle.rope(e, t, base)
    ang = t * base ** (-(hd - 2) / hd)
    assert abs(r[hd // 2 - 1] - math.cos(ang)) < 1e-12
    assert abs(r[hd - 1] - math.sin(ang)) < 1e-12


def test_rope_is_a_rotation_group():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(64)
    np.testing.assert_allclose(oracle.rope(oracle.rope(x, 11), 29), oracle.rope(x, 40), atol=1e-12)
    assert abs(np.linalg.norm(oracle.rope(x, 123)) - np.linalg.norm(x)) < 1e-12


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal(32), rng.standard_normal(32)
    s1 = oracle.rope(q, 50) @ oracle.rope(k, 20)
    s2 = oracle.rope(q, 530) @ oracle.rope(k, 500)
    s3 = oracle.rope(q, 30) @ oracle.rope(k, 0)
    assert abs(s1 - s2) < 1e-10 and abs(s1 - s3) < 1e-10


# ---- attention ----------------------------------------------------------------------------

def test_attention_equal_keys_give_mean_of_values():
    rng = np.random.default_rng(7)
    q = rng.standard_normal(16)
    K = np.tile(rng.standard_normal(16), (9, 1))
    V = rng.standard_normal((9, 16))
    np.testing.assert_allclose(oracle.attention_row(q, K, V), V.mean(axis=0), rtol=1e-13, atol=1e-14)


def test_attention_single_key_returns_its_value():
    rng = np.random.default_rng(8)
    q, K, V = rng.standard_normal(16), rng.standard_normal((1, 16)), rng.standard_normal((1, 16))
    np.testing.assert_allclose(oracle.attention_row(q, K, V), V[0], rtol=1e-15)


def test_attention_two_keys_logistic_closed_form():
    # With scores s0, s1 the weight of key 0 is the logistic function of (s0 - s1) / sqrt(hd).
    from scipy.special import expit
    hd = 16
    q = np.zeros(hd)
    q[3] = 2.0
    K = np.zeros((2, hd))
    K[0, 3], K[1, 3] = 1.5, -0.25
    V = np.zeros((2, hd))
    V[0, 0], V[1, 1] = 1.0, 1.0
    out = oracle.attention_row(q, K, V)
    w0 = expit((2.0 * 1.5 - 2.0 * -0.25) / math.sqrt(hd))
    assert abs(out[0] - w0) < 1e-15 and abs(out[1] - (1 - w0)) < 1e-15


def test_attention_permutation_invariant_and_shift_invariant():
    rng = np.random.default_rng(9)
    q = rng.standard_normal(8)
    K, V = rng.standard_normal((11, 8)), rng.standard_normal((11, 8))
    base = oracle.attention_row(q, K, V)
    perm = rng.permutation(11)
    np.testing.assert_allclose(oracle.attention_row(q, K[perm], V[perm]), base, rtol=1e-12, atol=1e-14)
    # adding a vector orthogonal to q to every key changes no score
    c = rng.standard_normal(8)
    c -= (c @ q) / (q @ q) * q
    np.testing.assert_allclose(oracle.attention_row(q, K + c, V), base, rtol=1e-11, atol=1e-13)


def test_attention_huge_score_selects_value():
    rng = np.random.default_rng(10)
    q = np.zeros(8)
    q[0] = 1.0
    K = rng.standard_normal((5, 8)) * 0.01
    K[3, 0] = 1e4
    V = rng.standard_normal((5, 8))
    np.testing.assert_allclose(oracle.attention_row(q, K, V), V[3], rtol=1e-12)


# ---- SiLU and argmax ----------------------------------------------------------------------

def test_silu_identities():
    from scipy.special import expit
    assert oracle.silu(0.0) == 0.0
    for x in [-7.5, -1.0, -0.1, 0.3, 2.0, 11.0]:
        assert abs(oracle.silu(-x) - (oracle.silu(x) - x)) < 1e-14
        assert abs(oracle.silu(x) - x * expit(x)) < 1e-14
    assert abs(oracle.silu(40.0) - 40.0) < 1e-12


def test_argmax_matches_numpy_and_breaks_ties_low():
    rng = np.random.default_rng(11)
    for _ in range(50):
        x = rng.standard_normal(300)
        assert oracle.argmax(x) == int(np.argmax(x.astype(np.float32)))
    x = np.zeros(10)
    x[[4, 7]] = 3.0
    assert oracle.argmax(x) == 4
    # values equal after rounding to fp32 tie as well (the decision is taken in fp32)
    y = np.zeros(10)
    y[6], y[2] = 1.0 + 1e-12, 1.0
    assert oracle.argmax(y) == 2
    z = np.zeros(5)
    z[1] = np.nan
    assert oracle.argmax(z) == -1


# ---- acceptance scan ----------------------------------------------------------------------

@pytest.mark.parametrize("m", list(range(1, 13)))
def test_accept_len_exhaustive(m):
    # For every pattern of which block positions k >= 1 agree with the prediction of row k-1,
    # the accepted length is one plus the length of the leading run of agreements.
    for bits in range(1 << max(m - 1, 0)):
        pred = np.arange(100, 100 + m, dtype=np.int32)
        z = np.empty(m, dtype=np.int32)
        z[0] = 7
        run, broken = 1, False
        for k in range(1, m):
            ok = (bits >> (k - 1)) & 1
            z[k] = pred[k - 1] if ok else pred[k - 1] + 1000
            if ok and not broken:
                run += 1
            else:
                broken = True
        assert oracle.accept_len(z, pred) == run


def test_accept_len_m64_all_and_none():
    pred = np.arange(64, dtype=np.int32)
    z = np.concatenate([[5], pred[:63]]).astype(np.int32)
    assert oracle.accept_len(z, pred) == 64
    z2 = z.copy()
    z2[1] += 1
    assert oracle.accept_len(z2, pred) == 1
