"""Pins of the oracle's quantizer steps (ranges, AGP, stochastic rounding, planes, packing)
against what the paper and the mathematics fix."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import fqt, philox

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "quantizer_examples.json")))
F32 = np.float32
ALL_U24 = (np.arange(1 << 24, dtype=np.uint32) << np.uint32(8))   # every 24-bit uniform once


# ----------------------------------------------------------------------------- stochastic rounding

def test_sr_worked_example_exact_frequencies():
    """Section 3.2 / Prop. B.1 example: over every 24-bit uniform, the round-up frequency is
    exactly frac(v); the dequantized mean is exactly x and the variance (R/B)^2 f(1-f)."""
    g = GOLD["sr_b1"]
    x = np.array(g["x"], dtype=F32)
    R, Z, b = F32(g["R"]), F32(g["Z"]), g["bits"]
    B = (1 << b) - 1
    for xi, p_up, fl, var in zip(x, g["prob_round_up"], g["code_floor"], g["dequant_variance"]):
        q = fqt.sr_codes(np.full(ALL_U24.size, xi, dtype=F32), Z, R, b, ALL_U24).astype(np.int64)
        n_up = int((q > fl).sum())
        assert Fraction(n_up, 1 << 24) == Fraction(p_up)
        deq = q.astype(np.float64) * float(R) / B + float(Z)
        assert deq.mean() == pytest.approx(float(xi), abs=1e-12)
        assert deq.var() == pytest.approx(var, abs=1e-12)


def test_sr_integral_value_never_rounds_up():
    q = fqt.sr_codes(np.full(ALL_U24.size, 3.0, dtype=F32), F32(0.0), F32(15.0), 4, ALL_U24)
    assert np.all(q == 3)


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_sr_unbiased_and_variance_prop_b1(bits):
    """E[Q(x)] = x and Var = (R/B)^2 f(1-f) <= R^2/(4B^2) per element (Prop. B.1; Section 4.2)."""
    rng = np.random.default_rng(bits)
    x = rng.standard_normal(40).astype(F32) * F32(3)
    Z, R = x.min(), x.max() - x.min()
    B = (1 << bits) - 1
    q = fqt.sr_codes(x[None, :], Z, R, bits, ALL_U24[::64, None]).astype(np.float64)
    deq = q * float(R) / B + float(Z)
    v = np.minimum((x.astype(np.float32) - Z) * (F32(B) / R), F32(B)).astype(np.float64)
    f = v - np.floor(v)
    np.testing.assert_allclose(deq.mean(axis=0), float(Z) + v * float(R) / B, rtol=0, atol=2.0 ** -17 * float(R) / B)
    # 2^18 stratified uniforms, plus the three float32 roundings in v (relative 3 * 2^-24)
    np.testing.assert_allclose(deq.mean(axis=0), x, rtol=0,
                               atol=(2.0 ** -17 + 3 * 2.0 ** -24 * B) * float(R) / B)
    np.testing.assert_allclose(deq.var(axis=0), (float(R) / B) ** 2 * f * (1 - f),
                               rtol=0, atol=1e-5 * (float(R) / B) ** 2)
    assert np.all(deq.var(axis=0) <= float(R) ** 2 / (4 * B * B) + 1e-9)


def test_sr_range_zero_gives_code_zero():
    q = fqt.sr_codes(np.full(8, 2.5, dtype=F32), F32(2.5), F32(0.0), 4, np.arange(8, dtype=np.uint32))
    assert np.all(q == 0)


def test_psq_variance_bound_monte_carlo():
    """PSQ variance <= D/(4B^2) sum_i R_i^2 (Section 5.2), estimated with Philox draws."""
    rng = np.random.default_rng(5)
    N, D, b = 6, 32, 1
    g = (rng.standard_normal((N, D)) * np.exp(rng.standard_normal((N, 1)))).astype(F32)
    tot = np.zeros((N, D))
    sq = np.zeros((N, D))
    S = 3000
    st = fqt.group_stats(g[:, :, None, None])
    for seed in range(S):
        u = philox.uniform_words(np.arange(N * D), philox.STREAM_ELEM, seed, 0, 0).reshape(N, D)
        q = fqt.sr_codes(g, st.Z_s[:, None], st.R_s[:, None], b, u).astype(np.float64)
        deq = q * st.R_s[:, None].astype(np.float64) + st.Z_s[:, None]
        tot += deq
        sq += deq * deq
    mean = tot / S
    var = sq / S - mean ** 2
    assert var.sum() <= D / 4.0 * float((st.R_s.astype(np.float64) ** 2).sum()) * 1.02
    sd = np.sqrt(np.maximum(var, 1e-30))
    assert np.all(np.abs(mean - g) <= 6 * sd / np.sqrt(S) + 1e-6)


# ----------------------------------------------------------------------------- ranges

def test_group_stats_linear_and_conv():
    rng = np.random.default_rng(0)
    dy = rng.standard_normal((3, 5, 2, 2)).astype(F32)
    st = fqt.group_stats(dy)
    for n in range(3):
        assert st.Z_s[n] == dy[n].min() and st.R_s[n] == F32(dy[n].max() - dy[n].min())
    for d in range(5):
        assert st.Z_c[d] == dy[:, d].min() and st.R_c[d] == F32(dy[:, d].max() - dy[:, d].min())


def test_group_stats_negative_zero_is_canonical():
    dy = np.array([[-0.0, -0.0], [1.0, -0.0]], dtype=F32)[:, :, None, None]
    st = fqt.group_stats(dy)
    assert not np.signbit(st.Z_s[0]) and not np.signbit(st.R_s[0])


# ----------------------------------------------------------------------------- AGP

def _p(R, bits):
    R = np.array(R, dtype=F32)
    r = fqt.agp_select(R, np.zeros_like(R), bits, fqt.AGP_BERNOULLI, np.zeros(R.size, np.uint32))
    return r.prob.astype(np.float64), r


def test_agp_worked_example():
    g = GOLD["agp_b2"]
    p, _ = _p(g["R"], g["bits"])
    np.testing.assert_allclose(p, g["p"], rtol=1e-7)
    assert p.sum() == pytest.approx(len(g["R"]) / g["bits"])


def test_agp_waterfill_example():
    """The paper's formula would give p > 1 here; the capped probabilities keep sum = G/b."""
    g = GOLD["agp_waterfill_b4"]
    R = np.array(g["R"], dtype=np.float64)
    np.testing.assert_allclose(len(R) * R / (g["bits"] * R.sum()), g["p_uncapped_formula"])
    p, r = _p(g["R"], g["bits"])
    np.testing.assert_allclose(p, g["p"], rtol=1e-7)
    assert r.saturated == 1


def _pps_reference(R, b):
    """Independent characterization: the unique p = min(1, c R) with sum p = G/b (bisection)."""
    R = np.asarray(R, dtype=np.float64)
    G = R.size
    target = G / b
    if R.max() <= 0:
        return np.zeros(G)
    if (R > 0).sum() <= target:
        return (R > 0).astype(np.float64)
    lo, hi = 0.0, 1.0 / R[R > 0].min() * 2
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if np.minimum(1.0, mid * R).sum() < target:
            lo = mid
        else:
            hi = mid
    return np.minimum(1.0, hi * R)


@pytest.mark.parametrize("seed", range(12))
def test_agp_probabilities_match_pps_fixed_point(seed):
    rng = np.random.default_rng(seed)
    G = int(rng.integers(2, 400))
    b = int(rng.choice([1, 2, 3, 4, 8]))
    R = np.exp(rng.standard_normal(G) * float(rng.choice([0.5, 2.0, 4.0]))).astype(F32)
    R[rng.random(G) < 0.1] = 0
    p, r = _p(R, b)
    ref = _pps_reference(R, b)
    np.testing.assert_allclose(p, ref, rtol=2e-6, atol=1e-9)
    assert np.all(p <= 1.0)
    if R.max() > 0:
        assert p.sum() == pytest.approx(min(G / b, (R > 0).sum()), rel=1e-5)


def test_agp_masks_unbiased():
    """E[m_i / p_i] = 1 and E[#kept] = G/b over Philox seeds (Section 5.2: Q_g is unbiased)."""
    rng = np.random.default_rng(3)
    G, b = 24, 4
    R = np.exp(rng.standard_normal(G) * 1.5).astype(F32)
    S = 4000
    acc = np.zeros(G)
    cnt = []
    for seed in range(S):
        u = philox.uniform_words(np.arange(G), philox.STREAM_SAMPLE, seed, 0, 0)
        r = fqt.agp_select(R, np.zeros(G, F32), b, fqt.AGP_BERNOULLI, u)
        acc += r.keep / np.where(r.prob > 0, r.prob.astype(np.float64), 1.0)
        cnt.append(r.count)
    p = r.prob.astype(np.float64)
    sd = np.sqrt((1 - p) / p)
    assert np.all(np.abs(acc / S - 1) <= 5 * sd / np.sqrt(S) + 1e-12)
    assert np.mean(cnt) == pytest.approx(G / b, abs=5 * np.sqrt((p * (1 - p)).sum() / S))


def test_agp_b1_and_off_reduce_to_plain_quantizer():
    R = np.array([3.0, 0.0, 1.0, 7.0], dtype=F32)
    Z = np.array([-1.0, 2.0, -0.5, 0.25], dtype=F32)
    r1 = fqt.agp_select(R, Z, 1, fqt.AGP_BERNOULLI, np.zeros(4, np.uint32) + 0xFFFFFFFF)
    assert list(r1.keep) == [True, False, True, True]            # R = 0 has weight 0
    roff = fqt.agp_select(R, Z, 4, fqt.AGP_OFF, np.zeros(4, np.uint32))
    assert roff.keep.all() and np.all(roff.prob == 1)
    np.testing.assert_array_equal(roff.scale, (R / F32(15)).astype(F32))
    np.testing.assert_array_equal(roff.offset, Z)


def test_topk_and_separated_bernoulli_agree():
    """Appendix B.2's limit: when the large groups exactly fill the budget, p is in {0,1}."""
    R = np.array([0, 100, 0, 0, 100, 0, 0, 0], dtype=F32)
    for seed in range(20):
        u = philox.uniform_words(np.arange(8), philox.STREAM_CHANNEL, seed, 0, 0)
        rb = fqt.agp_select(R, np.zeros(8, F32), 4, fqt.AGP_BERNOULLI, u)
        rt = fqt.agp_select(R, np.zeros(8, F32), 4, fqt.AGP_TOPK, u)
        assert list(np.flatnonzero(rb.keep)) == [1, 4] == list(np.flatnonzero(rt.keep))


def test_topk_tie_break_lower_index():
    R = np.array([1, 2, 2, 2, 1, 0], dtype=F32)
    rt = fqt.agp_select(R, np.zeros(6, F32), 3, fqt.AGP_TOPK, np.zeros(6, np.uint32))
    assert list(np.flatnonzero(rt.keep)) == [1, 2]
    assert list(rt.kept_ids) == [1, 2, 0, 3, 4, 5] and rt.count == 2


def test_agp_scale_and_offset_fold_one_over_p():
    rng = np.random.default_rng(9)
    R = np.exp(rng.standard_normal(50)).astype(F32)
    Z = (-rng.random(50)).astype(F32)
    u = philox.uniform_words(np.arange(50), philox.STREAM_SAMPLE, 1, 0, 0)
    r = fqt.agp_select(R, Z, 4, fqt.AGP_BERNOULLI, u)
    k = r.keep
    np.testing.assert_allclose(r.scale[k].astype(np.float64) * 15 * r.prob[k], R[k], rtol=1e-6)
    np.testing.assert_allclose(r.offset[k].astype(np.float64) * r.prob[k], Z[k], rtol=1e-6)
    assert np.all(r.scale[~k] == 0) and np.all(r.offset[~k] == 0)
    assert sorted(r.kept_ids.tolist()) == list(range(50))
    assert list(r.kept_ids[:r.count]) == list(np.flatnonzero(k))


# ----------------------------------------------------------------------------- planes, packing, identities

def test_planes_worked_example():
    g = GOLD["planes"]
    pl = fqt.bit_planes(np.array(g["q"]), g["bits"])
    assert pl[0].astype(int).tolist() == g["plane0"] and pl[1].astype(int).tolist() == g["plane1"]


def test_planes_lossless_exhaustive():
    q = np.arange(256, dtype=np.uint8)
    pl = fqt.bit_planes(q, 8).astype(np.int64)
    assert np.array_equal(sum(pl[k] << k for k in range(8)), q.astype(np.int64))


def test_pack_lsb_first_and_tail():
    bits = np.zeros(70, dtype=bool)
    bits[[0, 2, 3, 64, 69]] = True
    w = fqt.pack_words(bits)
    assert w.tolist() == [0b1101, (1 << 0) | (1 << 5)]
    rng = np.random.default_rng(0)
    for L in (1, 63, 64, 65, 200):
        b = rng.random((3, L)) < 0.5
        assert np.array_equal(fqt.unpack_words(fqt.pack_words(b), L), b)


def _popc(v):
    return bin(int(v)).count("1")


def test_and_popcount_example_and_exhaustive():
    g = GOLD["and_popcount"]
    assert 2 * _popc(g["a"] & g["t"]) - _popc(g["a"]) == g["dot"]
    assert sum(a * s for a, s in zip(g["a_values"], g["t_signs"])) == g["dot"]
    L = 8
    for a in range(256):
        for t in range(256):
            dot = sum(((a >> j) & 1) * (2 * ((t >> j) & 1) - 1) for j in range(L))
            assert 2 * _popc(a & t) - _popc(a) == dot


def test_xnor_popcount_example_and_random():
    g = GOLD["xnor_popcount"]
    m = 0xFFFFFFFF
    assert (_popc(~(g["x1"] ^ g["x2"]) & m) << 1) - 32 == g["dot"]
    rng = np.random.default_rng(1)
    for _ in range(200):
        x1, x2 = (int(v) for v in rng.integers(0, 2 ** 32, 2))
        dot = sum((2 * ((x1 >> j) & 1) - 1) * (2 * ((x2 >> j) & 1) - 1) for j in range(32))
        assert (_popc(~(x1 ^ x2) & m) << 1) - 32 == dot


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_average_one_bit_product_identity(bits):
    """Appendix C: a b-bit product equals b packed 1-bit products merged by shifts
    (sum_k 2^k (2 popc(a_k & t) - popc(a_k)) == sum_j q_j s_j), ragged lengths included."""
    rng = np.random.default_rng(bits)
    for L in (1, 64, 130, 200):
        q = rng.integers(0, 1 << bits, L).astype(np.uint8)
        t = rng.random(L) < 0.5
        A = fqt.pack_words(fqt.bit_planes(q, bits))
        T = fqt.pack_words(t)
        acc = 0
        for k in range(bits):
            acc += (2 * sum(_popc(int(a) & int(tt)) for a, tt in zip(A[k], T))
                    - sum(_popc(int(a)) for a in A[k])) << k
        assert acc == int((q.astype(np.int64) * (2 * t.astype(np.int64) - 1)).sum())
