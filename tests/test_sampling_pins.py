"""Pins for the sampling oracle (temperature drafting and speculative-sampling
verification), on the CPU.  Each check is fixed by something outside the
oracle: the generator's published known answers, the exactness of the uniform
map, the distribution a Gumbel-max draw must follow, the greedy limit, and the
lossless property of the speculative-sampling rule (its first emitted token is
distributed as the target's distribution)."""
import json
import os

import numpy as np
import pytest

import oracle

so = oracle.sampling_oracle
HERE = os.path.dirname(__file__)


def _chi2_ok(counts, probs, n):
    """Pearson chi-square against probs at the 0.1% level (critical values for k-1 <= 9 dof)."""
    crit = {1: 10.83, 2: 13.82, 3: 16.27, 4: 18.47, 5: 20.52, 6: 22.46, 7: 24.32, 8: 26.12, 9: 27.88}
    exp = probs * n
    stat = float(np.sum((counts - exp) ** 2 / exp))
    return stat < crit[len(probs) - 1], stat


def test_philox_known_answers():
    kat = json.load(open(os.path.join(HERE, "golden", "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        ctr = np.array([[int(x, 16) for x in v["counter"]]], dtype=np.uint32)
        key = [int(x, 16) for x in v["key"]]
        got = so.philox4x32_10(ctr, key)[0]
        assert [int(x) for x in got] == [int(x, 16) for x in v["out"]]


def test_uniform_map_exact_and_open():
    x = np.array([0, 511, 512, 0xFFFFFFFF, 0x80000000, 0x12345678], dtype=np.uint32)
    u = so.uniform01(x)
    assert np.all(u > 0) and np.all(u < 1)
    k = u * (1 << 23) - 0.5
    assert np.array_equal(k, np.floor(k))                   # on the 2^-23 grid, offset by half a step
    assert u[0] == u[1] == 0.5 / (1 << 23) and u[2] == 1.5 / (1 << 23) and u[3] == 1 - 0.5 / (1 << 23)
    assert np.all(u.astype(np.float32).astype(np.float64) == u)  # every value exact in fp32


def test_streams_are_distinct_and_positional():
    a = so.words(7, so.STREAM_DRAFT, 3, 5, 16)
    assert np.array_equal(a, so.words(7, so.STREAM_DRAFT, 3, 5, 16))
    for other in (so.words(7, so.STREAM_BONUS, 3, 5, 16), so.words(7, so.STREAM_DRAFT, 4, 5, 16),
                  so.words(7, so.STREAM_DRAFT, 3, 6, 16), so.words(8, so.STREAM_DRAFT, 3, 5, 16)):
        assert not np.array_equal(a, other)
    # word v of a longer request is the same word (a draw depends on v, not on V)
    assert np.array_equal(so.words(7, so.STREAM_DRAFT, 3, 5, 40)[:16], a)


def test_gumbel_max_draws_follow_softmax():
    z = np.array([0.3, -1.0, 1.2, 0.0, -0.4, 0.9])
    T = 0.7
    n = 8000
    counts = np.zeros(len(z))
    for r in range(n):
        tok, _ = so.sample_draft(z, T, seed=11, row=r, depth=1)
        counts[tok] += 1
    ok, stat = _chi2_ok(counts, so.softmax_t(z, T), n)
    assert ok, stat


def test_small_temperature_is_greedy():
    rng = np.random.default_rng(0)
    for r in range(20):
        z = rng.normal(size=50)
        tok, _ = so.sample_draft(z, 1e-6, seed=3, row=r, depth=2)
        assert tok == int(np.argmax(z))


def test_equal_distributions_accept_every_draft():
    rng = np.random.default_rng(1)
    bs, B, V = 20, 16, 9
    lg = rng.normal(size=(bs, B, V))
    draft = lg[:, :B - 1].copy()
    tok = np.zeros((bs, B), np.int32)
    for b in range(bs):
        for j in range(1, B):
            tok[b, j], _ = so.sample_draft(draft[b, j - 1], 1.0, 5, b, j)
    res = so.verify_sample(tok, lg, draft, 1.0, seed=5)
    assert np.all(res["accept_len"] == B - 1)
    assert np.array_equal(res["out_tokens"][:, :B - 1], tok[:, 1:])
    assert np.all(res["accepted_nodes"] == np.arange(1, B))


def test_verification_is_lossless_at_depth_one():
    """The first emitted token (accepted draft or residual draw) is distributed
    as the target's p_1, whatever the draft distribution q_1 is."""
    rng = np.random.default_rng(2)
    V, B, n = 5, 16, 5000
    t1 = np.array([0.5, -0.3, 1.1, 0.0, -1.5])        # target row after the anchor
    d1 = np.array([1.4, 0.2, -0.6, 0.8, 0.0])          # drafter's logits at depth 1
    lg = np.broadcast_to(rng.normal(size=(1, B, V)), (n, B, V)).copy()
    lg[:, 0] = t1
    draft = np.broadcast_to(rng.normal(size=(1, B - 1, V)), (n, B - 1, V)).copy()
    draft[:, 0] = d1
    tok = np.zeros((n, B), np.int32)
    for b in range(n):
        for j in range(1, B):
            tok[b, j], _ = so.sample_draft(draft[b, j - 1], 1.0, 9, b, j)
    res = so.verify_sample(tok, lg, draft, 1.0, seed=9)
    first = res["out_tokens"][:, 0]
    counts = np.bincount(first, minlength=V).astype(float)
    ok, stat = _chi2_ok(counts, so.softmax_t(t1, 1.0), n)
    assert ok, stat
    # and the draft tokens themselves follow q_1
    ok, stat = _chi2_ok(np.bincount(tok[:, 1], minlength=V).astype(float), so.softmax_t(d1, 1.0), n)
    assert ok, stat
    assert np.all((res["accept_len"] >= 0) & (res["accept_len"] <= B - 1))


def test_rejection_probability_matches_closed_form():
    """P(accept at depth 1) = sum_x min(p(x), q(x)) (the speculative-sampling identity)."""
    V, B, n = 4, 16, 5000
    t1 = np.array([0.0, 1.0, -1.0, 0.5])
    d1 = np.array([1.5, -0.5, 0.0, 0.0])
    lg = np.zeros((n, B, V)); lg[:, 0] = t1
    draft = np.zeros((n, B - 1, V)); draft[:, 0] = d1
    tok = np.zeros((n, B), np.int32)
    for b in range(n):
        for j in range(1, B):
            tok[b, j], _ = so.sample_draft(draft[b, j - 1], 1.0, 4, b, j)
    res = so.verify_sample(tok, lg, draft, 1.0, seed=4)
    p, q = so.softmax_t(t1, 1.0), so.softmax_t(d1, 1.0)
    want = float(np.sum(np.minimum(p, q)))
    got = float(np.mean(res["accept_len"] >= 1))
    assert abs(got - want) < 4 * np.sqrt(want * (1 - want) / n), (got, want)
