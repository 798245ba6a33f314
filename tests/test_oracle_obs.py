"""Pins of the OBS calibration oracle (channel scores, column swap).

Paper: "CLQ" (arXiv 2509.24416), Sec. 3.3 (Orthogonal-Based Smoothing: batch
mean, per-channel outlier metric, top half of the channels to the left) and
Sec. 4.2 (the five outlier metrics of the ablation).  Each test checks the
oracle against a hand-worked value, an independent library routine, a
closed form, or an invariant of the definition.
"""
import numpy as np
import pytest

from oracle import obs
import workloads


# ---- batch mean ----------------------------------------------------------------

def test_batch_mean_identical_samples_is_exact():
    x = workloads.activations(32, 64, seed=11)          # fp16
    X = np.stack([x] * 24)                                # B = 24: B * x exact in fp32
    assert np.array_equal(obs.batch_mean(X), x.astype(np.float32))


def test_batch_mean_hand_values():
    X = np.array([1.0, 2.0, 4.0], np.float16).reshape(3, 1, 1)
    assert obs.batch_mean(X)[0, 0] == np.float32(7.0) / np.float32(3.0)
    # the samples are added in batch order before one division
    X = np.array([2.0 ** 11, 1.0, 1.0, 1.0], np.float16).reshape(4, 1, 1)
    assert obs.batch_mean(X)[0, 0] == np.float32(2051.0 / 4.0)


# ---- pairwise summation ----------------------------------------------------------

def test_pairwise_order_hand_example():
    # tree: (1 + 2^24) + (1 + 0) = 2^24 + 1 -> 2^24 (ties to even);
    # a left-to-right sum would give 2^24 + 2
    v = np.array([1.0, 1.0, 2.0 ** 24, 0.0], np.float32)
    assert obs.pairwise_sum(v) == np.float32(2.0 ** 24)
    # three values are padded to four: (a + c) + (b + 0)
    v = np.array([2.0 ** 24, 1.0, 1.0], np.float32)
    assert obs.pairwise_sum(v) == np.float32(2.0 ** 24 + 1) + np.float32(1.0)


@pytest.mark.parametrize("n", [1, 2, 3, 7, 64, 1000])
def test_pairwise_exact_on_small_integers(n):
    v = np.arange(n, dtype=np.float32)
    assert obs.pairwise_sum(v) == np.float32(n * (n - 1) // 2)


# ---- the five metrics -------------------------------------------------------------

def test_absmax_and_range_hand():
    S = np.array([[1.0, -3.0], [-2.0, 0.5], [0.25, 2.0]], np.float32)
    assert np.array_equal(obs.channel_scores(S, "absmax"), np.array([2.0, 3.0], np.float32))
    assert np.array_equal(obs.channel_scores(S, "range"), np.array([3.0, 5.0], np.float32))


def test_par_closed_forms():
    N = 256
    S = np.zeros((N, 3), np.float32)
    S[:, 0] = -0.75              # constant magnitude: peak = average
    S[17, 1] = 5.0               # one non-zero: peak / (5 / N) = N
    par = obs.channel_scores(S, "par")
    assert par[0] == 1.0 and par[1] == np.float32(N) and par[2] == 0.0


def test_topk_mean_closed_form():
    N = 1000                     # k = 10: the top ten of 0..999
    S = np.arange(N, dtype=np.float32)[:, None] - np.float32(500.0)   # |.| peaks at 500
    v = np.abs(np.arange(N) - 500.0)
    k = obs.topk_count(N)
    assert k == 10
    assert obs.channel_scores(S, "topk_mean")[0] == np.float32(np.sort(v)[::-1][:k].mean())


@pytest.mark.parametrize("N", [1, 2, 99, 1000, 4096, 21600])
def test_topk_count_is_one_percent(N):
    k = obs.topk_count(N)
    assert k >= 1 and abs(k - N / 100) <= 0.5 + 1e-9 or (N < 50 and k == 1)


@pytest.mark.parametrize("N", [1000, 4096, 777])
def test_percentile_against_numpy_order_statistics(N):
    rng = np.random.default_rng(N)
    S = rng.standard_normal((N, 4)).astype(np.float32)
    got = obs.channel_scores(S, "percentile")
    p1 = np.percentile(S, 1, axis=0, method="lower")
    p99 = np.percentile(S, 99, axis=0, method="higher")
    assert np.array_equal(got, (p99 - p1).astype(np.float32))


def test_percentile_on_ranks():
    N = 1000
    S = np.arange(N, dtype=np.float32)[:, None]
    lo, hi = obs.percentile_ranks(N)
    assert (lo, hi) == (9, 990)
    assert obs.channel_scores(S, "percentile")[0] == np.float32(hi - lo)


# ---- the column swap ---------------------------------------------------------------

def test_permutation_hand_example():
    s = obs.permutation(np.array([0.5, 3.0, 1.0, 3.0], np.float32))
    assert s.tolist() == [1, 3, 0, 2]


def test_permutation_all_ties_is_identity():
    assert obs.permutation(np.ones(64, np.float32)).tolist() == list(range(64))


@pytest.mark.parametrize("D", [2, 64, 1152])
def test_permutation_properties(D):
    rng = np.random.default_rng(D)
    sc = rng.integers(0, 20, size=D).astype(np.float32)   # many ties
    s = obs.permutation(sc)
    assert sorted(s.tolist()) == list(range(D))
    left, right = s[:D // 2], s[D // 2:]
    assert np.all(np.diff(left) > 0) and np.all(np.diff(right) > 0)
    # brute force: channel d is in the top half iff fewer than D/2 channels
    # beat it (higher score, or equal score and lower index)
    for d in range(D):
        beaten_by = np.sum((sc > sc[d]) | ((sc == sc[d]) & (np.arange(D) < d)))
        assert (d in set(left.tolist())) == (beaten_by < D // 2)


@pytest.mark.parametrize("metric", obs.METRICS)
def test_power_of_two_scaling(metric):
    X = workloads.calibration(3, 128, 64, seed=7)
    S = obs.batch_mean(X)
    a = obs.channel_scores(S, metric)
    b = obs.channel_scores(S * np.float32(4.0), metric)
    if metric == "par":
        assert np.array_equal(a, b)
    else:
        assert np.array_equal(b, a * np.float32(4.0))
    assert np.array_equal(obs.permutation(a), obs.permutation(b))


def test_planted_outliers_go_left():
    # the swap gathers the outlier channels into the left half (the point
    # of S in G = S.H)
    D = 1152
    X = workloads.calibration(4, 256, D, seed=9)
    ch = workloads.calibration_outliers(D, seed=9)
    _, _, s = obs.obs(X, "absmax")
    assert set(ch.tolist()) <= set(s[:D // 2].tolist())
