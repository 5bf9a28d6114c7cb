"""The comparison rules of the GPU parity tests, pinned on the CPU: each
check must accept what the contract allows and reject each plausible
mistake of a GPU result (a swap outside the near-tie window, duplicates,
descending order, out-of-range positions, bad padding, a wrong count, a
score just outside the fp32 bound, a finite score past n_b)."""
from __future__ import annotations

import numpy as np
import pytest

from helpers import SCALE, SCORE_REL, TIE_REL, check_index_sets, check_scores


def _case(seed=0, n=64, k=8):
    """One unit: distinct fp64 scores, the oracle's top-k set ascending."""
    rng = np.random.default_rng(seed)
    S = rng.standard_normal((1, 1, n))
    top = np.sort(np.argsort(-S[0, 0], kind="stable")[:k])
    idx = np.full((1, 1, k), -1, np.int32)
    idx[0, 0, :k] = top
    nsel = np.array([[k]], np.int32)
    lens = np.array([n], np.int32)
    return S, idx, nsel, lens


def test_identical_sets_pass():
    S, idx, nsel, lens = _case()
    assert check_index_sets(idx.copy(), nsel.copy(), idx, nsel, S, lens) == 0


def _swap_last_for_next(S, idx, rel_gap):
    """The GPU set with the oracle's k-th entry swapped for the (k+1)-th,
    whose score is set rel_gap * |tau| below tau."""
    k = idx.shape[2]
    order = np.argsort(-S[0, 0], kind="stable")
    kth, nxt = order[k - 1], order[k]
    S = S.copy()
    tau = S[0, 0, kth]
    S[0, 0, nxt] = tau - rel_gap * abs(tau)
    g = idx.copy()
    g[0, 0, :k] = np.sort(np.where(g[0, 0, :k] == kth, nxt, g[0, 0, :k]))
    return S, g


def test_swap_inside_the_window_passes():
    S, idx, nsel, lens = _case()
    S2, g = _swap_last_for_next(S, idx, 0.5 * TIE_REL)
    assert check_index_sets(g, nsel.copy(), idx, nsel, S2, lens) == 1


def test_swap_outside_the_window_fails():
    S, idx, nsel, lens = _case()
    S2, g = _swap_last_for_next(S, idx, 3 * TIE_REL)
    with pytest.raises(AssertionError):
        check_index_sets(g, nsel.copy(), idx, nsel, S2, lens)


@pytest.mark.parametrize("mistake", ["duplicate", "descending", "past_n", "negative",
                                     "bad_padding", "wrong_count", "oracle_count"])
def test_malformed_gpu_sets_fail(mistake):
    n, k = 64, 8
    # a unit with a budget of k + 2 slots holding k selected positions (the
    # rest -1), as the GPU and the oracle write it for m = k
    S, idx, nsel, lens = _case(seed=3, n=n, k=k)
    gi, gn = np.full((1, 1, k + 2), -1, np.int32), nsel.copy()
    oi = gi.copy()
    gi[0, 0, :k] = idx[0, 0]
    oi[0, 0, :k] = idx[0, 0]
    lens_small = lens
    if mistake == "duplicate":
        gi[0, 0, 1] = gi[0, 0, 0]
    elif mistake == "descending":
        gi[0, 0, :k] = gi[0, 0, :k][::-1]
    elif mistake == "past_n":
        lens_small = np.array([gi[0, 0, k - 1]], np.int32)  # n_b at the last position
    elif mistake == "negative":
        gi[0, 0, 0] = -1
    elif mistake == "bad_padding":
        gi[0, 0, k] = 5
    elif mistake == "wrong_count":
        gn = gn + 1
    elif mistake == "oracle_count":
        gi[0, 0, :k] = idx[0, 0]
        gn = np.array([[k - 1]], np.int32)
    with pytest.raises(AssertionError):
        check_index_sets(gi, gn, oi, nsel, S, lens_small)


def test_short_context_selects_everything():
    """n_b <= k: the set is every position, then -1."""
    S = np.arange(5, dtype=np.float64).reshape(1, 1, 5)
    idx = np.array([[[0, 1, 2, 3, 4, -1, -1, -1]]], np.int32)
    nsel = np.array([[5]], np.int32)
    lens = np.array([5], np.int32)
    assert check_index_sets(idx.copy(), nsel.copy(), idx, nsel, S, lens) == 0
    bad = idx.copy()
    bad[0, 0, 5] = 0
    with pytest.raises(AssertionError):
        check_index_sets(bad, nsel.copy(), idx, nsel, S, lens)


def _bf16(x):
    """fp32 values -> bf16 bit patterns (round to nearest even)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _score_case():
    rng = np.random.default_rng(1)
    G, n = 4, 40
    q = _bf16(rng.standard_normal((1, G, 128)))
    K = _bf16(rng.standard_normal((1, 1, n + 5, 128)))
    qf = (q.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kf = (K.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    S = (qf[0] @ kf[0, 0].T).max(axis=0)[None, None] * SCALE   # [1][1][n+5]
    lens = np.array([n], np.int32)
    mag = (np.abs(qf[0]) @ np.abs(kf[0, 0, :n]).T).max(axis=0) * SCALE
    gpu = S.astype(np.float32).copy()
    gpu[0, 0, n:] = -np.inf
    return q, K, S, gpu, lens, mag, G, n


def test_scores_within_the_bound_pass():
    q, K, S, gpu, lens, mag, G, n = _score_case()
    check_scores(gpu, S, q, K, lens, G)
    # anything up to the bound itself is accepted
    edge = gpu.astype(np.float64)
    edge[0, 0, :n] = S[0, 0, :n] + 0.9 * SCORE_REL * mag
    check_scores(edge, S, q, K, lens, G)


def test_score_just_outside_the_bound_fails():
    q, K, S, gpu, lens, mag, G, n = _score_case()
    bad = gpu.astype(np.float64)
    bad[0, 0, 7] = S[0, 0, 7] + 1.5 * SCORE_REL * mag[7]
    with pytest.raises(AssertionError):
        check_scores(bad, S, q, K, lens, G)


def test_finite_score_past_the_context_fails():
    q, K, S, gpu, lens, mag, G, n = _score_case()
    bad = gpu.copy()
    bad[0, 0, n + 2] = 0.0
    with pytest.raises(AssertionError):
        check_scores(bad, S, q, K, lens, G)


def test_scores_of_the_wrong_query_head_fail():
    """max over the group replaced by one head's score: outside the bound."""
    q, K, S, gpu, lens, mag, G, n = _score_case()
    qf = (q.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kf = (K.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    one = (qf[0, 0] @ kf[0, 0].T)[None, None] * SCALE
    bad = gpu.copy()
    bad[0, 0, :n] = one[0, 0, :n]
    with pytest.raises(AssertionError):
        check_scores(bad, S, q, K, lens, G)
