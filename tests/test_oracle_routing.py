"""Pins of the oracle's router logits and softmax/top-k selection (Sec. 3.3 router-logit
computation; Sec. 4.1 softmax routing with top-k).

Independent references: numpy's float64 matmul on torch-decoded bf16 values, scipy's
softmax, and brute-force sorting in Python.
"""
import numpy as np
import pytest
import torch
from scipy.special import softmax


def bf16_bits(a):
    return torch.as_tensor(a, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_value(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()


@pytest.mark.parametrize("T,H,E", [(1, 256, 8), (3, 384, 17), (8, 2048, 128)])
@pytest.mark.parametrize("with_bias", [False, True])
def test_router_logits_match_numpy(orc, T, H, E, with_bias):
    rng = np.random.default_rng(T * 1000 + E)
    x = bf16_bits(rng.standard_normal((T, H)))
    rw = bf16_bits(rng.standard_normal((E, H)) * 0.02)
    bias = rng.standard_normal(E).astype(np.float32) if with_bias else None
    got = orc.router_logits(x, rw, bias)
    ref = bf16_value(x) @ bf16_value(rw).T
    if with_bias:
        ref = ref + bias.astype(np.float64)[None, :]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def brute_topk(l, k):
    order = sorted(range(len(l)), key=lambda e: (-l[e], e))
    return order[:k]


@pytest.mark.parametrize("renorm", [True, False])
def test_select_matches_brute_force_and_scipy(orc, renorm):
    rng = np.random.default_rng(1 + renorm)
    for trial in range(40):
        T, E = int(rng.integers(1, 6)), int(rng.integers(2, 40))
        k = int(rng.integers(1, E + 1))
        logits = rng.standard_normal((T, E))
        if trial % 3 == 0:   # exact ties, to exercise the lower-index rule
            logits = np.round(logits * 2) / 2
        ids, w = orc.select(logits, k, renorm)
        for t in range(T):
            assert ids[t].tolist() == brute_topk(logits[t].tolist(), k)
            p = softmax(logits[t])
            sel = p[ids[t]]
            ref = sel / sel.sum() if renorm else sel
            np.testing.assert_allclose(w[t], ref, rtol=1e-13, atol=1e-15)
            if renorm:
                assert abs(w[t].sum() - 1.0) < 1e-13
            else:
                assert w[t].sum() <= 1.0 + 1e-13


def test_select_all_experts_uniform(orc):
    for E in (1, 4, 8, 33):
        ids, w = orc.select(np.zeros((2, E)), E, True)
        assert ids.tolist() == [list(range(E))] * 2
        np.testing.assert_allclose(w, 1.0 / E, rtol=1e-15)
        ids, w = orc.select(np.zeros((1, E)), E, False)
        np.testing.assert_allclose(w, 1.0 / E, rtol=1e-15)


def test_select_permutation_equivariance(orc):
    rng = np.random.default_rng(9)
    E, k = 32, 5
    logits = rng.standard_normal((4, E))
    perm = rng.permutation(E)
    ids, w = orc.select(logits, k, True)
    ids_p, w_p = orc.select(logits[:, perm], k, True)
    inv = np.argsort(perm)
    # expert e of the original appears as expert inv[e] after permutation
    assert np.array_equal(inv[ids], ids_p)
    np.testing.assert_allclose(w, w_p, rtol=1e-15)


def test_weight_ratios_follow_logit_gaps(orc):
    rng = np.random.default_rng(4)
    logits = rng.standard_normal((3, 64)) * 3
    for renorm in (True, False):
        ids, w = orc.select(logits, 8, renorm)
        for t in range(3):
            for j in range(1, 8):
                r = w[t, 0] / w[t, j]
                assert abs(r / np.exp(logits[t, ids[t, 0]] - logits[t, ids[t, j]]) - 1) < 1e-12


# ---- sigmoid routing with an expert-selection bias and a routed scaling factor ----
# Independent references: scipy's logistic function (expit), brute-force sorting, and
# relations that hold whatever the implementation.
from scipy.special import expit


def test_sigmoid_select_matches_brute_force_and_expit(orc):
    rng = np.random.default_rng(21)
    for trial in range(40):
        T, E = int(rng.integers(1, 6)), int(rng.integers(2, 40))
        k = int(rng.integers(1, E + 1))
        logits = rng.standard_normal((T, E))
        bias = (rng.standard_normal(E) * 0.3).astype(np.float32)
        if trial % 3 == 0:   # exact score ties: equal logits and equal biases
            logits = np.round(logits)
            bias = np.round(bias * 2).astype(np.float32) / 2
        scale = float(rng.choice([1.0, 2.5]))
        ids, w = orc.select_sigmoid(logits, k, bias, scale)
        for t in range(T):
            a = expit(logits[t])
            score = a + bias.astype(np.float64)
            assert ids[t].tolist() == brute_topk(score.tolist(), k)
            sel = a[ids[t]]
            np.testing.assert_allclose(w[t], scale * sel / sel.sum(), rtol=1e-13)
            assert abs(w[t].sum() - scale) < 1e-12


def test_sigmoid_bias_steers_selection_not_weights(orc):
    # a large bias on experts 3 and 7 forces them in; their weights still come from the
    # unbiased affinities
    rng = np.random.default_rng(22)
    logits = rng.standard_normal((2, 16))
    bias = np.zeros(16, np.float32)
    bias[[3, 7]] = 10.0
    ids, w = orc.select_sigmoid(logits, 4, bias, 2.5)
    for t in range(2):
        assert set(ids[t][:2].tolist()) == {3, 7}
        a = expit(logits[t])
        np.testing.assert_allclose(w[t], 2.5 * a[ids[t]] / a[ids[t]].sum(), rtol=1e-13)


def test_sigmoid_without_bias_selects_like_softmax(orc):
    # the logistic function is increasing, so with no bias it ranks experts as the logits do
    rng = np.random.default_rng(23)
    logits = rng.standard_normal((5, 64)) * 2
    ids_s, _ = orc.select_sigmoid(logits, 8, None, 2.5)
    ids_m, _ = orc.select(logits, 8, True)
    assert np.array_equal(ids_s, ids_m)


def test_sigmoid_equal_logits_gives_equal_scaled_weights(orc):
    bias = np.arange(12, dtype=np.float32) * 0.01      # ranks experts 11, 10, 9, ...
    ids, w = orc.select_sigmoid(np.full((1, 12), 0.3), 5, bias, 2.5)
    assert ids[0].tolist() == [11, 10, 9, 8, 7]
    np.testing.assert_allclose(w[0], 0.5, rtol=1e-15)
