"""Pins of the decode exit-decision oracle (oracle/decode.py)."""

import math

import numpy as np
import pytest
import scipy.special

from oracle import Exit, EXIT_EMBEDDING, EXIT_MLP, EXIT_NORM
from oracle import decode as D


def rand_exit(rng, kind, h, V, I=0):
    e = Exit(kind=kind, w_out=rng.normal(0, 0.5, (V, h)))
    if kind != EXIT_EMBEDDING:
        e.gamma = rng.normal(1, 0.1, h)
    if kind == EXIT_MLP:
        e.gamma_mlp = rng.normal(1, 0.1, h)
        e.w_gate = rng.normal(0, 0.1, (I, h))
        e.w_up = rng.normal(0, 0.1, (I, h))
        e.w_down = rng.normal(0, 0.1, (h, I))
    return e


def test_uniform_logits():
    # W_out = 0: every logit is 0, so the confidence is 1/V and the tie goes to id 0.
    e = Exit(kind=EXIT_NORM, w_out=np.zeros((37, 8)), gamma=np.ones(8))
    r = D.exit_decide(e, np.random.default_rng(0).normal(size=(5, 8)), threshold=0.01)
    np.testing.assert_allclose(r["confidence"], 1 / 37, rtol=1e-15)
    assert (r["token"] == 0).all()
    assert r["exit"].all()                                     # 1/37 > 0.01
    assert not D.exit_decide(e, np.ones((2, 8)), 1 / 37)["exit"].any()   # strict "above"


def test_ties_go_to_the_lowest_id():
    rng = np.random.default_rng(1)
    w = rng.normal(0, 0.1, (50, 16))
    x = rng.normal(size=(3, 16))
    w[7] = w[31] = 10 * x.mean(axis=0)     # two identical, dominant rows
    e = Exit(kind=EXIT_EMBEDDING, w_out=w)
    r = D.exit_decide(e, x, 0.5)
    s = x @ w.T
    tied = [n for n in range(3) if s[n, 7] == s[n].max()]
    assert tied, "the fixture must make rows 7 and 31 the tied maximum"
    for n in tied:
        assert s[n, 31] == s[n, 7] and r["token"][n] == 7


def test_threshold_one_never_exits():
    # A dominant logit makes the fp64 probability round to exactly 1.0; "above 1" is still false.
    e = Exit(kind=EXIT_EMBEDDING, w_out=np.array([[100.0], [0.0], [-5.0]]))
    r = D.exit_decide(e, np.array([[1.0], [2.0]]), threshold=1.0)
    assert (r["confidence"] == 1.0).all() and not r["exit"].any()
    assert (r["token"] == 0).all()


@pytest.mark.parametrize("kind", [EXIT_EMBEDDING, EXIT_NORM, EXIT_MLP])
def test_matches_scipy_softmax_and_brute_force(kind):
    rng = np.random.default_rng(2 + kind)
    h, V, I = 12, 23, 20
    e = rand_exit(rng, kind, h, V, I)
    x = rng.normal(size=(6, h))
    r = D.exit_decide(e, x, 0.2)
    p = scipy.special.softmax(r["logits"], axis=1)
    np.testing.assert_allclose(r["confidence"], p.max(axis=1), rtol=1e-13)
    # pure-Python loops over the logits for the argmax (first maximum)
    for n in range(x.shape[0]):
        row = [float(v) for v in r["logits"][n]]
        best = 0
        for v in range(1, V):
            if row[v] > row[best]:
                best = v
        assert r["token"][n] == best
        denom = sum(math.exp(v - row[best]) for v in row)
        assert r["confidence"][n] == pytest.approx(1.0 / denom, rel=1e-13)
        assert r["exit"][n] == (r["confidence"][n] > 0.2)


def test_norm_exit_logits_are_the_training_forward():
    # The decision reads the same logits the training loss uses: with one
    # target per row, -log(conf) is the NLL of the argmax token.
    from oracle import token_nll
    rng = np.random.default_rng(5)
    e = rand_exit(rng, EXIT_NORM, 16, 40)
    x = rng.normal(size=(4, 16))
    r = D.exit_decide(e, x, 0.0)
    np.testing.assert_allclose(-np.log(r["confidence"]), token_nll(r["logits"], r["token"]), rtol=1e-12)
