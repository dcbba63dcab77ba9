"""Pins of the oracle's synthetic LM head and remasking sampler (CPU).

* confidence: the prediction's softmax probability (scipy's softmax) and, for
  two-token vocabularies, the logistic closed form; ties go to the smaller
  token index; the RMSNorm scale does not change the argmax;
* commit count: ceil(n / s), all at the last step, zero with nothing masked;
* remask: brute force over all k-subsets on tiny windows (the committed set
  maximises the summed confidence, smallest positions among equals);
  committed tokens never change; positions at or past `used` are untouched;
  after s steps with s steps left everything is committed;
* next inputs: embedding rows for committed positions, the step-0 row for
  masked ones, zero padding.
"""
import itertools

import numpy as np
from scipy.special import softmax

from oracle.sampler import MASKED, commit_count, lm_head_predict, next_inputs, remask_step


def test_confidence_and_argmax():
    rng = np.random.default_rng(0)
    h = rng.standard_normal((7, 16))
    W = rng.standard_normal((50, 16))
    tok, conf = lm_head_predict(h, W, 1e-5)
    a = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + 1e-5)
    p = softmax(a @ W.T, axis=1)
    np.testing.assert_array_equal(tok, np.argmax(p, axis=1))
    np.testing.assert_allclose(conf, p.max(axis=1), rtol=1e-12)
    # scaling a row does not move its argmax (RMSNorm removes the scale)
    tok2, conf2 = lm_head_predict(h * 7.5, W, 0.0)
    tok3, conf3 = lm_head_predict(h, W, 0.0)
    np.testing.assert_array_equal(tok2, tok3)
    np.testing.assert_allclose(conf2, conf3, rtol=1e-12)
    # two tokens: conf = logistic(|l0 - l1|)
    W2 = rng.standard_normal((2, 16))
    tok, conf = lm_head_predict(h, W2, 1e-5)
    l = a @ W2.T
    np.testing.assert_allclose(conf, 1.0 / (1.0 + np.exp(-np.abs(l[:, 0] - l[:, 1]))), rtol=1e-12)
    # exact tie: the smaller index wins, confidence 1/2
    Wt = np.stack([W2[0], W2[0]])
    tok, conf = lm_head_predict(h, Wt, 1e-5)
    assert np.all(tok == 0) and np.allclose(conf, 0.5)


def test_commit_count():
    assert [commit_count(10, s) for s in (1, 2, 3, 4, 10, 11)] == [10, 5, 4, 3, 1, 1]
    assert commit_count(0, 5) == 0 and commit_count(7, 0) == 7


def test_remask_brute_force():
    rng = np.random.default_rng(1)
    for trial in range(200):
        n = int(rng.integers(1, 8))
        used = int(rng.integers(0, n + 1))
        tokens = np.where(rng.random(n) < 0.4, rng.integers(0, 9, n), MASKED)
        pred = rng.integers(0, 9, n)
        conf = rng.choice([0.1, 0.2, 0.3], n)          # many ties
        steps = int(rng.integers(1, 4))
        new = remask_step(tokens, pred, conf, used, steps)
        masked = [i for i in range(used) if tokens[i] == MASKED]
        k = commit_count(len(masked), steps)
        best = max(itertools.combinations(masked, k),
                   key=lambda c: (round(sum(conf[i] for i in c), 12), [-i for i in sorted(c)]))
        expect = np.array(tokens, copy=True)
        for i in best:
            expect[i] = pred[i]
        np.testing.assert_array_equal(new, expect)
        # committed tokens stay; rows past `used` untouched
        keep = tokens != MASKED
        np.testing.assert_array_equal(new[keep], tokens[keep])
        np.testing.assert_array_equal(new[used:], tokens[used:])


def test_all_committed_after_the_last_step():
    rng = np.random.default_rng(2)
    n, used, S = 37, 33, 6
    tokens = np.full(n, MASKED)
    for s in range(S, 0, -1):
        pred = rng.integers(0, 100, n)
        conf = rng.random(n)
        before = int(np.sum(tokens[:used] == MASKED))
        tokens = remask_step(tokens, pred, conf, used, s)
        after = int(np.sum(tokens[:used] == MASKED))
        assert before - after == commit_count(before, s)
    assert np.all(tokens[:used] != MASKED) and np.all(tokens[used:] == MASKED)


def test_next_inputs():
    rng = np.random.default_rng(3)
    emb = rng.standard_normal((10, 4))
    x0 = rng.standard_normal((6, 4))
    tokens = np.array([3, MASKED, 9, MASKED, 1, 2])
    out = next_inputs(tokens, x0, emb, used=5)
    np.testing.assert_array_equal(out[0], emb[3])
    np.testing.assert_array_equal(out[1], x0[1])
    np.testing.assert_array_equal(out[2], emb[9])
    np.testing.assert_array_equal(out[4], emb[1])
    np.testing.assert_array_equal(out[5], 0.0)
