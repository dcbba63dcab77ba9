"""Synthetic LM head and low-confidence remasking sampler (oracle, fp64).

TEST INFRASTRUCTURE ONLY (part of the oracle package).

Each denoising step of a diffusion LLM predicts every masked position of the
window at once (Sec. 3.1, the per-step factorisation over positions) and then
commits some of the predictions before the next step.  The paper does not
describe its sampler; the LLaDA-family backbones it runs on commit, per step,
the masked positions whose prediction is most confident and leave the rest
masked.  Readings (no trained weights exist here, so the head is random):

  * logits of a window row = RMSNorm(h) (unit gain, the layer's eps) times the
    LM head W [V, d] transposed; prediction = argmax over the vocabulary
    (smallest index on ties); confidence = the prediction's softmax
    probability, 1 / sum_v exp(l_v - l_max);
  * per sequence, with n masked positions among its first `used` rows and
    s >= 1 steps left, k = ceil(n / s) of them are committed: the k largest
    confidences, ties to the smaller position; committed tokens never change;
  * the next step's input row of a committed position is the embedding row
    of its token; an uncommitted position keeps its step-0 input row (the
    synthetic batches carry their planted structure there, in place of a
    single mask embedding); rows at or past `used` are zero.
"""
import numpy as np

from .layer import rms_norm

MASKED = -1


def lm_head_predict(h, W_lm, rms_eps):
    """(token [n] int64, confidence [n] float64) for rows h [n, d]."""
    a = rms_norm(np.asarray(h, np.float64), 1.0, rms_eps)
    logits = a @ np.asarray(W_lm, np.float64).T
    tok = np.argmax(logits, axis=1)                   # first maximum: smallest index
    lmax = logits[np.arange(len(tok)), tok]
    conf = 1.0 / np.sum(np.exp(logits - lmax[:, None]), axis=1)
    return tok.astype(np.int64), conf


def commit_count(n_masked, steps_left):
    """Positions committed this step: ceil(n / s) (all of them when s <= 1)."""
    if steps_left <= 1:
        return int(n_masked)
    return int(-(-int(n_masked) // int(steps_left)))


def remask_step(tokens, pred, conf, used, steps_left):
    """One sequence: commit the k most confident masked positions among the
    first `used`; returns the new token array (MASKED where still masked)."""
    tokens = np.array(tokens, np.int64, copy=True)
    masked = [i for i in range(int(used)) if tokens[i] == MASKED]
    k = commit_count(len(masked), steps_left)
    order = sorted(masked, key=lambda i: (-float(conf[i]), i))
    for i in order[:k]:
        tokens[i] = int(pred[i])
    return tokens


def next_inputs(tokens, x0, emb, used):
    """Next step's input rows of one sequence (see the module readings)."""
    x0 = np.asarray(x0, np.float64)
    out = np.zeros_like(x0)
    for i in range(int(used)):
        out[i] = np.asarray(emb[int(tokens[i])], np.float64) if tokens[i] != MASKED else x0[i]
    return out
