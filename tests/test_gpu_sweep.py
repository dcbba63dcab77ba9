"""Detector-sensitivity sweep on the GPU (sweep_small, 32 sequences).

* every grid point (look-ahead 2..10; tau_jump 0.01..0.06 x gamma 0.2..1.0;
  detection layers 0..5): the GPU detector's boundaries equal the oracle's
  SNR criterion (exact rationals) on the same GPU counts, bit for bit;
* the synthetic batch shows the trends the paper reports: a look-ahead of 2
  cuts inside the content (its confounder runs), 3 and more do not, and the
  kept window grows with the look-ahead; a small tau_jump with a large gamma
  cuts early, a large tau_jump with a small gamma barely cuts; only the
  layer whose weights the EOS direction was planted for shows the boundary.
"""
from fractions import Fraction

import numpy as np
import pytest

from gpu_util import log
from oracle.detect import detect_batch
from workloads import WORKLOADS, scaled

pytestmark = pytest.mark.gpu


def test_sweep_small():
    from paper_2607_14557_amd import seer
    from paper_2607_14557_amd.sweep import run_sweep, markdown
    seer.load_library()
    w = scaled(WORKLOADS["sweep_small"], batch=32)
    log("sweep %s (B=%d)" % (w.name, w.batch))
    res = run_sweep(w, keep_counts=True)
    log(markdown(res))
    counts, batch = res["_counts"], res["_batch"]
    I = w.shape.d_ff
    for p in res["points"]:
        tau, gamma = Fraction(*p["tau"]), Fraction(*p["gamma"])
        ref, _ = detect_batch(counts[p["layer"]], batch.cu_seqlens, batch.win_off, batch.win_len, I,
                              tau, gamma, p["lookahead"])
        assert np.array_equal(np.asarray(p["boundary"]), ref), p
    la = {r["lookahead"]: r for r in res["lookahead"]}
    assert la[2]["premature"] >= 0.3
    assert all(la[k]["premature"] == 0.0 for k in la if k >= 3)
    kept = [la[k]["kept"] for k in sorted(la) if k >= 3]
    assert kept == sorted(kept) and kept[-1] > kept[0] + 0.1
    tg = {(r["tau_jump"], r["gamma"]): r for r in res["tau_gamma"]}
    assert tg[("1/100", "1")]["premature"] >= 0.5
    assert tg[("3/50", "1/5")]["premature"] == 0.0 and tg[("3/50", "1/5")]["kept"] >= 0.85
    lay = {r["layer"]: r for r in res["layer"]}
    assert lay[w.l_det]["exact"] >= 0.5
    assert all(lay[l]["exact"] <= 0.1 for l in lay if l != w.l_det)
