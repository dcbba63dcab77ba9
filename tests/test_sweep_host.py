"""Host-side checks of the detector-sensitivity sweep inputs and metrics (CPU).

* the confounder runs of the sweep workloads are EOS rows (the shared EOS
  vector plus the workload's noise), disjoint, inside the content and at
  least two positions before the planted boundary; workloads without them
  are unchanged;
* the sweep's summary metrics on hand-made boundaries.
"""
import numpy as np

from workloads import WORKLOADS, scaled
from workloads.generate import make_workload


def test_confounder_runs():
    w = scaled(WORKLOADS["sweep_small"], batch=12)
    _, b = make_workload(w, with_weights=False)
    d = w.shape.d_model
    S = w.seq_len_full
    n_runs = 0
    for s in range(w.batch):
        r2 = s * S + w.prefix_len
        p = int(b.planted[s])
        runs = b.dips[s]
        assert len(runs) <= w.dips[0]
        prev_end = -10
        for st0, ln in runs:
            assert 1 <= ln <= w.dips[1]
            assert st0 >= 1 and st0 + ln <= p - 2
            assert st0 > prev_end                       # disjoint, in order, not touching
            prev_end = st0 + ln
            rows = b.x[r2 + st0:r2 + st0 + ln] - b.eos[None, :]
            # EOS rows: the residual is the N(0, noise^2) noise (bf16-rounded)
            assert abs(np.std(rows) / w.noise_std - 1.0) < 0.1
            n_runs += 1
        # content rows outside the runs are N(0, 1), far from the EOS vector
        content = [i for i in range(p) if not any(a <= i < a + n for a, n in runs)]
        dist = np.linalg.norm(b.x[r2 + np.array(content)] - b.eos[None, :], axis=1)
        assert np.all(dist > 0.5 * np.linalg.norm(b.eos))
    assert n_runs >= w.batch                            # runs are actually planted
    for name in ("tiny_f32", "small_bf16_ragged", "small_bf16_stack"):
        _, b0 = make_workload(WORKLOADS[name], with_weights=False)
        assert all(len(r) == 0 for r in b0.dips)


def test_summary_metrics():
    from paper_2607_14557_amd.sweep import summarize
    planted = np.array([10, 20, 30, 40])
    win = np.array([100, 100, 100, 100])
    bnd = np.array([10, 15, 35, 100])
    keep = np.array([11, 16, 36, 100])
    m = summarize(bnd, keep, planted, win)
    assert m["exact"] == 0.25 and m["premature"] == 0.25 and m["late"] == 0.25 and m["none"] == 0.25
    assert abs(m["kept"] - (11 + 16 + 36 + 100) / 400) < 1e-12
    assert m["mean_abs_err"] == (0 + 5 + 5 + 60) / 4
