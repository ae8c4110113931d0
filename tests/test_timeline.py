"""The timeline tool's summary of a trace buffer (CPU; synthetic stamps)."""
import numpy as np

from paper_2607_02043_amd import timeline as T


def test_summary_of_a_synthetic_trace():
    buf = np.zeros((T.MAX_ITEMS, T.SLOTS), dtype=np.uint64)
    # (start, end) in 10 ns ticks, kind, tiles or units, workgroup id
    t = 10 ** 9
    items = [(t, t + 2000, 1, 10, 5), (t, t + 1000, 1, 5, 6), (t + 1100, t + 1600, 2, 3, 6)]
    for i, (s, e, k, n, hw) in enumerate(items):
        buf[i, 0], buf[i, 3], buf[i, 4], buf[i, 7] = s, s + 100, e - 100, e
        buf[i, 8], buf[i, 9] = k * 1000000 + n, hw
        if k == 1:  # third-tile shader clocks
            buf[i, 11], buf[i, 12], buf[i, 14], buf[i, 15], buf[i, 13] = 10, 40, 50, 90, 150
    # a stale item of an earlier launch (10 ms before) is left out
    buf[7, 0], buf[7, 7], buf[7, 8], buf[7, 9] = t - 10 ** 6, t - 10 ** 6 + 500, 1000004, 9
    r = T.summarize(buf)
    assert r["items"] == 3 and abs(r["span_us"] - 20.0) < 1e-9
    c = r["kinds"]["chunk"]
    assert c["n"] == 2 and c["dur_max"] == 20.0 and c["units_max"] == 10
    assert abs(c["prologue"] - 1.0) < 1e-9 and abs(c["epilogue"] - 1.0) < 1e-9
    assert r["kinds"]["decode"]["n"] == 1
    assert r["chunk_tile_clocks"] == {"barrier": 30.0, "dma_issue": 10.0, "pv": 40.0, "scores_softmax": 60.0,
                                      "total": 140.0}
    w = r["workgroups"]
    assert w["n"] == 2 and w["busy_max"] == 20.0 and abs(w["idle_share"] - 0.125) < 1e-9
    assert r["longest"][0]["item"] == 0
