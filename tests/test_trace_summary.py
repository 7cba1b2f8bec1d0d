"""The single-pass trace summary (paper_1904_00962_amd.trace) on synthetic
stamps: two rounds of four tiles whose phases are known."""

import numpy as np

from paper_1904_00962_amd import trace


def test_summary_of_known_stamps():
    # ticks of 10 ns: tile j of round r starts at r * 4000, reads for 1000 +
    # 100 j ticks, learns its scale at the round's last read end + 200 ticks,
    # writes for 300 ticks
    rows, et, el = [], [], []
    for r in range(2):
        base = r * 4000
        read_end = [base + 1000 + 100 * j for j in range(4)]
        scale = max(read_end) + 200
        for j in range(4):
            rows.append([base, read_end[j], scale, scale + 300])
            et.append(0 if j < 2 else 1)
            el.append(8192)
    info = dict(name="synthetic", algo="lamb", tensors=2, params=8 * 8192, g_dtype="bf16",
                groups=8, width=4, step_ms=[0.05], bytes_per_param=26)
    text = trace.summarize(np.asarray(rows, np.int64), np.asarray(et), np.asarray(el),
                           np.asarray([2, 2]), info)
    assert "for 8 tiles in 2 rounds" in text
    # read phases 10, 11, 12, 13 us: mean 11.5, max 13
    assert "| read (start to partial norms) | 11.50 | 11.50 |" in text
    # per round the reads end 3 us apart, and the scale comes 2 us later
    assert "finish reading 3.0 us apart" in text and "known 2.0 us after" in text
    # the kernel ends 5 us (2 + 3) after the last read
    assert "Kernel tail after the last read ends: 5.0 us." in text
