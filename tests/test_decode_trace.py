"""The decode loop's synthetic inputs (datagen.decode_trace): deterministic,
one prompt per layer from its own seeds, one generated row and one query per
step."""
import numpy as np

import datagen


def test_decode_trace_shapes_and_determinism():
    wl = datagen.WORKLOADS["tiny"].with_(N=256, P=64, R=4)
    a = datagen.decode_trace(wl, layers=2, steps=5)
    b = datagen.decode_trace(wl, layers=2, steps=5)
    assert len(a) == 2
    for (ba, qa), (bb, qb) in zip(a, b):
        assert qa.shape == (5, wl.B, wl.Hq, wl.d) and qa.dtype == np.float32
        assert ba.sK.shape == (wl.B, wl.Hkv, 5, wl.d)
        np.testing.assert_array_equal(qa, qb)
        np.testing.assert_array_equal(ba.K, bb.K)
        np.testing.assert_array_equal(ba.sK, bb.sK)
    # the layers are different prompts, and the queries drift from step to step
    assert not np.array_equal(a[0][0].K, a[1][0].K)
    assert not np.array_equal(a[0][1][0], a[0][1][1])
