"""Host-side logic of bench.py (no GPU)."""
import numpy as np

import bench


def test_stage_bench_output_gradient_alternates_sign():
    """The stage bench feeds a fixed synthetic output gradient; applied every
    step with the same sign, momentum SGD drives the weights without bound, so
    consecutive steps must see g and -g in turn."""
    g1 = np.arange(6, dtype=np.float32).reshape(2, 3)
    g2 = -2.0 * g1
    t = dict(db1=g1, db2=g2, nb1=-g1, nb2=-g2, flip=0)
    seen = [bench.output_grad(t) for _ in range(4)]
    assert seen[0][0] is g1 and seen[0][1] is g2
    assert seen[2][0] is g1 and seen[2][1] is g2
    for d1, d2 in (seen[1], seen[3]):
        assert np.array_equal(d1, -g1) and np.array_equal(d2, -g2)
    # over a pair of steps the gradients cancel exactly
    assert np.array_equal(seen[0][0] + seen[1][0], np.zeros_like(g1))

