"""The CPU oracle against its pins (no GPU)."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.fixture(scope="module")
def o():
    oracle.build()
    return oracle.get()


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(o, pin):
    pin(o)


def test_thread_count_changes_nothing(o):
    """The single-thread timing of the benchmark runs the same oracle: every
    output of a short chain is the same bytes on 1 thread and on all."""
    import numpy as np
    import dfssm_synth as S
    layers = [S.weights(K, N, 8, key=(90, i)) for i, (K, N) in enumerate([(256, 512), (512, 256), (256, 300)])]
    q0, s0 = o.quantize_act(S.activations(2, 256, key=(91,)))
    n = o.threads()
    try:
        o.set_threads(1)
        one, _ = o.chain(layers, q0, s0)
    finally:
        o.set_threads(n)
    many, _ = o.chain(layers, q0, s0)
    for a, b in zip(one, many):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
