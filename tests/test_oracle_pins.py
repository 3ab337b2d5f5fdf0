"""The fp64 oracle against facts that do not come from the oracle (CPU only)."""
import pytest

import oracle
import oracle_pins as P


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.attention_full)


def test_rejects_bad_arguments():
    import numpy as np
    q, k, v = P.rand_qkv(np.random.default_rng(0), 4, 3, 2, 8, 8)
    with pytest.raises((RuntimeError, ValueError)):
        oracle.attention_full(q, k, v, [0, 4], [0], [0])          # 3 % 2 != 0
    q, k, v = P.rand_qkv(np.random.default_rng(0), 4, 2, 2, 8, 8)
    with pytest.raises(ValueError):
        oracle.attention_full(q, k, v, [0, 4], [0], [3])          # runs off the cache
    with pytest.raises(RuntimeError):
        oracle.attention(q, k, v, [0, 4], [0], [0], rows=[4], heads=[0])


def test_threads_agree():
    import numpy as np
    q, k, v = P.rand_qkv(np.random.default_rng(1), 64, 4, 2, 16, 16)
    o1, l1 = oracle.attention_full(q, k, v, [0, 64], [0], [0], n_threads=1)
    o8, l8 = oracle.attention_full(q, k, v, [0, 64], [0], [0], n_threads=8)
    assert (o1 == o8).all() and (l1 == l8).all()
