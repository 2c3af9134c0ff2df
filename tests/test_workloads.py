"""The seeded input generator (no method arithmetic): reproducible bytes and
the digest logged beside every benchmark line."""
import numpy as np

from paper_2507_05687_amd import workloads


def _inputs(**kw):
    w = workloads.scaled(workloads.WORKLOADS["fwdbwd_bf16"], prompts=2, group=4, seq_len=24,
                         hidden=64, vocab=300, **kw)
    return workloads.make_weight(w), workloads.make_hidden(w), workloads.make_batch(w)


def test_same_seed_same_bytes_and_digest():
    a, b = _inputs(seed=5), _inputs(seed=5)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert workloads.batch_digest(*a) == workloads.batch_digest(*b)


def test_digest_sees_seed_bytes_and_shape():
    W, h, b = _inputs(seed=5)
    d = workloads.batch_digest(W, h, b)
    assert workloads.batch_digest(*_inputs(seed=6)) != d
    W2 = W.copy()
    W2.flat[123] ^= 1
    assert workloads.batch_digest(W2, h, b) != d
    # same bytes in another shape or dtype are other inputs
    assert workloads.input_digest(W.reshape(-1)) != workloads.input_digest(W)
    assert workloads.input_digest(W.view(np.int16)) != workloads.input_digest(W)
