"""The test helpers themselves (no GPU needed)."""
import numpy as np

from gpu_util import dev


def test_dev_accepts_a_reversed_length_one_axis():
    """Reversing an axis of length 1 leaves a negative stride that
    ascontiguousarray keeps (the array still counts as contiguous); the helper
    must still hand torch a positive-stride copy."""
    X = np.arange(3, dtype=np.int32).reshape(3, 1)
    t = dev(X[:, ::-1], device="cpu")
    assert t.tolist() == [[0], [1], [2]]
    t = dev(np.arange(6, dtype=np.int32).reshape(2, 3)[:, ::-1], device="cpu")
    assert t.tolist() == [[2, 1, 0], [5, 4, 3]]
