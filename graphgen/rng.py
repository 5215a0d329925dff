"""Independent numpy random streams, one per input array.

Every input draws from its own ``Generator(Philox(key=[seed, stream_id]))`` so
that changing the size of one array never shifts the values of another.
"""
import numpy as np

GRAPH = 1      # edge draws
RELABEL = 2    # vertex relabelling permutation
FEATURES = 3   # X
W1 = 4         # first weight matrix
W2 = 5         # second weight matrix
LABELS = 6     # node classes for the training loss
GRADS = 7      # upstream gradients fed to single backward steps


def stream(seed: int, stream_id: int) -> np.random.Generator:
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, stream_id], dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))
