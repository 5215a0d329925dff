"""Feature matrices and Glorot-uniform weight matrices (float32, row-major)."""
import numpy as np

from . import rng as _rng


def features_uniform(n, f, seed=0, stream_id=_rng.FEATURES):
    gen = _rng.stream(seed, stream_id)
    return (gen.random((n, f), dtype=np.float32) * np.float32(2.0) - np.float32(1.0))


def features_normal(n, f, seed=0, stream_id=_rng.FEATURES):
    gen = _rng.stream(seed, stream_id)
    return gen.standard_normal((n, f), dtype=np.float32)


def glorot(fan_in, fan_out, seed=0, stream_id=_rng.W1):
    gen = _rng.stream(seed, stream_id)
    lim = np.sqrt(6.0 / (fan_in + fan_out))
    return gen.uniform(-lim, lim, (fan_in, fan_out)).astype(np.float32)


def labels(n, classes, seed=0, labeled_fraction=1.0, stream_id=_rng.LABELS):
    """int32 class ids in [0, classes), -1 on the rows left unlabeled (a uniform draw)."""
    gen = _rng.stream(seed, stream_id)
    y = gen.integers(0, classes, n, dtype=np.int64).astype(np.int32)
    if labeled_fraction < 1.0:
        y[gen.random(n) >= labeled_fraction] = -1
    return y
