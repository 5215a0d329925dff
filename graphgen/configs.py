"""The five synthetic workloads (graph, features, walk parameters, weights).

=====  ==========================================================================
c1     R-MAT n=4096, 32768 undirected edges, X 4096x16 ~U(-1,1), walks 8 x 4 steps
c2     R-MAT n=2^17, avg degree 10 (incl. self-loop), X n x 64 ~N(0,1), walks 16 x 5
c3     SBM n=2^18, 512 communities of 64..1024 nodes, p_in=0.2, n Zipf(2.1) bridges,
       X n x 128 ~N(0,1), walks 16 x 5
c4     R-MAT n=2^21, avg degree 30, X n x 128 ~N(0,1), walks 16 x 5
c5     R-MAT n=2^22, avg degree 16, X n x 256 ~N(0,1), W1 256x128, W2 128x64
       Glorot-uniform; two GCN layers with ReLU between; walks 16 x 5
=====  ==========================================================================

"avg degree" counts the self-loop: an R-MAT graph with avg degree D has
m = n (D - 1) / 2 undirected edges and nnz = 2 m + n.

Generated arrays are cached as .npy files under ``$DUALGCN_INPUT_CACHE``
(default ``<repo>/_cache``; set it to ``off`` to disable).
"""
from dataclasses import dataclass, field
import os
import time

import numpy as np

from . import rmat, sbm, dense
from . import rng as _rng
from .csr import Graph

GEN_VERSION = 1


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str             # "rmat" | "sbm"
    n: int
    m: int                # undirected non-loop edges (R-MAT); 0 for SBM
    F: int
    x_dist: str           # "uniform" | "normal"
    walks: int
    steps: int
    layers: tuple = ()    # ((F_in, F_out), ...) for a GCN forward, else ()
    desc: str = ""

    @property
    def is_gcn(self):
        return bool(self.layers)


WORKLOADS = {
    "c1": Workload("c1", "rmat", 4096, 32768, 16, "uniform", 8, 4,
                   desc="R-MAT n=4096 m=32768, F=16, one SpMM"),
    "c2": Workload("c2", "rmat", 1 << 17, (1 << 17) * 9 // 2, 64, "normal", 16, 5,
                   desc="R-MAT n=2^17 avg deg 10, F=64, partition + SpMM"),
    "c3": Workload("c3", "sbm", 1 << 18, 0, 128, "normal", 16, 5,
                   desc="SBM n=2^18 512 communities p_in=0.2 + Zipf bridges, F=128"),
    "c4": Workload("c4", "rmat", 1 << 21, (1 << 21) * 29 // 2, 128, "normal", 16, 5,
                   desc="R-MAT n=2^21 avg deg 30, F=128, partition + SpMM"),
    "c5": Workload("c5", "rmat", 1 << 22, (1 << 22) * 15 // 2, 256, "normal", 16, 5,
                   layers=((256, 128), (128, 64)),
                   desc="2-layer GCN forward, R-MAT n=2^22 avg deg 16, 256->128->64"),
}


def _cache_dir():
    d = os.environ.get("DUALGCN_INPUT_CACHE")
    if d == "off":
        return None
    if not d:
        d = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "_cache")
    os.makedirs(d, exist_ok=True)
    return d


def _cached(tag, build):
    """build() -> dict of arrays; cached as <tag>.<key>.npy files."""
    d = _cache_dir()
    if d is not None:
        stamp = os.path.join(d, f"{tag}.v{GEN_VERSION}.done")
        if os.path.exists(stamp):
            with open(stamp) as fh:
                keys = fh.read().split()
            return {k: np.load(os.path.join(d, f"{tag}.{k}.npy"), mmap_mode=None) for k in keys}
    arrays = build()
    if d is not None:
        for k, a in arrays.items():
            np.save(os.path.join(d, f"{tag}.{k}.npy"), a)
        with open(os.path.join(d, f"{tag}.v{GEN_VERSION}.done"), "w") as fh:
            fh.write(" ".join(arrays))
    return arrays


def load_graph(name: str, seed: int = 0) -> Graph:
    w = WORKLOADS[name]

    def build():
        t0 = time.time()
        if w.kind == "rmat":
            g = rmat.graph(w.n, w.m, seed=seed)
        else:
            g = sbm.graph(w.n, seed=seed)
        sizes = np.array(g.meta.get("sizes", []), dtype=np.int64)
        return dict(rowptr=g.rowptr, col=g.col, val=g.val, sizes=sizes,
                    gen_seconds=np.array([time.time() - t0]))

    a = _cached(f"{name}.s{seed}.graph", build)
    meta = dict(name=name, kind=w.kind, n=w.n, seed=seed)
    if a["sizes"].size:
        meta["community_sizes"] = a["sizes"]
    g = Graph(n=w.n, rowptr=a["rowptr"], col=a["col"], val=a["val"], meta=meta)
    g.meta["max_degree"] = g.max_degree()
    return g


def load_features(name: str, seed: int = 0) -> np.ndarray:
    w = WORKLOADS[name]

    def build():
        if w.x_dist == "uniform":
            x = dense.features_uniform(w.n, w.F, seed)
        else:
            x = dense.features_normal(w.n, w.F, seed)
        return dict(x=x)

    return _cached(f"{name}.s{seed}.x", build)["x"]


def load_weights(name: str, seed: int = 0):
    w = WORKLOADS[name]
    out = []
    for i, (fi, fo) in enumerate(w.layers):
        out.append(dense.glorot(fi, fo, seed, _rng.W1 + i))
    return out
