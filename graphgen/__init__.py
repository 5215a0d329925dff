"""Seeded synthetic inputs for the DualGCN aggregation path.

This package builds graphs, feature matrices and weight matrices only. It holds
none of the method's arithmetic (no walks, no scores, no products): both the
CPU oracle and the GPU path take its outputs as inputs.

* :mod:`graphgen.rmat`   -- R-MAT power-law edge lists
* :mod:`graphgen.sbm`    -- stochastic block model with power-law bridges
* :mod:`graphgen.csr`    -- symmetrise, add self-loops, CSR, D^-1/2 (A+I) D^-1/2
* :mod:`graphgen.small`  -- tiny named graphs (path, star, clique, cycle, ...)
* :mod:`graphgen.dense`  -- feature and weight matrices
* :mod:`graphgen.configs`-- the five benchmark workloads
"""
from .csr import Graph, from_undirected_edges, normalised_values
from .rng import stream
from . import rmat, sbm, small, dense, configs

__all__ = ["Graph", "from_undirected_edges", "normalised_values", "stream",
           "rmat", "sbm", "small", "dense", "configs"]
