"""Seeded multi-tenant serving workload: many registered models, open-loop arrivals.

Model i is workload 2 + (i mod 3) (24 x 4096 bf16 MLP, ResNet-50 shape, BERT-base shape),
weight seed 1000 + i, following the paper's round-robin distribution of models across
functions. Requests arrive as a Poisson process (exponential inter-arrival times, seed
42); each picks a popularity rank from a Zipf law truncated to the number of models
(p_k proportional to k^-s, seed 44), and ranks map to models through a seeded permutation
(seed 43). Request r's input is drawn with seed 20000 + r.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .models import config_model, config_input


def tenant_models(n_models: int = 100, first_seed: int = 1000, kinds=(2, 3, 4)):
    """[(workload number, weight seed)] for models 0..n-1."""
    return [(kinds[i % len(kinds)], first_seed + i) for i in range(n_models)]


@dataclass
class Trace:
    arrival_s: np.ndarray      # float64 seconds from the start, non-decreasing
    model: np.ndarray          # int model index per request
    input_seed: np.ndarray     # int per request


def tenant_trace(n_requests: int = 3000, rate_per_s: float = 50.0, zipf_s: float = 1.1, n_models: int = 100,
                 arrival_seed: int = 42, perm_seed: int = 43, rank_seed: int = 44,
                 input_seed0: int = 20000) -> Trace:
    gaps = np.random.Generator(np.random.PCG64(arrival_seed)).exponential(1.0 / rate_per_s, n_requests)
    arrival = np.cumsum(gaps)
    k = np.arange(1, n_models + 1, dtype=np.float64)
    p = k ** (-zipf_s)
    p /= p.sum()
    ranks = np.random.Generator(np.random.PCG64(rank_seed)).choice(n_models, size=n_requests, p=p)
    perm = np.random.Generator(np.random.PCG64(perm_seed)).permutation(n_models)
    return Trace(arrival, perm[ranks], input_seed0 + np.arange(n_requests))


def build_models(specs, workers: int = 8):
    """Yields (index, Model) with weights drawn, drawing up to `workers` models at once
    (the generator releases the GIL); models come back in index order."""
    from concurrent.futures import ThreadPoolExecutor

    def make(i):
        cfg, seed = specs[i]
        m = config_model(cfg, seed)
        m.blob()
        return m

    with ThreadPoolExecutor(max_workers=workers) as ex:
        futs = {}
        nxt = 0
        for i in range(len(specs)):
            while nxt < len(specs) and nxt < i + workers:
                futs[nxt] = ex.submit(make, nxt)
                nxt += 1
            yield i, futs.pop(i).result()


def request_input(model, seed: int, batch: int = 1):
    return config_input(model, batch, seed)
