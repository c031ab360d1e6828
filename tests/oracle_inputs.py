"""Turn seeded bf16 workloads into the oracle's float64 inputs (test helper)."""
from __future__ import annotations

import numpy as np

from oracle import bf16_bits_to_f64
from paper_2609_33184_amd.workloads import bf16_bits


def f64(t) -> np.ndarray:
    return bf16_bits_to_f64(bf16_bits(t))


def oracle_inputs(w, layer: int = 0, requests=None):
    """Lists (per request) of float64 arrays: q, k_hist, v_hist, k_cand, v_cand."""
    bs = range(w.B) if requests is None else requests
    q = [f64(w.q(b, layer)) for b in bs]
    kh = [f64(w.k_hist(b, layer=layer)) for b in bs]
    vh = [f64(w.v_hist(b, layer=layer)) for b in bs]
    kc = [f64(w.k_cand(b, layer=layer)) for b in bs]
    vc = [f64(w.v_cand(b, layer=layer)) for b in bs]
    return q, kh, vh, kc, vc
