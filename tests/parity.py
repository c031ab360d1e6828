"""Parity helpers: compare GPU outputs with the fp64 oracle (test helper).

The bar: max-abs error <= 2e-3 and relative L2 error <= 1e-3 on
the fp32 outputs, for bf16 inputs with fp32 accumulation.
"""
from __future__ import annotations

from typing import Iterable, Tuple

import numpy as np
import torch

import oracle
from oracle_inputs import f64

MAX_ABS = 2e-3
REL_L2 = 1e-3


def errors(gpu: np.ndarray, ref: np.ndarray) -> Tuple[float, float]:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), "non-finite GPU output"
    max_abs = float(np.max(np.abs(gpu - ref))) if gpu.size else 0.0
    rel = float(np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-300)) if gpu.size else 0.0
    return max_abs, rel


def assert_parity(gpu, ref, what: str = "", max_abs: float = MAX_ABS, rel_l2: float = REL_L2):
    ma, rl = errors(gpu, ref)
    print(f"parity {what}: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert ma <= max_abs and rl <= rel_l2, f"{what}: max_abs={ma:.3e} rel_l2={rl:.3e}"
    return ma, rl


def oracle_group(w, b: int, g: int, layer: int = 0):
    """Oracle output of request b's rows for KV head g: O [n_b, G, d], LSE [n_b, G].

    Regenerates on the CPU only the slices it needs (one KV head)."""
    G = w.group
    q = f64(w.q(b, layer))[:, g * G:(g + 1) * G, :]
    kh = f64(w.k_hist(b, heads=[g], layer=layer))
    vh = f64(w.v_hist(b, heads=[g], layer=layer))
    kc = f64(w.k_cand(b, heads=[g], layer=layer))
    vc = f64(w.v_cand(b, heads=[g], layer=layer))
    return oracle.verify_attention([q], [kh], [vh], [kc], [vc], scale=w.softmax_scale)


def oracle_full(w, layer: int = 0):
    """Oracle output of every row: O [sum n_b, Hq, d], LSE [sum n_b, Hq]."""
    from oracle_inputs import oracle_inputs
    q, kh, vh, kc, vc = oracle_inputs(w, layer)
    return oracle.verify_attention(q, kh, vh, kc, vc, scale=w.softmax_scale)


def gpu_group(w, out: torch.Tensor, lse: torch.Tensor, b: int, g: int):
    off = w.row_offsets()[b]
    n, G = w.num_cand[b], w.group
    o = out[off:off + n, g * G:(g + 1) * G, :].double().cpu().numpy()
    l = lse[off:off + n, g * G:(g + 1) * G].double().cpu().numpy()
    return o, l


def check_sampled(w, out, lse, pairs: Iterable[Tuple[int, int]], layer: int = 0, what: str = ""):
    """Parity on sampled (request, KV head) groups, pooled over the samples."""
    gs, rs, gl, rl = [], [], [], []
    for b, g in pairs:
        ro, rlse = oracle_group(w, b, g, layer)
        go, glse = gpu_group(w, out, lse, b, g)
        gs.append(go.ravel())
        rs.append(ro.ravel())
        gl.append(glse.ravel())
        rl.append(rlse.ravel())
        assert_parity(go, ro, f"{what} b={b} g={g}")
    assert_parity(np.concatenate(gs), np.concatenate(rs), f"{what} pooled")
    assert_parity(np.concatenate(gl), np.concatenate(rl), f"{what} lse", max_abs=1e-3, rel_l2=1e-4)
