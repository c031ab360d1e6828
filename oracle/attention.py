"""fp64 oracle: masked softmax attention over committed history + candidates.

Test infrastructure only (see the package docstring).  Reference passages:
Sec. 4.2 of the paper, "KV Streaming for Multi-Query Verification":

* Eq. 12: O = softmax(Q [K_H; K_G]^T / sqrt(d_h) + M) [V_H; V_G], M causal;
* the candidate region is masked by each query's absolute position, so
  candidate query i (position C_b + i) sees candidate key j (position
  C_b + j) iff j <= i, while the whole committed history is visible to
  every query of the round;
* Eq. 13 / Eq. 14: chunk-local (m_j, l_j, a_j) and the rescaled merge,
  state initialised to (-inf, 0, 0) per query and head; O = a / l at the end.

Readings where the paper leaves a choice: query head h reads KV head
floor(h / G) with G = Hq / Hkv (contiguous GQA groups); Q and K arrive with
positional encoding already applied; the scale is sigma = 1/sqrt(d).

Inputs are float64 numpy arrays, per request ``b``::

    q[b]      [n_b, Hq, d]
    k_hist[b] [C_b, Hkv, d]    v_hist[b] same
    k_cand[b] [n_b, Hkv, d]    v_cand[b] same

Outputs: O [sum n_b, Hq, d] and LSE [sum n_b, Hq] (natural log), packed in
request order.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# input decoding
# ---------------------------------------------------------------------------
def bf16_bits_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64, exactly.

    A bfloat16 value is the binary32 value whose upper 16 bits are the
    pattern and whose lower 16 bits are zero."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# the two readings that the paper leaves implicit
# ---------------------------------------------------------------------------
def kv_head_of(h: int, group: int) -> int:
    """GQA: query head h shares KV head floor(h / G)."""
    return h // group


def candidate_visible(i: int, j: int) -> bool:
    """Causal rule in the Speculative Frontier (Sec. 4.2, GPU-resident pass):
    query i (position C + i) may attend candidate key j (position C + j)
    iff j <= i."""
    return j <= i


def _cand_mask(n: int) -> np.ndarray:
    return np.array([[candidate_visible(i, j) for j in range(n)] for i in range(n)], dtype=bool)


# ---------------------------------------------------------------------------
# direct definition (Eq. 12)
# ---------------------------------------------------------------------------
def attend_heads(qh: np.ndarray, keys: np.ndarray, values: np.ndarray, visible: np.ndarray,
                 scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Masked softmax attention for one query head.

    qh [n, d], keys/values [T, d], visible [n, T] bool.
    Returns O [n, d] and LSE [n]."""
    s = scale * (qh @ keys.T)                      # scores s_t
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)               # m = max over visible keys
    w = np.where(visible, np.exp(s - m), 0.0)      # w_t = e^{s_t - m}
    l = w.sum(axis=1, keepdims=True)               # l = sum_t w_t
    o = (w @ values) / l                           # O = sum_t w_t v_t / l
    lse = (m + np.log(l))[:, 0]
    return o, lse


def verify_attention(q: Sequence[np.ndarray], k_hist: Sequence[np.ndarray], v_hist: Sequence[np.ndarray],
                     k_cand: Sequence[np.ndarray], v_cand: Sequence[np.ndarray],
                     scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 12 for every request of a Cohort, every candidate query and head."""
    outs, lses = [], []
    for b in range(len(q)):
        qb = np.asarray(q[b], dtype=np.float64)
        n, Hq, d = qb.shape
        kh, vh = np.asarray(k_hist[b], np.float64), np.asarray(v_hist[b], np.float64)
        kc, vc = np.asarray(k_cand[b], np.float64), np.asarray(v_cand[b], np.float64)
        C, Hkv = kh.shape[0], kc.shape[1]
        G = Hq // Hkv
        sc = 1.0 / math.sqrt(d) if scale is None else scale
        visible = np.concatenate([np.ones((n, C), dtype=bool), _cand_mask(n)], axis=1)
        ob = np.empty((n, Hq, d))
        lb = np.empty((n, Hq))
        for h in range(Hq):
            g = kv_head_of(h, G)
            keys = np.concatenate([kh[:, g, :], kc[:, g, :]], axis=0)
            vals = np.concatenate([vh[:, g, :], vc[:, g, :]], axis=0)
            ob[:, h, :], lb[:, h] = attend_heads(qb[:, h, :], keys, vals, visible, sc)
        outs.append(ob)
        lses.append(lb)
    return np.concatenate(outs, 0), np.concatenate(lses, 0)


# ---------------------------------------------------------------------------
# the paper's chunked procedure (Eq. 13, Eq. 14)
# ---------------------------------------------------------------------------
def _empty_state(n: int, d: int):
    """Initial state (-inf, 0, 0) per query."""
    return np.full(n, -np.inf), np.zeros(n), np.zeros((n, d))


def _chunk_local_state(s: np.ndarray, vis: np.ndarray, vals: np.ndarray):
    """Eq. 13 over the keys of one chunk visible to each query.

    A query that sees no key of the chunk gets the empty state."""
    if s.shape[1] == 0:                            # an empty chunk
        return _empty_state(s.shape[0], vals.shape[1])
    s = np.where(vis, s, -np.inf)
    m_j = s.max(axis=1)
    has = np.isfinite(m_j)
    e = np.where(vis & has[:, None], np.exp(s - np.where(has, m_j, 0.0)[:, None]), 0.0)
    l_j = e.sum(axis=1)
    a_j = e @ vals
    return m_j, l_j, a_j


def _merge(state, local):
    """Eq. 14: m' = max(m, m_j), alpha = e^{m - m'}, beta = e^{m_j - m'},
    l' = alpha l + beta l_j, a' = alpha a + beta a_j.

    An empty operand (m = -inf) has weight 0, so empty (+) X = X."""
    m, l, a = state
    m_j, l_j, a_j = local
    m_new = np.maximum(m, m_j)
    safe = np.where(np.isfinite(m_new), m_new, 0.0)
    alpha = np.where(np.isfinite(m), np.exp(m - safe), 0.0)
    beta = np.where(np.isfinite(m_j), np.exp(m_j - safe), 0.0)
    return m_new, alpha * l + beta * l_j, alpha[:, None] * a + beta[:, None] * a_j


def verify_attention_chunked(q, k_hist, v_hist, k_cand, v_cand, chunks: Sequence[Sequence[np.ndarray]],
                             scale: Optional[float] = None, cand_position: Optional[int] = None
                             ) -> Tuple[np.ndarray, np.ndarray]:
    """Online-softmax verification following Sec. 4.2 step by step.

    ``chunks[b]`` is a list of int index arrays, a partition of request b's
    history tokens [0, C_b) in processing order (any partition and order).
    The candidate pass runs after all history chunks (the paper's order) or,
    if ``cand_position`` is given, before history chunk ``cand_position``.
    """
    outs, lses = [], []
    for b in range(len(q)):
        qb = np.asarray(q[b], np.float64)
        n, Hq, d = qb.shape
        kh, vh = np.asarray(k_hist[b], np.float64), np.asarray(v_hist[b], np.float64)
        kc, vc = np.asarray(k_cand[b], np.float64), np.asarray(v_cand[b], np.float64)
        Hkv = kc.shape[1]
        G = Hq // Hkv
        sc = 1.0 / math.sqrt(d) if scale is None else scale
        cmask = _cand_mask(n)
        ob = np.empty((n, Hq, d))
        lb = np.empty((n, Hq))
        order: List = list(chunks[b])
        pos = len(order) if cand_position is None else cand_position
        order = order[:pos] + ["cand"] + order[pos:]
        for h in range(Hq):
            g = kv_head_of(h, G)
            state = _empty_state(n, d)
            for item in order:
                if isinstance(item, str):
                    keys, vals, vis = kc[:, g, :], vc[:, g, :], cmask
                else:
                    idx = np.asarray(item, dtype=np.int64)
                    keys, vals = kh[idx, g, :], vh[idx, g, :]
                    vis = np.ones((n, len(idx)), dtype=bool)   # history: visible to all
                s = sc * (qb[:, h, :] @ keys.T)               # S_j = Q K_j^T / sqrt(d)
                state = _merge(state, _chunk_local_state(s, vis, vals))
            m, l, a = state
            ob[:, h, :] = a / l[:, None]                       # O = a / l
            lb[:, h] = m + np.log(l)
        outs.append(ob)
        lses.append(lb)
    return np.concatenate(outs, 0), np.concatenate(lses, 0)


def contiguous_chunks(C: int, S: int) -> List[np.ndarray]:
    """[0, C) split into consecutive chunks of S tokens (partial last)."""
    return [np.arange(s, min(C, s + S)) for s in range(0, C, S)]
