"""Pins of the fp64 oracle against things other than itself (CPU only).

Each ``pin_*`` function checks the oracle against something the paper or the
mathematics fixes:

* hand-derived closed-form golden cases (tests/golden/closed_form_cases.json);
* 50-digit decimal brute force of Eq. 12 on tiny inputs;
* torch's scaled_dot_product_attention in float64 (a library routine for
  masked GQA softmax attention), with the candidate causal mask;
* k = 0 (one candidate) reducing to ordinary single-token decode;
* Eq. 17: the chunked Eq. 13/14 procedure equals the direct definition for
  every partition and order of the history (and any position of the
  candidate pass); LSE agrees too;
* a candidate never sees later candidates (their K/V may change freely);
* softmax weights sum to 1 (V = 1 gives O = 1), identical keys give the mean
  of the visible values, V x 2 gives O x 2 exactly, permuting history tokens
  changes nothing.

``test_planted_mistakes`` plants plausible mistakes in the oracle (dropped
scale, wrong GQA mapping, diagonal excluded, mask dropped, merge without
rescaling, missing normalisation, LSE sign) and requires each to be caught.
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
import oracle.attention as OA
from oracle.attention import contiguous_chunks
from paper_2609_33184_amd import workloads as W
from oracle_inputs import oracle_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_form_cases.json")


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(1e-300, float(np.max(np.abs(b)))))


def _tiny(seed, C, n, Hq=4, Hkv=2, d=8, B=1):
    w = W.custom([C] * B, [n] * B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, chunk_tokens=4,
                 seed_base=seed)
    return w, oracle_inputs(w)


# ---------------------------------------------------------------------------
# pins (raise AssertionError on failure)
# ---------------------------------------------------------------------------
def _eval_expr(s: str) -> float:
    return float(eval(s, {"__builtins__": {}}, {"e": math.e, "exp": math.exp, "ln": math.log}))


def pin_golden():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        d = len(c["q"][0][0][0])
        arr = lambda x, shape_tail: np.array(x, dtype=np.float64).reshape((-1,) + shape_tail)
        q = [np.array(x, np.float64) for x in c["q"]]
        Hkv = len(c["k_cand"][0][0])
        kh = [arr(x, (Hkv, d)) for x in c["k_hist"]]
        vh = [arr(x, (Hkv, d)) for x in c["v_hist"]]
        kc = [np.array(x, np.float64) for x in c["k_cand"]]
        vc = [np.array(x, np.float64) for x in c["v_cand"]]
        eo = np.array([[[_eval_expr(e) for e in row_h] for row_h in row] for row in c["expect_o"]])
        el = np.array([[_eval_expr(e) for e in row] for row in c["expect_lse"]])
        o, l = oracle.verify_attention(q, kh, vh, kc, vc)
        assert np.allclose(o, eo, rtol=1e-12, atol=1e-14), (c["name"], o, eo)
        assert np.allclose(l, el, rtol=1e-12, atol=1e-12), (c["name"], l, el)
        chunks = [contiguous_chunks(x.shape[0], 1) for x in kh]
        o2, l2 = oracle.verify_attention_chunked(q, kh, vh, kc, vc, chunks)
        assert np.allclose(o2, eo, rtol=1e-12, atol=1e-14), (c["name"], "chunked")
        assert np.allclose(l2, el, rtol=1e-12, atol=1e-12), (c["name"], "chunked lse")


def pin_decimal(cases=((0, 1), (1, 1), (5, 3), (13, 3), (0, 3)), B=2):
    for k, (C, n) in enumerate(cases):
        w, (q, kh, vh, kc, vc) = _tiny(100 + k, C, n, B=B)
        O_dec, L_dec = oracle.verify_attention_decimal(q, kh, vh, kc, vc)
        o_ref = np.array([[[float(x) for x in hrow] for hrow in row] for row in O_dec])
        l_ref = np.array([[float(x) for x in row] for row in L_dec])
        o, l = oracle.verify_attention(q, kh, vh, kc, vc)
        assert _rel(o, o_ref) <= 1e-12, ("direct", C, n, _rel(o, o_ref))
        assert _rel(l, l_ref) <= 1e-12, ("direct lse", C, n)
        chunks = [contiguous_chunks(C, 2) for _ in range(B)]
        o2, l2 = oracle.verify_attention_chunked(q, kh, vh, kc, vc, chunks)
        assert _rel(o2, o_ref) <= 1e-12, ("chunked", C, n)
        assert _rel(l2, l_ref) <= 1e-12, ("chunked lse", C, n)


def _sdpa(q, kh, vh, kc, vc, scale=None):
    """torch SDPA (math backend, float64) with the candidate causal mask."""
    outs = []
    for b in range(len(q)):
        n, Hq, d = q[b].shape
        C = kh[b].shape[0]
        Q = torch.from_numpy(q[b]).permute(1, 0, 2)[None]                       # [1, Hq, n, d]
        K = torch.from_numpy(np.concatenate([kh[b], kc[b]], 0)).permute(1, 0, 2)[None]
        V = torch.from_numpy(np.concatenate([vh[b], vc[b]], 0)).permute(1, 0, 2)[None]
        mask = torch.ones(n, C + n, dtype=torch.bool)
        mask[:, C:] = torch.tril(torch.ones(n, n, dtype=torch.bool))
        o = torch.nn.functional.scaled_dot_product_attention(Q, K, V, attn_mask=mask, scale=scale,
                                                             enable_gqa=True)
        outs.append(o[0].permute(1, 0, 2).numpy())
    return np.concatenate(outs, 0)


def pin_sdpa(shapes=((37, 3, 8, 2, 16), (0, 4, 4, 4, 8), (64, 1, 8, 1, 32), (5, 8, 32, 8, 16))):
    for k, (C, n, Hq, Hkv, d) in enumerate(shapes):
        w, (q, kh, vh, kc, vc) = _tiny(200 + k, C, n, Hq, Hkv, d, B=2)
        o, _ = oracle.verify_attention(q, kh, vh, kc, vc)
        ref = _sdpa(q, kh, vh, kc, vc)
        assert _rel(o, ref) <= 1e-12, ("sdpa", C, n, Hq, Hkv, d, _rel(o, ref))


def pin_decode():
    """k = 0: one candidate that sees the whole history and itself."""
    for k, C in enumerate((1, 17, 300)):
        w, (q, kh, vh, kc, vc) = _tiny(300 + k, C, 1, 8, 2, 16)
        o, l = oracle.verify_attention(q, kh, vh, kc, vc)
        Q = torch.from_numpy(q[0]).permute(1, 0, 2)[None]
        K = torch.from_numpy(np.concatenate([kh[0], kc[0]], 0)).permute(1, 0, 2)[None]
        V = torch.from_numpy(np.concatenate([vh[0], vc[0]], 0)).permute(1, 0, 2)[None]
        ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, enable_gqa=True)
        assert _rel(o, ref[0].permute(1, 0, 2).numpy()) <= 1e-12
        # textbook decode: p = softmax(K q / sqrt(d)), o = V^T p, lse = log sum exp
        for h in range(8):
            g = h // 4
            keys = np.concatenate([kh[0][:, g], kc[0][:, g]], 0)
            vals = np.concatenate([vh[0][:, g], vc[0][:, g]], 0)
            s = keys @ q[0][0, h] / math.sqrt(16)
            lse = np.logaddexp.reduce(s)
            p = np.exp(s - lse)
            assert _rel(o[0, h], vals.T @ p) <= 1e-12
            assert abs(l[0, h] - lse) <= 1e-12 * max(1.0, abs(lse))


def pin_chunk_invariance(seed=0, C=29, n=4, trials=6):
    w, (q, kh, vh, kc, vc) = _tiny(400 + seed, C, n, 4, 2, 8, B=2)
    o, l = oracle.verify_attention(q, kh, vh, kc, vc)
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        chunks = []
        for b in range(2):
            perm = rng.permutation(C)
            cuts = np.sort(rng.choice(np.arange(1, C), size=rng.integers(0, min(6, C - 1) + 1),
                                      replace=False)) if C > 1 else []
            parts = np.split(perm, cuts)
            chunks.append([p for p in parts])
        pos = int(rng.integers(0, len(chunks[0]) + 1))
        o2, l2 = oracle.verify_attention_chunked(q, kh, vh, kc, vc, chunks, cand_position=min(pos, len(chunks[1])))
        assert _rel(o2, o) <= 1e-12, ("chunk order/partition", _rel(o2, o))
        assert _rel(l2, l) <= 1e-12


def pin_mask():
    """Later candidates' K/V scaled x64 leave earlier queries' outputs bitwise unchanged."""
    w, (q, kh, vh, kc, vc) = _tiny(500, 7, 5, 4, 2, 8)
    o, l = oracle.verify_attention(q, kh, vh, kc, vc)
    for j in range(1, 5):
        kc2, vc2 = kc[0].copy(), vc[0].copy()
        kc2[j:] *= 64.0
        vc2[j:] *= 64.0
        o2, l2 = oracle.verify_attention(q, kh, vh, [kc2], [vc2])
        assert np.array_equal(o2[:j], o[:j]) and np.array_equal(l2[:j], l[:j]), ("mask", j)
        assert not np.allclose(o2[j:], o[j:]), ("later queries must see the change", j)


def pin_weights_and_closed_forms():
    w, (q, kh, vh, kc, vc) = _tiny(600, 11, 4, 4, 2, 8)
    ones = lambda a: np.ones_like(a)
    o, _ = oracle.verify_attention(q, kh, [ones(vh[0])], kc, [ones(vc[0])])
    assert np.max(np.abs(o - 1.0)) <= 1e-15, "weights must sum to 1"
    # identical keys -> mean of the visible values
    kconst = np.broadcast_to(kh[0][:1], kh[0].shape).copy()
    kcc = np.broadcast_to(kh[0][:1], kc[0].shape).copy()
    o, _ = oracle.verify_attention(q, [kconst], vh, [kcc], vc)
    for i in range(4):
        for h in range(4):
            g = h // 2
            vis = np.concatenate([vh[0][:, g], vc[0][: i + 1, g]], 0)
            assert _rel(o[i, h], vis.mean(0)) <= 1e-13
    # V x 2 -> O x 2 exactly
    o1, _ = oracle.verify_attention(q, kh, vh, kc, vc)
    o2, _ = oracle.verify_attention(q, kh, [2 * vh[0]], kc, [2 * vc[0]])
    assert np.array_equal(o2, 2 * o1)
    # C = 0, i = 0 -> O = v_cand0 exactly
    w0, (q0, kh0, vh0, kc0, vc0) = _tiny(601, 0, 3, 4, 2, 8)
    o, _ = oracle.verify_attention(q0, kh0, vh0, kc0, vc0)
    for h in range(4):
        assert np.array_equal(o[0, h], vc0[0][0, h // 2])
    # permuting history tokens changes nothing (up to rounding)
    perm = np.random.default_rng(1).permutation(11)
    o3, _ = oracle.verify_attention(q, [kh[0][perm]], [vh[0][perm]], kc, vc)
    assert _rel(o3, o1) <= 1e-13


ALL_PINS = [pin_golden, pin_decimal, pin_sdpa, pin_decode, pin_chunk_invariance, pin_mask,
            pin_weights_and_closed_forms]


# ---------------------------------------------------------------------------
# tests
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


@settings(max_examples=25, deadline=None)
@given(seed=st.integers(0, 10_000), C=st.integers(0, 40), n=st.integers(1, 8))
def test_chunk_invariance_property(seed, C, n):
    w, (q, kh, vh, kc, vc) = _tiny(seed, C, n, 4, 2, 8, B=1)
    o, l = oracle.verify_attention(q, kh, vh, kc, vc)
    rng = np.random.default_rng(seed)
    perm = rng.permutation(C)
    parts = np.array_split(perm, int(rng.integers(1, 6))) if C else []
    parts = [p for p in parts if len(p)] + ([np.array([], dtype=np.int64)] if rng.random() < 0.3 else [])
    o2, l2 = oracle.verify_attention_chunked(q, kh, vh, kc, vc, [parts],
                                             cand_position=int(rng.integers(0, len(parts) + 1)))
    assert _rel(o2, o) <= 1e-12
    assert _rel(l2, l) <= 1e-12


def test_bf16_decoding():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x4049, 0x7F7F, 0x0001], dtype=np.uint16)
    vals = OA.bf16_bits_to_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0 and vals[2] == 0.0
    assert np.signbit(vals[3]) and vals[3] == 0.0
    assert vals[4] == 3.140625
    assert vals[5] == float.fromhex("0x1.fep127")
    assert vals[6] == 2.0 ** -133
    t = torch.tensor([1.0, -2.5, 3.140625], dtype=torch.bfloat16)
    assert np.array_equal(OA.bf16_bits_to_f64(W.bf16_bits(t)), np.array([1.0, -2.5, 3.140625]))


# ---------------------------------------------------------------------------
# planted mistakes: every one must be caught by at least one pin
# ---------------------------------------------------------------------------
def _mutant_no_scale(mp):
    class FakeMath:
        sqrt = staticmethod(lambda x: 1.0)
    mp.setattr(OA, "math", FakeMath)


def _mutant_gqa_interleaved(mp):
    mp.setattr(OA, "kv_head_of", lambda h, G: h % 2)


def _mutant_diag_excluded(mp):
    mp.setattr(OA, "candidate_visible", lambda i, j: j < i)


def _mutant_no_mask(mp):
    mp.setattr(OA, "candidate_visible", lambda i, j: True)


def _mutant_merge_no_rescale(mp):
    def bad_merge(state, local):
        m, l, a = state
        m_j, l_j, a_j = local
        return np.maximum(m, m_j), l + l_j, a + a_j
    mp.setattr(OA, "_merge", bad_merge)


def _mutant_no_normalise(mp):
    orig = OA.attend_heads

    def bad(qh, keys, values, visible, scale):
        o, lse = orig(qh, keys, values, visible, scale)
        s = np.where(visible, scale * (qh @ keys.T), -np.inf)
        l = np.exp(s - s.max(1, keepdims=True)).sum(1, keepdims=True)
        return o * l, lse
    mp.setattr(OA, "attend_heads", bad)


def _mutant_lse_sign(mp):
    orig = OA.attend_heads

    def bad(qh, keys, values, visible, scale):
        o, lse = orig(qh, keys, values, visible, scale)
        s = np.where(visible, scale * (qh @ keys.T), -np.inf)
        m = s.max(1)
        return o, m - (lse - m)
    mp.setattr(OA, "attend_heads", bad)


def _mutant_transposed_values(mp):
    orig = OA.attend_heads

    def bad(qh, keys, values, visible, scale):
        # weights applied to the values of the reversed token order
        return orig(qh, keys, values[::-1].copy(), visible, scale)
    mp.setattr(OA, "attend_heads", bad)


MUTANTS = [_mutant_no_scale, _mutant_gqa_interleaved, _mutant_diag_excluded, _mutant_no_mask,
           _mutant_merge_no_rescale, _mutant_no_normalise, _mutant_lse_sign, _mutant_transposed_values]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_planted_mistakes(mutant, monkeypatch):
    with monkeypatch.context() as mp:
        mutant(mp)
        caught = []
        for pin in ALL_PINS:
            try:
                with np.errstate(all="ignore"):
                    pin()
            except (AssertionError, ValueError, FloatingPointError, IndexError):
                caught.append(pin.__name__)
        assert caught, f"{mutant.__name__} was not caught by any pin"
