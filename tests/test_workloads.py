"""Seeded input generator: determinism, path equivalence, workload shapes (CPU)."""
import hashlib

import numpy as np
import torch

from paper_2609_33184_amd import workloads as W


def _sha(t):
    return hashlib.sha256(W.bf16_bits(t).tobytes()).hexdigest()


def test_numpy_and_torch_paths_identical():
    # the CPU (numpy) and device (torch int64) hash paths must agree bit for bit,
    # including indices beyond 2**32
    idx = torch.cat([torch.arange(0, 4096), torch.arange((1 << 32) - 2048, (1 << 32) + 2048),
                     torch.arange(9 * (1 << 30), 9 * (1 << 30) + 1000)]).to(torch.int64)
    for seed in (0, 1, 0xDEADBEEF):
        assert torch.equal(W.normal_f32(seed, idx), W.normal_f32(seed, idx, force_torch=True))
        assert torch.equal(W.uniform01_f32(seed, idx), W.uniform01_f32(seed, idx, force_torch=True))
        assert torch.equal(W.bernoulli(seed, idx, 100), W.bernoulli(seed, idx, 100, force_torch=True))


def test_determinism_and_slicing():
    w = W.workload(1)
    a = w.k_hist(0)
    b = w.k_hist(0)
    assert _sha(a) == _sha(b)
    # any slice regenerates independently
    assert torch.equal(w.k_hist(0, 100, 200), a[100:200])
    assert torch.equal(w.k_hist(0, heads=[1]), a[:, 1:2])
    # different tensors differ
    assert not torch.equal(w.v_hist(0), a)


def test_distribution():
    x = W.normal_f32(W.seed_key(7), torch.arange(1 << 20))
    assert abs(float(x.mean())) < 5e-3
    assert abs(float(x.var()) - 1.0) < 5e-3
    assert float(x.abs().max()) <= 6.0
    u = W.uniform01_f32(W.seed_key(8), torch.arange(1 << 16))
    assert 0.0 <= float(u.min()) and float(u.max()) < 1.0


def test_config_shapes():
    w1, w2, w3, w4, w5 = (W.workload(i) for i in range(1, 6))
    assert (w1.B, w1.num_q_heads, w1.num_kv_heads, w1.hist_len, w1.num_cand, w1.num_chunks) == \
        (1, 8, 2, [4096], [5], 4)
    assert (w2.num_q_heads, w2.num_kv_heads, w2.chunk_tokens, w2.num_chunks, w2.kscale) == (32, 8, 2048, 8, True)
    assert (w3.B, w3.hist_len[0], w3.num_chunks, w3.num_cand[0]) == (16, 32768, 8, 6)
    assert w3.history_kv_bytes() == 2 * 1024 ** 3
    assert w4.B == 64 and min(w4.hist_len) >= 2048 and max(w4.hist_len) <= 65536
    assert set(w4.num_cand) <= set(range(1, 9)) and len(set(w4.num_cand)) > 4
    assert any(c % 4096 for c in w4.hist_len)           # partial last chunks exist
    assert (w5.B, w5.layers, w5.hist_len[0], w5.chunk_tokens, w5.num_cand[0]) == (32, 36, 131072, 8192, 8)
    assert w5.history_kv_bytes() == 16 * 1024 ** 3
    for j in range(w4.num_chunks):
        lens = w4.chunk_lens(j)
        assert all(0 <= x <= 4096 for x in lens)
    assert [sum(w4.chunk_lens(j)[b] for j in range(w4.num_chunks)) for b in range(w4.B)] == w4.hist_len


def test_kscale_and_outliers():
    w2 = W.workload(2)
    s = w2._kscale_vec(0, 0, "cpu")
    assert float(s.min()) >= 0.5 and float(s.max()) < 2.0
    w5 = W.workload(5)
    k = w5.k_hist(0, 0, 4096).float()
    frac = float((k.abs().amax(-1) > 6.01).float().mean())
    assert 0.005 < frac < 0.015


def test_chunk_packing():
    w = W.custom([5, 0, 9], [1, 2, 3], chunk_tokens=4)
    k, v = w.chunk_kv(1)
    assert w.chunk_lens(1) == [1, 0, 4]
    assert torch.equal(k[0:1], w.k_hist(0, 4, 5)) and torch.equal(k[1:5], w.k_hist(2, 4, 8))
    assert torch.equal(v[1:5], w.v_hist(2, 4, 8))
