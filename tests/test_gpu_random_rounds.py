"""Seeded random rounds on the GPU against the fp64 oracle, through the C ABI.

Each case draws a small ragged cohort and a way of running its round:
request count, history lengths (empty, below one tile, across several tiles
and chunks), candidate counts, query-group shape (1 to 64 rows per KV head),
the value distribution (per-channel K scales, outlier key rows), chunk size,
chunk layout, workgroup share size, balancing tail, the row count from which
the MFMA body runs, call batching, chunk order and where the candidate call
falls among the history calls.  Every output row and LSE is compared with
the oracle at the bar of the other parity tests; a second round on the same
buffers, with the counter block promised zero, must give the same bits.
The draws are fixed by the seed, so a failing case is named by its index
and its printed parameters.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2609_33184_amd import harness as H
from paper_2609_33184_amd import specstream as ss
from paper_2609_33184_amd import workloads as W
from parity import assert_parity, oracle_full

NUM_RANDOM = 24          # cases with every option drawn
NUM_CASES = 28           # the last ones with shares large enough for the balancing tail
LAYOUTS = (ss.SS_KV_TOKEN_MAJOR, ss.SS_KV_HEAD_MAJOR, ss.SS_KV_HEAD_MAJOR_KV)


def _draw_len(rng) -> int:
    u = rng.random()
    if u < 0.12:
        return 0
    if u < 0.35:
        return int(rng.integers(1, 65))
    if u < 0.8:
        return int(rng.integers(65, 3001))
    return int(rng.integers(3001, 12001))


def draw_case(k: int) -> dict:
    """Case k's workload and call parameters (a pure function of k).  Cases
    from NUM_RANDOM on put 12000 to 40000 history tokens into one batched
    call with shares of 8192 tokens and an explicit tail fraction, the
    smallest shares for which the library builds a balancing tail."""
    rng = np.random.default_rng(20260 + k)
    tail = k >= NUM_RANDOM
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 6, 8]))
    hq = g * hkv
    max_cand = min(8, 64 // g)
    B = int(rng.integers(1, 6)) if not tail else 3
    lens = [_draw_len(rng) for _ in range(B)] if not tail else [int(rng.integers(4000, 13334)) for _ in range(B)]
    cands = [int(rng.integers(1, max_cand + 1)) for _ in range(B)]
    chunk_tokens = int(rng.choice([64, 200, 1024, 4096, 100000] if not tail else [1024, 4096, 100000]))
    split = int(rng.choice([0, 0, 32, 96, 512, 4096])) if not tail else 8192
    balance = int(rng.choice([0, -1, 100, 500])) if not tail else int(rng.choice([100, 500]))
    return dict(
        lens=lens, cands=cands, hq=hq, hkv=hkv, chunk_tokens=chunk_tokens,
        kscale=bool(rng.random() < 0.3), outliers=int(rng.choice([0, 0, 100])),
        layout=int(rng.choice(LAYOUTS)), split=split, balance=balance,
        mfma_min_rows=int(rng.choice([0, 1, 3, 5])),
        batch_choice=int(rng.integers(0, 3)) if not tail else 2,   # 0: per chunk, 1: pairs, 2: up to 32 chunks per call
        shuffle=bool(rng.random() < 0.5), cand_pos_u=float(rng.random()),
        seed=1000 + k)


@pytest.fixture(scope="module")
def stream():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.load()
    s = torch.cuda.Stream()
    yield s
    torch.cuda.synchronize()


def test_draws_cover_the_options():
    """The fixed draws reach every layout, batching mode and body choice, an
    empty history, a unit of more than 32 rows per KV head and a call whose
    shares are large enough for the balancing tail."""
    cases = [draw_case(k) for k in range(NUM_CASES)]
    assert {c["layout"] for c in cases} == set(LAYOUTS)
    assert {c["batch_choice"] for c in cases} == {0, 1, 2}
    assert {c["mfma_min_rows"] for c in cases} >= {1, 5}
    assert any(0 in c["lens"] for c in cases)
    assert any(max(n * (c["hq"] // c["hkv"]) for n in c["cands"]) > 32 for c in cases)
    tails = [c for c in cases if c["balance"] > 0 and c["split"] >= 4096 and c["batch_choice"] == 2]
    assert len(tails) >= 4 and all(sum(c["lens"]) >= 12000 for c in tails)
    assert {c["balance"] for c in tails} == {100, 500}


@pytest.mark.gpu
@pytest.mark.parametrize("k", range(NUM_CASES))
def test_random_round(stream, k):
    c = draw_case(k)
    w = W.custom(c["lens"], c["cands"], num_q_heads=c["hq"], num_kv_heads=c["hkv"],
                 chunk_tokens=c["chunk_tokens"], seed_base=c["seed"], kscale=c["kscale"],
                 outlier_per_10000=c["outliers"])
    nch = w.num_chunks
    batch = (1, 2, min(32, max(1, nch)))[c["batch_choice"]]
    order = None
    if c["shuffle"] and batch == 1 and nch > 1:
        order = list(np.random.default_rng(c["seed"]).permutation(nch))
    cand_pos = int(c["cand_pos_u"] * (nch + 1)) if batch == 1 else None
    print(f"random case {k}: {c} chunks={nch} batch={batch} order={order} cand_pos={cand_pos}", flush=True)

    b = H.RoundBuffers(w, split_tokens=c["split"], mfma_min_rows=c["mfma_min_rows"], kv_layout=c["layout"],
                       balance_permille=c["balance"], counters_zeroed=1)
    chunks = H.hbm_history(w, kv_layout=c["layout"])
    outs = []
    for rep in range(2):
        b.out.fill_(float("nan"))
        b.lse.fill_(float("nan"))
        torch.cuda.synchronize()
        H.run_round(b, chunks, stream.cuda_stream, order=order, cand_position=cand_pos, batch=batch)
        stream.synchronize()
        outs.append((b.out.clone(), b.lse.clone()))
    ref_o, ref_l = oracle_full(w)
    assert_parity(outs[0][0].double().cpu().numpy(), ref_o, f"random {k}")
    assert_parity(outs[0][1].double().cpu().numpy(), ref_l, f"random {k} lse", max_abs=1e-3, rel_l2=1e-4)
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1]), \
        f"random {k}: the second round on the same workspace differs"


def capacity_case(name: str):
    """Cohorts whose history launches overflow the smaller kernel-argument
    tables: more than 64 requests (finalize's larger item table), more than
    512 units, 1024 items or 256 workgroups per KV head (the largest chunk
    table), and the same with 64 rows per KV head (the wide kernel's
    medium and largest tables)."""
    rng = np.random.default_rng({"req100_split32": 1, "req100_batched": 2, "req300_split96": 3,
                                 "wide100_split32": 4, "wide100_auto": 5}[name])
    if name.startswith("req100"):
        B, hq, hkv, S, layout = 100, 8, 2, 256, ss.SS_KV_TOKEN_MAJOR
        cands = rng.integers(1, 9, B)
        lens = rng.integers(0, 601, B)
        split, batch = (32, 3) if name == "req100_split32" else (0, 3)
    elif name == "req300_split96":
        B, hq, hkv, S, layout = 300, 8, 2, 512, ss.SS_KV_HEAD_MAJOR_KV
        cands = rng.integers(1, 5, B)
        lens = rng.integers(100, 401, B)
        split, batch = 96, 1
    else:
        B, hq, hkv, S, layout = 100, 64, 8, 1024, ss.SS_KV_HEAD_MAJOR_KV
        cands = np.full(B, 8)
        lens = rng.integers(100, 701, B)
        split, batch = (32 if name == "wide100_split32" else 0), 1
    return dict(B=B, hq=hq, hkv=hkv, S=S, layout=layout, cands=[int(x) for x in cands],
                lens=[int(x) for x in lens], split=split, batch=batch)


CAPACITY_CASES = ["req100_split32", "req100_batched", "req300_split96", "wide100_split32", "wide100_auto"]


@pytest.mark.gpu
@pytest.mark.parametrize("name", CAPACITY_CASES)
def test_table_capacities(stream, name):
    c = capacity_case(name)
    w = W.custom(c["lens"], c["cands"], num_q_heads=c["hq"], num_kv_heads=c["hkv"], chunk_tokens=c["S"],
                 seed_base=77)
    print(f"capacity case {name}: B={c['B']} {c['hq']}q/{c['hkv']}kv chunks={w.num_chunks} split={c['split']} "
          f"batch={c['batch']} layout={c['layout']}", flush=True)
    b = H.RoundBuffers(w, split_tokens=c["split"], kv_layout=c["layout"])
    chunks = H.hbm_history(w, kv_layout=c["layout"])
    torch.cuda.synchronize()
    H.run_round(b, chunks, stream.cuda_stream, batch=c["batch"])
    stream.synchronize()
    ref_o, ref_l = oracle_full(w)
    assert_parity(b.out.double().cpu().numpy(), ref_o, f"capacity {name}")
    assert_parity(b.lse.double().cpu().numpy(), ref_l, f"capacity {name} lse", max_abs=1e-3, rel_l2=1e-4)


STREAMED_CASES = [k for k in range(NUM_CASES) if k % 3 == 0]


@pytest.mark.gpu
@pytest.mark.parametrize("k", STREAMED_CASES)
def test_random_streamed_round(stream, k):
    """The same random rounds with the history streamed from pinned host
    memory through the two-slot pipeline: one chunk per transfer (in the
    drawn order) or transfer batches of adjacent chunks.  The result equals,
    bitwise, the in-HBM round that makes the same history calls, and
    matches the oracle."""
    c = draw_case(k)
    w = W.custom(c["lens"], c["cands"], num_q_heads=c["hq"], num_kv_heads=c["hkv"],
                 chunk_tokens=c["chunk_tokens"], seed_base=c["seed"], kscale=c["kscale"],
                 outlier_per_10000=c["outliers"])
    nch = w.num_chunks
    if nch == 0:
        pytest.skip("no history to stream")
    batch = (1, 2, min(32, nch))[c["batch_choice"]]
    order = list(np.random.default_rng(c["seed"]).permutation(nch)) if batch == 1 and c["shuffle"] else None
    print(f"random streamed case {k}: chunks={nch} batch={batch} order={order} layout={c['layout']}", flush=True)
    kw = dict(split_tokens=c["split"], mfma_min_rows=c["mfma_min_rows"], kv_layout=c["layout"],
              balance_permille=c["balance"])
    ref = H.RoundBuffers(w, **kw)
    chunks = H.hbm_history(w, kv_layout=c["layout"])
    torch.cuda.synchronize()
    H.run_round(ref, chunks, stream.cuda_stream, order=order, batch=batch)
    stream.synchronize()
    del chunks
    host = H.HostHistory(w, kv_layout=c["layout"])
    pipe = H.Pipeline(H.batch_bytes(host, batch) if batch > 1 else host.max_chunk_bytes())
    try:
        b = H.RoundBuffers(w, **kw)
        b.out.fill_(float("nan"))
        torch.cuda.synchronize()
        H.run_round_streamed(b, host, pipe, stream.cuda_stream, order=order, batch=batch)
        stream.synchronize()
    finally:
        pipe.close()
    assert torch.equal(b.out, ref.out) and torch.equal(b.lse, ref.lse), f"streamed case {k} differs from in-HBM"
    ref_o, ref_l = oracle_full(w)
    assert_parity(b.out.double().cpu().numpy(), ref_o, f"streamed {k}")
    assert_parity(b.lse.double().cpu().numpy(), ref_l, f"streamed {k} lse", max_abs=1e-3, rel_l2=1e-4)
