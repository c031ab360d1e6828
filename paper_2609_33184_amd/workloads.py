"""Seeded synthetic inputs for verification-attention rounds.

This module only *produces inputs*: query, history and candidate K/V tensors
in bfloat16, per-request history lengths and candidate counts.  It holds no
attention arithmetic, so both the fp64 oracle (on the CPU) and the HIP path
(on the GPU) may draw from it without sharing any of the method.

Generator
---------
Every value is a pure function of ``(seed, element index)``:

* a 32-bit key is derived from ``(0x55C0DE, config, layer, request, tensor)``
  with the MurmurHash3 32-bit finaliser (``fmix32``, Appleby) applied to
  running sums;
* each element draws six ``fmix32`` hashes of its index (counter-based
  generation), giving twelve 16-bit uniforms ``u_k``;
* the Irwin-Hall sum ``x = sum_k (u_k + 1/2)/65536 - 6`` has mean 0 and
  variance 1 (the classical twelve-uniform approximation of N(0,1), bounded
  to +-6).  ``x`` is an integer over 65536, so it is exact in float32;
* optional transforms are single IEEE float32 operations (a per-channel K
  scale in [0.5, 2], an exact x8 for outlier key rows);
* the result is rounded once to bfloat16 with round-to-nearest-even.

Only integer arithmetic (kept below 2**63) and correctly rounded float32
operations are used, so the CPU and the GPU produce bit-identical tensors.
That lets the GPU generate the multi-GiB histories quickly while the oracle
regenerates, on the CPU, exactly the slices it samples.

Workloads
---------
The five workloads below stand in for the paper's long-context serving
workloads (Sec. 5.1: LongBench v2 / MRCR long inputs, 16K-32K ablation
inputs, up to 32 concurrent requests, widths q in {2,4,6,8}); the paper
gives no activation statistics, so standard-normal Q/K/V with the stated
transforms are used.  No item of any dataset is used or reproduced.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import torch

M32 = 0xFFFFFFFF
GOLDEN = 0x9E3779B9

# tensor ids (part of the seed key)
TID_Q, TID_KH, TID_VH, TID_KC, TID_VC, TID_KSCALE, TID_OUT_H, TID_OUT_C, TID_LEN = range(9)


# ----------------------------------------------------------------------------
# 32-bit counter hash, host (python int) and tensor (int64) versions
# ----------------------------------------------------------------------------
def _mul32_int(x: int, c: int) -> int:
    return (x * c) & M32


def fmix32_int(h: int) -> int:
    h &= M32
    h ^= h >> 16
    h = _mul32_int(h, 0x85EBCA6B)
    h ^= h >> 13
    h = _mul32_int(h, 0xC2B2AE35)
    h ^= h >> 16
    return h


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2**32 for int64 tensors holding values in [0, 2**32).

    Split into 16-bit halves so no intermediate exceeds 2**49 (int64 never
    overflows, the result is the same on every device)."""
    c_lo = c & 0xFFFF
    x_lo = x & 0xFFFF
    x_hi = x >> 16
    return (x_lo * c + ((x_hi * c_lo) << 16)) & M32


def fmix32(h: torch.Tensor) -> torch.Tensor:
    h = h ^ (h >> 16)
    h = _mul32(h, 0x85EBCA6B)
    h = h ^ (h >> 13)
    h = _mul32(h, 0xC2B2AE35)
    h = h ^ (h >> 16)
    return h


def seed_key(*parts: int) -> int:
    """32-bit key for a (config, layer, request, tensor) tuple."""
    h = fmix32_int(0x55C0DE)
    for p in parts:
        h = fmix32_int((h + (int(p) & M32) * GOLDEN) & M32)
    return h


def _fmix32_np(h):
    """fmix32 on a numpy uint32 array (multiplication wraps mod 2**32)."""
    import numpy as np
    h = h ^ (h >> np.uint32(16))
    h = h * np.uint32(0x85EBCA6B)
    h = h ^ (h >> np.uint32(13))
    h = h * np.uint32(0xC2B2AE35)
    h = h ^ (h >> np.uint32(16))
    return h


def _hash_sums_np(seed: int, idx, ndraw: int, mode: str):
    """CPU path of the counter hash (numpy uint32, threaded over blocks)."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor

    idx = np.ascontiguousarray(idx, dtype=np.int64)
    flat = idx.reshape(-1)
    out = np.empty(flat.shape, dtype=np.float32 if mode != "bern" else np.uint32)
    bases = [fmix32_int((seed + k * GOLDEN) & M32) for k in range(ndraw)]

    def work(a, b):
        x = flat[a:b]
        lo = (x & M32).astype(np.uint32)
        hi = (x >> 32).astype(np.uint32)
        acc = np.zeros(b - a, dtype=np.int64) if mode == "normal" else None
        for k in range(ndraw):
            t = _fmix32_np(hi ^ np.uint32(bases[k]))
            h = _fmix32_np(lo + t)
            if mode == "normal":
                acc += (h & np.uint32(0xFFFF)).astype(np.int64) + (h >> np.uint32(16)).astype(np.int64)
            elif mode == "uniform":
                out[a:b] = (h >> np.uint32(8)).astype(np.float32) / np.float32(16777216.0)
            else:
                out[a:b] = h
        if mode == "normal":
            out[a:b] = (acc - 393210).astype(np.float32) / np.float32(65536.0)

    n = flat.shape[0]
    blk = 1 << 20
    if n <= blk:
        work(0, n)
    else:
        with ThreadPoolExecutor(max_workers=min(16, (n + blk - 1) // blk)) as ex:
            list(ex.map(lambda a: work(a, min(n, a + blk)), range(0, n, blk)))
    return out.reshape(idx.shape)


def _draw_hashes(seed: int, idx: torch.Tensor, ndraw: int) -> List[torch.Tensor]:
    """``ndraw`` independent 32-bit hashes of each int64 index (counter mode),
    as int64 tensors on the index's device."""
    lo = idx & M32
    hi = idx >> 32
    out = []
    for k in range(ndraw):
        base = fmix32_int((seed + k * GOLDEN) & M32)
        out.append(fmix32((lo + fmix32(hi ^ base)) & M32))
    return out


def _use_numpy(idx: torch.Tensor, force_torch: bool) -> bool:
    return idx.device.type == "cpu" and not force_torch


def normal_f32(seed: int, idx: torch.Tensor, force_torch: bool = False) -> torch.Tensor:
    """Irwin-Hall(12) standard-normal stand-in, exact in float32."""
    if _use_numpy(idx, force_torch):
        return torch.from_numpy(_hash_sums_np(seed, idx.numpy(), 6, "normal"))
    s = torch.zeros_like(idx)
    for h in _draw_hashes(seed, idx, 6):
        s += (h & 0xFFFF) + (h >> 16)
    return (s - 393210).to(torch.float32) / 65536.0


def uniform01_f32(seed: int, idx: torch.Tensor, force_torch: bool = False) -> torch.Tensor:
    """Uniform in [0, 1) with 24 random bits (exact in float32)."""
    if _use_numpy(idx, force_torch):
        return torch.from_numpy(_hash_sums_np(seed, idx.numpy(), 1, "uniform"))
    (h,) = _draw_hashes(seed, idx, 1)
    return (h >> 8).to(torch.float32) / 16777216.0


def bernoulli(seed: int, idx: torch.Tensor, per_10000: int, force_torch: bool = False) -> torch.Tensor:
    if _use_numpy(idx, force_torch):
        h = torch.from_numpy(_hash_sums_np(seed, idx.numpy(), 1, "bern").astype("int64"))
        return (h % 10000) < per_10000
    (h,) = _draw_hashes(seed, idx, 1)
    return (h % 10000) < per_10000


def _index_range(start: int, count: int, device) -> torch.Tensor:
    return torch.arange(start, start + count, dtype=torch.int64, device=device)


# ----------------------------------------------------------------------------
# Workload descriptions
# ----------------------------------------------------------------------------
@dataclass
class Workload:
    """One verification-round workload (one Cohort of requests)."""

    cfg_id: int
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    chunk_tokens: int
    hist_len: List[int]
    num_cand: List[int]
    layers: int = 1
    kscale: bool = False          # per-(request, kv head, channel) K scale U[0.5, 2]
    outlier_per_10000: int = 0    # K rows (token, kv head) scaled x8
    seed_base: int = 0

    # -- shapes --------------------------------------------------------------
    @property
    def B(self) -> int:
        return len(self.hist_len)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def total_rows(self) -> int:
        return sum(self.num_cand)

    def row_offsets(self) -> List[int]:
        off, acc = [], 0
        for n in self.num_cand:
            off.append(acc)
            acc += n
        return off

    @property
    def num_chunks(self) -> int:
        return max((c + self.chunk_tokens - 1) // self.chunk_tokens for c in self.hist_len) if self.hist_len else 0

    def chunk_lens(self, j: int) -> List[int]:
        """Tokens of each request in history chunk j (partial last chunk)."""
        S = self.chunk_tokens
        return [max(0, min(S, c - j * S)) for c in self.hist_len]

    def token_bytes(self) -> int:
        """K+V bytes of one token of one layer (all KV heads, bf16)."""
        return self.num_kv_heads * self.head_dim * 2 * 2

    def history_kv_bytes(self) -> int:
        return sum(self.hist_len) * self.token_bytes()

    def algorithmic_kv_bytes(self) -> int:
        """Sum_b (C_b + n_b) * Hkv * d * 2 (K,V) * 2 B."""
        return (sum(self.hist_len) + sum(self.num_cand)) * self.token_bytes()

    # -- seeds ---------------------------------------------------------------
    def _seed(self, layer: int, b: int, tid: int) -> int:
        return seed_key(self.seed_base, self.cfg_id, layer, b, tid)

    def _kv_layer(self, layer: int) -> int:
        # every layer of a multi-layer round shares one history (host memory
        # holds one layer); queries differ per layer
        return 0

    # -- element generators ----------------------------------------------------
    def _kscale_vec(self, b: int, layer: int, device) -> torch.Tensor:
        """[Hkv, d] float32 scale in [0.5, 2]."""
        n = self.num_kv_heads * self.head_dim
        u = uniform01_f32(self._seed(self._kv_layer(layer), b, TID_KSCALE), _index_range(0, n, device))
        return (u * 1.5 + 0.5).view(self.num_kv_heads, self.head_dim)

    def _gen_k(self, b: int, layer: int, tid: int, out_tid: int, t0: int, t1: int,
               heads: Optional[Sequence[int]], device) -> torch.Tensor:
        Hkv, d = self.num_kv_heads, self.head_dim
        kl = self._kv_layer(layer)
        hs = list(range(Hkv)) if heads is None else list(heads)
        t = torch.arange(t0, t1, dtype=torch.int64, device=device)
        g = torch.tensor(hs, dtype=torch.int64, device=device)
        c = torch.arange(d, dtype=torch.int64, device=device)
        idx = (t.view(-1, 1, 1) * Hkv + g.view(1, -1, 1)) * d + c.view(1, 1, -1)
        x = normal_f32(self._seed(kl, b, tid), idx)
        if self.kscale:
            s = self._kscale_vec(b, layer, device)[g]
            x = x * s.view(1, len(hs), d)
        kb = x.to(torch.bfloat16)
        if self.outlier_per_10000:
            ridx = t.view(-1, 1) * Hkv + g.view(1, -1)
            m = bernoulli(self._seed(kl, b, out_tid), ridx, self.outlier_per_10000)
            kb = torch.where(m.unsqueeze(-1), kb * 8, kb)
        return kb

    def _gen_v(self, b: int, layer: int, tid: int, t0: int, t1: int,
               heads: Optional[Sequence[int]], device) -> torch.Tensor:
        Hkv, d = self.num_kv_heads, self.head_dim
        hs = list(range(Hkv)) if heads is None else list(heads)
        t = torch.arange(t0, t1, dtype=torch.int64, device=device)
        g = torch.tensor(hs, dtype=torch.int64, device=device)
        c = torch.arange(d, dtype=torch.int64, device=device)
        idx = (t.view(-1, 1, 1) * Hkv + g.view(1, -1, 1)) * d + c.view(1, 1, -1)
        return normal_f32(self._seed(self._kv_layer(layer), b, tid), idx).to(torch.bfloat16)

    # -- public tensors (bf16) --------------------------------------------------
    def q(self, b: int, layer: int = 0, device="cpu") -> torch.Tensor:
        """[n_b, Hq, d]"""
        n = self.num_cand[b] * self.num_q_heads * self.head_dim
        x = normal_f32(self._seed(layer, b, TID_Q), _index_range(0, n, device))
        return x.to(torch.bfloat16).view(self.num_cand[b], self.num_q_heads, self.head_dim)

    def q_all(self, layer: int = 0, device="cpu") -> torch.Tensor:
        """[sum n_b, Hq, d] packed in request order."""
        return torch.cat([self.q(b, layer, device) for b in range(self.B)], 0)

    def k_hist(self, b: int, t0: int = 0, t1: Optional[int] = None, heads=None,
               layer: int = 0, device="cpu") -> torch.Tensor:
        """[t1-t0, Hkv or len(heads), d] history keys of request b."""
        t1 = self.hist_len[b] if t1 is None else t1
        return self._gen_k(b, layer, TID_KH, TID_OUT_H, t0, t1, heads, device)

    def v_hist(self, b: int, t0: int = 0, t1: Optional[int] = None, heads=None,
               layer: int = 0, device="cpu") -> torch.Tensor:
        t1 = self.hist_len[b] if t1 is None else t1
        return self._gen_v(b, layer, TID_VH, t0, t1, heads, device)

    def k_cand(self, b: int, heads=None, layer: int = 0, device="cpu") -> torch.Tensor:
        """[n_b, Hkv, d] candidate (Speculative Frontier) keys."""
        return self._gen_k(b, layer, TID_KC, TID_OUT_C, 0, self.num_cand[b], heads, device)

    def v_cand(self, b: int, heads=None, layer: int = 0, device="cpu") -> torch.Tensor:
        return self._gen_v(b, layer, TID_VC, 0, self.num_cand[b], heads, device)

    def k_cand_all(self, layer: int = 0, device="cpu") -> torch.Tensor:
        return torch.cat([self.k_cand(b, layer=layer, device=device) for b in range(self.B)], 0)

    def v_cand_all(self, layer: int = 0, device="cpu") -> torch.Tensor:
        return torch.cat([self.v_cand(b, layer=layer, device=device) for b in range(self.B)], 0)

    def chunk_kv(self, j: int, layer: int = 0, device="cpu", out_k=None, out_v=None, head_major: bool = False,
                 kv_interleaved: bool = False) -> Tuple[torch.Tensor, torch.Tensor]:
        """History chunk j packed in request order: [sum_b len_bj, Hkv, d] each
        (token-major), or [Hkv, sum_b len_bj, d] with ``head_major``.  With
        ``kv_interleaved`` both live in one [Hkv, sum_b len_bj, 2, d] buffer
        (a token's K row, then its V row) and K, V are views of it."""
        if kv_interleaved:
            k, v = self.chunk_kv(j, layer, device)
            kv = torch.stack((k.transpose(0, 1), v.transpose(0, 1)), dim=2).contiguous()
            return kv[:, :, 0], kv[:, :, 1]
        if head_major:
            k, v = self.chunk_kv(j, layer, device)
            return k.transpose(0, 1).contiguous(), v.transpose(0, 1).contiguous()
        lens = self.chunk_lens(j)
        tot = sum(lens)
        shape = (tot, self.num_kv_heads, self.head_dim)
        k = torch.empty(shape, dtype=torch.bfloat16, device=device) if out_k is None else out_k
        v = torch.empty(shape, dtype=torch.bfloat16, device=device) if out_v is None else out_v
        off = 0
        S = self.chunk_tokens
        for b, n in enumerate(lens):
            if n == 0:
                continue
            # generate in slices to bound temporary memory
            step = max(1, (1 << 22) // (self.num_kv_heads * self.head_dim))
            for s0 in range(0, n, step):
                s1 = min(n, s0 + step)
                k[off + s0: off + s1] = self.k_hist(b, j * S + s0, j * S + s1, layer=layer, device=device)
                v[off + s0: off + s1] = self.v_hist(b, j * S + s0, j * S + s1, layer=layer, device=device)
            off += n
        return k, v


def _log_uniform_lengths(cfg_id: int, B: int, lo: int, hi: int) -> Tuple[List[int], List[int]]:
    """Per-request history length log-U[lo, hi] and candidate count U{1..8}."""
    lens, cands = [], []
    for b in range(B):
        h1 = fmix32_int(seed_key(0, cfg_id, 0, b, TID_LEN))
        h2 = fmix32_int(h1 ^ 0xA5A5A5A5)
        u = h1 / 4294967296.0
        c = int(round(math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))))
        lens.append(min(hi, max(lo, c)))
        cands.append(1 + (h2 % 8))
    return lens, cands


def workload(cfg_id: int) -> Workload:
    """The five workload configurations (seeded synthetic inputs of the paper's shapes)."""
    if cfg_id == 1:
        return Workload(1, "tiny-1req-8q2kv-4096ctx", 8, 2, 128, 1024, [4096], [5])
    if cfg_id == 2:
        return Workload(2, "7-8B-layer-1req-32q8kv-16384ctx-kscale", 32, 8, 128, 2048, [16384], [5],
                        kscale=True)
    if cfg_id == 3:
        return Workload(3, "batch16-32q8kv-32768ctx-6cand", 32, 8, 128, 4096, [32768] * 16, [6] * 16)
    if cfg_id == 4:
        lens, cands = _log_uniform_lengths(4, 64, 2048, 65536)
        return Workload(4, "ragged64-32q8kv-logU2048-65536-cand1to8", 32, 8, 128, 4096, lens, cands)
    if cfg_id == 5:
        return Workload(5, "fulldepth-36L-batch32-32q8kv-131072ctx-8cand-outliers", 32, 8, 128, 8192,
                        [131072] * 32, [8] * 32, layers=36, outlier_per_10000=100)
    raise ValueError(f"unknown config {cfg_id}")


def custom(hist_len: Sequence[int], num_cand: Sequence[int], num_q_heads: int = 8, num_kv_heads: int = 2,
           head_dim: int = 128, chunk_tokens: int = 1024, seed_base: int = 1, kscale: bool = False,
           outlier_per_10000: int = 0, cfg_id: int = 100) -> Workload:
    """A small seeded workload for tests."""
    return Workload(cfg_id, "custom", num_q_heads, num_kv_heads, head_dim, chunk_tokens,
                    list(hist_len), list(num_cand), kscale=kscale,
                    outlier_per_10000=outlier_per_10000, seed_base=seed_base)


def bf16_bits(t: torch.Tensor):
    """uint16 numpy view of a bf16 tensor (moved to the CPU)."""
    import numpy as np
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)
