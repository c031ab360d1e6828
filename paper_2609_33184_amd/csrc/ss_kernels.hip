// gfx950 (MI355X) kernels of chunk-streamed speculative-verification attention.
//
// Paper Sec. 4.2: every history chunk (K_j, V_j) is read once for the whole
// query group of a request (all n_b candidates x all G query heads sharing a
// KV head); the chunk-local online-softmax state (Eq. 13) is merged into the
// running state with the rescaled update of Eq. 14; the Speculative Frontier
// is attended with the causal candidate mask; O = a / l (Eq. 17).
//
// Layout and precision
//   * scores are kept in the log2 domain: x = sigma * log2(e) * q.k, so every
//     exponential is one v_exp_f32; the state's m is in that domain as well.
//   * all accumulation is fp32.  In the MFMA path the softmax weights P
//     (fp32) are split into bf16 hi + lo parts and both are multiplied with V
//     (two bf16 MFMAs), which keeps P to ~2^-16 relative; rounding P once to
//     bf16 would cost ~1.6e-3 relative L2 error.  The denominator l sums the
//     fp32 weights themselves, which hi + lo carry to that precision.
//   * a running state is split into kNumSlots slots per query row so that
//     several workgroups can fold disjoint token ranges of one chunk into the
//     same row without atomics; the finalize kernel merges the slots.
#include <hip/hip_runtime.h>

#include "ss_kernels.h"

#include <cstddef>
#include <cstring>

#include <math.h>

#include <mutex>
#include <type_traits>

namespace ss {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kAwPitch = 132;  // floats per row of a wave's partial accumulator
constexpr int kBufferFlags = 0x00020000;   // buffer resource word 3: 32-bit data format, raw offsets
// Cache policy of the history K/V loads: non-temporal.  Every history byte
// is read once per round, so the streaming loads should not displace
// reusable lines; measured on MI355X, this took config 3's round from 378 to
// 354 us and config 4's from 786 to 743 us (means over 40 rounds).
constexpr int kStreamLoad = 2;
constexpr int kMaxDevices = 64;   // devices whose scratch address is cached

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Sum over the 16 lanes of a DPP row; every lane of the row gets the total.
__device__ __forceinline__ float row16_sum(float x) {
  int v;
  v = __builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xf, 0xf, false);  // quad_perm [1,0,3,2]
  x += __int_as_float(v);
  v = __builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xf, 0xf, false);  // quad_perm [2,3,0,1]
  x += __int_as_float(v);
  v = __builtin_amdgcn_mov_dpp(__float_as_int(x), 0x124, 0xf, 0xf, false); // row_ror:4
  x += __int_as_float(v);
  v = __builtin_amdgcn_mov_dpp(__float_as_int(x), 0x128, 0xf, 0xf, false); // row_ror:8
  x += __int_as_float(v);
  return x;
}

// Max / sum across the four 16-lane groups of a wave (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float xgroup_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}
__device__ __forceinline__ float xgroup_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

template <typename P>
__device__ __forceinline__ int global_row(const P &p, int q_row0, int g, int r) {
  // local row r of (request, kv head g) -> packed query row (off_b + i) * Hq + h
  const int i = r / p.G;
  const int h = g * p.G + (r - i * p.G);
  return (q_row0 + i) * p.Hq + h;
}

// ---------------------------------------------------------------------------
// Workgroup epilogue shared by the chunk kernels: the kWaves waves have left
// their partial states in LDS (aw[w][row][kAwPitch], mw[w][row], lw[w][row],
// all relative to their own maxima); combine them (Eq. 14 over the waves) and
// fold the result into the item's slot of the running state (Eq. 14 again).
// ---------------------------------------------------------------------------
template <int ROWS, typename P>
__device__ __forceinline__ void fold_into_slot(const P &p, const Item &it, int q_row0, int g, int M, int tx,
                                               const float *aw, const float *mw, const float *lw) {
  // SEGS threads per row (the largest power of two with SEGS * ROWS <= 256,
  // at most 32), SEGLEN (a multiple of 4) values each
  constexpr int SEGS = (256 / ROWS) >= 32 ? 32 : (256 / ROWS) >= 16 ? 16 : (256 / ROWS) >= 8 ? 8 : 4;
  constexpr int SEGLEN = kHeadDim / SEGS;
  static_assert(SEGLEN % 4 == 0 && SEGS * ROWS <= 256, "fold layout");
  const int r = tx / SEGS;
  const int seg = tx % SEGS;
  if (r >= M) return;
  float mwv[kWaves];
  float mstar = kNegInf;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    mwv[w] = mw[w * ROWS + r];
    mstar = fmaxf(mstar, mwv[w]);
  }
  float f[kWaves];
  float lstar = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    f[w] = exp2_fast(mwv[w] - mstar);   // a wave without tokens has m = -inf -> 0
    lstar += f[w] * lw[w * ROWS + r];
  }
  float a[SEGLEN];
#pragma unroll
  for (int c = 0; c < SEGLEN; ++c) a[c] = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float *src = aw + (w * ROWS + r) * kAwPitch + seg * SEGLEN;
#pragma unroll
    for (int c = 0; c < SEGLEN; c += 4) {
      const f32x4_t x = *reinterpret_cast<const f32x4_t *>(src + c);
      a[c] += f[w] * x[0];
      a[c + 1] += f[w] * x[1];
      a[c + 2] += f[w] * x[2];
      a[c + 3] += f[w] * x[3];
    }
  }
  const size_t idx = (size_t)it.slot * p.st.R + global_row(p, q_row0, g, r);
  float *ap = p.st.a + idx * kHeadDim + seg * SEGLEN;
  if (it.flags & kSlotFresh) {       // first write of this slot in the round: store
#pragma unroll
    for (int c = 0; c < SEGLEN; c += 4)
      *reinterpret_cast<f32x4_t *>(ap + c) = f32x4_t{a[c], a[c + 1], a[c + 2], a[c + 3]};
    if (seg == 0) {
      p.st.m[idx] = mstar;
      p.st.l[idx] = lstar;
    }
  } else {
    const float ms = p.st.m[idx];
    const float mn = fmaxf(ms, mstar);
    const float alpha = exp2_fast(ms - mn);
    const float beta = exp2_fast(mstar - mn);
#pragma unroll
    for (int c = 0; c < SEGLEN; c += 4) {
      f32x4_t o = *reinterpret_cast<const f32x4_t *>(ap + c);
      o[0] = alpha * o[0] + beta * a[c];
      o[1] = alpha * o[1] + beta * a[c + 1];
      o[2] = alpha * o[2] + beta * a[c + 2];
      o[3] = alpha * o[3] + beta * a[c + 3];
      *reinterpret_cast<f32x4_t *>(ap + c) = o;
    }
    if (seg == 0) {
      p.st.m[idx] = mn;
      p.st.l[idx] = alpha * p.st.l[idx] + beta * lstar;
    }
  }
}

// ---------------------------------------------------------------------------
// MFMA chunk body.  Workgroup = (kv head, unit); 4 waves; wave w takes the
// 32-token tiles w, w+4, ... of the unit's chain of items (one request's
// token ranges, possibly from several chunks, attended as one sequence).
// Per tile:
//   K, V tiles -> LDS        coalesced 16-byte loads: one instruction reads 4
//                            whole 256-byte token rows (16 lanes per row)
//   S^T[t][row] = K Q^T      v_mfma_f32_16x16x32_bf16, A = K (16 tokens x 32 d,
//                            one ds_read_b128 per k-step), B = Q^T (from an
//                            LDS copy of the group's query rows)
//   online softmax per row   (row = lane % 16; the four lane groups share it)
//   O^T[d][row] += V^T P^T   A = V^T via the LDS transpose read, B = P^T
//                            straight from the S accumulators (hi and lo parts)
// Lane l: lr = l % 16, lq = l / 16.  In the S tile lane (lr, lq) holds
// tokens 16u + 4*lq + r (u = 0,1; r = 0..3) of row lr; in O it holds
// d = 16*db + 4*lq + r.  The reduction index of both MFMAs is permuted so
// every operand is contiguous: for QK^T lane group lq, k-step s covers the
// d-chunk 4*s + lq (8 values); for PV lane group lq covers tokens
// {4lq..4lq+3, 16+4lq..16+4lq+3}, exactly the S values the lane holds.
//
// LDS tiles are 32 rows of 256 bytes; 16-byte chunk c of token row t is
// stored at chunk position c ^ (t & 15) for K and c ^ 2(t & 7) for V, which
// makes the row-wise stores, the K operand reads (16 rows, same chunk) and
// the transpose reads of V (8 rows, 32 bytes each per half-wave) free of
// bank conflicts.
//
// ds_read_b64_tr_b16: within each 16-lane group, result lane i, element e is
// element (i % 4) of what source lane 4e + i/4 addressed.  Source lane j of
// group lq addresses row 4lq + j/4 (+16 for the second half), columns
// 16db + 4(j%4) .. +3, so result lane i receives V[4lq + e][16db + i].
//
// Each wave keeps the next tile's K and V in flight in registers for the
// whole compute of the current tile: a tile's loads are written to LDS at
// the top of the iteration and the next loads are issued right after.  The
// last tile is peeled so the in-loop prefetch is unconditional (a
// conditional load would make the compiler wait for every outstanding load).
// ---------------------------------------------------------------------------
constexpr int kRowBytes = kHeadDim * 2;          // 256
constexpr int kTileBytes = kTile * kRowBytes;    // 8 KiB per K or V tile

__device__ __forceinline__ int tiles_of(const Item &it) { return (it.tok_count + kTile - 1) / kTile; }

// Chunk-table index of an item.  The item is read as whole dwords: a
// byte-sized read of a kernel argument becomes a vector memory load, and the
// wait for it would also wait for every K/V load in flight.
__device__ __forceinline__ int item_chunk(const Item &it) {
  uint32_t w[4];
  __builtin_memcpy(w, &it, sizeof w);
  return (int)((w[3] >> 8) & 0xffu);
}
static_assert(offsetof(Item, chunk) == 13, "Item layout");

// Buffer resource over item `it`'s rows of KV head g in the chunk that
// starts at `base` (K or V) with head_stride `hs` elements: loads past the
// item's last token return zero, so no clamping is needed.  Offsets are
// 32-bit (the host keeps an item below 2^31 bytes).
template <typename P>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t item_rsrc_at(const P &p, const Item &it, const uint16_t *base,
                                                               uint64_t hs, int g) {
  const uint32_t nrec = (uint32_t)(it.tok_count - 1) * (p.tok_stride * 2) + kRowBytes;
  const size_t first = (size_t)it.tok_begin * p.tok_stride + (size_t)g * hs;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(base + first), (short)0, (int)nrec, kBufferFlags);
}
// The same through the launch's chunk table `tab` (p.k or p.v).
template <typename P>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t item_rsrc(const P &p, const Item &it, int chunk, int g,
                                                            const uint16_t *const *tab) {
  return item_rsrc_at(p, it, tab[chunk], p.head_stride[chunk], g);
}

// A unit's first item and its chunk-table entries.  The item is read as
// whole dwords, and the item and the three entries are forced into
// registers at one point, so their loads go out together (the chunk comes
// from the unit record, not from the item) and are waited for once.
struct FirstItem {
  Item it;
  const uint16_t *k, *v;
  uint64_t hs;
};
template <typename P>
__device__ __forceinline__ FirstItem load_first_item(const P &p, const UnitRec &ur) {
  const int i0 = unit_i0(ur.word), c = unit_chunk(ur.word);
  uint32_t w[4];
  __builtin_memcpy(w, &p.items[i0], sizeof w);
  const uint16_t *k = p.k[c];
  const uint16_t *v = p.v[c];
  uint64_t hs = p.head_stride[c];
  asm volatile("" : "+s"(w[0]), "+s"(w[1]), "+s"(w[2]), "+s"(w[3]), "+s"(k), "+s"(v), "+s"(hs));
  FirstItem f;
  __builtin_memcpy(&f.it, w, sizeof w);
  f.k = k;
  f.v = v;
  f.hs = hs;
  return f;
}

// A unit's tiles are numbered across its chain of items (item 0's tiles
// first).  The cursor maps a global tile T to (item k, k's first global
// tile); it only moves forward, and never past the chain's last item.
struct TileCursor {
  int k = 0;
  int base = 0;
};
template <typename P>
__device__ __forceinline__ void seek(const P &p, int i0, int nit, TileCursor &c, int T) {
  while (c.k + 1 < nit && T - c.base >= tiles_of(p.items[i0 + c.k])) {
    c.base += tiles_of(p.items[i0 + c.k]);
    ++c.k;
  }
}

// Resources and item-local token base of the next tile a wave loads.
struct NextTile {
  __amdgpu_buffer_rsrc_t krs, vrs;
  int tb;
};

template <int RB>
struct MfmaLds {
  static constexpr int kQBytes = RB * 16 * kRowBytes;               // Q rows, shared by the waves
  static constexpr int kStageBytes = kQBytes + kWaves * 2 * kTileBytes;
  static constexpr int kMergeBytes = kWaves * RB * 16 * (kAwPitch + 2) * 4;
  static constexpr int kBytes = kStageBytes > kMergeBytes ? kStageBytes : kMergeBytes;
};

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ s16x4_t lds_read_tr16(const unsigned char *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4_t *)(reinterpret_cast<uintptr_t>(p)));
}

template <int RB, typename P>
__device__ __forceinline__ void mfma_unit(const P &p, unsigned char *smem, const UnitRec &ur, int tx, int g, int nxt) {
  const int w = __builtin_amdgcn_readfirstlane(tx >> 6);   // wave-uniform
  const int lane = tx & 63;
  const int lr = lane & 15;
  const int lq = lane >> 4;
  const int i0 = unit_i0(ur.word), nit = unit_nit(ur.word);
  const int q_row0 = ur.q_row0;
  const int M = ur.n_cand * p.G;
  const int ntiles = (int)ur.ntiles;

  float m_run[RB], l_run[RB];
  f32x4_t acc[RB][8];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_run[rb] = kNegInf;
    l_run[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[rb][db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  const uint32_t stride_b = p.tok_stride * 2;                      // bytes between tokens
  const uint32_t voff = lq * stride_b + 16 * lr;                     // token lq, chunk lr
  unsigned char *qs = smem;
  unsigned char *ks = smem + MfmaLds<RB>::kQBytes + w * (2 * kTileBytes);
  unsigned char *vs = ks + kTileBytes;
  const float sl2 = p.scale_log2;

  u32x4_t kr[8], vr[8];
  // coalesced loads: instruction i reads tokens tb + 4i + lq, chunk lr.  The
  // whole offset goes in the VGPR operand: the buffer range check covers the
  // VGPR (and immediate) offset only, not the scalar one, and rows past the
  // item must come back as zeros rather than read beyond the buffer.
  auto load_kv = [&](const NextTile &nx) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      kr[i] = __builtin_amdgcn_raw_buffer_load_b128(nx.krs, voff + (uint32_t)(nx.tb + 4 * i) * stride_b, 0, kStreamLoad);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      vr[i] = __builtin_amdgcn_raw_buffer_load_b128(nx.vrs, voff + (uint32_t)(nx.tb + 4 * i) * stride_b, 0, kStreamLoad);
  };
  // K operand read: row 16u + lr, chunk 4s + lq at position (4s + lq) ^ lr
  // V transpose read: row 4lq + lr/4 (+16), chunk 2db + (lr&3)/2, half lr&1
  const int vrow = 4 * lq + (lr >> 2);
  const int vrd = vrow * kRowBytes + 8 * (lr & 1);
  const int vsw = 2 * (vrow & 7);
  const int vc0 = (lr & 3) >> 1;

  // one tile: tokens [tb, tb + 32) of an item with `count` tokens, already in
  // kr / vr; `nx` is the tile to load next (unused for a wave's last tile)
  auto tile = [&](int tb, int count, auto prefetch, const NextTile &nx) {
    constexpr bool kPrefetch = decltype(prefetch)::value;
    // stage K(i), V(i) in LDS, then issue the loads of the next tile
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = 4 * i + lq;
      *reinterpret_cast<u32x4_t *>(ks + t * kRowBytes + 16 * (lr ^ (t & 15))) = kr[i];
      *reinterpret_cast<u32x4_t *>(vs + t * kRowBytes + 16 * (lr ^ (2 * (t & 7)))) = vr[i];
    }
    if constexpr (kPrefetch) load_kv(nx);
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch here, ahead of the math

    // S^T = K Q^T
    f32x4_t sacc[2][RB];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      bf16x8_t kop[4];
      const int t = 16 * u + lr;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        kop[s] = *reinterpret_cast<const bf16x8_t *>(ks + t * kRowBytes + 16 * ((4 * s + lq) ^ lr));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        f32x4_t c = {0.f, 0.f, 0.f, 0.f};
        const unsigned char *qrow = qs + (16 * rb + lr) * kRowBytes;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const bf16x8_t qop = *reinterpret_cast<const bf16x8_t *>(qrow + 16 * ((4 * s + lq) ^ lr));
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[s], qop, c, 0, 0, 0);
        }
        sacc[u][rb] = c;
      }
    }

    __builtin_amdgcn_sched_barrier(0);   // phases stay apart: bounded register pressure

    // online softmax (Eq. 13 local terms merged per Eq. 14 into the wave's state)
    bf16x8_t phi[RB], plo[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // raw scores up to the exponent (sigma log2(e) > 0 commutes with the
      // maximum); only an item's last, partial tile needs the token mask
      float x[8];
      float mx = kNegInf;
      if (tb + kTile <= count) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            x[4 * u + r] = sacc[u][rb][r];
            mx = fmaxf(mx, sacc[u][rb][r]);
          }
      } else {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int t = tb + 16 * u + 4 * lq + r;
            const float v = t < count ? sacc[u][rb][r] : kNegInf;
            x[4 * u + r] = v;
            mx = fmaxf(mx, v);
          }
      }
      const float mn = fmaxf(m_run[rb], xgroup_max(mx) * sl2);
      // Eq. 14's rescale, only when some row's maximum rose (elsewhere the
      // factor is exactly 1)
      if (__builtin_amdgcn_ballot_w64(mn > m_run[rb])) {
        const float alpha = exp2_fast(m_run[rb] - mn);
        l_run[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < 8; ++db) acc[rb][db] *= alpha;
        m_run[rb] = mn;
      }
      float ls = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pe = exp2_fast(__builtin_fmaf(x[e], sl2, -mn));
        const __bf16 h = (__bf16)pe;
        const float hf = (float)h;
        const __bf16 lo = (__bf16)(pe - hf);
        phi[rb][e] = h;
        plo[rb][e] = lo;
        ls += pe;
      }
      l_run[rb] += ls;
    }

    __builtin_amdgcn_sched_barrier(0);

    // O^T += V^T P^T  (hi and lo parts of P)
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const int off = vrd + 16 * ((2 * db + vc0) ^ vsw);
      const s16x4_t v0 = lds_read_tr16(vs + off);
      const s16x4_t v1 = lds_read_tr16(vs + off + 16 * kRowBytes);
      const bf16x8_t vop = __builtin_bit_cast(
          bf16x8_t, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        acc[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, phi[rb], acc[rb][db], 0, 0, 0);
        acc[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, plo[rb], acc[rb][db], 0, 0, 0);
      }
    }
  };

  // Q rows of this (request, kv head) -> LDS, chunk c of row r at c ^ (r & 15);
  // rows >= M are zero.  The Q^T operand (B[k = d][j = row]) of lane (lr, lq),
  // k-step s, is row lr's d-chunk 4s + lq.  The query loads are issued first,
  // then the first K/V tile, so staging Q waits only for the query rows.
  // They are buffer loads over the whole Q tensor: a padding row (r >= M)
  // gets an offset past the end and reads zero, so no load sits behind a
  // branch (whose merge with the zero default would force an early wait).
  constexpr int kQPerThread = RB * 16 * 16 / 256;
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t *>(p.q), (short)0, (int)((uint32_t)p.st.R * kRowBytes), kBufferFlags);
  u32x4_t qv[kQPerThread];
#pragma unroll
  for (int e = 0; e < kQPerThread; ++e) {
    const int c = tx + 256 * e, r = c >> 4, ch = c & 15;
    const uint32_t qoff = r < M ? (uint32_t)global_row(p, q_row0, g, r) * kRowBytes + 16 * ch : 0x80000000u;
    qv[e] = __builtin_amdgcn_raw_buffer_load_b128(qrs, qoff, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);   // the query loads go out before the wait for the first item
  // wave w takes the chain's tiles T = w, w + 4, ...  The first tile's loads
  // are issued unconditionally (a wave without tiles loads through an empty
  // resource, which reads nothing), so the wait for the query rows below
  // does not have to include them.  The first item (slot and flags of the
  // whole chain) comes with its chunk; a wave whose first tile lies in a
  // later item of the chain rebuilds its resources from that item.
  const FirstItem fi = load_first_item(p, ur);
  const Item &it = fi.it;
  // The workgroup's next unit of its own list (nxt >= 0): its first item's
  // resources, read now, so that each wave can bring the lines of its first
  // tile of that unit into the L2 cache during its last tile of this one.
  __amdgpu_buffer_rsrc_t wkrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.q), (short)0, 0, kBufferFlags);
  __amdgpu_buffer_rsrc_t wvrs = wkrs;
  if (nxt >= 0) {
    const UnitRec un = p.units[nxt];
    const Item in0 = p.items[unit_i0(un.word)];
    const int cn = unit_chunk(un.word);
    wkrs = item_rsrc(p, in0, cn, g, p.k);
    wvrs = item_rsrc(p, in0, cn, g, p.v);
  }
  int T = w;
  TileCursor cur;
  NextTile nx;
  const __amdgpu_buffer_rsrc_t empty =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.q), (short)0, 0, kBufferFlags);
  const bool has_tile = T < ntiles;
  nx.krs = has_tile ? item_rsrc_at(p, it, fi.k, fi.hs, g) : empty;
  nx.vrs = has_tile ? item_rsrc_at(p, it, fi.v, fi.hs, g) : empty;
  nx.tb = T * kTile;
  if (has_tile && T >= tiles_of(it)) {
    seek(p, i0, nit, cur, T);
    const Item ic = p.items[i0 + cur.k];
    nx.krs = item_rsrc(p, ic, item_chunk(ic), g, p.k);
    nx.vrs = item_rsrc(p, ic, item_chunk(ic), g, p.v);
    nx.tb = (T - cur.base) * kTile;
  }
  load_kv(nx);
#pragma unroll
  for (int e = 0; e < kQPerThread; ++e) {
    const int c = tx + 256 * e, r = c >> 4, ch = c & 15;
    *reinterpret_cast<u32x4_t *>(qs + r * kRowBytes + 16 * (ch ^ (r & 15))) = qv[e];
  }
  __syncthreads();

  if (T < ntiles) {
    int tb = nx.tb;
    int count = cur.k == 0 ? it.tok_count : p.items[i0 + cur.k].tok_count;
    for (; T + kWaves < ntiles; T += kWaves) {
      const int kprev = cur.k;
      seek(p, i0, nit, cur, T + kWaves);
      if (cur.k != kprev) {
        const Item in = p.items[i0 + cur.k];
        nx.krs = item_rsrc(p, in, item_chunk(in), g, p.k);
        nx.vrs = item_rsrc(p, in, item_chunk(in), g, p.v);
      }
      nx.tb = (T + kWaves - cur.base) * kTile;
      tile(tb, count, std::integral_constant<bool, true>{}, nx);
      tb = nx.tb;
      count = p.items[i0 + cur.k].tok_count;
    }
    // one 4-byte read per 128-byte line of this wave's first tile of the
    // next unit (tokens 32w .. 32w+31 of its first item, K and V; reads
    // past the item return zero without touching memory), at the default
    // cache policy so the lines stay in L2; the values are only kept alive
    // until the last tile is done, where the wait for them is free
    uint32_t warm_k = 0, warm_v = 0;
    if (nxt >= 0) {
      const uint32_t wo = (uint32_t)(kTile * w + (lane >> 1)) * stride_b + 128u * (uint32_t)(lane & 1);
      warm_k = __builtin_amdgcn_raw_buffer_load_b32(wkrs, wo, 0, 0);
      warm_v = __builtin_amdgcn_raw_buffer_load_b32(wvrs, wo, 0, 0);
    }
    tile(tb, count, std::integral_constant<bool, false>{}, nx);
    asm volatile("" ::"v"(warm_k), "v"(warm_v));
  }

  // wave partials -> LDS
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) l_run[rb] = xgroup_sum(l_run[rb]);
  __syncthreads();
  float *aw = reinterpret_cast<float *>(smem);
  float *mw = aw + kWaves * RB * 16 * kAwPitch;
  float *lw = mw + kWaves * RB * 16;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    float *row = aw + (w * RB * 16 + rb * 16 + lr) * kAwPitch + 4 * lq;
#pragma unroll
    for (int db = 0; db < 8; ++db) *reinterpret_cast<f32x4_t *>(row + 16 * db) = acc[rb][db];
    if (lq == 0) {
      mw[w * RB * 16 + rb * 16 + lr] = m_run[rb];
      lw[w * RB * 16 + rb * 16 + lr] = l_run[rb];
    }
  }
  __syncthreads();
  fold_into_slot<RB * 16>(p, it, q_row0, g, M, tx, aw, mw, lw);
}

// ---------------------------------------------------------------------------
// Row-split MFMA body for wide query groups (33..64 rows per KV head).  Wave
// w owns rows 16w .. 16w+15 and attends every tile of the unit, so no
// cross-wave merge is needed: a wave holds one 16-row block of accumulators
// and its query operand in registers, and the wide kernel keeps two
// workgroups per CU.  The four waves stage each 32-token tile together
// (wave w loads tokens 8w .. 8w+7 of K and of V) into one of two LDS tile
// buffers, with one workgroup barrier per tile; each wave keeps the loads of
// the next kRowsAhead tiles in flight in registers.  Per tile a wave runs
// the one-block math of the body above (same LDS swizzle and operand
// layouts): S^T = K Q^T, the online softmax, O^T += V^T P^T with P as hi + lo.
//
// Tile t is staged in buffer t % 2.  A wave writes buffer t % 2 only after
// the barrier of tile t - 1, which every wave reaches after attending tile
// t - 2, the buffer's previous contents; the barrier of tile t then makes
// the whole tile visible.  Every wave runs the same number of barriers:
// the steps run in groups of kRowsAhead, and a step past the unit's last
// tile (up to kRowsAhead - 1 of them) stages zeros and attends nothing.
// Loads for tiles past the end (the last kRowsAhead issued are never
// staged) go through an empty buffer resource, which reads zeros without
// touching memory.
// ---------------------------------------------------------------------------
constexpr int kRowsAhead = 4;   // tiles of loads in flight per wave; even, so step i of a group uses buffer i % 2
constexpr int kRowsLdsBytes = 2 * 2 * kTileBytes;  // two K + V tile buffers

template <typename P>
__device__ __forceinline__ void rows_unit(const P &p, unsigned char *smem, const UnitRec &ur, int tx, int g) {
  const int w = __builtin_amdgcn_readfirstlane(tx >> 6);   // wave-uniform
  const int lane = tx & 63;
  const int lr = lane & 15;
  const int lq = lane >> 4;
  const int i0 = unit_i0(ur.word);
  const int q_row0 = ur.q_row0;
  const int M = ur.n_cand * p.G;
  const bool active = 16 * w < M;       // wave-uniform: the wave has rows
  const int ntiles = (int)ur.ntiles;

  const uint32_t stride_b = p.tok_stride * 2;                // bytes between tokens
  const uint32_t voff = (8 * w + lq) * stride_b + 16 * lr;     // token 8w + lq, chunk lr
  const float sl2 = p.scale_log2;

  // Q^T operand (B[k = d][j = row]) of row 16w + lr, k-step s: d-chunk
  // 4s + lq.  A padding row (>= M) gets an offset past the end: zeros.
  const int row = 16 * w + lr;
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t *>(p.q), (short)0, (int)((uint32_t)p.st.R * kRowBytes), kBufferFlags);
  const uint32_t qoff = row < M ? (uint32_t)global_row(p, q_row0, g, row) * kRowBytes + 16 * lq : 0x80000000u;
  bf16x8_t qop[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qop[s] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(qrs, qoff + 64 * s, 0, 0));
  __builtin_amdgcn_sched_barrier(0);   // the query loads go out before the wait for the first item
  const FirstItem fi = load_first_item(p, ur);   // slot and flags of the whole chain
  const Item &it = fi.it;

  // loads of tile t: K rows 8w + lq and 8w + 4 + lq, then the same V rows.
  // Tiles are requested in order; the resources of the current item are
  // kept and rebuilt only when the tile moves on to the next item, so a
  // step issues its loads without a chain of dependent argument reads.
  // The loads themselves are unconditional (a conditional load would make
  // the compiler wait for every outstanding one): past the unit's last tile
  // they go through an empty resource.
  const __amdgpu_buffer_rsrc_t empty =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.q), (short)0, 0, kBufferFlags);
  int lk = 0, lbase = 0, lend = tiles_of(it);
  __amdgpu_buffer_rsrc_t lkrs = item_rsrc_at(p, it, fi.k, fi.hs, g);
  __amdgpu_buffer_rsrc_t lvrs = item_rsrc_at(p, it, fi.v, fi.hs, g);
  auto issue = [&](u32x4_t (&d)[4], int t) {
    if (t >= lend && t < ntiles) {
      while (t >= lend) {
        lbase = lend;
        lend += tiles_of(p.items[i0 + ++lk]);
      }
      const Item il = p.items[i0 + lk];
      lkrs = item_rsrc(p, il, item_chunk(il), g, p.k);
      lvrs = item_rsrc(p, il, item_chunk(il), g, p.v);
    }
    const bool in = t < ntiles;
    const __amdgpu_buffer_rsrc_t krs = in ? lkrs : empty;
    const __amdgpu_buffer_rsrc_t vrs = in ? lvrs : empty;
    const uint32_t o = voff + (uint32_t)(in ? (t - lbase) * kTile : 0) * stride_b;
    d[0] = __builtin_amdgcn_raw_buffer_load_b128(krs, o, 0, kStreamLoad);
    d[1] = __builtin_amdgcn_raw_buffer_load_b128(krs, o + 4 * stride_b, 0, kStreamLoad);
    d[2] = __builtin_amdgcn_raw_buffer_load_b128(vrs, o, 0, kStreamLoad);
    d[3] = __builtin_amdgcn_raw_buffer_load_b128(vrs, o + 4 * stride_b, 0, kStreamLoad);
  };
  auto stage = [&](const u32x4_t (&d)[4], unsigned char *buf) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int t = 8 * w + 4 * j + lq;
      *reinterpret_cast<u32x4_t *>(buf + t * kRowBytes + 16 * (lr ^ (t & 15))) = d[j];
      *reinterpret_cast<u32x4_t *>(buf + kTileBytes + t * kRowBytes + 16 * (lr ^ (2 * (t & 7)))) = d[2 + j];
    }
  };

  float m_run = kNegInf, l_run = 0.f;
  f32x4_t acc[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) acc[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int vrow = 4 * lq + (lr >> 2);
  const int vrd = vrow * kRowBytes + 8 * (lr & 1);
  const int vsw = 2 * (vrow & 7);
  const int vc0 = (lr & 3) >> 1;
  // item of the tile being attended: index, first tile, end tile, tokens
  int ck = 0, cbase = 0, cend = lend, count = it.tok_count;

  // attend staged tile t (tokens [tb, tb + 32) of an item with `count` tokens)
  auto attend = [&](const unsigned char *buf, int t) {
    if (t >= cend) {
      while (t >= cend) {
        cbase = cend;
        cend += tiles_of(p.items[i0 + ++ck]);
      }
      count = p.items[i0 + ck].tok_count;
    }
    const int tb = (t - cbase) * kTile;
    const unsigned char *ks = buf;
    const unsigned char *vs = buf + kTileBytes;
    f32x4_t sacc[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int tk = 16 * u + lr;
      f32x4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bf16x8_t kop = *reinterpret_cast<const bf16x8_t *>(ks + tk * kRowBytes + 16 * ((4 * s + lq) ^ lr));
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[s], c, 0, 0, 0);
      }
      sacc[u] = c;
    }
    // the V^T operands go out now, so their LDS latency hides behind the softmax
    bf16x8_t vop[8];
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const int off = vrd + 16 * ((2 * db + vc0) ^ vsw);
      const s16x4_t v0 = lds_read_tr16(vs + off);
      const s16x4_t v1 = lds_read_tr16(vs + off + 16 * kRowBytes);
      vop[db] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
    }

    __builtin_amdgcn_sched_barrier(0);

    // Scores stay unscaled up to the exponent: the row maximum of the raw
    // scores times sigma log2(e) (> 0) is the maximum of the scaled ones,
    // and each weight is 2^(x sigma log2(e) - m) with one fma.  Only an
    // item's last, partial tile needs the token mask.
    float x[8];
    float mx = kNegInf;
    if (tb + kTile <= count) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          x[4 * u + r] = sacc[u][r];
          mx = fmaxf(mx, sacc[u][r]);
        }
    } else {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tt = tb + 16 * u + 4 * lq + r;
          const float v = tt < count ? sacc[u][r] : kNegInf;
          x[4 * u + r] = v;
          mx = fmaxf(mx, v);
        }
    }
    const float mn = fmaxf(m_run, xgroup_max(mx) * sl2);
    // Eq. 14's rescale, only when some row's maximum rose (elsewhere the
    // factor is exactly 1)
    if (__builtin_amdgcn_ballot_w64(mn > m_run)) {
      const float alpha = exp2_fast(m_run - mn);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < 8; ++db) acc[db] *= alpha;
      m_run = mn;
    }
    bf16x8_t phi, plo;
    float ls = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pe = exp2_fast(__builtin_fmaf(x[e], sl2, -mn));
      const __bf16 h = (__bf16)pe;
      const float hf = (float)h;
      const __bf16 lo = (__bf16)(pe - hf);
      phi[e] = h;
      plo[e] = lo;
      ls += pe;
    }
    l_run += ls;

    __builtin_amdgcn_sched_barrier(0);

#pragma unroll
    for (int db = 0; db < 8; ++db) {
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[db], phi, acc[db], 0, 0, 0);
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[db], plo, acc[db], 0, 0, 0);
    }
  };

  u32x4_t ld[kRowsAhead][4];
#pragma unroll
  for (int i = 0; i < kRowsAhead; ++i) issue(ld[i], i);
  for (int t0 = 0; t0 < ntiles; t0 += kRowsAhead) {
#pragma unroll
    for (int i = 0; i < kRowsAhead; ++i) {
      const int t = t0 + i;
      unsigned char *buf = smem + (i & 1) * (2 * kTileBytes);
      stage(ld[i], buf);
      issue(ld[i], t + kRowsAhead);
      __syncthreads();
      if (active && t < ntiles) attend(buf, t);
    }
  }

  // the wave's rows -> their slot (Eq. 14 with the slot's state unless the
  // slot is fresh).  Lane (lr, lq) holds d = 16db + 4lq .. +3 of row 16w + lr.
  if (!active) return;
  l_run = xgroup_sum(l_run);
  if (row >= M) return;
  const size_t idx = (size_t)it.slot * p.st.R + global_row(p, q_row0, g, row);
  float *ap = p.st.a + idx * kHeadDim + 4 * lq;
  if (it.flags & kSlotFresh) {
#pragma unroll
    for (int db = 0; db < 8; ++db) *reinterpret_cast<f32x4_t *>(ap + 16 * db) = acc[db];
    if (lq == 0) {
      p.st.m[idx] = m_run;
      p.st.l[idx] = l_run;
    }
  } else {
    const float ms = p.st.m[idx];
    const float ls = p.st.l[idx];
    const float mn = fmaxf(ms, m_run);
    const float alpha = exp2_fast(ms - mn);
    const float beta = exp2_fast(m_run - mn);
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      f32x4_t o = *reinterpret_cast<const f32x4_t *>(ap + 16 * db);
      o = alpha * o + beta * acc[db];
      *reinterpret_cast<f32x4_t *>(ap + 16 * db) = o;
    }
    if (lq == 0) {
      p.st.m[idx] = mn;
      p.st.l[idx] = alpha * ls + beta * l_run;
    }
  }
}

// ---------------------------------------------------------------------------
// VALU chunk body for sparse query groups (few rows per KV head), used when
// the round's mfma_min_rows asks for it: fp32 dot products on the vector
// ALUs, exact fp32 softmax weights.  Lane l: d-chunk
// c = l % 16 (8 values), token group tg = l / 16; a 32-token tile is 8
// coalesced loads (4 token rows of 256 B each) of K and of V.  Scores are
// reduced over the 16 lanes of a DPP row.
// ---------------------------------------------------------------------------
template <int MAXR, typename P>
__device__ __forceinline__ void valu_unit(const P &p, float *smem, const UnitRec &ur, int tx, int g) {
  const int w = __builtin_amdgcn_readfirstlane(tx >> 6);   // wave-uniform
  const int lane = tx & 63;
  const int c = lane & 15;
  const int tg = lane >> 4;
  const int i0 = unit_i0(ur.word), nit = unit_nit(ur.word);
  const int q_row0 = ur.q_row0;
  const int M = ur.n_cand * p.G;
  const int ntiles = (int)ur.ntiles;
  const FirstItem fi = load_first_item(p, ur);   // slot and flags of the whole chain
  const Item &it = fi.it;

  float qf[MAXR][8];
#pragma unroll
  for (int r = 0; r < MAXR; ++r) {
    if (r < M) {
      const u32x4_t q4 = reinterpret_cast<const u32x4_t *>(p.q + (size_t)global_row(p, q_row0, g, r) * kHeadDim)[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qf[r][2 * e] = bf16_lo(q4[e]);
        qf[r][2 * e + 1] = bf16_hi(q4[e]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[r][e] = 0.f;
    }
  }
  float m_run[MAXR], l_run[MAXR], acc[MAXR][8];
#pragma unroll
  for (int r = 0; r < MAXR; ++r) {
    m_run[r] = kNegInf;
    l_run[r] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
  }
  const uint32_t stride_b = p.tok_stride * 2;
  const uint32_t voff = tg * stride_b + 16 * c;
  const float sl2 = p.scale_log2;

  // coalesced loads (4 token rows per instruction); tokens past the item read 0
  u32x4_t kr[8], vr[8];
  // the whole offset goes in the range-checked VGPR operand (see the MFMA kernel)
  auto load_k = [&](const NextTile &nx) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      kr[i] = __builtin_amdgcn_raw_buffer_load_b128(nx.krs, voff + (uint32_t)(nx.tb + 4 * i) * stride_b, 0, kStreamLoad);
  };
  auto load_v = [&](const NextTile &nx) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      vr[i] = __builtin_amdgcn_raw_buffer_load_b128(nx.vrs, voff + (uint32_t)(nx.tb + 4 * i) * stride_b, 0, kStreamLoad);
  };
  // one tile per iteration (tokens [tb, tb + 32) of an item with `count`
  // tokens); the next tile's K is issued after the scores, its V after the
  // PV update; the last tile is peeled (unconditional prefetch)
  auto tile = [&](int tb, int count, auto prefetch, const NextTile &nx) {
    constexpr bool more = decltype(prefetch)::value;
    float x[8][MAXR];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float kf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kf[2 * e] = bf16_lo(kr[i][e]);
        kf[2 * e + 1] = bf16_hi(kr[i][e]);
      }
      const bool valid = tb + 4 * i + tg < count;
#pragma unroll
      for (int r = 0; r < MAXR; ++r) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d = fmaf(qf[r][e], kf[e], d);
        d = row16_sum(d);
        x[i][r] = valid ? d * sl2 : kNegInf;
      }
    }
    if constexpr (more) load_k(nx);
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
      float mx = kNegInf;
#pragma unroll
      for (int i = 0; i < 8; ++i) mx = fmaxf(mx, x[i][r]);
      mx = xgroup_max(mx);
      const float mn = fmaxf(m_run[r], mx);
      const float alpha = exp2_fast(m_run[r] - mn);
      m_run[r] = mn;
      l_run[r] *= alpha;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[r][e] *= alpha;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float pe = exp2_fast(x[i][r] - mn);
        x[i][r] = pe;
        l_run[r] += pe;
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float vf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[2 * e] = bf16_lo(vr[i][e]);
        vf[2 * e + 1] = bf16_hi(vr[i][e]);
      }
#pragma unroll
      for (int r = 0; r < MAXR; ++r)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[r][e] = fmaf(x[i][r], vf[e], acc[r][e]);
    }
    if constexpr (more) load_v(nx);
  };
  // wave w takes the chain's tiles T = w, w + 4, ...
  int T = w;
  if (T < ntiles) {
    TileCursor cur;
    NextTile nx;
    nx.krs = item_rsrc_at(p, it, fi.k, fi.hs, g);
    nx.vrs = item_rsrc_at(p, it, fi.v, fi.hs, g);
    nx.tb = T * kTile;
    if (T >= tiles_of(it)) {
      seek(p, i0, nit, cur, T);
      const Item ic = p.items[i0 + cur.k];
      nx.krs = item_rsrc(p, ic, item_chunk(ic), g, p.k);
      nx.vrs = item_rsrc(p, ic, item_chunk(ic), g, p.v);
      nx.tb = (T - cur.base) * kTile;
    }
    load_k(nx);
    load_v(nx);
    int tb = nx.tb;
    int count = cur.k == 0 ? it.tok_count : p.items[i0 + cur.k].tok_count;
    for (; T + kWaves < ntiles; T += kWaves) {
      const int kprev = cur.k;
      seek(p, i0, nit, cur, T + kWaves);
      if (cur.k != kprev) {
        const Item in = p.items[i0 + cur.k];
        nx.krs = item_rsrc(p, in, item_chunk(in), g, p.k);
        nx.vrs = item_rsrc(p, in, item_chunk(in), g, p.v);
      }
      nx.tb = (T + kWaves - cur.base) * kTile;
      tile(tb, count, std::integral_constant<bool, true>{}, nx);
      tb = nx.tb;
      count = p.items[i0 + cur.k].tok_count;
    }
    tile(tb, count, std::integral_constant<bool, false>{}, nx);
  }

  // reduce over the token groups, partials -> LDS
#pragma unroll
  for (int r = 0; r < MAXR; ++r) {
    l_run[r] = xgroup_sum(l_run[r]);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = xgroup_sum(acc[r][e]);
  }
  float *aw = smem;
  float *mw = aw + kWaves * MAXR * kAwPitch;
  float *lw = mw + kWaves * MAXR;
  if (tg == 0) {
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
      float *row = aw + (w * MAXR + r) * kAwPitch + 8 * c;
      *reinterpret_cast<f32x4_t *>(row) = f32x4_t{acc[r][0], acc[r][1], acc[r][2], acc[r][3]};
      *reinterpret_cast<f32x4_t *>(row + 4) = f32x4_t{acc[r][4], acc[r][5], acc[r][6], acc[r][7]};
      if (c == 0) {
        mw[w * MAXR + r] = m_run[r];
        lw[w * MAXR + r] = l_run[r];
      }
    }
  }
  __syncthreads();
  fold_into_slot<MAXR>(p, it, q_row0, g, M, tx, aw, mw, lw);
}

constexpr int kValuLdsBytes = kWaves * kMaxValuRows * (kAwPitch + 2) * 4;
constexpr int kChunkLdsBytes = MfmaLds<2>::kBytes > kValuLdsBytes ? MfmaLds<2>::kBytes : kValuLdsBytes;
static_assert(MfmaLds<1>::kBytes <= kChunkLdsBytes, "LDS sizes");
static_assert(kNumSlots == 32, "finalize builds for 8, 16, 24 and 32 slots");
static_assert(kRowsLdsBytes <= kChunkLdsBytes && 2 * kChunkLdsBytes <= 160 * 1024, "LDS sizes");

// ---------------------------------------------------------------------------
// History kernel: one launch for every unit of a call.  Workgroup w of KV
// head g first attends the units of its own list in order (the host gives
// every workgroup an equal share of the call's tokens, which may span
// several requests); each unit's kind selects the body: MFMA with two or
// one 16-row blocks, the row-split body for three or four (only on the wide
// instantiation, which a launch with such a unit runs on), or the VALU path
// for <= 4 rows (built for 1, 2 and 4 rows).  The grid is (g, w) with the
// heads as the fast dimension for token-major chunks, where the eight XCDs
// then read the eight heads of the same tokens, and (w, g) for head-major
// chunks, where every XCD then reads every head's plane: on MI355X a
// head-major launch over 16 x 32768 tokens took 354 us with the heads fast
// and 323 us the other way round (the same box; a loads-only copy of the
// kernel 347 against 318 us, and a plain read of the same 2 GiB 301 us).
//
// The XCDs do not stream at the same rate (on MI355X some finish an equal
// share 10% later than others), so the host may hold back the last part of
// every share as a tail of small units, largest first.  A workgroup that has
// finished its own list claims (tail unit, KV head) pairs from a counter
// until none is left, whatever its own head; each tail unit still owns a
// fixed state slot, so the result does not depend on who attends it.  Every
// workgroup makes exactly one claim past the last pair and then stops, so a
// launch makes num_tail * Hkv + (workgroups) claims; the one that receives
// the last number sets the counter back to zero for the next launch.
// Claims are compared without sign: a counter that is not zero at launch
// (garbage, or a broken workspace promise) gives large numbers, which end
// the loop instead of indexing outside the tail.
// ---------------------------------------------------------------------------
template <bool Wide, typename P>
__global__ void __launch_bounds__(256, 2) chunk_attn(const P p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[kChunkLdsBytes];
  __shared__ uint32_t claim_sh;
  const int y = p.heads_fast ? blockIdx.y : blockIdx.x;     // workgroup of its KV head
  const int g_own = p.heads_fast ? blockIdx.x : blockIdx.y;  // KV head of its own units
  // The workgroup's first unit record and the range of its further units
  // are read together at the start and forced into registers here, so
  // neither the first unit's loads nor its end wait for a second round of
  // argument reads.
  UnitRec ur = p.units[y];
  uint32_t more0 = p.more[y], more1 = p.more[y + 1];
  asm volatile("" : "+s"(ur.word), "+s"(ur.ntiles), "+s"(ur.q_row0), "+s"(ur.n_cand), "+s"(more0), "+s"(more1));
  const uint32_t nclaims = (uint32_t)p.num_tail * (uint32_t)p.Hkv;
  const uint32_t last_claim = nclaims + (uint32_t)p.Hkv * (uint32_t)p.num_wgs - 1u;
  uint32_t u = more0;
  bool first = true;
  for (;;) {
    int g = g_own;
    if (first) {
      first = false;
      if (unit_nit(ur.word) == 0) continue;   // a workgroup without units of its own
    } else if (u < more1) {
      __syncthreads();   // the previous unit's fold has read the LDS this unit restages
      ur = p.units[u++];
    } else {
      if (nclaims == 0) break;
      __syncthreads();   // ... and every thread has read the previous claim
      if (threadIdx.x == 0) {
        const uint32_t c = atomicAdd(p.claim, 1u);
        if (c == last_claim) __hip_atomic_store(p.claim, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        claim_sh = c;
      }
      __syncthreads();
      const uint32_t c = __builtin_amdgcn_readfirstlane(claim_sh);
      if (c >= nclaims) break;
      const uint32_t t = c / (uint32_t)p.Hkv;
      ur = p.units[p.tail_first + (int)t];
      g = (int)(c - t * (uint32_t)p.Hkv);
    }
    // The bodies derive their per-lane addresses from tx.  Passing it
    // through an empty asm each unit keeps the compiler from computing
    // them once before the loop and holding all three bodies' worth live
    // across it (that spilled 14 registers and cost 6% on one-unit calls).
    int tx = threadIdx.x;
    asm volatile("" : "+v"(tx));
    const int kind = unit_kind(ur.word);
    if constexpr (Wide) {
      if (kind >= kUnitMfma3) {
        rows_unit(p, smem, ur, tx, g);
        continue;
      }
    }
    const int nxt = u < more1 ? (int)u : -1;   // the next unit of the workgroup's own list
    if (kind == kUnitMfma2)
      mfma_unit<2>(p, smem, ur, tx, g, nxt);
    else if (kind == kUnitMfma1)
      mfma_unit<1>(p, smem, ur, tx, g, nxt);
    else {
      // the VALU body's work grows with the rows it is built for: build it
      // for 1, 2 and 4 rows and take the smallest that holds the unit
      const int rows = ur.n_cand * p.G;
      float *lds = reinterpret_cast<float *>(smem);
      if (rows <= 1)
        valu_unit<1>(p, lds, ur, tx, g);
      else if (rows <= 2)
        valu_unit<2>(p, lds, ur, tx, g);
      else
        valu_unit<kMaxValuRows>(p, lds, ur, tx, g);
    }
  }
}

__global__ void __launch_bounds__(64) clear_counters_kernel(uint32_t *c, int n) {
  for (int i = threadIdx.x; i < n; i += 64) c[i] = 0u;
}

// ---------------------------------------------------------------------------
// Finalize: for every query row (request b, candidate i, head h)
//   * attend the Speculative Frontier: candidate keys j <= i of the same
//     request, causal by absolute position (Sec. 4.2, GPU-resident pass),
//   * merge the split slots the history calls wrote (Eq. 14; slot count per
//     request from the host, unwritten slots are never read),
//   * write O = a / l and LSE = m ln 2 + ln l (Eq. 17).
// One wave per row (4 rows of one request per workgroup); lane l
// holds d = 2l, 2l+1.  The kernel is latency-bound, so a row costs one
// memory round trip: every load is issued before any use (the query, the
// visible candidates' K/V, each slot's m and l - lane s loads slot s - and
// every slot's a values).  The row's maximum over the frontier scores and
// the slot maxima then gives each term its scale 2^(m_s - m*) once (Eq. 14
// applied to all pieces together), so the slots need no step-by-step
// rescaling.  Slot loads past the request's count go through empty buffer
// resources or offsets past the end and read zeros.
// ---------------------------------------------------------------------------
//
// The grid is (request, block of 4 rows), sized for the request with the
// most rows; a block past a request's rows exits at once.  Workgroups are
// dispatched in grid order, so with the requests as the fast dimension the
// blocks of the requests with the most rows come last, behind every idle
// block: with ragged row counts the grid is built the other way round
// (RowsFast), which spreads the idle blocks over the dispatch.
template <int MS, bool RowsFast, typename P>
__global__ void __launch_bounds__(256) finalize_kernel(const P p) {
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const Item it = p.items[RowsFast ? blockIdx.y : blockIdx.x];
  const int r = (RowsFast ? blockIdx.x : blockIdx.y) * kWaves + w;   // local row = i * Hq + h
  if (r >= it.n_cand * p.Hq) return;
  const int i = r / p.Hq;
  const int h = r - i * p.Hq;
  const int g = h / p.G;
  const int row = __builtin_amdgcn_readfirstlane(it.q_row0 * p.Hq + r);   // (off_b + i) * Hq + h
  const int nslot = it.tok_count;

  const uint32_t qw = reinterpret_cast<const uint32_t *>(p.q + (size_t)row * kHeadDim)[lane];
  uint32_t kw[kMaxCand], vw[kMaxCand];
#pragma unroll
  for (int j = 0; j < kMaxCand; ++j) {
    kw[j] = 0;
    vw[j] = 0;
    if (j <= i) {
      const size_t kv = ((size_t)(it.q_row0 + j) * p.Hkv + g) * kHeadDim;
      kw[j] = reinterpret_cast<const uint32_t *>(p.kc + kv)[lane];
      vw[j] = reinterpret_cast<const uint32_t *>(p.vc + kv)[lane];
    }
  }
  // slot s's m and l in lane s (offsets past the array read zero)
  const __amdgpu_buffer_rsrc_t mrs = __builtin_amdgcn_make_buffer_rsrc(
      p.st.m, (short)0, (int)((uint32_t)kNumSlots * (uint32_t)p.st.R * 4), kBufferFlags);
  const __amdgpu_buffer_rsrc_t lrs = __builtin_amdgcn_make_buffer_rsrc(
      p.st.l, (short)0, (int)((uint32_t)kNumSlots * (uint32_t)p.st.R * 4), kBufferFlags);
  const uint32_t moff = lane < nslot ? ((uint32_t)lane * (uint32_t)p.st.R + (uint32_t)row) * 4 : 0xfffffff0u;
  const float m_lane = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, moff, 0, 0));
  const float l_lane = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(lrs, moff, 0, 0));
  // every slot's a values of this row: slot s through a resource over the
  // row's 512 bytes in that slot (empty past the count); the launch is built
  // for MS >= every request's slot count
  float2 as[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s) {
    const float *base = p.st.a + ((size_t)s * p.st.R + row) * kHeadDim;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(base), (short)0, s < nslot ? kRowBytes * 2 : 0, kBufferFlags);
    const uint64_t v = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(rs, (uint32_t)lane * 8, 0, 0));
    as[s] = __builtin_bit_cast(float2, v);
  }

  // frontier scores: the <= 8 dot products reduced as independent chains
  const float q0 = bf16_lo(qw), q1 = bf16_hi(qw);
  float x[kMaxCand];
#pragma unroll
  for (int j = 0; j < kMaxCand; ++j) x[j] = fmaf(q0, bf16_lo(kw[j]), q1 * bf16_hi(kw[j]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
    for (int j = 0; j < kMaxCand; ++j) x[j] += __shfl_xor(x[j], off);
  float m = kNegInf;
#pragma unroll
  for (int j = 0; j < kMaxCand; ++j) {
    x[j] = j <= i ? x[j] * p.scale_log2 : kNegInf;
    m = fmaxf(m, x[j]);
  }
  // m* over the frontier (finite: every query sees candidate 0) and the slots
  const float ms_lane = lane < nslot ? m_lane : kNegInf;
  float mslot = ms_lane;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mslot = fmaxf(mslot, __shfl_xor(mslot, off));
  m = fmaxf(m, mslot);
  const float f_lane = exp2_fast(ms_lane - m);    // slot scale in lane s; 0 past the count
  float lsum = f_lane * l_lane;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) lsum += __shfl_xor(lsum, off);
  float l = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxCand; ++j) {
    if (j <= i) {
      const float pj = exp2_fast(x[j] - m);
      l += pj;
      a0 = fmaf(pj, bf16_lo(vw[j]), a0);
      a1 = fmaf(pj, bf16_hi(vw[j]), a1);
    }
  }
  l += lsum;
#pragma unroll
  for (int s = 0; s < MS; ++s) {
    const float f = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, f_lane), s));
    a0 = fmaf(f, as[s].x, a0);
    a1 = fmaf(f, as[s].y, a1);
  }
  const float inv = 1.0f / l;
  reinterpret_cast<float2 *>(p.out + (size_t)row * kHeadDim)[lane] = make_float2(a0 * inv, a1 * inv);
  if (p.lse != nullptr && lane == 0) p.lse[row] = m * 0.69314718055994531f + logf(l);
}

// Read-bandwidth probe: workgroup w XOR-folds the 32-bit words of bytes
// [w * share, min((w + 1) * share, bytes)) of buf and stores the fold to
// sink[w].  The loads are the history kernel's: 16 bytes per lane, non-
// temporal, through a range-checked buffer resource (reads past the slice
// return zero, which the fold ignores), eight per lane in flight.
__global__ void __launch_bounds__(256) read_probe_kernel(const uint8_t *buf, uint64_t bytes, uint64_t share,
                                                         uint32_t *sink) {
  const uint64_t first = (uint64_t)blockIdx.x * share;
  const uint32_t n = first >= bytes ? 0u : (uint32_t)(bytes - first < share ? bytes - first : share);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(buf) + (first < bytes ? first : 0), (short)0, (int)n,
                                        kBufferFlags);
  constexpr uint32_t kStep = 256 * 16;   // bytes one load instruction of the workgroup reads
  constexpr int kDepth = 8;
  const uint32_t t = threadIdx.x * 16u;
  u32x4_t acc = {0u, 0u, 0u, 0u};
  uint32_t o = 0;
  for (; o + kDepth * kStep <= n; o += kDepth * kStep) {
    u32x4_t v[kDepth];
#pragma unroll
    for (int i = 0; i < kDepth; ++i)
      v[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, o + i * kStep + t, 0, kStreamLoad));
#pragma unroll
    for (int i = 0; i < kDepth; ++i) acc ^= v[i];
  }
  for (; o < n; o += kStep)
    acc ^= __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, o + t, 0, kStreamLoad));
  uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x ^= (uint32_t)__shfl_xor((int)x, m, 64);
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

// The library's device scratch (see scratch_address).  Each GPU the library
// runs on holds its own copy until the process ends.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

}  // namespace

namespace {

// Table capacities of the launches: a Cohort's whole history call usually
// fits the small class (config 3: 32 workgroups per KV head, 32 units, 128
// items), large ragged batches the medium one.
using ChunkSmall = ChunkParamsT<128, 256, 128>;
using ChunkMedium = ChunkParamsT<512, 1024, 256>;
using FinalSmall = FinalParamsT<64>;

template <bool Wide, typename D>
hipError_t launch_chunk_as(const ChunkParams &p, hipStream_t s) {
  static thread_local D d;
  static_cast<ChunkHeader &>(d) = p;
  std::memcpy(d.units, p.units, sizeof(UnitRec) * p.num_units);
  std::memcpy(d.more, p.more, sizeof(uint32_t) * (p.num_wgs + 1));
  std::memcpy(d.items, p.items, sizeof(Item) * p.num_items);
  const dim3 grid = p.heads_fast ? dim3(p.Hkv, p.num_wgs) : dim3(p.num_wgs, p.Hkv);
  hipLaunchKernelGGL((chunk_attn<Wide, D>), grid, dim3(256), 0, s, d);
  return hipGetLastError();
}

template <bool Wide>
hipError_t launch_chunk_sized(const ChunkParams &p, hipStream_t s) {
  auto fits = [&](int units, int items, int wgs) {
    return p.num_units <= units && p.num_items <= items && p.num_wgs <= wgs;
  };
  if (fits(ChunkSmall::kUnits, ChunkSmall::kItems, ChunkSmall::kWgs)) return launch_chunk_as<Wide, ChunkSmall>(p, s);
  if (fits(ChunkMedium::kUnits, ChunkMedium::kItems, ChunkMedium::kWgs)) return launch_chunk_as<Wide, ChunkMedium>(p, s);
  const dim3 grid = p.heads_fast ? dim3(p.Hkv, p.num_wgs) : dim3(p.num_wgs, p.Hkv);
  hipLaunchKernelGGL((chunk_attn<Wide, ChunkParams>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_chunk(const ChunkParams &p, hipStream_t s) {
  // a launch with any unit of more than two 16-row blocks runs on the wide kernel
  for (int u = 0; u < p.num_units; ++u)
    if (unit_kind(p.units[u].word) >= kUnitMfma3) return launch_chunk_sized<true>(p, s);
  return launch_chunk_sized<false>(p, s);
}

hipError_t launch_clear_counters(uint32_t *counters, int n, hipStream_t s) {
  hipLaunchKernelGGL(clear_counters_kernel, dim3(1), dim3(64), 0, s, counters, n);
  return hipGetLastError();
}
template <int MS, bool RowsFast>
hipError_t launch_finalize_as(const FinalParams &p, int row_blocks, hipStream_t s) {
  const dim3 grid = RowsFast ? dim3(row_blocks, p.num_items) : dim3(p.num_items, row_blocks);
  if (p.num_items <= FinalSmall::kItems) {
    static thread_local FinalSmall d;
    static_cast<FinalHeader &>(d) = p;
    std::memcpy(d.items, p.items, sizeof(Item) * p.num_items);
    hipLaunchKernelGGL((finalize_kernel<MS, RowsFast, FinalSmall>), grid, dim3(256), 0, s, d);
  } else {
    hipLaunchKernelGGL((finalize_kernel<MS, RowsFast, FinalParams>), grid, dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

template <int MS>
hipError_t launch_finalize_ms(const FinalParams &p, int row_blocks, bool rows_fast, hipStream_t s) {
  return rows_fast ? launch_finalize_as<MS, true>(p, row_blocks, s) : launch_finalize_as<MS, false>(p, row_blocks, s);
}

hipError_t launch_finalize(const FinalParams &p, hipStream_t s) {
  // Built for 8, 16, 24 or 32 slots: each slot a row may read costs the
  // wave a load and two registers, so the smallest build that holds every
  // request's slot count keeps more waves resident.  Measured on MI355X:
  // 16 x 32768 tokens (14 slots) 7.3 -> 6.0 us, 64 ragged requests (16
  // slots) 19.8 -> 13.6 us against the 32-slot build.
  // Row-block order: the requests-fast grid keeps a request's blocks on one
  // XCD (the grid's request count is a multiple of 8 in the common case),
  // which measured faster for uniform cohorts; with more than a quarter of
  // the blocks idle the rows-fast grid is faster.  Measured on MI355X
  // (medians, alternated in one run): 64 ragged requests (42% idle) 16.5 us
  // requests-fast, 14.5-14.9 us rows-fast; 16 x 6 candidates 6.8-7.0 us
  // requests-fast, 7.0-7.1 us rows-fast.
  int rows = 0, slots = 0;
  long busy = 0;
  for (int i = 0; i < p.num_items; ++i) {
    const int ri = p.items[i].n_cand * p.Hq;
    rows = rows > ri ? rows : ri;
    busy += (ri + kWaves - 1) / kWaves;
    slots = slots > p.items[i].tok_count ? slots : p.items[i].tok_count;
  }
  const int row_blocks = (rows + kWaves - 1) / kWaves;
  const bool rows_fast = 4 * busy < 3 * (long)row_blocks * p.num_items;
  if (slots <= 8) return launch_finalize_ms<8>(p, row_blocks, rows_fast, s);
  if (slots <= 16) return launch_finalize_ms<16>(p, row_blocks, rows_fast, s);
  if (slots <= 24) return launch_finalize_ms<24>(p, row_blocks, rows_fast, s);
  return launch_finalize_ms<kNumSlots>(p, row_blocks, rows_fast, s);
}

hipError_t launch_read_probe(const void *buf, uint64_t bytes, uint64_t share, uint32_t *sink, int workgroups,
                             hipStream_t s) {
  hipLaunchKernelGGL(read_probe_kernel, dim3(workgroups), dim3(256), 0, s, static_cast<const uint8_t *>(buf), bytes,
                     share, sink);
  return hipGetLastError();
}

hipError_t scratch_address(void **ptr) {
  // One lookup per device, with that device current; the array's name is a
  // host-side stand-in, so only the looked-up address may reach a kernel.
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void *a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (a == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = a;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace ss
