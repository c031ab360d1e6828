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
//     bf16 would cost ~1.6e-3 relative L2 error.  The denominator l is summed
//     from the same hi + lo values, so numerator and denominator agree.
//   * a running state is split into kNumSlots slots per query row so that
//     several workgroups can fold disjoint token ranges of one chunk into the
//     same row without atomics; the finalize kernel merges the slots.
#include <hip/hip_runtime.h>

#include "ss_kernels.h"

#include <math.h>

#include <type_traits>

namespace ss {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kAwPitch = 132;  // floats per row of a wave's partial accumulator

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

__device__ __forceinline__ int global_row(const ChunkParams &p, const Item &it, int g, int r) {
  // local row r of (request, kv head g) -> packed query row (off_b + i) * Hq + h
  const int i = r / p.G;
  const int h = g * p.G + (r - i * p.G);
  return (it.q_row0 + i) * p.Hq + h;
}

// ---------------------------------------------------------------------------
// Workgroup epilogue shared by the chunk kernels: the kWaves waves have left
// their partial states in LDS (aw[w][row][kAwPitch], mw[w][row], lw[w][row],
// all relative to their own maxima); combine them (Eq. 14 over the waves) and
// fold the result into the item's slot of the running state (Eq. 14 again).
// ---------------------------------------------------------------------------
template <int ROWS>
__device__ __forceinline__ void fold_into_slot(const ChunkParams &p, const Item &it, int g, int M,
                                               const float *aw, const float *mw, const float *lw) {
  // SEGS threads per row, SEGLEN (a multiple of 4) values each
  constexpr int SEGS = (256 / ROWS) < 32 ? (256 / ROWS) : 32;
  constexpr int SEGLEN = kHeadDim / SEGS;
  static_assert(SEGLEN % 4 == 0 && SEGS * ROWS <= 256, "fold layout");
  const int r = threadIdx.x / SEGS;
  const int seg = threadIdx.x % SEGS;
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
  const size_t idx = (size_t)it.slot * p.st.R + global_row(p, it, g, r);
  float *ap = p.st.a + idx * kHeadDim + seg * SEGLEN;
  const float ms = p.st.m[idx];
  if (ms == kNegInf) {               // empty slot: empty (+) X = X, old a is not read
#pragma unroll
    for (int c = 0; c < SEGLEN; c += 4)
      *reinterpret_cast<f32x4_t *>(ap + c) = f32x4_t{a[c], a[c + 1], a[c + 2], a[c + 3]};
    if (seg == 0) {
      p.st.m[idx] = mstar;
      p.st.l[idx] = lstar;
    }
  } else {
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
// MFMA chunk kernel.  Workgroup = (item, kv head); 4 waves; wave w takes the
// 32-token tiles w, w+4, ... of the item.  Per tile:
//   S^T[t][row] = K Q^T      v_mfma_f32_16x16x32_bf16, A = K (16 tokens x 32 d
//                            from registers), B = Q^T (held in registers)
//   online softmax per row   (row = lane % 16; the four lane groups share it)
//   O^T[d][row] += V^T P^T   A = V^T read from a row-major LDS tile with the
//                            LDS transpose read, B = P^T straight from the S
//                            accumulators (hi and lo parts)
// Lane l: lr = l % 16, lq = l / 16.  In the S tile lane (lr, lq) holds
// tokens 16u + 4*lq + r (u = 0,1; r = 0..3) of row lr; in O it holds
// d = 16*db + 4*lq + r.  The reduction index of both MFMAs is permuted so
// every operand is contiguous: for QK^T lane group lq, k-step s covers the
// d-chunk 4*s + lq (8 values); for PV lane group lq covers tokens
// {4lq..4lq+3, 16+4lq..16+4lq+3}, exactly the S values the lane holds.
//
// ds_read_b64_tr_b16: within each 16-lane group, result lane i, element e is
// element (i % 4) of what source lane 4e + i/4 addressed.  Source lane j of
// group lq addresses row 4lq + j/4 (+16 for the second half), columns
// 16db + 4(j%4) .. +3, so result lane i receives V[4lq + e][16db + i].
//
// Each wave keeps the next tile's K and V in flight in registers: K(i+1) is
// issued as soon as S(i) has consumed K(i), V(i+1) as soon as V(i) is staged
// in LDS, so at the top of an iteration only K is waited for.  The last tile
// is peeled so the in-loop prefetch is unconditional (a conditional load
// would make the compiler wait for every outstanding load).
// ---------------------------------------------------------------------------
constexpr int kVPitch = 144;   // bf16 per LDS V row (128 + 16): rows 288 B apart

template <int RB>
struct MfmaLds {
  static constexpr int kVBytes = kWaves * kTile * kVPitch * 2;
  static constexpr int kMergeBytes = kWaves * RB * 16 * (kAwPitch + 2) * 4;
  static constexpr int kBytes = kVBytes > kMergeBytes ? kVBytes : kMergeBytes;
};

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ s16x4_t lds_read_tr16(const uint16_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4_t *)(reinterpret_cast<uintptr_t>(p)));
}

template <int RB>
__global__ void __launch_bounds__(256, 2) chunk_attn_mfma(const ChunkParams p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[MfmaLds<RB>::kBytes];
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15;
  const int lq = lane >> 4;
  const Item it = p.items[blockIdx.x];
  const int g = blockIdx.y;
  const int M = it.n_cand * p.G;
  const int count = it.tok_count;

  // Q^T operand: B[k = d][j = row]; lane (lr, lq), k-step s -> row lr, d-chunk 4s+lq
  bf16x8_t qop[RB][4];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = rb * 16 + lr;
    if (r < M) {
      const u32x4_t *qp = reinterpret_cast<const u32x4_t *>(p.q + (size_t)global_row(p, it, g, r) * kHeadDim);
#pragma unroll
      for (int s = 0; s < 4; ++s) qop[rb][s] = __builtin_bit_cast(bf16x8_t, qp[4 * s + lq]);
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s) qop[rb][s] = __builtin_bit_cast(bf16x8_t, u32x4_t{0, 0, 0, 0});
    }
  }

  float m_run[RB], l_run[RB];
  f32x4_t acc[RB][8];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_run[rb] = kNegInf;
    l_run[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[rb][db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // 32-bit element offsets inside the item (the host keeps an item < 2^30 elements)
  const uint32_t tok_stride = (uint32_t)p.Hkv * kHeadDim;
  const uint16_t *kbase = p.k + ((size_t)it.tok_begin * p.Hkv + g) * kHeadDim;
  const uint16_t *vbase = p.v + ((size_t)it.tok_begin * p.Hkv + g) * kHeadDim;
  uint16_t *vs = reinterpret_cast<uint16_t *>(smem) + w * (kTile * kVPitch);
  const int ntiles = (count + kTile - 1) / kTile;
  const float sl2 = p.scale_log2;

  u32x4_t kr[2][4];
  u32x4_t vr[8];
  auto load_k = [&](int tb) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint32_t t = (uint32_t)min(tb + 16 * u + lr, count - 1);
      const u32x4_t *src = reinterpret_cast<const u32x4_t *>(kbase + t * tok_stride);
#pragma unroll
      for (int s = 0; s < 4; ++s) kr[u][s] = src[4 * s + lq];
    }
  };
  auto load_v = [&](int tb) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t t = (uint32_t)min(tb + 4 * i + lq, count - 1);
      vr[i] = reinterpret_cast<const u32x4_t *>(vbase + t * tok_stride)[lr];
    }
  };
  // V operand read addresses (row 4lq + lr/4, column 4*(lr%4)), first half
  const uint16_t *vrd = vs + (4 * lq + (lr >> 2)) * kVPitch + 4 * (lr & 3);

  auto tile = [&](int tb, auto prefetch) {
    constexpr bool kPrefetch = decltype(prefetch)::value;
    // S^T = K Q^T
    f32x4_t sacc[2][RB];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        f32x4_t c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4; ++s)
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[u][s]), qop[rb][s], c, 0, 0, 0);
        sacc[u][rb] = c;
      }
    if constexpr (kPrefetch) load_k(tb + kWaves * kTile);
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch here, ahead of the softmax

    // online softmax (Eq. 13 local terms merged per Eq. 14 into the wave's state)
    bf16x8_t phi[RB], plo[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float x[8];
      float mx = kNegInf;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tb + 16 * u + 4 * lq + r;
          const float v = t < count ? sacc[u][rb][r] * sl2 : kNegInf;
          x[4 * u + r] = v;
          mx = fmaxf(mx, v);
        }
      mx = xgroup_max(mx);
      const float mn = fmaxf(m_run[rb], mx);
      const float alpha = exp2_fast(m_run[rb] - mn);
      m_run[rb] = mn;
      float ls = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pe = exp2_fast(x[e] - mn);
        const __bf16 h = (__bf16)pe;
        const float hf = (float)h;
        const __bf16 lo = (__bf16)(pe - hf);
        phi[rb][e] = h;
        plo[rb][e] = lo;
        ls += hf + (float)lo;
      }
      l_run[rb] = alpha * l_run[rb] + ls;
#pragma unroll
      for (int db = 0; db < 8; ++db) acc[rb][db] *= alpha;
    }

    // V tile -> LDS, row-major (token 4i + lq, 16-byte chunk lr); then prefetch
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4_t *>(vs + (4 * i + lq) * kVPitch + 8 * lr) = vr[i];
    if constexpr (kPrefetch) load_v(tb + kWaves * kTile);
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch here, ahead of PV

    // O^T += V^T P^T  (hi and lo parts of P)
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const s16x4_t v0 = lds_read_tr16(vrd + 16 * db);
      const s16x4_t v1 = lds_read_tr16(vrd + 16 * kVPitch + 16 * db);
      const bf16x8_t vop = __builtin_bit_cast(
          bf16x8_t, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        acc[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, phi[rb], acc[rb][db], 0, 0, 0);
        acc[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, plo[rb], acc[rb][db], 0, 0, 0);
      }
    }
  };

  int t0 = w;
  if (t0 < ntiles) {
    load_k(t0 * kTile);   // same issue order as the loop body: K, then V
    load_v(t0 * kTile);
    for (; t0 + kWaves < ntiles; t0 += kWaves) tile(t0 * kTile, std::integral_constant<bool, true>{});
    tile(t0 * kTile, std::integral_constant<bool, false>{});
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
  fold_into_slot<RB * 16>(p, it, g, M, aw, mw, lw);
}
// ---------------------------------------------------------------------------
// VALU chunk kernel for sparse query groups (few rows per KV head): fp32 dot
// products on the vector ALUs, exact fp32 softmax weights.  Lane l: d-chunk
// c = l % 16 (8 values), token group tg = l / 16; a 32-token tile is 8
// coalesced loads (4 token rows of 256 B each) of K and of V.  Scores are
// reduced over the 16 lanes of a DPP row.
// ---------------------------------------------------------------------------
template <int MAXR>
__global__ void __launch_bounds__(256, 2) chunk_attn_valu(const ChunkParams p) {
  __shared__ __attribute__((aligned(16))) float smem[kWaves * MAXR * (kAwPitch + 2)];
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int c = lane & 15;
  const int tg = lane >> 4;
  const Item it = p.items[blockIdx.x];
  const int g = blockIdx.y;
  const int M = it.n_cand * p.G;
  const int count = it.tok_count;

  float qf[MAXR][8];
#pragma unroll
  for (int r = 0; r < MAXR; ++r) {
    if (r < M) {
      const u32x4_t q4 = reinterpret_cast<const u32x4_t *>(p.q + (size_t)global_row(p, it, g, r) * kHeadDim)[c];
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
  const size_t tok_stride = (size_t)p.Hkv * kHeadDim;
  const uint16_t *kbase = p.k + ((size_t)it.tok_begin * p.Hkv + g) * kHeadDim;
  const uint16_t *vbase = p.v + ((size_t)it.tok_begin * p.Hkv + g) * kHeadDim;
  const int ntiles = (count + kTile - 1) / kTile;
  const float sl2 = p.scale_log2;

  u32x4_t kr[8], vr[8];
  auto load_k = [&](int tb) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = min(tb + 4 * i + tg, count - 1);
      kr[i] = reinterpret_cast<const u32x4_t *>(kbase + (size_t)t * tok_stride)[c];
    }
  };
  auto load_v = [&](int tb) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = min(tb + 4 * i + tg, count - 1);
      vr[i] = reinterpret_cast<const u32x4_t *>(vbase + (size_t)t * tok_stride)[c];
    }
  };
  int tile = w;
  if (tile < ntiles) {
    load_k(tile * kTile);
    load_v(tile * kTile);
  }
  for (; tile < ntiles; tile += kWaves) {
    const int tb = tile * kTile;
    const bool more = tile + kWaves < ntiles;
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
    if (more) load_k(tb + kWaves * kTile);
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
    if (more) load_v(tb + kWaves * kTile);
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
  fold_into_slot<MAXR>(p, it, g, M, aw, mw, lw);
}

// ---------------------------------------------------------------------------
// Speculative Frontier: query i of request b sees candidate keys j <= i.
// Workgroup = (request, kv head); wave w takes rows w, w+4, ...; lane l holds
// d = 2l, 2l+1.  The local state is merged into slot 0 (Eq. 14).
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) candidates_kernel(const ChunkParams p) {
  const int w = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const Item it = p.items[blockIdx.x];
  const int g = blockIdx.y;
  const int n = it.n_cand;
  const int M = n * p.G;
  for (int r = w; r < M; r += kWaves) {
    const int i = r / p.G;
    const int row = global_row(p, it, g, r);
    const uint32_t qw = reinterpret_cast<const uint32_t *>(p.q + (size_t)row * kHeadDim)[lane];
    const float q0 = bf16_lo(qw), q1 = bf16_hi(qw);
    float x[kMaxCand];
    float mx = kNegInf;
#pragma unroll
    for (int j = 0; j < kMaxCand; ++j) {
      x[j] = kNegInf;
      if (j <= i) {
        const size_t krow = ((size_t)(it.q_row0 + j) * p.Hkv + g) * kHeadDim;
        const uint32_t kw = reinterpret_cast<const uint32_t *>(p.k + krow)[lane];
        float d = fmaf(q0, bf16_lo(kw), q1 * bf16_hi(kw));
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) d += __shfl_xor(d, off);
        x[j] = d * p.scale_log2;
        mx = fmaxf(mx, x[j]);
      }
    }
    float l = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxCand; ++j) {
      if (j <= i) {
        const float pj = exp2_fast(x[j] - mx);
        const size_t vrow = ((size_t)(it.q_row0 + j) * p.Hkv + g) * kHeadDim;
        const uint32_t vw = reinterpret_cast<const uint32_t *>(p.v + vrow)[lane];
        l += pj;
        a0 = fmaf(pj, bf16_lo(vw), a0);
        a1 = fmaf(pj, bf16_hi(vw), a1);
      }
    }
    const size_t idx = (size_t)row;          // slot 0
    float *ap = p.st.a + idx * kHeadDim + 2 * lane;
    const float ms = p.st.m[idx];
    if (ms == kNegInf) {
      ap[0] = a0;
      ap[1] = a1;
      if (lane == 0) {
        p.st.m[idx] = mx;
        p.st.l[idx] = l;
      }
    } else {
      const float mn = fmaxf(ms, mx);
      const float alpha = exp2_fast(ms - mn);
      const float beta = exp2_fast(mx - mn);
      ap[0] = alpha * ap[0] + beta * a0;
      ap[1] = alpha * ap[1] + beta * a1;
      if (lane == 0) {
        p.st.m[idx] = mn;
        p.st.l[idx] = alpha * p.st.l[idx] + beta * l;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Split-KV state merge + normalisation: for each query row merge the
// kNumSlots slot states (Eq. 14; empty slots have weight 0) and write
// O = a / l and LSE = m ln 2 + ln l.  One wave per row, lane l holds d = 2l, 2l+1.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) finalize_kernel(const State st, float *out, float *lse) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= st.R) return;
  float ms[kNumSlots];
  float mstar = kNegInf;
#pragma unroll
  for (int s = 0; s < kNumSlots; ++s) {
    ms[s] = st.m[(size_t)s * st.R + row];
    mstar = fmaxf(mstar, ms[s]);
  }
  float l = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int s = 0; s < kNumSlots; ++s) {
    if (ms[s] != kNegInf) {
      const size_t idx = (size_t)s * st.R + row;
      const float f = exp2_fast(ms[s] - mstar);
      const float2 a = reinterpret_cast<const float2 *>(st.a + idx * kHeadDim)[lane];
      l += f * st.l[idx];
      a0 = fmaf(f, a.x, a0);
      a1 = fmaf(f, a.y, a1);
    }
  }
  const float inv = 1.0f / l;
  reinterpret_cast<float2 *>(out + (size_t)row * kHeadDim)[lane] = make_float2(a0 * inv, a1 * inv);
  if (lse != nullptr && lane == 0) lse[row] = mstar * 0.69314718055994531f + logf(l);
}

__global__ void init_state_kernel(const State st) {
  const size_t n = (size_t)kNumSlots * st.R;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    st.m[i] = kNegInf;
    st.l[i] = 0.f;
  }
}

}  // namespace

hipError_t launch_init_state(const State &st, hipStream_t s) {
  const size_t n = (size_t)kNumSlots * st.R;
  const int blocks = (int)((n + 255) / 256 < 2048 ? (n + 255) / 256 : 2048);
  hipLaunchKernelGGL(init_state_kernel, dim3(blocks), dim3(256), 0, s, st);
  return hipGetLastError();
}

hipError_t launch_chunk_mfma(const ChunkParams &p, int row_blocks, hipStream_t s) {
  const dim3 grid(p.num_items, p.Hkv);
  if (row_blocks == 1)
    hipLaunchKernelGGL(chunk_attn_mfma<1>, grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(chunk_attn_mfma<2>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_chunk_valu(const ChunkParams &p, int max_rows, hipStream_t s) {
  const dim3 grid(p.num_items, p.Hkv);
  (void)max_rows;  // rows per KV head <= kMaxValuRows, checked by the host
  hipLaunchKernelGGL(chunk_attn_valu<kMaxValuRows>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_candidates(const ChunkParams &p, hipStream_t s) {
  hipLaunchKernelGGL(candidates_kernel, dim3(p.num_items, p.Hkv), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_finalize(const State &st, float *out, float *lse, hipStream_t s) {
  hipLaunchKernelGGL(finalize_kernel, dim3((st.R + 3) / 4), dim3(256), 0, s, st, out, lse);
  return hipGetLastError();
}

}  // namespace ss
