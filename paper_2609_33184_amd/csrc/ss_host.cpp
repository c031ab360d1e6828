// Host side of libspecstream: argument validation, the round state machine,
// the work planner that splits each history chunk into workgroup pieces, the
// upload call and the two-slot transfer pipeline (paper Sec. 4.2).
#include "specstream.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "ss_error.h"
#include "ss_kernels.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace ss {

ss_status fail(ss_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

ss_status hip_fail(hipError_t e, const char *what) {
  return fail(SS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace ss

namespace {

using ss::fail;
using ss::hip_fail;

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workgroups of a history call: the call's tokens (every request's, in
// request order) are cut into equal shares, one per workgroup and KV head
// (stream-K style), so every workgroup has the same work however ragged the
// requests are; a share may span several requests.  Large shares amortise
// each unit's fixed costs (query staging, wave merge, state fold); aim for
// one workgroup per CU (256 on MI355X).  Measured per round: 16 x 32768
// tokens, 8 KV heads: shares of 8192 tokens (512 workgroups) 340 us, 16384
// (256) 329 us; 32 x 131072 tokens: 256 workgroups 2545 us, 1024 2577 us.
// 64 ragged requests of 2048..65536 tokens took 698-702 us with
// per-request pieces in longest-first order and 678-681 us with equal
// shares (same GPU, same run).
constexpr long kTargetWorkgroups = 256;
// Calls whose shares would be shorter than kSmallShare tokens at one
// workgroup per CU are latency-bound: each wave walks its few tiles one
// HBM round trip after another.  They get twice the workgroups (two fit on
// a CU), with shares of at least kMinPiece tokens (one tile per wave), as
// far as the state slots allow.  Measured on MI355X: 1 x 4096 tokens, 2 KV
// heads, one batched call, 9.9 -> 7.5 us (64 workgroups instead of 32);
// 1 x 16384 tokens, 8 KV heads (which would need 64 slots) took 16.5
// against 17.0 us with 64 slots, which made finalize slower.
constexpr long kSmallShare = 2048;
constexpr int kMinPiece = 128;
// Balancing tail (see the history kernel): the last kDefaultTailPermille
// thousandths of every share become tail units of guided sizes, each about
// 2 (tail tokens left) / W tokens, clamped to [kTailMin, kTailMax] and to
// the share's own tail, so the first claims are large and the last ones
// small.  Only calls whose shares have at least kTailMinShare tokens get
// the default tail (kTailMinShareExplicit for a fraction the caller set).
// Measured on MI355X, one batched call, tail on against off, alternated in
// one session: 64 ragged requests (shares of ~32K tokens) 667 -> 642 us;
// 32 x 131072 tokens (shares of 131072) 2505 -> 2423 us; 16 x 32768 tokens
// (shares of 16384) 321.0 -> 319.6 us on a GPU whose XCDs finished their
// shares within 278-309 us, and 344.2 -> 337.4 us on one where they
// finished within 290-340 us.  A tail of 150 thousandths, or pieces a
// quarter of that size, gained less.  A claimed unit costs about 4 us of
// start-up, claim and merge, and a round's first balanced launch needs the
// counter clear (about 4 us), so shorter shares are left alone.
constexpr int kDefaultTailPermille = 100;
constexpr long kTailMin = 256;
constexpr long kTailMax = 4096;
constexpr long kTailMinShare = 16384;          // with the default tail
constexpr long kTailMinShareExplicit = 4096;   // with a tail the caller asked for
// Density dispatch: units of 1 or 2 rows per KV head run the fp32 VALU body
// (built for that many rows), units of 3 or more the bf16 MFMA body, whose
// 16-row blocks would be 7/8 padding or more below that.  Measured on
// MI355X, one launch over 16 x 32768 tokens (same box, same run): 1 row per
// KV head 305.4 us on VALU against 307.1 us on MFMA, 2 rows 305.3-305.9
// against 301.8-305.9 us; at 4 rows the VALU body is bound by its own
// arithmetic (358.2 against 301.4 us), so it takes no unit of 3-4 rows by
// default.
constexpr int kDefaultMfmaMinRows = 3;

ss_status validate_desc(const ss_round_desc *d) {
  if (d == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "desc is null");
  if (d->num_requests < 1) return fail(SS_ERR_INVALID_ARGUMENT, "num_requests must be >= 1 (got %d)", d->num_requests);
  if (d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "head counts must be >= 1 (Hq=%d, Hkv=%d)", d->num_q_heads, d->num_kv_heads);
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(SS_ERR_INVALID_ARGUMENT, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)", d->num_q_heads,
                d->num_kv_heads);
  if (d->head_dim != ss::kHeadDim)
    return fail(SS_ERR_UNSUPPORTED, "head_dim %d is not built (only %d)", d->head_dim, ss::kHeadDim);
  if (!(d->softmax_scale > 0.f) || !std::isfinite(d->softmax_scale))
    return fail(SS_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  if (d->num_cand == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "num_cand is null");
  if (d->max_chunk_tokens < 1) return fail(SS_ERR_INVALID_ARGUMENT, "max_chunk_tokens must be >= 1");
  if (d->balance_permille > 500)
    return fail(SS_ERR_INVALID_ARGUMENT, "balance_permille = %d > 500 (a tail holds at most half of each share)",
                d->balance_permille);
  if (d->split_tokens < 0 || d->split_tokens % ss::kTile != 0)
    return fail(SS_ERR_INVALID_ARGUMENT, "split_tokens must be 0 or a positive multiple of %d", ss::kTile);
  if (d->mfma_min_rows < 0 || d->mfma_min_rows > ss::kMaxValuRows + 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "mfma_min_rows must be in [0, %d]", ss::kMaxValuRows + 1);
  if (d->counters_zeroed != 0 && d->counters_zeroed != 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "counters_zeroed must be 0 or 1");
  if (d->kv_layout != SS_KV_TOKEN_MAJOR && d->kv_layout != SS_KV_HEAD_MAJOR && d->kv_layout != SS_KV_HEAD_MAJOR_KV)
    return fail(SS_ERR_INVALID_ARGUMENT, "kv_layout must be SS_KV_TOKEN_MAJOR, SS_KV_HEAD_MAJOR or SS_KV_HEAD_MAJOR_KV");
  const int G = d->num_q_heads / d->num_kv_heads;
  long rows = 0;
  for (int b = 0; b < d->num_requests; ++b) {
    const int n = d->num_cand[b];
    if (n < 1 || n > SS_MAX_CANDIDATES)
      return fail(SS_ERR_INVALID_ARGUMENT, "num_cand[%d] = %d outside [1, %d]", b, n, SS_MAX_CANDIDATES);
    if (n * G > SS_MAX_ROWS_PER_KV_HEAD)
      return fail(SS_ERR_UNSUPPORTED, "request %d: n_b * Hq/Hkv = %d rows per KV head exceeds %d", b, n * G,
                  SS_MAX_ROWS_PER_KV_HEAD);
    rows += (long)n * d->num_q_heads;
  }
  if (rows * (long)ss::kNumSlots * ss::kHeadDim > (1L << 40))
    return fail(SS_ERR_INVALID_ARGUMENT, "round too large");
  if (rows * ss::kHeadDim * 2 >= (1L << 31))   // the kernels address Q with 32-bit byte offsets
    return fail(SS_ERR_INVALID_ARGUMENT, "round too large: the query tensor must stay below 2^31 bytes");
  return SS_OK;
}

// Workspace: slot states a, m, l, then the counter block of kClaimCounters
// words (the first is the balancing tail's claim counter).
size_t workspace_bytes_rows(long R) {
  const size_t a = align_up((size_t)ss::kNumSlots * R * ss::kHeadDim * sizeof(float), 256);
  const size_t m = align_up((size_t)ss::kNumSlots * R * sizeof(float), 256);
  return a + 2 * m + align_up(ss::kClaimCounters * sizeof(uint32_t), 256);
}

}  // namespace

struct ss_round {
  int32_t B, Hq, Hkv, G;
  float scale;
  int32_t max_chunk_tokens, split_tokens, mfma_min_rows, kv_layout, tail_permille;
  std::vector<int32_t> n_cand, row_off;
  uint32_t *counters = nullptr;      // the workspace's counter block (kClaimCounters words)
  bool counters_ready = false;       // the block is known to be zero (cleared, or the caller said so)
  std::vector<int32_t> slots_used;   // per request: state slots written so far this round
  const uint16_t *q;
  const uint16_t *kc = nullptr, *vc = nullptr;   // candidate K/V, attended by finalize
  ss::State st;
  bool cand_done = false;
  bool finalized = false;
  // A call failed after part of its work was enqueued (a launch or an
  // event record returned an error): the slots that work writes and the
  // host's record of them may disagree, so every later call is refused.
  bool failed = false;
};

struct ss_pipeline {
  char *slot[2];
  size_t slot_bytes;
  hipStream_t copy;
  hipEvent_t ready[2];
  hipEvent_t freed[2];
  bool used[2];
  int next;
  // An upload or the attention after it failed part-way: a slot's events
  // no longer describe its contents, so every later call is refused.
  bool failed = false;
};

namespace {

ss_status check_round(const ss_round *r) {
  if (r == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "round handle is null");
  if (r->failed) return fail(SS_ERR_BAD_STATE, "an earlier call of this round failed part-way; destroy the round");
  if (r->finalized) return fail(SS_ERR_BAD_STATE, "round already finalized");
  return SS_OK;
}

// Elements between consecutive tokens of one KV head in a chunk.
uint32_t tok_stride(const ss_round *r) {
  switch (r->kv_layout) {
    case SS_KV_TOKEN_MAJOR: return (uint32_t)(r->Hkv * ss::kHeadDim);
    case SS_KV_HEAD_MAJOR_KV: return 2 * ss::kHeadDim;
    default: return ss::kHeadDim;
  }
}

long max_piece_tokens(const ss_round *r) {
  // an item must stay below 2^31 bytes of one KV head (32-bit buffer offsets)
  const long per_tok = 2 * (long)tok_stride(r);
  return ((1L << 31) - 1024) / per_tok / ss::kTile * ss::kTile;
}

// Validate a (batched) history call; per-chunk totals in tot[c].
ss_status check_history_args(const ss_round *r, int nchunks, const void *const *k, const void *const *v,
                             const int32_t *len, std::vector<long> *tot) {
  ss_status s = check_round(r);
  if (s != SS_OK) return s;
  if (nchunks < 1 || nchunks > ss::kMaxChunks)
    return fail(SS_ERR_INVALID_ARGUMENT, "num_chunks = %d outside [1, %d]", nchunks, ss::kMaxChunks);
  if (len == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "len is null");
  const long cap = max_piece_tokens(r) * ss::kNumSlots;
  tot->assign(nchunks, 0);
  for (int c = 0; c < nchunks; ++c) {
    long t = 0;
    for (int b = 0; b < r->B; ++b) {
      const int32_t n = len[(size_t)c * r->B + b];
      if (n < 0) return fail(SS_ERR_INVALID_ARGUMENT, "len[%d][%d] = %d < 0", c, b, n);
      if ((long)n > cap) return fail(SS_ERR_INVALID_ARGUMENT, "len[%d][%d] = %d is too large", c, b, n);
      t += n;
    }
    if (t > r->max_chunk_tokens)
      return fail(SS_ERR_INVALID_ARGUMENT, "chunk %d has %ld tokens > max_chunk_tokens %d", c, t, r->max_chunk_tokens);
    if (t > 0 && (k == nullptr || v == nullptr || k[c] == nullptr || v[c] == nullptr || !aligned(k[c], 16) ||
                  !aligned(v[c], 16)))
      return fail(SS_ERR_INVALID_ARGUMENT, "chunk %d: k and v must be non-null and 16-byte aligned", c);
    if (t > 0 && r->kv_layout == SS_KV_HEAD_MAJOR_KV &&
        static_cast<const char *>(v[c]) != static_cast<const char *>(k[c]) + ss::kHeadDim * 2)
      return fail(SS_ERR_INVALID_ARGUMENT, "chunk %d: with SS_KV_HEAD_MAJOR_KV, v must be k + %d elements", c,
                  ss::kHeadDim);
    (*tot)[c] = t;
  }
  return SS_OK;
}

// Work of one history call.  Unit u = items [unit_first[u],
// unit_first[u + 1]): a chain of at most kMaxChain token ranges of one
// request, attended as one sequence into its own state slot by body
// kind[u].  Workgroup w (of every KV head) attends units [wg_first[w],
// wg_first[w + 1]) in order; units [tail_first, units()) are the balancing
// tail, claimed at run time by any workgroup for any KV head.
struct Plan {
  std::vector<ss::Item> items;
  std::vector<uint32_t> unit_first{0};
  std::vector<uint8_t> kind;
  std::vector<uint32_t> wg_first;
  std::vector<int32_t> slots_after;   // per request: slots in use after this call
  size_t tail_first = 0, num_tail = 0;
  size_t units() const { return kind.size(); }
};

// Kernel body of request b's units: VALU for few rows per KV head when the
// round asks for it, else MFMA with one to four 16-row blocks (three or four
// only on the wide kernel, which a launch with such a unit runs on, as
// row-split units).
int kind_of(const ss_round *r, int b) {
  const int min_rows = r->mfma_min_rows > 0 ? r->mfma_min_rows : kDefaultMfmaMinRows;
  const int M = r->n_cand[b] * r->G;
  if (M < min_rows && M <= ss::kMaxValuRows) return ss::kUnitValu;
  return M <= 16 ? ss::kUnitMfma1 : M <= 32 ? ss::kUnitMfma2 : M <= 48 ? ss::kUnitMfma3 : ss::kUnitMfma4;
}

// Split this call's tokens into W shares.  The requests' tokens (each
// request's ranges in chunk order) are concatenated in request order; share
// w is [x_w, x_{w+1}) with x_w = w * L / W moved down to a tile boundary of
// its request.  With tail_permille > 0, workgroup w keeps [x_w, y_w), y_w
// the same fraction (1 - tail_permille / 1000) of its share, and the rest
// of every share becomes tail pieces of about 2 (tail tokens left) / W
// tokens, at least tail_min and at most kTailMax, cut at tile boundaries
// (a remainder below tail_min joins the piece before it).
// Each request's part of a share or piece becomes units: its token ranges,
// cut at chunk boundaries and at pmax tokens, in chains of at most
// kMaxChain.  Returns false if a request would need more than kNumSlots
// slots.
bool build_plan(const ss_round *r, int nchunks, const int32_t *len, long W, long pmax, int tail_permille,
                long tail_min, Plan *plan) {
  const int B = r->B;
  *plan = Plan();
  plan->slots_after = r->slots_used;
  // per request: tokens before chunk c (cum), and offset of the request in chunk c (off)
  std::vector<long> cum((size_t)B * (nchunks + 1), 0), off((size_t)nchunks * B, 0), start(B + 1, 0);
  for (int c = 0; c < nchunks; ++c) {
    long o = 0;
    for (int b = 0; b < B; ++b) {
      off[(size_t)c * B + b] = o;
      o += len[(size_t)c * B + b];
    }
  }
  for (int b = 0; b < B; ++b) {
    for (int c = 0; c < nchunks; ++c)
      cum[(size_t)b * (nchunks + 1) + c + 1] = cum[(size_t)b * (nchunks + 1) + c] + len[(size_t)c * B + b];
    start[b + 1] = start[b] + cum[(size_t)b * (nchunks + 1) + nchunks];
  }
  const long L = start[B];
  // request holding global token position pos < L (skips requests without tokens)
  auto request_of = [&](long pos) {
    return (int)(std::upper_bound(start.begin(), start.end(), pos) - start.begin()) - 1;
  };
  // raw moved down to a tile boundary of its request, not below lo
  auto cut = [&](long raw, long lo) {
    if (raw >= L) return L;
    const int b = request_of(raw);
    const long o = raw - start[b];
    return std::max(lo, start[b] + o - o % ss::kTile);
  };
  std::vector<long> x(W + 1, L), y(W, 0);
  x[0] = 0;
  for (long w = 1; w < W; ++w) x[w] = cut(L * w / W, x[w - 1]);
  for (long w = 0; w < W; ++w)
    y[w] = tail_permille > 0 ? cut(x[w] + (x[w + 1] - x[w]) * (1000 - tail_permille) / 1000, x[w]) : x[w + 1];

  std::vector<int> slot(B, 0);
  long ranges = 0;   // items in the open unit
  int ub = -1;       // request of the open unit
  auto close = [&]() {
    if (ranges == 0) return;
    plan->unit_first.push_back((uint32_t)plan->items.size());
    plan->kind.push_back((uint8_t)kind_of(r, ub));
    ++slot[ub];
    ranges = 0;
  };
  // units of the global token range [lo_g, hi_g)
  auto emit = [&](long lo_g, long hi_g) {
    long pos = lo_g;
    while (pos < hi_g) {
      const int b = request_of(pos);
      const long lo = pos - start[b], hi = std::min(hi_g, start[b + 1]) - start[b];
      const long *cb = &cum[(size_t)b * (nchunks + 1)];
      int c = 0;
      for (long t = lo; t < hi;) {
        while (cb[c + 1] <= t) ++c;
        const long take = std::min({hi, cb[c + 1]}) - t;
        for (long q = 0; q < take;) {
          if (ranges == ss::kMaxChain) close();
          if (ranges == 0) {
            if (slot[b] >= ss::kNumSlots) return false;
            ub = b;
          }
          const long n = std::min(take - q, pmax);
          ss::Item it;
          it.tok_begin = (int32_t)(off[(size_t)c * B + b] + (t - cb[c]) + q);
          it.tok_count = (int32_t)n;
          it.q_row0 = r->row_off[b];
          it.n_cand = (uint8_t)r->n_cand[b];
          it.chunk = (uint8_t)c;
          it.slot = (uint8_t)slot[b];
          it.flags = slot[b] >= r->slots_used[b] ? ss::kSlotFresh : 0;
          plan->items.push_back(it);
          ++ranges;
          q += n;
        }
        t += take;
      }
      close();
      pos = start[b] + hi;
    }
    return true;
  };
  for (long w = 0; w < W; ++w) {
    plan->wg_first.push_back((uint32_t)plan->units());
    if (!emit(x[w], y[w])) return false;
  }
  plan->wg_first.push_back((uint32_t)plan->units());
  plan->tail_first = plan->units();
  long left = 0;
  for (long w = 0; w < W; ++w) left += x[w + 1] - y[w];
  for (long w = 0; w < W; ++w) {
    for (long pos = y[w]; pos < x[w + 1];) {
      long size = std::min(kTailMax, std::max(tail_min, 2 * left / W));
      size = (size + ss::kTile - 1) / ss::kTile * ss::kTile;
      // a remainder below the smallest piece joins this one
      const long end = pos + size + tail_min >= x[w + 1] ? x[w + 1] : cut(pos + size, pos + 1);
      if (!emit(pos, end)) return false;
      left -= end - pos;
      pos = end;
    }
  }
  plan->num_tail = plan->units() - plan->tail_first;
  for (int b = 0; b < B; ++b) plan->slots_after[b] = std::max(plan->slots_after[b], slot[b]);
  return true;
}

size_t unit_records(const Plan &plan, size_t w0, size_t w1);

bool fits_one_launch(const Plan &plan) {
  const size_t W = plan.wg_first.size() - 1;
  return W <= (size_t)ss::kMaxWgs && unit_records(plan, 0, W) + plan.num_tail <= (size_t)ss::kMaxUnits &&
         plan.items.size() <= (size_t)ss::kMaxItems;
}

ss_status plan_chunks(const ss_round *r, int nchunks, const int32_t *len, const std::vector<long> &tot,
                      Plan *plan) {
  long total = 0;
  for (long t : tot) total += t;
  long W;
  if (r->split_tokens > 0) {
    W = (total + r->split_tokens - 1) / r->split_tokens;
  } else {
    // Row-split units (three or four 16-row blocks) also get two workgroups
    // per CU: each of their tile steps is a barrier-bound chain of LDS and
    // MFMA latencies, which a second workgroup on the CU overlaps.
    bool wide = false;
    for (int c = 0; c < nchunks && !wide; ++c)
      for (int b = 0; b < r->B && !wide; ++b)
        wide = len[(size_t)c * r->B + b] > 0 && kind_of(r, b) >= ss::kUnitMfma3;
    W = std::max<long>(1, kTargetWorkgroups / r->Hkv);
    if (total / W < kSmallShare || wide) W = std::max<long>(1, 2 * kTargetWorkgroups / r->Hkv);
    W = std::min(W, std::max<long>(1, total / kMinPiece));
  }
  W = std::max<long>(1, std::min<long>(W, total));
  const long pmax = max_piece_tokens(r);
  // Fewer, larger shares until every request fits its units into the
  // slots; more, smaller ones while a share would exceed one launch's unit
  // or item table.
  bool shrunk = false;
  for (;;) {
    if (!build_plan(r, nchunks, len, W, pmax, 0, kTailMin, plan)) {
      if (W == 1) return fail(SS_ERR_INVALID_ARGUMENT, "too many token ranges per request for one history call");
      W = (W + 1) / 2;
      shrunk = true;
      continue;
    }
    bool fits = true;
    for (size_t w = 0; w + 1 < plan->wg_first.size(); ++w)
      if (plan->wg_first[w + 1] - plan->wg_first[w] > (uint32_t)ss::kMaxUnits ||
          plan->unit_first[plan->wg_first[w + 1]] - plan->unit_first[plan->wg_first[w]] > (uint32_t)ss::kMaxItems)
        fits = false;
    if (fits) break;
    if (shrunk || W >= total) return fail(SS_ERR_INVALID_ARGUMENT, "history call too fragmented for one workgroup's tables");
    W *= 2;
  }
  // Balancing tail: only for large shares, within one launch, while a claim
  // counter is left; coarser pieces if the finer ones need too many slots
  // or table entries, else none.
  const int permille = r->tail_permille == 0 ? kDefaultTailPermille : r->tail_permille;
  const long min_share = r->tail_permille == 0 ? kTailMinShare : kTailMinShareExplicit;
  if (permille > 0 && total / W >= min_share && fits_one_launch(*plan)) {
    Plan t;
    for (long tmin = kTailMin; tmin <= kTailMax; tmin *= 2)
      if (build_plan(r, nchunks, len, W, pmax, permille, tmin, &t) && fits_one_launch(t)) {
        *plan = std::move(t);
        break;
      }
  }
  return SS_OK;
}

ss::ChunkParams *base_params(const ss_round *r, int nchunks, const void *const *k, const void *const *v,
                             const std::vector<long> &tot) {
  static thread_local ss::ChunkParams p;
  p.q = r->q;
  p.st = r->st;
  p.Hq = r->Hq;
  p.Hkv = r->Hkv;
  p.G = r->G;
  p.scale_log2 = r->scale * 1.4426950408889634f;
  p.tok_stride = tok_stride(r);
  p.heads_fast = r->kv_layout == SS_KV_TOKEN_MAJOR ? 1 : 0;
  for (int c = 0; c < nchunks; ++c) {
    p.k[c] = static_cast<const uint16_t *>(k[c]);
    p.v[c] = static_cast<const uint16_t *>(v[c]);
    p.head_stride[c] = r->kv_layout == SS_KV_TOKEN_MAJOR ? (uint64_t)ss::kHeadDim : (uint64_t)tot[c] * tok_stride(r);
  }
  p.num_items = 0;
  p.num_units = 0;
  p.claim = nullptr;
  p.tail_first = 0;
  p.num_tail = 0;
  return &p;
}

// Launch the workgroups of `plan` in batches of at most kMaxWgs workgroups,
// kMaxUnits unit records and kMaxItems items with `launch(params)`.  A
// batch's records are the first unit of each of its workgroups (an empty
// record for a workgroup without units), then the further units in
// workgroup order, then the balancing tail.  A plan with a balancing tail
// is launched whole, tail units after the workgroups' own.
size_t unit_records(const Plan &plan, size_t w0, size_t w1) {
  size_t n = plan.wg_first[w1] - plan.wg_first[w0];
  for (size_t w = w0; w < w1; ++w) n += plan.wg_first[w + 1] == plan.wg_first[w];
  return n;
}

template <typename F>
hipError_t launch_units(ss::ChunkParams *p, const Plan &plan, F launch) {
  const size_t W = plan.wg_first.size() - 1;
  const size_t tail = plan.num_tail;
  size_t w0 = 0;
  while (w0 < W) {
    const uint32_t u0 = plan.wg_first[w0];
    const uint32_t i0 = plan.unit_first[u0];
    size_t w1 = w0, nrec = 0;   // records of workgroups [w0, w1)
    for (;;) {
      if (w1 == W || w1 - w0 == (size_t)ss::kMaxWgs) break;
      const size_t add = std::max<size_t>(1, plan.wg_first[w1 + 1] - plan.wg_first[w1]);
      if (nrec + add + tail > (size_t)ss::kMaxUnits ||
          plan.unit_first[plan.wg_first[w1 + 1]] - i0 > (uint32_t)ss::kMaxItems)
        break;
      nrec += add;
      ++w1;
    }
    if (w1 == w0) return hipErrorInvalidValue;   // one share over the table sizes (plan_chunks prevents it)
    const uint32_t u1 = plan.wg_first[w1];
    if (tail > 0 && !(w0 == 0 && w1 == W)) return hipErrorInvalidValue;   // plan_chunks keeps such plans whole
    const uint32_t uend = tail > 0 ? (uint32_t)plan.units() : u1;
    const uint32_t n = plan.unit_first[uend] - i0;
    std::memcpy(p->items, plan.items.data() + i0, n * sizeof(ss::Item));
    auto rec = [&](uint32_t u) {
      ss::UnitRec ur;
      const uint32_t f = plan.unit_first[u], nit = plan.unit_first[u + 1] - f;
      uint32_t ntiles = 0;
      for (uint32_t i = f; i < f + nit; ++i) ntiles += (uint32_t)((plan.items[i].tok_count + ss::kTile - 1) / ss::kTile);
      ur.word = ss::unit_word(f - i0, nit, plan.kind[u], plan.items[f].chunk);
      ur.ntiles = ntiles;
      ur.q_row0 = plan.items[f].q_row0;
      ur.n_cand = plan.items[f].n_cand;
      return ur;
    };
    const size_t nw = w1 - w0;
    size_t next = nw;   // further units start after the first-unit records
    for (size_t w = w0; w < w1; ++w) {
      const uint32_t a = plan.wg_first[w], b = plan.wg_first[w + 1];
      p->units[w - w0] = a < b ? rec(a) : ss::UnitRec{0u, 0u, 0, 0};
      p->more[w - w0] = (uint32_t)next;
      for (uint32_t u = a + 1; u < b; ++u) p->units[next++] = rec(u);
    }
    p->more[nw] = (uint32_t)next;
    const size_t tail_first = next;
    for (uint32_t u = u1; u < uend; ++u) p->units[next++] = rec(u);
    p->num_items = (int32_t)n;
    p->num_units = (int32_t)next;
    p->num_wgs = (int32_t)nw;
    p->tail_first = tail > 0 ? (int32_t)tail_first : 0;
    p->num_tail = tail > 0 ? (int32_t)tail : 0;
    const hipError_t e = launch(*p);
    if (e != hipSuccess) return e;
    w0 = w1;
  }
  return hipSuccess;
}

// Launch `items` in batches of kMaxItems with `launch(params)`.
template <typename P, typename F>
hipError_t launch_items(P *p, const std::vector<ss::Item> &items, F launch) {
  for (size_t i0 = 0; i0 < items.size(); i0 += ss::kMaxItems) {
    const size_t n = std::min<size_t>(ss::kMaxItems, items.size() - i0);
    std::memcpy(p->items, items.data() + i0, n * sizeof(ss::Item));
    p->num_items = (int32_t)n;
    const hipError_t e = launch(*p);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Before the round's first launch that uses the workspace's counter block:
// zero the block with a one-wave kernel unless it is known to be zero
// (ss_round_desc.counters_zeroed).  Every launch leaves the counters it used
// at zero, so one clear serves the whole round.
ss_status ensure_counters(ss_round *r, hipStream_t stream) {
  if (r->counters_ready) return SS_OK;
  const hipError_t e = ss::launch_clear_counters(r->counters, ss::kClaimCounters, stream);
  if (e != hipSuccess) {
    r->failed = true;
    return hip_fail(e, "counter clear launch");
  }
  r->counters_ready = true;
  return SS_OK;
}

// A validated and planned history call, ready to enqueue.
struct Prepared {
  std::vector<long> tot;
  long total = 0;
  Plan plan;
};

// Validate a history call and plan its launches; enqueues nothing.
ss_status prepare_history(const ss_round *r, int nchunks, const void *const *k, const void *const *v,
                          const int32_t *len, Prepared *pr) {
  ss_status s = check_history_args(r, nchunks, k, v, len, &pr->tot);
  if (s != SS_OK) return s;
  pr->total = 0;
  for (long t : pr->tot) pr->total += t;
  if (pr->total == 0) return SS_OK;
  return plan_chunks(r, nchunks, len, pr->tot, &pr->plan);
}

// Enqueue a prepared call: the stream waits for wait_before, the launches
// run, signal_after is recorded.  A HIP error after the first enqueued
// operation marks the round failed (its slots_used would no longer match
// what the device writes).
ss_status enqueue_history(ss_round *r, int nchunks, const void *const *k, const void *const *v,
                          const Prepared &pr, hipEvent_t wait_before, hipEvent_t signal_after, hipStream_t stream) {
  hipError_t e;
  if (wait_before != nullptr && (e = hipStreamWaitEvent(stream, wait_before, 0)) != hipSuccess)
    return hip_fail(e, "hipStreamWaitEvent (history)");
  if (pr.total > 0) {
    const Plan &plan = pr.plan;
    ss::ChunkParams *p = base_params(r, nchunks, k, v, pr.tot);
    if (plan.num_tail > 0) {
      ss_status s = ensure_counters(r, stream);
      if (s != SS_OK) return s;
      p->claim = r->counters;   // zero at launch; the launch's last claim leaves it zero
    }
    e = launch_units(p, plan, [&](const ss::ChunkParams &q) { return ss::launch_chunk(q, stream); });
    if (e != hipSuccess) {
      r->failed = true;
      return hip_fail(e, "history chunk kernel launch");
    }
    r->slots_used = plan.slots_after;   // the slots written by this call are valid from now on
  }
  if (signal_after != nullptr && (e = hipEventRecord(signal_after, stream)) != hipSuccess) {
    r->failed = true;
    return hip_fail(e, "hipEventRecord (history)");
  }
  return SS_OK;
}

ss_status attend_history(ss_round *r, int nchunks, const void *const *k, const void *const *v, const int32_t *len,
                         hipEvent_t wait_before, hipEvent_t signal_after, hipStream_t stream) {
  Prepared pr;
  ss_status s = prepare_history(r, nchunks, k, v, len, &pr);
  if (s != SS_OK) return s;
  return enqueue_history(r, nchunks, k, v, pr, wait_before, signal_after, stream);
}

// Finalize item of request b: the slots its history calls wrote.
ss::Item fin_item(const ss_round *r, int b) {
  ss::Item it{};
  it.tok_begin = 0;
  it.tok_count = r->slots_used[b];
  it.q_row0 = r->row_off[b];
  it.n_cand = (uint8_t)r->n_cand[b];
  return it;
}

bool check_out(float *out, float *lse, ss_status *s) {
  if (out == nullptr || !aligned(out, 16)) {
    *s = fail(SS_ERR_INVALID_ARGUMENT, "out must be non-null and 16-byte aligned");
    return false;
  }
  if (lse != nullptr && !aligned(lse, 4)) {
    *s = fail(SS_ERR_INVALID_ARGUMENT, "lse must be 4-byte aligned");
    return false;
  }
  return true;
}

// The finalize kernel: one wave per query row.
ss_status enqueue_finalize(ss_round *r, float *out, float *lse, hipStream_t stream) {
  static thread_local ss::FinalParams p;
  p.kc = r->kc;
  p.vc = r->vc;
  p.q = r->q;
  p.out = out;
  p.lse = lse;
  p.st = r->st;
  p.Hq = r->Hq;
  p.Hkv = r->Hkv;
  p.G = r->G;
  p.scale_log2 = r->scale * 1.4426950408889634f;
  std::vector<ss::Item> items(r->B);
  for (int b = 0; b < r->B; ++b) items[b] = fin_item(r, b);
  const hipError_t e = launch_items(&p, items, [&](const ss::FinalParams &q) { return ss::launch_finalize(q, stream); });
  if (e != hipSuccess) {
    r->failed = true;
    return hip_fail(e, "finalize kernel launch");
  }
  r->finalized = true;
  return SS_OK;
}

// Pointer checks of a host<->device copy: the host side must be pinned
// (page-locked) memory, the device side device memory.
ss_status check_copy(const void *dst, const void *src, size_t bytes, hipMemcpyKind kind) {
  const bool h2d = kind == hipMemcpyHostToDevice;
  const void *host = h2d ? src : dst;
  const void *dev = h2d ? dst : src;
  if (dst == nullptr || src == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "copy pointers must be non-null");
  if (bytes == 0) return fail(SS_ERR_INVALID_ARGUMENT, "copy of 0 bytes");
  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof attr);
  hipError_t e = hipPointerGetAttributes(&attr, host);
  if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return fail(SS_ERR_NOT_PINNED, "%s %p is not pinned host memory", h2d ? "upload source" : "download destination",
                host);
  }
  std::memset(&attr, 0, sizeof attr);
  e = hipPointerGetAttributes(&attr, dev);
  if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(SS_ERR_INVALID_ARGUMENT, "%s %p is not device memory", h2d ? "upload destination" : "download source",
                dev);
  }
  return SS_OK;
}

// Enqueue a checked copy on copy_stream: wait for wait_before, copy, record
// signal_after.  *enqueued (nullable) tells whether any of it reached the
// stream before an error.
ss_status enqueue_copy(void *dst, const void *src, size_t bytes, hipMemcpyKind kind, hipStream_t copy_stream,
                       hipEvent_t wait_before, hipEvent_t signal_after, bool *enqueued) {
  if (enqueued != nullptr) *enqueued = false;
  hipError_t e;
  if (wait_before != nullptr && (e = hipStreamWaitEvent(copy_stream, wait_before, 0)) != hipSuccess)
    return hip_fail(e, "hipStreamWaitEvent (copy)");
  if (enqueued != nullptr) *enqueued = wait_before != nullptr;
  if ((e = hipMemcpyAsync(dst, src, bytes, kind, copy_stream)) != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  if (enqueued != nullptr) *enqueued = true;
  if (signal_after != nullptr && (e = hipEventRecord(signal_after, copy_stream)) != hipSuccess)
    return hip_fail(e, "hipEventRecord (copy)");
  return SS_OK;
}

// Run an entry point's body with C++ exceptions turned into statuses: host
// allocation failures (std::vector, new) become SS_ERR_OUT_OF_MEMORY and
// nothing escapes the C ABI.  Every body allocates before it enqueues
// anything, so such a failure leaves the device work untouched.
template <typename F>
ss_status guarded(F body) {
  try {
    return body();
  } catch (const std::bad_alloc &) {
    return fail(SS_ERR_OUT_OF_MEMORY, "out of host memory");
  } catch (...) {
    return fail(SS_ERR_INVALID_ARGUMENT, "unexpected C++ exception in the library");
  }
}

}  // namespace

extern "C" {

size_t ss_round_workspace_bytes(const ss_round_desc *desc) {
  if (validate_desc(desc) != SS_OK) return 0;
  long R = 0;
  for (int b = 0; b < desc->num_requests; ++b) R += (long)desc->num_cand[b] * desc->num_q_heads;
  return workspace_bytes_rows(R);
}

}  // extern "C"

namespace {

// The common part of the round-init entry points: validate, lay out the
// workspace (slot states a, m, l, then the claim counters) and create the
// host handle.
ss_status init_round(ss_round **out, const ss_round_desc *desc, const void *q, void *workspace,
                     size_t workspace_bytes) {
  if (out == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  ss_status s = validate_desc(desc);
  if (s != SS_OK) return s;
  if (q == nullptr || !aligned(q, 16)) return fail(SS_ERR_INVALID_ARGUMENT, "q must be non-null and 16-byte aligned");
  long R = 0;
  for (int b = 0; b < desc->num_requests; ++b) R += (long)desc->num_cand[b] * desc->num_q_heads;
  const size_t need = workspace_bytes_rows(R);
  if (workspace == nullptr || !aligned(workspace, 256))
    return fail(SS_ERR_WORKSPACE, "workspace must be non-null and 256-byte aligned");
  if (workspace_bytes < need)
    return fail(SS_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);

  ss_round *r = new (std::nothrow) ss_round();
  if (r == nullptr) return fail(SS_ERR_OUT_OF_MEMORY, "out of host memory");
  r->B = desc->num_requests;
  r->Hq = desc->num_q_heads;
  r->Hkv = desc->num_kv_heads;
  r->G = r->Hq / r->Hkv;
  r->scale = desc->softmax_scale;
  r->max_chunk_tokens = desc->max_chunk_tokens;
  r->split_tokens = desc->split_tokens;
  r->mfma_min_rows = desc->mfma_min_rows;
  try {
    r->n_cand.assign(desc->num_cand, desc->num_cand + desc->num_requests);
    r->row_off.resize(r->B);
    r->slots_used.assign(r->B, 0);   // every slot starts empty: nothing to enqueue
  } catch (const std::bad_alloc &) {
    delete r;
    return fail(SS_ERR_OUT_OF_MEMORY, "out of host memory");
  }
  int32_t acc = 0;
  for (int b = 0; b < r->B; ++b) {
    r->row_off[b] = acc;
    acc += r->n_cand[b];
  }
  r->q = static_cast<const uint16_t *>(q);
  char *ws = static_cast<char *>(workspace);
  const size_t a_bytes = align_up((size_t)ss::kNumSlots * R * ss::kHeadDim * sizeof(float), 256);
  const size_t m_bytes = align_up((size_t)ss::kNumSlots * R * sizeof(float), 256);
  r->st.a = reinterpret_cast<float *>(ws);
  r->st.m = reinterpret_cast<float *>(ws + a_bytes);
  r->st.l = reinterpret_cast<float *>(ws + a_bytes + m_bytes);
  r->counters = reinterpret_cast<uint32_t *>(ws + a_bytes + 2 * m_bytes);
  r->counters_ready = desc->counters_zeroed != 0;
  r->tail_permille = desc->balance_permille;
  r->st.R = (int32_t)R;
  r->kv_layout = desc->kv_layout;
  *out = r;
  return SS_OK;
}

}  // namespace

extern "C" {

ss_status ss_round_init(ss_round **out, const ss_round_desc *desc, const void *q, void *workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  (void)stream;   // the empty state is tracked on the host: nothing to enqueue
  return init_round(out, desc, q, workspace, workspace_bytes);
}

ss_status ss_upload_chunk(void *dst_device, const void *src_pinned_host, size_t bytes, hipStream_t copy_stream,
                          hipEvent_t wait_before, hipEvent_t signal_after) {
  ss_status s = check_copy(dst_device, src_pinned_host, bytes, hipMemcpyHostToDevice);
  if (s != SS_OK) return s;
  return enqueue_copy(dst_device, src_pinned_host, bytes, hipMemcpyHostToDevice, copy_stream, wait_before,
                      signal_after, nullptr);
}

ss_status ss_attend_history_chunk(ss_round *r, const void *k, const void *v, const int32_t *len,
                                  hipEvent_t wait_before, hipEvent_t signal_after, hipStream_t stream) {
  const void *kk[1] = {k};
  const void *vv[1] = {v};
  return guarded([&] { return attend_history(r, 1, kk, vv, len, wait_before, signal_after, stream); });
}

ss_status ss_attend_history_chunks(ss_round *r, int32_t num_chunks, const void *const *k, const void *const *v,
                                   const int32_t *len, hipEvent_t wait_before, hipEvent_t signal_after,
                                   hipStream_t stream) {
  return guarded([&] { return attend_history(r, num_chunks, k, v, len, wait_before, signal_after, stream); });
}

ss_status ss_attend_local_candidates(ss_round *r, const void *k_cand, const void *v_cand, hipStream_t stream) {
  ss_status s = check_round(r);
  if (s != SS_OK) return s;
  if (r->cand_done) return fail(SS_ERR_BAD_STATE, "local candidates already attended for this round");
  if (k_cand == nullptr || v_cand == nullptr || !aligned(k_cand, 16) || !aligned(v_cand, 16))
    return fail(SS_ERR_INVALID_ARGUMENT, "k_cand and v_cand must be non-null and 16-byte aligned");
  // the frontier pass runs inside the finalize kernel (fused with the slot
  // merge and the normalisation); the result does not depend on the order
  (void)stream;
  r->kc = static_cast<const uint16_t *>(k_cand);
  r->vc = static_cast<const uint16_t *>(v_cand);
  r->cand_done = true;
  return SS_OK;
}

ss_status ss_round_finalize(ss_round *r, float *out, float *lse, hipStream_t stream) {
  return guarded([&]() -> ss_status {
    ss_status s = check_round(r);
    if (s != SS_OK) return s;
    if (!r->cand_done) return fail(SS_ERR_BAD_STATE, "finalize before ss_attend_local_candidates");
    if (!check_out(out, lse, &s)) return s;
    return enqueue_finalize(r, out, lse, stream);
  });
}

ss_status ss_round_init_scratch(ss_round **out, const ss_round_desc *desc, const void *q, hipStream_t stream) {
  (void)stream;
  if (out == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  const size_t need = ss_round_workspace_bytes(desc);
  if (need == 0) return validate_desc(desc);   // sets the detail
  if (need > ss::kScratchBytes)
    return fail(SS_ERR_WORKSPACE, "the round needs %zu bytes of workspace; the library's scratch holds %zu",
                need, ss::kScratchBytes);
  void *scratch = nullptr;
  const hipError_t e = ss::scratch_address(&scratch);
  if (e != hipSuccess) return hip_fail(e, "scratch address lookup");
  const ss_status st = init_round(out, desc, q, scratch, ss::kScratchBytes);
  // The counter block sits at the end of this round's share of the scratch,
  // where an earlier round of another size may have left state: always clear.
  if (st == SS_OK) (*out)->counters_ready = false;
  return st;
}

void ss_round_destroy(ss_round *r) { delete r; }

ss_status ss_pipeline_create(ss_pipeline **out, void *staging0, void *staging1, size_t slot_bytes,
                             hipStream_t copy_stream) {
  if (out == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (staging0 == nullptr || staging1 == nullptr || !aligned(staging0, 256) || !aligned(staging1, 256))
    return fail(SS_ERR_INVALID_ARGUMENT, "staging slots must be non-null and 256-byte aligned");
  if (slot_bytes == 0) return fail(SS_ERR_INVALID_ARGUMENT, "slot_bytes must be > 0");
  ss_pipeline *p = new (std::nothrow) ss_pipeline();
  if (p == nullptr) return fail(SS_ERR_OUT_OF_MEMORY, "out of host memory");
  p->slot[0] = static_cast<char *>(staging0);
  p->slot[1] = static_cast<char *>(staging1);
  p->slot_bytes = slot_bytes;
  p->copy = copy_stream;
  p->used[0] = p->used[1] = false;
  p->next = 0;
  for (int i = 0; i < 2; ++i) {
    hipError_t e = hipEventCreateWithFlags(&p->ready[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&p->freed[i], hipEventDisableTiming);
    if (e != hipSuccess) {
      for (int j = 0; j < i; ++j) {
        (void)hipEventDestroy(p->ready[j]);
        (void)hipEventDestroy(p->freed[j]);
      }
      delete p;
      return hip_fail(e, "pipeline event creation");
    }
  }
  *out = p;
  return SS_OK;
}

ss_status ss_pipeline_attend_chunks(ss_pipeline *p, ss_round *r, int32_t num_chunks, const void *host_kv,
                                    const int32_t *len, hipStream_t stream) {
  return guarded([&]() -> ss_status {
  if (p == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "pipeline is null");
  if (p->failed) return fail(SS_ERR_BAD_STATE, "an earlier call of this pipeline failed part-way; destroy it");
  ss_status s = check_round(r);
  if (s != SS_OK) return s;
  if (num_chunks < 1 || num_chunks > ss::kMaxChunks)
    return fail(SS_ERR_INVALID_ARGUMENT, "num_chunks = %d outside [1, %d]", num_chunks, ss::kMaxChunks);
  if (len == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "len is null");
  // chunk c occupies [off[c], off[c] + 2 * half[c]) of the slot: its K, then
  // its V (SS_KV_HEAD_MAJOR_KV: one buffer of K and V rows)
  const int sl = p->next;
  std::vector<const void *> kk(num_chunks), vv(num_chunks);
  size_t bytes = 0;
  for (int c = 0; c < num_chunks; ++c) {
    long total = 0;
    for (int b = 0; b < r->B; ++b) total += std::max<int32_t>(0, len[(size_t)c * r->B + b]);
    const size_t half = (size_t)total * r->Hkv * ss::kHeadDim * 2;
    kk[c] = p->slot[sl] + bytes;
    vv[c] = p->slot[sl] + bytes + (r->kv_layout == SS_KV_HEAD_MAJOR_KV ? ss::kHeadDim * 2 : half);
    bytes += 2 * half;
  }
  // everything that can be refused is checked (and the launches planned)
  // before the upload is enqueued
  Prepared pr;
  s = prepare_history(r, num_chunks, kk.data(), vv.data(), len, &pr);
  if (s != SS_OK) return s;
  if (bytes == 0) return SS_OK;
  if (host_kv == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "host_kv is null");
  if (bytes > p->slot_bytes)
    return fail(SS_ERR_INVALID_ARGUMENT, "chunks need %zu bytes > slot_bytes %zu", bytes, p->slot_bytes);
  s = check_copy(p->slot[sl], host_kv, bytes, hipMemcpyHostToDevice);
  if (s != SS_OK) return s;
  bool enqueued = false;
  s = enqueue_copy(p->slot[sl], host_kv, bytes, hipMemcpyHostToDevice, p->copy, p->used[sl] ? p->freed[sl] : nullptr,
                   p->ready[sl], &enqueued);
  if (s != SS_OK) {
    // a wait or copy already on the copy stream leaves the slot's events
    // out of step with its contents
    if (enqueued) p->failed = true;
    return s;
  }
  s = enqueue_history(r, num_chunks, kk.data(), vv.data(), pr, p->ready[sl], p->freed[sl], stream);
  if (s != SS_OK) {
    // the upload is in flight and the slot's free event may never be
    // recorded after its readers
    p->failed = true;
    return s;
  }
  p->used[sl] = true;
  p->next = sl ^ 1;
  return SS_OK;
  });
}

ss_status ss_pipeline_attend_chunk(ss_pipeline *p, ss_round *r, const void *host_kv, const int32_t *len,
                                   hipStream_t stream) {
  return ss_pipeline_attend_chunks(p, r, 1, host_kv, len, stream);
}

void ss_pipeline_destroy(ss_pipeline *p) {
  if (p == nullptr) return;
  for (int i = 0; i < 2; ++i) {
    (void)hipEventDestroy(p->ready[i]);
    (void)hipEventDestroy(p->freed[i]);
  }
  delete p;
}

ss_status ss_probe_read(const void *buf, size_t bytes, uint32_t *sink, int32_t workgroups, hipStream_t stream) {
  if (buf == nullptr || sink == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "buffer and sink must be non-null");
  if (bytes == 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return fail(SS_ERR_INVALID_ARGUMENT, "the buffer must be 16-byte aligned and a non-zero multiple of 16 bytes");
  if (reinterpret_cast<uintptr_t>(sink) % 4 != 0) return fail(SS_ERR_INVALID_ARGUMENT, "sink is not 4-byte aligned");
  if (workgroups < 1 || workgroups > 65536) return fail(SS_ERR_INVALID_ARGUMENT, "workgroups must be in 1..65536");
  const uint64_t share = (bytes / 16 + (uint64_t)workgroups - 1) / (uint64_t)workgroups * 16;
  if (share > ss::kProbeMaxShare)
    return fail(SS_ERR_INVALID_ARGUMENT, "%llu bytes per workgroup; at most %llu", (unsigned long long)share,
                (unsigned long long)ss::kProbeMaxShare);
  for (const void *ptr : {static_cast<const void *>(buf), static_cast<const void *>(sink)}) {
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof attr);
    const hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
      (void)hipGetLastError();
      return fail(SS_ERR_INVALID_ARGUMENT, "%p is not device memory", ptr);
    }
  }
  const hipError_t e = ss::launch_read_probe(buf, bytes, share, sink, workgroups, stream);
  if (e != hipSuccess) return hip_fail(e, "read probe launch");
  return SS_OK;
}

ss_status ss_event_create(hipEvent_t *e) {
  if (e == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "event pointer is null");
  const hipError_t h = hipEventCreateWithFlags(e, hipEventDisableTiming);
  if (h != hipSuccess) return hip_fail(h, "hipEventCreateWithFlags");
  return SS_OK;
}

void ss_event_destroy(hipEvent_t e) {
  if (e != nullptr) (void)hipEventDestroy(e);
}

const char *ss_status_string(ss_status s) {
  switch (s) {
    case SS_OK: return "SS_OK";
    case SS_ERR_INVALID_ARGUMENT: return "SS_ERR_INVALID_ARGUMENT";
    case SS_ERR_UNSUPPORTED: return "SS_ERR_UNSUPPORTED";
    case SS_ERR_BAD_STATE: return "SS_ERR_BAD_STATE";
    case SS_ERR_NOT_PINNED: return "SS_ERR_NOT_PINNED";
    case SS_ERR_WORKSPACE: return "SS_ERR_WORKSPACE";
    case SS_ERR_HIP: return "SS_ERR_HIP";
    case SS_ERR_OUT_OF_MEMORY: return "SS_ERR_OUT_OF_MEMORY";
    default: return "SS_ERR_UNKNOWN";
  }
}

const char *ss_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
