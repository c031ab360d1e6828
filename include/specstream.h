/*
 * specstream.h -- C ABI of the chunk-streamed speculative-verification
 * attention library (libspecstream.so, gfx950 / MI355X).
 *
 * What it computes (paper Sec. 4.2, "KV Streaming for Multi-Query
 * Verification"): in one verification round every request b of a Cohort has
 * n_b candidate queries (the k_b draft tokens plus one, at positions C_b + i)
 * that attend to
 *   - the committed history [0, C_b), delivered as chunks of tokens that are
 *     each read once for all n_b * Hq queries of the request (Sec. 4.2,
 *     "chunked verification shared across queries"), and
 *   - the GPU-resident Speculative Frontier (Eq. 8): candidate keys j with
 *     j <= i (causal mask by absolute position, Sec. 4.2).
 * The result equals full attention (Eq. 12, Eq. 17): per query and head an
 * online-softmax state (m, l, a) starts at (-inf, 0, 0) (Sec. 4.2), each chunk
 * contributes its local state (Eq. 13) through the rescaled merge (Eq. 14),
 * and O = a / l at the end.
 *
 * Conventions shared by every call
 *   - bf16 = IEEE bfloat16 bit patterns (uint16); all device arrays are
 *     row-major and 16-byte aligned.
 *   - Query rows are packed in request order: row (b, i) = off_b + i with
 *     off_b = sum_{b'<b} n_b'.  Q and O are [sum n_b, Hq, d]; candidate K/V
 *     are [sum n_b, Hkv, d].
 *   - A history chunk is token-major [sum_b len_b, Hkv, d] with request b's
 *     len_b tokens contiguous and requests in order, so a Cohort's chunk is
 *     one contiguous buffer (K and V are two such buffers).
 *   - GQA: query head h reads KV head floor(h / G), G = Hq / Hkv.
 *   - Q and K arrive with any positional encoding applied; softmax_scale
 *     multiplies the dot product (1/sqrt(d) in the paper, Sec. 4.2).
 *   - Ownership: the caller owns every buffer, stream and event and keeps
 *     them alive until the enqueued work has finished.  The library never
 *     allocates device memory at run time; its state is the host handles
 *     and the static device scratch that ss_round_init_scratch uses.
 *   - Asynchrony: calls validate, enqueue on the given stream and return.
 *     A non-OK status means nothing was enqueued by that call, except
 *     SS_ERR_HIP, reported when a HIP call itself fails: if part of the
 *     call's work had already been enqueued, the round (and a pipeline the
 *     call went through) is marked failed and refuses every later call with
 *     SS_ERR_BAD_STATE; destroy it.  Device faults surface at the caller's
 *     synchronisation.
 *   - All calls of one round go to one stream (or are ordered by events);
 *     calls of one round that overlap on different streams race.
 *   - Threading: one host thread per handle at a time.  ss_last_error() is
 *     thread-local.
 */
#ifndef SPECSTREAM_H
#define SPECSTREAM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ss_round ss_round;       /* opaque host handle of one round */
typedef struct ss_pipeline ss_pipeline; /* opaque two-slot upload pipeline */
typedef int32_t ss_status;

enum {
  SS_OK = 0,
  SS_ERR_INVALID_ARGUMENT = -1, /* null/misaligned pointer, bad size or count */
  SS_ERR_UNSUPPORTED = -2,      /* valid but not built: head_dim != 128, rows per KV head > 64 */
  SS_ERR_BAD_STATE = -3,        /* call out of order for this round */
  SS_ERR_NOT_PINNED = -4,       /* upload source is not pinned (page-locked) host memory */
  SS_ERR_WORKSPACE = -5,        /* workspace null, misaligned or too small */
  SS_ERR_HIP = -6,              /* a HIP runtime call failed (detail in ss_last_error) */
  SS_ERR_OUT_OF_MEMORY = -7     /* a host allocation of the library failed; nothing was enqueued */
};

/* Largest candidate count per request (k_b + 1).  The paper's widths are
 * q in {2, 4, 6, 8} (Sec. 5.1). */
#define SS_MAX_CANDIDATES 8
/* Rows that share one KV head, n_b * Hq / Hkv, must not exceed this (64
 * covers GQA groups of 8 query heads at the paper's largest width, q = 8).
 * A history call with a request of more than 32 such rows runs on a kernel
 * variant in which each wave attends every tile for 16 of the rows, with
 * two workgroups per CU. */
#define SS_MAX_ROWS_PER_KV_HEAD 64

typedef struct {
  int32_t num_requests;     /* B >= 1: one Cohort (Sec. 4.2, Cohort batching)  */
  int32_t num_q_heads;      /* Hq >= 1, Hq % Hkv == 0                          */
  int32_t num_kv_heads;     /* Hkv >= 1                                        */
  int32_t head_dim;         /* d; only 128 is built (else SS_ERR_UNSUPPORTED)  */
  float softmax_scale;      /* sigma > 0, finite; 1/sqrt(d) in the paper       */
  const int32_t *num_cand;  /* host [B]: n_b = k_b + 1, 1 <= n_b <= 8, copied  */
  int32_t max_chunk_tokens; /* >= 1: bound on sum_b len_b of one history call  */
  int32_t split_tokens;     /* tokens per workgroup share: a history call's
                               tokens (all requests, in request order) are
                               split into equal shares of about this many,
                               one per workgroup and KV head; 0 = automatic
                               (one workgroup per CU, two per CU for calls
                               whose shares would be below 2048 tokens or
                               with a request of more than 32 rows per KV
                               head);
                               else a multiple of 32                           */
  int32_t mfma_min_rows;    /* rows per KV head (n_b * G) from which the bf16
                               MFMA path is used; fewer (at most 4) use the
                               fp32 VALU path.  0 = default (3: VALU for 1-2
                               rows, where MFMA blocks would be mostly
                               padding and both bodies run at the HBM rate;
                               MFMA from 3 rows); 1 = always MFMA; 2..5 =
                               VALU below that many rows; range 0..5           */
  int32_t kv_layout;        /* layout of history chunks: SS_KV_TOKEN_MAJOR
                               [sum_b len_b][Hkv][d], SS_KV_HEAD_MAJOR
                               [Hkv][sum_b len_b][d] or SS_KV_HEAD_MAJOR_KV
                               [Hkv][sum_b len_b][2][d] (K and V rows of a
                               token adjacent)                                 */
  int32_t balance_permille; /* thousandths of every workgroup share held back
                               as a tail of small units that workgroups of
                               any KV head claim once their own share is done
                               (the GPU's dies stream at different rates);
                               0 = default (100), < 0 = no tail, at most 500.
                               The default applies to history calls whose
                               shares hold at least 16384 tokens, a value set
                               here from 4096; the result is the same bitwise
                               whichever workgroup attends a unit              */
  int32_t counters_zeroed;  /* the workspace ends with a block of counters
                               (the balancing tail's claim counter) that must
                               be zero when a history launch that uses it
                               starts; every such launch leaves it zero.
                               0 = the library zeroes the block with a
                               one-wave kernel before the round's first launch
                               that uses it.  1 = the caller guarantees it is
                               zero: the workspace was zero-filled when it was
                               allocated and has since been written only by
                               rounds of this library whose work completed
                               without error (a serving loop reusing one
                               workspace), so no clear is enqueued.  A block
                               that is not zero when promised gives wrong
                               results (never an access outside the
                               workspace).                                    */
} ss_round_desc;

/* History chunk layouts (ss_round_desc.kv_layout).  In all, request b's
 * len_b tokens follow request b-1's; head-major keeps each KV head's tokens
 * contiguous (one contiguous stream per workgroup for K and one for V).
 * SS_KV_HEAD_MAJOR_KV keeps K and V of one chunk in one buffer, each token's
 * K row followed by its V row, so a workgroup reads a single contiguous
 * stream; the chunk's v pointer must then be its k pointer + d elements. */
#define SS_KV_TOKEN_MAJOR 0
#define SS_KV_HEAD_MAJOR 1
#define SS_KV_HEAD_MAJOR_KV 2

/* Bytes of device workspace a round with this descriptor needs (fp32
 * online-softmax states of every query row, per split slot, then a 256-byte
 * counter block whose first word is the balancing tail's claim counter).  0
 * if the descriptor is invalid (see ss_last_error). */
size_t ss_round_workspace_bytes(const ss_round_desc *desc);

/* Start a round (paper Sec. 4.2: state (m, l, a) = (-inf, 0, 0) per query and
 * head).  q: device bf16 [sum n_b, Hq, d], read by the later calls, so it
 * must stay unchanged until ss_round_finalize's work has completed.
 * workspace: device, 256-byte aligned, >= ss_round_workspace_bytes(desc);
 * owned by the round until finalize's work has completed.  The empty state
 * is tracked on the host (a split slot is written before it is ever read),
 * so this call enqueues nothing on `stream`; unless desc->counters_zeroed is
 * set, the round's first history call with a balancing tail enqueues a
 * one-wave kernel that zeroes the counter block before its attention
 * launch.
 * On success *out receives a new handle (free with ss_round_destroy). */
ss_status ss_round_init(ss_round **out, const ss_round_desc *desc, const void *q,
                        void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Copy one history chunk (or any byte range) from pinned host memory to the
 * device on a side stream (paper Sec. 4.2, "Pipelined KV transfers": chunks
 * move host->device while the previous chunk is being attended).
 * If wait_before is non-null, copy_stream first waits for it (the staging
 * slot's "free" event); if signal_after is non-null it is recorded on
 * copy_stream after the copy (the slot's "ready" event).  src must be
 * page-locked host memory (hipHostMalloc / pinned tensors), else
 * SS_ERR_NOT_PINNED; dst must be device memory.  bytes > 0. */
ss_status ss_upload_chunk(void *dst_device, const void *src_pinned_host, size_t bytes,
                          hipStream_t copy_stream, hipEvent_t wait_before, hipEvent_t signal_after);

/* Attend one history chunk for every request of the round (paper Sec. 4.2:
 * S_j = Q K_j^T / sqrt(d) for the whole query group, Eq. 13 local state,
 * Eq. 14 merge into the running state).  k, v: device bf16 chunks in the
 * round's kv_layout (token-major [sum_b len_b, Hkv, d] or head-major
 * [Hkv, sum_b len_b, d]).  len: host [B], len_b >= 0 (0 = request has no tokens in
 * this chunk), sum <= max_chunk_tokens.  History tokens are visible to every
 * candidate query.  Chunks may come in any order and any number (>= 0),
 * before or after ss_attend_local_candidates.  If wait_before is non-null the
 * stream waits for it first (chunk ready); if signal_after is non-null it is
 * recorded after the last kernel reading k and v (chunk buffer free). */
ss_status ss_attend_history_chunk(ss_round *r, const void *k, const void *v, const int32_t *len,
                                  hipEvent_t wait_before, hipEvent_t signal_after, hipStream_t stream);

/* Attend several history chunks in one launch (paper Sec. 4.2, transfer
 * batching: one launch serves a group of adjacent chunks, so its fixed
 * costs are paid once for the group).  Same semantics as num_chunks calls of
 * ss_attend_history_chunk, in any order.  k, v: host arrays [num_chunks] of
 * device chunk pointers (each chunk in the round's kv_layout); len: host
 * [num_chunks][B] token counts; 1 <= num_chunks <= 32.  wait_before and
 * signal_after bracket the whole batch. */
ss_status ss_attend_history_chunks(ss_round *r, int32_t num_chunks, const void *const *k,
                                   const void *const *v, const int32_t *len, hipEvent_t wait_before,
                                   hipEvent_t signal_after, hipStream_t stream);

/* Attend the Speculative Frontier (paper Sec. 4.2, GPU-resident pass): query
 * i of request b sees candidate keys j <= i of the same request.  k_cand,
 * v_cand: device bf16 [sum n_b, Hkv, d].  Exactly once per round.  The pass
 * is executed by the kernel ss_round_finalize enqueues (fused with the split
 * merge and the normalisation), so k_cand and v_cand must stay valid and
 * unchanged until finalize's work has completed; this call enqueues nothing. */
ss_status ss_attend_local_candidates(ss_round *r, const void *k_cand, const void *v_cand,
                                     hipStream_t stream);

/* Finish the round: merge the split states (Eq. 14) and write O = a / l
 * (paper Sec. 4.2, Eq. 17).  out: device fp32 [sum n_b, Hq, d].  lse: null or
 * device fp32 [sum n_b, Hq], natural-log sum of exp of the scaled scores
 * (m + ln l).  Requires ss_attend_local_candidates to have been called.
 * After finalize the handle accepts no more calls except destroy. */
ss_status ss_round_finalize(ss_round *r, float *out, float *lse, hipStream_t stream);

/* Free the host handle (never device memory).  Null is ignored.  Call it
 * after enqueueing finalize; enqueued work does not use the handle. */
void ss_round_destroy(ss_round *r);

/* Two-slot host->device pipeline (paper Sec. 4.2: two GPU staging buffers,
 * separate transfer and compute streams; buffer A is attended while B
 * receives the next chunk, and a buffer is refilled only after the whole
 * query group has consumed it).  staging0/1: device buffers of slot_bytes
 * each, owned by the caller.  copy_stream: the transfer stream.  The
 * pipeline owns four events (ready/free per slot), created here. */
ss_status ss_pipeline_create(ss_pipeline **out, void *staging0, void *staging1, size_t slot_bytes,
                             hipStream_t copy_stream);

/* Upload one history chunk into the next staging slot and attend it:
 *   copy_stream: wait free[s]; copy host_kv -> slot s; record ready[s]
 *   stream:      wait ready[s]; ss_attend_history_chunk; record free[s]
 * host_kv: pinned host bf16, the chunk's K then its V, each in the round's
 * kv_layout ([sum_b len_b][Hkv][d] or [Hkv][sum_b len_b][d]), contiguous
 * (SS_KV_HEAD_MAJOR_KV: the chunk's one [Hkv][sum_b len_b][2][d] buffer);
 * len as in ss_attend_history_chunk.  The chunk may belong
 * to any round (e.g. the next layer), so transfers run ahead across layer
 * boundaries. */
ss_status ss_pipeline_attend_chunk(ss_pipeline *p, ss_round *r, const void *host_kv,
                                   const int32_t *len, hipStream_t stream);

/* Transfer batch (paper Sec. 4.2): num_chunks adjacent history chunks go to
 * the next staging slot as one copy and are attended by one launch, as
 * ss_attend_history_chunks does, so the copy's and the launch's fixed costs
 * are paid once for the group.  host_kv: pinned host memory holding chunk 0's K, chunk 0's V, chunk
 * 1's K, ... contiguously (each in the round's kv_layout; with
 * SS_KV_HEAD_MAJOR_KV each chunk's one K-and-V buffer); len: host
 * [num_chunks][B]; 1 <= num_chunks <= 32; the batch must fit slot_bytes. */
ss_status ss_pipeline_attend_chunks(ss_pipeline *p, ss_round *r, int32_t num_chunks, const void *host_kv,
                                    const int32_t *len, hipStream_t stream);

/* Destroy the pipeline's events (after its work has completed). */
void ss_pipeline_destroy(ss_pipeline *p);

/* ---- Commit-aware KV tiering (paper Sec. 4.1) ------------------------------
 * Per request the Target KV is split at 0 <= H <= C <= L (Eq. 8):
 *   [0, H)  Sealed History       host (pinned memory), streamed as chunks
 *   [H, C)  Active Tail          GPU, committed tokens not yet migrated
 *   [C, L)  Speculative Frontier GPU, candidates awaiting verification
 * Committed tokens more than T behind C move to the host in blocks of g
 * tokens.  The boundary H moves forward only once a migration's copy is
 * done (ss_tier_complete).  A rejected suffix of the frontier lies at or
 * after C >= H, so releasing it touches GPU memory only and never the
 * host copy. */

/* Eq. 9: end of the next migration, E = max(H, g * floor(max(0, C - T) / g)).
 * Requires H >= 0, C >= H, T >= 0, g >= 1 and H a multiple of g; returns -1
 * otherwise.  E == H means nothing to migrate. */
int64_t ss_tier_endpoint(int64_t H, int64_t C, int64_t T, int64_t g);

typedef struct ss_tier ss_tier;   /* opaque host-side boundaries of a Cohort */

/* New tiering state for num_requests requests, all boundaries 0; tail_target
 * = T >= 0 tokens kept on the GPU, granularity = g >= 1 tokens per migration
 * block.  Host memory only; free with ss_tier_destroy. */
ss_status ss_tier_create(ss_tier **out, int32_t num_requests, int64_t tail_target, int64_t granularity);
void ss_tier_destroy(ss_tier *t);

/* Boundaries of request b (each pointer nullable). */
ss_status ss_tier_get(const ss_tier *t, int32_t b, int64_t *H, int64_t *C, int64_t *L);

/* n >= 0 new tokens enter the frontier (the round's candidates, or a
 * prompt before its commit): L += n. */
ss_status ss_tier_extend(ss_tier *t, int32_t b, int64_t n);

/* Verification kept the first `accepted` frontier tokens (0 <= accepted <=
 * L - C): C' = C + accepted; the suffix [C', L) is released (its range is
 * returned through the nullable released_* pointers) and L = C'. */
ss_status ss_tier_commit(ss_tier *t, int32_t b, int64_t accepted, int64_t *released_begin,
                         int64_t *released_end);

/* Plan request b's next migration (Eq. 9).  If none is in flight and E > H,
 * [H, E) is marked in flight and returned; otherwise begin == end.  The
 * caller copies those tokens' K/V (ss_download_range) and calls
 * ss_tier_complete once the copy has completed. */
ss_status ss_tier_plan(ss_tier *t, int32_t b, int64_t *begin, int64_t *end);

/* The in-flight migration of request b has completed: H = E, and the GPU
 * space of the migrated tokens may be reclaimed.  SS_ERR_BAD_STATE if none
 * is in flight. */
ss_status ss_tier_complete(ss_tier *t, int32_t b);

/* Device -> pinned host copy on copy_stream (a migration's copy); the same
 * event conventions as ss_upload_chunk.  dst must be page-locked host memory
 * (else SS_ERR_NOT_PINNED), src device memory; bytes > 0. */
ss_status ss_download_range(void *dst_pinned_host, const void *src_device, size_t bytes,
                            hipStream_t copy_stream, hipEvent_t wait_before, hipEvent_t signal_after);

/* ---- I/O-aware dynamic verification width (paper Sec. 4.2) ----------------
 * Chooses the next round's width q (candidate rows per request, 1..8) as
 * q* = argmin_q T_round(q) / U(q): estimated round time per committed token.
 * T_round = max(history transfer, verification compute) + draft generation +
 * rejection correction (transfer and compute overlap in the pipeline, so
 * they are not counted twice); U = committed tokens.  Each width is sampled
 * min_samples times first (ascending); later, widths without records are
 * estimated from the measured ones (transfer constant in q, compute and
 * draft time linear in q, U from the geometric acceptance model
 * (1 - a^q) / (1 - a) fitted to the measured widths).  The width changes
 * only if the estimate improves on the current one by more than
 * switch_threshold (a fraction).  A width's observations are averaged
 * plainly over its first 1 / decay rounds, then exponentially weighted with
 * factor `decay` (1 = keep only the latest); its committed-token record is
 * blended with the acceptance model in proportion to its rounds (the model
 * weighs as much as 16 rounds). */
typedef struct ss_width_ctl ss_width_ctl;

/* widths: host [num_widths], ascending, each in 1..8; copied. */
ss_status ss_width_create(ss_width_ctl **out, const int32_t *widths, int32_t num_widths,
                          double switch_threshold, int32_t min_samples, double decay);
void ss_width_destroy(ss_width_ctl *c);

/* Record a finished round run at `width`: seconds of history transfer,
 * verification compute, draft generation and rejection correction, and the
 * tokens it committed (averaged over the Cohort's requests). */
ss_status ss_width_observe(ss_width_ctl *c, int32_t width, double transfer_s, double compute_s,
                           double draft_s, double correct_s, double committed_tokens);

/* The width for the next round (-1 if c is null). */
int32_t ss_width_select(ss_width_ctl *c);

/* The controller's estimate of seconds per committed token at `width` (-1
 * for an unknown width). */
double ss_width_estimate(const ss_width_ctl *c, int32_t width);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): start a
 * round as ss_round_init does, but with the library's own device scratch as
 * its workspace instead of a caller buffer, so no device memory is allocated
 * and no workspace argument is needed.  The scratch is a 64 MiB device array
 * per GPU (ss_round_workspace_bytes(desc) must not exceed it, else
 * SS_ERR_WORKSPACE), held from the library's first use on that GPU until the
 * process ends; its address is looked up on the calling thread's current
 * device at the first call there.  Every round started this way on one GPU
 * shares that scratch, which keeps the previous round's contents: rounds
 * whose work overlaps on one GPU (other streams, or a round started before
 * the previous one's work completed without a stream order between them)
 * race.  desc->counters_zeroed is ignored: the counter block's place in the
 * scratch depends on the round's size, so the round's first history call
 * with a balancing tail always clears it.  Every other call of the round is
 * the ordinary one; the host handle is freed with ss_round_destroy. */
ss_status ss_round_init_scratch(ss_round **out, const ss_round_desc *desc, const void *q, hipStream_t stream);

/* Measurement helper, not a step of the method: the read-bandwidth ceiling
 * that the history launches are judged against.  Reads `bytes` of device
 * memory at buf (16-byte aligned, a non-zero multiple of 16) with the
 * history kernel's load form (16 bytes per lane, non-temporal), split over
 * `workgroups` (1..65536) workgroups of 256 threads in equal contiguous
 * slices of ceil(bytes / 16 / workgroups) * 16 bytes (at most 1 GiB each;
 * trailing workgroups may get empty slices).  Workgroup w stores the XOR of
 * its slice's 32-bit words to sink[w] (device, 4-byte aligned, `workgroups`
 * words), so the reads cannot be elided and the result is checkable.
 * Enqueues one launch on `stream`; both buffers stay the caller's. */
ss_status ss_probe_read(const void *buf, size_t bytes, uint32_t *sink, int32_t workgroups, hipStream_t stream);

/* Event helpers so callers need no HIP binding of their own.  Events are
 * created with timing disabled. */
ss_status ss_event_create(hipEvent_t *e);
void ss_event_destroy(hipEvent_t e);

/* Static description of a status code. */
const char *ss_status_string(ss_status s);
/* Detail of the last failure on this thread ("" if none). */
const char *ss_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPECSTREAM_H */
