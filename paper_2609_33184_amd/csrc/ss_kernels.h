// Internal interface between the host library (ss_host.cpp) and the gfx950
// kernels (ss_kernels.hip).  Not part of the public ABI.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace ss {

constexpr int kHeadDim = 128;       // d
constexpr int kNumSlots = 32;       // split slots of the running state per row
constexpr int kMaxItems = 2048;     // work items per launch (kernel-argument list)
constexpr int kMaxUnits = 1024;     // units per launch (x all KV heads)
constexpr int kMaxWgs = 1024;       // workgroups per KV head per launch
constexpr int kMaxChain = 16;       // items (token ranges) per unit
constexpr int kMaxChunks = 32;      // history chunks per launch
constexpr int kTile = 32;           // history tokens per wave iteration
constexpr int kWaves = 4;           // waves per workgroup of the chunk kernels
constexpr int kMaxCand = 8;         // candidates per request (k_b + 1)
constexpr int kMaxValuRows = 4;     // rows per KV head the VALU chunk kernel handles
constexpr int kMaxRows = 64;        // rows per KV head the MFMA chunk kernels handle
constexpr int kClaimCounters = 64;  // words of the workspace's counter block (the first is the claim counter)

// Unit kinds: the chunk kernel body that attends a unit (rows per KV head
// M = n_b * G: <= 4 on the VALU path, else MFMA with ceil(M / 16) blocks).
constexpr int kUnitValu = 0;
constexpr int kUnitMfma1 = 1;
constexpr int kUnitMfma2 = 2;
constexpr int kUnitMfma3 = 3;       // wide units (row-split body): only the wide kernel runs them
constexpr int kUnitMfma4 = 4;

// Item flag: the slot has not been written in this round yet, so the kernel
// stores its result instead of merging with (uninitialised) workspace.
constexpr int kSlotFresh = 1;

// History item: one token range of one chunk for one request: tokens
// [tok_begin, tok_begin + tok_count) of chunk `chunk` (tok_count >= 1).
// A unit (one workgroup per KV head, blockIdx.x) is a chain of consecutive
// items of one request, attended as one token sequence with one running
// state that is folded into split slot `slot`; every item of a chain carries
// the same q_row0, n_cand, slot and flags.
// Finalize item: one request; tok_count = number of slots written by
// history calls (slots >= that are empty), other token fields unused.
struct Item {
  int32_t tok_begin;
  int32_t tok_count;
  int32_t q_row0;   // off_b: first packed candidate row of the request
  uint8_t n_cand;   // n_b
  uint8_t chunk;    // index into the launch's chunk table
  uint8_t slot;     // state slot
  uint8_t flags;    // kSlotFresh
};
static_assert(sizeof(Item) == 16, "Item layout");

// Running state in the workspace, per slot s and query row R_idx = (off_b+i)*Hq+h:
//   m[s*R + R_idx]   running max of sigma*log2(e)*q.k (log2 domain)
//   l[s*R + R_idx]   running sum of 2^(x - m)
//   a[(s*R + R_idx)*d + c]  running weighted value sum (same scale as l)
// A slot is valid only once a history item has written it in this round.
struct State {
  float *m;
  float *l;
  float *a;
  int32_t R;        // rows = sum n_b * Hq
};

// Kernel arguments.  The unit and item tables travel by value in the
// kernel-argument segment; the launch wrappers pick the smallest of three
// table capacities that holds a launch, so a typical round passes a few KB
// (large by-value arguments fill the runtime's argument pool quickly, and a
// full pool makes the next launch wait for the queue to drain).
struct ChunkHeader {
  const uint16_t *q;    // bf16 [sum n_b, Hq, d]
  State st;
  int32_t Hq, Hkv, G;
  float scale_log2;     // softmax_scale * log2(e)
  uint32_t tok_stride;  // elements between consecutive tokens of one KV head
  int32_t num_items;
  // chunk table: bf16 chunks, token-major [sum len][Hkv][d] or head-major [Hkv][sum len][d]
  const uint16_t *k[kMaxChunks];
  const uint16_t *v[kMaxChunks];
  uint64_t head_stride[kMaxChunks];   // elements between KV heads at the same token
  int32_t num_units;    // unit records (num_wgs first-unit records included)
  int32_t num_wgs;      // workgroups per KV head
  // Grid order: 1 = (KV head, workgroup) with the heads as the fast
  // dimension, 0 = (workgroup, KV head).  Workgroups are placed on the XCDs
  // round-robin in grid order, so with the heads fast XCD g streams only KV
  // head g; that suits token-major chunks, where a token's heads are
  // adjacent, and not head-major ones, where each head is its own plane.
  int32_t heads_fast;
  // Balancing tail: units [tail_first, tail_first + num_tail) are claimed at
  // run time, for every KV head, by whichever workgroup has finished its own
  // units: claim c = atomicAdd(claim, 1) < num_tail * Hkv attends unit
  // tail_first + c / Hkv for KV head c % Hkv.  The counter is zero at launch;
  // the launch's last claim sets it back to zero.
  uint32_t *claim;
  int32_t tail_first;
  int32_t num_tail;
};

// Unit record: what a workgroup needs to start a unit, so that its first
// loads depend on one record and the item and chunk-table entries it names
// (kernel arguments are read with dependent loads of about a microsecond
// each at the start of a launch).  word packs the unit's first item i0
// (within the launch), its item count nit (1..kMaxChain; 0 = no unit), the
// body kind and the chunk of item i0; ntiles is the chain's tile count.
struct UnitRec {
  uint32_t word;
  uint32_t ntiles;
  int32_t q_row0;   // off_b of the unit's request
  int32_t n_cand;   // n_b of the unit's request
};
static_assert(sizeof(UnitRec) == 16, "UnitRec layout");
constexpr uint32_t unit_word(uint32_t i0, uint32_t nit, uint32_t kind, uint32_t chunk) {
  return i0 | (nit << 16) | (kind << 21) | (chunk << 24);
}
constexpr int unit_i0(uint32_t w) { return (int)(w & 0xffffu); }
constexpr int unit_nit(uint32_t w) { return (int)((w >> 16) & 0x1fu); }
constexpr int unit_kind(uint32_t w) { return (int)((w >> 21) & 0x7u); }
constexpr int unit_chunk(uint32_t w) { return (int)((w >> 24) & 0x1fu); }
static_assert(kMaxItems <= 0x10000 && kMaxChain <= 0x1f && kUnitMfma4 <= 7 && kMaxChunks <= 0x20, "unit word fields");

template <int MaxUnits, int MaxItems, int MaxWgs>
struct ChunkParamsT : ChunkHeader {
  static constexpr int kUnits = MaxUnits;
  static constexpr int kItems = MaxItems;
  static constexpr int kWgs = MaxWgs;
  // Units of workgroup w (of every KV head): units[w] (its first unit; a
  // record with nit = 0 if it has none), then units [more[w], more[w + 1]).
  // Units [num_wgs, tail_first) are these further units in workgroup order.
  UnitRec units[MaxUnits];
  uint32_t more[MaxWgs + 1];
  Item items[MaxItems];
};
using ChunkParams = ChunkParamsT<kMaxUnits, kMaxItems, kMaxWgs>;   // what the host fills

struct FinalHeader {
  const uint16_t *kc;   // bf16 candidate K [sum n_b, Hkv, d]
  const uint16_t *vc;   // bf16 candidate V
  const uint16_t *q;
  float *out;           // fp32 [sum n_b, Hq, d]
  float *lse;           // fp32 [sum n_b, Hq] or null
  State st;
  int32_t Hq, Hkv, G;
  float scale_log2;
  int32_t num_items;
};

template <int MaxItems>
struct FinalParamsT : FinalHeader {
  static constexpr int kItems = MaxItems;
  Item items[MaxItems];
};
using FinalParams = FinalParamsT<kMaxItems>;

// Launch wrappers; return hipGetLastError() of the launch.
// History units of every kind, grid (Hkv, num_wgs) or (num_wgs, Hkv) by heads_fast.
hipError_t launch_chunk(const ChunkParams &p, hipStream_t s);
// Speculative Frontier pass fused with the split-slot merge and O = a / l.
hipError_t launch_finalize(const FinalParams &p, hipStream_t s);
// Zero n counters (a kernel rather than a memset node, so the call can be
// captured in a graph).
hipError_t launch_clear_counters(uint32_t *counters, int n, hipStream_t s);

// Read-bandwidth probe over `bytes` (a multiple of 16) of device memory:
// workgroup w < workgroups XOR-folds bytes [w * share, (w + 1) * share)
// (share a multiple of 16, at most kProbeMaxShare) into sink[w].
constexpr uint64_t kProbeMaxShare = uint64_t(1) << 30;
hipError_t launch_read_probe(const void *buf, uint64_t bytes, uint64_t share, uint32_t *sink, int workgroups,
                             hipStream_t s);

// The library's own device scratch: a file-scope device array of
// kScratchBytes that serves as the workspace of rounds started with
// ss_round_init_scratch.  scratch_address returns its address on the
// current device (looked up once per device, then cached).
constexpr size_t kScratchBytes = size_t(64) << 20;
hipError_t scratch_address(void **ptr);

}  // namespace ss
