// CPU check of the history-call planner together with the chunk kernels' tile
// traversal: every token of every request is visited exactly once per KV
// head, every buffer resource stays inside its chunk, chains are
// single-request and single-slot, slots and fresh flags are consistent, the
// workgroup lists cover every unit once, and every workgroup's share of the
// call is within one tile of the mean.  The balancing tail's claim loop is
// emulated with the workgroups interleaved at random, from a zero counter
// (every (tail unit, KV head) pair claimed once, the counter left at zero)
// and from counters that are not zero (no claim outside the tail's range).
// The kernel launchers are stubs that record the launch tables.
#include "ss_kernels.h"
#include "specstream.h"
#include <cstdio>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <map>
#include <random>
#include <vector>
#include <set>

namespace {
struct Rec {
  std::vector<ss::Item> items; std::vector<uint32_t> units; std::vector<uint32_t> wg_first; int kind;
  int tail_first, num_tail; uint32_t *claim; int clears_before; int Hkv;
};
int g_finalize_launches = 0;
long g_empty_wgs = 0;             // workgroups launched without a unit of their own
int g_clear_n = 0;
std::vector<Rec> g_recs;
const ss::ChunkParams *g_last = nullptr;
int g_clears = 0;                 // claim-counter clear launches so far
uint32_t *g_clear_ptr = nullptr;
}

namespace ss {
// Record a launch.  The unit records are checked against the items they
// name, then flattened into the order the kernel attends them: workgroup w's
// first unit (record w, unless empty), its further units [more[w],
// more[w + 1]), ..., then the tail; the tables below use that order, with
// unit words (i0 | nit << 16 | kind << 24).
static void rec(const ChunkParams &p, int kind) {
  Rec r;
  r.items.assign(p.items, p.items + p.num_items);
  if (p.num_wgs < 1 || p.num_wgs > kMaxWgs) { printf("bad workgroup count\n"); exit(1); }
  if (p.num_units < p.num_wgs || p.num_units > kMaxUnits || p.num_items < 1 || p.num_items > kMaxItems) { printf("bad counts\n"); exit(1); }
  const int W = p.num_wgs;
  const int tail_first = p.num_tail > 0 ? p.tail_first : p.num_units;
  bool ok = p.more[0] == (uint32_t)W && p.more[W] == (uint32_t)tail_first &&
            tail_first + (p.num_tail > 0 ? p.num_tail : 0) == p.num_units;
  for (int w = 0; w < W; ++w) ok = ok && p.more[w] <= p.more[w + 1];
  if (!ok) { printf("bad unit ranges\n"); exit(1); }
  auto word = [&](int u) {
    const UnitRec &ur = p.units[u];
    const int i0 = unit_i0(ur.word), nit = unit_nit(ur.word);
    if (nit < 1 || i0 + nit > p.num_items) { printf("unit %d: items [%d, +%d) outside the table\n", u, i0, nit); exit(1); }
    uint32_t tiles = 0;
    for (int i = i0; i < i0 + nit; ++i) tiles += (uint32_t)((p.items[i].tok_count + kTile - 1) / kTile);
    const Item &it = p.items[i0];
    if (ur.ntiles != tiles || ur.q_row0 != it.q_row0 || ur.n_cand != it.n_cand || unit_chunk(ur.word) != it.chunk) {
      printf("unit %d: record does not match its items\n", u);
      exit(1);
    }
    return (uint32_t)i0 | ((uint32_t)nit << 16) | ((uint32_t)unit_kind(ur.word) << 24);
  };
  for (int w = 0; w < W; ++w) {
    r.wg_first.push_back((uint16_t)r.units.size());
    if (unit_nit(p.units[w].word) > 0) r.units.push_back(word(w));
    else g_empty_wgs++;
    for (uint32_t u = p.more[w]; u < p.more[w + 1]; ++u) r.units.push_back(word((int)u));
  }
  r.wg_first.push_back((uint16_t)r.units.size());
  r.tail_first = (int)r.units.size();
  for (int u = tail_first; u < p.num_units; ++u) r.units.push_back(word(u));
  r.kind = kind;
  r.num_tail = p.num_tail; r.claim = p.claim; r.clears_before = g_clears;
  r.Hkv = p.Hkv;
  g_recs.push_back(r);
  g_last = &p;
}
hipError_t launch_chunk(const ChunkParams &p, hipStream_t) { rec(p, -1); return hipSuccess; }
hipError_t launch_finalize(const FinalParams &, hipStream_t) { ++g_finalize_launches; return hipSuccess; }

hipError_t launch_clear_counters(uint32_t *c, int n, hipStream_t) {
  ++g_clears; g_clear_ptr = c; g_clear_n = n; return hipSuccess;
}
// The scratch stands at the same address as the caller workspaces below.
hipError_t launch_read_probe(const void *, uint64_t, uint64_t, uint32_t *, int, hipStream_t) { return hipSuccess; }
hipError_t scratch_address(void **p) { *p = (void *)0x7f1000000000ull; return hipSuccess; }
}

static const ss_round_desc *g_desc = nullptr;
static bool g_trust_zeroed = false;   // the round may skip the counter clear
static int g_tail_calls = 0;
static std::mt19937 g_emu(11);

static int tiles_of(const ss::Item &it) { return (it.tok_count + ss::kTile - 1) / ss::kTile; }

static int fails = 0;
#define CHECK(c, ...) do { if (!(c)) { printf("FAIL %s:%d: ", __FILE__, __LINE__); printf(__VA_ARGS__); printf("\n"); if (++fails > 20) exit(1); } } while (0)

struct UnitF { int i0, nit, kind; };
static UnitF unit_fields(uint32_t u) { return UnitF{(int)(u & 0xffff), (int)((u >> 16) & 0xff), (int)(u >> 24)}; }

// The history kernel's claim loop, with the launch's workgroups interleaved
// at random: a workgroup claims only after its own units, makes claims until
// it receives a number >= nclaims, and the claim that receives the launch's
// last number stores zero.  Returns the (tail unit, KV head) pairs attended.
static std::vector<std::pair<int, int>> emulate_claims(const Rec &rc, uint32_t start, uint32_t *end_value) {
  const uint32_t Hkv = (uint32_t)rc.Hkv, W = (uint32_t)rc.wg_first.size() - 1;
  const uint32_t nclaims = (uint32_t)rc.num_tail * Hkv, last = nclaims + Hkv * W - 1u;
  uint32_t ctr = start;
  std::vector<std::pair<int, int>> got;
  std::vector<int> active;
  for (uint32_t w = 0; w < Hkv * W; ++w) active.push_back((int)w);
  while (!active.empty()) {
    const size_t k = g_emu() % active.size();
    const uint32_t c = ctr++;            // atomicAdd
    if (c == last) ctr = 0u;             // the launch's last claim
    if (c >= nclaims) {                  // compared without sign
      active.erase(active.begin() + k);
      continue;
    }
    const uint32_t t = c / Hkv;
    got.push_back({rc.tail_first + (int)t, (int)(c - t * Hkv)});
  }
  *end_value = ctr;
  return got;
}

// emulate one history call
static void check_call(int B, int Hq, int Hkv, const std::vector<int> &ncand, const std::vector<std::vector<int>> &lens,
                       int split, int layout, int mfma_min_rows, std::vector<int> &slots_used, ss_round *r) {
  const int nch = (int)lens.size();
  std::vector<int32_t> flat;
  std::vector<long> tot(nch, 0);
  for (int c = 0; c < nch; ++c) for (int b = 0; b < B; ++b) { flat.push_back(lens[c][b]); tot[c] += lens[c][b]; }
  std::vector<const void *> kp(nch), vp(nch);
  // fake aligned chunk pointers; never dereferenced
  for (int c = 0; c < nch; ++c) {
    kp[c] = (const void *)(uintptr_t)(0x100000000ull * (c + 1));
    vp[c] = (const void *)(uintptr_t)(0x100000000ull * (c + 1) + (layout == SS_KV_HEAD_MAJOR_KV ? 256 : 0x80000000ull));
  }
  g_recs.clear();
  g_finalize_launches = 0;
  const ss_status s = ss_attend_history_chunks(r, nch, kp.data(), vp.data(), flat.data(), nullptr, nullptr, nullptr);
  CHECK(s == SS_OK, "status %d: %s", s, ss_last_error());
  if (s != SS_OK) return;
  long total = 0;
  for (auto &row : lens) for (int x : row) total += x;
  // coverage[b][c] token counts
  std::vector<std::vector<std::vector<int>>> cov(B, std::vector<std::vector<int>>(nch));
  for (int b = 0; b < B; ++b) for (int c = 0; c < nch; ++c) cov[b][c].assign(lens[c][b], 0);
  std::map<std::pair<int,int>, int> slot_writes;   // (request, slot) -> units
  const int G = Hq / Hkv;
  std::vector<int> off_rows(B, 0);
  for (int b = 1; b < B; ++b) off_rows[b] = off_rows[b - 1] + ncand[b - 1];
  // workgroup lists: cover every unit once, in order; shares are equal
  long wgs = 0, max_share = 0;
  for (auto &rc : g_recs) {
    CHECK(rc.wg_first.front() == 0 && rc.wg_first.back() + rc.num_tail == rc.units.size(), "workgroup table ends");
    for (size_t w = 0; w + 1 < rc.wg_first.size(); ++w) {
      CHECK(rc.wg_first[w] <= rc.wg_first[w + 1], "workgroup table order");
      long share = 0;
      for (int u = rc.wg_first[w]; u < rc.wg_first[w + 1]; ++u) {
        const UnitF f = unit_fields(rc.units[u]);
        for (int k = 0; k < f.nit; ++k) share += rc.items[f.i0 + k].tok_count;
      }
      max_share = std::max(max_share, share);
      ++wgs;
    }
  }
  if (total >= 32 * wgs) CHECK(max_share <= (total + wgs - 1) / wgs + 31, "share %ld > mean %ld + a tile", max_share, total / wgs);
  // counter block: at the workspace's end, cleared once per round (before
  // the first launch that uses it) unless the caller said it is zero
  const size_t ws_end = 0x7f1000000000ull + ss_round_workspace_bytes(g_desc);
  const size_t block_words = ss::kClaimCounters;
  const uintptr_t block = ws_end - (block_words * 4 + 255) / 256 * 256;
  for (auto &rc : g_recs) {
    if (rc.num_tail == 0) {
      CHECK(rc.wg_first.back() == rc.units.size(), "units beyond the workgroup lists");
      continue;
    }
    CHECK(g_recs.size() == 1, "a call with a tail took %zu launches", g_recs.size());
    if (g_trust_zeroed) {
      CHECK(g_clears == 0, "counters cleared although the caller said they are zero");
    } else {
      CHECK(rc.clears_before == 1 && (uintptr_t)g_clear_ptr == block && g_clear_n == (int)block_words,
            "counter block cleared %d times (at %p, %d words) before the launch", rc.clears_before, (void *)g_clear_ptr,
            g_clear_n);
    }
    if (rc.num_tail > 0) {
      CHECK(rc.tail_first == (int)rc.wg_first.back() && rc.tail_first + rc.num_tail == (int)rc.units.size(), "tail range");
      CHECK((uintptr_t)rc.claim == block, "claim counter is not the block's first word");
      g_tail_calls++;
      // claim loop from a zero counter: every pair once, counter back to zero
      for (int rep = 0; rep < 3; ++rep) {
        uint32_t end = 1;
        auto got = emulate_claims(rc, 0u, &end);
        std::set<std::pair<int, int>> seen(got.begin(), got.end());
        CHECK(got.size() == seen.size() && got.size() == (size_t)rc.num_tail * Hkv, "claims: %zu pairs, %zu distinct",
              got.size(), seen.size());
        CHECK(end == 0u, "claim counter left at %u", end);
      }
      // from counters that are not zero (a broken workspace contract): no pair outside the tail
      for (uint32_t start : {1u, 7u, (uint32_t)rc.num_tail * Hkv, 0x7fffffffu, 0x80000000u, 0xfffffff0u, 0xffffffffu,
                             (uint32_t)g_emu()}) {
        uint32_t end = 0;
        for (auto &pr : emulate_claims(rc, start, &end))
          CHECK(pr.first >= rc.tail_first && pr.first < rc.tail_first + rc.num_tail && pr.second >= 0 && pr.second < Hkv,
                "claim from counter %u outside the tail: unit %d head %d", start, pr.first, pr.second);
      }
    }
  }
  for (auto &rc : g_recs) {
    for (size_t u = 0; u < rc.units.size(); ++u) {
      const UnitF f = unit_fields(rc.units[u]);
      const int i0 = f.i0, nit = f.nit, kind = f.kind;
      CHECK(nit >= 1 && nit <= ss::kMaxChain && i0 + nit <= (int)rc.items.size(), "unit table");
      const ss::Item &it = rc.items[i0];
      int b = -1;
      for (int bb = 0; bb < B; ++bb) if (off_rows[bb] == it.q_row0) b = bb;
      CHECK(b >= 0, "q_row0");
      const int M = it.n_cand * G;
      // mfma_min_rows 0 is the library's default, 3 (ss_round_desc)
      const int want_kind = (M < (mfma_min_rows ? mfma_min_rows : 3) && M <= 4) ? 0 : (M + 15) / 16;
      CHECK(kind == want_kind, "unit kind %d want %d (M=%d)", kind, want_kind, M);
      int ntiles = 0;
      long toks = 0;
      for (int k = 0; k < nit; ++k) {
        const ss::Item &ik = rc.items[i0 + k];
        CHECK(ik.q_row0 == it.q_row0 && ik.slot == it.slot && ik.flags == it.flags && ik.n_cand == it.n_cand, "chain mixes");
        CHECK(ik.tok_count >= 1, "empty item");
        CHECK(ik.chunk < nch, "chunk index");
        ntiles += tiles_of(ik);
        toks += ik.tok_count;
        // the item is request b's tokens of chunk ik.chunk
        long ofs = 0;
        for (int bb = 0; bb < b; ++bb) ofs += lens[ik.chunk][bb];
        CHECK(ik.tok_begin >= ofs && ik.tok_begin + ik.tok_count <= ofs + lens[ik.chunk][b], "item outside request range");
        // buffer resource bounds for every head: [first, first + nrec) inside the chunk
        const bool il = layout == SS_KV_HEAD_MAJOR_KV;
        const long stride = layout == SS_KV_TOKEN_MAJOR ? (long)Hkv * 128 : il ? 256 : 128;
        const long hstride = layout == SS_KV_TOKEN_MAJOR ? 128 : tot[ik.chunk] * stride;
        const long bytes = tot[ik.chunk] * Hkv * 256 * (il ? 2 : 1);   // the buffer K (and V) offsets index
        for (int g = 0; g < Hkv; ++g) {
          const long first = (long)ik.tok_begin * stride + (long)g * hstride;
          const long nrec = (long)(ik.tok_count - 1) * stride * 2 + 256;
          CHECK(first * 2 + nrec <= bytes, "K rsrc past chunk");
          CHECK(first * 2 + (il ? 256 : 0) + nrec <= bytes, "V rsrc past chunk");
          CHECK(nrec < (1L << 31), "nrec 32-bit");
        }
      }
      CHECK(toks >= 1, "empty unit");
      slot_writes[{b, it.slot}]++;
      CHECK(((it.flags & ss::kSlotFresh) != 0) == (it.slot >= slots_used[b]), "fresh flag");
      // emulate the 4 waves' traversal (same as the kernels)
      for (int w = 0; w < ss::kWaves; ++w) {
        int T = w;
        int ck = 0, cbase = 0;
        auto seek = [&](int TT) {
          while (ck + 1 < nit && TT - cbase >= tiles_of(rc.items[i0 + ck])) { cbase += tiles_of(rc.items[i0 + ck]); ++ck; }
        };
        for (; T < ntiles; T += ss::kWaves) {
          seek(T);
          const ss::Item &ic = rc.items[i0 + ck];
          const int tb = (T - cbase) * ss::kTile;
          CHECK(tb >= 0 && tb < ic.tok_count, "tile outside item (tb %d count %d)", tb, ic.tok_count);
          long ofs = 0;
          for (int bb = 0; bb < b; ++bb) ofs += lens[ic.chunk][bb];
          for (int t = tb; t < tb + ss::kTile && t < ic.tok_count; ++t) cov[b][ic.chunk][ic.tok_begin - ofs + t]++;
        }
      }
    }
  }
  for (int b = 0; b < B; ++b)
    for (int c = 0; c < nch; ++c)
      for (int t = 0; t < lens[c][b]; ++t) CHECK(cov[b][c][t] == 1, "token b=%d c=%d t=%d visited %d times", b, c, t, cov[b][c][t]);
  for (auto &kv : slot_writes) CHECK(kv.second == 1, "slot (%d,%d) written by %d units", kv.first.first, kv.first.second, kv.second);
  for (auto &kv : slot_writes) CHECK(kv.first.second < ss::kNumSlots, "slot index");
  for (int b = 0; b < B; ++b) {
    int mx = -1;
    for (auto &kv : slot_writes) if (kv.first.first == b) mx = std::max(mx, kv.first.second);
    for (int s2 = 0; s2 <= mx; ++s2) CHECK(slot_writes.count({b, s2}), "slot gap b=%d s=%d", b, s2);
    slots_used[b] = std::max(slots_used[b], mx + 1);
  }
}

// One round of history calls in batches of `batch` chunks, then the
// finalize, on a workspace of unknown contents, on one the caller declared
// zeroed, and (when it fits) on the library's scratch with counters_zeroed
// set, which the scratch round must ignore.
static void scenario(const char *name, int B, int Hq, int Hkv, std::vector<int> ncand, std::vector<int> hist, int S,
                     int split, int layout, int batch, int mfma_min_rows = 0, int balance = 0, int expect_tail = -1,
                     int expect_wgs = -1) {
  const int nch = [&] { int m = 0; for (int h : hist) m = std::max(m, (h + S - 1) / S); return m; }();
  std::vector<std::vector<int>> lens(nch, std::vector<int>(B));
  long maxc = 1;
  for (int c = 0; c < nch; ++c) { long t = 0; for (int b = 0; b < B; ++b) { lens[c][b] = std::max(0, std::min(S, hist[b] - c * S)); t += lens[c][b]; } maxc = std::max(maxc, t); }
  for (int mode = 0; mode < 3; ++mode) {
    ss_round_desc d{};
    d.num_requests = B; d.num_q_heads = Hq; d.num_kv_heads = Hkv; d.head_dim = 128; d.softmax_scale = 0.088f;
    d.num_cand = ncand.data(); d.max_chunk_tokens = (int)maxc; d.split_tokens = split; d.mfma_min_rows = mfma_min_rows; d.kv_layout = layout;
    d.balance_permille = balance;
    d.counters_zeroed = mode >= 1;
    g_trust_zeroed = mode == 1;
    g_desc = &d; g_clears = 0; g_clear_ptr = nullptr; g_tail_calls = 0;
    ss_round *r = nullptr;
    size_t ws = ss_round_workspace_bytes(&d);
    if (mode == 2 && ws > ss::kScratchBytes) {
      CHECK(ss_round_init_scratch(&r, &d, (const void *)0x7f0000000000ull, nullptr) == SS_ERR_WORKSPACE && r == nullptr,
            "%s: a round beyond the scratch was accepted", name);
      continue;
    }
    ss_status s = mode == 2 ? ss_round_init_scratch(&r, &d, (const void *)0x7f0000000000ull, nullptr)
                            : ss_round_init(&r, &d, (const void *)0x7f0000000000ull, (void *)0x7f1000000000ull, ws, nullptr);
    if (s != SS_OK) { printf("%s: init failed %s\n", name, ss_last_error()); fails++; return; }
    std::vector<int> used(B, 0);
    const int before = fails;
    // chunk batches
    for (int c0 = 0; c0 < nch; c0 += batch) {
      std::vector<std::vector<int>> part(lens.begin() + c0, lens.begin() + std::min(nch, c0 + batch));
      check_call(B, Hq, Hkv, ncand, part, split, layout, mfma_min_rows, used, r);
    }
    g_finalize_launches = 0;
    s = ss_attend_local_candidates(r, (const void *)0x7f2000000000ull, (const void *)0x7f3000000000ull, nullptr);
    if (s == SS_OK) s = ss_round_finalize(r, (float *)0x7f4000000000ull, nullptr, nullptr);
    CHECK(s == SS_OK && g_finalize_launches == 1, "finalize: %s", ss_last_error());
    ss_round_destroy(r);
    const int want_clears = g_trust_zeroed ? 0 : g_tail_calls > 0 ? 1 : 0;
    CHECK(g_clears == want_clears, "%d clears for %d balanced calls", g_clears, g_tail_calls);
    if (expect_tail >= 0) CHECK((g_tail_calls > 0) == (expect_tail > 0), "%s: %d balanced calls", name, g_tail_calls);
    // workgroups per KV head of the last call's launches
    if (expect_wgs >= 0)
      for (auto &rc : g_recs)
        CHECK((int)rc.wg_first.size() - 1 == expect_wgs, "%s: %d workgroups per KV head, want %d", name,
              (int)rc.wg_first.size() - 1, expect_wgs);
    printf("%-44s %-7s %s (launches in last call: %zu, balanced calls: %d)\n", name,
           mode == 0 ? "" : mode == 1 ? "zeroed" : "scratch",
           fails == before ? "ok" : "FAILED", g_recs.size(), g_tail_calls);
  }
}

int main() {
  std::mt19937 rng(7);
  for (int layout : {SS_KV_TOKEN_MAJOR, SS_KV_HEAD_MAJOR, SS_KV_HEAD_MAJOR_KV}) {
    scenario("config1 per-chunk", 1, 8, 2, {5}, {4096}, 1024, 0, layout, 1);
    scenario("config1 split 32", 1, 8, 2, {5}, {4096}, 1024, 32, layout, 1);
    scenario("config1 split 96", 1, 8, 2, {5}, {4096}, 1024, 96, layout, 1);
    scenario("config1 batched", 1, 8, 2, {5}, {4096}, 1024, 0, layout, 4);
    // shares of 16.5 tokens: the first share ends below the first tile boundary, so workgroup 0 has no unit
    scenario("33 tokens, split 32 (a workgroup without units)", 1, 8, 2, {5}, {33}, 64, 32, layout, 1);
    scenario("ragged, split 32 (workgroups without units)", 3, 32, 8, {2, 7, 1}, {33, 97, 65}, 64, 32, layout, 2);
    scenario("config2 per-chunk", 1, 32, 8, {5}, {16384}, 2048, 0, layout, 1);
    // one workgroup per CU: 8 KV heads x 32
    scenario("config3 batched 8", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 0, 1, 32);
    scenario("16 x 16384 batched 4 (no tail: shares of 8192)", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 16384), 4096, 0, layout, 4, 0, 0, 0);
    scenario("16 x 65536 batched 16 (tail)", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 65536), 4096, 0, layout, 16, 0, 0, 1);
    scenario("config3 batched 8, no tail", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, -1, 0);
    scenario("config3 batched 8, tail 500", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 500, 1);
    scenario("config3 batched 8, tail 1", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 1, 1);
    scenario("config3 per-chunk", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 1);
    scenario("config3 batched 3", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 0, layout, 3);
    scenario("config3 split 2048 batched", 16, 32, 8, std::vector<int>(16, 6), std::vector<int>(16, 32768), 4096, 2048, layout, 8);
    scenario("config5 per-chunk", 32, 32, 8, std::vector<int>(32, 8), std::vector<int>(32, 131072), 8192, 0, layout, 1, 0, 0, 0);
    scenario("config5 batched 4 (tail)", 32, 32, 8, std::vector<int>(32, 8), std::vector<int>(32, 131072), 8192, 0, layout, 4, 0, 0, 1);
    {
      std::mt19937 g4(4);
      std::vector<int> h4(64), n4(64);
      for (int b = 0; b < 64; ++b) {
        h4[b] = (int)std::lround(std::exp(std::log(2048.0) + (std::log(65536.0) - std::log(2048.0)) * (g4() / 4294967296.0)));
        n4[b] = 1 + g4() % 8;
      }
      scenario("config4-like ragged batched 16", 64, 32, 8, n4, h4, 4096, 0, layout, 16, 0, 0, 1);
      scenario("config4-like ragged per-chunk", 64, 32, 8, n4, h4, 4096, 0, layout, 1, 0, 0, -1);
    }
    // row-split units get two workgroups per CU (8 KV heads x 64): 8192-token shares, below the default
    // tail's threshold
    scenario("64q/8kv x 8 candidates (64 rows), batched", 16, 64, 8, std::vector<int>(16, 8), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 0, 0, 64);
    scenario("64q/8kv x 8 candidates, batched, tail 100", 16, 64, 8, std::vector<int>(16, 8), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 100, 1, 64);
    scenario("64q/8kv x 4 candidates (32 rows), batched", 16, 64, 8, std::vector<int>(16, 4), std::vector<int>(16, 32768), 4096, 0, layout, 8, 0, 0, 1, 32);
    scenario("48q/8kv ragged candidates, per-chunk", 12, 48, 8, {1, 8, 3, 6, 2, 7, 8, 5, 4, 1, 6, 8}, std::vector<int>(12, 9000), 2048, 0, layout, 1);
    scenario("config2 per-chunk (no tail: small shares)", 1, 32, 8, {5}, {16384}, 2048, 0, layout, 8, 0, 0, 0);
    scenario("config5 batched 16", 32, 32, 8, std::vector<int>(32, 8), std::vector<int>(32, 131072), 8192, 0, layout, 16);
    scenario("many units (8192 chains)", 256, 8, 2, std::vector<int>(256, 3), std::vector<int>(256, 4096), 512, 128, layout, 8);
    // one share of 2.2M tokens: with 8 KV heads token-major, a KV head's
    // rows span more than 2^31 bytes, so the share is cut into pieces below
    // that (32-bit buffer offsets)
    scenario("one share over 2^31 bytes per head", 1, 8, 8, {2}, {2200000}, 2200000, 2199968, layout, 1);
    scenario("many items (chains of 16)", 128, 8, 2, std::vector<int>(128, 2), std::vector<int>(128, 8192), 32, 512, layout, 32);
    for (int rep = 0; rep < 40; ++rep) {
      const int B = 1 + rng() % 64;
      std::vector<int> nc(B), h(B);
      for (int b = 0; b < B; ++b) { nc[b] = 1 + rng() % 8; h[b] = (rng() % 4 == 0) ? (int)(rng() % 70) : (int)(rng() % 66000); }
      const int S = 32 * (1 + rng() % 256);
      const int split = (rng() % 3 == 0) ? 32 * (1 + rng() % 64) : 0;
      int nch = 0; for (int x : h) nch = std::max(nch, (x + S - 1) / S);
      if (nch == 0) continue;
      const int batch = 1 + rng() % 32;
      const int hsel = rng() % 6;   // GQA groups of 4, 4, 8, 6, 1 and 2 query heads
      const int hq = hsel == 0 ? 32 : hsel == 1 ? 8 : hsel == 2 ? 64 : hsel == 3 ? 48 : hsel == 4 ? 8 : 16;
      const int hkv = hsel == 1 ? 2 : 8;
      char nm[64]; snprintf(nm, sizeof nm, "random %d B=%d S=%d split=%d batch=%d", rep, B, S, split, batch);
      const int bal = (rng() % 4 == 0) ? -1 : (rng() % 2 ? 0 : (int)(1 + rng() % 500));
      scenario(nm, B, hq, hkv, nc, h, S, split, layout, batch, (int)(rng() % 6), bal);
    }
  }
  printf("workgroups without units of their own: %ld\n", g_empty_wgs);
  CHECK(g_empty_wgs > 0, "no launch had a workgroup without units of its own");
  printf("%s\n", fails ? "FAILURES" : "all ok");
  return fails ? 1 : 0;
}
