// CPU check of the library's error paths.  The host code (ss_host.cpp) is
// linked with stub kernel launchers and stub HIP runtime calls that can be
// told to fail at the n-th call, and with a global operator new that can be
// told to throw.  Checked: a call that fails after part of its work was
// enqueued marks the round (and a pipeline it went through) failed, so every
// later call returns SS_ERR_BAD_STATE; a call that fails before enqueueing
// anything leaves the round usable; host allocation failures return
// SS_ERR_OUT_OF_MEMORY and leave the round usable.
#include "ss_kernels.h"
#include "specstream.h"

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

namespace {
int g_launches = 0, g_fail_launch = -1;   // kernel launches so far; fail the launch with this index
int g_hip_calls = 0, g_fail_hip = -1;     // HIP runtime calls so far; fail the call with this index
bool g_throw_new = false;
int fails = 0;
#define CHECK(c, ...) do { if (!(c)) { printf("FAIL %s:%d: ", __FILE__, __LINE__); printf(__VA_ARGS__); printf("\n"); ++fails; } } while (0)

hipError_t launch_result() { return g_launches++ == g_fail_launch ? hipErrorLaunchFailure : hipSuccess; }
hipError_t hip_result() { return g_hip_calls++ == g_fail_hip ? hipErrorInvalidValue : hipSuccess; }
void arm(int launch, int hip) {
  g_launches = 0; g_fail_launch = launch; g_hip_calls = 0; g_fail_hip = hip;
}
}  // namespace

void *operator new(size_t n) {
  if (g_throw_new) throw std::bad_alloc();
  if (void *p = std::malloc(n ? n : 1)) return p;
  throw std::bad_alloc();
}
void operator delete(void *p) noexcept { std::free(p); }
void operator delete(void *p, size_t) noexcept { std::free(p); }

namespace ss {
hipError_t launch_chunk(const ChunkParams &, hipStream_t) { return launch_result(); }
hipError_t launch_finalize(const FinalParams &, hipStream_t) { return launch_result(); }
hipError_t launch_clear_counters(uint32_t *, int, hipStream_t) { return launch_result(); }
hipError_t launch_read_probe(const void *, uint64_t, uint64_t, uint32_t *, int, hipStream_t) { return launch_result(); }
hipError_t scratch_address(void **) { return hipErrorNotSupported; }
}  // namespace ss

// HIP runtime stand-ins: host pointers below 0x100000000000, device above.
extern "C" {
const char *hipGetErrorString(hipError_t) { return "stub error"; }
hipError_t hipGetLastError(void) { return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned int) { return hip_result(); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hip_result(); }
hipError_t hipMemcpyAsync(void *, const void *, size_t, hipMemcpyKind, hipStream_t) { return hip_result(); }
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) {
  static uintptr_t next = 0x1000;
  *e = reinterpret_cast<hipEvent_t>(next += 0x10);
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
hipError_t hipPointerGetAttributes(hipPointerAttribute_t *a, const void *p) {
  a->type = reinterpret_cast<uintptr_t>(p) < 0x100000000000ull ? hipMemoryTypeHost : hipMemoryTypeDevice;
  return hipSuccess;
}
}

namespace {
const void *Q = (const void *)0x7f0000000000ull;
void *WS = (void *)0x7f1000000000ull;
const void *KC = (const void *)0x7f2000000000ull, *VC = (const void *)0x7f3000000000ull;
float *OUT = (float *)0x7f4000000000ull;
const void *HOST = (const void *)0x10000000ull;
hipEvent_t EV = reinterpret_cast<hipEvent_t>(0x900);

struct Shape {
  std::vector<int> ncand, lens;
  int Hq, Hkv, balance, split = 0;
  ss_round_desc desc() {
    ss_round_desc d{};
    d.num_requests = (int)ncand.size(); d.num_q_heads = Hq; d.num_kv_heads = Hkv; d.head_dim = 128;
    d.softmax_scale = 0.088f; d.num_cand = ncand.data(); d.max_chunk_tokens = 1 << 30; d.balance_permille = balance;
    d.kv_layout = SS_KV_HEAD_MAJOR;
    d.split_tokens = split;
    return d;
  }
};
// 16 x 32768 tokens, 32q/8kv: one launch with a balancing tail (counter clear first)
Shape tailed() { return Shape{std::vector<int>(16, 6), std::vector<int>(16, 32768), 32, 8, 0}; }
// 256 requests x 4096 tokens, 8q/2kv, shares of 128 tokens: several launches, no tail
Shape many() { return Shape{std::vector<int>(256, 3), std::vector<int>(256, 4096), 8, 2, -1, 128}; }

ss_round *init(Shape &s, ss_round_desc &d) {
  d = s.desc();
  ss_round *r = nullptr;
  const ss_status st = ss_round_init(&r, &d, Q, WS, ss_round_workspace_bytes(&d), nullptr);
  CHECK(st == SS_OK && r != nullptr, "init: %s", ss_last_error());
  return r;
}

ss_status history(ss_round *r, Shape &s, hipEvent_t wait = nullptr, hipEvent_t signal = nullptr) {
  const void *k = (const void *)0x200000000000ull, *v = (const void *)0x300000000000ull;
  return ss_attend_history_chunks(r, 1, &k, &v, s.lens.data(), wait, signal, nullptr);
}

void expect_failed(ss_round *r, Shape &s, const char *what) {
  arm(-1, -1);
  CHECK(history(r, s) == SS_ERR_BAD_STATE, "%s: history after failure", what);
  CHECK(ss_attend_local_candidates(r, KC, VC, nullptr) == SS_ERR_BAD_STATE, "%s: candidates after failure", what);
  CHECK(ss_round_finalize(r, OUT, nullptr, nullptr) == SS_ERR_BAD_STATE, "%s: finalize after failure", what);
  CHECK(g_launches == 0 && g_hip_calls == 0, "%s: a refused call enqueued work", what);
}

void expect_usable(ss_round *r, Shape &s, const char *what) {
  arm(-1, -1);
  CHECK(history(r, s) == SS_OK, "%s: history after a refused call: %s", what, ss_last_error());
  CHECK(ss_attend_local_candidates(r, KC, VC, nullptr) == SS_OK, "%s: candidates", what);
  CHECK(ss_round_finalize(r, OUT, nullptr, nullptr) == SS_OK, "%s: finalize: %s", what, ss_last_error());
}
}  // namespace

int main() {
  ss_round_desc d;
  {  // the counter clear fails
    Shape s = tailed();
    ss_round *r = init(s, d);
    arm(0, -1);
    CHECK(history(r, s) == SS_ERR_HIP, "clear failure not reported");
    expect_failed(r, s, "clear failure");
    ss_round_destroy(r);
  }
  {  // the attention launch after the clear fails
    Shape s = tailed();
    ss_round *r = init(s, d);
    arm(1, -1);
    CHECK(history(r, s) == SS_ERR_HIP, "launch failure not reported");
    expect_failed(r, s, "launch after clear");
    ss_round_destroy(r);
  }
  {  // the second launch of a multi-launch call fails
    Shape s = many();
    ss_round *r = init(s, d);
    arm(1, -1);
    CHECK(history(r, s) == SS_ERR_HIP, "second launch failure not reported");
    CHECK(g_launches >= 2, "the call stopped before its second launch");
    expect_failed(r, s, "second launch");
    ss_round_destroy(r);
  }
  {  // the wait before the call fails: nothing enqueued, the round stays usable
    Shape s = many();
    ss_round *r = init(s, d);
    arm(-1, 0);
    CHECK(history(r, s, EV, nullptr) == SS_ERR_HIP, "wait failure not reported");
    CHECK(g_launches == 0, "launched after a failed wait");
    expect_usable(r, s, "failed wait");
    ss_round_destroy(r);
  }
  {  // the event record after the launches fails
    Shape s = many();
    ss_round *r = init(s, d);
    arm(-1, 0);
    CHECK(history(r, s, nullptr, EV) == SS_ERR_HIP, "record failure not reported");
    expect_failed(r, s, "failed record");
    ss_round_destroy(r);
  }
  {  // the finalize launch fails
    Shape s = many();
    ss_round *r = init(s, d);
    arm(-1, -1);
    CHECK(history(r, s) == SS_OK && ss_attend_local_candidates(r, KC, VC, nullptr) == SS_OK, "setup");
    arm(0, -1);
    CHECK(ss_round_finalize(r, OUT, nullptr, nullptr) == SS_ERR_HIP, "finalize failure not reported");
    expect_failed(r, s, "finalize launch");
    ss_round_destroy(r);
  }
  {  // host allocation failures: init, a history call, pipeline creation
    Shape s = many();
    d = s.desc();
    ss_round *r = nullptr;
    g_throw_new = true;
    CHECK(ss_round_init(&r, &d, Q, WS, ss_round_workspace_bytes(&d), nullptr) == SS_ERR_OUT_OF_MEMORY && r == nullptr,
          "init: out of memory not reported");
    g_throw_new = false;
    r = init(s, d);
    arm(-1, -1);
    g_throw_new = true;
    CHECK(history(r, s) == SS_ERR_OUT_OF_MEMORY, "history: out of memory not reported");
    g_throw_new = false;
    CHECK(g_launches == 0, "launched after an allocation failure");
    expect_usable(r, s, "allocation failure");
    ss_round_destroy(r);
    ss_pipeline *p = nullptr;
    g_throw_new = true;
    CHECK(ss_pipeline_create(&p, WS, WS, 1 << 20, nullptr) == SS_ERR_OUT_OF_MEMORY && p == nullptr,
          "pipeline: out of memory not reported");
    g_throw_new = false;
    CHECK(std::strcmp(ss_status_string(SS_ERR_OUT_OF_MEMORY), "SS_ERR_OUT_OF_MEMORY") == 0, "status string");
  }
  {  // pipeline: the attention after an enqueued upload fails
    Shape s{std::vector<int>(2, 4), std::vector<int>(2, 1024), 8, 2, -1};
    ss_round *r = init(s, d);
    ss_pipeline *p = nullptr;
    char *slot0 = (char *)0x200000000000ull, *slot1 = (char *)0x210000000000ull;
    CHECK(ss_pipeline_create(&p, slot0, slot1, 64 << 20, nullptr) == SS_OK, "pipeline create");
    arm(-1, -1);
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_OK, "first pipelined chunk: %s",
          ss_last_error());
    arm(0, -1);   // the next chunk's upload goes out, its launch fails
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_ERR_HIP, "attend failure not reported");
    arm(-1, -1);
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_ERR_BAD_STATE, "pipeline not failed");
    CHECK(g_hip_calls == 0 && g_launches == 0, "a failed pipeline enqueued work");
    ss_round *r2 = init(s, d);   // a fresh round does not revive the pipeline
    CHECK(ss_pipeline_attend_chunk(p, r2, HOST, s.lens.data(), nullptr) == SS_ERR_BAD_STATE,
          "failed pipeline accepted a new round");
    ss_round_destroy(r2);
    expect_failed(r, s, "pipelined attend");
    ss_pipeline_destroy(p);
    ss_round_destroy(r);
  }
  {  // pipeline: an upload whose copy fails after its slot-free wait went out
    Shape s{std::vector<int>(2, 4), std::vector<int>(2, 1024), 8, 2, -1};
    ss_round *r = init(s, d);
    ss_pipeline *p = nullptr;
    char *slot0 = (char *)0x200000000000ull, *slot1 = (char *)0x210000000000ull;
    CHECK(ss_pipeline_create(&p, slot0, slot1, 64 << 20, nullptr) == SS_OK, "pipeline create");
    arm(-1, -1);
    for (int c = 0; c < 2; ++c)
      CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_OK, "chunk %d: %s", c, ss_last_error());
    arm(-1, 1);   // slot 0 again: the free wait (call 0) goes out, the copy (call 1) fails
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_ERR_HIP, "copy failure not reported");
    arm(-1, -1);
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_ERR_BAD_STATE, "pipeline not failed");
    ss_pipeline_destroy(p);
    ss_round_destroy(r);
  }
  {  // pipeline: a first upload whose copy fails enqueued nothing: pipeline and round stay usable
    Shape s{std::vector<int>(2, 4), std::vector<int>(2, 1024), 8, 2, -1};
    ss_round *r = init(s, d);
    ss_pipeline *p = nullptr;
    char *slot0 = (char *)0x200000000000ull, *slot1 = (char *)0x210000000000ull;
    CHECK(ss_pipeline_create(&p, slot0, slot1, 64 << 20, nullptr) == SS_OK, "pipeline create");
    arm(-1, 0);
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_ERR_HIP, "copy failure not reported");
    arm(-1, -1);
    CHECK(ss_pipeline_attend_chunk(p, r, HOST, s.lens.data(), nullptr) == SS_OK, "pipeline unusable: %s",
          ss_last_error());
    ss_pipeline_destroy(p);
    ss_round_destroy(r);
  }
  printf("%s\n", fails ? "FAILURES" : "all ok");
  return fails ? 1 : 0;
}
