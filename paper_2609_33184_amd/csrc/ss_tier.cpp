// Commit-aware KV tiering (paper Sec. 4.1): per request the Target KV is
// split at H <= C <= L (Eq. 8) into the Sealed History [0, H) on the host,
// the Active Tail [H, C) and the Speculative Frontier [C, L) on the GPU.
// Committed tokens older than the tail target T migrate to the host in
// blocks of g tokens (Eq. 9); H advances only once a migration's copy has
// completed, and a verification result releases only the frontier's
// rejected suffix, which never overlaps the host copy.
#include <hip/hip_runtime_api.h>

#include <cstring>
#include <new>
#include <vector>

#include "specstream.h"
#include "ss_error.h"

using ss::fail;
using ss::hip_fail;

struct ss_tier {
  int64_t T;   // Active Tail target length
  int64_t g;   // migration granularity
  struct Req {
    int64_t H = 0, C = 0, L = 0;
    bool inflight = false;
    int64_t E = 0;   // end of the in-flight migration
  };
  std::vector<Req> req;
};

namespace {

ss_status check_req(const ss_tier *t, int32_t b) {
  if (t == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "tier handle is null");
  if (b < 0 || b >= (int32_t)t->req.size())
    return fail(SS_ERR_INVALID_ARGUMENT, "request %d outside [0, %d)", b, (int)t->req.size());
  return SS_OK;
}

}  // namespace

extern "C" {

int64_t ss_tier_endpoint(int64_t H, int64_t C, int64_t T, int64_t g) {
  if (H < 0 || C < H || T < 0 || g < 1 || H % g != 0) return -1;
  const int64_t over = C - T > 0 ? C - T : 0;
  const int64_t E = g * (over / g);
  return E > H ? E : H;
}

ss_status ss_tier_create(ss_tier **out, int32_t num_requests, int64_t tail_target, int64_t granularity) {
  if (out == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (num_requests < 1) return fail(SS_ERR_INVALID_ARGUMENT, "num_requests must be >= 1 (got %d)", num_requests);
  if (tail_target < 0) return fail(SS_ERR_INVALID_ARGUMENT, "tail_target must be >= 0");
  if (granularity < 1) return fail(SS_ERR_INVALID_ARGUMENT, "granularity must be >= 1");
  ss_tier *t = new (std::nothrow) ss_tier();
  if (t == nullptr) return fail(SS_ERR_INVALID_ARGUMENT, "out of host memory");
  t->T = tail_target;
  t->g = granularity;
  t->req.resize(num_requests);
  *out = t;
  return SS_OK;
}

void ss_tier_destroy(ss_tier *t) { delete t; }

ss_status ss_tier_get(const ss_tier *t, int32_t b, int64_t *H, int64_t *C, int64_t *L) {
  ss_status s = check_req(t, b);
  if (s != SS_OK) return s;
  const ss_tier::Req &r = t->req[b];
  if (H != nullptr) *H = r.H;
  if (C != nullptr) *C = r.C;
  if (L != nullptr) *L = r.L;
  return SS_OK;
}

ss_status ss_tier_extend(ss_tier *t, int32_t b, int64_t n) {
  ss_status s = check_req(t, b);
  if (s != SS_OK) return s;
  if (n < 0) return fail(SS_ERR_INVALID_ARGUMENT, "cannot extend the frontier by %ld tokens", (long)n);
  t->req[b].L += n;
  return SS_OK;
}

ss_status ss_tier_commit(ss_tier *t, int32_t b, int64_t accepted, int64_t *released_begin, int64_t *released_end) {
  ss_status s = check_req(t, b);
  if (s != SS_OK) return s;
  ss_tier::Req &r = t->req[b];
  if (accepted < 0 || accepted > r.L - r.C)
    return fail(SS_ERR_INVALID_ARGUMENT, "accepted = %ld outside [0, %ld]", (long)accepted, (long)(r.L - r.C));
  const int64_t C2 = r.C + accepted;
  if (released_begin != nullptr) *released_begin = C2;
  if (released_end != nullptr) *released_end = r.L;
  r.C = C2;
  r.L = C2;
  return SS_OK;
}

ss_status ss_tier_plan(ss_tier *t, int32_t b, int64_t *begin, int64_t *end) {
  ss_status s = check_req(t, b);
  if (s != SS_OK) return s;
  ss_tier::Req &r = t->req[b];
  int64_t E = r.H;
  if (!r.inflight) E = ss_tier_endpoint(r.H, r.C, t->T, t->g);
  if (E < 0) return fail(SS_ERR_BAD_STATE, "tier state of request %d is inconsistent", b);
  if (begin != nullptr) *begin = r.H;
  if (end != nullptr) *end = E;
  if (E > r.H) {
    r.inflight = true;
    r.E = E;
  }
  return SS_OK;
}

ss_status ss_tier_complete(ss_tier *t, int32_t b) {
  ss_status s = check_req(t, b);
  if (s != SS_OK) return s;
  ss_tier::Req &r = t->req[b];
  if (!r.inflight) return fail(SS_ERR_BAD_STATE, "request %d has no migration in flight", b);
  r.H = r.E;
  r.inflight = false;
  return SS_OK;
}

ss_status ss_download_range(void *dst_pinned_host, const void *src_device, size_t bytes, hipStream_t copy_stream,
                            hipEvent_t wait_before, hipEvent_t signal_after) {
  if (dst_pinned_host == nullptr || src_device == nullptr)
    return fail(SS_ERR_INVALID_ARGUMENT, "download pointers must be non-null");
  if (bytes == 0) return fail(SS_ERR_INVALID_ARGUMENT, "download of 0 bytes");
  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof attr);
  hipError_t e = hipPointerGetAttributes(&attr, dst_pinned_host);
  if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return fail(SS_ERR_NOT_PINNED, "download destination %p is not pinned host memory", dst_pinned_host);
  }
  std::memset(&attr, 0, sizeof attr);
  e = hipPointerGetAttributes(&attr, src_device);
  if (e != hipSuccess || attr.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(SS_ERR_INVALID_ARGUMENT, "download source %p is not device memory", src_device);
  }
  if (wait_before != nullptr && (e = hipStreamWaitEvent(copy_stream, wait_before, 0)) != hipSuccess)
    return hip_fail(e, "hipStreamWaitEvent (download)");
  if ((e = hipMemcpyAsync(dst_pinned_host, src_device, bytes, hipMemcpyDeviceToHost, copy_stream)) != hipSuccess)
    return hip_fail(e, "hipMemcpyAsync (download)");
  if (signal_after != nullptr && (e = hipEventRecord(signal_after, copy_stream)) != hipSuccess)
    return hip_fail(e, "hipEventRecord (download)");
  return SS_OK;
}

}  // extern "C"
