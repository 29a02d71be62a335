// The asynchronous deployment loop (Sec. 3.3, Fig. 1): the expert runs every control tick on one stream and reads
// the cache as it stands; the slow system's new rows are appended on a second stream (same priority) every K
// ticks.  The ring state (start / len / pos per agent) is double-buffered on the host: ticks read the FRONT state,
// appends advance the BACK state; an append is published to the ticks (front = back) by an event-ordered hand-off,
// as soon as it has completed, and at the latest K-1 ticks after it was submitted (the tick then waits for it on
// its stream), so no tick reads a cache older than K-1 ticks of the newest rows.  An append whose rows overwrite
// rows the ticks can see (a full ring) waits for the last enqueued tick and is published to the very next tick.
//
// Built on the public entry points only (fsx_expert_forward, fsx_cache_append_rows[_quantize]) plus HIP events.

#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"

struct fsx_loop {
  fsx_expert* ex = nullptr;
  fsx_cache_desc front{}, back{};
  std::vector<int64_t> fs, fl, fp, bs, bl, bp;  // front / back start, len, pos
  int32_t K = 1, policy = FSX_APPEND_RING;
  hipStream_t es = nullptr, as = nullptr;
  hipEvent_t tick_done = nullptr, append_done = nullptr;
  bool any_tick = false;
  bool pending = false;      // submitted rows the ticks do not see yet
  bool must_wait = false;    // a pending append overwrites rows visible in the front state
  int64_t ticks = 0;         // ticks enqueued so far
  int64_t first_unseen = 0;  // tick index of the first tick enqueued after the oldest pending submission
};

namespace {
thread_local std::string g_loop_err;
int lfail(int code, const std::string& m) {
  g_loop_err = m;
  return code;
}
#define LOOP_HIP(expr)                                                                                       \
  do {                                                                                                       \
    hipError_t e_ = (expr);                                                                                  \
    if (e_ != hipSuccess) return lfail(FSX_E_HIP, std::string(#expr ": ") + hipGetErrorString(e_));         \
  } while (0)
int from_api(int rc) {
  if (rc != FSX_OK) g_loop_err = fsx_last_error();
  return rc;
}
void point(fsx_cache_desc& d, std::vector<int64_t>& s, std::vector<int64_t>& l, std::vector<int64_t>& p) {
  d.start = s.data();
  d.len = l.data();
  d.pos = p.data();
}
}  // namespace

extern "C" const char* fsx_loop_last_error(void) { return g_loop_err.c_str(); }

extern "C" int fsx_loop_create(fsx_expert* ex, const fsx_cache_desc* cache, int32_t append_every, int32_t policy,
                               void* expert_stream, void* append_stream, fsx_loop** out) {
  if (!out) return lfail(FSX_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!ex || !cache) return lfail(FSX_E_INVALID, "expert and cache must be non-NULL");
  if (append_every < 1) return lfail(FSX_E_INVALID, "append_every (K) must be >= 1");
  if (policy != FSX_APPEND_RING && policy != FSX_APPEND_ERROR) return lfail(FSX_E_INVALID, "unknown append policy");
  if (cache->batch <= 0 || cache->batch > FSX_MAX_BATCH || !cache->start || !cache->len || !cache->pos)
    return lfail(FSX_E_INVALID, "cache batch must be in 1..64 with host start/len/pos arrays");
  if (cache->layout & FSX_CACHE_SHARED) return lfail(FSX_E_UNSUPPORTED, "the loop appends, a shared cache cannot");
  if (expert_stream == append_stream && expert_stream != nullptr)
    return lfail(FSX_E_INVALID, "the expert and the appends need two different streams");
  fsx_loop* lp = new fsx_loop();
  lp->ex = ex;
  lp->K = append_every;
  lp->policy = policy;
  lp->es = (hipStream_t)expert_stream;
  lp->as = (hipStream_t)append_stream;
  const int B = cache->batch;
  lp->fs.assign(cache->start, cache->start + B);
  lp->fl.assign(cache->len, cache->len + B);
  lp->fp.assign(cache->pos, cache->pos + B);
  lp->bs = lp->fs;
  lp->bl = lp->fl;
  lp->bp = lp->fp;
  lp->front = *cache;
  lp->back = *cache;
  point(lp->front, lp->fs, lp->fl, lp->fp);
  point(lp->back, lp->bs, lp->bl, lp->bp);
  if (hipEventCreateWithFlags(&lp->tick_done, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&lp->append_done, hipEventDisableTiming) != hipSuccess) {
    if (lp->tick_done) (void)hipEventDestroy(lp->tick_done);
    delete lp;
    return lfail(FSX_E_HIP, "hipEventCreateWithFlags failed");
  }
  *out = lp;
  g_loop_err.clear();
  return FSX_OK;
}

extern "C" int fsx_loop_append(fsx_loop* lp, const void* k_rows, const void* v_rows, int32_t rows_dtype,
                               int32_t n_rows) {
  if (!lp) return lfail(FSX_E_INVALID, "loop is NULL");
  if (n_rows <= 0) return lfail(FSX_E_INVALID, "n_rows must be positive");
  const int B = lp->back.batch;
  // rows visible to the ticks are overwritten when the ring wraps: wait for the ticks enqueued so far first
  bool overwrites = false;
  for (int b = 0; b < B; ++b) overwrites = overwrites || lp->bl[b] + n_rows > lp->back.capacity;
  if (overwrites && lp->policy == FSX_APPEND_ERROR)
    return lfail(FSX_E_CAPACITY, "ring full (policy FSX_APPEND_ERROR)");
  if (overwrites && lp->any_tick) LOOP_HIP(hipStreamWaitEvent(lp->as, lp->tick_done, 0));
  const int rc = rows_dtype == lp->back.dtype
                     ? fsx_cache_append_rows(&lp->back, k_rows, v_rows, n_rows, lp->policy, lp->as)
                     : fsx_cache_append_rows_quantize(&lp->back, k_rows, v_rows, rows_dtype, n_rows, lp->policy, lp->as);
  if (rc != FSX_OK) return from_api(rc);
  LOOP_HIP(hipEventRecord(lp->append_done, lp->as));
  if (!lp->pending) lp->first_unseen = lp->ticks;
  lp->pending = true;
  lp->must_wait = lp->must_wait || overwrites;
  g_loop_err.clear();
  return FSX_OK;
}

extern "C" int fsx_loop_tick(fsx_loop* lp, const void* tokens, int32_t batch, int32_t n_frame_tokens,
                             float* waypoints, float* hidden, fsx_loop_tick_info* info) {
  if (!lp) return lfail(FSX_E_INVALID, "loop is NULL");
  if (batch <= 0 || batch > lp->front.batch) return lfail(FSX_E_INVALID, "batch outside 1..cache batch");
  int32_t published = 0;
  if (lp->pending) {
    const bool forced = lp->must_wait || lp->ticks - lp->first_unseen >= lp->K - 1;
    const hipError_t q = forced ? hipErrorNotReady : hipEventQuery(lp->append_done);
    if (q != hipSuccess && q != hipErrorNotReady) return lfail(FSX_E_HIP, std::string("hipEventQuery: ") + hipGetErrorString(q));
    if (forced || q == hipSuccess) {
      // event-ordered hand-off: this tick (and every later one) runs after the appended rows are written
      LOOP_HIP(hipStreamWaitEvent(lp->es, lp->append_done, 0));
      lp->fs = lp->bs;
      lp->fl = lp->bl;
      lp->fp = lp->bp;
      point(lp->front, lp->fs, lp->fl, lp->fp);
      lp->pending = false;
      lp->must_wait = false;
      published = 1;
    }
  }
  const int rc = fsx_expert_forward(lp->ex, &lp->front, tokens, batch, n_frame_tokens, waypoints, hidden, lp->es);
  if (rc != FSX_OK) return from_api(rc);
  LOOP_HIP(hipEventRecord(lp->tick_done, lp->es));
  lp->any_tick = true;
  if (info) {
    info->tick = lp->ticks;
    info->published = published;
    info->staleness = lp->pending ? (int32_t)(lp->ticks - lp->first_unseen + 1) : 0;
    for (int b = 0; b < batch; ++b) {
      info->start[b] = lp->fs[b];
      info->len[b] = lp->fl[b];
      info->pos[b] = lp->fp[b];
    }
  }
  ++lp->ticks;
  g_loop_err.clear();
  return FSX_OK;
}

extern "C" int fsx_loop_sync(fsx_loop* lp, fsx_cache_desc* cache_out) {
  if (!lp) return lfail(FSX_E_INVALID, "loop is NULL");
  LOOP_HIP(hipStreamSynchronize(lp->as));
  LOOP_HIP(hipStreamSynchronize(lp->es));
  if (cache_out) {
    if (cache_out->batch != lp->back.batch || !cache_out->start || !cache_out->len || !cache_out->pos)
      return lfail(FSX_E_INVALID, "cache_out must have the loop's batch and host start/len/pos arrays");
    std::memcpy(cache_out->start, lp->bs.data(), sizeof(int64_t) * lp->bs.size());
    std::memcpy(cache_out->len, lp->bl.data(), sizeof(int64_t) * lp->bl.size());
    std::memcpy(cache_out->pos, lp->bp.data(), sizeof(int64_t) * lp->bp.size());
  }
  g_loop_err.clear();
  return FSX_OK;
}

extern "C" void fsx_loop_destroy(fsx_loop* lp) {
  if (!lp) return;
  if (lp->append_done) (void)hipEventSynchronize(lp->append_done);
  if (lp->tick_done) (void)hipEventSynchronize(lp->tick_done);
  (void)hipEventDestroy(lp->append_done);
  (void)hipEventDestroy(lp->tick_done);
  delete lp;
}
