// Event-pair profiler of the kernel families (janus_profile_enable / _read)
// and the fork / join events between the caller's stream and the side stream.
#include <cstring>

#include "internal.h"

namespace janus {

static const char* kProfNames[PROF_NCLASS] = {"expert_gemm", "expert_wgrad", "dense_gemm", "edge",     "atom",
                                              "route",       "graph",        "other",      "attention"};

static hipEvent_t take_event(janus_ctx* c) {
  if (c->prof_used == c->prof_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->prof_pool.push_back(e);
  }
  return c->prof_pool[c->prof_used++];
}

ProfScope::ProfScope(janus_ctx* ctx, hipStream_t s, int cls, double flops, double bytes)
    : c(ctx), st(s), on(ctx && ctx->prof_on && (ctx->prof_mask >> cls & 1u)) {
  if (!on) return;
  rec.cls = cls;
  rec.flops = flops;
  rec.bytes = bytes;
  rec.a = take_event(c);
  rec.b = take_event(c);
  if (!rec.a || !rec.b) {
    on = false;
    return;
  }
  (void)hipEventRecord(rec.a, st);
}

ProfScope::~ProfScope() {
  if (!on) return;
  (void)hipEventRecord(rec.b, st);
  c->prof_recs.push_back(rec);
}

SideSync::SideSync(janus_ctx* ctx, hipStream_t main) : c(ctx), st(main), sd(main) {
  if (c->concurrent && c->side) sd = c->side;
}

hipEvent_t SideSync::record(hipStream_t from) {
  if (sd == st || err != hipSuccess) return nullptr;
  if (c->sync_used == c->sync_pool.size()) {
    hipEvent_t e;
    err = hipEventCreateWithFlags(&e, hipEventDisableTiming);
    if (err != hipSuccess) return nullptr;
    c->sync_pool.push_back(e);
  }
  hipEvent_t e = c->sync_pool[c->sync_used++];
  err = hipEventRecord(e, from);
  return err == hipSuccess ? e : nullptr;
}

void SideSync::order(hipStream_t from, hipStream_t to) {
  hipEvent_t e = record(from);
  if (e) err = hipStreamWaitEvent(to, e, 0);
}

void SideSync::wait(hipEvent_t e) {
  if (e && err == hipSuccess) err = hipStreamWaitEvent(st, e, 0);
}

}  // namespace janus

using namespace janus;

extern "C" int janus_profile_enable(janus_ctx* ctx, int mask) {
  if (!ctx) return JANUS_EINVAL;
  ctx->prof_on = mask != 0;
  ctx->prof_mask = (unsigned)mask;
  if (mask) {
    ctx->prof_recs.clear();
    ctx->prof_used = 0;
  }
  return JANUS_OK;
}

extern "C" int janus_profile_read(janus_ctx* ctx, janus_profile_entry* out, int32_t cap) {
  if (!ctx || (cap > 0 && !out) || cap < 0) return JANUS_EINVAL;
  janus_profile_entry acc[PROF_NCLASS];
  std::memset(acc, 0, sizeof(acc));
  for (const auto& r : ctx->prof_recs) {
    JANUS_HIP_TRY(hipEventSynchronize(r.b));
    float ms = 0.f;
    JANUS_HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
    acc[r.cls].launches += 1;
    acc[r.cls].ms += ms;
    acc[r.cls].flops += r.flops;
    acc[r.cls].bytes += r.bytes;
  }
  ctx->prof_recs.clear();
  ctx->prof_used = 0;
  int n = 0;
  for (int q = 0; q < PROF_NCLASS; ++q) {
    if (!acc[q].launches) continue;
    if (n < cap) {
      out[n] = acc[q];
      std::strncpy(out[n].name, kProfNames[q], sizeof(out[n].name) - 1);
    }
    ++n;
  }
  return n < cap ? n : cap;
}
