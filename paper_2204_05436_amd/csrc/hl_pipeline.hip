// The pipelined schedule of one mini-batch (Sec. IV and Fig. "hotlinepipe":
// the popular mu-batch runs while the non-popular mu-batch's working
// parameters are gathered), as a native scheduler: three streams of default
// priority and the events that order them, enqueued by one host call.
//
//   main  : dispatch, cold plan | fwd(popular), hot half of fwd(non-popular) |
//           wait fetch: cold half of fwd(non-popular) | wait group: staging
//           row updates
//   fetch : wait plan: row fetch over the host link [| wait updates: write-back]
//   group : wait plan: the backward's grouping | wait hot halves of the
//           forwards: dY reduction, hot-row updates, staging-row sums
//
// The fetch stream runs on a few compute units of its own and the others on
// the rest: the copy keeps its units' memory queues full of slow host reads,
// and a kernel with a block on such a unit would wait for them.
#include <vector>

#include "hl_internal.h"

struct hl_pipeline {
  hl_handle* h;
  hipStream_t main, fetch, group;
  hipEvent_t ev_in, ev_plan, ev_fetch, ev_fwdhot, ev_group, ev_apply, ev_out, ev_wb[2];
  const void* wb_ids[2];  // the cold list each write-back event covers
  int wb_next;
};

extern "C" hl_status hl_pipeline_destroy(hl_pipeline* p) {
  if (!p) return HL_ERR_INVALID_ARG;
  hl_status st = HL_OK;
  if (hipDeviceSynchronize() != hipSuccess) st = HL_ERR_HIP;
  hipEvent_t evs[] = {p->ev_in, p->ev_plan, p->ev_fetch, p->ev_fwdhot, p->ev_group, p->ev_apply, p->ev_out,
                      p->ev_wb[0], p->ev_wb[1]};
  for (hipEvent_t e : evs)
    if (e && hipEventDestroy(e) != hipSuccess) st = HL_ERR_HIP;
  hipStream_t ss[] = {p->main, p->fetch, p->group};
  for (hipStream_t s : ss)
    if (s && hipStreamDestroy(s) != hipSuccess) st = HL_ERR_HIP;
  delete p;
  return st;
}

extern "C" hl_status hl_pipeline_create(hl_handle* h, int32_t fetch_cus, hl_pipeline** out) {
  if (!h || !out || fetch_cus < 0) return HL_ERR_INVALID_ARG;
  hl_pipeline* p = new hl_pipeline();
  p->h = h;
  hl_stream s[3] = {nullptr, nullptr, nullptr};
  hl_status st = hl_stream_create(0, fetch_cus, 0, &s[0]);
  if (st == HL_OK) st = hl_stream_create(0, fetch_cus, 1, &s[1]);
  if (st == HL_OK) st = hl_stream_create(0, fetch_cus, 1, &s[2]);
  p->fetch = (hipStream_t)s[0];
  p->main = (hipStream_t)s[1];
  p->group = (hipStream_t)s[2];
  hipEvent_t* evs[] = {&p->ev_in, &p->ev_plan, &p->ev_fetch, &p->ev_fwdhot, &p->ev_group, &p->ev_apply,
                       &p->ev_out, &p->ev_wb[0], &p->ev_wb[1]};
  for (hipEvent_t* e : evs)
    if (st == HL_OK && hipEventCreateWithFlags(e, hipEventDisableTiming) != hipSuccess) st = HL_ERR_HIP;
  if (st != HL_OK) {
    hl_pipeline_destroy(p);
    return st;
  }
  // the write-back events start recorded (nothing to wait for)
  for (int i = 0; i < 2; ++i)
    if (hipEventRecord(p->ev_wb[i], p->fetch) != hipSuccess) st = HL_ERR_HIP;
  *out = p;
  return st;
}

#define HL_TRY(x)                     \
  do {                                \
    hl_status _st = (x);              \
    if (_st != HL_OK) return _st;     \
  } while (0)
#define HL_HIPTRY(x)                                \
  do {                                              \
    if ((x) != hipSuccess) return HL_ERR_HIP;       \
  } while (0)

extern "C" hl_status hl_pipeline_step(hl_pipeline* p, const hl_step_io* io, hl_stream stream) {
  if (!p || !io) return HL_ERR_INVALID_ARG;
  hl_handle* h = p->h;
  // not under stream capture: a graph keeps no stream's compute-unit mask, and
  // capturing these masked streams is not supported
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing((hipStream_t)stream, &cs) != hipSuccess) return HL_ERR_HIP;
  if (cs != hipStreamCaptureStatusNone) return HL_ERR_UNSUPPORTED;
  const int32_t B = io->n_samples, bps = io->bags_per_sample, cap = io->staging_cap;
  const int64_t L = io->n_lookups;
  hipStream_t caller = (hipStream_t)stream, m = p->main, f = p->fetch, g = p->group;
  const hl_stream M = (hl_stream)m, F = (hl_stream)f, G = (hl_stream)g;
  // the write-back that last read this cold list (if any) must end before the plan rewrites it
  int slot = -1;
  for (int i = 0; i < 2; ++i)
    if (p->wb_ids[i] == io->cold_ids) slot = i;
  const bool tie = !(io->step_flags & HL_STEP_UNTIED);
  if (tie) {
    HL_HIPTRY(hipEventRecord(p->ev_in, caller));
    HL_HIPTRY(hipStreamWaitEvent(m, p->ev_in, 0));
  }
  HL_TRY(hl_dispatch(h, io->rows, io->bag_ptr, B, bps, L, io->gids, io->codes, io->flags, io->pop_ids,
                     io->nonpop_ids, io->counts, io->workspace, io->ws_bytes, M));
  if (slot >= 0) HL_HIPTRY(hipStreamWaitEvent(m, p->ev_wb[slot], 0));
  // a cold lookup makes its sample non-popular: no sample list needed
  HL_TRY(hl_cold_plan(h, io->gids, io->codes, io->bag_ptr, B, bps, L, nullptr, nullptr, B, cap, io->cold_ids,
                      io->n_cold, io->workspace, io->ws_bytes, M));
  HL_HIPTRY(hipEventRecord(p->ev_plan, m));
  HL_HIPTRY(hipStreamWaitEvent(f, p->ev_plan, 0));
  HL_TRY(hl_cold_fetch(h, io->cold_ids, io->n_cold, cap, io->w_host, io->staging, F));
  HL_HIPTRY(hipEventRecord(p->ev_fetch, f));
  HL_HIPTRY(hipStreamWaitEvent(g, p->ev_plan, 0));
  if (io->dY)
    HL_TRY(hl_embbag_bwd_plan(h, cap, io->codes, io->bag_ptr, B, bps, L, nullptr, nullptr, B, io->workspace,
                              io->ws_bytes, G));
  HL_TRY(hl_embbag_fwd_part(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L, io->pop_ids,
                            io->counts, B, io->out, 0, M));
  HL_TRY(hl_embbag_fwd_part(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L, io->nonpop_ids,
                            io->counts + 1, B, io->out, 1, M));
  HL_HIPTRY(hipEventRecord(p->ev_fwdhot, m));
  HL_HIPTRY(hipStreamWaitEvent(g, p->ev_fwdhot, 0));
  if (io->dY)
    HL_TRY(hl_embbag_bwd_apply_part(h, io->w_hot, io->staging, cap, B, bps, L, io->dY, io->lr, 1, io->workspace,
                                    io->ws_bytes, G));
  HL_HIPTRY(hipEventRecord(p->ev_group, g));
  HL_HIPTRY(hipStreamWaitEvent(m, p->ev_fetch, 0));
  HL_TRY(hl_embbag_fwd_part(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L, io->nonpop_ids,
                            io->counts + 1, B, io->out, 2, M));
  HL_HIPTRY(hipStreamWaitEvent(m, p->ev_group, 0));
  if (io->dY)
    HL_TRY(hl_embbag_bwd_apply_part(h, io->w_hot, io->staging, cap, B, bps, L, io->dY, io->lr, 2, io->workspace,
                                    io->ws_bytes, M));
  if (io->write_back) {
    HL_HIPTRY(hipEventRecord(p->ev_apply, m));
    HL_HIPTRY(hipStreamWaitEvent(f, p->ev_apply, 0));
    HL_TRY(hl_cold_scatter(h, io->cold_ids, io->n_cold, cap, io->staging, const_cast<void*>(io->w_host), F));
    if (slot < 0) {
      slot = p->wb_next;
      p->wb_next ^= 1;
    }
    p->wb_ids[slot] = io->cold_ids;
    HL_HIPTRY(hipEventRecord(p->ev_wb[slot], f));
  }
  HL_HIPTRY(hipEventRecord(p->ev_out, m));
  if (tie) HL_HIPTRY(hipStreamWaitEvent(caller, p->ev_out, 0));
  return HL_OK;
}

extern "C" hl_status hl_pipeline_sync_writeback(hl_pipeline* p, hl_stream stream) {
  if (!p) return HL_ERR_INVALID_ARG;
  HL_HIPTRY(hipStreamWaitEvent((hipStream_t)stream, p->ev_wb[0], 0));
  HL_HIPTRY(hipStreamWaitEvent((hipStream_t)stream, p->ev_wb[1], 0));
  return HL_OK;
}

extern "C" hl_status hl_pipeline_streams(const hl_pipeline* p, hl_stream* main, hl_stream* fetch, hl_stream* group) {
  if (!p) return HL_ERR_INVALID_ARG;
  if (main) *main = (hl_stream)p->main;
  if (fetch) *fetch = (hl_stream)p->fetch;
  if (group) *group = (hl_stream)p->group;
  return HL_OK;
}

extern "C" hl_status hl_pipeline_sync(hl_pipeline* p, hl_stream stream) {
  if (!p) return HL_ERR_INVALID_ARG;
  HL_HIPTRY(hipStreamWaitEvent((hipStream_t)stream, p->ev_out, 0));
  return hl_pipeline_sync_writeback(p, stream);
}
