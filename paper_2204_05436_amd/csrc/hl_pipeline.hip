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
//
// Streams hand over through flags in device memory rather than events: after
// the producing kernel, a one-wave kernel stores the step's sequence number
// into the flag (the producer's writes are complete and written back at its
// kernel boundary); before the consuming kernels, a one-wave kernel waits until
// the flag reaches that number (a bounded wait: past the limit it sets
// HL_DEVERR_STALL and returns).  A handover costs two small kernels (~3 us
// each) instead of an event dependency between streams (~17 us measured).
// Handovers that meet at one point of a stream share one launch (pl_hand): the
// fetch's two waits, the fetch's end signal with the next plan's fetch waits
// (the copies follow one another with one launch between them), and a plan's
// grouping signal with the next plan's waits.
// On the main stream of a planned step they ride on the kernels themselves
// (hl_hook): the forward signals the previous step's end as it starts and
// waits for the grouping as it ends, the reduction waits for the fetch, and
// the step's last kernel waits for the next plan's cold list, so main runs its
// kernels back to back (each handover launch measured ~2-3 us of main's time
// per step).
// Flags need streams that progress independently: a stream with a compute-unit
// mask has a hardware queue of its own.  Without masks (fetch_cus = 0) streams
// may share a hardware queue, where a wait ahead of its signal would stall, so
// the handovers are events then.  hl_pipeline_create checks it: for each pair
// of streams that hand over, a bounded wait is enqueued on one stream before
// the signal on the other; a wait that runs out (the two shared a queue)
// makes the creation fail (HL_ERR_UNSUPPORTED) instead of a later step
// stalling.
//
// Look-ahead (hl_pipeline_plan): the dispatch, the cold plan and the
// backward's grouping of the next mini-batch, which read only its inputs and
// the fixed hot set, run on a fourth stream while the current step trains, as
// the accelerator segregates the next mini-batch while the GPUs train (Sec. IV,
// pipeline figure).  Only that work moves ahead: the next step's row fetch
// still waits for the end of the current step (its staging rows and, with
// write-back, their write-back), so no row is read before the update that
// precedes it.  A plan waits for every step enqueued before it (their per-step
// buffers and workspace are the plan's to rewrite), so two alternating sets of
// per-step buffers suffice.  The planned step's main stream runs the forwards
// and the backward's apply, the fetch stream the copy.  (The grouping on a
// stream of its own, beside the next plan, measured slower: four busy streams
// slowed every kernel.)
#include <vector>

#include "hl_internal.h"

#define PF_PLAN 0
#define PF_FETCH 1
#define PF_FWDHOT 2
#define PF_GROUP 3
#define PF_WB 5   // the last step whose write-back has ended (write-backs run in order)
#define PF_LOOK 7 // a look-ahead plan: its own sequence
#define PF_DONE 8 // the end of a step on the main stream
#define PF_SORT 9 // a look-ahead plan's grouping (plan sequence)
#define PF_COLD 10 // a fused look-ahead plan's cold list (plan sequence; codes follow with PF_LOOK)
#define PF_N 16
#define PL_PLANS 4 // look-ahead plans not yet stepped

__global__ void pl_signal(uint32_t* flag, uint32_t v) {
  if (threadIdx.x == 0) __hip_atomic_store(flag, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// The creation's check of a pair of streams: waits up to `limit` sleeps for
// *flag to reach v; *stalled = 1 if it did not.
__global__ void pl_probe_wait(const uint32_t* flag, uint32_t v, uint32_t limit, uint32_t* stalled) {
  if (threadIdx.x != 0) return;
  uint32_t spins = 0;
  while ((int32_t)(__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) - v) < 0) {
    if (++spins > limit) {
      __hip_atomic_store(stalled, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}

__global__ void pl_wait(const uint32_t* flag, uint32_t v, uint32_t* err) {
  if (threadIdx.x != 0) return;
  uint32_t spins = 0;
  // (int32_t)(x - v) >= 0: x has reached v (sequence numbers wrap)
  while ((int32_t)(__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) - v) < 0) {
    if (++spins > HL_SPIN_LIMIT) {
      hl_flag(err, HL_DEVERR_STALL);
      return;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}

// Several handovers of one stream at one point in a single launch: the
// signal (if any), then each wait in turn.  The signal tells that the kernels
// before it on the stream are complete, as a separate pl_signal would.
__global__ void pl_hand(uint32_t* sflag, uint32_t sv, const uint32_t* w1, uint32_t v1, const uint32_t* w2,
                        uint32_t v2, const uint32_t* w3, uint32_t v3, uint32_t* err) {
  if (threadIdx.x != 0) return;
  if (sflag) __hip_atomic_store(sflag, sv, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t* wf[3] = {w1, w2, w3};
  const uint32_t wv[3] = {v1, v2, v3};
  for (int k = 0; k < 3; ++k) {
    if (!wf[k]) continue;
    uint32_t spins = 0;
    while ((int32_t)(__hip_atomic_load(wf[k], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) - wv[k]) < 0) {
      if (++spins > HL_SPIN_LIMIT) {
        hl_flag(err, HL_DEVERR_STALL);
        return;
      }
      __builtin_amdgcn_s_sleep(8);
    }
  }
}

struct pl_plan {
  hl_step_io io;      // the inputs and per-step buffers it ran with
  uint32_t seq;       // its PF_LOOK value
  uint32_t need;      // the step whose end it waits for (0: none)
  int cold_flag;      // the flag that tells its cold list is ready (PF_COLD, or PF_LOOK with the codes)
  bool pending;       // enqueued, not yet consumed by a step
};

struct hl_pipeline {
  hl_handle* h;
  hipStream_t main, fetch, group, plan;
  int32_t fetch_cus, plan_cus;
  pl_plan plans[PL_PLANS];
  uint32_t plan_seq;      // sequence number of the last look-ahead plan
  uint32_t* flags;        // [PF_N] device
  uint32_t seq;           // sequence number of the last step
  const void* wb_ids[8];  // cold lists of recent write-backs, and the step of each one's last
  uint32_t wb_seq[8];     // (a list not among them was last written back before all of these)
  int wb_next;
  bool use_flags;         // handovers through device flags (masked streams)
  bool sep_hand;          // this call's handovers as kernels of their own (HL_STEP_HANDOVER_KERNELS)
  hipEvent_t ev[PF_N];    // the same handovers as events (pipelines without masks)
  hipEvent_t ev_in, ev_out, ev_pin, ev_plan, ev_f, ev_g;
  const void* stg_ptr[4]; // staging buffers of recent steps, and the last step that used each
  uint32_t stg_seq[4];
  int stg_next;
  bool sort_pend;         // the last plan's grouping signal (value sort_v) is not enqueued yet: it
  uint32_t sort_v;        // rides on the next plan's first wait, or is enqueued alone when awaited
  bool done_pend;         // the last step's end signal (value done_v) likewise: it rides on the
  uint32_t done_v;        // next step's first main-stream wait
  const void* use_ptr[32];  // per-step buffers of recent steps, and the last step that used each
  uint32_t use_seq[32];
  int use_next;
  uint32_t np_last;       // last step that ran its own dispatch and cold plan (cold-gather hash table)
  uint32_t np_synced;     // the np_last a plan has waited for with a launch of its own
  uint32_t look_seen;     // the plan whose "cold list" the last step's last kernel waited for (0: none)
  bool fetch_pend;        // the last copy's end signal (value fetch_pv) rides on the next copy, that of
  uint32_t fetch_pv;      // plan fetch_plan (its kernel signals as it starts, and waits for its inputs)
  uint32_t fetch_plan;
  uint32_t fetch_seen;    // the plan whose fetch waits the fetch stream's last signal launch also took
  uint32_t fetch_last;    // (0: none), and the step whose end it awaited for that plan's staging rows
};

static hl_status pl_flush(hl_pipeline* p);

extern "C" hl_status hl_pipeline_destroy(hl_pipeline* p) {
  if (!p) return HL_ERR_INVALID_ARG;
  hl_status st = pl_flush(p);
  if (hipDeviceSynchronize() != hipSuccess) st = HL_ERR_HIP;
  for (hipEvent_t e : p->ev)
    if (e && hipEventDestroy(e) != hipSuccess) st = HL_ERR_HIP;
  for (hipEvent_t e : {p->ev_in, p->ev_out, p->ev_pin, p->ev_plan, p->ev_f, p->ev_g})
    if (e && hipEventDestroy(e) != hipSuccess) st = HL_ERR_HIP;
  hipStream_t ss[] = {p->main, p->fetch, p->group, p->plan};
  for (hipStream_t s : ss)
    if (s && hipStreamDestroy(s) != hipSuccess) st = HL_ERR_HIP;
  if (p->flags && hipFree(p->flags) != hipSuccess) st = HL_ERR_HIP;
  delete p;
  return st;
}

extern "C" hl_status hl_pipeline_create(hl_handle* h, int32_t fetch_cus, int32_t plan_cus, hl_pipeline** out) {
  if (!h || !out || fetch_cus < 0 || plan_cus < 0 || (plan_cus > 0 && fetch_cus == 0)) return HL_ERR_INVALID_ARG;
  hl_pipeline* p = new hl_pipeline();
  p->h = h;
  // the group stream is created on first use: look-ahead steps leave it idle,
  // and every stream takes a hardware queue
  // compute units [0, fetch_cus) for the copy, the next plan_cus for the
  // look-ahead plans (0: with main), the rest for main (and group)
  hl_stream s[3] = {nullptr, nullptr, nullptr};
  hl_status st = hl_stream_create(0, fetch_cus, 0, &s[0]);
  if (st == HL_OK) st = hl_stream_create(0, fetch_cus + plan_cus, 1, &s[1]);
  if (st == HL_OK)
    st = plan_cus ? hl_stream_create(fetch_cus, plan_cus, 0, &s[2]) : hl_stream_create(0, fetch_cus, 1, &s[2]);
  p->fetch = (hipStream_t)s[0];
  p->main = (hipStream_t)s[1];
  p->plan = (hipStream_t)s[2];
  p->fetch_cus = fetch_cus;
  p->plan_cus = plan_cus;
  p->use_flags = fetch_cus > 0;
  hipEvent_t* extra[] = {&p->ev_in, &p->ev_out, &p->ev_pin, &p->ev_plan, &p->ev_f, &p->ev_g};
  for (int i = 0; i < PF_N + 6; ++i) {
    hipEvent_t* e = i < PF_N ? &p->ev[i] : extra[i - PF_N];
    // ordering between streams of this device: a device-scope release suffices
    if (st == HL_OK && hipEventCreateWithFlags(e, hipEventDisableTiming | hipEventReleaseToDevice) != hipSuccess)
      st = HL_ERR_HIP;
  }
  // PF_N handover flags, then two words for the creation's check
  if (st == HL_OK && hipMalloc(&p->flags, (PF_N + 2) * sizeof(uint32_t)) != hipSuccess) st = HL_ERR_HIP;
  if (st == HL_OK && hipMemset(p->flags, 0, (PF_N + 2) * sizeof(uint32_t)) != hipSuccess) st = HL_ERR_HIP;
  if (st == HL_OK && p->use_flags) {
    // each pair of streams that hand over: the wait enqueued first (~10 ms at
    // most if it runs out), the signal second; sequence numbers 1, 2, ...
    uint32_t* pf = p->flags + PF_N;
    const hipStream_t pairs[][2] = {{p->fetch, p->main}, {p->main, p->fetch}, {p->plan, p->main}, {p->main, p->plan},
                                    {p->fetch, p->plan}};
    uint32_t seq = 0;
    for (const auto& pr : pairs) {
      if (st != HL_OK || pr[0] == pr[1]) continue;
      ++seq;
      hipLaunchKernelGGL(pl_probe_wait, dim3(1), dim3(64), 0, pr[0], pf, seq, 50000u, pf + 1);
      hipLaunchKernelGGL(pl_signal, dim3(1), dim3(64), 0, pr[1], pf, seq);
      if (hipGetLastError() != hipSuccess || hipStreamSynchronize(pr[0]) != hipSuccess ||
          hipStreamSynchronize(pr[1]) != hipSuccess)
        st = HL_ERR_HIP;
    }
    uint32_t stalled = 0;
    if (st == HL_OK && hipMemcpy(&stalled, pf + 1, sizeof(stalled), hipMemcpyDeviceToHost) != hipSuccess) st = HL_ERR_HIP;
    if (st == HL_OK && stalled) st = HL_ERR_UNSUPPORTED;  // two of the streams share a hardware queue
  }
  if (st != HL_OK) {
    hl_pipeline_destroy(p);
    return st;
  }
  // the write-back event starts recorded (nothing to wait for)
  if (!p->use_flags && hipEventRecord(p->ev[PF_WB], p->fetch) != hipSuccess) st = HL_ERR_HIP;
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

// handover f of step v: stream s has enqueued the producer.  (Flag mode
// records no event: event records in every step measured ~12 us slower steps.)
static hl_status pl_sig(hl_pipeline* p, hipStream_t s, int f, uint32_t v) {
  if (p->use_flags) {
    hipLaunchKernelGGL(pl_signal, dim3(1), dim3(64), 0, s, p->flags + f, v);
    return hipGetLastError() == hipSuccess ? HL_OK : HL_ERR_HIP;
  }
  return hipEventRecord(p->ev[f], s) == hipSuccess ? HL_OK : HL_ERR_HIP;
}
// stream s waits for handover f of step v
static hl_status pl_wt(hl_pipeline* p, hipStream_t s, int f, uint32_t v) {
  if (!p->use_flags) return hipStreamWaitEvent(s, p->ev[f], 0) == hipSuccess ? HL_OK : HL_ERR_HIP;
  hipLaunchKernelGGL(pl_wait, dim3(1), dim3(64), 0, s, p->flags + f, v, p->h->d_err);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_ERR_HIP;
}

// flag mode: stream s signals flag sf = sv (sf < 0: none), then waits for
// flags w1 >= v1 and w2 >= v2 (w < 0: none), in one launch
static hl_status pl_hw(hl_pipeline* p, hipStream_t s, int sf, uint32_t sv, int w1, uint32_t v1, int w2, uint32_t v2,
                       int w3 = -1, uint32_t v3 = 0) {
  if (sf < 0 && w1 < 0 && w2 < 0 && w3 < 0) return HL_OK;
  if (!p->use_flags) {
    if (sf >= 0) HL_TRY(pl_sig(p, s, sf, sv));
    if (w1 >= 0) HL_TRY(pl_wt(p, s, w1, v1));
    if (w2 >= 0) HL_TRY(pl_wt(p, s, w2, v2));
    if (w3 >= 0) HL_TRY(pl_wt(p, s, w3, v3));
    return HL_OK;
  }
  uint32_t* F = p->flags;
  hipLaunchKernelGGL(pl_hand, dim3(1), dim3(64), 0, s, sf >= 0 ? F + sf : nullptr, sv, w1 >= 0 ? F + w1 : nullptr, v1,
                     w2 >= 0 ? F + w2 : nullptr, v2, w3 >= 0 ? F + w3 : nullptr, v3, p->h->d_err);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_ERR_HIP;
}
// Flag mode: the next kernel of the path launched on the stream signals sf = sv
// as it starts and waits for wf >= wv as it ends (hl_hook_head, hl_hook_tail),
// which spares the handover launch and its kernel boundary.  A call that
// launched no such kernel leaves the handover to pl_unhook, which enqueues it
// alone (the same order: nothing ran in between).
static void pl_hook(hl_pipeline* p, int sf, uint32_t sv, int wf, uint32_t wv) {
  hl_hook& k = p->h->hook;
  k = hl_hook{};
  k.sflag = sf >= 0 ? p->flags + sf : nullptr;
  k.sv = sv;
  k.wflag = wf >= 0 ? p->flags + wf : nullptr;
  k.wv = wv;
  k.err = p->h->d_err;
}
static hl_status pl_unhook(hl_pipeline* p, hipStream_t s) {
  const hl_hook k = hl_hook_take(p->h);
  if (!k.sflag && !k.wflag && !k.w2flag) return HL_OK;
  if (k.gate) return HL_ERR_UNSUPPORTED;  // unreachable: a gate is set only for a call whose first kernel takes it
  hipLaunchKernelGGL(pl_hand, dim3(1), dim3(64), 0, s, k.sflag, k.sv, k.wflag, k.wv, k.w2flag, k.w2v, nullptr, 0u,
                     p->h->d_err);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_ERR_HIP;
}
// HL_STEP_HANDOVER_KERNELS: the waits of the handover set by pl_hook taken
// out of the call on stream s.  A gate's waits (and its signal) go into a
// pl_hand launched now, before the call; otherwise the signal stays with the
// kernel that takes the handover (not always the call's first: the grouping's
// sort gives the plan's signal once its first kernel has completed the codes)
// and the waits go into *rest, for pl_unhook after the call.
static hl_status pl_hand_split(hl_pipeline* p, hipStream_t s, hl_hook* rest) {
  hl_hook& k = p->h->hook;
  *rest = hl_hook{};
  if (!k.gate) {
    rest->wflag = k.wflag;
    rest->wv = k.wv;
    rest->w2flag = k.w2flag;
    rest->w2v = k.w2v;
    rest->err = k.err;
    k.wflag = k.w2flag = nullptr;
    return HL_OK;
  }
  const hl_hook g = hl_hook_take(p->h);
  if (!g.sflag && !g.wflag && !g.w2flag) return HL_OK;
  hipLaunchKernelGGL(pl_hand, dim3(1), dim3(64), 0, s, g.sflag, g.sv, g.wflag, g.wv, g.w2flag, g.w2v, nullptr, 0u,
                     p->h->d_err);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_ERR_HIP;
}
// a call on stream s with the handover set by pl_hook (dropped if the call
// fails); what no kernel of the call took is enqueued after it
#define PL_HOOKED(s, call)                                    \
  do {                                                        \
    hl_hook _rest{};                                          \
    if (p->sep_hand) HL_TRY(pl_hand_split(p, (s), &_rest));   \
    const hl_status _st = (call);                             \
    if (_st != HL_OK) {                                       \
      (void)hl_hook_take(p->h);                               \
      return _st;                                             \
    }                                                         \
    if (p->sep_hand) {                                        \
      _rest.sflag = p->h->hook.sflag; /* (a signal not taken) */ \
      _rest.sv = p->h->hook.sv;                               \
      p->h->hook = _rest;                                     \
    }                                                         \
    HL_TRY(pl_unhook(p, (s)));                                \
  } while (0)

// the pending signals, enqueued alone
static hl_status pl_flush_sort(hl_pipeline* p) {
  if (!p->sort_pend) return HL_OK;
  p->sort_pend = false;
  return pl_sig(p, p->plan, PF_SORT, p->sort_v);
}
static hl_status pl_flush_done(hl_pipeline* p) {
  if (!p->done_pend) return HL_OK;
  p->done_pend = false;
  return pl_sig(p, p->main, PF_DONE, p->done_v);
}
static hl_status pl_flush_fetch(hl_pipeline* p) {
  if (!p->fetch_pend) return HL_OK;
  p->fetch_pend = false;
  return pl_sig(p, p->fetch, PF_FETCH, p->fetch_pv);
}
static hl_status pl_flush(hl_pipeline* p) {
  HL_TRY(pl_flush_sort(p));
  HL_TRY(pl_flush_fetch(p));
  return pl_flush_done(p);
}
// a before b in sequence order (sequence numbers wrap)
static bool pl_before(uint32_t a, uint32_t b) { return (int32_t)(a - b) < 0; }
// the last step that used buffer x (0: none seen)
static uint32_t pl_use_last(const hl_pipeline* p, const void* x) {
  for (int i = 0; i < 32; ++i)
    if (p->use_ptr[i] == x) return p->use_seq[i];
  return 0;
}
static void pl_use_note(hl_pipeline* p, const void* x, uint32_t q) {
  if (!x) return;
  for (int i = 0; i < 32; ++i)
    if (p->use_ptr[i] == x) {
      p->use_seq[i] = q;
      return;
    }
  p->use_ptr[p->use_next] = x;
  p->use_seq[p->use_next] = q;
  p->use_next = (p->use_next + 1) % 32;
}
// the per-step buffers a plan rewrites (and a step uses)
static void pl_step_bufs(const hl_step_io* io, const void* (&b)[9]) {
  const void* v[9] = {io->gids, io->codes, io->flags, io->pop_ids, io->nonpop_ids, io->counts, io->cold_ids,
                      io->n_cold, io->workspace};
  for (int i = 0; i < 9; ++i) b[i] = v[i];
}

static hl_status pl_group(hl_pipeline* p) {
  if (p->group) return HL_OK;
  hl_stream g = nullptr;
  HL_TRY(hl_stream_create(0, p->fetch_cus + p->plan_cus, 1, &g));
  p->group = (hipStream_t)g;
  return HL_OK;
}

static hl_status pl_not_capturing(hipStream_t s) {
  // a graph keeps no stream's compute-unit mask, and capturing these masked
  // streams is not supported
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess) return HL_ERR_HIP;
  return cs == hipStreamCaptureStatusNone ? HL_OK : HL_ERR_UNSUPPORTED;
}

// the inputs, sizes and per-step buffers that a plan reads or writes
static bool pl_same_plan(const hl_step_io& a, const hl_step_io& b) {
  return a.rows == b.rows && a.bag_ptr == b.bag_ptr && a.n_samples == b.n_samples &&
         a.bags_per_sample == b.bags_per_sample && a.n_lookups == b.n_lookups && a.gids == b.gids &&
         a.codes == b.codes && a.flags == b.flags && a.pop_ids == b.pop_ids && a.nonpop_ids == b.nonpop_ids &&
         a.counts == b.counts && a.cold_ids == b.cold_ids && a.n_cold == b.n_cold &&
         a.staging_cap == b.staging_cap && a.workspace == b.workspace && a.ws_bytes == b.ws_bytes &&
         (a.dY != nullptr) == (b.dY != nullptr);
}

static pl_plan* pl_pending(hl_pipeline* p, const void* ws) {
  for (pl_plan& e : p->plans)
    if (e.pending && e.io.workspace == ws) return &e;
  return nullptr;
}

// the last step that used this staging buffer (0: none seen)
static uint32_t pl_stg_last(const hl_pipeline* p, const void* stg) {
  for (int i = 0; i < 4; ++i)
    if (p->stg_ptr[i] == stg) return p->stg_seq[i];
  return 0;
}
static void pl_stg_note(hl_pipeline* p, const void* stg, uint32_t q) {
  for (int i = 0; i < 4; ++i)
    if (p->stg_ptr[i] == stg) {
      p->stg_seq[i] = q;
      return;
    }
  p->stg_ptr[p->stg_next] = stg;
  p->stg_seq[p->stg_next] = q;
  p->stg_next = (p->stg_next + 1) % 4;
}

// the step of the last write-back that read this cold list (0: none): a list
// not among the recent ones was written back before all of them, so the
// oldest recent one bounds it
static uint32_t pl_wb_last(const hl_pipeline* p, const uint32_t* cold_ids) {
  uint32_t oldest = 0;
  for (int i = 0; i < 8; ++i) {
    if (!p->wb_ids[i]) continue;
    if (p->wb_ids[i] == cold_ids) return p->wb_seq[i];
    if (!oldest || pl_before(p->wb_seq[i], oldest)) oldest = p->wb_seq[i];
  }
  return oldest;
}
static void pl_wb_note(hl_pipeline* p, const uint32_t* cold_ids, uint32_t q) {
  for (int i = 0; i < 8; ++i)
    if (p->wb_ids[i] == cold_ids) {
      p->wb_seq[i] = q;
      return;
    }
  p->wb_ids[p->wb_next] = cold_ids;
  p->wb_seq[p->wb_next] = q;
  p->wb_next = (p->wb_next + 1) % 8;
}

// The popular mu-batch and the hot rows of the non-popular one in one launch:
// the hot half of the forward over every sample equals the popular mu-batch's
// whole forward (its rows are all hot) and the non-popular one's hot half, bit
// for bit (the same sums in the same order), so one pass over the samples
// replaces two over the two lists.
static hl_status pl_fwd_hot(hl_handle* h, const hl_step_io* io, hl_stream s) {
  return hl_embbag_fwd_part(h, io->w_hot, io->staging, io->staging_cap, io->codes, io->bag_ptr, io->n_samples,
                            io->bags_per_sample, io->n_lookups, nullptr, nullptr, io->n_samples, io->out, 1, s);
}

extern "C" hl_status hl_pipeline_plan(hl_pipeline* p, const hl_step_io* io, hl_stream stream) {
  if (!p || !io) return HL_ERR_INVALID_ARG;
  if (!p->use_flags) return HL_ERR_UNSUPPORTED;
  HL_TRY(pl_not_capturing((hipStream_t)stream));
  if (pl_pending(p, io->workspace)) return HL_ERR_INVALID_ARG;  // that plan has not been stepped yet
  p->sep_hand = io->step_flags & HL_STEP_HANDOVER_KERNELS;
  pl_plan* e = nullptr;
  for (pl_plan& c : p->plans)
    if (!c.pending) e = &c;
  if (!e) return HL_ERR_INVALID_ARG;  // too many plans ahead
  hl_handle* h = p->h;
  hipStream_t P = p->plan;
  const hl_stream PS = (hl_stream)P;
  if (!(io->step_flags & HL_STEP_UNTIED)) {
    HL_HIPTRY(hipEventRecord(p->ev_pin, (hipStream_t)stream));
    HL_HIPTRY(hipStreamWaitEvent(P, p->ev_pin, 0));
  }
  // every step that used one of the plan's per-step buffers or workspace has
  // finished with it, and so has every step that ran its own cold plan (the
  // cold-gather hash table, which plans share; steps are in order on the main
  // stream, so one wait covers them all); the previous plan's grouping signal
  // goes in the same launch
  const void* bufs[9];
  pl_step_bufs(io, bufs);
  uint32_t need = p->np_last;
  for (const void* b : bufs) {
    const uint32_t u = pl_use_last(p, b);
    if (u && (!need || pl_before(need, u))) need = u;
  }
  if (need && p->done_pend && p->done_v == need) HL_TRY(pl_flush_done(p));
  const uint32_t wb = pl_wb_last(p, io->cold_ids);
  const bool sp = p->sort_pend;
  p->sort_pend = false;
  const int32_t B = io->n_samples, bps = io->bags_per_sample;
  // the fused plan (five launches) with the grouping, when the workspace and
  // the hash table allow it
  hl_cg_fused cf{};
  bool fuse = io->dY && io->n_lookups > 0 && B > 0 &&
              hl_dispatch_fused(h, B, bps, io->n_lookups, io->workspace, io->ws_bytes);
  if (fuse)
    fuse = hl_cold_fused_begin(h, io->n_lookups, (int64_t)B * bps, B, io->staging_cap, io->workspace, io->ws_bytes, P,
                               &cf) == HL_OK;
  // The waits order the plan's writes after the reads of the steps that used
  // its buffers, and it reads nothing they wrote, except the cold-gather hash
  // table after a step that ran its own cold plan: then one launch waits
  // (its end makes that step's writes visible to the plan); otherwise the
  // dispatch kernel's blocks wait as they start, and its block 0 gives the
  // previous plan's grouping signal.
  if (p->np_last == p->np_synced && hl_dispatch_fused(h, B, bps, io->n_lookups, io->workspace, io->ws_bytes)) {
    pl_hook(p, sp ? PF_SORT : -1, p->sort_v, need ? PF_DONE : -1, need);
    h->hook.w2flag = wb ? p->flags + PF_WB : nullptr;
    h->hook.w2v = wb;
    h->hook.gate = 1;
  } else {
    HL_TRY(pl_hw(p, P, sp ? PF_SORT : -1, p->sort_v, need ? PF_DONE : -1, need, wb ? PF_WB : -1, wb));
    p->np_synced = p->np_last;
  }
  PL_HOOKED(P, hl_dispatch_ex(h, io->rows, io->bag_ptr, B, bps, io->n_lookups, io->gids, io->codes, io->flags,
                              io->pop_ids, io->nonpop_ids, io->counts, io->workspace, io->ws_bytes, PS,
                              fuse ? &cf : nullptr));
  const uint32_t v = ++p->plan_seq;
  bool sent = false;
  if (fuse) {
    // the rank scan writes the cold list: the fetch may start once it ends
    // (the grouping's first kernel signals it as it starts); that kernel also
    // completes the codes, which the first sort pass then signals as it starts
    HL_TRY(hl_cold_rank_fused(h, io->gids, io->codes, io->n_lookups, io->cold_ids, io->n_cold, io->workspace, cf, P));
    pl_hook(p, PF_LOOK, v, -1, 0);
    PL_HOOKED(P, hl_embbag_bwd_plan_signal(h, io->staging_cap, io->codes, io->bag_ptr, B, bps, io->n_lookups, nullptr,
                                           nullptr, B, io->workspace, io->ws_bytes, PS, p->flags + PF_COLD, v, &sent,
                                           &cf));
    if (!sent) HL_TRY(pl_sig(p, P, PF_COLD, v));
  } else {
    HL_TRY(hl_cold_plan(h, io->gids, io->codes, io->bag_ptr, B, bps, io->n_lookups, nullptr, nullptr, B,
                        io->staging_cap, io->cold_ids, io->n_cold, io->workspace, io->ws_bytes, PS));
    // the cold list and the codes are ready: the fetch may start while the
    // grouping runs (the grouping's first kernel gives the signal as it starts)
    if (io->dY)
      HL_TRY(hl_embbag_bwd_plan_signal(h, io->staging_cap, io->codes, io->bag_ptr, B, bps, io->n_lookups, nullptr,
                                       nullptr, B, io->workspace, io->ws_bytes, PS, p->flags + PF_LOOK, v, &sent,
                                       nullptr));
    if (!sent) HL_TRY(pl_sig(p, P, PF_LOOK, v));
  }
  p->sort_pend = true;
  p->sort_v = v;
  e->io = *io;
  e->seq = v;
  e->need = need;
  e->cold_flag = fuse ? PF_COLD : PF_LOOK;
  e->pending = true;
  return HL_OK;
}

extern "C" hl_status hl_pipeline_step(hl_pipeline* p, const hl_step_io* io, hl_stream stream) {
  if (!p || !io) return HL_ERR_INVALID_ARG;
  hl_handle* h = p->h;
  HL_TRY(pl_not_capturing((hipStream_t)stream));
  p->sep_hand = io->step_flags & HL_STEP_HANDOVER_KERNELS;
  const bool planned = io->step_flags & HL_STEP_PLANNED;
  pl_plan* e = pl_pending(p, io->workspace);
  if (planned ? !e || !pl_same_plan(e->io, *io) : e != nullptr) return HL_ERR_INVALID_ARG;
  if (!planned) HL_TRY(pl_group(p));
  // the last copy's end signal rides on this step's copy only if this is the
  // plan it was kept for
  if (p->fetch_pend && (!planned || e->seq != p->fetch_plan || io->staging_cap <= 0)) HL_TRY(pl_flush_fetch(p));
  const int32_t B = io->n_samples, bps = io->bags_per_sample, cap = io->staging_cap;
  const int64_t L = io->n_lookups;
  hipStream_t caller = (hipStream_t)stream, m = p->main, f = p->fetch, g = p->group;
  const hl_stream M = (hl_stream)m, F = (hl_stream)f, G = (hl_stream)g;
  const uint32_t q = ++p->seq;
  const uint32_t wbl = pl_wb_last(p, io->cold_ids);
  const bool tie = !(io->step_flags & HL_STEP_UNTIED);
  if (tie) {
    HL_HIPTRY(hipEventRecord(p->ev_in, caller));
    HL_HIPTRY(hipStreamWaitEvent(m, p->ev_in, 0));
    HL_HIPTRY(hipStreamWaitEvent(planned ? f : g, p->ev_in, 0));
  }
  if (planned) {
    e->pending = false;
    // main: the forwards and the backward on the planned grouping; fetch: the
    // copy, once the last step that used these staging rows has ended (a
    // write-back of the previous step precedes it on the fetch stream).  With
    // two staging buffers alternating, the copy overlaps the previous step.
    // (a pending end signal of the previous step is given by this step's
    // first main-stream launch, enqueued below)
    const uint32_t last = pl_stg_last(p, io->staging);
    if (p->fetch_pend) {
      // the copy itself gives the last copy's end signal as it starts and
      // waits for its inputs (every block, before it reads)
      pl_hook(p, PF_FETCH, p->fetch_pv, e->cold_flag, e->seq);
      h->hook.w2flag = last ? p->flags + PF_DONE : nullptr;
      h->hook.w2v = last;
      h->hook.gate = 1;
      p->fetch_pend = false;
      p->fetch_seen = 0;
      PL_HOOKED(f, hl_cold_fetch(h, io->cold_ids, io->n_cold, cap, io->w_host, io->staging, F));
    } else {
      if (p->fetch_seen != e->seq || p->fetch_last != last)
        HL_TRY(pl_hw(p, f, -1, 0, e->cold_flag, e->seq, last ? PF_DONE : -1, last));
      p->fetch_seen = 0;
      HL_TRY(hl_cold_fetch(h, io->cold_ids, io->n_cold, cap, io->w_host, io->staging, F));
    }
    // the end signal rides on the next pending plan's copy, which also waits
    // for its own inputs (its cold list, and the end of the last step that
    // used its staging rows), so the copies follow one another with no launch
    // between them.  Only for a plan that waits for no step from this one on
    // and has staging rows of its own: every signal it awaits is then enqueued
    // by the end of this call (the signal is enqueued alone if anything else
    // comes first, or at a sync).
    pl_plan* fx = nullptr;
    if (p->use_flags && !io->write_back)
      for (pl_plan& c : p->plans)
        if (c.pending && (!fx || pl_before(c.seq, fx->seq))) fx = &c;
    if (fx && ((fx->need && !pl_before(fx->need, q)) || fx->io.staging == io->staging)) fx = nullptr;
    if (fx && fx->io.staging_cap > 0) {
      p->fetch_pend = true;
      p->fetch_pv = q;
      p->fetch_plan = fx->seq;
    } else if (fx) {
      const uint32_t lx = pl_stg_last(p, fx->io.staging);
      HL_TRY(pl_hw(p, f, PF_FETCH, q, fx->cold_flag, fx->seq, lx ? PF_DONE : -1, lx));
      p->fetch_seen = fx->seq;
      p->fetch_last = lx;
    } else {
      HL_TRY(pl_sig(p, f, PF_FETCH, q));
    }
    // main: the previous step's end signal and the wait for the plan (in the
    // previous step's last kernel when it waited for this plan already, else
    // one launch); the grouping is awaited after the hot forward (the plan
    // stream carries as much work per step as main: awaiting the grouping
    // before the forward measured slower, also with plans two steps ahead).
    // The waits between main's kernels ride on the kernels before them.
    if (io->dY && p->sort_pend && p->sort_v == e->seq) HL_TRY(pl_flush_sort(p));
    const bool dp = p->done_pend;
    p->done_pend = false;
    const bool bwd = io->dY != nullptr;
    if (p->look_seen == e->seq) {
      pl_hook(p, dp ? PF_DONE : -1, p->done_v, bwd ? PF_SORT : PF_FETCH, bwd ? e->seq : q);
    } else {
      HL_TRY(pl_hw(p, m, dp ? PF_DONE : -1, p->done_v, PF_LOOK, e->seq, -1, 0));
      pl_hook(p, -1, 0, bwd ? PF_SORT : PF_FETCH, bwd ? e->seq : q);
    }
    p->look_seen = 0;
    PL_HOOKED(m, pl_fwd_hot(h, io, M));
    // the step's last kernel waits for the next pending plan's cold list (the
    // oldest; it waits only for steps before this one, so it ends without it)
    pl_plan* nx = nullptr;
    for (pl_plan& c : p->plans)
      if (c.pending && (!nx || pl_before(c.seq, nx->seq))) nx = &c;
    if (nx && nx->need && !pl_before(nx->need, q)) nx = nullptr;
    if (bwd) {
      // the reduction of the hot runs and of the staging runs inside a tile
      pl_hook(p, -1, 0, PF_FETCH, q);
      PL_HOOKED(m, hl_embbag_bwd_apply_any(h, io->w_hot, io->staging, cap, B, bps, L, io->dY, io->lr, 3,
                                           io->workspace, io->ws_bytes, M));
      // the cold half of the forward from the grouping's tail (cold lookups
      // only) with the runs that span tiles, then the staging-row updates
      pl_hook(p, -1, 0, nx ? PF_LOOK : -1, nx ? nx->seq : 0);
      PL_HOOKED(m, hl_embbag_finish_cold(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L, io->lr,
                                         io->out, io->workspace, io->ws_bytes, M));
    } else {
      pl_hook(p, -1, 0, nx ? PF_LOOK : -1, nx ? nx->seq : 0);
      PL_HOOKED(m, hl_embbag_fwd_part(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L,
                                      io->nonpop_ids, io->counts + 1, B, io->out, 2, M));
    }
    if (nx) p->look_seen = nx->seq;
  } else {
    // the look-ahead plans use the same cold-gather hash table
    const bool dp = p->done_pend;
    p->done_pend = false;
    p->look_seen = 0;
    HL_TRY(pl_hw(p, m, dp ? PF_DONE : -1, p->done_v, p->plan_seq ? PF_LOOK : -1, p->plan_seq, -1, 0));
    p->np_last = q;
    HL_TRY(hl_dispatch(h, io->rows, io->bag_ptr, B, bps, L, io->gids, io->codes, io->flags, io->pop_ids,
                       io->nonpop_ids, io->counts, io->workspace, io->ws_bytes, M));
    // the write-back that last read this cold list must end before the plan rewrites it
    if (wbl) HL_TRY(pl_wt(p, m, PF_WB, wbl));
    // a cold lookup makes its sample non-popular: no sample list needed
    HL_TRY(hl_cold_plan(h, io->gids, io->codes, io->bag_ptr, B, bps, L, nullptr, nullptr, B, cap, io->cold_ids,
                        io->n_cold, io->workspace, io->ws_bytes, M));
    HL_TRY(pl_sig(p, m, PF_PLAN, q));
    // the working parameters of the non-popular mu-batch over the host link
    p->fetch_seen = 0;
    HL_TRY(pl_wt(p, f, PF_PLAN, q));
    HL_TRY(hl_cold_fetch(h, io->cold_ids, io->n_cold, cap, io->w_host, io->staging, F));
    HL_TRY(pl_sig(p, f, PF_FETCH, q));
    // the backward's grouping needs only the codes
    HL_TRY(pl_wt(p, g, PF_PLAN, q));
    if (io->dY)
      HL_TRY(hl_embbag_bwd_plan(h, cap, io->codes, io->bag_ptr, B, bps, L, nullptr, nullptr, B, io->workspace,
                                io->ws_bytes, G));
    // the popular mu-batch and the hot rows of the non-popular one while the fetch runs
    HL_TRY(pl_fwd_hot(h, io, M));
    HL_TRY(pl_sig(p, m, PF_FWDHOT, q));
    // the reduction and the hot-row updates once both forwards have read the hot rows
    HL_TRY(pl_wt(p, g, PF_FWDHOT, q));
    if (io->dY)
      HL_TRY(hl_embbag_bwd_apply_part(h, io->w_hot, io->staging, cap, B, bps, L, io->dY, io->lr, 1, io->workspace,
                                      io->ws_bytes, G));
    HL_TRY(pl_sig(p, g, PF_GROUP, q));
    // the staging rows: cold half of the non-popular forward, then their updates
    HL_TRY(pl_wt(p, m, PF_FETCH, q));
    HL_TRY(hl_embbag_fwd_part(h, io->w_hot, io->staging, cap, io->codes, io->bag_ptr, B, bps, L, io->nonpop_ids,
                              io->counts + 1, B, io->out, 2, M));
    HL_TRY(pl_wt(p, m, PF_GROUP, q));
    if (io->dY)
      HL_TRY(hl_embbag_bwd_apply_part(h, io->w_hot, io->staging, cap, B, bps, L, io->dY, io->lr, 2, io->workspace,
                                      io->ws_bytes, M));
  }
  // the end signal waits for the next step's first main-stream launch, unless
  // the write-back below needs it now
  if (io->write_back || !p->use_flags) {
    HL_TRY(pl_sig(p, m, PF_DONE, q));
  } else {
    p->done_pend = true;
    p->done_v = q;
  }
  pl_stg_note(p, io->staging, q);
  {
    const void* bufs[9];
    pl_step_bufs(io, bufs);
    for (const void* b : bufs) pl_use_note(p, b, q);
  }
  if (io->write_back) {
    HL_TRY(pl_wt(p, f, PF_DONE, q));
    HL_TRY(hl_cold_scatter(h, io->cold_ids, io->n_cold, cap, io->staging, const_cast<void*>(io->w_host), F));
    pl_wb_note(p, io->cold_ids, q);
    HL_TRY(pl_sig(p, f, PF_WB, q));
  }
  if (tie) {
    // (the step's end waits for its copy's end signal, which would otherwise
    // ride on the next step's copy)
    HL_TRY(pl_flush_fetch(p));
    HL_HIPTRY(hipEventRecord(p->ev_out, m));
    HL_HIPTRY(hipStreamWaitEvent(caller, p->ev_out, 0));
  }
  return HL_OK;
}

extern "C" hl_status hl_pipeline_sync_writeback(hl_pipeline* p, hl_stream stream) {
  if (!p) return HL_ERR_INVALID_ARG;
  HL_TRY(pl_flush(p));
  if (!p->use_flags) {
    HL_HIPTRY(hipStreamWaitEvent((hipStream_t)stream, p->ev[PF_WB], 0));
    return HL_OK;
  }
  // the write-backs run in order on the fetch stream
  HL_HIPTRY(hipEventRecord(p->ev_f, p->fetch));
  HL_HIPTRY(hipStreamWaitEvent((hipStream_t)stream, p->ev_f, 0));
  return HL_OK;
}

extern "C" hl_status hl_pipeline_streams(const hl_pipeline* p, hl_stream* main, hl_stream* fetch, hl_stream* group) {
  if (!p) return HL_ERR_INVALID_ARG;
  if (main) *main = (hl_stream)p->main;
  if (fetch) *fetch = (hl_stream)p->fetch;
  if (group) {
    HL_TRY(pl_group(const_cast<hl_pipeline*>(p)));
    *group = (hl_stream)p->group;
  }
  return HL_OK;
}

extern "C" hl_status hl_pipeline_sync(hl_pipeline* p, hl_stream stream) {
  if (!p) return HL_ERR_INVALID_ARG;
  HL_TRY(pl_flush(p));
  hipStream_t c = (hipStream_t)stream;
  // events recorded now, behind everything enqueued on each stream
  HL_HIPTRY(hipEventRecord(p->ev_out, p->main));
  HL_HIPTRY(hipEventRecord(p->ev_plan, p->plan));
  HL_HIPTRY(hipEventRecord(p->ev_f, p->fetch));
  HL_HIPTRY(hipStreamWaitEvent(c, p->ev_out, 0));
  HL_HIPTRY(hipStreamWaitEvent(c, p->ev_plan, 0));
  HL_HIPTRY(hipStreamWaitEvent(c, p->ev_f, 0));
  if (p->group) {
    HL_HIPTRY(hipEventRecord(p->ev_g, p->group));
    HL_HIPTRY(hipStreamWaitEvent(c, p->ev_g, 0));
  }
  return HL_OK;
}
