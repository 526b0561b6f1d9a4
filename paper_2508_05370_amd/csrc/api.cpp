// api.cpp -- the C ABI (include/hetsim.h): context lifetime, workspace, launches.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "hetsim.h"
#include "internal.h"

namespace hetsim {
hipError_t launch_fill32(uint32_t* p, uint32_t n, uint32_t v, hipStream_t s);
hipError_t launch_prep(const Tab& t, const sim_plans& p, int64_t n, uint64_t* out, PackedPlan* packed, uint4* pcut,
                       uint32_t* meta, uint32_t* hist, uint16_t* keys, hipStream_t s);
hipError_t launch_memory(const Tab& t, const sim_plans& p, int64_t n, uint64_t* out, hipStream_t s);
hipError_t launch_plan_syncs(const Tab& t, const PackedPlan* packed, const uint4* pcut, const uint32_t* meta,
                             int64_t n, uint64_t* hdp, uint32_t* pc, uint32_t* perm, hipStream_t s);
hipError_t launch_stages(const Tab& t, const PackedPlan* packed, const uint4* pcut, const uint32_t* meta, int64_t n,
                         uint64_t* out_stage, hipStream_t s);
hipError_t launch_scan(const uint32_t* hist, uint32_t* cursor, uint32_t* sstart, uint32_t* sbase, bool grouped,
                       uint32_t* ids, hipStream_t s);
hipError_t launch_scatter(const uint16_t* keys, uint32_t nslots, uint32_t* cursor, const uint32_t* sbase, bool grouped,
                          uint32_t* ids, hipStream_t s);
hipError_t launch_first(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s);
hipError_t launch_group(const Tab& t, const EvalArgs& a, uint32_t max_tasks, int g, hipStream_t s);
hipError_t launch_variant(const Tab& t, const EvalArgs& a, int g, hipStream_t s);
hipError_t launch_deferred(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s);
hipError_t launch_argmin(const uint64_t* t, int64_t n, int64_t base, sim_best* b, hipStream_t s);
hipError_t launch_best_reduce(const sim_best* in, int64_t n, sim_best* out, hipStream_t s);
hipError_t launch_node_probe(double* sink, int blocks, int iters, hipStream_t s);
}  // namespace hetsim

using namespace hetsim;

namespace {
// plans per internal chunk: bounds the temporary memory of one call
constexpr int64_t kChunk = 1 << 21;

struct EventPair {
  hipEvent_t a, b;
};
}  // namespace

// Side streams of multi-chunk calls made on one caller stream: two for the
// four first-pass groups and one for the deferred pass.  Each caller stream
// gets its own set, so calls on different caller streams do not queue behind
// each other.  The groups pair up long with short -- 13-16 with 1-4 stages,
// 9-12 with 5-8 -- so two evaluation kernels run at once: measured on the
// 16M-plan sweep, four at once (one stream each, with enough hardware
// queues) ran 13 % slower, and the other pairings 2-6 % slower.
constexpr int kGroupStreams = 2;
constexpr int kGroupStream[4] = {0, 1, 1, 0};
struct SideStreams {
  hipStream_t caller;
  hipStream_t aux;
  hipStream_t grp[kGroupStreams];
};

// Streams this context has launched work on, each with an event recorded
// after its latest call: sim_destroy waits for these (and the side streams)
// rather than for the whole device.  The events are created with the
// context, so that recording one allocates nothing.
constexpr int kTracked = 16;

struct sim_ctx {
  Tab tab;
  int device;
  void* tables;        // one device allocation holding every table
  hipMemPool_t pool;   // stream-ordered pool for per-call workspace
  std::mutex mu;
  bool timing;
  std::vector<EventPair> ev[4];
  uint64_t* skipped_ops;   // device counter, inside `tables`
  Tab* dtab;               // copy of `tab` in device memory, inside `tables`
  std::vector<SideStreams> side;   // per caller stream, created on first use
  hipStream_t seen[kTracked];      // caller streams of calls so far
  hipEvent_t seen_ev[kTracked];    // recorded after the latest call on seen[j]
  int nseen;
  bool untracked;                  // more than kTracked streams were used
};

constexpr size_t kSkipBytes = (size_t)kSkipSlots * kSkipStride * 8;

extern "C" const char* sim_strerror(int code) {
  switch (code) {
    case SIM_OK: return "ok";
    case SIM_EINVAL: return "invalid argument or descriptor";
    case SIM_ERANGE: return "descriptor could overflow 64-bit picosecond arithmetic";
    case SIM_ENOMEM: return "out of memory";
    case SIM_EHIP: return "HIP runtime error";
    case SIM_ESIZE: return "more plans than the allocation-free entry point's workspace holds (SIM_NOALLOC_MAX_PLANS)";
    default: return "unknown error";
  }
}

extern "C" int sim_create(const sim_model_desc* model, const sim_cluster_desc* cluster, sim_ctx** out) {
  if (!out) return SIM_EINVAL;
  *out = nullptr;
  HostTables* ht = new (std::nothrow) HostTables();
  if (!ht) return SIM_ENOMEM;
  int rc = build_tables(model, cluster, ht);
  if (rc != SIM_OK) { delete ht; return rc; }
  sim_ctx* c = new (std::nothrow) sim_ctx();
  if (!c) { delete ht; return SIM_ENOMEM; }
  c->tab = ht->tab;
  c->timing = false;
  c->tables = nullptr;
  c->pool = nullptr;
  c->nseen = 0;
  c->untracked = false;
  for (auto& e : c->seen_ev) e = nullptr;
  if (hipGetDevice(&c->device) != hipSuccess) { delete ht; delete c; return SIM_EHIP; }
  for (auto& e : c->seen_ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      for (auto& x : c->seen_ev)
        if (x) (void)hipEventDestroy(x);
      delete ht; delete c; return SIM_EHIP;
    }
  // this device's copy of the allocation-free workspace (resolved once per device)
  void* scratch = nullptr;
  auto fail = [&](int rc) {
    for (auto& x : c->seen_ev) (void)hipEventDestroy(x);
    if (c->tables) (void)hipFree(c->tables);
    delete ht;
    delete c;
    return rc;
  };
  if (noalloc_scratch(c->device, &scratch) != 0) return fail(SIM_EHIP);
  // the table image, then the skipped-work counter slots
  const size_t img = align256(ht->img.size());
  if (hipMalloc(&c->tables, img + kSkipBytes + align256(sizeof(Tab))) != hipSuccess) {
    c->tables = nullptr;
    return fail(SIM_ENOMEM);
  }
  if (hipMemcpy(c->tables, ht->img.data(), ht->img.size(), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset((char*)c->tables + img, 0, kSkipBytes) != hipSuccess)
    return fail(SIM_EHIP);
  c->tab.img = c->tables;
  if (eval_grids(&c->tab) != 0) return fail(SIM_EHIP);
  c->skipped_ops = (uint64_t*)((char*)c->tables + img);
  c->dtab = (Tab*)((char*)c->tables + img + kSkipBytes);
  if (hipMemcpy(c->dtab, &c->tab, sizeof(Tab), hipMemcpyHostToDevice) != hipSuccess) return fail(SIM_EHIP);
  hipMemPoolProps props;
  memset(&props, 0, sizeof(props));
  props.allocType = hipMemAllocationTypePinned;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = c->device;
  if (hipMemPoolCreate(&c->pool, &props) != hipSuccess) {
    c->pool = nullptr;
    return fail(SIM_EHIP);
  }
  delete ht;
  uint64_t keep = UINT64_MAX;   // keep workspace memory cached between calls
  (void)hipMemPoolSetAttribute(c->pool, hipMemPoolAttrReleaseThreshold, &keep);
  *out = c;
  return SIM_OK;
}

// Record that a call has been launched on stream s (after its last launch).
static void track(sim_ctx* c, hipStream_t s) {
  std::lock_guard<std::mutex> g(c->mu);
  int j = 0;
  while (j < c->nseen && c->seen[j] != s) ++j;
  if (j == c->nseen) {
    if (j == kTracked) {
      c->untracked = true;
      return;
    }
    c->seen[c->nseen++] = s;
  }
  (void)hipEventRecord(c->seen_ev[j], s);
}

extern "C" void sim_destroy(sim_ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  // wait for this context's work: its side streams and the latest call on
  // every caller stream it was given (the whole device only if it was given
  // more streams than it tracks)
  for (auto& q : c->side) {
    (void)hipStreamSynchronize(q.aux);
    for (auto g : q.grp) (void)hipStreamSynchronize(g);
  }
  if (c->untracked) (void)hipDeviceSynchronize();
  for (int j = 0; j < c->nseen; ++j) (void)hipEventSynchronize(c->seen_ev[j]);
  for (auto& v : c->ev)
    for (auto& e : v) { (void)hipEventDestroy(e.a); (void)hipEventDestroy(e.b); }
  for (auto& e : c->seen_ev) (void)hipEventDestroy(e);
  for (auto& q : c->side) {
    (void)hipStreamDestroy(q.aux);
    for (auto g : q.grp) (void)hipStreamDestroy(g);
  }
  if (c->pool) (void)hipMemPoolDestroy(c->pool);
  if (c->tables) (void)hipFree(c->tables);
  delete c;
}

static bool plans_ok(const sim_plans* p, int64_t n) {
  return p && p->hdr && (p->chdr ? p->ccut != nullptr : p->cut != nullptr) && p->cls && p->types &&
         p->stride >= n && n >= 0;
}

static bool begin_event(sim_ctx* c, int kind, hipStream_t s, EventPair* e) {
  if (!c->timing) return false;
  if (hipEventCreate(&e->a) != hipSuccess) return false;
  if (hipEventCreate(&e->b) != hipSuccess) { (void)hipEventDestroy(e->a); return false; }
  (void)hipEventRecord(e->a, s);
  (void)kind;
  return true;
}
static void end_event(sim_ctx* c, int kind, hipStream_t s, EventPair* e) {
  (void)hipEventRecord(e->b, s);
  std::lock_guard<std::mutex> g(c->mu);
  c->ev[kind].push_back(*e);
}

// The side streams of caller stream s (created on its first multi-chunk call).
static bool side_streams(sim_ctx* c, hipStream_t s, SideStreams* out) {
  std::lock_guard<std::mutex> g(c->mu);
  for (auto& q : c->side)
    if (q.caller == s) {
      *out = q;
      return true;
    }
  SideStreams q = {s, nullptr, {nullptr, nullptr}};
  bool ok = hipStreamCreateWithFlags(&q.aux, hipStreamNonBlocking) == hipSuccess;
  for (auto& x : q.grp) ok = ok && hipStreamCreateWithFlags(&x, hipStreamNonBlocking) == hipSuccess;
  if (!ok) {
    if (q.aux) (void)hipStreamDestroy(q.aux);
    for (auto x : q.grp)
      if (x) (void)hipStreamDestroy(x);
    return false;
  }
  c->side.push_back(q);
  *out = q;
  return true;
}

// Chunks of kChunk plans (one chunk up to 2 kChunk).  With more than one chunk, the four stage-count
// groups of chunk i's first pass run on two side streams (paired as
// kGroupStream says), and its deferred pass on a third that waits for them,
// while the call's stream packs and sorts chunk i + 1.  The two workspaces alternate; the call's
// stream waits for chunk i's deferred pass before reusing its workspace for
// chunk i + 2 and, at the end, for the last one.
extern "C" int sim_eval_plans(sim_ctx* c, const sim_plans* plans, int64_t n, uint64_t* out, void* stream) {
  if (!c || !plans_ok(plans, n) || (n > 0 && !out)) return SIM_EINVAL;
  if (n == 0) return SIM_OK;
  hipStream_t s = (hipStream_t)stream;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  // up to two chunks' worth of plans run as one chunk on the caller's stream
  // alone (so that calls on several caller streams overlap each other);
  // larger calls are worked in kChunk chunks, double-buffered, with side
  // streams
  const int64_t ch = n <= 2 * kChunk ? n : kChunk;
  const int nbuf = n > ch ? 2 : 1;
  hipStream_t aux = s;
  SideStreams side = {};
  constexpr int kEv = 2 * 6;   // per buffer: sorted, four group ends, deferred end
  hipEvent_t evs[kEv] = {};
  auto sorted = [&](int b) { return evs[b * 6]; };
  auto fin = [&](int b, int g) { return evs[b * 6 + 1 + g]; };
  auto done = [&](int b) { return evs[b * 6 + 5]; };
  if (nbuf == 2) {
    if (!side_streams(c, s, &side)) return SIM_EHIP;
    aux = side.aux;
    for (int j = 0; j < kEv; ++j)
      if (hipEventCreateWithFlags(&evs[j], hipEventDisableTiming) != hipSuccess) {
        for (auto& x : evs)
          if (x) (void)hipEventDestroy(x);
        return SIM_EHIP;
      }
  }
  void* ws = nullptr;
  const bool het = plans->chdr != nullptr;
  hipError_t e = hipMallocFromPoolAsync(&ws, nbuf * work_bytes(ch, het), c->pool, s);
  if (e != hipSuccess) ws = nullptr;
  Work w[2];
  for (int j = 0; ws && j < nbuf; ++j) w[j] = carve((char*)ws + j * work_bytes(ch, het), ch, het);
  EventPair call, ev;
  bool tcall = ws && begin_event(c, 2, s, &call);
  bool joined = true;
  int64_t i = 0;
  for (int64_t off = 0; ws && off < n && e == hipSuccess; off += ch, ++i) {
    const int64_t cn = n - off < ch ? n - off : ch;
    const int b = (int)(i % nbuf);
    const Work& W = w[b];
    sim_plans p = *plans;
    p.hdr += off; p.cls += off; p.types += off;
    if (p.cut) p.cut += off;
    if (het) { p.chdr += off; p.ccut += off; }
    if (i >= 2) e = hipStreamWaitEvent(s, done(b), 0);
    if (e == hipSuccess) e = launch_fill32(W.hist, kCounters, 0, s);
    bool t1 = e == hipSuccess && begin_event(c, 1, s, &ev);
    if (e == hipSuccess) e = launch_prep(c->tab, p, cn, out + off, W.packed, W.pcut, W.meta, W.hist, W.keys, s);
    if (t1) end_event(c, 1, s, &ev);
    // (the plan order goes to the variant-tile array, unused in this layout until the deferred sort)
    if (e == hipSuccess && het)
      e = launch_plan_syncs(c->tab, W.packed, W.pcut, W.meta, cn, W.hdp, W.ctr + kEvalCounters, W.vlist, s);
    // shared-layout calls sort plans by plan: the scan and the scatter mark
    // the padding lanes
    if (e == hipSuccess) e = launch_scan(W.hist, W.cursor, W.sstart, W.sbase, !het, W.ids, s);
    if (e == hipSuccess) e = launch_scatter(W.keys, (uint32_t)(cn * 4), W.cursor, W.sbase, !het, W.ids, s);
    const EvalArgs a = {W.packed, W.pcut, W.hdp, W.meta, W.ids, W.sstart, out + off, W.ctr, W.deferred, W.vlist,
                        c->timing ? c->skipped_ops : nullptr, c->dtab};
    EventPair e0;
    bool t0 = e == hipSuccess && begin_event(c, 0, s, &e0);
    if (nbuf == 1) {
      if (e == hipSuccess) e = launch_first(c->tab, a, (uint32_t)(cn * 4), s);
      if (t0) end_event(c, 0, s, &e0);
      if (e != hipSuccess) break;
    } else {
      if (e == hipSuccess) e = hipEventRecord(sorted(b), s);
      joined = false;
      for (int g = 0; g < 4 && e == hipSuccess; ++g) {
        const hipStream_t gs = side.grp[kGroupStream[g]];
        e = hipStreamWaitEvent(gs, sorted(b), 0);
        if (e == hipSuccess) e = launch_group(c->tab, a, (uint32_t)(cn * 4), g, gs);
        if (e == hipSuccess) e = launch_variant(c->tab, a, g, gs);
        if (e == hipSuccess) e = hipEventRecord(fin(b, g), gs);
        if (e == hipSuccess) e = hipStreamWaitEvent(aux, fin(b, g), 0);
      }
      if (t0) end_event(c, 0, aux, &e0);
      if (e != hipSuccess) break;
    }
    bool t3 = begin_event(c, 3, aux, &ev);
    e = launch_deferred(c->tab, a, (uint32_t)(cn * 4), aux);
    if (t3) end_event(c, 3, aux, &ev);
    if (nbuf == 2) {
      const hipError_t r = hipEventRecord(done(b), aux);
      if (e == hipSuccess) e = r;
    }
  }
  // the call's stream takes over everything the side streams were given (after
  // a failed launch, drain them before the workspace is released)
  if (nbuf == 2 && e != hipSuccess) {
    for (auto q : side.grp) (void)hipStreamSynchronize(q);
    (void)hipStreamSynchronize(aux);
  } else if (!joined) {
    for (int g = 0; g < 4; ++g) {
      const hipError_t r = hipStreamWaitEvent(s, fin((int)((i - 1) % 2), g), 0);
      if (e == hipSuccess) e = r;
    }
    const hipError_t r = hipStreamWaitEvent(s, done((int)((i - 1) % 2)), 0);
    if (e == hipSuccess) e = r;
  }
  if (tcall) end_event(c, 2, s, &call);
  if (ws) (void)hipFreeAsync(ws, s);
  track(c, s);
  for (auto& x : evs)
    if (x) (void)hipEventDestroy(x);
  if (!ws) return SIM_ENOMEM;
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

static_assert(SIM_NOALLOC_MAX_PLANS == kNoAllocPlans && SIM_NOALLOC_MAX_PLANS_PER_CLASS == kNoAllocPlansHet,
              "allocation-free limits");

// One chunk on the caller's stream, with the workspace in the static device
// array: no allocation, no side streams, no events.
extern "C" int sim_eval_plans_noalloc(sim_ctx* c, const sim_plans* plans, int64_t n, uint64_t* out, void* stream) {
  if (!c || !plans_ok(plans, n) || (n > 0 && !out)) return SIM_EINVAL;
  if (n == 0) return SIM_OK;
  const bool het = plans->chdr != nullptr;
  if (n > (het ? kNoAllocPlansHet : kNoAllocPlans)) return SIM_ESIZE;
  hipStream_t s = (hipStream_t)stream;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  void* ws = nullptr;
  if (noalloc_scratch(c->device, &ws) != 0) return SIM_EHIP;
  const Work W = carve(ws, n, het);
  hipError_t e = launch_fill32(W.hist, kCounters, 0, s);
  if (e == hipSuccess) e = launch_prep(c->tab, *plans, n, out, W.packed, W.pcut, W.meta, W.hist, W.keys, s);
  if (e == hipSuccess && het)
    e = launch_plan_syncs(c->tab, W.packed, W.pcut, W.meta, n, W.hdp, W.ctr + kEvalCounters, W.vlist, s);
  if (e == hipSuccess) e = launch_scan(W.hist, W.cursor, W.sstart, W.sbase, !het, W.ids, s);
  if (e == hipSuccess) e = launch_scatter(W.keys, (uint32_t)(n * 4), W.cursor, W.sbase, !het, W.ids, s);
  const EvalArgs a = {W.packed, W.pcut, W.hdp, W.meta, W.ids, W.sstart, out, W.ctr, W.deferred, W.vlist,
                      c->timing ? c->skipped_ops : nullptr, c->dtab};
  if (e == hipSuccess) e = launch_first(c->tab, a, (uint32_t)(n * 4), s);
  if (e == hipSuccess) e = launch_deferred(c->tab, a, (uint32_t)(n * 4), s);
  // a stream under graph capture records nothing here: the launches become
  // graph nodes, and the caller owns the graph's completion
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cap) == hipSuccess && cap == hipStreamCaptureStatusNone) track(c, s);
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

extern "C" int sim_eval_stages(sim_ctx* c, const sim_plans* plans, int64_t n, uint64_t* out_stage,
                               uint32_t* out_class, void* stream) {
  if (!c || !plans_ok(plans, n) || (n > 0 && (!out_stage || !out_class))) return SIM_EINVAL;
  if (n == 0) return SIM_OK;
  hipStream_t s = (hipStream_t)stream;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  void* ws = nullptr;
  const bool het = plans->chdr != nullptr;
  const int64_t ch = n < kChunk ? n : kChunk;
  if (hipMallocFromPoolAsync(&ws, align256((size_t)ch * sizeof(PackedPlan)) + cut_rows_bytes(ch, het), c->pool, s) !=
      hipSuccess)
    return SIM_ENOMEM;
  PackedPlan* packed = (PackedPlan*)ws;
  uint4* pcut = het ? (uint4*)((char*)ws + align256((size_t)ch * sizeof(PackedPlan))) : nullptr;
  hipError_t e = hipSuccess;
  // chunks of kChunk plans through one workspace, in order on the stream
  for (int64_t off = 0; off < n && e == hipSuccess; off += ch) {
    const int64_t cn = n - off < ch ? n - off : ch;
    sim_plans p = *plans;
    p.hdr += off; p.cls += off; p.types += off;
    if (p.cut) p.cut += off;
    if (het) { p.chdr += off; p.ccut += off; }
    e = launch_prep(c->tab, p, cn, nullptr, packed, pcut, out_class + off * 4, nullptr, nullptr, s);
    if (e == hipSuccess)
      e = launch_stages(c->tab, packed, pcut, out_class + off * 4, cn, out_stage + off * 4 * kMaxStages * 4, s);
  }
  (void)hipFreeAsync(ws, s);
  track(c, s);
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

extern "C" int sim_eval_memory(sim_ctx* c, const sim_plans* plans, int64_t n, uint64_t* out_mem, void* stream) {
  if (!c || !plans_ok(plans, n) || (n > 0 && !out_mem)) return SIM_EINVAL;
  if (n == 0) return SIM_OK;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  for (int64_t off = 0; off < n && e == hipSuccess; off += kChunk) {
    const int64_t cn = n - off < kChunk ? n - off : kChunk;
    sim_plans p = *plans;
    p.hdr += off; p.cls += off; p.types += off;
    if (p.cut) p.cut += off;
    if (p.chdr) { p.chdr += off; p.ccut += off; }
    e = launch_memory(c->tab, p, cn, out_mem + off * 4 * kMaxStages, s);
  }
  track(c, s);
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

extern "C" int sim_argmin(sim_ctx* c, const uint64_t* t, int64_t n, int64_t base, sim_best* out, void* stream) {
  if (!c || !out || n < 0 || (n > 0 && !t)) return SIM_EINVAL;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  const hipError_t e = launch_argmin(t, n, base, out, (hipStream_t)stream);
  track(c, (hipStream_t)stream);
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

extern "C" int sim_best_reduce(sim_ctx* c, const sim_best* in, int64_t n, sim_best* out, void* stream) {
  if (!c || !out || n < 0 || (n > 0 && !in)) return SIM_EINVAL;
  if (hipSetDevice(c->device) != hipSuccess) return SIM_EHIP;
  const hipError_t e = launch_best_reduce(in, n, out, (hipStream_t)stream);
  track(c, (hipStream_t)stream);
  return e == hipSuccess ? SIM_OK : SIM_EHIP;
}

extern "C" int sim_set_timing(sim_ctx* c, int enable) {
  if (!c) return SIM_EINVAL;
  c->timing = enable != 0;
  return SIM_OK;
}

extern "C" int sim_get_skipped_ops(sim_ctx* c, uint64_t* ops) {
  if (!c || !ops) return SIM_EINVAL;
  std::vector<uint64_t> v((size_t)kSkipSlots * kSkipStride);
  if (hipSetDevice(c->device) != hipSuccess || hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(v.data(), c->skipped_ops, kSkipBytes, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemset(c->skipped_ops, 0, kSkipBytes) != hipSuccess)
    return SIM_EHIP;
  uint64_t sum = 0;
  for (uint32_t j = 0; j < kSkipSlots; ++j) sum += v[(size_t)j * kSkipStride];
  *ops = sum;
  return SIM_OK;
}

extern "C" int sim_get_timing(sim_ctx* c, int kind, double* total_ms, int64_t* launches) {
  if (!c || kind < 0 || kind > 3 || !total_ms || !launches) return SIM_EINVAL;
  std::vector<EventPair> v;
  {
    std::lock_guard<std::mutex> g(c->mu);
    v.swap(c->ev[kind]);
  }
  double sum = 0;
  int rc = SIM_OK;
  for (auto& e : v) {
    float ms = 0;
    if (hipEventSynchronize(e.b) != hipSuccess || hipEventElapsedTime(&ms, e.a, e.b) != hipSuccess) rc = SIM_EHIP;
    sum += ms;
    (void)hipEventDestroy(e.a);
    (void)hipEventDestroy(e.b);
  }
  *total_ms = sum;
  *launches = (int64_t)v.size();
  return rc;
}

// Times the node probe on `stream` (blocking): 32 blocks of 256 threads per
// CU, 8 chains per thread, 4096 nodes per chain; the faster of two timed runs
// after one warm-up.
extern "C" int sim_measure_node_rate(double* nodes_per_s, void* stream) {
  if (!nodes_per_s) return SIM_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return SIM_EHIP;
  const int blocks = 32 * cus, iters = 4096;
  double* sink = nullptr;
  if (hipMalloc(&sink, (size_t)blocks * 256 * sizeof(double)) != hipSuccess) return SIM_ENOMEM;
  hipEvent_t a = nullptr, b = nullptr;
  int rc = SIM_OK;
  float best = 0;
  if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) rc = SIM_EHIP;
  for (int r = 0; r < 3 && rc == SIM_OK; ++r) {
    if (hipEventRecord(a, s) != hipSuccess || launch_node_probe(sink, blocks, iters, s) != hipSuccess ||
        hipEventRecord(b, s) != hipSuccess || hipEventSynchronize(b) != hipSuccess) {
      rc = SIM_EHIP;
      break;
    }
    float ms = 0;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) rc = SIM_EHIP;
    if (r > 0 && (best == 0 || ms < best)) best = ms;
  }
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  (void)hipFree(sink);
  if (rc != SIM_OK) return rc;
  if (best <= 0) return SIM_EHIP;
  *nodes_per_s = (double)blocks * 256 * 8 * iters / (best * 1e-3);
  return SIM_OK;
}
