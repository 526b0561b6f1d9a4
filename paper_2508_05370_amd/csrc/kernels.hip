// kernels.hip -- the plan evaluator's kernels other than the evaluation
// passes (those are in eval_pass.hip): packing and checking, bucketing,
// per-stage records, device memory, the u64 redo and the argmin; and the
// launchers the C ABI calls.  The data flow is described in device.h.
#include <mutex>

#include "launch.h"

namespace hetsim {

// ---------------------------------------------------------------- allocation-free workspace
// The workspace of sim_eval_plans_noalloc: one chunk's buffers (kNoAllocBytes,
// about 46 MiB) in a static device array.  Every GPU the library runs on holds
// its own copy until the process ends; host code reaches it only through the
// address hipGetSymbolAddress returns for the current device (the array's
// name in host code is a host-side stand-in, not a device address).
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices];
}  // namespace

int noalloc_scratch(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices || !ptr) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(scratch_mu);
  if (!scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess) return (int)r;
    if (!p) return (int)hipErrorInvalidSymbol;
    scratch_ptr[device] = p;
  }
  *ptr = scratch_ptr[device];
  return 0;
}

// ---------------------------------------------------------------- bucketing
__global__ void k_fill32(uint32_t* p, uint32_t n, uint32_t v) {
  for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < n; j += gridDim.x * blockDim.x) p[j] = v;
}

// Bucket offsets.  Plain buckets come in 64 groups of kBucketsM (one group
// per (stages, classes), more stages first, then more classes), the
// interleaved buckets after them.  With `grouped` (a shared-layout call),
// the plain groups count plans, not pipelines: a group of G classes then
// takes ceil(plans / plans_per_wave(G)) whole wavefronts of lanes, its
// buckets' cursors count plans from the group's start, and sbase[group] is
// the group's first lane.  Otherwise (per-class layout) they count pipelines
// and their cursors are lanes.  sstart[16 - S] = first lane of
// the S-stage pipelines, sstart[16 + q] = first lane of interleaved group q,
// sstart[16 + kIlGroups] = all lanes.  Thread tid takes plain buckets
// [8 tid, 8 tid + 8) (sixteen threads per group) and interleaved bucket
// kPlainBuckets + tid; one block scan of (plain, interleaved) pairs, then one
// of the 64 groups' lane counts.
__global__ void __launch_bounds__(1024) k_scan(const uint32_t* __restrict__ hist, uint32_t* __restrict__ cursor,
                                               uint32_t* __restrict__ sstart, uint32_t* __restrict__ sbase,
                                               uint32_t grouped, uint32_t* __restrict__ ids) {
  constexpr int kPer = kPlainBuckets / 1024;
  constexpr int kThreadsPerGroup = kBucketsM / kPer;
  static_assert(kPlainBuckets % 1024 == 0 && kBuckets - kPlainBuckets == 1024, "bucket count");
  static_assert(kThreadsPerGroup * kSuperBuckets == 1024, "sixteen threads per (stages, classes) group");
  __shared__ uint2 part[1024];
  __shared__ uint32_t lanes[kSuperBuckets + 1];
  uint32_t v[kPer], sum = 0;
  const uint32_t tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < kPer; ++j) { v[j] = hist[tid * kPer + j]; sum += v[j]; }
  const uint32_t vi = hist[kPlainBuckets + tid];
  part[tid] = make_uint2(sum, vi);
  __syncthreads();
  for (uint32_t off = 1; off < 1024; off <<= 1) {
    const uint2 x = tid >= off ? part[tid - off] : make_uint2(0, 0);
    __syncthreads();
    part[tid].x += x.x;
    part[tid].y += x.y;
    __syncthreads();
  }
  // the group of this thread's buckets, its entries before this thread's
  const uint32_t grp = tid / kThreadsPerGroup, g0 = grp * kThreadsPerGroup;
  const uint32_t before_grp = g0 ? part[g0 - 1].x : 0;
  const bool by_plan = grouped != 0;
  uint32_t ngrp = 0;
  if (tid < kSuperBuckets) {
    // lanes of group tid
    const uint32_t a = tid * kThreadsPerGroup;
    ngrp = part[a + kThreadsPerGroup - 1].x - (a ? part[a - 1].x : 0);
    const uint32_t pw = plans_per_wave(kMaxClasses - tid % kMaxClasses);
    lanes[tid] = grouped ? (ngrp + pw - 1) / pw * 64u : ngrp;
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t run = 0;
    for (uint32_t q = 0; q < kSuperBuckets; ++q) {
      const uint32_t x = lanes[q];
      lanes[q] = run;
      run += x;
    }
    lanes[kSuperBuckets] = run;
  }
  __syncthreads();
  if (tid < kSuperBuckets) sbase[tid] = lanes[tid];
  // a plan-sorted group's last wavefront, when partly filled: its lanes past
  // the plans hold no pipeline (k_scatter marks the unused lanes of the full ones)
  if (grouped && tid < kSuperBuckets) {
    const uint32_t G = kMaxClasses - tid % kMaxClasses, pw = plans_per_wave(G), r = ngrp % pw;
    const uint32_t w0 = lanes[tid] + ngrp / pw * 64u;
    if (r)
      for (uint32_t q = G * r; q < 64u; ++q) ids[w0 + q] = kNoSlot;
  }
  // pipelines of S stages start at group (16 - S) * 4 (four classes first)
  if (tid < kMaxStages) sstart[tid] = lanes[tid * kMaxClasses];
  uint32_t run = part[tid].x - sum - before_grp;
  if (!by_plan) run += lanes[grp];
#pragma unroll
  for (int j = 0; j < kPer; ++j) { cursor[tid * kPer + j] = run; run += v[j]; }
  const uint32_t irun = lanes[kSuperBuckets] + part[tid].y - vi;
  if (tid % kIlBucketsQ == 0 && tid / kIlBucketsQ <= (uint32_t)kIlGroups) sstart[kMaxStages + tid / kIlBucketsQ] = irun;
  cursor[kPlainBuckets + tid] = irun;
}

// Place every pipeline id at its bucket's next free lane.  A plain key of a
// grouped call sits on the plan's class-0 slot and stands for the whole plan: the plan's rank r in its
// group puts its G pipeline ids on lanes sbase[group] + 64 (r / P) + G (r % P)
// onward (P = plans_per_wave(G)); the lanes no plan fills are set to kNoSlot
// here (64 mod G per full wavefront) and by k_scan (a group's last one).
constexpr int kScatterPer = 64;
__global__ void __launch_bounds__(256) k_scatter(const uint16_t* __restrict__ keys, uint32_t nslots,
                                                 uint32_t* __restrict__ cursor, const uint32_t* __restrict__ sbase,
                                                 uint32_t grouped, uint32_t* __restrict__ ids) {
  constexpr int kPer = kScatterPer;
  __shared__ uint32_t lc[kBuckets];
  for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x) lc[j] = 0;
  __syncthreads();
  uint32_t key[kPer], rank[kPer];
  const uint32_t first = blockIdx.x * blockDim.x * kPer + threadIdx.x;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const uint32_t slot = first + j * blockDim.x;
    key[j] = 0xffffffffu;
    rank[j] = 0;
    if (slot < nslots) {
      const uint32_t k = keys[slot];
      if (k != kNoKey) {
        key[j] = k;
        rank[j] = atomicAdd(&lc[k], 1u);
      }
    }
  }
  __syncthreads();
  for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x)
    if (lc[j]) lc[j] = atomicAdd(&cursor[j], lc[j]);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    if (key[j] == 0xffffffffu) continue;
    const uint32_t slot = first + j * blockDim.x, pos = lc[key[j]] + rank[j];
    const uint32_t grp = key[j] / kBucketsM, G = kMaxClasses - grp % kMaxClasses;
    if (grouped && key[j] < kPlainBuckets) {
      const uint32_t pw = plans_per_wave(G), lane = sbase[grp] + pos / pw * 64u + pos % pw * G;
      for (uint32_t c = 0; c < G; ++c) ids[lane + c] = slot + c;
      // the wavefront's last plan marks the lanes that no plan fills (64 mod G)
      if (pos % pw == pw - 1)
        for (uint32_t q = G * pw; q < 64u; ++q) ids[lane - (pw - 1) * G + q] = kNoSlot;
    } else {
      ids[pos] = slot;
    }
  }
}

// ---------------------------------------------------------------- per-class layout: plan order
// k_plan_syncs walks each plan's layer segments, one plan per lane, so a
// wavefront lasts as long as its longest walk.  The valid plans are first
// counting-sorted by (classes, total stages over the classes), a close proxy
// for the number of segments (the union of the classes' cuts), into perm;
// pc as kPlanSortWords describes.  The key comes from the pipeline metadata
// k_prep wrote (S | G << 5 | ..., per class; zero past the classes and for
// invalid plans).
__device__ __forceinline__ uint32_t plan_key(uint4 m) {
  const uint32_t G = (m.x >> 5) & 7, st = (m.x & 31) + (m.y & 31) + (m.z & 31) + (m.w & 31);
  return (G - 1) * 64 + st - 1;
}
constexpr int kPlanPer = 8;   // plans per thread of the plan-order kernels
__global__ void __launch_bounds__(256) k_plan_hist(const uint4* __restrict__ meta, uint32_t n, uint32_t* __restrict__ pc) {
  __shared__ uint32_t lh[kPlanBuckets];
  lh[threadIdx.x] = 0;
  __syncthreads();
  for (int j = 0; j < kPlanPer; ++j) {
    const uint32_t i = (blockIdx.x * kPlanPer + j) * 256 + threadIdx.x;
    if (i >= n) break;
    const uint4 m = meta[i];
    if (m.x) atomicAdd(&lh[plan_key(m)], 1u);
  }
  __syncthreads();
  if (lh[threadIdx.x]) atomicAdd(&pc[threadIdx.x], lh[threadIdx.x]);
}
__global__ void __launch_bounds__(256) k_plan_scatter(const uint4* __restrict__ meta, uint32_t n,
                                                      uint32_t* __restrict__ pc, uint32_t* __restrict__ perm) {
  static_assert(kPlanBuckets == 256, "one bucket per thread");
  __shared__ uint32_t base[kPlanBuckets], lc[kPlanBuckets];
  const uint32_t b = threadIdx.x;
  base[b] = pc[b];
  lc[b] = 0;
  __syncthreads();
  for (uint32_t off = 1; off < kPlanBuckets; off <<= 1) {   // inclusive scan of the counts
    const uint32_t x = b >= off ? base[b - off] : 0;
    __syncthreads();
    base[b] += x;
    __syncthreads();
  }
  if (blockIdx.x == 0 && b == kPlanBuckets - 1) pc[2 * kPlanBuckets] = base[b];   // valid plans
  const uint32_t excl = base[b] - pc[b];
  __syncthreads();
  base[b] = excl;
  uint32_t key[kPlanPer], rank[kPlanPer];
  for (int j = 0; j < kPlanPer; ++j) {
    const uint32_t i = (blockIdx.x * kPlanPer + j) * 256 + threadIdx.x;
    key[j] = kNoSlot;
    if (i < n) {
      const uint4 m = meta[i];
      if (m.x) {
        key[j] = plan_key(m);
        rank[j] = atomicAdd(&lc[key[j]], 1u);
      }
    }
  }
  __syncthreads();
  if (lc[b]) lc[b] = atomicAdd(&pc[kPlanBuckets + b], lc[b]);
  __syncthreads();
  for (int j = 0; j < kPlanPer; ++j)
    if (key[j] != kNoSlot) perm[base[key[j]] + lc[key[j]] + rank[j]] = (blockIdx.x * kPlanPer + j) * 256 + threadIdx.x;
}

// ---------------------------------------------------------------- deferred lists
// Counting sort of the deferred lists by micro-batch count (bucket
// min(31, M / 16), largest first) into vlist, which the variant pass has
// finished with: the deferred pass then runs wavefronts of similar trip
// counts rather than waiting in every wavefront for its longest chain.
__device__ __forceinline__ uint32_t defer_bucket(const EvalBufs& e, uint32_t slot) {
  const uint32_t w = e.packed[slot >> 2].cls[slot & 3], reps = w & 0xffff, M = ((w >> 16) + reps - 1) / reps;
  const uint32_t b = M >> 4;
  return b < kSortBuckets - 1 ? b : kSortBuckets - 1;
}
// entry idx of the concatenated lists -> (list j, position k in it)
__device__ __forceinline__ bool defer_entry(const EvalBufs& e, uint32_t idx, uint32_t& j, uint32_t& k) {
  uint32_t before = 0;
  for (j = 0; j < (uint32_t)kMaxStages; ++j) {
    const uint32_t n = e.ctr[1 + j];
    if (idx < before + n) {
      k = idx - before;
      return true;
    }
    before += n;
  }
  return false;
}
__global__ void __launch_bounds__(256) k_defer_hist(EvalBufs e) {
  __shared__ uint32_t hs[kMaxStages * kSortBuckets];
  for (uint32_t i = threadIdx.x; i < kMaxStages * kSortBuckets; i += blockDim.x) hs[i] = 0;
  __syncthreads();
  uint32_t total = 0;
  for (uint32_t j = 0; j < (uint32_t)kMaxStages; ++j) total += e.ctr[1 + j];
  for (uint32_t idx = blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += gridDim.x * blockDim.x) {
    uint32_t j, k;
    if (!defer_entry(e, idx, j, k)) break;
    atomicAdd(&hs[j * kSortBuckets + defer_bucket(e, e.deferred[e.sstart[j] + k])], 1u);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < kMaxStages * kSortBuckets; i += blockDim.x)
    if (hs[i]) atomicAdd(&e.ctr[kSortCtr + i], hs[i]);
}
__global__ void __launch_bounds__(256) k_defer_sort(EvalBufs e) {
  constexpr uint32_t kN = kMaxStages * kSortBuckets;
  __shared__ uint32_t base[kN], lc[kN];
  if (threadIdx.x < (uint32_t)kMaxStages) {   // list j's buckets, largest micro-batch counts first
    uint32_t run = 0;
    for (int b = kSortBuckets - 1; b >= 0; --b) {
      base[threadIdx.x * kSortBuckets + b] = run;
      run += e.ctr[kSortCtr + threadIdx.x * kSortBuckets + b];
    }
  }
  uint32_t total = 0;
  for (uint32_t j = 0; j < (uint32_t)kMaxStages; ++j) total += e.ctr[1 + j];
  // one entry per thread per round; ranks within the block from LDS counters,
  // then one global cursor update per (round, bucket)
  for (uint32_t r0 = blockIdx.x * blockDim.x; r0 < total; r0 += gridDim.x * blockDim.x) {
    for (uint32_t i = threadIdx.x; i < kN; i += blockDim.x) lc[i] = 0;
    __syncthreads();
    uint32_t j = 0, k = 0, slot = 0, b = 0, rank = 0;
    const bool has = r0 + threadIdx.x < total && defer_entry(e, r0 + threadIdx.x, j, k);
    if (has) {
      slot = e.deferred[e.sstart[j] + k];
      b = j * kSortBuckets + defer_bucket(e, slot);
      rank = atomicAdd(&lc[b], 1u);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < kN; i += blockDim.x)
      if (lc[i]) lc[i] = atomicAdd(&e.ctr[kSortCtr + kN + i], lc[i]);
    __syncthreads();
    if (has) e.vlist[e.sstart[j] + base[b] + lc[b] + rank] = slot;
    __syncthreads();
  }
}

// ---------------------------------------------------------------- argmin
__global__ void k_best_init(sim_best* b) {
  b->time_ps = kInvalid;
  b->index = INT64_MAX;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o);
    v = w < v ? w : v;
  }
  return v;
}

__global__ void __launch_bounds__(256) k_min_time(const uint64_t* __restrict__ t, int64_t n, sim_best* b) {
  __shared__ uint64_t part[4];
  uint64_t v = kInvalid;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    v = t[i] < v ? t[i] : v;
  v = wave_min_u64(v);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) v = part[w] < v ? part[w] : v;
    if (v != kInvalid) atomicMin((unsigned long long*)&b->time_ps, (unsigned long long)v);
  }
}

__global__ void __launch_bounds__(256) k_min_index(const uint64_t* __restrict__ t, int64_t n, int64_t base,
                                                   sim_best* b) {
  __shared__ uint64_t part[4];
  const uint64_t best = b->time_ps;
  uint64_t v = kInvalid;
  if (best != kInvalid)
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
      if (t[i] == best) { v = (uint64_t)i; break; }
  v = wave_min_u64(v);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) v = part[w] < v ? part[w] : v;
    if (v != kInvalid) atomicMin((long long*)&b->index, (long long)(base + (int64_t)v));
  }
}

__global__ void k_best_fix(sim_best* b) {
  if (b->time_ps == kInvalid) b->index = -1;
}

__global__ void __launch_bounds__(256) k_best_reduce(const sim_best* __restrict__ in, int64_t n, sim_best* out) {
  __shared__ uint64_t tpart[4], ipart[4];
  uint64_t bt = kInvalid, bi = kInvalid;
  for (int64_t j = threadIdx.x; j < n; j += blockDim.x) {
    const uint64_t tt = in[j].time_ps;
    const int64_t ii = in[j].index;
    if (tt == kInvalid || ii < 0) continue;
    if (tt < bt || (tt == bt && (uint64_t)ii < bi)) { bt = tt; bi = (uint64_t)ii; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t t2 = __shfl_xor(bt, o), i2 = __shfl_xor(bi, o);
    if (t2 < bt || (t2 == bt && i2 < bi)) { bt = t2; bi = i2; }
  }
  if ((threadIdx.x & 63) == 0) { tpart[threadIdx.x >> 6] = bt; ipart[threadIdx.x >> 6] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (tpart[w] < bt || (tpart[w] == bt && ipart[w] < bi)) { bt = tpart[w]; bi = ipart[w]; }
    out->time_ps = bt;
    out->index = bt == kInvalid ? -1 : (int64_t)bi;
  }
}


// ---------------------------------------------------------------- launchers
static int blocks_for(int64_t n, int per) { return (int)((n + per - 1) / per); }

hipError_t launch_fill32(uint32_t* p, uint32_t n, uint32_t v, hipStream_t s) {
  k_fill32<<<blocks_for(n, 256) < 1024 ? blocks_for(n, 256) : 1024, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}
hipError_t launch_prep(const Tab& t, const sim_plans& p, int64_t n, uint64_t* out, PackedPlan* packed, uint4* pcut,
                       uint32_t* meta, uint32_t* hist, uint16_t* keys, hipStream_t s) {
  const int g = blocks_for(n, 256 * kPrepPerThread);
  if (p.chdr) k_prep<true><<<g, 256, 0, s>>>(t, p, n, out, packed, pcut, meta, hist, keys);
  else k_prep<false><<<g, 256, 0, s>>>(t, p, n, out, packed, pcut, meta, hist, keys);
  return hipGetLastError();
}
hipError_t launch_memory(const Tab& t, const sim_plans& p, int64_t n, uint64_t* out, hipStream_t s) {
  if (p.chdr) k_memory<true><<<blocks_for(n, 256), 256, 0, s>>>(t, p, n, out);
  else k_memory<false><<<blocks_for(n, 256), 256, 0, s>>>(t, p, n, out);
  return hipGetLastError();
}

// pc: the plan-order counters (zero on entry); perm: n words
hipError_t launch_plan_syncs(const Tab& t, const PackedPlan* packed, const uint4* pcut, const uint32_t* meta,
                             int64_t n, uint64_t* hdp, uint32_t* pc, uint32_t* perm, hipStream_t s) {
  const int go = blocks_for(n, 256 * kPlanPer);
  k_plan_hist<<<go, 256, 0, s>>>((const uint4*)meta, (uint32_t)n, pc);
  k_plan_scatter<<<go, 256, 0, s>>>((const uint4*)meta, (uint32_t)n, pc, perm);
  const int g = blocks_for(n, 256);
  const size_t lds = t.mode < 2 ? t.lds_bytes : 0;
  if (t.mode == 0) k_plan_syncs<0><<<g, 256, lds, s>>>(t, packed, pcut, perm, pc, n, hdp);
  else if (t.mode == 1) k_plan_syncs<1><<<g, 256, lds, s>>>(t, packed, pcut, perm, pc, n, hdp);
  else k_plan_syncs<2><<<g, 256, 0, s>>>(t, packed, pcut, perm, pc, n, hdp);
  return hipGetLastError();
}

hipError_t launch_stages(const Tab& t, const PackedPlan* packed, const uint4* pcut, const uint32_t* meta, int64_t n,
                         uint64_t* out_stage, hipStream_t s) {
  if (pcut) k_stages<true><<<blocks_for(n * 4, 256), 256, 0, s>>>(t, packed, pcut, meta, n, out_stage);
  else k_stages<false><<<blocks_for(n * 4, 256), 256, 0, s>>>(t, packed, pcut, meta, n, out_stage);
  return hipGetLastError();
}
hipError_t launch_scan(const uint32_t* hist, uint32_t* cursor, uint32_t* sstart, uint32_t* sbase, bool grouped,
                       uint32_t* ids, hipStream_t s) {
  k_scan<<<1, 1024, 0, s>>>(hist, cursor, sstart, sbase, grouped ? 1u : 0u, ids);
  return hipGetLastError();
}
hipError_t launch_scatter(const uint16_t* keys, uint32_t nslots, uint32_t* cursor, const uint32_t* sbase, bool grouped,
                          uint32_t* ids, hipStream_t s) {
  k_scatter<<<blocks_for(nslots, 256 * kScatterPer), 256, 0, s>>>(keys, nslots, cursor, sbase, grouped ? 1u : 0u, ids);
  return hipGetLastError();
}
// ---------------------------------------------------------------- node-rate probe
// Peak rate of the recurrence's schedule-node operation on this device:
// end = max(end, input + hop) + duration, in fp64 (add, max, add), over
// kProbeChains independent chains per lane so that issue, not latency,
// bounds it.  The result feeds roofline reports; it is not part of any
// evaluation.
constexpr int kProbeChains = 8;
__global__ void __launch_bounds__(256) k_node_probe(double* __restrict__ sink, int iters, double c, double d) {
  double a[kProbeChains];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) a[j] = (double)(i + j);
  for (int k = 0; k < iters; ++k) {
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j) a[j] = __builtin_fmax(a[j], a[(j + 1) % kProbeChains] + c) + d;
  }
  double t = 0;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) t += a[j];
  sink[i] = t;
}

hipError_t launch_node_probe(double* sink, int blocks, int iters, hipStream_t s) {
  k_node_probe<<<blocks, 256, 0, s>>>(sink, iters, 3.0, 1.0);
  return hipGetLastError();
}

// ---------------------------------------------------------------- evaluation passes
EvalBufs eval_bufs(const EvalArgs& a) {
  return {a.packed, (const uint4*)a.pcut, a.hdp, a.meta, a.ids, a.sstart, a.out, a.ctr,
          a.ctr + kEvalCounters + kPlanSortWords, a.deferred,
          a.vlist, (unsigned long long*)a.skipped_ops, a.dtab};
}

// Blocks of each evaluation kernel that fit the device at once.
int eval_grids(Tab* t) {
  int cus = 0, dev = 0;
  hipError_t r = hipGetDevice(&dev);
  if (r == hipSuccess) r = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (r != hipSuccess) return (int)r;
  const size_t lds = t->mode < 2 ? t->lds_bytes : 0;
  int nb[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0}, nbc[4] = {0, 0, 0, 0};
  if (t->mode == 0) r = occupancy_first_v<0>(nb, lds, 0);
  else if (t->mode == 1) r = occupancy_first_v<1>(nb, lds, 0);
  else r = occupancy_first_v<2>(nb, lds, 0);
  // the stage-placement cache of the first pass's long groups, where it costs no blocks
  if (r == hipSuccess) {
    if (t->mode == 0) r = occupancy_first_v<0>(nbc, lds, 3u);
    else if (t->mode == 1) r = occupancy_first_v<1>(nbc, lds, 3u);
    else r = occupancy_first_v<2>(nbc, lds, 3u);
  }
  t->bcache = 0;
  for (int i = 0; i < 2; ++i)
    if (nbc[i] == nb[i]) t->bcache |= 1u << i;
  if (r == hipSuccess) {
    if (t->mode == 0) r = occupancy_deferred_v<0>(nb + 4, lds);
    else if (t->mode == 1) r = occupancy_deferred_v<1>(nb + 4, lds);
    else r = occupancy_deferred_v<2>(nb + 4, lds);
  }
  if (r == hipSuccess) {
    if (t->mode == 0) r = occupancy_variant_v<0>(nb + 5, lds);
    else if (t->mode == 1) r = occupancy_variant_v<1>(nb + 5, lds);
    else r = occupancy_variant_v<2>(nb + 5, lds);
  }
  if (r != hipSuccess) return (int)r;
  for (int i = 0; i < 4; ++i) t->grid_eval[i] = (uint32_t)((nb[i] > 0 ? nb[i] : 1) * cus);
  t->grid_deferred = (uint32_t)((nb[4] > 0 ? nb[4] : 1) * cus);
  for (int i = 0; i < 4; ++i) t->grid_variant[i] = (uint32_t)((nb[5 + i] > 0 ? nb[5 + i] : 1) * cus);
  return 0;
}

// first pass of one stage-count group (g = 0..3) over a chunk
hipError_t launch_group(const Tab& t, const EvalArgs& a, uint32_t max_tasks, int g, hipStream_t s) {
  const bool het = a.pcut != nullptr;
  if (t.mode == 0) return het ? launch_group_v<0, true>(t, a, max_tasks, g, s) : launch_group_v<0, false>(t, a, max_tasks, g, s);
  if (t.mode == 1) return het ? launch_group_v<1, true>(t, a, max_tasks, g, s) : launch_group_v<1, false>(t, a, max_tasks, g, s);
  return het ? launch_group_v<2, true>(t, a, max_tasks, g, s) : launch_group_v<2, false>(t, a, max_tasks, g, s);
}

// variant pass of one stage-count group: the overlap and zero-bubble
// pipelines the group's first pass listed (none with the per-class layout)
hipError_t launch_variant(const Tab& t, const EvalArgs& a, int g, hipStream_t s) {
  if (a.pcut) return hipSuccess;
  if (t.mode == 0) return launch_variant_v<0>(t, a, g, s);
  if (t.mode == 1) return launch_variant_v<1>(t, a, g, s);
  return launch_variant_v<2>(t, a, g, s);
}

// first pass over a chunk: k_eval of each stage-count group, in order, then
// the variant passes
hipError_t launch_first(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s) {
  hipError_t r = hipSuccess;
  for (int g = 0; g < 4 && r == hipSuccess; ++g) r = launch_group(t, a, max_tasks, g, s);
  for (int g = 0; g < 4 && r == hipSuccess; ++g) r = launch_variant(t, a, g, s);
  return r;
}

// then the interleaved and the deferred pipelines, and the u64 redo of the
// overflowed ones
hipError_t launch_deferred(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s) {
  const bool het = a.pcut != nullptr;
  hipError_t r;
  {
    // the deferred lists, sorted by micro-batch count into vlist
    const EvalBufs e = eval_bufs(a);
    k_defer_hist<<<64, 256, 0, s>>>(e);
    k_defer_sort<<<64, 256, 0, s>>>(e);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  }
  if (t.mode == 0) r = het ? launch_deferred_v<0, true>(t, a, max_tasks, s) : launch_deferred_v<0, false>(t, a, max_tasks, s);
  else if (t.mode == 1) r = het ? launch_deferred_v<1, true>(t, a, max_tasks, s) : launch_deferred_v<1, false>(t, a, max_tasks, s);
  else r = het ? launch_deferred_v<2, true>(t, a, max_tasks, s) : launch_deferred_v<2, false>(t, a, max_tasks, s);
  if (r != hipSuccess) return r;
  const EvalBufs e = eval_bufs(a);
  if (het) k_redo_u64<true><<<32, 64, 0, s>>>(t, e);
  else k_redo_u64<false><<<32, 64, 0, s>>>(t, e);
  return hipGetLastError();
}

hipError_t launch_argmin(const uint64_t* t, int64_t n, int64_t base, sim_best* b, hipStream_t s) {
  int g = blocks_for(n, 256 * 8);
  g = g < 1 ? 1 : (g > 2048 ? 2048 : g);
  k_best_init<<<1, 1, 0, s>>>(b);
  if (n > 0) {
    k_min_time<<<g, 256, 0, s>>>(t, n, b);
    k_min_index<<<g, 256, 0, s>>>(t, n, base, b);
  }
  k_best_fix<<<1, 1, 0, s>>>(b);
  return hipGetLastError();
}
hipError_t launch_best_reduce(const sim_best* in, int64_t n, sim_best* out, hipStream_t s) {
  k_best_reduce<<<1, 256, 0, s>>>(in, n, out);
  return hipGetLastError();
}

}  // namespace hetsim

