// device.h -- device code of the plan evaluator, shared by the library's
// translation units (kernels.hip and the evaluation-pass variants).
//
// Data flow of one chunk of plans (all in HBM):
//   k_prep     one plan per lane: decode and check the plan, pack it into 80
//              contiguous bytes, and count it per bucket: in the shared
//              layout the whole plan by (stages, classes, longest
//              micro-batch count), otherwise each pipeline (one per replica
//              class) by its own.
//   k_scan     one block: bucket offsets, longest pipelines first; a
//              plan-sorted (stages, classes) group takes whole wavefronts.
//   k_scatter  places the ids: a plan-sorted plan's G pipelines on adjacent
//              lanes of one wavefront, so that a wavefront runs one stage
//              count, one class count and similar micro-batch counts.
//   k_plan_hist, k_plan_scatter, k_plan_syncs (per-class layout only) the
//              syncs of every (class, stage), once per plan, plans sorted by
//              the length of their segment walks.
//   k_eval     one pipeline per lane, one launch per group of four stage
//              counts.  Overlap and zero-bubble plans are handed to the
//              variant pass first.  Setup: place the class on its device
//              pools, read stage compute from the layer prefix tables, find
//              each group's slowest link with range-max tables, and cost the
//              TP/EP/PP collectives.  Then the 1F1B recurrence, unrolled per
//              stage count so that all per-stage state stays in VGPRs; times
//              are integers carried exactly in fp64 (3 VALU ops per schedule
//              node).  Once a steady iteration advances the whole schedule
//              state by one constant, the remaining steady iterations are
//              added in one step (periodic shortcut); lanes still aperiodic
//              after a fixed budget are deferred.  Then the DP syncs, shared
//              over a plan's lanes, and one store of the plan's time.
//   k_variant  the overlap and zero-bubble plans of each group, the same way.
//   k_defer_hist, k_defer_sort  the deferred lists sorted by micro-batch count.
//   k_deferred the interleaved-1F1B pipelines, then the deferred pipelines of
//              all stage counts (full steady loop).
//   k_redo_u64 pipelines whose time reached 2^53 ps, again in u64.
//              Later passes raise a plan's time with atomic max.
#pragma once
#include <hip/hip_runtime.h>

#include <type_traits>

#include "internal.h"

namespace hetsim {

constexpr uint64_t kInvalid = ~0ull;

// ---------------------------------------------------------------- helpers
// ceil(bytes * bq / 2^16) with bytes < 2^48 and bq < 2^32 (80-bit product)
__device__ __forceinline__ uint64_t link_ps(uint64_t bytes, uint32_t bq) {
  uint64_t lo = bytes * (uint64_t)bq;
  uint64_t hi = __umul64hi(bytes, (uint64_t)bq);
  return ((hi << 48) | (lo >> 16)) + ((lo & 0xffffull) != 0);
}

// max over [lo, hi] of a range-max table with row length n
__device__ __forceinline__ uint32_t range_max(const uint32_t* __restrict__ tb, uint32_t n, uint32_t lo, uint32_t hi) {
  uint32_t j = 31u - __clz(hi - lo + 1);
  uint32_t a = tb[j * n + lo], b = tb[j * n + hi + 1 - (1u << j)];
  return a > b ? a : b;
}

// number of the nibbles selected by `sel` that equal k
__device__ __forceinline__ uint32_t count_type(uint64_t types, uint32_t k, uint64_t sel) {
  const uint64_t ones = 0x1111111111111111ull;
  uint64_t x = types ^ (ones * k);
  uint64_t nz = (x | (x >> 1) | (x >> 2) | (x >> 3)) & ones;
  return (uint32_t)__popcll(~nz & ones & sel);
}

// ceil(x / p) for x < 2^53 and p >= 1, given rp = RN(1/p): the rounded
// product is within 1 of x/p, so one correction each way makes it exact
// (two are applied).
__device__ __forceinline__ uint64_t div_up(uint64_t x, uint64_t p, double rp) {
  uint64_t q = (uint64_t)((double)x * rp);
  int64_t r = (int64_t)(x - q * p);
  const int64_t ps = (int64_t)p;
  if (r < 0) { --q; r += ps; }
  if (r < 0) { --q; r += ps; }
  if (r >= ps) { ++q; r -= ps; }
  if (r >= ps) { ++q; r -= ps; }
  return q + (r != 0);
}

// ceil(x / p) for any x: div_up below 2^53, the integer division above
// (never on the workloads here; a branch the wavefront skips when no lane
// takes it)
__device__ __forceinline__ uint64_t div_up_u64(uint64_t x, uint64_t p, double rp) {
  if (x < (1ull << 53)) return div_up(x, p, rp);
  return x / p + (x % p != 0);
}

// DP gradient sync of one stage over a ring of p members.  tree: an
// all-reduce takes the faster of the ring and a pipelined binary tree
// (reduce up, broadcast down: 2 ceil(log2 p) latencies, each member's
// gradient twice over the slowest link); ZeRO's reduce-scatter and
// all-gather stay rings.
__device__ __forceinline__ uint64_t ring_sync(uint32_t p, double rp, uint32_t zero, uint64_t grads, uint64_t params,
                                              uint64_t alpha, uint32_t bq, uint32_t tree) {
  uint64_t g = div_up(grads, p, rp);
  if (!zero) {
    uint64_t steps = 2ull * (p - 1);
    uint64_t r = steps * alpha + link_ps(steps * g, bq);
    if (tree && p > 1) {
      const uint64_t lg = 32 - __builtin_clz(p - 1);
      const uint64_t tt = 2 * lg * alpha + link_ps(2 * grads, bq);
      r = tt < r ? tt : r;
    }
    return r;
  }
  uint64_t steps = p - 1;
  return 2 * steps * alpha + link_ps(steps * g, bq) + link_ps(steps * div_up(params, p, rp), bq);
}

// The same sync as latency steps and link time (the part that concurrent
// syncs over the same links share); the tree only when strictly faster.
__device__ __forceinline__ void ring_parts(uint32_t p, double rp, uint32_t zero, uint64_t grads, uint64_t params,
                                           uint64_t alpha, uint32_t bq, uint32_t tree, uint64_t& lat, uint64_t& bw) {
  const uint64_t g = div_up(grads, p, rp);
  lat = 2ull * (p - 1) * alpha;
  if (!zero) {
    bw = link_ps(2ull * (p - 1) * g, bq);
    if (tree && p > 1) {
      const uint64_t lg = 32 - __builtin_clz(p - 1);
      const uint64_t tl = 2 * lg * alpha, tb = link_ps(2 * grads, bq);
      if (tl + tb < lat + bw) {
        lat = tl;
        bw = tb;
      }
    }
  } else {
    const uint64_t steps = p - 1;
    bw = link_ps(steps * g, bq) + link_ps(steps * div_up(params, p, rp), bq);
  }
}

// micro-batch counts: exact up to 64, then steps of 16 up to 1088
__device__ __forceinline__ uint32_t m_bucket(uint32_t M) {
  if (M <= 64) return M - 1;
  const uint32_t b = 64 + (M - 65) / 16;
  return b < kBucketsM - 1 ? b : kBucketsM - 1;
}
// ascending key: more stages first, then more classes, then more micro-batches
__device__ __forceinline__ uint32_t bucket_key(uint32_t S, uint32_t G, uint32_t M) {
  return ((kMaxStages - S) * kMaxClasses + (kMaxClasses - G)) * kBucketsM + (kBucketsM - 1 - m_bucket(M));
}
// interleaved pipelines: after all others, one group per (S, v), more
// micro-batches first (q = M / S exact from 2 to 49).  M is a multiple of S
// below 2^16, so M times the approximate reciprocal of S rounds to q.
__device__ __forceinline__ uint32_t il_group(uint32_t S, uint32_t v) { return (S - 2) * 3 + (v - 2); }
__device__ __forceinline__ uint32_t il_key(uint32_t S, uint32_t v, uint32_t M) {
  const uint32_t q = (uint32_t)((float)M * __builtin_amdgcn_rcpf((float)S) + 0.5f) - 2;
  return kPlainBuckets + il_group(S, v) * kIlBucketsQ + (kIlBucketsQ - 1 - (q < kIlBucketsQ - 1 ? q : kIlBucketsQ - 1));
}
// (S, v) shapes of interleaved pipelines: S v <= 16 virtual stages
#define HETSIM_IL_SHAPES(X) \
  X(2, 2) X(2, 3) X(2, 4) X(3, 2) X(3, 3) X(3, 4) X(4, 2) X(4, 3) X(4, 4) X(5, 2) X(5, 3) X(6, 2) X(7, 2) X(8, 2)

// pipeline metadata word: S | G << 5 | M << 8 | (v - 1) << 24 (0 = no pipeline);
// bucket keys travel as u16, kNoKey = no pipeline
constexpr uint32_t kNoKey = 0xffff;
static_assert(kBuckets < kNoKey, "bucket keys fit 16 bits");

// ---------------------------------------------------------------- plan validation
// Decoded plan fields used by every pipeline of the plan.
struct Plan {
  uint32_t tpl, epl, S, G, zero, mi, tp, ep, psum;
  uint32_t overlap;         // gradient sync overlapped with the last backward pass
  uint32_t v;               // model chunks per device: 1, or 2..4 for interleaved 1F1B
  uint32_t zb;              // zero-bubble order: backward split into input and weight gradients
  uint64_t cut_lo, cut_hi;  // cut bytes of stages 0-7 and 8-15, eight per word (virtual stages when v > 1)
  uint32_t reps[4], nmb[4];
  uint64_t tv[4];           // stage types, nibbles past S cleared
  // the class a pipeline evaluates: index, replicas, micro-batches, types.
  // Read here, from the packed plan in memory, so that no per-lane class
  // index ever selects among the fields above (that would put them in
  // private memory).
  uint32_t c, rc, nc;
  uint64_t tc;
  // per-class layout: byte c = log2 TP | (PP - 1) << 2 | micro-batch size
  // index << 6 of class c (0 with the shared layout, where tpl, S, mi and
  // the cuts above hold for every class; with the per-class layout they are
  // the pipeline's own class's)
  uint32_t chdr;
};

__device__ __forceinline__ uint32_t cls_tpl(uint32_t chdr, uint32_t c) { return (chdr >> (8 * c)) & 3; }
__device__ __forceinline__ uint32_t cls_S(uint32_t chdr, uint32_t c) { return ((chdr >> (8 * c + 2)) & 15) + 1; }
__device__ __forceinline__ uint32_t cls_mi(uint32_t chdr, uint32_t c) { return (chdr >> (8 * c + 6)) & 3; }
__device__ __forceinline__ uint64_t stage_sel(uint32_t S) { return S == 16 ? ~0ull : ((1ull << (4 * S)) - 1); }

// cut of stage s (a run-time index): mask arithmetic rather than a select,
// which the compiler may turn into an indexed load of the plan in private
// memory
__device__ __forceinline__ uint32_t cut_at(const Plan& p, uint32_t s) {
  const uint64_t m = 0ull - (uint64_t)(s >> 3);
  const uint64_t w = (p.cut_lo & ~m) | (p.cut_hi & m);
  return (uint32_t)(w >> (8 * (s & 7))) & 0xff;
}

__device__ __forceinline__ Plan unpack(const PackedPlan& q, uint32_t c = 0) {
  Plan p;
  p.c = c;
  const uint32_t cc = q.cls[c];
  p.rc = cc & 0xffff;
  p.nc = cc >> 16;
  p.tc = q.types[c];
  const uint32_t hdr = q.hdr;
  p.tpl = hdr & 3; p.epl = (hdr >> 2) & 3; p.S = ((hdr >> 4) & 15) + 1; p.G = ((hdr >> 8) & 3) + 1;
  p.zero = (hdr >> 10) & 1; p.mi = (hdr >> 11) & 3; p.tp = 1u << p.tpl; p.ep = 1u << p.epl; p.psum = q.psum;
  p.overlap = (hdr >> 13) & 1;
  p.v = ((hdr >> 14) & 3) + 1;
  p.zb = (hdr >> 16) & 1;
  p.chdr = q.pad0;
  const uint64_t* cw = reinterpret_cast<const uint64_t*>(q.cut);
  p.cut_lo = cw[0];
  p.cut_hi = cw[1];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    p.reps[j] = q.cls[j] & 0xffff;
    p.nmb[j] = q.cls[j] >> 16;
    p.tv[j] = q.types[j];
  }
  return p;
}

// The plan of pipeline `slot` (plan slot / 4, class slot % 4).  With the
// per-class layout the own class's TP degree, depth and cuts replace the
// header's; its cut row is row `slot` of the per-class cut array.
template <bool kHet>
__device__ __forceinline__ Plan load_plan(const PackedPlan* packed, const uint4* pcut, uint32_t slot) {
  Plan p = unpack(packed[slot >> 2], slot & 3);
  if (kHet) {
    p.tpl = cls_tpl(p.chdr, p.c);
    p.tp = 1u << p.tpl;
    p.S = cls_S(p.chdr, p.c);
    p.mi = cls_mi(p.chdr, p.c);
    const uint4 r = pcut[slot];
    p.cut_lo = (uint64_t)r.y << 32 | r.x;
    p.cut_hi = (uint64_t)r.w << 32 | r.z;
  }
  return p;
}

// micro-batches per replica of the pipeline's class (its M)
__device__ __forceinline__ uint32_t class_mb(const Plan& p) { return (p.nc + p.rc - 1) / p.rc; }

constexpr int kPrepPerThread = 4;

// Plan i as loaded and checked by one lane: every rule of the plan layout
// except the memory check.  Per-class quantities are kept per class; with
// the shared layout every class has the header's.
struct Checked {
  bool ok;
  uint32_t hdr, psum, chdr;
  uint32_t tpl[4], S[4];   // per class (devices per replica)
  uint32_t v;              // model chunks per device (interleaved 1F1B when > 1)
  uint32_t cw[4][4];       // per class: cut bytes, four per word, 0 past the class's (virtual) stages
  uint32_t cls[4];         // 0 past the class count
  uint64_t tv[4];          // stage types, nibbles past the class's stages cleared; 0 past the class count
};

template <bool kHet>
__device__ __forceinline__ Checked check_plan(const Tab& t, const sim_plans& pl, int64_t i) {
  Checked r;
  const int64_t st = pl.stride;
  // every plane exists: load before any use
  const uint32_t hdr = pl.hdr[i];
  uint32_t cb[kHet ? 64 : 16];
#pragma unroll
  for (int s = 0; s < (kHet ? 64 : 16); ++s) cb[s] = kHet ? pl.ccut[s * st + i] : pl.cut[s * st + i];
  const uint32_t chdr = kHet ? pl.chdr[i] : 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    r.cls[c] = pl.cls[c * st + i];
    r.tv[c] = pl.types[c * st + i];
  }
  const uint32_t epl = (hdr >> 2) & 3, G = ((hdr >> 8) & 3) + 1, mi = (hdr >> 11) & 3;
  const uint32_t ep = 1u << epl, v = ((hdr >> 14) & 3) + 1;
  bool ok = (hdr >> 17) == 0 && mi < t.n_mbs && ((t.ep_ok >> epl) & 1);
  // the per-class layout leaves the header's TP and PP fields unused (0) and
  // has no overlap, interleaving or zero-bubble order
  if (kHet) ok = ok && (hdr & 0x1f8f3) == 0;   // and its micro-batch size: every class has its own
  // the zero-bubble order goes with neither overlap nor interleaving
  if (!kHet && ((hdr >> 16) & 1)) ok = ok && (hdr & 0xe000) == 0;
  // interleaving: no overlap, at least two devices, at most 16 virtual stages
  if (!kHet && v > 1) {
    const uint32_t S0 = ((hdr >> 4) & 15) + 1;
    ok = ok && ((hdr >> 13) & 1) == 0 && S0 >= 2 && S0 * v <= (uint32_t)kMaxStages;
  }
  uint32_t batch = 0, psum = 0;
#pragma unroll
  for (uint32_t c = 0; c < 4; ++c) {
    const uint32_t lay = kHet ? (chdr >> (8 * c)) & 0xff : (hdr & 3) | (((hdr >> 4) & 15) << 2);
    const uint32_t tpl = lay & 3, S = ((lay >> 2) & 15) + 1;
    r.tpl[c] = tpl;
    r.S[c] = S;
#pragma unroll
    for (int j = 0; j < 4; ++j) r.cw[c][j] = 0;
    if (c < G) {
      const uint32_t mic = kHet ? lay >> 6 : mi;   // the class's micro-batch size index
      if (kHet) ok = ok && mic < t.n_mbs;
      if (kHet || c == 0) {   // the shared layout's cuts are checked once
        ok = ok && ((t.tp_ok >> tpl) & 1);
        const uint32_t ncut = kHet ? S : S * v;
        uint32_t prev = 0;
#pragma unroll
        for (uint32_t s = 0; s < 16; ++s) {
          if (s < ncut) {
            const uint32_t v = cb[(kHet ? 16 * c : 0) + s];
            ok = ok && v > prev;
            prev = v;
            r.cw[c][s >> 2] |= v << (8 * (s & 3));
          }
        }
        ok = ok && prev == t.L;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) r.cw[c][j] = r.cw[0][j];
      }
      r.tv[c] &= stage_sel(S);
      const uint32_t reps = r.cls[c] & 0xffff, nmb = r.cls[c] >> 16;
      ok = ok && reps >= 1 && nmb >= reps && (reps & (ep - 1)) == 0;
      if (!kHet && v > 1 && ok) {   // interleaving: M a multiple of S and at least 2 S
        const uint32_t M = (nmb + reps - 1) / reps;
        ok = M % S == 0 && M >= 2 * S;
      }
      batch += nmb * t.mbs[mic];
      psum += reps;
      // every stage's type exists and holds whole TP groups in a node
      const uint32_t okm = t.type_ok[tpl];
      for (uint32_t s = 0; s < S; ++s) ok = ok && ((okm >> ((uint32_t)(r.tv[c] >> (4 * s)) & 15)) & 1);
    } else {
      r.cls[c] = 0;
      r.tv[c] = 0;
    }
  }
  ok = ok && batch == t.gbs;
  // capacity of every pool under the packing (blocks aligned to their TP degree)
  for (uint32_t k = 0; ok && k < t.K; ++k) {
    uint32_t need = 0;
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c) {
      const uint32_t nk = c < G ? count_type(r.tv[c], k, stage_sel(r.S[c])) : 0;
      if (nk) need = ((need + (1u << r.tpl[c]) - 1) >> r.tpl[c] << r.tpl[c]) + (((r.cls[c] & 0xffff) * nk) << r.tpl[c]);
    }
    ok = need <= t.cap[k];
  }
  r.ok = ok;
  r.hdr = hdr;
  r.psum = psum;
  r.chdr = chdr;
  r.v = kHet ? 1 : v;
  return r;
}

// Peak bytes of one device of a stage of ns layers at TP 2^tpl apart from
// its stored activations: weights and gradients of the parameters its TP
// rank holds, and the optimizer state, split with ZeRO over the DP group
// (all replicas for the non-expert parameters, replicas / EP for the
// experts).
__device__ __forceinline__ uint64_t state_bytes(const Tab& t, uint32_t tpl, uint32_t epl, uint32_t zero,
                                                uint32_t psum, bool first, bool last, uint32_t ns) {
  uint64_t pd = (uint64_t)ns * t.par_layer[tpl];
  if (first) pd += t.par_embed[tpl];
  if (last) pd += t.par_head[tpl];
  const uint64_t pe = (uint64_t)ns * t.par_expert[tpl][epl];
  uint64_t od = t.opt_bytes * pd, oe = t.opt_bytes * pe;
  if (zero) {
    const uint32_t pdx = psum >> epl;
    od = (od + psum - 1) / psum;
    oe = (oe + pdx - 1) / pdx;
  }
  return (t.param_bytes + t.grad_bytes) * (pd + pe) + od + oe;
}

// cut byte of stage s (run-time index) of class c (a compile-time index) of a checked plan
__device__ __forceinline__ uint32_t checked_cut(const Checked& r, uint32_t c, uint32_t s) {
  const uint64_t lo = (uint64_t)r.cw[c][0] | ((uint64_t)r.cw[c][1] << 32);
  const uint64_t hi = (uint64_t)r.cw[c][2] | ((uint64_t)r.cw[c][3] << 32);
  const uint64_t m = 0ull - (uint64_t)(s >> 3);
  return (uint32_t)(((lo & ~m) | (hi & m)) >> (8 * (s & 7))) & 0xff;
}

// State bytes of stage s (ns layers) of class c of a checked plan.
__device__ __forceinline__ uint64_t class_state_bytes(const Tab& t, const Checked& r, uint32_t c, uint32_t s,
                                                      uint32_t ns) {
  const uint32_t epl = (r.hdr >> 2) & 3, zero = (r.hdr >> 10) & 1;
  return state_bytes(t, r.tpl[c], epl, zero, r.psum, s == 0, s == r.S[c] - 1, ns);
}

// Peak bytes of the devices of stage s (ns layers) of class c: its state plus
// the activations of the min(PP - s, M) micro-batches 1F1B keeps in flight
// there (min(PP, M) on every stage under the zero-bubble order, where a
// micro-batch's activations stay until its weight-gradient pass).
__device__ __forceinline__ uint64_t class_stage_bytes(const Tab& t, const Checked& r, uint32_t c, uint32_t s,
                                                      uint32_t ns, uint64_t state) {
  // the micro-batch size: the header's (shared layout) or the class's (per-class layout, header field 0)
  const uint32_t mi = ((r.hdr >> 11) & 3) | cls_mi(r.chdr, c), S = r.S[c];
  const uint32_t reps = r.cls[c] & 0xffff, M = ((r.cls[c] >> 16) + reps - 1) / reps;
  const uint32_t held = ((r.hdr >> 16) & 1) ? S : S - s;
  const uint32_t fly = held < M ? held : M;
  return state + (uint64_t)ns * fly * t.act_layer[r.tpl[c]][mi];
}

// Interleaved 1F1B: device s holds virtual stages j S + s (j < v), so its
// state covers the layers of all of them (ns; the embedding on device 0, the
// head on device S - 1), and its activations are those of its
// 2 (S - 1 - s) + (v - 1) S warm-up passes plus one (at most M v passes),
// each counted at the device's largest chunk (nmax layers).
__device__ __forceinline__ void il_device_layers(const Checked& r, uint32_t s, uint32_t& ns, uint32_t& nmax) {
  const uint32_t S = r.S[0];
  ns = 0;
  nmax = 0;
  for (uint32_t j = 0; j < r.v; ++j) {
    const uint32_t vs = j * S + s;
    const uint32_t n = checked_cut(r, 0, vs) - (vs ? checked_cut(r, 0, vs - 1) : 0);
    ns += n;
    nmax = n > nmax ? n : nmax;
  }
}
__device__ __forceinline__ uint64_t il_stage_bytes(const Tab& t, const Checked& r, uint32_t c, uint32_t s,
                                                   uint32_t nmax, uint64_t state) {
  const uint32_t mi = (r.hdr >> 11) & 3, S = r.S[c], v = r.v;
  const uint32_t reps = r.cls[c] & 0xffff, M = ((r.cls[c] >> 16) + reps - 1) / reps;
  const uint32_t w = 2 * (S - 1 - s) + (v - 1) * S + 1;
  const uint32_t fly = w < M * v ? w : M * v;
  return state + (uint64_t)nmax * fly * t.act_layer[r.tpl[c]][mi];
}

// Every device of a checked plan fits its type's memory.  With one layout
// for all classes a stage's state is the same for every class: computed once.
template <bool kHet>
__device__ __forceinline__ bool fits_memory(const Tab& t, const Checked& r) {
  const uint32_t G = ((r.hdr >> 8) & 3) + 1;
  bool ok = true;
  if (!kHet && r.v > 1) {
    for (uint32_t s = 0; s < r.S[0]; ++s) {
      uint32_t ns, nmax;
      il_device_layers(r, s, ns, nmax);
      const uint64_t state = class_state_bytes(t, r, 0, s, ns);
#pragma unroll
      for (uint32_t c = 0; c < 4; ++c)
        if (c < G)
          ok = ok && il_stage_bytes(t, r, c, s, nmax, state) <= t.mem_cap[(uint32_t)(r.tv[c] >> (4 * s)) & 15];
    }
    return ok;
  }
  if (!kHet) {
    uint32_t prev = 0;
    for (uint32_t s = 0; s < r.S[0]; ++s) {
      const uint32_t cut = checked_cut(r, 0, s), ns = cut - prev;
      prev = cut;
      const uint64_t state = class_state_bytes(t, r, 0, s, ns);
#pragma unroll
      for (uint32_t c = 0; c < 4; ++c)
        if (c < G)
          ok = ok && class_stage_bytes(t, r, c, s, ns, state) <= t.mem_cap[(uint32_t)(r.tv[c] >> (4 * s)) & 15];
    }
    return ok;
  }
#pragma unroll
  for (uint32_t c = 0; c < 4; ++c) {
    if (c >= G) continue;
    uint32_t prev = 0;
    for (uint32_t s = 0; s < r.S[c]; ++s) {
      const uint32_t cut = checked_cut(r, c, s), ns = cut - prev;
      prev = cut;
      const uint64_t v = class_stage_bytes(t, r, c, s, ns, class_state_bytes(t, r, c, s, ns));
      ok = ok && v <= t.mem_cap[(uint32_t)(r.tv[c] >> (4 * s)) & 15];
    }
  }
  return ok;
}

// Decode and check plan i (every rule of the plan layout); on success pack it
// (with the per-class layout, the class header word goes to pad0 and each
// class's cut row to pcut[4 i + c]).  Writes out[i] (0 = valid, to be raised
// by the pipelines; else invalid) and the per-pipeline metadata
// S | G << 5 | M << 8 | (v - 1) << 24 with the class's own S (0 = no pipeline),
// and (keys, when given) each pipeline's bucket (kNoKey = no pipeline); with
// keys, valid plans sorted by plan get no metadata.
template <bool kHet>
__global__ void __launch_bounds__(256) k_prep(Tab t, sim_plans pl, int64_t n, uint64_t* __restrict__ out,
                                              PackedPlan* __restrict__ packed, uint4* __restrict__ pcut,
                                              uint32_t* __restrict__ meta, uint32_t* __restrict__ hist,
                                              uint16_t* __restrict__ keys) {
  __shared__ uint32_t lh[kBuckets];
  if (hist) {
    for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x) lh[j] = 0;
    __syncthreads();
  }
  for (int rep = 0; rep < kPrepPerThread; ++rep) {
    const int64_t i = ((int64_t)blockIdx.x * kPrepPerThread + rep) * blockDim.x + threadIdx.x;
    if (i >= n) break;
    const Checked r = check_plan<kHet>(t, pl, i);
    const bool ok = r.ok && (!t.mem_check || fits_memory<kHet>(t, r));
    const uint32_t G = ((r.hdr >> 8) & 3) + 1;
    if (out) out[i] = ok ? 0 : kInvalid;
    if (ok) {
      PackedPlan q;
      q.hdr = r.hdr; q.psum = r.psum; q.pad0 = r.chdr; q.pad1 = 0;
      uint32_t* qc = reinterpret_cast<uint32_t*>(q.cut);
#pragma unroll
      for (int j = 0; j < 4; ++j) { qc[j] = r.cw[0][j]; q.cls[j] = r.cls[j]; q.types[j] = r.tv[j]; }
      packed[i] = q;
      if (kHet) {
#pragma unroll
        for (int c = 0; c < 4; ++c) pcut[4 * i + c] = make_uint4(r.cw[c][0], r.cw[c][1], r.cw[c][2], r.cw[c][3]);
      }
    }
    uint32_t m[4], key[4], Mmax = 0;
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c) {
      m[c] = 0;
      key[c] = kNoKey;
      if (ok && c < G) {
        const uint32_t reps = r.cls[c] & 0xffff, M = ((r.cls[c] >> 16) + reps - 1) / reps;
        m[c] = r.S[c] | (G << 5) | (M << 8) | ((r.v - 1) << 24);
        Mmax = M > Mmax ? M : Mmax;
      }
    }
    // plans sorted by plan (their class 0 carries the key, ranked by the
    // longest class), the others by pipeline
    const bool by_plan = !kHet && ok && r.v == 1;
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c) {
      if (ok && c < G && (!by_plan || c == 0)) {
        const uint32_t M = by_plan ? Mmax : m[c] >> 8 & 0xffff;
        key[c] = r.v > 1 ? il_key(r.S[c], r.v, M) : bucket_key(r.S[c], G, M);
        if (hist) atomicAdd(&lh[key[c]], 1u);
      }
    }
    // one 16-byte and one 8-byte store per plan (the workspace is 256-byte
    // aligned; a caller's class array may be aligned to 4 bytes only).  An
    // evaluation call (keys given) reads no metadata of the plans it sorts by
    // plan: only its other pipelines get it
    if (!keys || !by_plan) {
      if (((uintptr_t)meta & 15) == 0) {
        reinterpret_cast<uint4*>(meta)[i] = make_uint4(m[0], m[1], m[2], m[3]);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) meta[i * 4 + c] = m[c];
      }
    }
    if (keys) reinterpret_cast<uint2*>(keys)[i] = make_uint2(key[0] | key[1] << 16, key[2] | key[3] << 16);
  }
  if (hist) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x)
      if (lh[j]) atomicAdd(&hist[j], lh[j]);
  }
}

// Peak memory of every (class, stage) device of plan i (one plan per lane).
template <bool kHet>
__global__ void __launch_bounds__(256) k_memory(Tab t, sim_plans pl, int64_t n, uint64_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const Checked r = check_plan<kHet>(t, pl, i);
  const uint32_t G = ((r.hdr >> 8) & 3) + 1;
  uint64_t* o = out + i * (kMaxClasses * kMaxStages);
#pragma unroll
  for (uint32_t c = 0; c < 4; ++c) {
    uint32_t prev = 0;
    for (uint32_t s = 0; s < (uint32_t)kMaxStages; ++s) {
      uint64_t v = kInvalid;
      if (r.ok) {
        v = 0;
        if (c < G && s < r.S[c] && r.v > 1) {
          uint32_t ns, nmax;
          il_device_layers(r, s, ns, nmax);
          v = il_stage_bytes(t, r, c, s, nmax, class_state_bytes(t, r, c, s, ns));
        } else if (c < G && s < r.S[c]) {
          const uint32_t cut = checked_cut(r, c, s);
          v = class_stage_bytes(t, r, c, s, cut - prev, class_state_bytes(t, r, c, s, cut - prev));
          prev = cut;
        }
      }
      o[c * kMaxStages + s] = v;
    }
  }
}

// ---------------------------------------------------------------- table image
// Reads of the setup tables (the image described with Tab).  kMode 0: the
// whole image is in LDS; 1: all but the device range-max rows; 2: all in
// device memory.
template <int kMode>
struct Hot {
  const uint8_t* b;       // image base for every section but the device rows
  const uint32_t* rmn;    // device range-max rows
  const Tab& t;
  __device__ __forceinline__ Hot(const Tab& tab, const uint4* lds)
      : b(kMode < 2 ? (const uint8_t*)lds : (const uint8_t*)tab.img),
        rmn((const uint32_t*)((kMode == 0 ? (const uint8_t*)lds : (const uint8_t*)tab.img) + tab.o_rmn)),
        t(tab) {}
  __device__ __forceinline__ TypeInfo type(uint32_t k) const {
    const uint4* q = (const uint4*)(b + k * sizeof(TypeInfo));
    const uint4 x = q[0], y = q[1];
    TypeInfo r;
    r.node_off = x.x; r.dev_off = x.y; r.dpl = x.z; r.bq_pcie = x.w;
    r.a_intra = (uint64_t)y.y << 32 | y.x;
    r.a_side = (uint64_t)y.w << 32 | y.z;
    return r;
  }
  // {forward, backward} prefix entry
  __device__ __forceinline__ ulonglong2 pfb(uint32_t i) const { return ((const ulonglong2*)(b + t.o_pfb))[i]; }
  __device__ __forceinline__ ulonglong2 emb(uint32_t i) const { return ((const ulonglong2*)(b + t.o_emb))[i]; }
  __device__ __forceinline__ ulonglong2 head(uint32_t i) const { return ((const ulonglong2*)(b + t.o_head))[i]; }
  __device__ __forceinline__ uint64_t pa(uint32_t i) const { return ((const uint64_t*)(b + t.o_pa))[i]; }
  __device__ __forceinline__ const uint32_t* rmi() const { return (const uint32_t*)(b + t.o_rmi); }
};

// Copy the LDS part of the image (every thread of the block takes part).
template <int kMode>
__device__ __forceinline__ void fill_lds(const Tab& t, uint4* lds) {
  if (kMode < 2) {
    const uint32_t n = t.lds_bytes >> 4;
    const uint4* img = (const uint4*)t.img;
    for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) lds[i] = img[i];
    __syncthreads();
  }
}

// ---------------------------------------------------------------- per-pipeline setup
// Stage quantities of class c of a valid plan: rec[s] = {forward and backward
// time of one micro-batch on stage s, hop s -> s+1, DP sync of stage s}.
//
// Placement: every pool is filled in (class, stage) order, reps*tp devices per
// (class, stage), so a (class, stage) of type k starts after the devices of
// type k used by earlier classes and by earlier stages of its own class.
// Devices of type k taken before (class c2, stage s) for a class index c2
// that is a compile-time constant once the callers' class loops unroll.
__device__ __forceinline__ uint32_t placed_before(const Plan& p, uint32_t c2, uint32_t s, uint32_t k) {
  const uint64_t sel = p.S == 16 ? ~0ull : ((1ull << (4 * p.S)) - 1);
  uint32_t below = 0;
#pragma unroll
  for (uint32_t c3 = 0; c3 < 4; ++c3)
    if (c3 < c2) below += p.reps[c3] * count_type(p.tv[c3], k, sel);
  return below + p.reps[c2] * count_type(p.tv[c2], k, (1ull << (4 * s)) - 1);
}

// The same for the pipeline's own class (a per-lane index).
__device__ __forceinline__ uint32_t placed_before_own(const Plan& p, uint32_t s, uint32_t k) {
  const uint64_t sel = p.S == 16 ? ~0ull : ((1ull << (4 * p.S)) - 1);
  uint32_t below = 0;
#pragma unroll
  for (uint32_t c3 = 0; c3 < 4; ++c3)
    if (c3 < p.c) below += p.reps[c3] * count_type(p.tv[c3], k, sel);
  return below + p.rc * count_type(p.tc, k, (1ull << (4 * s)) - 1);
}

// Devices of type k taken before (class c2, stage s), and the same for the
// pipeline's own class, under either layout.  With the per-class layout each
// class takes reps * its own TP degree devices per stage, and its blocks
// start at a multiple of that degree (so no TP group spans two nodes): a
// class's blocks in a pool are contiguous after its first one is aligned.
__device__ __forceinline__ uint32_t align_up(uint32_t x, uint32_t tpl) { return ((x + (1u << tpl) - 1) >> tpl) << tpl; }

template <bool kHet>
__device__ __forceinline__ uint32_t dev_before(const Plan& p, uint32_t c2, uint32_t s, uint32_t k) {
  if (!kHet) return placed_before(p, c2, s, k) * p.tp;
  uint32_t ptr = 0;
#pragma unroll
  for (uint32_t c3 = 0; c3 < 4; ++c3) {
    if (c3 < c2) {
      const uint32_t tl = cls_tpl(p.chdr, c3), nk = count_type(p.tv[c3], k, stage_sel(cls_S(p.chdr, c3)));
      if (nk) ptr = align_up(ptr, tl) + ((p.reps[c3] * nk) << tl);
    }
  }
  const uint32_t tl = cls_tpl(p.chdr, c2);
  return align_up(ptr, tl) + ((p.reps[c2] * count_type(p.tv[c2], k, (1ull << (4 * s)) - 1)) << tl);
}
template <bool kHet>
__device__ __forceinline__ uint32_t dev_before_own(const Plan& p, uint32_t s, uint32_t k) {
  if (!kHet) return placed_before_own(p, s, k) * p.tp;
  uint32_t ptr = 0;
#pragma unroll
  for (uint32_t c3 = 0; c3 < 4; ++c3) {
    if (c3 < p.c) {
      const uint32_t tl = cls_tpl(p.chdr, c3), nk = count_type(p.tv[c3], k, stage_sel(cls_S(p.chdr, c3)));
      if (nk) ptr = align_up(ptr, tl) + ((p.reps[c3] * nk) << tl);
    }
  }
  return align_up(ptr, p.tpl) + ((p.rc * count_type(p.tc, k, (1ull << (4 * s)) - 1)) << p.tpl);
}

// DP sync of stage s (layers [lo, hi), ns = hi - lo) over every replica of
// every class: one ring across all replicas on the slowest NIC of the
// participating devices, or inside one node when every replica of the stage
// sits in the same node; MoE models add the expert ring over the EP-sized
// groups.  The same for every class of the plan.
// With two-level collectives enabled, hs is the group's shape for them:
// usable when every class's devices of the stage fill whole nodes with the
// same number g > 1 of TP groups per node, over N > 1 nodes in all; a_in
// and bq_in are the worst node latency and fabric rate over them.
struct HierShape {
  bool ok;
  uint32_t g, N, bq_in;
  uint64_t a_in;
};

template <int kMode, bool kHier>
__device__ __forceinline__ void stage_link(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                           uint64_t& alpha, uint32_t& bq, HierShape& hs,
                                           const uint32_t* __restrict__ bl = nullptr) {
  const uint32_t G = p.G, tp = p.tp;
  bool same = true;
  uint32_t k0 = 0, nmin = 0xffffffffu, nmax = 0, bq_dp = 0;
  uint64_t a_dp = 0;
  hs.ok = kHier && t.ccl_hier != 0;
  hs.g = 0; hs.N = 0; hs.bq_in = 0; hs.a_in = 0;
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2) {
    if (c2 >= G) continue;
    const uint32_t k2 = (uint32_t)(p.tv[c2] >> (4 * s)) & 15;
    const TypeInfo t2 = h.type(k2);
    // (bl: the plan's lanes' stage placements, class-major, p.S per class)
    const uint32_t b2 = bl ? bl[c2 * p.S + s] : placed_before(p, c2, s, k2) * tp, n2 = p.reps[c2] * tp, d2 = t2.dpl;
    const uint32_t l2 = t2.node_off + (b2 >> d2), h2 = t2.node_off + ((b2 + n2 - 1) >> d2);
    const uint32_t dl2 = t2.dev_off + b2;
    const uint32_t nic2 = range_max(h.rmn, t.D, dl2, dl2 + n2 - 1);
    if (c2 == 0) k0 = k2; else same = same && k2 == k0;
    nmin = l2 < nmin ? l2 : nmin;
    nmax = h2 > nmax ? h2 : nmax;
    const uint32_t bx = nic2 > t2.bq_pcie ? nic2 : t2.bq_pcie;
    bq_dp = bx > bq_dp ? bx : bq_dp;
    a_dp = 2 * t2.a_side > a_dp ? 2 * t2.a_side : a_dp;
    if (kHier && t.ccl_hier) {
      const uint32_t dm = (1u << d2) - 1, gm = (1u << d2) >> p.tpl;
      hs.ok = hs.ok && (b2 & dm) == 0 && (n2 & dm) == 0 && (c2 == 0 || gm == hs.g);
      hs.g = gm;
      hs.N += n2 >> d2;
      hs.a_in = t2.a_intra > hs.a_in ? t2.a_intra : hs.a_in;
      const uint32_t bi = range_max(h.rmi(), t.N, l2, h2);
      hs.bq_in = bi > hs.bq_in ? bi : hs.bq_in;
    }
  }
  hs.ok = hs.ok && hs.g > 1 && hs.N > 1;
  const bool intra = same && nmin == nmax;
  alpha = intra ? h.type(k0).a_intra : a_dp;
  bq = intra ? h.rmi()[nmin] : bq_dp;
}

// A dense all-reduce of `grads` bytes per member over the group, with the
// two-level algorithm when the shape allows it and it is faster: the
// node-local ring over the whole gradient (g members), then the ring
// across the N nodes over a 1/g shard (g is a power of two).
__device__ __forceinline__ uint64_t with_hier(uint64_t ring, const HierShape& hs, uint32_t zero, uint64_t grads,
                                              uint64_t alpha, uint32_t bq) {
  if (!hs.ok || zero) return ring;
  const uint32_t lg = __builtin_ctz(hs.g);
  const uint64_t sh = (grads + hs.g - 1) >> lg;
  const uint64_t intra = 2ull * (hs.g - 1) * hs.a_in + link_ps(2ull * (hs.g - 1) * sh, hs.bq_in);
  const uint64_t inter = 2ull * (hs.N - 1) * alpha +
                         link_ps(2ull * (hs.N - 1) * div_up(sh, hs.N, 1.0 / (double)hs.N), bq);
  return intra + inter < ring ? intra + inter : ring;
}

// kHier: the two-level all-reduce is considered (the first-pass kernels,
// compiled without it, defer every pipeline when it is enabled).
template <int kMode, bool kHier = true>
__device__ __forceinline__ uint64_t stage_dp(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                             uint32_t ns, double rp, double rpe, const uint32_t* bl = nullptr) {
  if (p.psum <= 1) return 0;
  const uint32_t tpl = p.tpl, epl = p.epl, S = p.S;
  uint64_t alpha;
  uint32_t bq;
  HierShape hs;
  stage_link<kMode, kHier>(t, h, p, s, alpha, bq, hs, bl);
  const uint64_t pd = (uint64_t)ns * t.par_layer[tpl] + (s == 0 ? t.par_embed[tpl] : 0) +
                      (s == S - 1 ? t.par_head[tpl] : 0);
  uint64_t tdp = ring_sync(p.psum, rp, p.zero, t.grad_bytes * pd, t.param_bytes * pd, alpha, bq, t.ccl_tree);
  if (kHier) tdp = with_hier(tdp, hs, p.zero, t.grad_bytes * pd, alpha, bq);
  const uint32_t pe = p.psum >> epl;
  if (t.E && pe > 1) {
    const uint64_t px = (uint64_t)ns * t.par_expert[tpl][epl];
    tdp += ring_sync(pe, rpe, p.zero, t.grad_bytes * px, t.param_bytes * px, alpha, bq, t.ccl_tree);
  }
  return tdp;
}

// Gradient sync overlapped with stage s's last backward pass (shared layout;
// stage s holds layers [lo, hi) on device type k in the pipeline's class).
// Buckets -- the head on the last stage, the layers from the top, the
// embedding on the first stage -- each start once their backward is done,
// one after another on the stage's ring.  Bucket j is ready at
// r_j = end - R_j (R_j: backward compute of the buckets after it), so the
// queue completes at end + max_j (D_j - R_j) (D_j: syncs of bucket j and
// the later ones); that tail is returned, walked from the last bucket.
// The plan-level part of stage s's overlapped sync: the sync of one layer's
// bucket (dl; every layer bucket of the stage has the same size) and, on
// the first and last stages, of the embedding's and the head's buckets.
struct OvlSyncs {
  uint64_t dl, demb, dhead;
};
template <int kMode, bool kHier>
__device__ __forceinline__ OvlSyncs overlap_syncs(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                                  double rp, double rpe) {
  OvlSyncs r = {0, 0, 0};
  if (p.psum <= 1) return r;
  const uint32_t tpl = p.tpl, epl = p.epl;
  uint64_t alpha;
  uint32_t bq;
  HierShape hs;
  stage_link<kMode, kHier>(t, h, p, s, alpha, bq, hs);
  const uint64_t gb = t.grad_bytes, pb = t.param_bytes;
  uint64_t dl = ring_sync(p.psum, rp, p.zero, gb * t.par_layer[tpl], pb * t.par_layer[tpl], alpha, bq, t.ccl_tree);
  dl = with_hier(dl, hs, p.zero, gb * t.par_layer[tpl], alpha, bq);
  const uint32_t pe = p.psum >> epl;
  if (t.E && pe > 1)
    dl += ring_sync(pe, rpe, p.zero, gb * t.par_expert[tpl][epl], pb * t.par_expert[tpl][epl], alpha, bq, t.ccl_tree);
  r.dl = dl;
  if (s == 0)
    r.demb = with_hier(
        ring_sync(p.psum, rp, p.zero, gb * t.par_embed[tpl], pb * t.par_embed[tpl], alpha, bq, t.ccl_tree), hs, p.zero,
        gb * t.par_embed[tpl], alpha, bq);
  if (s == p.S - 1)
    r.dhead = with_hier(
        ring_sync(p.psum, rp, p.zero, gb * t.par_head[tpl], pb * t.par_head[tpl], alpha, bq, t.ccl_tree), hs, p.zero,
        gb * t.par_head[tpl], alpha, bq);
  return r;
}

// The class's part: its buckets' readiness from its own backward compute on
// device type k, walked against the syncs.
template <int kMode>
__device__ __forceinline__ uint64_t overlap_walk(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                                 uint32_t lo, uint32_t hi, uint32_t k, const OvlSyncs& y) {
  if (p.psum <= 1) return 0;
  const uint32_t tpl = p.tpl, mi = p.mi;
  const uint32_t L1 = t.L + 1, epq = t.E ? p.epl : 0;
  const uint32_t row = ((k * 4 + tpl) * t.n_mbs + mi) * t.nep + epq;
  int64_t D = 0, R = 0, X = 0;
  if (s == 0) {
    D += (int64_t)y.demb;
    X = D;
    R += (int64_t)h.emb(k * t.n_mbs + mi).y;
  }
  if (t.uniform_layers) {
    // every layer's backward costs the same r: after layer i of the n the
    // value D - R is (D + dl - R) + i (dl - r), linear in i, so its largest
    // is at the first or the last layer
    const int64_t n = (int64_t)(hi - lo), dl = (int64_t)y.dl, r = (int64_t)h.pfb(row).y;
    const int64_t v0 = D + dl - R, v1 = v0 + (n - 1) * (dl - r);
    X = v0 > X ? v0 : X;
    X = v1 > X ? v1 : X;
    D += n * dl;
    R += n * r;
  } else {
    for (uint32_t l = lo; l < hi; ++l) {
      D += (int64_t)y.dl;
      X = D - R > X ? D - R : X;
      R += (int64_t)(h.pfb(row * L1 + l + 1).y - h.pfb(row * L1 + l).y);
    }
  }
  if (s == p.S - 1) {
    D += (int64_t)y.dhead;
    X = D - R > X ? D - R : X;
  }
  return (uint64_t)X;
}

template <int kMode, bool kHier = true>
__device__ __forceinline__ uint64_t overlap_tail(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                                 uint32_t lo, uint32_t hi, uint32_t k, double rp, double rpe) {
  return overlap_walk<kMode>(t, h, p, s, lo, hi, k, overlap_syncs<kMode, kHier>(t, h, p, s, rp, rpe));
}

// The sync that follows stage s of the pipeline's class (shared layout):
// the stage's whole ring, or with overlap the part of its bucket syncs left
// after its last backward pass.
template <int kMode>
__device__ __forceinline__ uint64_t stage_sync(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s,
                                               uint32_t lo, uint32_t hi, double rp, double rpe) {
  if (p.overlap) return overlap_tail(t, h, p, s, lo, hi, (uint32_t)(p.tc >> (4 * s)) & 15, rp, rpe);
  return stage_dp(t, h, p, s, hi - lo, rp, rpe);
}

// Per-class layout.  The gradients of layers [a, e) -- a segment between
// consecutive cuts of any class, so inside one stage of every class -- sync
// in one ring over every replica, on the coarsest TP layout among the
// classes; before it, each class with finer shards gathers the coarse shard
// inside its TP groups (ring all-gather over 2^(tpl - tpl_min) members of
// the class's own shard, on the node fabric; classes at the same time, so
// the slowest counts).  rows: the plan's four class cut rows.
__device__ __forceinline__ uint32_t row_word(const uint4 (&rows)[4], uint32_t c, uint32_t j) {
  const uint4 v = rows[c];
  return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

// Weighting of a gradient shard of n elements by the class's share of the
// global batch, on a device of type k: one multiply per element, the fp32
// shard read and written (the roofline time of one elementwise op)
// (the ceilings through fp64 reciprocals: a 64-bit integer division is a
// long instruction loop on this ISA)
__device__ __forceinline__ uint64_t weigh_ps(const Tab& t, uint32_t k, uint64_t n) {
  const uint64_t by = 2000 * t.grad_bytes * n;
  const uint64_t tc = div_up_u64(n, t.tflops[k], t.rtflops[k]), tm = div_up_u64(by, t.hbm[k], t.rhbm[k]);
  return tc > tm ? tc : tm;
}

template <int kMode>
__device__ __forceinline__ uint64_t seg_dp(const Tab& t, const Hot<kMode>& h, const Plan& p, const uint4 (&rows)[4],
                                           uint32_t a, uint32_t e, double rp, double rpe, uint64_t& lat,
                                           uint64_t& bw) {
  const uint32_t G = p.G, epl = p.epl, ns = e - a;
  uint32_t tmin = 3;
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2)
    if (c2 < G) tmin = cls_tpl(p.chdr, c2) < tmin ? cls_tpl(p.chdr, c2) : tmin;
  // classes at different micro-batch sizes weight their gradients first
  bool mixed = false;
#pragma unroll
  for (uint32_t c2 = 1; c2 < 4; ++c2)
    if (c2 < G) mixed = mixed || cls_mi(p.chdr, c2) != cls_mi(p.chdr, 0);
  bool same = true;
  uint32_t k0 = 0, nmin = 0xffffffffu, nmax = 0, bq_dp = 0;
  uint64_t a_dp = 0, rs = 0, rs_l = 0, rs_b = 0;
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2) {
    if (c2 >= G) continue;
    const uint32_t tpl2 = cls_tpl(p.chdr, c2);
    // the stage of class c2 holding layer a: its cuts in (0, a] (bytes past its stages are 0)
    uint32_t s2 = 0;
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j) {
      const uint32_t w = row_word(rows, c2, j);
#pragma unroll
      for (uint32_t q = 0; q < 4; ++q) {
        const uint32_t v = (w >> (8 * q)) & 0xff;
        s2 += (v != 0 && v <= a) ? 1u : 0u;
      }
    }
    const uint32_t k2 = (uint32_t)(p.tv[c2] >> (4 * s2)) & 15;
    const TypeInfo t2 = h.type(k2);
    const uint32_t b2 = dev_before<true>(p, c2, s2, k2), n2 = p.reps[c2] << tpl2, d2 = t2.dpl;
    const uint32_t l2 = t2.node_off + (b2 >> d2), h2 = t2.node_off + ((b2 + n2 - 1) >> d2);
    const uint32_t dl2 = t2.dev_off + b2;
    const uint32_t nic2 = range_max(h.rmn, t.D, dl2, dl2 + n2 - 1);
    if (c2 == 0) k0 = k2; else same = same && k2 == k0;
    nmin = l2 < nmin ? l2 : nmin;
    nmax = h2 > nmax ? h2 : nmax;
    const uint32_t bx = nic2 > t2.bq_pcie ? nic2 : t2.bq_pcie;
    bq_dp = bx > bq_dp ? bx : bq_dp;
    a_dp = 2 * t2.a_side > a_dp ? 2 * t2.a_side : a_dp;
    if (tpl2 > tmin || mixed) {
      // the class's shard: weighted (one multiply per element, read and
      // written at the device's HBM rate) when micro-batch sizes differ,
      // then gathered to the coarsest TP layout inside each TP group
      const uint64_t g1 = (1u << (tpl2 - tmin)) - 1;
      const uint64_t sh = (uint64_t)ns * (t.par_layer[tpl2] + t.par_expert[tpl2][epl]) +
                          (a == 0 ? t.par_embed[tpl2] : 0) + (e == t.L ? t.par_head[tpl2] : 0);
      const uint64_t sc = mixed ? weigh_ps(t, k2, sh) : 0;
      const uint32_t bq_in = range_max(h.rmi(), t.N, l2, h2);
      const uint64_t rl = sc + g1 * t2.a_intra, rb = link_ps(g1 * t.grad_bytes * sh, bq_in), r = rl + rb;
      if (r > rs) {
        rs = r;
        rs_l = rl;
        rs_b = rb;
      }
    }
  }
  const bool intra = same && nmin == nmax;
  const uint64_t alpha = intra ? h.type(k0).a_intra : a_dp;
  const uint32_t bq = intra ? h.rmi()[nmin] : bq_dp;
  const uint64_t pd = (uint64_t)ns * t.par_layer[tmin] + (a == 0 ? t.par_embed[tmin] : 0) +
                      (e == t.L ? t.par_head[tmin] : 0);
  uint64_t ld = 0, bd = 0, le = 0, be = 0;
  if (p.psum > 1) ring_parts(p.psum, rp, p.zero, t.grad_bytes * pd, t.param_bytes * pd, alpha, bq, t.ccl_tree, ld, bd);
  const uint32_t pe = p.psum >> epl;
  if (t.E && pe > 1) {
    const uint64_t px = (uint64_t)ns * t.par_expert[tmin][epl];
    ring_parts(pe, rpe, p.zero, t.grad_bytes * px, t.param_bytes * px, alpha, bq, t.ccl_tree, le, be);
  }
  lat = ld + le + rs_l;
  bw = bd + be + rs_b;
  return lat + bw;
}

// The sync a stage [lo, hi) of the pipeline's class waits for: the longest
// of the segments inside it, or with contention the largest latency part
// plus the sum of the link-time parts.
template <int kMode>
__device__ __forceinline__ uint64_t het_stage_dp(const Tab& t, const Hot<kMode>& h, const Plan& p,
                                                 const uint4 (&rows)[4], uint32_t lo, uint32_t hi, double rp,
                                                 double rpe) {
  uint64_t best = 0, lmax = 0, bsum = 0;
  for (uint32_t a = lo; a < hi;) {
    uint32_t e = hi;   // the next cut of any class above a
#pragma unroll
    for (uint32_t c2 = 0; c2 < 4; ++c2)
#pragma unroll
      for (uint32_t j = 0; j < 4; ++j) {
        const uint32_t w = row_word(rows, c2, j);
#pragma unroll
        for (uint32_t q = 0; q < 4; ++q) {
          const uint32_t v = (w >> (8 * q)) & 0xff;
          e = (v > a && v < e) ? v : e;
        }
      }
    uint64_t sl, sb;
    const uint64_t x = seg_dp(t, h, p, rows, a, e, rp, rpe, sl, sb);
    best = x > best ? x : best;
    lmax = sl > lmax ? sl : lmax;
    bsum += sb;
    a = e;
  }
  return t.contention ? lmax + bsum : best;
}

__device__ __forceinline__ void load_rows(const uint4* prow, uint4 (&rows)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) rows[c] = prow[c];
}

// cut byte of stage s (run-time index) of class c of the plan's cut rows
__device__ __forceinline__ uint32_t row_cut(const uint4 (&rows)[4], uint32_t c, uint32_t s) {
  const uint4 r = rows[c];
  const uint64_t lo = (uint64_t)r.y << 32 | r.x, hi = (uint64_t)r.w << 32 | r.z;
  const uint64_t m = 0ull - (uint64_t)(s >> 3);
  return (uint32_t)(((lo & ~m) | (hi & m)) >> (8 * (s & 7))) & 0xff;
}

// Per-class layout: the sync each (class, stage) of a valid plan waits for
// -- the same values as het_stage_dp -- found by one walk over the segments
// of the whole model.  Each class's stage holding the current segment, with
// its placement and links, is recomputed only when the walk crosses one of
// that class's cuts; a class's running max is stored when it leaves a stage.
// drow: the plan's four rows of 16 entries (class c, stage s at c*16 + s).
template <int kMode>
__device__ __forceinline__ void het_plan_syncs(const Tab& t, const Hot<kMode>& h, const Plan& p,
                                               const uint4 (&rows)[4], uint64_t* __restrict__ drow) {
  const uint32_t G = p.G, epl = p.epl;
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> epl);
  uint32_t tmin = 3;
  bool mixed = false;   // classes at different micro-batch sizes weight their gradients first
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2)
    if (c2 < G) {
      tmin = cls_tpl(p.chdr, c2) < tmin ? cls_tpl(p.chdr, c2) : tmin;
      mixed = mixed || cls_mi(p.chdr, c2) != cls_mi(p.chdr, 0);
    }
  // per class: current stage and its end, and that stage's type, node range,
  // worst NIC/PCIe rate, inter-node latency, node latency, worst node fabric;
  // classes enter their first stage at the walk's first step
  // cur: the stage's sync so far -- the longest segment, or with contention
  // the largest latency part (cur) and the summed link times (curb)
  uint32_t stg[4], nxt[4], kk[4], nl[4], nh[4], bx[4], bin[4];
  uint64_t as2[4], ain[4], cur[4], curb[4];
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2) {
    stg[c2] = 0xffffffffu; nxt[c2] = c2 < G ? 0 : 0xffffffffu; kk[c2] = 0; nl[c2] = 0; nh[c2] = 0; bx[c2] = 0;
    bin[c2] = 0; as2[c2] = 0; ain[c2] = 0; cur[c2] = 0; curb[c2] = 0;
  }
  for (uint32_t a = 0; a < t.L;) {
#pragma unroll
    for (uint32_t c2 = 0; c2 < 4; ++c2) {
      if (nxt[c2] == a) {   // the walk crossed one of class c2's cuts (or starts)
        if (a > 0) drow[c2 * kMaxStages + stg[c2]] = cur[c2] + curb[c2];
        cur[c2] = 0;
        curb[c2] = 0;
        const uint32_t s2 = ++stg[c2], tpl2 = cls_tpl(p.chdr, c2);
        const uint32_t k2 = (uint32_t)(p.tv[c2] >> (4 * s2)) & 15;
        const TypeInfo t2 = h.type(k2);
        const uint32_t b2 = dev_before<true>(p, c2, s2, k2), n2 = p.reps[c2] << tpl2, d2 = t2.dpl;
        const uint32_t l2 = t2.node_off + (b2 >> d2), h2 = t2.node_off + ((b2 + n2 - 1) >> d2);
        const uint32_t dl2 = t2.dev_off + b2;
        const uint32_t nic2 = range_max(h.rmn, t.D, dl2, dl2 + n2 - 1);
        nxt[c2] = row_cut(rows, c2, s2);
        kk[c2] = k2;
        nl[c2] = l2;
        nh[c2] = h2;
        bx[c2] = nic2 > t2.bq_pcie ? nic2 : t2.bq_pcie;
        as2[c2] = 2 * t2.a_side;
        ain[c2] = t2.a_intra;
        bin[c2] = tpl2 > tmin ? range_max(h.rmi(), t.N, l2, h2) : 0;
      }
    }
    uint32_t e = t.L;
#pragma unroll
    for (uint32_t c2 = 0; c2 < 4; ++c2)
      if (c2 < G) e = nxt[c2] < e ? nxt[c2] : e;
    // the sync of layers [a, e)
    const uint32_t ns = e - a;
    bool same = true;
    uint32_t nmin = 0xffffffffu, nmax = 0, bq_dp = 0;
    uint64_t a_dp = 0, rs = 0, rs_l = 0, rs_b = 0;
#pragma unroll
    for (uint32_t c2 = 0; c2 < 4; ++c2) {
      if (c2 >= G) continue;
      same = same && kk[c2] == kk[0];
      nmin = nl[c2] < nmin ? nl[c2] : nmin;
      nmax = nh[c2] > nmax ? nh[c2] : nmax;
      bq_dp = bx[c2] > bq_dp ? bx[c2] : bq_dp;
      a_dp = as2[c2] > a_dp ? as2[c2] : a_dp;
      const uint32_t tpl2 = cls_tpl(p.chdr, c2);
      if (tpl2 > tmin || mixed) {
        const uint64_t g1 = (1u << (tpl2 - tmin)) - 1;
        const uint64_t sh = (uint64_t)ns * (t.par_layer[tpl2] + t.par_expert[tpl2][epl]) +
                            (a == 0 ? t.par_embed[tpl2] : 0) + (e == t.L ? t.par_head[tpl2] : 0);
        const uint64_t rl = (mixed ? weigh_ps(t, kk[c2], sh) : 0) + g1 * ain[c2];
        const uint64_t rb = link_ps(g1 * t.grad_bytes * sh, bin[c2]), r = rl + rb;
        if (r > rs) {
          rs = r;
          rs_l = rl;
          rs_b = rb;
        }
      }
    }
    const bool intra = same && nmin == nmax;
    const uint64_t alpha = intra ? ain[0] : a_dp;
    const uint32_t bq = intra ? h.rmi()[nmin] : bq_dp;
    const uint64_t pd = (uint64_t)ns * t.par_layer[tmin] + (a == 0 ? t.par_embed[tmin] : 0) +
                        (e == t.L ? t.par_head[tmin] : 0);
    if (!t.contention) {
      uint64_t x = p.psum <= 1 ? 0 : ring_sync(p.psum, rp, p.zero, t.grad_bytes * pd, t.param_bytes * pd, alpha, bq, t.ccl_tree);
      const uint32_t pe = p.psum >> epl;
      if (t.E && pe > 1) {
        const uint64_t px = (uint64_t)ns * t.par_expert[tmin][epl];
        x += ring_sync(pe, rpe, p.zero, t.grad_bytes * px, t.param_bytes * px, alpha, bq, t.ccl_tree);
      }
      x += rs;
#pragma unroll
      for (uint32_t c2 = 0; c2 < 4; ++c2)
        if (c2 < G) cur[c2] = x > cur[c2] ? x : cur[c2];
    } else {
      uint64_t ld = 0, bd = 0, le = 0, be = 0;
      if (p.psum > 1) ring_parts(p.psum, rp, p.zero, t.grad_bytes * pd, t.param_bytes * pd, alpha, bq, t.ccl_tree, ld, bd);
      const uint32_t pe = p.psum >> epl;
      if (t.E && pe > 1) {
        const uint64_t px = (uint64_t)ns * t.par_expert[tmin][epl];
        ring_parts(pe, rpe, p.zero, t.grad_bytes * px, t.param_bytes * px, alpha, bq, t.ccl_tree, le, be);
      }
      const uint64_t l = ld + le + rs_l, b = bd + be + rs_b;
#pragma unroll
      for (uint32_t c2 = 0; c2 < 4; ++c2)
        if (c2 < G) {
          cur[c2] = l > cur[c2] ? l : cur[c2];
          curb[c2] += b;
        }
    }
    a = e;
  }
#pragma unroll
  for (uint32_t c2 = 0; c2 < 4; ++c2)
    if (c2 < G) drow[c2 * kMaxStages + stg[c2]] = cur[c2] + curb[c2];
}

// Forward and backward time of one micro-batch over layers [lo, hi) on the
// reps * tp devices of the pipeline's class from `base` on in pool k (type
// ti; bq_in, bq_nic: slowest node fabric and NIC rates over them): the
// layers, the embedding if `first`, the head if `last`, the TP all-reduces
// exposed in the forward pass and the MoE all-to-all in both passes.  wc:
// the weight-gradient pass of the zero-bubble order, half of the backward
// compute rounded down (the all-to-all carries input gradients: it stays in
// the input-gradient pass).
template <int kMode, bool kHet>
__device__ __forceinline__ void stage_cost(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t k,
                                           const TypeInfo& ti, uint32_t base, uint32_t bq_in, uint32_t bq_nic,
                                           uint32_t lo, uint32_t hi, bool first, bool last, uint64_t& fc,
                                           uint64_t& bc, uint64_t& wc) {
  const uint32_t tp = p.tp, ep = p.ep, tpl = p.tpl, epl = p.epl, mi = p.mi, ns = hi - lo, dpl = ti.dpl;
  const uint64_t act = t.act[mi], act_tp = (act + tp - 1) >> tpl;
  const uint32_t L1 = t.L + 1, epq = t.E ? p.epl : 0;
  const uint32_t reps = p.rc;
  const uint32_t row = ((k * 4 + tpl) * t.n_mbs + mi) * t.nep + epq;
  if (t.uniform_layers) {
    const ulonglong2 lc = h.pfb(row);
    fc = lc.x * ns;
    bc = lc.y * ns;
  } else {
    const ulonglong2 ph = h.pfb(row * L1 + hi), pl = h.pfb(row * L1 + lo);
    fc = ph.x - pl.x;
    bc = ph.y - pl.y;
  }
  if (first) {
    const ulonglong2 em = h.emb(k * t.n_mbs + mi);
    fc += em.x;
    bc += em.y;
  }
  if (last) {
    const ulonglong2 hd = h.head((k * 4 + tpl) * t.n_mbs + mi);
    fc += hd.x;
    bc += hd.y;
  }
  wc = bc >> 1;
  if (tp > 1) {  // TP all-reduces of this stage, exposed in the forward pass
    const uint64_t steps = (uint64_t)(2 * ns + first) * 2 * (tp - 1);
    fc += steps * ti.a_intra + link_ps(steps * act_tp, bq_in);
  }
  if (t.E && ep > 1) {  // dispatch + combine all-to-all in each pass
    // EP groups are blocks of ep*tp devices from base on.  With one TP
    // degree for all classes base is a multiple of ep*tp, and the groups
    // are inside nodes iff one fits a node.  With per-class degrees, a
    // group of E = ep*tp <= node size starting at offset r in its node
    // fits iff r <= node - E; the offsets of the successive groups are
    // base's in-node offset plus multiples of E, so with b = base mod E
    // != 0 the first group to cross is number node/E - 1 - (in-node offset div E).
    const uint32_t E = ep * tp;
    bool intra = E <= (1u << dpl);
    if (kHet && intra && (base & (E - 1)) != 0) {
      const uint32_t q = (base & ((1u << dpl) - 1)) / E;
      intra = reps / ep <= (1u << dpl) / E - 1 - q;
    }
    const uint64_t alpha = intra ? ti.a_intra : 2 * ti.a_side;
    const uint32_t bq = intra ? bq_in : (bq_nic > ti.bq_pcie ? bq_nic : ti.bq_pcie);
    const uint32_t pa = (epl * t.n_mbs + mi) * L1;
    const uint64_t e = (uint64_t)ns * 2 * (ep - 1) * alpha + link_ps(2 * (h.pa(pa + hi) - h.pa(pa + lo)), bq);
    fc += e;
    bc += e;
  }
}

// Where the devices of stage s of the pipeline's class sit: type k, its
// pool's info, the first device in the pool, and the slowest node fabric
// and NIC rates over the stage's reps * tp devices.
template <int kMode, bool kHet>
__device__ __forceinline__ void stage_place(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t s, uint32_t& k,
                                            TypeInfo& ti, uint32_t& base, uint32_t& bq_in, uint32_t& bq_nic) {
  k = (uint32_t)(p.tc >> (4 * s)) & 15;
  ti = h.type(k);
  base = dev_before_own<kHet>(p, s, k);
  const uint32_t nd = p.rc * p.tp, dpl = ti.dpl;
  const uint32_t gnl = ti.node_off + (base >> dpl), gnh = ti.node_off + ((base + nd - 1) >> dpl);
  bq_in = range_max(h.rmi(), t.N, gnl, gnh);
  const uint32_t dlo = ti.dev_off + base;
  bq_nic = range_max(h.rmn, t.D, dlo, dlo + nd - 1);
}

// Rail-only network (Fig. 2): the NIC of local rank r of every node joins
// rail r and rails do not meet.  A pipeline hop between nodes pairs device i
// of the sending stage (from bs on, n = reps * tp devices) with device i of
// the receiving one (from br on); a pair at different local ranks is
// forwarded over a node's fabric first -- the sender's, or the receiver's
// when the sender's nodes hold one device -- which adds that node's latency
// and the activation at its slowest fabric rate (ins / inr over the
// stage's nodes).  Offsets os, or in their nodes: every pair shares a rank
// iff os == or and, with different node sizes, the n pairs do not reach the
// end of the smaller node (past it one rank wraps and the other does not).
__device__ __forceinline__ uint64_t rail_extra(uint32_t n, const TypeInfo& ts, uint32_t bs, uint32_t ins,
                                               const TypeInfo& tr, uint32_t br, uint32_t inr, uint64_t act) {
  const uint32_t ds = 1u << ts.dpl, dr = 1u << tr.dpl, os = bs & (ds - 1), orr = br & (dr - 1);
  const bool same = os == orr && (ds == dr || os + n <= (ds < dr ? ds : dr));
  if (same) return 0;
  const bool at_s = ts.dpl > 0;
  return (at_s ? ts.a_intra : tr.a_intra) + link_ps(act, at_s ? ins : inr);
}

template <int kMode, bool kHet, typename Sink>
__device__ __forceinline__ void class_setup(const Tab& t, const Hot<kMode>& h, const Plan& p, uint32_t c,
                                            Sink& sink, const uint4* prow) {
  // register sinks fix the stage count at compile time (the plan's S equals it)
  const uint32_t S = Sink::kS ? (uint32_t)Sink::kS : p.S, tp = p.tp, epl = p.epl;
  const uint64_t act = t.act[p.mi];
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> epl);
  const uint32_t reps = p.rc;
  uint32_t pk = 0, pbase = 0, pnic = 0, pin = 0, lo = 0;
  TypeInfo pti = {};
#pragma unroll Sink::kUnroll
  for (uint32_t s = 0; s < S; ++s) {
    const uint32_t hi = cut_at(p, s);
    // ---- this class: compute, TP, EP, hop from the previous stage
    uint32_t k, base, bq_in, bq_nic;
    TypeInfo ti;
    stage_place<kMode, kHet>(t, h, p, s, k, ti, base, bq_in, bq_nic);
    sink.base(s, base);
    const uint32_t dpl = ti.dpl;
    uint64_t fc, bc, wc;
    stage_cost<kMode, kHet>(t, h, p, k, ti, base, bq_in, bq_nic, lo, hi, s == 0, s == S - 1, fc, bc, wc);
    uint64_t hop = 0;
    if (s > 0) {  // hop (s-1) -> s
      // same pool means the two ranges are adjacent: intra iff the pair spans one node
      const bool intra = pk == k && (pbase >> dpl) == ((pbase + (2 * reps - 1) * tp) >> dpl);
      const uint64_t alpha = intra ? ti.a_intra : pti.a_side + ti.a_side;
      uint32_t bq;
      if (intra) {
        bq = pin > bq_in ? pin : bq_in;
      } else {
        const uint32_t a = pnic > bq_nic ? pnic : bq_nic;
        const uint32_t b = pti.bq_pcie > ti.bq_pcie ? pti.bq_pcie : ti.bq_pcie;
        bq = a > b ? a : b;
      }
      hop = alpha + link_ps(act, bq);
      if (t.rail_only && !intra) hop += rail_extra(reps * tp, pti, pbase, pin, ti, base, bq_in, act);
    }
    pk = k; pbase = base; pnic = bq_nic; pin = bq_in; pti = ti;
    // ---- DP sync of this stage (the sink may leave it for later)
    uint64_t tdp = 0;
    if (Sink::kDp) {
      if (kHet) {
        uint4 rows[4];
        load_rows(prow, rows);
        tdp = het_stage_dp(t, h, p, rows, lo, hi, rp, rpe);
      } else {
        tdp = stage_sync(t, h, p, s, lo, hi, rp, rpe);
      }
    }
    sink.put(s, fc, bc, wc, hop, tdp);
    lo = hi;
  }
}

// Sinks of class_setup.  RecSink stores whole stage records in memory order
// (the hop of the last stage is 0), and, given `w`, each stage's
// weight-gradient pass.
struct RecSink {
  static constexpr bool kDp = true;
  static constexpr int kS = 0, kUnroll = 1;   // stage count taken from the plan
  __device__ __forceinline__ void base(uint32_t, uint32_t) {}
  uint64_t (&rec)[kMaxStages][kRecWords];
  uint64_t* w = nullptr;
  __device__ __forceinline__ void put(uint32_t s, uint64_t fc, uint64_t bc, uint64_t wc, uint64_t hop,
                                      uint64_t tdp) {
    rec[s][0] = fc;
    rec[s][1] = bc;
    rec[s][2] = 0;
    rec[s][3] = tdp;
    if (w) w[s] = wc;
    if (s > 0) rec[s - 1][2] = hop;
  }
};

// RegSink keeps forward, backward and hop times of an S-stage pipeline in
// registers as fp64 (every stage quantity is below 2^52, so exact): each
// stage shifts the arrays down by one and appends, so after S stages stage s
// sits at index s; a runtime-indexed array would go through private memory.
// The stage loop runs S (a compile-time count) times, unrolled by
// kSetupUnroll: within an unrolled body the shifts are register renames, so
// the copies are paid once per kSetupUnroll stages.  The DP sync is left to
// dp_tail, after the recurrence.
constexpr int kSetupUnroll = 4;

template <int S>
struct RegSink {
  static constexpr bool kDp = false;
  static constexpr int kS = S, kUnroll = kSetupUnroll;
  double f[S], b[S], c[S];
  uint32_t* bs = nullptr;   // optional: each stage's first device in its pool (LDS)
  __device__ __forceinline__ void base(uint32_t s, uint32_t b0) {
    if (bs) bs[s] = b0;
  }
  __device__ __forceinline__ RegSink() {
#pragma unroll
    for (int i = 0; i < S; ++i) f[i] = b[i] = c[i] = 0;
  }
  __device__ __forceinline__ void put(uint32_t s, uint64_t fc, uint64_t bc, uint64_t, uint64_t hop, uint64_t) {
#pragma unroll
    for (int i = 0; i + 1 < S; ++i) {
      f[i] = f[i + 1];
      b[i] = b[i + 1];
      c[i] = c[i + 1];
    }
    f[S - 1] = (double)fc;
    b[S - 1] = (double)bc;
    c[S - 1] = 0;
    if (S > 1 && s > 0) c[S - 2] = (double)hop;
  }
};

// ZbSink: the same with the backward split for the zero-bubble order: bi,
// the input-gradient pass, and w, the weight-gradient pass.
template <int S>
struct ZbSink {
  static constexpr bool kDp = false;
  static constexpr int kS = S, kUnroll = kSetupUnroll;
  __device__ __forceinline__ void base(uint32_t, uint32_t) {}
  double f[S], bi[S], w[S], c[S];
  __device__ __forceinline__ ZbSink() {
#pragma unroll
    for (int i = 0; i < S; ++i) f[i] = bi[i] = w[i] = c[i] = 0;
  }
  __device__ __forceinline__ void put(uint32_t s, uint64_t fc, uint64_t bc, uint64_t wc, uint64_t hop, uint64_t) {
#pragma unroll
    for (int i = 0; i + 1 < S; ++i) {
      f[i] = f[i + 1];
      bi[i] = bi[i + 1];
      w[i] = w[i + 1];
      c[i] = c[i + 1];
    }
    f[S - 1] = (double)fc;
    bi[S - 1] = (double)(bc - wc);
    w[S - 1] = (double)wc;
    c[S - 1] = 0;
    if (S > 1 && s > 0) c[S - 2] = (double)hop;
  }
};

// Iteration time from the end of each stage's last op: the max over stages
// of that end plus the stage's DP sync, walking the stages with the same
// shift so that no array is indexed at run time.
template <int S, int kMode, bool kHet, bool kOvl, bool kHier>
__device__ __forceinline__ double dp_tail(const Tab& t, const Hot<kMode>& h, const Plan& p, double (&last)[S],
                                          const uint64_t* drow) {
  if constexpr (kHet) {
    // per-class layout: the syncs the plan pass stored for this pipeline's stages
    double T = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      const double e = last[s] + (double)drow[s];
      T = e > T ? e : T;
    }
    return T;
  }
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> p.epl);
  double T = 0;
  uint32_t lo = 0;
  for (uint32_t s = 0; s < (uint32_t)S; ++s) {
    const uint32_t hi = cut_at(p, s);
    const uint64_t d = kOvl ? overlap_tail<kMode, kHier>(t, h, p, s, lo, hi, (uint32_t)(p.tc >> (4 * s)) & 15, rp, rpe)
                            : stage_dp<kMode, kHier>(t, h, p, s, hi - lo, rp, rpe);
    const double e = last[0] + (double)d;
    T = e > T ? e : T;
#pragma unroll
    for (int i = 0; i + 1 < S; ++i) last[i] = last[i + 1];
    lo = hi;
  }
  return T;
}

template <int S, int v>
__device__ __forceinline__ void il_records(const Tab& t, const Hot<2>& h, const Plan& p, uint64_t* o);
__device__ __forceinline__ uint32_t il_shape(uint32_t S, uint32_t v) { return S | (v - 1) << 5; }

// per (class, stage) quantities of every plan, in plan order; for an
// interleaved pipeline per virtual stage (hops and syncs per device, in the
// first S records, the last hop being the wrap hop)
template <bool kHet>
__global__ void __launch_bounds__(256) k_stages(Tab t, const PackedPlan* __restrict__ packed,
                                                const uint4* __restrict__ pcut, const uint32_t* __restrict__ meta,
                                                int64_t n, uint64_t* __restrict__ out_stage) {
  const int64_t slot = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (slot >= n * 4 || meta[slot] == 0) return;
  const Plan p = load_plan<kHet>(packed, pcut, (uint32_t)slot);
  const Hot<2> h(t, nullptr);
  if (!kHet && p.v > 1) {
    uint64_t* o = out_stage + slot * (kMaxStages * kRecWords);
    switch (il_shape(p.S, p.v)) {
#define X(S_, V_)                        \
  case S_ | (V_ - 1) << 5:               \
    il_records<S_, V_>(t, h, p, o);      \
    break;
      HETSIM_IL_SHAPES(X)
#undef X
      default: break;
    }
    return;
  }
  uint64_t rec[kMaxStages][kRecWords];
  RecSink sink{rec};
  class_setup<2, kHet>(t, h, p, (uint32_t)(slot & 3), sink, kHet ? pcut + (slot & ~3ll) : nullptr);
  uint64_t* o = out_stage + slot * (kMaxStages * kRecWords);
  for (uint32_t s = 0; s < p.S; ++s)
#pragma unroll
    for (int q = 0; q < kRecWords; ++q) o[s * kRecWords + q] = rec[s][q];
}

// Per-class layout: the syncs of every (class, stage) of every valid plan
// (one plan per lane), once per plan rather than once per pipeline; lane j
// takes plan perm[j] of the pc[512] valid plans (sorted by the length of
// their walks).
template <int kMode>
__global__ void __launch_bounds__(256) k_plan_syncs(Tab t, const PackedPlan* __restrict__ packed,
                                                    const uint4* __restrict__ pcut, const uint32_t* __restrict__ perm,
                                                    const uint32_t* __restrict__ pc, int64_t n,
                                                    uint64_t* __restrict__ hdp) {
  extern __shared__ uint4 lds[];
  fill_lds<kMode>(t, lds);
  const Hot<kMode> h(t, lds);
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n || j >= (int64_t)pc[2 * kPlanBuckets]) return;
  const uint32_t i = perm[j];
  const Plan p = unpack(packed[i], 0);
  uint4 rows[4];
  load_rows(pcut + 4 * (size_t)i, rows);
  het_plan_syncs(t, h, p, rows, hdp + (size_t)i * (kMaxClasses * kMaxStages));
}


// ---------------------------------------------------------------- 1F1B pipeline
// Schedule of one class (S stages, M micro-batches per replica): stage s runs
// W_s = min(S-1-s, M) forwards, then pairs (forward, backward), then its last
// W_s backwards.  Evaluation order that respects every dependency:
//   warm-up rows m = 0..: stages s < S-1-m run F(s, m), ascending s;
//   then for each backward index i, descending s: F(s, i + W_s) if it exists,
//   then B(s, i).
// Descending s lets B(s, i) read B(s+1, i) just computed while F(s, .) still
// sees stage s-1's previous forward.  Iterations where every stage has its
// forward form the steady loop; the last min(S-1, M) iterations, where the
// upper stages have run out of forwards, are unrolled.
//   out_f[s] end of the latest forward on stage s, last[s] end of its latest op.
// Each schedule node is end = max(previous end on the stage, input end + hop)
// + duration: 3 VALU ops in fp64, 5 in u64 (64-bit add is one v_lshl_add_u64,
// max is a compare and two selects).
typedef uint64_t StageRec[kMaxStages][kRecWords];

__device__ __forceinline__ double vmax(double a, double b) { return __builtin_fmax(a, b); }
__device__ __forceinline__ uint64_t vmax(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Periodic regime.  One steady iteration maps the state x = (out_f[0..S-2],
// last[0..S-1]) to a max of (component + constant) terms, so adding a constant
// lam to every component of x adds lam to every component of the result.
// Hence once an iteration advances every component by the same lam, every
// later one does too, and the remaining r steady iterations collapse into
// x += r * lam, exactly (in fp64 every value stays below 2^53 or the pipeline
// is redone in u64).  On the workloads here most schedules reach that regime
// within a few iterations after the warm-up, against a hundred or more
// micro-batches.  A wave waits at most kPeriodicBudget steady iterations for
// its lanes; a lane still aperiodic by then is deferred to a full-loop pass,
// so one aperiodic schedule does not hold 63 periodic ones.
constexpr int kPeriodicBudget = 40;

template <int S, typename V>
__device__ __forceinline__ void steady_iter(const V (&f)[S], const V (&b)[S], const V (&c)[S], V (&out_f)[S],
                                            V (&last)[S]) {
#pragma unroll
  for (int s = S - 1; s >= 0; --s) {
    const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
    out_f[s] = st + f[s];
    const V sb = s == S - 1 ? out_f[s] : vmax(out_f[s], last[s + 1] + c[s]);
    last[s] = sb + b[s];
  }
}

// kJump: take the periodic shortcut; then `skipped` returns the steady
// iterations it skipped, or -1 if the lane is deferred (result not computed).
// Returns false for a deferred lane; else last[s] = end of stage s's last op.
template <int S, typename V, bool kJump, bool kFallback = false>
__device__ __forceinline__ bool pipe(const V (&f)[S], const V (&b)[S], const V (&c)[S], uint32_t M, int& skipped,
                                     V (&last)[S]) {
  V out_f[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    out_f[s] = 0;
    last[s] = 0;
  }
  const int m_ = (int)M;
#pragma unroll
  for (int m = 0; m < S - 1; ++m) {
    if (m < m_) {
#pragma unroll
      for (int s = 0; s < S - 1 - m; ++s) {
        const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
        out_f[s] = st + f[s];
        last[s] = out_f[s];
      }
    }
  }
  int left = m_ - (S - 1);
  skipped = 0;
  if (kJump) {
    int budget = kPeriodicBudget;
    while (left >= 2 && budget > 0) {
      steady_iter<S, V>(f, b, c, out_f, last);
      // second iteration of the pair: does every state value advance by lam?
      bool same = true;
      V lam = 0;
#pragma unroll
      for (int s = S - 1; s >= 0; --s) {
        const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
        const V nf = st + f[s];
        if (s < S - 1) same = same && nf - out_f[s] == lam;
        out_f[s] = nf;
        const V nl = (s == S - 1 ? nf : vmax(nf, last[s + 1] + c[s])) + b[s];
        if (s == S - 1) lam = nl - last[s];
        else same = same && nl - last[s] == lam;
        last[s] = nl;
      }
      left -= 2;
      budget -= 2;
      if (same) {
        const V k = (V)left * lam;
#pragma unroll
        for (int s = 0; s < S; ++s) {
          out_f[s] += k;
          last[s] += k;
        }
        skipped = left;
        left = 0;
      }
    }
    if (left == 1) {
      steady_iter<S, V>(f, b, c, out_f, last);
      left = 0;
    }
    if (kFallback) {
      // still aperiodic after the budget: the rest of the steady loop here
      for (; left > 0; --left) steady_iter<S, V>(f, b, c, out_f, last);
    } else if (left > 0) {
      skipped = -1;
      return false;
    }
  } else {
    // two iterations per trip: the next iteration's upper stages overlap
    // this one's backward chain
#pragma unroll 2
    for (int i = 0; i < left; ++i) steady_iter<S, V>(f, b, c, out_f, last);
  }
#pragma unroll
  for (int tr = 0; tr < S - 1; ++tr) {
    if (tr >= S - 1 - m_) {
#pragma unroll
      for (int s = S - 1; s >= 0; --s) {
        if (s > tr) {
          const V st = vmax(last[s], out_f[s - 1] + c[s - 1]);
          out_f[s] = st + f[s];
          const V sb = s == S - 1 ? out_f[s] : vmax(out_f[s], last[s + 1] + c[s]);
          last[s] = sb + b[s];
        } else {
          last[s] = (s == S - 1 ? last[s] : vmax(last[s], last[s + 1] + c[s])) + b[s];
        }
      }
    }
  }
  return true;
}

// Zero-bubble order (ZB-H1, Qi et al. 2024): pipe's evaluation order with a
// stage's backward pass split into bi, the input gradient stage s-1 waits
// for (eb = its end), and w, the weight gradient (half of the backward
// compute; the MoE all-to-all stays in bi).  After B(s, i) stage s runs
// W(s, i - s) once i >= s -- a pure delay on the stage, its B having run
// before -- and its last min(s, M) W passes at the end.  From i = S - 1 on
// every steady iteration runs every stage's W, so the same map repeats and
// the periodic shortcut applies as in pipe (state out_f[0..S-2],
// last[0..S-1]; the B end of stage s + 1 is read only by stage s, right
// after, in the same iteration, so it is one carried value).  kJump:
// shortcut pairs within the budget, then the whole loop; otherwise the
// whole loop.
template <int S, typename V>
__device__ __forceinline__ void zb_iter(const V (&f)[S], const V (&bi)[S], const V (&w)[S], const V (&c)[S], int i,
                                        int tr, V (&out_f)[S], V (&last)[S]) {
  V eb = 0;
#pragma unroll
  for (int s = S - 1; s >= 0; --s) {
    if (s > tr) {   // the stage still runs a forward in this iteration
      const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
      out_f[s] = st + f[s];
      const V sb = s == S - 1 ? out_f[s] : vmax(out_f[s], eb + c[s]);
      eb = sb + bi[s];
    } else {
      eb = (s == S - 1 ? last[s] : vmax(last[s], eb + c[s])) + bi[s];
    }
    last[s] = i >= s ? eb + w[s] : eb;
  }
}

template <int S, typename V, bool kJump, bool kFallback = false>
__device__ __forceinline__ bool pipe_zb(const V (&f)[S], const V (&bi)[S], const V (&w)[S], const V (&c)[S], uint32_t M,
                                        int& skipped,
                                        V (&last)[S]) {
  V out_f[S];
#pragma unroll
  for (int s = 0; s < S; ++s) out_f[s] = last[s] = 0;
  const int m_ = (int)M;
#pragma unroll
  for (int m = 0; m < S - 1; ++m) {
    if (m < m_) {
#pragma unroll
      for (int s = 0; s < S - 1 - m; ++s) {
        const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
        out_f[s] = st + f[s];
        last[s] = out_f[s];
      }
    }
  }
  const int left = m_ - (S - 1);
  skipped = 0;
  int i = 0;
  for (; i < left && i < S - 1; ++i) zb_iter<S, V>(f, bi, w, c, i, -1, out_f, last);
  int rem = left - i;
  if (kJump) {
    int budget = kPeriodicBudget;
    while (rem >= 2 && budget > 0) {
      zb_iter<S, V>(f, bi, w, c, S, -1, out_f, last);
      bool same = true;
      V lam = 0, eb = 0;
#pragma unroll
      for (int s = S - 1; s >= 0; --s) {
        const V st = s == 0 ? last[0] : vmax(last[s], out_f[s - 1] + c[s - 1]);
        const V nf = st + f[s];
        if (s < S - 1) same = same && nf - out_f[s] == lam;
        out_f[s] = nf;
        const V sb = s == S - 1 ? nf : vmax(nf, eb + c[s]);
        eb = sb + bi[s];
        const V nl = eb + w[s];
        if (s == S - 1) lam = nl - last[s];
        else same = same && nl - last[s] == lam;
        last[s] = nl;
      }
      rem -= 2;
      budget -= 2;
      if (same) {
        const V k = (V)rem * lam;
#pragma unroll
        for (int s = 0; s < S; ++s) {
          out_f[s] += k;
          last[s] += k;
        }
        skipped = rem;
        rem = 0;
      }
    }
    if (rem == 1) {
      zb_iter<S, V>(f, bi, w, c, S, -1, out_f, last);
      rem = 0;
    }
    if (rem > 0 && !kFallback) {   // still aperiodic: the deferred pass runs the whole loop
      skipped = -1;
      return false;
    }
  }
  for (; rem > 0; --rem) zb_iter<S, V>(f, bi, w, c, S, -1, out_f, last);
#pragma unroll
  for (int tr = 0; tr < S - 1; ++tr)
    if (tr >= S - 1 - m_) zb_iter<S, V>(f, bi, w, c, m_ - S + 1 + tr, tr, out_f, last);
#pragma unroll
  for (int s = 0; s < S; ++s) last[s] += (V)(s < m_ ? s : m_) * w[s];
  return true;
}

// Integers below 2^53 are exact in fp64.  Every value the fp64 pass computes
// is at most the end of some op, which is at most T, so if T < 2^53 no
// rounding ever happened.  Otherwise the pipeline goes on an overflow list
// and k_redo_u64 evaluates it again in u64, outside the hot kernels.
constexpr double kExact = 9007199254740992.0;

// Device buffers of one evaluation pass over a chunk.
struct EvalBufs {
  const PackedPlan* packed;
  const uint4* pcut;        // per-class layout: cut row of pipeline slot at [slot]
  const uint64_t* hdp;      // per-class layout: the syncs of pipeline slot's stages at [16 slot, + 16)
  const uint32_t* meta;
  const uint32_t* ids;      // pipeline ids sorted by bucket
  const uint32_t* sstart;   // [16 - S]: start of the S-stage pipelines in ids; [16] = total
  uint64_t* out;
  uint32_t* ctr;            // [0] overflow count, [1 + 16 - S] deferred S-stage pipelines,
                            // [kVariantCtr + 16 - S] S-stage overlap and zero-bubble pipelines
  uint32_t* ovf;            // overflow list (fp64 result reached 2^53)
  uint32_t* deferred;       // deferred S-stage pipelines at [sstart[16 - S], ...)
  uint32_t* vlist;          // S-stage overlap and zero-bubble tiles at [sstart[16 - S], ...): each a
                            // first-pass wavefront's lanes as they were (kNoSlot elsewhere)
  unsigned long long* skipped_ops;   // optional: recurrence ops skipped by the shortcut
  const Tab* dtab;          // the Tab in device memory
};

// Pipelines are sorted by stage count (descending), so each group of four
// stage counts is a contiguous range of ids; one kernel per group keeps the
// register footprint, and so the occupancy, of small pipelines independent of
// the 16-stage code.  Block b of group g runs the g-th range's pipelines
// [64b, 64b + 64); blocks past the range return at once.  This first pass
// takes the periodic shortcut and defers the lanes still aperiodic after the
// budget; k_deferred runs those through the whole steady loop.
// kOvl: the pipeline's plan overlaps its gradient sync with the last
// backward pass; kZb: it runs the zero-bubble order.  The first pass (kFull
// false) sends both kinds to the variant lists, so that its kernels carry
// neither; k_variant runs them with the shortcut (the whole loop where they
// stay aperiodic).  With a context that enables two-level collectives, whose
// sync code the first pass lacks, it sends every other shared-layout
// pipeline to the deferred lists.
// DP tail of a plan-sorted pipeline (first pass, shared layout, G > 1 classes
// on G adjacent lanes): the lane of class c costs the syncs of stages c,
// c + G, ... (each the same for every class of the plan) into its plan's row
// of the wavefront's LDS exchange area, then every lane of the plan reads
// the whole row.  Every lane of the plan takes part, deferred ones included
// (the syncs do not depend on the recurrence).
template <int S, int kMode, bool kHier>
__device__ __forceinline__ double grouped_tail(const Tab& t, const Hot<kMode>& h, const Plan& p, const double (&last)[S],
                                               double* xw, const uint32_t* bw = nullptr) {
  const uint32_t G = p.G, lane = threadIdx.x & 63u;
  double* x = xw + (lane / G) * xchg_row(S);
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> p.epl);
  // bw: every lane's stage placements from its setup (S per lane); the
  // plan's G lanes start at lane - c
  const uint32_t* bl = bw ? bw + (lane - p.c) * S : nullptr;
  if (bw) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  for (uint32_t s = p.c; s < (uint32_t)S; s += G) {
    const uint32_t lo = s ? cut_at(p, s - 1) : 0;
    x[s] = (double)stage_dp<kMode, kHier>(t, h, p, s, cut_at(p, s) - lo, rp, rpe, bl);
  }
  // the rows are written and read by the lanes of one wavefront, whose LDS
  // accesses complete in order; the fences keep the compiler from moving
  // the reads above the writes of the other lanes
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  double T = 0;
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const double v = last[s] + x[s];
    T = v > T ? v : T;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  return T;
}

// The same for an overlapped plan (variant pass): the lane of class c costs
// the syncs of stages c, c + G, ... (one layer's bucket per stage, the
// embedding's and the head's) into its plan's row, then every lane walks its
// own buckets' readiness against them.
template <int S, int kMode>
__device__ __forceinline__ double grouped_overlap_tail(const Tab& t, const Hot<kMode>& h, const Plan& p,
                                                       double (&last)[S], double* xw) {
  const uint32_t G = p.G, lane = threadIdx.x & 63u;
  double* x = xw + (lane / G) * xchg_row(S);
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> p.epl);
  for (uint32_t s = p.c; s < (uint32_t)S; s += G) {
    const OvlSyncs y = overlap_syncs<kMode, true>(t, h, p, s, rp, rpe);
    x[s] = (double)y.dl;
    if (s == 0) x[xchg_row(S) - 2] = (double)y.demb;
    if (s == (uint32_t)S - 1) x[xchg_row(S) - 1] = (double)y.dhead;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const OvlSyncs ends = {0, (uint64_t)x[xchg_row(S) - 2], (uint64_t)x[xchg_row(S) - 1]};
  double T = 0;
  uint32_t lo = 0;
  for (uint32_t s = 0; s < (uint32_t)S; ++s) {
    const uint32_t hi = cut_at(p, s);
    const OvlSyncs y = {(uint64_t)x[s], ends.demb, ends.dhead};
    const double e = last[0] + (double)overlap_walk<kMode>(t, h, p, s, lo, hi, (uint32_t)(p.tc >> (4 * s)) & 15, y);
    T = e > T ? e : T;
#pragma unroll
    for (int i = 0; i + 1 < S; ++i) last[i] = last[i + 1];
    lo = hi;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  return T;
}

template <int S, bool kFull, int kMode, bool kHet, bool kOvl = false, bool kZb = false>
__device__ __forceinline__ void eval_one(const Tab& t, const Hot<kMode>& h, const EvalBufs& e, uint32_t slot,
                                         double* xw = nullptr, uint32_t* bw = nullptr) {
  // plan-sorted pipelines of the first or the variant pass (shared layout)
  constexpr bool kGrouped = !kFull && !kHet;
  typename std::conditional<kZb, ZbSink<S>, RegSink<S>>::type r;
  uint32_t M;
  const Plan p = load_plan<kHet>(e.packed, e.pcut, slot);
  {
    if (!kFull && !kHet && !kOvl && !kZb) {
      // (overlap and zero-bubble plans left for the variant pass in k_eval)
      if (t.ccl_hier) {
        e.deferred[e.sstart[kMaxStages - S] + atomicAdd(&e.ctr[1 + kMaxStages - S], 1u)] = slot;
        return;
      }
    }
    M = class_mb(p);
    if constexpr (kGrouped && !kZb)
      if (bw) r.bs = bw + (threadIdx.x & 63u) * S;
    class_setup<kMode, kHet>(t, h, p, slot & 3, r, nullptr);
  }
  int skipped;
  double last[S];
  bool done = true;
  // the first and variant passes take the periodic shortcut and defer the
  // lanes still aperiodic after the budget; the deferred pass runs the whole loop
  if constexpr (kZb) done = pipe_zb<S, double, !kFull>(r.f, r.bi, r.w, r.c, M, skipped, last);
  else done = pipe<S, double, !kFull>(r.f, r.b, r.c, M, skipped, last);
  // With up to kKeepPlanS stages the plan stays in registers through the
  // recurrence (whose state is small); longer pipelines read it again for
  // the DP tail (an L2 hit) rather than hold it: the lane's own slot passed
  // through a shuffle is opaque to the compiler, which would otherwise reuse
  // the first load
  constexpr int kKeepPlanS = 8;
  const uint32_t slot2 = S <= kKeepPlanS ? slot : __shfl(slot, (int)(threadIdx.x & 63u));
  double T;
  const Plan p2 = S <= kKeepPlanS ? p : load_plan<kHet>(e.packed, e.pcut, slot2);
  if (kGrouped && p2.G > 1) {   // G is the same in the whole wavefront
    if constexpr (kOvl) T = grouped_overlap_tail<S, kMode>(t, h, p2, last, xw);
    else T = grouped_tail<S, kMode, kZb>(t, h, p2, last, xw, kZb ? nullptr : bw);
  } else {
    T = done ? dp_tail<S, kMode, kHet, kOvl, kFull || kOvl || kZb>(t, h, p2, last,
                                                                   kHet ? e.hdp + (size_t)slot2 * kMaxStages : nullptr)
             : 0;
  }
  if constexpr (kGrouped) {
    // the plan's G pipelines sit on adjacent lanes from a multiple of G, all
    // of them here: the first one stores the largest result of the finished
    // ones (one store per plan; the deferred and the u64 passes, later in
    // stream order, raise it with atomicMax)
    const uint32_t G = p2.G, lane = threadIdx.x & 63u, lead = lane - lane % G;
    const bool mine = done && T < kExact;
    double v = mine ? T : 0;
    for (uint32_t c = 1; c < G; ++c) {
      const double u = __shfl(v, (int)(lead + c));
      if (lane == lead) v = u > v ? u : v;
    }
    if (lane == lead && v > 0) e.out[slot >> 2] = (uint64_t)v;
    if (!done) {
      e.deferred[e.sstart[kMaxStages - S] + atomicAdd(&e.ctr[1 + kMaxStages - S], 1u)] = slot;
      return;
    }
    if (!mine) e.ovf[atomicAdd(&e.ctr[0], 1u)] = slot;
  } else {
    if (!done) {
      e.deferred[e.sstart[kMaxStages - S] + atomicAdd(&e.ctr[1 + kMaxStages - S], 1u)] = slot;
      return;
    }
    if (T < kExact) {
      atomicMax((unsigned long long*)&e.out[slot >> 2], (unsigned long long)T);
    } else {
      e.ovf[atomicAdd(&e.ctr[0], 1u)] = slot;
    }
  }
  if (e.skipped_ops && skipped > 0)
    atomicAdd(e.skipped_ops + ((blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) % kSkipSlots) * kSkipStride,
              (unsigned long long)skipped * (unsigned long long)(6 * (S - 1) + 2));
}

// Deferred pass of one pipeline: the whole loop (plain, overlap or zero-bubble, by its header).
template <int S, int kMode, bool kHet>
__device__ __forceinline__ void eval_deferred(const Tab& t, const Hot<kMode>& h, const EvalBufs& e, uint32_t slot) {
  const uint32_t hdr = kHet ? 0 : e.packed[slot >> 2].hdr;
  if (!kHet && ((hdr >> 16) & 1)) eval_one<S, true, kMode, false, false, true>(t, h, e, slot);
  else if (!kHet && ((hdr >> 13) & 1)) eval_one<S, true, kMode, false, true, false>(t, h, e, slot);
  else eval_one<S, true, kMode, kHet>(t, h, e, slot);
}

// Variant pass of one pipeline (shared layout): overlapped gradient sync or
// the zero-bubble order, with the periodic shortcut; lanes still aperiodic
// after the budget go to the deferred lists (the deferred pass runs them
// through the whole loop).
template <int S, int kMode>
__device__ __forceinline__ void eval_variant(const Tab& t, const Hot<kMode>& h, const EvalBufs& e, uint32_t slot,
                                             double* xw) {
  if ((e.packed[slot >> 2].hdr >> 16) & 1) eval_one<S, false, kMode, false, false, true>(t, h, e, slot, xw);
  else eval_one<S, false, kMode, false, true>(t, h, e, slot, xw);
}

// ---------------------------------------------------------------- interleaved 1F1B
// Schedule (Narayanan et al. 2021): device s of an S-device pipeline holds
// chunks j = 0..v-1 of the model, virtual stage j S + s.  It runs
// W_s = 2 (S-1-s) + (v-1) S warm-up forwards, then (forward, backward) pairs,
// then its last W_s backwards; its k-th forward runs chunk (k mod S v) / S,
// its k-th backward chunk v-1 - (k mod S v) / S, both on micro-batch
// (k div S v) S + k mod S.  With M a multiple of S and M >= 2 S the devices
// advance in lockstep: at step t device s runs forward k = t - s, then
// backward k = t - s - W_s (each where 0 <= k < M v), and each op's input is
// an op of a neighbouring device at step t - 1: for a forward on device
// s > 0 the forward of device s - 1, on device 0 (chunk j > 0) the forward
// of device S - 1 across the wrap hop; for a backward on device s < S - 1
// the backward of device s + 1, on device S - 1 (chunk j < v - 1) the
// backward of device 0 across the wrap hop; the last virtual stage's
// backward takes its own forward of the same step.  Steps run
// t = 0 .. M v + W_0 - 1.  Within a trip of S v steps starting at a multiple
// of S v, the chunk of every op is a compile-time constant, so every
// duration is a register.

// Hop between the devices of two stages of one class, a placed before b
// when they share a pool: inside a node iff every replica's pair is, i.e.
// iff a's first device and b's last one share a node.
__device__ __forceinline__ uint64_t il_hop(const Tab& t, uint32_t ka, const TypeInfo& ta, uint32_t basea,
                                           uint32_t ina, uint32_t nica, uint32_t kb, const TypeInfo& tb,
                                           uint32_t baseb, uint32_t inb, uint32_t nicb, uint32_t reps, uint32_t tp,
                                           uint64_t act, bool a_sends) {
  const uint32_t dpl = tb.dpl;
  const bool intra = ka == kb && (basea >> dpl) == ((baseb + (reps - 1) * tp) >> dpl);
  const uint64_t alpha = intra ? tb.a_intra : ta.a_side + tb.a_side;
  uint32_t bq;
  if (intra) {
    bq = ina > inb ? ina : inb;
  } else {
    const uint32_t x = nica > nicb ? nica : nicb;
    const uint32_t y = ta.bq_pcie > tb.bq_pcie ? ta.bq_pcie : tb.bq_pcie;
    bq = x > y ? x : y;
  }
  uint64_t hop = alpha + link_ps(act, bq);
  if (t.rail_only && !intra)
    hop += a_sends ? rail_extra(reps * tp, ta, basea, ina, tb, baseb, inb, act)
                   : rail_extra(reps * tp, tb, baseb, inb, ta, basea, ina, act);
  return hop;
}

// Per virtual stage forward and backward time (f, b), hops between devices
// (c[s]: s -> s + 1, c[S - 1]: the wrap hop S - 1 -> 0).
template <int S, int v, int kMode, typename V>
__device__ __forceinline__ void il_setup(const Tab& t, const Hot<kMode>& h, const Plan& p, V (&f)[S * v],
                                         V (&b)[S * v], V (&c)[S]) {
  constexpr int NV = S * v;
  const uint64_t act = t.act[p.mi];
  uint32_t k0 = 0, base0 = 0, in0 = 0, nic0 = 0, pk = 0, pbase = 0, pin = 0, pnic = 0;
  TypeInfo ti0 = {}, pti = {};
#pragma unroll
  for (int s = 0; s < S; ++s) {
    uint32_t k, base, bq_in, bq_nic;
    TypeInfo ti;
    stage_place<kMode, false>(t, h, p, s, k, ti, base, bq_in, bq_nic);
#pragma unroll
    for (int j = 0; j < v; ++j) {
      const int vs = j * S + s;
      const uint32_t lo = vs ? cut_at(p, vs - 1) : 0, hi = cut_at(p, vs);
      uint64_t fc, bc, wc;
      stage_cost<kMode, false>(t, h, p, k, ti, base, bq_in, bq_nic, lo, hi, vs == 0, vs == NV - 1, fc, bc, wc);
      f[vs] = (V)fc;
      b[vs] = (V)bc;
    }
    if (s > 0) c[s - 1] = (V)il_hop(t, pk, pti, pbase, pin, pnic, k, ti, base, bq_in, bq_nic, p.rc, p.tp, act, true);
    if (s == 0) {
      k0 = k; ti0 = ti; base0 = base; in0 = bq_in; nic0 = bq_nic;
    }
    if (s == S - 1)   // the wrap hop: device S - 1 sends to device 0, placed before it
      c[S - 1] = (V)il_hop(t, k0, ti0, base0, in0, nic0, k, ti, base, bq_in, bq_nic, p.rc, p.tp, act, false);
    pk = k; pti = ti; pbase = base; pin = bq_in; pnic = bq_nic;
  }
}

// One trip of S v steps from step t0 (a multiple of S v).  kPred: some op of
// the trip may lie outside its device's schedule (warm-up, cool-down);
// otherwise every device runs a forward and a backward at every step.
// F[s], B[s]: end of device s's latest forward / backward; busy[s]: of its
// latest op.
template <int S, int v, typename V, bool kPred>
__device__ __forceinline__ void il_trip(int t0, int n, const V (&f)[S * v], const V (&b)[S * v], const V (&c)[S],
                                        V (&F)[S], V (&B)[S], V (&busy)[S]) {
  constexpr int NV = S * v;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    V nF[S], nB[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
      const int W = 2 * (S - 1 - s) + (v - 1) * S;
      const int jf = ((u - s) % NV + NV) % NV / S, vf = jf * S + s;
      const int jb = v - 1 - ((u - s - W) % NV + NV) % NV / S, vb = jb * S + s;
      V x = busy[s];
      const V rf = s > 0 ? F[s - 1] + c[s - 1] : jf > 0 ? F[S - 1] + c[S - 1] : (V)0;
      V ef = vmax(x, rf) + f[vf];
      if (kPred) {
        const bool a = (unsigned)(t0 + u - s) < (unsigned)n;
        ef = a ? ef : F[s];
        x = a ? ef : x;
      } else {
        x = ef;
      }
      nF[s] = ef;
      const V rb = vb == NV - 1 ? ef : s < S - 1 ? B[s + 1] + c[s] : B[0] + c[S - 1];
      V eb = vmax(x, rb) + b[vb];
      if (kPred) {
        const bool a = (unsigned)(t0 + u - s - W) < (unsigned)n;
        eb = a ? eb : B[s];
        x = a ? eb : x;
      } else {
        x = eb;
      }
      nB[s] = eb;
      busy[s] = x;
    }
#pragma unroll
    for (int s = 0; s < S; ++s) {
      F[s] = nF[s];
      B[s] = nB[s];
    }
  }
}

// The whole schedule; busy[s] = end of device s's last op.  kJump: a trip
// in the steady part maps the state (F, B; busy = B there) to a max of
// (component + constant) terms, so once a steady trip advances every
// component by one constant lam the later steady trips do too, and they are
// taken in one step (the argument of the plain pipeline's shortcut).
template <int S, int v, typename V, bool kJump>
__device__ __forceinline__ void il_pipe(const V (&f)[S * v], const V (&b)[S * v], const V (&c)[S], uint32_t M,
                                        V (&busy)[S], int& skipped) {
  constexpr int NV = S * v, W0 = 2 * (S - 1) + (v - 1) * S;
  const int n = (int)M * v, steps = n + W0;
  V F[S], B[S], pF[S], pB[S];
#pragma unroll
  for (int s = 0; s < S; ++s) F[s] = B[s] = busy[s] = pF[s] = pB[s] = 0;
  skipped = 0;
  bool prev_steady = false;
  for (int t0 = 0; t0 < steps; t0 += NV) {
    if (t0 >= W0 && t0 + NV <= n) {
      if (kJump) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          pF[s] = F[s];
          pB[s] = B[s];
        }
      }
      il_trip<S, v, V, false>(t0, n, f, b, c, F, B, busy);
      if (kJump && prev_steady) {
        const V lam = B[0] - pB[0];
        bool same = true;
#pragma unroll
        for (int s = 0; s < S; ++s) same = same && F[s] - pF[s] == lam && B[s] - pB[s] == lam;
        const int r = (n - (t0 + NV)) / NV;
        if (same && r > 0) {
          const V k = (V)r * lam;
#pragma unroll
          for (int s = 0; s < S; ++s) {
            F[s] += k;
            B[s] += k;
            busy[s] += k;
          }
          t0 += r * NV;
          skipped += r;
        }
      }
      prev_steady = true;
    } else {
      il_trip<S, v, V, true>(t0, n, f, b, c, F, B, busy);
      prev_steady = false;
    }
  }
}

// Layers on device s: the sum over its chunks.
template <int S, int v>
__device__ __forceinline__ uint32_t il_device_ns(const Plan& p, int s) {
  uint32_t ns = 0;
#pragma unroll
  for (int j = 0; j < v; ++j) {
    const int vs = j * S + s;
    ns += cut_at(p, vs) - (vs ? cut_at(p, vs - 1) : 0);
  }
  return ns;
}

// The iteration time of one interleaved pipeline: the latest device end
// plus that device's DP sync over the parameters of all its chunks.
template <int S, int v, int kMode, typename V>
__device__ __forceinline__ V il_tail(const Tab& t, const Hot<kMode>& h, const Plan& p, const V (&busy)[S]) {
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> p.epl);
  V T = 0;
#pragma unroll
  for (int s = 0; s < S; ++s) T = vmax(T, busy[s] + (V)stage_dp(t, h, p, s, il_device_ns<S, v>(p, s), rp, rpe));
  return T;
}

template <int S, int v, int kMode, typename V, bool kJump>
__device__ __forceinline__ V il_time(const Tab& t, const Hot<kMode>& h, const Plan& p, int& skipped) {
  V f[S * v], b[S * v], c[S], busy[S];
  il_setup<S, v, kMode, V>(t, h, p, f, b, c);
  il_pipe<S, v, V, kJump>(f, b, c, class_mb(p), busy, skipped);
  return il_tail<S, v, kMode, V>(t, h, p, busy);
}

// Stage records of an interleaved pipeline: {forward, backward, hop, sync}
// per virtual stage; hop and sync only in the first S records (per device).
template <int S, int v>
__device__ __forceinline__ void il_records(const Tab& t, const Hot<2>& h, const Plan& p, uint64_t* o) {
  uint64_t f[S * v], b[S * v], c[S];
  il_setup<S, v, 2, uint64_t>(t, h, p, f, b, c);
  const double rp = 1.0 / (double)p.psum, rpe = 1.0 / (double)(p.psum >> p.epl);
#pragma unroll
  for (int vs = 0; vs < S * v; ++vs) {
    o[vs * kRecWords + 0] = f[vs];
    o[vs * kRecWords + 1] = b[vs];
    o[vs * kRecWords + 2] = vs < S ? c[vs < S ? vs : 0] : 0;
    o[vs * kRecWords + 3] = vs < S ? stage_dp(t, h, p, vs, il_device_ns<S, v>(p, vs < S ? vs : 0), rp, rpe) : 0;
  }
}

template <int S, int v, int kMode>
__device__ __forceinline__ void eval_il(const Tab& t, const Hot<kMode>& h, const EvalBufs& e, uint32_t slot) {
  double busy[S];
  int skipped;
  {
    double f[S * v], b[S * v], c[S];
    uint32_t M;
    {
      const Plan p = load_plan<false>(e.packed, e.pcut, slot);
      il_setup<S, v, kMode, double>(t, h, p, f, b, c);
      M = class_mb(p);
    }
    il_pipe<S, v, double, true>(f, b, c, M, busy, skipped);
  }
  // the tail reads the plan again (as eval_one does) rather than keeping it
  // in registers through the recurrence
  const uint32_t slot2 = __shfl(slot, (int)(threadIdx.x & 63u));
  const double T = il_tail<S, v, kMode, double>(t, h, load_plan<false>(e.packed, e.pcut, slot2), busy);
  if (T < kExact) atomicMax((unsigned long long*)&e.out[slot >> 2], (unsigned long long)T);
  else e.ovf[atomicAdd(&e.ctr[0], 1u)] = slot;
}

// Blocks of four waves share one LDS copy of the table image.
constexpr uint32_t kEvalThreads = 256;

// The grid is capped at a few times the blocks that fit at once (a launch
// over the whole chunk would mostly start blocks past the group's range,
// each holding a full LDS allocation); the waves of the grid take the
// group's 64-pipeline tiles in a fixed stride, heaviest tiles first.
template <int GRP, int kMode, bool kHet>
__global__ void __launch_bounds__(kEvalThreads) k_eval(Tab t, EvalBufs e) {
  constexpr int kTop = kMaxStages - 4 * GRP;   // stage counts kTop-3 .. kTop
  extern __shared__ uint4 lds[];
  const uint32_t lo = e.sstart[4 * GRP], hi = e.sstart[4 * GRP + 4];
  if (lo + blockIdx.x * kEvalThreads >= hi) return;   // the whole block, before any barrier
  fill_lds<kMode>(t, lds);
  const Hot<kMode> h(t, lds);
  const uint32_t stride = gridDim.x * kEvalThreads;
  // the wavefront's row of the plan-sorted groups' LDS exchange area
  double* xw = nullptr;
  uint32_t* bw = nullptr;   // and its stage-placement cache, when the group has one
  if constexpr (!kHet) {
    char* const x0 = (char*)lds + (kMode < 2 ? t.lds_bytes : 0);
    xw = (double*)x0 + (threadIdx.x >> 6) * xchg_wave(GRP);
    if (GRP < 2 && ((t.bcache >> GRP) & 1))
      bw = (uint32_t*)(x0 + xchg_bytes(GRP)) + (threadIdx.x >> 6) * bcache_words(GRP);
  }
  for (uint32_t base = lo + blockIdx.x * kEvalThreads + (threadIdx.x & ~63u); base < hi; base += stride) {
    const uint32_t pos = base + (threadIdx.x & 63u);
    bool pending = pos < hi;
    const uint32_t slot = pending ? e.ids[pos] : 0;
    pending = pending && slot != kNoSlot;   // padding lanes of plan-sorted groups
    const uint32_t hdr = !pending || kHet ? 0 : e.packed[slot >> 2].hdr;
    const uint32_t S = !pending ? 0 : kHet ? e.meta[slot] & 31 : ((hdr >> 4) & 15) + 1;
    if constexpr (!kHet) {
      // overlap and zero-bubble plans go to the variant pass: the wavefront
      // (one stage count: the plan-sorted groups are padded to whole
      // wavefronts) takes one 64-slot tile and every lane writes its own
      // position, the slot of an overlap or zero-bubble plan or kNoSlot, so
      // that the tile keeps its plans' lanes together; the lane that takes
      // the tile is the one readfirstlane reads.  That needs every lane of
      // the wavefront here, which the loop's single uniform latch gives; if
      // a compiler ever split the wavefront at this point, the tile would
      // have holes, so a partial wavefront hands such lanes to the deferred
      // lists instead (whole loop per lane, plans need not stay whole there).
      const bool var = pending && (((hdr >> 13) & 1) | ((hdr >> 16) & 1));
      const uint64_t vb = __ballot(var);
      if (vb) {
        if (__ballot(1) == ~0ull) {
          const uint32_t Sv = __builtin_amdgcn_readfirstlane(__shfl(S, __ffsll((unsigned long long)vb) - 1));
          uint32_t tile = 0;
          if ((threadIdx.x & 63u) == 0) tile = atomicAdd(&e.ctr[kVariantCtr + kMaxStages - Sv], 64u);
          tile = __builtin_amdgcn_readfirstlane(tile);
          e.vlist[e.sstart[kMaxStages - Sv] + tile + (threadIdx.x & 63u)] = var ? slot : kNoSlot;
        } else if (var) {
          e.deferred[e.sstart[kMaxStages - S] + atomicAdd(&e.ctr[1 + kMaxStages - S], 1u)] = slot;
        }
        pending = pending && !var;
      }
    }
    // one pass per distinct stage count present in the wavefront (usually one)
    while (true) {
      const uint64_t live = __ballot(pending);
      if (!live) break;
      const uint32_t S0 = __builtin_amdgcn_readfirstlane(__shfl(S, __ffsll((unsigned long long)live) - 1));
      if (pending && S == S0) {
        if (S0 == kTop) eval_one<kTop, false, kMode, kHet>(t, h, e, slot, xw, bw);
        else if (S0 == kTop - 1) eval_one<kTop - 1, false, kMode, kHet>(t, h, e, slot, xw, bw);
        else if (S0 == kTop - 2) eval_one<kTop - 2, false, kMode, kHet>(t, h, e, slot, xw, bw);
        else eval_one<kTop - 3, false, kMode, kHet>(t, h, e, slot, xw, bw);
        pending = false;
      }
    }
  }
}

// Interleaved pipelines (shared layout) of one 64-pipeline tile starting at
// sorted id `base` (ids below hi): one pass per (S, v) present in the tile.
template <int kMode>
__device__ __forceinline__ void il_tile(const Tab& t, const Hot<kMode>& h, const EvalBufs& e, uint32_t base,
                                        uint32_t hi) {
  const uint32_t pos = base + (threadIdx.x & 63u);
  bool pending = pos < hi;
  const uint32_t slot = pending ? e.ids[pos] : 0;
  const uint32_t m = pending ? e.meta[slot] : 0;
  const uint32_t key = il_shape(m & 31, (m >> 24) + 1);
  while (true) {
    const uint64_t live = __ballot(pending);
    if (!live) break;
    const uint32_t k0 = __builtin_amdgcn_readfirstlane(__shfl(key, __ffsll((unsigned long long)live) - 1));
    if (pending && key == k0) {
      switch (k0) {
#define X(S_, V_)                          \
  case S_ | (V_ - 1) << 5:                 \
    eval_il<S_, V_, kMode>(t, h, e, slot); \
    break;
        HETSIM_IL_SHAPES(X)
#undef X
        default: break;
      }
      pending = false;
    }
  }
}

// Deferred pipelines of every stage count in one launch, so that the long
// serial chains of the different stage counts overlap.  Tiles of 64 are
// dealt round-robin to the waves of the grid: first the interleaved
// pipelines (shared layout; sorted ids [sstart[16], sstart[16 + 21]), so a
// tile mostly holds one (S, v) and one micro-batch count), then the
// deferred S-stage pipelines at [sstart[16 - S], + ctr[1 + 16 - S]), tile q
// located by walking the sixteen list lengths (16 stages first).  The Tab
// is read from its copy in device memory: this kernel holds every pipeline
// kind's code, and with the Tab as a by-value argument the compiler copied
// the whole argument block to private memory in every wave.
template <int kMode, bool kHet>
__global__ void __launch_bounds__(kEvalThreads) k_deferred(const Tab* __restrict__ tp, EvalBufs e) {
  const Tab& t = *tp;
  extern __shared__ uint4 lds[];
  fill_lds<kMode>(t, lds);
  const Hot<kMode> h(t, lds);
  const uint32_t waves = gridDim.x * (kEvalThreads / 64);
  const uint32_t il_lo = kHet ? 0 : e.sstart[kMaxStages], il_hi = kHet ? 0 : e.sstart[kMaxStages + kIlGroups];
  const uint32_t il_tiles = (il_hi - il_lo + 63) >> 6;
  for (uint32_t q = blockIdx.x * (kEvalThreads / 64) + (threadIdx.x >> 6);; q += waves) {
    if (!kHet && q < il_tiles) {
      il_tile<kMode>(t, h, e, il_lo + q * 64u, il_hi);
      continue;
    }
    uint32_t j = 0, before = il_tiles, nt = 0;
    for (; j < kMaxStages; ++j) {
      nt = (e.ctr[1 + j] + 63) >> 6;
      if (q < before + nt) break;
      before += nt;
    }
    if (j == kMaxStages) return;
    const uint32_t off = (q - before) * 64u + (threadIdx.x & 63u);
    if (off >= e.ctr[1 + j]) continue;
    const uint32_t slot = e.vlist[e.sstart[j] + off];   // the deferred list, sorted
    switch (kMaxStages - j) {
      case 1: eval_deferred<1, kMode, kHet>(t, h, e, slot); break;
      case 2: eval_deferred<2, kMode, kHet>(t, h, e, slot); break;
      case 3: eval_deferred<3, kMode, kHet>(t, h, e, slot); break;
      case 4: eval_deferred<4, kMode, kHet>(t, h, e, slot); break;
      case 5: eval_deferred<5, kMode, kHet>(t, h, e, slot); break;
      case 6: eval_deferred<6, kMode, kHet>(t, h, e, slot); break;
      case 7: eval_deferred<7, kMode, kHet>(t, h, e, slot); break;
      case 8: eval_deferred<8, kMode, kHet>(t, h, e, slot); break;
      case 9: eval_deferred<9, kMode, kHet>(t, h, e, slot); break;
      case 10: eval_deferred<10, kMode, kHet>(t, h, e, slot); break;
      case 11: eval_deferred<11, kMode, kHet>(t, h, e, slot); break;
      case 12: eval_deferred<12, kMode, kHet>(t, h, e, slot); break;
      case 13: eval_deferred<13, kMode, kHet>(t, h, e, slot); break;
      case 14: eval_deferred<14, kMode, kHet>(t, h, e, slot); break;
      case 15: eval_deferred<15, kMode, kHet>(t, h, e, slot); break;
      default: eval_deferred<16, kMode, kHet>(t, h, e, slot); break;
    }
  }
}

// Overlap and zero-bubble pipelines of the four stage counts of group GRP
// (as k_eval's groups), taken from the tiles the first pass filled: the
// S-stage tiles start at sstart[16 - S] and take ctr[kVariantCtr + 16 - S]
// slots, each tile one first-pass wavefront's lanes (plans whole, kNoSlot
// elsewhere), dealt round-robin to the waves of the grid.  The Tab is read from its copy
// in device memory, as in k_deferred.  A block with no tile returns before
// touching LDS, so a launch over empty lists costs next to nothing.
template <int GRP, int kMode>
__global__ void __launch_bounds__(kEvalThreads) k_variant(const Tab* __restrict__ tp, EvalBufs e) {
  constexpr int kTop = kMaxStages - 4 * GRP;   // stage counts kTop-3 .. kTop
  const uint32_t c0 = e.ctr[kVariantCtr + kMaxStages - kTop], c1 = e.ctr[kVariantCtr + kMaxStages - kTop + 1];
  const uint32_t c2 = e.ctr[kVariantCtr + kMaxStages - kTop + 2], c3 = e.ctr[kVariantCtr + kMaxStages - kTop + 3];
  // first tile of each list
  const uint32_t q1 = (c0 + 63) >> 6, q2 = q1 + ((c1 + 63) >> 6), q3 = q2 + ((c2 + 63) >> 6);
  const uint32_t tiles = q3 + ((c3 + 63) >> 6);
  const uint32_t wpb = kEvalThreads / 64;
  if (blockIdx.x * wpb >= tiles) return;   // the whole block, before any barrier
  const Tab& t = *tp;
  extern __shared__ uint4 lds[];
  fill_lds<kMode>(t, lds);
  const Hot<kMode> h(t, lds);
  const uint32_t waves = gridDim.x * wpb;
  // the wavefront's row of the zero-bubble plans' DP exchange area (as k_eval's)
  double* xw = (double*)((char*)lds + (kMode < 2 ? t.lds_bytes : 0)) + (threadIdx.x >> 6) * xchg_wave(GRP);
  for (uint32_t q = blockIdx.x * wpb + (threadIdx.x >> 6); q < tiles; q += waves) {
    const uint32_t j = (q >= q1) + (q >= q2) + (q >= q3);
    const uint32_t first = j == 0 ? 0 : j == 1 ? q1 : j == 2 ? q2 : q3;
    const uint32_t cnt = j == 0 ? c0 : j == 1 ? c1 : j == 2 ? c2 : c3;
    const uint32_t off = (q - first) * 64u + (threadIdx.x & 63u);
    if (off >= cnt) continue;
    const uint32_t S = kTop - j;
    const uint32_t slot = e.vlist[e.sstart[kMaxStages - S] + off];
    if (slot == kNoSlot) continue;
    if (j == 0) eval_variant<kTop, kMode>(t, h, e, slot, xw);
    else if (j == 1) eval_variant<kTop - 1, kMode>(t, h, e, slot, xw);
    else if (j == 2) eval_variant<kTop - 2, kMode>(t, h, e, slot, xw);
    else eval_variant<kTop - 3, kMode>(t, h, e, slot, xw);
  }
}

// Pipelines whose fp64 time reached 2^53 ps, again in u64 (exact below 2^64).
// zb: the zero-bubble order, W[s] each stage's weight-gradient pass.
template <int S>
__device__ __forceinline__ uint64_t redo_one(const StageRec& R, const uint64_t (&W)[kMaxStages], bool zb,
                                             uint32_t M) {
  uint64_t f[S], b[S], w[S], c[S], last[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    f[s] = R[s][0];
    w[s] = zb ? W[s] : 0;
    b[s] = R[s][1] - w[s];
    c[s] = R[s][2];
  }
  // the periodic shortcut holds in any exact arithmetic: pairs within the
  // budget, then the rest of the loop in place
  int skipped;
  if (zb) pipe_zb<S, uint64_t, true, true>(f, b, w, c, M, skipped, last);
  else pipe<S, uint64_t, true, true>(f, b, c, M, skipped, last);
  uint64_t T = 0;
#pragma unroll
  for (int s = 0; s < S; ++s) T = vmax(T, last[s] + R[s][3]);
  return T;
}

template <bool kHet>
__global__ void __launch_bounds__(64) k_redo_u64(Tab t, EvalBufs e) {
  const uint32_t n = e.ctr[0];
  for (uint32_t j = blockIdx.x * 64u + threadIdx.x; j < n; j += gridDim.x * 64u) {
    const uint32_t slot = e.ovf[j];
    const Plan p = load_plan<kHet>(e.packed, e.pcut, slot);
    const uint32_t S = p.S, M = class_mb(p);
    const Hot<2> h(t, nullptr);
    if (!kHet && p.v > 1) {
      uint64_t r = 0;
      int skipped;
      switch (il_shape(S, p.v)) {
#define X(S_, V_)                                                    \
  case S_ | (V_ - 1) << 5:                                           \
    r = il_time<S_, V_, 2, uint64_t, true>(t, h, p, skipped);        \
    break;
        HETSIM_IL_SHAPES(X)
#undef X
        default: break;
      }
      atomicMax((unsigned long long*)&e.out[slot >> 2], (unsigned long long)r);
      continue;
    }
    StageRec R;
    uint64_t W[kMaxStages];
    const bool w = !kHet && p.zb;
    RecSink sink{R, W};
    class_setup<2, kHet>(t, h, p, slot & 3, sink, kHet ? e.pcut + (slot & ~3u) : nullptr);
    uint64_t r;
    switch (S) {
      case 1: r = redo_one<1>(R, W, w, M); break;
      case 2: r = redo_one<2>(R, W, w, M); break;
      case 3: r = redo_one<3>(R, W, w, M); break;
      case 4: r = redo_one<4>(R, W, w, M); break;
      case 5: r = redo_one<5>(R, W, w, M); break;
      case 6: r = redo_one<6>(R, W, w, M); break;
      case 7: r = redo_one<7>(R, W, w, M); break;
      case 8: r = redo_one<8>(R, W, w, M); break;
      case 9: r = redo_one<9>(R, W, w, M); break;
      case 10: r = redo_one<10>(R, W, w, M); break;
      case 11: r = redo_one<11>(R, W, w, M); break;
      case 12: r = redo_one<12>(R, W, w, M); break;
      case 13: r = redo_one<13>(R, W, w, M); break;
      case 14: r = redo_one<14>(R, W, w, M); break;
      case 15: r = redo_one<15>(R, W, w, M); break;
      default: r = redo_one<16>(R, W, w, M); break;
    }
    atomicMax((unsigned long long*)&e.out[slot >> 2], (unsigned long long)r);
  }
}
}  // namespace hetsim
