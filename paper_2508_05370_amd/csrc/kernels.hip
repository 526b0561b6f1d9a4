// kernels.hip -- gfx950 kernels of the plan evaluator.
//
// Data flow of one chunk of plans (all in HBM):
//   k_setup    one plan per lane: decode and validate the plan, place every
//              (class, stage) on its device pool, read stage compute from the
//              layer prefix tables, find each group's slowest link with
//              range-max tables, and write per (class, stage) the forward and
//              backward time of one micro-batch, the pipeline hop and the DP
//              sync; counts pipelines per (stages, micro-batches) bucket.
//   k_scan     one block: bucket offsets, longest pipelines first.
//   k_scatter  groups pipeline ids by bucket, so a wavefront runs pipelines of
//              one stage count and similar micro-batch counts.
//   k_pipe     one pipeline per lane: the 1F1B recurrence, unrolled per stage
//              count so that all per-stage state stays in VGPRs; times are
//              integers carried exactly in fp64 (3 VALU ops per schedule
//              node); a pipeline whose time reaches 2^53 ps is redone in u64.
//              The plan's time is the max over its classes (atomic max).
#include <hip/hip_runtime.h>

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
  uint32_t a = tb[(size_t)j * n + lo], b = tb[(size_t)j * n + hi + 1 - (1u << j)];
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

// DP gradient sync of one stage over a ring of p members
__device__ __forceinline__ uint64_t ring_sync(uint32_t p, double rp, uint32_t zero, uint64_t grads, uint64_t params,
                                              uint64_t alpha, uint32_t bq) {
  uint64_t g = div_up(grads, p, rp);
  if (!zero) {
    uint64_t steps = 2ull * (p - 1);
    return steps * alpha + link_ps(steps * g, bq);
  }
  uint64_t steps = p - 1;
  return 2 * steps * alpha + link_ps(steps * g, bq) + link_ps(steps * div_up(params, p, rp), bq);
}

__device__ __host__ __forceinline__ uint32_t m_bucket(uint32_t M) {
  if (M <= 128) return M - 1;
  if (M <= 1152) return 128 + (M - 129) / 16;
  uint32_t b = 192 + (M - 1153) / 256;
  return b > 255 ? 255 : b;
}
// ascending key: more stages first, then more micro-batches first
__device__ __forceinline__ uint32_t bucket_key(uint32_t S, uint32_t M) {
  return (kMaxStages - S) * kBucketsM + (kBucketsM - 1 - m_bucket(M));
}

// ---------------------------------------------------------------- setup
__device__ void setup_plan(const Tab& t, const sim_plans& pl, int64_t i, uint64_t* __restrict__ out,
                           uint64_t* __restrict__ rec, uint32_t* __restrict__ meta, uint32_t* lh) {
  const int64_t st = pl.stride;
  const uint32_t hdr = pl.hdr[i];
  const uint32_t tpl = hdr & 3, epl = (hdr >> 2) & 3, S = ((hdr >> 4) & 15) + 1, G = ((hdr >> 8) & 3) + 1;
  const uint32_t zero = (hdr >> 10) & 1, mi = (hdr >> 11) & 3;
  const uint32_t tp = 1u << tpl, ep = 1u << epl;
  bool ok = (hdr >> 13) == 0 && mi < t.n_mbs && ((t.tp_ok >> tpl) & 1) && ((t.ep_ok >> epl) & 1);

  uint32_t prev = 0;
  for (uint32_t s = 0; s < S; ++s) {
    uint32_t c = pl.cut[s * st + i];
    ok = ok && c > prev;
    prev = c;
  }
  ok = ok && prev == t.L;

  const uint64_t sel = S == 16 ? ~0ull : ((1ull << (4 * S)) - 1);
  uint32_t reps[4], nmb[4];
  uint64_t tv[4];
  uint32_t batch = 0, psum = 0;
#pragma unroll
  for (uint32_t c = 0; c < 4; ++c) {
    reps[c] = 0; nmb[c] = 0; tv[c] = 0;
    if (c < G) {
      uint32_t w = pl.cls[c * st + i];
      reps[c] = w & 0xffff;
      nmb[c] = w >> 16;
      tv[c] = pl.types[c * st + i] & sel;
      ok = ok && reps[c] >= 1 && nmb[c] >= reps[c] && (reps[c] & (ep - 1)) == 0;
      batch += nmb[c] * t.mbs[mi];
      psum += reps[c];
      for (uint32_t s = 0; s < S; ++s) {
        uint32_t k = (uint32_t)(tv[c] >> (4 * s)) & 15;
        ok = ok && k < t.K && t.dpn_log2[k] >= tpl;
      }
    }
  }
  ok = ok && batch == t.gbs;
  for (uint32_t k = 0; ok && k < t.K; ++k) {
    uint32_t need = 0;
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c)
      if (c < G) need += reps[c] * count_type(tv[c], k, sel);
    ok = need * tp <= t.cap[k];
  }
  if (!ok) {
    if (out) out[i] = kInvalid;
    if (meta)
#pragma unroll
      for (uint32_t c = 0; c < 4; ++c) meta[i * 4 + c] = 0;
    return;
  }
  if (out) out[i] = 0;

  const uint64_t act = t.act[mi], act_tp = (act + tp - 1) >> tpl;
  const double rp = 1.0 / (double)psum, rpe = 1.0 / (double)(psum >> epl);
  const size_t L1 = t.L + 1;
  uint64_t* R = rec + (size_t)i * kPlanWords;
  uint32_t pk[4] = {0, 0, 0, 0}, pbase[4] = {0, 0, 0, 0}, pnic[4] = {0, 0, 0, 0}, pin[4] = {0, 0, 0, 0};
  uint32_t lo = 0;
  for (uint32_t s = 0; s < S; ++s) {
    const uint32_t hi = pl.cut[s * st + i], ns = hi - lo;
    bool same = true;
    uint32_t k0 = 0, nmin = 0xffffffffu, nmax = 0, bq_dp = 0;
    uint64_t a_dp = 0;
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c) {
      if (c >= G) continue;
      const uint32_t k = (uint32_t)(tv[c] >> (4 * s)) & 15;
      // canonical packing: this (class, stage) follows everything placed before it in pool k
      uint32_t below = reps[c] * count_type(tv[c], k, (1ull << (4 * s)) - 1);
#pragma unroll
      for (uint32_t c2 = 0; c2 < c; ++c2) below += reps[c2] * count_type(tv[c2], k, sel);
      const uint32_t base = below * tp, nd = reps[c] * tp, dpl = t.dpn_log2[k];
      const uint32_t gnl = t.node_off[k] + (base >> dpl), gnh = t.node_off[k] + ((base + nd - 1) >> dpl);
      const uint32_t bq_in = range_max(t.rm_intra, t.N, gnl, gnh);
      const uint32_t dlo = t.dev_off[k] + base;
      const uint32_t bq_nic = range_max(t.rm_nic, t.D, dlo, dlo + nd - 1);
      const size_t tb = ((((size_t)k * 4 + tpl) * t.n_mbs + mi) * 4 + epl) * L1;
      uint64_t fc = t.pf[tb + hi] - t.pf[tb + lo];
      uint64_t bc = t.pb[tb + hi] - t.pb[tb + lo];
      if (s == 0) {
        fc += t.emb[((size_t)k * t.n_mbs + mi) * 2];
        bc += t.emb[((size_t)k * t.n_mbs + mi) * 2 + 1];
      }
      if (s == S - 1) {
        const size_t hb = (((size_t)k * 4 + tpl) * t.n_mbs + mi) * 2;
        fc += t.head[hb];
        bc += t.head[hb + 1];
      }
      if (tp > 1) {  // TP all-reduces of this stage, exposed in the forward pass
        const uint64_t steps = (uint64_t)(2 * ns + (s == 0)) * 2 * (tp - 1);
        fc += steps * t.a_intra[k] + link_ps(steps * act_tp, bq_in);
      }
      if (t.E && ep > 1) {  // dispatch + combine all-to-all in each pass
        // EP groups are aligned blocks of ep*tp devices: inside a node iff they fit one
        const bool intra = ep * tp <= (1u << dpl);
        const uint64_t alpha = intra ? t.a_intra[k] : 2 * t.a_side[k];
        const uint32_t bq = intra ? bq_in : (bq_nic > t.bq_pcie[k] ? bq_nic : t.bq_pcie[k]);
        const size_t pb = ((size_t)epl * t.n_mbs + mi) * L1;
        const uint64_t e = (uint64_t)ns * 2 * (ep - 1) * alpha + link_ps(2 * (t.pa[pb + hi] - t.pa[pb + lo]), bq);
        fc += e;
        bc += e;
      }
      uint64_t* r = R + (c * kMaxStages + s) * kRecWords;
      r[0] = fc;
      r[1] = bc;
      if (s > 0) {  // hop (s-1) -> s of this class
        // same pool means the two ranges are adjacent: intra iff the pair spans one node
        const bool intra = pk[c] == k && (pbase[c] >> dpl) == ((pbase[c] + (2 * reps[c] - 1) * tp) >> dpl);
        const uint64_t alpha = intra ? t.a_intra[k] : t.a_side[pk[c]] + t.a_side[k];
        uint32_t bq;
        if (intra) {
          bq = pin[c] > bq_in ? pin[c] : bq_in;
        } else {
          uint32_t a = pnic[c] > bq_nic ? pnic[c] : bq_nic;
          uint32_t b = t.bq_pcie[pk[c]] > t.bq_pcie[k] ? t.bq_pcie[pk[c]] : t.bq_pcie[k];
          bq = a > b ? a : b;
        }
        R[(c * kMaxStages + s - 1) * kRecWords + 2] = alpha + link_ps(act, bq);
      }
      pk[c] = k; pbase[c] = base; pnic[c] = bq_nic; pin[c] = bq_in;
      if (c == 0) k0 = k; else same = same && k == k0;
      nmin = gnl < nmin ? gnl : nmin;
      nmax = gnh > nmax ? gnh : nmax;
      const uint32_t bx = bq_nic > t.bq_pcie[k] ? bq_nic : t.bq_pcie[k];
      bq_dp = bx > bq_dp ? bx : bq_dp;
      a_dp = 2 * t.a_side[k] > a_dp ? 2 * t.a_side[k] : a_dp;
    }
    // DP sync of this stage over every replica of every class
    uint64_t tdp = 0;
    if (psum > 1) {
      const bool intra = same && nmin == nmax;
      const uint64_t alpha = intra ? t.a_intra[k0] : a_dp;
      const uint32_t bq = intra ? t.rm_intra[nmin] : bq_dp;
      const uint64_t pd = (uint64_t)ns * t.par_layer[tpl] + (s == 0 ? t.par_embed[tpl] : 0) +
                          (s == S - 1 ? t.par_head[tpl] : 0);
      tdp = ring_sync(psum, rp, zero, t.grad_bytes * pd, t.param_bytes * pd, alpha, bq);
      const uint32_t pe = psum >> epl;
      if (t.E && pe > 1) {
        const uint64_t px = (uint64_t)ns * t.par_expert[tpl][epl];
        tdp += ring_sync(pe, rpe, zero, t.grad_bytes * px, t.param_bytes * px, alpha, bq);
      }
    }
#pragma unroll
    for (uint32_t c = 0; c < 4; ++c)
      if (c < G) R[(c * kMaxStages + s) * kRecWords + 3] = tdp;
    lo = hi;
  }
#pragma unroll
  for (uint32_t c = 0; c < 4; ++c) {
    uint32_t m = 0;
    if (c < G) {
      R[(c * kMaxStages + S - 1) * kRecWords + 2] = 0;
      const uint32_t M = (nmb[c] + reps[c] - 1) / reps[c];
      m = S | (M << 8);
      if (lh) atomicAdd(&lh[bucket_key(S, M)], 1u);
    }
    if (meta) meta[i * 4 + c] = m;
  }
}

__global__ void __launch_bounds__(256) k_setup(Tab t, sim_plans pl, int64_t n, uint64_t* __restrict__ out,
                                               uint64_t* __restrict__ rec, uint32_t* __restrict__ meta,
                                               uint32_t* __restrict__ hist) {
  __shared__ uint32_t lh[kBuckets];
  if (hist) {
    for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x) lh[j] = 0;
    __syncthreads();
  }
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) setup_plan(t, pl, i, out, rec, meta, hist ? lh : nullptr);
  if (hist) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x)
      if (lh[j]) atomicAdd(&hist[j], lh[j]);
  }
}

__global__ void k_fill32(uint32_t* p, uint32_t n, uint32_t v) {
  for (uint32_t j = blockIdx.x * blockDim.x + threadIdx.x; j < n; j += gridDim.x * blockDim.x) p[j] = v;
}

// exclusive scan of the bucket counts; total pipelines into *total
__global__ void __launch_bounds__(1024) k_scan(const uint32_t* __restrict__ hist, uint32_t* __restrict__ cursor,
                                               uint32_t* __restrict__ total) {
  constexpr int kPer = kBuckets / 1024;
  __shared__ uint32_t part[1024];
  uint32_t v[kPer], sum = 0;
  const uint32_t tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < kPer; ++j) { v[j] = hist[tid * kPer + j]; sum += v[j]; }
  part[tid] = sum;
  __syncthreads();
  for (uint32_t off = 1; off < 1024; off <<= 1) {
    uint32_t x = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  uint32_t run = part[tid] - sum;
#pragma unroll
  for (int j = 0; j < kPer; ++j) { cursor[tid * kPer + j] = run; run += v[j]; }
  if (tid == 1023) *total = part[1023];
}

// place every pipeline id at its bucket's next free position
__global__ void __launch_bounds__(256) k_scatter(const uint32_t* __restrict__ meta, uint32_t nslots,
                                                 uint32_t* __restrict__ cursor, uint32_t* __restrict__ ids) {
  constexpr int kPer = 4;
  __shared__ uint32_t lc[kBuckets];
  for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x) lc[j] = 0;
  __syncthreads();
  uint32_t key[kPer], rank[kPer];
  const uint32_t first = blockIdx.x * blockDim.x * kPer + threadIdx.x;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const uint32_t slot = first + j * blockDim.x;
    key[j] = 0xffffffffu;
    if (slot < nslots) {
      const uint32_t m = meta[slot];
      if (m) {
        key[j] = bucket_key(m & 255, m >> 8);
        rank[j] = atomicAdd(&lc[key[j]], 1u);
      }
    }
  }
  __syncthreads();
  for (uint32_t j = threadIdx.x; j < kBuckets; j += blockDim.x)
    if (lc[j]) lc[j] = atomicAdd(&cursor[j], lc[j]);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPer; ++j)
    if (key[j] != 0xffffffffu) ids[lc[key[j]] + rank[j]] = first + j * blockDim.x;
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
template <int S>
__device__ __forceinline__ uint64_t pipe_fp64(const uint64_t* __restrict__ R, uint32_t M) {
  double f[S], b[S], c[S], out_f[S], last[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    f[s] = (double)R[s * kRecWords + 0];
    b[s] = (double)R[s * kRecWords + 1];
    c[s] = (double)R[s * kRecWords + 2];
    out_f[s] = 0.0;
    last[s] = 0.0;
  }
  const int m_ = (int)M;
#pragma unroll
  for (int m = 0; m < S - 1; ++m) {
    if (m < m_) {
#pragma unroll
      for (int s = 0; s < S - 1 - m; ++s) {
        const double st = s == 0 ? last[0] : __builtin_fmax(last[s], out_f[s - 1] + c[s - 1]);
        out_f[s] = st + f[s];
        last[s] = out_f[s];
      }
    }
  }
  const int steady = m_ - (S - 1);
  for (int i = 0; i < steady; ++i) {
#pragma unroll
    for (int s = S - 1; s >= 0; --s) {
      const double st = s == 0 ? last[0] : __builtin_fmax(last[s], out_f[s - 1] + c[s - 1]);
      out_f[s] = st + f[s];
      const double sb = s == S - 1 ? out_f[s] : __builtin_fmax(out_f[s], last[s + 1] + c[s]);
      last[s] = sb + b[s];
    }
  }
#pragma unroll
  for (int tr = 0; tr < S - 1; ++tr) {
    if (tr >= S - 1 - m_) {
#pragma unroll
      for (int s = S - 1; s >= 0; --s) {
        if (s > tr) {
          const double st = __builtin_fmax(last[s], out_f[s - 1] + c[s - 1]);
          out_f[s] = st + f[s];
          const double sb = s == S - 1 ? out_f[s] : __builtin_fmax(out_f[s], last[s + 1] + c[s]);
          last[s] = sb + b[s];
        } else {
          last[s] = (s == S - 1 ? last[s] : __builtin_fmax(last[s], last[s + 1] + c[s])) + b[s];
        }
      }
    }
  }
  double T = 0.0;
#pragma unroll
  for (int s = 0; s < S; ++s) T = __builtin_fmax(T, last[s] + (double)R[s * kRecWords + 3]);
  // integers below 2^53 are exact in fp64; if no value ever reached 2^53 every
  // add was exact, and the result bounds every intermediate value
  return T < 9007199254740992.0 ? (uint64_t)T : kInvalid;
}

// same schedule in u64, for pipelines whose time reaches 2^53 ps
__device__ __noinline__ uint64_t pipe_u64(const uint64_t* __restrict__ R, int S, uint32_t M) {
  uint64_t out_f[kMaxStages], last[kMaxStages];
  for (int s = 0; s < S; ++s) { out_f[s] = 0; last[s] = 0; }
  const int m_ = (int)M;
  auto fwd = [&](int s) {
    uint64_t st = last[s];
    if (s > 0) { uint64_t r = out_f[s - 1] + R[(s - 1) * kRecWords + 2]; st = st > r ? st : r; }
    out_f[s] = st + R[s * kRecWords + 0];
    last[s] = out_f[s];
  };
  auto bwd = [&](int s) {
    uint64_t st = last[s];
    if (s < S - 1) { uint64_t r = last[s + 1] + R[s * kRecWords + 2]; st = st > r ? st : r; }
    last[s] = st + R[s * kRecWords + 1];
  };
  for (int m = 0; m < S - 1 && m < m_; ++m)
    for (int s = 0; s < S - 1 - m; ++s) fwd(s);
  for (int i = 0; i < m_ - (S - 1); ++i)
    for (int s = S - 1; s >= 0; --s) { fwd(s); bwd(s); }
  for (int tr = (S - 1 - m_ > 0 ? S - 1 - m_ : 0); tr < S - 1; ++tr)
    for (int s = S - 1; s >= 0; --s) {
      if (s > tr) fwd(s);
      bwd(s);
    }
  uint64_t T = 0;
  for (int s = 0; s < S; ++s) {
    uint64_t v = last[s] + R[s * kRecWords + 3];
    T = T > v ? T : v;
  }
  return T;
}

template <int S>
__device__ __forceinline__ uint64_t run_pipe(const uint64_t* R, uint32_t M) {
  uint64_t r = pipe_fp64<S>(R, M);
  return r != kInvalid ? r : pipe_u64(R, S, M);
}

__global__ void __launch_bounds__(64) k_pipe(const uint64_t* __restrict__ rec, const uint32_t* __restrict__ meta,
                                             const uint32_t* __restrict__ ids, const uint32_t* __restrict__ total,
                                             uint64_t* __restrict__ out) {
  const uint32_t tot = *total;
  if (blockIdx.x * 64u >= tot) return;
  const uint32_t pos = blockIdx.x * 64u + threadIdx.x;
  bool pending = pos < tot;
  const uint32_t slot = pending ? ids[pos] : 0;
  const uint32_t m = pending ? meta[slot] : 0;
  const uint32_t S = m & 255, M = m >> 8;
  const uint64_t* R = rec + (size_t)(slot >> 2) * kPlanWords + (slot & 3) * (kMaxStages * kRecWords);
  // one pass per distinct stage count present in the wavefront (usually one)
  while (true) {
    const uint64_t live = __ballot(pending);
    if (!live) break;
    const uint32_t S0 = __builtin_amdgcn_readfirstlane(__shfl(S, __ffsll((unsigned long long)live) - 1));
    if (pending && S == S0) {
      uint64_t r;
      switch (S0) {
        case 1: r = run_pipe<1>(R, M); break;
        case 2: r = run_pipe<2>(R, M); break;
        case 3: r = run_pipe<3>(R, M); break;
        case 4: r = run_pipe<4>(R, M); break;
        case 5: r = run_pipe<5>(R, M); break;
        case 6: r = run_pipe<6>(R, M); break;
        case 7: r = run_pipe<7>(R, M); break;
        case 8: r = run_pipe<8>(R, M); break;
        case 9: r = run_pipe<9>(R, M); break;
        case 10: r = run_pipe<10>(R, M); break;
        case 11: r = run_pipe<11>(R, M); break;
        case 12: r = run_pipe<12>(R, M); break;
        case 13: r = run_pipe<13>(R, M); break;
        case 14: r = run_pipe<14>(R, M); break;
        case 15: r = run_pipe<15>(R, M); break;
        default: r = run_pipe<16>(R, M); break;
      }
      atomicMax((unsigned long long*)&out[slot >> 2], (unsigned long long)r);
      pending = false;
    }
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
hipError_t launch_setup(const Tab& t, const sim_plans& p, int64_t n, uint64_t* out, uint64_t* rec, uint32_t* meta,
                        uint32_t* hist, hipStream_t s) {
  k_setup<<<blocks_for(n, 256), 256, 0, s>>>(t, p, n, out, rec, meta, hist);
  return hipGetLastError();
}
hipError_t launch_scan(const uint32_t* hist, uint32_t* cursor, uint32_t* total, hipStream_t s) {
  k_scan<<<1, 1024, 0, s>>>(hist, cursor, total);
  return hipGetLastError();
}
hipError_t launch_scatter(const uint32_t* meta, uint32_t nslots, uint32_t* cursor, uint32_t* ids, hipStream_t s) {
  k_scatter<<<blocks_for(nslots, 256 * 4), 256, 0, s>>>(meta, nslots, cursor, ids);
  return hipGetLastError();
}
hipError_t launch_pipe(const uint64_t* rec, const uint32_t* meta, const uint32_t* ids, const uint32_t* total,
                       uint32_t max_tasks, uint64_t* out, hipStream_t s) {
  k_pipe<<<blocks_for(max_tasks, 64), 64, 0, s>>>(rec, meta, ids, total, out);
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
