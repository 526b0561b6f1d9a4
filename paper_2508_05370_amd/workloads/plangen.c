/*
 * plangen.c -- seeded synthetic candidate-plan generator.
 *
 * Input generation only: it draws plan descriptors (parallel degrees, a
 * non-uniform layer split, replica classes with device types and a
 * non-uniform micro-batch split) and computes no time.  Both the HIP path
 * and the CPU oracle consume its output.
 *
 * Randomness: SplitMix64 (Steele, Lea, Flood, OOPSLA 2014) used
 * counter-based: draw(seed, c) = mix(seed + (c + 1) * 0x9E3779B97F4A7C15),
 * with counter c = plan_index * 4096 + draw_number, so every plan is
 * reproducible on its own and generation parallelises by index.
 *
 * Plan layout (structure of arrays, plane stride `stride`):
 *   hdr[i]            tp_log2:2 | ep_log2:2 | (pp-1):4 | (G-1):2 | zero:1 | mbs_idx:2 | 0:19
 *   cut[s*stride+i]   cumulative layer end of stage s (u8)
 *   cls[c*stride+i]   replicas (low 16 bits) | micro-batches (high 16 bits)
 *   types[c*stride+i] 4-bit device type of stage s in bits [4s, 4s+4)
 */
#include <stdint.h>
#include <string.h>
#include <pthread.h>

static uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
uint64_t plangen_draw(uint64_t seed, uint64_t counter) { return mix(seed + (counter + 1) * 0x9E3779B97F4A7C15ull); }

typedef struct { uint64_t seed, i, d; } rng;
static uint64_t next(rng* r) { return plangen_draw(r->seed, r->i * 4096 + r->d++); }
/* uniform integer in [lo, hi] */
static uint64_t uni(rng* r, uint64_t lo, uint64_t hi) { return lo + next(r) % (hi - lo + 1); }

typedef struct {
  uint64_t seed;
  uint32_t L;            /* layers */
  uint32_t K;            /* device types */
  uint32_t cap[16];      /* devices per type */
  uint32_t batches;      /* micro-batches per iteration (global batch / micro-batch size) */
  uint32_t experts;      /* 0 = dense (EP fixed to 1) */
} pg_params;

static void gen_one(const pg_params* P, uint64_t i, uint32_t* hdr, uint8_t* cut, uint32_t* cls, uint64_t* types,
                    int64_t stride, int64_t slot) {
  rng r = {P->seed, i, 0};
  uint32_t tpl = 0, pp = 1, epl = 0, G = 0, zero = 0;
  uint32_t reps[4] = {0}, nmb[4] = {0};
  uint64_t tv[4] = {0};
  uint32_t sumreps = 0;
  for (int attempt = 0; attempt < 16 && G == 0; ++attempt) {
    r.d = (uint64_t)attempt * 256;
    tpl = (uint32_t)uni(&r, 0, 3);
    pp = (uint32_t)uni(&r, 1, P->L < 16 ? P->L : 16);   /* at most one stage per layer */
    epl = 0;
    if (P->experts) {
      epl = (uint32_t)uni(&r, 0, 3);
      while ((1u << epl) > P->experts || P->experts % (1u << epl)) --epl;
    }
    uint32_t want = (uint32_t)uni(&r, 1, 4);
    zero = (uint32_t)uni(&r, 0, 1);
    uint32_t tp = 1u << tpl, ep = 1u << epl;
    uint32_t left[16];
    memcpy(left, P->cap, sizeof(left));
    sumreps = 0;
    for (uint32_t c = 0; c < want; ++c) {
      uint32_t cnt[16] = {0};
      uint64_t t = 0;
      for (uint32_t s = 0; s < pp; ++s) {
        uint64_t k = uni(&r, 0, P->K - 1);
        t |= k << (4 * s);
        cnt[k]++;
      }
      uint32_t maxr = 0xffffffffu;
      for (uint32_t k = 0; k < P->K; ++k)
        if (cnt[k]) { uint32_t m = left[k] / (cnt[k] * tp); if (m < maxr) maxr = m; }
      if (maxr > P->batches - sumreps) maxr = P->batches - sumreps;
      if (maxr > 0xffff) maxr = 0xffff;
      maxr = maxr / ep * ep;
      if (maxr < ep) break;
      uint32_t rr = ep * (uint32_t)uni(&r, 1, maxr / ep);
      for (uint32_t k = 0; k < P->K; ++k) left[k] -= rr * cnt[k] * tp;
      reps[c] = rr; tv[c] = t; sumreps += rr; G = c + 1;
    }
    if (G == 0 && attempt == 15) {      /* give up: emit a plan that fails the capacity check */
      G = 1; reps[0] = ep; tv[0] = 0; sumreps = ep;
      if (sumreps > P->batches) sumreps = P->batches;
    }
  }
  /* non-uniform layer split: pp-1 distinct cut points in [1, L-1], sorted */
  uint8_t pts[256];
  for (uint32_t l = 1; l < P->L; ++l) pts[l - 1] = (uint8_t)l;
  r.d = 16 * 256;
  for (uint32_t j = 0; j + 1 < pp; ++j) {
    uint32_t pick = j + (uint32_t)uni(&r, 0, P->L - 2 - j);
    uint8_t tmp = pts[j]; pts[j] = pts[pick]; pts[pick] = tmp;
  }
  for (uint32_t j = 1; j + 1 < pp; ++j) {         /* insertion sort of the chosen points */
    uint8_t v = pts[j]; int q = (int)j - 1;
    while (q >= 0 && pts[q] > v) { pts[q + 1] = pts[q]; --q; }
    pts[q + 1] = v;
  }
  for (uint32_t s = 0; s < 16; ++s) cut[s * stride + slot] = 0;
  for (uint32_t s = 0; s + 1 < pp; ++s) cut[s * stride + slot] = pts[s];
  cut[(pp - 1) * stride + slot] = (uint8_t)P->L;
  /* non-uniform batch split: every replica gets one micro-batch, the rest by random weights */
  uint32_t extra = P->batches > sumreps ? P->batches - sumreps : 0;
  uint64_t w[4], W = 0;
  for (uint32_t c = 0; c < G; ++c) { w[c] = uni(&r, 1, 1000); W += w[c]; }
  uint32_t given = 0;
  for (uint32_t c = 1; c < G; ++c) { uint32_t x = (uint32_t)((uint64_t)extra * w[c] / W); nmb[c] = reps[c] + x; given += x; }
  nmb[0] = reps[0] + (extra - given);
  for (uint32_t c = 0; c < 4; ++c) {
    cls[c * stride + slot] = c < G ? (reps[c] & 0xffff) | ((nmb[c] & 0xffff) << 16) : 0;
    types[c * stride + slot] = c < G ? tv[c] : 0;
  }
  hdr[slot] = tpl | (epl << 2) | ((pp - 1) << 4) | ((G - 1) << 8) | (zero << 10);
}

typedef struct {
  const pg_params* P; uint64_t first; int64_t lo, hi, stride;
  uint32_t* hdr; uint8_t* cut; uint32_t* cls; uint64_t* types;
} pg_job;

static void* run(void* a) {
  pg_job* j = (pg_job*)a;
  for (int64_t s = j->lo; s < j->hi; ++s) gen_one(j->P, j->first + (uint64_t)s, j->hdr, j->cut, j->cls, j->types, j->stride, s);
  return 0;
}

/* Plans first .. first+n-1 into slots 0 .. n-1 of the given planes. */
void plangen_random(const pg_params* P, uint64_t first, int64_t n, uint32_t* hdr, uint8_t* cut, uint32_t* cls,
                    uint64_t* types, int64_t stride, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  pthread_t th[64];
  pg_job jobs[64];
  for (int t = 0; t < nthreads; ++t) {
    pg_job j = {P, first, n * t / nthreads, n * (t + 1) / nthreads, stride, hdr, cut, cls, types};
    jobs[t] = j;
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], 0, run, &jobs[t]);
  run(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], 0);
}

/* ------------------------------------------------------------------ */
/* plans with a per-class layout: every replica class draws its own TP
 * degree, pipeline depth and layer split (per-class planes):
 *   chdr[i]                    byte c = tp_log2:2 | (pp_c-1):4 | 0:2
 *   ccut[(c*16+s)*stride+i]    cumulative layer end of stage s of class c
 * and hdr carries only ep_log2, G-1, zero (TP and PP fields 0). */
static void gen_one_het(const pg_params* P, uint64_t i, uint32_t* hdr, uint8_t* ccut, uint32_t* cls,
                        uint64_t* types, uint32_t* chdr, int64_t stride, int64_t slot) {
  rng r = {P->seed, i, 0};
  uint32_t tpl[4] = {0}, pp[4] = {1, 1, 1, 1}, epl = 0, G = 0, zero = 0;
  uint32_t reps[4] = {0}, nmb[4] = {0};
  uint64_t tv[4] = {0};
  uint32_t sumreps = 0;
  for (int attempt = 0; attempt < 16 && G == 0; ++attempt) {
    r.d = (uint64_t)attempt * 256;
    epl = 0;
    if (P->experts) {
      epl = (uint32_t)uni(&r, 0, 3);
      while ((1u << epl) > P->experts || P->experts % (1u << epl)) --epl;
    }
    uint32_t want = (uint32_t)uni(&r, 1, 4);
    zero = (uint32_t)uni(&r, 0, 1);
    uint32_t ep = 1u << epl;
    uint32_t left[16];
    memcpy(left, P->cap, sizeof(left));
    sumreps = 0;
    for (uint32_t c = 0; c < want; ++c) {
      tpl[c] = (uint32_t)uni(&r, 0, 3);
      pp[c] = (uint32_t)uni(&r, 1, P->L < 16 ? P->L : 16);
      uint32_t tp = 1u << tpl[c];
      uint32_t cnt[16] = {0};
      uint64_t t = 0;
      for (uint32_t s = 0; s < pp[c]; ++s) {
        uint64_t k = uni(&r, 0, P->K - 1);
        t |= k << (4 * s);
        cnt[k]++;
      }
      uint32_t maxr = 0xffffffffu;
      for (uint32_t k = 0; k < P->K; ++k)
        if (cnt[k]) { uint32_t m = left[k] / (cnt[k] * tp); if (m < maxr) maxr = m; }
      if (maxr > P->batches - sumreps) maxr = P->batches - sumreps;
      if (maxr > 0xffff) maxr = 0xffff;
      maxr = maxr / ep * ep;
      if (maxr < ep) break;
      uint32_t rr = ep * (uint32_t)uni(&r, 1, maxr / ep);
      for (uint32_t k = 0; k < P->K; ++k) left[k] -= rr * cnt[k] * tp;
      reps[c] = rr; tv[c] = t; sumreps += rr; G = c + 1;
    }
    if (G == 0 && attempt == 15) {      /* give up: emit a plan that fails the capacity check */
      G = 1; reps[0] = ep; tv[0] = 0; sumreps = ep; tpl[0] = 0; pp[0] = 1;
      if (sumreps > P->batches) sumreps = P->batches;
    }
  }
  for (uint32_t c = 0; c < 4; ++c) {
    for (uint32_t s = 0; s < 16; ++s) ccut[(c * 16 + s) * stride + slot] = 0;
    if (c >= G) continue;
    /* this class's layer split: pp-1 distinct cut points in [1, L-1], sorted */
    uint8_t pts[256];
    for (uint32_t l = 1; l < P->L; ++l) pts[l - 1] = (uint8_t)l;
    r.d = 16 * 256 + c * 64;
    for (uint32_t j = 0; j + 1 < pp[c]; ++j) {
      uint32_t pick = j + (uint32_t)uni(&r, 0, P->L - 2 - j);
      uint8_t tmp = pts[j]; pts[j] = pts[pick]; pts[pick] = tmp;
    }
    for (uint32_t j = 1; j + 1 < pp[c]; ++j) {
      uint8_t v = pts[j]; int q = (int)j - 1;
      while (q >= 0 && pts[q] > v) { pts[q + 1] = pts[q]; --q; }
      pts[q + 1] = v;
    }
    for (uint32_t s = 0; s + 1 < pp[c]; ++s) ccut[(c * 16 + s) * stride + slot] = pts[s];
    ccut[(c * 16 + pp[c] - 1) * stride + slot] = (uint8_t)P->L;
  }
  r.d = 16 * 256 + 4 * 64;
  uint32_t extra = P->batches > sumreps ? P->batches - sumreps : 0;
  uint64_t w[4], W = 0;
  for (uint32_t c = 0; c < G; ++c) { w[c] = uni(&r, 1, 1000); W += w[c]; }
  uint32_t given = 0;
  for (uint32_t c = 1; c < G; ++c) { uint32_t x = (uint32_t)((uint64_t)extra * w[c] / W); nmb[c] = reps[c] + x; given += x; }
  nmb[0] = reps[0] + (extra - given);
  uint32_t ch = 0;
  for (uint32_t c = 0; c < 4; ++c) {
    cls[c * stride + slot] = c < G ? (reps[c] & 0xffff) | ((nmb[c] & 0xffff) << 16) : 0;
    types[c * stride + slot] = c < G ? tv[c] : 0;
    if (c < G) ch |= (tpl[c] | ((pp[c] - 1) << 2)) << (8 * c);
  }
  chdr[slot] = ch;
  hdr[slot] = (epl << 2) | ((G - 1) << 8) | (zero << 10);
}

typedef struct {
  const pg_params* P; uint64_t first; int64_t lo, hi, stride;
  uint32_t* hdr; uint8_t* ccut; uint32_t* cls; uint64_t* types; uint32_t* chdr;
} pg_job_het;

static void* run_het(void* a) {
  pg_job_het* j = (pg_job_het*)a;
  for (int64_t s = j->lo; s < j->hi; ++s)
    gen_one_het(j->P, j->first + (uint64_t)s, j->hdr, j->ccut, j->cls, j->types, j->chdr, j->stride, s);
  return 0;
}

/* Per-class-layout plans first .. first+n-1 into slots 0 .. n-1. */
void plangen_random_het(const pg_params* P, uint64_t first, int64_t n, uint32_t* hdr, uint8_t* ccut, uint32_t* cls,
                        uint64_t* types, uint32_t* chdr, int64_t stride, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  pthread_t th[64];
  pg_job_het jobs[64];
  for (int t = 0; t < nthreads; ++t) {
    pg_job_het j = {P, first, n * t / nthreads, n * (t + 1) / nthreads, stride, hdr, ccut, cls, types, chdr};
    jobs[t] = j;
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], 0, run_het, &jobs[t]);
  run_het(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], 0);
}

/* ------------------------------------------------------------------ */
/* interleaved plans: hdr bits 14-15 = v - 1 (v = 2..4 model chunks per
 * device), PP = S devices, S*v virtual-stage cuts; every class runs a
 * micro-batch count per replica M that is a multiple of S and at least 2S. */
static void gen_one_il(const pg_params* P, uint64_t i, uint32_t* hdr, uint8_t* cut, uint32_t* cls, uint64_t* types,
                       int64_t stride, int64_t slot) {
  rng r = {P->seed, i, 0};
  uint32_t tpl = 0, v = 2, S = 2, epl = 0, G = 0, zero = 0;
  uint32_t reps[4] = {0}, nmb[4] = {0};
  uint64_t tv[4] = {0};
  for (int attempt = 0; attempt < 32 && G == 0; ++attempt) {
    r.d = (uint64_t)attempt * 256;
    tpl = (uint32_t)uni(&r, 0, 3);
    v = (uint32_t)uni(&r, 2, 4);
    S = (uint32_t)uni(&r, 2, 16 / v);
    if (S * v > P->L) continue;
    epl = 0;
    if (P->experts) {
      epl = (uint32_t)uni(&r, 0, 3);
      while ((1u << epl) > P->experts || P->experts % (1u << epl)) --epl;
    }
    uint32_t want = (uint32_t)uni(&r, 1, 4);
    zero = (uint32_t)uni(&r, 0, 1);
    uint32_t tp = 1u << tpl, ep = 1u << epl;
    uint32_t left[16];
    memcpy(left, P->cap, sizeof(left));
    /* every replica runs at least 2S micro-batches (2S-1 of them can be short) */
    uint32_t budget = P->batches, g = 0;
    for (uint32_t c = 0; c < want; ++c) {
      uint32_t cnt[16] = {0};
      uint64_t t = 0;
      for (uint32_t s = 0; s < S; ++s) {
        uint64_t k = uni(&r, 0, P->K - 1);
        t |= k << (4 * s);
        cnt[k]++;
      }
      uint32_t maxr = 0xffffffffu;
      for (uint32_t k = 0; k < P->K; ++k)
        if (cnt[k]) { uint32_t m = left[k] / (cnt[k] * tp); if (m < maxr) maxr = m; }
      uint32_t per = 2 * S * 2 - 1;     /* a little more than the minimum per replica */
      if (maxr > budget / per) maxr = budget / per;
      maxr = maxr / ep * ep;
      if (maxr < ep) break;
      uint32_t rr = ep * (uint32_t)uni(&r, 1, maxr / ep);
      for (uint32_t k = 0; k < P->K; ++k) left[k] -= rr * cnt[k] * tp;
      reps[c] = rr; tv[c] = t; budget -= rr * (2 * S - 1) + rr; g = c + 1;
    }
    if (g == 0) continue;
    /* micro-batches: class c runs M_c = S q_c per replica, so it takes between
     * reps (M_c - 1) + 1 and reps M_c of them; raise q until the windows reach
     * the global batch, then fill the windows */
    uint32_t q[4] = {2, 2, 2, 2};
    uint64_t lo_sum = 0, hi_sum = 0;
    for (int guard = 0; guard < 100000; ++guard) {
      lo_sum = hi_sum = 0;
      for (uint32_t c = 0; c < g; ++c) {
        lo_sum += (uint64_t)reps[c] * (S * q[c] - 1) + 1;
        hi_sum += (uint64_t)reps[c] * S * q[c];
      }
      if (hi_sum >= P->batches) break;
      q[uni(&r, 0, g - 1)]++;
    }
    if (lo_sum > P->batches || hi_sum < P->batches) continue;
    uint64_t extra = P->batches - lo_sum;
    for (uint32_t c = 0; c < g; ++c) {
      uint64_t lo = (uint64_t)reps[c] * (S * q[c] - 1) + 1, width = reps[c] - 1;
      uint64_t add = extra < width ? extra : width;
      nmb[c] = (uint32_t)(lo + add);
      extra -= add;
    }
    if (extra) continue;
    G = g;
  }
  if (G == 0) {        /* give up: a plan that fails the micro-batch rule */
    G = 1; reps[0] = 1u << epl; tv[0] = 0; nmb[0] = P->batches; S = 2; v = 2;
  }
  uint8_t pts[256];
  for (uint32_t l = 1; l < P->L; ++l) pts[l - 1] = (uint8_t)l;
  uint32_t V = S * v;
  r.d = 32 * 256;
  for (uint32_t j = 0; j + 1 < V; ++j) {
    uint32_t pick = j + (uint32_t)uni(&r, 0, P->L - 2 - j);
    uint8_t tmp = pts[j]; pts[j] = pts[pick]; pts[pick] = tmp;
  }
  for (uint32_t j = 1; j + 1 < V; ++j) {
    uint8_t vv = pts[j]; int qq = (int)j - 1;
    while (qq >= 0 && pts[qq] > vv) { pts[qq + 1] = pts[qq]; --qq; }
    pts[qq + 1] = vv;
  }
  for (uint32_t s = 0; s < 16; ++s) cut[s * stride + slot] = 0;
  for (uint32_t s = 0; s + 1 < V; ++s) cut[s * stride + slot] = pts[s];
  cut[(V - 1) * stride + slot] = (uint8_t)P->L;
  for (uint32_t c = 0; c < 4; ++c) {
    cls[c * stride + slot] = c < G ? (reps[c] & 0xffff) | ((nmb[c] & 0xffff) << 16) : 0;
    types[c * stride + slot] = c < G ? tv[c] : 0;
  }
  hdr[slot] = tpl | (epl << 2) | ((S - 1) << 4) | ((G - 1) << 8) | (zero << 10) | ((v - 1) << 14);
}

static void* run_il(void* a) {
  pg_job* j = (pg_job*)a;
  for (int64_t s = j->lo; s < j->hi; ++s)
    gen_one_il(j->P, j->first + (uint64_t)s, j->hdr, j->cut, j->cls, j->types, j->stride, s);
  return 0;
}

/* Interleaved plans first .. first+n-1 into slots 0 .. n-1. */
void plangen_random_interleaved(const pg_params* P, uint64_t first, int64_t n, uint32_t* hdr, uint8_t* cut,
                                uint32_t* cls, uint64_t* types, int64_t stride, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 64) nthreads = 64;
  pthread_t th[64];
  pg_job jobs[64];
  for (int t = 0; t < nthreads; ++t) {
    pg_job j = {P, first, n * t / nthreads, n * (t + 1) / nthreads, stride, hdr, cut, cls, types};
    jobs[t] = j;
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], 0, run_il, &jobs[t]);
  run_il(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], 0);
}
