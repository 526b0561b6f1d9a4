/*
 * oracle.c -- plain, slow, obviously-correct CPU evaluator of candidate
 * deployment plans for heterogeneous LLM training (arXiv 2508.05370).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference against which the
 * HIP path is checked.  Only tests/, the smoke entry point and the CPU
 * baseline leg of the benchmark may load it.  It shares no code, header,
 * table or constant generator with the HIP library.
 *
 * Every quantity is an unsigned integer; time is picoseconds.  Each step
 * follows the paper's statement of the problem:
 *   - input description: model, framework (device groups, TP/PP/DP degrees,
 *     parallelism-to-device-group mapping) and heterogeneous topology
 *     (Sec. 4.2 "Input Description", Tables 5 and 6);
 *   - a device group (DG) forms one pipeline replica; the DP group spans all
 *     replicas (Sec. 3 "Device grouping");
 *   - non-uniform layer and batch partitioning (Sec. 3 "Non-uniform workload
 *     partitioning");
 *   - exposed communication: TP exposed in forward only, PP in both passes,
 *     DP after the backward pass (Table 1);
 *   - interconnect delay = jumbo frame bits / unidirectional bandwidth, two
 *     PCIe trips for inter-node traffic (Sec. 5 "Interconnect configuration");
 *   - the slowest link or device of a collective sets its time (Sec. 4.1
 *     [C4], Sec. 5 [Q2]);
 *   - parallelism exists to fit the model within device memory (Sec. 2),
 *     and device types differ in capacity (Sec. 3 example, Table 5: A100
 *     40 GB, H100 80 GB): a plan that overflows a device is infeasible;
 *   - device groups may differ in TP degree, layer split and micro-batch
 *     size (Sec. 3); then the gradient sync is preceded by resharding
 *     (Sec. 3 "Resharding", both of its conditions; Sec. 4.1 [C2]).
 * Where the paper is silent the reading used is named R1..R51 in comments;
 * the design notes of the repository list every reading.
 *
 * Parity notes: the recurrence, the collective formulas, the interconnect
 * delays, the parameter counts and the FLOP counts are pinned by tests
 * (closed forms, Table 5, Table 6, Table 1, a brute-force event simulator).
 * The per-op byte accounting of the roofline (R6/R8) has no printed value
 * to compare against: parity unpinned beyond scaling invariants.  The
 * per-class layout (R35-R37) is pinned by its encoding of a shared layout,
 * by classes that do not interact without links, and by the ring closed
 * forms of its segment syncs and its resharding all-gather.  The
 * stored-activation count (R32) is pinned for GPT-shaped layers to
 * Korthikanti et al. 2022; its gated-MLP and MoE terms are parity unpinned
 * beyond the reduction of a one-expert top-1 MoE layer to a gated dense one.
 * The gradient-sync overlap (R38-R40) is pinned by an event queue over the
 * same buckets and by its communication- and compute-bound extremes.
 * Interleaved 1F1B (R41-R43) is pinned by the bubble closed form of
 * Narayanan et al. 2021, an event-driven replay of the same op lists, the
 * per-virtual-stage costs of a plain plan over the same cuts and the ring
 * closed form of its per-device sync; its in-flight activation count (each
 * pass counted at the device's largest chunk) is a bound of this reading,
 * pinned only by its own differences.  Per-class micro-batch sizes and the
 * gradient weighting they trigger (R51) are pinned by Sec. 3's worked example
 * composed by hand from pinned pieces; the weighting's cost itself is a
 * reading with no printed value: parity unpinned beyond that.  Whole plans of
 * the exhaustive 8-device workload are checked against a second, independent
 * evaluator (brute_plan.py).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <stdio.h>
#include <pthread.h>

#define OR_INVALID UINT64_MAX
#define OR_MAXK 16
#define OR_MAXS 16
#define OR_MAXG 4

/* ------------------------------------------------------------------ */
/* checked integer arithmetic: the oracle never wraps silently         */
/* ------------------------------------------------------------------ */
static void or_die(const char* what) {
  fprintf(stderr, "oracle: arithmetic overflow in %s\n", what);
  abort();
}
static uint64_t add(uint64_t a, uint64_t b) {
  uint64_t r;
  if (__builtin_add_overflow(a, b, &r)) or_die("add");
  return r;
}
static uint64_t mul(uint64_t a, uint64_t b) {
  uint64_t r;
  if (__builtin_mul_overflow(a, b, &r)) or_die("mul");
  return r;
}
/* R1: every division rounds up. */
static uint64_t cdiv(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }
static uint64_t umax(uint64_t a, uint64_t b) { return a > b ? a : b; }

/* ------------------------------------------------------------------ */
/* inputs                                                              */
/* ------------------------------------------------------------------ */
typedef struct {
  uint64_t L, h, heads, kv_heads, ffn, gated, vocab, learned_pos, seq, e;
  uint64_t gbs, n_mbs, mbs[4], grad_bytes, param_bytes, E, topk, effn;
  uint64_t opt_bytes; /* optimizer-state bytes per parameter (R31) */
  uint32_t* q; /* [L][E] expert shares in units of 2^-16 */
} or_model;

typedef struct {
  uint64_t K;
  uint64_t n_nodes[OR_MAXK], dpn[OR_MAXK], tflops[OR_MAXK], hbm[OR_MAXK];
  uint64_t intra[OR_MAXK], pcie[OR_MAXK], nic[OR_MAXK];
  uint64_t a_intra[OR_MAXK], a_pcie[OR_MAXK], a_nic[OR_MAXK];
  uint64_t dev_off[OR_MAXK], node_off[OR_MAXK];
  uint64_t mem[OR_MAXK]; /* device memory capacity in bytes (R34) */
  int mem_check;         /* 0: capacities not given, memory not checked */
  int rail_only;         /* 1: rail-only inter-node network (R47) */
  int ccl_tree;          /* 1: all-reduces take the faster of ring and tree (R48) */
  int contention;        /* 1: concurrent segment syncs of a stage share its links (R49) */
  int ccl_hier;          /* 1: all-reduces over whole nodes may take the two-level algorithm (R50) */
  uint32_t* nic_dev;    /* NULL or per-device NIC MB/s, pool order */
  uint32_t* intra_node; /* NULL or per-node intra MB/s, pool order */
} or_cluster;

typedef struct {
  or_model m;
  or_cluster c;
  uint64_t Vp; /* vocabulary padded to a multiple of 128 (R7) */
  /* memo of per-layer forward/backward times, computed by the plain
   * per-layer functions below: [k][tpl][mi][epl][l] */
  uint64_t* lf;
  uint64_t* lb;
} or_ctx;

/* ------------------------------------------------------------------ */
/* R2: roofline time of one op on device type k                        */
/* ------------------------------------------------------------------ */
static uint64_t op_time(const or_ctx* x, int k, uint64_t F, uint64_t B) {
  uint64_t tc = cdiv(F, x->c.tflops[k]);               /* F / (TFLOPS*1e12) s = F/TFLOPS ps */
  uint64_t tm = cdiv(mul(1000, B), x->c.hbm[k]);       /* B / (GB/s*1e9) s = 1000*B/GBps ps */
  return umax(tc, tm);
}

/* an op is (F flops, B bytes); a layer is a list of ops */
typedef struct { uint64_t F, B; } op;
typedef struct { op v[16]; int n; } oplist;

static void push(oplist* l, uint64_t F, uint64_t B) { l->v[l->n].F = F; l->v[l->n].B = B; l->n++; }
/* GEMM [m x k] x [k x n]: 2mkn flops; reads A and B, writes C */
static void push_gemm(oplist* l, uint64_t m, uint64_t k, uint64_t n, uint64_t e) {
  push(l, mul(2, mul(m, mul(k, n))), mul(e, add(add(mul(m, k), mul(k, n)), mul(m, n))));
}

/* forward time of a list; backward evaluates every op with 2F and 2B (R12) */
static uint64_t list_fwd(const or_ctx* x, int k, const oplist* l) {
  uint64_t t = 0;
  for (int i = 0; i < l->n; ++i) t = add(t, op_time(x, k, l->v[i].F, l->v[i].B));
  return t;
}
static uint64_t list_bwd(const or_ctx* x, int k, const oplist* l) {
  uint64_t t = 0;
  for (int i = 0; i < l->n; ++i) t = add(t, op_time(x, k, mul(2, l->v[i].F), mul(2, l->v[i].B)));
  return t;
}

/* attention + norms + residuals of one transformer layer, per TP rank
 * (R6/R8).  T = b*s tokens, hq = h/t query width, hkv = kv width per rank. */
static void attn_ops(const or_ctx* x, uint64_t t, uint64_t b, oplist* l) {
  const or_model* m = &x->m;
  uint64_t T = b * m->seq, e = m->e, h = m->h;
  uint64_t hd = h / m->heads, hq = h / t, hkv = m->kv_heads * hd / t;
  push(l, 0, mul(2, mul(T, mul(h, e))));                                   /* norm1 */
  push_gemm(l, T, h, hq + 2 * hkv, e);                                     /* QKV projection */
  push(l, mul(4, mul(b, mul(m->seq, mul(m->seq, hq)))),                    /* attention core, non-causal count */
       mul(e, mul(b, mul(m->seq, 2 * hq + 2 * hkv))));                     /* read Q,K,V write O */
  push_gemm(l, T, hq, h, e);                                               /* output projection */
  push(l, 0, mul(3, mul(T, mul(h, e))));                                   /* residual add */
  push(l, 0, mul(2, mul(T, mul(h, e))));                                   /* norm2 */
}
/* dense MLP, per TP rank: gated (three matrices) or plain (two) */
static void mlp_ops(const or_ctx* x, uint64_t t, uint64_t T, uint64_t f, int gated, oplist* l) {
  uint64_t e = x->m.e, h = x->m.h, ft = f / t;
  if (gated) {
    push_gemm(l, T, h, 2 * ft, e);                                         /* up + gate */
    push(l, 0, mul(3, mul(T, mul(ft, e))));                                /* activation * gate */
  } else {
    push_gemm(l, T, h, ft, e);                                             /* up */
    push(l, 0, mul(2, mul(T, mul(ft, e))));                                /* activation */
  }
  push_gemm(l, T, ft, h, e);                                               /* down */
}

/* R9: expert part of an MoE layer.  EP rank j hosts experts
 * [j*E/ep, (j+1)*E/ep); expert e receives cdiv(ep*T*topk*q, 2^16) tokens;
 * the layer waits for the slowest EP rank (Sec. 4.1 [C4]). */
static uint64_t expert_time(const or_ctx* x, int k, uint64_t t, uint64_t b, uint64_t ep, uint64_t layer, int bwd) {
  const or_model* m = &x->m;
  uint64_t T = b * m->seq, per = m->E / ep, worst = 0;
  for (uint64_t j = 0; j < ep; ++j) {
    uint64_t sum = 0;
    for (uint64_t ex = j * per; ex < (j + 1) * per; ++ex) {
      uint64_t n_e = cdiv(mul(mul(ep, T), mul(m->topk, m->q[layer * m->E + ex])), 65536);
      oplist l = {{{0, 0}}, 0};
      mlp_ops(x, t, n_e, m->effn, 1, &l);
      sum = add(sum, bwd ? list_bwd(x, k, &l) : list_fwd(x, k, &l));
    }
    worst = umax(worst, sum);
  }
  return worst;
}

/* time of transformer layer `layer` on type k, TP t, micro-batch b, EP ep */
static uint64_t layer_time(const or_ctx* x, int k, uint64_t t, uint64_t b, uint64_t ep, uint64_t layer, int bwd) {
  const or_model* m = &x->m;
  uint64_t T = b * m->seq;
  oplist l = {{{0, 0}}, 0};
  attn_ops(x, t, b, &l);
  if (m->E == 0) {
    mlp_ops(x, t, T, m->ffn, (int)m->gated, &l);
  } else {
    push_gemm(&l, T, m->h, m->E, m->e);                                    /* router, replicated */
  }
  push(&l, 0, mul(3, mul(T, mul(m->h, m->e))));                            /* residual add */
  uint64_t tt = bwd ? list_bwd(x, k, &l) : list_fwd(x, k, &l);
  if (m->E) tt = add(tt, expert_time(x, k, t, b, ep, layer, bwd));
  return tt;
}

/* input embedding (stage 0): gather rows, plus learned positions if any */
static uint64_t embed_time(const or_ctx* x, int k, uint64_t b, int bwd) {
  const or_model* m = &x->m;
  uint64_t T = b * m->seq;
  uint64_t B = mul(m->e, mul(T, mul(m->h, 2 + 2 * (m->learned_pos > 0))));
  return bwd ? op_time(x, k, 0, mul(2, B)) : op_time(x, k, 0, B);
}
/* output head (last stage): final norm, vocab-parallel LM head, loss (R13) */
static uint64_t head_time(const or_ctx* x, int k, uint64_t t, uint64_t b, int bwd) {
  const or_model* m = &x->m;
  uint64_t T = b * m->seq, vt = x->Vp / t;
  oplist l = {{{0, 0}}, 0};
  push(&l, 0, mul(2, mul(T, mul(m->h, m->e))));
  push_gemm(&l, T, m->h, vt, m->e);
  push(&l, 0, mul(2, mul(T, mul(vt, m->e))));
  return bwd ? list_bwd(x, k, &l) : list_fwd(x, k, &l);
}

/* parameters held by one TP rank (biases ignored, R13) */
static uint64_t layer_params_dense(const or_ctx* x, uint64_t t) {
  const or_model* m = &x->m;
  uint64_t h = m->h, hd = h / m->heads, hq = h / t, hkv = m->kv_heads * hd / t;
  uint64_t p = h * (hq + 2 * hkv) + hq * h + 2 * h;                      /* attention + two norms */
  if (m->E == 0) p += (m->gated ? 3 : 2) * h * (m->ffn / t);
  else p += h * m->E;                                                    /* router */
  return p;
}
static uint64_t layer_params_expert(const or_ctx* x, uint64_t t, uint64_t ep) {
  const or_model* m = &x->m;
  if (m->E == 0) return 0;
  return (m->E / ep) * 3 * m->h * (m->effn / t);
}
static uint64_t embed_params(const or_ctx* x, uint64_t t) { return x->Vp * x->m.h / t + x->m.learned_pos * x->m.h; }
static uint64_t head_params(const or_ctx* x, uint64_t t) { return x->Vp * x->m.h / t + x->m.h; }

/* R32: bytes one TP rank keeps from the forward pass of one transformer
 * layer for its backward pass, for a micro-batch of b sequences: the inputs
 * of the layer's ops (the stored-activation count of Korthikanti et al.
 * 2022, "Reducing Activation Recomputation in Large Transformer Models",
 * without dropout masks and without the s x s attention scores, which a
 * fused attention kernel recomputes).  No sequence parallelism: the inputs
 * of the norms and of the first projections are full width on every rank.
 * Counted per token, in elements: */
static uint64_t layer_act_bytes(const or_ctx* x, uint64_t t, uint64_t b) {
  const or_model* m = &x->m;
  uint64_t h = m->h, hd = h / m->heads, hq = h / t, hkv = m->kv_heads * hd / t;
  uint64_t w = 0;
  w += h;                          /* input of the first norm */
  w += h;                          /* normed input of the QKV projection */
  w += hq + 2 * hkv;               /* Q, K and V, inputs of the attention core */
  w += hq;                         /* attention output, input of the output projection */
  w += h;                          /* input of the second norm */
  if (m->E == 0) {
    uint64_t ft = m->ffn / t;
    w += h;                        /* normed input of the up (and gate) projection */
    w += m->gated ? 2 * ft : ft;   /* up (and gate) outputs, inputs of the activation */
    w += ft;                       /* activation output, input of the down projection */
  } else {
    uint64_t ft = m->effn / t;
    w += h;                        /* normed input of the router */
    /* each token goes to topk experts (balanced, R32); per routed copy: the
     * expert's input, its up and gate outputs, its down projection's input */
    w += m->topk * (h + 3 * ft);
  }
  return mul(m->e, mul(b * m->seq, w));
}

/* ------------------------------------------------------------------ */
/* links (R3, R4, R5)                                                  */
/* ------------------------------------------------------------------ */
/* ps per byte in units of 2^-16; 0 = tier absent */
static uint64_t beta_q(uint64_t MBps) { return MBps ? cdiv(65536ull * 1000000ull, MBps) : 0; }
static uint64_t link_time(uint64_t bytes, uint64_t bq) {
  unsigned __int128 p = (unsigned __int128)bytes * bq;
  unsigned __int128 r = p / 65536 + (p % 65536 != 0);
  if (r >> 64) or_die("link_time");
  return (uint64_t)r;
}
static uint64_t nic_bq(const or_ctx* x, int k, uint64_t dev) {
  return beta_q(x->c.nic_dev ? x->c.nic_dev[x->c.dev_off[k] + dev] : x->c.nic[k]);
}
static uint64_t intra_bq(const or_ctx* x, int k, uint64_t node) {
  return beta_q(x->c.intra_node ? x->c.intra_node[x->c.node_off[k] + node] : x->c.intra[k]);
}
/* one endpoint of an inter-node path: GPU->switch->NIC (two PCIe trips)
 * plus NIC processing (Sec. 5, Table 5) */
static uint64_t alpha_side(const or_ctx* x, int k) { return add(mul(2, x->c.a_pcie[k]), x->c.a_nic[k]); }

/* worst NIC over devices [lo, lo+n) of pool k */
static uint64_t nic_max(const or_ctx* x, int k, uint64_t lo, uint64_t n) {
  uint64_t w = 0;
  for (uint64_t d = lo; d < lo + n; ++d) w = umax(w, nic_bq(x, k, d));
  return w;
}
/* worst intra-node fabric over the nodes touched by devices [lo, lo+n) */
static uint64_t intra_max(const or_ctx* x, int k, uint64_t lo, uint64_t n) {
  uint64_t w = 0;
  for (uint64_t d = lo; d < lo + n; ++d) w = umax(w, intra_bq(x, k, d / x->c.dpn[k]));
  return w;
}

/* ------------------------------------------------------------------ */
/* pipeline: non-interleaved 1F1B (R24, R25)                           */
/* ------------------------------------------------------------------ */
/* Stage s runs, in order: W = min(S-1-s, M) forwards, then M-W pairs
 * (forward, backward), then the remaining W backwards.  F(s,m) may start
 * once F(s-1,m) has ended and its activation crossed hop s-1; B(s,m) once
 * B(s+1,m) has ended and its gradient crossed hop s; on the last stage
 * B(S-1,m) needs F(S-1,m).  A stage runs one op at a time; sends do not
 * block the sender.  The result is the longest path of that DAG, so any
 * evaluation order that respects it gives the same numbers.  This one
 * sweeps the stages repeatedly, advancing each while its next op is
 * ready. */
typedef struct { int isB; uint64_t m; } slot;
static slot op_at(uint64_t S, uint64_t M, uint64_t s, uint64_t pos) {
  uint64_t W = (S - 1 - s) < M ? (S - 1 - s) : M;
  slot r;
  if (pos < W) { r.isB = 0; r.m = pos; return r; }
  if (pos < 2 * M - W) {
    uint64_t i = (pos - W) / 2;
    if ((pos - W) % 2 == 0) { r.isB = 0; r.m = W + i; } else { r.isB = 1; r.m = i; }
    return r;
  }
  r.isB = 1; r.m = pos - M; /* B(M-W+j) sits at position 2M-W+j */
  return r;
}

/* end[s] := end time of stage s's last op.  scratch holds 2*S*M words. */
static void pipeline(uint64_t S, uint64_t M, const uint64_t* f, const uint64_t* b, const uint64_t* c,
                     uint64_t* end, uint64_t* scratch) {
  uint64_t* endF = scratch;          /* [S][M], OR_INVALID = not yet run */
  uint64_t* endB = scratch + S * M;
  for (uint64_t i = 0; i < 2 * S * M; ++i) scratch[i] = OR_INVALID;
  uint64_t pos[OR_MAXS], last[OR_MAXS];
  for (uint64_t s = 0; s < S; ++s) { pos[s] = 0; last[s] = 0; }
  int progress = 1;
  while (progress) {
    progress = 0;
    for (uint64_t s = 0; s < S; ++s) {
      while (pos[s] < 2 * M) {
        slot o = op_at(S, M, s, pos[s]);
        uint64_t ready;
        if (!o.isB) {
          if (s == 0) ready = 0;
          else if (endF[(s - 1) * M + o.m] == OR_INVALID) break;
          else ready = add(endF[(s - 1) * M + o.m], c[s - 1]);
        } else {
          if (s == S - 1) {
            if (endF[s * M + o.m] == OR_INVALID) break;
            ready = endF[s * M + o.m];
          } else if (endB[(s + 1) * M + o.m] == OR_INVALID) break;
          else ready = add(endB[(s + 1) * M + o.m], c[s]);
        }
        uint64_t start = umax(last[s], ready);
        uint64_t e = add(start, o.isB ? b[s] : f[s]);
        if (o.isB) endB[s * M + o.m] = e; else endF[s * M + o.m] = e;
        last[s] = e;
        pos[s]++;
        progress = 1;
      }
    }
  }
  for (uint64_t s = 0; s < S; ++s) {
    if (pos[s] != 2 * M) { fprintf(stderr, "oracle: pipeline deadlock\n"); abort(); }
    end[s] = last[s];
  }
}

/* ------------------------------------------------------------------ */
/* one plan                                                            */
/* ------------------------------------------------------------------ */
/* A plan's replica classes either share one TP degree, pipeline depth and
 * layer split (the header and the cut planes say which), or, with the
 * per-class layout, each class has its own (Sec. 3: more layers to faster
 * devices, TP degrees that follow each device group's size; R35). */
typedef struct {
  uint64_t ep, G, zero, mi;
  uint64_t mi_c[OR_MAXG];  /* micro-batch size index of each class (R51; the plan's mi in the shared layout) */
  uint64_t overlap;      /* 1: gradient sync overlapped with the last backward pass (R38) */
  uint64_t v;            /* model chunks per device: 1 = plain 1F1B, 2..4 interleaved (R41) */
  uint64_t zb;           /* 1: backward split into input and weight gradients, zero-bubble order (R44) */
  int het;               /* 1: per-class layout */
  uint64_t tp[OR_MAXG], S[OR_MAXG];
  uint64_t cut[OR_MAXG][OR_MAXS];
  uint64_t reps[OR_MAXG], nmb[OR_MAXG];
  int type[OR_MAXG][OR_MAXS];
} or_plan;

/* per-stage quantities of one plan, exposed for tests; tdp[g][s] is the
 * longest layer-segment sync (resharding included) that waits for stage s
 * of class g, or with overlap the part of the stage's bucket syncs left
 * after its last backward ends */
typedef struct {
  uint64_t valid, G;
  uint64_t S[OR_MAXG];
  uint64_t M[OR_MAXG];
  uint64_t f[OR_MAXG][OR_MAXS], b[OR_MAXG][OR_MAXS], c[OR_MAXG][OR_MAXS];
  uint64_t w[OR_MAXG][OR_MAXS];   /* zero-bubble order: the weight-gradient part of b */
  uint64_t tdp[OR_MAXG][OR_MAXS];
  uint64_t end[OR_MAXG][OR_MAXS];
  uint64_t time;
} or_detail;

/* the input planes of a batch of plans */
typedef struct {
  const uint32_t* hdr;
  const uint8_t* cut;    /* [16][stride]; unused with the per-class layout */
  const uint32_t* cls;   /* [4][stride] */
  const uint64_t* types; /* [4][stride] */
  const uint32_t* chdr;  /* NULL, or [stride]: per-class layout, byte c = log2 TP | (PP-1) << 2 */
  const uint8_t* ccut;   /* with chdr: [4*16][stride], cut of stage s of class c at row c*16+s */
  int64_t stride;
} or_planes;

static int heads_split(const or_model* m, uint64_t tp) {
  if (m->heads % tp || m->kv_heads % tp) return 0;
  if (m->E == 0 && m->ffn % tp) return 0;
  if (m->E != 0 && m->effn % tp) return 0;
  return 1;
}

static int decode_rules(const or_ctx* x, const or_planes* q, int64_t i, or_plan* p) {
  const or_model* m = &x->m;
  const int64_t stride = q->stride;
  const uint32_t hdr = q->hdr[i];
  if (hdr >> 17) return 0;                                   /* V7 reserved bits */
  p->overlap = (hdr >> 13) & 1;
  p->v = ((hdr >> 14) & 3) + 1;
  p->het = q->chdr != NULL;
  p->zb = (hdr >> 16) & 1;
  if (p->zb && (p->overlap || p->v > 1)) return 0;           /* V13 (R45) */
  p->ep = 1ull << ((hdr >> 2) & 3);
  p->G = ((hdr >> 8) & 3) + 1;
  p->zero = (hdr >> 10) & 1;
  p->mi = (hdr >> 11) & 3;
  if (p->mi >= m->n_mbs) return 0;                           /* V8 */
  if (q->chdr) {
    if (hdr & 0x18f3) return 0;                              /* V10 the header's TP, PP and micro-batch size are unused (0) */
    if (p->overlap) return 0;                                /* V11 overlap needs the shared layout */
    if (p->v > 1) return 0;                                  /* V12 interleaving needs the shared layout */
    if (p->zb) return 0;                                     /* V13 so does the zero-bubble order */
    uint32_t w = q->chdr[i];
    for (uint64_t g = 0; g < p->G; ++g) {
      uint32_t bt = (w >> (8 * g)) & 0xff;
      p->tp[g] = 1ull << (bt & 3);
      p->S[g] = ((bt >> 2) & 15) + 1;
      p->mi_c[g] = bt >> 6;                                  /* R51 the class's own micro-batch size */
      if (p->mi_c[g] >= m->n_mbs) return 0;                  /* V8 */
    }
  } else {
    for (uint64_t g = 0; g < p->G; ++g) {
      p->tp[g] = 1ull << (hdr & 3);
      p->S[g] = ((hdr >> 4) & 15) + 1;
      p->mi_c[g] = p->mi;
    }
  }
  if (p->v > 1 && (p->overlap || p->S[0] < 2 || p->S[0] * p->v > OR_MAXS)) return 0;   /* V12 */
  for (uint64_t g = 0; g < p->G; ++g) {                      /* V2, per class; S*v virtual stages */
    uint64_t prev = 0;
    for (uint64_t s = 0; s < p->S[g] * p->v; ++s) {
      p->cut[g][s] = q->chdr ? q->ccut[(g * OR_MAXS + s) * stride + i] : q->cut[s * stride + i];
      if (p->cut[g][s] <= prev) return 0;
      prev = p->cut[g][s];
    }
    if (prev != m->L) return 0;
  }
  uint64_t batch = 0;
  for (uint64_t g = 0; g < p->G; ++g) {
    uint32_t w = q->cls[g * stride + i];
    p->reps[g] = w & 0xffff;
    p->nmb[g] = w >> 16;
    if (p->reps[g] == 0) return 0;                           /* V1 */
    if (p->nmb[g] < p->reps[g]) return 0;                    /* V4 every replica gets work */
    batch += p->nmb[g] * m->mbs[p->mi_c[g]];
    uint64_t tv = q->types[g * stride + i];
    for (uint64_t s = 0; s < p->S[g]; ++s) {
      p->type[g][s] = (int)((tv >> (4 * s)) & 15);
      if ((uint64_t)p->type[g][s] >= x->c.K) return 0;       /* V1 */
      if (x->c.dpn[p->type[g][s]] % p->tp[g]) return 0;      /* V5 TP stays inside a node */
    }
    if (!heads_split(m, p->tp[g])) return 0;                 /* V5 */
  }
  if (batch != m->gbs) return 0;                             /* V4 exactly the global batch (R14) */
  if (p->v > 1)                                              /* V12 (R42) */
    for (uint64_t g = 0; g < p->G; ++g) {
      uint64_t M = cdiv(p->nmb[g], p->reps[g]);
      if (M % p->S[g] || M < 2 * p->S[g]) return 0;
    }
  if (m->E == 0) {                                           /* V3 */
    if (p->ep != 1) return 0;
  } else {
    if (p->ep > m->E || m->E % p->ep) return 0;
    for (uint64_t g = 0; g < p->G; ++g) if (p->reps[g] % p->ep) return 0;
  }
  uint64_t need[OR_MAXK] = {0};                              /* V6 capacity of the packing (R18) */
  for (uint64_t g = 0; g < p->G; ++g)
    for (uint64_t s = 0; s < p->S[g]; ++s) {
      int k = p->type[g][s];
      need[k] = cdiv(need[k], p->tp[g]) * p->tp[g] + p->reps[g] * p->tp[g];
    }
  for (uint64_t k = 0; k < x->c.K; ++k)
    if (need[k] > x->c.n_nodes[k] * x->c.dpn[k]) return 0;
  return 1;
}

/* R33: micro-batches whose activations stage s holds at once under 1F1B.
 * The stage runs W = min(S-1-s, M) forwards before its first backward,
 * then alternates forward and backward, so right after each of those
 * forwards it holds W+1 of them (all M when M <= W). */
static uint64_t in_flight(uint64_t S, uint64_t M, uint64_t s) {
  uint64_t W = (S - 1 - s) < M ? (S - 1 - s) : M;
  return W + 1 < M ? W + 1 : M;
}

/* R46: micro-batches whose activations stage s holds at once under the
 * zero-bubble order: a forward's activations stay until the micro-batch's
 * weight-gradient pass (W) has run.  Counted by walking the stage's ops. */
static void zb_ops(uint64_t S, uint64_t M, uint64_t s, char* kind, uint64_t* mb);
static uint64_t in_flight_zb(uint64_t S, uint64_t M, uint64_t s) {
  char* kind = (char*)malloc(3 * M + 1);
  uint64_t* mb = (uint64_t*)malloc(8 * (3 * M + 1));
  if (!kind || !mb) or_die("in_flight_zb: out of memory");
  zb_ops(S, M, s, kind, mb);
  uint64_t live = 0, peak = 0;
  for (uint64_t j = 0; j < 3 * M; ++j) {
    if (kind[j] == 'F') { ++live; if (live > peak) peak = live; }
    if (kind[j] == 'W') --live;
  }
  free(kind);
  free(mb);
  return peak;
}

/* R41: the warm-up forwards of device s under interleaved 1F1B with S
 * devices, v chunks and M micro-batches. */
static uint64_t interleaved_warmup(uint64_t S, uint64_t v, uint64_t M, uint64_t s) {
  uint64_t w = 2 * (S - 1 - s) + (v - 1) * S;
  return w < M * v ? w : M * v;
}

/* R31 for interleaved 1F1B (R43): device s holds the layers of its v chunks
 * (virtual stages j*S + s), the embedding with virtual stage 0 and the head
 * with the last one; it keeps at most W_s + 1 chunk forwards in flight, each
 * counted at its largest chunk (a bound, not the exact mix). */
static uint64_t stage_mem_interleaved(const or_ctx* x, const or_plan* p, uint64_t g, uint64_t s) {
  const or_model* m = &x->m;
  uint64_t tp = p->tp[g], ep = p->ep, S = p->S[g], v = p->v, ns = 0, nmax = 0;
  for (uint64_t j = 0; j < v; ++j) {
    uint64_t vs = j * S + s, lo = vs ? p->cut[g][vs - 1] : 0, n = p->cut[g][vs] - lo;
    ns += n;
    if (n > nmax) nmax = n;
  }
  uint64_t pd = mul(ns, layer_params_dense(x, tp)), pe = mul(ns, layer_params_expert(x, tp, ep));
  if (s == 0) pd = add(pd, embed_params(x, tp));
  if (s == S - 1) pd = add(pd, head_params(x, tp));
  uint64_t p_all = 0;
  for (uint64_t c = 0; c < p->G; ++c) p_all += p->reps[c];
  uint64_t wg = mul(add(m->param_bytes, m->grad_bytes), add(pd, pe));
  uint64_t opt;
  if (p->zero) opt = add(cdiv(mul(m->opt_bytes, pd), p_all), cdiv(mul(m->opt_bytes, pe), p_all / ep));
  else opt = mul(m->opt_bytes, add(pd, pe));
  uint64_t M = cdiv(p->nmb[g], p->reps[g]);
  uint64_t fly = interleaved_warmup(S, v, M, s) + 1;
  if (fly > M * v) fly = M * v;
  uint64_t act = mul(mul(nmax, layer_act_bytes(x, tp, m->mbs[p->mi])), fly);
  return add(add(wg, opt), act);
}

/* R31: peak bytes on one device of stage s of class g.  Every replica keeps
 * the weights and gradients of the parameters its TP rank holds; the
 * optimizer state is kept whole, or, with ZeRO, split over the DP group
 * (all replicas for the non-expert parameters, replicas/EP for the
 * experts), rounded up; the activations of the in-flight micro-batches come
 * on top (R32, R33). */
static uint64_t stage_mem(const or_ctx* x, const or_plan* p, uint64_t g, uint64_t s) {
  const or_model* m = &x->m;
  uint64_t tp = p->tp[g], ep = p->ep;
  if (p->v > 1) return stage_mem_interleaved(x, p, g, s);
  uint64_t lo = s ? p->cut[g][s - 1] : 0, ns = p->cut[g][s] - lo;
  uint64_t pd = mul(ns, layer_params_dense(x, tp)), pe = mul(ns, layer_params_expert(x, tp, ep));
  if (s == 0) pd = add(pd, embed_params(x, tp));
  if (s == p->S[g] - 1) pd = add(pd, head_params(x, tp));
  uint64_t p_all = 0;
  for (uint64_t c = 0; c < p->G; ++c) p_all += p->reps[c];
  uint64_t wg = mul(add(m->param_bytes, m->grad_bytes), add(pd, pe));
  uint64_t opt;
  if (p->zero) opt = add(cdiv(mul(m->opt_bytes, pd), p_all), cdiv(mul(m->opt_bytes, pe), p_all / ep));
  else opt = mul(m->opt_bytes, add(pd, pe));
  uint64_t M = cdiv(p->nmb[g], p->reps[g]);
  uint64_t fly = p->zb ? in_flight_zb(p->S[g], M, s) : in_flight(p->S[g], M, s);
  uint64_t act = mul(mul(ns, layer_act_bytes(x, tp, m->mbs[p->mi_c[g]])), fly);
  return add(add(wg, opt), act);
}

/* V9 (R34): when capacities are given, every device of the plan fits. */
static int decode(const or_ctx* x, const or_planes* q, int64_t i, or_plan* p) {
  if (!decode_rules(x, q, i, p)) return 0;
  if (!x->c.mem_check) return 1;
  for (uint64_t g = 0; g < p->G; ++g)
    for (uint64_t s = 0; s < p->S[g]; ++s)
      if (stage_mem(x, p, g, s) > x->c.mem[p->type[g][s]]) return 0;
  return 1;
}

static const uint64_t* LF(const or_ctx* x, int k, uint64_t tpl, uint64_t mi, uint64_t epl) {
  return x->lf + ((((uint64_t)k * 4 + tpl) * 4 + mi) * 4 + epl) * x->m.L;
}
static const uint64_t* LB(const or_ctx* x, int k, uint64_t tpl, uint64_t mi, uint64_t epl) {
  return x->lb + ((((uint64_t)k * 4 + tpl) * 4 + mi) * 4 + epl) * x->m.L;
}
static uint64_t log2u(uint64_t v) { uint64_t r = 0; while ((1ull << r) < v) ++r; return r; }

/* one DP ring phase: `steps` transfers of `chunk` bytes each (R23) */
static uint64_t ring(uint64_t steps, uint64_t chunk, uint64_t alpha, uint64_t bq) {
  return add(mul(steps, alpha), link_time(mul(steps, chunk), bq));
}
/* gradient sync of one stage over a p-member ring (R11, R26, R27) */
static uint64_t dp_sync(uint64_t p, uint64_t zero, uint64_t grads, uint64_t params, uint64_t alpha, uint64_t bq) {
  if (p <= 1) return 0;
  if (!zero) return ring(2 * (p - 1), cdiv(grads, p), alpha, bq);          /* ring all-reduce */
  return add(ring(p - 1, cdiv(grads, p), alpha, bq),                       /* reduce-scatter of gradients */
             ring(p - 1, cdiv(params, p), alpha, bq));                     /* all-gather of parameters */
}

/* R48: pipelined binary-tree all-reduce over p members (reduce up the tree,
 * broadcast down it, in chunks): 2 ceil(log2 p) message latencies, and
 * every member's gradient crosses its busiest link twice. */
static uint64_t umin(uint64_t a, uint64_t b) { return a < b ? a : b; }
static uint64_t tree_allreduce(uint64_t p, uint64_t grads, uint64_t alpha, uint64_t bq) {
  if (p <= 1) return 0;
  uint64_t lg = 0;
  while ((1ull << lg) < p) ++lg;
  return add(mul(2 * lg, alpha), link_time(mul(2, grads), bq));
}
/* a stage's DP sync on the cluster's collectives: the ring, or with tree
 * collectives enabled the faster of ring and tree for an all-reduce (NCCL
 * picks an algorithm per call); reduce-scatter and all-gather are rings */
static uint64_t dp_sync_cl(const or_ctx* x, uint64_t p, uint64_t zero, uint64_t grads, uint64_t params, uint64_t alpha,
                           uint64_t bq) {
  uint64_t r = dp_sync(p, zero, grads, params, alpha, bq);
  if (x->c.ccl_tree && !zero && p > 1) r = umin(r, tree_allreduce(p, grads, alpha, bq));
  return r;
}

/* R49: the same sync split into its latency steps and the time its bytes
 * take on the link (the part concurrent collectives on one link share); the
 * tree is taken only when strictly faster, as above.  A shared-layout plan
 * also splits the two-level all-reduce (dp_parts_h, after its definition),
 * so that a stage holding one segment keeps its sync time. */
static void dp_parts(const or_ctx* x, uint64_t p, uint64_t zero, uint64_t grads, uint64_t params, uint64_t alpha,
                     uint64_t bq, uint64_t* lat, uint64_t* bw) {
  *lat = 0;
  *bw = 0;
  if (p <= 1) return;
  *lat = mul(2 * (p - 1), alpha);
  if (!zero) *bw = link_time(mul(2 * (p - 1), cdiv(grads, p)), bq);
  else *bw = add(link_time(mul(p - 1, cdiv(grads, p)), bq), link_time(mul(p - 1, cdiv(params, p)), bq));
  if (x->c.ccl_tree && !zero) {
    uint64_t lg = 0;
    while ((1ull << lg) < p) ++lg;
    uint64_t tl = mul(2 * lg, alpha), tb = link_time(mul(2, grads), bq);
    if (add(tl, tb) < add(*lat, *bw)) { *lat = tl; *bw = tb; }
  }
}

/* parameters of layers [a, b) held by one rank at TP t, EP ep: non-expert
 * part (with the embedding if a = 0 and the head if b = L) and expert part */
static void span_params(const or_ctx* x, uint64_t a, uint64_t b, uint64_t t, uint64_t ep, uint64_t* pd,
                        uint64_t* pe) {
  *pd = mul(b - a, layer_params_dense(x, t));
  if (a == 0) *pd = add(*pd, embed_params(x, t));
  if (b == x->m.L) *pd = add(*pd, head_params(x, t));
  *pe = mul(b - a, layer_params_expert(x, t, ep));
}

/* R18 canonical packing: per pool, a bump pointer in (class, stage) order;
 * a block starts at a multiple of its class's TP degree so that no TP group
 * spans two nodes (with one TP degree for all classes every block already
 * does) */
static void place(const or_plan* p, uint64_t base[OR_MAXG][OR_MAXS]) {
  uint64_t ptr[OR_MAXK] = {0};
  for (uint64_t g = 0; g < p->G; ++g)
    for (uint64_t s = 0; s < p->S[g]; ++s) {
      int k = p->type[g][s];
      base[g][s] = cdiv(ptr[k], p->tp[g]) * p->tp[g];
      ptr[k] = base[g][s] + p->reps[g] * p->tp[g];
    }
}

/* Forward and backward time of one micro-batch over layers [lo, hi) on the
 * devices of class g's stage on pool k from device `base` on: the layers
 * (Sec. 3 non-uniform layer split), the embedding if `first`, the head if
 * `last`, the TP all-reduces exposed in forward (Table 1, R22) and the MoE
 * all-to-all in both passes (R20). */
static void stage_compute(const or_ctx* x, const or_plan* p, uint64_t g, int k, uint64_t base, uint64_t lo,
                          uint64_t hi, int first, int last, uint64_t* F, uint64_t* B, uint64_t* Wg) {
  const or_model* m = &x->m;
  const or_cluster* cl = &x->c;
  uint64_t ep = p->ep, epl = log2u(ep), tp = p->tp[g], tpl = log2u(tp);
  uint64_t mi = p->mi_c[g], b = m->mbs[mi], T = b * m->seq, ns = hi - lo, n = p->reps[g] * tp;
  uint64_t act = mul(T, mul(m->h, m->e));                      /* one micro-batch activation (Table 1, R10) */
  uint64_t Fc = 0, Bc = 0;
  for (uint64_t l = lo; l < hi; ++l) {
    Fc = add(Fc, LF(x, k, tpl, mi, epl)[l]);
    Bc = add(Bc, LB(x, k, tpl, mi, epl)[l]);
  }
  if (first) { Fc = add(Fc, embed_time(x, k, b, 0)); Bc = add(Bc, embed_time(x, k, b, 1)); }
  if (last) { Fc = add(Fc, head_time(x, k, tp, b, 0)); Bc = add(Bc, head_time(x, k, tp, b, 1)); }
  uint64_t tpf = 0;
  if (tp > 1) {
    uint64_t nar = 2 * ns + (first != 0);
    uint64_t steps = nar * 2 * (tp - 1);
    tpf = add(mul(steps, cl->a_intra[k]), link_time(mul(steps, cdiv(act, tp)), intra_max(x, k, base, n)));
  }
  uint64_t epc = 0;
  if (m->E && ep > 1) {
    int intra = 1;
    for (uint64_t grp = 0; grp < p->reps[g] / ep; ++grp) {
      uint64_t f0 = base + grp * ep * tp, f1 = f0 + ep * tp - 1;
      if (f0 / cl->dpn[k] != f1 / cl->dpn[k]) intra = 0;
    }
    uint64_t alpha, bq;
    if (intra) { alpha = cl->a_intra[k]; bq = intra_max(x, k, base, n); }
    else { alpha = mul(2, alpha_side(x, k)); bq = umax(nic_max(x, k, base, n), beta_q(cl->pcie[k])); }
    uint64_t bytes = 0;
    for (uint64_t l = lo; l < hi; ++l) {
      uint64_t per = m->E / ep, wmax = 0;
      for (uint64_t j = 0; j < ep; ++j) {
        uint64_t w = 0;
        for (uint64_t ex = j * per; ex < (j + 1) * per; ++ex) w += m->q[l * m->E + ex];
        wmax = umax(wmax, w);
      }
      bytes = add(bytes, cdiv(mul(mul(ep - 1, T), mul(m->topk, mul(wmax, mul(m->h, m->e)))), 65536));
    }
    epc = add(mul(ns * 2 * (ep - 1), alpha), link_time(mul(2, bytes), bq));
  }
  *F = add(add(Fc, tpf), epc);
  *B = add(Bc, epc);
  /* R44: W, the weight gradient, is half of the backward compute (rounded
   * down); the MoE all-to-all of the backward pass carries the input
   * gradient between EP ranks, so it stays in B with the other half */
  if (Wg) *Wg = Bc / 2;
}

/* PP hop between class g's stage on pool k (devices from b1 on) and its
 * stage on pool k2 (from b2 on): activation forward, gradient backward
 * (Table 1); intra-node iff same pool and every replica's pair of devices
 * shares a node (R20) */
static uint64_t hop_cost(const or_ctx* x, const or_plan* p, uint64_t g, int k, uint64_t b1, int k2, uint64_t b2) {
  const or_model* m = &x->m;
  const or_cluster* cl = &x->c;
  uint64_t tp = p->tp[g], n = p->reps[g] * tp;
  uint64_t act = mul(m->mbs[p->mi_c[g]] * m->seq, mul(m->h, m->e));
  int intra = (k == k2);
  for (uint64_t r = 0; intra && r < p->reps[g]; ++r)
    if ((b1 + r * tp) / cl->dpn[k] != (b2 + r * tp) / cl->dpn[k]) intra = 0;
  uint64_t alpha, bq;
  if (intra) {
    alpha = cl->a_intra[k];
    bq = umax(intra_max(x, k, b1, n), intra_max(x, k, b2, n));
  } else {
    alpha = add(alpha_side(x, k), alpha_side(x, k2));
    bq = umax(umax(nic_max(x, k, b1, n), nic_max(x, k2, b2, n)), umax(beta_q(cl->pcie[k]), beta_q(cl->pcie[k2])));
  }
  uint64_t t = add(alpha, link_time(act, bq));
  if (cl->rail_only) {
    /* R47 (Fig. 2c): device i of the earlier stage sends to device i of the
     * later one (i < reps * tp); a pair in two nodes at different local
     * ranks crosses rails, so its data first crosses a node's fabric to the
     * receiver's rank: that of the sender's node, or of the receiver's when
     * the sender's node holds one device */
    int cross = 0;
    for (uint64_t i = 0; i < n; ++i) {
      uint64_t d1 = b1 + i, d2 = b2 + i;
      int other_node = k != k2 || d1 / cl->dpn[k] != d2 / cl->dpn[k2];
      if (other_node && d1 % cl->dpn[k] != d2 % cl->dpn[k2]) cross = 1;
    }
    if (cross) {
      int kf = cl->dpn[k] > 1 ? k : k2;
      uint64_t bf = cl->dpn[k] > 1 ? b1 : b2;
      t = add(t, add(cl->a_intra[kf], link_time(act, intra_max(x, kf, bf, n))));
    }
  }
  return t;
}

/* the DP ring's latency and rate over the devices of stage sg[g] of every
 * class (R20, R21) */
static void dp_link(const or_ctx* x, const or_plan* p, uint64_t base[OR_MAXG][OR_MAXS], const uint64_t* sg,
                    uint64_t* alpha_out, uint64_t* bq_out) {
  const or_cluster* cl = &x->c;
  int k0 = p->type[0][sg[0]], same = 1;
  uint64_t nlo = UINT64_MAX, nhi = 0;
  for (uint64_t g = 0; g < p->G; ++g) {
    int k = p->type[g][sg[g]];
    if (k != k0) same = 0;
    uint64_t n = p->reps[g] * p->tp[g];
    for (uint64_t dv = base[g][sg[g]]; dv < base[g][sg[g]] + n; ++dv) {
      uint64_t node = dv / cl->dpn[k];
      if (node < nlo) nlo = node;
      if (node > nhi) nhi = node;
    }
  }
  uint64_t alpha, bq;
  if (same && nlo == nhi) { alpha = cl->a_intra[k0]; bq = intra_bq(x, k0, nlo); }
  else {
    alpha = 0; bq = 0;
    for (uint64_t g = 0; g < p->G; ++g) {
      int k = p->type[g][sg[g]];
      alpha = umax(alpha, mul(2, alpha_side(x, k)));                    /* R21 */
      bq = umax(bq, umax(nic_max(x, k, base[g][sg[g]], p->reps[g] * p->tp[g]), beta_q(cl->pcie[k])));
    }
  }
  *alpha_out = alpha;
  *bq_out = bq;
}

/* R50: the shape of the DP group of stage sg[g] of every class for the
 * two-level all-reduce: usable when the classes' devices fill whole nodes
 * with the same number g > 1 of members (TP groups) in every node, over
 * N > 1 nodes; a_in, bq_in: the worst node latency and fabric rate. */
typedef struct { int ok; uint64_t g, N, a_in, bq_in; } or_hier;
static or_hier hier_shape(const or_ctx* x, const or_plan* p, uint64_t base[OR_MAXG][OR_MAXS], const uint64_t* sg) {
  const or_cluster* cl = &x->c;
  or_hier h = {1, 0, 0, 0, 0};
  for (uint64_t g = 0; g < p->G; ++g) {
    int k = p->type[g][sg[g]];
    uint64_t b = base[g][sg[g]], n = p->reps[g] * p->tp[g], d = cl->dpn[k];
    if (b % d || n % d) { h.ok = 0; return h; }
    uint64_t gm = d / p->tp[g];
    if (g > 0 && gm != h.g) { h.ok = 0; return h; }
    h.g = gm;
    h.N += n / d;
    h.a_in = umax(h.a_in, cl->a_intra[k]);
    h.bq_in = umax(h.bq_in, intra_max(x, k, b, n));
  }
  h.ok = h.g > 1 && h.N > 1;
  return h;
}
/* two-level all-reduce: reduce-scatter inside each node (g - 1 steps of a
 * 1/g shard on the node fabric), ring all-reduce of each shard across the
 * N nodes on the group's inter-node tier, all-gather inside each node */
static uint64_t hier_allreduce(const or_hier* h, uint64_t grads, uint64_t alpha, uint64_t bq) {
  uint64_t sh = cdiv(grads, h->g);
  return add(add(mul(2 * (h->g - 1), h->a_in), link_time(mul(2 * (h->g - 1), sh), h->bq_in)),
             add(mul(2 * (h->N - 1), alpha), link_time(mul(2 * (h->N - 1), cdiv(sh, h->N)), bq)));
}
/* a dense DP sync with the cluster's algorithms: ring, tree (R48), and
 * the two-level all-reduce where the group allows it (R50; no ZeRO) */
static uint64_t dp_sync_h(const or_ctx* x, const or_hier* h, uint64_t p, uint64_t zero, uint64_t grads,
                          uint64_t params, uint64_t alpha, uint64_t bq) {
  uint64_t r = dp_sync_cl(x, p, zero, grads, params, alpha, bq);
  if (x->c.ccl_hier && h && h->ok && !zero && p > 1) r = umin(r, hier_allreduce(h, grads, alpha, bq));
  return r;
}

/* the split of dp_sync_h: the two-level all-reduce's latency steps on both
 * tiers and its bytes on both tiers, taken where it is strictly faster */
static void dp_parts_h(const or_ctx* x, const or_hier* h, uint64_t p, uint64_t zero, uint64_t grads, uint64_t params,
                       uint64_t alpha, uint64_t bq, uint64_t* lat, uint64_t* bw) {
  dp_parts(x, p, zero, grads, params, alpha, bq, lat, bw);
  if (!(x->c.ccl_hier && h && h->ok && !zero && p > 1)) return;
  uint64_t sh = cdiv(grads, h->g);
  uint64_t hl = add(mul(2 * (h->g - 1), h->a_in), mul(2 * (h->N - 1), alpha));
  uint64_t hb = add(link_time(mul(2 * (h->g - 1), sh), h->bq_in), link_time(mul(2 * (h->N - 1), cdiv(sh, h->N)), bq));
  if (add(hl, hb) < add(*lat, *bw)) { *lat = hl; *bw = hb; }
}

static void eval_plan_interleaved(const or_ctx* x, const or_plan* p, or_detail* d, uint64_t* scratch);

/* R44-R46: zero-bubble order (ZB-H1 of Qi et al. 2024, "Zero Bubble
 * Pipeline Parallelism").  The backward pass of a stage splits into B, the
 * gradient of its input (what stage s-1 waits for), and W, the gradient of
 * its weights (needed by nobody downstream).  Stage s runs min(S-1-s, M)
 * warm-up forwards, then for i = 0..M-1: the next forward if any is left,
 * B(i), and W(i-s) once i >= s; then its last min(s, M) W passes.  So W of
 * stage s trails its B by s micro-batches, which fills the cool-down and
 * keeps at most S micro-batches' activations on any stage. */
static void zb_ops(uint64_t S, uint64_t M, uint64_t s, char* kind, uint64_t* mb) {
  uint64_t Wu = (S - 1 - s) < M ? (S - 1 - s) : M, n = 0, nextF = 0, nextW = 0;
  for (; nextF < Wu; ++nextF) { kind[n] = 'F'; mb[n++] = nextF; }
  for (uint64_t i = 0; i < M; ++i) {
    if (nextF < M) { kind[n] = 'F'; mb[n++] = nextF++; }
    kind[n] = 'B'; mb[n++] = i;
    if (i >= s) { kind[n] = 'W'; mb[n++] = nextW++; }
  }
  while (nextW < M) { kind[n] = 'W'; mb[n++] = nextW++; }
}

/* end[s] := end of stage s's last op; bi, w: B and W durations per stage.
 * F and B wait as in 1F1B; W(s,m) needs B(s,m), which precedes it on the
 * stage.  scratch holds 2 S M words. */
static void pipeline_zb(uint64_t S, uint64_t M, const uint64_t* f, const uint64_t* bi, const uint64_t* w,
                        const uint64_t* c, uint64_t* end, uint64_t* scratch) {
  char* kind[OR_MAXS];
  uint64_t* mb[OR_MAXS];
  for (uint64_t s = 0; s < S; ++s) {
    kind[s] = (char*)malloc(3 * M + 1);
    mb[s] = (uint64_t*)malloc(8 * (3 * M + 1));
    if (!kind[s] || !mb[s]) or_die("pipeline_zb: out of memory");
  }
  uint64_t* endF = scratch;
  uint64_t* endB = scratch + S * M;
  for (uint64_t i = 0; i < 2 * S * M; ++i) scratch[i] = OR_INVALID;
  uint64_t pos[OR_MAXS], last[OR_MAXS];
  for (uint64_t s = 0; s < S; ++s) { pos[s] = 0; last[s] = 0; zb_ops(S, M, s, kind[s], mb[s]); }
  int progress = 1;
  while (progress) {
    progress = 0;
    for (uint64_t s = 0; s < S; ++s) {
      while (pos[s] < 3 * M) {
        char k = kind[s][pos[s]];
        uint64_t m = mb[s][pos[s]], ready, dur;
        if (k == 'F') {
          if (s == 0) ready = 0;
          else if (endF[(s - 1) * M + m] == OR_INVALID) break;
          else ready = add(endF[(s - 1) * M + m], c[s - 1]);
          dur = f[s];
        } else if (k == 'B') {
          if (s == S - 1) {
            if (endF[s * M + m] == OR_INVALID) break;
            ready = endF[s * M + m];
          } else if (endB[(s + 1) * M + m] == OR_INVALID) break;
          else ready = add(endB[(s + 1) * M + m], c[s]);
          dur = bi[s];
        } else {
          if (endB[s * M + m] == OR_INVALID) or_die("pipeline_zb: W before its B");
          ready = endB[s * M + m];
          dur = w[s];
        }
        uint64_t e = add(umax(last[s], ready), dur);
        if (k == 'F') endF[s * M + m] = e;
        else if (k == 'B') endB[s * M + m] = e;
        last[s] = e;
        pos[s]++;
        progress = 1;
      }
    }
  }
  for (uint64_t s = 0; s < S; ++s) {
    if (pos[s] != 3 * M) or_die("pipeline_zb: deadlock");
    end[s] = last[s];
    free(kind[s]);
    free(mb[s]);
  }
}

static void eval_plan(const or_ctx* x, const or_plan* p, or_detail* d, uint64_t* scratch) {
  if (p->v > 1) { eval_plan_interleaved(x, p, d, scratch); return; }
  const or_model* m = &x->m;
  const or_cluster* cl = &x->c;
  uint64_t G = p->G, ep = p->ep, epl = log2u(ep), b = m->mbs[p->mi];
  d->valid = 1; d->G = G;
  uint64_t base[OR_MAXG][OR_MAXS];
  place(p, base);

  for (uint64_t g = 0; g < G; ++g) {
    uint64_t S = p->S[g];
    d->S[g] = S;
    d->M[g] = cdiv(p->nmb[g], p->reps[g]);                     /* R16 */
    for (uint64_t s = 0; s < S; ++s) {
      int k = p->type[g][s];
      uint64_t lo = s ? p->cut[g][s - 1] : 0, hi = p->cut[g][s];
      stage_compute(x, p, g, k, base[g][s], lo, hi, s == 0, s == S - 1, &d->f[g][s], &d->b[g][s], &d->w[g][s]);
      d->c[g][s] = s + 1 < S ? hop_cost(x, p, g, k, base[g][s], p->type[g][s + 1], base[g][s + 1]) : 0;
    }
  }

  /* DP sync per layer segment across all classes (Sec. 3: DP group = all
   * replicas; R35-R37).  The segments are the layer ranges between
   * consecutive cuts of any class, so each lies inside one stage of every
   * class; with one layout for all classes they are the stages. */
  uint64_t p_all = 0, tp_min = 8;
  for (uint64_t g = 0; g < G; ++g) { p_all += p->reps[g]; if (p->tp[g] < tp_min) tp_min = p->tp[g]; }
  uint64_t bnd[OR_MAXG * OR_MAXS + 1], nb = 0;
  bnd[nb++] = 0;
  for (uint64_t g = 0; g < G; ++g)
    for (uint64_t s = 0; s < p->S[g]; ++s) {
      uint64_t v = p->cut[g][s], j = nb;
      int seen = 0;
      for (uint64_t t = 0; t < nb; ++t) if (bnd[t] == v) seen = 1;
      if (seen) continue;
      while (j > 0 && bnd[j - 1] > v) { bnd[j] = bnd[j - 1]; --j; }   /* insertion sort */
      bnd[j] = v;
      ++nb;
    }
  for (uint64_t g = 0; g < G; ++g) for (uint64_t s = 0; s < OR_MAXS; ++s) d->tdp[g][s] = 0;
  uint64_t seg_alpha[OR_MAXG * OR_MAXS], seg_bq[OR_MAXG * OR_MAXS];
  uint64_t seg_lat[OR_MAXG][OR_MAXS], seg_bw[OR_MAXG][OR_MAXS];
  or_hier seg_h[OR_MAXG * OR_MAXS];
  memset(seg_lat, 0, sizeof(seg_lat));
  memset(seg_bw, 0, sizeof(seg_bw));
  for (uint64_t j = 0; j + 1 < nb; ++j) {
    uint64_t a = bnd[j], e = bnd[j + 1];
    uint64_t sg[OR_MAXG];
    for (uint64_t g = 0; g < G; ++g) {                          /* the stage of class g holding [a, e) */
      uint64_t s = 0;
      while (p->cut[g][s] <= a) ++s;
      sg[g] = s;
    }
    uint64_t alpha, bq;
    dp_link(x, p, base, sg, &alpha, &bq);
    seg_alpha[j] = alpha;
    seg_bq[j] = bq;
    seg_h[j] = hier_shape(x, p, base, sg);
    /* R36: the ring runs on the coarsest TP layout among the classes */
    uint64_t pd, pe;
    span_params(x, a, e, tp_min, ep, &pd, &pe);
    uint64_t t = dp_sync_h(x, p->het ? NULL : &seg_h[j], p_all, p->zero, mul(m->grad_bytes, pd),
                           mul(m->param_bytes, pd), alpha, bq);
    if (m->E) t = add(t, dp_sync_cl(x, p_all / ep, p->zero, mul(m->grad_bytes, pe), mul(m->param_bytes, pe), alpha, bq));
    /* R51: when the classes holding the segment run different micro-batch
     * sizes, each class first weights its gradient shard by its share of
     * the global batch (one elementwise pass: a multiply per element, the
     * shard read and written at the device's HBM rate).
     * R36: classes with finer shards then gather the coarse shard inside
     * each TP group: a ring all-gather over tp/tp_min members of the
     * class's own gradient shard, on the group's node fabric.  Classes
     * reshard at the same time, so the slowest class counts. */
    int mixed = 0;
    for (uint64_t g = 1; g < G; ++g) if (p->mi_c[g] != p->mi_c[0]) mixed = 1;
    uint64_t rs = 0, rs_lat = 0, rs_bw = 0;
    for (uint64_t g = 0; g < G; ++g) {
      if (p->tp[g] == tp_min && !mixed) continue;
      uint64_t qd, qe;
      span_params(x, a, e, p->tp[g], ep, &qd, &qe);
      int k = p->type[g][sg[g]];
      uint64_t elems = add(qd, qe);
      uint64_t sc = mixed ? op_time(x, k, elems, mul(2 * m->grad_bytes, elems)) : 0;
      uint64_t steps = p->tp[g] / tp_min - 1, chunk = mul(m->grad_bytes, elems);
      uint64_t bqi = intra_max(x, k, base[g][sg[g]], p->reps[g] * p->tp[g]);
      uint64_t r = add(sc, ring(steps, chunk, cl->a_intra[k], bqi));
      if (r > rs) { rs = r; rs_lat = add(sc, mul(steps, cl->a_intra[k])); rs_bw = link_time(mul(steps, chunk), bqi); }
    }
    t = add(t, rs);
    if (!cl->contention) {
      for (uint64_t g = 0; g < G; ++g) d->tdp[g][sg[g]] = umax(d->tdp[g][sg[g]], t);
    } else {
      /* R49: the segments a stage holds sync at the same time over the same
       * devices, so their link times add up while their latencies overlap */
      uint64_t ld, bd, le = 0, be = 0;
      dp_parts_h(x, p->het ? NULL : &seg_h[j], p_all, p->zero, mul(m->grad_bytes, pd), mul(m->param_bytes, pd),
                 alpha, bq, &ld, &bd);
      if (m->E) dp_parts(x, p_all / ep, p->zero, mul(m->grad_bytes, pe), mul(m->param_bytes, pe), alpha, bq, &le, &be);
      uint64_t lat = add(add(ld, le), rs_lat), bw = add(add(bd, be), rs_bw);
      if (add(lat, bw) != t) or_die("contention: split does not add up");
      for (uint64_t g = 0; g < G; ++g) {
        seg_lat[g][sg[g]] = umax(seg_lat[g][sg[g]], lat);
        seg_bw[g][sg[g]] = add(seg_bw[g][sg[g]], bw);
        d->tdp[g][sg[g]] = add(seg_lat[g][sg[g]], seg_bw[g][sg[g]]);
      }
    }
  }

  /* per class pipeline; a segment's sync starts when every stage holding it
   * has finished, so T = max over classes and stages (R27, R28) */
  uint64_t T_iter = 0;
  for (uint64_t g = 0; g < G; ++g) {
    if (p->zb) {
      uint64_t bi[OR_MAXS];
      for (uint64_t s = 0; s < p->S[g]; ++s) bi[s] = d->b[g][s] - d->w[g][s];
      pipeline_zb(p->S[g], d->M[g], d->f[g], bi, d->w[g], d->c[g], d->end[g], scratch);
    } else {
      pipeline(p->S[g], d->M[g], d->f[g], d->b[g], d->c[g], d->end[g], scratch);
    }
    if (!p->overlap)
      for (uint64_t s = 0; s < p->S[g]; ++s) T_iter = umax(T_iter, add(d->end[g][s], d->tdp[g][s]));
  }
  if (p->overlap) {
    /* R38-R40 (shared layout: segment s is stage s).  The last backward pass
     * of stage s (it ends the stage's schedule) first runs the stage's MoE
     * all-to-all share, then the head (last stage), layers hi-1 .. lo and
     * the embedding (first stage); each of these is a gradient bucket whose
     * sync may start once its backward is done and the stage's previous
     * bucket has synced (one queue per stage and class) */
    uint64_t S = p->S[0], tp = p->tp[0], tpl = log2u(tp);
    for (uint64_t g = 0; g < G; ++g)
      for (uint64_t s = 0; s < S; ++s) {
        int k = p->type[g][s];
        uint64_t lo = s ? p->cut[g][s - 1] : 0, hi = p->cut[g][s];
        uint64_t comp[OR_MAXS * 16 + 2], pd[OR_MAXS * 16 + 2], pe[OR_MAXS * 16 + 2], nbk = 0, bsum = 0;
        if (s == S - 1) {
          comp[nbk] = head_time(x, k, tp, b, 1); pd[nbk] = head_params(x, tp); pe[nbk] = 0; ++nbk;
        }
        for (uint64_t l = hi; l-- > lo;) {
          comp[nbk] = LB(x, k, tpl, p->mi, epl)[l];
          pd[nbk] = layer_params_dense(x, tp);
          pe[nbk] = layer_params_expert(x, tp, ep);
          ++nbk;
        }
        if (s == 0) {
          comp[nbk] = embed_time(x, k, b, 1); pd[nbk] = embed_params(x, tp); pe[nbk] = 0; ++nbk;
        }
        for (uint64_t j = 0; j < nbk; ++j) bsum = add(bsum, comp[j]);
        /* the last backward starts at end - b; the all-to-all share b - bsum comes first */
        uint64_t ready = d->end[g][s] - bsum, c = 0;
        for (uint64_t j = 0; j < nbk; ++j) {
          ready = add(ready, comp[j]);
          uint64_t dj = dp_sync_h(x, &seg_h[s], p_all, p->zero, mul(m->grad_bytes, pd[j]),
                                  mul(m->param_bytes, pd[j]), seg_alpha[s], seg_bq[s]);
          if (m->E && pe[j])
            dj = add(dj, dp_sync_cl(x, p_all / ep, p->zero, mul(m->grad_bytes, pe[j]), mul(m->param_bytes, pe[j]),
                                 seg_alpha[s], seg_bq[s]));
          c = add(umax(c, ready), dj);
        }
        d->tdp[g][s] = c - d->end[g][s];        /* the sync time left after the stage's end */
        T_iter = umax(T_iter, c);
      }
  }
  d->time = T_iter;
}

/* R41: interleaved 1F1B (Narayanan et al. 2021, as in Megatron-LM).  Device
 * s runs chunks j = 0..v-1 of the model, virtual stage vs = j S + s.  Its
 * ops: W_s forwards, then (forward, backward) pairs, then the remaining
 * backwards; forward number k runs micro-batch (k / (S v)) S + k mod S of
 * chunk (k mod S v) / S, backward number k the same micro-batch of chunk
 * v - 1 - (k mod S v) / S.  A forward of vs waits for vs - 1's forward of
 * the micro-batch plus the hop between their devices (the wrap hop cw from
 * the last device to the first between chunks); a backward for vs + 1's
 * backward plus the hop back, or on the last virtual stage for its own
 * forward.  Evaluated by sweeping the devices as pipeline() does.
 * f, b: [S v] per virtual stage; c: [S] hops s -> s+1. */
static void pipeline_interleaved(uint64_t S, uint64_t v, uint64_t M, const uint64_t* f, const uint64_t* b,
                                 const uint64_t* c, uint64_t cw, uint64_t* end, uint64_t* scratch) {
  uint64_t V = S * v, n = M * v;
  uint64_t* endF = scratch;          /* [V][M] */
  uint64_t* endB = scratch + V * M;
  for (uint64_t i = 0; i < 2 * V * M; ++i) scratch[i] = OR_INVALID;
  uint64_t pos[OR_MAXS], last[OR_MAXS], W[OR_MAXS];
  for (uint64_t s = 0; s < S; ++s) { pos[s] = 0; last[s] = 0; W[s] = interleaved_warmup(S, v, M, s); }
  int progress = 1;
  while (progress) {
    progress = 0;
    for (uint64_t s = 0; s < S; ++s) {
      while (pos[s] < 2 * n) {
        uint64_t q = pos[s], k;
        int isB;
        if (q < W[s]) { isB = 0; k = q; }
        else if (q < 2 * n - W[s]) {
          uint64_t i = (q - W[s]) / 2;
          if ((q - W[s]) % 2 == 0) { isB = 0; k = W[s] + i; } else { isB = 1; k = i; }
        } else { isB = 1; k = q - n; }
        uint64_t r = k % V, mb = (k / V) * S + r % S;
        uint64_t j = isB ? v - 1 - r / S : r / S, vs = j * S + s;
        uint64_t ready;
        if (!isB) {
          if (vs == 0) ready = 0;
          else if (endF[(vs - 1) * M + mb] == OR_INVALID) break;
          else ready = add(endF[(vs - 1) * M + mb], s > 0 ? c[s - 1] : cw);
        } else {
          if (vs == V - 1) {
            if (endF[vs * M + mb] == OR_INVALID) break;
            ready = endF[vs * M + mb];
          } else if (endB[(vs + 1) * M + mb] == OR_INVALID) break;
          else ready = add(endB[(vs + 1) * M + mb], s < S - 1 ? c[s] : cw);
        }
        uint64_t e = add(umax(last[s], ready), isB ? b[vs] : f[vs]);
        if (isB) endB[vs * M + mb] = e; else endF[vs * M + mb] = e;
        last[s] = e;
        pos[s]++;
        progress = 1;
      }
    }
  }
  for (uint64_t s = 0; s < S; ++s) {
    if (pos[s] != 2 * n) { fprintf(stderr, "oracle: interleaved pipeline deadlock\n"); abort(); }
    end[s] = last[s];
  }
}

/* An interleaved plan (shared layout): per class, virtual stage costs, the
 * hops between devices (c[g][S-1] holds the wrap hop), the DP sync of each
 * device over the parameters of all its chunks, and T = max over classes
 * and devices of the device's last op end plus its sync. */
static void eval_plan_interleaved(const or_ctx* x, const or_plan* p, or_detail* d, uint64_t* scratch) {
  const or_model* m = &x->m;
  uint64_t G = p->G, ep = p->ep, v = p->v;
  d->valid = 1; d->G = G;
  uint64_t base[OR_MAXG][OR_MAXS];
  place(p, base);
  for (uint64_t g = 0; g < G; ++g) {
    uint64_t S = p->S[g], V = S * v;
    d->S[g] = V;
    d->M[g] = cdiv(p->nmb[g], p->reps[g]);
    for (uint64_t vs = 0; vs < V; ++vs) {
      uint64_t s = vs % S;
      uint64_t lo = vs ? p->cut[g][vs - 1] : 0, hi = p->cut[g][vs];
      stage_compute(x, p, g, p->type[g][s], base[g][s], lo, hi, vs == 0, vs == V - 1, &d->f[g][vs], &d->b[g][vs],
                    NULL);
    }
    for (uint64_t s = 0; s < S; ++s) {
      uint64_t s2 = s + 1 < S ? s + 1 : 0;
      d->c[g][s] = hop_cost(x, p, g, p->type[g][s], base[g][s], p->type[g][s2], base[g][s2]);
    }
    for (uint64_t s = S; s < OR_MAXS; ++s) d->c[g][s] = 0;
  }
  /* DP sync of each device over all its chunks' parameters (R43) */
  uint64_t p_all = 0, S = p->S[0], tp = p->tp[0];
  for (uint64_t g = 0; g < G; ++g) p_all += p->reps[g];
  uint64_t tdp[OR_MAXS];
  for (uint64_t s = 0; s < S; ++s) {
    uint64_t sg[OR_MAXG];
    for (uint64_t g = 0; g < G; ++g) sg[g] = s;
    uint64_t alpha, bq, ns = 0;
    dp_link(x, p, base, sg, &alpha, &bq);
    for (uint64_t j = 0; j < v; ++j) {
      uint64_t vs = j * S + s;
      ns += p->cut[0][vs] - (vs ? p->cut[0][vs - 1] : 0);
    }
    uint64_t pd = mul(ns, layer_params_dense(x, tp)), pe = mul(ns, layer_params_expert(x, tp, ep));
    if (s == 0) pd = add(pd, embed_params(x, tp));
    if (s == S - 1) pd = add(pd, head_params(x, tp));
    or_hier hs = hier_shape(x, p, base, sg);
    uint64_t t = dp_sync_h(x, &hs, p_all, p->zero, mul(m->grad_bytes, pd), mul(m->param_bytes, pd), alpha, bq);
    if (m->E) t = add(t, dp_sync_cl(x, p_all / ep, p->zero, mul(m->grad_bytes, pe), mul(m->param_bytes, pe), alpha, bq));
    tdp[s] = t;
  }
  uint64_t T_iter = 0;
  for (uint64_t g = 0; g < G; ++g) {
    pipeline_interleaved(S, v, d->M[g], d->f[g], d->b[g], d->c[g], d->c[g][S - 1], d->end[g], scratch);
    for (uint64_t s = 0; s < S; ++s) {
      d->tdp[g][s] = tdp[s];
      T_iter = umax(T_iter, add(d->end[g][s], tdp[s]));
    }
  }
  d->time = T_iter;
}

/* ------------------------------------------------------------------ */
/* context                                                             */
/* ------------------------------------------------------------------ */
/* mp: L h heads kv_heads ffn gated vocab learned_pos seq e gbs n_mbs mbs0..3
 *     grad_bytes param_bytes E topk effn opt_bytes  (22 words)
 * cp: K, then for each type k: n_nodes dpn tflops hbm intra pcie nic
 *     a_intra a_pcie a_nic mem  (1 + 11K words; mem = device memory in
 *     bytes, 0 for every type = memory not checked) */
or_ctx* oracle_new(const uint64_t* mp, const uint32_t* q, const uint64_t* cp,
                   const uint32_t* nic_dev, const uint32_t* intra_node) {
  or_ctx* x = (or_ctx*)calloc(1, sizeof(or_ctx));
  or_model* m = &x->m;
  m->L = mp[0]; m->h = mp[1]; m->heads = mp[2]; m->kv_heads = mp[3]; m->ffn = mp[4]; m->gated = mp[5];
  m->vocab = mp[6]; m->learned_pos = mp[7]; m->seq = mp[8]; m->e = mp[9]; m->gbs = mp[10]; m->n_mbs = mp[11];
  for (int i = 0; i < 4; ++i) m->mbs[i] = mp[12 + i];
  m->grad_bytes = mp[16]; m->param_bytes = mp[17]; m->E = mp[18]; m->topk = mp[19]; m->effn = mp[20];
  m->opt_bytes = mp[21];
  if (m->E) {
    m->q = (uint32_t*)malloc(sizeof(uint32_t) * m->L * m->E);
    memcpy(m->q, q, sizeof(uint32_t) * m->L * m->E);
  }
  or_cluster* c = &x->c;
  c->K = cp[0];
  uint64_t dsum = 0, nsum = 0;
  for (uint64_t k = 0; k < c->K; ++k) {
    const uint64_t* r = cp + 1 + 11 * k;
    c->n_nodes[k] = r[0]; c->dpn[k] = r[1]; c->tflops[k] = r[2]; c->hbm[k] = r[3];
    c->intra[k] = r[4]; c->pcie[k] = r[5]; c->nic[k] = r[6];
    c->a_intra[k] = r[7]; c->a_pcie[k] = r[8]; c->a_nic[k] = r[9];
    c->mem[k] = r[10];
    if (r[10]) c->mem_check = 1;
    c->dev_off[k] = dsum; c->node_off[k] = nsum;
    dsum += r[0] * r[1]; nsum += r[0];
  }
  c->rail_only = cp[1 + 11 * c->K] != 0;
  c->ccl_tree = cp[2 + 11 * c->K] != 0;
  c->contention = cp[3 + 11 * c->K] != 0;
  c->ccl_hier = cp[4 + 11 * c->K] != 0;
  if (nic_dev) { c->nic_dev = (uint32_t*)malloc(4 * dsum); memcpy(c->nic_dev, nic_dev, 4 * dsum); }
  if (intra_node) { c->intra_node = (uint32_t*)malloc(4 * nsum); memcpy(c->intra_node, intra_node, 4 * nsum); }
  x->Vp = cdiv(m->vocab, 128) * 128;
  /* per-layer memo, filled by the per-layer definitions above for every
   * (type, TP, micro-batch size, EP) whose divisibility holds */
  uint64_t cells = c->K * 4 * 4 * 4 * m->L;
  x->lf = (uint64_t*)calloc(cells, 8);
  x->lb = (uint64_t*)calloc(cells, 8);
  for (uint64_t k = 0; k < c->K; ++k)
    for (uint64_t tpl = 0; tpl < 4; ++tpl) {
      uint64_t t = 1ull << tpl;
      if (m->heads % t || m->kv_heads % t) continue;
      if (m->E == 0 && m->ffn % t) continue;
      if (m->E && m->effn % t) continue;
      for (uint64_t mi = 0; mi < m->n_mbs; ++mi)
        for (uint64_t epl = 0; epl < 4; ++epl) {
          uint64_t ep = 1ull << epl;
          if (m->E == 0 && ep > 1) continue;
          if (m->E && (ep > m->E || m->E % ep)) continue;
          uint64_t* f = x->lf + (((k * 4 + tpl) * 4 + mi) * 4 + epl) * m->L;
          uint64_t* b = x->lb + (((k * 4 + tpl) * 4 + mi) * 4 + epl) * m->L;
          for (uint64_t l = 0; l < m->L; ++l) {
            f[l] = layer_time(x, (int)k, t, m->mbs[mi], ep, l, 0);
            b[l] = layer_time(x, (int)k, t, m->mbs[mi], ep, l, 1);
          }
        }
    }
  return x;
}

void oracle_free(or_ctx* x) {
  if (!x) return;
  free(x->m.q); free(x->c.nic_dev); free(x->c.intra_node); free(x->lf); free(x->lb); free(x);
}

typedef struct {
  const or_ctx* x;
  or_planes q;
  int64_t lo, hi;
  uint64_t* out;
} or_job;

static or_planes planes(const uint32_t* hdr, const uint8_t* cut, const uint32_t* cls, const uint64_t* types,
                        const uint32_t* chdr, const uint8_t* ccut, int64_t stride) {
  or_planes q = {hdr, cut, cls, types, chdr, ccut, stride};
  return q;
}

static void* worker(void* arg) {
  or_job* j = (or_job*)arg;
  uint64_t Mmax = j->x->m.gbs;                 /* nmb <= global batch, so M <= global batch */
  uint64_t* scratch = (uint64_t*)malloc(8 * 2 * OR_MAXS * (Mmax + 1));
  or_detail d;
  for (int64_t i = j->lo; i < j->hi; ++i) {
    or_plan p;
    if (!decode(j->x, &j->q, i, &p)) { j->out[i] = OR_INVALID; continue; }
    eval_plan(j->x, &p, &d, scratch);
    j->out[i] = d.time;
  }
  free(scratch);
  return NULL;
}

/* Evaluate plans [0, n) of SoA planes with plane stride `stride` (chdr and
 * ccut NULL unless the plans use the per-class layout). */
void oracle_eval(const or_ctx* x, const uint32_t* hdr, const uint8_t* cut, const uint32_t* cls,
                 const uint64_t* types, const uint32_t* chdr, const uint8_t* ccut, int64_t stride, int64_t n,
                 uint64_t* out, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  pthread_t th[256];
  or_job jobs[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].x = x; jobs[t].q = planes(hdr, cut, cls, types, chdr, ccut, stride); jobs[t].out = out;
    jobs[t].lo = n * t / nthreads; jobs[t].hi = n * (t + 1) / nthreads;
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, worker, &jobs[t]);
  worker(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
}

/* Stage-level detail of plan i (for tests and debugging). */
int oracle_detail(const or_ctx* x, const uint32_t* hdr, const uint8_t* cut, const uint32_t* cls,
                  const uint64_t* types, const uint32_t* chdr, const uint8_t* ccut, int64_t stride, int64_t i,
                  or_detail* d) {
  memset(d, 0, sizeof(*d));
  or_plan p;
  or_planes q = planes(hdr, cut, cls, types, chdr, ccut, stride);
  if (!decode(x, &q, i, &p)) { d->time = OR_INVALID; return 0; }
  uint64_t* scratch = (uint64_t*)malloc(8 * 2 * OR_MAXS * (x->m.gbs + 1));
  eval_plan(x, &p, d, scratch);
  free(scratch);
  return 1;
}
size_t oracle_detail_size(void) { return sizeof(or_detail); }

/* ------------------------------------------------------------------ */
/* pieces exposed for pinning                                          */
/* ------------------------------------------------------------------ */
void oracle_pipeline(uint64_t S, uint64_t M, const uint64_t* f, const uint64_t* b, const uint64_t* c, uint64_t* end) {
  uint64_t* scratch = (uint64_t*)malloc(8 * 2 * S * M + 8);
  pipeline(S, M, f, b, c, end, scratch);
  free(scratch);
}
/* Sec. 5: delay = jumbo frame (9200 B) * 8 / unidirectional Gb/s, in ps, rounded up */
void oracle_pipeline_interleaved(uint64_t S, uint64_t v, uint64_t M, const uint64_t* f, const uint64_t* b,
                                 const uint64_t* c, uint64_t cw, uint64_t* end) {
  uint64_t* scratch = (uint64_t*)malloc(8 * 2 * S * v * M + 8);
  pipeline_interleaved(S, v, M, f, b, c, cw, end, scratch);
  free(scratch);
}
uint64_t oracle_alpha_ps(uint64_t gbps_unidir) { return cdiv(9200ull * 8 * 1000, gbps_unidir); }
uint64_t oracle_beta_q(uint64_t MBps) { return beta_q(MBps); }
uint64_t oracle_link_time(uint64_t bytes, uint64_t bq) { return link_time(bytes, bq); }
uint64_t oracle_hier_allreduce(uint64_t g, uint64_t N, uint64_t grads, uint64_t a_in, uint64_t MBps_in, uint64_t alpha,
                               uint64_t MBps) {
  or_hier h = {1, g, N, a_in, beta_q(MBps_in)};
  return hier_allreduce(&h, grads, alpha, beta_q(MBps));
}
uint64_t oracle_tree_allreduce(uint64_t p, uint64_t grads, uint64_t alpha, uint64_t MBps) {
  return tree_allreduce(p, grads, alpha, beta_q(MBps));
}
uint64_t oracle_dp_sync(uint64_t p, uint64_t zero, uint64_t grads, uint64_t params, uint64_t alpha, uint64_t MBps) {
  return dp_sync(p, zero, grads, params, alpha, beta_q(MBps));
}
uint64_t oracle_layer_time(const or_ctx* x, int k, uint64_t t, uint64_t b, uint64_t ep, uint64_t layer, int bwd) {
  return layer_time(x, k, t, b, ep, layer, bwd);
}
uint64_t oracle_embed_time(const or_ctx* x, int k, uint64_t b, int bwd) { return embed_time(x, k, b, bwd); }
uint64_t oracle_head_time(const or_ctx* x, int k, uint64_t t, uint64_t b, int bwd) { return head_time(x, k, t, b, bwd); }
/* total parameters of the model at TP=1, EP=1: layers, embedding, head */
uint64_t oracle_param_count(const or_ctx* x, int with_head) {
  uint64_t p = x->m.L * (layer_params_dense(x, 1) + layer_params_expert(x, 1, 1)) + embed_params(x, 1);
  if (with_head) p += head_params(x, 1);
  return p;
}
/* parameters of the layers [lo, hi) held by one rank at TP t, EP ep */
uint64_t oracle_rank_params(const or_ctx* x, uint64_t t, uint64_t ep, uint64_t nlayers) {
  return nlayers * (layer_params_dense(x, t) + layer_params_expert(x, t, ep));
}
uint64_t oracle_act_bytes(const or_ctx* x, uint64_t b) { return b * x->m.seq * x->m.h * x->m.e; }
uint64_t oracle_layer_act_bytes(const or_ctx* x, uint64_t t, uint64_t b) { return layer_act_bytes(x, t, b); }
uint64_t oracle_in_flight(uint64_t S, uint64_t M, uint64_t s) { return in_flight(S, M, s); }
uint64_t oracle_in_flight_zb(uint64_t S, uint64_t M, uint64_t s) { return in_flight_zb(S, M, s); }
void oracle_pipeline_zb(uint64_t S, uint64_t M, const uint64_t* f, const uint64_t* bi, const uint64_t* w,
                        const uint64_t* c, uint64_t* end) {
  uint64_t* scratch = (uint64_t*)malloc(8 * 2 * S * M + 8);
  pipeline_zb(S, M, f, bi, w, c, end, scratch);
  free(scratch);
}
/* Peak memory of every (class, stage) device of plan i into mem[c*16 + s]
 * (entries of absent classes and stages 0).  Returns 0 if the plan breaks
 * a rule other than the memory check (mem then all 0), else 1. */
int oracle_stage_mem(const or_ctx* x, const uint32_t* hdr, const uint8_t* cut, const uint32_t* cls,
                     const uint64_t* types, const uint32_t* chdr, const uint8_t* ccut, int64_t stride, int64_t i,
                     uint64_t* mem) {
  memset(mem, 0, 8 * OR_MAXG * OR_MAXS);
  or_plan p;
  or_planes q = planes(hdr, cut, cls, types, chdr, ccut, stride);
  if (!decode_rules(x, &q, i, &p)) return 0;
  for (uint64_t g = 0; g < p.G; ++g)
    for (uint64_t s = 0; s < p.S[g]; ++s) mem[g * OR_MAXS + s] = stage_mem(x, &p, g, s);
  return 1;
}
