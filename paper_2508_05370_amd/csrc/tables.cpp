// tables.cpp -- descriptor validation and cost/link tables for one (model, cluster).
//
// Cost model (per transformer op, per device type): roofline time
// max(FLOPs / TFLOPS, bytes / HBM bandwidth), rounded up to whole ps; a layer
// is the sum of its ops, the backward pass charges every op twice its FLOPs
// and bytes.  Device-type profiles stand in for the paper's per-device layer
// profiling (Sec. 4.2 "Workload layer").  Link delays come from the cluster
// description (Table 5, Sec. 5); a message of B bytes over a link of rate r
// MB/s costs ceil(B * ceil(2^16 * 10^6 / r) / 2^16) ps.
#include <string.h>

#include <algorithm>

#include "internal.h"

namespace hetsim {
namespace {

typedef unsigned __int128 u128;

// A quantity that may overflow 64 bits while tables are built; any use past
// the limit turns the descriptor into SIM_ERANGE.
struct Wide {
  u128 v;
};
constexpr u128 kLimit = (u128)1 << 62;

u128 up(u128 a, u128 b) { return (a + b - 1) / b; }

struct TypeRates {
  u128 tflops, hbm;
};

// one op: FLOPs and bytes moved
struct Op {
  u128 flops, bytes;
};

u128 roofline_ps(const TypeRates& r, const Op& o, int passes) {
  u128 f = o.flops * passes, b = o.bytes * passes;
  u128 tc = up(f, r.tflops);             // F / (TFLOPS * 1e12) s  ==  F / TFLOPS ps
  u128 tm = up(b * 1000, r.hbm);         // B / (GB/s * 1e9) s     ==  1000 B / GBps ps
  return tc > tm ? tc : tm;
}

Op matmul(u128 m, u128 k, u128 n, u128 e) { return Op{2 * m * k * n, e * (m * k + k * n + m * n)}; }
Op stream(u128 bytes) { return Op{0, bytes}; }

struct Shape {
  u128 L, h, heads, kv, ffn, gated, vpad, lpos, seq, e, E, topk, effn;
};

// ops of one layer on one TP rank that do not depend on the routed tokens
int dense_layer_ops(const Shape& s, u128 t, u128 b, Op* ops) {
  u128 T = b * s.seq, hd = s.h / s.heads, q = s.h / t, kv = s.kv * hd / t;
  int n = 0;
  ops[n++] = stream(2 * T * s.h * s.e);                              // first norm
  ops[n++] = matmul(T, s.h, q + 2 * kv, s.e);                        // fused Q, K, V
  ops[n++] = Op{4 * b * s.seq * s.seq * q, s.e * b * s.seq * (2 * q + 2 * kv)};  // scores + context
  ops[n++] = matmul(T, q, s.h, s.e);                                 // attention output
  ops[n++] = stream(3 * T * s.h * s.e);                              // residual
  ops[n++] = stream(2 * T * s.h * s.e);                              // second norm
  if (s.E == 0) {
    u128 w = s.ffn / t;
    if (s.gated) {
      ops[n++] = matmul(T, s.h, 2 * w, s.e);
      ops[n++] = stream(3 * T * w * s.e);
    } else {
      ops[n++] = matmul(T, s.h, w, s.e);
      ops[n++] = stream(2 * T * w * s.e);
    }
    ops[n++] = matmul(T, w, s.h, s.e);
  } else {
    ops[n++] = matmul(T, s.h, s.E, s.e);                             // router (not split by TP)
  }
  ops[n++] = stream(3 * T * s.h * s.e);                              // residual
  return n;
}

u128 sum_ops(const TypeRates& r, const Op* ops, int n, int passes) {
  u128 t = 0;
  for (int i = 0; i < n; ++i) t += roofline_ps(r, ops[i], passes);
  return t;
}

// one gated expert MLP with `tok` tokens on one TP rank
u128 expert_ps(const Shape& s, const TypeRates& r, u128 t, u128 tok, int passes) {
  u128 w = s.effn / t;
  Op ops[3] = {matmul(tok, s.h, 2 * w, s.e), stream(3 * tok * w * s.e), matmul(tok, w, s.h, s.e)};
  return sum_ops(r, ops, 3, passes);
}

u128 beta_q(uint64_t MBps) { return MBps ? up((u128)65536 * 1000000, MBps) : 0; }

u128 link_ps(u128 bytes, u128 bq) { return up(bytes * bq, 65536); }

bool pow2(uint32_t v) { return v && !(v & (v - 1)); }
uint32_t ilog2(uint32_t v) {
  uint32_t r = 0;
  while ((1u << (r + 1)) <= v) ++r;
  return r;
}

// range-max table: level j holds max over [i, i + 2^j)
void build_rmax(const std::vector<uint32_t>& v, std::vector<uint32_t>* out, uint32_t* levels) {
  uint32_t n = (uint32_t)v.size(), lv = ilog2(n) + 1;
  out->assign((size_t)lv * n, 0);
  std::copy(v.begin(), v.end(), out->begin());
  for (uint32_t j = 1; j < lv; ++j)
    for (uint32_t i = 0; i + (1u << j) <= n; ++i)
      (*out)[(size_t)j * n + i] =
          std::max((*out)[(size_t)(j - 1) * n + i], (*out)[(size_t)(j - 1) * n + i + (1u << (j - 1))]);
  *levels = lv;
}

// Lay the setup tables out as the device image (see Tab).
void build_image(HostTables* h) {
  Tab& t = h->tab;
  const uint32_t K = t.K, nm = t.n_mbs, L1 = t.L + 1;
  t.nep = t.E ? 4 : 1;
  // every layer of a dense model costs the same on a given (type, TP,
  // micro-batch size): then one {fwd, bwd} entry per table row replaces the
  // L+1 prefix sums, and a stage costs ns times it (the same integers)
  bool uniform = t.E == 0;
  for (size_t r = 0; uniform && r < h->pf.size() / L1; ++r)
    for (uint32_t l = 1; uniform && l < t.L; ++l) {
      const size_t b = r * L1;
      uniform = h->pf[b + l + 1] - h->pf[b + l] == h->pf[b + 1] - h->pf[b] &&
                h->pb[b + l + 1] - h->pb[b + l] == h->pb[b + 1] - h->pb[b];
    }
  t.uniform_layers = uniform ? 1 : 0;
  const uint32_t row = uniform ? 1 : L1;   // entries per (type, TP, mbs, EP slot)
  auto a16 = [](size_t x) { return (uint32_t)((x + 15) & ~(size_t)15); };
  const uint32_t n_pfb = K * 4 * nm * t.nep * row;
  t.o_pfb = a16((size_t)K * sizeof(TypeInfo));
  t.o_emb = t.o_pfb + n_pfb * 16;
  t.o_head = t.o_emb + K * nm * 16;
  t.o_pa = t.o_head + K * 4 * nm * 16;
  t.o_rmi = t.o_pa + a16(t.E ? (size_t)4 * nm * L1 * 8 : 0);
  t.o_rmn = t.o_rmi + a16(h->rm_intra.size() * 4);
  t.img_bytes = t.o_rmn + a16(h->rm_nic.size() * 4);
  t.mode = t.img_bytes <= kLdsBudget ? 0 : t.o_rmn <= kLdsBudget ? 1 : 2;
  t.lds_bytes = t.mode == 0 ? t.img_bytes : t.mode == 1 ? t.o_rmn : 0;
  h->img.assign(t.img_bytes, 0);
  uint8_t* b = h->img.data();
  memcpy(b, h->ty.data(), K * sizeof(TypeInfo));
  uint64_t* pfb = (uint64_t*)(b + t.o_pfb);
  for (uint32_t k = 0; k < K; ++k)
    for (uint32_t j = 0; j < 4; ++j)
      for (uint32_t mi = 0; mi < nm; ++mi)
        for (uint32_t g = 0; g < t.nep; ++g)
          for (uint32_t l = 0; l < row; ++l) {
            const size_t src = ((((size_t)k * 4 + j) * nm + mi) * 4 + g) * L1 + l + (uniform ? 1 : 0);
            const size_t dst = ((((size_t)k * 4 + j) * nm + mi) * t.nep + g) * row + l;
            pfb[2 * dst] = h->pf[src];        // uniform: pf[1] - pf[0] = the layer's cost
            pfb[2 * dst + 1] = h->pb[src];
          }
  memcpy(b + t.o_emb, h->emb.data(), h->emb.size() * 8);
  memcpy(b + t.o_head, h->head.data(), h->head.size() * 8);
  if (t.E) memcpy(b + t.o_pa, h->pa.data(), h->pa.size() * 8);
  memcpy(b + t.o_rmi, h->rm_intra.data(), h->rm_intra.size() * 4);
  memcpy(b + t.o_rmn, h->rm_nic.data(), h->rm_nic.size() * 4);
}

}  // namespace

int build_tables(const sim_model_desc* md, const sim_cluster_desc* cd, HostTables* out) {
  const int INV = SIM_EINVAL, RNG = SIM_ERANGE;
  if (!md || !cd || !out) return INV;
  // ---------------- model
  if (md->n_layers < 1 || md->n_layers > 255) return INV;
  if (md->hidden < 1 || md->hidden > (1u << 17)) return INV;
  if (md->heads < 1 || md->hidden % md->heads) return INV;
  if (md->kv_heads < 1 || md->heads % md->kv_heads) return INV;
  if (md->gated > 1) return INV;
  if (md->vocab < 1 || md->vocab > (1u << 24)) return INV;
  if (md->learned_pos > (1u << 24)) return INV;
  if (md->seq < 1 || md->seq > (1u << 20)) return INV;
  if (md->dtype_bytes < 1 || md->dtype_bytes > 16) return INV;
  if (md->global_batch < 1) return INV;
  if (md->n_mbs < 1 || md->n_mbs > 4) return INV;
  for (uint32_t i = 0; i < md->n_mbs; ++i)
    if (md->mbs[i] < 1 || md->mbs[i] > 1024) return INV;
  if (md->grad_bytes < 1 || md->grad_bytes > 16 || md->param_bytes < 1 || md->param_bytes > 16) return INV;
  if (md->opt_bytes > 64) return INV;
  if (md->experts > 256) return INV;
  if (md->experts == 0) {
    if (md->ffn < 1 || md->ffn > (1u << 20)) return INV;
  } else {
    if (md->topk < 1 || md->topk > md->experts) return INV;
    if (md->expert_ffn < 1 || md->expert_ffn > (1u << 20)) return INV;
    if (!md->load_q16) return INV;
    for (uint32_t l = 0; l < md->n_layers; ++l) {
      uint64_t sum = 0;
      for (uint32_t e = 0; e < md->experts; ++e) sum += md->load_q16[(size_t)l * md->experts + e];
      if (sum != 65536) return INV;
    }
  }
  // ---------------- cluster
  const uint32_t K = cd->n_types;
  if (K < 1 || K > (uint32_t)kMaxTypes) return INV;
  if (!cd->n_nodes || !cd->dev_per_node || !cd->tflops || !cd->hbm_GBps || !cd->intra_MBps || !cd->pcie_MBps ||
      !cd->nic_MBps || !cd->intra_alpha_ps || !cd->pcie_alpha_ps || !cd->nic_alpha_ps)
    return INV;
  const uint64_t kMaxAlpha = (uint64_t)1 << 40;
  uint64_t D = 0, N = 0;
  for (uint32_t k = 0; k < K; ++k) {
    if (cd->n_nodes[k] < 1 || !pow2(cd->dev_per_node[k]) || cd->dev_per_node[k] > 64) return INV;
    if (cd->tflops[k] < 1 || cd->hbm_GBps[k] < 1) return INV;
    if (cd->dev_per_node[k] > 1 && cd->intra_MBps[k] < 16) return INV;
    if (cd->intra_MBps[k] && cd->intra_MBps[k] < 16) return INV;
    if (cd->pcie_MBps[k] && cd->pcie_MBps[k] < 16) return INV;
    if (cd->nic_MBps[k] < 16) return INV;
    if (cd->intra_alpha_ps[k] > kMaxAlpha || cd->pcie_alpha_ps[k] > kMaxAlpha || cd->nic_alpha_ps[k] > kMaxAlpha)
      return INV;
    if (cd->mem_bytes && cd->mem_bytes[k] < 1) return INV;
    D += (uint64_t)cd->n_nodes[k] * cd->dev_per_node[k];
    N += cd->n_nodes[k];
  }
  if (D > (1u << 20)) return INV;
  Tab& t = out->tab;
  memset(&t, 0, sizeof(t));
  t.L = md->n_layers;
  t.K = K;
  t.E = md->experts;
  t.n_mbs = md->n_mbs;
  t.gbs = md->global_batch;
  for (uint32_t i = 0; i < 4; ++i) t.mbs[i] = i < md->n_mbs ? md->mbs[i] : 0;
  t.D = (uint32_t)D;
  t.N = (uint32_t)N;
  t.grad_bytes = md->grad_bytes;
  t.param_bytes = md->param_bytes;

  Shape s;
  s.L = md->n_layers; s.h = md->hidden; s.heads = md->heads; s.kv = md->kv_heads; s.ffn = md->ffn;
  s.gated = md->gated; s.vpad = up(md->vocab, 128) * 128; s.lpos = md->learned_pos; s.seq = md->seq;
  s.e = md->dtype_bytes; s.E = md->experts; s.topk = md->topk; s.effn = md->expert_ffn;

  for (uint32_t j = 0; j < 4; ++j) {
    uint32_t tp = 1u << j;
    bool ok = md->heads % tp == 0 && md->kv_heads % tp == 0;
    ok = ok && (md->experts ? md->expert_ffn % tp == 0 : md->ffn % tp == 0);
    if (ok) t.tp_ok |= 1u << j;
    uint32_t ep = 1u << j;
    if (md->experts ? (ep <= md->experts && md->experts % ep == 0) : ep == 1) t.ep_ok |= 1u << j;
  }

  // links
  u128 bq_max = 0, a_max = 0;
  std::vector<uint32_t> nic(D), intra(N);
  uint64_t d0 = 0, n0 = 0;
  for (uint32_t k = 0; k < K; ++k) {
    t.dpn_log2[k] = ilog2(cd->dev_per_node[k]);
    t.cap[k] = cd->n_nodes[k] * cd->dev_per_node[k];
    t.tflops[k] = cd->tflops[k];
    t.hbm[k] = cd->hbm_GBps[k];
    t.rtflops[k] = 1.0 / (double)cd->tflops[k];
    t.rhbm[k] = 1.0 / (double)cd->hbm_GBps[k];
    t.dev_off[k] = (uint32_t)d0;
    t.node_off[k] = (uint32_t)n0;
    t.bq_pcie[k] = (uint32_t)beta_q(cd->pcie_MBps[k]);
    t.a_intra[k] = cd->intra_alpha_ps[k];
    t.a_side[k] = 2 * cd->pcie_alpha_ps[k] + cd->nic_alpha_ps[k];
    a_max = std::max<u128>(a_max, std::max<u128>(t.a_intra[k], 2 * (u128)t.a_side[k]));
    bq_max = std::max<u128>(bq_max, t.bq_pcie[k]);
    for (uint64_t i = 0; i < t.cap[k]; ++i) {
      uint32_t r = cd->nic_MBps_dev ? cd->nic_MBps_dev[d0 + i] : cd->nic_MBps[k];
      if (r < 16) return INV;
      nic[d0 + i] = (uint32_t)beta_q(r);
      bq_max = std::max<u128>(bq_max, nic[d0 + i]);
    }
    for (uint64_t i = 0; i < cd->n_nodes[k]; ++i) {
      uint32_t r = cd->intra_MBps_node ? cd->intra_MBps_node[n0 + i] : cd->intra_MBps[k];
      if (r && r < 16) return INV;
      if (cd->dev_per_node[k] > 1 && r == 0) return INV;
      intra[n0 + i] = (uint32_t)beta_q(r);
      bq_max = std::max<u128>(bq_max, intra[n0 + i]);
    }
    d0 += t.cap[k];
    n0 += cd->n_nodes[k];
  }
  for (uint32_t j = 0; j < 4; ++j)
    for (uint32_t k = 0; k < K; ++k)
      if (t.dpn_log2[k] >= j) t.type_ok[j] |= 1u << k;
  out->ty.assign(K, TypeInfo{});
  for (uint32_t k = 0; k < K; ++k)
    out->ty[k] = TypeInfo{t.node_off[k], t.dev_off[k], t.dpn_log2[k], t.bq_pcie[k], t.a_intra[k], t.a_side[k]};
  build_rmax(nic, &out->rm_nic, &t.lvl_dev);
  build_rmax(intra, &out->rm_intra, &t.lvl_node);

  // parameters held by one TP rank (biases ignored)
  for (uint32_t j = 0; j < 4; ++j) {
    u128 tp = (u128)1 << j;
    if (!(t.tp_ok >> j & 1)) continue;
    u128 hd = s.h / s.heads, q = s.h / tp, kv = s.kv * hd / tp;
    u128 p = s.h * (q + 2 * kv) + q * s.h + 2 * s.h;
    p += s.E ? s.h * s.E : (s.gated ? 3 : 2) * s.h * (s.ffn / tp);
    t.par_layer[j] = (uint64_t)p;
    t.par_embed[j] = (uint64_t)(s.vpad * s.h / tp + s.lpos * s.h);
    t.par_head[j] = (uint64_t)(s.vpad * s.h / tp + s.h);
    for (uint32_t g = 0; g < 4; ++g)
      if (s.E && (t.ep_ok >> g & 1)) t.par_expert[j][g] = (uint64_t)((s.E >> g) * 3 * s.h * (s.effn / tp));
  }
  for (uint32_t mi = 0; mi < md->n_mbs; ++mi) t.act[mi] = (uint64_t)((u128)md->mbs[mi] * s.seq * s.h * s.e);

  // Memory check: capacities, optimizer bytes, and the activations one layer
  // keeps for its backward pass on one TP rank: the inputs of its ops (no
  // dropout masks; attention scores are recomputed by a fused kernel), per
  // token: norm input, QKV input, Q/K/V, attention output, second norm
  // input, then the MLP's input, its activation input(s) and the down
  // projection's input -- or, for MoE layers, the router input and per
  // routed token copy (top-k of them, balanced) the same three MLP tensors.
  t.rail_only = cd->rail_only != 0;
  t.ccl_tree = cd->ccl_tree != 0;
  t.contention = cd->contention != 0;
  t.ccl_hier = cd->ccl_hier != 0;
  // The per-device bytes that sim_eval_memory reports are defined with or
  // without capacities; the capacities only switch the feasibility check on.
  u128 mem_max = 0;
  if (cd->mem_bytes) {
    t.mem_check = 1;
    for (uint32_t k = 0; k < K; ++k) t.mem_cap[k] = cd->mem_bytes[k];
  }
  {
    t.opt_bytes = md->opt_bytes;
    for (uint32_t j = 0; j < 4; ++j) {
      if (!(t.tp_ok >> j & 1)) continue;
      u128 tp = (u128)1 << j, hd = s.h / s.heads, q = s.h / tp, kv = s.kv * hd / tp;
      u128 per_tok = 3 * s.h + q + 2 * kv + q;
      if (s.E) per_tok += s.h + s.topk * (s.h + 3 * (s.effn / tp));
      else per_tok += s.h + (s.gated ? 3 : 2) * (s.ffn / tp);
      for (uint32_t mi = 0; mi < md->n_mbs; ++mi) {
        u128 a = per_tok * md->mbs[mi] * s.seq * s.e;
        t.act_layer[j][mi] = (uint64_t)a;
        u128 par = (u128)t.par_layer[j] * s.L + t.par_embed[j] + t.par_head[j] + (u128)t.par_expert[j][0] * s.L;
        mem_max = std::max(mem_max, par * (md->param_bytes + md->grad_bytes + md->opt_bytes) +
                                        a * s.L * kMaxStages);
      }
    }
    // a device's bytes are summed in 64 bits
    if (mem_max >= ((u128)1 << 63)) return RNG;
  }

  // per-layer roofline times and their prefix sums
  const uint64_t L1 = s.L + 1, nm = md->n_mbs;
  out->pf.assign((size_t)K * 4 * nm * 4 * L1, 0);
  out->pb.assign(out->pf.size(), 0);
  out->emb.assign((size_t)K * nm * 2, 0);
  out->head.assign((size_t)K * 4 * nm * 2, 0);
  out->pa.assign((size_t)4 * nm * L1, 0);
  u128 stage_max = 0;   // largest compute of any stage (all layers + embedding + head)
  for (uint32_t k = 0; k < K; ++k) {
    TypeRates r{cd->tflops[k], cd->hbm_GBps[k]};
    for (uint32_t mi = 0; mi < nm; ++mi) {
      u128 b = md->mbs[mi], T = b * s.seq;
      Op em = stream(s.e * T * s.h * (2 + (s.lpos ? 2 : 0)));
      u128 ef = roofline_ps(r, em, 1), eb = roofline_ps(r, em, 2);
      out->emb[((size_t)k * nm + mi) * 2] = (uint64_t)ef;
      out->emb[((size_t)k * nm + mi) * 2 + 1] = (uint64_t)eb;
      for (uint32_t j = 0; j < 4; ++j) {
        if (!(t.tp_ok >> j & 1)) continue;
        u128 tp = (u128)1 << j, vt = s.vpad / tp;
        Op hd[3] = {stream(2 * T * s.h * s.e), matmul(T, s.h, vt, s.e), stream(2 * T * vt * s.e)};
        u128 hf = sum_ops(r, hd, 3, 1), hb = sum_ops(r, hd, 3, 2);
        if (hf + hb + ef + eb >= kLimit) return RNG;
        out->head[(((size_t)k * 4 + j) * nm + mi) * 2] = (uint64_t)hf;
        out->head[(((size_t)k * 4 + j) * nm + mi) * 2 + 1] = (uint64_t)hb;
        Op ops[16];
        int no = dense_layer_ops(s, tp, b, ops);
        u128 df = sum_ops(r, ops, no, 1), db = sum_ops(r, ops, no, 2);
        for (uint32_t g = 0; g < 4; ++g) {
          if (!(t.ep_ok >> g & 1)) continue;
          u128 ep = (u128)1 << g, per = s.E ? s.E / ep : 0;
          size_t base = ((((size_t)k * 4 + j) * nm + mi) * 4 + g) * L1;
          u128 accf = 0, accb = 0;
          for (uint32_t l = 0; l < s.L; ++l) {
            u128 lf = df, lb = db;
            if (s.E) {
              // the MoE layer waits for its busiest EP rank
              u128 wf = 0, wb = 0;
              for (u128 rank = 0; rank < ep; ++rank) {
                u128 sf = 0, sb = 0;
                for (u128 x = rank * per; x < (rank + 1) * per; ++x) {
                  u128 share = md->load_q16[(size_t)l * s.E + (size_t)x];
                  u128 tok = up(ep * T * s.topk * share, 65536);
                  sf += expert_ps(s, r, tp, tok, 1);
                  sb += expert_ps(s, r, tp, tok, 2);
                }
                wf = std::max(wf, sf);
                wb = std::max(wb, sb);
              }
              lf += wf;
              lb += wb;
            }
            accf += lf;
            accb += lb;
            if (accf + accb >= kLimit) return RNG;
            out->pf[base + l + 1] = (uint64_t)accf;
            out->pb[base + l + 1] = (uint64_t)accb;
          }
          stage_max = std::max(stage_max, accf + accb + ef + eb + hf + hb);
        }
      }
    }
  }
  // all-to-all bytes of one all-to-all on the busiest EP rank, per layer, prefix summed
  u128 a2a_max = 0;
  for (uint32_t g = 0; g < 4; ++g) {
    if (!s.E || !(t.ep_ok >> g & 1) || g == 0) continue;
    u128 ep = (u128)1 << g, per = s.E / ep;
    for (uint32_t mi = 0; mi < nm; ++mi) {
      u128 T = (u128)md->mbs[mi] * s.seq, acc = 0;
      size_t base = ((size_t)g * nm + mi) * L1;
      for (uint32_t l = 0; l < s.L; ++l) {
        u128 w = 0;
        for (u128 rank = 0; rank < ep; ++rank) {
          u128 sum = 0;
          for (u128 x = rank * per; x < (rank + 1) * per; ++x) sum += md->load_q16[(size_t)l * s.E + (size_t)x];
          w = std::max(w, sum);
        }
        acc += up((ep - 1) * T * s.topk * w * s.h * s.e, 65536);
        if (acc >= ((u128)1 << 46)) return RNG;
        out->pa[base + l + 1] = (uint64_t)acc;
      }
      a2a_max = std::max(a2a_max, acc);
    }
  }

  // Overflow guard.  Every message stays below 2^48 bytes so that bytes * rate
  // fits 80 bits; a stage's per-micro-batch time and DP sync stay below 2^52;
  // the whole iteration (bounded by the sum over all pipeline nodes of their
  // duration and incoming hop, plus the DP sync) stays below 2^62.
  u128 act_max = 0;
  for (uint32_t mi = 0; mi < nm; ++mi) act_max = std::max<u128>(act_max, t.act[mi]);
  u128 steps_tp = (2 * s.L + 1) * 2 * 7, steps_ep = s.L * 2 * 7;
  u128 tp_max = steps_tp * a_max + link_ps(steps_tp * act_max, bq_max);
  u128 ep_max = steps_ep * a_max + link_ps(2 * a2a_max, bq_max);
  u128 hop_max = a_max + link_ps(act_max, bq_max);
  if (t.rail_only) hop_max *= 2;   // a cross-rail hop adds one intra-node step
  u128 par_max = 0;
  for (uint32_t j = 0; j < 4; ++j)
    par_max = std::max<u128>(par_max, (u128)t.par_layer[j] * s.L + t.par_embed[j] + t.par_head[j] +
                                          (u128)t.par_expert[j][0] * s.L);
  u128 bytes_dp = par_max * std::max(md->grad_bytes, md->param_bytes);
  if (act_max * steps_tp >= ((u128)1 << 48) || bytes_dp * 2 + 2 * D >= ((u128)1 << 48)) return RNG;
  u128 dp_max = 4 * (2 * (u128)D * a_max + link_ps(2 * bytes_dp + 2 * D, bq_max));
  u128 node_max = stage_max + 2 * tp_max + 2 * ep_max + 2 * hop_max;
  if (node_max >= ((u128)1 << 52) || dp_max >= ((u128)1 << 52)) return RNG;
  u128 total = (u128)md->global_batch * kMaxStages * node_max + dp_max;
  if (total >= kLimit) return RNG;
  build_image(out);
  return SIM_OK;
}

}  // namespace hetsim
