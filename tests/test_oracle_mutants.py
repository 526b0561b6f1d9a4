"""The oracle's pins reject the mistakes they name.

Each case plants one plausible mistake in a copy of oracle.c (a dropped term, a wrong count, a
swapped operand), builds that copy on the CPU into a temporary directory, and runs the pins that
claim to catch it against the mutated build (the wrapper loads the library named by
HETSIM_ORACLE_LIB).  A case passes when those pins fail.  The product and the real oracle are
untouched; the mutated copies live only in the temporary directory.
"""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

PINS = "tests/test_oracle_pins.py::"
ZB = "tests/test_oracle_zb.py::"
FIG3 = "tests/test_oracle_fig3.py::"

# name: (text in oracle.c, the mistake, pins that must fail)
MUTANTS = {
    "zb_w_takes_all_to_all": (
        "  if (Wg) *Wg = Bc / 2;",
        "  if (Wg) *Wg = *B / 2;",
        [ZB + "test_moe_split_keeps_all_to_all_in_input_gradient"]),
    "tp_steps_not_doubled": (
        "uint64_t steps = nar * 2 * (tp - 1);",
        "uint64_t steps = nar * (tp - 1);",
        [PINS + "test_tp_allreduce_closed_form"]),
    "tp_no_embedding_allreduce": (
        "uint64_t nar = 2 * ns + (first != 0);",
        "uint64_t nar = 2 * ns;",
        [PINS + "test_tp_allreduce_closed_form"]),
    "tp_whole_activation_per_step": (
        "link_time(mul(steps, cdiv(act, tp)), intra_max(x, k, base, n))",
        "link_time(mul(steps, act), intra_max(x, k, base, n))",
        [PINS + "test_tp_allreduce_closed_form"]),
    "tp_in_backward": (
        "  *B = add(Bc, epc);",
        "  *B = add(add(Bc, epc), tpf);",
        [PINS + "test_tp_allreduce_closed_form"]),
    "hop_latency_one_end": (
        "    alpha = add(alpha_side(x, k), alpha_side(x, k2));",
        "    alpha = alpha_side(x, k2);",
        [PINS + "test_pp_hop_inter_node_with_pcie"]),
    "hop_one_pcie_trip": (
        "static uint64_t alpha_side(const or_ctx* x, int k) { return add(mul(2, x->c.a_pcie[k]), x->c.a_nic[k]); }",
        "static uint64_t alpha_side(const or_ctx* x, int k) { return add(x->c.a_pcie[k], x->c.a_nic[k]); }",
        [PINS + "test_pp_hop_inter_node_with_pcie"]),
    "hop_pcie_rate_ignored": (
        "bq = umax(umax(nic_max(x, k, b1, n), nic_max(x, k2, b2, n)), umax(beta_q(cl->pcie[k]), beta_q(cl->pcie[k2])));",
        "bq = umax(nic_max(x, k, b1, n), nic_max(x, k2, b2, n));",
        [PINS + "test_pp_hop_inter_node_with_pcie"]),
    "hop_intra_per_pool": (
        "    if ((b1 + r * tp) / cl->dpn[k] != (b2 + r * tp) / cl->dpn[k]) intra = 0;",
        "    if (0) intra = 0;",
        [PINS + "test_pp_hop_intra_vs_inter_in_one_pool"]),
    "expert_sum_over_ranks": (
        "    worst = umax(worst, sum);",
        "    worst = add(worst, sum);",
        [PINS + "test_expert_imbalance_takes_busiest_rank"]),
    "expert_mean_over_ranks": (
        "    worst = umax(worst, sum);",
        "    worst = add(worst, cdiv(sum, ep));",
        [PINS + "test_expert_imbalance_takes_busiest_rank"]),
    "embedding_positions_dropped": (
        "uint64_t B = mul(m->e, mul(T, mul(m->h, 2 + 2 * (m->learned_pos > 0))));",
        "uint64_t B = mul(m->e, mul(T, mul(m->h, 2)));",
        [PINS + "test_embedding_bytes"]),
    "embedding_reads_whole_table": (
        "uint64_t B = mul(m->e, mul(T, mul(m->h, 2 + 2 * (m->learned_pos > 0))));",
        "uint64_t B = add(mul(m->e, mul(T, mul(m->h, 2 + 2 * (m->learned_pos > 0)))), mul(m->e, mul(x->Vp, m->h)));",
        [PINS + "test_embedding_bytes"]),
    "pipeline_gradient_hop_dropped": (
        "          else ready = add(endB[(s + 1) * M + o.m], c[s]);",
        "          else ready = endB[(s + 1) * M + o.m];",
        [PINS + "test_pipeline_uniform_with_comm", PINS + "test_pipeline_vs_event_simulation"]),
    "ring_allreduce_half_steps": (
        "  if (!zero) return ring(2 * (p - 1), cdiv(grads, p), alpha, bq);",
        "  if (!zero) return ring(p - 1, cdiv(grads, p), alpha, bq);",
        [PINS + "test_ring_allreduce_closed_form"]),
    "dp_ring_latency_one_end": (
        "      alpha = umax(alpha, mul(2, alpha_side(x, k)));                    /* R21 */",
        "      alpha = umax(alpha, alpha_side(x, k));                    /* R21 */",
        [PINS + "test_dp_ring_inter_node_latency"]),
    "all_to_all_sends_own_share": (
        "bytes = add(bytes, cdiv(mul(mul(ep - 1, T), mul(m->topk, mul(wmax, mul(m->h, m->e)))), 65536));",
        "bytes = add(bytes, cdiv(mul(mul(ep, T), mul(m->topk, mul(wmax, mul(m->h, m->e)))), 65536));",
        [PINS + "test_moe_all_to_all_closed_form"]),
    # R51 and the Fig. 3 composition (per-class micro-batch sizes)
    "weighting_reads_only": (
        "      uint64_t sc = mixed ? op_time(x, k, elems, mul(2 * m->grad_bytes, elems)) : 0;",
        "      uint64_t sc = mixed ? op_time(x, k, elems, mul(m->grad_bytes, elems)) : 0;",
        [FIG3 + "test_fig3_worked_example"]),
    "weighting_always": (
        "      uint64_t sc = mixed ? op_time(x, k, elems, mul(2 * m->grad_bytes, elems)) : 0;",
        "      uint64_t sc = op_time(x, k, elems, mul(2 * m->grad_bytes, elems));",
        [FIG3 + "test_fig3_worked_example"]),
    "weighting_at_coarse_shard": (
        "      span_params(x, a, e, p->tp[g], ep, &qd, &qe);\n      int k = p->type[g][sg[g]];\n      uint64_t elems",
        "      span_params(x, a, e, tp_min, ep, &qd, &qe);\n      int k = p->type[g][sg[g]];\n      uint64_t elems",
        [FIG3 + "test_fig3_worked_example"]),
    "hop_at_plan_micro_batch": (
        "  uint64_t act = mul(m->mbs[p->mi_c[g]] * m->seq, mul(m->h, m->e));\n  int intra = (k == k2);",
        "  uint64_t act = mul(m->mbs[p->mi] * m->seq, mul(m->h, m->e));\n  int intra = (k == k2);",
        [FIG3 + "test_fig3_worked_example"]),
    "reshard_gather_not_before_ring": (
        "    t = add(t, rs);\n    if (!cl->contention) {",
        "    if (!cl->contention) {",
        [FIG3 + "test_fig3_worked_example"]),
}


def _run_mutant(name):
    old, new, pins = MUTANTS[name]
    with open(SRC) as fh:
        text = fh.read()
    if text.count(old) != 1:
        return "site", "the mutation site occurs %d times in oracle.c" % text.count(old)
    with tempfile.TemporaryDirectory(prefix="oracle_mutant_") as tmp:
        src = os.path.join(tmp, "oracle.c")
        lib = os.path.join(tmp, "liboracle.so")
        with open(src, "w") as fh:
            fh.write(text.replace(old, new))
        cc = subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread", src, "-o", lib],
                            capture_output=True, text=True)
        if cc.returncode != 0:
            return "build", cc.stderr[-2000:]
        env = dict(os.environ, HETSIM_ORACLE_LIB=lib)
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", *pins], cwd=ROOT, env=env,
                           capture_output=True, text=True, timeout=600)
        return r.returncode, r.stdout[-3000:]


@pytest.fixture(scope="module")
def mutant_results():
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as pool:
        names = list(MUTANTS)
        return dict(zip(names, pool.map(_run_mutant, names)))


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_reject_mutant(mutant_results, name):
    rc, text = mutant_results[name]
    assert rc not in ("site", "build"), text
    # pytest exits 1 when tests ran and some failed; anything else (0 = the mistake went unnoticed,
    # 2-5 = the run itself broke) does not count as the pins catching the mistake
    assert rc == 1, "pins did not reject mutant %s (pytest exit %s):\n%s" % (name, rc, text)
