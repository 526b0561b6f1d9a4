/*
 * hetsim.h -- C ABI of the MI355X evaluator of heterogeneous LLM-training
 * deployment plans (arXiv 2508.05370, "Simulating LLM training workloads for
 * heterogeneous compute and network infrastructure").
 *
 * The library estimates the iteration time of many candidate plans at once.
 * A plan maps one model onto a heterogeneous cluster: TP/PP/DP/EP degrees,
 * a non-uniform split of the layers into pipeline stages, and up to four
 * replica classes (a device group composition, Sec. 3 "Device grouping", and
 * how many replicas of it run), each with its own share of the global batch
 * (Sec. 3 "Non-uniform workload partitioning").  The inputs follow the
 * paper's input description: model parameters, framework parameters and a
 * heterogeneous topology with per-tier bandwidth and latency (Sec. 4.2
 * "Input Description", Tables 5 and 6).
 *
 * All times are unsigned 64-bit picoseconds and every division rounds up,
 * so results are exact integers, reproducible bit for bit.
 *
 * Threading: a context is immutable after sim_create and may be used from
 * several host threads and HIP streams at once.  Calls that take a stream
 * are asynchronous: they enqueue work and return; results are valid once
 * the stream has been synchronised.
 */
#ifndef HETSIM_H
#define HETSIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
#define SIM_OK 0
#define SIM_EINVAL (-1)   /* malformed descriptor or argument */
#define SIM_ERANGE (-2)   /* descriptor could overflow the 64-bit time arithmetic */
#define SIM_ENOMEM (-3)   /* host or device allocation failed */
#define SIM_EHIP (-4)     /* a HIP runtime call or kernel launch failed */
#define SIM_ESIZE (-5)    /* more plans than sim_eval_plans_noalloc's fixed workspace holds */

/* per-plan result of an invalid or infeasible plan */
#define SIM_TIME_INVALID UINT64_MAX

typedef struct sim_ctx sim_ctx;

/*
 * Model (Sec. 4.2 "Model parameters"; Table 6).  Host memory, owned by the
 * caller, deep-copied by sim_create.  Per-op costs follow a roofline of the
 * device type: each op takes max(FLOPs / TFLOPS, bytes / HBM bandwidth).
 */
typedef struct {
  uint32_t n_layers;      /* L, 1..255 transformer layers */
  uint32_t hidden;        /* h */
  uint32_t heads;         /* query heads; divides hidden */
  uint32_t kv_heads;      /* key/value heads (grouped-query attention); divides heads */
  uint32_t ffn;           /* dense MLP width; ignored when experts > 0 */
  uint32_t gated;         /* 1: gated MLP with three matrices (SwiGLU); 0: two matrices (GELU) */
  uint32_t vocab;         /* vocabulary; padded up to a multiple of 128 */
  uint32_t learned_pos;   /* rows of a learned position table; 0 = none (rotary) */
  uint32_t seq;           /* sequence length, tokens */
  uint32_t dtype_bytes;   /* bytes per activation/weight element (2 = bf16/fp16) */
  uint32_t global_batch;  /* sequences per iteration */
  uint32_t n_mbs;         /* 1..4 micro-batch sizes a plan may pick from */
  uint32_t mbs[4];        /* micro-batch sizes in sequences, 1..1024 */
  uint32_t grad_bytes;    /* bytes per gradient element in the DP sync (4 = fp32) */
  uint32_t param_bytes;   /* bytes per parameter in the ZeRO all-gather (2 = bf16) */
  uint32_t experts;       /* E: 0 = dense model; else experts per MoE layer (every layer) */
  uint32_t topk;          /* experts per token, 1..E */
  uint32_t expert_ffn;    /* width of one (gated) expert MLP */
  const uint32_t* load_q16; /* [n_layers][experts] token share of each expert in units of
                               2^-16, rows summing to 65536; NULL iff experts == 0 */
  uint32_t opt_bytes;     /* optimizer-state bytes per parameter, 0..64 (12 = fp32 master
                             weights and two Adam moments); used by the memory check only */
} sim_model_desc;

/*
 * Cluster (Sec. 4.2 "Heterogeneous host and cluster topology"; Table 5).
 * K device types; type k is a pool of n_nodes[k] homogeneous nodes of
 * dev_per_node[k] devices.  Devices are numbered pool by pool (type-major),
 * node-major inside a pool.  Links: an intra-node fabric per node, a PCIe
 * path from device to NIC, one NIC per device.  Bandwidths are MB/s per
 * direction (0 = tier absent, else >= 16); latencies are ps per message.
 * All arrays are host memory owned by the caller and deep-copied.
 */
typedef struct {
  uint32_t n_types;                 /* K, 1..16 */
  const uint32_t* n_nodes;          /* [K] >= 1 */
  const uint32_t* dev_per_node;     /* [K] power of two, 1..64 */
  const uint32_t* tflops;           /* [K] dense TFLOP/s, >= 1 */
  const uint32_t* hbm_GBps;         /* [K] memory bandwidth GB/s, >= 1 */
  const uint32_t* intra_MBps;       /* [K] intra-node fabric; required when dev_per_node > 1 */
  const uint32_t* pcie_MBps;        /* [K] device-to-NIC PCIe; 0 = not on the inter-node path */
  const uint32_t* nic_MBps;         /* [K] per-device NIC, required */
  const uint64_t* intra_alpha_ps;   /* [K] latency of one intra-node message */
  const uint64_t* pcie_alpha_ps;    /* [K] latency of one PCIe trip (an inter-node path makes two per side) */
  const uint64_t* nic_alpha_ps;     /* [K] NIC processing latency per side */
  const uint32_t* nic_MBps_dev;     /* optional [total devices] per-device NIC rate (overrides nic_MBps) */
  const uint32_t* intra_MBps_node;  /* optional [total nodes] per-node fabric rate (overrides intra_MBps) */
  const uint64_t* mem_bytes;        /* optional [K] device memory in bytes, each >= 1 (Table 5 names
                                       A100 40 GB and H100 80 GB); NULL = memory not checked */
  uint32_t rail_only;               /* nonzero: rail-only inter-node network (Fig. 2): the NIC of local rank r
                                       of every node joins rail r and rails do not meet, so a pipeline
                                       hop between nodes whose device pairs sit at different local ranks
                                       first crosses a node's fabric to the receiver's rank -- the
                                       sender's node, or the receiver's when the sender's type has one
                                       device per node -- adding that node's latency and the activation
                                       at its slowest fabric rate (Fig. 2c); 0: any NIC reaches any */
  uint32_t ccl_tree;                /* nonzero: every DP all-reduce (not the reduce-scatter and all-gather of
                                       ZeRO) takes the faster of the ring and a pipelined binary tree,
                                       2 ceil(log2 p) latencies plus twice the gradient bytes at the
                                       ring's slowest rate, as a collective library picks an algorithm
                                       per call (Sec. 4.1 [C3]); 0: rings only */
  uint32_t contention;              /* nonzero: with the per-class layout, the syncs of the layer segments a
                                       stage holds run at the same time over the same devices and share
                                       their links: the stage waits for the largest latency part plus
                                       the sum of the link-time parts (each segment: its rings' message
                                       latencies, then their bytes at the slowest rate, resharding
                                       included); 0: concurrent syncs do not slow each other */
  uint32_t ccl_hier;                /* nonzero: a dense DP all-reduce (shared layout, not ZeRO) whose group fills
                                       whole nodes with the same number g > 1 of members (TP groups) in
                                       every node, over N > 1 nodes, may take the two-level algorithm --
                                       reduce-scatter inside each node, ring all-reduce of each 1/g shard
                                       across the nodes, all-gather inside each node -- when faster */
} sim_cluster_desc;

/*
 * Candidate plans, structure of arrays in DEVICE memory (caller-owned),
 * plane stride `stride` elements (>= n).  Plan i, shared layout (every
 * replica class runs the same TP degree, pipeline depth and layer split):
 *   hdr[i]              bits 0-1 log2 TP, 2-3 log2 EP, 4-7 PP-1, 8-9 classes-1,
 *                       10 ZeRO (reduce-scatter + all-gather instead of
 *                       all-reduce), 11-12 micro-batch size index,
 *                       13 overlap: each stage's gradient sync runs in
 *                       buckets (head, every layer, embedding) that start as
 *                       soon as their part of the stage's last backward pass
 *                       is done, one after another on the stage's ring
 *                       (Sec. 6 on overlapping communication with
 *                       computation; shared layout only), 14-15 v-1:
 *                       with v > 1, interleaved 1F1B (Narayanan et al.
 *                       2021): each of the PP devices of a replica holds v
 *                       model chunks, virtual stage j*PP + s on device s
 *                       (shared layout only, no overlap, PP >= 2,
 *                       PP*v <= 16, micro-batches per replica of every
 *                       class a multiple of PP and at least 2 PP),
 *                       16 zero-bubble order (ZB-H1, Qi et al. 2024): the
 *                       backward pass splits into an input-gradient part
 *                       (what the previous stage waits for) and a
 *                       weight-gradient part, half of the backward time
 *                       rounded down; stage s runs 1F1B's order of forwards
 *                       and input-gradient passes and each weight-gradient
 *                       pass s micro-batches after its input-gradient pass,
 *                       the last s at the end (shared layout only, with
 *                       neither overlap nor interleaving),
 *                       17-31 zero
 *   cut[s*stride+i]     u8, last layer (exclusive) of stage s: 1 <= cut[0] <
 *                       ... < cut[PP-1] = L (the non-uniform layer split);
 *                       interleaved: PP*v cuts, one per virtual stage
 *   cls[c*stride+i]     u32, class c: replicas in bits 0-15, micro-batches in
 *                       bits 16-31 (the class's share of the global batch)
 *   types[c*stride+i]   u64, device type of stage s of class c in bits [4s, 4s+4)
 * Entries past PP stages or past the class count are ignored.
 *
 * Per-class layout (chdr != NULL): device groups may differ in TP degree,
 * in how many layers each stage takes and in micro-batch size (Sec. 3
 * "Non-uniform workload partitioning": TP=1 next to TP=3 groups, more
 * layers on faster devices, non-uniform batches).  Then hdr's TP, PP and
 * micro-batch size fields must be 0, `cut` is not read (may be NULL), and
 *   chdr[i]                 byte c (class c): bits 0-1 log2 TP, 2-5 PP-1,
 *                           6-7 micro-batch size index (into mbs[])
 *   ccut[(c*16+s)*stride+i] u8, last layer (exclusive) of stage s of class
 *                           c: 1 <= ... < ccut[(c*16+PP_c-1)*stride+i] = L
 * The classes' micro-batches times their micro-batch sizes sum to the
 * global batch.  The gradient sync of the layers between two consecutive
 * cuts of any class runs as one ring over every replica on the coarsest TP
 * layout among the classes.  Before it each class reshards its gradients
 * (Sec. 3 "Resharding", both conditions; Sec. 4.1 [C2]): when the classes
 * holding those layers differ in micro-batch size, each weights its shard
 * by its share of the batch (one elementwise pass: a multiply per element,
 * the fp32 shard read and written at its devices' HBM rate), and a class
 * with a finer shard gathers the coarse one inside its TP groups; the
 * classes do this at once and the slowest counts.  A stage's sync waits for
 * its own backward passes and those of the other classes' stages that hold
 * the same layers.  The rules above apply per class.
 * A plan that breaks any rule (ranges, divisibility of heads/widths by TP,
 * TP within a node, EP dividing every class's replicas, capacity of every
 * device pool, micro-batches summing to the global batch, at least one
 * micro-batch per replica, and, when the cluster gives mem_bytes, the peak
 * memory of every device as sim_eval_memory defines it) evaluates to
 * SIM_TIME_INVALID; that is not an error.
 */
typedef struct {
  const uint32_t* hdr;
  const uint8_t* cut;
  const uint32_t* cls;
  const uint64_t* types;
  int64_t stride;
  const uint32_t* chdr;   /* NULL = shared layout */
  const uint8_t* ccut;    /* with chdr: [64][stride] */
} sim_plans;

/* argmin result: lowest time, ties to the lowest plan index */
typedef struct {
  uint64_t time_ps;
  int64_t index;
} sim_best;

/*
 * Create a context on the current HIP device: validates the descriptors,
 * builds the per-device-type roofline cost tables (per layer, forward and
 * backward, for every TP degree, micro-batch size and EP degree, with layer
 * prefix sums), the link tables and range-maximum structures, and uploads
 * them.  Returns SIM_EINVAL for malformed descriptors, SIM_ERANGE when some
 * plan's time could exceed 2^62 ps, a per-stage quantity 2^52 ps or a
 * device's memory as sim_eval_memory defines it 2^63 bytes,
 * SIM_ENOMEM or SIM_EHIP on allocation/copy failure.  *out is NULL on error.
 */
int sim_create(const sim_model_desc* model, const sim_cluster_desc* cluster, sim_ctx** out);

/*
 * Iteration time of plans 0..n-1 into out_time_ps[0..n-1] (device memory,
 * caller-owned): per-stage compute from the cost tables, alpha-beta times of
 * the TP all-reduce (exposed in forward), the MoE all-to-all, the pipeline
 * point-to-point hops (Table 1 exposure) on each group's slowest link (Sec.
 * 4.1 [C4]), a 1F1B pipeline per class (interleaved when the header says
 * so), then the DP gradient sync per stage (per device) across all
 * replicas.  n = 0 is a no-op.  Temporary device memory is taken
 * from a stream-ordered pool on `stream` (a hipStream_t; NULL = null
 * stream).  Returns SIM_EINVAL for a NULL pointer, n < 0 or stride < n,
 * SIM_ENOMEM if the temporary memory cannot be allocated, SIM_EHIP if a
 * launch fails.
 */
int sim_eval_plans(sim_ctx* ctx, const sim_plans* plans, int64_t n, uint64_t* out_time_ps, void* stream);

/* Plans per call of sim_eval_plans_noalloc: shared layout, per-class layout. */
#define SIM_NOALLOC_MAX_PLANS (1 << 18)
#define SIM_NOALLOC_MAX_PLANS_PER_CLASS (1 << 16)

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * results as sim_eval_plans, computed by the same kernels, with no
 * hipMalloc, hipFree, pool allocation, stream or event creation.  The
 * workspace is a static device array of about 46 MiB that every GPU the
 * library runs on holds from the first sim_create on it until the process
 * ends.  Every call on one GPU shares that GPU's array: calls that overlap
 * in time on one GPU (on two streams, from two threads or two contexts)
 * race and give wrong results; serialize them.  The counters a call needs
 * are cleared by a fill kernel on `stream` (no memset node), and every other
 * buffer is rewritten before it is read, so consecutive calls need nothing
 * in between.  All work runs on `stream` in order.  Returns SIM_ESIZE when n
 * exceeds SIM_NOALLOC_MAX_PLANS (SIM_NOALLOC_MAX_PLANS_PER_CLASS for the
 * per-class layout), SIM_EINVAL and SIM_EHIP as sim_eval_plans.
 */
int sim_eval_plans_noalloc(sim_ctx* ctx, const sim_plans* plans, int64_t n, uint64_t* out_time_ps, void* stream);

/*
 * Measurement helper for roofline reports (no part of an evaluation): the
 * peak rate, in nodes per second, at which the current device runs the
 * recurrence's schedule-node operation -- end = max(end, input + hop) +
 * duration, three fp64 VALU operations -- over independent chains, so that
 * instruction issue and not latency bounds it.  Blocking: it allocates a
 * small buffer, launches on `stream`, waits for it and frees the buffer.
 * Returns SIM_EINVAL for a NULL result, SIM_ENOMEM or SIM_EHIP on failure.
 */
int sim_measure_node_rate(double* nodes_per_s, void* stream);

/*
 * Per-stage quantities of plans 0..n-1 (device memory, caller-owned):
 *   out_stage[((i*4 + c)*16 + s)*4 + q], q = 0 forward time of one
 *   micro-batch on stage s of class c, 1 backward time, 2 pipeline hop
 *   s -> s+1, 3 DP sync that waits for stage s of class c (with the
 *   per-class layout: the longest of the syncs of the layer segments the
 *   stage holds, resharding included);
 *   out_class[i*4 + c] = PP of the class | classes << 5 | M << 8 | (v-1) << 24
 *   where M is the micro-batches per replica of class c (0 for an absent
 *   class or an invalid plan).  For an interleaved plan s runs over the
 *   PP*v virtual stages for q = 0, 1; q = 2 and 3 are per device (s < PP;
 *   the hop of device PP-1 is the one back to device 0) and 0 past PP.
 * Entries of absent stages are left untouched.  Plans are worked in chunks
 * of 2^21 through one temporary workspace.  Same errors as sim_eval_plans.
 */
int sim_eval_stages(sim_ctx* ctx, const sim_plans* plans, int64_t n, uint64_t* out_stage, uint32_t* out_class,
                    void* stream);

/*
 * Peak device memory of plans 0..n-1: out_mem[(i*4 + c)*16 + s] (device
 * memory, caller-owned) = bytes one device of stage s of class c holds at
 * once.  Parallelism exists to fit the model in device memory (Sec. 2) and
 * device types differ in it (Sec. 3 example, Table 5), so with mem_bytes
 * given a plan is feasible only if every device fits.  The bytes are
 *   (param_bytes + grad_bytes) * P                 weights and gradients
 * + opt_bytes * P, or with ZeRO ceil(opt_bytes * P_dense / replicas)
 *   + ceil(opt_bytes * P_expert / (replicas / EP)) optimizer state, split
 *   over the stage's DP group as its gradient sync is
 * + layers * A * min(PP - s, M)                    stored activations
 * where P is the parameters the device's TP rank holds for the stage's
 * layers (and the embedding on the first stage, the head on the last), A
 * the bytes one layer keeps for its backward pass per micro-batch (the
 * inputs of its ops: the stored-activation count of Korthikanti et al.
 * 2022 without dropout masks and attention scores; routed MoE tokens
 * counted at the balanced top-k share) and min(PP - s, M) the micro-batches
 * stage s holds at once under 1F1B (min(PP, M) on every stage under the
 * zero-bubble order, whose activations stay until the weight-gradient
 * pass).  Interleaved plans: s is the device,
 * whose layers are those of all its chunks, and the activation term is
 * nmax * A * min(2 (PP-1-s) + (v-1) PP + 1, M v) with nmax the layers of the
 * device's largest chunk (its warm-up passes plus one, each counted at that
 * chunk).  Entries of absent classes and stages
 * are 0; all 64 entries of a plan that breaks another rule are
 * SIM_TIME_INVALID.  The memory check itself does not affect this output.
 * Any n; plans are worked in chunks of 2^21.  Errors as sim_eval_plans.
 */
int sim_eval_memory(sim_ctx* ctx, const sim_plans* plans, int64_t n, uint64_t* out_mem, void* stream);

/*
 * Lexicographic minimum of (time_ps[i], index_base + i) over i < n, written
 * to *out_best (device memory).  Invalid plans are skipped; if all are
 * invalid (or n = 0) the result is {SIM_TIME_INVALID, -1}.  Chunks of a
 * larger sweep may be reduced on different streams into separate slots and
 * combined with sim_best_reduce; the result does not depend on the order.
 */
int sim_argmin(sim_ctx* ctx, const uint64_t* time_ps, int64_t n, int64_t index_base, sim_best* out_best,
               void* stream);

/* Lexicographic minimum of n argmin slots (device memory) into *out_best. */
int sim_best_reduce(sim_ctx* ctx, const sim_best* bests, int64_t n, sim_best* out_best, void* stream);

/*
 * Kernel timing for measurement.  When enabled, sim_eval_plans records a
 * HIP event pair around each chunk's kernels of one kind and around the
 * whole call; sim_get_timing synchronises those events and returns the
 * accumulated milliseconds and pair counts, then clears them.
 * kind 0 = first evaluation pass (per-pipeline setup and 1F1B recurrence
 * with the periodic shortcut), 1 = plan check/pack kernel, 2 = whole
 * sim_eval_plans call, 3 = deferred pass (full-loop pipelines and the u64
 * redo).  A call of more than 2^22 plans works in chunks of 2^21 and runs
 * each chunk's first pass on two side streams of the context and its
 * deferred pass on a third, overlapped with the next chunk; the call's
 * stream waits for them before the call's work is complete, so kinds 0 and
 * 3 may overlap in time.
 */
int sim_set_timing(sim_ctx* ctx, int enable);
int sim_get_timing(sim_ctx* ctx, int kind, double* total_ms, int64_t* launches);

/*
 * Work measure of the periodic shortcut.  After its warm-up a 1F1B schedule
 * usually becomes periodic: one steady iteration advances every stage's
 * state by the same amount, and so does every later one (the recurrence is
 * a max of sums, Table 1's per-op costs being constants per stage), so the
 * remaining steady iterations are added in one step.  While timing is
 * enabled sim_eval_plans sums, on the device, the recurrence work this
 * skipped: s skipped iterations of an S-stage pipeline count
 * s * (6 (S - 1) + 2) VALU ops, the cost of S forward and S backward nodes
 * at 3 ops per node (1 for a node without a cross-stage input).
 * sim_get_skipped_ops synchronises the device, writes the sum to *ops (host
 * memory) and clears it (it starts at zero).
 */
int sim_get_skipped_ops(sim_ctx* ctx, uint64_t* ops);

/*
 * Release a context.  Waits for the context's own work only: its side
 * streams and the latest call it was given on each caller stream (up to 16
 * caller streams are tracked; past that it waits for the whole device).
 * Calls on a stream under graph capture are not tracked: the caller must
 * not destroy a context that a graph it has not yet finished still uses.
 */
void sim_destroy(sim_ctx* ctx);
const char* sim_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif
