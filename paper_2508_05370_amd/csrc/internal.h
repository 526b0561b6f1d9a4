// internal.h -- context tables shared by the host builder and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <vector>

#include "hetsim.h"

namespace hetsim {

constexpr int kMaxTypes = 16;
constexpr int kMaxStages = 16;
constexpr int kMaxClasses = 4;
constexpr int kRecWords = 4;                    // per (plan, class, stage): fwd, bwd, hop, dp
constexpr int kPlanWords = kMaxClasses * kMaxStages * kRecWords;
constexpr int kBucketsM = 128;                  // micro-batch-count buckets per (stages, classes)
constexpr int kPlainBuckets = kMaxStages * kMaxClasses * kBucketsM;
// Interleaved 1F1B pipelines (S = 2..8 devices, v = 2..4 chunks, S v <= 16)
// sort after all others, in groups keyed (S - 2) * 3 + (v - 2), each of
// kIlBucketsQ micro-batch buckets.
constexpr int kIlGroups = 21;
constexpr int kIlBucketsQ = 48;
constexpr int kBuckets = kPlainBuckets + 1024;
static_assert(kIlGroups * kIlBucketsQ <= 1024, "interleaved buckets");
// sstart: [16 - S] first sorted id of the S-stage pipelines, [16 + q] first
// id of interleaved group q, [16 + kIlGroups] the total
constexpr int kSstartWords = kMaxStages + kIlGroups + 1;
// Plans of the shared layout with one model chunk per device are sorted by
// plan: the G pipelines of a plan take G adjacent lanes of one wavefront,
// every wavefront holds plans of one stage count and one class count (64 / G
// plans of them, 21 when G = 3), and each (stages, classes) bucket starts on
// a wavefront boundary.  kGroupPad bounds the padding lanes this adds to a
// chunk; padding lanes hold kNoSlot.
constexpr uint32_t kSuperBuckets = kMaxStages * kMaxClasses;
constexpr uint32_t kGroupPad = 64 * kSuperBuckets;
constexpr uint32_t kNoSlot = 0xffffffffu;
__host__ __device__ constexpr uint32_t plans_per_wave(uint32_t G) { return G == 3 ? 21 : 64 / G; }
// LDS of the first and variant passes over plan-sorted pipelines: per
// wavefront, a row of DP syncs for each of up to 32 plans (one per stage of
// the kernel's largest stage count, and two more for the embedding's and the
// head's buckets of an overlapped sync), exchanged between the lanes of each
// plan
constexpr uint32_t kXchgPlans = 32;
__host__ __device__ constexpr uint32_t xchg_row(uint32_t S) { return (S + 3) / 4 * 4 + 2; }
__host__ __device__ constexpr uint32_t xchg_wave(int group) { return kXchgPlans * xchg_row(kMaxStages - 4 * group); }
__host__ __device__ constexpr uint32_t xchg_bytes(int group) { return 4 * xchg_wave(group) * 8; }
// The first pass of the two long stage-count groups keeps each lane's stage
// placements (first device in the pool, u32 per stage) in LDS from setup to
// the DP tail, where the plan's lanes read each other's instead of counting
// them again: 64 lanes x the group's longest stage count per wavefront.
__host__ __device__ constexpr uint32_t bcache_words(int group) { return group < 2 ? 64u * (kMaxStages - 4 * group) : 0u; }
__host__ __device__ constexpr uint32_t bcache_bytes(int group) { return 4 * bcache_words(group) * 4; }

// A validated plan packed into 80 contiguous bytes, so that the pipelines of
// one plan gather it with five 16-byte loads.
struct __attribute__((aligned(16))) PackedPlan {
  uint32_t hdr, psum, pad0, pad1;   // header; replicas summed over classes
  uint8_t cut[16];
  uint32_t cls[4];
  uint64_t types[4];
};

// Per-device-type fields a kernel reads together (32 bytes, two loads).
struct TypeInfo {
  uint32_t node_off, dev_off;     // first global node / device of the pool
  uint32_t dpl;                   // log2 devices per node
  uint32_t bq_pcie;               // PCIe ps/byte in 2^-16 units, 0 = absent
  uint64_t a_intra;               // intra-node message latency
  uint64_t a_side;                // one end of an inter-node path: two PCIe trips + NIC
};

// The tables of the per-pipeline setup form one byte image in device memory
// that the evaluation kernels copy into LDS, where lanes gather from it at
// LDS rather than vector-cache rates.  Sections, each 16-byte aligned:
//   TypeInfo [K]; {forward, backward} layer prefix sums
//   [K][4 log2 TP][n_mbs][nep][L+1] (nep = 4 EP slots for MoE models, 1 for
//   dense ones), or, when every layer costs the same (dense models), one
//   {forward, backward} layer cost [K][4][n_mbs] (uniform_layers);
//   {fwd, bwd} embedding [K][n_mbs]; {fwd, bwd} head
//   [K][4][n_mbs]; all-to-all bytes prefix [4][n_mbs][L+1] (MoE only);
//   range-max rows of the node fabric rates [lvl_node][N]; range-max rows
//   of the device NIC rates [lvl_dev][D] (last, the largest).
// mode 0: the whole image fits the LDS budget; 1: all but the device rows
// fit; 2: nothing is copied and every table is read from device memory.
constexpr uint32_t kLdsBudget = 64 * 1024;

// Everything a kernel needs about one (model, cluster) pair.  Scalars travel
// by value in the kernel argument block; tables live in device memory.
struct Tab {
  uint32_t L, K, E, n_mbs, gbs;
  uint32_t mbs[4];
  uint32_t tp_ok;                 // bit j: TP 2^j divides heads, kv heads and MLP widths
  uint32_t ep_ok;                 // bit j: EP 2^j allowed (dense models: EP 1 only)
  uint32_t type_ok[4];            // [log2 TP] bit k: type k exists and TP 2^j divides its node size
  uint32_t D, N;                  // total devices, total nodes
  uint32_t lvl_dev, lvl_node;     // levels of the range-max tables
  uint32_t dpn_log2[kMaxTypes];
  uint32_t cap[kMaxTypes];        // devices per pool
  uint32_t dev_off[kMaxTypes];    // first global device of pool k
  uint32_t node_off[kMaxTypes];   // first global node of pool k
  uint32_t bq_pcie[kMaxTypes];    // PCIe ps/byte in 2^-16 units, 0 = absent
  uint64_t a_intra[kMaxTypes];    // intra-node message latency
  uint64_t a_side[kMaxTypes];     // one end of an inter-node path: two PCIe trips + NIC
  uint32_t tflops[kMaxTypes];     // device speed of pool k (TFLOP/s, GB/s of HBM): the gradient
  uint32_t hbm[kMaxTypes];        // weighting of classes with different micro-batch sizes
  double rtflops[kMaxTypes];      // their reciprocals, rounded to nearest (for exact ceilings)
  double rhbm[kMaxTypes];
  uint64_t act[4];                // bytes of one micro-batch activation per mbs index
  uint64_t grad_bytes, param_bytes;
  uint64_t par_layer[4];          // non-expert parameters of one layer on one TP rank, by log2 TP
  uint64_t par_expert[4][4];      // expert parameters of one layer per rank [log2 TP][log2 EP]
  uint64_t par_embed[4], par_head[4];
  uint32_t mem_check;             // 1: device memory capacities given; plans must fit them
  uint32_t rail_only;             // 1: rail-only inter-node network (cross-rail hops forwarded in a node)
  uint32_t ccl_tree;              // 1: all-reduces take the faster of ring and tree
  uint32_t contention;            // 1: a stage's concurrent segment syncs share its links
  uint32_t ccl_hier;              // 1: whole-node DP groups may take the two-level all-reduce
  uint64_t mem_cap[kMaxTypes];    // device memory of type k, bytes
  uint64_t opt_bytes;             // optimizer-state bytes per parameter
  uint64_t act_layer[4][4];       // bytes one layer stores for backward per micro-batch [log2 TP][mbs index]
  uint32_t nep;                   // EP slots of the prefix tables
  uint32_t uniform_layers;        // 1: the layer table holds one layer's cost per row
  uint32_t o_pfb, o_emb, o_head, o_pa, o_rmi, o_rmn;   // section byte offsets (TypeInfo at 0)
  uint32_t img_bytes;             // whole image
  uint32_t lds_bytes;             // prefix copied to LDS: img_bytes, o_rmn or 0 by mode
  uint32_t mode;
  const void* img;                // the image in device memory (16-byte aligned)
  uint32_t grid_eval[4];          // blocks of each first-pass kernel that fit the device at once
  uint32_t grid_deferred;
  uint32_t grid_variant[4];       // blocks of each variant-pass kernel that fit the device at once
  uint32_t bcache;                // bit g: first-pass group g keeps stage placements in LDS (when that
                                  // costs no occupancy)
};

// Device buffers of one evaluation pass over a chunk, as the host hands them
// to the launcher.  sstart[16 - S] is the first sorted id of the S-stage
// pipelines, sstart[16] their total and the first id of the interleaved
// pipelines (layout above).  ctr[0] counts overflowed pipelines,
// ctr[1 + 16 - S] the S-stage pipelines deferred to the full-loop pass,
// ctr[kVariantCtr + 16 - S] the slots of the S-stage overlap and zero-bubble
// tiles of the variant pass (64 per tile); the per-class layout's plan-order
// counters (kPlanSortWords) follow the evaluation counters at ctr +
// kEvalCounters, and the overflow list follows them at ctr + kEvalCounters +
// kPlanSortWords.
constexpr uint32_t kVariantCtr = 1 + kMaxStages;
// The deferred lists are sorted by micro-batch count before the deferred
// pass (longest first, kSortBuckets buckets per stage count): their counts
// at ctr[kSortCtr + 32 j + b], cursors at ctr[kSortCtr + 512 + 32 j + b] for
// the list of 16 - j stages.
constexpr uint32_t kSortBuckets = 32;
constexpr uint32_t kSortCtr = 48;
constexpr uint32_t kEvalCounters = kSortCtr + 2 * kMaxStages * kSortBuckets;
// Per-class layout: plans counting-sorted by (classes, total stages) before
// the plan-level sync pass -- counts [0, 256), cursors [256, 512), the
// number of valid plans at 512.
constexpr uint32_t kPlanBuckets = 256;
constexpr uint32_t kPlanSortWords = 2 * kPlanBuckets + 1;
static_assert(kVariantCtr + kMaxStages <= kSortCtr, "evaluation counters");
// The skipped-work counter is spread over slots on separate cache lines so
// that the waves of a launch do not serialise on one address.
constexpr uint32_t kSkipSlots = 512, kSkipStride = 16;
struct EvalArgs {
  const PackedPlan* packed;
  const void* pcut;            // per-class layout: four 16-byte cut rows per plan; nullptr for the shared layout
  const uint64_t* hdp;         // per-class layout: per pipeline slot, the syncs its 16 stages wait for
  const uint32_t* meta;
  const uint32_t* ids;
  const uint32_t* sstart;
  uint64_t* out;
  uint32_t* ctr;
  uint32_t* deferred;          // as long as ids
  uint32_t* vlist;             // as long as ids: overlap and zero-bubble tiles (kNoSlot where empty)
  uint64_t* skipped_ops;       // optional: kSkipSlots counters, kSkipStride words apart
  const Tab* dtab;             // the context's Tab in device memory (read by the deferred pass)
};

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace of one chunk: packed plans, pipeline metadata, pipeline ids and
// the deferred lists, bucket counts followed by the evaluation counters and
// the overflow list (counts and counters cleared together), bucket cursors,
// the start of each stage count's pipelines, each pipeline's bucket key
// (u16, written with the metadata and read by the scatter), and with the
// per-class layout
// the plans' class cut rows (64 bytes per plan) and the syncs each pipeline's
// stages wait for (16 u64 per pipeline slot, 512 bytes per plan).
constexpr uint32_t kCounters = kBuckets + kEvalCounters + kPlanSortWords;
struct Work {
  PackedPlan* packed;
  uint4* pcut;
  uint64_t* hdp;
  uint32_t *meta, *ids, *deferred, *vlist, *hist, *ctr, *cursor, *sstart, *sbase;
  uint16_t* keys;
};
// sorted ids (and deferred lists) of a chunk: four lanes per plan at most,
// plus the padding of the plan-sorted buckets
constexpr size_t id_words(int64_t ch) { return (size_t)ch * 4 + kGroupPad; }
constexpr size_t cut_rows_bytes(int64_t ch, bool het) { return het ? align256((size_t)ch * 64) : 0; }
constexpr size_t het_sync_bytes(int64_t ch, bool het) {
  return het ? align256((size_t)ch * kMaxClasses * kMaxStages * 8) : 0;
}
constexpr size_t work_bytes(int64_t ch, bool het) {
  return align256((size_t)ch * sizeof(PackedPlan)) + align256((size_t)ch * 4 * 4) + 3 * align256(id_words(ch) * 4) +
         align256(kCounters * 4 + (size_t)ch * 4 * 4) + align256(kBuckets * 4) + align256(kSstartWords * 4) +
         align256(kSuperBuckets * 4) + align256((size_t)ch * 4 * 2) +
         cut_rows_bytes(ch, het) + het_sync_bytes(ch, het);
}
inline Work carve(void* base, int64_t ch, bool het) {
  Work w;
  char* p = (char*)base;
  w.pcut = het ? (uint4*)p : nullptr; p += cut_rows_bytes(ch, het);
  w.hdp = het ? (uint64_t*)p : nullptr; p += het_sync_bytes(ch, het);
  w.packed = (PackedPlan*)p; p += align256((size_t)ch * sizeof(PackedPlan));
  w.meta = (uint32_t*)p; p += align256((size_t)ch * 16);
  w.ids = (uint32_t*)p; p += align256(id_words(ch) * 4);
  w.deferred = (uint32_t*)p; p += align256(id_words(ch) * 4);
  w.vlist = (uint32_t*)p; p += align256(id_words(ch) * 4);
  w.hist = (uint32_t*)p; w.ctr = w.hist + kBuckets; p += align256(kCounters * 4 + (size_t)ch * 16);
  w.cursor = (uint32_t*)p; p += align256(kBuckets * 4);
  w.sstart = (uint32_t*)p; p += align256(kSstartWords * 4);
  w.sbase = (uint32_t*)p; p += align256(kSuperBuckets * 4);
  w.keys = (uint16_t*)p;
  return w;
}

// The allocation-free entry point's workspace: one chunk of at most
// kNoAllocPlans plans in the shared layout or kNoAllocPlansHet in the
// per-class layout, in a static device array (one per GPU).
constexpr int64_t kNoAllocPlans = 1 << 18;
constexpr int64_t kNoAllocPlansHet = 1 << 16;
constexpr size_t kNoAllocBytes = work_bytes(kNoAllocPlans, false) > work_bytes(kNoAllocPlansHet, true)
                                     ? work_bytes(kNoAllocPlans, false)
                                     : work_bytes(kNoAllocPlansHet, true);
// Address of this device's copy of that array (the current device); 0 or a
// HIP error code.
int noalloc_scratch(int device, void** ptr);

// Host side: validate descriptors and build the tables (host copies).
struct HostTables {
  Tab tab;
  // pf, pb [K][4][n_mbs][4][L+1]; emb [K][n_mbs][2]; head [K][4][n_mbs][2]; pa [4][n_mbs][L+1]
  std::vector<uint64_t> pf, pb, emb, head, pa;
  std::vector<uint32_t> rm_nic, rm_intra;
  std::vector<TypeInfo> ty;
  std::vector<uint8_t> img;       // the device image built from the above
};

// Blocks of each evaluation kernel that fit the current device at once (they
// size the capped grids).  Returns a HIP error code.
int eval_grids(Tab* t);

// Returns 0 (SIM_OK), SIM_EINVAL or SIM_ERANGE.
int build_tables(const sim_model_desc* model, const sim_cluster_desc* cluster, HostTables* out);

}  // namespace hetsim
