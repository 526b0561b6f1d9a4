// launch.h -- host-side launchers of the evaluation kernels.  The first and
// the deferred pass of each (table mode, plan layout) pair are compiled in
// translation units of their own (eval_pass.hip built once per variant), so
// that the library builds in parallel; kernels.hip dispatches to them.
#pragma once
#include "device.h"

namespace hetsim {

// First pass of stage-count group g (0..3: 16-13, 12-9, 8-5, 4-1 stages).
template <int kMode, bool kHet>
hipError_t launch_group_v(const Tab& t, const EvalArgs& a, uint32_t max_tasks, int g, hipStream_t s);
// Deferred pass: interleaved pipelines, then every deferred list.
template <int kMode, bool kHet>
hipError_t launch_deferred_v(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s);
// Blocks per CU of the shared-layout first-pass kernels (nb[0..3]) or of the
// deferred kernel (nb[0]) at the given LDS size.
// Variant pass of stage-count group g: overlap and zero-bubble pipelines.
template <int kMode>
hipError_t launch_variant_v(const Tab& t, const EvalArgs& a, int g, hipStream_t s);
template <int kMode>
hipError_t occupancy_first_v(int nb[4], size_t lds, uint32_t bcache);
template <int kMode>
hipError_t occupancy_variant_v(int nb[4], size_t lds);
template <int kMode>
hipError_t occupancy_deferred_v(int nb[1], size_t lds);

#define HETSIM_EXTERN_VARIANT(M, H)                                                                         \
  extern template hipError_t launch_group_v<M, H>(const Tab&, const EvalArgs&, uint32_t, int, hipStream_t); \
  extern template hipError_t launch_deferred_v<M, H>(const Tab&, const EvalArgs&, uint32_t, hipStream_t);
HETSIM_EXTERN_VARIANT(0, false)
HETSIM_EXTERN_VARIANT(0, true)
HETSIM_EXTERN_VARIANT(1, false)
HETSIM_EXTERN_VARIANT(1, true)
HETSIM_EXTERN_VARIANT(2, false)
HETSIM_EXTERN_VARIANT(2, true)
#undef HETSIM_EXTERN_VARIANT
extern template hipError_t launch_variant_v<0>(const Tab&, const EvalArgs&, int, hipStream_t);
extern template hipError_t launch_variant_v<1>(const Tab&, const EvalArgs&, int, hipStream_t);
extern template hipError_t launch_variant_v<2>(const Tab&, const EvalArgs&, int, hipStream_t);
extern template hipError_t occupancy_variant_v<0>(int[4], size_t);
extern template hipError_t occupancy_variant_v<1>(int[4], size_t);
extern template hipError_t occupancy_variant_v<2>(int[4], size_t);
extern template hipError_t occupancy_first_v<0>(int[4], size_t, uint32_t);
extern template hipError_t occupancy_first_v<1>(int[4], size_t, uint32_t);
extern template hipError_t occupancy_first_v<2>(int[4], size_t, uint32_t);
extern template hipError_t occupancy_deferred_v<0>(int[1], size_t);
extern template hipError_t occupancy_deferred_v<1>(int[1], size_t);
extern template hipError_t occupancy_deferred_v<2>(int[1], size_t);

// EvalArgs -> the kernels' buffer view
EvalBufs eval_bufs(const EvalArgs& a);

}  // namespace hetsim
