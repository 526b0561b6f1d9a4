// eval_pass.hip -- one evaluation pass of one variant: table mode HETSIM_MODE
// (0..2), plan layout HETSIM_HET (0 shared, 1 per class), pass HETSIM_PASS
// (0 the first pass's k_eval groups, 1 the deferred pass, 2 the variant pass
// of overlap and zero-bubble pipelines).  The build
// compiles this file once per variant; kernels.hip dispatches at run time.
#include "launch.h"

#if !defined(HETSIM_MODE) || !defined(HETSIM_HET) || !defined(HETSIM_PASS)
#error "eval_pass.hip is built once per variant: define HETSIM_MODE, HETSIM_HET and HETSIM_PASS"
#endif

namespace hetsim {

[[maybe_unused]] static int pass_blocks(uint32_t n, uint32_t per) { return (int)((n + per - 1) / per); }

#if HETSIM_PASS == 0
template <int kMode, bool kHet>
hipError_t launch_group_v(const Tab& t, const EvalArgs& a, uint32_t max_tasks, int g, hipStream_t s) {
  const EvalBufs e = eval_bufs(a);
  const int nb = pass_blocks(max_tasks, kEvalThreads);
  const uint32_t need = nb > 0 ? (uint32_t)nb : 1, grid = 4 * t.grid_eval[g] < need ? 4 * t.grid_eval[g] : need;
  // the shared layout's plan-sorted groups add their plans' DP exchange area
  const size_t lds = (kMode < 2 ? t.lds_bytes : 0) +
                    (!kHet ? xchg_bytes(g) + (((t.bcache >> g) & 1) ? bcache_bytes(g) : 0) : 0);
  if (g == 0) k_eval<0, kMode, kHet><<<grid, kEvalThreads, lds, s>>>(t, e);
  else if (g == 1) k_eval<1, kMode, kHet><<<grid, kEvalThreads, lds, s>>>(t, e);
  else if (g == 2) k_eval<2, kMode, kHet><<<grid, kEvalThreads, lds, s>>>(t, e);
  else k_eval<3, kMode, kHet><<<grid, kEvalThreads, lds, s>>>(t, e);
  return hipGetLastError();
}
template hipError_t launch_group_v<HETSIM_MODE, (bool)HETSIM_HET>(const Tab&, const EvalArgs&, uint32_t, int,
                                                                  hipStream_t);

#if !HETSIM_HET
// Grid caps come from the shared-layout kernels; the per-class-layout ones
// take the same caps (their fixed-stride loops cover any grid).
// bcache: the groups whose stage-placement cache is counted (bit g)
template <int kMode>
hipError_t occupancy_first_v(int nb[4], size_t lds, uint32_t bcache) {
  const void* k[4] = {(const void*)k_eval<0, kMode, false>, (const void*)k_eval<1, kMode, false>,
                      (const void*)k_eval<2, kMode, false>, (const void*)k_eval<3, kMode, false>};
  for (int i = 0; i < 4; ++i) {
    const size_t b = lds + xchg_bytes(i) + (((bcache >> i) & 1) ? bcache_bytes(i) : 0);
    hipError_t r = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb[i], k[i], kEvalThreads, b);
    if (r != hipSuccess) return r;
  }
  return hipSuccess;
}
template hipError_t occupancy_first_v<HETSIM_MODE>(int[4], size_t, uint32_t);
#endif

#elif HETSIM_PASS == 2
// overlap and zero-bubble pipelines exist in the shared layout only
#if HETSIM_HET
#error "the variant pass is built for the shared layout only"
#endif
template <int kMode>
hipError_t launch_variant_v(const Tab& t, const EvalArgs& a, int g, hipStream_t s) {
  const EvalBufs e = eval_bufs(a);
  const uint32_t grid = t.grid_variant[g];
  const size_t lds = (kMode < 2 ? t.lds_bytes : 0) + xchg_bytes(g);
  if (g == 0) k_variant<0, kMode><<<grid, kEvalThreads, lds, s>>>(e.dtab, e);
  else if (g == 1) k_variant<1, kMode><<<grid, kEvalThreads, lds, s>>>(e.dtab, e);
  else if (g == 2) k_variant<2, kMode><<<grid, kEvalThreads, lds, s>>>(e.dtab, e);
  else k_variant<3, kMode><<<grid, kEvalThreads, lds, s>>>(e.dtab, e);
  return hipGetLastError();
}
template hipError_t launch_variant_v<HETSIM_MODE>(const Tab&, const EvalArgs&, int, hipStream_t);

template <int kMode>
hipError_t occupancy_variant_v(int nb[4], size_t lds) {
  const void* k[4] = {(const void*)k_variant<0, kMode>, (const void*)k_variant<1, kMode>,
                      (const void*)k_variant<2, kMode>, (const void*)k_variant<3, kMode>};
  for (int i = 0; i < 4; ++i) {
    hipError_t r = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb[i], k[i], kEvalThreads, lds + xchg_bytes(i));
    if (r != hipSuccess) return r;
  }
  return hipSuccess;
}
template hipError_t occupancy_variant_v<HETSIM_MODE>(int[4], size_t);

#else
template <int kMode, bool kHet>
hipError_t launch_deferred_v(const Tab& t, const EvalArgs& a, uint32_t max_tasks, hipStream_t s) {
  const EvalBufs e = eval_bufs(a);
  int g = pass_blocks(max_tasks, kEvalThreads);
  g = g < 1 ? 1 : (g > (int)t.grid_deferred ? (int)t.grid_deferred : g);
  const size_t lds = kMode < 2 ? t.lds_bytes : 0;
  k_deferred<kMode, kHet><<<g, kEvalThreads, lds, s>>>(e.dtab, e);
  return hipGetLastError();
}
template hipError_t launch_deferred_v<HETSIM_MODE, (bool)HETSIM_HET>(const Tab&, const EvalArgs&, uint32_t,
                                                                     hipStream_t);

#if !HETSIM_HET
template <int kMode>
hipError_t occupancy_deferred_v(int nb[1], size_t lds) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb[0], (const void*)k_deferred<kMode, false>, kEvalThreads,
                                                      lds);
}
template hipError_t occupancy_deferred_v<HETSIM_MODE>(int[1], size_t);
#endif
#endif

}  // namespace hetsim
