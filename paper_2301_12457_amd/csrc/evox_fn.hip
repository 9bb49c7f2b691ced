// One benchmark function's instantiation of the generation kernels
// (compiled once per function with -DEVOX_FN=<id>).
#include "evox_kernels.hpp"

#ifndef EVOX_FN
#error "compile with -DEVOX_FN=<function id>"
#endif

namespace evox {

template hipError_t launch_pso_t<EVOX_FN>(Layout, int, const PsoArgs &, int, hipStream_t);
template hipError_t launch_pso_small_t<EVOX_FN>(Layout, const PsoArgs &, int64_t, float *, DevBest *, hipStream_t);
template hipError_t launch_eval_t<EVOX_FN>(Layout, bool, const EvalArgs &, int, hipStream_t);
template hipError_t launch_cso_t<EVOX_FN>(Layout, const CsoArgs &, int, hipStream_t);
template hipError_t launch_de_t<EVOX_FN>(Layout, const DeArgs &, int, hipStream_t);
template hipError_t launch_es_eval_t<EVOX_FN>(Layout, const EsArgs &, int, hipStream_t);
template hipError_t launch_mae_eval_t<EVOX_FN>(Layout, const MaeEvalArgs &, int, hipStream_t);
template int occupancy_cso_t<EVOX_FN>(Layout, bool);

}  // namespace evox
