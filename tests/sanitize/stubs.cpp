// Test infrastructure: stand-ins for the kernel launches, so that the host
// logic of the library (plans, job layouts, schedule, planner, argument
// checks) can be built with the host sanitizers into an executable that
// never touches a GPU (lin.hip is linked as it is: its host part sizes the
// wide-layer product's grid).  Every launch reports failure; the driver
// calls no entry point that would launch.
#include "../../paper_2510_12494_amd/csrc/kernels.h"

namespace vfl {
static hipError_t no_gpu() { return hipErrorNotSupported; }
hipError_t launch_tick_base(TickSrc*, int, hipStream_t) { return no_gpu(); }
hipError_t launch_tick_set(TickSrc*, const TickSrc&, hipStream_t) { return no_gpu(); }
hipError_t launch_fwd(Elt, int, int, const FwdJob*, int, int, const ChainCall&, TickRef, hipStream_t) { return no_gpu(); }
hipError_t launch_active(Elt, int, int, const ActiveJob*, int, int, const ChainCall&, TickRef, hipStream_t) { return no_gpu(); }
hipError_t launch_bwd(Elt, int, int, const BwdJob*, int, int, const ChainCall&, TickRef, hipStream_t) { return no_gpu(); }
hipError_t chain_init() { return no_gpu(); }
hipError_t launch_dw(Elt, const DwJob*, int, int, float, TickRef, hipStream_t) { return no_gpu(); }
hipError_t dwt_init() { return no_gpu(); }
hipError_t launch_dwt(const DwJob*, int, hipStream_t) { return no_gpu(); }
hipError_t launch_dw32(Elt, const DwJob*, int, int, float, float*, TickRef, float*, hipStream_t) { return no_gpu(); }
hipError_t launch_dw_reduce(Elt, const DwJob*, int, int, float, float*, TickRef, float*, hipStream_t) { return no_gpu(); }
hipError_t launch_avg(const AvgJob&, hipStream_t) { return no_gpu(); }
hipError_t launch_cast(Elt, const CastJob*, int, hipStream_t) { return no_gpu(); }
hipError_t launch_scatter_sgd(const ScatterJob&, hipStream_t) { return no_gpu(); }
hipError_t launch_philox_words(uint64_t, uint32_t, uint32_t, uint32_t, int, int, uint32_t*, hipStream_t) { return no_gpu(); }
}  // namespace vfl
