// Host-only stand-ins for the device launchers, so that the C-ABI layer can
// be built with g++ and run under AddressSanitizer / UBSan without a GPU.
// Only the schedule builder and the argument checks are exercised; a call
// that would reach a kernel returns hipErrorNotSupported.
#include "fg_internal.h"

namespace fg {

hipError_t launch_gspmm(const GraphView&, const PlanView*, int, int, int64_t, int64_t, const float*,
                        const float*, float*, int32_t*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_gsddmm(const GraphView&, const PlanView*, int64_t, int64_t, const float*,
                         const float*, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_edge_softmax(const GraphView&, const PlanView*, int64_t, const float*, bool, float,
                               float*, hipStream_t) {
  return hipErrorNotSupported;
}
bool gsddmm_softmax_fused(int64_t, int64_t, const float*, const float*) { return false; }
hipError_t launch_gsddmm_softmax(const GraphView&, const PlanView*, int64_t, const float*,
                                 const float*, bool, float, float*, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_gspmm_max_backward(const GraphView&, const int32_t*, int, int64_t, int64_t,
                                     const float*, const float*, const int32_t*, const float*, float*,
                                     float*, const BinWorkspace*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_edge_softmax_backward(const GraphView&, const PlanView*, int64_t, const float*,
                                        const float*, const float*, bool, float, float*,
                                        hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_gsddmm_softmax_backward(const GraphView&, const PlanView*, const PlanView*,
                                          int64_t, int64_t, const float*, const float*,
                                          const float*, const float*, bool, float, float*,
                                          hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t noalloc_scratch(void**) { return hipErrorNotSupported; }
hipError_t launch_build_eid_pos(const int32_t*, int64_t, int64_t, int32_t*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_dense_matmul(int64_t, int64_t, int64_t, const float*, const float*, float*,
                               hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_mlp_aggregate(const GraphView&, const PlanView*, int64_t, int64_t, const float*,
                                const float*, const float*, float*, int32_t*, float*, hipStream_t) {
  return hipErrorNotSupported;
}
bool gat_fused_supported(int64_t, int64_t) { return true; }
hipError_t launch_gat_fused(const GraphView&, const PlanView*, int64_t, int64_t, const float*,
                            const float*, bool, float, float*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace fg
