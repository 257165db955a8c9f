// Backward kernels (placeholder until the backward lands).
#include "tla_common.hpp"
#include "tla_internal.hpp"

namespace tla {

hipError_t launch_bwd_rec(const Shape&, const FwdIn&, const void*, const float*, const PrepBufs&,
                          const BwdBufs&, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_bwd_state(const Shape&, const FwdIn&, const void*, const PrepBufs&,
                            const SavedBufs&, const BwdBufs&, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_bwd_chunk(const Shape&, const FwdIn&, const void*, const SavedBufs&,
                            const BwdBufs&, void*, void*, void*, void*, void*, float*, float*,
                            hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace tla
