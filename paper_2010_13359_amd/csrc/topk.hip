// Top-k compressor (Theorem 1 of arXiv:2010.13359): placeholder launchers,
// replaced by the radix-select path.
#include "plan.hpp"

namespace dq {

hipError_t topk_alloc(dqgan_plan_s &) { return hipSuccess; }
void topk_free(dqgan_plan_s &) {}
hipError_t launch_topk_compress(const dqgan_plan_s &, float, const float *, float *, const dqgan_wire &, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_topk_select(const dqgan_plan_s &, float, const float *, const float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_topk_apply(const dqgan_plan_s &, float, const float *, float *, float *, float *, const dqgan_wire &,
                             float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_topk_unpack(const dqgan_plan_s &, const dqgan_wire &, float *, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_topk_aggregate(const dqgan_plan_s &, const dqgan_wire &, float *, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace dq
