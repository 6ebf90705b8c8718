// Construction kernels (placeholder until the construction pass lands).
#include "common.h"
#include "internal.h"

namespace reskv {

bool make_build_plan(const reskv_shape_t&, const reskv_build_params_t&, const int32_t*, const int32_t*,
                     const int32_t*, BuildPlan*) {
  return false;
}

hipError_t launch_build(const reskv_shape_t&, const reskv_build_params_t&, const BuildPlan&, const void*,
                        const void*, const int32_t*, const void*, const int32_t*, const int32_t*, void*, void*,
                        float*, int32_t*, int32_t*, int32_t*, float*, int32_t*, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace reskv
