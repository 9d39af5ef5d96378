// Instantiates the SHAP-interaction kernels for fp32 models (every launch shape and
// longest-path variant); kept apart so the variants compile in parallel.
#include "gts_shap_kernel.h"

namespace gts {

gts_status launch_inter_f32(const KernelArgs& a, const Plan& p) {
  return launch_plan<float, true>(a, p);
}

}  // namespace gts
