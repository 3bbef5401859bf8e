// Instantiations of the 64-worker worker-group step kernel (float32 and bf16
// parameter storage).
#include "kernels_wg.hpp"

namespace fgd {

namespace {
template <template <int> class PIOT>
const void *pick(int k1, int k2) {
    using P = PIOT<kWgV>;
    if (k1 == kTable && k2 == kTable) return reinterpret_cast<const void *>(&wg_step_kernel<P, kTable, kTable>);
    if (k1 == kGlobal && k2 == kTable) return reinterpret_cast<const void *>(&wg_step_kernel<P, kGlobal, kTable>);
    return nullptr;
}
}  // namespace

bool wg_kernel(bool bf16, int k1, int k2, WgKernel *out) {
    out->step = bf16 ? pick<ParamBF16>(k1, k2) : pick<ParamF32>(k1, k2);
    out->pattern = bf16 ? reinterpret_cast<const void *>(&wg_pattern_kernel<2>)
                        : reinterpret_cast<const void *>(&wg_pattern_kernel<4>);
    return out->step != nullptr;
}

}  // namespace fgd
