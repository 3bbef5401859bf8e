// Instantiations of the step and consensus kernels for bf16 parameter storage (float32 arithmetic).
#include "kernels.hpp"

namespace fgd {

namespace {
struct Sets {
    template <int MMAX, bool EXACT>
    static KernelSet get(int k1, int k2, bool subset) {
        return make_kernel_set<ParamBF16, MMAX, EXACT, lanes_v_bf16(MMAX)>(k1, k2, subset);
    }
};
}  // namespace

bool kernels_bf16(int M, int k1, int k2, bool subset, KernelSet *out) {
    return select_workers<Sets>(M, out, k1, k2, subset);
}

}  // namespace fgd
