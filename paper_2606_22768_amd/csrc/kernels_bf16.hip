// Instantiations of the step and consensus kernels for bf16 parameter storage (float32 arithmetic).
#include "kernels.hpp"

namespace fgd {

template <int MMAX, bool EXACT>
static KernelSet set_bf16(int k1, int k2) {
    return make_kernel_set<ParamBF16, MMAX, EXACT, lanes_v_bf16(MMAX)>(k1, k2);
}

bool kernels_bf16(int M, int k1, int k2, KernelSet *out) {
    if (M < 1 || M > 64) return false;
    if (M == 1) *out = set_bf16<1, true>(k1, k2);
    else if (M == 2) *out = set_bf16<2, true>(k1, k2);
    else if (M == 3) *out = set_bf16<4, false>(k1, k2);
    else if (M == 4) *out = set_bf16<4, true>(k1, k2);
    else if (M < 8) *out = set_bf16<8, false>(k1, k2);
    else if (M == 8) *out = set_bf16<8, true>(k1, k2);
    else if (M < 16) *out = set_bf16<16, false>(k1, k2);
    else if (M == 16) *out = set_bf16<16, true>(k1, k2);
    else if (M < 32) *out = set_bf16<32, false>(k1, k2);
    else if (M == 32) *out = set_bf16<32, true>(k1, k2);
    else if (M < 64) *out = set_bf16<64, false>(k1, k2);
    else *out = set_bf16<64, true>(k1, k2);
    return true;
}

}  // namespace fgd
