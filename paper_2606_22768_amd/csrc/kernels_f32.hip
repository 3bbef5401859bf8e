// Instantiations of the step and consensus kernels for float32 parameter storage.
#include "kernels.hpp"

namespace fgd {

template <int MMAX, bool EXACT>
static KernelSet set_f32(int k1, int k2) {
    return make_kernel_set<ParamF32, MMAX, EXACT, lanes_v_f32(MMAX)>(k1, k2);
}

bool kernels_f32(int M, int k1, int k2, KernelSet *out) {
    if (M < 1 || M > 64) return false;
    if (M == 1) *out = set_f32<1, true>(k1, k2);
    else if (M == 2) *out = set_f32<2, true>(k1, k2);
    else if (M == 3) *out = set_f32<4, false>(k1, k2);
    else if (M == 4) *out = set_f32<4, true>(k1, k2);
    else if (M < 8) *out = set_f32<8, false>(k1, k2);
    else if (M == 8) *out = set_f32<8, true>(k1, k2);
    else if (M < 16) *out = set_f32<16, false>(k1, k2);
    else if (M == 16) *out = set_f32<16, true>(k1, k2);
    else if (M < 32) *out = set_f32<32, false>(k1, k2);
    else if (M == 32) *out = set_f32<32, true>(k1, k2);
    else if (M < 64) *out = set_f32<64, false>(k1, k2);
    else *out = set_f32<64, true>(k1, k2);
    return true;
}

}  // namespace fgd
