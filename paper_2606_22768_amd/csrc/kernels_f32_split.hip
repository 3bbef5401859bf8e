// Split-execution kernels for float32 parameter storage: the Mix1 half and the blocking
// half of a round (Appendix A, Algorithm 1).
#include "kernels.hpp"

namespace fgd {

namespace {
struct Sets {
    template <int MMAX, bool EXACT>
    static SplitSet get(int k1, int k2, bool subset, bool mix_state) {
        return make_split_set<ParamF32, MMAX, EXACT, lanes_v_f32(MMAX)>(k1, k2, subset, mix_state);
    }
};
}  // namespace

bool split_kernels_f32(int M, int k1, int k2, bool subset, bool mix_state, SplitSet *out) {
    return select_workers<Sets>(M, out, k1, k2, subset, mix_state);
}

}  // namespace fgd
