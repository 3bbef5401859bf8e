// Kernels shared by every instantiation: consensus finalize and the plain
// streaming copy used as the bandwidth reference.
#include "kernels.hpp"

namespace fgd {

// One block per output entry i: thread t sums partials[b][i] for b = t, t +
// 256, ... in ascending b, then a fixed-shape tree in LDS adds the 256
// thread sums.  The order of additions never changes, so the result is
// deterministic.
__global__ __launch_bounds__(256) void finalize_kernel(const double *partials, int nblocks, int n, double *out) {
    __shared__ double s[256];
    const int i = blockIdx.x, t = threadIdx.x;
    double acc = 0.0;
    for (int b = t; b < nblocks; b += 256) acc += partials[static_cast<int64_t>(b) * n + i];
    s[t] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) s[t] += s[t + w];
        __syncthreads();
    }
    if (t == 0) out[i] = s[0];
}

__global__ void counter_reset_kernel(int *counter) {
    if (threadIdx.x == 0 && blockIdx.x == 0) counter[0] = 0;
}

// Each block iteration moves 4 vectors of 16 bytes per thread; all four loads
// are issued before the stores.
__global__ __launch_bounds__(256) void copy_kernel(const u32x4 *src, u32x4 *dst, int64_t n) {
    constexpr int kUnroll = 4;
    const int64_t chunk = static_cast<int64_t>(blockDim.x) * kUnroll;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * chunk; base < n; base += static_cast<int64_t>(gridDim.x) * chunk) {
        u32x4 r[kUnroll];
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const int64_t i = base + j * blockDim.x + threadIdx.x;
            if (i < n) r[j] = __builtin_nontemporal_load(src + i);
        }
#pragma unroll
        for (int j = 0; j < kUnroll; ++j) {
            const int64_t i = base + j * blockDim.x + threadIdx.x;
            if (i < n) __builtin_nontemporal_store(r[j], dst + i);
        }
    }
}

namespace {
template <int M>
void pattern_pick(bool bf16, const void **kernel, int *v, int *bpc) {
    if (bf16) {
        constexpr int V = lanes_v_bf16(M);
        *kernel = reinterpret_cast<const void *>(&pattern_kernel<M, V, 2>);
        *v = V;
    } else {
        constexpr int V = lanes_v_f32(M);
        *kernel = reinterpret_cast<const void *>(&pattern_kernel<M, V, 4>);
        *v = V;
    }
    *bpc = step_blocks_per_cu(M);
}
}  // namespace

bool pattern_kernel_for(int M, bool bf16, const void **kernel, int *v, int *blocks_per_cu) {
    switch (M) {
        case 1: pattern_pick<1>(bf16, kernel, v, blocks_per_cu); return true;
        case 2: pattern_pick<2>(bf16, kernel, v, blocks_per_cu); return true;
        case 4: pattern_pick<4>(bf16, kernel, v, blocks_per_cu); return true;
        case 8: pattern_pick<8>(bf16, kernel, v, blocks_per_cu); return true;
        case 16: pattern_pick<16>(bf16, kernel, v, blocks_per_cu); return true;
        case 32: pattern_pick<32>(bf16, kernel, v, blocks_per_cu); return true;
        case 64: pattern_pick<64>(bf16, kernel, v, blocks_per_cu); return true;
        default: return false;
    }
}

}  // namespace fgd
