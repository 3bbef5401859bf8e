// js.hip -- Jensen--Shannon functional distance between each worker's
// predicted token distribution and the parameter-averaged model's
// (Sec. 4.4, JS distance; Appendix D.2, JS functional disagreement).
//
// For token u (one block per token), in float64 and in the log domain:
//   lse_a        = log sum_i exp(zbar_i)              averaged model's row
//   T            = the k largest zbar_i (ties: lower index first), found by a
//                  radix select over order-preserving integer keys of the
//                  stored logits (exact comparisons: no rounding decides it)
//   for every worker m:
//     lse_m      = log sum_i exp(z_m,i)               a streaming pass over the row
//     JS_m       = sum over i in T of the per-token terms
//                  1/2 p (lp - lmix) + 1/2 q (lq - lmix), lp = z_m,i - lse_m,
//                  lq = zbar_i - lse_a, lmix = log((p + q) / 2)
//     d_m(u)     = sqrt(max(JS_m, 0) / log 2)
// Probabilities are those of the full softmax; only the sum is restricted to
// T.  The log-sum-exp of a row is an online (max, scaled sum) reduction, one
// float64 exp per element plus one per 16-byte vector when the running max
// grows; every reduction has a fixed order, so results are deterministic.
// The selected indices are rank-sorted so that the JS sum runs in index
// order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace fgd {

constexpr int kJsMaxTopK = 1024;

struct JsParams {
    const void *avg;      // [U][ldk] logits of the averaged model
    const void *workers;  // [M][U][ldk] logits of every worker
    double *d_out;        // [M][U]
    int32_t *topk_out;    // [U][k] or nullptr
    int64_t U, K, ldk;
    int32_t M, k;
};

// 16 bytes of logits: float values and order-preserving keys (ascending key
// = ascending value; -0 and +0 share the key of +0).
struct JsF32 {
    static constexpr int kPer = 4, kElem = 4, kKeyBits = 32;
    __device__ static void unpack(u32x4 t, float (&v)[kPer], uint32_t (&key)[kPer]) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t b = t[j];
            if ((b & 0x7FFFFFFFu) == 0) b = 0;
            v[j] = __uint_as_float(b);
            key[j] = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
        }
    }
    __device__ static float at(rsrc_t r, int64_t i) {
        return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, static_cast<uint32_t>(i * 4), 0, 0));
    }
};

struct JsBF16 {
    static constexpr int kPer = 8, kElem = 2, kKeyBits = 16;
    __device__ static void unpack(u32x4 t, float (&v)[kPer], uint32_t (&key)[kPer]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t h = (t[j / 2] >> (16 * (j % 2))) & 0xFFFFu;
            if ((h & 0x7FFFu) == 0) h = 0;
            v[j] = __uint_as_float(h << 16);
            key[j] = (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
        }
    }
    __device__ static float at(rsrc_t r, int64_t i) {
        const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(r, static_cast<uint32_t>(i * 2), 0, 0);
        return __uint_as_float(h << 16);
    }
};

__device__ inline rsrc_t js_row(const void *base, int64_t row, int64_t ldk, int es) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(base)) + row * ldk * es,
                                             static_cast<short>(0), 0x7fffffff, kRawBufferFlags);
}

// (max, sum of exp(x - max)) pairs: the combination is symmetric, so every
// lane of a butterfly ends with the same value.
__device__ inline void lse_combine(double &m, double &s, double m2, double s2) {
    const double mm = m > m2 ? m : m2;
    if (mm == -INFINITY) return;  // both empty
    const double a = m == -INFINITY ? 0.0 : s * exp(m - mm);
    const double b = m2 == -INFINITY ? 0.0 : s2 * exp(m2 - mm);
    m = mm;
    s = a + b;
}

__device__ inline double shfl_xor_d(double x, int mask) {
    const int64_t b = __double_as_longlong(x);
    const int lo = __shfl_xor(static_cast<int>(b & 0xFFFFFFFF), mask);
    const int hi = __shfl_xor(static_cast<int>(b >> 32), mask);
    return __longlong_as_double((static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo));
}

// Block-wide log-sum-exp of per-thread (m, s); every thread gets the result.
__device__ inline double block_lse(double m, double s, double *red) {
    for (int o = kWave / 2; o > 0; o >>= 1) lse_combine(m, s, shfl_xor_d(m, o), shfl_xor_d(s, o));
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) {
        red[2 * wave] = m;
        red[2 * wave + 1] = s;
    }
    __syncthreads();
    double M = red[0], S = red[1];
    for (int w = 1; w < kWavesPerBlock; ++w) lse_combine(M, S, red[2 * w], red[2 * w + 1]);
    return M == -INFINITY ? -INFINITY : M + log(S);
}

// Block-wide sum in a fixed order; every thread gets the result.
__device__ inline double block_sum(double x, double *red) {
    for (int o = kWave / 2; o > 0; o >>= 1) x += shfl_xor_d(x, o);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) red[wave] = x;
    __syncthreads();
    double t = red[0];
    for (int w = 1; w < kWavesPerBlock; ++w) t += red[w];
    return t;
}

// One 16-byte vector of a row: values, keys and how many lie below K.
template <class E>
__device__ inline int load_vec(rsrc_t r, int64_t i0, int64_t K, float (&v)[E::kPer], uint32_t (&key)[E::kPer]) {
    const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<uint32_t>(i0 * E::kElem), 0, kLoadPolicy);
    E::unpack(t, v, key);
    const int64_t left = K - i0;
    return left >= E::kPer ? E::kPer : static_cast<int>(left);
}

// Online (max, scaled sum) over the valid values of one vector.
template <int N>
__device__ inline void lse_add(double &m, double &s, const float (&v)[N], int n) {
    float vm = -INFINITY;
#pragma unroll
    for (int j = 0; j < N; ++j)
        if (j < n) vm = fmaxf(vm, v[j]);
    if (vm == -INFINITY) return;
    const double dm = vm;
    if (dm > m) {
        s = m == -INFINITY ? 0.0 : s * exp(m - dm);
        m = dm;
    }
#pragma unroll
    for (int j = 0; j < N; ++j)
        if (j < n) s += exp(static_cast<double>(v[j]) - m);
}

template <class E>
__global__ __launch_bounds__(kBlock) void js_kernel(JsParams a) {
    constexpr int P = E::kPer;
    constexpr int64_t kStride = static_cast<int64_t>(kBlock) * P;  // elements per block sweep
    __shared__ uint32_t hist[256];
    __shared__ int32_t sel_idx[kJsMaxTopK], sorted_idx[kJsMaxTopK];
    __shared__ float sel_val[kJsMaxTopK];
    __shared__ double la[kJsMaxTopK];
    __shared__ double red[2 * kWavesPerBlock];
    __shared__ uint32_t s_prefix;
    __shared__ int s_need, s_count_eq, s_nsel;
    __shared__ int s_scan[kBlock];

    const int tid = threadIdx.x;
    const int64_t u = blockIdx.x;
    const int k = a.k;
    const rsrc_t ra = js_row(a.avg, u, a.ldk, E::kElem);

    // Pass 1 over the averaged row: log-sum-exp and the histogram of the top
    // key byte.
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    double m = -INFINITY, s = 0.0;
    for (int64_t i0 = static_cast<int64_t>(tid) * P; i0 < a.K; i0 += kStride) {
        float v[P];
        uint32_t key[P];
        const int n = load_vec<E>(ra, i0, a.K, v, key);
        lse_add<P>(m, s, v, n);
#pragma unroll
        for (int j = 0; j < P; ++j)
            if (j < n) atomicAdd(&hist[key[j] >> (E::kKeyBits - 8)], 1u);
    }
    const double lse_a = block_lse(m, s, red);

    // Radix select of the k-th largest key, 8 bits per pass from the top.
    uint32_t prefix = 0;
    int need = k;
    for (int pass = 0; pass < E::kKeyBits / 8; ++pass) {
        const int shift = E::kKeyBits - 8 * (pass + 1);
        if (pass > 0) {
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
            for (int64_t i0 = static_cast<int64_t>(tid) * P; i0 < a.K; i0 += kStride) {
                float v[P];
                uint32_t key[P];
                const int n = load_vec<E>(ra, i0, a.K, v, key);
#pragma unroll
                for (int j = 0; j < P; ++j)
                    if (j < n && (key[j] >> (shift + 8)) == prefix) atomicAdd(&hist[(key[j] >> shift) & 255u], 1u);
            }
        }
        __syncthreads();
        if (tid == 0) {
            int above = 0, bin = 255;
            for (; bin > 0; --bin) {
                if (above + static_cast<int>(hist[bin]) >= need) break;
                above += hist[bin];
            }
            s_prefix = (prefix << 8) | static_cast<uint32_t>(bin);
            s_need = need - above;
            s_count_eq = hist[bin];
        }
        __syncthreads();
        prefix = s_prefix;
        need = s_need;
    }
    const uint32_t T = prefix;
    const int need_eq = need;
    const bool take_all_eq = s_count_eq == need_eq;

    // Collect the keys above T (and those equal to T when all of them are
    // taken); the list order does not matter, it is sorted below.
    if (tid == 0) s_nsel = 0;
    __syncthreads();
    for (int64_t i0 = static_cast<int64_t>(tid) * P; i0 < a.K; i0 += kStride) {
        float v[P];
        uint32_t key[P];
        const int n = load_vec<E>(ra, i0, a.K, v, key);
#pragma unroll
        for (int j = 0; j < P; ++j) {
            if (j < n && (key[j] > T || (take_all_eq && key[j] == T))) {
                const int slot = atomicAdd(&s_nsel, 1);
                sel_idx[slot] = static_cast<int32_t>(i0 + j);
                sel_val[slot] = v[j];
            }
        }
    }
    __syncthreads();
    if (!take_all_eq) {
        // Ties straddle the threshold: take the equal keys in index order,
        // one block sweep at a time, until need_eq are taken.
        int remaining = need_eq;
        for (int64_t base = 0; base < a.K && remaining > 0; base += kStride) {
            const int64_t i0 = base + static_cast<int64_t>(tid) * P;
            float v[P];
            uint32_t key[P];
            int n = 0, cnt = 0;
            if (i0 < a.K) {
                n = load_vec<E>(ra, i0, a.K, v, key);
#pragma unroll
                for (int j = 0; j < P; ++j) cnt += (j < n && key[j] == T) ? 1 : 0;
            }
            s_scan[tid] = cnt;
            __syncthreads();
            if (tid == 0) {
                int run = 0;
                for (int t = 0; t < kBlock; ++t) {
                    const int c = s_scan[t];
                    s_scan[t] = run;
                    run += c;
                }
            }
            __syncthreads();
            int rank = s_scan[tid];
            if (i0 < a.K) {
#pragma unroll
                for (int j = 0; j < P; ++j) {
                    if (j < n && key[j] == T) {
                        if (rank < remaining) {
                            const int slot = atomicAdd(&s_nsel, 1);
                            sel_idx[slot] = static_cast<int32_t>(i0 + j);
                            sel_val[slot] = v[j];
                        }
                        ++rank;
                    }
                }
            }
            __syncthreads();
            const int taken_total = s_nsel;
            remaining = k - taken_total;
            __syncthreads();
        }
    }

    // Rank sort by token index (indices are distinct), then the averaged
    // model's log-probabilities of the selected tokens.
    for (int t = tid; t < k; t += kBlock) {
        const int32_t my = sel_idx[t];
        int r = 0;
        for (int j = 0; j < k; ++j) r += sel_idx[j] < my ? 1 : 0;
        sorted_idx[r] = my;
        la[r] = static_cast<double>(sel_val[t]) - lse_a;
    }
    __syncthreads();
    if (a.topk_out)
        for (int t = tid; t < k; t += kBlock) a.topk_out[u * k + t] = sorted_idx[t];

    constexpr double kLog2 = 0.69314718055994530942;
    for (int w = 0; w < a.M; ++w) {
        const rsrc_t rw = js_row(a.workers, static_cast<int64_t>(w) * a.U + u, a.ldk, E::kElem);
        double mw = -INFINITY, sw = 0.0;
        for (int64_t i0 = static_cast<int64_t>(tid) * P; i0 < a.K; i0 += kStride) {
            float v[P];
            uint32_t key[P];
            const int n = load_vec<E>(rw, i0, a.K, v, key);
            lse_add<P>(mw, sw, v, n);
        }
        const double lse_w = block_lse(mw, sw, red);
        double part = 0.0;
        for (int t = tid; t < k; t += kBlock) {
            const double lp = static_cast<double>(E::at(rw, sorted_idx[t])) - lse_w;
            const double lq = la[t];
            const double hi = lp > lq ? lp : lq, lo = lp > lq ? lq : lp;
            if (hi == -INFINITY) continue;  // probability 0 on both sides
            const double lmix = hi + log1p(exp(lo - hi)) - kLog2;
            // A side of probability 0 adds nothing (0 log 0 = 0).
            if (lp != -INFINITY) part += 0.5 * exp(lp) * (lp - lmix);
            if (lq != -INFINITY) part += 0.5 * exp(lq) * (lq - lmix);
        }
        const double js = block_sum(part, red);
        if (tid == 0) a.d_out[static_cast<int64_t>(w) * a.U + u] = sqrt((js > 0.0 ? js : 0.0) / kLog2);
    }
}

// mean[m] = (1/U) sum_u d[m][u], one block per worker, fixed order.
__global__ __launch_bounds__(256) void js_mean_kernel(const double *d, int64_t U, double *mean) {
    __shared__ double s[256];
    const int m = blockIdx.x, t = threadIdx.x;
    double acc = 0.0;
    for (int64_t u = t; u < U; u += 256) acc += d[static_cast<int64_t>(m) * U + u];
    s[t] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) s[t] += s[t + w];
        __syncthreads();
    }
    if (t == 0) mean[m] = s[0] / static_cast<double>(U);
}

bool js_launch(const void *avg, const void *workers, int32_t bf16, int32_t M, int64_t U, int64_t K, int64_t ldk,
               int32_t k, double *d_out, double *mean_out, int32_t *topk_out, hipStream_t stream) {
    JsParams p{avg, workers, d_out, topk_out, U, K, ldk, M, k};
    if (bf16) hipLaunchKernelGGL(js_kernel<JsBF16>, dim3(static_cast<unsigned>(U)), dim3(kBlock), 0, stream, p);
    else hipLaunchKernelGGL(js_kernel<JsF32>, dim3(static_cast<unsigned>(U)), dim3(kBlock), 0, stream, p);
    if (hipGetLastError() != hipSuccess) return false;
    if (mean_out) {
        hipLaunchKernelGGL(js_mean_kernel, dim3(M), dim3(256), 0, stream, d_out, U, mean_out);
        if (hipGetLastError() != hipSuccess) return false;
    }
    return true;
}

}  // namespace fgd
