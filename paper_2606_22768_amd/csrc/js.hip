// js.hip -- Jensen--Shannon functional distance between each worker's
// predicted token distribution and the parameter-averaged model's
// (Sec. 4.4, JS distance; Appendix D.2, JS functional disagreement).
//
// For token u, in float64 and in the log domain:
//   lse_m      = log sum_i exp(z_m,i)               every worker row
//   lse_a      = log sum_i exp(zbar_i)              the averaged model's row
//   T          = the k largest zbar_i (ties: lower index first), selected on
//                order-preserving integer keys of the stored logits (exact
//                comparisons: no rounding decides it)
//   JS_m       = sum over i in T of the per-token terms
//                1/2 p (lp - lmix) + 1/2 q (lq - lmix), lp = z_m,i - lse_m,
//                lq = zbar_i - lse_a, lmix = log((p + q) / 2)
//   d_m(u)     = sqrt(max(JS_m, 0) / log 2)
// Probabilities are those of the full softmax; only the sum is restricted to
// T.  Kernels, in order on the call's stream, with a caller workspace between
// them:
//   js_rows_kernel         streams all (M + 1) U rows once (persistent, no
//                          barriers): per row, each wave's (shift, sum) part
//                          of the log-sum-exp; per averaged row, each row
//                          thread's four largest vector maxima (key, index)
//   js_token_wave_kernel   (k <= 512) one wave per token: the averaged row's
//                          lse from its parts, the selection (a threshold from
//                          the recorded maxima, a second read of only the
//                          vectors that reach it), the JS terms; a token with
//                          too many candidates is flagged
//   js_token_radix_kernel  per token, a radix select over the whole row: every
//                          token when k > 512, else only the flagged ones
//   js_mean_kernel         the per-worker mean of d
//
// Rows.  bf16 logits take only 65536 bit patterns, and the exp of every bf16
// value v with 2^-16 <= |v| < 64 (22 binades, both signs: 5632 values) is a
// table of 44 KB in LDS, filled once per block with the library's float64
// exp.  Such terms need no shift: each is below e^64, so their plain sum
// cannot overflow; a term costs an index from the bit pattern, one LDS read
// and one add.  A 16-byte vector of logits in which any lane of the wave
// holds another value (0, |v| < 2^-16, |v| >= 64, -inf, or the ragged end of
// the row) goes through the general path below, whose shifted sum is merged
// with the table sum at the end of the row.  float32 logits always take the
// general path.  The averaged rows and the worker rows run the same sums in
// the same lane order, so a worker whose logits equal the averaged model's
// gets exactly d = 0.
//
// General path.  The log-sum-exp of a row is a (shift, scaled sum)
// reduction: the shift is a lane's first finite value and moves only when a
// later value exceeds it by more than kLseSlack, so every exponent is at
// most kLseSlack and the sums cannot overflow.  exp is a table-driven
// float64 exp (Tang's method: ACM TOMS 15(2), 1989): x = (256 n + j) ln2/256
// + r with |r| <= ln2/512, exp(x) = 2^n 2^(j/256) (1 + q(r)), q the degree-4
// Taylor polynomial of e^r - 1 (truncation below 0.4 ulp), 2^(j/256) from a
// table in LDS; within 2 ulp of the correctly rounded value.  The factor 2^n
// is applied by an integer add to the table entry's exponent field (the
// entry is stored with j << 12 already subtracted from its high word, so
// adding n << 12 leaves the mantissa alone and adds n >> 8 to the
// exponent); x is clamped at -708 so that the scaled entry stays a normal
// double.  Lanes, then a row's waves, are combined through the largest
// shift (one exp per part, no pairwise rescaling).  Every reduction has a
// fixed order, so results are deterministic.  The selected indices are
// rank-sorted so that the JS sum runs in index order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "js.hpp"
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
    static constexpr bool kBf16 = false;
    __device__ static void unpack(u32x4 t, float (&v)[kPer], uint32_t (&key)[kPer]) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t b = t[j];
            if ((b & 0x7FFFFFFFu) == 0) b = 0;
            v[j] = __uint_as_float(b);
            key[j] = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
        }
    }
    __device__ static void values(u32x4 t, float (&v)[kPer]) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = __uint_as_float(t[j]);
    }
    // Element i of the row that starts at `row` (a gather; nontemporal: the
    // line is not kept).
    __device__ static float at_ptr(const char *row, int64_t i) {
        return __builtin_nontemporal_load(reinterpret_cast<const float *>(row) + i);
    }
    // The key of a value, and the value of a key that some value has.
    __device__ static uint32_t key_of(float v) {
        uint32_t b = __float_as_uint(v);
        if ((b & 0x7FFFFFFFu) == 0) b = 0;
        return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
    }
    __device__ static float value_of(uint32_t key) {
        return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
    }
};

struct JsBF16 {
    static constexpr int kPer = 8, kElem = 2, kKeyBits = 16;
    static constexpr bool kBf16 = true;
    __device__ static void unpack(u32x4 t, float (&v)[kPer], uint32_t (&key)[kPer]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t h = (t[j / 2] >> (16 * (j % 2))) & 0xFFFFu;
            if ((h & 0x7FFFu) == 0) h = 0;
            v[j] = __uint_as_float(h << 16);
            key[j] = (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
        }
    }
    __device__ static void values(u32x4 t, float (&v)[kPer]) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = __uint_as_float(t[j] << 16);
            v[2 * j + 1] = __uint_as_float(t[j] & 0xFFFF0000u);
        }
    }
    // Element i of the row that starts at `row` (a gather; nontemporal: the
    // line is not kept).
    __device__ static float at_ptr(const char *row, int64_t i) {
        const uint16_t h = __builtin_nontemporal_load(reinterpret_cast<const uint16_t *>(row) + i);
        return __uint_as_float(static_cast<uint32_t>(h) << 16);
    }
    // The key of a value (a bf16 widened to float), and the value of a key
    // that some value has.
    __device__ static uint32_t key_of(float v) {
        uint32_t h = __float_as_uint(v) >> 16;
        if ((h & 0x7FFFu) == 0) h = 0;
        return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u);
    }
    __device__ static float value_of(uint32_t key) {
        return __uint_as_float(((key & 0x8000u) ? (key & 0x7FFFu) : (~key & 0xFFFFu)) << 16);
    }
};

__device__ inline rsrc_t js_row(const void *base, int64_t row, int64_t ldk, int es) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(base)) + row * ldk * es,
                                             static_cast<short>(0), 0x7fffffff, kRawBufferFlags);
}

__device__ inline double shfl_xor_d(double x, int mask) {
    const int64_t b = __double_as_longlong(x);
    const int lo = __shfl_xor(static_cast<int>(b & 0xFFFFFFFF), mask);
    const int hi = __shfl_xor(static_cast<int>(b >> 32), mask);
    return __longlong_as_double((static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo));
}

// ------------------------------------------------------------ float64 exp
// 2^(j/256) for j = 0..255, each the double nearest to the exact value.
constexpr int kTabBits = 8;
constexpr int kTab = 1 << kTabBits;
static_assert(kTab <= kBlock, "one thread per table entry loads the LDS copy");
__constant__ double kExp2Frac[kTab] = {
    0x1.0000000000000p+0, 0x1.00b1afa5abcbfp+0, 0x1.0163da9fb3335p+0, 0x1.02168143b0281p+0,
    0x1.02c9a3e778061p+0, 0x1.037d42e11bbccp+0, 0x1.04315e86e7f85p+0, 0x1.04e5f72f654b1p+0,
    0x1.059b0d3158574p+0, 0x1.0650a0e3c1f89p+0, 0x1.0706b29ddf6dep+0, 0x1.07bd42b72a836p+0,
    0x1.0874518759bc8p+0, 0x1.092bdf66607e0p+0, 0x1.09e3ecac6f383p+0, 0x1.0a9c79b1f3919p+0,
    0x1.0b5586cf9890fp+0, 0x1.0c0f145e46c85p+0, 0x1.0cc922b7247f7p+0, 0x1.0d83b23395decp+0,
    0x1.0e3ec32d3d1a2p+0, 0x1.0efa55fdfa9c5p+0, 0x1.0fb66affed31bp+0, 0x1.1073028d7233ep+0,
    0x1.11301d0125b51p+0, 0x1.11edbab5e2ab6p+0, 0x1.12abdc06c31ccp+0, 0x1.136a814f204abp+0,
    0x1.1429aaea92de0p+0, 0x1.14e95934f312ep+0, 0x1.15a98c8a58e51p+0, 0x1.166a45471c3c2p+0,
    0x1.172b83c7d517bp+0, 0x1.17ed48695bbc0p+0, 0x1.18af9388c8deap+0, 0x1.1972658375d2fp+0,
    0x1.1a35beb6fcb75p+0, 0x1.1af99f8138a1cp+0, 0x1.1bbe084045cd4p+0, 0x1.1c82f95281c6bp+0,
    0x1.1d4873168b9aap+0, 0x1.1e0e75eb44027p+0, 0x1.1ed5022fcd91dp+0, 0x1.1f9c18438ce4dp+0,
    0x1.2063b88628cd6p+0, 0x1.212be3578a819p+0, 0x1.21f49917ddc96p+0, 0x1.22bdda27912d1p+0,
    0x1.2387a6e756238p+0, 0x1.2451ffb82140ap+0, 0x1.251ce4fb2a63fp+0, 0x1.25e85711ece75p+0,
    0x1.26b4565e27cddp+0, 0x1.2780e341ddf29p+0, 0x1.284dfe1f56381p+0, 0x1.291ba7591bb70p+0,
    0x1.29e9df51fdee1p+0, 0x1.2ab8a66d10f13p+0, 0x1.2b87fd0dad990p+0, 0x1.2c57e39771b2fp+0,
    0x1.2d285a6e4030bp+0, 0x1.2df961f641589p+0, 0x1.2ecafa93e2f56p+0, 0x1.2f9d24abd886bp+0,
    0x1.306fe0a31b715p+0, 0x1.31432edeeb2fdp+0, 0x1.32170fc4cd831p+0, 0x1.32eb83ba8ea32p+0,
    0x1.33c08b26416ffp+0, 0x1.3496266e3fa2dp+0, 0x1.356c55f929ff1p+0, 0x1.36431a2de883bp+0,
    0x1.371a7373aa9cbp+0, 0x1.37f26231e754ap+0, 0x1.38cae6d05d866p+0, 0x1.39a401b7140efp+0,
    0x1.3a7db34e59ff7p+0, 0x1.3b57fbfec6cf4p+0, 0x1.3c32dc313a8e5p+0, 0x1.3d0e544ede173p+0,
    0x1.3dea64c123422p+0, 0x1.3ec70df1c5175p+0, 0x1.3fa4504ac801cp+0, 0x1.40822c367a024p+0,
    0x1.4160a21f72e2ap+0, 0x1.423fb2709468ap+0, 0x1.431f5d950a897p+0, 0x1.43ffa3f84b9d4p+0,
    0x1.44e086061892dp+0, 0x1.45c2042a7d232p+0, 0x1.46a41ed1d0057p+0, 0x1.4786d668b3237p+0,
    0x1.486a2b5c13cd0p+0, 0x1.494e1e192aed2p+0, 0x1.4a32af0d7d3dep+0, 0x1.4b17dea6db7d7p+0,
    0x1.4bfdad5362a27p+0, 0x1.4ce41b817c114p+0, 0x1.4dcb299fddd0dp+0, 0x1.4eb2d81d8abffp+0,
    0x1.4f9b2769d2ca7p+0, 0x1.508417f4531eep+0, 0x1.516daa2cf6642p+0, 0x1.5257de83f4eefp+0,
    0x1.5342b569d4f82p+0, 0x1.542e2f4f6ad27p+0, 0x1.551a4ca5d920fp+0, 0x1.56070dde910d2p+0,
    0x1.56f4736b527dap+0, 0x1.57e27dbe2c4cfp+0, 0x1.58d12d497c7fdp+0, 0x1.59c0827ff07ccp+0,
    0x1.5ab07dd485429p+0, 0x1.5ba11fba87a03p+0, 0x1.5c9268a5946b7p+0, 0x1.5d84590998b93p+0,
    0x1.5e76f15ad2148p+0, 0x1.5f6a320dceb71p+0, 0x1.605e1b976dc09p+0, 0x1.6152ae6cdf6f4p+0,
    0x1.6247eb03a5585p+0, 0x1.633dd1d1929fdp+0, 0x1.6434634ccc320p+0, 0x1.652b9febc8fb7p+0,
    0x1.6623882552225p+0, 0x1.671c1c70833f6p+0, 0x1.68155d44ca973p+0, 0x1.690f4b19e9538p+0,
    0x1.6a09e667f3bcdp+0, 0x1.6b052fa75173ep+0, 0x1.6c012750bdabfp+0, 0x1.6cfdcddd47645p+0,
    0x1.6dfb23c651a2fp+0, 0x1.6ef9298593ae5p+0, 0x1.6ff7df9519484p+0, 0x1.70f7466f42e87p+0,
    0x1.71f75e8ec5f74p+0, 0x1.72f8286ead08ap+0, 0x1.73f9a48a58174p+0, 0x1.74fbd35d7cbfdp+0,
    0x1.75feb564267c9p+0, 0x1.77024b1ab6e09p+0, 0x1.780694fde5d3fp+0, 0x1.790b938ac1cf6p+0,
    0x1.7a11473eb0187p+0, 0x1.7b17b0976cfdbp+0, 0x1.7c1ed0130c132p+0, 0x1.7d26a62ff86f0p+0,
    0x1.7e2f336cf4e62p+0, 0x1.7f3878491c491p+0, 0x1.80427543e1a12p+0, 0x1.814d2add106d9p+0,
    0x1.82589994cce13p+0, 0x1.8364c1eb941f7p+0, 0x1.8471a4623c7adp+0, 0x1.857f4179f5b21p+0,
    0x1.868d99b4492edp+0, 0x1.879cad931a436p+0, 0x1.88ac7d98a6699p+0, 0x1.89bd0a478580fp+0,
    0x1.8ace5422aa0dbp+0, 0x1.8be05bad61778p+0, 0x1.8cf3216b5448cp+0, 0x1.8e06a5e0866d9p+0,
    0x1.8f1ae99157736p+0, 0x1.902fed0282c8ap+0, 0x1.9145b0b91ffc6p+0, 0x1.925c353aa2fe2p+0,
    0x1.93737b0cdc5e5p+0, 0x1.948b82b5f98e5p+0, 0x1.95a44cbc8520fp+0, 0x1.96bdd9a7670b3p+0,
    0x1.97d829fde4e50p+0, 0x1.98f33e47a22a2p+0, 0x1.9a0f170ca07bap+0, 0x1.9b2bb4d53fe0dp+0,
    0x1.9c49182a3f090p+0, 0x1.9d674194bb8d5p+0, 0x1.9e86319e32323p+0, 0x1.9fa5e8d07f29ep+0,
    0x1.a0c667b5de565p+0, 0x1.a1e7aed8eb8bbp+0, 0x1.a309bec4a2d33p+0, 0x1.a42c980460ad8p+0,
    0x1.a5503b23e255dp+0, 0x1.a674a8af46052p+0, 0x1.a799e1330b358p+0, 0x1.a8bfe53c12e59p+0,
    0x1.a9e6b5579fdbfp+0, 0x1.ab0e521356ebap+0, 0x1.ac36bbfd3f37ap+0, 0x1.ad5ff3a3c2774p+0,
    0x1.ae89f995ad3adp+0, 0x1.afb4ce622f2ffp+0, 0x1.b0e07298db666p+0, 0x1.b20ce6c9a8952p+0,
    0x1.b33a2b84f15fbp+0, 0x1.b468415b749b1p+0, 0x1.b59728de5593ap+0, 0x1.b6c6e29f1c52ap+0,
    0x1.b7f76f2fb5e47p+0, 0x1.b928cf22749e4p+0, 0x1.ba5b030a1064ap+0, 0x1.bb8e0b79a6f1fp+0,
    0x1.bcc1e904bc1d2p+0, 0x1.bdf69c3f3a207p+0, 0x1.bf2c25bd71e09p+0, 0x1.c06286141b33dp+0,
    0x1.c199bdd85529cp+0, 0x1.c2d1cd9fa652cp+0, 0x1.c40ab5fffd07ap+0, 0x1.c544778fafb22p+0,
    0x1.c67f12e57d14bp+0, 0x1.c7ba88988c933p+0, 0x1.c8f6d9406e7b5p+0, 0x1.ca3405751c4dbp+0,
    0x1.cb720dcef9069p+0, 0x1.ccb0f2e6d1675p+0, 0x1.cdf0b555dc3fap+0, 0x1.cf3155b5bab74p+0,
    0x1.d072d4a07897cp+0, 0x1.d1b532b08c968p+0, 0x1.d2f87080d89f2p+0, 0x1.d43c8eacaa1d6p+0,
    0x1.d5818dcfba487p+0, 0x1.d6c76e862e6d3p+0, 0x1.d80e316c98398p+0, 0x1.d955d71ff6075p+0,
    0x1.da9e603db3285p+0, 0x1.dbe7cd63a8315p+0, 0x1.dd321f301b460p+0, 0x1.de7d5641c0658p+0,
    0x1.dfc97337b9b5fp+0, 0x1.e11676b197d17p+0, 0x1.e264614f5a129p+0, 0x1.e3b333b16ee12p+0,
    0x1.e502ee78b3ff6p+0, 0x1.e653924676d76p+0, 0x1.e7a51fbc74c83p+0, 0x1.e8f7977cdb740p+0,
    0x1.ea4afa2a490dap+0, 0x1.eb9f4867cca6ep+0, 0x1.ecf482d8e67f1p+0, 0x1.ee4aaa2188510p+0,
    0x1.efa1bee615a27p+0, 0x1.f0f9c1cb6412ap+0, 0x1.f252b376bba97p+0, 0x1.f3ac948dd7274p+0,
    0x1.f50765b6e4540p+0, 0x1.f6632798844f8p+0, 0x1.f7bfdad9cbe14p+0, 0x1.f91d802243c89p+0,
    0x1.fa7c1819e90d8p+0, 0x1.fbdba3692d514p+0, 0x1.fd3c22b8f71f1p+0, 0x1.fe9d96b2a23d9p+0,
};

// The polynomial steps are written as three-address v_fma_f64 with the
// wave-uniform constant in scalar registers: the compiler's two-address
// v_fmac form would copy a constant register before every use.
__device__ __forceinline__ double fma_vvs(double a, double b, double c) {  // a * b + c, c uniform
    double d;
    asm("v_fma_f64 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "s"(c));
    return d;
}
__device__ __forceinline__ double fma_vsv(double a, double b, double c) {  // a * b + c, b uniform
    double d;
    asm("v_fma_f64 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
    return d;
}
__device__ __forceinline__ double fnma_vsv(double a, double b, double c) {  // c - a * b, b uniform
    double d;
    asm("v_fma_f64 %0, -%1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
    return d;
}

constexpr double kExpRound = 0x1.8p52;                   // adding it rounds to an integer, kept in the low word
constexpr double kExpInvL = 0x1.71547652b82fep+8;        // 256 / ln 2
constexpr double kExpL1 = 0x1.62e42fee00000p-9;          // ln2 / 256, high part (n * kExpL1 is exact)
constexpr double kExpL2 = 0x1.a39ef35793c76p-41;         // ln2 / 256 - kExpL1
constexpr double kExpFloor = -708.0;                     // 2^(n >> 8) 2^(j/256) stays normal above it

// The LDS copy of kExp2Frac with j << 12 subtracted from entry j's high
// word (see exp_table).  Block-wide; ends with a barrier.
__device__ inline void load_exp_table(double *tab) {
    const int tid = threadIdx.x;
    if (tid < kTab) {
        const double t = kExp2Frac[tid];
        tab[tid] = __hiloint2double(__double2hiint(t) - (tid << 12), __double2loint(t));
    }
    __syncthreads();
}

// exp(x) for x <= 700; x below -708 (and -inf) gives exp(-708) ~ 3.3e-308,
// which no sum it joins can notice (every sum it is added to holds a term
// of at least 1, or is discarded; see lse_add and the row kernels).  `tab`
// comes from load_exp_table.
__device__ __forceinline__ double exp_table(double x, const double *tab) {
    x = fmax(x, kExpFloor);
    const double y = fma_vsv(x, kExpInvL, kExpRound);
    const int n = __double2loint(y);                     // round(x * 256 / ln2)
    const double nd = y - kExpRound;
    const double r = fnma_vsv(nd, kExpL2, fnma_vsv(nd, kExpL1, x));
    double p = fma_vsv(r, 1.0 / 24.0, 1.0 / 6.0);
    p = fma_vvs(p, r, 0.5);
    p = fma_vvs(p, r, 1.0);
    const double q = p * r;                              // e^r - 1
    const double tb = tab[n & (kTab - 1)];
    // 2^(j/256) * 2^(n >> 8): the entry's high word already lacks j << 12.
    const double t = __hiloint2double(__double2hiint(tb) + (n << 12), __double2loint(tb));
    return fma(t, q, t);
}

// ------------------------------------------------------------ log-sum-exp
constexpr double kLseSlack = 64.0;     // largest exponent a sum may take
constexpr double kLseEmpty = -1e300;   // shift of a lane that has seen no finite value

// Values of one loaded 16-byte vector of a row that starts at element i0;
// those at or past K read as -inf, which the log-sum-exp ignores exactly.
template <class E>
__device__ inline void vec_values(u32x4 t, int64_t i0, int64_t K, float (&v)[E::kPer]) {
    E::values(t, v);
    if (i0 + E::kPer > K) {
#pragma unroll
        for (int j = 0; j < E::kPer; ++j)
            if (i0 + j >= K) v[j] = -INFINITY;
    }
}

// Values and keys of one vector and how many lie below K (values past K read
// as -inf; key users test the count).
template <class E>
__device__ inline int load_vec(rsrc_t r, int64_t i0, int64_t K, float (&v)[E::kPer], uint32_t (&key)[E::kPer]) {
    const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<uint32_t>(i0 * E::kElem), 0, kLoadPolicy);
    E::unpack(t, v, key);
    const int64_t left = K - i0;
    const int n = left >= E::kPer ? E::kPer : static_cast<int>(left);
    if (n < E::kPer) {
#pragma unroll
        for (int j = 0; j < E::kPer; ++j)
            if (j >= n) v[j] = -INFINITY;
    }
    return n;
}

// Largest of four or eight values (three-operand maxima; logits are never
// NaN).
__device__ __forceinline__ float max3f(float a, float b, float c) {
    float d;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
    return d;
}
template <int N>
__device__ __forceinline__ float vec_max(const float (&v)[N]) {
    static_assert(N == 4 || N == 8, "a 16-byte vector holds 4 or 8 logits");
    if constexpr (N == 8) return max3f(max3f(max3f(v[0], v[1], v[2]), v[3], v[4]), max3f(v[5], v[6], v[7]), v[0]);
    return max3f(max3f(v[0], v[1], v[2]), v[3], v[0]);
}

// Adds one vector to a lane's (shift m, sum s = sum exp(x - m)); thr is
// m + kLseSlack rounded to float (-inf while the lane is empty), the value
// above which the shift moves.  The terms are summed pairwise before they
// join the running sum.  Once a lane has seen a finite value, s holds a
// term of at least 1 (the one at the shift), so clamped terms (exp_table)
// vanish in it; the terms a still-empty lane gathers are scaled to 0 when
// its shift first moves, or dropped by lane_state.
template <int N>
__device__ inline void lse_add(double &m, float &thr, double &s, const float (&v)[N], const double *tab) {
    const float vm = vec_max<N>(v);
    if (vm > thr) {
        const double dm = vm;
        s *= exp_table(m - dm, tab);
        m = dm;
        thr = static_cast<float>(dm + kLseSlack);
    }
    double e[N];
#pragma unroll
    for (int j = 0; j < N; ++j) e[j] = exp_table(static_cast<double>(v[j]) - m, tab);
#pragma unroll
    for (int w = 1; w < N; w *= 2)
#pragma unroll
        for (int j = 0; j + w < N; j += 2 * w) e[j] += e[j + w];
    s += e[0];
}

// A lane's (shift, sum) at the end of a row: an empty lane reports no terms.
__device__ inline void lane_state(double &m, double &s) {
    if (m == kLseEmpty) s = 0.0;
}

// ------------------------------------------------ bf16 rows: exp table
constexpr int kBfTabE0 = 111;                              // exponent field of 2^-16
constexpr int kBfTabE1 = 132;                              // exponent field of [32, 64)
constexpr uint32_t kBfTabLo = kBfTabE0 << 7;               // first magnitude pattern in the table
constexpr uint32_t kBfTabN = (kBfTabE1 - kBfTabE0 + 1) << 7;  // magnitudes per sign (2816)
constexpr int kBfTabEntries = 2 * kBfTabN;

// Entry 2 (a - kBfTabLo) + s = exp of the bf16 value with magnitude
// pattern a and sign s, from the library's float64 exp.  Block-wide, no
// barrier of its own.
__device__ inline void fill_bf16_exp_table(double *etab) {
    for (int i = threadIdx.x; i < kBfTabEntries; i += blockDim.x) {
        const uint32_t h = (kBfTabLo + static_cast<uint32_t>(i >> 1)) | (static_cast<uint32_t>(i & 1) << 15);
        etab[i] = exp(static_cast<double>(__uint_as_float(h << 16)));
    }
}

// A lane's partial log-sum-exp of a row: table terms summed unshifted (s0)
// and general-path terms shifted by m (s1, thr as in lse_add).
struct RowLse {
    double s0 = 0.0, m = kLseEmpty, s1 = 0.0;
    float thr = -INFINITY;
};

// Adds the 16-byte vector `t` of bf16 logits (elements i0 .. i0 + 7 of a
// row of K).  When every active lane of the wave holds eight values inside
// the table, their terms are read from it; otherwise the vector takes the
// general path, one term at a time (which keeps the kernels' registers
// within their occupancy).  The choice depends only on the data and the
// lane-to-element map, so two rows with equal logits summed under the same
// map give bit-identical results.
__device__ inline void bf16_lse_add(RowLse &st, u32x4 t, int64_t i0, int64_t K, const double *etab,
                                    const double *tab) {
    constexpr int P = JsBF16::kPer;
    uint32_t idx[P];
    bool in_table = i0 + P <= K;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t w = t[j];
        const uint32_t d0 = (w & 0x7FFFu) - kBfTabLo, d1 = ((w >> 16) & 0x7FFFu) - kBfTabLo;
        in_table = in_table && d0 < kBfTabN && d1 < kBfTabN;
        idx[2 * j] = (d0 << 1) | ((w >> 15) & 1u);
        idx[2 * j + 1] = (d1 << 1) | (w >> 31);
    }
    if (__all(in_table)) {
        double e[P];
#pragma unroll
        for (int j = 0; j < P; ++j) e[j] = etab[idx[j]];
#pragma unroll
        for (int w = 1; w < P; w *= 2)
#pragma unroll
            for (int j = 0; j + w < P; j += 2 * w) e[j] += e[j + w];
        st.s0 += e[0];
    } else {
        float v[P];
        vec_values<JsBF16>(t, i0, K, v);
        const float vm = vec_max<P>(v);
        if (vm > st.thr) {
            const double dm = vm;
            st.s1 *= exp_table(st.m - dm, tab);
            st.m = dm;
            st.thr = static_cast<float>(dm + kLseSlack);
        }
#pragma unroll 1
        for (int j = 0; j < P; ++j) st.s1 += exp_table(static_cast<double>(v[j]) - st.m, tab);
    }
}

// The lane's (shift, sum) at the end of a row: the table sum has shift 0,
// the general one shift m; an empty lane reports no terms.
__device__ inline void row_lse_lane(RowLse st, double &ml, double &sl, const double *tab) {
    lane_state(st.m, st.s1);
    if (st.s1 == 0.0) {
        ml = st.s0 == 0.0 ? kLseEmpty : 0.0;
        sl = st.s0;
    } else if (st.s0 == 0.0) {
        ml = st.m;
        sl = st.s1;
    } else {
        ml = st.m > 0.0 ? st.m : 0.0;
        sl = st.s0 * exp_table(-ml, tab) + st.s1 * exp_table(st.m - ml, tab);
    }
}

// One token's term of the JS sum, 1/2 p log(p / mix) + 1/2 q log(q / mix),
// from the two log-probabilities.  With hi >= lo the larger and smaller of
// them and r = exp(lo - hi): log mix = hi + log1p(r) - log 2, so the term is
// 1/2 exp(hi) [(log 2 - log1p(r)) + r ((lo - hi) + log 2 - log1p(r))].  A
// side of probability 0 adds nothing (0 log 0 = 0), and equal sides add
// exactly 0 (p = q = mix).
__device__ inline double js_term(double lp, double lq) {
    constexpr double kLog2 = 0.69314718055994530942;
    const double hi = lp > lq ? lp : lq, lo = lp > lq ? lq : lp;
    if (hi == -INFINITY || lo == hi) return 0.0;
    const double r = exp(lo - hi);  // 0 when lo = -inf
    const double c = kLog2 - log1p(r);
    double t = c;
    if (r != 0.0) t += r * ((lo - hi) + c);
    return 0.5 * exp(hi) * t;
}

constexpr int kJsGroup = 8;  // workers whose logits are gathered together

// ------------------------------------------------------------ workspace
// From the row kernel to the per-token kernels: per row, the (shift, sum)
// of each of its kRowWaves waves; per token and row thread, the averaged
// row's kTopVecs largest vector maxima; a flag per token.
constexpr int kRowThreads = kBlock;                     // threads per row (the radix kernel's block)
constexpr int kRowWaves = kRowThreads / kWave;          // wave partials per row
constexpr int kRowsPerBlock = 2;                        // rows a js_rows_kernel block streams at once
constexpr int kRowsBlock = kRowThreads * kRowsPerBlock;
constexpr int kRowsBlocksPerCu = 3;                     // bf16 LDS: 3 x 46 KB of the CU's 160 KB
constexpr int kTopVecs = 4;                             // vector maxima a row thread of an averaged row keeps
constexpr int64_t kTopIndexLimit = 1 << 16;             // vectors per row thread their 16-bit indices can name

// A wave's part of a row's log-sum-exp: sum exp(z - m) over its lanes'
// elements (s = 0: none).
struct LsePart {
    double m, s;
};

struct JsWork {
    LsePart *part;   // [(M + 1) U][kRowWaves]: row u < U is token u's averaged row, U + m U + u worker m's
    u32x4 *top;      // [U][kRowThreads]: top entries, largest first (0: none; see TopVecs)
    int32_t *flag;   // [U]: 1 where the per-token wave kernel left the token to the radix kernel
};

// The kTopVecs largest vector maxima of a row thread, each entry the
// 16-bit key of the vector's largest element (the key itself for bf16, its
// top 16 bits for float32) above the vector's index among the thread's
// vectors: key16 << 16 | index, so entries order by key, then index.
template <class E>
struct TopVecs {
    uint32_t t[kTopVecs] = {0, 0, 0, 0};  // largest first; 0: no vector
    __device__ static uint32_t key16(uint32_t key) { return E::kBf16 ? key : key >> 16; }
    // Takes entry e in (entries are distinct): each slot keeps the median of
    // itself, the slot above and e, from the bottom up.
    __device__ void insert(uint32_t e) {
#pragma unroll
        for (int i = kTopVecs - 1; i > 0; --i) t[i] = med3(t[i], t[i - 1], e);
        t[0] = max(t[0], e);
    }
    __device__ static uint32_t med3(uint32_t a, uint32_t b, uint32_t c) { return max(min(a, b), min(max(a, b), c)); }
};

// The row streamed at position q of the row kernels' order: token-major,
// token u's averaged row (row u of the workspace parts) then its M worker
// rows (row U + m U + u), so every pass of the persistent grid holds the
// same share of averaged rows, whose terms cost more.
__device__ inline int64_t js_stream_row(int64_t q, int32_t M, int64_t U) {
    const int64_t u = q / (M + 1), j = q - u * (M + 1);
    return j == 0 ? u : U + (j - 1) * U + u;
}

// Vectors per row thread, at most (a row of K logits, P per vector).
inline int64_t js_thread_vectors(int64_t K, int per) {
    return ((K + per - 1) / per + kRowThreads - 1) / kRowThreads;
}

// A wave's (shift, sum) from its lanes' (m, s): the largest shift, then
// sum s exp(m - shift) in a fixed order; lane 0's copy is the one used.
__device__ inline LsePart wave_lse(double m, double s, const double *tab) {
    double M = m;
    for (int o = kWave / 2; o > 0; o >>= 1) M = fmax(M, shfl_xor_d(M, o));
    double t = s == 0.0 ? 0.0 : s * exp_table(m - M, tab);
    for (int o = kWave / 2; o > 0; o >>= 1) t += shfl_xor_d(t, o);
    return LsePart{M, t};
}

// A row's log-sum-exp from its wave parts, in wave order (-inf for a row of
// -inf logits).
__device__ inline double lse_of_parts(const LsePart (&q)[kRowWaves], const double *tab) {
    double M = q[0].m;
#pragma unroll
    for (int j = 1; j < kRowWaves; ++j) M = fmax(M, q[j].m);
    double S = 0.0;
#pragma unroll
    for (int j = 0; j < kRowWaves; ++j)
        if (q[j].s != 0.0) S += q[j].s * exp_table(q[j].m - M, tab);
    return S == 0.0 ? -INFINITY : M + log(S);
}
__device__ inline double row_lse(const LsePart *p, const double *tab) {
    LsePart q[kRowWaves];
#pragma unroll
    for (int j = 0; j < kRowWaves; ++j) q[j] = p[j];
    return lse_of_parts(q, tab);
}

// Packed 16-bit lanes: two bf16 logits of a 32-bit word at once.  The word
// is copied with memcpy: with this toolchain, __builtin_bit_cast of an
// element t[j] of a u32x4 compiled to a read of t[0] for every j.
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u16x2 as_u16x2(uint32_t x) {
    u16x2 r;
    __builtin_memcpy(&r, &x, sizeof(r));
    return r;
}

// bf16_lse_add for a whole vector inside the row (elements i0 .. i0 + 7 all
// below K): the table indices 2 (magnitude - kBfTabLo) + sign of both
// halves of a word at once.  Same terms, order and path choice.
__device__ inline void bf16_lse_add_whole(RowLse &st, u32x4 t, const double *etab, const double *tab) {
    constexpr int P = JsBF16::kPer;
    u16x2 d[4];
    u16x2 mx = {0, 0};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const u16x2 h = as_u16x2(t[j]);
        d[j] = ((h << 1) | (h >> 15)) - static_cast<u16x2>(static_cast<uint16_t>(2 * kBfTabLo));
        mx = __builtin_elementwise_max(mx, d[j]);
    }
    const uint32_t m = mx.x > mx.y ? mx.x : mx.y;
    if (__all(m < static_cast<uint32_t>(kBfTabEntries))) {
        double e[P];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            e[2 * j] = etab[d[j].x];
            e[2 * j + 1] = etab[d[j].y];
        }
#pragma unroll
        for (int w = 1; w < P; w *= 2)
#pragma unroll
            for (int j = 0; j + w < P; j += 2 * w) e[j] += e[j + w];
        st.s0 += e[0];
    } else {
        float v[P];
        JsBF16::values(t, v);
        const float vm = vec_max<P>(v);
        if (vm > st.thr) {
            const double dm = vm;
            st.s1 *= exp_table(st.m - dm, tab);
            st.m = dm;
            st.thr = static_cast<float>(dm + kLseSlack);
        }
#pragma unroll 1
        for (int j = 0; j < P; ++j) st.s1 += exp_table(static_cast<double>(v[j]) - st.m, tab);
    }
}

// One vector's terms: whole (every element below K) or the row's last,
// which may be partial.  With kAvg it also updates the thread's largest
// vector maxima (v: the vector's sweep).
template <class E, bool kAvg, bool kWhole>
__device__ __forceinline__ void vec_terms(u32x4 cur, int64_t i0, int64_t K, uint32_t v, RowLse &st,
                                          const double *etab, const double *tab, TopVecs<E> &top) {
    constexpr int P = E::kPer;
    if constexpr (kAvg || !E::kBf16) {
        float x[P];
        if constexpr (kWhole)
            E::values(cur, x);
        else
            vec_values<E>(cur, i0, K, x);  // past K: -inf
        if constexpr (kAvg) top.insert((TopVecs<E>::key16(E::key_of(vec_max<P>(x))) << 16) | (v & 0xFFFFu));
        if constexpr (!E::kBf16) lse_add<P>(st.m, st.thr, st.s1, x, tab);
    }
    if constexpr (E::kBf16) {
        if constexpr (kWhole)
            bf16_lse_add_whole(st, cur, etab, tab);
        else
            bf16_lse_add(st, cur, i0, K, etab, tab);
    }
}

// One row's log-sum-exp terms for the thread's elements i_first + s kStride
// (sweeps s = 0 .. nsw - 1) into st.  `nxt` holds the row's first vector on
// entry and, when has_next, the first vector of row rn on return, so that
// the next row's load overlaps this row's end.  Sweeps before the last are
// whole for every lane: their loads take the sweep's offset as a scalar.
// With kAvg it also keeps the thread's kTopVecs largest vector maxima (top,
// empty on entry; indices past 16 bits wrap, and the per-token wave kernel
// is then not used).
template <class E, bool kAvg>
__device__ inline void row_terms(rsrc_t r, rsrc_t rn, bool has_next, int64_t i_first, int64_t K, int nsw,
                                 u32x4 &nxt, RowLse &st, const double *etab, const double *tab, TopVecs<E> &top) {
    constexpr int64_t kStride = static_cast<int64_t>(kRowThreads) * E::kPer;
    constexpr uint32_t kSweepBytes = kRowThreads * 16;
    const uint32_t voff = static_cast<uint32_t>(i_first * E::kElem);
    const int64_t i_last = i_first + static_cast<int64_t>(nsw - 1) * kStride;  // the last sweep's element
    int s = 0;
    for (; s < nsw - 2; ++s) {
        const u32x4 cur = nxt;
        nxt = __builtin_amdgcn_raw_buffer_load_b128(r, voff, (s + 1) * kSweepBytes, kLoadPolicy);
        vec_terms<E, kAvg, true>(cur, 0, K, static_cast<uint32_t>(s), st, etab, tab, top);
    }
    if (nsw >= 2) {  // s = nsw - 2: the next load is the last sweep's, which a lane may lack
        const u32x4 cur = nxt;
        if (i_last < K) nxt = __builtin_amdgcn_raw_buffer_load_b128(r, voff, (nsw - 1) * kSweepBytes, kLoadPolicy);
        vec_terms<E, kAvg, true>(cur, 0, K, static_cast<uint32_t>(nsw - 2), st, etab, tab, top);
    }
    const u32x4 cur = nxt;
    if (has_next && i_first < K) nxt = __builtin_amdgcn_raw_buffer_load_b128(rn, voff, 0, kLoadPolicy);
    if (i_last < K) vec_terms<E, kAvg, false>(cur, i_last, K, static_cast<uint32_t>(nsw - 1), st, etab, tab, top);
}

// Every row's wave parts of its log-sum-exp, and the averaged rows'
// largest vector maxima per thread, into the workspace.  Persistent: thread group g
// (kRowThreads threads; two per block) streams the rows at positions g,
// g + G, ... (G groups) of js_stream_row's order; thread lt of a group takes the
// elements lt * P + s * kStride of its row.  No barriers after the tables
// are loaded: each wave streams on its own, its next row's first load
// issued before its row ends.
template <class E>
__global__ __launch_bounds__(kRowsBlock) __attribute__((amdgpu_waves_per_eu(6, 8)))
void js_rows_kernel(JsParams a, JsWork w) {
    constexpr int64_t kStride = static_cast<int64_t>(kRowThreads) * E::kPer;
    __shared__ double etab[E::kBf16 ? kBfTabEntries : 1];
    __shared__ double tab[kTab];
    if constexpr (E::kBf16) fill_bf16_exp_table(etab);
    load_exp_table(tab);  // its barrier also covers etab
    const int lt = threadIdx.x % kRowThreads;
    const int64_t i_first = static_cast<int64_t>(lt) * E::kPer;
    const int64_t G = static_cast<int64_t>(gridDim.x) * kRowsPerBlock;
    const int64_t R = static_cast<int64_t>(a.M + 1) * a.U;
    const int nsw = static_cast<int>((a.K + kStride - 1) / kStride);  // sweeps per row
    // Row r of the workspace parts: the averaged rows (token u at r = u),
    // then the worker rows (row m U + u at r = U + m U + u).
    auto row_of = [&](int64_t r) -> rsrc_t {
        return r < a.U ? js_row(a.avg, r, a.ldk, E::kElem) : js_row(a.workers, r - a.U, a.ldk, E::kElem);
    };
    // The group index is uniform in a wave: in a scalar register, the row's
    // buffer descriptor stays scalar (no per-load waterfall).
    const int g = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kRowThreads));
    int64_t q = static_cast<int64_t>(blockIdx.x) * kRowsPerBlock + g;  // streaming position
    u32x4 nxt = {0, 0, 0, 0};
    if (q < R && i_first < a.K)
        nxt = __builtin_amdgcn_raw_buffer_load_b128(row_of(js_stream_row(q, a.M, a.U)),
                                                    static_cast<uint32_t>(i_first * E::kElem), 0, kLoadPolicy);
    for (; q < R; q += G) {
        const int64_t r = js_stream_row(q, a.M, a.U);
        const bool has_next = q + G < R;
        const rsrc_t rr = row_of(r);
        const rsrc_t rn = has_next ? row_of(js_stream_row(q + G, a.M, a.U)) : rr;
        RowLse st;
        TopVecs<E> top;
        const bool avg = r < a.U;
        if (avg)
            row_terms<E, true>(rr, rn, has_next, i_first, a.K, nsw, nxt, st, etab, tab, top);
        else
            row_terms<E, false>(rr, rn, has_next, i_first, a.K, nsw, nxt, st, etab, tab, top);
        double ml, sl;
        row_lse_lane(st, ml, sl, tab);
        const LsePart p = wave_lse(ml, sl, tab);
        if ((threadIdx.x & (kWave - 1)) == 0) w.part[r * kRowWaves + lt / kWave] = p;
        if (avg) w.top[r * kRowThreads + lt] = u32x4{top.t[0], top.t[1], top.t[2], top.t[3]};
    }
}

// The bin of a 256-bin digit histogram in which the need-th largest of the
// counted keys falls, and how many keys of that bin are still needed:
// thread t takes bin 255 - t, and an inclusive scan over the threads finds
// the first bin (from the top) at which the running count reaches need
// (need <= the histogram's total).  Block-wide barriers; every thread gets
// the result.  s_wsum: kWavesPerBlock ints; s_pick: 2 ints.
__device__ inline void hist_pick(const uint32_t *hist, int need, int *s_wsum, int *s_pick, int &bin, int &need_in) {
    static_assert(kBlock == 256, "one histogram bin per thread");
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int c = static_cast<int>(hist[255 - tid]);
    int incl = c;
    for (int o = 1; o < kWave; o <<= 1) {
        const int t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) s_wsum[wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; ++w) incl += s_wsum[w];
    if (incl >= need && incl - c < need) {
        s_pick[0] = 255 - tid;
        s_pick[1] = need - (incl - c);
    }
    __syncthreads();
    bin = s_pick[0];
    need_in = s_pick[1];
}

// Per token (block u; thread t the row thread lt = t of js_rows_kernel):
// the averaged row's log-sum-exp from its wave parts, its top-k set by a
// radix select over the row (8 key bits per pass from the top, then a
// collection pass that splits the tie at the threshold in index order), then
// JS_m for every worker.  Any k up to kJsMaxTopK: the path for k above a
// block's threads, and for the tokens the wave kernel flags (flag !=
// nullptr: only those).
template <class E>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4, 8)))
void js_token_radix_kernel(JsParams a, JsWork w, const int32_t *flag) {
    constexpr int P = E::kPer;
    constexpr int kMaxK = kJsMaxTopK;
    constexpr int64_t kStride = static_cast<int64_t>(kBlock) * P;  // elements per block sweep
    constexpr int kWorkerLanes = kBlock / kJsGroup;                // threads per worker in the JS terms
    __shared__ uint32_t hist[256];
    __shared__ __align__(16) int32_t sel_idx[kMaxK];
    __shared__ float sel_val[kMaxK];
    __shared__ __align__(16) struct {
        int32_t idx[kMaxK];
        double la[kMaxK];
    } out;  // the selected tokens in index order, log pbar
    __shared__ double s_lse[kJsGroup];
    __shared__ int s_wsum[kWavesPerBlock], s_pick[2];
    __shared__ int s_nsel;
    __shared__ double tab[kTab];

    const int tid = threadIdx.x;
    const int k = a.k;
    __shared__ int64_t s_tok[kBlock];
    __shared__ int s_ntok;
    bool have_tab = false;
    // The block's tokens u = blockIdx.x + j gridDim.x, kBlock values of j at
    // a time: all of them, or (flag != nullptr) those flagged, their flags
    // read by the block's threads at once.
    const int64_t n_mine = (a.U - blockIdx.x + gridDim.x - 1) / gridDim.x;
    for (int64_t j0 = 0; j0 < n_mine; j0 += kBlock) {
        int ntok = static_cast<int>(n_mine - j0 < kBlock ? n_mine - j0 : kBlock);
        if (flag) {
            if (tid == 0) s_ntok = 0;
            __syncthreads();
            const int64_t uu = blockIdx.x + (j0 + tid) * gridDim.x;
            if (tid < ntok && flag[uu] != 0) s_tok[atomicAdd(&s_ntok, 1)] = uu;
            __syncthreads();
            ntok = s_ntok;
        }
        for (int q = 0; q < ntok; ++q) {
            const int64_t u = flag ? s_tok[q] : blockIdx.x + (j0 + q) * gridDim.x;
            if (!have_tab) {  // blocks without a flagged token leave without it
                load_exp_table(tab);
                have_tab = true;
            }
            const rsrc_t ra = js_row(a.avg, u, a.ldk, E::kElem);
            const double lse_a = row_lse(w.part + u * kRowWaves, tab);
            {
                // Radix select of the k-th largest key, 8 bits per pass from the top.
                uint32_t prefix = 0;
                int need = k, count_eq = 0;
                for (int pass = 0; pass < E::kKeyBits / 8; ++pass) {
                    const int shift = E::kKeyBits - 8 * (pass + 1);
                    hist[tid] = 0;
                    __syncthreads();
                    for (int64_t i0 = static_cast<int64_t>(tid) * P; i0 < a.K; i0 += kStride) {
                        float v[P];
                        uint32_t key[P];
                        const int n = load_vec<E>(ra, i0, a.K, v, key);
    #pragma unroll
                        for (int j = 0; j < P; ++j)
                            if (j < n && (pass == 0 || (key[j] >> (shift + 8)) == prefix))
                                atomicAdd(&hist[(key[j] >> shift) & 255u], 1u);
                    }
                    __syncthreads();
                    int bin, need_in;
                    hist_pick(hist, need, s_wsum, s_pick, bin, need_in);
                    count_eq = static_cast<int>(hist[bin]);  // read before the next pass clears it
                    prefix = (prefix << 8) | static_cast<uint32_t>(bin);
                    need = need_in;
                    __syncthreads();
                }
                const uint32_t T = prefix;
                const int need_eq = need;
                const bool take_all_eq = count_eq == need_eq;

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
                    // one block sweep at a time (thread order is element order within
                    // a sweep), until need_eq are taken.
                    const int lane = tid & (kWave - 1), wave = tid / kWave;
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
                        int incl = cnt;  // inclusive prefix over the wave's lanes
                        for (int o = 1; o < kWave; o <<= 1) {
                            const int t = __shfl_up(incl, o);
                            if (lane >= o) incl += t;
                        }
                        if (lane == kWave - 1) s_wsum[wave] = incl;
                        __syncthreads();
                        int rank = incl - cnt;
                        for (int wv = 0; wv < wave; ++wv) rank += s_wsum[wv];
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
                        remaining = k - s_nsel;
                        __syncthreads();  // every thread has read s_nsel before s_wsum is rewritten
                    }
                }
            }

            // Rank sort by token index (indices are distinct), then the averaged
            // model's log-probabilities of the selected tokens.
            // Pad to a multiple of 4 with an index above every token.
            if (tid < 4 && k + tid < ((k + 3) & ~3)) sel_idx[k + tid] = INT32_MAX;
            __syncthreads();
            for (int t = tid; t < k; t += kBlock) {
                const int32_t my = sel_idx[t];
                int r = 0;
                for (int j = 0; j < k; j += 4) {
                    const u32x4 o = *reinterpret_cast<const u32x4 *>(&sel_idx[j]);
    #pragma unroll
                    for (int q = 0; q < 4; ++q) r += static_cast<int32_t>(o[q]) < my ? 1 : 0;
                }
                out.idx[r] = my;
                out.la[r] = static_cast<double>(sel_val[t]) - lse_a;
            }
            __syncthreads();
            if (a.topk_out)
                for (int t = tid; t < k; t += kBlock) a.topk_out[u * k + t] = out.idx[t];

            // JS terms, kJsGroup workers at a time: worker j of the group takes
            // threads [j, j + 1) * kWorkerLanes (half a wave), thread l of them
            // the selected tokens l, l + kWorkerLanes, ... in index order; the
            // half-wave sum is d's.
            constexpr double kLog2 = 0.69314718055994530942;
            const int j = tid / kWorkerLanes, l = tid % kWorkerLanes;
            for (int64_t w0 = 0; w0 < a.M; w0 += kJsGroup) {
                const int nw = a.M - w0 < kJsGroup ? static_cast<int>(a.M - w0) : kJsGroup;
                if (tid < nw) s_lse[tid] = row_lse(w.part + (a.U + (w0 + tid) * a.U + u) * kRowWaves, tab);
                __syncthreads();
                double acc = 0.0;
                const int64_t row = (w0 + (j < nw ? j : 0)) * a.U + u;
                if (j < nw) {
                    const char *zrow = static_cast<const char *>(a.workers) + row * a.ldk * E::kElem;
                    const double lse_w = s_lse[j];
                    constexpr int kGather = 4;  // gathers a thread has in flight
                    for (int t0 = l; t0 < k; t0 += kGather * kWorkerLanes) {
                        float z[kGather];
    #pragma unroll
                        for (int q = 0; q < kGather; ++q) {
                            const int t = t0 + q * kWorkerLanes;
                            z[q] = t < k ? E::at_ptr(zrow, out.idx[t]) : 0.0f;
                        }
    #pragma unroll
                        for (int q = 0; q < kGather; ++q) {
                            const int t = t0 + q * kWorkerLanes;
                            if (t < k) acc += js_term(static_cast<double>(z[q]) - lse_w, out.la[t]);
                        }
                    }
                }
                for (int o = kWorkerLanes / 2; o > 0; o >>= 1) acc += shfl_xor_d(acc, o);
                if (l == 0 && j < nw) a.d_out[row] = sqrt((acc > 0.0 ? acc : 0.0) / kLog2);
                __syncthreads();  // s_lse is rewritten by the next group
            }
            // The next token reuses the shared arrays, and the next group of
            // tokens s_tok: the last barrier above follows every read of them.
        }
    }
}

// The row kernel's loads without its arithmetic: the same grid, row groups,
// streaming order, lane elements and prefetch, and no LDS table; each wave
// folds what it loads into one word (an XOR) and stores it over its part in
// the workspace, so no load can be dropped.  Its rate is the practical
// ceiling of the row kernel's access pattern.
template <class E>
__global__ __launch_bounds__(kRowsBlock) void js_rows_pattern_kernel(JsParams a, JsWork w) {
    const int lt = threadIdx.x % kRowThreads;
    const int64_t i_first = static_cast<int64_t>(lt) * E::kPer;
    constexpr int64_t kStride = static_cast<int64_t>(kRowThreads) * E::kPer;
    const int64_t G = static_cast<int64_t>(gridDim.x) * kRowsPerBlock;
    const int64_t R = static_cast<int64_t>(a.M + 1) * a.U;
    auto row_of = [&](int64_t r) -> rsrc_t {
        return r < a.U ? js_row(a.avg, r, a.ldk, E::kElem) : js_row(a.workers, r - a.U, a.ldk, E::kElem);
    };
    const int g = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kRowThreads));
    int64_t q = static_cast<int64_t>(blockIdx.x) * kRowsPerBlock + g;  // streaming position
    u32x4 nxt = {0, 0, 0, 0};
    if (q < R && i_first < a.K)
        nxt = __builtin_amdgcn_raw_buffer_load_b128(row_of(js_stream_row(q, a.M, a.U)),
                                                    static_cast<uint32_t>(i_first * E::kElem), 0, kLoadPolicy);
    for (; q < R; q += G) {
        const int64_t r = js_stream_row(q, a.M, a.U);
        const bool has_next = q + G < R;
        const rsrc_t rr = row_of(r);
        const rsrc_t rn = has_next ? row_of(js_stream_row(q + G, a.M, a.U)) : rr;
        uint32_t acc = 0;
        for (int64_t i0 = i_first; i0 < a.K; i0 += kStride) {
            const u32x4 cur = nxt;
            if (i0 + kStride < a.K)
                nxt = __builtin_amdgcn_raw_buffer_load_b128(rr, static_cast<uint32_t>((i0 + kStride) * E::kElem), 0,
                                                            kLoadPolicy);
            else if (has_next)
                nxt = __builtin_amdgcn_raw_buffer_load_b128(rn, static_cast<uint32_t>(i_first * E::kElem), 0,
                                                            kLoadPolicy);
            acc ^= cur[0] ^ cur[1] ^ cur[2] ^ cur[3];
        }
        for (int o = kWave / 2; o > 0; o >>= 1) acc ^= static_cast<uint32_t>(__shfl_xor(static_cast<int>(acc), o));
        if ((threadIdx.x & (kWave - 1)) == 0) reinterpret_cast<uint32_t *>(w.part)[r * kRowWaves + lt / kWave] = acc;
    }
}

// ------------------------------------------------- per token, one wave each
constexpr int kWaveTokens = kBlock / kWave;            // tokens per block of js_token_wave_kernel
constexpr int kRtPerLane = kRowThreads / kWave;        // row threads whose recorded maxima a lane takes
constexpr int kRecords = kRowThreads * kTopVecs;       // recorded vector maxima per token
constexpr int kWaveCandSmall = 512;                    // candidates a token may have, k <= 256
constexpr int kWaveCandLarge = 1024;                   // the same, 256 < k <= 512
constexpr int kWaveMaxK = kWaveCandLarge / 2;          // k the wave kernel takes (at most half its candidates)
constexpr int kJsLanes = kWave / kJsGroup;             // lanes per worker in the JS terms
constexpr int kReadRound = 4;                          // recorded vectors a lane reads at once
constexpr int kWaveGather = 16;                        // worker logits a lane gathers at once

// Orders a wave's LDS accesses: what a lane wrote before it is visible to
// every lane of the wave after it.
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Slots, in lane order, for the lanes that set `pred`: base, base + 1, ...;
// base (wave-uniform) grows by their number.  Every lane of the wave calls it.
__device__ inline int wave_append(bool pred, int &base) {
    const uint64_t m = __ballot(pred);
    const uint32_t below = __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u);  // set lanes before this one
    const int slot = base + static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32), below));
    base += __popcll(m);
    return slot;
}

// One wave's LDS in js_token_wave_kernel with up to kCand candidates and
// k <= kCand / 2.
template <int kCand>
struct __align__(16) WaveLds {
    uint64_t comp[kCand];  // candidates: key << 32 | ~index, larger = earlier in (key desc, index asc)
    union {
        uint32_t queue[kRecords];  // first elements of the recorded vectors to read again
        struct {
            int32_t idx[kCand / 2];
            double la[kCand / 2];
        } out;  // the selected tokens in index order, log pbar
    } u;
    double lse[kJsGroup];
};

__device__ inline uint64_t shfl_xor_u64(uint64_t x, int mask) {
    const uint32_t lo = static_cast<uint32_t>(__shfl_xor(static_cast<int>(static_cast<uint32_t>(x)), mask));
    const uint32_t hi = static_cast<uint32_t>(__shfl_xor(static_cast<int>(x >> 32), mask));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sorts the wave's 64 R words (word p = lane + 64 r in v[r] of lane
// `lane`) in place, descending or ascending: Batcher's bitonic network,
// partners in other lanes exchanged by shuffles, partners in the same lane
// (distances of 64 and more) in registers.
template <int R, bool kDescending>
__device__ inline void wave_bitonic_sort(uint64_t (&v)[R], int lane) {
#pragma unroll
    for (int k = 2; k <= kWave * R; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= kWave) {
                const int jr = j / kWave;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    if (r & jr) continue;
                    const bool down = ((r * kWave) & k) == 0;  // this pair's block sorts downwards
                    const uint64_t x = v[r], y = v[r | jr];
                    const bool big_first = down == kDescending;
                    const uint64_t hi = x > y ? x : y, lo = x > y ? y : x;
                    v[r] = big_first ? hi : lo;
                    v[r | jr] = big_first ? lo : hi;
                }
            } else {
                const bool lower = (lane & j) == 0;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const uint64_t o = shfl_xor_u64(v[r], j);
                    const bool down = ((lane + r * kWave) & k) == 0;
                    const bool take_big = (lower == (down == kDescending));
                    v[r] = take_big ? (v[r] > o ? v[r] : o) : (v[r] > o ? o : v[r]);
                }
            }
        }
    }
}

// The selection from C candidates (candidate c in slot c of L.comp, as
// key << 32 | ~index; 64 R slots at least): the candidates sorted
// descending, the first k selected, those sorted by index; into L.u.out
// the selected tokens in index order with log pbar = value - lse_a (the
// value recovered from the key).
template <class E, int R>
__device__ inline void select_sorted(const uint64_t *comp, int C, int k, int lane, double lse_a, int32_t *out_idx,
                                     double *out_la) {
    uint64_t v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int c = lane + r * kWave;
        v[r] = c < C ? comp[c] : 0;  // 0: below every candidate
    }
    wave_bitonic_sort<R, true>(v, lane);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int p = lane + r * kWave;
        // index << 32 | key for the selected, above every index otherwise
        v[r] = p < k ? (static_cast<uint64_t>(0xFFFFFFFFu - static_cast<uint32_t>(v[r])) << 32) | (v[r] >> 32)
                     : ~0ull;
    }
    wave_bitonic_sort<R, false>(v, lane);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int p = lane + r * kWave;
        if (p < k) {
            out_idx[p] = static_cast<int32_t>(v[r] >> 32);
            out_la[p] = static_cast<double>(E::value_of(static_cast<uint32_t>(v[r]))) - lse_a;
        }
    }
}

// Per token, one wave (token u = blockIdx.x * kWaveTokens + wave; no block
// barriers after the exp table): the averaged row's log-sum-exp from its
// wave parts; T0, the k-th largest of the 1024 recorded vector maxima (16-bit
// keys, built from the top bit down by counting with ballots), which is at
// most the row's k-th largest key, so the selected tokens are among the
// elements with key >= T0 (on these inputs a little over k); the vectors
// whose maxima reach T0 go to a queue and are read again in one round, and
// their elements at or above T0 are appended to the candidates in lane
// order; the candidates are sorted under (key descending, index ascending)
// by a bitonic network across the wave, the first k then by index; then
// the JS terms, kJsLanes lanes per worker, with a lane's gathers issued
// together.  A token with more than kCand candidates (a row of many equal
// logits) is flagged and left to js_token_radix_kernel.  k <= kCand / 2:
// kCand 512 keeps a block's LDS at 35 KB, 1024 (for 256 < k <= 512) takes
// 58 KB.
template <class E, int kCand>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kCand == kWaveCandSmall ? 4 : 2, 8)))
void js_token_wave_kernel(JsParams a, JsWork w) {
    constexpr int P = E::kPer;
    constexpr int64_t kStride = static_cast<int64_t>(kRowThreads) * P;  // elements per row sweep
    __shared__ double tab[kTab];
    __shared__ WaveLds<kCand> lds[kWaveTokens];
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t u = static_cast<int64_t>(blockIdx.x) * kWaveTokens + wave;
    const bool live = u < a.U;  // the whole wave

    // The largest vector maxima of row threads lane + q kWave (entries
    // key16 << 16 | vector index, largest first; 0: none) and the averaged
    // row's wave parts, loaded while the exp table is.
    u32x4 tq[kRtPerLane];
    LsePart pa[kRowWaves];
    if (live) {
#pragma unroll
        for (int q = 0; q < kRtPerLane; ++q) tq[q] = w.top[u * kRowThreads + lane + q * kWave];
#pragma unroll
        for (int j = 0; j < kRowWaves; ++j) pa[j] = w.part[u * kRowWaves + j];
    }
    load_exp_table(tab);
    if (!live) return;
    WaveLds<kCand> &L = lds[wave];
    const int k = a.k;
    const rsrc_t ra = js_row(a.avg, u, a.ldk, E::kElem);
    const double lse_a = lse_of_parts(pa, tab);

    // T0: the largest t with at least k entries whose key reaches it (an
    // empty entry counts as key 0), one bit at a time from the top.
    uint32_t T0 = 0;
    for (int b = 15; b >= 0; --b) {
        const uint32_t t = T0 | (1u << b);
        int cnt = 0;
#pragma unroll
        for (int q = 0; q < kRtPerLane; ++q)
#pragma unroll
            for (int i = 0; i < kTopVecs; ++i) cnt += __popcll(__ballot((tq[q][i] >> 16) >= t));
        if (cnt >= k) T0 = t;
    }

    // The k-th largest of distinct vectors' maxima is at most the row's
    // k-th largest key, so the selected tokens are among the candidates: the
    // elements whose key reaches kthr (key16 T0, widened to a full key for
    // float32; T0 = 0 takes every element).  They lie in vectors whose maxima
    // reach T0: a row thread's recorded ones, or any of its vectors when even
    // its fourth entry reaches T0 (it may have more).
    const uint32_t kthr = E::kBf16 ? T0 : T0 << 16;
    int nsel = 0;  // candidates appended so far (wave-uniform)
    auto collect = [&](bool have, u32x4 t, int64_t i0) {
        float v[P];
        E::values(t, v);
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const uint32_t key = E::key_of(v[j]);
            const bool c = have && i0 + j < a.K && key >= kthr;
            const int slot = wave_append(c, nsel);
            if (c && slot < kCand)
                L.comp[slot] = (static_cast<uint64_t>(key) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(i0 + j));
        }
    };
    int nq = 0;
#pragma unroll
    for (int q = 0; q < kRtPerLane; ++q) {
        const uint32_t last = tq[q][kTopVecs - 1];
        const bool crowded = last != 0 && (last >> 16) >= T0;  // read below, by the whole wave
        const int64_t rt = lane + q * kWave;
#pragma unroll
        for (int i = 0; i < kTopVecs; ++i) {
            const uint32_t e = tq[q][i];
            const int64_t at = rt * P + static_cast<int64_t>(e & 0xFFFFu) * kStride;
            const bool use = !crowded && e != 0 && (e >> 16) >= T0 && at < a.K;
            const int slot = wave_append(use, nq);
            if (use) L.u.queue[slot] = static_cast<uint32_t>(at);
        }
    }
    nq = __builtin_amdgcn_readfirstlane(nq);
    wave_sync();
    for (int s0 = 0; s0 < nq; s0 += kReadRound * kWave) {
        u32x4 t[kReadRound];
        int64_t at[kReadRound];
        bool have[kReadRound];
#pragma unroll
        for (int j = 0; j < kReadRound; ++j) {
            const int s = s0 + j * kWave + lane;
            have[j] = s < nq;
            at[j] = have[j] ? static_cast<int64_t>(L.u.queue[s]) : 0;
            t[j] = u32x4{0, 0, 0, 0};
            if (have[j])
                t[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, static_cast<uint32_t>(at[j] * E::kElem), 0,
                                                             kLoadPolicy);
        }
#pragma unroll
        for (int j = 0; j < kReadRound; ++j)
            if (s0 + j * kWave < nq) collect(have[j], t[j], at[j]);
    }
    // A row thread whose fourth entry reaches T0 may have more such vectors
    // (rare): the whole wave reads all of its vectors, one per lane.
#pragma unroll
    for (int q = 0; q < kRtPerLane; ++q) {
        const uint32_t last = tq[q][kTopVecs - 1];
        uint64_t scan = __ballot(last != 0 && (last >> 16) >= T0);
        while (scan != 0) {
            const int64_t rt = __builtin_ctzll(scan) + q * kWave;
            scan &= scan - 1;
            for (int64_t b0 = rt * P; b0 < a.K; b0 += kWave * kStride) {
                const int64_t i0 = b0 + lane * kStride;
                const bool have = i0 < a.K;
                u32x4 t = u32x4{0, 0, 0, 0};
                if (have) t = __builtin_amdgcn_raw_buffer_load_b128(ra, static_cast<uint32_t>(i0 * E::kElem), 0,
                                                                    kLoadPolicy);
                collect(have, t, i0);
            }
        }
    }
    // More candidates than the wave holds go to the radix kernel; fewer than
    // k cannot occur (each of the k entries at or above T0 names a distinct
    // vector holding an element at or above it) and would leave selected
    // slots without a token, so that too is handed on rather than gathered.
    const int C = __builtin_amdgcn_readfirstlane(nsel);
    if (C > kCand || C < k) {  // the same in every lane
        if (lane == 0) w.flag[u] = 1;
        return;
    }
    wave_sync();

    // The selection, by sorting: the queue is no longer read, and its space
    // takes the selected tokens in index order, with the averaged model's
    // log-probabilities.
    if (C <= 2 * kWave)
        select_sorted<E, 2>(L.comp, C, k, lane, lse_a, L.u.out.idx, L.u.out.la);
    else if (C <= 8 * kWave || kCand <= 8 * kWave)  // 8 per lane holds every candidate of the small kernel
        select_sorted<E, 8>(L.comp, C, k, lane, lse_a, L.u.out.idx, L.u.out.la);
    else
        select_sorted<E, kCand / kWave>(L.comp, C, k, lane, lse_a, L.u.out.idx, L.u.out.la);
    wave_sync();
    if (a.topk_out)
        for (int t = lane; t < k; t += kWave) a.topk_out[u * k + t] = L.u.out.idx[t];

    // JS terms, kJsGroup workers at a time: worker jw of the group takes
    // lanes [jw, jw + 1) * kJsLanes, lane l of them the selected tokens l,
    // l + kJsLanes, ... in index order; their sum is d's.  The workers'
    // log-sum-exp parts are loaded while the first gathers are in flight.
    constexpr double kLog2 = 0.69314718055994530942;
    const int jw = lane / kJsLanes, l = lane % kJsLanes;
    for (int64_t w0 = 0; w0 < a.M; w0 += kJsGroup) {
        const int nw = a.M - w0 < kJsGroup ? static_cast<int>(a.M - w0) : kJsGroup;
        const bool mine_w = jw < nw;
        const int64_t row = (w0 + (mine_w ? jw : 0)) * a.U + u;
        const char *zrow = static_cast<const char *>(a.workers) + row * a.ldk * E::kElem;
        double acc = 0.0;
        for (int t0 = 0; t0 < k; t0 += kWaveGather * kJsLanes) {
            float z[kWaveGather];
#pragma unroll
            for (int q = 0; q < kWaveGather; ++q) {
                const int t = t0 + l + q * kJsLanes;
                z[q] = mine_w && t < k ? E::at_ptr(zrow, L.u.out.idx[t]) : 0.0f;
            }
            if (t0 == 0) {
                if (lane < nw) L.lse[lane] = row_lse(w.part + (a.U + (w0 + lane) * a.U + u) * kRowWaves, tab);
                wave_sync();
            }
            const double lse_w = L.lse[mine_w ? jw : 0];
#pragma unroll
            for (int q = 0; q < kWaveGather; ++q) {
                const int t = t0 + l + q * kJsLanes;
                if (mine_w && t < k) acc += js_term(static_cast<double>(z[q]) - lse_w, L.u.out.la[t]);
            }
        }
        for (int o = kJsLanes / 2; o > 0; o >>= 1) acc += shfl_xor_d(acc, o);
        if (l == 0 && mine_w) a.d_out[row] = sqrt((acc > 0.0 ? acc : 0.0) / kLog2);
        wave_sync();  // L.lse is rewritten by the next group
    }
    if (lane == 0) w.flag[u] = 0;
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

namespace {
int64_t js_part_bytes(int32_t M, int64_t U) {
    return (static_cast<int64_t>(M) + 1) * U * kRowWaves * static_cast<int64_t>(sizeof(LsePart));
}
int64_t js_top_bytes(int64_t U) { return U * kRowThreads * static_cast<int64_t>(sizeof(u32x4)); }
}  // namespace

int64_t js_workspace_bytes(int32_t bf16, int32_t M, int64_t U) {
    (void)bf16;
    return js_part_bytes(M, U) + js_top_bytes(U) + (U * 4 + 15) / 16 * 16;
}

bool js_launch(const void *avg, const void *workers, int32_t bf16, int32_t M, int64_t U, int64_t K, int64_t ldk,
               int32_t k, double *d_out, double *mean_out, int32_t *topk_out, void *workspace, int num_cus,
               hipStream_t stream) {
    JsParams p{avg, workers, d_out, topk_out, U, K, ldk, M, k};
    char *ws = static_cast<char *>(workspace);
    const int64_t o_top = js_part_bytes(M, U), o_flag = o_top + js_top_bytes(U);
    JsWork w{reinterpret_cast<LsePart *>(ws), reinterpret_cast<u32x4 *>(ws + o_top),
             reinterpret_cast<int32_t *>(ws + o_flag)};
    const int64_t groups = ((static_cast<int64_t>(M) + 1) * U + kRowsPerBlock - 1) / kRowsPerBlock;
    const int64_t grid = std::min<int64_t>(groups, static_cast<int64_t>(kRowsBlocksPerCu) * std::max(num_cus, 1));
    const dim3 token_waves(static_cast<unsigned>((U + kWaveTokens - 1) / kWaveTokens));
    // The wave kernel names a row thread's vectors by 16-bit indices.
    const bool wave_path =
        k <= kWaveMaxK && js_thread_vectors(K, bf16 ? JsBF16::kPer : JsF32::kPer) <= kTopIndexLimit;
    // The radix kernel takes every token, or after the wave kernel only the
    // flagged ones (few): then a few blocks per CU walk the flags.
    const dim3 tokens(static_cast<unsigned>(wave_path ? std::min<int64_t>(U, 4 * std::max(num_cus, 1)) : U));
    if (bf16) {
        hipLaunchKernelGGL(js_rows_kernel<JsBF16>, dim3(static_cast<unsigned>(grid)), dim3(kRowsBlock), 0, stream, p, w);
        if (wave_path && k <= kWaveCandSmall / 2)
            hipLaunchKernelGGL((js_token_wave_kernel<JsBF16, kWaveCandSmall>), token_waves, dim3(kBlock), 0, stream, p, w);
        else if (wave_path)
            hipLaunchKernelGGL((js_token_wave_kernel<JsBF16, kWaveCandLarge>), token_waves, dim3(kBlock), 0, stream, p, w);
        hipLaunchKernelGGL(js_token_radix_kernel<JsBF16>, tokens, dim3(kBlock), 0, stream, p, w,
                           wave_path ? static_cast<const int32_t *>(w.flag) : nullptr);
    } else {
        hipLaunchKernelGGL(js_rows_kernel<JsF32>, dim3(static_cast<unsigned>(grid)), dim3(kRowsBlock), 0, stream, p, w);
        if (wave_path && k <= kWaveCandSmall / 2)
            hipLaunchKernelGGL((js_token_wave_kernel<JsF32, kWaveCandSmall>), token_waves, dim3(kBlock), 0, stream, p, w);
        else if (wave_path)
            hipLaunchKernelGGL((js_token_wave_kernel<JsF32, kWaveCandLarge>), token_waves, dim3(kBlock), 0, stream, p, w);
        hipLaunchKernelGGL(js_token_radix_kernel<JsF32>, tokens, dim3(kBlock), 0, stream, p, w,
                           wave_path ? static_cast<const int32_t *>(w.flag) : nullptr);
    }
    if (hipGetLastError() != hipSuccess) return false;
    if (mean_out) {
        hipLaunchKernelGGL(js_mean_kernel, dim3(M), dim3(256), 0, stream, d_out, U, mean_out);
        if (hipGetLastError() != hipSuccess) return false;
    }
    return true;
}

bool js_pattern_launch(const void *avg, const void *workers, int32_t bf16, int32_t M, int64_t U, int64_t K,
                       int64_t ldk, void *workspace, int num_cus, hipStream_t stream) {
    JsParams p{avg, workers, nullptr, nullptr, U, K, ldk, M, 1};
    JsWork w{static_cast<LsePart *>(workspace), nullptr, nullptr};
    const int64_t groups = ((static_cast<int64_t>(M) + 1) * U + kRowsPerBlock - 1) / kRowsPerBlock;
    const int64_t grid = std::min<int64_t>(groups, static_cast<int64_t>(kRowsBlocksPerCu) * std::max(num_cus, 1));
    if (bf16)
        hipLaunchKernelGGL(js_rows_pattern_kernel<JsBF16>, dim3(static_cast<unsigned>(grid)), dim3(kRowsBlock), 0,
                           stream, p, w);
    else
        hipLaunchKernelGGL(js_rows_pattern_kernel<JsF32>, dim3(static_cast<unsigned>(grid)), dim3(kRowsBlock), 0,
                           stream, p, w);
    return hipGetLastError() == hipSuccess;
}

}  // namespace fgd
