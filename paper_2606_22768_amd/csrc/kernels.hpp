// kernels.hpp -- HIP kernels of the fused outer step for gfx950 (CDNA4).
//
// The step (Sec. 4.1 factored formulation; Appendix A, Algorithm 1, outer
// step; Appendix B Nesterov form) is a bandwidth-bound pass over M worker
// rows.  Every parameter index p is independent given W, so one lane owns V
// consecutive parameters of *all* M workers and keeps them in registers:
//
//   phase A  load theta_prev and theta_local rows (nontemporal buffer loads,
//            16 bytes per lane where V allows), g0 = theta_prev - theta_local
//   mix      Mix2 on g and Mix1 on x = theta_prev: a global mean in registers,
//            or CSR rounds.  A CSR round needs u[col] for a run-time col that
//            is the same for the whole wave, so the lane parks its M values
//            in its own column of an LDS array [M][block][V] (plus a zero
//            row M when some table pads a short row) and gathers from there
//            (no barrier: a lane touches only its own column).
//            Per round the host supplies a padded table [width][M] of
//            (column, weight): the d-th live entry of every row, in ascending
//            column order, so the sum runs in the CSR row's order.
//   phase D  load momentum rows, v' = mu v + g, theta' = x - lr (g + mu v')
//            (plain momentum: theta' = x - lr v'), store theta' (RNE to bf16
//            for bf16 storage) and v'.  With the optimizer state mixed
//            (Appendix B, GlobalM1S) all momentum rows are loaded first and
//            Mix1 is applied to them before the update.
//   subset   Mix2 restricted to parameter segments (the Mix2-subset
//            configuration): after every round the elements outside the
//            subset are restored from the lane's own LDS column, which still
//            holds the round's input.
//   CD       S_m(u) = sum_p (u_m - mean_n u_n)^2 for every intermediate u
//            (Sec. 4.4; Appendix D.1): float32 deviations, a reduce-scatter
//            across the wave's lanes (cross-row lane swaps, then DPP),
//            double accumulation per (row, worker) in LDS, per-block partials
//            and a fixed-order finalize kernel, so results are deterministic.
//
// Global memory is addressed through buffer descriptors: each row's address
// is formed in scalar registers and every lane adds one 32-bit byte offset,
// so a lane needs a single address register however many rows it streams.
// No matrix cores: the work is a sparse weighted reduction across rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fgd {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int kBlock = 256;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = kBlock / kWave;

enum MixKind : int32_t { kIdentity = 0, kGlobal = 1, kTable = 2 };

struct MixDev {
    int32_t kind;       // MixKind
    int32_t rounds;     // table rounds (kTable)
    int32_t width;      // entries per row in each round's table
    int32_t pad_;
    const int2 *table;  // [rounds][width][M] of (column, bit pattern of float weight)
};

struct StepParams {
    const void *theta_prev;   // [M][ld] storage type, read
    void *theta_out;          // the same array, written (a separate argument so the
                              // row descriptors of the loads and of the stores are
                              // formed independently and none stays live across the tile)
    const void *theta_local;  // [M][ld] storage type
    const float *mom;         // [M][ld] float32, read
    float *mom_out;           // the same array, written (separate for the same reason)
    double *cd_partials;      // [gridDim.x][n_cd][M] or nullptr
    int64_t P, ld, ntiles;
    int32_t M, n_cd;
    int32_t lds_rows;         // rows of the LDS gather array: 0 (no CSR mix), M, or M + 1
                              // when some table pads a short row (row M is then zero)
    int32_t nesterov;         // 1: theta' = x - lr (g + mu v'); 0: theta' = x - lr v'
    float lr, mu;
    int32_t n_seg, pad_;      // Mix2 subset: number of segments (0: Mix2 everywhere)
    const int64_t *seg;       // [n_seg][2] ascending half-open [begin, end) parameter ranges
    MixDev mix1, mix2;
    // Split execution (the Mix1 half and the blocking half of a round):
    const void *x;            // blocking half: the stored Mix1 output, [M][ld] storage type
    void *x_out;              // Mix1 half: where it stores x
    void *local_out;          // blocking half: theta_local, receives theta' (nullptr: no write-back)
    int *chunk_counter;       // Mix1 half: next chunk to take (0 at launch)
    int64_t nchunks;          // Mix1 half: chunks of chunk_tiles tiles; cd_partials is [nchunks][n_cd][M]
    int64_t chunk_tiles;
};

struct ConsensusParams {
    const void *x;            // [M][ld] storage type
    double *partials;         // [gridDim.x][M]
    int64_t P, ld, ntiles;
    int32_t M, pad_;
};

constexpr int pow2_at_least(int m) { return m <= 1 ? 1 : 2 * pow2_at_least((m + 1) / 2); }
constexpr int ilog2(int m) { return m <= 1 ? 0 : 1 + ilog2(m / 2); }

// ------------------------------------------------------------ tuning knobs
// Defaults are the shipped configuration; variants are built with -D.

#ifndef FGD_NT
#define FGD_NT 1  // nontemporal hint on the streaming accesses
#endif
#ifndef FGD_WAVES_M8
#define FGD_WAVES_M8 2  // occupancy hint for up to 8 workers
#endif
#ifndef FGD_V_F32_M16
#define FGD_V_F32_M16 4  // float32 parameters per lane at 16 workers
#endif
#ifndef FGD_V_BF16_M8
#define FGD_V_BF16_M8 4  // bf16 parameters per lane up to 8 workers
#endif

// ------------------------------------------------------------ storage access

#ifndef FGD_NT_LOAD
#define FGD_NT_LOAD FGD_NT
#endif
#ifndef FGD_NT_STORE
#define FGD_NT_STORE FGD_NT
#endif
// Buffer-instruction cache bits of the streaming loads and stores (2: nontemporal).
constexpr int kLoadPolicy = FGD_NT_LOAD ? 2 : 0;
constexpr int kStorePolicy = FGD_NT_STORE ? 2 : 0;
constexpr int kRawBufferFlags = 0x00020000;   // raw (untyped) buffer descriptor, dword 3

// Descriptor of the row that starts `elem` elements (of `es` bytes) past
// `base`.  Offsets used with it stay far below the 2^31-byte record count.
__device__ __forceinline__ rsrc_t row_rsrc(const void *base, int64_t elem, int es) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(base)) + elem * es,
                                             static_cast<short>(0), 0x7fffffff, kRawBufferFlags);
}

// float32 values, V in {1, 2, 4}; `off` is the lane's byte offset in the row.
template <int V>
struct F32Io {
    __device__ static void load(rsrc_t r, uint32_t off, float (&o)[V]) {
        if constexpr (V == 4) {
            const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kLoadPolicy);
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = __uint_as_float(t[v]);
        } else if constexpr (V == 2) {
            const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kLoadPolicy);
            o[0] = __uint_as_float(t[0]);
            o[1] = __uint_as_float(t[1]);
        } else {
            o[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kLoadPolicy));
        }
    }
    __device__ static void store(rsrc_t r, uint32_t off, const float (&i)[V]) {
        if constexpr (V == 4) {
            const u32x4 t = {__float_as_uint(i[0]), __float_as_uint(i[1]), __float_as_uint(i[2]), __float_as_uint(i[3])};
            __builtin_amdgcn_raw_buffer_store_b128(t, r, off, 0, kStorePolicy);
        } else if constexpr (V == 2) {
            const u32x2 t = {__float_as_uint(i[0]), __float_as_uint(i[1])};
            __builtin_amdgcn_raw_buffer_store_b64(t, r, off, 0, kStorePolicy);
        } else {
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(i[0]), r, off, 0, kStorePolicy);
        }
    }
    // Writes only the first n < V values (ragged end of a row).
    __device__ static void store_part(rsrc_t r, uint32_t off, int n, const float (&i)[V]) {
#pragma unroll
        for (int v = 0; v < V; ++v)
            if (v < n) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(i[v]), r, off + 4 * v, 0, kStorePolicy);
    }
};

// Parameter storage: float32 (ParamF32) or bf16 bit patterns (ParamBF16).
// store() writes the values in the storage type and returns, in `s`, what
// was stored, widened back to float.
template <int V>
struct ParamF32 {
    static constexpr int kElem = 4;
    __device__ static void load(rsrc_t r, uint32_t off, float (&o)[V]) { F32Io<V>::load(r, off, o); }
    __device__ static void store(rsrc_t r, uint32_t off, const float (&i)[V], float (&s)[V]) {
        F32Io<V>::store(r, off, i);
#pragma unroll
        for (int v = 0; v < V; ++v) s[v] = i[v];
    }
    __device__ static void store_part(rsrc_t r, uint32_t off, int n, const float (&i)[V], float (&s)[V]) {
        F32Io<V>::store_part(r, off, n, i);
#pragma unroll
        for (int v = 0; v < V; ++v) s[v] = v < n ? i[v] : 0.0f;
    }
};

__device__ inline float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack_bf16(float a, float b) {
    f32x2 f = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

template <int V>
struct ParamBF16 {
    static constexpr int kElem = 2;
    __device__ static void load(rsrc_t r, uint32_t off, float (&o)[V]) {
        if constexpr (V == 8) {
            const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kLoadPolicy);
#pragma unroll
            for (int k = 0; k < 4; ++k) { o[2 * k] = bf16_lo(t[k]); o[2 * k + 1] = bf16_hi(t[k]); }
        } else if constexpr (V == 4) {
            const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kLoadPolicy);
            o[0] = bf16_lo(t[0]); o[1] = bf16_hi(t[0]); o[2] = bf16_lo(t[1]); o[3] = bf16_hi(t[1]);
        } else if constexpr (V == 2) {
            const uint32_t t = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kLoadPolicy);
            o[0] = bf16_lo(t); o[1] = bf16_hi(t);
        } else {
            const uint16_t t = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kLoadPolicy);
            o[0] = __uint_as_float(static_cast<uint32_t>(t) << 16);
        }
    }
    __device__ static void store(rsrc_t r, uint32_t off, const float (&i)[V], float (&s)[V]) {
        if constexpr (V == 1) {
            const uint32_t w = pack_bf16(i[0], 0.0f);
            __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(w & 0xFFFFu), r, off, 0, kStorePolicy);
            s[0] = bf16_lo(w);
        } else {
            uint32_t w[V / 2];
#pragma unroll
            for (int k = 0; k < V / 2; ++k) {
                w[k] = pack_bf16(i[2 * k], i[2 * k + 1]);
                s[2 * k] = bf16_lo(w[k]);
                s[2 * k + 1] = bf16_hi(w[k]);
            }
            if constexpr (V == 8) {
                const u32x4 t = {w[0], w[1], w[2], w[3]};
                __builtin_amdgcn_raw_buffer_store_b128(t, r, off, 0, kStorePolicy);
            } else if constexpr (V == 4) {
                const u32x2 t = {w[0], w[1]};
                __builtin_amdgcn_raw_buffer_store_b64(t, r, off, 0, kStorePolicy);
            } else {
                __builtin_amdgcn_raw_buffer_store_b32(w[0], r, off, 0, kStorePolicy);
            }
        }
    }
    __device__ static void store_part(rsrc_t r, uint32_t off, int n, const float (&i)[V], float (&s)[V]) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const uint32_t w = pack_bf16(i[v], 0.0f);
            if (v < n) __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(w & 0xFFFFu), r, off + 2 * v, 0,
                                                             kStorePolicy);
            s[v] = v < n ? bf16_lo(w) : 0.0f;
        }
    }
};

// ------------------------------------------------------- consensus pieces

// Cross-lane moves used by the reduce-scatter.  swap32 / swap16 exchange the
// upper half of `a` with the lower half of `b` across the two 32-lane halves
// (v_permlane32_swap) or across adjacent 16-lane rows (v_permlane16_swap).
__device__ __forceinline__ void swap32(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap16(float &a, float &b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
}
// DPP lane permutations inside a 16-lane row; each pairs lanes whose bit
// 3, 2, 1 or 0 differs and keeps the higher bits.
constexpr int kDppRowMirror = 0x140;      // l <-> 15 - l
constexpr int kDppRowHalfMirror = 0x141;  // l <-> 7 - l inside each 8
constexpr int kDppQuadXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppQuadXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// One step of the reduce-scatter on lane bit B: with n values left, lanes
// whose bit B is clear keep the lower n/2 values and lanes whose bit is set
// keep the upper n/2, each summed with its partner's copy; with one value
// left it is a plain all-reduce step.
template <int B, int C>
__device__ __forceinline__ void rs_step(float (&part)[C], int &n, int lane) {
    constexpr int ctrl = B == 3 ? kDppRowMirror : (B == 2 ? kDppRowHalfMirror : (B == 1 ? kDppQuadXor2 : kDppQuadXor1));
    if (n > 1) {
        n >>= 1;
#pragma unroll
        for (int i = 0; i < C / 2; ++i) {
            if (i < n) {
                // Read both values first: a select between two array lvalues
                // would index the register array dynamically.
                float lower_half = part[i], upper_half = part[i + n];
                if constexpr (B == 5 || B == 4) {
                    if constexpr (B == 5) swap32(lower_half, upper_half);
                    else swap16(lower_half, upper_half);
                    part[i] = lower_half + upper_half;
                } else {
                    const bool upper = (lane >> B) & 1;
                    const float send = upper ? lower_half : upper_half;
                    const float keep = upper ? upper_half : lower_half;
                    part[i] = keep + dpp<ctrl>(send);
                }
            }
        }
    } else {
        if constexpr (B == 5 || B == 4) {
            float a = part[0], b = part[0];
            if constexpr (B == 5) swap32(a, b);
            else swap16(a, b);
            part[0] = a + b;
        } else {
            part[0] += dpp<ctrl>(part[0]);
        }
    }
}

// Sum over the wave of part[j] for every j < C, scattered so that lane l ends
// up with the total of j = l >> (6 - log2 C) (every lane of that group of
// 64 / C lanes holds it).  The order of additions is fixed, so results are
// deterministic.  Needs all 64 lanes active.
template <int C>
__device__ inline float wave_reduce_scatter(float (&part)[C], int lane) {
    int n = C;
    rs_step<5>(part, n, lane);
    rs_step<4>(part, n, lane);
    rs_step<3>(part, n, lane);
    rs_step<2>(part, n, lane);
    rs_step<1>(part, n, lane);
    rs_step<0>(part, n, lane);
    return part[0];
}

// Sum of element v of rows [LO, LO + N) of u, rows at or past M counting as
// 0, as a balanced tree: each rounding chain has about log2(N) additions
// instead of N - 1 (64 workers of zero-mean values otherwise lose a few
// parts in 1e7 of their mean to float32 rounding).
template <int MMAX, bool EXACT, int V, int LO, int N>
__device__ __forceinline__ float tree_sum(const float (&u)[MMAX][V], int M, int v) {
    if constexpr (N == 1) {
        return (EXACT || LO < M) ? u[LO][v] : 0.0f;
    } else {
        return tree_sum<MMAX, EXACT, V, LO, N / 2>(u, M, v) + tree_sum<MMAX, EXACT, V, LO + N / 2, N - N / 2>(u, M, v);
    }
}

// Mean over the M rows of u, per element (float32, fixed pairwise order).
template <int MMAX, bool EXACT, int V>
__device__ inline void row_mean(const float (&u)[MMAX][V], int M, float (&mean)[V]) {
#pragma unroll
    for (int v = 0; v < V; ++v) mean[v] = tree_sum<MMAX, EXACT, V, 0, MMAX>(u, M, v) / static_cast<float>(EXACT ? MMAX : M);
}

// Adds this lane-column's contribution to S_m(u) = sum_p (u_m - mean)^2 into
// the wave's double accumulators acc[m], for a given per-element worker mean.
// Workers are reduced in chunks of at most 16 to bound register use.
template <int MMAX, bool EXACT, int V>
__device__ inline void cd_accumulate_about(const float (&u)[MMAX][V], const float (&mean)[V], int M, double *acc,
                                           int lane) {
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int C = MP < 16 ? MP : 16;
    constexpr int kShift = 6 - ilog2(C);
#pragma unroll
    for (int c = 0; c < MP / C; ++c) {
        float part[C];
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int m = c * C + j;
            float t = 0.0f;
            if (m < MMAX && (EXACT || m < M)) {
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    const float d = u[m < MMAX ? m : 0][v] - mean[v];
                    t = fmaf(d, d, t);
                }
            }
            part[j] = t;
        }
        const float tot = wave_reduce_scatter<C>(part, lane);
        const int m = c * C + (lane >> kShift);
        if ((lane & ((1 << kShift) - 1)) == 0 && m < M) acc[m] += static_cast<double>(tot);
    }
}

// S_m(u) contribution about the worker mean of u itself.
template <int MMAX, bool EXACT, int V>
__device__ inline void cd_accumulate(const float (&u)[MMAX][V], int M, double *acc, int lane) {
    float mean[V];
    row_mean<MMAX, EXACT, V>(u, M, mean);
    cd_accumulate_about<MMAX, EXACT, V>(u, mean, M, acc, lane);
}

// ------------------------------------------------------------------ mixing

// Mix kinds as template arguments; kAny reads the kind at run time.
// kStored (Mix1 only): x is read from the array a Mix1 launch stored (the
// blocking half of split execution).
constexpr int kAny = 3;
constexpr int kStored = 4;

// The tables are read through the constant address space: they are never
// written by the kernel, and this lets every (column, weight) pair arrive in
// scalar registers, shared by the wave.
typedef const __attribute__((address_space(4))) int32_t *const_table_ptr;

// The lane's V values of row `col` in its LDS column.
template <int V>
__device__ __forceinline__ void lds_row(const float *rows, int col, int tid, float (&r)[V]) {
    const float *src = rows + (static_cast<int64_t>(col) * kBlock + tid) * V;
    if constexpr (V == 4) {
        const f32x4 t = *reinterpret_cast<const f32x4 *>(src);
        r[0] = t.x; r[1] = t.y; r[2] = t.z; r[3] = t.w;
    } else if constexpr (V == 2) {
        const f32x2 t = *reinterpret_cast<const f32x2 *>(src);
        r[0] = t.x; r[1] = t.y;
    } else {
#pragma unroll
        for (int v = 0; v < V; ++v) r[v] = src[v];
    }
}

// Tables at least this wide (in kernels for more than 16 workers) are summed
// four entries at a time, each four as a small tree added to the running
// sum: one float32 chain over a dense row of W (up to 64 entries) would
// otherwise lose up to a part in 1e6 of a mixed value that is much smaller
// than its terms.  Narrower tables (the sparse graphs: rings, exponential
// and regular graphs) take one fused multiply-add per entry.
constexpr int kWideTable = 16;

// One table round applied in place, u_m <- sum_d w[d][m] * u_{col[d][m]},
// gathering through the lane's LDS column.
template <int MMAX, bool EXACT, int V>
__device__ inline void table_round_lds(const_table_ptr tab, int width, int M, float (&u)[MMAX][V], float *rows,
                                       int tid) {
    const int Mr = EXACT ? MMAX : M;
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        if (EXACT || m < M) {
            float *dst = rows + (static_cast<int64_t>(m) * kBlock + tid) * V;
            if constexpr (V == 4) {
                *reinterpret_cast<f32x4 *>(dst) = f32x4{u[m][0], u[m][1], u[m][2], u[m][3]};
            } else if constexpr (V == 2) {
                *reinterpret_cast<f32x2 *>(dst) = f32x2{u[m][0], u[m][1]};
            } else {
#pragma unroll
                for (int v = 0; v < V; ++v) dst[v] = u[m][v];
            }
        }
#pragma unroll
        for (int v = 0; v < V; ++v) u[m][v] = 0.0f;
    }
    int d = 0;
    // Kernels for up to 16 workers leave this path out: their tables are at
    // most 16 wide, short enough for one chain, and the path's presence alone
    // made the compiler schedule their narrow path 8-14% slower.
    if constexpr (MMAX > kWideTable) {
        for (; width >= kWideTable && d + 4 <= width; d += 4) {
            const_table_ptr td = tab + 2 * d * Mr;
#pragma unroll
            for (int m = 0; m < MMAX; ++m) {
                if (m % 8 == 0 && m > 0) __builtin_amdgcn_sched_barrier(0);
                if (EXACT || m < M) {
                    float r0[V], r1[V], r2[V], r3[V];
                    lds_row<V>(rows, td[2 * m], tid, r0);
                    lds_row<V>(rows, td[2 * Mr + 2 * m], tid, r1);
                    lds_row<V>(rows, td[4 * Mr + 2 * m], tid, r2);
                    lds_row<V>(rows, td[6 * Mr + 2 * m], tid, r3);
                    const float w0 = __int_as_float(td[2 * m + 1]), w1 = __int_as_float(td[2 * Mr + 2 * m + 1]);
                    const float w2 = __int_as_float(td[4 * Mr + 2 * m + 1]), w3 = __int_as_float(td[6 * Mr + 2 * m + 1]);
#pragma unroll
                    for (int v = 0; v < V; ++v) {
                        const float a = fmaf(w0, r0[v], w1 * r1[v]);
                        const float b = fmaf(w2, r2[v], w3 * r3[v]);
                        u[m][v] += a + b;
                    }
                }
            }
        }
    }
    for (; d < width; ++d) {
        const_table_ptr td = tab + 2 * d * Mr;
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            // Keep the scheduler from hoisting every row's table entry into
            // scalar registers at once.
            if (m % 16 == 0 && m > 0) __builtin_amdgcn_sched_barrier(0);
            if (EXACT || m < M) {
                const float w = __int_as_float(td[2 * m + 1]);
                float r[V];
                lds_row<V>(rows, td[2 * m], tid, r);
#pragma unroll
                for (int v = 0; v < V; ++v) u[m][v] = fmaf(w, r[v], u[m][v]);
            }
        }
    }
}

template <int MMAX, bool EXACT, int V>
__device__ __forceinline__ void table_round(const_table_ptr tab, int width, int M, float (&u)[MMAX][V], float *rows,
                                            int tid) {
    table_round_lds<MMAX, EXACT, V>(tab, width, M, u, rows, tid);
}

// Applies one Mix slot to u.  `mean` holds the worker mean of u on entry.
// A global mean leaves the result in `mean` (KIND == kGlobal) or in every row
// (KIND == kAny).  cd_acc: the wave's accumulators of the slot's first
// round-output row (nullptr: no consensus); consecutive rounds use
// consecutive rows, `cd_stride` doubles apart.  A doubly-stochastic W keeps
// the worker mean (Sec. 3), so every round's consensus row is taken about
// the input mean.
// Restores the elements whose bit is set in `keep` to the values the round
// started from, which are still in the lane's LDS column (identity outside a
// Mix2 subset).
template <int MMAX, bool EXACT, int V>
__device__ inline void keep_own(float (&u)[MMAX][V], const float *rows, int tid, int M, uint32_t keep) {
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
        if (EXACT || m < M) {
            const float *own = rows + (static_cast<int64_t>(m) * kBlock + tid) * V;
#pragma unroll
            for (int v = 0; v < V; ++v)
                if ((keep >> v) & 1u) u[m][v] = own[v];
        }
    }
}

// Consensus row of a global-mean output: every worker holds the mean, so
// S_m = sum_p (mean_p - mean_p)^2 is 0 where the mean is finite and NaN
// where it is not (IEEE: inf - inf and NaN - NaN are NaN).  Only that case
// needs work: when some lane's mean is non-finite the wave's accumulators
// of the row become NaN for every worker.
template <int V>
__device__ inline void cd_global_row(const float (&mean)[V], int M, double *acc, int lane) {
    bool bad = false;
#pragma unroll
    for (int v = 0; v < V; ++v) bad |= !__builtin_isfinite(mean[v]);
    if (__builtin_amdgcn_ballot_w64(bad)) {
        for (int m = lane; m < M; m += kWave) acc[m] = __builtin_nan("");
    }
}

// keep: bit v set = element v of this lane is outside the Mix's subset and
// passes through unchanged (0 for a Mix over every element).
template <int MMAX, bool EXACT, int V, int KIND>
__device__ inline void mix_apply(const MixDev &mx, int M, float (&u)[MMAX][V], const float (&mean)[V], float *rows,
                                 int tid, double *cd_acc, int cd_stride, int lane, uint32_t keep) {
    if constexpr (KIND == kIdentity) {
        return;
    } else if constexpr (KIND == kGlobal) {
        if (cd_acc) cd_global_row<V>(mean, M, cd_acc, lane);
        return;
    } else {
        if (KIND == kAny && mx.kind == kGlobal) {
#pragma unroll
            for (int m = 0; m < MMAX; ++m)
#pragma unroll
                for (int v = 0; v < V; ++v) u[m][v] = mean[v];
            // Every row equal (subsets need a table Mix).
            if (cd_acc) cd_global_row<V>(mean, M, cd_acc, lane);
            return;
        }
        if (KIND == kAny && mx.kind != kTable) return;
        const int Mr = EXACT ? MMAX : M;
        for (int k = 0; k < mx.rounds; ++k) {
            const_table_ptr tab = (const_table_ptr)(mx.table) + 2 * static_cast<int64_t>(k) * mx.width * Mr;
            table_round<MMAX, EXACT, V>(tab, mx.width, M, u, rows, tid);
            if (keep) keep_own<MMAX, EXACT, V>(u, rows, tid, M, keep);
            if (cd_acc) cd_accumulate_about<MMAX, EXACT, V>(u, mean, M, cd_acc + k * cd_stride, lane);
        }
    }
}

// ------------------------------------------------------------ step kernel

// Waves per SIMD the register allocator is asked to leave room for: enough
// waves in flight to keep HBM busy while others mix.
constexpr int waves_per_simd_target(int mmax) { return mmax <= 4 ? 4 : (mmax <= 8 ? FGD_WAVES_M8 : 1); }

// Per-tile state shared by the full-tile and ragged-tile paths.
struct TileCtx {
    float *rows;      // LDS rows (CSR mixes gathered through LDS)
    double *cd_acc;   // this wave's consensus accumulators, or nullptr
    int M, tid, lane, n1, n2;
};

// One tile of kBlock * V parameters.  FULL: every lane's vector lies below P
// (uniform; all tiles but the last), so no lane needs bounds logic.
// MS: Mix1 is also applied to the momentum rows before the update.
// keep: the lane's elements outside a Mix2 subset (bit v for element v);
// they pass through Mix2 unchanged.
template <int MMAX, bool EXACT, int V, class PIO, int K1, int K2, bool MS, bool FULL>
__device__ __forceinline__ void step_tile(const StepParams &a, const TileCtx &c, int64_t tb, uint32_t lo,
                                          uint32_t keep) {
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int kCdStride = kWavesPerBlock * MP;  // doubles between consensus rows
    constexpr int kE = PIO::kElem;
    const int M = c.M;
    int nv = V;
    if constexpr (!FULL) {
        const int64_t rem = a.P - tb - lo;
        nv = rem >= V ? V : (rem > 0 ? static_cast<int>(rem) : 0);
    }
    const uint32_t off_p = lo * kE, off_v = lo * 4;  // lane byte offsets in parameter / momentum rows

    // Phase A: every row's loads are issued before the first use.  On the
    // ragged tile a lane whose vector straddles P still loads the whole
    // vector (the row's ld span covers it) and zeroes the elements at or
    // beyond P; lanes entirely beyond P load nothing.
    float u1[MMAX][V];  // theta_prev, then Mix1 output (unless global)
    float u2[MMAX][V];  // theta_local, then g0, then Mix2 output (unless global)
    if (FULL || nv > 0) {
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            if (EXACT || m < M) {
                PIO::load(row_rsrc(a.theta_prev, m * a.ld + tb, kE), off_p, u1[m]);
                PIO::load(row_rsrc(a.theta_local, m * a.ld + tb, kE), off_p, u2[m]);
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
            if ((EXACT || m < M) && (FULL || v < nv)) u2[m][v] = u1[m][v] - u2[m][v];
            else { u1[m][v] = 0.0f; u2[m][v] = 0.0f; }
        }
    }

    // Worker means of the mix inputs: the global-mean outputs themselves and
    // the centres of every consensus row of the slot.
    float xbar[V], gbar[V];
    row_mean<MMAX, EXACT, V>(u2, M, gbar);
    if (c.cd_acc) cd_accumulate_about<MMAX, EXACT, V>(u2, gbar, M, c.cd_acc, c.lane);
    if constexpr (K1 != kStored) {
        row_mean<MMAX, EXACT, V>(u1, M, xbar);
        if (c.cd_acc) cd_accumulate_about<MMAX, EXACT, V>(u1, xbar, M, c.cd_acc + (c.n2 + 1) * kCdStride, c.lane);
        mix_apply<MMAX, EXACT, V, K1>(a.mix1, M, u1, xbar, c.rows, c.tid,
                                      c.cd_acc ? c.cd_acc + (c.n2 + 2) * kCdStride : nullptr, kCdStride, c.lane, 0u);
    }
    // A tile wholly outside a Mix2 subset runs the rounds too, with every
    // element kept: one code path keeps the register budget of the kernel.
    mix_apply<MMAX, EXACT, V, K2>(a.mix2, M, u2, gbar, c.rows, c.tid, c.cd_acc ? c.cd_acc + 1 * kCdStride : nullptr,
                                  kCdStride, c.lane, keep);

    // Phase D: the outer optimizer and the stores.  The stored theta'
    // replaces the row's dead input registers.
    constexpr bool kStoreInU2 = K2 != kGlobal;
    constexpr bool kStoreInU1 = !kStoreInU2 && K1 != kGlobal;
    constexpr int kSep = (!kStoreInU2 && !kStoreInU1) ? MMAX : 1;
    float sep[kSep][V];
    const float mu = a.mu, lr = a.lr;
    const bool nesterov = a.nesterov != 0;

    // v' = mu v + g ; theta' = x - lr (g + mu v') or x - lr v'; stores row m.
    // xs: the row's stored x (kStored only).
    auto finish_row = [&](int m, float (&vr)[V], const float (&xs)[V]) {
        float stored[V];
        if ((EXACT || m < M) && (FULL || nv > 0)) {
            float t[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const float g = K2 == kGlobal ? gbar[e] : u2[m][e];
                const float x = K1 == kStored ? xs[e] : (K1 == kGlobal ? xbar[e] : u1[m][e]);
                vr[e] = fmaf(mu, vr[e], g);
                const float step = nesterov ? fmaf(mu, vr[e], g) : vr[e];
                t[e] = fmaf(-lr, step, x);
            }
            const rsrc_t rv = row_rsrc(a.mom_out, m * a.ld + tb, 4);
            const rsrc_t rp = row_rsrc(a.theta_out, m * a.ld + tb, kE);
            if (FULL || nv == V) {
                F32Io<V>::store(rv, off_v, vr);
                PIO::store(rp, off_p, t, stored);
            } else {
                F32Io<V>::store_part(rv, off_v, nv, vr);
                PIO::store_part(rp, off_p, nv, t, stored);
            }
            if constexpr (K1 == kStored) {
                if (a.local_out) {  // theta' (already in storage precision) as the next inner start
                    float again[V];
                    const rsrc_t rl = row_rsrc(a.local_out, m * a.ld + tb, kE);
                    if (FULL || nv == V) PIO::store(rl, off_p, stored, again);
                    else PIO::store_part(rl, off_p, nv, stored, again);
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < V; ++e) stored[e] = 0.0f;
        }
#pragma unroll
        for (int e = 0; e < V; ++e) {
            if constexpr (kStoreInU2) u2[m][e] = stored[e];
            else if constexpr (kStoreInU1) u1[m][e] = stored[e];
            else sep[kSep == 1 ? 0 : m][e] = stored[e];
        }
    };

    if constexpr (MS) {
        // Optimizer state mixed by Mix1: every momentum row first.
        float vm[MMAX][V];
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            if ((EXACT || m < M) && (FULL || nv > 0)) F32Io<V>::load(row_rsrc(a.mom, m * a.ld + tb, 4), off_v, vm[m]);
            else {
#pragma unroll
                for (int e = 0; e < V; ++e) vm[m][e] = 0.0f;
            }
        }
        float vbar[V];
        row_mean<MMAX, EXACT, V>(vm, M, vbar);
        if constexpr (K1 == kGlobal) {
#pragma unroll
            for (int m = 0; m < MMAX; ++m)
#pragma unroll
                for (int e = 0; e < V; ++e) vm[m][e] = vbar[e];
        } else {
            mix_apply<MMAX, EXACT, V, K1>(a.mix1, M, vm, vbar, c.rows, c.tid, nullptr, 0, c.lane, 0u);
        }
#pragma unroll
        for (int m = 0; m < MMAX; ++m) finish_row(m, vm[m], vm[m]);
    } else {
        // A group of rows at a time bounds the momentum (and stored x) registers.
        constexpr int G = (MMAX * V <= 32) ? MMAX : (32 / V > 0 ? 32 / V : 1);
        constexpr int GX = K1 == kStored ? G : 1;
#pragma unroll
        for (int m0 = 0; m0 < MMAX; m0 += G) {
            float vm[G][V];
            float xm[GX][V];
            if (FULL || nv > 0) {
#pragma unroll
                for (int j = 0; j < G; ++j) {
                    const int m = m0 + j;
                    if (m < MMAX && (EXACT || m < M)) {
                        F32Io<V>::load(row_rsrc(a.mom, m * a.ld + tb, 4), off_v, vm[j]);
                        if constexpr (K1 == kStored) PIO::load(row_rsrc(a.x, m * a.ld + tb, kE), off_p, xm[j]);
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < G; ++j)
                if (m0 + j < MMAX) finish_row(m0 + j, vm[j], xm[GX == 1 ? 0 : j]);
        }
    }
    if (c.cd_acc) {
        // The stored theta' row follows the Mix2 rows, then (fused step) the Mix1 rows.
        double *acc = c.cd_acc + (K1 == kStored ? c.n2 + 1 : c.n2 + c.n1 + 2) * kCdStride;
        if constexpr (kStoreInU2) cd_accumulate<MMAX, EXACT, V>(u2, M, acc, c.lane);
        else if constexpr (kStoreInU1) cd_accumulate<MMAX, EXACT, V>(u1, M, acc, c.lane);
        else cd_accumulate<MMAX, EXACT, V>(sep, M, acc, c.lane);
    }
}

// Parameter segments of a Mix2 subset, read as scalar loads (never written).
typedef const __attribute__((address_space(4))) int64_t *const_seg_ptr;

// Step-kernel variant flags.
constexpr int kMixState = 1;  // Mix1 also mixes the optimizer state
constexpr int kSubset = 2;    // Mix2 may be restricted to a parameter subset

// K1, K2: compile-time kinds of Mix1 and Mix2 (kAny = decided at run time).
// FLAGS: kMixState | kSubset.
template <int MMAX, bool EXACT, int V, class PIO, int K1, int K2, int FLAGS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(waves_per_simd_target(MMAX))))
void outer_step_kernel(StepParams a) {
    constexpr bool MS = (FLAGS & kMixState) != 0;
    constexpr bool SUB = (FLAGS & kSubset) != 0 && (K2 == kTable || K2 == kAny);
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int kCdStride = kWavesPerBlock * MP;
    constexpr int64_t kTile = static_cast<int64_t>(kBlock) * V;
    TileCtx c;
    c.M = EXACT ? MMAX : a.M;
    c.tid = threadIdx.x;
    c.lane = c.tid & (kWave - 1);
    const int wave = c.tid / kWave;
    c.rows = reinterpret_cast<float *>(smem);
    const int64_t rows_bytes = static_cast<int64_t>(a.lds_rows) * kBlock * V * 4;
    c.cd_acc = a.cd_partials ? reinterpret_cast<double *>(smem + rows_bytes) + wave * MP : nullptr;
    c.n2 = a.mix2.kind == kTable ? a.mix2.rounds : (a.mix2.kind == kGlobal ? 1 : 0);
    c.n1 = a.mix1.kind == kTable ? a.mix1.rounds : (a.mix1.kind == kGlobal ? 1 : 0);

    if (a.lds_rows > c.M) {
        float *z = c.rows + (static_cast<int64_t>(c.M) * kBlock + c.tid) * V;
#pragma unroll
        for (int v = 0; v < V; ++v) z[v] = 0.0f;
    }
    if (c.cd_acc) {
        for (int i = c.lane; i < a.n_cd * MP; i += kWave) c.cd_acc[(i / MP) * kCdStride + i % MP] = 0.0;
    }

    const uint32_t lo = static_cast<uint32_t>(c.tid) * V;  // lane offset inside a tile, in elements
    const const_seg_ptr seg = (const_seg_ptr)(a.seg);
    int s = 0;  // first segment that ends after the tile start; tiles ascend, so it only moves forward
    // Bounds of segment s, kept in (scalar) registers: reloaded only when s
    // moves, so a tile's classification costs no memory access.
    int64_t s_begin = 0, s_end = 0;
    if constexpr (SUB) {
        if (a.n_seg > 0) {
            s_begin = seg[0];
            s_end = seg[1];
        }
    }
    for (int64_t tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int64_t tb = tile * kTile;  // first parameter of the tile (uniform)
        uint32_t keep = 0;                // elements of this lane outside the Mix2 subset
        if constexpr (SUB) {
            if (a.n_seg > 0) {
                const int64_t te = tb + kTile < a.P ? tb + kTile : a.P;
                while (s < a.n_seg && s_end <= tb) {
                    ++s;
                    if (s < a.n_seg) {
                        s_begin = seg[2 * s];
                        s_end = seg[2 * s + 1];
                    }
                }
                if (s == a.n_seg || s_begin >= te) {
                    keep = (1u << V) - 1u;  // wholly outside
                } else if (s_begin <= tb && s_end >= te) {
                    keep = 0u;  // wholly inside
                } else {
                    keep = (1u << V) - 1u;
                    for (int i = s; i < a.n_seg && seg[2 * i] < te; ++i) {
                        const int64_t b = seg[2 * i], e = seg[2 * i + 1];
#pragma unroll
                        for (int v = 0; v < V; ++v) {
                            const int64_t p = tb + lo + v;
                            if (p >= b && p < e) keep &= ~(1u << v);
                        }
                    }
                }
            }
        }
        if (tb + kTile <= a.P) step_tile<MMAX, EXACT, V, PIO, K1, K2, MS, true>(a, c, tb, lo, keep);
        else step_tile<MMAX, EXACT, V, PIO, K1, K2, MS, false>(a, c, tb, lo, keep);
    }

    if (c.cd_acc) {
        __syncthreads();
        const double *base = reinterpret_cast<const double *>(smem + rows_bytes);
        for (int i = c.tid; i < a.n_cd * c.M; i += kBlock) {
            const int r = i / c.M, m = i % c.M;
            double s = 0.0;
#pragma unroll
            for (int w = 0; w < kWavesPerBlock; ++w) s += base[r * kCdStride + w * MP + m];
            a.cd_partials[(static_cast<int64_t>(blockIdx.x) * a.n_cd + r) * c.M + m] = s;
        }
    }
}

// ------------------------------------------------ split execution: Mix1 half

// x = Mix1(theta_prev) stored in the parameter type (Appendix A, Algorithm
// 1: the non-blocking mix launched at the start of a round), with consensus
// rows x^0..x^K1; MS: the momentum is replaced by Mix1 of itself.
template <int MMAX, bool EXACT, int V, class PIO, int K1, bool MS, bool FULL>
__device__ __forceinline__ void mix1_tile(const StepParams &a, const TileCtx &c, int64_t tb, uint32_t lo) {
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int kCdStride = kWavesPerBlock * MP;
    constexpr int kE = PIO::kElem;
    const int M = c.M;
    int nv = V;
    if constexpr (!FULL) {
        const int64_t rem = a.P - tb - lo;
        nv = rem >= V ? V : (rem > 0 ? static_cast<int>(rem) : 0);
    }
    const uint32_t off_p = lo * kE, off_v = lo * 4;
    float u[MMAX][V];
    if (FULL || nv > 0) {
#pragma unroll
        for (int m = 0; m < MMAX; ++m)
            if (EXACT || m < M) PIO::load(row_rsrc(a.theta_prev, m * a.ld + tb, kE), off_p, u[m]);
    }
#pragma unroll
    for (int m = 0; m < MMAX; ++m)
#pragma unroll
        for (int v = 0; v < V; ++v)
            if (!((EXACT || m < M) && (FULL || v < nv))) u[m][v] = 0.0f;
    float xbar[V];
    row_mean<MMAX, EXACT, V>(u, M, xbar);
    if (c.cd_acc) cd_accumulate_about<MMAX, EXACT, V>(u, xbar, M, c.cd_acc, c.lane);
    mix_apply<MMAX, EXACT, V, K1>(a.mix1, M, u, xbar, c.rows, c.tid, c.cd_acc ? c.cd_acc + kCdStride : nullptr,
                                  kCdStride, c.lane, 0u);
    if (FULL || nv > 0) {
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            if (EXACT || m < M) {
                float stored[V];
                const rsrc_t rx = row_rsrc(a.x_out, m * a.ld + tb, kE);
                if (FULL || nv == V) PIO::store(rx, off_p, K1 == kGlobal ? xbar : u[m], stored);
                else PIO::store_part(rx, off_p, nv, K1 == kGlobal ? xbar : u[m], stored);
            }
        }
    }
    if constexpr (MS) {
        float vm[MMAX][V];
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            if ((EXACT || m < M) && (FULL || nv > 0)) F32Io<V>::load(row_rsrc(a.mom, m * a.ld + tb, 4), off_v, vm[m]);
            else {
#pragma unroll
                for (int e = 0; e < V; ++e) vm[m][e] = 0.0f;
            }
        }
        float vbar[V];
        row_mean<MMAX, EXACT, V>(vm, M, vbar);
        mix_apply<MMAX, EXACT, V, K1>(a.mix1, M, vm, vbar, c.rows, c.tid, nullptr, 0, c.lane, 0u);
        if (FULL || nv > 0) {
#pragma unroll
            for (int m = 0; m < MMAX; ++m) {
                if (EXACT || m < M) {
                    const rsrc_t rv = row_rsrc(a.mom_out, m * a.ld + tb, 4);
                    if (FULL || nv == V) F32Io<V>::store(rv, off_v, K1 == kGlobal ? vbar : vm[m]);
                    else F32Io<V>::store_part(rv, off_v, nv, K1 == kGlobal ? vbar : vm[m]);
                }
            }
        }
    }
}

// The Mix1 half is meant to run beside other kernels (the inner loop), where
// a grid of resident blocks can be placed unevenly: blocks dispatched while
// another kernel holds most CUs pile up on the few that are free.  So blocks
// take fixed chunks of tiles from a counter instead of a fixed stride, and
// each chunk leaves its own consensus partials, summed in chunk order: the
// work balances itself and the result does not depend on which block took
// which chunk.
template <int MMAX, bool EXACT, int V, class PIO, int K1, bool MS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(waves_per_simd_target(MMAX))))
void mix1_kernel(StepParams a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    __shared__ int64_t s_chunk;
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int kCdStride = kWavesPerBlock * MP;
    constexpr int64_t kTile = static_cast<int64_t>(kBlock) * V;
    TileCtx c;
    c.M = EXACT ? MMAX : a.M;
    c.tid = threadIdx.x;
    c.lane = c.tid & (kWave - 1);
    const int wave = c.tid / kWave;
    c.rows = reinterpret_cast<float *>(smem);
    const int64_t rows_bytes = static_cast<int64_t>(a.lds_rows) * kBlock * V * 4;
    c.cd_acc = a.cd_partials ? reinterpret_cast<double *>(smem + rows_bytes) + wave * MP : nullptr;
    c.n1 = c.n2 = 0;
    if (a.lds_rows > c.M) {
        float *z = c.rows + (static_cast<int64_t>(c.M) * kBlock + c.tid) * V;
#pragma unroll
        for (int v = 0; v < V; ++v) z[v] = 0.0f;
    }
    const uint32_t lo = static_cast<uint32_t>(c.tid) * V;
    for (;;) {
        if (c.tid == 0) s_chunk = atomicAdd(a.chunk_counter, 1);
        __syncthreads();
        const int64_t chunk = s_chunk;
        __syncthreads();  // every thread has its copy before thread 0 takes the next chunk
        if (chunk >= a.nchunks) break;
        if (c.cd_acc) {
            for (int i = c.lane; i < a.n_cd * MP; i += kWave) c.cd_acc[(i / MP) * kCdStride + i % MP] = 0.0;
        }
        const int64_t t0 = chunk * a.chunk_tiles;
        const int64_t t1 = t0 + a.chunk_tiles < a.ntiles ? t0 + a.chunk_tiles : a.ntiles;
        for (int64_t tile = t0; tile < t1; ++tile) {
            const int64_t tb = tile * kTile;
            if (tb + kTile <= a.P) mix1_tile<MMAX, EXACT, V, PIO, K1, MS, true>(a, c, tb, lo);
            else mix1_tile<MMAX, EXACT, V, PIO, K1, MS, false>(a, c, tb, lo);
        }
        if (c.cd_acc) {
            __syncthreads();
            const double *base = reinterpret_cast<const double *>(smem + rows_bytes);
            for (int i = c.tid; i < a.n_cd * c.M; i += kBlock) {
                const int r = i / c.M, m = i % c.M;
                double s = 0.0;
#pragma unroll
                for (int w = 0; w < kWavesPerBlock; ++w) s += base[r * kCdStride + w * MP + m];
                a.cd_partials[(chunk * a.n_cd + r) * c.M + m] = s;
            }
            __syncthreads();  // partials read before the accumulators are cleared for the next chunk
        }
    }
}

// Sets the chunk counter of a Mix1 launch to 0 (one thread; stream-ordered
// before the launch).
__global__ void counter_reset_kernel(int *counter);

// ------------------------------------------------- standalone consensus

template <int MMAX, bool EXACT, int V, class PIO>
__global__ __launch_bounds__(kBlock) void consensus_kernel(ConsensusParams a) {
    constexpr int MP = pow2_at_least(MMAX);
    constexpr int kE = PIO::kElem;
    __shared__ double acc[kWavesPerBlock * MP];
    const int M = EXACT ? MMAX : a.M;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    for (int i = tid; i < kWavesPerBlock * MP; i += kBlock) acc[i] = 0.0;
    __syncthreads();
    const uint32_t lo = static_cast<uint32_t>(tid) * V;
    for (int64_t tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int64_t tb = tile * (kBlock * V);
        const int64_t rem = a.P - tb - lo;
        const int nv = rem >= V ? V : (rem > 0 ? static_cast<int>(rem) : 0);
        float u[MMAX][V];
        if (nv > 0) {
#pragma unroll
            for (int m = 0; m < MMAX; ++m)
                if (EXACT || m < M) PIO::load(row_rsrc(a.x, m * a.ld + tb, kE), lo * kE, u[m]);
        }
#pragma unroll
        for (int m = 0; m < MMAX; ++m)
#pragma unroll
            for (int v = 0; v < V; ++v)
                if (!((EXACT || m < M) && v < nv)) u[m][v] = 0.0f;
        cd_accumulate<MMAX, EXACT, V>(u, M, acc + wave * MP, lane);
    }
    __syncthreads();
    for (int m = tid; m < M; m += kBlock) {
        double s = 0.0;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) s += acc[w * MP + m];
        a.partials[static_cast<int64_t>(blockIdx.x) * M + m] = s;
    }
}

// out[i] = sum over blocks b of partials[b][i], i < n, in a fixed order (one
// block per entry; launch with n blocks of 256 threads).
__global__ void finalize_kernel(const double *partials, int nblocks, int n, double *out);

// Plain 16-byte streaming copy.
__global__ void copy_kernel(const u32x4 *src, u32x4 *dst, int64_t n);

// ----------------------------------------------- access-pattern reference

// Raw 2-, 4-, 8- or 16-byte lane accesses with the step's cache policy (a
// 2-byte value travels in the low half of its word).
template <int N>
struct RawIo {
    static constexpr int kW = N >= 4 ? N / 4 : 1;  // words per lane
    __device__ static void load(rsrc_t r, uint32_t off, uint32_t (&o)[kW]) {
        if constexpr (N == 16) {
            const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kLoadPolicy);
            o[0] = t[0]; o[1] = t[1]; o[2] = t[2]; o[3] = t[3];
        } else if constexpr (N == 8) {
            const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kLoadPolicy);
            o[0] = t[0]; o[1] = t[1];
        } else if constexpr (N == 4) {
            o[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kLoadPolicy);
        } else {
            o[0] = __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kLoadPolicy);
        }
    }
    __device__ static void store(rsrc_t r, uint32_t off, const uint32_t (&i)[kW]) {
        if constexpr (N == 16) {
            const u32x4 t = {i[0], i[1], i[2], i[3]};
            __builtin_amdgcn_raw_buffer_store_b128(t, r, off, 0, kStorePolicy);
        } else if constexpr (N == 8) {
            const u32x2 t = {i[0], i[1]};
            __builtin_amdgcn_raw_buffer_store_b64(t, r, off, 0, kStorePolicy);
        } else if constexpr (N == 4) {
            __builtin_amdgcn_raw_buffer_store_b32(i[0], r, off, 0, kStorePolicy);
        } else {
            __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(i[0] & 0xFFFFu), r, off, 0, kStorePolicy);
        }
    }
};

// The fused step's memory traffic without its arithmetic: the tiles, lane
// vectors, cache policy and launch shape of outer_step_kernel, every
// theta_prev and theta_local row of a tile loaded before first use, then row
// by row the momentum loaded and theta_prev and the momentum stored.  The
// stored words are the loaded ones OR (theta_local word AND mask) with mask =
// 0 passed at run time, so the arrays keep their exact bits while no load can
// be dropped.  A lane whose vector straddles P loads it and stores nothing.
// Its rate is the practical ceiling of the step's read/write mix.
struct PatternParams {
    const void *theta_prev;
    void *theta_out;
    const void *theta_local;
    const float *mom;
    float *mom_out;
    int64_t P, ld, ntiles;
    uint32_t mask;
};

template <int MMAX, int V, int kE>
__global__ __launch_bounds__(kBlock) void pattern_kernel(PatternParams a) {
    constexpr int NP = V * kE, NV = V * 4;  // bytes per lane vector: parameters, momentum
    constexpr int64_t kTile = static_cast<int64_t>(kBlock) * V;
    const uint32_t lo = static_cast<uint32_t>(threadIdx.x) * V;
    for (int64_t tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int64_t tb = tile * kTile;
        const int64_t rem = a.P - tb - lo;
        if (rem <= 0) continue;
        const bool whole = rem >= V;
        constexpr int WP = RawIo<NP>::kW, WV = RawIo<NV>::kW;
        uint32_t u1[MMAX][WP], u2[MMAX][WP];
#pragma unroll
        for (int m = 0; m < MMAX; ++m) {
            RawIo<NP>::load(row_rsrc(a.theta_prev, m * a.ld + tb, kE), lo * kE, u1[m]);
            RawIo<NP>::load(row_rsrc(a.theta_local, m * a.ld + tb, kE), lo * kE, u2[m]);
        }
        // Momentum rows in the step's groups (all of a group's loads first).
        constexpr int G = (MMAX * V <= 32) ? MMAX : (32 / V > 0 ? 32 / V : 1);
#pragma unroll
        for (int m0 = 0; m0 < MMAX; m0 += G) {
            uint32_t vm[G][WV];
#pragma unroll
            for (int j = 0; j < G; ++j)
                RawIo<NV>::load(row_rsrc(a.mom, (m0 + j) * a.ld + tb, 4), lo * 4, vm[j]);
#pragma unroll
            for (int j = 0; j < G; ++j) {
                const int m = m0 + j;
                uint32_t t[WP];
#pragma unroll
                for (int k = 0; k < WP; ++k) t[k] = u1[m][k] | (u2[m][k] & a.mask);
#pragma unroll
                for (int k = 0; k < WV; ++k) vm[j][k] |= u2[m][k % WP] & a.mask;
                if (whole) {
                    RawIo<NV>::store(row_rsrc(a.mom_out, m * a.ld + tb, 4), lo * 4, vm[j]);
                    RawIo<NP>::store(row_rsrc(a.theta_out, m * a.ld + tb, kE), lo * kE, t);
                }
            }
        }
    }
}

// ------------------------------------------------------------ dispatch

// Launch description of one (M, dtype) instantiation.
struct KernelSet {
    const void *step;       // outer_step_kernel instantiation for the requested kinds
    const void *consensus;  // consensus_kernel instantiation
    int v;                  // elements per lane per row
    int mmax;               // compile-time worker bound
    int step_blocks_per_cu; // cap on resident step blocks per compute unit
};

#ifndef FGD_STEP_BLOCKS_PER_CU_SMALL
#define FGD_STEP_BLOCKS_PER_CU_SMALL 1
#endif
// Step blocks per compute unit.  Up to 16 workers a block streams 3M rows of
// 16-byte (8-byte bf16) accesses per tile, all issued before first use, which
// keeps enough bytes in flight with one block per CU; more resident blocks
// only add DRAM contention (measured 5-7% slower with 4 at 8 workers).  With
// 32 or 64 workers a lane holds one or two parameters and the rows are
// gathered through LDS, so a second block is needed to cover that latency.
constexpr int step_blocks_per_cu(int mmax) { return mmax <= 16 ? FGD_STEP_BLOCKS_PER_CU_SMALL : 8; }

// Kernel set of one instantiation; the step kernel is specialised on the
// (Mix1, Mix2) kinds of the paper's configurations (Appendix A table:
// GlobalM1LocalM2, LocalM1M2, GlobalM1, DiLoCo) when M is exact.  `subset`:
// a Mix2 subset is set; only GlobalM1LocalM2 has a specialisation for it
// (the paper's subset configuration), the rest run on the run-time-kind
// kernel, which always handles subsets.
template <template <int> class PIOT, int MMAX, bool EXACT, int V>
KernelSet make_kernel_set(int k1, int k2, bool subset) {
    using P = PIOT<V>;
    KernelSet ks;
    ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kAny, kAny, kSubset>);
    if constexpr (EXACT) {
        if (subset) {
            if (k1 == kGlobal && k2 == kTable)
                ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kTable, kSubset>);
        } else if (k1 == kGlobal && k2 == kTable) {
            ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kTable, 0>);
        } else if (k1 == kTable && k2 == kTable) {
            ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kTable, kTable, 0>);
        } else if (k1 == kGlobal && k2 == kIdentity) {
            ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kIdentity, 0>);
        } else if (k1 == kIdentity && k2 == kGlobal) {
            ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kIdentity, kGlobal, 0>);
        }
    }
    ks.consensus = reinterpret_cast<const void *>(&consensus_kernel<MMAX, EXACT, V, P>);
    ks.v = V;
    ks.mmax = MMAX;
    ks.step_blocks_per_cu = step_blocks_per_cu(MMAX);
    return ks;
}

// The same with the optimizer state mixed by Mix1 (Appendix B: GlobalM1S,
// GlobalM1SLocalM2 and GlobalM1SLocalM2-subset are specialised when M is
// exact).
template <template <int> class PIOT, int MMAX, bool EXACT, int V>
KernelSet make_kernel_set_ms(int k1, int k2, bool subset) {
    using P = PIOT<V>;
    constexpr int MSF = kMixState;
    KernelSet ks;
    ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kAny, kAny, MSF | kSubset>);
    if constexpr (EXACT) {
        if (k1 == kGlobal && k2 == kTable)
            ks.step = subset ? reinterpret_cast<const void *>(
                                   &outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kTable, MSF | kSubset>)
                             : reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kTable, MSF>);
        else if (k1 == kGlobal && k2 == kIdentity && !subset)
            ks.step = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kGlobal, kIdentity, MSF>);
    }
    ks.consensus = reinterpret_cast<const void *>(&consensus_kernel<MMAX, EXACT, V, P>);
    ks.v = V;
    ks.mmax = MMAX;
    // With both the state mix and a subset the kernel's per-tile work no
    // longer hides behind one block's loads: at 8 workers x 1.1e9 bf16 it
    // took 22.9 ms with one block per CU and 21.6 ms with two (the other
    // variants are faster with one).
    ks.step_blocks_per_cu = (subset && MMAX <= 16) ? 2 : step_blocks_per_cu(MMAX);
    return ks;
}

// Split-execution kernels of one instantiation: the Mix1 half (global mean
// specialised when M is exact, run-time kinds otherwise) and the blocking
// half (CSR Mix2 specialised when M is exact, with and without a subset).
struct SplitSet {
    const void *mix1;
    const void *blocking;
    int v;
    int mmax;
    int blocks_per_cu;
};

template <template <int> class PIOT, int MMAX, bool EXACT, int V>
SplitSet make_split_set(int k1, int k2, bool subset, bool mix_state) {
    using P = PIOT<V>;
    SplitSet ks;
    ks.mix1 = mix_state ? reinterpret_cast<const void *>(&mix1_kernel<MMAX, EXACT, V, P, kAny, true>)
                        : reinterpret_cast<const void *>(&mix1_kernel<MMAX, EXACT, V, P, kAny, false>);
    ks.blocking = reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kStored, kAny, kSubset>);
    if constexpr (EXACT) {
        if (k1 == kGlobal)
            ks.mix1 = mix_state ? reinterpret_cast<const void *>(&mix1_kernel<MMAX, EXACT, V, P, kGlobal, true>)
                                : reinterpret_cast<const void *>(&mix1_kernel<MMAX, EXACT, V, P, kGlobal, false>);
        if (k2 == kTable)
            ks.blocking = subset ? reinterpret_cast<const void *>(
                                       &outer_step_kernel<MMAX, EXACT, V, P, kStored, kTable, kSubset>)
                                 : reinterpret_cast<const void *>(&outer_step_kernel<MMAX, EXACT, V, P, kStored, kTable, 0>);
    }
    ks.v = V;
    ks.mmax = MMAX;
    ks.blocks_per_cu = step_blocks_per_cu(MMAX);
    return ks;
}

// Elements per lane per row: 16-byte float32 accesses up to 8 workers; bf16
// parameters use 8-byte accesses (4 elements) so that momentum still moves in
// 16-byte accesses and the register and LDS footprint per lane stays small.
constexpr int lanes_v_f32(int mmax) { return mmax <= 8 ? 4 : (mmax == 16 ? FGD_V_F32_M16 : (mmax == 32 ? 2 : 1)); }
constexpr int lanes_v_bf16(int mmax) {
    return mmax <= 8 ? FGD_V_BF16_M8 : (mmax == 16 ? 4 : (mmax == 32 ? 2 : 1));
}

// Calls F::get<MMAX, EXACT>(args...) for the instantiation that serves M
// workers: exact for M in {1, 2, 4, 8, 16, 32, 64}, else the next power of
// two with M read at run time.
template <class F, class Out, class... A>
bool select_workers(int M, Out *out, A... args) {
    if (M < 1 || M > 64) return false;
    if (M == 1) *out = F::template get<1, true>(args...);
    else if (M == 2) *out = F::template get<2, true>(args...);
    else if (M == 3) *out = F::template get<4, false>(args...);
    else if (M == 4) *out = F::template get<4, true>(args...);
    else if (M < 8) *out = F::template get<8, false>(args...);
    else if (M == 8) *out = F::template get<8, true>(args...);
    else if (M < 16) *out = F::template get<16, false>(args...);
    else if (M == 16) *out = F::template get<16, true>(args...);
    else if (M < 32) *out = F::template get<32, false>(args...);
    else if (M == 32) *out = F::template get<32, true>(args...);
    else if (M < 64) *out = F::template get<64, false>(args...);
    else *out = F::template get<64, true>(args...);
    return true;
}

// Defined per storage type.  k1, k2: Mix kinds (kIdentity, kGlobal, kTable);
// subset: a Mix2 subset is set.  A specialised step kernel is returned when
// one exists, else the one that reads the kinds at run time.  Returns false
// if M is outside [1, 64].
bool kernels_f32(int M, int k1, int k2, bool subset, KernelSet *out);
bool kernels_bf16(int M, int k1, int k2, bool subset, KernelSet *out);
// Step kernels that also mix the optimizer state with Mix1.
bool kernels_f32_ms(int M, int k1, int k2, bool subset, KernelSet *out);
bool kernels_bf16_ms(int M, int k1, int k2, bool subset, KernelSet *out);
// Split-execution kernels.
bool split_kernels_f32(int M, int k1, int k2, bool subset, bool mix_state, SplitSet *out);
bool split_kernels_bf16(int M, int k1, int k2, bool subset, bool mix_state, SplitSet *out);
// The access-pattern reference for exact M in {1, 2, 4, 8, 16, 32, 64}: the
// pattern_kernel instance, its lane vector and the step's blocks per CU.
bool pattern_kernel_for(int M, bool bf16, const void **kernel, int *v, int *blocks_per_cu);

}  // namespace fgd
