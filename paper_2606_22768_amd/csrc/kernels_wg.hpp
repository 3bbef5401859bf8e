// kernels_wg.hpp -- the fused outer step for 64 workers, worker-group layout.
//
// Same step as outer_step_kernel (Sec. 4.1 factored formulation; Appendix
// A, Algorithm 1, outer step; Appendix B Nesterov form; Sec. 4.4 and
// Appendix D.1 consensus), laid out for sparse mixing over many workers.
// outer_step_kernel gives each lane one parameter of all 64 workers: every
// table gather then costs an address computation and a 4-byte LDS read per
// value, and every consensus row a reduce-scatter of 64 values across the
// whole wave.  Here a lane holds 16 workers x 4 consecutive parameters:
//
//   lane = 16 * wg + pg        wg = lane bits 4-5: worker group 0..3
//                              pg = lane bits 0-3: parameter group 0..15
//   register row j (0..15) of a lane holds worker m = 4 j + wg,
//   parameters tb + 64 wave + 4 pg + (0..3)
//
// so a wave covers 64 parameters of all 64 workers, a block (4 waves) 256.
//
//   loads    one 16-byte (bf16: 8-byte) access per row and array: the four
//            groups of 16 lanes read four worker rows, 256 contiguous bytes
//            each (per-lane row offsets wg * ld stay below 2^32 bytes)
//   means    worker means of the mix inputs: a tree over the lane's 16
//            workers, then a sum over the four groups (lane swaps across
//            lane bits 5 and 4), identical in every lane of a parameter
//   mixing   a CSR round writes the rows to the wave's LDS region [64][64
//            parameters] and gathers 16 bytes (4 parameters) per table
//            entry; the entries of the four groups differ, so the tables
//            are staged in LDS as [round][entry][j][wg] of (LDS row offset,
//            weight) and read per lane
//   CD       S_m contributions: squared deviations summed over the lane's 4
//            parameters, then reduce-scattered over the 16 parameter groups
//            (DPP inside each 16-lane row), so each lane ends with one
//            worker's sum, added to a double register accumulator
//
// Only sparse tables qualify (fewer than 16 entries per row, and the staged
// tables must fit in LDS beside the rows); denser W, Mix2 subsets and state
// mixing run on outer_step_kernel.
#pragma once

#include "kernels.hpp"

namespace fgd {

constexpr int kWgWorkers = 64;
constexpr int kWgGroups = 4;                          // worker groups (lane bits 4-5)
constexpr int kWgJ = kWgWorkers / kWgGroups;          // workers per lane
constexpr int kWgPg = kWave / kWgGroups;              // parameter groups (lane bits 0-3)
constexpr int kWgV = 4;                               // parameters per lane
constexpr int kWgWaveParams = kWgPg * kWgV;           // 64 parameters per wave
constexpr int64_t kWgTile = kWavesPerBlock * kWgWaveParams;  // 256 per block tile
constexpr int kWgRowBytes = kWgWaveParams * 4;        // one LDS row: 64 floats
constexpr int kWgR1 = 2;                              // Mix1 rounds the kernel unrolls
constexpr int kWgR2 = 4;                              // Mix2 rounds the kernel unrolls
constexpr int kWgSlots = (kWgR2 + 1) + (kWgR1 + 1) + 1;  // consensus accumulators per lane
constexpr int kWgMaxWidth = 15;                       // widest table row (entries)
#ifndef FGD_WG_BATCH
#define FGD_WG_BATCH 4  // table entries whose gathers are in flight together
#endif

struct WgMix {
    int32_t kind;        // MixKind
    int32_t rounds;      // table rounds (kTable), at most kWgR1 / kWgR2
    int32_t width;       // entries per row in each round's table
    int32_t lds_entry;   // first LDS table entry of this slot
    const int2 *table;   // [rounds][width][64] of (column, bit pattern of float weight)
};

struct WgParams {
    const void *theta_prev;   // [64][ld] storage type, read
    void *theta_out;          // the same array, written
    const void *theta_local;  // [64][ld] storage type
    const float *mom;         // [64][ld] float32, read
    float *mom_out;           // the same array, written
    double *cd_partials;      // [gridDim.x][n_cd][64] or nullptr
    int64_t P, ld, ntiles;
    int32_t n_cd;
    int32_t wave_rows;        // LDS rows per wave: 64, or 65 when some table pads a short row
    int32_t nesterov;
    float lr, mu;
    int32_t rows_bytes;       // LDS bytes of the rows of the four waves (tables follow)
    WgMix mix1, mix2;
};

// Descriptor of a row with a record count of 2^32 - 1 bytes: the per-lane
// offsets of this layout reach 3 ld elements (the worker groups' rows).
__device__ __forceinline__ rsrc_t row_rsrc_wide(const void *base, int64_t elem, int es) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(base)) + elem * es,
                                             static_cast<short>(0), -1, kRawBufferFlags);
}

// Sum of x over the four worker groups (lanes l, l ^ 16, l ^ 32, l ^ 48), the
// same bits in all four lanes.
__device__ __forceinline__ float wg_group_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);  // groups (0 + 2), (1 + 3)
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Balanced tree over the lane's rows [LO, LO + N) of element v.
template <int LO, int N>
__device__ __forceinline__ float wg_tree(const float (&u)[kWgJ][kWgV], int v) {
    if constexpr (N == 1) return u[LO][v];
    else return wg_tree<LO, N / 2>(u, v) + wg_tree<LO + N / 2, N - N / 2>(u, v);
}

// Worker mean of every element of the lane's parameter vector.
__device__ __forceinline__ void wg_mean(const float (&u)[kWgJ][kWgV], float (&mean)[kWgV]) {
#pragma unroll
    for (int v = 0; v < kWgV; ++v) mean[v] = wg_group_sum(wg_tree<0, kWgJ>(u, v)) * (1.0f / kWgWorkers);
}

// This tile's S_m contribution sum_p (u_m,p - mean_p)^2 for the lane's
// worker 4 pg + wg, added to acc: squares summed over the lane's 4
// parameters, then reduce-scattered over the 16 parameter groups (lane bits
// 3..0), so lane pg keeps the total of its row j = pg.
__device__ __forceinline__ void wg_cd(const float (&u)[kWgJ][kWgV], const float (&mean)[kWgV], double &acc,
                                      int lane) {
    float part[kWgJ];
#pragma unroll
    for (int j = 0; j < kWgJ; ++j) {
        float t = 0.0f;
#pragma unroll
        for (int v = 0; v < kWgV; ++v) {
            const float d = u[j][v] - mean[v];
            t = fmaf(d, d, t);
        }
        part[j] = t;
    }
    int n = kWgJ;
    rs_step<3, kWgJ>(part, n, lane);
    rs_step<2, kWgJ>(part, n, lane);
    rs_step<1, kWgJ>(part, n, lane);
    rs_step<0, kWgJ>(part, n, lane);
    acc += static_cast<double>(part[0]);
}

// Consensus of a global-mean output (every worker holds the mean): 0 where
// the mean is finite, NaN where it is not (see cd_global_row).
__device__ __forceinline__ void wg_cd_global(const float (&mean)[kWgV], double &acc) {
    bool bad = false;
#pragma unroll
    for (int v = 0; v < kWgV; ++v) bad |= !__builtin_isfinite(mean[v]);
    if (__builtin_amdgcn_ballot_w64(bad)) acc = __builtin_nan("");
}

// One table round in place, u_m <- sum_d w[d][m] u_{col[d][m]}: the lane's
// rows go to the wave's LDS region, then every entry gathers 4 parameters.
// tab: this round's staged entries, [width][16][4] of (row byte offset,
// weight bits); the lane reads those of its group wg.
__device__ __forceinline__ void wg_round(float (&u)[kWgJ][kWgV], unsigned char *rows, int lane_row, int lane_col,
                                         const int2 *tab, int width, int wg) {
#pragma unroll
    for (int j = 0; j < kWgJ; ++j)
        *reinterpret_cast<f32x4 *>(rows + lane_row + j * kWgGroups * kWgRowBytes) =
            f32x4{u[j][0], u[j][1], u[j][2], u[j][3]};
    // Lanes read rows other lanes of the wave wrote: LDS operations of a
    // wave complete in order; the fence keeps the compiler from moving the
    // reads above the writes.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // Entries are taken in batches of B rows: the B table reads, then the B
    // gathers they address, then the multiply-adds, so that B pairs of
    // dependent LDS reads are in flight together.
    constexpr int B = FGD_WG_BATCH;
    const int2 *t = tab + wg;
    for (int d = 0; d < width; ++d) {
        const int2 *td = t + d * kWgJ * kWgGroups;
#pragma unroll
        for (int j0 = 0; j0 < kWgJ; j0 += B) {
            int2 e[B];
            f32x4 r[B];
#pragma unroll
            for (int q = 0; q < B; ++q) e[q] = td[(j0 + q) * kWgGroups];
#pragma unroll
            for (int q = 0; q < B; ++q) r[q] = *reinterpret_cast<const f32x4 *>(rows + e[q].x + lane_col);
#pragma unroll
            for (int q = 0; q < B; ++q) {
                const int j = j0 + q;
                const float w = __int_as_float(e[q].y);
                if (d == 0) {
                    u[j][0] = w * r[q].x; u[j][1] = w * r[q].y; u[j][2] = w * r[q].z; u[j][3] = w * r[q].w;
                } else {
                    u[j][0] = fmaf(w, r[q].x, u[j][0]);
                    u[j][1] = fmaf(w, r[q].y, u[j][1]);
                    u[j][2] = fmaf(w, r[q].z, u[j][2]);
                    u[j][3] = fmaf(w, r[q].w, u[j][3]);
                }
            }
        }
    }
    // The next round's writes must not pass this round's reads.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One Mix slot on u (mean: the worker mean of u).  Table kinds run up to R
// unrolled rounds (so each round's consensus accumulator is a register);
// acc0 is the accumulator of the slot's first output row.
template <int KIND, int R>
__device__ __forceinline__ void wg_mix(const WgMix &mx, float (&u)[kWgJ][kWgV], const float (&mean)[kWgV],
                                       unsigned char *rows, const int2 *tab_lds, int lane_row, int lane_col, int wg,
                                       int lane, bool cd, double *acc0) {
    const bool table = KIND == kTable || (KIND == kAny && mx.kind == kTable);
    const bool global = KIND == kGlobal || (KIND == kAny && mx.kind == kGlobal);
    if (table) {
#pragma unroll
        for (int k = 0; k < R; ++k) {
            if (k < mx.rounds) {
                wg_round(u, rows, lane_row, lane_col, tab_lds + mx.lds_entry + k * mx.width * kWgJ * kWgGroups,
                         mx.width, wg);
                if (cd) wg_cd(u, mean, acc0[k], lane);
            }
        }
    } else if (global && cd) {
        wg_cd_global(mean, acc0[0]);
    }
}

// Per-lane constants of the step kernel.
struct WgLane {
    unsigned char *rows;    // the wave's LDS rows
    const int2 *tab_lds;    // staged tables
    int lane_row, lane_col, wg, lane, lane_param;
    uint32_t off_p, off_v;  // lane byte offsets in parameter / momentum rows (worker group's row included)
};

// One tile of 256 parameters.  FULL: every lane's 4 parameters lie below P
// (uniform; all tiles but the last), so no lane needs bounds logic.
template <class PIO, int K1, int K2, bool FULL>
__device__ __forceinline__ void wg_tile(const WgParams &a, const WgLane &c, int64_t tb, bool cd,
                                        double (&acc)[kWgSlots]) {
    constexpr int kE = PIO::kElem;
    constexpr int kSlotX = kWgR2 + 1, kSlotT = kWgR2 + kWgR1 + 2;
    unsigned char *rows = c.rows;
    const int2 *tab_lds = c.tab_lds;
    const int lane_row = c.lane_row, lane_col = c.lane_col, wg = c.wg, lane = c.lane;
    const uint32_t off_p = c.off_p, off_v = c.off_v;
    const float mu = a.mu, lr = a.lr;
    const bool nesterov = a.nesterov != 0;
    int nv = kWgV;
    if constexpr (!FULL) {
        const int64_t rem = a.P - tb - c.lane_param;
        nv = rem >= kWgV ? kWgV : (rem > 0 ? static_cast<int>(rem) : 0);
    }

    // Phase A: every row's loads before first use.
    float u1[kWgJ][kWgV], u2[kWgJ][kWgV];
    if (FULL || nv > 0) {
#pragma unroll
        for (int j = 0; j < kWgJ; ++j) {
            const int64_t e = static_cast<int64_t>(kWgGroups * j) * a.ld + tb;
            PIO::load(row_rsrc_wide(a.theta_prev, e, kE), off_p, u1[j]);
            PIO::load(row_rsrc_wide(a.theta_local, e, kE), off_p, u2[j]);
        }
    }
#pragma unroll
    for (int j = 0; j < kWgJ; ++j)
#pragma unroll
        for (int v = 0; v < kWgV; ++v) {
            if (FULL || v < nv) u2[j][v] = u1[j][v] - u2[j][v];
            else { u1[j][v] = 0.0f; u2[j][v] = 0.0f; }
        }

    float gbar[kWgV], xbar[kWgV];
    wg_mean(u2, gbar);
    wg_mean(u1, xbar);
    if (cd) {
        wg_cd(u2, gbar, acc[0], lane);
        wg_cd(u1, xbar, acc[kSlotX], lane);
    }
    wg_mix<K2, kWgR2>(a.mix2, u2, gbar, rows, tab_lds, lane_row, lane_col, wg, lane, cd, acc + 1);
    wg_mix<K1, kWgR1>(a.mix1, u1, xbar, rows, tab_lds, lane_row, lane_col, wg, lane, cd, acc + kSlotX + 1);
    const bool g2 = K2 == kGlobal || (K2 == kAny && a.mix2.kind == kGlobal);
    const bool g1 = K1 == kGlobal || (K1 == kAny && a.mix1.kind == kGlobal);

    // Phase D: the optimizer, four rows at a time; the stored theta'
    // replaces the row's mixed gradient.
    constexpr int G = 4;
#pragma unroll
    for (int j0 = 0; j0 < kWgJ; j0 += G) {
        float vm[G][kWgV];
        if (FULL || nv > 0) {
#pragma unroll
            for (int i = 0; i < G; ++i)
                F32Io<kWgV>::load(row_rsrc_wide(a.mom, static_cast<int64_t>(kWgGroups * (j0 + i)) * a.ld + tb, 4),
                                  off_v, vm[i]);
        } else {
#pragma unroll
            for (int i = 0; i < G; ++i)
#pragma unroll
                for (int v = 0; v < kWgV; ++v) vm[i][v] = 0.0f;
        }
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const int j = j0 + i;
            float t[kWgV], stored[kWgV];
#pragma unroll
            for (int v = 0; v < kWgV; ++v) {
                const float g = g2 ? gbar[v] : u2[j][v];
                const float x = g1 ? xbar[v] : u1[j][v];
                vm[i][v] = fmaf(mu, vm[i][v], g);
                const float step = nesterov ? fmaf(mu, vm[i][v], g) : vm[i][v];
                t[v] = fmaf(-lr, step, x);
            }
            if (FULL || nv > 0) {
                const int64_t e = static_cast<int64_t>(kWgGroups * j) * a.ld + tb;
                const rsrc_t rv = row_rsrc_wide(a.mom_out, e, 4);
                const rsrc_t rp = row_rsrc_wide(a.theta_out, e, kE);
                if (FULL || nv == kWgV) {
                    F32Io<kWgV>::store(rv, off_v, vm[i]);
                    PIO::store(rp, off_p, t, stored);
                } else {
                    F32Io<kWgV>::store_part(rv, off_v, nv, vm[i]);
                    PIO::store_part(rp, off_p, nv, t, stored);
                }
            } else {
#pragma unroll
                for (int v = 0; v < kWgV; ++v) stored[v] = 0.0f;
            }
#pragma unroll
            for (int v = 0; v < kWgV; ++v) u2[j][v] = stored[v];
        }
    }
    if (cd) {
        float tbar[kWgV];
        wg_mean(u2, tbar);
        wg_cd(u2, tbar, acc[kSlotT], lane);
    }
}

template <class PIO, int K1, int K2>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(2))) void wg_step_kernel(WgParams a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    constexpr int kE = PIO::kElem;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int wg = lane >> 4, pg = lane & (kWgPg - 1);
    unsigned char *rows = smem + wave * a.wave_rows * kWgRowBytes;  // this wave's rows
    int2 *tab_lds = reinterpret_cast<int2 *>(smem + a.rows_bytes);
    const int lane_row = wg * kWgRowBytes + pg * 16;  // byte offset of the lane's row 0 (worker wg)
    const int lane_col = pg * 16;                     // byte offset of the lane's 4 parameters in a row

    // Stage the tables: entry (k, d, m) at [k][d][m >> 2][m & 3], with the
    // column turned into its LDS row offset.
    for (int s = 0; s < 2; ++s) {
        const WgMix &mx = s == 0 ? a.mix1 : a.mix2;
        if (mx.kind != kTable) continue;
        const int n = mx.rounds * mx.width * kWgWorkers;
        for (int i = tid; i < n; i += kBlock) {
            const int2 e = mx.table[i];
            const int m = i % kWgWorkers, kd = i / kWgWorkers;
            tab_lds[mx.lds_entry + (kd * kWgJ + (m >> 2)) * kWgGroups + (m & 3)] = int2{e.x * kWgRowBytes, e.y};
        }
    }
    if (a.wave_rows > kWgWorkers && lane < kWgRowBytes / 4)  // the all-zero row of padded tables
        reinterpret_cast<float *>(rows + kWgWorkers * kWgRowBytes)[lane] = 0.0f;
    __syncthreads();

    const bool cd = a.cd_partials != nullptr;
    double acc[kWgSlots];
#pragma unroll
    for (int s = 0; s < kWgSlots; ++s) acc[s] = 0.0;
    constexpr int kSlotX = kWgR2 + 1, kSlotT = kWgR2 + kWgR1 + 2;

    WgLane c;
    c.rows = rows;
    c.tab_lds = tab_lds;
    c.lane_row = lane_row;
    c.lane_col = lane_col;
    c.wg = wg;
    c.lane = lane;
    c.lane_param = wave * kWgWaveParams + pg * kWgV;  // parameter offset in a tile
    c.off_p = static_cast<uint32_t>((wg * a.ld + c.lane_param) * kE);
    c.off_v = static_cast<uint32_t>((wg * a.ld + c.lane_param) * 4);

    for (int64_t tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int64_t tb = tile * kWgTile;
        if (tb + kWgTile <= a.P) wg_tile<PIO, K1, K2, true>(a, c, tb, cd, acc);
        else wg_tile<PIO, K1, K2, false>(a, c, tb, cd, acc);
    }

    if (cd) {
        // Block partials: the four waves' accumulators through LDS (the rows
        // region is free now), summed in wave order.
        __syncthreads();
        double *red = reinterpret_cast<double *>(smem);  // [wave][slot][lane]
#pragma unroll
        for (int s = 0; s < kWgSlots; ++s) red[(wave * kWgSlots + s) * kWave + lane] = acc[s];
        __syncthreads();
        const int n2 = a.mix2.kind == kTable ? a.mix2.rounds : (a.mix2.kind == kGlobal ? 1 : 0);
        const int n1 = a.mix1.kind == kTable ? a.mix1.rounds : (a.mix1.kind == kGlobal ? 1 : 0);
        for (int i = tid; i < a.n_cd * kWgWorkers; i += kBlock) {
            const int r = i / kWgWorkers, m = i % kWgWorkers;
            // Output rows g^0..g^n2, x^0..x^n1, theta'; worker m = 4 pg + wg
            // sits in lane 16 wg + pg.
            const int s = r <= n2 ? r : (r <= n2 + n1 + 1 ? kSlotX + (r - n2 - 1) : kSlotT);
            const int l = (m & 3) * kWgPg + (m >> 2);
            double sum = 0.0;
#pragma unroll
            for (int w = 0; w < kWavesPerBlock; ++w) sum += red[(w * kWgSlots + s) * kWave + l];
            a.cd_partials[(static_cast<int64_t>(blockIdx.x) * a.n_cd + r) * kWgWorkers + m] = sum;
        }
    }
}

// The worker-group step's memory traffic without its arithmetic (the
// access-pattern reference of fgd_stream_step_pattern for this layout):
// same tiles, per-lane rows and vectors, cache policy and launch shape;
// every theta_prev and theta_local row of a tile loaded before first use,
// then four momentum rows at a time loaded and theta_prev and the momentum
// stored back with their own bits (OR of theta_local AND mask, mask = 0 at
// run time, keeps every load live).  Lanes of a ragged vector store nothing.
template <int kE>
__global__ __launch_bounds__(kBlock) void wg_pattern_kernel(PatternParams a) {
    constexpr int NP = kWgV * kE, WP = RawIo<NP>::kW, WV = RawIo<kWgV * 4>::kW;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int wg = lane >> 4, pg = lane & (kWgPg - 1);
    const int lane_param = wave * kWgWaveParams + pg * kWgV;
    const uint32_t off_p = static_cast<uint32_t>((wg * a.ld + lane_param) * kE);
    const uint32_t off_v = static_cast<uint32_t>((wg * a.ld + lane_param) * 4);
    for (int64_t tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int64_t tb = tile * kWgTile;
        const int64_t rem = a.P - tb - lane_param;
        if (rem <= 0) continue;
        const bool whole = rem >= kWgV;
        uint32_t u1[kWgJ][WP], u2[kWgJ][WP];
#pragma unroll
        for (int j = 0; j < kWgJ; ++j) {
            const int64_t e = static_cast<int64_t>(kWgGroups * j) * a.ld + tb;
            RawIo<NP>::load(row_rsrc_wide(a.theta_prev, e, kE), off_p, u1[j]);
            RawIo<NP>::load(row_rsrc_wide(a.theta_local, e, kE), off_p, u2[j]);
        }
        constexpr int G = 4;
#pragma unroll
        for (int j0 = 0; j0 < kWgJ; j0 += G) {
            uint32_t vm[G][WV];
#pragma unroll
            for (int i = 0; i < G; ++i)
                RawIo<kWgV * 4>::load(row_rsrc_wide(a.mom, static_cast<int64_t>(kWgGroups * (j0 + i)) * a.ld + tb, 4),
                                      off_v, vm[i]);
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const int j = j0 + i;
                uint32_t t[WP];
#pragma unroll
                for (int k = 0; k < WP; ++k) t[k] = u1[j][k] | (u2[j][k] & a.mask);
#pragma unroll
                for (int k = 0; k < WV; ++k) vm[i][k] |= u2[j][k % WP] & a.mask;
                if (whole) {
                    const int64_t e = static_cast<int64_t>(kWgGroups * j) * a.ld + tb;
                    RawIo<kWgV * 4>::store(row_rsrc_wide(a.mom_out, e, 4), off_v, vm[i]);
                    RawIo<NP>::store(row_rsrc_wide(a.theta_out, e, kE), off_p, t);
                }
            }
        }
    }
}

// Worker-group kernel for the (Mix1, Mix2) kinds of the paper's sparse
// configurations at 64 workers: LocalM1M2 (CSR, CSR) and GlobalM1LocalM2
// (global mean, CSR).  False for other kinds (their run-time-kind form
// needs more registers than two waves per SIMD leave, so they run on
// outer_step_kernel).
struct WgKernel {
    const void *step;
    const void *pattern;  // wg_pattern_kernel of the storage
};
bool wg_kernel(bool bf16, int k1, int k2, WgKernel *out);

}  // namespace fgd
