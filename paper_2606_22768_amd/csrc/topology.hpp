// topology.hpp -- host-side mixing topology of one Mix slot.
//
// A Mix round maps worker m to sum_n w_{m,n} u_n (Sec. 3, gossip mixing
// operator).  W must be doubly stochastic; the paper also takes it
// symmetric, which this engine only requires where the reweighting rule
// needs it (a directed, doubly-stochastic exponential graph is accepted).
// Links that drop in a round are described by per-round masks; the
// effective weights of the round follow the reweighting rule documented in
// include/fgd.h.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace fgd {

enum class TopoStatus { ok, invalid_arg, topology };

struct MixTopology {
    int32_t kind = 0;                  // 0 identity, 1 global mean, 2 CSR
    int32_t rounds = 0;                // CSR rounds
    int32_t num_workers = 0;
    std::vector<int32_t> row_ptr;      // [M+1]
    std::vector<int32_t> col_idx;      // [nnz]
    std::vector<float> eff;            // [rounds][nnz], 0 where dropped
    std::vector<uint8_t> live;         // [rounds][nnz]
    int32_t width = 0;                 // max live entries of a row over all rounds
    bool padded = false;               // some row of some round has fewer than `width` live entries

    // Rounds of this slot as the kernel counts them (global mean = 1).
    int32_t effective_rounds() const { return kind == 0 ? 0 : (kind == 1 ? 1 : rounds); }

    // Padded per-round tables for the kernel: [rounds][width][M] pairs of
    // (column, float bits); the d-th live entry of each row in ascending
    // column order, then (M, 0) padding that points at an all-zero row.
    void pack_tables(std::vector<int32_t> &out) const;
};

// Validates the inputs and fills `out`.  On failure `err` says why.
TopoStatus build_mix_topology(int32_t M, int32_t kind, const int32_t *row_ptr, const int32_t *col_idx,
                              const float *weights, int32_t rounds, const uint8_t *masks, int32_t reweight,
                              MixTopology &out, std::string &err);

// Effective weights of a single round (mask may be NULL).
TopoStatus effective_round_weights(int32_t M, const int32_t *row_ptr, const int32_t *col_idx,
                                   const float *weights, const uint8_t *mask, int32_t reweight, float *out,
                                   std::string &err);

}  // namespace fgd
