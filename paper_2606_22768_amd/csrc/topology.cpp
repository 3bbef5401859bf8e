// topology.cpp -- validation and per-round effective weights of a Mix slot.
#include "topology.hpp"

#include <algorithm>
#include <cmath>
#include <cstdio>

namespace fgd {

namespace {

constexpr int32_t kMaxWorkers = 64;
constexpr int32_t kMaxRounds = 8;
constexpr double kSumTolerance = 1e-6;

std::string fmt(const char *f, long a = 0, long b = 0, long c = 0) {
    char buf[256];
    std::snprintf(buf, sizeof buf, f, a, b, c);
    return buf;
}

// Index of entry (i, j) in the CSR, or -1.
int32_t find_entry(const int32_t *row_ptr, const int32_t *col_idx, int32_t i, int32_t j) {
    const int32_t *b = col_idx + row_ptr[i], *e = col_idx + row_ptr[i + 1];
    const int32_t *it = std::lower_bound(b, e, j);
    return (it != e && *it == j) ? static_cast<int32_t>(it - col_idx) : -1;
}

TopoStatus check_structure(int32_t M, const int32_t *row_ptr, const int32_t *col_idx, std::string &err) {
    if (!row_ptr || !col_idx) {
        err = "row_ptr and col_idx are required for a CSR topology";
        return TopoStatus::invalid_arg;
    }
    if (row_ptr[0] != 0) {
        err = "row_ptr[0] must be 0";
        return TopoStatus::topology;
    }
    for (int32_t i = 0; i < M; ++i) {
        if (row_ptr[i + 1] < row_ptr[i]) {
            err = fmt("row_ptr decreases at row %ld", i);
            return TopoStatus::topology;
        }
    }
    if (row_ptr[M] > M * M) {
        err = fmt("nnz %ld exceeds M*M = %ld", row_ptr[M], static_cast<long>(M) * M);
        return TopoStatus::topology;
    }
    for (int32_t i = 0; i < M; ++i) {
        bool diag = false;
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            const int32_t j = col_idx[e];
            if (j < 0 || j >= M) {
                err = fmt("column %ld of row %ld is out of range", j, i);
                return TopoStatus::topology;
            }
            if (e > row_ptr[i] && col_idx[e - 1] >= j) {
                err = fmt("columns of row %ld are not strictly ascending", i);
                return TopoStatus::topology;
            }
            diag = diag || j == i;
        }
        if (!diag) {
            err = fmt("row %ld has no diagonal entry", i);
            return TopoStatus::topology;
        }
    }
    return TopoStatus::ok;
}

bool structurally_symmetric(int32_t M, const int32_t *row_ptr, const int32_t *col_idx) {
    for (int32_t i = 0; i < M; ++i)
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
            if (find_entry(row_ptr, col_idx, col_idx[e], i) < 0) return false;
    return true;
}

TopoStatus check_mask(int32_t M, const int32_t *row_ptr, const int32_t *col_idx, const uint8_t *mask, bool sym,
                      std::string &err) {
    for (int32_t i = 0; i < M; ++i) {
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            const int32_t j = col_idx[e];
            if (mask[e] > 1) {
                err = fmt("mask entry (%ld,%ld) is %ld, not 0/1", i, j, mask[e]);
                return TopoStatus::topology;
            }
            if (j == i && mask[e] != 1) {
                err = fmt("diagonal entry of row %ld is masked", i);
                return TopoStatus::topology;
            }
            if (sym) {
                const int32_t t = find_entry(row_ptr, col_idx, j, i);
                if (mask[t] != mask[e]) {
                    err = fmt("masks of (%ld,%ld) and its transpose differ", i, j);
                    return TopoStatus::topology;
                }
            }
        }
    }
    return TopoStatus::ok;
}

}  // namespace

TopoStatus effective_round_weights(int32_t M, const int32_t *row_ptr, const int32_t *col_idx,
                                   const float *weights, const uint8_t *mask, int32_t reweight, float *out,
                                   std::string &err) {
    if (M < 1 || M > kMaxWorkers) {
        err = fmt("num_workers %ld is outside [1, %ld]", M, kMaxWorkers);
        return TopoStatus::invalid_arg;
    }
    if (!out) {
        err = "output array is NULL";
        return TopoStatus::invalid_arg;
    }
    TopoStatus st = check_structure(M, row_ptr, col_idx, err);
    if (st != TopoStatus::ok) return st;
    const bool sym = structurally_symmetric(M, row_ptr, col_idx);
    if (mask) {
        st = check_mask(M, row_ptr, col_idx, mask, sym, err);
        if (st != TopoStatus::ok) return st;
    }
    const int32_t nnz = row_ptr[M];
    auto is_live = [&](int32_t e) { return !mask || mask[e] != 0; };

    if (reweight == 0 || reweight == 2) {
        if (!weights) {
            err = "weights are required unless the reweighting is Metropolis";
            return TopoStatus::invalid_arg;
        }
        for (int32_t e = 0; e < nnz; ++e) {
            if (!std::isfinite(weights[e]) || weights[e] < 0.0f) {
                err = fmt("weight of entry %ld is negative or not finite", e);
                return TopoStatus::topology;
            }
        }
    }
    if (reweight == 0) {
        for (int32_t e = 0; e < nnz; ++e) {
            if (!is_live(e)) {
                err = "masks drop links but the reweighting is NONE";
                return TopoStatus::topology;
            }
            out[e] = weights[e];
        }
        return TopoStatus::ok;
    }
    if (reweight == 1) {
        if (!sym) {
            err = "Metropolis weights need a structurally symmetric graph";
            return TopoStatus::topology;
        }
        int32_t degree[kMaxWorkers] = {0};
        for (int32_t i = 0; i < M; ++i)
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
                degree[i] += (col_idx[e] != i && is_live(e)) ? 1 : 0;
        for (int32_t i = 0; i < M; ++i) {
            double taken = 0.0;
            int32_t self = -1;
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                const int32_t j = col_idx[e];
                if (j == i) {
                    self = e;
                } else if (is_live(e)) {
                    const double w = 1.0 / (1.0 + static_cast<double>(std::max(degree[i], degree[j])));
                    taken += w;
                    out[e] = static_cast<float>(w);
                } else {
                    out[e] = 0.0f;
                }
            }
            out[self] = static_cast<float>(1.0 - taken);
        }
        return TopoStatus::ok;
    }
    if (reweight == 2) {
        for (int32_t i = 0; i < M; ++i) {
            const int32_t self = find_entry(row_ptr, col_idx, i, i);
            double diag = static_cast<double>(weights[self]);
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                if (e == self) continue;
                if (is_live(e)) {
                    out[e] = weights[e];
                } else {
                    diag += static_cast<double>(weights[e]);
                    out[e] = 0.0f;
                }
            }
            out[self] = static_cast<float>(diag);
        }
        return TopoStatus::ok;
    }
    err = fmt("unknown reweighting %ld", reweight);
    return TopoStatus::invalid_arg;
}

TopoStatus build_mix_topology(int32_t M, int32_t kind, const int32_t *row_ptr, const int32_t *col_idx,
                              const float *weights, int32_t rounds, const uint8_t *masks, int32_t reweight,
                              MixTopology &out, std::string &err) {
    MixTopology t;
    t.num_workers = M;
    if (M < 1 || M > kMaxWorkers) {
        err = fmt("num_workers %ld is outside [1, %ld]", M, kMaxWorkers);
        return TopoStatus::invalid_arg;
    }
    if (kind == 0 || kind == 1) {
        t.kind = kind;
        out = std::move(t);
        return TopoStatus::ok;
    }
    if (kind != 2) {
        err = fmt("unknown topology kind %ld", kind);
        return TopoStatus::invalid_arg;
    }
    if (rounds < 0 || rounds > kMaxRounds) {
        err = fmt("num_rounds %ld is outside [0, %ld]", rounds, kMaxRounds);
        return TopoStatus::invalid_arg;
    }
    if (reweight < 0 || reweight > 2) {
        err = fmt("unknown reweighting %ld", reweight);
        return TopoStatus::invalid_arg;
    }
    if (rounds == 0) {  // zero rounds: the identity
        t.kind = 0;
        out = std::move(t);
        return TopoStatus::ok;
    }
    TopoStatus st = check_structure(M, row_ptr, col_idx, err);
    if (st != TopoStatus::ok) return st;
    const int32_t nnz = row_ptr[M];
    t.kind = 2;
    t.rounds = rounds;
    t.row_ptr.assign(row_ptr, row_ptr + M + 1);
    t.col_idx.assign(col_idx, col_idx + nnz);
    t.eff.assign(static_cast<size_t>(rounds) * nnz, 0.0f);
    t.live.assign(static_cast<size_t>(rounds) * nnz, 1);
    for (int32_t k = 0; k < rounds; ++k) {
        const uint8_t *mask = masks ? masks + static_cast<size_t>(k) * nnz : nullptr;
        std::string e2;
        st = effective_round_weights(M, row_ptr, col_idx, weights, mask, reweight, t.eff.data() + k * nnz, e2);
        if (st != TopoStatus::ok) {
            err = fmt("round %ld: ", k) + e2;
            return st;
        }
        if (mask) std::copy(mask, mask + nnz, t.live.begin() + static_cast<size_t>(k) * nnz);
        // Row and column sums of the effective W (live entries), in double.
        double col_sum[kMaxWorkers] = {0.0};
        for (int32_t i = 0; i < M; ++i) {
            double row_sum = 0.0;
            int32_t nlive = 0;
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                if (!t.live[static_cast<size_t>(k) * nnz + e]) continue;
                const double w = t.eff[static_cast<size_t>(k) * nnz + e];
                row_sum += w;
                col_sum[col_idx[e]] += w;
                ++nlive;
            }
            t.width = std::max(t.width, nlive);
            if (std::fabs(row_sum - 1.0) > kSumTolerance) {
                err = fmt("round %ld: row %ld of W does not sum to 1", k, i);
                return TopoStatus::topology;
            }
        }
        for (int32_t j = 0; j < M; ++j) {
            if (std::fabs(col_sum[j] - 1.0) > kSumTolerance) {
                err = fmt("round %ld: column %ld of W does not sum to 1 (W must be doubly stochastic)", k, j);
                return TopoStatus::topology;
            }
        }
    }
    for (int32_t k = 0; k < rounds && !t.padded; ++k) {
        for (int32_t i = 0; i < M; ++i) {
            int32_t nlive = 0;
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) nlive += t.live[static_cast<size_t>(k) * nnz + e];
            if (nlive < t.width) {
                t.padded = true;
                break;
            }
        }
    }
    out = std::move(t);
    return TopoStatus::ok;
}

void MixTopology::pack_tables(std::vector<int32_t> &out) const {
    out.clear();
    if (kind != 2) return;
    const int32_t M = num_workers;
    const int32_t nnz = row_ptr[M];
    out.assign(static_cast<size_t>(rounds) * width * M * 2, 0);
    for (int32_t k = 0; k < rounds; ++k) {
        for (int32_t m = 0; m < M; ++m) {
            int32_t d = 0;
            for (int32_t e = row_ptr[m]; e < row_ptr[m + 1]; ++e) {
                if (!live[static_cast<size_t>(k) * nnz + e]) continue;
                const size_t at = ((static_cast<size_t>(k) * width + d) * M + m) * 2;
                float w = eff[static_cast<size_t>(k) * nnz + e];
                int32_t bits;
                static_assert(sizeof bits == sizeof w, "float is 32-bit");
                std::copy(reinterpret_cast<const char *>(&w), reinterpret_cast<const char *>(&w) + 4,
                          reinterpret_cast<char *>(&bits));
                out[at] = col_idx[e];
                out[at + 1] = bits;
                ++d;
            }
            for (; d < width; ++d) {
                const size_t at = ((static_cast<size_t>(k) * width + d) * M + m) * 2;
                out[at] = M;  // the all-zero LDS row
                out[at + 1] = 0;
            }
        }
    }
}

}  // namespace fgd
