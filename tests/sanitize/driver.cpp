// Sanitizer driver: runs the CPU oracle (oracle/fgd_oracle.c) and the
// library's host topology code (paper_2606_22768_amd/csrc/topology.cpp) on
// seeded random and malformed inputs, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitize.py.  Both parse
// caller-supplied CSR structures, masks and subset segments; any
// out-of-bounds access, leak or undefined operation aborts the run.
//
// The driver also checks what it can cheaply: the two implementations'
// effective weights agree bit for bit, malformed topologies are rejected,
// and the oracle's steps, split halves and consensus run on random sizes
// (P = 0 and padded rows included) and reject bad arguments.  Prints "ok"
// and exits 0 on success.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "topology.hpp"

// The oracle's C interface, declared here (the oracle ships no header).
extern "C" {
typedef struct {
    float lr, mu;
    int32_t nesterov, mix1_state, n_seg;
    const int64_t *seg;
} fgdo_opts;
typedef struct {
    int32_t kind, rounds;
    const int32_t *row_ptr, *col_idx;
    const float *weights;
    const uint8_t *masks;
    int32_t reweight;
} fgdo_mix;
int fgdo_round_weights(int32_t M, const int32_t *row_ptr, const int32_t *col_idx, const float *w_in,
                       const uint8_t *mask, int32_t reweight, float *w_out);
int fgdo_outer_step(int32_t M, int64_t P, int64_t ld, int32_t dtype, void *theta_prev, const void *theta_local,
                    float *mom, const fgdo_mix *mix1, const fgdo_mix *mix2, const fgdo_opts *opt, double *cd);
int fgdo_mix1_split(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *theta_prev, void *x_out, float *mom,
                    const fgdo_mix *mix1, int32_t mix1_state, double *cd);
int fgdo_outer_blocking(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *x_in, void *theta_prev,
                        void *theta_local, float *mom, const fgdo_mix *mix2, const fgdo_opts *opt,
                        int32_t write_local, double *cd);
int fgdo_consensus(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *x, double *S);
int fgdo_num_cd(const fgdo_mix *mix1, const fgdo_mix *mix2);
uint16_t fgdo_bf16_from_double(double d);
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {  // xorshift64*
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return g_state * 0x2545F4914F6CDD1Dull;
}
int rnd(int n) { return static_cast<int>(next() % static_cast<uint64_t>(n)); }
double unif() { return (next() >> 11) * (1.0 / 9007199254740992.0); }
double normal() {
    double u = unif() + 1e-300, v = unif();
    return std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
}

int g_fail = 0;
void check(bool ok, const char *what, int a = 0, int b = 0) {
    if (!ok) {
        std::printf("FAIL: %s (%d, %d)\n", what, a, b);
        ++g_fail;
    }
}

struct Csr {
    int M = 0;
    std::vector<int32_t> row_ptr, col_idx;
};

// Random structurally symmetric graph with every diagonal entry.
Csr random_graph(int M, double p) {
    std::vector<std::vector<char>> adj(M, std::vector<char>(M, 0));
    for (int i = 0; i < M; ++i) {
        adj[i][i] = 1;
        for (int j = i + 1; j < M; ++j)
            if (unif() < p) adj[i][j] = adj[j][i] = 1;
    }
    Csr g;
    g.M = M;
    g.row_ptr.push_back(0);
    for (int i = 0; i < M; ++i) {
        for (int j = 0; j < M; ++j)
            if (adj[i][j]) g.col_idx.push_back(j);
        g.row_ptr.push_back(static_cast<int32_t>(g.col_idx.size()));
    }
    return g;
}

int32_t entry(const Csr &g, int i, int j) {
    for (int e = g.row_ptr[i]; e < g.row_ptr[i + 1]; ++e)
        if (g.col_idx[e] == j) return e;
    return -1;
}

// Symmetric per-round masks: every undirected link dropped with probability p.
std::vector<uint8_t> random_masks(const Csr &g, int rounds, double p) {
    const int nnz = g.row_ptr[g.M];
    std::vector<uint8_t> m(static_cast<size_t>(rounds) * nnz, 1);
    for (int k = 0; k < rounds; ++k)
        for (int i = 0; i < g.M; ++i)
            for (int e = g.row_ptr[i]; e < g.row_ptr[i + 1]; ++e) {
                const int j = g.col_idx[e];
                if (j <= i) continue;
                if (unif() < p) {
                    m[static_cast<size_t>(k) * nnz + e] = 0;
                    m[static_cast<size_t>(k) * nnz + entry(g, j, i)] = 0;
                }
            }
    return m;
}

void weights_agree() {
    for (int it = 0; it < 300; ++it) {
        const int M = 1 + rnd(40);
        Csr g = random_graph(M, 0.05 + 0.9 * unif());
        const int nnz = g.row_ptr[M];
        std::vector<float> base(nnz), a(nnz), b(nnz);
        check(fgdo_round_weights(M, g.row_ptr.data(), g.col_idx.data(), nullptr, nullptr, 1, base.data()) == 0,
              "oracle Metropolis base weights", it);
        std::vector<uint8_t> mask = random_masks(g, 1, unif());
        for (int rw = 1; rw <= 2; ++rw) {
            std::string err;
            auto st = fgd::effective_round_weights(M, g.row_ptr.data(), g.col_idx.data(), base.data(), mask.data(), rw,
                                                   a.data(), err);
            check(st == fgd::TopoStatus::ok, "library weights", it, rw);
            check(fgdo_round_weights(M, g.row_ptr.data(), g.col_idx.data(), base.data(), mask.data(), rw, b.data()) == 0,
                  "oracle weights", it, rw);
            check(std::memcmp(a.data(), b.data(), nnz * sizeof(float)) == 0, "weights differ in bits", it, rw);
        }
        // Several rounds through the slot builder and its packed tables.
        const int rounds = 1 + rnd(8);
        std::vector<uint8_t> masks = random_masks(g, rounds, 0.3 * unif());
        fgd::MixTopology t;
        std::string err;
        auto st = fgd::build_mix_topology(M, 2, g.row_ptr.data(), g.col_idx.data(), nullptr, rounds, masks.data(), 1, t,
                                          err);
        check(st == fgd::TopoStatus::ok, "slot with several rounds", it);
        std::vector<int32_t> tab;
        t.pack_tables(tab);
        check(tab.size() == static_cast<size_t>(rounds) * t.width * M * 2, "packed table size", it);
        for (size_t i = 0; i < tab.size(); i += 2) check(tab[i] >= 0 && tab[i] <= M, "packed column in range", it);
    }
}

void malformed_rejected() {
    const int M = 6;
    Csr g = random_graph(M, 0.6);
    const int nnz = g.row_ptr[M];
    std::vector<float> w(nnz);
    fgdo_round_weights(M, g.row_ptr.data(), g.col_idx.data(), nullptr, nullptr, 1, w.data());
    std::vector<float> out(nnz);
    // slot_only: a defect only the slot builder sees (the one-round weight
    // computation does not check that W is doubly stochastic).
    auto reject = [&](const std::vector<int32_t> &rp, const std::vector<int32_t> &ci, const float *wt,
                      const uint8_t *mask, int rw, const char *what, bool slot_only = false) {
        std::string err;
        // The column array is given with room for any row_ptr[M] <= M * M, so
        // the checks (not the buffer) decide.
        std::vector<int32_t> cols(ci);
        cols.resize(M * M, 0);
        auto st = fgd::effective_round_weights(M, rp.data(), cols.data(), wt, mask, rw, out.data(), err);
        check(slot_only || (st != fgd::TopoStatus::ok && !err.empty()), what);
        fgd::MixTopology t;
        std::vector<uint8_t> masks2;
        if (mask) masks2.assign(mask, mask + nnz);
        st = fgd::build_mix_topology(M, 2, rp.data(), cols.data(), wt, 1, mask ? masks2.data() : nullptr, rw, t, err);
        check(st != fgd::TopoStatus::ok, what);
    };
    {
        auto rp = g.row_ptr;
        std::swap(rp[2], rp[3]);
        if (rp[2] != rp[3]) reject(rp, g.col_idx, w.data(), nullptr, 0, "decreasing row_ptr");
    }
    {
        auto rp = g.row_ptr;
        rp[0] = 1;
        reject(rp, g.col_idx, w.data(), nullptr, 0, "row_ptr[0] != 0");
    }
    {
        auto rp = g.row_ptr;
        rp[M] = M * M + 1;
        reject(rp, g.col_idx, w.data(), nullptr, 0, "nnz beyond M*M");
    }
    {
        auto ci = g.col_idx;
        ci[0] = M;
        reject(g.row_ptr, ci, w.data(), nullptr, 0, "column out of range");
        ci[0] = -1;
        reject(g.row_ptr, ci, w.data(), nullptr, 0, "negative column");
    }
    {
        auto ci = g.col_idx;
        for (int i = 0; i < M; ++i)
            if (g.row_ptr[i + 1] - g.row_ptr[i] >= 2) {
                std::swap(ci[g.row_ptr[i]], ci[g.row_ptr[i] + 1]);
                break;
            }
        reject(g.row_ptr, ci, w.data(), nullptr, 0, "unsorted columns");
    }
    {
        // Row 0 without its diagonal: drop column 0 from row 0.
        std::vector<int32_t> rp{0}, ci;
        for (int i = 0; i < M; ++i) {
            for (int e = g.row_ptr[i]; e < g.row_ptr[i + 1]; ++e)
                if (!(i == 0 && g.col_idx[e] == 0)) ci.push_back(g.col_idx[e]);
            rp.push_back(static_cast<int32_t>(ci.size()));
        }
        std::vector<float> w2(ci.size(), 0.1f);
        reject(rp, ci, w2.data(), nullptr, 0, "missing diagonal");
    }
    std::vector<uint8_t> mask(nnz, 1);
    mask[entry(g, 1, 1)] = 0;
    reject(g.row_ptr, g.col_idx, w.data(), mask.data(), 1, "masked diagonal");
    mask.assign(nnz, 1);
    mask[0] = 2;
    reject(g.row_ptr, g.col_idx, w.data(), mask.data(), 1, "mask not 0/1");
    mask.assign(nnz, 1);
    for (int e = g.row_ptr[0]; e < g.row_ptr[1]; ++e)
        if (g.col_idx[e] != 0) {
            mask[e] = 0;  // (0, j) dropped, (j, 0) live
            reject(g.row_ptr, g.col_idx, w.data(), mask.data(), 1, "asymmetric mask");
            reject(g.row_ptr, g.col_idx, w.data(), mask.data(), 0, "masks under NONE");
            break;
        }
    {
        std::vector<float> bad(w);
        bad[0] = -0.5f;
        reject(g.row_ptr, g.col_idx, bad.data(), nullptr, 0, "negative weight");
        bad[0] = NAN;
        reject(g.row_ptr, g.col_idx, bad.data(), nullptr, 0, "NaN weight");
        bad[0] = w[0] + 0.25f;
        reject(g.row_ptr, g.col_idx, bad.data(), nullptr, 0, "row sum != 1", true);
    }
    reject(g.row_ptr, g.col_idx, nullptr, nullptr, 0, "NONE without weights");
    reject(g.row_ptr, g.col_idx, w.data(), nullptr, 7, "unknown reweighting");
    {
        std::string err;
        fgd::MixTopology t;
        check(fgd::build_mix_topology(0, 2, g.row_ptr.data(), g.col_idx.data(), w.data(), 1, nullptr, 0, t, err) !=
                  fgd::TopoStatus::ok, "M = 0");
        check(fgd::build_mix_topology(65, 1, nullptr, nullptr, nullptr, 1, nullptr, 0, t, err) != fgd::TopoStatus::ok,
              "M = 65");
        check(fgd::build_mix_topology(M, 2, g.row_ptr.data(), g.col_idx.data(), w.data(), 9, nullptr, 0, t, err) !=
                  fgd::TopoStatus::ok, "9 rounds");
        check(fgd::build_mix_topology(M, 2, nullptr, nullptr, w.data(), 1, nullptr, 0, t, err) != fgd::TopoStatus::ok,
              "NULL structure");
        check(fgd::build_mix_topology(M, 5, nullptr, nullptr, nullptr, 1, nullptr, 0, t, err) != fgd::TopoStatus::ok,
              "unknown kind");
    }
    // Metropolis on a structurally non-symmetric graph: directed ring with self loops.
    {
        std::vector<int32_t> rp{0}, ci;
        for (int i = 0; i < M; ++i) {
            int a = i, b = (i + 1) % M;
            ci.push_back(a < b ? a : b);
            ci.push_back(a < b ? b : a);
            rp.push_back(static_cast<int32_t>(ci.size()));
        }
        std::vector<float> w2(ci.size(), 0.5f);
        reject(rp, ci, w2.data(), nullptr, 1, "Metropolis on a directed graph");
    }
}

// The oracle's fused step, split halves and consensus on random sizes,
// kinds, masks, subsets and storages, then its argument rejections.
void oracle_steps() {
    for (int it = 0; it < 120; ++it) {
        const int M = 1 + rnd(12);
        const int64_t P = rnd(4) == 0 ? 0 : 1 + rnd(300);
        const int64_t ld = P + rnd(9);
        const int dtype = rnd(2);
        Csr g = random_graph(M, 0.2 + 0.7 * unif());
        const int nnz = g.row_ptr[M];
        std::vector<float> base(nnz);
        fgdo_round_weights(M, g.row_ptr.data(), g.col_idx.data(), nullptr, nullptr, 1, base.data());
        const int k1 = rnd(4), k2 = rnd(4);
        std::vector<uint8_t> m1 = random_masks(g, k1 > 0 ? k1 : 1, 0.3), m2 = random_masks(g, k2 > 0 ? k2 : 1, 0.3);
        fgdo_mix mix1{rnd(3), k1, g.row_ptr.data(), g.col_idx.data(), base.data(), m1.data(), 1 + rnd(2)};
        fgdo_mix mix2{rnd(3), k2, g.row_ptr.data(), g.col_idx.data(), base.data(), m2.data(), 1 + rnd(2)};
        std::vector<int64_t> seg;
        for (int64_t p = 0; P > 0 && p < P;) {
            const int64_t b = p + rnd(20), e = b + 1 + rnd(30);
            if (e > P) break;
            seg.push_back(b);
            seg.push_back(e);
            p = e;
        }
        fgdo_opts opt{0.7f, 0.9f, rnd(2), rnd(2), static_cast<int32_t>(seg.size() / 2), seg.data()};
        // One element more than the arrays hold, so an empty array (P = 0,
        // ld = 0) still has a non-NULL base; the oracle never touches it.
        const size_t n = static_cast<size_t>(M) * ld;
        std::vector<float> tp(n + 1), tl(n + 1), mom(n + 1), x(n + 1);
        std::vector<uint16_t> tpb(n + 1), tlb(n + 1), xb(n + 1);
        for (size_t i = 0; i < n; ++i) {
            tp[i] = static_cast<float>(0.02 * normal());
            tl[i] = tp[i] + static_cast<float>(1e-3 * normal());
            mom[i] = static_cast<float>(1e-4 * normal());
            tpb[i] = fgdo_bf16_from_double(tp[i]);
            tlb[i] = fgdo_bf16_from_double(tl[i]);
        }
        void *P_tp = dtype ? static_cast<void *>(tpb.data()) : tp.data();
        void *P_tl = dtype ? static_cast<void *>(tlb.data()) : tl.data();
        void *P_x = dtype ? static_cast<void *>(xb.data()) : x.data();
        const int ncd = fgdo_num_cd(&mix1, &mix2);
        check(ncd > 0, "consensus row count", it);
        std::vector<double> cd(static_cast<size_t>(ncd) * M);
        std::vector<float> mom1(mom);
        int rc = fgdo_outer_step(M, P, ld, dtype, P_tp, P_tl, mom1.data(), &mix1, &mix2, &opt, cd.data());
        check(rc == 0, "oracle step", it, rc);
        // Split halves on fresh copies.
        std::vector<float> mom2(mom);
        std::vector<double> cd1(static_cast<size_t>(ncd) * M), cd2(static_cast<size_t>(ncd) * M);
        rc = fgdo_mix1_split(M, P, ld, dtype, P_tp, P_x, mom2.data(), &mix1, opt.mix1_state, cd1.data());
        check(rc == 0, "oracle Mix1 half", it, rc);
        rc = fgdo_outer_blocking(M, P, ld, dtype, P_x, P_tp, P_tl, mom2.data(), &mix2, &opt, rnd(2), cd2.data());
        check(rc == 0, "oracle blocking half", it, rc);
        std::vector<double> S(M);
        check(fgdo_consensus(M, P, ld, dtype, P_tp, S.data()) == 0, "oracle consensus", it);
        for (int m = 0; m < M; ++m) check(std::isfinite(S[m]) && S[m] >= 0.0, "consensus finite", it, m);
    }
    // Rejected arguments.
    float f[8] = {0};
    double d[8] = {0};
    fgdo_mix id{0, 0, nullptr, nullptr, nullptr, nullptr, 0};
    fgdo_opts opt{0.7f, 0.9f, 1, 0, 0, nullptr};
    check(fgdo_outer_step(0, 1, 1, 0, f, f, f, &id, &id, &opt, d) != 0, "oracle M = 0");
    check(fgdo_outer_step(1, 2, 1, 0, f, f, f, &id, &id, &opt, d) != 0, "oracle ld < P");
    check(fgdo_outer_step(1, 1, 1, 3, f, f, f, &id, &id, &opt, d) != 0, "oracle dtype");
    check(fgdo_outer_step(1, 1, 1, 0, nullptr, f, f, &id, &id, &opt, d) != 0, "oracle NULL");
    fgdo_mix bad{2, 1, nullptr, nullptr, nullptr, nullptr, 1};
    check(fgdo_outer_step(1, 1, 1, 0, f, f, f, &bad, &id, &opt, d) != 0, "oracle CSR without structure");
    int64_t seg_bad[2] = {3, 2};
    fgdo_opts opt2{0.7f, 0.9f, 1, 0, 1, seg_bad};
    check(fgdo_outer_step(1, 4, 4, 0, f, f, f, &id, &id, &opt2, d) != 0, "oracle empty subset segment");
}

}  // namespace

int main() {
    weights_agree();
    malformed_rejected();
    oracle_steps();
    if (g_fail) {
        std::printf("%d checks failed\n", g_fail);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
