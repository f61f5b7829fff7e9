// Host-side helpers shared by the packing code and the plan-execution code
// of libfate: input validation of clusters and DAG batches, device masks
// and a small thread pool over independent items.
#pragma once

#include <algorithm>
#include <atomic>
#include <cmath>
#include <thread>
#include <vector>

#include "fate.h"

namespace fate_host {

inline bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.0f; }
inline uint64_t dev_mask(int D) { return D >= 64 ? ~0ull : ((1ull << D) - 1ull); }

inline unsigned worker_count() {
    unsigned n = std::thread::hardware_concurrency();
    if (n == 0) n = 1;
    return std::min(n, 16u);
}

template <class F>
void parallel_for(int64_t count, F &&fn) {
    unsigned nw = worker_count();
    if (count < 4 || nw == 1) {
        for (int64_t i = 0; i < count; ++i) fn(i);
        return;
    }
    std::atomic<int64_t> next(0);
    std::vector<std::thread> ts;
    for (unsigned t = 0; t < nw; ++t)
        ts.emplace_back([&] {
            for (;;) {
                int64_t i = next.fetch_add(1);
                if (i >= count) break;
                fn(i);
            }
        });
    for (auto &t : ts) t.join();
}

inline fate_status_t validate_cluster(const fate_cluster_t *c) {
    if (!c) return FATE_EINVAL;
    if (c->D < 1 || c->D > FATE_MAX_DEVICES || c->M < 1 || c->M > FATE_MAX_MODELS) return FATE_ERANGE;
    if (!c->exec || !c->switch_s || !c->weight_bytes || !c->cap_bytes || !c->beta) return FATE_EINVAL;
    const int D = c->D, M = c->M;
    for (int i = 0; i < M * D; ++i)
        if (!finite_nonneg(c->exec[i]) || !finite_nonneg(c->switch_s[i])) return FATE_EINVAL;
    for (int i = 0; i < D * D; ++i)
        if (!finite_nonneg(c->beta[i])) return FATE_EINVAL;
    for (int m = 0; m < M; ++m)
        if (c->weight_bytes[m] <= 0) return FATE_EINVAL;
    for (int d = 0; d < D; ++d)
        if (c->cap_bytes[d] <= 0) return FATE_EINVAL;
    return FATE_OK;
}

inline std::vector<uint64_t> fit_masks(const fate_cluster_t *c) {
    std::vector<uint64_t> fits(c->M, 0);
    for (int m = 0; m < c->M; ++m)
        for (int d = 0; d < c->D; ++d)
            if (c->weight_bytes[m] <= c->cap_bytes[d]) fits[m] |= 1ull << d;
    return fits;
}

// Structural checks of the flat batch: offsets, parent order, attributes.
inline fate_status_t validate_batch(const fate_cluster_t *c, const fate_dag_batch_t *g, int64_t *N_out,
                             int64_t *E_out) {
    if (!g || g->B < 0 || !g->stage_off) return FATE_EINVAL;
    const int B = g->B;
    if (g->stage_off[0] != 0) return FATE_EINVAL;
    for (int b = 0; b < B; ++b)
        if (g->stage_off[b + 1] < g->stage_off[b]) return FATE_EINVAL;
    const int64_t N = g->stage_off[B];
    if (N > FATE_MAX_TOTAL_STAGES) return FATE_ERANGE;
    if (N > 0 && (!g->par_off || !g->model || !g->elig || !g->shard_max || !g->prefix_hash ||
                  !g->prefix_tokens || !g->out_bytes))
        return FATE_EINVAL;
    if (N > 0 && g->par_off[0] != 0) return FATE_EINVAL;
    for (int64_t i = 0; i < N; ++i)
        if (g->par_off[i + 1] < g->par_off[i]) return FATE_EINVAL;
    const int64_t E = N > 0 ? g->par_off[N] : 0;
    if (E > 0 && !g->par_idx) return FATE_EINVAL;
    if (E >= (int64_t(1) << 32)) return FATE_ERANGE;
    const std::vector<uint64_t> fits = fit_masks(c);
    const uint64_t dm = dev_mask(c->D);
    for (int b = 0; b < B; ++b) {
        const int64_t base = g->stage_off[b];
        const int64_t n = g->stage_off[b + 1] - base;
        for (int64_t v = 0; v < n; ++v) {
            const int64_t s = base + v;
            const int64_t np = g->par_off[s + 1] - g->par_off[s];
            if (np > FATE_MAX_PARENTS) return FATE_ERANGE;
            int64_t prev = -1;
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q) {
                const int64_t p = g->par_idx[q];
                if (p < 0) return FATE_EINVAL;
                if (p >= v || p <= prev) return FATE_ECYCLE;
                prev = p;
            }
            const int m = g->model[s];
            if (m < 0 || m >= c->M) return FATE_EINVAL;
            const uint64_t e = g->elig[s];
            if (e == 0 || (e & ~dm) != 0) return FATE_EINVAL;
            if (g->shard_max[s] < 1) return FATE_EINVAL;
            if (g->shard_max[s] > 255) return FATE_ERANGE;
            if (!finite_nonneg(g->prefix_tokens[s]) || !finite_nonneg(g->out_bytes[s])) return FATE_EINVAL;
            if ((e & fits[m]) == 0) return FATE_ENOFEAS;
        }
    }
    *N_out = N;
    *E_out = E;
    return FATE_OK;
}

}  // namespace fate_host
