// Plan execution and baseline placements (host side of libfate).
//
// fate_simulate executes a placement - the devices S(v) of every pending
// stage and an order key per stage - on every instance of a batch and
// reports the makespan, the p95 completion of the sink stages and the
// mechanism proxies of App. C.2 (cross-device parent edges, estimated prefix
// hits, same-model continuations).  Each device runs its stages in key
// order; processing an instance's placed stages in (key, id) order computes
// that schedule exactly when the keys respect the DAG, which is checked.  A
// shard of v on d (k = |S(v)|) starts when d is free and every parent's
// output has arrived (1/k of a remote parent's output, from its cheapest
// holder), pays the switch time if m(v) is absent (then Load), and saves
// kappa_prefix * L(v) / k of its runtime c(v, d) / k on a prefix hit; grp(v)
// then joins d's prefix slots (oldest dropped when full).
//
// fate_place_baseline builds the two comparison placements: round robin
// (each pending stage, in id order, on the next feasible device after the
// previous one) and an HEFT-style list schedule (pending stages by upward
// rank, each on the feasible device with the earliest finish under the rule
// above).  Instances are independent and run on a small thread pool.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "fate_host_common.h"

namespace {

using fate_host::dev_mask;
using fate_host::finite_nonneg;
using fate_host::parallel_for;

constexpr uint8_t kCompleted = FATE_COMPLETED;

// One instance's execution state.
struct Exec {
    const fate_cluster_t *c;
    const fate_dag_batch_t *g;
    int D, M, K;
    int64_t base, n;
    double t0, kpf;
    std::vector<double> free, fin;
    std::vector<uint64_t> res, ring, holders;
    std::vector<int> last_model;
    std::vector<char> done;
    std::vector<std::vector<int32_t>> children;

    Exec(const fate_cluster_t *c_, const fate_dag_batch_t *g_, const fate_state_t *s, int b, double kpf_)
        : c(c_), g(g_), D(c_->D), M(c_->M), K(s->K), kpf(kpf_) {
        base = g->stage_off[b];
        n = g->stage_off[b + 1] - base;
        t0 = (double)s->t_now[b];
        free.resize(D);
        res.resize(D);
        last_model.assign(D, -1);
        ring.assign((size_t)D * K, 0);
        for (int d = 0; d < D; ++d) {
            free[d] = std::max((double)s->tau_free[(int64_t)b * D + d], t0);
            res[d] = s->resident[(int64_t)b * D + d];
            for (int e = 0; e < K; ++e) ring[(size_t)d * K + e] = s->prefix_cache[((int64_t)b * D + d) * K + e];
        }
        fin.assign(n, 0.0);
        done.assign(n, 0);
        holders.assign(n, 0);
        children.assign(n, {});
        for (int64_t v = 0; v < n; ++v) {
            const int64_t gv = base + v;
            if (s->status[gv] == kCompleted) {
                fin[v] = t0;
                done[v] = 1;
                holders[v] = s->holders[gv];
            }
            for (int64_t q = g->par_off[gv]; q < g->par_off[gv + 1]; ++q) children[g->par_idx[q]].push_back((int32_t)v);
        }
    }

    bool feasible(int64_t v, int d) const {
        const int m = g->model[base + v];
        return ((g->elig[base + v] >> d) & 1ull) && c->weight_bytes[m] <= c->cap_bytes[d];
    }

    uint64_t load(uint64_t r, int m, int d) const {
        if ((r >> m) & 1ull) return r;
        r |= 1ull << m;
        int64_t total = 0;
        for (int i = 0; i < M; ++i)
            if ((r >> i) & 1ull) total += c->weight_bytes[i];
        for (int i = 0; i < M && total > c->cap_bytes[d]; ++i) {
            if (i == m || !((r >> i) & 1ull)) continue;
            r &= ~(1ull << i);
            total -= c->weight_bytes[i];
        }
        return r;
    }

    bool cached(int d, uint64_t h) const {
        if (h == 0) return false;
        for (int e = 0; e < K; ++e)
            if (ring[(size_t)d * K + e] == h) return true;
        return false;
    }

    // Finish time of v's shard on d (k shards), without side effects.
    double shard(int64_t v, int d, int k, bool &hit) const {
        const int64_t gv = base + v;
        double ready = t0;
        for (int64_t q = g->par_off[gv]; q < g->par_off[gv + 1]; ++q) {
            const int32_t u = g->par_idx[q];
            const uint64_t hu = holders[u];
            double arr;
            if ((hu >> d) & 1ull) {
                arr = fin[u];
            } else {
                double bmin = INFINITY;
                for (uint64_t t = hu; t; t &= t - 1) bmin = std::min(bmin, (double)c->beta[__builtin_ctzll(t) * D + d]);
                arr = fin[u] + (double)g->out_bytes[base + u] * bmin / k;
            }
            ready = std::max(ready, arr);
        }
        const double start = std::max(free[d], ready);
        const int m = g->model[gv];
        const double sw = ((res[d] >> m) & 1ull) ? 0.0 : (double)c->switch_s[m * D + d];
        hit = cached(d, g->prefix_hash[gv]);
        double run = (double)c->exec[m * D + d] / k;
        if (hit) run = std::max(0.0, run - kpf * (double)g->prefix_tokens[gv] / k);
        return start + sw + run;
    }

    void ring_push(int d, uint64_t h) {
        if (h == 0 || K == 0 || cached(d, h)) return;
        uint64_t *r = &ring[(size_t)d * K];
        for (int e = 0; e < K; ++e)
            if (r[e] == 0) {
                r[e] = h;
                return;
            }
        for (int e = 0; e + 1 < K; ++e) r[e] = r[e + 1];
        r[K - 1] = h;
    }

    // Execute v on S; returns whether its first device hit the prefix cache
    // and continued the same model.
    void run(int64_t v, uint64_t S, bool &hit0, bool &cont0) {
        const int k = __builtin_popcountll(S);
        const int m = g->model[base + v];
        double f = t0;
        bool first = true;
        for (uint64_t t = S; t; t &= t - 1) {
            const int d = __builtin_ctzll(t);
            bool hit;
            const double fd = shard(v, d, k, hit);
            if (first) {
                hit0 = hit;
                cont0 = last_model[d] == m;
                first = false;
            }
            free[d] = fd;
            res[d] = load(res[d], m, d);
            ring_push(d, g->prefix_hash[base + v]);
            last_model[d] = m;
            f = std::max(f, fd);
        }
        fin[v] = f;
        holders[v] = S;
        done[v] = 1;
    }
};

fate_status_t check_state(const fate_cluster_t *c, const fate_dag_batch_t *g, const fate_state_t *s, int64_t N) {
    if (!s || s->K < 0 || s->K > FATE_MAX_PREFIX_SLOTS) return FATE_EINVAL;
    const int B = g->B, D = c->D;
    if (B > 0 && (!s->resident || !s->tau_free || !s->t_now || (s->K > 0 && !s->prefix_cache))) return FATE_EINVAL;
    if (N > 0 && (!s->holders || !s->status)) return FATE_EINVAL;
    for (int64_t i = 0; i < (int64_t)B * D; ++i)
        if (!std::isfinite(s->tau_free[i])) return FATE_EINVAL;
    for (int b = 0; b < B; ++b)
        if (!std::isfinite(s->t_now[b])) return FATE_EINVAL;
    const uint64_t dm = dev_mask(D);
    for (int64_t i = 0; i < N; ++i) {
        if (s->status[i] != FATE_PENDING && s->status[i] != kCompleted) return FATE_ESTATE;
        if ((s->status[i] == kCompleted) != (s->holders[i] != 0)) return FATE_ESTATE;
        if (s->holders[i] & ~dm) return FATE_ESTATE;
    }
    return FATE_OK;
}

fate_status_t check_inputs(const fate_cluster_t *c, const fate_dag_batch_t *g, const fate_state_t *s) {
    fate_status_t st = fate_host::validate_cluster(c);
    if (st != FATE_OK) return st;
    int64_t N = 0, E = 0;
    st = fate_host::validate_batch(c, g, &N, &E);
    if (st != FATE_OK) return st;
    return check_state(c, g, s, N);
}

}  // namespace

extern "C" {

fate_status_t fate_simulate(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, const fate_state_t *state,
                            const uint64_t *devices, const int64_t *order, float kappa_prefix,
                            fate_sim_metrics_t *out) {
    fate_status_t st = check_inputs(cluster, dags, state);
    if (st != FATE_OK) return st;
    const int64_t N = dags->stage_off[dags->B];
    if ((N > 0 && (!devices || !order)) || (dags->B > 0 && !out) || !finite_nonneg(kappa_prefix)) return FATE_EINVAL;
    const uint64_t dm = dev_mask(cluster->D);
    for (int64_t i = 0; i < N; ++i)
        if (devices[i] & ~dm) return FATE_EINVAL;
    std::vector<fate_status_t> rc(dags->B, FATE_OK);
    parallel_for(dags->B, [&](int64_t b) {
        Exec x(cluster, dags, state, (int)b, (double)kappa_prefix);
        std::vector<int64_t> todo;
        for (int64_t v = 0; v < x.n; ++v)
            if (!x.done[v] && devices[x.base + v] != 0) todo.push_back(v);
        std::sort(todo.begin(), todo.end(), [&](int64_t p, int64_t q) {
            const int64_t kp = order[x.base + p], kq = order[x.base + q];
            return kp != kq ? kp < kq : p < q;
        });
        fate_sim_metrics_t m;
        std::memset(&m, 0, sizeof(m));
        for (int64_t v : todo) {
            const uint64_t S = devices[x.base + v];
            for (int64_t q = dags->par_off[x.base + v]; q < dags->par_off[x.base + v + 1]; ++q) {
                const int32_t u = dags->par_idx[q];
                if (!x.done[u]) {  // the order runs v before a parent
                    rc[b] = FATE_ESTATE;
                    return;
                }
                m.xdev_edges += (x.holders[u] & S) == 0 ? 1 : 0;
            }
            bool hit = false, cont = false;
            x.run(v, S, hit, cont);
            m.tasks += 1;
            m.cache_hits += hit ? 1 : 0;
            m.model_cont += cont ? 1 : 0;
        }
        double last = x.t0;
        std::vector<double> sinks;
        for (int64_t v : todo) {
            last = std::max(last, x.fin[v]);
            if (x.children[v].empty()) sinks.push_back(x.fin[v] - x.t0);
        }
        m.makespan = last - x.t0;
        if (!sinks.empty()) {
            std::sort(sinks.begin(), sinks.end());
            const int64_t r = (int64_t)std::ceil(0.95 * (double)sinks.size());
            m.p95 = sinks[(size_t)std::max<int64_t>(0, r - 1)];
        }
        out[b] = m;
    });
    for (fate_status_t r : rc)
        if (r != FATE_OK) return r;
    return FATE_OK;
}

fate_status_t fate_place_baseline(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                  const fate_state_t *state, int32_t policy, float kappa_prefix, uint64_t *devices,
                                  int64_t *order) {
    if (policy != FATE_PLACE_ROUND_ROBIN && policy != FATE_PLACE_HEFT) return FATE_EINVAL;
    fate_status_t st = check_inputs(cluster, dags, state);
    if (st != FATE_OK) return st;
    const int64_t N = dags->stage_off[dags->B];
    if ((N > 0 && (!devices || !order)) || !finite_nonneg(kappa_prefix)) return FATE_EINVAL;
    const int D = cluster->D;
    double bmean = 0.0;
    int nb = 0;
    for (int i = 0; i < D; ++i)
        for (int j = 0; j < D; ++j)
            if (i != j) {
                bmean += (double)cluster->beta[i * D + j];
                ++nb;
            }
    bmean = nb ? bmean / nb : 0.0;
    parallel_for(dags->B, [&](int64_t b) {
        Exec x(cluster, dags, state, (int)b, (double)kappa_prefix);
        for (int64_t v = 0; v < x.n; ++v) {
            devices[x.base + v] = 0;
            order[x.base + v] = 0;
        }
        if (policy == FATE_PLACE_ROUND_ROBIN) {
            int nxt = 0;
            for (int64_t v = 0; v < x.n; ++v) {
                if (x.done[v]) continue;
                for (int q = 0; q < D; ++q) {
                    const int d = (nxt + q) % D;
                    if (x.feasible(v, d)) {
                        devices[x.base + v] = 1ull << d;
                        nxt = d + 1;
                        break;
                    }
                }
                order[x.base + v] = v;
            }
            return;
        }
        // HEFT-style: upward ranks (children have larger ids), then earliest finish
        std::vector<double> rank(x.n, 0.0);
        for (int64_t v = x.n - 1; v >= 0; --v) {
            const int m = dags->model[x.base + v];
            double wsum = 0.0;
            int nf = 0;
            for (int d = 0; d < D; ++d)
                if (x.feasible(v, d)) {
                    wsum += (double)cluster->exec[m * D + d];
                    ++nf;
                }
            double tail = 0.0;
            bool any = false;
            for (int32_t ch : x.children[v]) {
                const double t = (double)dags->out_bytes[x.base + v] * bmean + rank[ch];
                tail = any ? std::max(tail, t) : t;
                any = true;
            }
            rank[v] = wsum / nf + tail;
        }
        std::vector<int64_t> todo;
        for (int64_t v = 0; v < x.n; ++v)
            if (!x.done[v]) todo.push_back(v);
        std::sort(todo.begin(), todo.end(), [&](int64_t p, int64_t q) {
            return rank[p] != rank[q] ? rank[p] > rank[q] : p < q;
        });
        for (size_t pos = 0; pos < todo.size(); ++pos) {
            const int64_t v = todo[pos];
            int best = -1;
            double bf = INFINITY;
            for (int d = 0; d < D; ++d) {
                if (!x.feasible(v, d)) continue;
                bool hit;
                const double f = x.shard(v, d, 1, hit);
                if (f < bf) {
                    best = d;
                    bf = f;
                }
            }
            bool h0, c0;
            x.run(v, 1ull << best, h0, c0);
            devices[x.base + v] = 1ull << best;
            order[x.base + v] = (int64_t)pos;
        }
    });
    return FATE_OK;
}

}  // extern "C"
