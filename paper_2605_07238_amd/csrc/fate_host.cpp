// Host half of libfate: validation, packing of DAG batches and states into
// flat device images, and the C ABI entry points declared in fate.h.
//
// Packing does no scoring arithmetic.  It checks the inputs, lays out the
// stage records and parent lists, derives each stage's horizon descendants
// (breadth-first levels 1..H below it, Sec. 3.3) and the ready frontier
// (pending stages whose parents are all completed, Sec. 2 / App. A.1), and
// copies the image to the caller's device buffer.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "fate_host_common.h"
#include "fate_internal.h"

namespace {

// memcpy for byte counts that may be 0 (the source of an empty copy may be null)
void copy_bytes(void *dst, const void *src, size_t n) {
    if (n) std::memcpy(dst, src, n);
}

using fate::StageRec;
using fate_host::dev_mask;
using fate_host::finite_nonneg;
using fate_host::fit_masks;
using fate_host::parallel_for;
using fate_host::validate_batch;
using fate_host::validate_cluster;

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// ---------------------------------------------------------------------------
// horizon descendants
// ---------------------------------------------------------------------------

// Horizon descendants of every stage of instance b (Sec. 3.3): with
// FATE_LEVELS_HOP the stages at breadth-first distance 1..H, each at its
// minimum distance; with FATE_LEVELS_TOPO the stages reachable from v whose
// topological level (longest path from a stage without parents) exceeds v's
// by 1..H, at that difference.  With `out`, stores each stage's entries (flat
// id | depth << 28) ordered by (depth, id); always stores the per-stage
// counts into count[] (indexed by flat id).
void instance_horizons(const fate_dag_batch_t *g, int b, int H, int levels, uint32_t *count,
                       std::vector<uint32_t> *out) {
    const int64_t base = g->stage_off[b];
    const int64_t n = g->stage_off[b + 1] - base;
    if (n == 0) return;
    std::vector<int64_t> cptr(n + 1, 0);
    for (int64_t v = 0; v < n; ++v)
        for (int64_t q = g->par_off[base + v]; q < g->par_off[base + v + 1]; ++q) cptr[g->par_idx[q] + 1]++;
    for (int64_t v = 0; v < n; ++v) cptr[v + 1] += cptr[v];
    std::vector<int32_t> cidx(cptr[n]);
    std::vector<int64_t> fill(cptr.begin(), cptr.end() - 1);
    for (int64_t v = 0; v < n; ++v)
        for (int64_t q = g->par_off[base + v]; q < g->par_off[base + v + 1]; ++q)
            cidx[fill[g->par_idx[q]]++] = (int32_t)v;
    std::vector<int64_t> stamp(n, -1);
    std::vector<int32_t> cur, nxt;
    if (out) out->clear();
    if (levels == FATE_LEVELS_TOPO) {
        std::vector<int32_t> lv(n, 0);  // parents have smaller ids
        for (int64_t v = 0; v < n; ++v)
            for (int64_t q = g->par_off[base + v]; q < g->par_off[base + v + 1]; ++q)
                lv[v] = std::max(lv[v], lv[g->par_idx[q]] + 1);
        std::vector<int32_t> reach;
        for (int64_t v = 0; v < n; ++v) {
            // levels rise along every edge, so nothing below a stage past the
            // window is inside it
            reach.clear();
            stamp[v] = v;
            cur.assign(1, (int32_t)v);
            while (!cur.empty()) {
                nxt.clear();
                for (int32_t x : cur)
                    for (int64_t q = cptr[x]; q < cptr[x + 1]; ++q) {
                        const int32_t c = cidx[q];
                        if (stamp[c] == v || lv[c] - lv[v] > H) continue;
                        stamp[c] = v;
                        nxt.push_back(c);
                        reach.push_back(c);
                    }
                cur.swap(nxt);
            }
            std::sort(reach.begin(), reach.end(), [&](int32_t x, int32_t y) {
                return lv[x] != lv[y] ? lv[x] < lv[y] : x < y;
            });
            count[base + v] = (uint32_t)reach.size();
            if (out)
                for (int32_t c : reach)
                    out->push_back((uint32_t)(base + c) | ((uint32_t)(lv[c] - lv[v]) << fate::kDescDepthShift));
        }
        return;
    }
    for (int64_t v = 0; v < n; ++v) {
        uint32_t cnt = 0;
        stamp[v] = v;
        cur.assign(1, (int32_t)v);
        for (int h = 1; h <= H && !cur.empty(); ++h) {
            nxt.clear();
            for (int32_t x : cur)
                for (int64_t q = cptr[x]; q < cptr[x + 1]; ++q) {
                    const int32_t c = cidx[q];
                    if (stamp[c] == v) continue;
                    stamp[c] = v;
                    nxt.push_back(c);
                }
            std::sort(nxt.begin(), nxt.end());
            cnt += (uint32_t)nxt.size();
            if (out)
                for (int32_t c : nxt)
                    out->push_back((uint32_t)(base + c) | ((uint32_t)h << fate::kDescDepthShift));
            cur.swap(nxt);
        }
        count[base + v] = cnt;
    }
}

struct DagLayout {
    size_t exec, ksw, beta, weight, cap, fits, stage_off, rec, rowrec, par, desc_off, desc, desc_w, ch_off, ch_idx, total;
};

// Whether the batch gets 16-byte row records: the row kernel for at most 16
// devices and 32 models reads them, and their packed word holds |Pa(v)| in 11 bits.
inline bool row_records_fit(int D, int M, int64_t max_npar) {
    return D <= 16 && M <= 32 && max_npar <= fate::kRowRecMaxNpar;
}

// desc_w (one float per horizon entry) only with level weights
DagLayout dag_layout(int B, int D, int M, int64_t N, int64_t E, int64_t ndesc, bool level_weights, bool rows) {
    DagLayout L;
    size_t o = 0;
    L.exec = o; o = align_up(o + sizeof(float) * M * D);
    L.ksw = o; o = align_up(o + sizeof(float) * M * D);
    L.beta = o; o = align_up(o + sizeof(float) * D * D);
    L.weight = o; o = align_up(o + sizeof(uint64_t) * M);
    L.cap = o; o = align_up(o + sizeof(uint64_t) * D);
    L.fits = o; o = align_up(o + sizeof(uint64_t) * M);
    L.stage_off = o; o = align_up(o + sizeof(int64_t) * (B + 1));
    L.rec = o; o = align_up(o + sizeof(StageRec) * N);
    L.rowrec = o; o = align_up(o + (rows ? sizeof(fate::RowRec) * N : 0));
    L.par = o; o = align_up(o + sizeof(uint32_t) * E);
    L.desc_off = o; o = align_up(o + sizeof(uint32_t) * (N + 1));
    L.desc = o; o = align_up(o + sizeof(uint32_t) * ndesc);
    L.desc_w = o; o = align_up(o + (level_weights ? sizeof(float) * ndesc : 0));
    L.ch_off = o; o = align_up(o + sizeof(uint32_t) * (N + 1));
    L.ch_idx = o; o = align_up(o + sizeof(uint32_t) * E);
    L.total = o;
    return L;
}

struct DagsPlan {
    int64_t N = 0, E = 0, ndesc = 0, max_npar = 0;
    bool rows = false;  // row records (row_records_fit)
    std::vector<uint32_t> count;
    std::vector<std::vector<uint32_t>> lists;  // per instance, when building
};

bool opts_ok(const fate_pack_opts_t *o) {
    return o && (o->levels == FATE_LEVELS_HOP || o->levels == FATE_LEVELS_TOPO) &&
           (o->level_weights == 0 || o->level_weights == 1);
}

fate_status_t plan_dags(const fate_cluster_t *c, const fate_dag_batch_t *g, const fate_pack_opts_t &o, bool keep,
                        DagsPlan *p) {
    fate_status_t st = validate_cluster(c);
    if (st != FATE_OK) return st;
    const int H = o.H;
    if (H < 0 || H > FATE_MAX_HORIZON) return FATE_ERANGE;
    st = validate_batch(c, g, &p->N, &p->E);
    if (st != FATE_OK) return st;
    for (int64_t s = 0; s < p->N; ++s) p->max_npar = std::max(p->max_npar, g->par_off[s + 1] - g->par_off[s]);
    p->rows = row_records_fit(c->D, c->M, p->max_npar);
    p->count.assign(p->N, 0);
    if (keep) p->lists.assign(g->B, {});
    parallel_for(g->B, [&](int64_t b) {
        instance_horizons(g, (int)b, H, o.levels, p->count.data(), keep ? &p->lists[b] : nullptr);
    });
    int64_t tot = 0;
    for (uint32_t x : p->count) tot += x;
    if (tot >= (int64_t(1) << 32)) return FATE_ERANGE;
    p->ndesc = tot;
    return FATE_OK;
}

void fill_dags_handle(const fate_cluster_t *c, const fate_dag_batch_t *g, const fate_pack_opts_t &o,
                      const DagsPlan &p, const DagLayout &L, uint8_t *base, size_t bytes, fate_dags_t *out) {
    std::memset(out, 0, sizeof(*out));
    out->B = g->B;
    out->D = c->D;
    out->M = c->M;
    out->H = o.H;
    out->levels = o.levels;
    out->desc_w = o.level_weights ? reinterpret_cast<const float *>(base + L.desc_w) : nullptr;
    out->N = p.N;
    out->E = p.E;
    out->n_desc = p.ndesc;
    int uniform = 1;
    float b0 = 0.0f;
    bool first = true;
    for (int i = 0; i < c->D; ++i)
        for (int j = 0; j < c->D; ++j) {
            if (i == j) continue;
            float x = c->beta[i * c->D + j];
            if (first) { b0 = x; first = false; }
            else if (std::memcmp(&x, &b0, sizeof(float)) != 0) uniform = 0;
        }
    out->beta_uniform = uniform;
    out->beta0 = b0;
    int32_t max_r = 1;
    for (int64_t i = 0; i < p.N; ++i) max_r = std::max(max_r, (int32_t)g->shard_max[i]);
    out->max_r = max_r;
    int64_t max_stages = 0;
    for (int b = 0; b < g->B; ++b) max_stages = std::max(max_stages, g->stage_off[b + 1] - g->stage_off[b]);
    out->max_stages = max_stages;
    out->base = base;
    out->bytes = bytes;
    out->exec = reinterpret_cast<const float *>(base + L.exec);
    out->switch_s = reinterpret_cast<const float *>(base + L.ksw);
    out->beta = reinterpret_cast<const float *>(base + L.beta);
    out->weight = reinterpret_cast<const uint64_t *>(base + L.weight);
    out->cap = reinterpret_cast<const uint64_t *>(base + L.cap);
    out->fits = reinterpret_cast<const uint64_t *>(base + L.fits);
    out->stage_off = reinterpret_cast<const int64_t *>(base + L.stage_off);
    out->records = base + L.rec;
    out->par_idx = reinterpret_cast<const uint32_t *>(base + L.par);
    out->desc_off = reinterpret_cast<const uint32_t *>(base + L.desc_off);
    out->desc = reinterpret_cast<const uint32_t *>(base + L.desc);
    out->ch_off = reinterpret_cast<const uint32_t *>(base + L.ch_off);
    out->ch_idx = reinterpret_cast<const uint32_t *>(base + L.ch_idx);
    out->row_records = p.rows ? base + L.rowrec : nullptr;
}

void write_dags_image(const fate_cluster_t *c, const fate_dag_batch_t *g, const DagsPlan &p,
                      const DagLayout &L, bool level_weights, uint8_t *img) {
    float *wts = level_weights ? reinterpret_cast<float *>(img + L.desc_w) : nullptr;
    const int D = c->D, M = c->M;
    copy_bytes(img + L.exec, c->exec, sizeof(float) * M * D);
    copy_bytes(img + L.ksw, c->switch_s, sizeof(float) * M * D);
    copy_bytes(img + L.beta, c->beta, sizeof(float) * D * D);
    uint64_t *w = reinterpret_cast<uint64_t *>(img + L.weight);
    uint64_t *cp = reinterpret_cast<uint64_t *>(img + L.cap);
    uint64_t *ft = reinterpret_cast<uint64_t *>(img + L.fits);
    const std::vector<uint64_t> fits = fit_masks(c);
    for (int m = 0; m < M; ++m) { w[m] = (uint64_t)c->weight_bytes[m]; ft[m] = fits[m]; }
    for (int d = 0; d < D; ++d) cp[d] = (uint64_t)c->cap_bytes[d];
    copy_bytes(img + L.stage_off, g->stage_off, sizeof(int64_t) * (g->B + 1));
    StageRec *rec = reinterpret_cast<StageRec *>(img + L.rec);
    uint32_t *par = reinterpret_cast<uint32_t *>(img + L.par);
    uint32_t *doff = reinterpret_cast<uint32_t *>(img + L.desc_off);
    uint32_t *desc = reinterpret_cast<uint32_t *>(img + L.desc);
    uint32_t acc = 0;
    for (int64_t s = 0; s < p.N; ++s) { doff[s] = acc; acc += p.count[s]; }
    doff[p.N] = acc;
    parallel_for(g->B, [&](int64_t b) {
        const int64_t base = g->stage_off[b];
        const int64_t n = g->stage_off[b + 1] - base;
        for (int64_t v = 0; v < n; ++v) {
            const int64_t s = base + v;
            StageRec r;
            r.elig = g->elig[s];
            r.hash = g->prefix_hash[s];
            r.tokens = g->prefix_tokens[s];
            r.sigma = g->out_bytes[s];
            r.par_begin = (uint32_t)g->par_off[s];
            r.model = (uint8_t)g->model[s];
            r.shard = (uint8_t)g->shard_max[s];
            r.npar = (uint16_t)(g->par_off[s + 1] - g->par_off[s]);
            rec[s] = r;
            if (p.rows) {
                fate::RowRec rr;
                rr.hash = r.hash;
                rr.tokens = r.tokens;
                rr.meta = (uint32_t)(r.elig & 0xffffull) | ((uint32_t)r.model << 16) | ((uint32_t)r.npar << 21);
                reinterpret_cast<fate::RowRec *>(img + L.rowrec)[s] = rr;
            }
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q) par[q] = (uint32_t)(base + g->par_idx[q]);
        }
        if (n > 0 && !p.lists[b].empty())
            copy_bytes(desc + doff[base], p.lists[b].data(), sizeof(uint32_t) * p.lists[b].size());
    });
    // children lists: stages visited in ascending id append themselves to
    // their parents' lists, so every list ascends
    uint32_t *choff = reinterpret_cast<uint32_t *>(img + L.ch_off);
    uint32_t *chidx = reinterpret_cast<uint32_t *>(img + L.ch_idx);
    for (int b = 0; b < g->B; ++b)
        for (int64_t s = g->stage_off[b]; s < g->stage_off[b + 1]; ++s)
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q) ++choff[g->stage_off[b] + g->par_idx[q]];
    uint32_t run = 0;
    for (int64_t s = 0; s <= p.N; ++s) {
        const uint32_t c = s < p.N ? choff[s] : 0u;
        choff[s] = run;
        run += c;
    }
    std::vector<uint32_t> fillc(choff, choff + p.N);
    for (int b = 0; b < g->B; ++b)
        for (int64_t s = g->stage_off[b]; s < g->stage_off[b + 1]; ++s)
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q)
                chidx[fillc[g->stage_off[b] + g->par_idx[q]]++] = (uint32_t)s;
    if (!wts) return;
    // level weights: 1 / (number of v's horizon stages at that depth), for
    // the mean-per-level tail; the entries of a stage are ordered by depth
    parallel_for(p.N, [&](int64_t s) {
        uint32_t e = doff[s];
        while (e < doff[s + 1]) {
            uint32_t f = e;
            while (f < doff[s + 1] && (desc[f] >> fate::kDescDepthShift) == (desc[e] >> fate::kDescDepthShift)) ++f;
            const float w = 1.0f / (float)(f - e);
            for (uint32_t q = e; q < f; ++q) wts[q] = w;
            e = f;
        }
    });
}

// ---------------------------------------------------------------------------
// state
// ---------------------------------------------------------------------------

inline int shard_cap(int R, int max_shard, int D) { return std::max(1, std::min(std::min(R, max_shard), D)); }
inline int64_t candidates_of(int r, int D) {
    int64_t c = D;
    for (int k = 2; k <= r; ++k) c += D - k + 1;
    return c;
}

struct StatePlan {
    std::vector<uint32_t> frontier;  // pairs
    std::vector<uint32_t> cand_off;
    std::vector<uint32_t> slices;    // triples
    std::vector<uint32_t> fr_off;    // [B+1]
    std::vector<uint32_t> order;     // [B]: by decreasing frontier size, ties by instance
    std::vector<uint32_t> done_n;    // [N]
    std::vector<fate::DoneParent> done;  // [E]: stage s's slots from par_off[s]
    int64_t nF = 0, nC = 0, nS = 0;
};

fate_status_t plan_state(const fate_dags_t *pk, const fate_dag_batch_t *g, const fate_state_t *st,
                         int max_shard, StatePlan *p) {
    if (!pk || !g || !st) return FATE_EINVAL;
    if (max_shard < 1 || max_shard > FATE_MAX_SHARD) return FATE_ERANGE;
    if (st->K < 0 || st->K > FATE_MAX_PREFIX_SLOTS) return FATE_ERANGE;
    if (g->B != pk->B || !g->stage_off || g->stage_off[g->B] != pk->N) return FATE_ESTATE;
    const int B = g->B, D = pk->D, K = st->K;
    const int64_t N = pk->N;
    if (B > 0 && (!st->resident || !st->tau_free || !st->t_now)) return FATE_EINVAL;
    if (N > 0 && (!st->holders || !st->status || !g->par_off || !g->shard_max)) return FATE_EINVAL;
    if (pk->E > 0 && !g->par_idx) return FATE_EINVAL;
    if (B > 0 && K > 0 && !st->prefix_cache) return FATE_EINVAL;
    if (N > 0 && g->par_off[N] != pk->E) return FATE_ESTATE;
    const uint64_t mm = pk->M >= 64 ? ~0ull : ((1ull << pk->M) - 1ull);
    const uint64_t dm = dev_mask(D);
    for (int64_t i = 0; i < (int64_t)B * D; ++i) {
        if (st->resident[i] & ~mm) return FATE_EINVAL;
        if (!std::isfinite(st->tau_free[i])) return FATE_EINVAL;
    }
    for (int b = 0; b < B; ++b)
        if (!std::isfinite(st->t_now[b])) return FATE_EINVAL;
    p->cand_off.clear();
    p->frontier.clear();
    p->slices.clear();
    p->fr_off.assign(B + 1, 0);
    const int64_t slice = fate::slice_len(D);
    int64_t nc = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t base = g->stage_off[b];
        const int64_t n = g->stage_off[b + 1] - base;
        const int64_t first = (int64_t)p->frontier.size() / 2;
        p->fr_off[b] = (uint32_t)first;
        for (int64_t v = 0; v < n; ++v) {
            const int64_t s = base + v;
            const uint8_t status = st->status[s];
            const uint64_t hold = st->holders[s];
            if (status > FATE_COMMITTED) return FATE_EINVAL;
            if (hold & ~dm) return FATE_ESTATE;
            if ((status == FATE_COMPLETED) != (hold != 0)) return FATE_ESTATE;
            bool parents_done = true;
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q) {
                const int64_t u = g->par_idx[q];
                if (u < 0 || u >= v) return FATE_ECYCLE;
                if (st->status[base + u] != FATE_COMPLETED) parents_done = false;
            }
            if ((status == FATE_COMPLETED || status == FATE_RUNNING) && !parents_done) return FATE_ESTATE;
            if (status == FATE_PENDING && parents_done) {
                p->frontier.push_back((uint32_t)s);
                p->frontier.push_back((uint32_t)b);
                p->cand_off.push_back((uint32_t)nc);
                nc += candidates_of(shard_cap(g->shard_max[s], max_shard, D), D);
                if (nc >= (int64_t(1) << 32)) return FATE_ERANGE;
            }
        }
    }
    p->fr_off[B] = (uint32_t)(p->frontier.size() / 2);
    // per-instance launches take the largest frontiers first, so that the
    // last workgroups to start are short ones; the scoring slices follow the
    // same order where the general scoring kernel uses them
    p->order.resize(B);
    uint32_t mx = 0;
    for (int b = 0; b < B; ++b) {
        p->order[b] = (uint32_t)b;
        mx = std::max(mx, p->fr_off[b + 1] - p->fr_off[b]);
    }
    std::stable_sort(p->order.begin(), p->order.end(), [&](uint32_t x, uint32_t y) {
        return fate::order_class(p->fr_off[x + 1] - p->fr_off[x], mx) <
               fate::order_class(p->fr_off[y + 1] - p->fr_off[y], mx);
    });
    const bool in_order = !fate::rows_batch(pk, max_shard, K);
    for (int i = 0; i < B; ++i) {
        const uint32_t b = in_order ? p->order[i] : (uint32_t)i;
        const int64_t first = p->fr_off[b], last = p->fr_off[b + 1];
        for (int64_t f = first; f < last; f += slice) {
            p->slices.push_back(b);
            p->slices.push_back((uint32_t)f);
            p->slices.push_back((uint32_t)std::min(last, f + slice));
        }
    }
    p->nS = (int64_t)p->slices.size() / 3;
    // completed parents of every pending stage (only pending stages are
    // scored, in the frontier or in a horizon), with their holders and
    // sizes, in the first of the stage's parent slots
    p->done_n.assign(N, 0);
    fate::DoneParent zero;
    zero.holders = 0;
    zero.sigma = 0.0f;
    zero.pad = 0;
    p->done.assign(pk->E, zero);
    for (int b = 0; b < B; ++b) {
        const int64_t base = g->stage_off[b];
        for (int64_t s = base; s < g->stage_off[b + 1]; ++s) {
            if (st->status[s] != FATE_PENDING) continue;
            uint32_t k = 0;
            for (int64_t q = g->par_off[s]; q < g->par_off[s + 1]; ++q) {
                const int64_t u = base + g->par_idx[q];
                if (st->holders[u] == 0) continue;
                fate::DoneParent &e = p->done[g->par_off[s] + k++];
                e.holders = st->holders[u];
                e.sigma = g->out_bytes[u];
            }
            p->done_n[s] = k;
        }
    }
    p->cand_off.push_back((uint32_t)nc);
    p->nF = (int64_t)p->frontier.size() / 2;
    p->nC = nc;
    return FATE_OK;
}

struct StateLayout {
    size_t resident, pcache, holders, tau, tnow, frontier, cand_off, slices, done_n, done, fr_off, order, status,
        finish, counts, total;
};

// Section sizes: nF frontier slots, nS slices (the exact counts, or the
// capacities of a planning state, which also carries the stage statuses and
// the device counters), nDone = E completed-parent slots.
StateLayout state_layout(int B, int D, int K, int64_t N, int64_t nF, int64_t nS, int64_t nDone,
                         bool advance = false) {
    StateLayout L;
    size_t o = 0;
    L.resident = o; o = align_up(o + sizeof(uint64_t) * B * D);
    L.pcache = o; o = align_up(o + sizeof(uint64_t) * (size_t)B * D * K);
    L.holders = o; o = align_up(o + sizeof(uint64_t) * N);
    L.tau = o; o = align_up(o + sizeof(float) * B * D);
    L.tnow = o; o = align_up(o + sizeof(float) * B);
    L.frontier = o; o = align_up(o + sizeof(uint32_t) * 2 * nF);
    L.cand_off = o; o = align_up(o + sizeof(uint32_t) * (nF + 1));
    L.slices = o; o = align_up(o + sizeof(uint32_t) * 3 * nS);
    L.done_n = o; o = align_up(o + sizeof(uint32_t) * N);
    L.done = o; o = align_up(o + sizeof(fate::DoneParent) * nDone);
    L.fr_off = o; o = align_up(o + sizeof(uint32_t) * (B + 1));
    L.order = o; o = align_up(o + sizeof(uint32_t) * B);
    L.status = o;
    if (advance) o = align_up(o + (size_t)N);
    L.finish = o;
    if (advance) o = align_up(o + sizeof(float) * (size_t)N);
    L.counts = o;
    if (advance) o = align_up(o + 4 * sizeof(uint32_t));
    L.total = o;
    return L;
}

// Capacities of a planning state: every pending stage may join the frontier
// later, every parent may complete.
struct AdvanceCaps {
    int64_t nF = 0, nC = 0, nS = 0, nDone = 0;
};
fate_status_t advance_caps(const fate_dags_t *pk, const fate_dag_batch_t *g, const fate_state_t *st,
                           int max_shard, AdvanceCaps *c) {
    const int64_t slice = fate::slice_len(pk->D);
    for (int b = 0; b < pk->B; ++b) {
        int64_t pend = 0;
        for (int64_t s = g->stage_off[b]; s < g->stage_off[b + 1]; ++s) {
            if (st->status[s] != FATE_PENDING) continue;
            ++pend;
            c->nC += candidates_of(shard_cap(g->shard_max[s], max_shard, pk->D), pk->D);
        }
        c->nF += pend;
        c->nS += (pend + slice - 1) / slice;
    }
    c->nDone = pk->E;
    if (c->nC >= (int64_t(1) << 32)) return FATE_ERANGE;
    return FATE_OK;
}

void write_state_image(const fate_dags_t *pk, const fate_dag_batch_t *g, const fate_state_t *st, const StatePlan &p,
                       const StateLayout &L, uint8_t *img) {
    const int B = pk->B, D = pk->D, K = st->K;
    copy_bytes(img + L.resident, st->resident, sizeof(uint64_t) * B * D);
    copy_bytes(img + L.pcache, st->prefix_cache, sizeof(uint64_t) * (size_t)B * D * K);
    copy_bytes(img + L.holders, st->holders, sizeof(uint64_t) * pk->N);
    copy_bytes(img + L.tau, st->tau_free, sizeof(float) * B * D);
    copy_bytes(img + L.tnow, st->t_now, sizeof(float) * B);
    copy_bytes(img + L.frontier, p.frontier.data(), sizeof(uint32_t) * p.frontier.size());
    copy_bytes(img + L.cand_off, p.cand_off.data(), sizeof(uint32_t) * p.cand_off.size());
    copy_bytes(img + L.slices, p.slices.data(), sizeof(uint32_t) * p.slices.size());
    copy_bytes(img + L.done_n, p.done_n.data(), sizeof(uint32_t) * p.done_n.size());
    copy_bytes(img + L.done, p.done.data(), sizeof(fate::DoneParent) * p.done.size());
    copy_bytes(img + L.fr_off, p.fr_off.data(), sizeof(uint32_t) * p.fr_off.size());
    copy_bytes(img + L.order, p.order.data(), sizeof(uint32_t) * p.order.size());
    if (L.counts > L.status) {  // planning state
        copy_bytes(img + L.status, st->status, (size_t)pk->N);
        // planned finish: t for the stages completed when planning begins
        float *fin = reinterpret_cast<float *>(img + L.finish);
        for (int b = 0; b < B; ++b)
            for (int64_t s = g->stage_off[b]; s < g->stage_off[b + 1]; ++s)
                fin[s] = st->status[s] == FATE_COMPLETED ? st->t_now[b] : 0.0f;
        const uint32_t counts[4] = {(uint32_t)p.nF, (uint32_t)p.nC, (uint32_t)p.nS, 0u};
        std::memcpy(img + L.counts, counts, sizeof(counts));
    }
}

void fill_state_handle(const fate_dags_t *pk, const fate_state_t *st, int max_shard, const StatePlan &p,
                       const StateLayout &L, uint8_t *base, size_t bytes, fate_state_h *out) {
    std::memset(out, 0, sizeof(*out));
    out->B = pk->B;
    out->D = pk->D;
    out->K = st->K;
    out->max_shard = max_shard;
    out->N = pk->N;
    out->n_frontier = p.nF;
    out->n_cand = p.nC;
    out->base = base;
    out->bytes = bytes;
    out->resident = reinterpret_cast<const uint64_t *>(base + L.resident);
    out->prefix_cache = reinterpret_cast<const uint64_t *>(base + L.pcache);
    out->holders = reinterpret_cast<const uint64_t *>(base + L.holders);
    out->tau_free = reinterpret_cast<const float *>(base + L.tau);
    out->t_now = reinterpret_cast<const float *>(base + L.tnow);
    out->frontier = reinterpret_cast<const uint32_t *>(base + L.frontier);
    out->cand_off = reinterpret_cast<const uint32_t *>(base + L.cand_off);
    out->n_slices = p.nS;
    out->slices = reinterpret_cast<const uint32_t *>(base + L.slices);
    out->n_done_edges = (int64_t)p.done.size();
    out->done_n = reinterpret_cast<const uint32_t *>(base + L.done_n);
    out->done = base + L.done;
    out->fr_off = reinterpret_cast<const uint32_t *>(base + L.fr_off);
    out->order = reinterpret_cast<const uint32_t *>(base + L.order);
    out->slice = (int32_t)fate::slice_len(pk->D);
}

void fill_advance_handle(const AdvanceCaps &c, const StateLayout &L, uint8_t *base, fate_state_h *out) {
    out->n_frontier = c.nF;
    out->n_cand = c.nC;
    out->n_slices = c.nS;
    out->n_done_edges = c.nDone;
    out->advance = 1;
    out->status = base + L.status;
    out->finish = reinterpret_cast<const float *>(base + L.finish);
    out->counts = reinterpret_cast<const uint32_t *>(base + L.counts);
}

fate_status_t copy_to_device(void *d_buf, const void *h, size_t bytes, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (hipMemcpyAsync(d_buf, h, bytes, hipMemcpyHostToDevice, s) != hipSuccess) return FATE_EHIP;
    if (hipStreamSynchronize(s) != hipSuccess) return FATE_EHIP;
    return FATE_OK;
}

bool params_ok(const fate_params_t *p) {
    const float v[] = {p->lam_q, p->lam_s, p->lam_tr, p->lam_c, p->lam_p, p->kappa_prefix, p->gamma, p->lam_m};
    for (float x : v)
        if (!finite_nonneg(x)) return false;
    return (p->flags & ~(FATE_MEAN_PER_LEVEL | FATE_NO_WINDOWS)) == 0;
}

}  // namespace

extern "C" {

const char *fate_version(void) { return "fate-mi355x 0.1.0 (gfx950)"; }

const char *fate_strerror(fate_status_t s) {
    // a caller may pass any int; read it as one (an enum value outside the
    // enumerators' range is not a valid fate_status_t in C++)
    int code;
    std::memcpy(&code, &s, sizeof code);
    switch (code) {
        case FATE_OK: return "ok";
        case FATE_EINVAL: return "invalid argument";
        case FATE_ERANGE: return "value out of supported range";
        case FATE_ECYCLE: return "parent id not below child id (not a DAG in topological order)";
        case FATE_ENOFEAS: return "stage has no eligible device that can hold its model";
        case FATE_ESIZE: return "caller buffer too small";
        case FATE_ESTATE: return "inconsistent execution state or handle";
        case FATE_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

fate_status_t fate_pack_dags_opt_size(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                      const fate_pack_opts_t *opts, size_t *bytes) {
    if (!bytes || !opts_ok(opts)) return FATE_EINVAL;
    DagsPlan p;
    fate_status_t st = plan_dags(cluster, dags, *opts, false, &p);
    if (st != FATE_OK) return st;
    *bytes = dag_layout(dags->B, cluster->D, cluster->M, p.N, p.E, p.ndesc, opts->level_weights != 0, p.rows).total;
    return FATE_OK;
}

static fate_status_t build_dags(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                const fate_pack_opts_t &o, size_t bytes, std::vector<uint8_t> &img, DagsPlan &p,
                                DagLayout &L) {
    fate_status_t st = plan_dags(cluster, dags, o, true, &p);
    if (st != FATE_OK) return st;
    L = dag_layout(dags->B, cluster->D, cluster->M, p.N, p.E, p.ndesc, o.level_weights != 0, p.rows);
    if (bytes < L.total) return FATE_ESIZE;
    img.assign(L.total, 0);
    write_dags_image(cluster, dags, p, L, o.level_weights != 0, img.data());
    return FATE_OK;
}

fate_status_t fate_layout_dags_opt(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                   const fate_pack_opts_t *opts, void *h_buf, size_t bytes, fate_dags_t *out) {
    if (!h_buf || !out || !opts_ok(opts)) return FATE_EINVAL;
    std::vector<uint8_t> img;
    DagsPlan p;
    DagLayout L;
    fate_status_t st = build_dags(cluster, dags, *opts, bytes, img, p, L);
    if (st != FATE_OK) return st;
    copy_bytes(h_buf, img.data(), L.total);
    fill_dags_handle(cluster, dags, *opts, p, L, static_cast<uint8_t *>(h_buf), bytes, out);
    return FATE_OK;
}

fate_status_t fate_pack_dags_opt(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                 const fate_pack_opts_t *opts, void *d_buf, size_t bytes, void *stream,
                                 fate_dags_t *out) {
    if (!d_buf || !out || !opts_ok(opts)) return FATE_EINVAL;
    std::vector<uint8_t> img;
    DagsPlan p;
    DagLayout L;
    fate_status_t st = build_dags(cluster, dags, *opts, bytes, img, p, L);
    if (st != FATE_OK) return st;
    st = copy_to_device(d_buf, img.data(), L.total, stream);
    if (st != FATE_OK) return st;
    fill_dags_handle(cluster, dags, *opts, p, L, static_cast<uint8_t *>(d_buf), bytes, out);
    return FATE_OK;
}

static fate_pack_opts_t hop_opts(int32_t H) {
    fate_pack_opts_t o;
    o.H = H;
    o.levels = FATE_LEVELS_HOP;
    o.level_weights = 0;
    return o;
}

fate_status_t fate_pack_dags_size(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, int32_t H,
                                  size_t *bytes) {
    const fate_pack_opts_t o = hop_opts(H);
    return fate_pack_dags_opt_size(cluster, dags, &o, bytes);
}

fate_status_t fate_layout_dags(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, int32_t H,
                               void *h_buf, size_t bytes, fate_dags_t *out) {
    const fate_pack_opts_t o = hop_opts(H);
    return fate_layout_dags_opt(cluster, dags, &o, h_buf, bytes, out);
}

fate_status_t fate_pack_dags(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, int32_t H,
                             void *d_buf, size_t bytes, void *stream, fate_dags_t *out) {
    const fate_pack_opts_t o = hop_opts(H);
    return fate_pack_dags_opt(cluster, dags, &o, d_buf, bytes, stream, out);
}

fate_status_t fate_pack_state_size(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                   const fate_state_t *state, int32_t max_shard, size_t *bytes,
                                   int64_t *n_frontier, int64_t *n_cand) {
    if (!bytes) return FATE_EINVAL;
    StatePlan p;
    fate_status_t st = plan_state(packed, dags, state, max_shard, &p);
    if (st != FATE_OK) return st;
    *bytes = state_layout(packed->B, packed->D, state->K, packed->N, p.nF, p.nS, packed->E).total;
    if (n_frontier) *n_frontier = p.nF;
    if (n_cand) *n_cand = p.nC;
    return FATE_OK;
}

static fate_status_t build_state(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                 const fate_state_t *state, int32_t max_shard, size_t bytes,
                                 std::vector<uint8_t> &img, StatePlan &p, StateLayout &L) {
    fate_status_t st = plan_state(packed, dags, state, max_shard, &p);
    if (st != FATE_OK) return st;
    L = state_layout(packed->B, packed->D, state->K, packed->N, p.nF, p.nS, packed->E);
    if (bytes < L.total) return FATE_ESIZE;
    img.assign(L.total, 0);
    write_state_image(packed, dags, state, p, L, img.data());
    return FATE_OK;
}

fate_status_t fate_layout_state(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                const fate_state_t *state, int32_t max_shard, void *h_buf, size_t bytes,
                                fate_state_h *out) {
    if (!h_buf || !out) return FATE_EINVAL;
    std::vector<uint8_t> img;
    StatePlan p;
    StateLayout L;
    fate_status_t st = build_state(packed, dags, state, max_shard, bytes, img, p, L);
    if (st != FATE_OK) return st;
    copy_bytes(h_buf, img.data(), L.total);
    fill_state_handle(packed, state, max_shard, p, L, static_cast<uint8_t *>(h_buf), bytes, out);
    return FATE_OK;
}

fate_status_t fate_pack_state(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                              const fate_state_t *state, int32_t max_shard, void *d_buf, size_t bytes,
                              void *stream, fate_state_h *out) {
    if (!d_buf || !out) return FATE_EINVAL;
    std::vector<uint8_t> img;
    StatePlan p;
    StateLayout L;
    fate_status_t st = build_state(packed, dags, state, max_shard, bytes, img, p, L);
    if (st != FATE_OK) return st;
    st = copy_to_device(d_buf, img.data(), L.total, stream);
    if (st != FATE_OK) return st;
    fill_state_handle(packed, state, max_shard, p, L, static_cast<uint8_t *>(d_buf), bytes, out);
    return FATE_OK;
}

fate_status_t fate_pack_state_advance_size(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                           const fate_state_t *state, int32_t max_shard, size_t *bytes) {
    if (!bytes) return FATE_EINVAL;
    StatePlan p;
    fate_status_t st = plan_state(packed, dags, state, max_shard, &p);
    if (st != FATE_OK) return st;
    AdvanceCaps c;
    st = advance_caps(packed, dags, state, max_shard, &c);
    if (st != FATE_OK) return st;
    *bytes = state_layout(packed->B, packed->D, state->K, packed->N, c.nF, c.nS, c.nDone, true).total;
    return FATE_OK;
}

fate_status_t fate_pack_state_advance(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                      const fate_state_t *state, int32_t max_shard, void *d_buf, size_t bytes,
                                      void *stream, fate_state_h *out) {
    if (!d_buf || !out) return FATE_EINVAL;
    StatePlan p;
    fate_status_t st = plan_state(packed, dags, state, max_shard, &p);
    if (st != FATE_OK) return st;
    AdvanceCaps c;
    st = advance_caps(packed, dags, state, max_shard, &c);
    if (st != FATE_OK) return st;
    const StateLayout L = state_layout(packed->B, packed->D, state->K, packed->N, c.nF, c.nS, c.nDone, true);
    if (bytes < L.total) return FATE_ESIZE;
    std::vector<uint8_t> img(L.total, 0);
    write_state_image(packed, dags, state, p, L, img.data());
    st = copy_to_device(d_buf, img.data(), L.total, stream);
    if (st != FATE_OK) return st;
    fill_state_handle(packed, state, max_shard, p, L, static_cast<uint8_t *>(d_buf), bytes, out);
    fill_advance_handle(c, L, static_cast<uint8_t *>(d_buf), out);
    return FATE_OK;
}

static fate_status_t check_pair(const fate_dags_t *dags, const fate_state_h *state) {
    if (!dags || !state) return FATE_EINVAL;
    if (dags->B != state->B || dags->D != state->D || dags->N != state->N) return FATE_ESTATE;
    // the scoring kernel's LDS holds one slice of this build's length
    if (state->slice != fate::slice_len(dags->D)) return FATE_ESTATE;
    if (!dags->records || !state->frontier || !state->cand_off || !state->slices || !state->done_n ||
        !state->fr_off || !state->order)
        return FATE_EINVAL;
    return FATE_OK;
}

fate_status_t fate_commit_ws_size(const fate_dags_t *dags, const fate_state_h *state, size_t *bytes) {
    if (!bytes) return FATE_EINVAL;
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    if (!state->advance) return FATE_EINVAL;
    *bytes = fate::commit_ws_layout(state->N, state->B).total;
    return FATE_OK;
}

fate_status_t fate_commit_advance(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                                  int32_t sel_stride, void *d_ws, size_t ws_bytes, void *stream) {
    return fate::commit_impl(dags, state, d_sel, sel_stride, d_ws, ws_bytes, stream);
}

}  // extern "C"

namespace fate {

fate_status_t commit_check(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                           int32_t sel_stride, size_t *ws_total) {
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    if (!state->advance || !state->status || !state->counts || sel_stride < 1) return FATE_EINVAL;
    if (state->n_frontier > 0 && !d_sel) return FATE_EINVAL;
    if (!dags->ch_off || (dags->E > 0 && !dags->ch_idx)) return FATE_EINVAL;
    *ws_total = fate::commit_ws_layout(state->N, state->B).total;
    return FATE_OK;
}

fate_status_t commit_impl(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                          int32_t sel_stride, void *d_ws, size_t ws_bytes, void *stream) {
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    if (!state->advance || !state->status || !state->counts || sel_stride < 1) return FATE_EINVAL;
    if (state->n_frontier > 0 && !d_sel) return FATE_EINVAL;
    if (!dags->ch_off || (dags->E > 0 && !dags->ch_idx)) return FATE_EINVAL;
    const fate::CommitWs W = fate::commit_ws_layout(state->N, state->B);
    if (ws_bytes < W.total) return FATE_ESIZE;
    if (W.total > 0 && !d_ws) return FATE_EINVAL;
    uint8_t *ws = static_cast<uint8_t *>(d_ws);
    fate::CommitLaunch a;
    a.rec = static_cast<const StageRec *>(dags->records);
    a.par_idx = dags->par_idx;
    a.stage_off = dags->stage_off;
    a.exec = dags->exec;
    a.ksw = dags->switch_s;
    a.weight = dags->weight;
    a.cap = dags->cap;
    a.fits = dags->fits;
    // the planning state's buffer is the caller's, handed over for update
    a.resident = const_cast<uint64_t *>(state->resident);
    a.pcache = const_cast<uint64_t *>(state->prefix_cache);
    a.holders = const_cast<uint64_t *>(state->holders);
    a.tau = const_cast<float *>(state->tau_free);
    a.fin = const_cast<float *>(state->finish);
    a.beta = dags->beta;
    a.tnow = state->t_now;
    a.status = const_cast<uint8_t *>(state->status);
    a.frontier = const_cast<uint32_t *>(state->frontier);
    a.cand_off = const_cast<uint32_t *>(state->cand_off);
    a.slices = const_cast<uint32_t *>(state->slices);
    a.done_n = const_cast<uint32_t *>(state->done_n);
    a.fr_off = const_cast<uint32_t *>(state->fr_off);
    a.order = const_cast<uint32_t *>(state->order);
    a.done = static_cast<fate::DoneParent *>(const_cast<void *>(state->done));
    a.counts = const_cast<uint32_t *>(state->counts);
    a.sel = d_sel;
    a.sel_stride = sel_stride;
    a.ch_off = dags->ch_off;
    a.ch_idx = dags->ch_idx;
    a.list = reinterpret_cast<uint32_t *>(ws + W.list);
    a.tot = reinterpret_cast<uint32_t *>(ws + W.tot);
    a.base = reinterpret_cast<uint32_t *>(ws + W.base);
    a.nsp = reinterpret_cast<uint32_t *>(ws + W.nsp);
    a.gbm = reinterpret_cast<uint32_t *>(ws + W.gbm);
    // the largest instance's bitmap, with the slack of an unaligned start in
    // the workspace
    a.bm_words = (int32_t)((dags->max_stages + 31 + 31) / 32);
    a.bm_lds = a.bm_words <= fate::kCommitLdsBitmapWords ? 1 : 0;
    a.slice_order = fate::rows_batch(dags, state->max_shard, state->K) ? 0 : 1;
    a.beta_uniform = dags->beta_uniform;
    a.beta0 = dags->beta0;
    a.N = state->N;
    a.B = state->B;
    a.D = dags->D;
    a.M = dags->M;
    a.K = state->K;
    a.max_shard = state->max_shard;
    a.slice = fate::slice_len(dags->D);
    return fate::launch_commit(a, stream) == 0 ? FATE_OK : FATE_EHIP;
}

}  // namespace fate

extern "C" {

fate_status_t fate_score_ws_size(const fate_dags_t *dags, const fate_state_h *state, size_t *bytes) {
    if (!bytes) return FATE_EINVAL;
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    *bytes = 0;
    return FATE_OK;
}

// Scoring launch over P parameter sets: set p writes d_scores + p * stride.
static fate_status_t score_impl(const fate_dags_t *dags, const fate_state_h *state, const fate_params_t *params,
                                int32_t P, float *d_scores, int64_t n_scores, int64_t stride, int32_t k,
                                int32_t *d_idx, float *d_val, void *stream) {
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    if (!params) return FATE_EINVAL;
    if (P < 1 || P > FATE_MAX_SWEEP) return FATE_ERANGE;
    for (int p = 0; p < P; ++p) {
        if (!params_ok(&params[p])) return FATE_EINVAL;
        if (params[p].H < 0 || params[p].H > dags->H) return FATE_EINVAL;
        if ((params[p].flags & FATE_MEAN_PER_LEVEL) && !dags->desc_w) return FATE_EINVAL;
    }
    if (stride < state->n_cand) return FATE_ESIZE;
    if (n_scores < stride * (P - 1) + state->n_cand) return FATE_ESIZE;
    // the instance's prefix table, model tables and staging must fit one workgroup's LDS
    if (!fate::score_fits(dags->D, state->K, dags->M, dags->beta_uniform)) return FATE_ERANGE;
    if (state->n_frontier == 0) return FATE_OK;
    if (!d_scores) return FATE_EINVAL;
    fate::ScoreLaunch a;
    a.rec = static_cast<const StageRec *>(dags->records);
    a.rowrec = static_cast<const fate::RowRec *>(dags->row_records);
    a.par_idx = dags->par_idx;
    a.desc_off = dags->desc_off;
    a.desc = dags->desc;
    a.desc_w = dags->desc_w;
    a.exec = dags->exec;
    a.ksw = dags->switch_s;
    a.beta = dags->beta;
    a.weight = dags->weight;
    a.cap = dags->cap;
    a.fits = dags->fits;
    a.resident = state->resident;
    a.pcache = state->prefix_cache;
    a.holders = state->holders;
    a.tau = state->tau_free;
    a.tnow = state->t_now;
    a.frontier = state->frontier;
    a.cand_off = state->cand_off;
    a.slices = state->slices;
    a.done_n = state->done_n;
    a.done = static_cast<const fate::DoneParent *>(state->done);
    a.order = state->order;
    a.fr_off = state->fr_off;
    a.scores = d_scores;
    a.score_stride = stride;
    a.dcounts = state->advance ? state->counts : nullptr;
    a.topk = k;
    a.tk_idx = d_idx;
    a.tk_val = d_val;
    a.nF = state->n_frontier;
    a.n_slices = state->n_slices;
    a.B = dags->B;
    a.D = dags->D;
    a.M = dags->M;
    a.K = state->K;
    a.max_shard = state->max_shard;
    a.beta_uniform = dags->beta_uniform;
    a.slice = fate::slice_len(dags->D);
    a.beta0 = dags->beta0;
    a.topo = dags->levels == FATE_LEVELS_TOPO ? 1 : 0;
    a.Hpack = dags->H;
    // a window needs a stage with R(v) > 1, a shard cap above 1 and two devices
    a.singles = std::min(std::min(dags->max_r, state->max_shard), dags->D) <= 1 ? 1 : 0;
    a.nsets = P;
    for (int p = 0; p < fate::kMaxSets; ++p) {
        const fate_params_t &q = params[p < P ? p : 0];
        fate::ParamSet &ps = a.ps[p];
        ps.lam_q = q.lam_q;
        ps.lam_s = q.lam_s;
        ps.lam_tr = q.lam_tr;
        ps.lam_c = q.lam_c;
        ps.lam_p = q.lam_p;
        ps.kpf = q.kappa_prefix;
        ps.gamma = q.gamma;
        ps.lam_m = q.lam_m;
        ps.H = q.H;
        ps.flags = q.flags;
        a.set_of[p] = p;
    }
    return fate::launch_score(a, stream) == 0 ? FATE_OK : FATE_EHIP;
}

fate_status_t fate_score_frontier(const fate_dags_t *dags, const fate_state_h *state,
                                  const fate_params_t *params, float *d_scores, int64_t n_scores,
                                  void *d_ws, size_t ws_bytes, void *stream) {
    (void)d_ws;
    (void)ws_bytes;
    return score_impl(dags, state, params, 1, d_scores, n_scores, state ? state->n_cand : 0, 0, nullptr, nullptr,
                      stream);
}

fate_status_t fate_score_sweep(const fate_dags_t *dags, const fate_state_h *state, const fate_params_t *params,
                               int32_t n_sets, float *d_scores, int64_t n_scores, int64_t score_stride,
                               void *d_ws, size_t ws_bytes, void *stream) {
    (void)d_ws;
    (void)ws_bytes;
    return score_impl(dags, state, params, n_sets, d_scores, n_scores, score_stride, 0, nullptr, nullptr, stream);
}

fate_status_t fate_score_topk(const fate_dags_t *dags, const fate_state_h *state, const fate_params_t *params,
                              float *d_scores, int64_t n_scores, int32_t k, int32_t *d_idx, float *d_val,
                              void *d_ws, size_t ws_bytes, void *stream) {
    (void)d_ws;
    (void)ws_bytes;
    if (k < 1 || k > FATE_MAX_TOPK) return FATE_ERANGE;
    if (state && state->n_frontier > 0 && (!d_idx || !d_val)) return FATE_EINVAL;
    return score_impl(dags, state, params, 1, d_scores, n_scores, state ? state->n_cand : 0, k, d_idx, d_val,
                      stream);
}

static fate_status_t topk_impl(const fate_state_h *state, const float *d_scores, int64_t n_scores,
                               int64_t score_stride, int32_t n_sets, int32_t k, int32_t *d_idx, float *d_val,
                               void *stream) {
    if (!state) return FATE_EINVAL;
    if (k < 1 || k > FATE_MAX_TOPK) return FATE_ERANGE;
    if (n_sets < 1 || n_sets > FATE_MAX_SWEEP) return FATE_ERANGE;
    if (score_stride < state->n_cand) return FATE_ESIZE;
    if (n_scores < score_stride * (n_sets - 1) + state->n_cand) return FATE_ESIZE;
    if (state->n_frontier == 0) return FATE_OK;
    if (!d_scores || !d_idx || !d_val || !state->cand_off) return FATE_EINVAL;
    fate::TopkLaunch a;
    a.cand_off = state->cand_off;
    a.scores = d_scores;
    a.idx = d_idx;
    a.val = d_val;
    a.dcounts = state->advance ? state->counts : nullptr;
    a.nF = state->n_frontier;
    a.score_stride = score_stride;
    a.out_stride = state->n_frontier * (int64_t)k;
    a.nsets = n_sets;
    a.D = state->D;
    a.k = k;
    return fate::launch_topk(a, stream) == 0 ? FATE_OK : FATE_EHIP;
}

fate_status_t fate_topk(const fate_state_h *state, const float *d_scores, int64_t n_scores, int32_t k,
                        int32_t *d_idx, float *d_val, void *stream) {
    return topk_impl(state, d_scores, n_scores, state ? state->n_cand : 0, 1, k, d_idx, d_val, stream);
}

fate_status_t fate_topk_sweep(const fate_state_h *state, const float *d_scores, int64_t n_scores,
                              int64_t score_stride, int32_t n_sets, int32_t k, int32_t *d_idx, float *d_val,
                              void *stream) {
    return topk_impl(state, d_scores, n_scores, score_stride, n_sets, k, d_idx, d_val, stream);
}

fate_status_t fate_plan_wave(const fate_state_h *state, const int32_t *d_idx, const float *d_val, int32_t k,
                             int32_t *d_sel, void *stream) {
    if (!state) return FATE_EINVAL;
    if (k < 1 || k > FATE_MAX_TOPK) return FATE_ERANGE;
    if (state->n_frontier == 0) return FATE_OK;
    if (!d_idx || !d_val || !d_sel || !state->frontier || !state->cand_off || !state->fr_off || !state->order)
        return FATE_EINVAL;
    if (state->n_frontier * (int64_t)k >= (int64_t(1) << 32)) return FATE_ERANGE;
    fate::PlanLaunch a;
    a.frontier = state->frontier;
    a.cand_off = state->cand_off;
    a.idx = d_idx;
    a.val = d_val;
    a.sel = d_sel;
    a.fr_off = state->fr_off;
    a.order = state->order;
    a.nF = state->n_frontier;
    a.B = state->B;
    a.D = state->D;
    a.k = k;
    return fate::launch_plan(a, stream) == 0 ? FATE_OK : FATE_EHIP;
}

}  // extern "C"

// ---- plan execution and baseline placements on the device ------------------

static fate_status_t sim_check(const fate_dags_t *dags, const fate_state_h *state, float kappa_prefix,
                               int32_t *d_status, void *d_ws, size_t ws_bytes) {
    fate_status_t st = check_pair(dags, state);
    if (st != FATE_OK) return st;
    if (!finite_nonneg(kappa_prefix)) return FATE_EINVAL;
    if (state->B > 0 && (!d_status || !state->resident || !state->tau_free || !state->t_now || !dags->stage_off))
        return FATE_EINVAL;
    if (state->K > 0 && state->B > 0 && !state->prefix_cache) return FATE_EINVAL;
    if (state->N > 0 && !state->holders) return FATE_EINVAL;
    const fate::SimWs W = fate::sim_ws_layout(state->N);
    if (ws_bytes < W.total) return FATE_ESIZE;
    if (W.total > 0 && !d_ws) return FATE_EINVAL;
    return FATE_OK;
}

static void sim_fill(const fate_dags_t *dags, const fate_state_h *state, float kappa_prefix, int32_t *d_status,
                     void *d_ws, fate::SimLaunch &a) {
    const fate::SimWs W = fate::sim_ws_layout(state->N);
    uint8_t *ws = static_cast<uint8_t *>(d_ws);
    a.rec = static_cast<const StageRec *>(dags->records);
    a.par_idx = dags->par_idx;
    a.stage_off = dags->stage_off;
    a.exec = dags->exec;
    a.ksw = dags->switch_s;
    a.beta = dags->beta;
    a.weight = dags->weight;
    a.cap = dags->cap;
    a.fits = dags->fits;
    a.resident = state->resident;
    a.pcache = state->prefix_cache;
    a.holders = state->holders;
    a.tau = state->tau_free;
    a.tnow = state->t_now;
    a.devices = nullptr;
    a.order = nullptr;
    a.dev_out = nullptr;
    a.ord_out = nullptr;
    a.out = nullptr;
    a.status = d_status;
    a.fin = reinterpret_cast<double *>(ws + W.fin);
    a.aux = reinterpret_cast<double *>(ws + W.aux);
    a.tail = reinterpret_cast<double *>(ws + W.tail);
    a.hold = reinterpret_cast<uint64_t *>(ws + W.hold);
    a.keys = reinterpret_cast<uint64_t *>(ws + W.keys);
    a.ids = reinterpret_cast<uint32_t *>(ws + W.ids);
    a.todo = reinterpret_cast<uint32_t *>(ws + W.todo);
    a.flags = ws + W.flags;
    a.kpf = (double)kappa_prefix;
    a.B = state->B;
    a.D = dags->D;
    a.K = state->K;
}

extern "C" {

fate_status_t fate_sim_ws_size(const fate_dags_t *dags, size_t *bytes) {
    if (!dags || !bytes) return FATE_EINVAL;
    *bytes = fate::sim_ws_layout(dags->N).total;
    return FATE_OK;
}

fate_status_t fate_simulate_device(const fate_dags_t *dags, const fate_state_h *state, const uint64_t *d_devices,
                                   const int64_t *d_order, float kappa_prefix, fate_sim_metrics_t *d_out,
                                   int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream) {
    fate_status_t st = sim_check(dags, state, kappa_prefix, d_status, d_ws, ws_bytes);
    if (st != FATE_OK) return st;
    if (state->B > 0 && !d_out) return FATE_EINVAL;
    if (state->N > 0 && (!d_devices || !d_order)) return FATE_EINVAL;
    fate::SimLaunch a;
    sim_fill(dags, state, kappa_prefix, d_status, d_ws, a);
    a.devices = d_devices;
    a.order = d_order;
    a.out = d_out;
    return fate::launch_sim(a, 0, stream) == 0 ? FATE_OK : FATE_EHIP;
}

fate_status_t fate_place_baseline_device(const fate_dags_t *dags, const fate_state_h *state, int32_t policy,
                                         float kappa_prefix, uint64_t *d_devices, int64_t *d_order,
                                         int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream) {
    if (policy != FATE_PLACE_ROUND_ROBIN && policy != FATE_PLACE_HEFT) return FATE_EINVAL;
    fate_status_t st = sim_check(dags, state, kappa_prefix, d_status, d_ws, ws_bytes);
    if (st != FATE_OK) return st;
    if (state->N > 0 && (!d_devices || !d_order)) return FATE_EINVAL;
    fate::SimLaunch a;
    sim_fill(dags, state, kappa_prefix, d_status, d_ws, a);
    a.dev_out = d_devices;
    a.ord_out = d_order;
    return fate::launch_sim(a, policy == FATE_PLACE_ROUND_ROBIN ? 1 : 2, stream) == 0 ? FATE_OK : FATE_EHIP;
}

}  // extern "C"
