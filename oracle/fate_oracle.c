/*
 * fp64 CPU oracle for FATE horizon-aware candidate scoring (arXiv 2605.07238).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this library.  It shares no
 * code, header, table or helper with the HIP scoring library; it reads the
 * same flat input arrays that the seeded workload generator produces and
 * computes every score from scratch, slowly and literally.
 *
 * What is computed, step by step, per workflow instance (Sec. 2, Sec. 3.3-3.5,
 * App. A.1-A.4).  Readings of passages the paper leaves open are marked
 * [reading]; each is listed in the design notes of the repository.
 *
 *  1. Frontier (Sec. 2 ready set; App. A.1 implementation frontier): stages
 *     that are pending (not completed, running or committed) and whose
 *     parents are all completed, in ascending stage id.
 *  2. Candidates of a frontier stage v: single devices {0}..{D-1}, then
 *     contiguous windows {i..i+k-1} for k = 2..r, i = 0..D-k, where
 *     r = min(R(v), max_shard, D)  (Sec. 3.3 shard slots; App. A.2 bounded
 *     shard execution) [reading: shard slots occupy a contiguous window].
 *  3. Feasibility (Sec. 2 feasible set; App. A.2 eligibility constraint):
 *     every device of the candidate is in A(v) and holds the model's weights
 *     (W(m(v)) <= cap(d)); otherwise the score is -infinity.
 *  4. Term functions, evaluated in a state s (App. A.3):
 *       Wait(d)    = max(0, tau_d - t)
 *       Sw(x,d)    = 0 if m(x) resident on d, else kappa_switch(m(x), d)
 *       Tr(x,d)    = sum over completed parents u of x with d not holding u's
 *                    output of sigma(u) * min_{i holding u} beta[i][d]
 *                    [reading: a parent output may sit on several devices]
 *       Colo(x,d)  = (1/|Pa(x)|) * #parents whose output d holds; 0 if no
 *                    parents
 *       Pf(x,d)    = kappa_prefix * L(x) if grp(x) != 0 and grp(x) is cached
 *                    on d [reading of Overlap()]
 *       c_hat(x,d) = c(x,d) + l_s Sw + l_tr Tr - l_c Colo - l_p Pf
 *                    (App. A.1 additive decomposition, App. A.4 estimator)
 *  5. Immediate cost of candidate S with k = |S| devices [reading of
 *     B_parallel]: per device d in S
 *       T(d) = l_q Wait(d) + c(v,d)/k + l_s Sw(v,d)
 *              + (l_tr Tr(v,d) - l_p Pf(v,d))/k - l_c Colo(v,d)
 *     G(S) = min_{p in S} sum_{d in S, d != p} beta[d][p] sigma(v) / k
 *     J0 = max_{d in S} T(d) + l_tr G(S).
 *  6. Post-state s' (Sec. 3.2 future state): for d in S the model of v is
 *     loaded (Load: add it, then while the resident weights exceed the
 *     capacity remove the smallest-id other model), grp(v) joins the prefix
 *     set of d, and v's output is held by exactly the devices of S.
 *  7. Horizon set (Sec. 3.3; App. D.4 treats H = 0 as no lookahead): stages
 *     at breadth-first hop distance h = 1..H from v, each counted once at its
 *     minimum distance.
 *  8. Descendant value [reading of future device reachability]: the minimum
 *     of c_hat(w, d' | s') over the devices d' feasible for w.
 *  9. J = J0 + sum_h gamma^h sum_{w at distance h} value(w); Psi = -J
 *     (higher is better).
 * 10. Top-k per frontier stage: candidates ordered by (Psi descending,
 *     candidate index ascending), infeasible ones skipped, padded with
 *     (-1, -infinity).
 * 11. Commit-and-advance of the planning state (Alg. 1: materialise the
 *     selected placements, then advance the frontier and update the
 *     planning state; Alg. 2: commit into the action pool and update the
 *     state as the stages complete) [reading: one planning-state update per
 *     planning step].  Per instance, the selected frontier stages are applied
 *     in ascending stage id; for each device d of the chosen candidate S
 *     (k = |S|), in ascending device id:
 *       ready  = max over parents u of fin(u) + (0 if d holds u's output, else
 *                sigma(u) * min over u's holders i of beta[i][d] / k)
 *                [reading: a shard cannot start before its inputs arrive;
 *                fin(u) is u's planned finish, t for a stage completed when
 *                planning began]
 *       start  = max(tau_d, t, ready)
 *       switch = kappa_switch(m(v), d) if m(v) is not resident on d, else 0
 *       rho_d  = Load(rho_d, m(v))                      (as in step 6)
 *       grp(v) joins the prefix slots of d if it is nonzero and absent: the
 *         first empty slot takes it, or, when all K slots are full, the slots
 *         move down by one (slot 0, the oldest, is dropped) and slot K-1
 *         takes it  [reading: the slots are kept oldest first]
 *       tau_d  = start + c(v,d)/k + switch
 *     then v is completed with its output held by exactly S, and fin(v) is
 *     the largest of those tau_d.  The next
 *     frontier follows from step 1 on the updated state.
 *
 * 12. Frontier planning wave (App. A.2 frontier placement problem: each
 *     device takes at most one shard-slot assignment per wave, each shard
 *     slot at most one device, slots enabled in order; Alg. 1 solves it with
 *     CP-SAT) [reading: the top-k candidates of each frontier stage are the
 *     choices; a candidate uses the devices of its window, which is the
 *     stage's slots 0..k-1 on k devices, so slot order holds by itself; the
 *     wave is built greedily]: among the choices whose stage has no
 *     assignment yet and whose devices are all still free in this wave, take
 *     the one with the highest score (ties: lower frontier slot, then lower
 *     rank), mark its stage assigned and its devices used, and repeat until
 *     no choice is left.  Choices scored -infinity, padded (-1) or past the
 *     stage's candidates are never taken.  Instances plan independently.
 *
 * Scoring variants (all off by default):
 *   V1. Same-model preference (Sec. 4 implementation summary: model-
 *       specialised placement preferences; App. C.3, "w/o same-model bonus"
 *       removes the reward for continuing with a model already resident
 *       while keeping the switch cost) [reading]: every place a switch cost
 *       Sw(x,d) enters (steps 4 and 5), the term - l_m SM(x,d) enters beside
 *       it, SM(x,d) = 1 if m(x) is resident on d in the state at hand, else 0.
 *   V2. Topological levels (Sec. 3.3 "downstream DAG levels", the other
 *       reading of step 7) [reading]: level(x) = 0 for a stage without
 *       parents, else 1 + the largest level of its parents; the horizon set of
 *       v is every stage reachable from v with 1 <= level(w) - level(v) <= H,
 *       at depth level(w) - level(v).
 *   V3. Mean per level (the alternative to the sum in step 9) [reading]: the
 *       values of the stages at depth h are averaged, each weighted
 *       gamma^h / n_h, n_h the number of horizon stages at depth h.
 *   V4. No windows (App. C.3, "w/o shard parallelism"): candidates with
 *       k > 1 keep their slots but score -infinity.
 *
 * Alongside Psi the oracle reports A, the sum of the absolute values of every
 * weighted term it added (for the maximising device of step 5 and the
 * minimising device of step 8).  Parity tolerances are relative to A.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC fate_oracle.c -o libfate_oracle.so -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int D, M, K, H, max_shard;
    const float *exec, *switch_s, *beta;      /* [M*D], [M*D], [D*D] */
    const int64_t *weight, *cap;              /* [M], [D] */
    const int64_t *stage_off, *par_off;       /* [B+1], [N+1] */
    const int32_t *par_idx, *model, *shard;   /* [E], [N], [N] */
    const uint64_t *elig, *hash;              /* [N], [N] */
    const float *tokens, *sigma;              /* [N], [N] */
    const uint64_t *resident, *cache;         /* [B*D], [B*D*K] */
    const uint64_t *holders;                  /* [N] */
    const uint8_t *status;                    /* [N] */
    const float *tau, *t_now;                 /* [B*D], [B] */
    double lam_q, lam_s, lam_tr, lam_c, lam_p, kappa_prefix, gamma;
    /* variants V1-V4 */
    double lam_m;
    int topo_levels, mean_levels, no_windows;
} oracle_in_t;

enum { ST_PENDING = 0, ST_COMPLETED = 1 };

/* State view used by the term functions: either the current state s or a
 * post-state s' that differs on the devices of one candidate. */
typedef struct {
    const oracle_in_t *in;
    int64_t base;            /* global index of the instance's stage 0 */
    int b;
    uint64_t res[64];        /* resident-model bitmask per device */
    uint64_t extra_hash[64]; /* one extra cached prefix group per device, 0 = none */
    int over_stage;          /* stage whose holders are overridden, -1 = none */
    uint64_t over_holders;
} view_t;

static int has_bit(uint64_t m, int i) { return (int)((m >> i) & 1u); }

static double exec_c(const oracle_in_t *in, int m, int d) { return (double)in->exec[m * in->D + d]; }

static uint64_t holders_of(const view_t *s, int u) {
    if (u == s->over_stage) return s->over_holders;
    return s->in->holders[s->base + u];
}

static int fits(const oracle_in_t *in, int m, int d) { return in->weight[m] <= in->cap[d]; }

static int feasible(const oracle_in_t *in, int64_t g, int d) {
    return has_bit(in->elig[g], d) && fits(in, in->model[g], d);
}

/* App. A.3 waiting cost. */
static double wait_cost(const view_t *s, int d) {
    double w = (double)s->in->tau[s->b * s->in->D + d] - (double)s->in->t_now[s->b];
    return w > 0.0 ? w : 0.0;
}

/* App. A.3 model-switch cost. */
static double switch_cost(const view_t *s, int x, int d) {
    const oracle_in_t *in = s->in;
    int m = in->model[s->base + x];
    if (has_bit(s->res[d], m)) return 0.0;
    return (double)in->switch_s[m * in->D + d];
}

/* App. A.3 cross-device transfer cost from completed parents. */
static double transfer_cost(const view_t *s, int x, int d) {
    const oracle_in_t *in = s->in;
    int64_t g = s->base + x;
    double tr = 0.0;
    for (int64_t q = in->par_off[g]; q < in->par_off[g + 1]; ++q) {
        int u = in->par_idx[q];
        uint64_t hu = holders_of(s, u);
        if (hu == 0 || has_bit(hu, d)) continue;
        double bmin = INFINITY;
        for (int i = 0; i < in->D; ++i)
            if (has_bit(hu, i) && (double)in->beta[i * in->D + d] < bmin)
                bmin = (double)in->beta[i * in->D + d];
        tr += (double)in->sigma[s->base + u] * bmin;
    }
    return tr;
}

/* App. A.3 parent-colocation benefit. */
static double colo_benefit(const view_t *s, int x, int d) {
    const oracle_in_t *in = s->in;
    int64_t g = s->base + x;
    int64_t np = in->par_off[g + 1] - in->par_off[g];
    if (np == 0) return 0.0;
    int cnt = 0;
    for (int64_t q = in->par_off[g]; q < in->par_off[g + 1]; ++q)
        if (has_bit(holders_of(s, in->par_idx[q]), d)) ++cnt;
    return (double)cnt / (double)np;
}

/* App. A.3 prefix-reuse benefit with Overlap = L(x) on a cached group. */
static double prefix_benefit(const view_t *s, int x, int d) {
    const oracle_in_t *in = s->in;
    int64_t g = s->base + x;
    uint64_t h = in->hash[g];
    if (h == 0) return 0.0;
    int hit = (s->extra_hash[d] == h);
    const uint64_t *slots = in->cache + ((int64_t)s->b * in->D + d) * in->K;
    for (int k = 0; k < in->K && !hit; ++k)
        if (slots[k] == h) hit = 1;
    return hit ? in->kappa_prefix * (double)in->tokens[g] : 0.0;
}

/* V1: 1 if the model of stage x is already resident on d. */
static double same_model(const view_t *s, int x, int d) {
    return has_bit(s->res[d], s->in->model[s->base + x]) ? 1.0 : 0.0;
}

/* App. A.1 / A.4 state-corrected cost of stage x on device d, plus the sum
 * of the absolute values of its weighted terms. */
static double c_hat(const view_t *s, int x, int d, double *mag) {
    const oracle_in_t *in = s->in;
    int m = in->model[s->base + x];
    double c = exec_c(in, m, d);
    double t_sw = in->lam_s * switch_cost(s, x, d);
    double t_tr = in->lam_tr * transfer_cost(s, x, d);
    double t_co = in->lam_c * colo_benefit(s, x, d);
    double t_pf = in->lam_p * prefix_benefit(s, x, d);
    double t_sm = in->lam_m * same_model(s, x, d);
    if (mag) *mag = fabs(c) + fabs(t_sw) + fabs(t_tr) + fabs(t_co) + fabs(t_pf) + fabs(t_sm);
    return c + t_sw + t_tr - t_co - t_pf - t_sm;
}

/* Model load under capacity: add m, then evict the smallest-id other
 * resident models while the resident weights exceed the device capacity. */
static uint64_t load_model(const oracle_in_t *in, uint64_t res, int m, int d) {
    if (has_bit(res, m)) return res;
    res |= (uint64_t)1 << m;
    int64_t total = 0;
    for (int i = 0; i < in->M; ++i)
        if (has_bit(res, i)) total += in->weight[i];
    for (int i = 0; i < in->M && total > in->cap[d]; ++i) {
        if (i == m || !has_bit(res, i)) continue;
        res &= ~((uint64_t)1 << i);
        total -= in->weight[i];
    }
    return res;
}

static void init_view(view_t *s, const oracle_in_t *in, int b) {
    s->in = in;
    s->b = b;
    s->base = in->stage_off[b];
    for (int d = 0; d < in->D; ++d) {
        s->res[d] = in->resident[(int64_t)b * in->D + d];
        s->extra_hash[d] = 0;
    }
    s->over_stage = -1;
    s->over_holders = 0;
}

static int shard_cap(const oracle_in_t *in, int64_t g) {
    int r = in->shard[g];
    if (r > in->max_shard) r = in->max_shard;
    if (r > in->D) r = in->D;
    if (r < 1) r = 1;
    return r;
}

static int64_t n_candidates(const oracle_in_t *in, int64_t g) {
    int r = shard_cap(in, g);
    int64_t c = in->D;
    for (int k = 2; k <= r; ++k) c += in->D - k + 1;
    return c;
}

/* Candidate j of a stage with D devices -> window start i and size k. */
static void window_of(int D, int64_t j, int *i_out, int *k_out) {
    if (j < D) { *i_out = (int)j; *k_out = 1; return; }
    j -= D;
    for (int k = 2;; ++k) {
        int64_t nw = D - k + 1;
        if (j < nw) { *i_out = (int)j; *k_out = k; return; }
        j -= nw;
    }
}

/* Candidate j of a stage -> window start i and size k. */
static void candidate(const oracle_in_t *in, int64_t j, int *i_out, int *k_out) {
    if (j < in->D) { *i_out = (int)j; *k_out = 1; return; }
    j -= in->D;
    for (int k = 2;; ++k) {
        int64_t nw = in->D - k + 1;
        if (j < nw) { *i_out = (int)j; *k_out = k; return; }
        j -= nw;
    }
}

static int is_frontier(const oracle_in_t *in, int64_t base, int v) {
    int64_t g = base + v;
    if (in->status[g] != ST_PENDING) return 0;
    for (int64_t q = in->par_off[g]; q < in->par_off[g + 1]; ++q)
        if (in->status[base + in->par_idx[q]] != ST_COMPLETED) return 0;
    return 1;
}

/* Count frontier stages and candidates of every instance. */
int oracle_count(const oracle_in_t *in, int B, int64_t *nf, int64_t *nc) {
    for (int b = 0; b < B; ++b) {
        int64_t base = in->stage_off[b], n = in->stage_off[b + 1] - base;
        nf[b] = 0;
        nc[b] = 0;
        for (int v = 0; v < n; ++v)
            if (is_frontier(in, base, v)) { nf[b] += 1; nc[b] += n_candidates(in, base + v); }
    }
    return 0;
}

/* Frontier stages of every instance (instance-local ids), slots as in
 * oracle_score: f_off[b] is the first slot of instance b. */
int oracle_frontier(const oracle_in_t *in, int B, const int64_t *f_off, int32_t *front_v) {
    for (int b = 0; b < B; ++b) {
        int64_t base = in->stage_off[b], n = in->stage_off[b + 1] - base, f = f_off[b];
        for (int v = 0; v < n; ++v)
            if (is_frontier(in, base, v)) front_v[f++] = v;
    }
    return 0;
}

typedef struct { int *depth; int *queue; int *list; int *cptr; int *cidx; int *level; int *nlev; } scratch_t;

/* V2 horizon set of v: every stage reachable from v whose topological level
 * exceeds v's by 1..H, at depth = that difference.  Levels rise along every
 * edge, so a stage beyond the window has no descendant inside it. */
static int horizon_levels(const scratch_t *sc, int n, int v, int H) {
    for (int i = 0; i < n; ++i) sc->depth[i] = -1;
    sc->depth[v] = 0;
    int head = 0, tail = 0, count = 0;
    sc->queue[tail++] = v;
    while (head < tail) {
        int x = sc->queue[head++];
        for (int q = sc->cptr[x]; q < sc->cptr[x + 1]; ++q) {
            int c = sc->cidx[q];
            int dl = sc->level[c] - sc->level[v];
            if (sc->depth[c] >= 0 || dl > H) continue;
            sc->depth[c] = dl;
            sc->queue[tail++] = c;
            sc->list[count++] = c;
        }
    }
    return count;
}

/* Breadth-first horizon set of v: fills list[0..count) with stages at hop
 * distance 1..H (each once, at its minimum distance) and depth[] for them. */
static int horizon(const scratch_t *sc, int n, int v, int H) {
    for (int i = 0; i < n; ++i) sc->depth[i] = -1;
    sc->depth[v] = 0;
    int head = 0, tail = 0, count = 0;
    sc->queue[tail++] = v;
    while (head < tail) {
        int x = sc->queue[head++];
        if (sc->depth[x] >= H) continue;
        for (int q = sc->cptr[x]; q < sc->cptr[x + 1]; ++q) {
            int c = sc->cidx[q];
            if (sc->depth[c] >= 0) continue;
            sc->depth[c] = sc->depth[x] + 1;
            sc->queue[tail++] = c;
            sc->list[count++] = c;
        }
    }
    return count;
}

static void score_instance(const oracle_in_t *in, int b, int64_t f0, int64_t c0, int32_t *front_v,
                           int64_t *cand_off, double *psi, double *mag) {
    int64_t base = in->stage_off[b];
    int n = (int)(in->stage_off[b + 1] - base);
    int D = in->D;
    scratch_t sc;
    sc.depth = (int *)malloc(sizeof(int) * (size_t)(n + 1));
    sc.queue = (int *)malloc(sizeof(int) * (size_t)(n + 1));
    sc.list = (int *)malloc(sizeof(int) * (size_t)(n + 1));
    sc.cptr = (int *)calloc((size_t)n + 2, sizeof(int));
    int64_t E = in->par_off[base + n] - in->par_off[base];
    sc.cidx = (int *)malloc(sizeof(int) * (size_t)(E + 1));
    /* children lists, built from the parent lists */
    for (int x = 0; x < n; ++x)
        for (int64_t q = in->par_off[base + x]; q < in->par_off[base + x + 1]; ++q)
            sc.cptr[in->par_idx[q] + 1] += 1;
    for (int x = 0; x < n; ++x) sc.cptr[x + 1] += sc.cptr[x];
    int *fill = (int *)calloc((size_t)n + 1, sizeof(int));
    for (int x = 0; x < n; ++x)
        for (int64_t q = in->par_off[base + x]; q < in->par_off[base + x + 1]; ++q) {
            int u = in->par_idx[q];
            sc.cidx[sc.cptr[u] + fill[u]++] = x;
        }
    free(fill);
    /* V2: topological levels (parents have smaller ids) */
    sc.level = (int *)calloc((size_t)n + 1, sizeof(int));
    for (int x = 0; x < n; ++x)
        for (int64_t q = in->par_off[base + x]; q < in->par_off[base + x + 1]; ++q) {
            int l = sc.level[in->par_idx[q]] + 1;
            if (l > sc.level[x]) sc.level[x] = l;
        }
    sc.nlev = (int *)calloc(17, sizeof(int));

    view_t cur;
    init_view(&cur, in, b);
    int64_t f = f0, c = c0;
    for (int v = 0; v < n; ++v) {
        if (!is_frontier(in, base, v)) continue;
        int64_t g = base + v;
        int mv = in->model[g];
        int64_t nc = n_candidates(in, g);
        front_v[f] = v;
        cand_off[f] = c;
        int count = in->topo_levels ? horizon_levels(&sc, n, v, in->H) : horizon(&sc, n, v, in->H);
        for (int h = 0; h <= 16; ++h) sc.nlev[h] = 0;
        for (int q = 0; q < count; ++q) sc.nlev[sc.depth[sc.list[q]]] += 1;
        for (int64_t j = 0; j < nc; ++j, ++c) {
            int i0, k;
            candidate(in, j, &i0, &k);
            int ok = 1;
            for (int d = i0; d < i0 + k; ++d)
                if (!feasible(in, g, d)) ok = 0;
            if (!ok || (k > 1 && in->no_windows)) { psi[c] = -INFINITY; mag[c] = 0.0; continue; }
            /* step 5: immediate cost */
            double best_t = -INFINITY, best_mag = 0.0;
            for (int d = i0; d < i0 + k; ++d) {
                double a_q = in->lam_q * wait_cost(&cur, d);
                double a_c = exec_c(in, mv, d) / k;
                double a_s = in->lam_s * switch_cost(&cur, v, d);
                double a_tr = in->lam_tr * transfer_cost(&cur, v, d) / k;
                double a_pf = in->lam_p * prefix_benefit(&cur, v, d) / k;
                double a_co = in->lam_c * colo_benefit(&cur, v, d);
                double a_sm = in->lam_m * same_model(&cur, v, d);
                double t = a_q + a_c + a_s + a_tr - a_pf - a_co - a_sm;
                if (t > best_t) {
                    best_t = t;
                    best_mag = fabs(a_q) + fabs(a_c) + fabs(a_s) + fabs(a_tr) + fabs(a_pf) + fabs(a_co) +
                               fabs(a_sm);
                }
            }
            double gsum = 0.0;
            if (k > 1) {
                gsum = INFINITY;
                for (int p = i0; p < i0 + k; ++p) {
                    double s = 0.0;
                    for (int d = i0; d < i0 + k; ++d)
                        if (d != p) s += (double)in->beta[d * D + p] * (double)in->sigma[g] / k;
                    if (s < gsum) gsum = s;
                }
            }
            double J = best_t + in->lam_tr * gsum;
            double A = best_mag + fabs(in->lam_tr * gsum);
            /* step 6: post-state */
            view_t post = cur;
            uint64_t smask = 0;
            for (int d = i0; d < i0 + k; ++d) {
                smask |= (uint64_t)1 << d;
                post.res[d] = load_model(in, cur.res[d], mv, d);
                post.extra_hash[d] = in->hash[g];
            }
            post.over_stage = v;
            post.over_holders = smask;
            /* steps 7-9: horizon */
            for (int q = 0; q < count; ++q) {
                int w = sc.list[q];
                int64_t gw = base + w;
                double gw_pow = pow(in->gamma, (double)sc.depth[w]);
                if (in->mean_levels) gw_pow /= (double)sc.nlev[sc.depth[w]];
                double vbest = INFINITY, vmag = 0.0;
                for (int d = 0; d < D; ++d) {
                    if (!feasible(in, gw, d)) continue;
                    double m_;
                    double val = c_hat(&post, w, d, &m_);
                    if (val < vbest) { vbest = val; vmag = m_; }
                }
                J += gw_pow * vbest;
                A += gw_pow * vmag;
            }
            psi[c] = -J;
            mag[c] = A;
        }
        ++f;
    }
    free(sc.depth); free(sc.queue); free(sc.list); free(sc.cptr); free(sc.cidx); free(sc.level); free(sc.nlev);
}

/* Score every candidate of every frontier stage.  f_off/c_off[b] are the
 * first frontier slot and first candidate of instance b (prefix sums of
 * oracle_count).  Outputs: front_v[slot] (instance-local stage id),
 * cand_off[slot] (global candidate offset), psi[cand], mag[cand]. */
int oracle_score(const oracle_in_t *in, int B, const int64_t *f_off, const int64_t *c_off,
                 int32_t *front_v, int64_t *cand_off, double *psi, double *mag, int threads) {
    if (in->D < 1 || in->D > 64 || in->M < 1 || in->M > 64) return -1;
    if (in->H < 0 || in->H > 16) return -1;
    if (threads < 1) threads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(threads)
    for (int b = 0; b < B; ++b) score_instance(in, b, f_off[b], c_off[b], front_v, cand_off, psi, mag);
    return 0;
}

/* Top-k of one frontier stage: (Psi descending, index ascending), skipping
 * -infinity, padded with (-1, -infinity). */
int oracle_topk(const double *psi, int64_t nc, int k, int32_t *idx, double *val) {
    unsigned char *taken = (unsigned char *)calloc((size_t)nc + 1, 1);
    for (int r = 0; r < k; ++r) {
        int64_t best = -1;
        for (int64_t j = 0; j < nc; ++j) {
            if (taken[j] || psi[j] == -INFINITY) continue;
            if (best < 0 || psi[j] > psi[best]) best = j;
        }
        if (best < 0) { idx[r] = -1; val[r] = -INFINITY; continue; }
        taken[best] = 1;
        idx[r] = (int32_t)best;
        val[r] = psi[best];
    }
    free(taken);
    return 0;
}

/* Step 11: commit the selected candidates of the current frontier and
 * advance the planning state.  sel[f] is the chosen candidate of frontier
 * slot f (slots as oracle_score lists them, f_off[b] the first slot of
 * instance b), or -1 to leave the stage pending.  The output arrays start as
 * copies of the current state and are updated in place; tau_out is fp64.
 * Returns the number of selections rejected (candidate index out of range,
 * or a device of the candidate infeasible for the stage); those stages stay
 * pending. */
int oracle_commit(const oracle_in_t *in, int B, const int64_t *f_off, const int32_t *front_v,
                  const int32_t *sel, uint64_t *res_out, uint64_t *cache_out, uint64_t *holders_out,
                  uint8_t *status_out, double *tau_out, double *fin_io) {
    const int D = in->D, K = in->K;
    int rejected = 0;
    for (int b = 0; b < B; ++b) {
        int64_t base = in->stage_off[b];
        for (int64_t f = f_off[b]; f < f_off[b + 1]; ++f) {
            if (sel[f] < 0) continue;
            int64_t g = base + front_v[f];
            if (sel[f] >= n_candidates(in, g)) { ++rejected; continue; }
            int i0, k;
            candidate(in, sel[f], &i0, &k);
            int ok = 1;
            for (int d = i0; d < i0 + k; ++d)
                if (!feasible(in, g, d)) ok = 0;
            if (!ok) { ++rejected; continue; }
            int m = in->model[g];
            uint64_t h = in->hash[g];
            uint64_t held = 0;
            double fin = -INFINITY;
            for (int d = i0; d < i0 + k; ++d) {
                int64_t bd = (int64_t)b * D + d;
                double start = tau_out[bd] > (double)in->t_now[b] ? tau_out[bd] : (double)in->t_now[b];
                for (int64_t q = in->par_off[g]; q < in->par_off[g + 1]; ++q) {
                    int64_t u = base + in->par_idx[q];
                    double arr = fin_io[u];
                    if (!has_bit(holders_out[u], d)) {
                        double bmin = INFINITY;
                        for (int i = 0; i < D; ++i)
                            if (has_bit(holders_out[u], i) && (double)in->beta[i * D + d] < bmin)
                                bmin = (double)in->beta[i * D + d];
                        arr = fin_io[u] + (double)in->sigma[u] * bmin / (double)k;
                    }
                    if (arr > start) start = arr;
                }
                double sw = has_bit(res_out[bd], m) ? 0.0 : (double)in->switch_s[m * D + d];
                res_out[bd] = load_model(in, res_out[bd], m, d);
                if (h != 0 && K > 0) {
                    uint64_t *slots = cache_out + bd * K;
                    int present = 0, empty = -1;
                    for (int q = 0; q < K; ++q) {
                        if (slots[q] == h) present = 1;
                        if (slots[q] == 0 && empty < 0) empty = q;
                    }
                    if (!present) {
                        if (empty >= 0) {
                            slots[empty] = h;
                        } else {
                            for (int q = 0; q + 1 < K; ++q) slots[q] = slots[q + 1];
                            slots[K - 1] = h;
                        }
                    }
                }
                tau_out[bd] = start + exec_c(in, m, d) / (double)k + sw;
                if (tau_out[bd] > fin) fin = tau_out[bd];
                held |= (uint64_t)1 << d;
            }
            holders_out[g] = held;
            status_out[g] = ST_COMPLETED;
            fin_io[g] = fin;
        }
    }
    return rejected;
}

/* Step 12: one frontier planning wave per instance.  For frontier slot f
 * (f_off[b] the first slot of instance b, n_cand[f] its stage's number of
 * candidates) the choices are idx[f*k + r], r < k (local candidate indices,
 * -1 = none) with scores val[f*k + r].  sel_out[f] receives the chosen
 * candidate or -1.  Returns the number of stages assigned. */
int oracle_plan_wave(int B, int D, const int64_t *f_off, const int64_t *n_cand, const int32_t *idx,
                     const float *val, int k, int32_t *sel_out) {
    int total = 0;
    for (int b = 0; b < B; ++b) {
        int64_t f0 = f_off[b], f1 = f_off[b + 1];
        for (int64_t f = f0; f < f1; ++f) sel_out[f] = -1;
        uint64_t used = 0;
        for (;;) {
            int64_t best_f = -1;
            int best_r = -1;
            double best_v = -INFINITY;
            uint64_t best_m = 0;
            for (int64_t f = f0; f < f1; ++f) {
                if (sel_out[f] >= 0) continue;
                for (int r = 0; r < k; ++r) {
                    int32_t j = idx[f * k + r];
                    double v = (double)val[f * k + r];
                    if (j < 0 || j >= n_cand[f] || v == -INFINITY) continue;
                    int i0, w;
                    window_of(D, j, &i0, &w);
                    uint64_t m = 0;
                    for (int d = i0; d < i0 + w; ++d) m |= (uint64_t)1 << d;
                    if (m & used) continue;
                    /* strictly better only: earlier slots and ranks win ties */
                    if (best_f < 0 || v > best_v) { best_f = f; best_r = r; best_v = v; best_m = m; }
                }
            }
            if (best_f < 0) break;
            sel_out[best_f] = idx[best_f * k + best_r];
            used |= best_m;
            ++total;
        }
    }
    return total;
}
