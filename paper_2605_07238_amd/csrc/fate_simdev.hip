// Plan execution and baseline placements on the device (App. C.2 metrics,
// App. B comparison schedulers), in fp64 like the host executor.
//
// One 64-lane wave per instance; lane d stands for device d and keeps that
// device's state in registers (free time, resident models, the model it ran
// last) and its prefix slots in LDS, so a stage's shards on the devices of
// S(v) are computed side by side, and the HEFT-style scheduler tries every
// feasible device at once.  A stage's parents are loaded one per lane and
// handed to the device lanes with readlane.  Stages run in (order key, id)
// order; the order is found by counting, for each stage, the stages that
// precede it (the keys staged through LDS).
//
// Execution rule (the same as the host executor): a shard of v on d (k =
// |S(v)|) starts when d is free and every parent's output has arrived (1/k of
// a remote parent's output from its cheapest holder); it pays the switch
// time if m(v) is absent (then Load with eviction), and runs c(v, d) / k, less
// kappa_prefix * L(v) / k (not below 0) when grp(v) is in d's prefix slots;
// grp(v) then joins the slots.  v finishes with its last shard and is then
// held by S(v).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fate_device.h"
#include "fate_internal.h"

// The host executor rounds every product and quotient before it adds; so does this code.
#pragma clang fp contract(off)

namespace fate {
namespace {

constexpr int kRing = FATE_MAX_DEVICES * FATE_MAX_PREFIX_SLOTS;  // prefix slots of one instance
constexpr int kChunk = 512;  // keys per LDS chunk of the ordering count
constexpr int kPer = 4;      // stages ranked per lane and pass

__device__ __forceinline__ uint64_t rl64(uint64_t x, int l) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, l);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ double rld(double x, int l) { return __longlong_as_double((long long)rl64((uint64_t)__double_as_longlong(x), l)); }

// Order-preserving image of a double (no NaN): a larger value, a larger key.
__device__ __forceinline__ uint64_t dkey(double x) {
    const uint64_t u = (uint64_t)__double_as_longlong(x + 0.0);
    return (u >> 63) ? ~u : (u | (1ull << 63));
}
__device__ __forceinline__ double dkey_inv(uint64_t k) {
    const uint64_t u = (k >> 63) ? (k & ~(1ull << 63)) : ~k;
    return __longlong_as_double((long long)u);
}

// Maximum / minimum of a 64-bit key over the wave (every lane active).
__device__ __forceinline__ uint64_t wave_max64(uint64_t x) {
    for (int off = 32; off >= 1; off >>= 1) {
        const uint64_t y = ((uint64_t)(uint32_t)__shfl_xor((int)(x >> 32), off) << 32) | (uint32_t)__shfl_xor((int)(uint32_t)x, off);
        x = y > x ? y : x;
    }
    return x;
}
__device__ __forceinline__ uint64_t wave_min64(uint64_t x) { return ~wave_max64(~x); }

// Make this wave's global and LDS writes visible to its own later reads.
__device__ __forceinline__ void wave_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Per-instance context of the walk.
struct Inst {
    int64_t base, n;
    double t0;
    int lane, D, K;
    bool live;
    // lane d: device d
    double fr;       // free time
    uint64_t res;    // resident models
    int lastm;       // model of the stage it ran last, -1 before the first
};

// Position of each of the cnt stages ids[0..cnt) in (key ascending, index
// ascending) order: out[position] = ids[i].
__device__ void order_by_count(const uint64_t *keys, const uint32_t *ids, int64_t cnt, uint32_t *out,
                               uint64_t *chunk, int lane) {
    for (int64_t i0 = 0; i0 < cnt; i0 += 64 * kPer) {  // uniform
        uint64_t ki[kPer];
        int64_t ii[kPer];
        uint32_t r[kPer];
#pragma unroll
        for (int p = 0; p < kPer; ++p) {
            ii[p] = i0 + p * 64 + lane;
            ki[p] = ii[p] < cnt ? keys[ii[p]] : ~0ull;
            r[p] = 0u;
        }
        for (int64_t j0 = 0; j0 < cnt; j0 += kChunk) {  // uniform
            const int jn = (int)min((int64_t)kChunk, cnt - j0);
            wave_fence();
            for (int t = lane; t < jn; t += 64) chunk[t] = keys[j0 + t];
            wave_fence();
            for (int t = 0; t < jn; ++t) {
                const uint64_t kj = chunk[t];
                const int64_t j = j0 + t;
#pragma unroll
                for (int p = 0; p < kPer; ++p) r[p] += (kj < ki[p] || (kj == ki[p] && j < ii[p])) ? 1u : 0u;
            }
        }
#pragma unroll
        for (int p = 0; p < kPer; ++p)
            if (ii[p] < cnt) out[r[p]] = ids[ii[p]];
    }
    wave_fence();
}

// Finish time of v's shard on this lane's device (k shards) with the parent
// data one per lane in (ph, pf, ps) for parents q0 .. q0+nq-1, folded into
// `ready`; the caller loops over chunks of 64 parents.
__device__ __forceinline__ double arrivals(const SimLaunch &a, const Inst &x, int d, int k, uint64_t ph, double pf,
                                           float ps, int nq, double ready) {
    for (int q = 0; q < nq; ++q) {  // uniform
        const uint64_t h = rl64(ph, q);
        const double f = rld(pf, q);
        const float s = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ps), q));
        double arr;
        if ((h >> d) & 1ull) {
            arr = f;
        } else {
            double bmin = __builtin_huge_val();
            for (uint64_t t = h; t; t &= t - 1) bmin = fmin(bmin, (double)a.beta[__builtin_ctzll(t) * x.D + d]);
            arr = f + ((double)s * bmin) / (double)k;
        }
        ready = fmax(ready, arr);
    }
    return ready;
}

// Shard of stage g (flat) on this lane's device d after the parents' latest
// arrival `ready`: finish time, and whether grp(g) is cached on d.
__device__ __forceinline__ double shard_finish(const SimLaunch &a, const Inst &x, const uint64_t *ring, const StageRec &r,
                                               int d, int k, double ready, bool &hit) {
    const double start = fmax(x.fr, ready);
    const int m = r.model;
    const double sw = ((x.res >> m) & 1ull) ? 0.0 : (double)a.ksw[m * x.D + d];
    hit = false;
    if (r.hash != 0)
        for (int e = 0; e < x.K; ++e) hit = hit || ring[d * x.K + e] == r.hash;
    double run = (double)a.exec[m * x.D + d] / (double)k;
    if (hit) run = fmax(0.0, run - ((a.kpf * (double)r.tokens) / (double)k));
    return (start + sw) + run;
}

// The parents' latest arrival on this lane's device for stage g with k
// shards; also whether every parent has finished (held somewhere) and how
// many parent edges reach no device of S (S = 0: not counted).
__device__ __forceinline__ double parent_ready(const SimLaunch &a, const Inst &x, const StageRec &r, int d, int k,
                                               uint64_t S, bool &all_done, int64_t &xdev) {
    double ready = x.t0;
    all_done = true;
    for (int q0 = 0; q0 < (int)r.npar; q0 += 64) {  // uniform
        const int nq = min(64, (int)r.npar - q0);
        uint64_t ph = 1ull;
        double pf = 0.0;
        float ps = 0.0f;
        if (x.lane < nq) {
            const uint32_t u = a.par_idx[r.par_begin + q0 + x.lane];
            ph = a.hold[u];
            pf = a.fin[u];
            ps = a.rec[u].sigma;
        }
        all_done = all_done && __ballot(ph == 0ull) == 0ull;
        xdev += __popcll(__ballot(x.lane < nq && (ph & S) == 0ull));
        ready = arrivals(a, x, d, k, ph, pf, ps, nq, ready);
    }
    return ready;
}

// Run stage g on the devices of S (lanes of S apply the shard's effects);
// returns its finish, and whether the first device of S hit the prefix
// cache and continued the same model.
__device__ __forceinline__ double run_stage(const SimLaunch &a, Inst &x, uint64_t *ring, const StageRec &r, int64_t g,
                                            uint64_t S, double ready, bool &hit0, bool &cont0) {
    const int k = __popcll(S);
    const int d = x.lane;
    const bool mine = x.live && ((S >> d) & 1ull);
    bool hit = false;
    double fd = x.t0;
    if (mine) fd = shard_finish(a, x, ring, r, d, k, ready, hit);
    const int d0 = __builtin_ctzll(S);
    hit0 = __builtin_amdgcn_readlane(hit ? 1 : 0, d0) != 0;
    cont0 = __builtin_amdgcn_readlane(x.lastm, d0) == (int)r.model;
    if (mine) {
        x.fr = fd;
        x.res = load_model(x.res, r.model, a.cap[d], a.weight);
        // grp(v) joins the slots: the first empty one, else drop the oldest and append
        if (r.hash != 0 && x.K > 0) {
            uint64_t *row = ring + d * x.K;
            bool have = false;
            int empty = -1;
            for (int e = 0; e < x.K; ++e) {
                have = have || row[e] == r.hash;
                if (empty < 0 && row[e] == 0ull) empty = e;
            }
            if (!have) {
                if (empty >= 0) {
                    row[empty] = r.hash;
                } else {
                    for (int e = 0; e + 1 < x.K; ++e) row[e] = row[e + 1];
                    row[x.K - 1] = r.hash;
                }
            }
        }
        x.lastm = r.model;
    }
    const double f = dkey_inv(wave_max64(mine ? dkey(fd) : dkey(x.t0)));  // max(t0, shard finishes)
    if (d == 0) {
        a.fin[g] = f;
        a.hold[g] = S;
    }
    wave_fence();
    return f;
}

template <int MODE>  // 0: execute a plan; 1: round-robin placement; 2: HEFT-style placement
__global__ __launch_bounds__(64) void k_sim(SimLaunch a) {
    __shared__ uint64_t ring[kRing];
    __shared__ uint64_t chunk[kChunk];
    const int b = blockIdx.x;
    Inst x;
    x.lane = threadIdx.x;
    x.D = a.D;
    x.K = a.K;
    x.base = a.stage_off[b];
    x.n = a.stage_off[b + 1] - x.base;
    x.t0 = (double)a.tnow[b];
    x.live = x.lane < x.D;
    const int D = x.D, K = x.K, lane = x.lane;
    const uint64_t dm = D >= 64 ? ~0ull : ((1ull << D) - 1ull);
    x.fr = x.live ? fmax((double)a.tau[(int64_t)b * D + lane], x.t0) : 0.0;
    x.res = x.live ? a.resident[(int64_t)b * D + lane] : 0ull;
    x.lastm = -1;
    for (int e = lane; e < D * K; e += 64) ring[e] = a.pcache[(int64_t)b * D * K + e];
    const int64_t base = x.base, n = x.n;

    // working copies of finish times and holders; children marks
    bool bad = false;
    for (int64_t v = lane; v < n; v += 64) {
        const int64_t g = base + v;
        const uint64_t h = a.holders[g];
        a.hold[g] = h;
        a.fin[g] = h != 0 ? x.t0 : 0.0;
        a.flags[g] = 0;
        if (MODE == 0 && (a.devices[g] & ~dm) != 0) bad = true;
        if (MODE != 0 && h != 0) {  // completed stages are not placed
            a.dev_out[g] = 0ull;
            a.ord_out[g] = 0;
        }
    }
    if (__ballot(bad) != 0ull) {
        if (lane == 0) {
            a.status[b] = FATE_EINVAL;
            a.out[b] = fate_sim_metrics_t{};
        }
        return;
    }
    wave_fence();
    for (int64_t v = lane; v < n; v += 64) {  // a stage with a child is no sink
        const StageRec r = a.rec[base + v];
        for (uint32_t q = 0; q < r.npar; ++q) a.flags[a.par_idx[r.par_begin + q]] = 1;
    }
    wave_fence();

    if (MODE == 1) {  // round robin: each pending stage, in id order, on the next feasible device
        int nxt = 0;
        for (int64_t v = 0; v < n; ++v) {  // uniform
            const int64_t g = base + v;
            uint64_t dev = 0;
            if (a.hold[g] == 0ull) {
                const StageRec r = a.rec[g];
                const uint64_t fm = r.elig & a.fits[r.model] & dm;
                const uint64_t hi = nxt < 64 ? fm & (~0ull << nxt) : 0ull;
                const int d = hi ? __builtin_ctzll(hi) : __builtin_ctzll(fm);
                dev = 1ull << d;
                nxt = d + 1;
            }
            if (lane == 0) {
                a.dev_out[g] = dev;
                a.ord_out[g] = dev ? v : 0;
            }
        }
        if (lane == 0) a.status[b] = FATE_OK;
        return;
    }

    // the stages to run and their order keys
    int64_t cnt = 0;
    if (MODE == 2) {  // HEFT-style: upward ranks, children first (a child has a larger id)
        double bmean = 0.0;  // mean off-diagonal transfer coefficient, summed in row order
        for (int i = 0; i < D; ++i)
            for (int j = 0; j < D; ++j)
                if (i != j) bmean += (double)a.beta[i * D + j];
        bmean = D > 1 ? bmean / (double)(D * (D - 1)) : 0.0;
        double rank_v = 0.0;
        for (int64_t v = n - 1; v >= 0; --v) {  // uniform
            const int64_t g = base + v;
            const StageRec r = a.rec[g];
            double wsum = 0.0;
            int nf = 0;
            const uint64_t fm = r.elig & a.fits[r.model] & dm;
            for (int d = 0; d < D; ++d)
                if ((fm >> d) & 1ull) {
                    wsum += (double)a.exec[r.model * D + d];
                    ++nf;
                }
            const double tail = (a.flags[g] & 2) ? a.tail[g] : 0.0;
            rank_v = wsum / (double)nf + tail;
            // each parent's tail: the largest sigma(u) * mean beta + rank over its children
            for (uint32_t q0 = 0; q0 < r.npar; q0 += 64) {
                const uint32_t q = q0 + lane;
                if (q < r.npar) {
                    const uint32_t u = a.par_idx[r.par_begin + q];
                    const double t = ((double)a.rec[u].sigma * bmean) + rank_v;
                    const uint8_t fl = a.flags[u];
                    a.tail[u] = (fl & 2) ? fmax(a.tail[u], t) : t;
                    a.flags[u] = fl | 2;
                }
            }
            if (lane == 0) a.aux[g] = rank_v;
            wave_fence();
        }
        // pending stages by rank descending, then id
        for (int64_t v0 = 0; v0 < n; v0 += 64) {
            const int64_t v = v0 + lane;
            const bool take = v < n && a.hold[base + v] == 0ull;
            const uint64_t bal = __ballot(take);
            if (take) {
                const int64_t o = cnt + __popcll(bal & ((1ull << lane) - 1ull));
                a.keys[base + o] = ~dkey(a.aux[base + v]);
                a.ids[base + o] = (uint32_t)v;
            }
            cnt += __popcll(bal);
        }
    } else {  // placed pending stages by (order key, id)
        for (int64_t v0 = 0; v0 < n; v0 += 64) {
            const int64_t v = v0 + lane;
            const bool take = v < n && a.hold[base + v] == 0ull && a.devices[base + v] != 0ull;
            const uint64_t bal = __ballot(take);
            if (take) {
                const int64_t o = cnt + __popcll(bal & ((1ull << lane) - 1ull));
                a.keys[base + o] = (uint64_t)a.order[base + v] ^ (1ull << 63);
                a.ids[base + o] = (uint32_t)v;
            }
            cnt += __popcll(bal);
        }
    }
    wave_fence();
    order_by_count(a.keys + base, a.ids + base, cnt, a.todo + base, chunk, lane);

    // the walk
    fate_sim_metrics_t m{};
    int32_t st = FATE_OK;
    for (int64_t p = 0; p < cnt; ++p) {  // uniform
        const int64_t g = base + a.todo[base + p];
        const StageRec r = a.rec[g];
        uint64_t S;
        bool all_done;
        int64_t xdev = 0;
        double ready;
        if (MODE == 2) {  // every feasible device at once; the earliest finish, ties to the lower device
            const int d = lane;
            const bool feas = x.live && ((r.elig & a.fits[r.model]) >> d) & 1ull;
            ready = parent_ready(a, x, r, x.live ? d : 0, 1, ~0ull, all_done, xdev);
            bool hit;
            const double fd = feas ? shard_finish(a, x, ring, r, d, 1, ready, hit) : 0.0;
            const uint64_t best = wave_min64(feas ? dkey(fd) : ~0ull);
            const int bd = (int)wave_min64(feas && dkey(fd) == best ? (uint64_t)d : ~0ull);
            S = 1ull << bd;
            if (lane == 0) {
                a.dev_out[g] = S;
                a.ord_out[g] = p;
            }
        } else {
            S = a.devices[g];
            ready = parent_ready(a, x, r, x.live ? lane : 0, __popcll(S), S, all_done, xdev);
        }
        if (!all_done) {  // the order runs a stage before one of its parents
            st = FATE_ESTATE;
            break;
        }
        bool hit0, cont0;
        run_stage(a, x, ring, r, g, S, ready, hit0, cont0);
        m.tasks += 1;
        m.xdev_edges += xdev;
        m.cache_hits += hit0 ? 1 : 0;
        m.model_cont += cont0 ? 1 : 0;
    }
    if (st != FATE_OK) {
        if (lane == 0) {
            a.status[b] = st;
            a.out[b] = fate_sim_metrics_t{};
        }
        return;
    }
    if (MODE == 2) {
        if (lane == 0) a.status[b] = FATE_OK;
        return;
    }

    // makespan and the p95 of the sinks' completion times
    uint64_t lastk = dkey(x.t0);
    int64_t ns = 0;
    for (int64_t p0 = 0; p0 < cnt; p0 += 64) {
        const int64_t p = p0 + lane;
        bool sink = false;
        double f = x.t0;
        if (p < cnt) {
            const int64_t g = base + a.todo[base + p];
            f = a.fin[g];
            sink = (a.flags[g] & 1) == 0;
        }
        const uint64_t fk = dkey(f);
        lastk = fk > lastk ? fk : lastk;
        const uint64_t bal = __ballot(sink);
        if (sink) a.aux[base + ns + __popcll(bal & ((1ull << lane) - 1ull))] = f - x.t0;
        ns += __popcll(bal);
    }
    m.makespan = dkey_inv(wave_max64(lastk)) - x.t0;
    wave_fence();
    if (ns > 0) {  // nearest rank: the element at 0-based position ceil(0.95 ns) - 1 in ascending order
        const int64_t rk = max((int64_t)0, (int64_t)ceil(0.95 * (double)ns) - 1);
        uint64_t pick = 0ull;
        for (int64_t i0 = 0; i0 < ns; i0 += 64) {
            const int64_t i = i0 + lane;
            const double xi = i < ns ? a.aux[base + i] : 0.0;
            int64_t lt = 0, le = 0;
            for (int64_t j = 0; j < ns; ++j) {
                const double xj = a.aux[base + j];
                lt += xj < xi ? 1 : 0;
                le += xj <= xi ? 1 : 0;
            }
            if (i < ns && lt <= rk && rk < le) pick = dkey(xi);
        }
        m.p95 = dkey_inv(wave_max64(pick));
    }
    if (lane == 0) {
        a.out[b] = m;
        a.status[b] = FATE_OK;
    }
}

}  // namespace

int launch_sim(const SimLaunch &a, int mode, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (a.B <= 0) return 0;
    if (mode == 0) hipLaunchKernelGGL(k_sim<0>, dim3((unsigned)a.B), dim3(64), 0, s, a);
    else if (mode == 1) hipLaunchKernelGGL(k_sim<1>, dim3((unsigned)a.B), dim3(64), 0, s, a);
    else hipLaunchKernelGGL(k_sim<2>, dim3((unsigned)a.B), dim3(64), 0, s, a);
    return (int)hipGetLastError();
}

}  // namespace fate
