// Commit-and-advance of a planning state on the device (Alg. 1: materialise
// the selected placements, then advance the planning frontier and update the
// planning state; Alg. 2: commit into the action pool and update the state
// as the stages complete).  Three launches on the caller's stream; only the
// instances' own frontiers and the children of the stages completed are
// visited, never the whole batch:
//
//   k_commit_apply  one wave per instance.  The wave keeps the instance's
//                   prefix slots, the exec and switch tables, the model
//                   weights and a bitmap over its stages in LDS.  It takes
//                   the instance's frontier slots 64 at a time: lane q
//                   checks slot q's selection and marks the stage completed
//                   with its output on the candidate's devices, or sets the
//                   stage's bit (it stays in the frontier); lane d (device d)
//                   applies, in ascending stage id, every placement whose
//                   candidate contains d: start at max(tau, t), switch time
//                   if the model was absent, Load, prefix slots, free time
//                   (summed in fp64 over the step, stored as fp32).  Then the
//                   children of the stages just completed, one (stage, child)
//                   pair per lane: the child's completed-parent list is
//                   rewritten in its parent slots, and a child whose parents
//                   are now all completed sets its bit.  The set bits, read
//                   in order, are the instance's new frontier: stage ids and
//                   candidate offsets within the instance, and its totals.
//   k_commit_scan   one workgroup: exclusive scan of the instances' totals
//                   (frontier stages, candidates, slices, rejected
//                   selections): frontier offsets per instance and the
//                   counters the scoring and top-k launches read; then the
//                   dispatch order (instances by size class of their
//                   frontier, largest first) and, for batches the general
//                   scoring kernel takes, the instances' slices placed in
//                   that order.
//   k_commit_fill   one wave per instance: its frontier slots, candidate
//                   offsets and scoring slices at the scanned offsets.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "fate_device.h"
#include "fate_internal.h"

namespace fate {
namespace {

constexpr uint8_t kCompleted = FATE_COMPLETED;

// Exclusive scan over the workgroup (NT threads, a multiple of 64) of F
// fields at once; total[] receives the sums.  sh holds F * NT / 64 words.
// Wave-level shuffle scans, one barrier to publish the wave totals (every
// thread adds the totals of the waves before its own), one barrier before sh
// may be reused.
template <int NT, int F>
__device__ void block_exscan(const uint32_t (&x)[F], uint32_t *sh, uint32_t (&ex)[F], uint32_t (&total)[F]) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    constexpr int NW = NT / 64;
    uint32_t v[F];
#pragma unroll
    for (int c = 0; c < F; ++c) v[c] = x[c];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
        for (int c = 0; c < F; ++c) {
            const uint32_t y = __shfl_up(v[c], off, 64);
            if (lane >= off) v[c] += y;
        }
    }
    if (lane == 63) {
#pragma unroll
        for (int c = 0; c < F; ++c) sh[c * NW + wid] = v[c];
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < F; ++c) {
        uint32_t before = 0, all = 0;
        for (int w = 0; w < NW; ++w) {
            const uint32_t t = sh[c * NW + w];
            before += w < wid ? t : 0u;
            all += t;
        }
        ex[c] = before + v[c] - x[c];
        total[c] = all;
    }
    __syncthreads();  // sh may be reused
}

// Parents whose loads one lane issues together.
constexpr int kParBatch = 8;

// One frontier slot of the instance, staged for the lanes of its wave:
// the devices of its selected candidate (0 when none or rejected), the
// stage's prefix group and model, and the candidate's size k.
struct SlotL {
    uint64_t win, hash, wm;  // wm: the model's weight
    double k;
    int32_t model, i0;       // i0: the window's first device
    double ready[FATE_MAX_SHARD];  // when the inputs are on window device i0 + p
};

// Prefix-slot rows in LDS are padded to a multiple of 8 entries so that a
// row is searched 8 entries per batch of loads.
__host__ __device__ inline int padded_slots(int K) { return (K + 7) & ~7; }

// LDS of k_commit_apply: the staged slots and their shards' finish times,
// the exec and switch tables, the model weights and fit masks, the instance's
// prefix-slot rows and each row's ring head, then the instance's bitmap when
// it is kept in LDS (bm_words words).
__host__ __device__ inline size_t apply_lds_bytes(int D, int M, int K, int bm_words) {
    return 64 * sizeof(SlotL) + 64 * 8 * FATE_MAX_SHARD + 8 * (size_t)M * D + 16 * (size_t)M +
           8 * (size_t)D * padded_slots(K) + 4 * (size_t)D + 4 * (size_t)bm_words;
}

// When the outputs of stage s's parents are on each device i0 + p (p < k) of
// a k-shard window: the latest parent finish plus, for a parent whose output
// that device does not hold, its size times the cheapest transfer coefficient
// into the device over k.  The parents' ids, then their holders, finish
// times and sizes, are loaded kParBatch at a time.
__device__ void inputs_ready(const CommitLaunch &a, const StageRec &r, int i0, int k, double (&ready)[FATE_MAX_SHARD]) {
#pragma unroll
    for (int p = 0; p < FATE_MAX_SHARD; ++p) ready[p] = -__builtin_inf();
    for (uint32_t q0 = 0; q0 < r.npar; q0 += kParBatch) {
        uint32_t u[kParBatch];
#pragma unroll
        for (int j = 0; j < kParBatch; ++j) u[j] = q0 + j < r.npar ? a.par_idx[r.par_begin + q0 + j] : 0u;
        uint64_t hu[kParBatch];
        float fu[kParBatch], su[kParBatch];
#pragma unroll
        for (int j = 0; j < kParBatch; ++j) {
            const bool in = q0 + j < r.npar;
            hu[j] = in ? a.holders[u[j]] : 0ull;
            fu[j] = in ? a.fin[u[j]] : 0.0f;
            su[j] = in ? a.rec[u[j]].sigma : 0.0f;
        }
        for (int j = 0; j < kParBatch && q0 + j < r.npar; ++j) {
            for (int p = 0; p < k; ++p) {
                const int d = i0 + p;
                double arr = (double)fu[j];
                if (!bit(hu[j], d)) {
                    double bmin = __builtin_inf();
                    if (a.beta_uniform) {
                        bmin = (double)a.beta0;  // every off-diagonal coefficient
                    } else {
                        for (uint64_t t = hu[j]; t; t &= t - 1) {
                            const double bt = (double)a.beta[__builtin_ctzll(t) * a.D + d];
                            bmin = bt < bmin ? bt : bmin;
                        }
                    }
                    arr = (double)fu[j] + (double)su[j] * bmin / (double)k;
                }
                ready[p] = arr > ready[p] ? arr : ready[p];
            }
        }
    }
}

// Is the nonzero group h in the padded row?  Empty and padding entries
// hold 0, which never equals h, so the whole padded row is compared.
__device__ __forceinline__ bool row_has(const uint64_t *row, int Kp, uint64_t h) {
    bool present = false;
    for (int g = 0; g < Kp; g += 8) {  // uniform
        uint64_t v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = row[g + e];
#pragma unroll
        for (int e = 0; e < 8; ++e) present |= v[e] == h;
    }
    return present;
}

// The first empty entry among the row's K slots (the caller knows one exists).
__device__ __forceinline__ int row_first_empty(const uint64_t *row, int K) {
    int e = 0;
    while (e + 1 < K && row[e] != 0ull) ++e;
    return e;
}

__global__ __launch_bounds__(64) void k_commit_apply(CommitLaunch a) {
    extern __shared__ uint64_t smem[];
    // largest frontiers first, so that the last waves to start are short
    const int b = (int)a.order[blockIdx.x], lane = threadIdx.x, D = a.D, K = a.K, M = a.M, Kp = padded_slots(K);
    SlotL *sl = reinterpret_cast<SlotL *>(smem);
    double *sfin = reinterpret_cast<double *>(smem + (64 * sizeof(SlotL)) / 8);  // [64][FATE_MAX_SHARD]
    uint64_t *wt = reinterpret_cast<uint64_t *>(sfin + 64 * FATE_MAX_SHARD);
    uint64_t *fit = wt + M;
    uint64_t *pslots = fit + M;
    float *ex = reinterpret_cast<float *>(pslots + (size_t)D * Kp);
    float *ks = ex + (size_t)M * D;
    int *heads = reinterpret_cast<int *>(ks + (size_t)M * D);
    // the instance's bitmap: bit bo + i for its stage i (frontier membership
    // after this step), in LDS or in its workspace region
    const int64_t sb = a.stage_off[b], nst = a.stage_off[b + 1] - sb;
    const uint32_t bo = a.bm_lds ? 0u : (uint32_t)(sb & 31);
    uint32_t *bm = a.bm_lds ? reinterpret_cast<uint32_t *>(heads + D) : a.gbm + (sb >> 5) + b;
    const uint32_t words = (uint32_t)((bo + nst + 31) / 32);
    auto mark = [&](int64_t s) {
        const uint32_t i = bo + (uint32_t)(s - sb);
        atomicOr(bm + (i >> 5), 1u << (i & 31));
    };
    for (uint32_t i = lane; i < words; i += 64) bm[i] = 0u;
    for (int i = lane; i < M * D; i += 64) {
        ex[i] = a.exec[i];
        ks[i] = a.ksw[i];
    }
    for (int i = lane; i < M; i += 64) {
        wt[i] = a.weight[i];
        fit[i] = a.fits[i];
    }
    for (int i = lane; i < D * Kp; i += 64) {
        const int dd = i / Kp, e = i - dd * Kp;
        pslots[i] = e < K ? a.pcache[((int64_t)b * D + dd) * K + e] : 0ull;
    }
    const int64_t lo = a.fr_off[b], hi = a.fr_off[b + 1];
    const bool live = lane < D;
    const int d = live ? lane : 0;
    const int64_t t = (int64_t)b * D + d;
    uint64_t res = live ? a.resident[t] : 0ull;
    const uint64_t cap = a.cap[d];
    // free time: summed in fp64 over the step, rounded once when stored
    double tau = live ? (double)a.tau[t] : 0.0;
    const double tn = (double)a.tnow[b];
    uint64_t *row = pslots + d * Kp;
    uint64_t last_h = 0;  // the group this device handled last: it is in its slots
    int last_m = -1;      // the model this device loaded last: it is resident
    uint32_t rejected = 0;
    __syncthreads();
    // resident weight, kept up to date by the loads below
    uint64_t total = 0;
    for (uint64_t r = res; r; r &= r - 1) total += wt[__builtin_ctzll(r)];
    // The row is kept as a ring: logical slot e is row[(head + e) mod K].
    // Dropping slot 0 and appending is then one store and head + 1.  Empty
    // slots exist only before the row first fills, and only then is an
    // empty slot filled, so head stays 0 while any slot is empty.
    int head = 0, nempty = 0;
    for (int e = 0; e < K; ++e) nempty += row[e] == 0ull ? 1 : 0;
    bool held = false;         // uniform: a chunk's children wait for the next pass
    uint32_t hcb = 0, hcn = 0;  // the held chunk's lane: its stage's first child, its pair count
    for (int64_t c0 = lo; c0 < hi; c0 += 64) {  // uniform: chunks of 64 slots
        // lane q checks slot c0 + q and records its stage as completed
        const int64_t f = c0 + lane;
        uint64_t win = 0;
        bool rej = false;
        uint32_t s = 0, cb = 0, cn = 0;
        int kq = 0;
        if (f < hi) {
            s = a.frontier[2 * f];
            const int j = a.sel[f * a.sel_stride];
            const StageRec r = a.rec[s];
            cb = a.ch_off[s];
            cn = a.ch_off[s + 1] - cb;
            SlotL x;
            x.hash = r.hash;
            x.model = r.model;
            x.wm = wt[r.model];
            x.i0 = 0;
            x.k = 1.0;
            if (j >= 0) {
                if (j >= candidates_of(shard_cap_of(r.shard, a.max_shard, D), D)) {
                    rej = true;
                } else {
                    int i0, k;
                    candidate_window(j, D, i0, k);
                    const uint64_t w = ((1ull << k) - 1ull) << i0;
                    if (((r.elig & fit[r.model]) & w) != w) {  // a device not eligible or too small
                        rej = true;
                    } else {
                        win = w;
                        kq = k;
                        x.k = (double)k;
                        x.i0 = i0;
                        // parents completed in earlier steps: their finish
                        // times and holders are settled
                        inputs_ready(a, r, i0, k, x.ready);
                        a.holders[s] = w;
                        a.status[s] = kCompleted;
                    }
                }
            }
            x.win = win;
            sl[lane] = x;
            if (win == 0) mark(s);  // still pending: it stays in the frontier
        }
        rejected += (uint32_t)__popcll(__ballot(rej));
        // lane d collects the slots whose candidate contains device d
        uint64_t mine = 0;
        for (int dd = 0; dd < D; ++dd) {  // uniform
            const uint64_t m = __ballot((win >> dd) & 1ull);
            if (lane == dd) mine = m;
        }
        __syncthreads();
        // each device applies its own placements in ascending stage id
        while (live && mine) {
            const int q = __builtin_ctzll(mine);
            mine &= mine - 1;
            const SlotL x = sl[q];
            const int m = x.model;
            const double ready = x.ready[d - x.i0];
            double start = tau > tn ? tau : tn;
            start = ready > start ? ready : start;
            const double c = (double)ex[m * D + d];
            double sw = 0.0;
            if (m != last_m) {
                last_m = m;
                if (!bit(res, m)) {  // Load, with the resident weight kept running
                    sw = (double)ks[m * D + d];
                    res |= 1ull << m;
                    total += x.wm;
                    for (uint64_t r = res & ~(1ull << m); r && total > cap; r &= r - 1) {
                        const int i = __builtin_ctzll(r);
                        res &= ~(1ull << i);
                        total -= wt[i];
                    }
                }
            }
            if (x.hash != 0 && K > 0 && x.hash != last_h) {  // placements often repeat a group
                last_h = x.hash;
                if (!row_has(row, Kp, x.hash)) {
                    if (nempty > 0) {  // head is 0: the first empty slot in order
                        row[row_first_empty(row, K)] = x.hash;
                        --nempty;
                    } else {  // oldest first: drop slot 0, append
                        row[head] = x.hash;
                        head = head + 1 == K ? 0 : head + 1;
                    }
                }
            }
            tau = start + (x.k == 1.0 ? c : c / x.k) + sw;  // c / 1 is c
            sfin[q * FATE_MAX_SHARD + (d - x.i0)] = tau;
        }
        __syncthreads();  // the next chunk overwrites the staged slots
        if (kq > 0) {  // the stage finishes with its latest shard
            double fs = sfin[lane * FATE_MAX_SHARD];
            for (int p = 1; p < kq; ++p) {
                const double t2 = sfin[lane * FATE_MAX_SHARD + p];
                fs = t2 > fs ? t2 : fs;
            }
            a.fin[s] = (float)fs;
        }
        // Children of the stages completed in this chunk and, every other
        // chunk, in the one before it (its pair counts wait in registers), one
        // (stage, child) pair per lane.  Every parent status and holder set so
        // far is visible to the wave (the barriers above).  A child with
        // several parents completed in this step is rewritten once per such
        // parent, each time from the statuses then settled: a later rewrite
        // sees more completed parents, and the last one sees them all
        // (parents in the same pass write the same list).  No child of a
        // stage pending before this step is in the frontier, so its bit is new.
        const uint32_t ncur = kq > 0 ? cn : 0u;
        if (!held && c0 + 64 < hi) {  // uniform: hold this chunk's children for the next pass
            held = true;
            hcb = cb;
            hcn = ncur;
            __syncthreads();
            continue;
        }
        uint32_t n0 = 0, n1 = 0;
        const uint32_t first0 = wave_exscan_u32(held ? hcn : 0u, n0);  // the held chunk's pairs, then this one's
        const uint32_t first1 = wave_exscan_u32(ncur, n1);
        const uint32_t cb0 = held ? hcb : 0u;
        held = false;
        const uint32_t npairs = n0 + n1;
        for (uint32_t p0 = 0; p0 < npairs; p0 += 64) {  // uniform
            const uint32_t pr = p0 + (uint32_t)lane;
            const bool in1 = pr >= n0;
            const uint32_t pl = in1 ? pr - n0 : pr;  // the pair within its chunk
            // the pair's stage: the last lane of its chunk whose first pair is at or before it
            int q = 0;
#pragma unroll
            for (int step = 32; step >= 1; step >>= 1) {
                const uint32_t f0 = (uint32_t)__shfl((int)first0, q + step), f1 = (uint32_t)__shfl((int)first1, q + step);
                if ((in1 ? f1 : f0) <= pl) q += step;
            }
            const uint32_t qb0 = (uint32_t)__shfl((int)cb0, q), qb1 = (uint32_t)__shfl((int)cb, q);
            const uint32_t qf0 = (uint32_t)__shfl((int)first0, q), qf1 = (uint32_t)__shfl((int)first1, q);
            if (pr < npairs) {
                const uint32_t w = a.ch_idx[in1 ? qb1 + (pl - qf1) : qb0 + (pl - qf0)];
                const StageRec rw = a.rec[w];
                uint32_t nd = 0;
                for (uint32_t q0 = 0; q0 < rw.npar; q0 += kParBatch) {  // the batch's loads are issued together
                    uint32_t u[kParBatch];
#pragma unroll
                    for (int j = 0; j < kParBatch; ++j) u[j] = q0 + j < rw.npar ? a.par_idx[rw.par_begin + q0 + j] : 0u;
                    bool dn[kParBatch];
#pragma unroll
                    for (int j = 0; j < kParBatch; ++j) dn[j] = q0 + j < rw.npar && a.status[u[j]] == kCompleted;
                    DoneParent e[kParBatch];
#pragma unroll
                    for (int j = 0; j < kParBatch; ++j) {
                        e[j].holders = dn[j] ? a.holders[u[j]] : 0ull;
                        e[j].sigma = dn[j] ? a.rec[u[j]].sigma : 0.0f;
                        e[j].pad = 0u;
                    }
#pragma unroll
                    for (int j = 0; j < kParBatch; ++j)
                        if (dn[j]) a.done[rw.par_begin + nd++] = e[j];
                }
                a.done_n[w] = nd;
                if (nd == rw.npar) mark(w);
            }
        }
        __syncthreads();
    }
    if (live) {
        a.resident[t] = res;
        a.tau[t] = (float)tau;
        heads[d] = head;
    }
    __syncthreads();
    for (int i = lane; i < D * K; i += 64) {  // rows back in slot order
        const int dd = i / K, e = i - dd * K;
        int p = heads[dd] + e;
        p = p >= K ? p - K : p;
        a.pcache[(int64_t)b * D * K + i] = pslots[dd * Kp + p];
    }
    // the new frontier in stage order: the set bits, 64 words at a time
    uint2 *lst = reinterpret_cast<uint2 *>(a.list) + sb;
    const bool singles = a.max_shard == 1 || D == 1;  // every stage has D candidates
    uint32_t nf = 0;
    for (uint32_t c = 0; c < words; c += 64) {  // uniform
        uint32_t x = c + lane < words ? bm[c + lane] : 0u;
        uint32_t cnt = 0;
        uint32_t pos = nf + wave_exscan_u32((uint32_t)__popc(x), cnt);
        while (x) {
            const uint32_t i = 32u * (c + lane) + (uint32_t)__builtin_ctz(x) - bo;
            x &= x - 1u;
            lst[pos] = make_uint2((uint32_t)sb + i, singles ? pos * (uint32_t)D : 0u);
            ++pos;
        }
        nf += cnt;
    }
    uint32_t ncand = nf * (uint32_t)D;
    if (!singles) {  // candidate offsets within the instance from the stages' shard caps
        __syncthreads();
        ncand = 0;
        for (uint32_t i0 = 0; i0 < nf; i0 += 64) {  // uniform
            const uint32_t i = i0 + lane;
            uint32_t s = 0, nc = 0;
            if (i < nf) {
                s = lst[i].x;
                nc = (uint32_t)candidates_of(shard_cap_of(a.rec[s].shard, a.max_shard, D), D);
            }
            uint32_t cnt = 0;
            const uint32_t off = ncand + wave_exscan_u32(nc, cnt);
            if (i < nf) lst[i] = make_uint2(s, off);
            ncand += cnt;
        }
    }
    if (lane == 0) {
        const uint32_t slice = (uint32_t)a.slice;
        reinterpret_cast<uint4 *>(a.tot)[b] = make_uint4(nf, ncand, (nf + slice - 1u) / slice, rejected);
    }
}

// Instances per thread of k_commit_scan: 4 K instances take one workgroup scan.
constexpr int kScanItems = 4;

// SLICES: the batch's slices follow the dispatch order (the general scoring
// kernel uses them); otherwise they stay in instance order.
template <bool SLICES>
__global__ __launch_bounds__(1024) void k_commit_scan(CommitLaunch a) {
    constexpr int C = kOrderClasses;
    static_assert(C * kScanItems * 16 < 1024, "one (class, item, wave) count per thread");
    __shared__ uint32_t sh[4 * (1024 / 64)];
    __shared__ uint32_t smax;
    __shared__ uint32_t gcnt[C * kScanItems * 16];      // per (class, item, wave): items
    __shared__ uint32_t gbase[C * kScanItems * 16 + 1];  // their first positions in the batch
    __shared__ uint32_t cstart[C + 1];                   // first position of each class (several batches)
    uint32_t run[4] = {0u, 0u, 0u, 0u};
    const uint4 *tot = reinterpret_cast<const uint4 *>(a.tot);
    if (threadIdx.x == 0) smax = 0u;
    __syncthreads();
    uint32_t mx = 0;  // the largest new frontier
    for (int batch = 0; batch < a.B; batch += kScanItems * 1024) {  // uniform
        const int b0 = batch + (int)threadIdx.x * kScanItems;
        uint4 t[kScanItems];
        uint32_t x[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            t[j] = b0 + j < a.B ? tot[b0 + j] : make_uint4(0u, 0u, 0u, 0u);
            x[0] += t[j].x;
            x[1] += t[j].y;
            x[2] += t[j].z;
            x[3] += t[j].w;
            mx = max(mx, t[j].x);
        }
        uint32_t ex[4], all[4];
        block_exscan<1024, 4>(x, sh, ex, all);
        uint32_t f = run[0] + ex[0], c = run[1] + ex[1], sl = run[2] + ex[2];
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            if (b0 + j >= a.B) break;
            a.fr_off[b0 + j] = f;
            a.base[2 * (b0 + j)] = c;
            if (!SLICES) a.base[2 * (b0 + j) + 1] = sl;  // slices in instance order
            f += t[j].x;
            c += t[j].y;
            sl += t[j].z;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) run[q] += all[q];
    }
    if (threadIdx.x == 0) {
        a.fr_off[a.B] = run[0];
        a.cand_off[run[0]] = run[1];
#pragma unroll
        for (int q = 0; q < 4; ++q) a.counts[q] = run[q];
    }
    // The dispatch order of the next per-instance launches: the instances by
    // size class of their new frontier, largest class first, each class in
    // instance order (a stable partition; no atomics, so the order is the
    // same on every run and equals the host packer's).  Per batch of 4,096
    // instances, item j of thread t is instance batch + 1024 j + t, so that
    // instance order is (j, wave, lane): ballots count each (class, j, wave),
    // one prefix sum over those counts in class-major order places every
    // (class, j, wave) group, and a lane's rank inside its wave's ballot
    // places the item.  Batches before this one put their items of each
    // class first.
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
    if ((threadIdx.x & 63) == 0) atomicMax(&smax, mx);
    __syncthreads();
    mx = smax;
    const int wv = (int)threadIdx.x >> 6, ln = (int)threadIdx.x & 63;
    const uint64_t below = ln ? (~0ull >> (64 - ln)) : 0ull;  // the lanes before this one
    // one batch: ballot counts, their class-major prefix sum into gbase, each
    // item's rank in its wave's ballot
    auto place = [&](int batch, uint32_t (&cl)[kScanItems], uint32_t (&rank)[kScanItems]) {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int b = batch + j * 1024 + (int)threadIdx.x;
            cl[j] = b < a.B ? order_class(tot[b].x, mx) : (uint32_t)C;
        }
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
#pragma unroll
            for (int q = 0; q < C; ++q) {
                const uint64_t m = __ballot(cl[j] == (uint32_t)q);
                if (cl[j] == (uint32_t)q) rank[j] = (uint32_t)__popcll(m & below);
                if (ln == 0) gcnt[(q * kScanItems + j) * 16 + wv] = (uint32_t)__popcll(m);
            }
        }
        __syncthreads();
        const uint32_t x[1] = {threadIdx.x < C * kScanItems * 16 ? gcnt[threadIdx.x] : 0u};
        uint32_t ex[1], all[1];
        block_exscan<1024, 1>(x, sh, ex, all);
        if (threadIdx.x < C * kScanItems * 16) gbase[threadIdx.x] = ex[0];
        if (threadIdx.x == 0) gbase[C * kScanItems * 16] = all[0];
        __syncthreads();
    };
    // the classes' starts over the whole batch of instances
    if (threadIdx.x <= C) cstart[threadIdx.x] = 0u;
    __syncthreads();
    const bool one = a.B <= kScanItems * 1024;  // uniform
    if (!one) {
        for (int batch = 0; batch < a.B; batch += kScanItems * 1024) {  // uniform
            uint32_t cl[kScanItems], rank[kScanItems];
            place(batch, cl, rank);
            if (threadIdx.x < C)
                cstart[threadIdx.x + 1] += gbase[(threadIdx.x + 1) * kScanItems * 16] - gbase[threadIdx.x * kScanItems * 16];
            __syncthreads();
        }
        if (threadIdx.x == 0)
            for (int q = 1; q <= C; ++q) cstart[q] += cstart[q - 1];
        __syncthreads();
    }
    for (int batch = 0; batch < a.B; batch += kScanItems * 1024) {  // uniform: positions
        uint32_t cl[kScanItems], rank[kScanItems];
        place(batch, cl, rank);
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            const int b = batch + j * 1024 + (int)threadIdx.x;
            if (b >= a.B) continue;
            const uint32_t g = (cl[j] * kScanItems + j) * 16 + wv;
            // the class's start over all batches, then this batch's items of
            // the class before this (j, wave) group
            const uint32_t pos = one ? gbase[g] + rank[j]
                                     : cstart[cl[j]] + gbase[g] - gbase[cl[j] * kScanItems * 16] + rank[j];
            a.order[pos] = (uint32_t)b;
            if (SLICES) a.nsp[pos] = tot[b].z;
        }
        __syncthreads();  // gbase is rewritten by the next batch
        if (!one && threadIdx.x < C)  // the next batch's items of a class follow this batch's
            cstart[threadIdx.x] += gbase[(threadIdx.x + 1) * kScanItems * 16] - gbase[threadIdx.x * kScanItems * 16];
        __syncthreads();
    }
    if (!SLICES) return;
    __syncthreads();  // the order and the slice counts by position are complete
    // the instances' first slices, in the dispatch order: the general scoring
    // kernel's workgroups then take the largest frontiers first too
    uint32_t srun = 0;
    for (int batch = 0; batch < a.B; batch += kScanItems * 1024) {  // uniform
        const int i0 = batch + (int)threadIdx.x * kScanItems;
        uint32_t n[kScanItems], bq[kScanItems], x[1] = {0u};
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            n[j] = i0 + j < a.B ? a.nsp[i0 + j] : 0u;
            bq[j] = i0 + j < a.B ? a.order[i0 + j] : 0u;
            x[0] += n[j];
        }
        uint32_t ex[1], all[1];
        block_exscan<1024, 1>(x, sh, ex, all);
        uint32_t sp = srun + ex[0];
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            if (i0 + j < a.B) a.base[2 * bq[j] + 1] = sp;
            sp += n[j];
        }
        srun += all[0];
    }
}

__global__ __launch_bounds__(64) void k_commit_fill(CommitLaunch a) {
    const int b = (int)a.order[blockIdx.x], lane = threadIdx.x;
    const uint32_t F = a.fr_off[b], n = a.fr_off[b + 1] - F;
    const uint2 cs = reinterpret_cast<const uint2 *>(a.base)[b];
    const uint2 *lst = reinterpret_cast<const uint2 *>(a.list) + a.stage_off[b];
    uint2 *fr = reinterpret_cast<uint2 *>(a.frontier);
    for (uint32_t i = lane; i < n; i += 64) {
        const uint2 e = lst[i];
        fr[F + i] = make_uint2(e.x, (uint32_t)b);
        a.cand_off[F + i] = cs.x + e.y;
    }
    const uint32_t slice = (uint32_t)a.slice, ns = (n + slice - 1u) / slice;
    for (uint32_t q = lane; q < ns; q += 64) {
        const int64_t o = 3 * (int64_t)(cs.y + q);
        a.slices[o] = (uint32_t)b;
        a.slices[o + 1] = F + q * slice;
        a.slices[o + 2] = F + min(n, (q + 1u) * slice);
    }
}

}  // namespace

int launch_commit(const CommitLaunch &a, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const size_t lds = apply_lds_bytes(a.D, a.M, a.K, a.bm_lds ? a.bm_words : 0);
    if (a.B > 0) hipLaunchKernelGGL(k_commit_apply, dim3((unsigned)a.B), dim3(64), lds, s, a);
    if (a.slice_order) hipLaunchKernelGGL(k_commit_scan<true>, dim3(1), dim3(1024), 0, s, a);
    else hipLaunchKernelGGL(k_commit_scan<false>, dim3(1), dim3(1024), 0, s, a);
    if (a.B > 0) hipLaunchKernelGGL(k_commit_fill, dim3((unsigned)a.B), dim3(64), 0, s, a);
    return (int)hipGetLastError();
}

}  // namespace fate

// ---- commit-and-advance without a caller workspace -------------------------
// The workspace of fate_commit_advance_noalloc lives in a file-scope device
// array, one copy per GPU, held until the process ends.  In host code the
// array's name is not a device address: its address on each device comes
// from hipGetSymbolAddress, taken once per device with that device current,
// and only that pointer is handed to the kernels.  Every word of the
// workspace is written before it is read within a call, so a call needs no
// clearing; calls that overlap on one GPU share the array and race.
namespace {

__device__ __align__(256) uint8_t scratch[FATE_NOALLOC_WS_BYTES];

std::mutex g_scratch_mu;
void *g_scratch_ptr[FATE_MAX_DEVICES_PER_PROCESS] = {};

// The current device's copy of the array (looked up on the first call).
fate_status_t scratch_of_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= FATE_MAX_DEVICES_PER_PROCESS) return FATE_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FATE_EHIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return FATE_OK;
}

}  // namespace

extern "C" fate_status_t fate_commit_advance_noalloc(const fate_dags_t *dags, const fate_state_h *state,
                                                     const int32_t *d_sel, int32_t sel_stride, void *stream) {
    size_t need = 0;
    fate_status_t st = fate::commit_check(dags, state, d_sel, sel_stride, &need);
    if (st != FATE_OK) return st;
    if (need > (size_t)FATE_NOALLOC_WS_BYTES) return FATE_ERANGE;
    void *ws = nullptr;
    st = scratch_of_current_device(&ws);
    if (st != FATE_OK) return st;
    return fate::commit_impl(dags, state, d_sel, sel_stride, ws, (size_t)FATE_NOALLOC_WS_BYTES, stream);
}
