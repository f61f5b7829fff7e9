// Commit-and-advance of a planning state on the device (Alg. 1: materialise
// the selected placements, then advance the planning frontier and update the
// planning state; Alg. 2: commit into the action pool and update the state
// as the stages complete).  Six launches on the caller's stream:
//
//   k_commit_apply  one wave per instance.  The wave keeps the instance's
//                   prefix slots, the exec and switch tables and the model
//                   weights in LDS.  It takes the frontier slots 64 at a
//                   time: lane q checks slot q's selection and marks the
//                   stage completed with its output on the candidate's
//                   devices; then lane d (device d) applies, in ascending
//                   stage id, every placement whose candidate contains d:
//                   start at max(tau, t), switch time if the model was
//                   absent, Load, prefix slots, free time (summed in fp64
//                   over the step, stored as fp32).
//   k_plan_count    per stage (kPlanItems consecutive stages per thread): for
//                   a pending stage its completed parents, and its candidate
//                   count when it is now in the frontier (every parent
//                   completed); workgroup totals.
//   k_plan_segscan  one workgroup per segment of kPlanSeg workgroup totals:
//                   offsets within the segment, segment totals.
//   k_plan_offsets  one workgroup: exclusive scan of the segment totals;
//                   frontier and candidate totals.  (One workgroup reading
//                   all the workgroup totals took 31 us: a single compute
//                   unit keeps too few loads in flight.)
//   k_plan_fill     per stage: offset and entries of its completed-parent
//                   list, its frontier slot, instance and first candidate.
//   k_plan_slices   one workgroup: each instance's frontier range cut into
//                   workgroup slices for the scoring kernel; the counts the
//                   scoring and top-k launches read.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "fate_device.h"
#include "fate_internal.h"

namespace fate {
namespace {

constexpr uint8_t kPending = FATE_PENDING, kCompleted = FATE_COMPLETED;

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

// Parents whose loads one thread issues together in the planning scans.
constexpr int kParBatch = 8;

// Instance of flat stage s: the last b with stage_off[b] <= s.
__device__ int instance_of(const int64_t *stage_off, int B, int64_t s) {
    int lo = 0, hi = B;  // stage_off[lo] <= s < stage_off[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (stage_off[mid] <= s) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Instance of each lane's stage sw + lane, for a wave whose 64 lanes hold
// consecutive stages from sw < N (all lanes active).  A 64-way search finds
// the instance of sw (each round of parallel loads narrows the range
// 64-fold), then the instance starts inside the wave's range, which form a
// prefix of the following instances, move each lane past the starts at or
// before its stage.  Many empty instances can put more than 63 starts in
// the range; those waves search per lane.
__device__ int instance_of_wave(const int64_t *stage_off, int B, int64_t sw) {
    const int lane = threadIdx.x & 63;
    int lo = 0, hi = B;  // stage_off[lo] <= sw < stage_off[hi] (stage_off[B] = N)
    while (hi - lo > 1) {  // uniform
        const int64_t n = hi - lo;
        auto probe = [&](int l) { return lo + 1 + (int)(((int64_t)l * (n - 1)) / 64); };  // in [lo + 1, hi - 1]
        const int cnt = __popcll(__ballot(stage_off[probe(lane)] <= sw));  // the probes at or below sw form a prefix
        const int nlo = cnt > 0 ? probe(cnt - 1) : lo;
        const int nhi = cnt < 64 ? probe(cnt) : hi;
        lo = nlo;
        hi = nhi;
    }
    const int64_t s = sw + lane;
    const int64_t st = stage_off[min(lo + 1 + lane, B)];  // starts after the instance of sw, ascending
    const int k = __popcll(__ballot(st <= sw + 63));
    if (k == 64) return instance_of(stage_off, B, s);
    int inst = lo;
    for (int j = 0; j < k; ++j) inst += s >= __shfl(st, j) ? 1 : 0;  // uniform trip count
    return inst;
}

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
// prefix-slot rows and each row's ring head.
__host__ __device__ inline size_t apply_lds_bytes(int D, int M, int K) {
    return 64 * sizeof(SlotL) + 64 * 8 * FATE_MAX_SHARD + 8 * (size_t)M * D + 16 * (size_t)M +
           8 * (size_t)D * padded_slots(K) + 4 * (size_t)D;
}

// When the outputs of stage s's parents are on device d for a k-shard
// placement: the latest parent finish plus, for a parent whose output d does
// not hold, its size times the cheapest transfer coefficient into d over k.
__device__ double inputs_ready(const CommitLaunch &a, const StageRec &r, int d, int k) {
    double ready = -__builtin_inf();
    for (uint32_t q = 0; q < r.npar; ++q) {
        const uint32_t u = a.par_idx[r.par_begin + q];
        const uint64_t hu = a.holders[u];
        double arr = (double)a.fin[u];
        if (!bit(hu, d)) {
            double bmin = __builtin_inf();
            for (uint64_t t = hu; t; t &= t - 1) {
                const double bt = (double)a.beta[__builtin_ctzll(t) * a.D + d];
                bmin = bt < bmin ? bt : bmin;
            }
            arr = (double)a.fin[u] + (double)a.rec[u].sigma * bmin / (double)k;
        }
        ready = arr > ready ? arr : ready;
    }
    return ready;
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
    const int b = blockIdx.x, lane = threadIdx.x, D = a.D, K = a.K, M = a.M, Kp = padded_slots(K);
    SlotL *sl = reinterpret_cast<SlotL *>(smem);
    double *sfin = reinterpret_cast<double *>(smem + (64 * sizeof(SlotL)) / 8);  // [64][FATE_MAX_SHARD]
    uint64_t *wt = reinterpret_cast<uint64_t *>(sfin + 64 * FATE_MAX_SHARD);
    uint64_t *fit = wt + M;
    uint64_t *pslots = fit + M;
    float *ex = reinterpret_cast<float *>(pslots + (size_t)D * Kp);
    float *ks = ex + (size_t)M * D;
    int *heads = reinterpret_cast<int *>(ks + (size_t)M * D);
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
    const int64_t nF = a.counts[0];
    const int64_t lo = first_slot_of_wave(a.frontier, nF, (uint32_t)b);
    const int64_t hi = first_slot_of_wave(a.frontier, nF, (uint32_t)b + 1u);
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
    for (int64_t c0 = lo; c0 < hi; c0 += 64) {  // uniform: chunks of 64 slots
        // lane q checks slot c0 + q and records its stage as completed
        const int64_t f = c0 + lane;
        uint64_t win = 0;
        bool rej = false;
        uint32_t s = 0;
        int kq = 0;
        if (f < hi) {
            s = a.frontier[2 * f];
            const int j = a.sel[f * a.sel_stride];
            const StageRec r = a.rec[s];
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
                        for (int p = 0; p < k; ++p) x.ready[p] = inputs_ready(a, r, i0 + p, k);
                        a.holders[s] = w;
                        a.status[s] = kCompleted;
                    }
                }
            }
            x.win = win;
            sl[lane] = x;
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
    if (lane == 0) a.rej[b] = rejected;
}

__global__ __launch_bounds__(kPlanBlock) void k_plan_count(CommitLaunch a) {
    __shared__ uint32_t sh[3 * (kPlanBlock / 64)];
    const int64_t s0 = (int64_t)blockIdx.x * kPlanStages + (int64_t)threadIdx.x * kPlanItems;
    uint32_t tcp = 0, tfr = 0, tnc = 0;
    for (int i = 0; i < kPlanItems; ++i) {
        const int64_t s = s0 + i;
        if (s >= a.N) break;
        // only pending stages can be scored (in the frontier or a horizon),
        // so only they carry completed-parent lists
        bool ready = a.status[s] == kPending;
        uint32_t cp = 0, nc = 0;
        if (ready) {
            const StageRec r = a.rec[s];
            for (uint32_t q0 = 0; q0 < r.npar; q0 += kParBatch) {  // the batch's loads are issued together
                uint32_t u[kParBatch];
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) u[j] = q0 + j < r.npar ? a.par_idx[r.par_begin + q0 + j] : 0u;
                uint8_t st[kParBatch];
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) st[j] = q0 + j < r.npar ? a.status[u[j]] : kCompleted;
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) {
                    if (q0 + j >= r.npar) break;
                    if (st[j] == kCompleted) ++cp;
                    else ready = false;
                }
            }
            nc = ready ? (uint32_t)candidates_of(shard_cap_of(r.shard, a.max_shard, a.D), a.D) : 0u;
        }
        a.cp[s] = cp;
        a.nc[s] = nc;
        tcp += cp;
        tfr += ready ? 1u : 0u;
        tnc += nc;
    }
    const uint32_t x[3] = {tcp, tfr, tnc};
    uint32_t ex[3], tot[3];
    block_exscan<kPlanBlock, 3>(x, sh, ex, tot);
    if (threadIdx.x == 0) {
        a.bsum[3 * blockIdx.x] = tot[0];
        a.bsum[3 * blockIdx.x + 1] = tot[1];
        a.bsum[3 * blockIdx.x + 2] = tot[2];
    }
}

// One workgroup per segment of kPlanSeg workgroup totals: the totals become
// offsets within the segment (in place), and the segment total is recorded.
__global__ __launch_bounds__(kPlanBlock) void k_plan_segscan(CommitLaunch a) {
    static_assert(kPlanSeg == kPlanBlock, "one workgroup total per thread");
    __shared__ uint32_t sh[3 * (kPlanBlock / 64)];
    const int seg = (int)blockIdx.x, i = seg * kPlanSeg + (int)threadIdx.x;
    uint32_t x[3] = {0u, 0u, 0u};
    if (i < a.nblk) {
#pragma unroll
        for (int c = 0; c < 3; ++c) x[c] = a.bsum[3 * i + c];
    }
    uint32_t ex[3], tot[3];
    block_exscan<kPlanBlock, 3>(x, sh, ex, tot);
    if (i < a.nblk) {
#pragma unroll
        for (int c = 0; c < 3; ++c) a.bsum[3 * i + c] = ex[c];
    }
    if (threadIdx.x == 0) {
#pragma unroll
        for (int c = 0; c < 3; ++c) a.segsum[3 * seg + c] = tot[c];
    }
}

__global__ __launch_bounds__(1024) void k_plan_offsets(CommitLaunch a) {
    // exclusive scan of the segment totals, 1024 at a time, in place
    __shared__ uint32_t sh[3 * (1024 / 64)];
    uint32_t run[3] = {0u, 0u, 0u};
    for (int batch = 0; batch < a.nseg; batch += 1024) {  // uniform
        const int i = batch + (int)threadIdx.x;
        uint32_t x[3];
#pragma unroll
        for (int c = 0; c < 3; ++c) x[c] = i < a.nseg ? a.segsum[3 * i + c] : 0u;
        uint32_t ex[3], tot[3];
        block_exscan<1024, 3>(x, sh, ex, tot);
        if (i < a.nseg) {
#pragma unroll
            for (int c = 0; c < 3; ++c) a.segsum[3 * i + c] = run[c] + ex[c];
        }
#pragma unroll
        for (int c = 0; c < 3; ++c) run[c] += tot[c];
    }
    if (threadIdx.x == 0) {
        a.done_off[a.N] = run[0];
        a.fidx[a.N] = run[1];
        a.cand_off[run[1]] = run[2];
        a.counts[0] = run[1];
        a.counts[1] = run[2];
    }
}

__global__ __launch_bounds__(kPlanBlock) void k_plan_fill(CommitLaunch a) {
    __shared__ uint32_t sh[3 * (kPlanBlock / 64)];
    const int64_t s0 = (int64_t)blockIdx.x * kPlanStages + (int64_t)threadIdx.x * kPlanItems;
    uint32_t cp[kPlanItems], nc[kPlanItems];
    uint32_t tcp = 0, tfr = 0, tnc = 0;
#pragma unroll
    for (int i = 0; i < kPlanItems; ++i) {
        const int64_t s = s0 + i;
        cp[i] = s < a.N ? a.cp[s] : 0u;
        nc[i] = s < a.N ? a.nc[s] : 0u;
        tcp += cp[i];
        tfr += nc[i] ? 1u : 0u;
        tnc += nc[i];
    }
    const uint32_t x[3] = {tcp, tfr, tnc};
    uint32_t ex[3], tot[3];
    block_exscan<kPlanBlock, 3>(x, sh, ex, tot);
    const int seg = (int)blockIdx.x / kPlanSeg;  // segment offset + offset within the segment + within the workgroup
    uint32_t dpos = a.segsum[3 * seg] + a.bsum[3 * blockIdx.x] + ex[0];
    uint32_t fpos = a.segsum[3 * seg + 1] + a.bsum[3 * blockIdx.x + 1] + ex[1];
    uint32_t cpos = a.segsum[3 * seg + 2] + a.bsum[3 * blockIdx.x + 2] + ex[2];
    static_assert(kPlanItems == 1, "the wave's stages are consecutive, one per lane");
    const int64_t sw = s0 - (threadIdx.x & 63);  // first stage of the wave
    const int inst = sw < a.N ? instance_of_wave(a.stage_off, a.B, sw) : 0;  // uniform condition
    for (int i = 0; i < kPlanItems; ++i) {
        const int64_t s = s0 + i;
        if (s >= a.N) break;
        a.done_off[s] = dpos;
        a.fidx[s] = fpos;
        if (nc[i]) {
            a.frontier[2 * (int64_t)fpos] = (uint32_t)s;
            a.frontier[2 * (int64_t)fpos + 1] = (uint32_t)inst;
            a.cand_off[fpos] = cpos;
            ++fpos;
            cpos += nc[i];
        }
        if (cp[i]) {
            const StageRec r = a.rec[s];
            uint32_t e = dpos;
            for (uint32_t q0 = 0; q0 < r.npar; q0 += kParBatch) {  // the batch's loads are issued together
                uint32_t u[kParBatch];
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) u[j] = q0 + j < r.npar ? a.par_idx[r.par_begin + q0 + j] : 0u;
                bool done[kParBatch];
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) done[j] = q0 + j < r.npar && a.status[u[j]] == kCompleted;
                DoneParent p[kParBatch];
#pragma unroll
                for (int j = 0; j < kParBatch; ++j) {
                    p[j].holders = done[j] ? a.holders[u[j]] : 0ull;
                    p[j].sigma = done[j] ? a.rec[u[j]].sigma : 0.0f;
                    p[j].pad = 0u;
                }
#pragma unroll
                for (int j = 0; j < kParBatch; ++j)
                    if (done[j]) a.done[e++] = p[j];
            }
            dpos += cp[i];
        }
    }
}

// Instances per thread of k_plan_slices: 4 K instances take one workgroup scan.
constexpr int kSliceItems = 4;

__global__ __launch_bounds__(1024) void k_plan_slices(CommitLaunch a) {
    // each thread takes kSliceItems consecutive instances: their frontier
    // ranges, slice and rejection counts; one workgroup scan places them
    __shared__ uint32_t sh[2 * (1024 / 64)];
    const uint32_t slice = (uint32_t)a.slice;
    uint32_t run[2] = {0u, 0u};
    for (int batch = 0; batch < a.B; batch += kSliceItems * 1024) {  // uniform
        const int b0 = batch + (int)threadIdx.x * kSliceItems;
        int64_t so[kSliceItems + 1];
#pragma unroll
        for (int j = 0; j <= kSliceItems; ++j) so[j] = b0 + j <= a.B ? a.stage_off[b0 + j] : 0;
        uint32_t f[kSliceItems + 1], r[kSliceItems];
#pragma unroll
        for (int j = 0; j <= kSliceItems; ++j) f[j] = b0 + j <= a.B ? a.fidx[so[j]] : 0u;
#pragma unroll
        for (int j = 0; j < kSliceItems; ++j) r[j] = b0 + j < a.B ? a.rej[b0 + j] : 0u;
        uint32_t ns[kSliceItems], t[2] = {0u, 0u};
#pragma unroll
        for (int j = 0; j < kSliceItems; ++j) {
            ns[j] = b0 + j < a.B ? (f[j + 1] - f[j] + slice - 1) / slice : 0u;
            t[0] += ns[j];
            t[1] += r[j];
        }
        uint32_t ex[2], tot[2];
        block_exscan<1024, 2>(t, sh, ex, tot);
        uint32_t off = run[0] + ex[0];
#pragma unroll
        for (int j = 0; j < kSliceItems; ++j) {
            if (b0 + j >= a.B) break;
            for (uint32_t q = 0; q < ns[j]; ++q, ++off) {
                const uint32_t fs = f[j] + q * slice;
                const int64_t o = 3 * (int64_t)off;
                a.slices[o] = (uint32_t)(b0 + j);
                a.slices[o + 1] = fs;
                a.slices[o + 2] = min(fs + slice, f[j + 1]);
            }
        }
        run[0] += tot[0];
        run[1] += tot[1];
    }
    if (threadIdx.x == 0) {
        a.counts[2] = run[0];
        a.counts[3] = run[1];
    }
}

}  // namespace

int launch_commit(const CommitLaunch &a, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (a.B > 0)
        hipLaunchKernelGGL(k_commit_apply, dim3((unsigned)a.B), dim3(64), apply_lds_bytes(a.D, a.M, a.K), s, a);
    if (a.nblk > 0) hipLaunchKernelGGL(k_plan_count, dim3((unsigned)a.nblk), dim3(kPlanBlock), 0, s, a);
    if (a.nseg > 0) hipLaunchKernelGGL(k_plan_segscan, dim3((unsigned)a.nseg), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_plan_offsets, dim3(1), dim3(1024), 0, s, a);
    if (a.nblk > 0) hipLaunchKernelGGL(k_plan_fill, dim3((unsigned)a.nblk), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_plan_slices, dim3(1), dim3(1024), 0, s, a);
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
