// Commit-and-advance of a planning state on the device (Alg. 1: materialise
// the selected placements, then advance the planning frontier and update the
// planning state; Alg. 2: commit into the action pool and update the state
// as the stages complete).  Five launches on the caller's stream:
//
//   k_commit_apply  one thread per (instance, device).  It walks the
//                   instance's frontier slots in ascending stage id and
//                   applies every valid selection whose candidate contains
//                   its device: start at max(tau, t), switch time if the
//                   model was absent, Load, prefix slots, free time (summed
//                   in fp64 over the step, stored as fp32).  The
//                   thread of the candidate's first device marks the stage
//                   completed with its output on the candidate's devices.
//   k_plan_count    per stage (kPlanItems consecutive stages per thread):
//                   completed parents, and the candidate count when the stage
//                   is now in the frontier (pending, every parent completed);
//                   workgroup totals.
//   k_plan_offsets  one workgroup: exclusive scan of the workgroup totals;
//                   frontier and candidate totals.
//   k_plan_fill     per stage: offset and entries of its completed-parent
//                   list, its frontier slot and first candidate.
//   k_plan_slices   one workgroup: each instance's frontier range cut into
//                   workgroup slices for the scoring kernel; the counts the
//                   scoring and top-k launches read.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fate_device.h"
#include "fate_internal.h"

namespace fate {
namespace {

constexpr uint8_t kPending = FATE_PENDING, kCompleted = FATE_COMPLETED;

// Exclusive scan over the workgroup (NT threads, a multiple of 64); `total`
// receives the sum.  sh holds NT/64 + 1 words.
template <int NT>
__device__ uint32_t block_exscan(uint32_t x, uint32_t *sh, uint32_t &total) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    uint32_t v = x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(v, off, 64);
        if (lane >= off) v += y;
    }
    if (lane == 63) sh[wid] = v;
    __syncthreads();
    if (tid == 0) {
        uint32_t run = 0;
        for (int w = 0; w < NT / 64; ++w) {
            const uint32_t t = sh[w];
            sh[w] = run;
            run += t;
        }
        sh[NT / 64] = run;
    }
    __syncthreads();
    const uint32_t r = sh[wid] + v - x;
    total = sh[NT / 64];
    __syncthreads();  // sh may be reused
    return r;
}

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

// First frontier slot whose instance is >= b (the frontier is ordered by instance).
__device__ int64_t first_slot_of(const uint32_t *frontier, int64_t nF, uint32_t b) {
    int64_t lo = 0, hi = nF;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (frontier[2 * mid + 1] < b) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(256) void k_commit_apply(CommitLaunch a) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)a.B * a.D) return;
    const int b = (int)(t / a.D), d = (int)(t % a.D), D = a.D, K = a.K;
    const int64_t nF = a.counts[0];
    const int64_t lo = first_slot_of(a.frontier, nF, (uint32_t)b);
    const int64_t hi = first_slot_of(a.frontier, nF, (uint32_t)b + 1u);
    uint64_t res = a.resident[t];
    // free time: summed in fp64 over the step, rounded once when stored
    double tau = (double)a.tau[t];
    const double tn = (double)a.tnow[b];
    uint64_t *slots = a.pcache + t * K;
    uint32_t rejected = 0;
    for (int64_t f = lo; f < hi; ++f) {
        const int j = a.sel[f * a.sel_stride];
        if (j < 0) continue;
        const uint32_t s = a.frontier[2 * f];
        const StageRec r = a.rec[s];
        const int m = r.model;
        if (j >= candidates_of(shard_cap_of(r.shard, a.max_shard, D), D)) {
            ++rejected;
            continue;
        }
        int i0, k;
        candidate_window(j, D, i0, k);
        const uint64_t win = ((1ull << k) - 1ull) << i0;
        if (((r.elig & a.fits[m]) & win) != win) {  // a device not eligible or too small
            ++rejected;
            continue;
        }
        if (d == i0) {
            a.holders[s] = win;
            a.status[s] = kCompleted;
        }
        if (d < i0 || d >= i0 + k) continue;
        const double start = tau > tn ? tau : tn;
        const double sw = bit(res, m) ? 0.0 : (double)a.ksw[m * D + d];
        res = load_model(res, m, a.cap[d], a.weight);
        const uint64_t h = r.hash;
        if (h != 0 && K > 0) {
            bool present = false;
            int empty = -1;
            for (int q = 0; q < K; ++q) {
                present = present || slots[q] == h;
                if (slots[q] == 0 && empty < 0) empty = q;
            }
            if (!present) {
                if (empty >= 0) {
                    slots[empty] = h;
                } else {  // oldest first: drop slot 0, append
                    for (int q = 0; q + 1 < K; ++q) slots[q] = slots[q + 1];
                    slots[K - 1] = h;
                }
            }
        }
        tau = start + (double)a.exec[m * D + d] / (double)k + sw;
    }
    a.resident[t] = res;
    a.tau[t] = (float)tau;
    if (d == 0) a.rej[b] = rejected;
}

__global__ __launch_bounds__(kPlanBlock) void k_plan_count(CommitLaunch a) {
    __shared__ uint32_t sh[kPlanBlock / 64 + 1];
    const int64_t s0 = (int64_t)blockIdx.x * kPlanStages + (int64_t)threadIdx.x * kPlanItems;
    uint32_t tcp = 0, tfr = 0, tnc = 0;
    for (int i = 0; i < kPlanItems; ++i) {
        const int64_t s = s0 + i;
        if (s >= a.N) break;
        const StageRec r = a.rec[s];
        bool ready = a.status[s] == kPending;
        uint32_t cp = 0;
        for (uint32_t q = 0; q < r.npar; ++q) {
            if (a.status[a.par_idx[r.par_begin + q]] == kCompleted) ++cp;
            else ready = false;
        }
        const uint32_t nc = ready ? (uint32_t)candidates_of(shard_cap_of(r.shard, a.max_shard, a.D), a.D) : 0u;
        a.cp[s] = cp;
        a.nc[s] = nc;
        tcp += cp;
        tfr += ready ? 1u : 0u;
        tnc += nc;
    }
    uint32_t tot_cp, tot_fr, tot_nc;
    block_exscan<kPlanBlock>(tcp, sh, tot_cp);
    block_exscan<kPlanBlock>(tfr, sh, tot_fr);
    block_exscan<kPlanBlock>(tnc, sh, tot_nc);
    if (threadIdx.x == 0) {
        a.bsum[3 * blockIdx.x] = tot_cp;
        a.bsum[3 * blockIdx.x + 1] = tot_fr;
        a.bsum[3 * blockIdx.x + 2] = tot_nc;
    }
}

__global__ __launch_bounds__(1024) void k_plan_offsets(CommitLaunch a) {
    __shared__ uint32_t sh[1024 / 64 + 1];
    uint32_t run_cp = 0, run_fr = 0, run_nc = 0;
    for (int base = 0; base < a.nblk; base += 1024) {  // uniform
        const int i = base + (int)threadIdx.x;
        const bool in = i < a.nblk;
        const uint32_t cp = in ? a.bsum[3 * i] : 0u, fr = in ? a.bsum[3 * i + 1] : 0u, nc = in ? a.bsum[3 * i + 2] : 0u;
        uint32_t t_cp, t_fr, t_nc;
        const uint32_t e_cp = block_exscan<1024>(cp, sh, t_cp);
        const uint32_t e_fr = block_exscan<1024>(fr, sh, t_fr);
        const uint32_t e_nc = block_exscan<1024>(nc, sh, t_nc);
        if (in) {
            a.bsum[3 * i] = run_cp + e_cp;
            a.bsum[3 * i + 1] = run_fr + e_fr;
            a.bsum[3 * i + 2] = run_nc + e_nc;
        }
        run_cp += t_cp;
        run_fr += t_fr;
        run_nc += t_nc;
    }
    if (threadIdx.x == 0) {
        a.done_off[a.N] = run_cp;
        a.fidx[a.N] = run_fr;
        a.cand_off[run_fr] = run_nc;
        a.counts[0] = run_fr;
        a.counts[1] = run_nc;
    }
}

__global__ __launch_bounds__(kPlanBlock) void k_plan_fill(CommitLaunch a) {
    __shared__ uint32_t sh[kPlanBlock / 64 + 1];
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
    uint32_t unused;
    uint32_t dpos = a.bsum[3 * blockIdx.x] + block_exscan<kPlanBlock>(tcp, sh, unused);
    uint32_t fpos = a.bsum[3 * blockIdx.x + 1] + block_exscan<kPlanBlock>(tfr, sh, unused);
    uint32_t cpos = a.bsum[3 * blockIdx.x + 2] + block_exscan<kPlanBlock>(tnc, sh, unused);
    for (int i = 0; i < kPlanItems; ++i) {
        const int64_t s = s0 + i;
        if (s >= a.N) break;
        a.done_off[s] = dpos;
        a.fidx[s] = fpos;
        if (nc[i]) {
            a.frontier[2 * (int64_t)fpos] = (uint32_t)s;
            a.frontier[2 * (int64_t)fpos + 1] = (uint32_t)instance_of(a.stage_off, a.B, s);
            a.cand_off[fpos] = cpos;
            ++fpos;
            cpos += nc[i];
        }
        if (cp[i]) {
            const StageRec r = a.rec[s];
            uint32_t e = dpos;
            for (uint32_t q = 0; q < r.npar; ++q) {
                const uint32_t u = a.par_idx[r.par_begin + q];
                if (a.status[u] != kCompleted) continue;
                DoneParent p;
                p.holders = a.holders[u];
                p.sigma = a.rec[u].sigma;
                p.pad = 0u;
                a.done[e++] = p;
            }
            dpos += cp[i];
        }
    }
}

__global__ __launch_bounds__(1024) void k_plan_slices(CommitLaunch a) {
    __shared__ uint32_t sh[1024 / 64 + 1];
    uint32_t run = 0, rej = 0;
    const uint32_t slice = (uint32_t)a.slice;
    for (int base = 0; base < a.B; base += 1024) {  // uniform
        const int b = base + (int)threadIdx.x;
        uint32_t f0 = 0, f1 = 0, nsl = 0, r = 0;
        if (b < a.B) {
            f0 = a.fidx[a.stage_off[b]];
            f1 = a.fidx[a.stage_off[b + 1]];
            nsl = (f1 - f0 + slice - 1) / slice;
            r = a.rej[b];
        }
        uint32_t t_sl, t_rej;
        const uint32_t off = run + block_exscan<1024>(nsl, sh, t_sl);
        block_exscan<1024>(r, sh, t_rej);
        for (uint32_t c = 0; c < nsl; ++c) {
            const int64_t o = 3 * (int64_t)(off + c);
            a.slices[o] = (uint32_t)b;
            a.slices[o + 1] = f0 + c * slice;
            a.slices[o + 2] = min(f0 + (c + 1) * slice, f1);
        }
        run += t_sl;
        rej += t_rej;
    }
    if (threadIdx.x == 0) {
        a.counts[2] = run;
        a.counts[3] = rej;
    }
}

}  // namespace

int launch_commit(const CommitLaunch &a, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t nthr = (int64_t)a.B * a.D;
    if (nthr > 0) hipLaunchKernelGGL(k_commit_apply, dim3((unsigned)((nthr + 255) / 256)), dim3(256), 0, s, a);
    if (a.nblk > 0) hipLaunchKernelGGL(k_plan_count, dim3((unsigned)a.nblk), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_plan_offsets, dim3(1), dim3(1024), 0, s, a);
    if (a.nblk > 0) hipLaunchKernelGGL(k_plan_fill, dim3((unsigned)a.nblk), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_plan_slices, dim3(1), dim3(1024), 0, s, a);
    return (int)hipGetLastError();
}

}  // namespace fate
