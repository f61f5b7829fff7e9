// Frontier planning wave on the device (Alg. 1 planner step, under the wave
// constraints of App. A.2: each device takes at most one shard-slot
// assignment per wave, each stage at most one choice; a window candidate is
// the stage's slots 0..k-1 on k devices, so slot order holds by itself).
// The choices of a frontier stage are its top-k (fate_topk's output); the
// wave is built greedily: the best remaining choice whose stage is still
// unassigned and whose devices are all free is taken, ties going to the
// lower frontier slot, then the lower rank, until no choice is left.
//
//   k_plan_wave  one 64-lane wave per instance.  The instance's choices are
//                staged in LDS as (device mask, order-preserving score key);
//                each round every lane takes the best valid choice among its
//                share, a wave-wide maximum picks the round's winner, and the
//                winner's stage's choices are cleared.  At most D rounds take
//                a choice.  Choices past the LDS capacity are read from HBM
//                each round.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fate_device.h"
#include "fate_internal.h"

namespace fate {
namespace {

// Choices of one instance staged in LDS: 16 KB, so that ten one-wave
// workgroups share a compute unit (2,048 choices, 32 KB, left room for five:
// 0.083 against 0.055 ms per fork-join wave).  Fork-join instances hold about
// 460 choices at k = 4.
constexpr int kPlanCap = 1024;

// Order-preserving map of a finite or +infinite score to a nonzero 32-bit key
// (a larger score gives a larger key, -0 and +0 the same one); 0 marks "no
// valid choice".
__device__ __forceinline__ uint32_t score_key(float v) {
    const uint32_t u = __float_as_uint(v + 0.0f);  // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Devices of candidate j of a stage with nc candidates, or 0 when j is not
// one of them; -infinity and padding are no choice.
__device__ __forceinline__ uint64_t choice_mask(int32_t j, float v, int D, uint32_t nc) {
    if (j < 0 || (uint32_t)j >= nc || !(v > -inf_f())) return 0ull;
    int i0, k;
    candidate_window(j, D, i0, k);
    return ((1ull << k) - 1ull) << i0;
}

struct ChoiceL {
    uint64_t mask;
    uint32_t key, pad;
};

// Maximum over the wave (all 64 lanes active), returned to every lane: DPP
// steps within each 16-lane row (pairs, quads, half-rows, rows), then the four
// row maxima through scalar registers.  No LDS round trips.
template <int CTRL>
__device__ __forceinline__ uint32_t umax_dpp(uint32_t x) {
    return max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = umax_dpp<0xB1>(x);   // quad_perm [1, 0, 3, 2]
    x = umax_dpp<0x4E>(x);   // quad_perm [2, 3, 0, 1]
    x = umax_dpp<0x141>(x);  // row_half_mirror
    x = umax_dpp<0x140>(x);  // row_mirror
    const uint32_t r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
    return max(max(r0, r1), max(r2, r3));
}
// 64-bit maximum: the high words first, then the low words of the lanes
// holding the highest high word.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
    const uint32_t hi = wave_max_u32((uint32_t)(x >> 32));
    const uint32_t lo = wave_max_u32((uint32_t)(x >> 32) == hi ? (uint32_t)x : 0u);
    return ((uint64_t)hi << 32) | lo;
}

__global__ __launch_bounds__(64) void k_plan_wave(PlanLaunch a) {
    __shared__ ChoiceL ch[kPlanCap];
    __shared__ uint32_t taken[64];  // local stages assigned so far (one device each at least)
    const int b = (int)a.order[blockIdx.x], lane = threadIdx.x, k = a.k;  // largest frontiers first
    const int64_t lo = a.fr_off[b], hi = a.fr_off[b + 1];
    const int64_t base = lo * k;
    const uint32_t n = (uint32_t)((hi - lo) * k);
    const uint32_t nl = n < (uint32_t)kPlanCap ? n : (uint32_t)kPlanCap;
    for (int64_t f = lo + lane; f < hi; f += 64) a.sel[f] = -1;
    for (uint32_t c = lane; c < nl; c += 64) {
        const int64_t f = lo + c / (uint32_t)k;
        ChoiceL x;
        x.mask = choice_mask(a.idx[base + c], a.val[base + c], a.D, a.cand_off[f + 1] - a.cand_off[f]);
        x.key = x.mask ? score_key(a.val[base + c]) : 0u;
        x.pad = 0u;
        ch[c] = x;
    }
    __syncthreads();
    uint64_t used = 0;
    int ntaken = 0;
    for (;;) {  // uniform: one assignment per round
        uint64_t best = 0;
        for (uint32_t c = lane; c < n; c += 64) {
            uint64_t m;
            uint32_t key;
            if (c < nl) {
                const ChoiceL x = ch[c];
                m = x.mask;
                key = x.key;
            } else {  // past the LDS capacity: read again, and skip assigned stages
                const float v = a.val[base + c];
                const uint32_t s = c / (uint32_t)k;
                m = choice_mask(a.idx[base + c], v, a.D, a.cand_off[lo + s + 1] - a.cand_off[lo + s]);
                key = m ? score_key(v) : 0u;
                for (int t = 0; t < ntaken; ++t) key = taken[t] == s ? 0u : key;
            }
            // highest key first; among equal keys the lowest choice index
            const uint64_t cand = ((uint64_t)key << 32) | (uint64_t)(0xffffffffu - c);
            if (key != 0u && (m & used) == 0ull && cand > best) best = cand;
        }
        best = wave_max_u64(best);
        if (best == 0ull) break;
        const uint32_t c = 0xffffffffu - (uint32_t)best;
        const uint32_t s = c / (uint32_t)k;
        const int32_t j = a.idx[base + c];
        used |= c < nl ? ch[c].mask
                       : choice_mask(j, a.val[base + c], a.D, a.cand_off[lo + s + 1] - a.cand_off[lo + s]);
        __syncthreads();  // every lane has read the winner's mask
        if (lane == 0) {
            a.sel[lo + s] = j;
            taken[ntaken] = s;
        }
        if (lane < k && s * (uint32_t)k + (uint32_t)lane < nl) ch[s * k + lane].key = 0u;
        ++ntaken;
        __syncthreads();
    }
}

}  // namespace

int launch_plan(const PlanLaunch &a, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (a.B > 0) hipLaunchKernelGGL(k_plan_wave, dim3((unsigned)a.B), dim3(64), 0, s, a);
    return (int)hipGetLastError();
}

}  // namespace fate
