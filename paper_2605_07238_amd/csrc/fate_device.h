// Device helpers shared by the scoring, commit-and-advance and planning
// kernels of libfate: bit tests, +infinity, the Load rule, the candidate
// numbering of a frontier stage and a wave prefix sum.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fate {

__device__ __forceinline__ bool bit(uint64_t m, int i) { return (m >> i) & 1ull; }

__device__ __forceinline__ float inf_f() { return __builtin_huge_valf(); }

// Load of model m on a device of capacity `cap` (Sec. 3.2 future state, with
// the eviction rule: add m, then drop the smallest-id other resident models
// while the resident weights exceed the capacity).
__device__ __forceinline__ uint64_t load_model(uint64_t res, int m, uint64_t cap, const uint64_t *weight) {
    if (bit(res, m)) return res;
    res |= 1ull << m;
    uint64_t total = 0;
    for (uint64_t t = res; t; t &= t - 1) total += weight[__builtin_ctzll(t)];
    for (uint64_t t = res & ~(1ull << m); t && total > cap; t &= t - 1) {
        const int i = __builtin_ctzll(t);
        res &= ~(1ull << i);
        total -= weight[i];
    }
    return res;
}

// Candidates of a stage with shard cap R (Sec. 3.3 shard slots): the D
// single devices, then the windows {i..i+k-1}, k = 2..r, i = 0..D-k, with
// r = min(R, max_shard, D).
__device__ __forceinline__ int shard_cap_of(int R, int max_shard, int D) {
    int r = R < max_shard ? R : max_shard;
    r = r < D ? r : D;
    return r < 1 ? 1 : r;
}
__device__ __forceinline__ int candidates_of(int r, int D) {
    int c = D;
    for (int k = 2; k <= r; ++k) c += D - k + 1;
    return c;
}
// Candidate j -> first device i and size k.
__device__ __forceinline__ void candidate_window(int j, int D, int &i, int &k) {
    if (j < D) {
        i = j;
        k = 1;
        return;
    }
    j -= D;
    k = 2;
    while (j >= D - k + 1) {
        j -= D - k + 1;
        ++k;
    }
    i = j;
}

// Sum and exclusive prefix sum over the 64 lanes of a wave (all active), in
// DPP moves only: shifts right by 1, 2, 4 and 8 within each row of 16 lanes
// (lanes shifted in from outside the row read 0), then the last lane of row
// 0 and of row 2 added to rows 1 and 3 (row_bcast:15), then the last lane
// of row 1 to rows 2 and 3 (row_bcast:31); the total is lane 63's.
__device__ __forceinline__ uint32_t wave_exscan_u32(uint32_t x, uint32_t &total) {
    uint32_t v = x;
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
    total = (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
    return v - x;
}

}  // namespace fate
