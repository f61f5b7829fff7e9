// HIP kernels of libfate for gfx950 (CDNA4, wave64).
//
// k_score: one lane group of G lanes (G = next power of two >= D, 4..64) per
// frontier stage v; lane d stands for device d.
//   1. Lane d evaluates the immediate terms of v on device d (App. A.3):
//      waiting, switch, transfer from completed parents, colocation, prefix
//      reuse, and the post-state of d after loading m(v) (Load with eviction
//      of the smallest-id other models while over capacity).
//   2. Lane d owns the candidates j = d, d+G, d+2G, d+3G (singletons first,
//      then contiguous windows).  For a window S of k devices the immediate
//      cost is the maximum over S of the per-device time with runtime,
//      transfer and prefix split k ways, plus the output gather term (the
//      cheapest gather target in S).
//   3. For each horizon descendant w of v (breadth-first levels 1..H, packed
//      by the host) lane d' computes B(d') = c_hat(w, d' | s) and the value it
//      takes once v sits on d' (model loaded, prefix group cached, v's output
//      local).  A group prefix/suffix minimum over B gives, for every window
//      S, the best device outside S in O(1); the best device inside S is a
//      minimum over at most four lanes.  min(outside, inside) is w's value
//      under candidate S, weighted by gamma^depth and added with compensated
//      summation.
//   This is an exact rearrangement of evaluating c_hat from scratch in the
//   post-state: only v's own output, the model loaded for v and v's prefix
//   group differ between s and s', and they only touch devices of S (plus
//   the transfer of v's output to devices outside S when w is a child of v).
//
// k_topk: same group layout; k rounds of a group-wide maximum over 64-bit
// keys (order-preserving score bits, then inverted candidate index).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fate_internal.h"

namespace fate {
namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ bool bit(uint64_t m, int i) { return (m >> i) & 1ull; }

__device__ __forceinline__ float inf_f() { return __builtin_huge_valf(); }

// Model load under capacity (post-state of a device receiving v).
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

// Cheapest transfer coefficient into device d from any device holding an output.
__device__ __forceinline__ float min_beta_into(const float *beta, uint64_t holders, int d, int D) {
    float m = inf_f();
    for (uint64_t t = holders; t; t &= t - 1) m = fminf(m, beta[__builtin_ctzll(t) * D + d]);
    return m;
}

__device__ __forceinline__ bool cached_on(const uint64_t *slots, int K, uint64_t h) {
    bool hit = false;
    for (int q = 0; q < K; ++q) hit |= (slots[q] == h);
    return hit;
}

// Candidate j of a stage -> window start i and size k (singletons first).
__device__ __forceinline__ void decode_candidate(int j, int D, int &i, int &k) {
    if (j < D) { i = j; k = 1; return; }
    j -= D;
    k = 2;
    while (j >= D - k + 1) { j -= D - k + 1; ++k; }
    i = j;
}

template <int G>
__device__ __forceinline__ float group_prefix_min(float x, int lane) {
#pragma unroll
    for (int off = 1; off < G; off <<= 1) {
        const float y = __shfl_up(x, off, G);
        if (lane >= off) x = fminf(x, y);
    }
    return x;
}

template <int G>
__device__ __forceinline__ float group_suffix_min(float x, int lane) {
#pragma unroll
    for (int off = 1; off < G; off <<= 1) {
        const float y = __shfl_down(x, off, G);
        if (lane + off < G) x = fminf(x, y);
    }
    return x;
}

__device__ __forceinline__ void kahan_add(float &sum, float &comp, float x) {
    const float t = sum + x;
    if (fabsf(sum) >= fabsf(x)) comp += (sum - t) + x;
    else comp += (x - t) + sum;
    sum = t;
}

// Transfer and colocation of stage x onto device d from its completed parents.
__device__ __forceinline__ void parent_terms(const ScoreLaunch &a, const StageRec &rx, int d, float &tr, int &cnt) {
    tr = 0.0f;
    cnt = 0;
    for (int q = 0; q < rx.npar; ++q) {
        const uint32_t u = a.par_idx[rx.par_begin + q];
        const uint64_t hu = a.holders[u];
        if (hu == 0) continue;
        if (bit(hu, d)) { ++cnt; continue; }
        tr += a.rec[u].sigma * min_beta_into(a.beta, hu, d, a.D);
    }
}

template <int G>
__global__ __launch_bounds__(kBlock) void k_score(ScoreLaunch a) {
    constexpr int kSlots = 4;
    const int tid = threadIdx.x;
    const int lane = tid & (G - 1);
    const int64_t f = (int64_t)blockIdx.x * (kBlock / G) + tid / G;
    if (f >= a.nF) return;  // uniform within the group
    const int D = a.D;
    const bool live = lane < D;
    const uint32_t v = a.frontier[2 * f];
    const uint32_t b = a.frontier[2 * f + 1];
    const StageRec rv = a.rec[v];
    const int mv = rv.model;
    const int64_t sd = (int64_t)b * D + (live ? lane : 0);

    // ---- 1. per-device immediate terms and post-state of v on device lane
    uint64_t rho = 0, rho_new = 0;
    bool hv_cached = false, feas_v = false;
    float a_imm = 0.0f, b_imm = 0.0f;
    if (live) {
        rho = a.resident[sd];
        const float wait = fmaxf(0.0f, a.tau[sd] - a.tnow[b]);
        if (rv.hash != 0) hv_cached = cached_on(a.pcache + sd * a.K, a.K, rv.hash);
        feas_v = bit(rv.elig, lane) && bit(a.fits[mv], lane);
        const float c = a.exec[mv * D + lane];
        const float sw = bit(rho, mv) ? 0.0f : a.ksw[mv * D + lane];
        float tr;
        int cnt;
        parent_terms(a, rv, lane, tr, cnt);
        const float colo = rv.npar ? (float)cnt / (float)rv.npar : 0.0f;
        const float pf = hv_cached ? a.kpf * rv.tokens : 0.0f;
        a_imm = a.lam_q * wait + a.lam_s * sw - a.lam_c * colo;
        b_imm = c + a.lam_tr * tr - a.lam_p * pf;
        rho_new = load_model(rho, mv, a.cap[lane], a.weight);
    }
    const bool prefix_added = live && rv.hash != 0 && !hv_cached;
    const int gbase = (tid & 63) & ~(G - 1);
    const uint64_t gmask = (G == 64) ? ~0ull : ((1ull << G) - 1ull);
    const uint64_t feas_mask = (__ballot(feas_v) >> gbase) & gmask;

    // ---- 2. candidates owned by this lane and their immediate cost
    const uint32_t c0 = a.cand_off[f];
    const int C = (int)(a.cand_off[f + 1] - c0);
    const int nslots = (C + G - 1) / G;
    int s_i[kSlots], s_k[kSlots];
    float j0[kSlots], acc[kSlots], comp[kSlots];
    bool ok[kSlots];
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        s_i[s] = 0; s_k[s] = 1; j0[s] = 0.0f; acc[s] = 0.0f; comp[s] = 0.0f; ok[s] = false;
        if (s >= nslots) continue;  // uniform
        const int j = lane + s * G;
        int i = 0, k = 1;
        if (j < C) decode_candidate(j, D, i, k);
        float tmax = -inf_f();
#pragma unroll
        for (int q = 0; q < kSlots; ++q) {
            const int src = min(i + q, G - 1);
            const float aq = __shfl(a_imm, src, G);
            const float bq = __shfl(b_imm, src, G);
            if (q < k) tmax = fmaxf(tmax, aq + bq / (float)k);
        }
        const uint64_t wmask = (k >= 64 ? ~0ull : ((1ull << k) - 1ull)) << i;
        const bool feasible = (j < C) && ((feas_mask & wmask) == wmask);
        float gat = 0.0f;
        if (feasible && k > 1) {
            gat = inf_f();
            for (int p = i; p < i + k; ++p) {
                float sum = 0.0f;
                for (int d = i; d < i + k; ++d)
                    if (d != p) sum += a.beta[d * D + p] * rv.sigma / (float)k;
                gat = fminf(gat, sum);
            }
        }
        s_i[s] = i;
        s_k[s] = k;
        ok[s] = feasible;
        j0[s] = tmax + a.lam_tr * gat;
    }

    // ---- 3. horizon descendants
    const uint32_t e0 = a.desc_off[v], e1 = a.desc_off[v + 1];
    const float t0 = a.lam_tr * rv.sigma * a.beta0;  // uniform-beta transfer of v's output
    const uint64_t *my_slots = a.pcache + sd * a.K;
    int cur_h = 0;
    float gh = 1.0f;
    for (uint32_t e = e0; e < e1; ++e) {
        const uint32_t ent = a.desc[e];
        const int h = (int)(ent >> kDescDepthShift);
        if (h > a.H) break;
        while (cur_h < h) { gh *= a.gamma; ++cur_h; }
        const uint32_t w = ent & kDescIdMask;
        const StageRec rw = a.rec[w];
        const int mw = rw.model;
        const bool child = (h == 1);
        float Bd = inf_f(), inval = inf_f();
        if (live && bit(rw.elig, lane) && bit(a.fits[mw], lane)) {
            const float c = a.exec[mw * D + lane];
            const float kswd = a.ksw[mw * D + lane];
            const bool in_old = bit(rho, mw);
            const bool in_new = bit(rho_new, mw);
            float tr;
            int cnt;
            parent_terms(a, rw, lane, tr, cnt);
            const float colo = rw.npar ? (float)cnt / (float)rw.npar : 0.0f;
            const bool pfw = rw.hash != 0 && cached_on(my_slots, a.K, rw.hash);
            const float pfv = a.kpf * rw.tokens;
            Bd = c + a.lam_s * (in_old ? 0.0f : kswd) + a.lam_tr * tr - a.lam_c * colo - (pfw ? a.lam_p * pfv : 0.0f);
            float dl = 0.0f;
            if (in_new && !in_old) dl -= a.lam_s * kswd;
            else if (!in_new && in_old) dl += a.lam_s * kswd;
            if (prefix_added && rw.hash == rv.hash) dl -= a.lam_p * pfv;
            if (child) dl -= a.lam_c / (float)rw.npar;
            inval = Bd + dl;
        }
        const float P = group_prefix_min<G>(Bd, lane);
        const float Q = group_suffix_min<G>(Bd, lane);
#pragma unroll
        for (int s = 0; s < kSlots; ++s) {
            if (s >= nslots) continue;  // uniform
            const int i = s_i[s], k = s_k[s];
            const float left = __shfl(P, max(i - 1, 0), G);
            const float right = __shfl(Q, min(i + k, G - 1), G);
            float excl = fminf(i > 0 ? left : inf_f(), i + k < G ? right : inf_f());
            if (child) {
                if (a.beta_uniform) {
                    excl += t0;
                } else {
                    excl = inf_f();
                    for (int dd = 0; dd < D; ++dd) {  // uniform trip count
                        const float bdd = __shfl(Bd, dd, G);
                        if (dd >= i && dd < i + k) continue;
                        float bmin = inf_f();
                        for (int q = 0; q < k; ++q) bmin = fminf(bmin, a.beta[(i + q) * D + dd]);
                        excl = fminf(excl, bdd + a.lam_tr * rv.sigma * bmin);
                    }
                }
            }
            float inside = inf_f();
#pragma unroll
            for (int q = 0; q < kSlots; ++q) {
                const float x = __shfl(inval, min(i + q, G - 1), G);
                if (q < k) inside = fminf(inside, x);
            }
            if (ok[s]) kahan_add(acc[s], comp[s], gh * fminf(excl, inside));
        }
    }

    // ---- 4. emit
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        if (s >= nslots) continue;
        const int j = lane + s * G;
        if (j >= C) continue;
        a.scores[c0 + j] = ok[s] ? -(j0[s] + (acc[s] + comp[s])) : -inf_f();
    }
}

__device__ __forceinline__ uint32_t order_bits(float x) {
    const uint32_t u = __float_as_uint(x + 0.0f);  // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float order_bits_inv(uint32_t o) {
    const uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

template <int G>
__global__ __launch_bounds__(kBlock) void k_topk(TopkLaunch a) {
    constexpr int kSlots = 4;
    const int tid = threadIdx.x;
    const int lane = tid & (G - 1);
    const int64_t f = (int64_t)blockIdx.x * (kBlock / G) + tid / G;
    if (f >= a.nF) return;
    const uint32_t c0 = a.cand_off[f];
    const int C = (int)(a.cand_off[f + 1] - c0);
    uint64_t key[kSlots];
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
        key[s] = 0;
        const int j = lane + s * G;
        if (j < C) {
            const float x = a.scores[c0 + j];
            if (x > -inf_f()) key[s] = ((uint64_t)order_bits(x) << 32) | (uint64_t)(0xffffffffu - (uint32_t)j);
        }
    }
    int32_t *out_i = a.idx + f * a.k;
    float *out_v = a.val + f * a.k;
    for (int r = 0; r < a.k; ++r) {
        uint64_t best = key[0];
#pragma unroll
        for (int s = 1; s < kSlots; ++s) best = key[s] > best ? key[s] : best;
#pragma unroll
        for (int off = G / 2; off >= 1; off >>= 1) {
            const uint64_t o = __shfl_xor(best, off, G);
            best = o > best ? o : best;
        }
        if (lane == 0) {
            if (best == 0) { out_i[r] = -1; out_v[r] = -inf_f(); }
            else {
                out_i[r] = (int32_t)(0xffffffffu - (uint32_t)(best & 0xffffffffu));
                out_v[r] = order_bits_inv((uint32_t)(best >> 32));
            }
        }
#pragma unroll
        for (int s = 0; s < kSlots; ++s)
            if (best != 0 && key[s] == best) key[s] = 0;
    }
}

int group_width(int D) {
    int g = 4;
    while (g < D) g <<= 1;
    return g;
}

}  // namespace

int launch_score(const ScoreLaunch &a, void *stream) {
    const int G = group_width(a.D);
    const int64_t groups = kBlock / G;
    const int64_t blocks = (a.nF + groups - 1) / groups;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    switch (G) {
        case 4: hipLaunchKernelGGL(k_score<4>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 8: hipLaunchKernelGGL(k_score<8>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 16: hipLaunchKernelGGL(k_score<16>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 32: hipLaunchKernelGGL(k_score<32>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        default: hipLaunchKernelGGL(k_score<64>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    }
    return (int)hipGetLastError();
}

int launch_topk(const TopkLaunch &a, void *stream) {
    const int G = group_width(a.D);
    const int64_t groups = kBlock / G;
    const int64_t blocks = (a.nF + groups - 1) / groups;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    switch (G) {
        case 4: hipLaunchKernelGGL(k_topk<4>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 8: hipLaunchKernelGGL(k_topk<8>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 16: hipLaunchKernelGGL(k_topk<16>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        case 32: hipLaunchKernelGGL(k_topk<32>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
        default: hipLaunchKernelGGL(k_topk<64>, dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    }
    return (int)hipGetLastError();
}

}  // namespace fate
