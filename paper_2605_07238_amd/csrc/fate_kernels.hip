// HIP kernels of libfate for gfx950 (CDNA4, wave64).
//
// k_score: one workgroup per (instance, slice of its frontier).  The
// prologue stages the instance's state in LDS: a hash table from prefix group
// to the devices caching it, per-model residency masks, per-device waits and
// capacity fits, and a work-sorted order of the slice's frontier stages (most
// horizon descendants first, so the lane groups of a wave stay balanced).
// Each frontier stage v is then handled by one lane group of G lanes (G =
// next power of two >= D, 4..64); lane d stands for device d.
//   1. Lane d evaluates the immediate terms of v on device d (App. A.3):
//      waiting, switch, transfer from completed parents, colocation, prefix
//      reuse, and the post-state of d after loading m(v) (Load with eviction
//      of the smallest-id other models while over capacity; the slot layout
//      reads it, and the cost terms, from per-block tables built once).
//   2. Slot 0 of lane d is the single-device candidate {d}; slots 1..3 hold
//      contiguous windows.  A window's immediate cost is the maximum over its
//      devices of the per-device time with runtime, transfer and prefix split
//      k ways, plus the output gather term (cheapest gather target).
//   3. For each horizon descendant w of v (breadth-first levels 1..H, packed
//      by the host) lane d' computes B(d') = c_hat(w, d' | s) and the value it
//      takes once v sits on d' (model loaded, prefix group cached, v's output
//      local).  Group prefix/suffix minimum scans over B (DPP row shifts for
//      G <= 16; the slot layout scans order-reversing integer keys with one
//      v_max_u32 per step; 32- and 64-lane groups add the other rows' minima
//      through scalar registers) give the best device outside any window in
//      O(1); the best device inside a window is a minimum over at most four
//      lanes.
//      min(outside, inside) is w's value under the candidate; it is weighted
//      by gamma^depth and accumulated in fp64.
//   This is an exact rearrangement of evaluating c_hat from scratch in the
//   post-state: only v's own output, the model loaded for v and v's prefix
//   group differ between s and s', and they only touch devices of S (plus
//   the transfer of v's output to devices outside S when w is a child of v).
//
// k_topk: one lane group per frontier stage; k rounds of a group-wide maximum
// of order-preserving score bits, then of the lowest candidate index holding it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "fate_device.h"
#include "fate_internal.h"

namespace fate {
namespace {

constexpr int kBlock = kScoreBlock;

// Cheapest transfer coefficient into device d from any device holding an output.
__device__ __forceinline__ float min_beta_into(const float *beta, uint64_t holders, int d, int D) {
    float m = inf_f();
    for (uint64_t t = holders; t; t &= t - 1) m = fminf(m, beta[__builtin_ctzll(t) * D + d]);
    return m;
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

// ---- per-workgroup LDS layout ----------------------------------------------
// Frontier stage of the slice, staged once per workgroup with its candidate
// offsets.
struct StageL {
    uint64_t elig, hash;
    float tokens, sigma;
    uint32_t v, e0, e1, dbeg;
    uint32_t c0, nc;      // first score and number of candidates
    uint16_t dn, npar;
    uint8_t model, shard, pad0, pad1;
    uint64_t pfm;         // devices caching grp(v), looked up once the prefix table is built
};
static_assert(sizeof(StageL) == 64, "StageL");

// Horizon descendant staged by one lane of a group for the whole group, with
// the per-descendant values every device lane needs precomputed.  For a
// uniform transfer coefficient the completed parents are folded into a base
// transfer term (every parent remote) and, per staged parent, the amount a
// device holding that parent's output saves (its transfer plus the
// colocation benefit).
constexpr int kCap = 3;  // completed parents staged per descendant
constexpr int kMore = 4;  // further completed parents loaded per round trip
template <class Mask>
struct EntryL {
    Mask feas;         // devices feasible for w: eligible and able to hold its model
    Mask pfdevs;       // devices whose prefix cache holds grp(w)
    Mask ph[kCap];     // holder masks of the first completed parents
    float gh;          // gamma^depth
    float base_tr;     // lam_tr * beta0 * sum of completed parents' sizes (uniform beta)
    float pfp;         // lam_p * kappa_prefix * L(w)
    float cw;          // lam_c / |Pa(w)|
    uint32_t moff;     // m(w) * D
    uint8_t model;
    uint8_t flags;     // bit 0: child of v; bit 1: same prefix group as v
    uint16_t dn;       // completed parents
    uint32_t dbeg;     // first completed parent
    float pw[kCap];    // uniform beta: lam_tr*beta0*sigma_u + cw; otherwise sigma_u
};
static_assert(sizeof(EntryL<uint32_t>) == 60, "EntryL<u32>");
static_assert(sizeof(EntryL<uint64_t>) == 80, "EntryL<u64>");

// Staging entry of the slot layout (16-lane groups, so D <= 16 and device
// masks fit in 16 bits; at most 32 models): four 16-byte words, read with
// wide LDS loads.  The parent words are read only when w has completed parents.
struct alignas(16) EntryS {
    uint32_t moff;  // m(w) * D: row of w's model in the block's cost table
    uint32_t m1;    // devices feasible for w | devices caching grp(w) << 16
    uint32_t m2;    // devices that gain grp(w) once v runs there | holders of parent 2 << 16
    uint32_t mdn;   // m(w) | completed parents << 8
    float gh;       // gamma^depth
    float xk;       // xbase + (child of v ? v's output to one more device : 0), where xbase =
                    // lam_tr * beta0 * sum of completed parents' sizes (every parent remote)
    float xn;       // xbase - (child of v ? lam_c / |Pa(w)| : 0)
    float pfp;      // lam_p * kappa_prefix * L(w)
    uint32_t dbeg;  // first completed parent
    uint32_t ph01;  // holders of parent 0 | holders of parent 1 << 16
    float pw0;      // what a device holding parent q saves: its transfer plus lam_c / |Pa(w)|
    float pw1;
    float pw2;
    float cw;       // lam_c / |Pa(w)|
    uint32_t pad0, pad1;
};
static_assert(sizeof(EntryS) == 64, "EntryS");

// The slot layout gives each 16-lane group G staging entries plus 16 bytes,
// so the four groups of a wave start on different LDS banks and their wide
// row reads do not conflict.
constexpr int kSlotGroupBytes = 16 * (int)sizeof(EntryS) + 16;

// Bytes of the staging area for lane-group width G in workgroups of BLK
// threads (host and device agree).
template <int G, int BLK>
constexpr int staging_bytes() {
    return G == 16 ? (BLK / 16) * kSlotGroupBytes
                   : BLK * (G <= 32 ? (int)sizeof(EntryL<uint32_t>) : (int)sizeof(EntryL<uint64_t>));
}

template <int G>
using MaskFor = typename std::conditional<(G <= 32), uint32_t, uint64_t>::type;

struct Lds {
    uint64_t *pkey, *rm, *rho, *fits, *wt, *cap, *keys;
    void *pmask;  // device masks of the prefix table: uint32_t when D <= 32, else uint64_t
    uint8_t *order;
    float *wait, *exec, *ksw, *gpow;
    uint32_t *next;  // next chunk of work positions to hand out
    StageL *stages;
    void *entries;
    int logT;
};

__host__ __device__ inline int table_log2(int D, int K) {
    int lt = 4;
    while ((1 << lt) < 2 * D * K) ++lt;
    return lt;
}

__host__ __device__ inline int pow2_at_least(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// Slot layout: per (model m, device d) under the instance's residency, the
// cost of running m on d with the switch term included, the switch term's
// magnitude (what it changes by when m's residency on d flips), and the
// execution and switch terms themselves.
struct alignas(16) CostS {
    float sw0, ksr, exec, swo;
};

// Byte offsets of every LDS array (shared by the launcher and the kernel).
struct LdsPlan {
    uint32_t pkey, pmask, rm, rho, fits, wt, cap, order, wait, gpow, next, exec, ksw, stages, entries, total;
    uint32_t items, parts, left, pbase, plen, pool;  // row splits of heavy stages (64-lane groups)
};

// 64-lane groups: a singletons-only stage with more than kSplitRows
// descendant rows is scored in parts of kSplitRows rows by several waves of
// its workgroup; each part's fp64 sums go to a pool slot, and the wave that
// finishes last adds them in part order and emits.  At most kSplitItems work
// items and kSplitSlots pool slots per workgroup: once they run short a stage
// gets fewer, longer parts (whole 64-row batches), and a stage that cannot
// have two stays whole.
constexpr int kSplitRows = 128, kSplitItems = 256, kSplitSlots = 32;
static_assert(kSplitRows % 64 == 0, "a part is whole 64-row batches");

__host__ __device__ inline LdsPlan lds_plan(int D, int K, int M, int slice, int staging, bool slots, bool split) {
    LdsPlan q;
    const uint32_t T = 1u << table_log2(D, K);
    const uint32_t mask_bytes = D <= 32 ? 4u : 8u;
    uint32_t o = 0;
    q.pkey = o; o += 8 * T;
    q.pmask = o; o += mask_bytes * T;
    o = (o + 7u) & ~7u;
    q.rm = o; o += 8 * (uint32_t)M;
    q.rho = o; o += 8 * (uint32_t)D;
    q.fits = o; o += 8 * (uint32_t)M;
    q.wt = o; o += 8 * (uint32_t)M;
    q.cap = o; o += 8 * (uint32_t)D;
    o = (o + 15u) & ~15u;
    q.stages = o; o += (uint32_t)sizeof(StageL) * (uint32_t)slice;
    q.entries = o; o += (uint32_t)staging;  // also holds the prologue's sort keys
    o = (o + 15u) & ~15u;
    q.order = o; o += ((uint32_t)slice + 15u) & ~15u;
    q.wait = o; o += 4 * (uint32_t)D;
    q.gpow = o; o += 4 * 16;
    q.next = o; o += 16;
    o = (o + 15u) & ~15u;
    if (slots) {  // [M][D] CostS table, then [M][D] residency after each load
        q.exec = o; o += (uint32_t)sizeof(CostS) * (uint32_t)(M * D);
        q.ksw = o; o += 4 * (uint32_t)(M * D);
    } else {  // [M][D] execution times and weighted switch times
        q.exec = o; o += 4 * (uint32_t)(M * D);
        q.ksw = o; o += 4 * (uint32_t)(M * D);
    }
    q.items = q.parts = q.left = q.pbase = q.plen = q.pool = o;
    if (split) {  // items (position | part << 8), parts, parts left, first pool slot, rows per part, then the pool
        q.items = o; o += 2 * kSplitItems;
        q.parts = o; o += ((uint32_t)slice + 3u) & ~3u;
        o = (o + 3u) & ~3u;
        q.left = o; o += 4 * (uint32_t)slice;
        q.pbase = o; o += ((uint32_t)slice + 3u) & ~3u;
        q.plen = o; o += 4 * (uint32_t)slice;
        o = (o + 7u) & ~7u;
        q.pool = o; o += 8 * 64 * kSplitSlots;
    }
    q.total = (o + 15u) & ~15u;
    return q;
}

__device__ __forceinline__ uint32_t table_slot(uint64_t h, int logT) {
    h ^= h >> 31;
    h *= 0x9E3779B97F4A7C15ull;
    return (uint32_t)(h >> (64 - logT));
}

template <class Mask>
__device__ __forceinline__ void table_insert(const Lds &L, uint64_t h, int d) {
    const uint32_t m = (1u << L.logT) - 1u;
    uint32_t s = table_slot(h, L.logT);
    Mask *pm = static_cast<Mask *>(L.pmask);
    for (;;) {
        const unsigned long long old = atomicCAS((unsigned long long *)&L.pkey[s], 0ull, (unsigned long long)h);
        if (old == 0ull || old == h) {
            atomicOr(&pm[s], (Mask)((Mask)1 << d));
            return;
        }
        s = (s + 1u) & m;
    }
}

// Devices whose prefix cache holds group h (0 for h == 0).  The table has
// more slots than distinct keys, so every probe sequence reaches an empty slot.
template <class Mask>
__device__ __forceinline__ Mask table_find(const Lds &L, uint64_t h) {
    if (h == 0) return 0;
    const uint32_t m = (1u << L.logT) - 1u;
    uint32_t s = table_slot(h, L.logT);
    const Mask *pm = static_cast<const Mask *>(L.pmask);
    for (;;) {
        const uint64_t k = L.pkey[s];
        if (k == h) return pm[s];
        if (k == 0) return 0;
        s = (s + 1u) & m;
    }
}

template <int CTRL>
__device__ __forceinline__ float dpp_move(float old, float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Order-reversing float <-> uint32 map (an involution; no NaNs): the larger
// the float, the smaller its key, so a minimum of floats is a maximum of
// keys.  +inf maps to 0x007fffff; key 0 lies below every float's key, so it
// is the identity of the maximum and stands for "no lane": a DPP move with
// bound_ctrl reads 0 where its source lane is outside the row, and the move
// folds into one v_max_u32 with no copy of the destination.
// The map is b ^ (~(b >> 31) & 0x7fffffff): one shift, then one three-input
// bitwise instruction (truth table A ^ (~B & C) = 0xD2 with A, B, C the
// tables 0xF0, 0xCC, 0xAA), written out because the compiler would turn the
// shifted sign into a compare and select.
__device__ __forceinline__ uint32_t key_map(int b) {
    return __builtin_amdgcn_bitop3_b32((uint32_t)b, (uint32_t)(b >> 31), 0x7fffffffu, 0xD2);
}
__device__ __forceinline__ uint32_t fkey(float x) { return key_map(__float_as_int(x)); }
__device__ __forceinline__ float unkey(uint32_t k) { return __uint_as_float(key_map((int)k)); }

constexpr uint32_t kKeyInf = 0x007fffffu;  // key of +inf

// max(x, x of the lane CTRL names); a lane without a source keeps x.
template <int CTRL>
__device__ __forceinline__ uint32_t kmax_dpp(uint32_t x) {
    return max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true));
}
// max(a, x of the lane CTRL names); a lane without a source gets a.
template <int CTRL>
__device__ __forceinline__ uint32_t kmax_from(uint32_t a, uint32_t x) {
    return max(a, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true));
}
// x of the lane CTRL names; 0 ("no lane") where there is none.
template <int CTRL>
__device__ __forceinline__ uint32_t kshift_in(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
// Inclusive prefix / suffix maximum of keys (minimum of the floats) over a
// 16-lane DPP row.
__device__ __forceinline__ uint32_t kscan_up16(uint32_t x) {
    x = kmax_dpp<0x111>(x);
    x = kmax_dpp<0x112>(x);
    x = kmax_dpp<0x114>(x);
    return kmax_dpp<0x118>(x);
}
__device__ __forceinline__ uint32_t kscan_down16(uint32_t x) {
    x = kmax_dpp<0x101>(x);
    x = kmax_dpp<0x102>(x);
    x = kmax_dpp<0x104>(x);
    return kmax_dpp<0x108>(x);
}
// x of the lane CTRL names, 0 where there is none: only for lanes whose
// result is discarded (lets a following min/max fold the move).
template <int CTRL>
__device__ __forceinline__ float dpp_b0(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Inclusive minimum over lanes 0..lane of the group.
template <int G>
__device__ __forceinline__ float scan_min_up(float x, int lane) {
    if constexpr (G == 16) {  // the group is one DPP row; lanes without a source keep x
        x = fminf(x, dpp_move<0x111>(x, x));
        x = fminf(x, dpp_move<0x112>(x, x));
        x = fminf(x, dpp_move<0x114>(x, x));
        x = fminf(x, dpp_move<0x118>(x, x));
        return x;
    } else if constexpr (G < 16) {  // groups sit inside one 16-lane DPP row
        float y = dpp_move<0x111>(inf_f(), x);
        if (lane >= 1) x = fminf(x, y);
        if constexpr (G > 2) { y = dpp_move<0x112>(inf_f(), x); if (lane >= 2) x = fminf(x, y); }
        if constexpr (G > 4) { y = dpp_move<0x114>(inf_f(), x); if (lane >= 4) x = fminf(x, y); }
        if constexpr (G > 8) { y = dpp_move<0x118>(inf_f(), x); if (lane >= 8) x = fminf(x, y); }
        return x;
    } else {
        return group_prefix_min<G>(x, lane);
    }
}

// Inclusive minimum over lanes lane..G-1 of the group.
template <int G>
__device__ __forceinline__ float scan_min_down(float x, int lane) {
    if constexpr (G == 16) {
        x = fminf(x, dpp_move<0x101>(x, x));
        x = fminf(x, dpp_move<0x102>(x, x));
        x = fminf(x, dpp_move<0x104>(x, x));
        x = fminf(x, dpp_move<0x108>(x, x));
        return x;
    } else if constexpr (G < 16) {
        float y = dpp_move<0x101>(inf_f(), x);
        if (lane + 1 < G) x = fminf(x, y);
        if constexpr (G > 2) { y = dpp_move<0x102>(inf_f(), x); if (lane + 2 < G) x = fminf(x, y); }
        if constexpr (G > 4) { y = dpp_move<0x104>(inf_f(), x); if (lane + 4 < G) x = fminf(x, y); }
        if constexpr (G > 8) { y = dpp_move<0x108>(inf_f(), x); if (lane + 8 < G) x = fminf(x, y); }
        return x;
    } else {
        return group_suffix_min<G>(x, lane);
    }
}

// Prefix and suffix minima of two independent rows, steps interleaved so the
// four dependency chains overlap.
template <int G>
__device__ __forceinline__ void scan_min_pair(float &p0, float &q0, float &p1, float &q1, int lane) {
    if constexpr (G == 16) {
        p0 = fminf(p0, dpp_move<0x111>(p0, p0)); q0 = fminf(q0, dpp_move<0x101>(q0, q0));
        p1 = fminf(p1, dpp_move<0x111>(p1, p1)); q1 = fminf(q1, dpp_move<0x101>(q1, q1));
        p0 = fminf(p0, dpp_move<0x112>(p0, p0)); q0 = fminf(q0, dpp_move<0x102>(q0, q0));
        p1 = fminf(p1, dpp_move<0x112>(p1, p1)); q1 = fminf(q1, dpp_move<0x102>(q1, q1));
        p0 = fminf(p0, dpp_move<0x114>(p0, p0)); q0 = fminf(q0, dpp_move<0x104>(q0, q0));
        p1 = fminf(p1, dpp_move<0x114>(p1, p1)); q1 = fminf(q1, dpp_move<0x104>(q1, q1));
        p0 = fminf(p0, dpp_move<0x118>(p0, p0)); q0 = fminf(q0, dpp_move<0x108>(q0, q0));
        p1 = fminf(p1, dpp_move<0x118>(p1, p1)); q1 = fminf(q1, dpp_move<0x108>(q1, q1));
    } else {
        p0 = scan_min_up<G>(p0, lane);
        q0 = scan_min_down<G>(q0, lane);
        p1 = scan_min_up<G>(p1, lane);
        q1 = scan_min_down<G>(q1, lane);
    }
}

// Value of lane-1 (lane 0 gets +inf) and of lane+1 (last lane gets +inf).
template <int G>
__device__ __forceinline__ float from_left(float x, int lane) {
    if constexpr (G == 16) return dpp_move<0x111>(inf_f(), x);
    float y;
    if constexpr (G < 16) y = dpp_move<0x111>(inf_f(), x);
    else y = __shfl_up(x, 1, G);
    return lane >= 1 ? y : inf_f();
}

template <int G>
__device__ __forceinline__ float from_right(float x, int lane) {
    if constexpr (G == 16) return dpp_move<0x101>(inf_f(), x);
    float y;
    if constexpr (G < 16) y = dpp_move<0x101>(inf_f(), x);
    else y = __shfl_down(x, 1, G);
    return lane + 1 < G ? y : inf_f();
}

// Minimum of x over the other lanes of a 32- or 64-lane group, for the lanes
// of a wave that hold whole groups (every lane of the group active): DPP
// prefix and suffix minima within each 16-lane row, then the other rows'
// minima of the group through scalar registers.  No LDS round trips (group
// shuffles take six dependent ones per scan).
template <int G>
__device__ __forceinline__ float others_min_wide(float x, int wl) {
    static_assert(G == 32 || G == 64, "groups of whole DPP rows");
    float p = x, q = x;
    p = fminf(p, dpp_move<0x111>(p, p)); q = fminf(q, dpp_move<0x101>(q, q));
    p = fminf(p, dpp_move<0x112>(p, p)); q = fminf(q, dpp_move<0x102>(q, q));
    p = fminf(p, dpp_move<0x114>(p, p)); q = fminf(q, dpp_move<0x104>(q, q));
    p = fminf(p, dpp_move<0x118>(p, p)); q = fminf(q, dpp_move<0x108>(q, q));
    const float in_row = fminf(dpp_move<0x111>(inf_f(), p), dpp_move<0x101>(inf_f(), q));  // lanes before / after in the row
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), 15));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), 31));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), 47));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p), 63));
    const int row = wl >> 4;
    float rows;
    if constexpr (G == 64) {
        const float m01 = fminf(r0, r1), m23 = fminf(r2, r3);
        rows = row == 0 ? fminf(r1, m23) : row == 1 ? fminf(r0, m23) : row == 2 ? fminf(m01, r3) : fminf(m01, r2);
    } else {  // rows 0, 1 and rows 2, 3 are two groups
        rows = row == 0 ? r1 : row == 1 ? r0 : row == 2 ? r3 : r2;
    }
    return fminf(in_row, rows);
}

// Window t (0-based among a stage's windows) -> start i and size k >= 2.
__device__ __forceinline__ void decode_window(int t, int D, int &i, int &k) {
    k = 2;
    while (t >= D - k + 1) { t -= D - k + 1; ++k; }
    i = t;
}

// Reciprocal to about 1 ulp (one instruction; an IEEE division takes about ten).
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Make the group's LDS writes visible to the other lanes of the same wave.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Lane J of each 16-lane row, to the whole row (DPP row_newbcast).
template <int J>
__device__ __forceinline__ int row_bcast(int x) {
    return __builtin_amdgcn_update_dpp(0, x, 0x150 + J, 0xF, 0xF, false);
}

// Order-preserving 32-bit image of a score (a larger score, a larger value;
// -0 and +0 alike), and its inverse.
__device__ __forceinline__ uint32_t order_bits(float x) {
    const uint32_t u = __float_as_uint(x + 0.0f);  // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float order_bits_inv(uint32_t o) {
    const uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

// Group-wide maximum / minimum of a 32-bit unsigned value.  Inside a 16-lane
// row: DPP steps (rotate by 8, mirror within halves, two quad swaps), each a
// single VALU op with its operand taken from another lane; wider groups finish
// across rows with shuffles.  The identity goes in as the DPP "old" value so
// the move folds into the min/max.
template <int G, bool MAX>
__device__ __forceinline__ uint32_t group_reduce_u32(uint32_t x) {
    constexpr int kId = MAX ? 0 : -1;
    auto op = [](uint32_t p, uint32_t q) { return MAX ? (p > q ? p : q) : (p < q ? p : q); };
    if constexpr (G >= 16) x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)x, 0x128, 0xF, 0xF, false));
    if constexpr (G >= 8) x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)x, 0x141, 0xF, 0xF, false));
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)x, 0xB1, 0xF, 0xF, false));
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)x, 0x4E, 0xF, 0xF, false));
#pragma unroll
    for (int off = 16; off < G; off <<= 1) x = op(x, (uint32_t)__shfl_xor((int)x, off, G));
    return x;
}

// Top-k of one stage held by a lane group: lane l owns candidates l + s*G
// (s < S) as order-preserving score bits, 0 for none or -inf.  Each of k
// rounds takes the group maximum of the bits, then the smallest candidate
// index holding it (ties go to the lower index), and clears that slot.  The
// pick is (index, score), or (-1, -inf) once the group runs out.  For k <= G
// lane r keeps round r's pick and lanes 0..k-1 store them together;
// otherwise lane 0 stores each round's pick.
// The candidate index of slot s on this lane is ci[s] (distinct over the
// group's lanes and slots).
template <int G, int S>
__device__ __forceinline__ void group_topk_at(uint32_t (&sb)[S], const uint32_t (&ci)[S], int lane, int k,
                                              int32_t *out_i, float *out_v) {
    int32_t my_i = -1;
    uint32_t my_m = 0u;
    for (int r = 0; r < k; ++r) {
        uint32_t m = sb[0];
#pragma unroll
        for (int s = 1; s < S; ++s) m = sb[s] > m ? sb[s] : m;
        m = group_reduce_u32<G, true>(m);
        uint32_t jm = 0xffffffffu;
#pragma unroll
        for (int s = S - 1; s >= 0; --s) jm = sb[s] == m && ci[s] < jm ? ci[s] : jm;
        jm = group_reduce_u32<G, false>(jm);
        const int32_t pick = m != 0 ? (int32_t)jm : -1;
        if (k <= G) {  // uniform
            if (lane == r) {
                my_i = pick;
                my_m = m;
            }
        } else if (lane == 0) {
            out_i[r] = pick;
            out_v[r] = m != 0 ? order_bits_inv(m) : -inf_f();
        }
#pragma unroll
        for (int s = 0; s < S; ++s) sb[s] = ci[s] == jm ? 0u : sb[s];
    }
    if (k <= G && lane < k) {
        out_i[lane] = my_i;
        out_v[lane] = my_m != 0 ? order_bits_inv(my_m) : -inf_f();
    }
}
// Candidate l + s*G on lane l, slot s.
template <int G, int S>
__device__ __forceinline__ void group_topk(uint32_t (&sb)[S], int lane, int k, int32_t *out_i, float *out_v) {
    uint32_t ci[S];
#pragma unroll
    for (int s = 0; s < S; ++s) ci[s] = (uint32_t)(lane + s * G);
    group_topk_at<G, S>(sb, ci, lane, k, out_i, out_v);
}

__device__ __forceinline__ uint32_t topk_bits(float x) { return x > -inf_f() ? order_bits(x) : 0u; }

// The slot layout ranks a singletons-only stage after its scoring loop, one
// lane per stage, for k up to kLaneTopk; a stage ranked inside the loop marks
// its slot with kRankedInLoop (the score bits of no float).
constexpr int kLaneTopk = 4;
constexpr uint32_t kRankedInLoop = 0xffffffffu;

// Top-k (k <= kLaneTopk) of up to 16 candidates held by one lane as score
// bits x[0..15] (0 for none or -inf): each candidate, in index order, enters
// a list sorted by bits descending and displaces only strictly smaller
// entries, so among equal scores the lower index ranks first.  The pick is
// (index, score), or (-1, -inf) once the candidates run out.
__device__ __forceinline__ void lane_topk16(const uint32_t (&x)[16], int k, int32_t *out_i, float *out_v) {
    uint32_t t[kLaneTopk];
    int32_t ix[kLaneTopk];
#pragma unroll
    for (int r = 0; r < kLaneTopk; ++r) { t[r] = 0u; ix[r] = -1; }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const uint32_t c = x[j];
        bool gt[kLaneTopk];
#pragma unroll
        for (int r = 0; r < kLaneTopk; ++r) gt[r] = c > t[r];  // gt[r] implies gt[r + 1]
#pragma unroll
        for (int r = kLaneTopk - 1; r > 0; --r) {
            t[r] = gt[r - 1] ? t[r - 1] : (gt[r] ? c : t[r]);
            ix[r] = gt[r - 1] ? ix[r - 1] : (gt[r] ? j : ix[r]);
        }
        t[0] = gt[0] ? c : t[0];
        ix[0] = gt[0] ? j : ix[0];
    }
#pragma unroll
    for (int r = 0; r < kLaneTopk; ++r) {
        if (r < k) {
            out_i[r] = ix[r];
            out_v[r] = t[r] != 0u ? order_bits_inv(t[r]) : -inf_f();
        }
    }
}

template <int G, int R>
__device__ __forceinline__ void rank_stages(const float *scores, const uint32_t (&c0)[R], const int (&C)[R],
                                            const int64_t (&f)[R], int lane, int k, int32_t *idx, float *val) {
    float x[R][4];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int j = lane + s * G;
            x[r][s] = (f[r] >= 0 && j < C[r]) ? scores[c0[r] + j] : -inf_f();
        }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (f[r] < 0) continue;  // uniform within the group
        if (C[r] <= G) {  // one candidate per lane
            uint32_t sb[1] = {topk_bits(x[r][0])};
            group_topk<G, 1>(sb, lane, k, idx + f[r] * k, val + f[r] * k);
        } else {
            uint32_t sb[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) sb[s] = topk_bits(x[r][s]);
            group_topk<G, 4>(sb, lane, k, idx + f[r] * k, val + f[r] * k);
        }
    }
}

// One completed parent's contribution on device d: its output is local
// (colocation count) or has to be transferred from the cheapest holder.
template <bool UNI>
__device__ __forceinline__ void add_parent(const ScoreLaunch &a, uint64_t hu, float su, int d, float &tr, float &cnt) {
    const bool local = bit(hu, d);
    const float bm = UNI ? a.beta0 : min_beta_into(a.beta, hu, d, a.D);
    cnt += local ? 1.0f : 0.0f;
    tr += local ? 0.0f : su * bm;
}

// Is horizon stage w (record rw, at `depth`) a child of the frontier stage v?
// With hop levels exactly the depth-1 stages are.  With topological levels a
// child can sit deeper (another of its parents may have a higher level), so
// its parent list is searched.
__device__ __forceinline__ bool child_of(const ScoreLaunch &a, const StageRec &rw, int depth, uint32_t v) {
    if (depth == 1) return true;
    if (!a.topo) return false;
    for (uint32_t q = 0; q < rw.npar; ++q)
        if (a.par_idx[rw.par_begin + q] == v) return true;
    return false;
}

// VAR = false compiles the scoring variants out (no same-model weight, sum
// over levels, windows on, hop levels); the launcher picks it when no
// parameter set of the launch uses a variant.  SPLIT (64-lane groups) scores
// heavy stages in parts; BLK is the workgroup size.  The launcher takes the
// first of (split, score_block(G)), (no split, score_block(G)), (no split,
// half that) whose LDS plan fits a workgroup.
template <int G, bool UNI, bool SLOTS, bool VAR, bool SPLIT, int BLK>
__global__ __launch_bounds__(BLK) void k_score(ScoreLaunch a) {
    constexpr int kBlock = BLK;  // threads of this workgroup
    static_assert(!SLOTS || (UNI && G == 16), "the slot layout needs 16-lane groups and uniform beta");
    static_assert(!SPLIT || (G == 64 && !SLOTS), "heavy-stage parts are for 64-lane groups");
    // a planning state is launched over its slice capacity; the current
    // number of slices is on the device
    const uint32_t slice = blockIdx.x;
    if (a.dcounts && slice >= a.dcounts[2]) return;
    // parameter set of this block (a sweep launches one grid row per set)
    const ParamSet ps = a.ps[blockIdx.y];
    float *const scores = a.scores + (int64_t)a.set_of[blockIdx.y] * a.score_stride;
    extern __shared__ uint64_t smem[];
    uint8_t *sb = reinterpret_cast<uint8_t *>(smem);
    const int tid = threadIdx.x;
    const int D = a.D, K = a.K, M = a.M;
    const uint32_t b = a.slices[3 * slice];
    const uint32_t f0 = a.slices[3 * slice + 1];
    // a slice holds at most a.slice stages (the LDS plan's size); a longer one,
    // from a state that another build packed, is cut rather than overrun LDS
    const int nF = min((int)(a.slices[3 * slice + 2] - f0), a.slice);
    const int P = pow2_at_least(nF);
    using Mask = MaskFor<G>;  // device bitmask
    // slot layout: 16-lane groups, uniform beta, at most 32 models (chosen by the launcher)
    constexpr bool kSlots = SLOTS;
    using Entry = EntryL<Mask>;
    constexpr bool kSplit = SPLIT;
    const LdsPlan plan = lds_plan(D, K, M, a.slice, staging_bytes<G, BLK>(), SLOTS, kSplit);

    Lds L;
    L.logT = table_log2(D, K);
    const int T = 1 << L.logT;
    L.pkey = reinterpret_cast<uint64_t *>(sb + plan.pkey);
    L.pmask = sb + plan.pmask;
    L.rm = reinterpret_cast<uint64_t *>(sb + plan.rm);
    L.rho = reinterpret_cast<uint64_t *>(sb + plan.rho);
    L.fits = reinterpret_cast<uint64_t *>(sb + plan.fits);
    L.order = sb + plan.order;
    L.keys = reinterpret_cast<uint64_t *>(sb + plan.entries);
    L.stages = reinterpret_cast<StageL *>(sb + plan.stages);
    L.entries = sb + plan.entries;
    L.wt = reinterpret_cast<uint64_t *>(sb + plan.wt);
    L.cap = reinterpret_cast<uint64_t *>(sb + plan.cap);
    L.wait = reinterpret_cast<float *>(sb + plan.wait);
    L.exec = reinterpret_cast<float *>(sb + plan.exec);
    L.ksw = reinterpret_cast<float *>(sb + plan.ksw);
    L.gpow = reinterpret_cast<float *>(sb + plan.gpow);
    L.next = reinterpret_cast<uint32_t *>(sb + plan.next);

    // ---- prologue: instance tables, cluster tables, the slice's stages
    for (int i = tid; i < T; i += kBlock) { L.pkey[i] = 0; static_cast<Mask *>(L.pmask)[i] = 0; }
    if (tid < D) {
        L.rho[tid] = a.resident[(int64_t)b * D + tid];
        L.wait[tid] = fmaxf(0.0f, a.tau[(int64_t)b * D + tid] - a.tnow[b]);
        L.cap[tid] = a.cap[tid];
    }
    if (tid < M) { L.fits[tid] = a.fits[tid]; L.wt[tid] = a.weight[tid]; }
    if (tid == 0) {
        float g = 1.0f;
        for (int h = 0; h < 16; ++h) { L.gpow[h] = g; g *= ps.gamma; }
        *L.next = 0u;
    }
    if constexpr (SLOTS) {
        // cost table (the residency after each load follows after the barrier)
        const float res = VAR ? -ps.lam_m : 0.0f;
        CostS *tab = reinterpret_cast<CostS *>(L.exec);
        for (int i = tid; i < M * D; i += kBlock) {
            const int m = i / D, d = i - m * D;
            const float ks = ps.lam_s * a.ksw[i];
            const uint64_t rd = a.resident[(int64_t)b * D + d];
            const float swo = bit(rd, m) ? res : ks;
            CostS c;
            c.sw0 = a.exec[i] + swo;
            c.ksr = ks - res;
            c.exec = a.exec[i];
            c.swo = swo;
            tab[i] = c;
        }
    } else {
        for (int i = tid; i < M * D; i += kBlock) { L.exec[i] = a.exec[i]; L.ksw[i] = ps.lam_s * a.ksw[i]; }
    }
    for (int i = tid; i < P; i += kBlock) {
        uint64_t key = ~0ull;
        if (i < nF) {
            const uint32_t v = a.frontier[2 * (f0 + i)];
            const StageRec r = a.rec[v];
            StageL st;
            st.elig = r.elig;
            st.hash = r.hash;
            st.tokens = r.tokens;
            st.sigma = r.sigma;
            st.v = v;
            st.e0 = a.desc_off[v];
            st.e1 = a.desc_off[v + 1];
            st.dbeg = r.par_begin;
            st.dn = (uint16_t)a.done_n[v];
            st.c0 = a.cand_off[f0 + i];
            st.nc = a.cand_off[f0 + i + 1] - st.c0;
            st.npar = r.npar;
            st.model = r.model;
            st.shard = r.shard;
            st.pad0 = st.pad1 = 0;
            st.pfm = 0;
            L.stages[i] = st;
            key = ((uint64_t)(0xffffffffu - (st.e1 - st.e0)) << 32) | (uint32_t)i;
        }
        L.keys[i] = key;
    }
    // prefix-cache entries are fetched before the barrier and inserted after it
    constexpr int kPre = 4;
    uint64_t pre[kPre];
#pragma unroll
    for (int r = 0; r < kPre; ++r) {
        const int i = tid + r * kBlock;
        pre[r] = i < D * K ? a.pcache[(int64_t)b * D * K + i] : 0ull;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPre; ++r)
        if (pre[r] != 0) table_insert<Mask>(L, pre[r], (tid + r * kBlock) / K);
    for (int i = tid + kPre * kBlock; i < D * K; i += kBlock) {  // D*K > 1024 only
        const uint64_t h = a.pcache[(int64_t)b * D * K + i];
        if (h != 0) table_insert<Mask>(L, h, i / K);
    }
    if (tid < M) {
        uint64_t m = 0;
        for (int d = 0; d < D; ++d)
            if (bit(L.rho[d], tid)) m |= 1ull << d;
        L.rm[tid] = m;
    }
    if constexpr (SLOTS) {  // residency of d after loading m, from the LDS tables (the Load rule's chain of reads)
        uint32_t *rnew = reinterpret_cast<uint32_t *>(L.ksw);
        for (int i = tid; i < M * D; i += kBlock) {
            const int m = i / D, d = i - m * D;
            rnew[i] = (uint32_t)load_model(L.rho[d], m, L.cap[d], L.wt);
        }
    }
    // work order: stage i goes to position = number of keys smaller than its
    // own (keys are distinct), so the most descendants come first
    for (int i = tid; i < nF; i += kBlock) {
        const uint64_t ki = L.keys[i];
        int rank = 0;
        for (int j = 0; j < nF; ++j) rank += L.keys[j] < ki ? 1 : 0;
        L.order[rank] = (uint8_t)i;
    }
    __syncthreads();  // the sort keys' space becomes staging slots; the prefix table is built
    for (int i = tid; i < nF; i += kBlock) L.stages[i].pfm = (uint64_t)table_find<Mask>(L, L.stages[i].hash);
    if (kSplit && tid == kBlock - 1) {  // work items in rank order; heavy singletons-only stages in parts
        uint16_t *items = reinterpret_cast<uint16_t *>(sb + plan.items);
        uint8_t *parts = sb + plan.parts, *pbase = sb + plan.pbase;
        uint32_t *left = reinterpret_cast<uint32_t *>(sb + plan.left);
        uint32_t *plen = reinterpret_cast<uint32_t *>(sb + plan.plen);
        int ni = 0, used = 0;
        for (int pos = 0; pos < nF; ++pos) {
            const StageL &st = L.stages[L.order[pos]];
            const int ne = (int)(st.e1 - st.e0);
            int np = 1;
            uint32_t pl = (uint32_t)ne;
            if (st.nc == (uint32_t)D && ne > kSplitRows) {
                // as many parts of kSplitRows rows as the pool slots and the
                // work items left allow (every later stage keeps one item)
                np = min((ne + kSplitRows - 1) / kSplitRows, min(kSplitSlots - used, kSplitItems - ni - (nF - 1 - pos)));
                if (np >= 2) {  // rows per part: whole 64-row batches; ne > 128 keeps np >= 2
                    pl = (uint32_t)((((ne + np - 1) / np) + 63) & ~63);
                    np = (ne + (int)pl - 1) / (int)pl;
                } else {
                    np = 1;
                }
            }
            parts[pos] = (uint8_t)np;
            left[pos] = (uint32_t)np;
            pbase[pos] = (uint8_t)used;
            plen[pos] = pl;
            if (np > 1) used += np;
            for (int q = 0; q < np; ++q) items[ni++] = (uint16_t)(pos | (q << 8));
        }
        L.next[1] = (uint32_t)ni;
    }
    __syncthreads();

    constexpr int kGroups = kBlock / G;
    const int lane = tid & (G - 1);
    const bool live = lane < D;
    const int dl = live ? lane : D - 1;  // clamped device index for table reads
    const int gbase = (tid & 63) & ~(G - 1);
    const uint64_t gmask = (G >= 64) ? ~0ull : ((1ull << (G & 63)) - 1ull);
    const uint64_t rho = L.rho[dl];
    const Mask mybit = live ? (Mask(1) << lane) : Mask(0);
    const float *exec_col = L.exec + dl;
    const float *ksw_col = L.ksw + dl;
    Entry *area = reinterpret_cast<Entry *>(L.entries) + (tid & ~(G - 1));  // this group's G staging slots
    const float lam_tr = ps.lam_tr, lam_c = ps.lam_c, lam_p = ps.lam_p;
    // same-model weight: a resident model costs -lam_m where an absent one
    // costs its (weighted) switch time
    const float res_cost = VAR ? -ps.lam_m : 0.0f;
    const bool mean_levels = VAR && (ps.flags & FATE_MEAN_PER_LEVEL) != 0;
    const bool windows_on = !VAR || (ps.flags & FATE_NO_WINDOWS) == 0;

    // Waves claim chunks of consecutive work positions (one per group of the
    // wave) from a shared counter: the largest stages go first and a wave
    // that finishes early takes the next chunk (list scheduling).
    constexpr int kGpw = 64 / G;  // lane groups per wave
    const int gw = (tid & 63) / G;
    const int nchunks = kSplit ? (int)L.next[1] : (nF + kGpw - 1) / kGpw;
    for (;;) {
        uint32_t chunk = 0;
        if ((tid & 63) == 0) chunk = atomicAdd(L.next, 1u);
        chunk = __builtin_amdgcn_readfirstlane(chunk);
        if ((int)chunk >= nchunks) break;  // uniform within the wave
        int pos = (int)chunk * kGpw + gw, part = 0;
        if constexpr (kSplit) {  // one group per wave: the work item names the position and part
            const uint32_t item = reinterpret_cast<const uint16_t *>(sb + plan.items)[chunk];
            pos = (int)(item & 0xffu);
            part = (int)(item >> 8);
        }
        if (pos >= nF) continue;  // the last chunk may be partial
        const int si = (int)L.order[pos];
        const StageL sv = L.stages[si];
        const int mv = sv.model;
        const bool hv_cached = bit(sv.pfm, lane);

        // ---- immediate terms of v on device `lane` and the post-state there
        float tr = 0.0f, cnt = 0.0f;
        // slot layout: lane j holds completed parent j of v (the first 16 are
        // loaded here, before the first horizon batch is staged, so that the
        // two chains of loads overlap)
        uint32_t par_h = 0u;
        float par_s = 0.0f;
        if constexpr (kSlots) {
            if (lane < (int)sv.dn) {
                const DoneParent pu = a.done[sv.dbeg + lane];
                par_h = (uint32_t)pu.holders;  // at most 16 devices
                par_s = pu.sigma;
            }
        }
        // each parent in turn goes to the whole row, in parent order (the first
        // by a DPP row broadcast, the rest by shuffles); one round trip per 16
        // parents
        auto add_parents16 = [&](uint32_t h, float sg, int n) {
            for (int j = 0; j < n; ++j) {
                const uint32_t hj = j == 0 ? (uint32_t)row_bcast<0>((int)h) : (uint32_t)__shfl((int)h, j, 16);
                const float sj = j == 0 ? __int_as_float(row_bcast<0>(__float_as_int(sg))) : __shfl(sg, j, 16);
                const bool local = ((hj >> dl) & 1u) != 0;
                cnt += local ? 1.0f : 0.0f;
                tr += local ? 0.0f : sj * a.beta0;
            }
        };
        if constexpr (!kSlots) {  // (the slot layout adds its parents once its first batch is staged)
            for (int q = 0; q < sv.dn; ++q) {  // uniform trip count
                const DoneParent pu = a.done[sv.dbeg + q];
                add_parent<UNI>(a, pu.holders, pu.sigma, dl, tr, cnt);
            }
        }
        const bool feas_v = live && bit(sv.elig, lane) && bit(L.fits[mv], lane);
        const float c_v = kSlots ? reinterpret_cast<const CostS *>(L.exec)[mv * D + dl].exec : L.exec[mv * D + dl];
        const float sw_v = kSlots ? reinterpret_cast<const CostS *>(L.exec)[mv * D + dl].swo
                                  : (bit(rho, mv) ? res_cost : L.ksw[mv * D + dl]);
        const float pf_v = hv_cached ? ps.kpf * sv.tokens : 0.0f;
        // the immediate cost's two parts, once the parents' transfer and colocation are summed
        auto imm_terms = [&](float &a_out, float &b_out) {
            const float colo_v = sv.npar ? cnt * fast_rcp((float)sv.npar) : 0.0f;
            a_out = ps.lam_q * L.wait[dl] + sw_v - lam_c * colo_v;  // the switch table holds lam_s * kappa
            b_out = c_v + lam_tr * tr - lam_p * pf_v;
        };
        float a_imm = 0.0f, b_imm = 0.0f;
        if constexpr (!kSlots) imm_terms(a_imm, b_imm);
        const uint64_t rho_new = kSlots ? (uint64_t)reinterpret_cast<const uint32_t *>(L.ksw)[mv * D + dl]
                                        : load_model(rho, mv, L.cap[dl], L.wt);
        const bool prefix_added = sv.hash != 0 && !hv_cached;
        const uint64_t feas_mask = (__ballot(feas_v) >> gbase) & gmask;

        // ---- horizon descendants: shared staging and row evaluation
        const float t0 = lam_tr * sv.sigma * a.beta0;  // v's output to one more device (uniform beta)
        // Lane j stages entry base + j of v's descendant list into the group's
        // LDS slots; returns how many entries the batch holds (they form a prefix).
        auto stage_batch = [&](uint32_t base) -> int {
            const uint32_t e = base + lane;
            bool valid = e < sv.e1;
            uint32_t ent = 0;
            if (valid) {
                ent = a.desc[e];
                valid = (int)(ent >> kDescDepthShift) <= ps.H;
            }
            if (valid) {
                const uint32_t w = ent & kDescIdMask;
                const int depth = (int)(ent >> kDescDepthShift);
                const StageRec rw = a.rec[w];
                const uint32_t db = rw.par_begin;
                const uint32_t dn = a.done_n[w];
                Entry &E = area[lane];
                E.feas = (Mask)(rw.elig & L.fits[rw.model]);
                E.pfdevs = table_find<Mask>(L, rw.hash);
                E.gh = mean_levels ? L.gpow[depth] * a.desc_w[e] : L.gpow[depth];
                const float cw = lam_c * fast_rcp((float)rw.npar);  // a descendant has at least one parent
                E.cw = cw;
                E.pfp = lam_p * ps.kpf * rw.tokens;
                E.moff = (uint32_t)rw.model * (uint32_t)D;
                E.model = rw.model;
                E.flags = (uint8_t)(((VAR ? child_of(a, rw, depth, sv.v) : depth == 1) ? 1 : 0) | (rw.hash != 0 && rw.hash == sv.hash ? 2 : 0));
                E.dn = (uint16_t)dn;
                E.dbeg = db;
                float base_tr = 0.0f;
                for (uint32_t q = 0; q < dn; ++q) {
                    const DoneParent pu = a.done[db + q];
                    const float t = lam_tr * a.beta0 * pu.sigma;
                    if (UNI) base_tr += t;
                    if (q < (uint32_t)kCap) {
                        E.ph[q] = (Mask)pu.holders;
                        E.pw[q] = UNI ? t + cw : pu.sigma;
                    }
                }
                E.base_tr = base_tr;
            }
            const int nb = __popcll((__ballot(valid) >> gbase) & gmask);
            wave_sync();
            return nb;
        };
        // Row of descendant E: B(d') = c_hat(w, d' | s) and its value once v
        // sits on d' (both +inf where w is infeasible).
        auto entry_row = [&](const Entry &E, float &Bd_out, float &inval_out, float &gh_out, bool &child_out) {
            const Mask feas = (Mask)E.feas, pfd = (Mask)E.pfdevs;
            const float gh = E.gh, pfp = E.pfp, cw = E.cw;
            const int mw = E.model, dn = E.dn, flags = E.flags;
            const bool child = (flags & 1) != 0;
            float X = exec_col[E.moff] + E.base_tr;
            const int ns = dn < kCap ? dn : kCap;
            if (UNI) {
                for (int q = 0; q < ns; ++q)  // uniform trip count
                    X -= ((Mask)E.ph[q] & mybit) != 0 ? E.pw[q] : 0.0f;
                for (int q = kCap; q < dn; ++q) {  // rare: more completed parents than staged
                    const DoneParent pu = a.done[E.dbeg + q];
                    X -= ((Mask)pu.holders & mybit) != 0 ? lam_tr * a.beta0 * pu.sigma + cw : 0.0f;
                }
            } else {
                float trw = 0.0f, cntw = 0.0f;
                for (int q = 0; q < ns; ++q) add_parent<false>(a, E.ph[q], E.pw[q], dl, trw, cntw);
                for (int q = kCap; q < dn; ++q) {
                    const DoneParent pu = a.done[E.dbeg + q];
                    add_parent<false>(a, pu.holders, pu.sigma, dl, trw, cntw);
                }
                X += lam_tr * trw - cntw * cw;
            }
            const float sw = ksw_col[E.moff];
            const bool in_old = ((rho >> mw) & 1ull) != 0;
            const bool in_new = ((rho_new >> mw) & 1ull) != 0;
            const bool pf_old = (pfd & mybit) != 0;
            const bool pf_new = pf_old || ((flags & 2) && prefix_added);
            const float Braw = X + (in_old ? res_cost : sw) - (pf_old ? pfp : 0.0f);
            const float Bnew = X + (in_new ? res_cost : sw) - (pf_new ? pfp : 0.0f) - (child ? cw : 0.0f);
            const bool fw = (feas & mybit) != 0;
            const float Bd = fw ? Braw : inf_f();
            const float inval = fw ? Bnew : inf_f();
            Bd_out = Bd;
            inval_out = inval;
            gh_out = gh;
            child_out = child;
        };

        if constexpr (kSlots) {
          {
            // ---- horizon rows, G at a time: lane j stages row j (EntryS)
            EntryS *areaS = reinterpret_cast<EntryS *>(static_cast<uint8_t *>(L.entries) + (tid / G) * kSlotGroupBytes);
            const uint32_t rho32 = (uint32_t)rho, rhon32 = (uint32_t)rho_new;
            const uint32_t chg32 = rho32 ^ rhon32, ld32 = rhon32 & ~rho32;  // models whose residency v's placement flips / loads
            const uint32_t bit_lo = (uint32_t)mybit, dlane = (uint32_t)lane;
            const CostS *tab_col = reinterpret_cast<const CostS *>(L.exec) + dl;
            // x where bit `pos` of m is set, else +0
            auto bit_sel = [](uint32_t m, uint32_t pos, float x) {
                return __uint_as_float(__float_as_uint(x) & (uint32_t)__builtin_amdgcn_sbfe((int)m, pos, 1u));
            };
            auto stage_rows = [&](uint32_t base) -> int {
                const uint32_t e = base + lane;
                bool valid = e < sv.e1;
                uint32_t ent = 0;
                if (valid) {
                    ent = a.desc[e];
                    valid = (int)(ent >> kDescDepthShift) <= ps.H;
                }
                if (valid) {
                    const uint32_t w = ent & kDescIdMask;
                    const int depth = (int)(ent >> kDescDepthShift);
                    const StageRec rw = a.rec[w];
                    const uint32_t db = rw.par_begin;
                    const uint32_t dn = a.done_n[w];
                    const uint32_t feas = (uint32_t)(rw.elig & L.fits[rw.model]);
                    const uint32_t pfo = table_find<uint32_t>(L, rw.hash);
                    const bool same = rw.hash != 0 && rw.hash == sv.hash;
                    const float cw = lam_c * fast_rcp((float)rw.npar);  // a descendant has at least one parent
                    float base_tr = 0.0f;
                    uint32_t ph[kCap] = {0u, 0u, 0u};
                    float pw[kCap] = {0.0f, 0.0f, 0.0f};
                    if (dn > 0) {  // the staged parents' loads are issued together
                        DoneParent pu[kCap];
#pragma unroll
                        for (int q = 0; q < kCap; ++q)
                            if ((uint32_t)q < dn) pu[q] = a.done[db + q];
#pragma unroll
                        for (int q = 0; q < kCap; ++q) {
                            if ((uint32_t)q < dn) {
                                const float t = lam_tr * a.beta0 * pu[q].sigma;
                                base_tr += t;
                                ph[q] = (uint32_t)pu[q].holders;
                                pw[q] = t + cw;
                            }
                        }
                        for (uint32_t q0 = kCap; q0 < dn; q0 += kMore) {  // rare: more completed parents than staged
                            float sg[kMore];  // loads issued together, added in parent order
#pragma unroll
                            for (int i = 0; i < kMore; ++i) sg[i] = q0 + i < dn ? a.done[db + q0 + i].sigma : 0.0f;
#pragma unroll
                            for (int i = 0; i < kMore; ++i)
                                if (q0 + i < dn) base_tr += lam_tr * a.beta0 * sg[i];
                        }
                    }
                    EntryS S;
                    const bool child = VAR ? child_of(a, rw, depth, sv.v) : depth == 1;
                    S.moff = (uint32_t)rw.model * (uint32_t)D;
                    S.m1 = feas | (pfo << 16);
                    // once v runs on a device, that device also caches grp(v)
                    S.m2 = (same ? (~pfo & 0xffffu) : 0u) | (ph[2] << 16);
                    S.mdn = (uint32_t)rw.model | (dn << 8);
                    S.gh = mean_levels ? L.gpow[depth] * a.desc_w[e] : L.gpow[depth];
                    S.xk = base_tr + (child ? t0 : 0.0f);
                    S.xn = base_tr + (child ? -cw : 0.0f);
                    S.pfp = lam_p * ps.kpf * rw.tokens;
                    S.dbeg = db;
                    S.ph01 = ph[0] | (ph[1] << 16);
                    S.pw0 = pw[0];
                    S.pw1 = pw[1];
                    S.pw2 = pw[2];
                    S.cw = cw;
                    areaS[lane] = S;
                }
                const int nb = __popcll((__ballot(valid) >> gbase) & gmask);
                wave_sync();
                return nb;
            };

            // the first batch is staged while v's parent loads are in flight
            int nb_first = 0;
            if (sv.e0 < sv.e1) nb_first = stage_rows(sv.e0);
            for (int q0 = 0; q0 < (int)sv.dn; q0 += 16) {  // uniform within the group
                uint32_t h = par_h;
                float sg = par_s;
                if (q0 > 0) {  // rare: more than 16 completed parents
                    h = 0u;
                    sg = 0.0f;
                    if (q0 + lane < (int)sv.dn) {
                        const DoneParent pu = a.done[sv.dbeg + q0 + lane];
                        h = (uint32_t)pu.holders;
                        sg = pu.sigma;
                    }
                }
                add_parents16(h, sg, min(16, (int)sv.dn - q0));
            }
            imm_terms(a_imm, b_imm);

            // ---- candidates: the single {lane} on its own lane; the window of
            // size k = s + 2 starting at device i on lane i of slot s (windows
            // are ordered by size, then start: slot s writes one contiguous run)
            const uint32_t c0 = sv.c0;
            int nk = 0;  // window sizes present: 2 .. nk + 1
            for (int rem = (int)sv.nc - D; rem > 0; rem -= D - nk) ++nk;
            const float j0_single = a_imm + b_imm;
            const uint32_t fm = (uint32_t)feas_mask;
            float w_j0[3] = {0.0f, 0.0f, 0.0f};
            bool w_ok[3] = {false, false, false};
            if (__ballot(nk != 0) != 0ull) {  // uniform over the wave: some stage of it has windows
#pragma unroll
                for (int s = 0; s < 3; ++s) {
                    const int k = s + 2;
                    const float y = a_imm + b_imm * (1.0f / (float)k);  // k is a constant here
                    // maximum over devices i..i+k-1 (a lane whose source is past the row holds no window)
                    float m = fmaxf(y, dpp_b0<0x101>(y));
                    if (k >= 3) m = fmaxf(m, dpp_b0<0x102>(y));
                    if (k >= 4) m = fmaxf(m, dpp_b0<0x103>(y));
                    const uint32_t wm = (1u << k) - 1u;
                    w_ok[s] = windows_on && s < nk && lane <= D - k && ((fm >> lane) & wm) == wm;
                    // gather with uniform beta: each of the k-1 other devices sends sigma/k
                    w_j0[s] = m + lam_tr * ((float)(k - 1) * a.beta0 * sv.sigma * (1.0f / (float)k));
                }
            }


            // ---- horizon rows.  Outside S the row is scanned as order-reversing
            // integer keys (prefix and suffix minima, one DPP op per step); the
            // minimum outside a window {i..i+k-1} is min(prefix(i-1), suffix(i+k)).
            // Inside S the window minimum of the post-state values slides by one
            // lane per size.  A batch's terms are summed in fp32, batches in fp64.
            double acc0 = 0.0, w_acc[3] = {0.0, 0.0, 0.0};
            for (uint32_t base = sv.e0; base < sv.e1; base += G) {  // uniform
                const int nb = base == sv.e0 ? nb_first : stage_rows(base);
                float f0 = 0.0f, f1 = 0.0f, f2 = 0.0f, f3 = 0.0f;
                // staged row jj: the key outside S, the value inside S, and gamma^depth.
                // Branch-free: a bit of a device mask selects a value by masking its bits.
                auto row = [&](int jj, uint32_t &key, float &inval, float &gh) {
                    const EntryS *E = areaS + jj;
                    const uint4 q0 = *reinterpret_cast<const uint4 *>(E);
                    const float4 q1 = *reinterpret_cast<const float4 *>(&E->gh);
                    // q0: moff, m1, m2, mdn; q1: gh, xk, xn, pfp
                    const float2 t = *reinterpret_cast<const float2 *>(&tab_col[q0.x]);  // cost with the old switch term, switch magnitude
                    float X = t.x;  // every completed parent remote (its transfer is in xk / xn)
                    if (q0.w > 255u) {  // completed parents: holding one's output saves its transfer and adds colocation
                        const uint4 q2 = *reinterpret_cast<const uint4 *>(&E->dbeg);
                        const float4 q3 = *reinterpret_cast<const float4 *>(&E->pw2);
                        X -= bit_sel(q2.y, dlane, __uint_as_float(q2.z));
                        X -= bit_sel(q2.y, dlane + 16u, __uint_as_float(q2.w));
                        X -= bit_sel(q0.z, dlane + 16u, q3.x);
                        const uint32_t dn = q0.w >> 8;
                        for (uint32_t p0 = kCap; p0 < dn; p0 += kMore) {  // rare: more completed parents than staged
                            uint32_t hq[kMore];  // loads issued together, subtracted in parent order
                            float sq[kMore];
#pragma unroll
                            for (int i = 0; i < kMore; ++i) {
                                hq[i] = 0u;
                                sq[i] = 0.0f;
                                if (p0 + i < dn) {
                                    hq[i] = (uint32_t)a.done[q2.x + p0 + i].holders;
                                    sq[i] = a.done[q2.x + p0 + i].sigma;
                                }
                            }
#pragma unroll
                            for (int i = 0; i < kMore; ++i)
                                if (p0 + i < dn) X -= (hq[i] & bit_lo) ? lam_tr * a.beta0 * sq[i] + q3.y : 0.0f;
                        }
                    }
                    X -= bit_sel(q0.y, dlane + 16u, q1.w);  // grp(w) already cached on this device
                    // v's placement flips m(w)'s residency here: loaded (switch term drops by the
                    // magnitude) or evicted (rises by it); the sign bit comes from the load bit
                    const uint32_t mw = q0.w;  // the bit-field offset uses bits 4:0, m(w)
                    const float dsw = __uint_as_float((__builtin_amdgcn_ubfe(ld32, mw, 1u) << 31) +
                                                      (__float_as_uint(t.y) & (uint32_t)__builtin_amdgcn_sbfe((int)chg32, mw, 1u)));
                    const float Bnew = X + q1.z + dsw - bit_sel(q0.z, dlane, q1.w);
                    const uint32_t fm = (uint32_t)__builtin_amdgcn_sbfe((int)q0.y, dlane, 1u);  // w feasible here
                    // outside S: a child also receives v's output here (in xk)
                    key = (fm & fkey(X + q1.y)) | (~fm & kKeyInf);
                    inval = __uint_as_float((fm & __float_as_uint(Bnew)) | (~fm & __float_as_uint(inf_f())));
                    gh = q1.x;
                };
                // one row's terms: outside S from the prefix / suffix scans, inside S
                // from the window minimum, each weighted by gamma^depth
                auto accumulate = [&](uint32_t Pl, uint32_t Q, float inval, float gh) {
                    f0 += gh * fminf(unkey(kmax_from<0x101>(Pl, Q)), inval);
                    if (nk >= 1) {  // uniform
                        float inside = fminf(inval, dpp_b0<0x101>(inval));
                        f1 += gh * fminf(unkey(kmax_from<0x102>(Pl, Q)), inside);
                        if (nk >= 2) {
                            inside = fminf(inside, dpp_b0<0x101>(inside));
                            f2 += gh * fminf(unkey(kmax_from<0x103>(Pl, Q)), inside);
                            if (nk >= 3) {
                                inside = fminf(inside, dpp_b0<0x101>(inside));
                                f3 += gh * fminf(unkey(kmax_from<0x104>(Pl, Q)), inside);
                            }
                        }
                    }
                };
                int jj = 0;
                // the wave's lane groups score different stages: the loop without
                // window terms only when none of them has windows, so that the
                // wave never runs both loops
                if (__ballot(nk != 0) == 0ull) {
                    for (; jj + 1 < nb; jj += 2) {  // two rows at a time, so their scans interleave
                        uint32_t k0, k1;
                        float v0, v1, g0, g1;
                        row(jj, k0, v0, g0);
                        row(jj + 1, k1, v1, g1);
                        const uint32_t P0 = kscan_up16(k0), P1 = kscan_up16(k1);
                        const uint32_t Q0 = kscan_down16(k0), Q1 = kscan_down16(k1);
                        const uint32_t L0 = kshift_in<0x111>(P0), L1 = kshift_in<0x111>(P1);  // prefix up to lane-1
                        f0 += g0 * fminf(unkey(kmax_from<0x101>(L0, Q0)), v0);
                        f0 += g1 * fminf(unkey(kmax_from<0x101>(L1, Q1)), v1);
                    }
                } else {
                    for (; jj + 1 < nb; jj += 2) {
                        uint32_t k0, k1;
                        float v0, v1, g0, g1;
                        row(jj, k0, v0, g0);
                        row(jj + 1, k1, v1, g1);
                        const uint32_t P0 = kscan_up16(k0), P1 = kscan_up16(k1);
                        const uint32_t Q0 = kscan_down16(k0), Q1 = kscan_down16(k1);
                        const uint32_t L0 = kshift_in<0x111>(P0), L1 = kshift_in<0x111>(P1);
                        accumulate(L0, Q0, v0, g0);
                        accumulate(L1, Q1, v1, g1);
                    }
                }
                if (jj < nb) {  // uniform: the odd row
                    uint32_t key;
                    float inval, gh;
                    row(jj, key, inval, gh);
                    const uint32_t P = kscan_up16(key), Q = kscan_down16(key);
                    accumulate(kshift_in<0x111>(P), Q, inval, gh);
                }
                acc0 += (double)f0;
                w_acc[0] += (double)f1;
                w_acc[1] += (double)f2;
                w_acc[2] += (double)f3;
                wave_sync();  // the next batch overwrites the staging slots
                if (nb < G) break;  // past the horizon depth or the list end
            }

            // ---- emit scores
            const float psi0 = feas_v ? (float)(-((double)j0_single + acc0)) : -inf_f();
            if (live) scores[c0 + lane] = psi0;
            uint32_t off = c0 + (uint32_t)D;
            float psiw[3] = {-inf_f(), -inf_f(), -inf_f()};
#pragma unroll
            for (int s = 0; s < 3; ++s) {
                if (s >= nk) break;  // uniform
                const int k = s + 2;
                psiw[s] = w_ok[s] ? (float)(-((double)w_j0[s] + w_acc[s])) : -inf_f();
                if (lane <= D - k) scores[off + lane] = psiw[s];
                off += (uint32_t)(D - k + 1);
            }
            // ---- fused top-k: the group ranks the scores it holds (the same
            // float values it stored), candidate index = offset within the stage
            if (a.topk > 0) {  // uniform over the launch
                const int64_t f = (int64_t)f0 + si;
                int32_t *ti = a.tk_idx + f * a.topk;
                float *tv = a.tk_val + f * a.topk;
                // the stage's record slot in LDS is dead once its group holds it
                // in registers: it takes the stage's score bits (one word per
                // device, 0 for none), ranked after the loop one lane per stage;
                // a stage ranked here marks the slot instead
                uint32_t *ranked = reinterpret_cast<uint32_t *>(L.stages + si);
                if (a.topk <= kLaneTopk && __ballot(nk != 0) == 0ull) {  // uniform over the wave
                    ranked[lane] = live ? topk_bits(psi0) : 0u;
                    continue;
                }
                if (lane == 0) ranked[0] = kRankedInLoop;
                if (__ballot(nk != 0) == 0ull) {  // uniform over the wave: singletons only
                    uint32_t sb[1] = {live ? topk_bits(psi0) : 0u};
                    const uint32_t ci[1] = {(uint32_t)lane};
                    group_topk_at<G, 1>(sb, ci, lane, a.topk, ti, tv);
                } else {
                    uint32_t sb[4], ci[4];
                    sb[0] = live ? topk_bits(psi0) : 0u;
                    ci[0] = (uint32_t)lane;
                    uint32_t base_c = (uint32_t)D;
#pragma unroll
                    for (int s = 0; s < 3; ++s) {
                        const int k = s + 2;
                        const bool has = s < nk && lane <= D - k;
                        sb[s + 1] = has ? topk_bits(psiw[s]) : 0u;
                        ci[s + 1] = has ? base_c + (uint32_t)lane : 0xfffffff0u + (uint32_t)s;  // distinct, never picked
                        base_c += s < nk ? (uint32_t)(D - k + 1) : 0u;
                    }
                    group_topk_at<G, 4>(sb, ci, lane, a.topk, ti, tv);
                }
            }
            continue;
          }
        }
        // ---- candidates: slot 0 = single device `lane`; slots 1..3 = windows
        const uint32_t c0 = sv.c0;
        const int nwin = (int)sv.nc - D;
        const int wslots = (nwin + G - 1) / G;
        const float j0_single = a_imm + b_imm;
        double acc0 = 0.0;
        int w_i[3], w_k[3];
        float w_j0[3];
        bool w_ok[3];
        double w_acc[3];
#pragma unroll
        for (int s = 0; s < 3; ++s) {
            w_i[s] = 0; w_k[s] = 2; w_j0[s] = 0.0f; w_ok[s] = false; w_acc[s] = 0.0;
            if (s >= wslots) continue;  // uniform
            const int t = lane + s * G;
            int i = 0, k = 2;
            if (t < nwin) decode_window(t, D, i, k);
            const float rk = fast_rcp((float)k);
            float tmax = -inf_f();
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int src = min(i + q, G - 1);
                const float aq = __shfl(a_imm, src, G);
                const float bq = __shfl(b_imm, src, G);
                if (q < k) tmax = fmaxf(tmax, aq + bq * rk);
            }
            const uint64_t wm = ((1ull << k) - 1ull) << i;
            const bool feasible = windows_on && (t < nwin) && ((feas_mask & wm) == wm);
            float gat = inf_f();
            if (feasible) {
                for (int p = i; p < i + k; ++p) {
                    float sum = 0.0f;
                    for (int d = i; d < i + k; ++d)
                        if (d != p) sum += a.beta[d * D + p] * sv.sigma * rk;
                    gat = fminf(gat, sum);
                }
            }
            w_i[s] = i;
            w_k[s] = k;
            w_ok[s] = feasible;
            w_j0[s] = tmax + lam_tr * gat;
        }

        // ---- horizon descendants, G at a time (a part of a heavy stage: its rows)
        const int nparts = kSplit ? (int)(sb + plan.parts)[pos] : 1;
        const uint32_t plen = kSplit && nparts > 1 ? reinterpret_cast<const uint32_t *>(sb + plan.plen)[pos] : 0u;
        const uint32_t b_lo = sv.e0 + (uint32_t)part * plen;
        const uint32_t b_hi = nparts > 1 ? min(sv.e1, b_lo + plen) : sv.e1;
        for (uint32_t base = b_lo; base < b_hi; base += G) {  // uniform; a part is whole G-row batches
            const int nb = stage_batch(base);
            int jj = 0;
            if (UNI && wslots == 0) {  // singletons only: two descendants per iteration
                for (; jj + 1 < nb; jj += 2) {
                    float B0, N0, g0, B1, N1, g1;
                    bool c0c, c1c;
                    entry_row(area[jj], B0, N0, g0, c0c);
                    entry_row(area[jj + 1], B1, N1, g1, c1c);
                    float o0, o1;  // minimum over the other devices
                    if constexpr (G >= 32) {
                        o0 = others_min_wide<G>(B0, tid & 63);
                        o1 = others_min_wide<G>(B1, tid & 63);
                    } else {
                        float p0 = B0, q0 = B0, p1 = B1, q1 = B1;
                        scan_min_pair<G>(p0, q0, p1, q1, lane);
                        o0 = fminf(from_left<G>(p0, lane), from_right<G>(q0, lane));
                        o1 = fminf(from_left<G>(p1, lane), from_right<G>(q1, lane));
                    }
                    const float e0 = o0 + (c0c ? t0 : 0.0f);
                    const float e1 = o1 + (c1c ? t0 : 0.0f);
                    acc0 += (double)(g0 * fminf(e0, N0));
                    acc0 += (double)(g1 * fminf(e1, N1));
                }
            }
            for (; jj < nb; ++jj) {  // uniform
                float Bd, inval, gh;
                bool child;
                entry_row(area[jj], Bd, inval, gh, child);
                const float Pm = scan_min_up<G>(Bd, lane);
                const float Qm = scan_min_down<G>(Bd, lane);
                {  // single device `lane`
                    float excl = fminf(from_left<G>(Pm, lane), from_right<G>(Qm, lane));
                    if (UNI) {
                        excl += child ? t0 : 0.0f;
                    } else if (child) {
                        {
                            excl = inf_f();
                            for (int dd = 0; dd < D; ++dd) {  // uniform trip count
                                const float bdd = __shfl(Bd, dd, G);
                                if (dd != lane)
                                    excl = fminf(excl, bdd + lam_tr * sv.sigma * a.beta[dl * D + dd]);
                            }
                        }
                    }
                    acc0 += (double)(gh * fminf(excl, inval));
                }
#pragma unroll
                for (int s = 0; s < 3; ++s) {  // windows
                    if (s >= wslots) continue;  // uniform
                    const int i = w_i[s], k = w_k[s];
                    const float left = __shfl(Pm, max(i - 1, 0), G);
                    const float right = __shfl(Qm, min(i + k, G - 1), G);
                    float excl = fminf(i > 0 ? left : inf_f(), i + k < G ? right : inf_f());
                    if (child) {
                        if (UNI) {
                            excl += t0;
                        } else {
                            excl = inf_f();
                            for (int dd = 0; dd < D; ++dd) {  // uniform trip count
                                const float bdd = __shfl(Bd, dd, G);
                                if (dd >= i && dd < i + k) continue;
                                float bmin = inf_f();
                                for (int q = 0; q < k; ++q) bmin = fminf(bmin, a.beta[(i + q) * D + dd]);
                                excl = fminf(excl, bdd + lam_tr * sv.sigma * bmin);
                            }
                        }
                    }
                    float inside = inf_f();
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float x = __shfl(inval, min(i + q, G - 1), G);
                        if (q < k) inside = fminf(inside, x);
                    }
                    w_acc[s] += (double)(gh * fminf(excl, inside));
                }
            }
            wave_sync();  // the next batch overwrites the staging slots
            if (nb < G) break;  // past the horizon depth or the list end
        }
        if (kSplit && nparts > 1) {  // uniform: the part's sum to its slot; the last part's wave emits
            double *pool = reinterpret_cast<double *>(sb + plan.pool);
            const int slot0 = (int)(sb + plan.pbase)[pos];
            pool[(slot0 + part) * 64 + lane] = acc0;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            uint32_t before = 0;
            if (lane == 0) before = atomicSub(reinterpret_cast<uint32_t *>(sb + plan.left) + pos, 1u);
            before = __builtin_amdgcn_readfirstlane(before);
            if (before != 1u) continue;  // another part is still being scored
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
            acc0 = 0.0;
            for (int q = 0; q < nparts; ++q) acc0 += pool[(slot0 + q) * 64 + lane];
        }

        // ---- emit scores
        const float psi0 = feas_v ? (float)(-((double)j0_single + acc0)) : -inf_f();
        if (live) scores[c0 + lane] = psi0;
#pragma unroll
        for (int s = 0; s < 3; ++s) {
            if (s >= wslots) continue;  // uniform
            const int t = lane + s * G;
            if (t < nwin) scores[c0 + D + t] = w_ok[s] ? (float)(-((double)w_j0[s] + w_acc[s])) : -inf_f();
        }
    }

    // ---- slot layout: the singletons-only stages' top-k, one lane per stage,
    // from the score bits their groups left in the stages' LDS slots
    if (kSlots && a.topk > 0 && a.topk <= kLaneTopk) {  // uniform over the block
        __syncthreads();  // every stage of the slice is scored
        for (int i = tid; i < nF; i += kBlock) {
            const uint4 *slot = reinterpret_cast<const uint4 *>(L.stages + i);
            uint32_t x[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint4 v = slot[q];
                x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
            }
            if (x[0] == kRankedInLoop) continue;
            const int64_t f = (int64_t)f0 + i;
            lane_topk16(x, a.topk, a.tk_idx + f * a.topk, a.tk_val + f * a.topk);
        }
    }

    // ---- fused top-k: after the block's scoring, each group ranks a fixed
    // share of its stages, re-reading the scores just written (outside the
    // scoring loop, so it adds no register pressure there)
    if (a.topk > 0 && !kSlots) {  // uniform over the block; the slot layout ranks in its loop
        __syncthreads();  // stages were scored by whichever wave claimed them
        constexpr int kRounds = 8;  // a slice holds at most eight rounds of groups
        uint32_t c0[kRounds];
        int C[kRounds];
        int64_t f[kRounds];
#pragma unroll
        for (int r = 0; r < kRounds; ++r) {
            const int pos = tid / G + r * kGroups;
            c0[r] = 0; C[r] = 0; f[r] = -1;
            if (pos < nF) {
                const int si = (int)L.order[pos];
                c0[r] = L.stages[si].c0;
                C[r] = (int)L.stages[si].nc;
                f[r] = (int64_t)f0 + si;
            }
        }
        rank_stages<G, kRounds>(scores, c0, C, f, lane, a.topk, a.tk_idx, a.tk_val);
    }
}

constexpr int kTopkRounds = 4;  // stages per lane group in k_topk

template <int G>
__global__ __launch_bounds__(kBlock) void k_topk(TopkLaunch a) {
    constexpr int kGroups = kBlock / G;
    const int tid = threadIdx.x;
    const int lane = tid & (G - 1);
    const int64_t nF = a.dcounts ? (int64_t)a.dcounts[0] : a.nF;  // planning state: current frontier
    const int64_t so = (int64_t)blockIdx.y * a.score_stride, oo = (int64_t)blockIdx.y * a.out_stride;
    // tiles of kTopkRounds * kGroups stages, grid-strided: a planning state's
    // grid covers its frontier capacity, mostly beyond the current frontier
    for (int64_t tile = blockIdx.x; tile * (kTopkRounds * kGroups) < nF; tile += gridDim.x) {  // uniform
        uint32_t c0[kTopkRounds];
        int C[kTopkRounds];
        int64_t f[kTopkRounds];
#pragma unroll
        for (int r = 0; r < kTopkRounds; ++r) {  // round r: the block's groups take consecutive stages
            const int64_t fr = (tile * kTopkRounds + r) * kGroups + tid / G;
            c0[r] = 0; C[r] = 0; f[r] = -1;
            if (fr < nF) {
                c0[r] = a.cand_off[fr];
                C[r] = (int)(a.cand_off[fr + 1] - c0[r]);
                f[r] = fr;
            }
        }
        rank_stages<G, kTopkRounds>(a.scores + so, c0, C, f, lane, a.k, a.idx + oo, a.val + oo);
    }
}

// ---- k_rows: one horizon row per lane ---------------------------------------
// For frontiers whose stages have single-device candidates only, with a
// uniform off-diagonal beta, D <= 16 and no scoring variant.  One workgroup
// per instance: it stages the instance's tables in LDS once (prefix-group
// table, per-(model, device) cost terms, and, per pair of models, the devices
// where loading the first flips the residency of the second), then takes the
// instance's frontier in chunks of kRowsChunk stages:
//   rows     the chunk's (frontier stage v, horizon row w) pairs are cut into
//            tasks of at most L consecutive rows of one stage, one task per
//            lane.  For each row the lane walks the devices d' in registers:
//            B(d') = c_hat(w, d' | s) (+infinity where w is infeasible), and,
//            for candidate d, the value C(d) once v sits on d (m(v) loaded,
//            grp(v) cached, v's output local).  The minimum of B over the
//            devices other than d is the second smallest B where B(d) is the
//            smallest and the smallest elsewhere (with a tie both are
//            equal), so the lane keeps the two smallest and adds
//            gamma^depth * min(that minimum (+ v's output transfer for a
//            child of v), C(d)) to its partial sum for candidate d.
//   combine  a group of lanes per stage (lane d = device d) computes the
//            immediate cost J0(v, d), adds the stage's task sums in task
//            order (fp64) and writes the scores.
//   top-k    one lane per stage ranks the scores left in LDS (k <= 4), or the
//            group ranks them in the combine step.
// Completed parents of a row lower B on the devices holding their outputs;
// a lane applies them in an LDS copy of its row (the devices are dynamic).
struct alignas(16) StageR {
    uint64_t elig, hash;
    float tokens, sigma;
    uint32_t e0, n;      // first descendant entry; rows within the horizon
    uint32_t c0, dbeg;   // first score; first completed parent
    uint32_t q0, nq;     // first full-length task and their number; the tail task (or 0xffffffff)
    uint16_t dn, npar;
    uint8_t model, pad0;
    uint16_t h0;         // devices holding the first completed parent's output (D <= 16)
    float s0;            // its output size
    uint32_t pfm;        // devices caching grp(v)
};
static_assert(sizeof(StageR) == 64, "StageR");

constexpr int kRowsChunk = 128;  // frontier stages per chunk of an instance

// floats per model row of the rows' cost table: (exec + switch term, switch
// magnitude) per device, plus four (rows of different models start on
// different LDS banks)
__host__ __device__ constexpr int rows_stride(int nd) { return 2 * nd + 4; }

struct RowsPlan {
    uint32_t pkey, pmask, rho, cap, wt, fits, wait, gpow, cst, rtab, fl, stages, tasks, part, misc, total;
    uint32_t ntask;  // task capacity
};

// The task sums are stored as float4 columns: column j of task t at
// part4[j * (ntask + 1) + t], so that lanes of consecutive tasks store to
// consecutive 16-byte slots, and the group reading a task's columns reads
// different banks.
__host__ __device__ inline RowsPlan rows_plan(int D, int K, int M, int nd, int blk) {
    RowsPlan q;
    const uint32_t T = 1u << table_log2(D, K);
    q.ntask = (uint32_t)(kRowsChunk > blk ? kRowsChunk : blk);
    uint32_t o = 0;
    q.pkey = o; o += 8 * T;
    q.pmask = o; o += 4 * T;
    o = (o + 7u) & ~7u;
    q.rho = o; o += 8 * (uint32_t)D;
    q.cap = o; o += 8 * (uint32_t)D;
    q.wt = o; o += 8 * (uint32_t)M;
    q.fits = o; o += 8 * (uint32_t)M;
    q.wait = o; o += 4 * (uint32_t)D;
    q.gpow = o; o += 4 * 16;
    o = (o + 15u) & ~15u;
    q.cst = o; o += (uint32_t)sizeof(CostS) * (uint32_t)(M * D);
    q.rtab = o; o += 4 * (uint32_t)(M * rows_stride(nd));
    q.fl = o; o += 4 * (uint32_t)(M * M);
    o = (o + 15u) & ~15u;
    q.stages = o; o += (uint32_t)sizeof(StageR) * (uint32_t)kRowsChunk;
    q.tasks = o; o += 4 * q.ntask;
    o = (o + 15u) & ~15u;
    q.part = o; o += 16 * (uint32_t)(nd / 4) * (q.ntask + 1);
    q.misc = o; o += 4 * 16;
    q.total = (o + 15u) & ~15u;
    return q;
}

// Four waves per SIMD (at most 128 VGPRs): four rows' loads in flight per lane
// need 129 without the bound, which would leave three.
template <int ND, int BLK>
__global__ __launch_bounds__(BLK) __attribute__((amdgpu_waves_per_eu(4))) void k_rows(ScoreLaunch a) {
    static_assert(BLK >= kRowsChunk && BLK % 64 == 0, "one thread per stage of a chunk");
    const int b = (int)a.order[blockIdx.x];  // largest frontiers first: the last workgroups to start are short
    const ParamSet ps = a.ps[blockIdx.y];
    float *const scores = a.scores + (int64_t)a.set_of[blockIdx.y] * a.score_stride;
    extern __shared__ uint64_t smem[];
    uint8_t *sb = reinterpret_cast<uint8_t *>(smem);
    const int tid = threadIdx.x;
    const int D = a.D, K = a.K, M = a.M;
    const RowsPlan plan = rows_plan(D, K, M, ND, BLK);
    constexpr int CS = rows_stride(ND), NJ = ND / 4;
    Lds L;
    L.logT = table_log2(D, K);
    L.pkey = reinterpret_cast<uint64_t *>(sb + plan.pkey);
    L.pmask = sb + plan.pmask;
    uint32_t *pmask = reinterpret_cast<uint32_t *>(sb + plan.pmask);
    uint64_t *rho = reinterpret_cast<uint64_t *>(sb + plan.rho);
    uint64_t *capd = reinterpret_cast<uint64_t *>(sb + plan.cap);
    uint64_t *wt = reinterpret_cast<uint64_t *>(sb + plan.wt);
    uint64_t *fits = reinterpret_cast<uint64_t *>(sb + plan.fits);
    float *wait = reinterpret_cast<float *>(sb + plan.wait);
    float *gpow = reinterpret_cast<float *>(sb + plan.gpow);
    CostS *cst = reinterpret_cast<CostS *>(sb + plan.cst);
    float *rtab = reinterpret_cast<float *>(sb + plan.rtab);
    uint32_t *fl = reinterpret_cast<uint32_t *>(sb + plan.fl);
    StageR *stg = reinterpret_cast<StageR *>(sb + plan.stages);
    uint32_t *tasks = reinterpret_cast<uint32_t *>(sb + plan.tasks);
    float4 *part4 = reinterpret_cast<float4 *>(sb + plan.part);
    float *partf = reinterpret_cast<float *>(sb + plan.part);
    uint32_t *misc = reinterpret_cast<uint32_t *>(sb + plan.misc);
    const uint32_t pcol = plan.ntask + 1;  // float4 slots per column of task sums

    // ---- prologue: the instance's frontier range and tables
    const int T = 1 << L.logT;
    for (int i = tid; i < T; i += BLK) { L.pkey[i] = 0; pmask[i] = 0u; }
    for (int i = tid; i < M * M; i += BLK) fl[i] = 0u;
    if (tid < D) {
        rho[tid] = a.resident[(int64_t)b * D + tid];
        wait[tid] = fmaxf(0.0f, a.tau[(int64_t)b * D + tid] - a.tnow[b]);
        capd[tid] = a.cap[tid];
    }
    if (tid < M) { fits[tid] = a.fits[tid]; wt[tid] = a.weight[tid]; }
    if (tid == 0) {
        float g = 1.0f;
        for (int h = 0; h < 16; ++h) { gpow[h] = g; g *= ps.gamma; }
    }
    for (int i = tid; i < M * ND; i += BLK) {  // cost terms under the instance's residency
        const int m = i / ND, d = i - m * ND;
        float sw0 = 0.0f, sks = 0.0f;
        if (d < D) {
            const int j = m * D + d;
            const float ks = ps.lam_s * a.ksw[j];
            const bool res = bit(a.resident[(int64_t)b * D + d], m);
            const float swo = res ? 0.0f : ks;
            sw0 = a.exec[j] + swo;
            CostS c;
            c.sw0 = sw0;
            c.ksr = ks;
            c.exec = a.exec[j];
            c.swo = swo;
            cst[j] = c;
            // a row's cost is +infinity where the model does not fit (its
            // feasibility then only needs A(w)); the magnitude carries the
            // sign of the change a flip of the residency makes: up where m is
            // resident now (evicted), down where it is not (loaded)
            if (!bit(a.fits[m], d)) sw0 = inf_f();
            sks = res ? ks : -ks;
        }
        rtab[m * CS + 2 * d] = sw0;  // devices past D: never feasible
        rtab[m * CS + 2 * d + 1] = sks;
    }
    constexpr int kPre = 4;  // prefix-cache entries fetched before the barrier
    uint64_t pre[kPre];
#pragma unroll
    for (int r = 0; r < kPre; ++r) {
        const int i = tid + r * BLK;
        pre[r] = i < D * K ? a.pcache[(int64_t)b * D * K + i] : 0ull;
    }
    if (tid == 0) {  // the instance's frontier range
        const uint32_t lo = a.fr_off[b], hi = a.fr_off[b + 1];
        misc[0] = lo;
        misc[1] = hi - lo;
    }
    __syncthreads();
    const int64_t lo = misc[0];
    const int nFi = (int)misc[1];
    if (nFi == 0) return;  // uniform
#pragma unroll
    for (int r = 0; r < kPre; ++r)
        if (pre[r] != 0) table_insert<uint32_t>(L, pre[r], (tid + r * BLK) / K);
    for (int i = tid + kPre * BLK; i < D * K; i += BLK) {
        const uint64_t h = a.pcache[(int64_t)b * D * K + i];
        if (h != 0) table_insert<uint32_t>(L, h, i / K);
    }
    // Load's effect on m(w)'s residency, per (m(v), m(w)): the devices where
    // it flips (high half) and where m(w) becomes resident (low half)
    for (int i = tid; i < M * D; i += BLK) {
        const int m = i / D, d = i - m * D;
        const uint64_t r0 = rho[d], r1 = load_model(r0, m, capd[d], wt);
        const uint64_t ldm = r1 & ~r0;
        for (uint64_t x = r0 ^ r1; x; x &= x - 1) {
            const int mw = __builtin_ctzll(x);
            atomicOr(&fl[m * M + mw], (1u << (16 + d)) | ((uint32_t)((ldm >> mw) & 1ull) << d));
        }
    }
    __syncthreads();

    const float lam_tr = ps.lam_tr, lam_c = ps.lam_c, lam_p = ps.lam_p, b0 = a.beta0;
    const uint32_t dmask = (1u << D) - 1u;  // D <= 16
    constexpr int G = ND, kGroups = BLK / G;
    const int lane = tid & (G - 1);
    const bool live = lane < D;
    const int dl = live ? lane : D - 1;
    const bool lane_rank = a.topk > 0 && a.topk <= kLaneTopk;

    for (int c0 = 0; c0 < nFi; c0 += kRowsChunk) {  // uniform: chunks of the instance's frontier
        const int nC = min(kRowsChunk, nFi - c0);
        const int64_t fc = lo + c0;  // frontier slot of the chunk's first stage
        if (tid < nC) {  // stage records, descendant ranges, v's first completed parent
            const uint32_t v = a.frontier[2 * (fc + tid)];
            const StageRec r = a.rec[v];
            StageR s;
            s.elig = r.elig;
            s.hash = r.hash;
            s.tokens = r.tokens;
            s.sigma = r.sigma;
            s.e0 = a.desc_off[v];
            uint32_t n = a.desc_off[v + 1] - s.e0;
            if (ps.H < a.Hpack && n > 0) {  // entries are ordered by depth: those within H form a prefix
                uint32_t l0 = 0, l1 = n;
                while (l0 < l1) {
                    const uint32_t mid = (l0 + l1) >> 1;
                    if ((int)(a.desc[s.e0 + mid] >> kDescDepthShift) <= ps.H) l0 = mid + 1;
                    else l1 = mid;
                }
                n = l0;
            }
            s.n = n;
            s.c0 = a.cand_off[fc + tid];
            s.dbeg = r.par_begin;
            s.dn = (uint16_t)a.done_n[v];
            s.npar = r.npar;
            s.model = r.model;
            s.pad0 = 0;
            s.h0 = 0;
            s.s0 = 0.0f;
            if (s.dn > 0) {
                const DoneParent pu = a.done[s.dbeg];
                s.h0 = (uint16_t)pu.holders;
                s.s0 = pu.sigma;
            }
            s.q0 = s.nq = 0;
            s.pfm = table_find<uint32_t>(L, r.hash);
            stg[tid] = s;
        }
        __syncthreads();
        if (tid < 64) {
            // tasks of L rows over the chunk's R rows in S stages, L the
            // shortest length whose tasks (ceil(n / L) per stage of n rows) fit
            // the cap task slots: every stage's full-length tasks first, then
            // its shorter tail task; the tail tasks ordered by length, longest
            // first (ties by stage), so that the lanes of a wave run the same
            // number of rows
            const int i0 = 2 * tid, i1 = 2 * tid + 1;
            const uint32_t n0 = i0 < nC ? stg[i0].n : 0u, n1 = i1 < nC ? stg[i1].n : 0u;
            uint32_t R = 0, S = 0;
            (void)wave_exscan_u32(n0 + n1, R);
            (void)wave_exscan_u32((n0 ? 1u : 0u) + (n1 ? 1u : 0u), S);
            // binary search between ceil(R / cap), below which the full tasks
            // alone overflow, and ceil(R / (cap - S)), where even one tail per
            // stage fits (S <= kRowsChunk < cap)
            uint32_t lo = R > 0 ? max(1u, (R + plan.ntask - 1u) / plan.ntask) : 1u;
            uint32_t hi = R > 0 ? max(1u, (R + plan.ntask - S - 1u) / (plan.ntask - S)) : 1u;
            while (lo < hi) {  // uniform
                const uint32_t mid = (lo + hi) >> 1;
                uint32_t cnt = 0;
                (void)wave_exscan_u32((n0 + mid - 1u) / mid + (n1 + mid - 1u) / mid, cnt);
                if (cnt <= plan.ntask) hi = mid;
                else lo = mid + 1u;
            }
            const uint32_t Lr = lo;
            const uint32_t f0n = n0 / Lr, f1n = n1 / Lr, t0n = n0 - f0n * Lr, t1n = n1 - f1n * Lr;
            uint32_t nfull = 0;
            const uint32_t off = wave_exscan_u32(f0n + f1n, nfull);
            // tail tasks by length buckets, longest first: a count per bucket,
            // then each tail takes the next slot of its bucket (which lane
            // runs which task does not change any sum: a stage adds its full
            // tasks, then its tail)
            uint32_t *bkt = reinterpret_cast<uint32_t *>(partf);  // scratch until the rows write their sums
            constexpr uint32_t kBuckets = 32;
            auto bucket = [&](uint32_t len) { return len >= kBuckets ? kBuckets - 1u : len; };
            if (tid < (int)kBuckets) bkt[tid] = 0u;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (i0 < nC && t0n) atomicAdd(&bkt[bucket(t0n)], 1u);
            if (i1 < nC && t1n) atomicAdd(&bkt[bucket(t1n)], 1u);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint32_t cb = tid < (int)kBuckets ? bkt[kBuckets - 1u - (uint32_t)tid] : 0u;  // longest first
            uint32_t ntail = 0;
            const uint32_t start = nfull + wave_exscan_u32(cb, ntail);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (tid < (int)kBuckets) bkt[kBuckets - 1u - (uint32_t)tid] = start;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint32_t k0 = (i0 < nC && t0n) ? atomicAdd(&bkt[bucket(t0n)], 1u) : 0u;
            const uint32_t k1 = (i1 < nC && t1n) ? atomicAdd(&bkt[bucket(t1n)], 1u) : 0u;
            if (i0 < nC) {
                stg[i0].q0 = off | (f0n << 16);
                stg[i0].nq = t0n ? k0 : 0xffffffffu;
                if (t0n) tasks[k0] = (uint32_t)i0 | (f0n << 16);
            }
            if (i1 < nC) {
                stg[i1].q0 = (off + f0n) | (f1n << 16);
                stg[i1].nq = t1n ? k1 : 0xffffffffu;
                if (t1n) tasks[k1] = (uint32_t)i1 | (f1n << 16);
            }
            for (uint32_t p = 0; p < f0n; ++p) tasks[off + p] = (uint32_t)i0 | (p << 16);
            for (uint32_t p = 0; p < f1n; ++p) tasks[off + f0n + p] = (uint32_t)i1 | (p << 16);
            if (tid == 0) {
                misc[2] = nfull + ntail;
                misc[3] = Lr;
            }
        }
        __syncthreads();
        const int ntask = (int)misc[2];
        const uint32_t Lr = misc[3];

        // ---- rows
        for (int t = tid; t < ntask; t += BLK) {
            const uint32_t tk = tasks[t];
            const int si = (int)(tk & 0xffffu);
            const uint32_t pt = tk >> 16;
            const StageR s = stg[si];
            const uint32_t r0 = pt * Lr, r1 = min(s.n, r0 + Lr);
            const uint64_t hv = s.hash;
            const float t0 = lam_tr * s.sigma * b0;  // v's output to one more device
            const uint32_t *flr = fl + (uint32_t)s.model * (uint32_t)M;
            // f[d]: the task's sums of gamma^depth * min(outside, C(d)) less
            // the row terms common to every device, which go to fx
            float f[ND], fx = 0.0f;
#pragma unroll
            for (int d = 0; d < ND; ++d) f[d] = 0.0f;
            // a row from w's row record: group hash, L(w), A(w) | m(w) << 16 | |Pa(w)| << 21
            auto row = [&](uint32_t ent, const RowRec &rw, uint32_t dn) {
                const int depth = (int)(ent >> kDescDepthShift);
                const uint32_t mw = (rw.meta >> 16) & 31u;
                const uint32_t feas = rw.meta & dmask;  // the row table is +infinity where m(w) does not fit
                const uint32_t pfo = table_find<uint32_t>(L, rw.hash);
                const bool same = rw.hash != 0 && rw.hash == hv;
                const float gh = gpow[depth];
                const float pfp = lam_p * ps.kpf * rw.tokens;
                const float cw = lam_c * fast_rcp((float)(rw.meta >> 21));  // a descendant has at least one parent
                const uint32_t flip = flr[mw] >> 16;
                const float *crow = rtab + mw * CS;
                // B without the completed parents: cost with the switch term, less the prefix benefit
                float B[ND];
#pragma unroll
                for (int j = 0; j < ND / 2; ++j) {
                    const float4 c = *reinterpret_cast<const float4 *>(crow + 4 * j);
                    B[2 * j] = c.x - __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)pfo, 2 * j, 1u));
                    B[2 * j + 1] = c.z - __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)pfo, 2 * j + 1, 1u));
                }
                // completed parents: every one's transfer (all remote), and on the
                // devices holding one its transfer saved and the colocation share
                float xb = 0.0f;
                if (dn > 0) {  // the row goes through the task's sum slots, indexed by device
                    const uint32_t db = a.rec[ent & kDescIdMask].par_begin;  // w's completed-parent slots
#pragma unroll
                    for (int j = 0; j < NJ; ++j) part4[j * pcol + t] = make_float4(B[4 * j], B[4 * j + 1], B[4 * j + 2], B[4 * j + 3]);
                    for (uint32_t q0 = 0; q0 < dn; q0 += 4) {  // the batch's loads are issued together
                        DoneParent pb[4];
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (q0 + j < dn) pb[j] = a.done[db + q0 + j];
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            if (q0 + j >= dn) break;
                            const float tq = lam_tr * b0 * pb[j].sigma;
                            xb += tq;
                            const float pw = tq + cw;
                            for (uint32_t h = (uint32_t)pb[j].holders & dmask; h; h &= h - 1u) {
                                const int d = __builtin_ctz(h);
                                partf[((d >> 2) * pcol + t) * 4 + (d & 3)] -= pw;
                            }
                        }
                    }
#pragma unroll
                    for (int j = 0; j < NJ; ++j) {
                        const float4 c = part4[j * pcol + t];
                        B[4 * j] = c.x; B[4 * j + 1] = c.y; B[4 * j + 2] = c.z; B[4 * j + 3] = c.w;
                    }
                }
                // feasibility, and the two smallest values of the row.  The
                // parents' transfer xb is common to every device of the row
                // (B, the outside minimum and C all carry it), and so is a
                // child's colocation share once it is moved to the outside
                // side: min(o, B - cw + ...) = min(o + cw, B + ...) - cw.
                // Both go to fx, once per row.
                float m1 = inf_f(), m2 = inf_f();
#pragma unroll
                for (int d = 0; d < ND; ++d) {
                    const uint32_t fm = (uint32_t)__builtin_amdgcn_sbfe((int)feas, d, 1u);
                    const float x = __uint_as_float((fm & __float_as_uint(B[d])) | (~fm & __float_as_uint(inf_f())));
                    B[d] = x;
                    m2 = __builtin_amdgcn_fmed3f(m1, x, m2);
                    m1 = fminf(m1, x);
                }
                const bool child = depth == 1;
                const float cwc = child ? cw : 0.0f;
                const float m1c = child ? (m1 + t0) + cw : m1, m2c = child ? (m2 + t0) + cw : m2;
                fx += gh * (xb - cwc);
                // devices that gain grp(w) once v runs there
                const uint32_t gain = same ? (~pfo & dmask) : 0u;
#pragma unroll
                for (int j = 0; j < ND / 2; ++j) {
                    const float4 c = *reinterpret_cast<const float4 *>(crow + 4 * j);
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const int d = 2 * j + u;
                        // m(w)'s switch term on d changes by the signed magnitude
                        // where v's Load flips m(w)'s residency there
                        const float dsw = __uint_as_float(__float_as_uint(u == 0 ? c.y : c.w) & (uint32_t)__builtin_amdgcn_sbfe((int)flip, d, 1u));
                        const float gp = __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)gain, d, 1u));
                        const float C = (B[d] + dsw) - gp;
                        const float o = B[d] == m1 ? m2c : m1c;
                        f[d] += gh * fminf(o, C);
                    }
                }
            };
            for (uint32_t r = r0; r < r1; r += 4) {  // four rows' loads in flight together
                uint32_t e[4];
                RowRec w[4];
                uint32_t dn[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) e[j] = r + j < r1 ? a.desc[s.e0 + r + j] : 0u;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    w[j] = a.rowrec[e[j] & kDescIdMask];
                    dn[j] = a.done_n[e[j] & kDescIdMask];
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (r + j < r1) row(e[j], w[j], dn[j]);
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                part4[j * pcol + t] = make_float4(f[4 * j] + fx, f[4 * j + 1] + fx, f[4 * j + 2] + fx, f[4 * j + 3] + fx);
        }
        __syncthreads();

        // ---- combine: immediate cost plus the stage's task sums; scores
        for (int i = tid / G; i < nC; i += kGroups) {  // uniform within the group
            const StageR s = stg[i];
            // completed parents of v, each to the whole group in order; the first was staged
            float tr = 0.0f, cnt = 0.0f;
            if (s.dn > 0) {
                const bool local = ((s.h0 >> dl) & 1u) != 0;
                cnt += local ? 1.0f : 0.0f;
                tr += local ? 0.0f : s.s0 * b0;
            }
            for (int q0 = 1; q0 < (int)s.dn; q0 += 4) {  // every lane loads the batch (one address per group), in order
                DoneParent pb[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (q0 + j < (int)s.dn) pb[j] = a.done[s.dbeg + q0 + j];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (q0 + j >= (int)s.dn) break;
                    const bool local = (((uint32_t)pb[j].holders >> dl) & 1u) != 0;
                    cnt += local ? 1.0f : 0.0f;
                    tr += local ? 0.0f : pb[j].sigma * b0;
                }
            }
            const CostS c = cst[s.model * D + dl];
            const float pf_v = ((s.pfm >> dl) & 1u) ? ps.kpf * s.tokens : 0.0f;
            const float colo = s.npar ? cnt * fast_rcp((float)s.npar) : 0.0f;
            const float a_imm = ps.lam_q * wait[dl] + c.swo - lam_c * colo;
            const float b_imm = c.exec + lam_tr * tr - lam_p * pf_v;
            // full-length tasks in row order, then the tail; task t's sum for
            // this lane's device at pc[4 t], four loads in flight per batch
            const uint32_t qf = s.q0 & 0xffffu, nf = s.q0 >> 16;
            const float *pc = partf + ((lane >> 2) * pcol + qf) * 4 + (lane & 3);
            const float xt = s.nq != 0xffffffffu ? partf[((lane >> 2) * pcol + s.nq) * 4 + (lane & 3)] : 0.0f;
            double acc = 0.0;
            uint32_t t = 0;
            for (; t + 4 <= nf; t += 4) {
                const float x0 = pc[4 * t], x1 = pc[4 * t + 4], x2 = pc[4 * t + 8], x3 = pc[4 * t + 12];
                acc += (double)x0;
                acc += (double)x1;
                acc += (double)x2;
                acc += (double)x3;
            }
            for (; t < nf; ++t) acc += (double)pc[4 * t];
            if (s.nq != 0xffffffffu) acc += (double)xt;
            const bool feas_v = live && bit(s.elig, lane) && bit(fits[s.model], lane);
            const float psi = feas_v ? (float)(-((double)(a_imm + b_imm) + acc)) : -inf_f();
            if (live) scores[s.c0 + lane] = psi;
            if (a.topk > 0) {
                if (lane_rank) {  // the stage's record slot takes its score bits
                    reinterpret_cast<uint32_t *>(stg + i)[lane] = live ? topk_bits(psi) : 0u;
                } else {
                    const int64_t f = fc + i;
                    uint32_t sbits[1] = {live ? topk_bits(psi) : 0u};
                    const uint32_t ci[1] = {(uint32_t)lane};
                    group_topk_at<G, 1>(sbits, ci, lane, a.topk, a.tk_idx + f * a.topk, a.tk_val + f * a.topk);
                }
            }
        }
        if (lane_rank) {  // uniform over the block
            __syncthreads();
            if (tid < nC) {
                const uint32_t *slot = reinterpret_cast<const uint32_t *>(stg + tid);
                uint32_t x[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) x[q] = q < ND ? slot[q] : 0u;
                const int64_t f = fc + tid;
                lane_topk16(x, a.topk, a.tk_idx + f * a.topk, a.tk_val + f * a.topk);
            }
        }
        if (c0 + kRowsChunk < nFi) __syncthreads();  // uniform: the next chunk reuses the stage slots and task sums
    }
}

// ---- k_rows4: one horizon row per four lanes (17 to 64 devices) -----------
// The rows kernel for wider clusters: a row's devices are split over the
// four lanes of a quad, lane ql of the quad holding devices 16 ql .. 16 ql +
// 15.  Each lane keeps the two smallest B of its sixteen, two exchanges
// within the quad give the row's two smallest, and each lane adds its
// devices' terms to its part of the task's sums (a task belongs to a quad).
// Device masks are 64-bit.  The combine gives each stage a whole wave (lane
// d = device d), which also ranks the stage's top-k.
struct alignas(16) StageR4 {
    uint64_t elig, hash;
    uint64_t pfm;        // devices caching grp(v)
    uint64_t h0;         // devices holding the first completed parent's output
    float tokens, sigma;
    uint32_t e0, n;      // first descendant entry; rows within the horizon
    uint32_t c0, dbeg;   // first score; first completed parent
    uint32_t q0, nq;     // first full-length task and their number; the tail task (or 0xffffffff)
    float s0;            // the first completed parent's output size
    uint16_t dn, npar;
    uint8_t model, pad0, pad1, pad2;
    uint32_t pad3;
};
static_assert(sizeof(StageR4) == 80, "StageR4");

constexpr int kRows4Devs = 64;                       // devices a row can span
constexpr int kRows4Stride = 2 * kRows4Devs + 4;     // floats per model row of the cost table

struct Rows4Plan {
    uint32_t pkey, pmask, rho, cap, wt, fits, wait, gpow, rtab, flf, stages, tasks, part, misc, total;
    uint32_t ntask;  // task slots: one per quad
};

// Task sums as float4 columns (16 of them: devices 4 j .. 4 j + 3), column j
// of task t at part4[j * (ntask + 1) + t].
__host__ __device__ inline Rows4Plan rows4_plan(int D, int K, int M, int blk) {
    Rows4Plan q;
    const uint32_t T = 1u << table_log2(D, K);
    q.ntask = (uint32_t)(blk / 4);
    uint32_t o = 0;
    q.pkey = o; o += 8 * T;
    q.pmask = o; o += 8 * T;
    q.rho = o; o += 8 * kRows4Devs;
    q.cap = o; o += 8 * kRows4Devs;
    q.wt = o; o += 8 * (uint32_t)M;
    q.fits = o; o += 8 * (uint32_t)M;
    q.wait = o; o += 4 * kRows4Devs;
    q.gpow = o; o += 4 * 16;
    o = (o + 15u) & ~15u;
    q.rtab = o; o += 4 * (uint32_t)(M * kRows4Stride);
    o = (o + 7u) & ~7u;
    q.flf = o; o += 8 * (uint32_t)(M * M);
    o = (o + 15u) & ~15u;
    q.stages = o; o += (uint32_t)sizeof(StageR4) * (uint32_t)kRowsChunk;
    q.tasks = o; o += 4 * q.ntask;
    o = (o + 15u) & ~15u;
    q.part = o; o += 16 * (uint32_t)(kRows4Devs / 4) * (q.ntask + 1);
    q.misc = o; o += 4 * 16;
    q.total = (o + 15u) & ~15u;
    return q;
}

// The two smallest of a quad's (m1, m2) pairs, on every lane of the quad.
template <int CTRL>
__device__ __forceinline__ float quad_move(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ void quad_two_smallest(float &m1, float &m2) {
    float x1 = quad_move<0xB1>(m1), x2 = quad_move<0xB1>(m2);  // quad_perm [1, 0, 3, 2]
    float lo = fminf(m1, x1);
    m2 = fminf(fmaxf(m1, x1), fminf(m2, x2));
    m1 = lo;
    x1 = quad_move<0x4E>(m1);  // quad_perm [2, 3, 0, 1]
    x2 = quad_move<0x4E>(m2);
    lo = fminf(m1, x1);
    m2 = fminf(fmaxf(m1, x1), fminf(m2, x2));
    m1 = lo;
}

template <int BLK>
__global__ __launch_bounds__(BLK) void k_rows4(ScoreLaunch a) {
    constexpr int ND = 16, NJ = ND / 4;  // devices per lane, float4 columns per lane
    constexpr int CS = kRows4Stride;
    static_assert(BLK / 4 >= kRowsChunk && BLK % 64 == 0, "a task slot per stage of a chunk, one thread per stage");
    const int b = (int)a.order[blockIdx.x];  // largest frontiers first: the last workgroups to start are short
    const ParamSet ps = a.ps[blockIdx.y];
    float *const scores = a.scores + (int64_t)a.set_of[blockIdx.y] * a.score_stride;
    extern __shared__ uint64_t smem[];
    uint8_t *sb = reinterpret_cast<uint8_t *>(smem);
    const int tid = threadIdx.x;
    const int D = a.D, K = a.K, M = a.M;
    const Rows4Plan plan = rows4_plan(D, K, M, BLK);
    Lds L;
    L.logT = table_log2(D, K);
    L.pkey = reinterpret_cast<uint64_t *>(sb + plan.pkey);
    L.pmask = sb + plan.pmask;
    uint64_t *pmask = reinterpret_cast<uint64_t *>(sb + plan.pmask);
    uint64_t *rho = reinterpret_cast<uint64_t *>(sb + plan.rho);
    uint64_t *capd = reinterpret_cast<uint64_t *>(sb + plan.cap);
    uint64_t *wt = reinterpret_cast<uint64_t *>(sb + plan.wt);
    uint64_t *fits = reinterpret_cast<uint64_t *>(sb + plan.fits);
    float *wait = reinterpret_cast<float *>(sb + plan.wait);
    float *gpow = reinterpret_cast<float *>(sb + plan.gpow);
    float *rtab = reinterpret_cast<float *>(sb + plan.rtab);
    uint64_t *flf = reinterpret_cast<uint64_t *>(sb + plan.flf);  // per (m(v), m(w)): devices where Load flips m(w)
    StageR4 *stg = reinterpret_cast<StageR4 *>(sb + plan.stages);
    uint32_t *tasks = reinterpret_cast<uint32_t *>(sb + plan.tasks);
    float4 *part4 = reinterpret_cast<float4 *>(sb + plan.part);
    float *partf = reinterpret_cast<float *>(sb + plan.part);
    uint32_t *misc = reinterpret_cast<uint32_t *>(sb + plan.misc);
    const uint32_t pcol = plan.ntask + 1;  // float4 slots per column of task sums

    // ---- prologue: the instance's frontier range and tables
    const int64_t lo = a.fr_off[b];
    const int nFi = (int)(a.fr_off[b + 1] - (uint32_t)lo);
    if (nFi == 0) return;  // uniform
    const int T = 1 << L.logT;
    for (int i = tid; i < T; i += BLK) { L.pkey[i] = 0; pmask[i] = 0ull; }
    for (int i = tid; i < M * M; i += BLK) flf[i] = 0ull;
    if (tid < D) {
        rho[tid] = a.resident[(int64_t)b * D + tid];
        wait[tid] = fmaxf(0.0f, a.tau[(int64_t)b * D + tid] - a.tnow[b]);
        capd[tid] = a.cap[tid];
    }
    if (tid < M) { fits[tid] = a.fits[tid]; wt[tid] = a.weight[tid]; }
    if (tid == 0) {
        float g = 1.0f;
        for (int h = 0; h < 16; ++h) { gpow[h] = g; g *= ps.gamma; }
    }
    for (int i = tid; i < M * kRows4Devs; i += BLK) {  // cost terms under the instance's residency
        const int m = i / kRows4Devs, d = i - m * kRows4Devs;
        float sw0 = 0.0f, sks = 0.0f;
        if (d < D) {
            const int j = m * D + d;
            const float ks = ps.lam_s * a.ksw[j];
            const bool res = bit(a.resident[(int64_t)b * D + d], m);
            sw0 = a.exec[j] + (res ? 0.0f : ks);
            // +infinity where the model does not fit; the magnitude signed by
            // the change a flip of the residency makes (up where resident now)
            if (!bit(a.fits[m], d)) sw0 = inf_f();
            sks = res ? ks : -ks;
        }
        rtab[m * CS + 2 * d] = sw0;  // devices past D: never feasible
        rtab[m * CS + 2 * d + 1] = sks;
    }
    constexpr int kPre = 4;  // prefix-cache entries fetched before the barrier
    uint64_t pre[kPre];
#pragma unroll
    for (int r = 0; r < kPre; ++r) {
        const int i = tid + r * BLK;
        pre[r] = i < D * K ? a.pcache[(int64_t)b * D * K + i] : 0ull;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPre; ++r)
        if (pre[r] != 0) table_insert<uint64_t>(L, pre[r], (tid + r * BLK) / K);
    for (int i = tid + kPre * BLK; i < D * K; i += BLK) {
        const uint64_t h = a.pcache[(int64_t)b * D * K + i];
        if (h != 0) table_insert<uint64_t>(L, h, i / K);
    }
    // Load's effect on m(w)'s residency, per (m(v), m(w))
    for (int i = tid; i < M * D; i += BLK) {
        const int m = i / D, d = i - m * D;
        const uint64_t r0 = rho[d], r1 = load_model(r0, m, capd[d], wt);
        for (uint64_t x = r0 ^ r1; x; x &= x - 1) {
            const int mw = __builtin_ctzll(x);
            atomicOr((unsigned long long *)&flf[m * M + mw], 1ull << d);
        }
    }
    __syncthreads();

    const float lam_tr = ps.lam_tr, lam_c = ps.lam_c, lam_p = ps.lam_p, b0 = a.beta0;
    const uint64_t dmask = D >= 64 ? ~0ull : ((1ull << D) - 1ull);
    constexpr int G = 64, kGroups = BLK / G;  // the combine: a wave per stage
    const int lane = tid & 63;
    const bool live = lane < D;
    const int dl = live ? lane : D - 1;
    const int ql = tid & 3, dq = ND * ql;  // this lane's devices within its quad's row
    const uint32_t qmask = (uint32_t)((dmask >> dq) & 0xffffull);

    for (int c0 = 0; c0 < nFi; c0 += kRowsChunk) {  // uniform: chunks of the instance's frontier
        const int nC = min(kRowsChunk, nFi - c0);
        const int64_t fc = lo + c0;  // frontier slot of the chunk's first stage
        if (tid < nC) {  // stage records, descendant ranges, v's first completed parent
            const uint32_t v = a.frontier[2 * (fc + tid)];
            const StageRec r = a.rec[v];
            StageR4 s;
            s.elig = r.elig;
            s.hash = r.hash;
            s.tokens = r.tokens;
            s.sigma = r.sigma;
            s.e0 = a.desc_off[v];
            uint32_t n = a.desc_off[v + 1] - s.e0;
            if (ps.H < a.Hpack && n > 0) {  // entries are ordered by depth: those within H form a prefix
                uint32_t l0 = 0, l1 = n;
                while (l0 < l1) {
                    const uint32_t mid = (l0 + l1) >> 1;
                    if ((int)(a.desc[s.e0 + mid] >> kDescDepthShift) <= ps.H) l0 = mid + 1;
                    else l1 = mid;
                }
                n = l0;
            }
            s.n = n;
            s.c0 = a.cand_off[fc + tid];
            s.dbeg = r.par_begin;
            s.dn = (uint16_t)a.done_n[v];
            s.npar = r.npar;
            s.model = r.model;
            s.pad0 = s.pad1 = s.pad2 = 0;
            s.pad3 = 0;
            s.h0 = 0;
            s.s0 = 0.0f;
            if (s.dn > 0) {
                const DoneParent pu = a.done[s.dbeg];
                s.h0 = pu.holders;
                s.s0 = pu.sigma;
            }
            s.q0 = s.nq = 0;
            s.pfm = table_find<uint64_t>(L, r.hash);
            stg[tid] = s;
        }
        __syncthreads();
        if (tid < 64) {
            // tasks of L rows over the chunk's R rows in S stages, L the
            // shortest length whose tasks (ceil(n / L) per stage of n rows) fit
            // the task slots: every stage's full-length tasks first, then its
            // shorter tail task; the tail tasks ordered by length, longest
            // first (ties by stage), so that the quads of a wave run the same
            // number of rows
            const int i0 = 2 * tid, i1 = 2 * tid + 1;
            const uint32_t n0 = i0 < nC ? stg[i0].n : 0u, n1 = i1 < nC ? stg[i1].n : 0u;
            uint32_t R = 0, S = 0;
            (void)wave_exscan_u32(n0 + n1, R);
            (void)wave_exscan_u32((n0 ? 1u : 0u) + (n1 ? 1u : 0u), S);
            uint32_t tlo = R > 0 ? max(1u, (R + plan.ntask - 1u) / plan.ntask) : 1u;
            uint32_t thi = R > 0 ? max(1u, (R + plan.ntask - S - 1u) / (plan.ntask - S)) : 1u;
            while (tlo < thi) {  // uniform
                const uint32_t mid = (tlo + thi) >> 1;
                uint32_t cnt = 0;
                (void)wave_exscan_u32((n0 + mid - 1u) / mid + (n1 + mid - 1u) / mid, cnt);
                if (cnt <= plan.ntask) thi = mid;
                else tlo = mid + 1u;
            }
            const uint32_t Lr = tlo;
            const uint32_t f0n = n0 / Lr, f1n = n1 / Lr, t0n = n0 - f0n * Lr, t1n = n1 - f1n * Lr;
            uint32_t nfull = 0;
            const uint32_t off = wave_exscan_u32(f0n + f1n, nfull);
            uint32_t *bkt = reinterpret_cast<uint32_t *>(partf);  // scratch until the rows write their sums
            constexpr uint32_t kBuckets = 32;
            auto bucket = [&](uint32_t len) { return len >= kBuckets ? kBuckets - 1u : len; };
            if (tid < (int)kBuckets) bkt[tid] = 0u;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (i0 < nC && t0n) atomicAdd(&bkt[bucket(t0n)], 1u);
            if (i1 < nC && t1n) atomicAdd(&bkt[bucket(t1n)], 1u);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint32_t cb = tid < (int)kBuckets ? bkt[kBuckets - 1u - (uint32_t)tid] : 0u;  // longest first
            uint32_t ntail = 0;
            const uint32_t start = nfull + wave_exscan_u32(cb, ntail);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (tid < (int)kBuckets) bkt[kBuckets - 1u - (uint32_t)tid] = start;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint32_t k0 = (i0 < nC && t0n) ? atomicAdd(&bkt[bucket(t0n)], 1u) : 0u;
            const uint32_t k1 = (i1 < nC && t1n) ? atomicAdd(&bkt[bucket(t1n)], 1u) : 0u;
            if (i0 < nC) {
                stg[i0].q0 = off | (f0n << 16);
                stg[i0].nq = t0n ? k0 : 0xffffffffu;
                if (t0n) tasks[k0] = (uint32_t)i0 | (f0n << 16);
            }
            if (i1 < nC) {
                stg[i1].q0 = (off + f0n) | (f1n << 16);
                stg[i1].nq = t1n ? k1 : 0xffffffffu;
                if (t1n) tasks[k1] = (uint32_t)i1 | (f1n << 16);
            }
            for (uint32_t p = 0; p < f0n; ++p) tasks[off + p] = (uint32_t)i0 | (p << 16);
            for (uint32_t p = 0; p < f1n; ++p) tasks[off + f0n + p] = (uint32_t)i1 | (p << 16);
            if (tid == 0) {
                misc[2] = nfull + ntail;
                misc[3] = Lr;
            }
        }
        __syncthreads();
        const int ntask = (int)misc[2];
        const uint32_t Lr = misc[3];

        // ---- rows: task t on quad t, lane ql taking devices dq .. dq + 15
        for (int t = tid >> 2; t < ntask; t += BLK / 4) {  // uniform within the quad
            const uint32_t tk = tasks[t];
            const int si = (int)(tk & 0xffffu);
            const uint32_t pt = tk >> 16;
            const StageR4 &s = stg[si];
            const uint32_t se0 = s.e0, sn = s.n;
            const uint32_t r0 = pt * Lr, r1 = min(sn, r0 + Lr);
            const uint64_t hv = s.hash;
            const float t0 = lam_tr * s.sigma * b0;  // v's output to one more device
            const uint32_t mrow = (uint32_t)s.model * (uint32_t)M;
            // f[d]: the task's sums less the row terms common to every device (fx)
            float f[ND], fx = 0.0f;
#pragma unroll
            for (int d = 0; d < ND; ++d) f[d] = 0.0f;
            auto row = [&](uint32_t ent, const StageRec &rw, uint32_t db, uint32_t dn) {
                const int depth = (int)(ent >> kDescDepthShift);
                const uint32_t mw = rw.model;
                const uint32_t feas = (uint32_t)((rw.elig >> dq) & 0xffffull) & qmask;  // +infinity in the row table where m(w) does not fit
                const uint64_t pfo64 = table_find<uint64_t>(L, rw.hash);
                const uint32_t pfo = (uint32_t)((pfo64 >> dq) & 0xffffull);
                const bool same = rw.hash != 0 && rw.hash == hv;
                const float gh = gpow[depth];
                const float pfp = lam_p * ps.kpf * rw.tokens;
                const float cw = lam_c * fast_rcp((float)rw.npar);  // a descendant has at least one parent
                const uint32_t flip = (uint32_t)((flf[mrow + mw] >> dq) & 0xffffull);
                const float *crow = rtab + mw * CS + 2 * dq;
                // B without the completed parents: cost with the switch term, less the prefix benefit
                float B[ND];
#pragma unroll
                for (int j = 0; j < ND / 2; ++j) {
                    const float4 c = *reinterpret_cast<const float4 *>(crow + 4 * j);
                    B[2 * j] = c.x - __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)pfo, 2 * j, 1u));
                    B[2 * j + 1] = c.z - __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)pfo, 2 * j + 1, 1u));
                }
                // completed parents: every one's transfer (all remote), and on the
                // devices holding one its transfer saved and the colocation share
                float xb = 0.0f;
                if (dn > 0) {  // the lane's devices go through its task sum slots, indexed by device
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        part4[(dq / 4 + j) * pcol + t] = make_float4(B[4 * j], B[4 * j + 1], B[4 * j + 2], B[4 * j + 3]);
                    for (uint32_t q0 = 0; q0 < dn; q0 += 4) {  // the batch's loads are issued together
                        DoneParent pb[4];
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            if (q0 + j < dn) pb[j] = a.done[db + q0 + j];
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            if (q0 + j >= dn) break;
                            const float tq = lam_tr * b0 * pb[j].sigma;
                            xb += tq;
                            const float pw = tq + cw;
                            for (uint32_t h = (uint32_t)((pb[j].holders >> dq) & 0xffffull) & qmask; h; h &= h - 1u) {
                                const int d = dq + __builtin_ctz(h);
                                partf[((d >> 2) * pcol + t) * 4 + (d & 3)] -= pw;
                            }
                        }
                    }
#pragma unroll
                    for (int j = 0; j < NJ; ++j) {
                        const float4 c = part4[(dq / 4 + j) * pcol + t];
                        B[4 * j] = c.x; B[4 * j + 1] = c.y; B[4 * j + 2] = c.z; B[4 * j + 3] = c.w;
                    }
                }
                // feasibility, and the two smallest values of the row
                float m1 = inf_f(), m2 = inf_f();
#pragma unroll
                for (int d = 0; d < ND; ++d) {
                    const uint32_t fm = (uint32_t)__builtin_amdgcn_sbfe((int)feas, d, 1u);
                    const float x = __uint_as_float((fm & __float_as_uint(B[d])) | (~fm & __float_as_uint(inf_f())));
                    B[d] = x;
                    m2 = __builtin_amdgcn_fmed3f(m1, x, m2);
                    m1 = fminf(m1, x);
                }
                quad_two_smallest(m1, m2);
                // the parents' transfer xb and a child's colocation share (moved
                // to the outside side) are common to every device: once per row
                const bool child = depth == 1;
                const float cwc = child ? cw : 0.0f;
                const float m1c = child ? (m1 + t0) + cw : m1, m2c = child ? (m2 + t0) + cw : m2;
                fx += gh * (xb - cwc);
                // devices that gain grp(w) once v runs there
                const uint32_t gain = same ? (~pfo & qmask) : 0u;
#pragma unroll
                for (int j = 0; j < ND / 2; ++j) {
                    const float4 c = *reinterpret_cast<const float4 *>(crow + 4 * j);
#pragma unroll
                    for (int u = 0; u < 2; ++u) {
                        const int d = 2 * j + u;
                        // m(w)'s switch term on d changes by the signed magnitude
                        // where v's Load flips m(w)'s residency there
                        const float dsw = __uint_as_float(__float_as_uint(u == 0 ? c.y : c.w) & (uint32_t)__builtin_amdgcn_sbfe((int)flip, d, 1u));
                        const float gp = __uint_as_float(__float_as_uint(pfp) & (uint32_t)__builtin_amdgcn_sbfe((int)gain, d, 1u));
                        const float C = (B[d] + dsw) - gp;
                        const float o = B[d] == m1 ? m2c : m1c;
                        f[d] += gh * fminf(o, C);
                    }
                }
            };
            // one row at a time with the next row's record and completed-parent
            // count in flight, and the descendant entry after it (a workgroup
            // has the compute unit to itself, so the lane's own rows hide the
            // loads' latency)
            uint32_t e = r0 < r1 ? a.desc[se0 + r0] : 0u;
            uint32_t en = r0 + 1 < r1 ? a.desc[se0 + r0 + 1] : 0u;
            StageRec w = a.rec[e & kDescIdMask];
            uint32_t dn = a.done_n[e & kDescIdMask];
            for (uint32_t r = r0; r < r1; ++r) {
                const uint32_t ec = e, dc = dn;
                const StageRec wc = w;
                if (r + 1 < r1) {
                    w = a.rec[en & kDescIdMask];
                    dn = a.done_n[en & kDescIdMask];
                    e = en;
                }
                if (r + 2 < r1) en = a.desc[se0 + r + 2];
                row(ec, wc, wc.par_begin, dc);
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                part4[(dq / 4 + j) * pcol + t] = make_float4(f[4 * j] + fx, f[4 * j + 1] + fx, f[4 * j + 2] + fx, f[4 * j + 3] + fx);
        }
        __syncthreads();

        // ---- combine: immediate cost plus the stage's task sums; scores and top-k
        for (int i = tid / G; i < nC; i += kGroups) {  // uniform within the wave
            const StageR4 s = stg[i];
            // completed parents of v, each to the whole wave in order; the first was staged
            float tr = 0.0f, cnt = 0.0f;
            if (s.dn > 0) {
                const bool local = ((s.h0 >> dl) & 1ull) != 0;
                cnt += local ? 1.0f : 0.0f;
                tr += local ? 0.0f : s.s0 * b0;
            }
            for (int q0 = 1; q0 < (int)s.dn; q0 += 4) {  // every lane loads the batch (one address per wave), in order
                DoneParent pb[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (q0 + j < (int)s.dn) pb[j] = a.done[s.dbeg + q0 + j];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (q0 + j >= (int)s.dn) break;
                    const bool local = ((pb[j].holders >> dl) & 1ull) != 0;
                    cnt += local ? 1.0f : 0.0f;
                    tr += local ? 0.0f : pb[j].sigma * b0;
                }
            }
            // the switch term where m(v) is not resident (the row table's
            // magnitude is negative there)
            const float swo = bit(rho[dl], s.model) ? 0.0f : -rtab[s.model * CS + 2 * dl + 1];
            const float ex = a.exec[s.model * D + dl];
            const float pf_v = ((s.pfm >> dl) & 1ull) ? ps.kpf * s.tokens : 0.0f;
            const float colo = s.npar ? cnt * fast_rcp((float)s.npar) : 0.0f;
            const float a_imm = ps.lam_q * wait[dl] + swo - lam_c * colo;
            const float b_imm = ex + lam_tr * tr - lam_p * pf_v;
            // full-length tasks in row order, then the tail; task t's sum for
            // this lane's device at pc[4 t], four loads in flight per batch
            const uint32_t qf = s.q0 & 0xffffu, nf = s.q0 >> 16;
            const float *pc = partf + ((lane >> 2) * pcol + qf) * 4 + (lane & 3);
            const float xt = s.nq != 0xffffffffu ? partf[((lane >> 2) * pcol + s.nq) * 4 + (lane & 3)] : 0.0f;
            double acc = 0.0;
            uint32_t t = 0;
            for (; t + 4 <= nf; t += 4) {
                const float x0 = pc[4 * t], x1 = pc[4 * t + 4], x2 = pc[4 * t + 8], x3 = pc[4 * t + 12];
                acc += (double)x0;
                acc += (double)x1;
                acc += (double)x2;
                acc += (double)x3;
            }
            for (; t < nf; ++t) acc += (double)pc[4 * t];
            if (s.nq != 0xffffffffu) acc += (double)xt;
            const bool feas_v = live && bit(s.elig, lane) && bit(fits[s.model], lane);
            const float psi = feas_v ? (float)(-((double)(a_imm + b_imm) + acc)) : -inf_f();
            if (live) scores[s.c0 + lane] = psi;
            if (a.topk > 0) {
                const int64_t f = fc + i;
                uint32_t sbits[1] = {live ? topk_bits(psi) : 0u};
                const uint32_t ci[1] = {(uint32_t)lane};
                group_topk_at<G, 1>(sbits, ci, lane, a.topk, a.tk_idx + f * a.topk, a.tk_val + f * a.topk);
            }
        }
        __syncthreads();  // the next chunk reuses the stage slots and task sums
    }
}

// Most workgroups of one top-k launch (sixteen per compute unit); larger
// frontiers loop over their tiles.
constexpr int64_t kTopkMaxBlocks = 4096;

}  // namespace

// Most LDS one workgroup may use on gfx950 (160 KiB per compute unit).
constexpr size_t kLdsLimit = 160 * 1024;

// Kernel instance of a launch and its LDS bytes.
struct ScoreShape {
    bool slots, split;
    int block;
    size_t lds;
};

// 16-lane groups with uniform beta and at most 32 models take the slot
// layout; 64-lane groups take the first of (heavy-stage parts, 1024 threads),
// (no parts, 1024 threads), (no parts, 512 threads) whose LDS fits.  False if
// none fits (the host rejects such shapes before anything is enqueued).
static bool score_shape(int D, int K, int M, int slice, bool uni, ScoreShape &sh) {
    const int G = group_width(D);
    sh.slots = uni && G == 16 && M <= 32;
    sh.split = false;
    sh.block = score_block(G);
    if (G < 64) {
        const int sb = G == 16 ? staging_bytes<16, score_block(16)>() : staging_bytes<8, score_block(8)>();
        sh.lds = lds_plan(D, K, M, slice, sb, sh.slots, false).total;
        return sh.lds <= kLdsLimit;
    }
    const bool split[3] = {true, false, false};
    const int block[3] = {score_block(64), score_block(64), score_block(64) / 2};
    for (int c = 0; c < 3; ++c) {
        const int sb = block[c] == score_block(64) ? staging_bytes<64, score_block(64)>()
                                                   : staging_bytes<64, score_block(64) / 2>();
        const size_t lds = lds_plan(D, K, M, slice, sb, false, split[c]).total;
        if (lds <= kLdsLimit) {
            sh.split = split[c];
            sh.block = block[c];
            sh.lds = lds;
            return true;
        }
    }
    return false;
}

bool score_fits(int D, int K, int M, int beta_uniform) {
    ScoreShape sh;
    return score_shape(D, K, M, slice_len(D), beta_uniform != 0, sh);
}

// Threads of a k_rows workgroup, and of a k_rows4 one (256 quads).
constexpr int kRowsBlock = 256;
constexpr int kRows4Block = 1024;

// The row kernels take frontiers with single-device candidates only, uniform
// beta, hop levels and parameter sets without a scoring variant: k_rows up
// to 16 devices and 32 models, k_rows4 up to 64 devices and 64 models, when
// their LDS fits.
bool rows_kernel_fits(int D, int K, int M) {
    if (D <= 16) {
        const int nd = D <= 4 ? 4 : D <= 8 ? 8 : 16;
        return M <= 32 && rows_plan(D, K, M, nd, kRowsBlock).total <= kLdsLimit;
    }
    return D <= kRows4Devs && M <= 64 && rows4_plan(D, K, M, kRows4Block).total <= kLdsLimit;
}

static bool rows_fit(const ScoreLaunch &a) {
    if (!a.beta_uniform || !a.singles || a.topo) return false;
    if (a.D <= 16 && !a.rowrec) return false;  // k_rows reads the row records
    return rows_kernel_fits(a.D, a.K, a.M);
}

static void launch_rows(const ScoreLaunch &a, hipStream_t s) {
    if (a.D > 16) {
        const size_t lds = rows4_plan(a.D, a.K, a.M, kRows4Block).total;
        hipLaunchKernelGGL((k_rows4<kRows4Block>), dim3((unsigned)a.B, (unsigned)a.nsets), dim3(kRows4Block), lds, s, a);
        return;
    }
    const int nd = a.D <= 4 ? 4 : a.D <= 8 ? 8 : 16;
    const size_t lds = rows_plan(a.D, a.K, a.M, nd, kRowsBlock).total;
    const dim3 grid((unsigned)a.B, (unsigned)a.nsets), block((unsigned)kRowsBlock);
    switch (nd) {
        case 4: hipLaunchKernelGGL((k_rows<4, kRowsBlock>), grid, block, lds, s, a); break;
        case 8: hipLaunchKernelGGL((k_rows<8, kRowsBlock>), grid, block, lds, s, a); break;
        default: hipLaunchKernelGGL((k_rows<16, kRowsBlock>), grid, block, lds, s, a); break;
    }
}

template <bool UNI>
static void launch_score_g(const ScoreLaunch &a0, const ScoreShape &sh, hipStream_t s) {
    ScoreLaunch a = a0;
    if (UNI && rows_fit(a0)) {
        // each parameter set goes where a launch of that set alone would go:
        // sets without a variant to k_rows, the others below
        ScoreLaunch r = a0;
        r.nsets = a.nsets = 0;
        for (int p = 0; p < a0.nsets; ++p) {
            ScoreLaunch &x = (a0.ps[p].lam_m != 0.0f || a0.ps[p].flags != 0) ? a : r;
            x.ps[x.nsets] = a0.ps[p];
            x.set_of[x.nsets] = a0.set_of[p];
            ++x.nsets;
        }
        if (r.nsets > 0) launch_rows(r, s);
        if (a.nsets == 0) return;
    }
    const int G = group_width(a.D);
    const dim3 grid((unsigned)a.n_slices, (unsigned)a.nsets), block((unsigned)sh.block);
    const size_t lds = sh.lds;
    bool var = a.topo != 0;
    for (int p = 0; p < a.nsets; ++p) var = var || a.ps[p].lam_m != 0.0f || a.ps[p].flags != 0;
    constexpr int B0 = kScoreBlock, B64 = score_block(64);
    switch (G) {
        case 4: hipLaunchKernelGGL((k_score<4, UNI, false, true, false, B0>), grid, block, lds, s, a); break;
        case 8: hipLaunchKernelGGL((k_score<8, UNI, false, true, false, B0>), grid, block, lds, s, a); break;
        case 16:
            if (UNI && sh.slots) {
                if (var) hipLaunchKernelGGL((k_score<16, UNI, UNI, true, false, B0>), grid, block, lds, s, a);
                else hipLaunchKernelGGL((k_score<16, UNI, UNI, false, false, B0>), grid, block, lds, s, a);
            } else {
                hipLaunchKernelGGL((k_score<16, UNI, false, true, false, B0>), grid, block, lds, s, a);
            }
            break;
        case 32: hipLaunchKernelGGL((k_score<32, UNI, false, true, false, B0>), grid, block, lds, s, a); break;
        default:
            if (sh.split) hipLaunchKernelGGL((k_score<64, UNI, false, true, true, B64>), grid, block, lds, s, a);
            else if (sh.block == B64) hipLaunchKernelGGL((k_score<64, UNI, false, true, false, B64>), grid, block, lds, s, a);
            else hipLaunchKernelGGL((k_score<64, UNI, false, true, false, B64 / 2>), grid, block, lds, s, a);
            break;
    }
}

int launch_score(const ScoreLaunch &a, void *stream) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    ScoreShape sh;
    if (!score_shape(a.D, a.K, a.M, a.slice, a.beta_uniform != 0, sh)) return (int)hipErrorInvalidValue;
    if (a.beta_uniform) launch_score_g<true>(a, sh, s);
    else launch_score_g<false>(a, sh, s);
    return (int)hipGetLastError();
}

int launch_topk(const TopkLaunch &a, void *stream) {
    const int G = group_width(a.D);
    const int64_t per_block = (int64_t)(kBlock / G) * kTopkRounds;
    const int64_t blocks = std::min((a.nF + per_block - 1) / per_block, kTopkMaxBlocks);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const dim3 grid((unsigned)blocks, (unsigned)a.nsets);
    switch (G) {
        case 4: hipLaunchKernelGGL(k_topk<4>, grid, dim3(kBlock), 0, s, a); break;
        case 8: hipLaunchKernelGGL(k_topk<8>, grid, dim3(kBlock), 0, s, a); break;
        case 16: hipLaunchKernelGGL(k_topk<16>, grid, dim3(kBlock), 0, s, a); break;
        case 32: hipLaunchKernelGGL(k_topk<32>, grid, dim3(kBlock), 0, s, a); break;
        default: hipLaunchKernelGGL(k_topk<64>, grid, dim3(kBlock), 0, s, a); break;
    }
    return (int)hipGetLastError();
}

}  // namespace fate
