// Internal layout shared by the host packer and the HIP kernels of libfate.
#pragma once

#include <stdint.h>

#include "fate.h"

namespace fate {

// 32-byte stage record, one per flat stage id (Sec. 2 stage tuple: model,
// eligible devices, shard cap, prefix group and length, output size, parents).
struct alignas(16) StageRec {
    uint64_t elig;       // A(v) device bitmask
    uint64_t hash;       // grp(v), 0 = none
    float tokens;        // L(v)
    float sigma;         // output bytes
    uint32_t par_begin;  // first entry of this stage in the flat parent list
    uint8_t model;       // m(v)
    uint8_t shard;       // R(v)
    uint16_t npar;       // |Pa(v)|
};
static_assert(sizeof(StageRec) == 32, "stage record must be 32 bytes");

// A completed parent of a stage as packed per planning step: the devices
// holding its output and its output size.
// The fields of a stage that a horizon row reads in the row kernel for at
// most 16 devices and 32 models, half a stage record: the group hash, L(v),
// and A(v) (16 bits) | m(v) << 16 (5 bits) | |Pa(v)| << 21 (11 bits).
struct alignas(16) RowRec {
    uint64_t hash;
    float tokens;
    uint32_t meta;
};
static_assert(sizeof(RowRec) == 16, "row record must be 16 bytes");
constexpr int kRowRecMaxNpar = 2047;

struct alignas(16) DoneParent {
    uint64_t holders;
    float sigma;
    uint32_t pad;
};
static_assert(sizeof(DoneParent) == 16, "completed-parent entry must be 16 bytes");

constexpr uint32_t kDescIdMask = (1u << 28) - 1u;
constexpr int kDescDepthShift = 28;

// One parameter set of a scoring launch (fate_params_t, as the kernels use
// it): Sec. 3.4 weights, App. A.3 kappa_prefix, Sec. 3.2 gamma, Sec. 3.3 H,
// the same-model weight and the variant flags.
struct ParamSet {
    float lam_q, lam_s, lam_tr, lam_c, lam_p, kpf, gamma, lam_m;
    int32_t H, flags;
};
constexpr int kMaxSets = FATE_MAX_SWEEP;

struct ScoreLaunch {
    const StageRec *rec;
    const RowRec *rowrec;  // row records (null unless D <= 16, M <= 32, |Pa| <= 2047)
    const uint32_t *par_idx;
    const uint32_t *desc_off;
    const uint32_t *desc;
    const float *desc_w;  // level weights (FATE_MEAN_PER_LEVEL), or null
    const float *exec;
    const float *ksw;
    const float *beta;
    const uint64_t *weight;
    const uint64_t *cap;
    const uint64_t *fits;
    const uint64_t *resident;
    const uint64_t *pcache;
    const uint64_t *holders;
    const float *tau;
    const float *tnow;
    const uint32_t *frontier;
    const uint32_t *cand_off;
    const uint32_t *slices;
    const uint32_t *done_n;  // completed parents of stage g: done[rec[g].par_begin ..] (done_n[g] of them)
    const DoneParent *done;
    const uint32_t *order;   // instances by decreasing frontier size (grid row x takes order[x])
    const uint32_t *fr_off;  // [B+1] instance b's frontier slots
    float *scores;            // parameter set p (blockIdx.y) writes scores + p * score_stride
    int64_t score_stride;
    const uint32_t *dcounts;  // planning state: counts[2] = current slices, else null
    int32_t *tk_idx;  // fused top-k outputs (topk > 0), [nF][topk]
    float *tk_val;
    int32_t topk;
    int64_t nF, n_slices;
    int32_t B, D, M, K, max_shard, beta_uniform, slice;
    float beta0;
    int32_t topo;  // descendant lists by topological level (FATE_LEVELS_TOPO)
    int32_t Hpack;      // horizon the descendant lists were packed with
    int32_t singles;    // every frontier stage has only single-device candidates
    int32_t nsets;
    ParamSet ps[kMaxSets];
    int32_t set_of[kMaxSets];  // grid row y scores parameter set set_of[y] (its place in the output)
};

struct TopkLaunch {
    const uint32_t *cand_off;
    const float *scores;
    int32_t *idx;
    float *val;
    const uint32_t *dcounts;  // planning state: counts[0] = current frontier size, else null
    int64_t nF;               // frontier size, or its capacity with dcounts
    int64_t score_stride;     // score set p (blockIdx.y) at scores + p * score_stride,
    int64_t out_stride;       // its top-k at idx / val + p * out_stride
    int32_t nsets;
    int32_t D, k;
};

// Commit-and-advance of a planning state (fate_commit.hip).
struct CommitLaunch {
    // packed DAGs
    const StageRec *rec;
    const uint32_t *par_idx;
    const int64_t *stage_off;
    const float *exec, *ksw, *beta;
    const uint64_t *weight, *cap, *fits;
    // planning state, updated in place
    uint64_t *resident, *pcache, *holders;
    float *tau, *fin;
    const float *tnow;
    uint8_t *status;
    uint32_t *frontier, *cand_off, *slices, *done_n, *fr_off;
    uint32_t *order;  // read by the apply kernel, re-sorted by the scan for the fill and the next step
    DoneParent *done;
    uint32_t *counts;
    // selections: sel[f * sel_stride] for frontier slot f
    const int32_t *sel;
    int32_t sel_stride;
    // packed DAGs: children lists
    const uint32_t *ch_off, *ch_idx;
    // workspace (commit_ws_layout)
    uint32_t *list;  // [N][2]: instance b's new frontier (stage, first candidate
                     // relative to the instance) from stage_off[b] on
    uint32_t *tot;   // [B][4]: new frontier stages, candidates, slices, rejected selections
    uint32_t *base;  // [B][2]: the instance's first candidate and first slice
    uint32_t *nsp;   // [B]: slices of the instance at each dispatch position
    uint32_t *gbm;   // frontier bitmaps of instances too large for LDS
    int32_t slice_order;  // 1: the slices follow the dispatch order (rows_batch false)
    int32_t bm_lds;  // 1: every instance's bitmap fits the apply kernel's LDS
    int32_t bm_words;  // bitmap words of the largest instance
    int64_t N;
    int32_t B, D, M, K, max_shard, slice;
    int32_t beta_uniform;  // every off-diagonal beta equals beta0
    float beta0;
};

// Whether a row kernel's LDS plan fits for D devices, K prefix slots and M
// models (fate_kernels.hip).
bool rows_kernel_fits(int D, int K, int M);

// Whether scoring on this batch takes a row kernel (k_rows, k_rows4) for
// parameter sets without a variant: single-device candidates only, uniform
// beta, hop levels, and tables that fit.  Its scoring slices then go unused,
// and the packer and the commit leave them in instance order; otherwise they
// follow the dispatch order (largest frontiers first).
inline bool rows_batch(const fate_dags_t *dags, int max_shard, int K) {
    const int r = dags->max_r < max_shard ? dags->max_r : max_shard;
    return dags->beta_uniform && (r < dags->D ? r : dags->D) <= 1 && dags->levels != FATE_LEVELS_TOPO &&
           rows_kernel_fits(dags->D, K, dags->M) && (dags->D > 16 || dags->row_records);
}

// The dispatch order of per-instance launches: instances by size class of
// their frontier, largest class first, each class in instance order.  Class
// 0 holds the largest frontiers: with mx the largest frontier of the batch,
// a frontier of n stages is in class C - 1 - min(C - 1, n * C / (mx + 1)).
// Longest-first list scheduling needs no finer order: eight classes keep
// within 2% of a full sort by size in a model of the fork-join launch.
constexpr int kOrderClasses = 8;
__host__ __device__ inline uint32_t order_class(uint32_t n, uint32_t mx) {
    const uint64_t c = (uint64_t)n * kOrderClasses / ((uint64_t)mx + 1u);
    return (uint32_t)(kOrderClasses - 1) - (uint32_t)(c < kOrderClasses - 1 ? c : kOrderClasses - 1);
}

// Bitmap words past which an instance's frontier bitmap moves from LDS to
// the workspace (instances of more than 32,768 stages).
constexpr int kCommitLdsBitmapWords = 1024;

// Workspace of the commit: the new frontier lists (one slot per stage), the
// per-instance totals, bases and slice counts by dispatch position, and the
// frontier bitmaps of large instances
// (instance b's from word (stage_off[b] >> 5) + b, covering bit
// (stage_off[b] & 31) + i for its stage i).
struct CommitWs {
    size_t list, tot, base, nsp, gbm, total;
};
inline CommitWs commit_ws_layout(int64_t N, int B) {
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    CommitWs w;
    size_t o = 0;
    w.list = o; o = up(o + 8 * (size_t)N);
    w.tot = o; o = up(o + 16 * (size_t)B);
    w.base = o; o = up(o + 8 * (size_t)B);
    w.nsp = o; o = up(o + 4 * (size_t)B);
    w.gbm = o; o = up(o + 4 * ((size_t)N / 32 + (size_t)B + 1));
    w.total = o;
    return w;
}

// Lane-group width for D devices (power of two, 4..64) and the number of
// frontier stages per scoring workgroup slice (eight rounds of its groups).
constexpr int kScoreBlock = 256;
// Threads per scoring workgroup: 1024 for 64-lane groups, whose instances
// have few frontier stages with many rows each, so that sixteen of them are
// in flight per workgroup; 256 otherwise.
constexpr int score_block(int G) { return G >= 64 ? 1024 : kScoreBlock; }
inline int group_width(int D) {
    int g = 4;
    while (g < D) g <<= 1;
    return g;
}
// Frontier stages per scoring workgroup: eight per lane group, but four for
// 16-lane groups, whose slot-layout staging leaves the least LDS for stage
// records (64 stages measured 2% faster than 128 on the 16-device fork-join
// batch; fewer, or other group widths, were slower).
inline int slice_len(int D) {
    const int G = group_width(D), groups = score_block(G) / G;
    const int per = G == 16 || G >= 64 ? 4 : 8;
    return groups * per > 256 ? 256 : groups * per;
}

// Kernel launchers (fate_kernels.hip).  Return a hipError_t as int.
int launch_score(const ScoreLaunch &a, void *stream);
// Whether some instance of the scoring kernel fits its LDS for this shape
// (devices, prefix slots, models, uniform beta).
bool score_fits(int D, int K, int M, int beta_uniform);
int launch_topk(const TopkLaunch &a, void *stream);
int launch_commit(const CommitLaunch &a, void *stream);  // fate_commit.hip

// Commit-and-advance behind both entry points (fate_host.cpp): validation,
// then the three launches with the workspace d_ws of ws_bytes.  commit_check
// runs the validation alone and returns the workspace bytes needed.
fate_status_t commit_check(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                           int32_t sel_stride, size_t *ws_total);
fate_status_t commit_impl(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                          int32_t sel_stride, void *d_ws, size_t ws_bytes, void *stream);

// Frontier planning wave (fate_plan.hip).
struct PlanLaunch {
    const uint32_t *frontier;  // [nF][2]: flat stage id, instance
    const uint32_t *cand_off;  // [nF + 1]: a stage's candidates are its choices' valid range
    const int32_t *idx;        // [nF][k] choices (local candidate indices, -1 = none)
    const float *val;          // [nF][k] their scores
    int32_t *sel;              // [nF] chosen candidate or -1
    const uint32_t *fr_off;    // [B+1] instance b's frontier slots
    const uint32_t *order;     // [B] instances by decreasing frontier size
    int64_t nF;                // frontier size, or its capacity with dcounts
    int32_t B, D, k;
};
int launch_plan(const PlanLaunch &a, void *stream);

// Plan execution and baseline placements on the device (fate_simdev.hip).
struct SimLaunch {
    // packed DAGs
    const StageRec *rec;
    const uint32_t *par_idx;
    const int64_t *stage_off;
    const float *exec, *ksw, *beta;
    const uint64_t *weight, *cap, *fits;
    // packed state (completed stages: holders != 0)
    const uint64_t *resident, *pcache, *holders;
    const float *tau, *tnow;
    // plan to execute, or the placement written
    const uint64_t *devices;
    const int64_t *order;
    uint64_t *dev_out;
    int64_t *ord_out;
    fate_sim_metrics_t *out;
    int32_t *status;
    // workspace (sim_ws_layout), per flat stage
    double *fin, *aux, *tail;
    uint64_t *hold, *keys;
    uint32_t *ids, *todo;
    uint8_t *flags;
    double kpf;
    int32_t B, D, K;
};
struct SimWs {
    size_t fin, aux, tail, hold, keys, ids, todo, flags, total;
};
inline SimWs sim_ws_layout(int64_t N) {
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    SimWs w;
    size_t o = 0;
    w.fin = o; o = up(o + 8 * (size_t)N);
    w.aux = o; o = up(o + 8 * (size_t)N);
    w.tail = o; o = up(o + 8 * (size_t)N);
    w.hold = o; o = up(o + 8 * (size_t)N);
    w.keys = o; o = up(o + 8 * (size_t)N);
    w.ids = o; o = up(o + 4 * (size_t)N);
    w.todo = o; o = up(o + 4 * (size_t)N);
    w.flags = o; o = up(o + (size_t)N);
    w.total = o;
    return w;
}
// mode 0: execute the plan; 1: round-robin placement; 2: HEFT-style placement
int launch_sim(const SimLaunch &a, int mode, void *stream);

}  // namespace fate
