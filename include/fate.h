/*
 * fate.h - C ABI of the MI355X horizon-aware candidate scoring library.
 *
 * The library scores, for a batch of B workflow-DAG instances, every
 * candidate placement (a single device, or a contiguous window of devices for
 * a shardable stage) of every ready-frontier stage, following FATE
 * (arXiv 2605.07238):
 *   - stage tuple (m(v), A(v), R(v), c_v, phi(v), Pa(v), Ch(v)): Sec. 2 and
 *     App. A.1;
 *   - execution state s_t = (rho_t, kappa_t, l_t, tau_t): Sec. 2, App. A.1;
 *   - ready frontier and feasible candidate set: Sec. 2, App. A.1;
 *   - score terms (waiting, switch, transfer, colocation, prefix, shard):
 *     Sec. 3.4 and App. A.3; additive state-conditional cost: App. A.1/A.4;
 *   - horizon-aware candidate score Psi(v, k, d | s_t, H): Sec. 3.3, App. A.2.
 * H counts downstream DAG levels beyond the frontier; H = 0 scores the
 * immediate cost only (App. D.4).  Psi is the negated estimated cost in
 * seconds: higher is better.
 *
 * Conventions for every entry point:
 *   - Every function returns a fate_status_t and is reentrant; the library
 *     keeps no global state and never allocates device memory.
 *   - Host arrays passed in are read during the call only and never retained.
 *   - Device buffers are allocated by the caller (sizes come from the *_size
 *     queries) and passed as a pointer plus a byte count.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Device work is
 *     enqueued on it.  The pack functions copy from pageable host memory and
 *     synchronise the stream before returning; scoring and top-k never
 *     synchronise.
 *   - Inputs are validated on the host before anything is enqueued; on an
 *     error nothing is written to device memory and outputs are untouched.
 *   - Devices are indexed 0..D-1 with D <= 64, models 0..M-1 with M <= 64;
 *     bitmasks over devices or models are uint64_t with bit i for index i.
 */
#ifndef FATE_H
#define FATE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FATE_MAX_DEVICES 64
#define FATE_MAX_MODELS 64
#define FATE_MAX_PREFIX_SLOTS 32
#define FATE_MAX_HORIZON 15
#define FATE_MAX_TOPK 64
#define FATE_MAX_SHARD 4
#define FATE_MAX_PARENTS 65535
#define FATE_MAX_SWEEP 16 /* parameter sets per fate_score_sweep / fate_topk_sweep launch */
/* Workspace that the library holds on each GPU for fate_commit_advance_noalloc
 * (32 MiB: planning states of up to about 2.7 million stages), and the number
 * of GPUs per process it keeps one for. */
#define FATE_NOALLOC_WS_BYTES (32u << 20)
#define FATE_MAX_DEVICES_PER_PROCESS 64
/* Total stages over the batch must fit 28 bits (stage ids share a 32-bit word
 * with their horizon depth in the packed descendant lists). */
#define FATE_MAX_TOTAL_STAGES ((1 << 28) - 1)

typedef enum {
    FATE_OK = 0,
    FATE_EINVAL = -1,  /* null pointer, negative size, non-finite or negative value, bad mask */
    FATE_ERANGE = -2,  /* a limit above is exceeded (D, M, K, H, k, R, parents, totals) */
    FATE_ECYCLE = -3,  /* a parent id is not smaller than its child's id, or parents unsorted */
    FATE_ENOFEAS = -4, /* a stage has no eligible device that can hold its model */
    FATE_ESIZE = -5,   /* a caller buffer is smaller than the size query returned */
    FATE_ESTATE = -6,  /* inconsistent state (status, holders, handle mismatch) */
    FATE_EHIP = -7     /* a HIP runtime call failed */
} fate_status_t;

/* Stage status codes (App. A.1 tracks completed, running and committed). */
enum { FATE_PENDING = 0, FATE_COMPLETED = 1, FATE_RUNNING = 2, FATE_COMMITTED = 3 };

/* Cluster tables (host memory), shared by every instance of a batch.
 *   exec[m*D + d]     base runtime c_v(d) of a stage using model m, seconds (>= 0)
 *   switch_s[m*D + d] kappa_switch(m, d), cost of loading model m on d, seconds (>= 0)
 *   weight_bytes[m]   memory footprint W(m) of model m, bytes (> 0)
 *   cap_bytes[d]      model memory capacity of device d, bytes (> 0)
 *   beta[i*D + j]     transfer coefficient beta_{i,j} from device i to j,
 *                     seconds per byte (>= 0; the diagonal is never used)  */
typedef struct {
    int32_t D, M;
    const float *exec;
    const float *switch_s;
    const int64_t *weight_bytes;
    const int64_t *cap_bytes;
    const float *beta;
} fate_cluster_t;

/* A batch of B DAG instances (host memory), stages stored flat.
 *   stage_off[B+1]  instance b owns flat stages [stage_off[b], stage_off[b+1]);
 *                   inside an instance stages are numbered 0..n_b-1 and
 *                   every edge goes from a smaller to a larger id
 *   par_off[N+1]    parents of flat stage g are par_idx[par_off[g] .. par_off[g+1])
 *   par_idx[E]      instance-local parent ids, strictly increasing per stage
 *   model[N]        m(v) in [0, M)
 *   elig[N]         A(v) as a device bitmask (non-zero, bits < D)
 *   shard_max[N]    R(v) in [1, 255]: maximum shard degree
 *   prefix_hash[N]  grp(v), the shared-prefix group; 0 = no group
 *   prefix_tokens[N] L(v), reusable prefix length in tokens (>= 0)
 *   out_bytes[N]    sigma(v), output size in bytes (>= 0)                  */
typedef struct {
    int32_t B;
    const int64_t *stage_off;
    const int64_t *par_off;
    const int32_t *par_idx;
    const int32_t *model;
    const uint64_t *elig;
    const int32_t *shard_max;
    const uint64_t *prefix_hash;
    const float *prefix_tokens;
    const float *out_bytes;
} fate_dag_batch_t;

/* Execution state of every instance (host memory), Sec. 2 s_t.
 *   K                  prefix-cache slots per device, 0..32
 *   resident[B*D]      rho: resident-model bitmask of device d of instance b
 *   prefix_cache[B*D*K] kappa: cached prefix groups per device, 0 = empty slot
 *   holders[N]         l: device bitmask holding a completed stage's output;
 *                      non-zero exactly for completed stages
 *   status[N]          FATE_PENDING / COMPLETED / RUNNING / COMMITTED; completed
 *                      and running stages have all parents completed
 *   tau_free[B*D]      tau_d^free: next time device d is free, seconds
 *   t_now[B]           current decision time t, seconds                    */
typedef struct {
    int32_t K;
    const uint64_t *resident;
    const uint64_t *prefix_cache;
    const uint64_t *holders;
    const uint8_t *status;
    const float *tau_free;
    const float *t_now;
} fate_state_t;

/* Scoring variants (fate_params_t.flags).
 *   FATE_MEAN_PER_LEVEL  the horizon tail averages the values of the stages at
 *                        each depth (weight gamma^h / n_h, n_h = v's horizon
 *                        stages at depth h) instead of summing them; needs
 *                        DAGs packed with level_weights
 *   FATE_NO_WINDOWS      shard windows (k > 1) keep their score slots but score
 *                        -infinity (App. C.3 "w/o shard parallelism")        */
enum { FATE_MEAN_PER_LEVEL = 1, FATE_NO_WINDOWS = 2 };

/* Score weights (Sec. 3.4 lambda_q, lambda_s, lambda_tr, lambda_c, lambda_p;
 * App. A.3 kappa_prefix), the horizon discount gamma (Sec. 3.2), the
 * horizon H (Sec. 3.3; 0 <= H <= the H the DAGs were packed with), the
 * same-model weight lam_m and the variant flags above.
 *   lam_m: the model-specialised placement preference (Sec. 4 implementation
 *   summary; App. C.3 "w/o same-model bonus"): wherever a switch cost
 *   Sw(x, d) enters a cost, -lam_m enters beside it when m(x) is resident on
 *   d in the state at hand (s_t for the frontier stage, on every shard
 *   device; s' for the horizon stages).  0 turns it off.
 * Every weight must be finite and >= 0; unknown flag bits are EINVAL. */
typedef struct {
    float lam_q, lam_s, lam_tr, lam_c, lam_p, kappa_prefix, gamma;
    int32_t H;
    float lam_m;
    int32_t flags;
} fate_params_t;

/* Horizon levels for packing (fate_pack_opts_t.levels; Sec. 3.3 "downstream
 * DAG levels").
 *   FATE_LEVELS_HOP   breadth-first hop distance from v, each stage once at
 *                     its minimum distance
 *   FATE_LEVELS_TOPO  topological level difference: level = 0 for a stage
 *                     without parents, else 1 + its parents' largest level;
 *                     the horizon of v is every stage reachable from v with
 *                     1 <= level(w) - level(v) <= H, at that depth           */
enum { FATE_LEVELS_HOP = 0, FATE_LEVELS_TOPO = 1 };

/* Packing options: the horizon H (0..15), the level definition, and
 * level_weights = 1 to also pack, per horizon entry, 1 / (number of v's
 * horizon stages at that depth) for FATE_MEAN_PER_LEVEL (4 bytes per entry). */
typedef struct {
    int32_t H;
    int32_t levels;
    int32_t level_weights;
} fate_pack_opts_t;

/* Packed DAG batch: plain data pointing into the caller's device buffer.
 * Valid while that buffer lives; filled by fate_pack_dags. */
typedef struct {
    int32_t B, D, M, H;
    int64_t N, E, n_desc;
    int32_t beta_uniform; /* 1 if every off-diagonal beta is equal */
    float beta0;          /* that common value */
    void *base;
    size_t bytes;
    const float *exec, *switch_s, *beta;
    const uint64_t *weight, *cap, *fits; /* fits[m]: devices that can hold model m */
    const void *records;                  /* 32-byte stage records [N] */
    const uint32_t *par_idx;              /* [E] flat parent ids */
    const uint32_t *desc_off;             /* [N+1] */
    const uint32_t *desc;                 /* [n_desc]: flat id | depth << 28 */
    const int64_t *stage_off;             /* [B+1] */
    int32_t levels;                       /* FATE_LEVELS_HOP or FATE_LEVELS_TOPO */
    const float *desc_w;                  /* [n_desc] level weights, or null */
    int32_t max_r;                        /* largest shard degree R(v) of the batch */
    const uint32_t *ch_off;               /* [N+1]: children of flat stage g are */
    const uint32_t *ch_idx;               /* ch_idx[ch_off[g] .. ch_off[g+1]), ascending flat ids */
    int64_t max_stages;                   /* stages of the largest instance */
    const void *row_records;              /* 16-byte row records [N] (group hash, L(v), then A(v) as 16 bits
                                             | m(v) << 16 | |Pa(v)| << 21), when D <= 16, M <= 32 and no
                                             stage has more than 2047 parents; else null */
} fate_dags_t;

/* Packed state of one planning step: plain data pointing into the caller's
 * device buffer; filled by fate_pack_state. */
typedef struct {
    int32_t B, D, K, max_shard;
    int64_t N, n_frontier, n_cand;
    void *base;
    size_t bytes;
    const uint64_t *resident, *prefix_cache, *holders;
    const float *tau_free, *t_now;
    const uint32_t *frontier; /* [n_frontier][2]: flat stage id, instance */
    const uint32_t *cand_off; /* [n_frontier+1]: first score of each frontier stage */
    int64_t n_slices;
    const uint32_t *slices;   /* [n_slices][3]: instance, first and end frontier slot; the
                                 scoring kernel runs one workgroup per slice */
    int64_t n_done_edges;     /* E: every stage has a slot per parent */
    const uint32_t *done_n;   /* [N]: the completed parents of pending flat stage g,
                                 in parent order, are done[p .. p + done_n[g]) with
                                 p = par_off[g], the first of g's |Pa(g)| slots;
                                 the counts and slots of other stages are stale */
    const void *done;         /* [E] 16-byte entries {uint64 holders; float out_bytes; pad} */
    /* Planning state (fate_pack_state_advance; all zero otherwise).  Its
     * sections are sized for any later planning step, so n_frontier,
     * n_cand and n_slices above hold those capacities, and the current
     * counts live in device memory: counts[0] frontier stages, counts[1]
     * candidates, counts[2] slices, counts[3] selections rejected by the
     * last fate_commit_advance. */
    int32_t advance;
    const uint8_t *status;    /* [N] stage status: FATE_PENDING .. FATE_COMMITTED */
    const uint32_t *counts;   /* [4] device counters, see above */
    const float *finish;      /* [N] planned finish of completed stages (t_now for
                                 those completed when planning began) */
    int32_t slice;            /* frontier stages per slice the state was cut into;
                                 scoring rejects a state whose slice length differs
                                 from this build's for the DAGs' device count (ESTATE) */
    const uint32_t *fr_off;   /* [B+1]: instance b's frontier slots are
                                 fr_off[b] .. fr_off[b+1] (current counts) */
    const uint32_t *order;    /* [B]: the order in which per-instance launches take
                                 the instances, largest frontiers first: instance b
                                 with a frontier of n stages, mx the largest, is in
                                 class 7 - min(7, 8 n / (mx + 1)), classes ascending,
                                 each in instance order (a dispatch order only: no
                                 result depends on it; a commit recomputes it) */
} fate_state_h;

const char *fate_version(void);
const char *fate_strerror(fate_status_t status);

/* fate_pack_dags_size: validate a DAG batch against the cluster and return
 * the device bytes fate_pack_dags needs for horizon H (0..15).
 * Errors: EINVAL, ERANGE, ECYCLE, ENOFEAS. */
fate_status_t fate_pack_dags_size(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                  int32_t H, size_t *bytes);

/* fate_pack_dags: validate, build the packed image on the host (cluster
 * tables, 32-byte stage records, flat parent lists, and for every stage its
 * horizon descendants: stages at breadth-first distance 1..H, each once at its
 * minimum distance, ordered by (distance, id) - Sec. 3.3), copy it to d_buf
 * on `stream` and synchronise.  `out` receives device pointers into d_buf.
 * Errors: as fate_pack_dags_size, plus ESIZE if bytes is too small, EHIP. */
fate_status_t fate_pack_dags(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, int32_t H,
                             void *d_buf, size_t bytes, void *stream, fate_dags_t *out);

/* fate_layout_dags: the host half of fate_pack_dags, writing the same image
 * into host memory h_buf (no HIP call; `out` points into h_buf). */
fate_status_t fate_layout_dags(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, int32_t H,
                               void *h_buf, size_t bytes, fate_dags_t *out);

/* fate_pack_dags_opt_size / fate_pack_dags_opt / fate_layout_dags_opt: as the
 * three calls above with the options of fate_pack_opts_t (horizon levels,
 * level weights); {H, FATE_LEVELS_HOP, 0} gives the same image.  Descendant
 * lists are ordered by (depth, id) either way.
 * Errors: as above, plus EINVAL for a null or unknown option. */
fate_status_t fate_pack_dags_opt_size(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                      const fate_pack_opts_t *opts, size_t *bytes);
fate_status_t fate_pack_dags_opt(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                 const fate_pack_opts_t *opts, void *d_buf, size_t bytes, void *stream,
                                 fate_dags_t *out);
fate_status_t fate_layout_dags_opt(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                   const fate_pack_opts_t *opts, void *h_buf, size_t bytes, fate_dags_t *out);

/* fate_pack_state_size: validate a state against a packed batch and the same
 * host DAG arrays it was packed from; return the device bytes needed, the
 * number of frontier stages (pending stages whose parents are all completed,
 * App. A.1) and of candidates.  A frontier stage v has D single-device
 * candidates followed by the windows {i..i+k-1}, k = 2..r, i = 0..D-k, with
 * r = min(R(v), max_shard, D) (Sec. 3.3 shard slots).  max_shard in 1..4.
 * Errors: EINVAL, ERANGE, ESTATE. */
fate_status_t fate_pack_state_size(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                   const fate_state_t *state, int32_t max_shard, size_t *bytes,
                                   int64_t *n_frontier, int64_t *n_cand);

/* fate_pack_state: validate, build the frontier list (ordered by instance,
 * then stage id) and candidate offsets, copy state and frontier to d_buf on
 * `stream` and synchronise.  Errors: as the size query, ESIZE, EHIP. */
fate_status_t fate_pack_state(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                              const fate_state_t *state, int32_t max_shard, void *d_buf, size_t bytes,
                              void *stream, fate_state_h *out);

/* fate_layout_state: the host half of fate_pack_state, into host memory. */
fate_status_t fate_layout_state(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                const fate_state_t *state, int32_t max_shard, void *h_buf, size_t bytes,
                                fate_state_h *out);

/* fate_pack_state_advance_size / fate_pack_state_advance: as
 * fate_pack_state_size / fate_pack_state, but the packed state is a planning
 * state that fate_commit_advance can update on the device, step after step:
 * it carries the stage statuses, and its frontier, candidate, slice and
 * completed-parent sections are sized for the largest possible frontier
 * (every stage of the batch).  The handle's n_frontier, n_cand and n_slices
 * are those capacities; the current counts are in the device array
 * `counts` (see fate_state_h).  Scoring and top-k accept such a handle:
 * their outputs are sized by the capacities, and slots past the current
 * counts are left untouched.
 * Errors: as fate_pack_state, plus ERANGE if the candidate capacity
 * reaches 2^32. */
fate_status_t fate_pack_state_advance_size(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                           const fate_state_t *state, int32_t max_shard, size_t *bytes);
fate_status_t fate_pack_state_advance(const fate_dags_t *packed, const fate_dag_batch_t *dags,
                                      const fate_state_t *state, int32_t max_shard, void *d_buf, size_t bytes,
                                      void *stream, fate_state_h *out);

/* fate_commit_ws_size: device workspace bytes fate_commit_advance needs
 * (about 8 bytes per stage).  Errors: EINVAL, ESTATE. */
fate_status_t fate_commit_ws_size(const fate_dags_t *dags, const fate_state_h *state, size_t *bytes);

/* fate_commit_advance: commit one planning step on the device and advance
 * the planning state (Alg. 1: materialise the selected placements, then
 * advance the frontier and update the planning state; Alg. 2: commit into
 * the action pool and update the state as the stages complete).
 *   d_sel[f * sel_stride], f < counts[0]: the candidate chosen for frontier
 *     slot f (the local index fate_topk reports, so a top-k array with
 *     sel_stride = k selects each stage's best candidate), or -1 to leave
 *     the stage pending.  Device memory, read only.
 * Per instance the selected stages are applied in ascending stage id, and on
 * each device d of the chosen candidate S (k = |S|):
 *   start = max(tau_d, t, every parent u's finish(u) + (0 if d holds u's
 *   output, else sigma(u) * min over u's holders i of beta[i][d] / k)), as a
 *   shard starts when its inputs are there; the switch time
 *   kappa_switch(m(v), d) counts if m(v) was not resident; m(v) is loaded
 *   (the smallest-id other models are
 *   evicted while the weights exceed the capacity, as in the post-state of
 *   fate_score_frontier); grp(v), if nonzero and absent, takes the first
 *   empty prefix slot of d or, with all slots full, is appended after
 *   dropping slot 0 (slots are kept oldest first); tau_d = start + c(v,d)/k
 *   + switch.  Then v is completed, its output is held by exactly S, and its
 *   finish is the largest of those tau_d.
 * A selection past the stage's candidates, or whose candidate has a device
 * that is not eligible or cannot hold the model, is skipped and counted in
 * counts[3].  Afterwards the frontier (pending stages whose parents are all
 * completed), its per-instance offsets, the candidate offsets and the
 * workgroup slices are rebuilt on the device, and so are the completed-parent
 * lists of the children of the stages just completed (no other list
 * changes).  t_now is unchanged.
 * `state` must come from fate_pack_state_advance; its buffer is updated in
 * place.  d_ws: at least fate_commit_ws_size bytes.  Enqueued on `stream`;
 * does not synchronise.
 * Errors: EINVAL (null pointers, sel_stride < 1, not a planning state),
 * ESIZE (workspace), ESTATE, EHIP. */
fate_status_t fate_commit_advance(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                                  int32_t sel_stride, void *d_ws, size_t ws_bytes, void *stream);

/* fate_commit_advance_noalloc: fate_commit_advance for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments without the workspace,
 * same kernels and results: the workspace is a library-held device array of
 * FATE_NOALLOC_WS_BYTES on each GPU, kept until the process ends; its
 * address is looked up on the first call on each device, which must be the
 * current device (the stream's device).  The call allocates and frees
 * nothing.  Every call on a GPU shares that GPU's array and leaves its
 * contents behind (nothing in it needs clearing), so calls that overlap on
 * one GPU - concurrent streams, threads or processes sharing the library's
 * copy - race and must be serialised by the caller.
 * Errors: as fate_commit_advance, except ESIZE; ERANGE when the planning
 * state needs more workspace than FATE_NOALLOC_WS_BYTES (fate_commit_ws_size
 * tells how much); EHIP if the array's device address cannot be found. */
fate_status_t fate_commit_advance_noalloc(const fate_dags_t *dags, const fate_state_h *state, const int32_t *d_sel,
                                          int32_t sel_stride, void *stream);

/* fate_score_ws_size: device workspace bytes fate_score_frontier needs
 * (may be 0).  Errors: EINVAL, ESTATE. */
fate_status_t fate_score_ws_size(const fate_dags_t *dags, const fate_state_h *state, size_t *bytes);

/* fate_score_frontier: for every frontier stage v and candidate S write
 *   Psi(v, S) = -( J0(v, S) + sum_{h=1..H} gamma^h sum_{w at distance h} min_{d' feasible for w} c_hat(w, d' | s') )
 * into d_scores[cand_off[f] + j] (float32, device memory, n_scores >= n_cand):
 *   J0(v, S) = max_{d in S} [ lam_q Wait(d) + c(v,d)/k + lam_s Sw(v,d)
 *                              + (lam_tr Tr(v,d) - lam_p Pf(v,d))/k - lam_c Colo(v,d) ]
 *              + lam_tr min_{p in S} sum_{d in S, d != p} beta[d][p] sigma(v)/k,
 * k = |S|; s' is the state after placing v on S (its model loaded on each
 * device of S, evicting the smallest-id other models while over capacity;
 * grp(v) cached there; v's output held by S).  Candidates with a device that
 * is not eligible or cannot hold the model score -infinity.
 * d_ws/ws_bytes: workspace of at least fate_score_ws_size bytes (may be NULL
 * when that size is 0).  Enqueued on `stream`; does not synchronise.
 * Errors: EINVAL (null, non-finite or negative weights, H out of range),
 * ESIZE, ESTATE (handles from different batches), EHIP. */
fate_status_t fate_score_frontier(const fate_dags_t *dags, const fate_state_h *state,
                                  const fate_params_t *params, float *d_scores, int64_t n_scores,
                                  void *d_ws, size_t ws_bytes, void *stream);

/* fate_score_topk: fate_score_frontier and fate_topk in one launch.  Writes
 * the same scores to d_scores and the same per-stage top-k to d_idx / d_val
 * ([n_frontier * k]) as the two calls in sequence would.
 * Errors: those of fate_score_frontier, plus ERANGE (k outside 1..64). */
fate_status_t fate_score_topk(const fate_dags_t *dags, const fate_state_h *state, const fate_params_t *params,
                              float *d_scores, int64_t n_scores, int32_t k, int32_t *d_idx, float *d_val,
                              void *d_ws, size_t ws_bytes, void *stream);

/* fate_topk: per frontier stage, the k (1..64) best candidates by
 * (score descending, candidate index ascending), skipping -infinity, padded
 * with (-1, -infinity).  d_idx/d_val: device arrays [n_frontier * k] of
 * local candidate indices and scores.  Enqueued on `stream`.
 * Errors: EINVAL, ERANGE (k), ESIZE (n_scores < n_cand), EHIP. */
fate_status_t fate_topk(const fate_state_h *state, const float *d_scores, int64_t n_scores, int32_t k,
                        int32_t *d_idx, float *d_val, void *stream);

/* fate_score_sweep: fate_score_frontier for n_sets (1..FATE_MAX_SWEEP)
 * parameter sets in one launch - the weight, horizon and variant grids of the
 * paper's ablations (App. C.3) and sensitivity study (App. D.4, Tab. 6) over
 * one packed state.  params[p] (host memory) scores into
 * d_scores + p * score_stride; score_stride >= n_cand, and d_scores holds
 * n_scores >= score_stride * (n_sets - 1) + n_cand floats.  Set p writes
 * exactly what fate_score_frontier with params[p] writes.
 * Errors: those of fate_score_frontier, plus ERANGE (n_sets), ESIZE (stride). */
fate_status_t fate_score_sweep(const fate_dags_t *dags, const fate_state_h *state, const fate_params_t *params,
                               int32_t n_sets, float *d_scores, int64_t n_scores, int64_t score_stride,
                               void *d_ws, size_t ws_bytes, void *stream);

/* fate_topk_sweep: fate_topk for n_sets score arrays at d_scores +
 * p * score_stride (the layout fate_score_sweep writes); set p's top-k goes to
 * d_idx / d_val + p * n_frontier * k (n_frontier of the handle: for a
 * planning state, its capacity).  One launch.
 * Errors: those of fate_topk, plus ERANGE (n_sets), ESIZE (stride). */
fate_status_t fate_topk_sweep(const fate_state_h *state, const float *d_scores, int64_t n_scores,
                              int64_t score_stride, int32_t n_sets, int32_t k, int32_t *d_idx, float *d_val,
                              void *stream);

/* fate_plan_wave: one frontier planning wave per instance on the device (the
 * planner step of Alg. 1 under the wave constraints of App. A.2: each device
 * takes at most one shard-slot assignment per wave, each stage at most one
 * placement; a window candidate is the stage's slots 0..k-1 on k devices,
 * so slots are enabled in order).  The choices of frontier slot f are
 * d_idx[f * k + r], r < k, with scores d_val[f * k + r] - the layout fate_topk
 * writes (device memory).  Greedy: the best remaining choice whose stage is
 * unassigned and whose devices are all free in this wave is taken (ties: the
 * lower frontier slot, then the lower rank), until none is left; choices of
 * -1, -infinity or an index past the stage's candidates are never taken.
 * d_sel[n_frontier] (device) receives each slot's chosen candidate or -1 (not
 * placed in this wave) - the selection fate_commit_advance takes with
 * sel_stride 1.  For a planning state the current frontier size is read on
 * the device.  Enqueued on `stream`.
 * Errors: EINVAL (null pointers), ERANGE (k outside 1..64, n_frontier * k
 * >= 2^32), EHIP. */
fate_status_t fate_plan_wave(const fate_state_h *state, const int32_t *d_idx, const float *d_val, int32_t k,
                             int32_t *d_sel, void *stream);

/* Plan execution (host memory, no device work).  Per instance:
 *   tasks       stages executed (the placed pending stages)
 *   makespan    latest finish - t_now, seconds
 *   p95         nearest-rank 95th percentile of finish - t_now over the
 *               executed stages without children
 *   xdev_edges  parent edges u -> v with v on no device holding u's output
 *   cache_hits  executed stages whose first device had grp(v) cached
 *   model_cont  executed stages whose first device ran the same model just
 *               before them
 * (App. C.2 makespan, p95 latency and mechanism proxies; normalising by the
 * task count or by a baseline is left to the caller.) */
typedef struct {
    int64_t tasks;
    double makespan, p95;
    int64_t xdev_edges, cache_hits, model_cont;
} fate_sim_metrics_t;

/* fate_simulate: execute a placement on every instance.  devices[N]: S(v)
 * as a device bitmask for each pending stage to run (0 = not run);
 * order[N]: each device runs its stages by (order, stage id).  A shard of v
 * on d, k = |S(v)|, starts when d is free and every parent's output has
 * arrived (finish(u) + sigma(u) * min over u's holders i of beta[i][d] / k,
 * or finish(u) when d holds it); it pays kappa_switch(m(v), d) if m(v) is not
 * resident (then m(v) is loaded with the eviction rule of scoring), and runs
 * c(v, d) / k, less kappa_prefix * L(v) / k (not below 0) when grp(v) is in
 * d's prefix slots; grp(v) then joins the slots (oldest dropped when full).
 * v finishes with its last shard; its output is then held by S(v).  The
 * state's statuses must be pending or completed (completed stages are
 * available at t_now on their holders).  Host memory; out[B].
 * Errors: EINVAL, ERANGE, ECYCLE, ENOFEAS (as packing), ESTATE (a status
 * other than pending / completed, holders inconsistent, or an order that runs
 * a stage before a parent that is not completed or run earlier). */
fate_status_t fate_simulate(const fate_cluster_t *cluster, const fate_dag_batch_t *dags, const fate_state_t *state,
                            const uint64_t *devices, const int64_t *order, float kappa_prefix,
                            fate_sim_metrics_t *out);

/* Baseline placements for fate_simulate (App. B comparison schedulers). */
enum { FATE_PLACE_ROUND_ROBIN = 0, FATE_PLACE_HEFT = 1 };

/* fate_place_baseline: FATE_PLACE_ROUND_ROBIN puts each pending stage, in id
 * order, on the next feasible device after the previous placement;
 * FATE_PLACE_HEFT orders pending stages by upward rank (mean runtime over
 * feasible devices plus the largest sigma * mean off-diagonal beta + rank over
 * its children; ties to the lower id) and gives each the feasible device with
 * the earliest finish under fate_simulate's rule (ties to the lower device).
 * Writes devices[N] and order[N] (host memory; 0 for completed stages).
 * Errors: EINVAL (policy, pointers), and those of fate_simulate's inputs. */
fate_status_t fate_place_baseline(const fate_cluster_t *cluster, const fate_dag_batch_t *dags,
                                  const fate_state_t *state, int32_t policy, float kappa_prefix, uint64_t *devices,
                                  int64_t *order);

/* Plan execution and baseline placements on the device (App. C.2 metrics,
 * App. B baselines): the rules of fate_simulate and fate_place_baseline,
 * computed in fp64 by one 64-lane wave per instance, on the packed DAGs and
 * a packed state instead of host arrays.  A stage is completed when its
 * holders in the packed state are non-zero, pending otherwise (so running and
 * committed stages count as pending).
 *
 * fate_sim_ws_size: bytes of device workspace the two calls below need
 * (about 50 bytes per stage of the batch).  Errors: EINVAL. */
fate_status_t fate_sim_ws_size(const fate_dags_t *dags, size_t *bytes);

/* fate_simulate_device: fate_simulate for d_devices[N] / d_order[N] (device
 * arrays, flat stage ids) from the packed state; writes d_out[B]
 * (fate_sim_metrics_t) and d_status[B] (device memory), and is enqueued on
 * `stream`.  Errors found in the device arrays are reported per instance in
 * d_status (FATE_OK, FATE_EINVAL for a device bit >= D, FATE_ESTATE for an
 * order that runs a placed stage before a parent that is neither completed
 * nor run earlier); such an instance's metrics are all zero.  The times
 * equal fate_simulate's bit for bit (the same fp64 operations in the same
 * order); d_ws is caller memory of fate_sim_ws_size bytes, overwritten.
 * Errors: EINVAL (null pointers, kappa_prefix negative or not finite),
 * ESTATE (handles of different batches), ESIZE (workspace), EHIP. */
fate_status_t fate_simulate_device(const fate_dags_t *dags, const fate_state_h *state, const uint64_t *d_devices,
                                   const int64_t *d_order, float kappa_prefix, fate_sim_metrics_t *d_out,
                                   int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream);

/* fate_place_baseline_device: fate_place_baseline on the device; writes
 * d_devices[N] and d_order[N] (0 for completed stages) and d_status[B]
 * (FATE_OK, or FATE_ESTATE if a stage's parent would run after it).
 * Errors: as fate_simulate_device, plus EINVAL for an unknown policy. */
fate_status_t fate_place_baseline_device(const fate_dags_t *dags, const fate_state_h *state, int32_t policy,
                                         float kappa_prefix, uint64_t *d_devices, int64_t *d_order,
                                         int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* FATE_H */
