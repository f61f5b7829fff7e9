"""Hand-derived micro scenarios that pin each term of the score.

Every expected value below was worked out by hand from the definitions the
paper gives (App. A.3 term definitions, App. A.1/A.4 additive estimator,
Sec. 3.3 horizon) under the readings recorded in the design notes.  Inputs are
exact binary fractions (powers of two for transfer coefficients and sizes,
lam_c = 1/8, kappa_prefix = 2^-10) so every expected value is exact in fp64
(the only exception is k = 3 windows, which divide by 3).

Each scenario is chosen so that a plausible slip (dropped term, wrong sign,
transposed transfer coefficient, wrong divisor, wrong eviction order, wrong
depth weight, missing de-duplication, ...) changes at least one number.

Where a scenario lists ``mag``, those are the hand-derived magnitudes A that
the parity tolerance divides by: the absolute values of the weighted terms
of the device that sets the immediate cost (the maximising shard device,
plus the gather term), plus gamma^depth times the absolute terms of the
device that gives each horizon stage its value (the minimising device).
A equals |Psi| when no benefit term (colocation, prefix, same model) enters.
"""

from __future__ import annotations

INF = float("inf")
P = dict(lam_c=0.125, kappa_prefix=2.0 ** -10)

# A: waiting cost is clamped at zero; switch only when the model is absent.
#   d0: wait max(0, 0.25-1) = 0, exec 1.0, m0 resident            -> 1.0
#   d1: wait 2-1 = 1, exec 0.5, switch 0.75                         -> 2.25
#   A: every term is a cost, so A = |Psi| = 1.0, 2.25.
WAIT_SWITCH = dict(
    spec=dict(D=2, M=1, K=1, exec=[[1.0, 0.5]], switch_s=[[0.75, 0.75]], weight_gb=[10], cap_gb=[20, 20],
              beta=[[0, 0], [0, 0]],
              instances=[dict(parents=[[]], model=[0], elig=[3], out_bytes=[1.0], status=[0], holders=[0],
                              resident=[1, 0], tau_free=[0.25, 2.0], t_now=1.0)]),
    H=0, params=P, front_v=[0], psi=[-1.0, -2.25], mag=[1.0, 2.25])

# B: transfer uses beta[from][to], the cheapest of several holders, and
#    colocation counts the fraction of parents held on the device.
#   u0 on {d0}, sigma 2^32; u1 on {d1,d2}, sigma 2^30; lam_c = 1/8.
#   d0: u1 -> 2^30 * min(beta[1][0]=2^-30, beta[2][0]=2^-31) = 0.5; colo 1/2
#       J0 = 1 + 0.5 - 1/16 = 1.4375
#   d1: u0 -> 2^32 * beta[0][1] (2^-32) = 1.0; colo 1/2  -> 1.9375
#   d2: u0 -> 2^32 * beta[0][2] (2^-31) = 2.0; colo 1/2  -> 2.9375
#   A adds the colocation benefit 1/16 instead of taking it off:
#   1 + 0.5 + 1/16 = 1.5625, 1 + 1 + 1/16 = 2.0625, 1 + 2 + 1/16 = 3.0625.
_B_BETA = [[0.0, 2.0 ** -32, 2.0 ** -31],
           [2.0 ** -30, 0.0, 2.0 ** -33],
           [2.0 ** -31, 2.0 ** -34, 0.0]]
TRANSFER_COLO = dict(
    spec=dict(D=3, M=1, K=1, exec=[[1.0, 1.0, 1.0]], switch_s=[[0.0, 0.0, 0.0]], weight_gb=[10],
              cap_gb=[20, 20, 20], beta=_B_BETA,
              instances=[dict(parents=[[], [], [0, 1]], model=[0, 0, 0], elig=[7, 7, 7],
                              out_bytes=[2.0 ** 32, 2.0 ** 30, 1.0], status=[1, 1, 0], holders=[1, 6, 0],
                              resident=[1, 1, 1], tau_free=[0.0, 0.0, 0.0], t_now=0.0)]),
    H=0, params=P, front_v=[2], psi=[-1.4375, -1.9375, -2.9375], mag=[1.5625, 2.0625, 3.0625])

# C: shard windows.  Per device (wait, exec, switch, transfer, colo, prefix):
#   d0: (2.0, 1.0, 0,   0,   1, 0)    d1: (0, 2.0, 0.5, 0.5, 0, 0)
#   d2: (0,   4.0, 0.5, 1.0, 0, 0.5)  with sigma(v) = 3*2^31.
#   T(d,k) = wait + exec/k + switch + (transfer - prefix)/k - colo/8.
#   k=1: T = 2.875, 3.0, 5.0
#   {0,1}: max(2.375, 1.75) + G; G = min(beta[1][0], beta[0][1])*sigma/2 = 0.375 -> 2.75
#   {1,2}: max(1.75, 2.75) + G; G = min(beta[2][1], beta[1][2])*sigma/2 = 0.1875 -> 2.9375
#   {0,1,2}: max(2 + 1/3 - 1/8, 2/3 + 1/2 + 1/6, 4/3 + 1/2 + 1/6) + G
#            G = min over p of the column sum into p times sigma/3
#              = min(1.25, 0.75, 0.625) = 0.625               -> 2.833333...
#   A, from the device that sets the maximum, plus the gather term:
#   k=1: d0 2 + 1 + 1/8 = 3.125; d1 3.0; d2 4 + 0.5 + 1 + 0.5 = 6.0
#   {0,1}: d0 (2.375 > 1.75): 2 + 0.5 + 1/8 = 2.625, + 0.375 = 3.0
#   {1,2}: d2 (2.75 > 1.75): 2 + 0.5 + 0.5 + 0.25 = 3.25, + 0.1875 = 3.4375
#   {0,1,2}: d0 (2.2083 > 2.0 > 1.3333): 2 + 1/3 + 1/8, + 0.625 = 3 + 1/12
_C_BETA = [[0.0, 2.0 ** -33, 2.0 ** -32],
           [2.0 ** -31, 0.0, 2.0 ** -34],
           [2.0 ** -33, 2.0 ** -32, 0.0]]
WINDOWS = dict(
    spec=dict(D=3, M=1, K=1, exec=[[1.0, 2.0, 4.0]], switch_s=[[0.5, 0.5, 0.5]], weight_gb=[10],
              cap_gb=[20, 20, 20], beta=_C_BETA,
              instances=[dict(parents=[[], [0]], model=[0, 0], elig=[7, 7], shard_max=[1, 3],
                              prefix_hash=[0, 7], prefix_tokens=[0.0, 512.0],
                              out_bytes=[2.0 ** 32, 3.0 * 2.0 ** 31], status=[1, 0], holders=[1, 0],
                              resident=[1, 0, 0], prefix_cache=[[0], [0], [7]],
                              tau_free=[3.0, 1.0, 1.0], t_now=1.0)]),
    H=0, params=P, front_v=[1],
    psi=[-2.875, -3.0, -5.0, -2.75, -2.9375, -(2.0 + 1.0 / 3.0 - 0.125 + 0.625)],
    mag=[3.125, 3.0, 6.0, 3.0, 3.4375, 2.0 + 1.0 / 3.0 + 0.125 + 0.625],
    topk3=[3, 5, 0])

# D: post-state seen by the descendants.
#   Models W = 10 GB each, capacity 25 GB; switch m0 0.25, m1 0.5, m2 1.0.
#   p (m0) completed on d1; v (m1, group 99, sigma 2^32) is the frontier stage;
#   q is running; w1 (m0, group 99, L 512, parents v and q); w2 (m2, parent v,
#   no prefix group, so its 256 tokens never count).
#   Immediate: d0 = 1 + 0.5 (switch) + 0.5 (p's output, 2^31*2^-32) = 2.0;
#              d1 = 1 + 0.5 - 1/8 (p colocated) = 1.375.
#   v on d0: loading m1 onto {m0,m2} overflows (30 > 25) and evicts m0.
#     w1: d0 = 1 + 0.25 - 1/16 - 0.5 = 0.6875; d1 = 1 + 0.25 + 1.0 = 2.25
#     w2: d0 = 1 - 1/8 = 0.875;              d1 = 1 + 1.0 = 2.0
#     J = 2.0 + 0.5 (0.6875 + 0.875) = 2.78125
#   v on d1: {m2} + m1 fits, nothing evicted.
#     w1: d0 = 1 + 1.0 = 2.0; d1 = 1 + 0.25 - 1/16 - 0.5 = 0.6875
#     w2: d0 = 1 + 1.0 = 2.0; d1 = 1 - 1/8 = 0.875
#     J = 1.375 + 0.78125 = 2.15625
#   A: immediate d0 1 + 0.5 + 0.5 = 2.0 (no benefit); d1 1 + 0.5 + 1/8 = 1.625.
#     Horizon (same minimising devices as above, each term's absolute value):
#     w1 1 + 0.25 + 1/16 + 0.5 = 1.8125, w2 1 + 1/8 = 1.125, times 0.5: 1.46875.
#     A = 3.46875 (v on d0), 3.09375 (v on d1); at H = 0: 2.0, 1.625.
_UNI = [[0.0, 2.0 ** -32], [2.0 ** -32, 0.0]]
POST_STATE = dict(
    spec=dict(D=2, M=3, K=1, exec=[[1.0, 1.0]] * 3, switch_s=[[0.25, 0.25], [0.5, 0.5], [1.0, 1.0]],
              weight_gb=[10, 10, 10], cap_gb=[25, 25], beta=_UNI,
              instances=[dict(parents=[[], [0], [], [1, 2], [1]], model=[0, 1, 0, 0, 2], elig=[3] * 5,
                              prefix_hash=[0, 99, 0, 99, 0], prefix_tokens=[0.0, 256.0, 0.0, 512.0, 256.0],
                              out_bytes=[2.0 ** 31, 2.0 ** 32, 1.0, 1.0, 1.0],
                              status=[1, 0, 2, 0, 0], holders=[2, 0, 0, 0, 0],
                              resident=[5, 4], prefix_cache=[[0], [0]],
                              tau_free=[1.0, 1.0], t_now=1.0)]),
    H=1, params=P, front_v=[1], psi=[-2.78125, -2.15625], mag=[3.46875, 3.09375])
POST_STATE_H0 = dict(POST_STATE, H=0, psi=[-2.0, -1.375], mag=[2.0, 1.625])

# E: horizon set = breadth-first levels 1..H, each stage once at its minimum
#    distance; descendants use only their feasible devices.  Only base
#    runtimes are non-zero (exec d0 = 1, d1 = 2; c is eligible on d1 only).
#    Levels from v: {a, b, f} at 1, {c} at 2, {e} at 3 (f is also a child of c).
#    H=2: J(d0) = 1 + 0.5*3 + 0.25*2 = 3.0; J(d1) = 4.0
#    H=3: plus 0.125*1 for e.
#    Only costs enter, so A = |Psi|.
_E_P = dict(lam_c=0.0, kappa_prefix=0.0)
HORIZON_SET = dict(
    spec=dict(D=2, M=1, K=1, exec=[[1.0, 2.0]], switch_s=[[0.0, 0.0]], weight_gb=[10], cap_gb=[20, 20],
              beta=[[0, 0], [0, 0]],
              instances=[dict(parents=[[], [0], [1], [1], [2, 3], [4], [1, 4]], model=[0] * 7,
                              elig=[3, 3, 3, 3, 2, 3, 3], out_bytes=[1.0] * 7,
                              status=[1, 0, 0, 0, 0, 0, 0], holders=[1, 0, 0, 0, 0, 0, 0],
                              resident=[1, 1], tau_free=[0.0, 0.0], t_now=0.0)]),
    H=2, params=_E_P, front_v=[1], psi=[-3.0, -4.0], mag=[3.0, 4.0])
HORIZON_SET_H3 = dict(HORIZON_SET, H=3, psi=[-3.125, -4.125], mag=[3.125, 4.125])

# F: feasibility needs eligibility and capacity; top-k skips -inf, breaks
#    ties by candidate index and pads with (-1, -inf).
#    v0 (m1, 30 GB) does not fit d0 (20 GB); v1 (m0) is eligible on d0, d2.
FEASIBILITY = dict(
    spec=dict(D=3, M=2, K=1, exec=[[1.0, 1.0, 1.0], [1.0, 1.0, 1.0]], switch_s=[[0.0] * 3, [0.0] * 3],
              weight_gb=[10, 30], cap_gb=[20, 40, 40], beta=[[0.0] * 3] * 3,
              instances=[dict(parents=[[], []], model=[1, 0], elig=[7, 5], shard_max=[1, 2],
                              out_bytes=[1.0, 1.0], status=[0, 0], holders=[0, 0],
                              resident=[1, 3, 3], tau_free=[0.0] * 3, t_now=0.0)]),
    H=0, params=P, front_v=[0, 1],
    psi=[-INF, -1.0, -1.0, -1.0, -INF, -1.0, -INF, -INF],
    topk4=[[1, 2, -1, -1], [0, 2, -1, -1]])

# G: the frontier holds pending stages whose parents are all completed;
#    running and committed stages are not in it.
FRONTIER = dict(
    spec=dict(D=2, M=1, K=1, exec=[[1.0, 1.0]], switch_s=[[0.0, 0.0]], weight_gb=[10], cap_gb=[20, 20],
              beta=[[0, 0], [0, 0]],
              instances=[dict(parents=[[], [], [], [0], [1], [], [0, 3]], model=[0] * 7, elig=[3] * 7,
                              out_bytes=[1.0] * 7, status=[1, 2, 3, 0, 0, 0, 0],
                              holders=[1, 0, 0, 0, 0, 0, 0], resident=[1, 1],
                              tau_free=[0.0, 0.0], t_now=0.0)]),
    H=0, params=P, front_v=[3, 5], psi=[-(1.0 - 0.125), -1.0, -1.0, -1.0])

ALL = dict(WAIT_SWITCH=WAIT_SWITCH, TRANSFER_COLO=TRANSFER_COLO, WINDOWS=WINDOWS, POST_STATE=POST_STATE,
           POST_STATE_H0=POST_STATE_H0, HORIZON_SET=HORIZON_SET, HORIZON_SET_H3=HORIZON_SET_H3,
           FEASIBILITY=FEASIBILITY, FRONTIER=FRONTIER)


# ---------------------------------------------------------------------------
# Commit-and-advance (oracle step 11).  Each scenario lists the selection per
# frontier slot and the hand-derived state after the commit.
# ---------------------------------------------------------------------------

# C1: one device each.  v1 (model 2) on d0: start = max(1.0, t=1.5) = 1.5;
#     model 2 absent -> switch 0.5; Load adds 2 (30 GB > 25 GB) and evicts
#     the smallest other id, model 0; grp 99 takes the empty slot 1;
#     tau0 = 1.5 + 0.75 + 0.5 = 2.75.  v4 (model 1) on d1: start 1.5, switch
#     0.5, Load adds 1 (20 GB fits); grp 7 already cached; tau1 = 1.5 + 1.0 +
#     0.5 = 3.0.  Next frontier: v2 (parent v1) and v3 (parents v0, v1).
COMMIT_SINGLE = dict(
    spec=dict(D=2, M=3, K=2, exec=[[0.5, 0.5], [1.0, 1.0], [0.75, 1.25]],
              switch_s=[[0.25, 0.25], [0.5, 0.5], [0.5, 1.0]], weight_gb=[10, 10, 10], cap_gb=[25, 25],
              beta=_UNI,
              instances=[dict(parents=[[], [0], [1], [0, 1], []], model=[0, 2, 1, 0, 1], elig=[3] * 5,
                              prefix_hash=[0, 99, 99, 0, 7], prefix_tokens=[0.0] * 5, out_bytes=[1.0] * 5,
                              status=[1, 0, 0, 0, 0], holders=[1, 0, 0, 0, 0],
                              resident=[3, 4], prefix_cache=[[5, 0], [7, 8]],
                              tau_free=[1.0, 0.5], t_now=1.5)]),
    front_v=[1, 4], sel=[0, 1],
    resident=[6, 6], prefix_cache=[[5, 99], [7, 8]], tau=[2.75, 3.0],
    holders=[1, 1, 0, 0, 2], status=[1, 1, 0, 0, 1], next_front_v=[2, 3], rejected=0)

# C2: a window and a second stage on a shared device.  v0 (model 0, R = 2)
#     on the window {d0, d1} (candidate D + 0): d0 start 2.0, model resident,
#     full prefix slots [3, 4] drop the oldest -> [4, 99], tau0 = 2.0 + 1/2;
#     d1 start max(0, 1) = 1.0, switch 0.25, empty slots -> [99, 0],
#     tau1 = 1.0 + 3/2 + 0.25 = 2.75; holders 0b11.  Then v1 (model 1) on d0:
#     start 2.5, switch 1.0, Load adds 1 (fits), grp 0 inserts nothing,
#     tau0 = 2.5 + 0.5 + 1.0 = 4.0.  Next frontier: v2.
COMMIT_WINDOW = dict(
    spec=dict(D=2, M=2, K=2, exec=[[1.0, 3.0], [0.5, 0.5]], switch_s=[[0.25, 0.25], [1.0, 1.0]],
              weight_gb=[10, 10], cap_gb=[25, 25], beta=_UNI, max_shard=2,
              instances=[dict(parents=[[], [], [0]], model=[0, 1, 0], elig=[3] * 3, shard_max=[2, 1, 1],
                              prefix_hash=[99, 0, 0], prefix_tokens=[0.0] * 3, out_bytes=[1.0] * 3,
                              status=[0, 0, 0], holders=[0, 0, 0],
                              resident=[1, 0], prefix_cache=[[3, 4], [0, 0]],
                              tau_free=[2.0, 0.0], t_now=1.0)]),
    front_v=[0, 1], sel=[2, 0],
    resident=[3, 1], prefix_cache=[[4, 99], [99, 0]], tau=[4.0, 2.75],
    holders=[3, 1, 0], status=[1, 1, 0], next_front_v=[2], rejected=0)

# C3: rejected selections leave the state unchanged: an index past the
#     candidates, and a window over a device where v is not eligible.
COMMIT_REJECT = dict(
    spec=dict(D=2, M=1, K=1, exec=[[1.0, 1.0]], switch_s=[[0.5, 0.5]], weight_gb=[10], cap_gb=[20, 20],
              beta=_UNI, max_shard=2,
              instances=[dict(parents=[[], []], model=[0, 0], elig=[3, 1], shard_max=[1, 2],
                              prefix_hash=[11, 12], prefix_tokens=[0.0, 0.0], out_bytes=[1.0, 1.0],
                              status=[0, 0], holders=[0, 0], resident=[0, 0], prefix_cache=[[0], [0]],
                              tau_free=[0.0, 0.0], t_now=0.0)]),
    front_v=[0, 1], sel=[5, 2],
    resident=[0, 0], prefix_cache=[[0], [0]], tau=[0.0, 0.0],
    holders=[0, 0], status=[0, 0], next_front_v=[0, 1], rejected=2)

# C4: a shard waits for its inputs.  Stage 0 is completed on d0 (2^31 bytes,
#     available at t = 1); beta = 2^-32 between the two devices; every
#     runtime is 1, the model is resident everywhere, tau = [0.5, 0.5].
#   Step 1: stage 1 on the window {d0, d1} (k = 2): d0 holds stage 0's output:
#     start max(0.5, 1, 1) = 1, tau0 = 1 + 1/2 = 1.5; d1 waits for half of it:
#     1 + 2^31 * 2^-32 / 2 = 1.25, tau1 = 1.25 + 0.5 = 1.75; fin(1) = 1.75.
#     Stage 2 on d1: all of stage 0's output, 1 + 0.5 = 1.5, but d1 is busy
#     until 1.75: tau1 = 2.75 = fin(2).
#   Step 2: stage 3 (parents 1 and 2) on d0: stage 1 is local (1.75); stage
#     2's 2^32 bytes arrive at 2.75 + 1 = 3.75: tau0 = 4.75 = fin(3).
COMMIT_READY = dict(
    spec=dict(D=2, M=1, K=1, exec=[[1.0, 1.0]], switch_s=[[0.0, 0.0]], weight_gb=[10], cap_gb=[25, 25],
              beta=[[1.0, 2.0 ** -32], [2.0 ** -32, 1.0]], max_shard=2,  # the diagonal is never used
              instances=[dict(parents=[[], [0], [0], [1, 2]], model=[0] * 4, elig=[3] * 4, shard_max=[1, 2, 1, 1],
                              out_bytes=[2.0 ** 31, 1.0, 2.0 ** 32, 1.0], status=[1, 0, 0, 0],
                              holders=[1, 0, 0, 0], resident=[1, 1], tau_free=[0.5, 0.5], t_now=1.0)]),
    steps=[dict(front_v=[1, 2], sel=[2, 1], tau=[1.5, 2.75], fin=[1.0, 1.75, 2.75, 0.0]),
           dict(front_v=[3], sel=[0], tau=[4.75, 2.75], fin=[1.0, 1.75, 2.75, 4.75])])

COMMITS = dict(COMMIT_SINGLE=COMMIT_SINGLE, COMMIT_WINDOW=COMMIT_WINDOW, COMMIT_REJECT=COMMIT_REJECT)


# ---------------------------------------------------------------------------
# Scoring variants (oracle V1-V4), each on an input of a scenario above.
# ---------------------------------------------------------------------------

# V1 same-model weight lam_m = 1/4, beside the switch cost.
#   WAIT_SWITCH: d0 holds m0 -> 1.0 - 0.25; d1 does not -> 2.25 unchanged.
_SM = dict(P, lam_m=0.25)
SM_IMMEDIATE = dict(WAIT_SWITCH, params=_SM, psi=[-0.75, -2.25])
#   WINDOWS (d0 holds m0, so only T(d0) drops by 1/4, inside the max):
#   k=1: 2.625, 3.0, 5.0; {0,1}: max(2.125, 1.75) + 0.375 = 2.5;
#   {1,2}: 2.9375; {0,1,2}: max(2 + 1/3 - 1/8 - 1/4, 4/3, 4/3 + 1/2 + 1/6) + 0.625
#   = 2.0 + 0.625 (d2 is now the slowest shard).
SM_WINDOWS = dict(WINDOWS, params=_SM, psi=[-2.625, -3.0, -5.0, -2.5, -2.9375, -(4.0 / 3.0 + 2.0 / 3.0 + 0.625)])
SM_WINDOWS.pop("topk3")
#   POST_STATE: m1 (v's model) is resident nowhere, so the immediate costs
#   stay 2.0 / 1.375; the descendants see s':
#   v on d0 -> d0 {m1, m2}, d1 {m2}: w1 (m0) 0.6875 / 2.25 (no bonus: m0 was
#     evicted from d0); w2 (m2) 0.875 - 0.25 / 2.0 - 0.25 -> 0.625.
#     J = 2.0 + 0.5 (0.6875 + 0.625) = 2.65625
#   v on d1 -> d0 {m0, m2}, d1 {m1, m2}: w1 2.0 - 0.25 / 0.6875; w2 2.0 - 0.25 /
#     0.875 - 0.25 -> 0.625.  J = 1.375 + 0.5 (0.6875 + 0.625) = 2.03125
SM_POST_STATE = dict(POST_STATE, params=_SM, psi=[-2.65625, -2.03125])

# V2 / V3 on the horizon scenario with f (stage 6) eligible on d1 only.
#   Hop distances from v: {2, 3, 6} at 1, {4} at 2, {5} at 3.
#   Topological levels: 0,1,2,2,3,4,4 -> from v: {2, 3} at 1, {4} at 2,
#   {5, 6} at 3 (6 has parents 1 and 4, so its level is 1 + 3).
#   Best runtimes: 2, 3, 5 -> 1 (d0); 4, 6 -> 2 (d1 only).
_HV_SPEC = dict(HORIZON_SET["spec"])
_HV_SPEC["instances"] = [dict(HORIZON_SET["spec"]["instances"][0], elig=[3, 3, 3, 3, 2, 3, 2])]
#   hop, sum:  tail = 0.5 (1 + 1 + 2) + 0.25 * 2 + 0.125 * 1 = 2.625
HV_HOP_SUM = dict(HORIZON_SET, spec=_HV_SPEC, H=3, psi=[-3.625, -4.625])
#   hop, mean: tail = 0.5 * 4/3 + 0.25 * 2 + 0.125 * 1 = 2/3 + 0.625
HV_HOP_MEAN = dict(HV_HOP_SUM, params=dict(_E_P, mean_levels=1),
                   psi=[-(1.0 + 2.0 / 3.0 + 0.625), -(2.0 + 2.0 / 3.0 + 0.625)])
#   topological, sum: tail = 0.5 (1 + 1) + 0.25 * 2 + 0.125 (1 + 2) = 1.875
HV_TOPO_SUM = dict(HV_HOP_SUM, params=dict(_E_P, topo_levels=1), psi=[-2.875, -3.875])
#   topological, H = 2: {5, 6} drop out -> tail = 1.5
HV_TOPO_SUM_H2 = dict(HV_TOPO_SUM, H=2, psi=[-2.5, -3.5])
#   topological, mean: tail = 0.5 * 1 + 0.25 * 2 + 0.125 * 1.5 = 1.1875
HV_TOPO_MEAN = dict(HV_HOP_SUM, params=dict(_E_P, topo_levels=1, mean_levels=1), psi=[-2.1875, -3.1875])

# V4 no windows: WINDOWS keeps its six slots, the three windows at -inf.
NO_WINDOWS = dict(WINDOWS, params=dict(P, no_windows=1), psi=[-2.875, -3.0, -5.0, -INF, -INF, -INF],
                  topk3=[0, 1, 2])

VARIANTS = dict(SM_IMMEDIATE=SM_IMMEDIATE, SM_WINDOWS=SM_WINDOWS, SM_POST_STATE=SM_POST_STATE,
                HV_HOP_SUM=HV_HOP_SUM, HV_HOP_MEAN=HV_HOP_MEAN, HV_TOPO_SUM=HV_TOPO_SUM,
                HV_TOPO_SUM_H2=HV_TOPO_SUM_H2, HV_TOPO_MEAN=HV_TOPO_MEAN, NO_WINDOWS=NO_WINDOWS)


# ---------------------------------------------------------------------------
# Frontier planning wave (oracle step 12).  Choices per frontier slot as
# (local candidate index, score); D devices per instance.
# ---------------------------------------------------------------------------

# W1: with D = 3, candidate 3 is the window {0, 1}.  Round 1 takes slot 0's
#     window (-1.0, the best score).  Round 2: slot 1 has {1} (used) or {2}
#     at -2.0; slot 2 has {2} at -1.2 or {0} (used).  It takes slot 2's {2}.
#     Every device is then used, so slot 1 waits for the next wave.
PLAN_WINDOW = dict(D=3, f_off=[0, 3], n_cand=[5, 5, 5], idx=[[3, 0], [1, 2], [2, 0]],
                   val=[[-1.0, -1.5], [-1.2, -2.0], [-1.2, -3.0]], sel=[3, -1, 2])
# W2: ties go to the lower frontier slot; -inf, padded and past-the-end
#     choices are never taken (slot 3's best, index 4, is past its 2
#     candidates); instances plan independently (both use device 0).
INF_ = float("inf")
PLAN_TIES = dict(D=2, f_off=[0, 2, 4], n_cand=[3, 3, 2, 2], idx=[[0, 1], [0, 1], [1, -1], [4, 0]],
                 val=[[-1.0, -2.0], [-1.0, -2.0], [-INF_, -INF_], [-0.5, -5.0]], sel=[0, 1, -1, 0])
# W3: a higher score on a later rank beats an earlier rank; a stage takes at
#     most one choice even when its devices are free.
PLAN_RANKS = dict(D=4, f_off=[0, 2], n_cand=[4, 4], idx=[[0, 1], [2, 3]], val=[[-3.0, -3.0], [-1.0, -0.5]],
                  sel=[0, 3])

# W4: -0 and +0 are the same score, so the lower slot wins the tie.
PLAN_SIGNED_ZERO = dict(D=1, f_off=[0, 2], n_cand=[1, 1], idx=[[0], [0]], val=[[-0.0], [0.0]], sel=[0, -1])

PLANS = dict(PLAN_WINDOW=PLAN_WINDOW, PLAN_TIES=PLAN_TIES, PLAN_RANKS=PLAN_RANKS, PLAN_SIGNED_ZERO=PLAN_SIGNED_ZERO)
