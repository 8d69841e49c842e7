/*
 * wf_plan.h -- C ABI of the MI355X (gfx950) candidate-plan scorer.
 *
 * The paper's scheduler (Sec. 3.5, Algorithm 1) ranks candidate physical
 * execution plans of a planning window by their predicted consequences on one
 * shared timeline; its Propagate step serialises co-located operations and
 * checks Eq. 9-11.  This library evaluates that forecast for a whole batch of
 * candidate plans at once on one GPU:
 *
 *   window (Sec. 3.2 window W_t of concurrent workflows, snapshot S_t of the
 *   pool, Predictor table of Eq. 1)  +  plans (device, priority, fuse bit,
 *   prefetch bit per activation)   ->   per-plan score and, optionally, the
 *   per-activation schedule.
 *
 * Semantics of one plan (each step cites the passage it follows):
 *   1. Units (Eq. 3, Eq. 4, Eq. 9).  Activation v is a chain member when its
 *      fuse bit is set and edge (u,v) satisfies Eq. 3: pred(v) = {u},
 *      succ(u) = {v}, same model.  Every other activation heads a unit: its
 *      chain of members runs back to back on the head's device under one
 *      grant; memory is the members' maximum; a member's own device entry
 *      is ignored.
 *   2. Resource order (Eq. 10; Sec. 3.5 tick-local planning).  Units are
 *      taken in ascending (topological level, priority, activation index).
 *   3. Lifecycle and memory (Eq. 5, Eq. 11; Sec. 3.5 reclamation).  A unit
 *      reuses its model if resident on its device, else loads it.  While the
 *      device cannot hold the resident models plus the load plus the unit's
 *      memory, the lease-free victim with no remaining use on the device is
 *      reclaimed first, then the least recently used, then the lower model
 *      id.  If it still does not fit the plan is flagged WF_ST_CAPACITY
 *      (memory equal to capacity fits).
 *   4. Timeline (Eq. 2, Eq. 7).  Release r = max(workflow arrival, latest
 *      predecessor finish).  A device runs one unit or one load at a time
 *      (unless the window sets batch limits, below).
 *      A load starts at max(r, device free) -- or max(arrival, device free)
 *      when the prefetch bit is set (Eq. 5, alpha_N = Prefetch) -- and the
 *      unit starts at max(r, load end); without a load at max(r, device
 *      free).  Reclamation takes no time.
 *   5. Score (Sec. 4 metrics).  makespan = last finish - first arrival;
 *      p95 = nearest-rank 95th percentile (the ceil(0.95 W)-th smallest) of
 *      per-workflow (last finish - arrival); objective = fp32(w_makespan *
 *      fp32(makespan)) + fp32(w_p95 * fp32(p95)), each operation rounded to
 *      nearest even, no fused multiply-add; min_headroom = min over devices
 *      of (capacity - peak memory).
 * Times are integer microseconds (int64), memory integer MiB (int32).
 *
 * Conventions
 *   - All functions are C, never throw, and return wf_status (0 = OK).
 *   - Validation failures return WF_EINVAL and change nothing; the message
 *     is available from wf_plan_last_error().
 *   - Plan, score, schedule and index buffers are caller-owned DEVICE
 *     memory of the context's GPU; they must stay alive until the work
 *     queued on the given stream has completed.  score_batch and argmin are
 *     asynchronous on that stream (NULL = the default stream); launch errors
 *     are reported on return as WF_EHIP.
 *   - A context is not thread-safe; use one per host thread.  Calls on one
 *     context must not run concurrently on different streams: the scoring
 *     calls may share the context's scratch area (per-wave regions of
 *     windows too large for LDS, allocated at upload, at most 1 GiB) and
 *     the argmins its work area.  A new upload must not race with queued
 *     work either (synchronise first).  Use one context per stream for
 *     concurrent scoring.
 */
#ifndef WF_PLAN_H
#define WF_PLAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WF_OK = 0,
  WF_EINVAL = 1,        /* invalid argument or window                       */
  WF_ENOWINDOW = 2,     /* score/argmin before a successful upload          */
  WF_ENOMEM = 3,        /* host or device allocation failed                 */
  WF_EHIP = 4,          /* HIP runtime error (message has the HIP string)   */
  WF_EUNSUPPORTED = 5   /* valid but outside the library's limits           */
} wf_status;

/* Limits of the library. */
#define WF_MAX_ACT 65535    /* activations per window                     */
#define WF_MAX_MODELS 64    /* models (resident sets are 64-bit masks)    */
#define WF_MAX_DEV 127      /* devices in the pool (plans carry int8 device ids) */
#define WF_MAX_MEM_MIB (1 << 28)   /* per weight / activation memory entry */
#define WF_MAX_CAP_MIB (1 << 30)   /* per device capacity                   */
#define WF_MAX_TIME_US (1LL << 52) /* arrivals and initial free times; every
                                      time then stays below 2^53 (exact in fp64) */
#define WF_MAX_MUT 64              /* mutations per generated candidate        */
#define WF_MAX_CLASSES 4           /* priority classes of the ranking key      */
#define WF_MAX_BATCH 4             /* batch limit of a device                  */

/* How generated candidates choose a re-placed device and a prefetch bit. */
enum { WF_SEARCH_UNIFORM = 0, WF_SEARCH_RULES = 1 };

/* Plan status bits; a plan is feasible iff status == 0. */
enum { WF_ST_INELIGIBLE = 1u, WF_ST_CAPACITY = 2u, WF_ST_REPLICA = 4u };

typedef struct wf_plan_ctx wf_plan_ctx; /* opaque; owns the device copy of a window */

/*
 * A planning window (Sec. 3.2) with its snapshot (S_t) and prediction table
 * (Eq. 1).  Host pointers, read during upload only (deep-copied).
 * Activations must be numbered in non-decreasing topological level (level 0
 * = no predecessor, else 1 + deepest predecessor).  Tables are row-major.
 */
typedef struct {
  int32_t n_act;                  /* N, 0..WF_MAX_ACT                          */
  int32_t n_wf;                   /* W >= 1 when N > 0; every workflow owns an activation */
  int32_t n_models;               /* M, 1..WF_MAX_MODELS                       */
  int32_t n_dev;                  /* D, 1..WF_MAX_DEV                          */
  const int32_t *act_wf;          /* [N] workflow id in [0, W)                 */
  const int32_t *act_model;       /* [N] model (deployment identity) in [0, M) */
  const int32_t *pred_off;        /* [N+1] CSR offsets, pred_off[0] = 0        */
  const int32_t *pred_idx;        /* [pred_off[N]] strictly increasing per row, each < its row */
  const int32_t *lat_us;          /* [N*D] predicted run time; -1 = ineligible (Eq. 8 cut) */
  const int32_t *mem_mib;         /* [N*D] activation memory M^inc (Eq. 11), 0..WF_MAX_MEM_MIB */
  const int64_t *wf_arrival_us;   /* [W] 0..WF_MAX_TIME_US                     */
  const int32_t *dev_cap_mib;     /* [D] 0..WF_MAX_CAP_MIB                     */
  const int32_t *model_mib;       /* [M] weights, 0..WF_MAX_MEM_MIB            */
  const int32_t *load_us;         /* [M*D] load time of model m on device d, >= 0 */
  const uint64_t *init_resident;  /* [D] resident-model bitmask; must fit the capacity */
  const int64_t *dev_free0_us;    /* [D] busy-until time, or NULL for all 0    */
  float w_makespan, w_p95;        /* objective weights, finite and >= 0        */
  const uint8_t *wf_class;        /* [W] priority class of each workflow for the ranking
                                     key (Eq. 12), 0..WF_MAX_CLASSES-1, class 0 ranked
                                     first; NULL = every workflow in class 0    */
  int32_t victim_order;           /* WF_VICTIM_REMAINING_LRU (0, step 3 above) or
                                     WF_VICTIM_PAPER (1, below)                 */
  const int32_t *dev_batch;       /* [D] batch limit 1..WF_MAX_BATCH (below), or NULL
                                     for 1 everywhere                           */
  const int32_t *model_replica_cap; /* [M] replica cap of each model >= 1 (below), or
                                     NULL for none; the initial residency must
                                     hold at most cap[m] copies of model m      */
  int64_t prefetch_slack_us;      /* dispatch slack of the rule-guided prefetch
                                     alternative (WF_SEARCH_RULES, below),
                                     0..WF_MAX_TIME_US                          */
} wf_window_desc;

/*
 * Replica cap (Sec. 3.5: scale-out -- a new replica of a deployment on
 * another device -- is subject to the replica cap).  A plan is flagged
 * WF_ST_REPLICA when, for some model m and some topological level L, the
 * devices that hold a copy of m as the units of L start (in resource order)
 * or load one for a unit of L outnumber model_replica_cap[m].  The flag is a
 * check only: no time, memory or count of the plan changes.
 */

/*
 * Batch limits (Eq. 11 and the replica batch limit B_q after it; Sec. 4,
 * continuous batching).  A device with batch limit B runs up to B units at
 * once, dispatched from its queue in resource order.  A unit takes the
 * device's slot that frees first (lowest slot on ties); its first action --
 * the load when its model is not resident, else the unit itself -- begins at
 *   t = max(release, or the workflow arrival for a prefetched load; the
 *           slot's free time; the previous unit's first action).
 * At t the device must hold its resident weights, the memory of every unit
 * still running at t (finish > t), the load and the unit's own memory.  Only
 * copies whose model no running unit uses (lease-free) may be reclaimed, in
 * the window's victim order.  If it still does not fit, t moves to the next
 * finish of a running unit and the check repeats; with no unit running the
 * plan is flagged WF_ST_CAPACITY and the unit proceeds.  A load ends L later
 * and the unit starts at max(release, load end); otherwise it starts at t.
 * Peak memory is taken at t.  B = 1 is the one-unit device of step 4.
 */

/*
 * Reclamation victim order.  WF_VICTIM_REMAINING_LRU is step 3 above.
 * WF_VICTIM_PAPER follows Sec. 3.5 (reclamation): among the resident copies
 * other than the unit's own, first those whose model is resident on another
 * device as the unit's topological level starts (redundant copies), then the
 * largest ratio of next-use distance to reload time -- distance = the number
 * of the device's units, in resource order, from the current one to the next
 * one that uses the model; the ratio distance / load time is infinite when
 * there is no next use or the load takes 0 us, and finite ratios compare by
 * cross-multiplication -- then least recently used, then the lower model id.
 */
enum { WF_VICTIM_REMAINING_LRU = 0, WF_VICTIM_PAPER = 1 };

/* Per-plan score, 32 bytes.  For a WF_ST_INELIGIBLE plan every other field
 * is 0. */
typedef struct {
  int64_t makespan_us;
  int64_t p95_us;
  float objective;
  uint32_t status;
  int32_t min_headroom_mib;
  uint16_t n_loads;   /* saturates at 65535 */
  uint16_t n_evicts;  /* saturates at 65535 */
} wf_plan_score;

/* Optional schedule output (device pointers, row-major per plan).  Rows of
 * WF_ST_INELIGIBLE plans are unspecified.  The first four arrays are
 * required when a schedule is requested; reclaimed_models may be NULL. */
typedef struct {
  int64_t *start_us;       /* [P][N] start of each activation                 */
  int64_t *finish_us;      /* [P][N] finish of each activation                */
  int64_t *load_start_us;  /* [P][N] load start of a unit head, -1 otherwise  */
  int32_t *peak_mib;       /* [P][D] peak memory of each device               */
  uint64_t *reclaimed_models; /* [P][N] at a unit head: bit m set when the copy
                                 of model m was reclaimed from the unit's device
                                 before the unit's first action (Eq. 5, Sec. 3.5
                                 reclamation); 0 for chain members          */
} wf_plan_sched;

/* Create a context on HIP device `hip_device`.  On failure *out is NULL and
 * wf_plan_last_error(NULL) describes the error. */
wf_status wf_plan_ctx_create(int hip_device, wf_plan_ctx **out);

/* Free the context and its device tables (NULL is a no-op).  Work queued on
 * the context must have completed. */
void wf_plan_ctx_destroy(wf_plan_ctx *ctx);

/* Message of the last failed call on `ctx` (or of the last failed
 * wf_plan_ctx_create / validation of this thread when ctx is NULL); "" if
 * none.  Valid until the next call on the context. */
const char *wf_plan_last_error(const wf_plan_ctx *ctx);

/* Host-only check of a window (no GPU needed): WF_OK or WF_EINVAL /
 * WF_EUNSUPPORTED with a message copied into err (NUL-terminated, may be
 * NULL). */
wf_status wf_plan_validate_window(const wf_window_desc *w, char *err, size_t err_len);

/* Validate the window, derive its structure (levels, Eq. 3 fusibility,
 * unique successors) and copy it to the device, replacing any previous
 * window.  Synchronous. */
wf_status wf_plan_upload_window(wf_plan_ctx *ctx, const wf_window_desc *w);

/* Score plans 0..n_plans-1.  dev [P][N] int8 device per activation; prio
 * [P][N] uint16 priority; flags [P][ceil(N/4)] where activation i owns bit
 * 2*(i%4) (fuse) and bit 2*(i%4)+1 (prefetch) of byte i/4 (padding bits are
 * ignored).  Out-of-range devices make a plan WF_ST_INELIGIBLE.  scores
 * [P]; sched may be NULL (scores only).  n_plans = 0 is a no-op. */
wf_status wf_plan_score_batch(wf_plan_ctx *ctx, const int8_t *dev, const uint16_t *prio,
                              const uint8_t *flags, int64_t n_plans, wf_plan_score *scores,
                              const wf_plan_sched *sched, void *hip_stream);

/* Among plans with status 0, the index of the smallest objective (lowest
 * index on ties), or -1 if none is feasible, written to the device int64
 * *out_index.  n_plans must be < 2^32; n_plans = 0 writes -1.  Uses a small
 * work area owned by the context (shared with wf_plan_argmin_keys): argmin
 * calls on one context must not run concurrently on different streams. */
wf_status wf_plan_argmin(wf_plan_ctx *ctx, const wf_plan_score *scores, int64_t n_plans,
                         int64_t *out_index, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * result of wf_plan_argmin without a context.  Runs on the calling thread's
 * current HIP device and allocates nothing: its partial minima (512 of 8
 * bytes, 4 KiB) live in a static array of the library that each GPU holds
 * for the life of the process.  Every call on one GPU shares that array, so
 * calls that overlap on one GPU (different streams or host threads) race;
 * each call writes every entry it reads, so nothing needs clearing.
 * n_plans must be < 2^32 (WF_EINVAL otherwise); n_plans = 0 writes -1.
 * Errors are reported by wf_plan_last_error(NULL).  Asynchronous on
 * hip_stream. */
wf_status wf_plan_argmin_noalloc(const wf_plan_score *scores, int64_t n_plans,
                                 int64_t *out_index, void *hip_stream);

/*
 * Candidate generation fused with scoring.  Algorithm 1 weighs alternatives
 * before Propagate checks one: another eligible device for a unit (the
 * binding choice, filtered by Eq. 8), another order among a level's units
 * (the ranked order of Eq. 10), another fusion choice (Eq. 3), another
 * lifecycle choice for near-ready work (Eq. 5, alpha_N = Prefetch).  These
 * calls draw such alternatives around an incumbent plan on the GPU, so the
 * candidates never exist in HBM.
 *
 * Candidate c is the incumbent with n_mut mutations applied in order
 * t = 0 .. n_mut-1.  Mutation t draws (r0, r1, r2, r3) = Philox4x32-10
 * (Salmon, Moraes, Dror and Shaw, SC'11) with counter (c mod 2^32,
 * c div 2^32, t, 0) and key (seed mod 2^32, seed div 2^32); then with
 * i = (r1 * N) div 2^32 and kind = r0 div 2^30:
 *   kind 0: the devices d with lat_us[i][d] >= 0, ascending, form E; when E
 *           is not empty, dev[i] = E[(r2 * |E|) div 2^32];
 *   kind 1: [lo, lo + w) is the index range of i's topological level;
 *           j = lo + (r2 * w) div 2^32; prio[i] and prio[j] are swapped;
 *   kind 2: the fuse bit of i is toggled;
 *   kind 3: the prefetch bit of i is toggled.
 * r3 is not used.  With N = 0 a candidate is the incumbent.  This is mode
 * WF_SEARCH_UNIFORM.  Mode WF_SEARCH_RULES draws the same (kind, i) and
 * takes kinds 0 and 3 from the rules Algorithm 1 names (Sec. 3.5) instead,
 * under these readings:
 *   - a unit is ready when activation i has no predecessor and its workflow
 *     has arrived by the window time 0; every other unit is near-ready;
 *   - kind 0, BestFeasibleBinding: among E, a device whose initial resident
 *     set holds i's model is reused first (the one with the smallest
 *     lat_us[i][d], then the lower id); with none, the load of largest value
 *     -- the summed lat_us[j][d] of the ready activations j of i's model
 *     eligible on d (the ready work the load unlocks) over load_us[m][d],
 *     a load time of 0 worth more than any ratio -- then the smallest
 *     lat_us[i][d], then the lower id.  With E empty dev[i] is unchanged;
 *   - kind 3, PlanPrefetch: with d = dev[i] as the earlier mutations left it
 *     (unchanged when d is outside 0..n_dev-1), the prefetch bit of i is set
 *     iff i is near-ready and its earliest release -- the longest path to it
 *     from its workflow's arrival over its predecessors, each on its fastest
 *     eligible device (0 with none) -- is at most load_us[m][d] +
 *     prefetch_slack_us; otherwise it is cleared.
 * Kinds 1 and 2 are as in the uniform mode.  Any other mode is WF_EINVAL.
 *
 * dev [N], prio [N], flags [ceil(N/4)] are the incumbent's rows (device
 * memory, layout of wf_plan_score_batch).  Candidates first ..
 * first+n_candidates-1 are generated; 0 <= n_mut <= WF_MAX_MUT, first >= 0
 * and first + n_candidates <= 2^62, else WF_EINVAL.
 */

/* Score the candidates: scores[k] is candidate first+k scored exactly as
 * wf_plan_score_batch would score its rows.  Asynchronous on hip_stream. */
wf_status wf_plan_search_batch(wf_plan_ctx *ctx, const int8_t *dev, const uint16_t *prio,
                               const uint8_t *flags, int32_t mode, uint64_t seed, int32_t n_mut,
                               int64_t first, int64_t n_candidates, wf_plan_score *scores,
                               void *hip_stream);

/* Write the candidates' rows (out_dev [n][N], out_prio [n][N], out_flags
 * [n][ceil(N/4)], device memory) -- to adopt a winner found by
 * wf_plan_search_batch and wf_plan_argmin.  Asynchronous on hip_stream. */
wf_status wf_plan_search_rows(wf_plan_ctx *ctx, const int8_t *dev, const uint16_t *prio,
                              const uint8_t *flags, int32_t mode, uint64_t seed, int32_t n_mut,
                              int64_t first, int64_t n_candidates, int8_t *out_dev,
                              uint16_t *out_prio, uint8_t *out_flags, void *hip_stream);

/*
 * Ranking keys.  The paper's scheduler ranks plans lexicographically by
 * Eq. 12 (Sec. 3.5),  Phi = (-A_1, ..., -A_K, C_F, -P_N, H_life):  ready-work
 * coverage per priority class first, then the latest completion of that
 * work, then timely prefetching and lifecycle overhead.  This library
 * computes the terms on the same simulation as wf_plan_score_batch, under
 * these readings:
 *   - a unit is ready (in F_t) when its head has no predecessor and its
 *     workflow has arrived by the window time 0; every other unit is
 *     near-ready (N_t);
 *   - the class of a ready unit is its workflow's wf_class (K =
 *     WF_MAX_CLASSES; classes the window does not use count 0);
 *   - A_k = the ready units of class k that are admitted: the memory check
 *     of step 3 holds at their turn;
 *   - C_F = the latest finish (absolute us) of an admitted ready unit, 0 if
 *     there is none;
 *   - P_N = the near-ready units with the prefetch bit whose model is loaded
 *     for them and whose load ends no later than their release;
 *   - H_life = for each ready unit that loads, its start minus the later of
 *     its release and the time its device became free (the delay the load
 *     adds), plus the load time of every load of a model that an earlier
 *     unit of the plan had reclaimed from that device (reload cost).
 * For a WF_ST_INELIGIBLE plan every field other than status is 0.
 */
typedef struct {
  int64_t c_ready_us;                  /* C_F                                   */
  int64_t h_life_us;                   /* H_life                                */
  uint16_t admitted[WF_MAX_CLASSES];   /* A_1 .. A_K                            */
  uint16_t timely_prefetch;            /* P_N, saturates at 65535               */
  uint16_t pad;                        /* 0                                     */
  uint32_t status;                     /* as wf_plan_score.status               */
} wf_plan_key;                         /* 32 bytes                              */

/* Ranking keys of plans 0..n_plans-1 (rows as for wf_plan_score_batch) into
 * keys [P] (device memory).  Asynchronous on hip_stream. */
wf_status wf_plan_score_keys(wf_plan_ctx *ctx, const int8_t *dev, const uint16_t *prio,
                             const uint8_t *flags, int64_t n_plans, wf_plan_key *keys,
                             void *hip_stream);

/* Ranking keys of generated candidates first .. first+n_candidates-1 around
 * an incumbent (arguments and limits as for wf_plan_search_batch). */
wf_status wf_plan_search_keys(wf_plan_ctx *ctx, const int8_t *dev, const uint16_t *prio,
                              const uint8_t *flags, int32_t mode, uint64_t seed, int32_t n_mut,
                              int64_t first, int64_t n_candidates, wf_plan_key *keys,
                              void *hip_stream);

/* Among keys with status 0, the index of the lexicographically smallest Phi
 * (lowest index on ties), or -1 if none is feasible, written to the device
 * int64 *out_index.  0 <= n_plans <= 2^62; n_plans = 0 writes -1.  Uses a
 * small work area owned by the context: calls on one context must not run
 * concurrently on different streams.  Asynchronous on hip_stream. */
wf_status wf_plan_argmin_keys(wf_plan_ctx *ctx, const wf_plan_key *keys, int64_t n_plans,
                              int64_t *out_index, void *hip_stream);

/* The prefix commit of Algorithm 1 (Prefix_t): of one selected plan, the
 * actions to commit before the window is planned again.  Inputs are the
 * plan's device row dev [N] and its schedule rows start_us, finish_us,
 * load_start_us, reclaimed [N] (as wf_plan_score_batch writes them for that
 * plan; all device memory).  Readings:
 *   - the window is planned again at the next predicted event after the
 *     window time 0: the earliest activation finish, load end (load start
 *     plus the model's load time on the unit's device) or workflow arrival
 *     that is later than 0; INT64_MAX when there is none -> *t_next_us;
 *   - every action that begins before that event is committed: commit[i]
 *     bit 0 when activation i starts before it (the unit's grant), bit 1
 *     when i's load starts before it;
 *   - the reclamations before a unit's first action (its load, else its
 *     start) are committed with it: commit_reclaimed[i] = reclaimed[i] when
 *     that action begins before the event, else 0.
 * Outputs commit [N] uint8, commit_reclaimed [N] uint64 and *t_next_us are
 * device memory.  A device entry outside 0..n_dev-1 (an ineligible plan)
 * gives unspecified results without touching memory outside the arrays.
 * N = 0 writes only *t_next_us.  Asynchronous on hip_stream. */
wf_status wf_plan_prefix(wf_plan_ctx *ctx, const int8_t *dev, const int64_t *start_us,
                         const int64_t *finish_us, const int64_t *load_start_us,
                         const uint64_t *reclaimed, uint8_t *commit,
                         uint64_t *commit_reclaimed, int64_t *t_next_us, void *hip_stream);

/* Time arithmetic the kernels use for the uploaded window: 32 when they
 * carry times as uint32 offsets from the window origin, 64 when they use
 * fp64 (exact for integers below 2^53); 0 when ctx is NULL or has no window.
 * uint32 is used when every time of every plan provably stays below 2^32 us
 * (a static bound: latest arrival or busy-until plus every activation's
 * longest run and load), and also when that bound is below 8 x 2^32 us: then
 * uint32 additions saturate, and every scoring call runs a second, fp64 pass
 * over the groups of plans whose times saturated.  Results are identical in
 * every case. */
int wf_plan_time_bits(const wf_plan_ctx *ctx);

/* Name of the kernel that scores plans read from HBM for the uploaded
 * window without a schedule: "score_lean" when the window qualifies for the
 * lean kernel (uint32 times, at most 16 models, at most 512 activations;
 * under the paper's reclamation order or with batch limits only without
 * replica caps, and not both), else "score_plans"; "" when ctx is NULL or
 * has no window.  Both give identical results.  Under the paper's order or
 * with batch limits the lean kernel serves wf_plan_score_batch only. */
const char *wf_plan_score_kernel(const wf_plan_ctx *ctx);

/* Library version string. */
const char *wf_plan_version(void);

#ifdef __cplusplus
}
#endif
#endif /* WF_PLAN_H */
