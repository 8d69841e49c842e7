/*
 * oracle.h -- plain, slow, single-threaded CPU reference scorer for candidate
 * physical execution plans.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this code; only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark load it.  It shares no header, helper, table
 * or constant with the GPU path.
 *
 * What it computes, per plan (paper Sec. 3.3-3.5):
 *   - fused units from the plan's fuse bits under the fusion condition
 *     (Eq. 3) with summed run time and maximal memory (Eq. 4);
 *   - the resource order: units sorted by (topological level, priority,
 *     activation index) -- ready work before near-ready work, priority
 *     within (Sec. 3.5, tick-local planning; Eq. 10);
 *   - per-device model lifecycle: reuse a resident replica or load it
 *     (Eq. 5), reclaiming lease-free victims first -- copies with no
 *     remaining use on the device, then least recently used, then the
 *     lower model id (Sec. 3.5, reclamation);
 *   - cumulative memory on every device at every unit transition (Eq. 11);
 *   - the max-plus timeline over graph and resource predecessors
 *     (Eq. 2, Eq. 7), loads starting at release, or at workflow arrival
 *     when prefetched;
 *   - makespan and p95 workflow completion (Sec. 4, metrics) and the
 *     fp32 objective  w_makespan * makespan + w_p95 * p95.
 * All times are integer microseconds, memory integer MiB.
 */
#ifndef WF_ORACLE_H
#define WF_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n_act, n_wf, n_models, n_dev;
  const int32_t *act_wf;        /* [n_act] workflow of each activation        */
  const int32_t *act_model;     /* [n_act] model (deployment identity)        */
  const int32_t *pred_off;      /* [n_act+1] CSR row offsets of predecessors  */
  const int32_t *pred_idx;      /* [nnz] predecessors, increasing, < row      */
  const int32_t *lat_us;        /* [n_act*n_dev] run time, < 0 = ineligible   */
  const int32_t *mem_mib;       /* [n_act*n_dev] activation memory            */
  const int64_t *wf_arrival_us; /* [n_wf]                                     */
  const int32_t *dev_cap_mib;   /* [n_dev]                                    */
  const int32_t *model_mib;     /* [n_models] weights                         */
  const int32_t *load_us;       /* [n_models*n_dev] load time                 */
  const uint64_t *init_resident;/* [n_dev] resident-model bitmask             */
  const int64_t *dev_free0_us;  /* [n_dev] busy-until, or NULL for all 0      */
  float w_makespan, w_p95;
  int32_t victim_order;         /* ORC_VICTIM_REMAINING_LRU or ORC_VICTIM_PAPER */
  const int32_t *dev_batch;     /* [n_dev] batch limit 1..ORC_MAX_BATCH, NULL = all 1 */
  const int32_t *replica_cap;   /* [n_models] replica cap >= 1, NULL = no cap (below) */
  int64_t prefetch_slack_us;    /* dispatch slack of the prefetch rule (below), >= 0 */
} orc_window;

/*
 * Replica cap (Sec. 3.5: scale-out, a new replica of a deployment on another
 * device, is subject to the replica cap).  With replica_cap set, a plan is
 * flagged ORC_REPLICA when, for some model m and some topological level L,
 * the devices that hold a copy of m as the units of L start (in resource
 * order) or load one for a unit of L outnumber replica_cap[m].  The flag is
 * a check only: no time, memory or count of the plan changes.  The initial
 * residency must respect the caps (ORC_ERR_REPLICA otherwise).
 */

/*
 * Batch limit (Eq. 11 and the replica batch limit B_q after it; Sec. 4,
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
 * plan is flagged ORC_CAPACITY and the unit proceeds.  A load ends L later
 * and the unit starts at max(release, load end); otherwise it starts at t.
 * Peak memory is taken at t.  With B = 1 this is exactly the one-unit device
 * of the semantics above.
 */
enum { ORC_MAX_BATCH = 4 };

/*
 * Reclamation victim order (Sec. 3.5, reclamation), among the resident
 * models of the device other than the unit's own:
 *   ORC_VICTIM_REMAINING_LRU -- copies with no remaining use on the device
 *     in the plan first, then least recently used (initial residents never
 *     used count as oldest), then the lower model id;
 *   ORC_VICTIM_PAPER -- redundant copies first (the model is resident on
 *     another device when the current topological level starts), then the
 *     largest ratio of next-use distance to reload time -- distance = the
 *     number of the device's units, in resource order, from the current one
 *     to the next one that uses the model, infinite without one; the ratio
 *     distance / load time is infinite when either the distance is infinite
 *     or the load time is 0; finite ratios compare by cross-multiplication --,
 *     then least recently used, then the lower model id.
 */
enum { ORC_VICTIM_REMAINING_LRU = 0, ORC_VICTIM_PAPER = 1 };

typedef struct {
  int64_t makespan_us;
  int64_t p95_us;
  float objective;
  uint32_t status;            /* ORC_INELIGIBLE | ORC_CAPACITY | ORC_REPLICA, 0 = feasible */
  int32_t min_headroom_mib;
  uint16_t n_loads, n_evicts; /* saturate at 65535                            */
} orc_score;

enum { ORC_INELIGIBLE = 1u, ORC_CAPACITY = 2u, ORC_REPLICA = 4u };

/* Error codes of orc_score_plans. */
enum {
  ORC_OK = 0,
  ORC_ERR_SIZE = 1,       /* negative sizes, n_models outside 1..64, n_dev < 1 */
  ORC_ERR_PRED = 2,       /* predecessor out of range or not increasing        */
  ORC_ERR_ORDER = 3,      /* activations not numbered in level order           */
  ORC_ERR_INDEX = 4,      /* workflow / model id out of range                  */
  ORC_ERR_EMPTY_WF = 5,   /* a workflow without activations                    */
  ORC_ERR_NOMEM = 6,
  ORC_ERR_CLASS = 7,      /* a workflow class outside 0 .. ORC_MAX_CLASSES-1    */
  ORC_ERR_VICTIM = 8,     /* victim_order is not one of ORC_VICTIM_*           */
  ORC_ERR_BATCH = 9,      /* a batch limit outside 1 .. ORC_MAX_BATCH          */
  ORC_ERR_REPLICA = 10    /* a replica cap below 1, or initial copies above it */
};

/*
 * Score plans [0, n_plans) of the row-major batch that starts at dev/prio/
 * flags (dev[p*N+i], prio[p*N+i], flags[p*ceil(N/4)+i/4]).  For a plan with
 * status ORC_INELIGIBLE every other score field is 0 and its schedule rows
 * are left untouched.  start/finish/load_start ([P][N]), peak ([P][D]) and
 * reclaimed ([P][N]: the mask of models whose copies were reclaimed from the
 * unit's device before the unit's first action, at the unit's head; 0 for
 * chain members) may each be NULL.  Thread-safe: no global state.
 */
int orc_score_plans(const orc_window *w, const int8_t *dev, const uint16_t *prio,
                    const uint8_t *flags, int64_t n_plans, orc_score *scores,
                    int64_t *start_us, int64_t *finish_us, int64_t *load_start_us,
                    int32_t *peak_mib, uint64_t *reclaimed);

/*
 * The prefix commit of Algorithm 1 (Prefix_t: of the selected plan, the
 * actions executable before the window is planned again), for one plan's
 * device row and schedule (as orc_score_plans writes them), read thus:
 *   - the window is planned again at the next predicted event after the
 *     window time 0: the earliest activation finish, load end (load start
 *     + the model's load time on the unit's device) or workflow arrival that
 *     is later than 0; INT64_MAX when there is none;
 *   - every action that begins before that event is committed: commit[i]
 *     bit 0 when activation i starts before it (the unit's grant), bit 1
 *     when i's load starts before it;
 *   - the reclamations of a unit whose first action (its load, else its
 *     start) begins before the event are committed with it:
 *     commit_reclaimed[i] = reclaimed[i] then, else 0.
 * Returns ORC_ERR_INDEX for a device entry outside 0 .. n_dev-1.
 */
int orc_prefix(const orc_window *w, const int8_t *dev, const int64_t *start_us,
               const int64_t *finish_us, const int64_t *load_start_us,
               const uint64_t *reclaimed, uint8_t *commit, uint64_t *commit_reclaimed,
               int64_t *t_next_us);

/*
 * The lexicographic ranking key of Eq. 12 (Sec. 3.5),
 *   Phi = (-A_1, ..., -A_K, C_F, -P_N, H_life),
 * under these readings (K <= ORC_MAX_CLASSES):
 *   - a unit is ready (in F_t) when its head has no predecessor and its
 *     workflow has arrived by the window time t = 0; every other unit is
 *     near-ready;
 *   - the priority class of a ready unit is its workflow's class
 *     (wf_class[w] in 0 .. K-1, class 0 ranked first; NULL puts every
 *     workflow in class 0);
 *   - A_k counts the ready units of class k that are admitted: their memory
 *     check (Eq. 11) holds at their turn;
 *   - C_F is the latest completion (absolute us) of an admitted ready unit,
 *     0 when there is none;
 *   - P_N counts timely prefetches: near-ready units with the prefetch bit
 *     whose model is loaded for them and whose load ends no later than
 *     their release;
 *   - H_life is the loading delay of ready work -- for a ready unit that
 *     loads, its start minus the later of its release and the time its
 *     device became free -- plus the reload cost of reclamation -- the load
 *     time of every load of a model that an earlier unit of the plan had
 *     reclaimed from that device.
 * The simulation is the one of orc_score_plans.  For a plan with status
 * ORC_INELIGIBLE every other field is 0.
 */
enum { ORC_MAX_CLASSES = 4 };

typedef struct {
  int64_t c_ready_us;                  /* C_F                                  */
  int64_t h_life_us;                   /* H_life                               */
  uint16_t admitted[ORC_MAX_CLASSES];  /* A_1 .. A_K (unused classes 0)        */
  uint16_t timely_prefetch;            /* P_N                                  */
  uint16_t pad;
  uint32_t status;                     /* as orc_score.status                  */
} orc_phi;

int orc_phi_keys(const orc_window *w, const uint8_t *wf_class, const int8_t *dev,
                 const uint16_t *prio, const uint8_t *flags, int64_t n_plans, orc_phi *keys);

/* Topological level of every activation (0 for sources).  Returns an error
 * code as above. */
int orc_levels(const orc_window *w, int32_t *level_out);

/*
 * Candidate plans around an incumbent (the alternatives Algorithm 1 weighs
 * before Propagate: another eligible device for a unit -- the binding choice
 * filtered by Eq. 8 --, another order among a level's units -- the ranked
 * order of Eq. 10 --, another fusion choice -- Eq. 3 --, another lifecycle
 * choice for near-ready work -- Eq. 5, alpha_N = Prefetch).
 *
 * Candidate c is the incumbent with n_mut mutations applied in order
 * t = 0 .. n_mut-1.  Mutation t draws (r0, r1, r2, r3) = Philox4x32-10 with
 * counter (c mod 2^32, c div 2^32, t, 0) and key (seed mod 2^32,
 * seed div 2^32), then with i = (r1 * N) div 2^32 and kind = r0 div 2^30:
 *   kind 0: the devices d with lat[i][d] >= 0, ascending, form E; when E is
 *           not empty, dev[i] = E[(r2 * |E|) div 2^32];
 *   kind 1: [lo, lo + w) is the index range of i's topological level;
 *           j = lo + (r2 * w) div 2^32; prio[i] and prio[j] are swapped;
 *   kind 2: the fuse bit of i is toggled;
 *   kind 3: the prefetch bit of i is toggled.
 * r3 is not used.  With N = 0 a candidate is the incumbent.
 */

/* Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds of the
 * Philox-4x32 bijection on the counter, the key bumped by the Weyl
 * constants after every round. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Rows of candidates first .. first+count-1 (out_dev [count][N], out_prio
 * [count][N], out_flags [count][ceil(N/4)]) around the incumbent rows dev,
 * prio, flags of one plan.  mode ORC_SEARCH_UNIFORM draws the alternatives
 * uniformly; ORC_SEARCH_RULES takes them from the rules below.  Returns an
 * error code as above (ORC_ERR_SIZE for an unknown mode). */
enum { ORC_SEARCH_UNIFORM = 0, ORC_SEARCH_RULES = 1 };
int orc_search_candidates(const orc_window *w, const int8_t *dev, const uint16_t *prio,
                          const uint8_t *flags, uint64_t seed, int32_t n_mut, int64_t first,
                          int64_t count, int32_t mode, int8_t *out_dev, uint16_t *out_prio,
                          uint8_t *out_flags);

/*
 * Rule-guided alternatives (Algorithm 1, Sec. 3.5).  A unit is ready when
 * its activation has no predecessor and its workflow has arrived by the
 * window time 0; every other one is near-ready.
 *   BestFeasibleBinding of activation i (mutation kind 0): among its
 *   eligible devices (Eq. 8), one that holds i's model in the snapshot is
 *   reused first -- the fastest for i, then the lower id; with no resident
 *   copy, the load whose value is largest: the ready work it unlocks (the
 *   summed run times on that device of the ready activations of the same
 *   model eligible there) per load time of the model there (a free load is
 *   worth the most; equal values: the faster device for i, then the lower
 *   id).  An activation without an eligible device keeps its device.
 *   PlanPrefetch of activation i (kind 3): the prefetch bit is set when i
 *   is near-ready and its earliest release -- the longest path to it from
 *   the workflow's arrival over predecessors on their fastest eligible
 *   devices -- is at most the load time of its model on its current device
 *   plus the window's dispatch slack; otherwise it is cleared (ready units
 *   load at their release anyway).  A current device outside 0..n_dev-1
 *   leaves the bit unchanged.
 * Kinds 1 (a priority swap in the level) and 2 (the fuse bit) are drawn as
 * in the uniform mode.
 */

#ifdef __cplusplus
}
#endif
#endif
