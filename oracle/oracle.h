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
} orc_window;

typedef struct {
  int64_t makespan_us;
  int64_t p95_us;
  float objective;
  uint32_t status;            /* ORC_INELIGIBLE | ORC_CAPACITY, 0 = feasible */
  int32_t min_headroom_mib;
  uint16_t n_loads, n_evicts; /* saturate at 65535                            */
} orc_score;

enum { ORC_INELIGIBLE = 1u, ORC_CAPACITY = 2u };

/* Error codes of orc_score_plans. */
enum {
  ORC_OK = 0,
  ORC_ERR_SIZE = 1,       /* negative sizes, n_models outside 1..64, n_dev < 1 */
  ORC_ERR_PRED = 2,       /* predecessor out of range or not increasing        */
  ORC_ERR_ORDER = 3,      /* activations not numbered in level order           */
  ORC_ERR_INDEX = 4,      /* workflow / model id out of range                  */
  ORC_ERR_EMPTY_WF = 5,   /* a workflow without activations                    */
  ORC_ERR_NOMEM = 6
};

/*
 * Score plans [0, n_plans) of the row-major batch that starts at dev/prio/
 * flags (dev[p*N+i], prio[p*N+i], flags[p*ceil(N/4)+i/4]).  For a plan with
 * status ORC_INELIGIBLE every other score field is 0 and its schedule rows
 * are left untouched.  start/finish/load_start ([P][N]) and peak ([P][D])
 * may be NULL.  Thread-safe: no global state.
 */
int orc_score_plans(const orc_window *w, const int8_t *dev, const uint16_t *prio,
                    const uint8_t *flags, int64_t n_plans, orc_score *scores,
                    int64_t *start_us, int64_t *finish_us, int64_t *load_start_us,
                    int32_t *peak_mib);

/* Topological level of every activation (0 for sources).  Returns an error
 * code as above. */
int orc_levels(const orc_window *w, int32_t *level_out);

#ifdef __cplusplus
}
#endif
#endif
