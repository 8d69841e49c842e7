// Internal interface between the host library (host.hip) and the gfx950
// kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wf_plan.h"

namespace wfp {

// Window tables resident in HBM (one allocation owned by the context).
struct WindowDev {
  int32_t N, W, M, D, NB;   // NB = ceil(N / 4) flag bytes per plan row
  int32_t n_levels, wmax;   // number of topological levels, widest level
  int64_t min_arrival;      // first workflow arrival (0 when N == 0)
  float w_mk, w_p95;
  const int32_t* act_model;   // [N]
  const int32_t* act_wf;      // [N]
  const uint8_t* fusible;     // [N] Eq. 3 holds for the edge into v
  const int32_t* chain_next;  // [N] v when succ(u) = {v} and v is fusible, else -1
  const int32_t* pred_off;    // [N+1]
  const int32_t* pred_idx;    // [nnz]
  const int32_t* lat;         // [N*D]
  const int32_t* mem;         // [N*D]
  const int64_t* arrival;     // [W]
  const int32_t* cap;         // [D]
  const int32_t* wmib;        // [M]
  const int32_t* load;        // [M*D]
  const uint64_t* init_res;   // [D]
  const int64_t* free0;       // [D]
  const int32_t* level_off;   // [n_levels+1]
};

// Launch geometry and LDS carve-up of the scoring kernel.
struct ScoreLaunch {
  int G;            // plans scored together by one wave (G * D <= 64)
  int nwords;       // 64-bit words per level bitmask = ceil(wmax / 64)
  int big;          // 1: finish times and workflow maxima live in global scratch
  int off_pos, off_claim, off_mask, off_cnt, off_last, off_acc, off_finish, off_wfmax;
  int lds_bytes;
  int grid;         // persistent grid (waves)
  int64_t scratch_per_wave;   // int64 entries of global scratch per wave (big mode)
};

hipError_t launch_score(const WindowDev& w, const ScoreLaunch& L, int64_t* scratch,
                        const int8_t* dev, const uint16_t* prio, const uint8_t* flags,
                        int64_t n_plans, wf_plan_score* scores, const wf_plan_sched* sched,
                        hipStream_t stream);

hipError_t launch_argmin(const wf_plan_score* scores, int64_t n_plans, int64_t* out_index,
                         int grid, hipStream_t stream);

// Per-plan accumulators kept in LDS by the scoring kernel.
struct PlanAcc {
  uint32_t status;
  int32_t headroom;
  uint32_t loads;
  uint32_t evicts;
  unsigned long long max_finish;
  long long p95;
};

}  // namespace wfp
