// Batched scoring of candidate physical execution plans on gfx950.
//
// One wave (64 lanes) scores a group of G plans at a time and loops over
// groups (persistent grid).  Lanes take two roles:
//   * lanes over activations -- per plan, decode the packed row, find unit
//     heads (Eq. 3), count heads per (device, model), and give every head of
//     a topological level its slot in the resource order (level, priority,
//     index) (Eq. 10);
//   * lane (g, d) = (lane / D, lane % D) -- simulates device d of plan g:
//     reuse / reclaim / load (Eq. 5, Eq. 11) and the max-plus timeline of
//     Eq. 2 and Eq. 7, walking its own units of each level in slot order.
// Levels are processed in order, so every predecessor finish a unit reads
// was written by an earlier level (all predecessors sit at lower levels; a
// fused member's finish is written with its head, which sits lower still).
// Residency, reclamation and memory depend only on each device's unit
// sequence, never on times, which is what makes the device lanes
// independent within a level.
#include "kernels.h"

namespace wfp {
namespace {

__device__ __forceinline__ int fuse_bit(const uint8_t* fl, int v) {
  return (fl[v >> 2] >> ((v & 3) << 1)) & 1;
}
__device__ __forceinline__ int pf_bit(const uint8_t* fl, int v) {
  return (fl[v >> 2] >> (((v & 3) << 1) + 1)) & 1;
}
__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

template <bool BIG>
__global__ __launch_bounds__(64) void score_plans(WindowDev w, ScoreLaunch L, int64_t* scratch,
                                                  const int8_t* __restrict__ dev_all,
                                                  const uint16_t* __restrict__ prio_all,
                                                  const uint8_t* __restrict__ flags_all,
                                                  int64_t P, wf_plan_score* __restrict__ scores,
                                                  wf_plan_sched sched, int has_sched) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x;
  const int G = L.G, D = w.D, N = w.N, M = w.M, NW = L.nwords, WF = w.W;
  uint16_t* pos2u = reinterpret_cast<uint16_t*>(lds + L.off_pos);          // [G][wmax]
  unsigned long long* claim = reinterpret_cast<unsigned long long*>(lds + L.off_claim);  // [G][NW]
  unsigned long long* mask = reinterpret_cast<unsigned long long*>(lds + L.off_mask);    // [G][D][NW]
  uint32_t* cnt = reinterpret_cast<uint32_t*>(lds + L.off_cnt);            // [G*D][M]
  int32_t* lastu = reinterpret_cast<int32_t*>(lds + L.off_last);           // [G*D][M]
  PlanAcc* acc = reinterpret_cast<PlanAcc*>(lds + L.off_acc);              // [G]
  int64_t* finish;
  unsigned long long* wfmax;
  if (BIG) {
    int64_t* mine = scratch + (int64_t)blockIdx.x * L.scratch_per_wave;
    finish = mine;                                                         // [G][N]
    wfmax = reinterpret_cast<unsigned long long*>(mine + (int64_t)G * N);  // [G][W]
  } else {
    finish = reinterpret_cast<int64_t*>(lds + L.off_finish);
    wfmax = reinterpret_cast<unsigned long long*>(lds + L.off_wfmax);
  }

  const int g_me = lane / D;
  const int d_me = lane - g_me * D;
  const int64_t n_groups = (P + G - 1) / G;

  for (int64_t grp = blockIdx.x; grp < n_groups; grp += gridDim.x) {
    const int64_t p0 = grp * G;
    const int gcount = (int)((P - p0) < G ? (P - p0) : G);

    // ---- per-group initialisation ----
    for (int i = lane; i < G * D * M; i += 64) {
      cnt[i] = 0;
      lastu[i] = -1;
    }
    for (int i = lane; i < G * WF; i += 64) wfmax[i] = 0ull;
    if (lane < G) {
      acc[lane].status = 0;
      acc[lane].headroom = 0x7fffffff;
      acc[lane].loads = 0;
      acc[lane].evicts = 0;
      acc[lane].max_finish = 0ull;
      acc[lane].p95 = 0;
    }
    __syncthreads();

    // ---- unit heads and remaining uses per (device, model) ----
    for (int g = 0; g < gcount; ++g) {
      const int64_t p = p0 + g;
      const int8_t* pdev = dev_all + p * N;
      const uint8_t* pfl = flags_all + p * w.NB;
      for (int u = lane; u < N; u += 64) {
        if (w.fusible[u] && fuse_bit(pfl, u)) continue;  // chain member
        const int d = pdev[u];
        if (d < 0 || d >= D) {
          atomicOr(&acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
          continue;
        }
        atomicAdd(&cnt[(g * D + d) * M + w.act_model[u]], 1u);
      }
    }
    __syncthreads();

    // ---- device-lane state ----
    const bool active = g_me < gcount;
    const int64_t pw = p0 + (active ? g_me : 0);
    const uint8_t* myfl = flags_all + pw * w.NB;
    int64_t* myfin = finish + (int64_t)(active ? g_me : 0) * N;
    uint32_t* mycnt = cnt + (active ? (g_me * D + d_me) * M : 0);
    int32_t* mylast = lastu + (active ? (g_me * D + d_me) * M : 0);
    uint64_t res = 0;
    int32_t used = 0, peak = 0;
    int64_t freet = 0;
    uint32_t nld = 0, nev = 0, capbad = 0, inel = 0;
    int32_t seq = 0;
    int32_t capd = 0;
    if (active) {
      res = w.init_res[d_me];
      for (int m = 0; m < M; ++m)
        if ((res >> m) & 1ull) used += w.wmib[m];
      peak = used;
      freet = w.free0[d_me];
      capd = w.cap[d_me];
    }

    for (int lv = 0; lv < w.n_levels; ++lv) {
      const int lo = w.level_off[lv], hi = w.level_off[lv + 1], wl = hi - lo;
      const int nwl = (wl + 63) >> 6;

      // ---- resource order of the level's heads (per plan) ----
      for (int g = 0; g < gcount; ++g) {
        const int64_t p = p0 + g;
        const int8_t* pdev = dev_all + p * N;
        const uint16_t* pprio = prio_all + p * N;
        const uint8_t* pfl = flags_all + p * w.NB;
        unsigned long long* cl = claim + g * NW;
        unsigned long long* mk = mask + g * D * NW;
        for (int i = lane; i < nwl; i += 64) cl[i] = 0ull;
        for (int i = lane; i < D * nwl; i += 64) mk[(i / nwl) * NW + (i % nwl)] = 0ull;
        __syncthreads();
        // fast path: priorities of the level's heads are distinct values in
        // [lo, hi) -- each head's slot is its priority minus lo
        int bad = 0;
        for (int u = lo + lane; u < hi; u += 64) {
          if (w.fusible[u] && fuse_bit(pfl, u)) continue;
          const int d = pdev[u];
          if (d < 0 || d >= D) continue;
          const int k = (int)pprio[u] - lo;
          if (k < 0 || k >= wl) {
            bad = 1;
            continue;
          }
          const unsigned long long bit = 1ull << (k & 63);
          if (atomicOr(&cl[k >> 6], bit) & bit) bad = 1;
        }
        bad = __any(bad);
        __syncthreads();
        for (int u = lo + lane; u < hi; u += 64) {
          if (w.fusible[u] && fuse_bit(pfl, u)) continue;
          const int d = pdev[u];
          if (d < 0 || d >= D) continue;
          const int pu = pprio[u];
          int k = pu - lo;
          if (bad) {  // general path: rank by (priority, index) among heads
            k = 0;
            for (int j = lo; j < hi; ++j) {
              if (w.fusible[j] && fuse_bit(pfl, j)) continue;
              const int dj = pdev[j];
              if (dj < 0 || dj >= D) continue;
              const int pj = pprio[j];
              k += (pj < pu) || (pj == pu && j < u);
            }
          }
          pos2u[g * w.wmax + k] = (uint16_t)u;
          atomicOr(&mk[d * NW + (k >> 6)], 1ull << (k & 63));
        }
        __syncthreads();
      }

      // ---- device lanes walk their units of this level in slot order ----
      if (active) {
        const unsigned long long* mymask = mask + (g_me * D + d_me) * NW;
        const uint16_t* mypos = pos2u + g_me * w.wmax;
        const int d = d_me;
        for (int j = 0; j < nwl; ++j) {
          unsigned long long bits = mymask[j];
          while (bits) {
            const int k = (j << 6) + __builtin_ctzll(bits);
            bits &= bits - 1;
            const int u = mypos[k];
            const int m = w.act_model[u];
            const int wf = w.act_wf[u];
            mycnt[m] -= 1u;
            // release (Eq. 2): arrival, or the latest predecessor finish
            int64_t r = w.arrival[wf];
            for (int e = w.pred_off[u]; e < w.pred_off[u + 1]; ++e) r = max64(r, myfin[w.pred_idx[e]]);
            // unit memory: maximum over the fused chain (Eq. 4)
            int32_t mx = w.mem[u * D + d];
            inel |= (uint32_t)(w.lat[u * D + d] < 0);
            for (int v = u;;) {
              const int c = w.chain_next[v];
              if (c < 0 || !fuse_bit(myfl, c)) break;
              v = c;
              const int32_t mv = w.mem[v * D + d];
              mx = mv > mx ? mv : mx;
              inel |= (uint32_t)(w.lat[v * D + d] < 0);
            }
            // lifecycle (Eq. 5) with reclamation, cumulative memory (Eq. 11)
            const uint64_t mbit = 1ull << m;
            const bool miss = !(res & mbit);
            const int32_t need = (miss ? w.wmib[m] : 0) + mx;
            while (used + need > capd) {
              uint64_t cand = res & ~mbit;
              if (!cand) break;
              int victim = 0, v_alive = 2, v_last = 0x7fffffff;
              while (cand) {
                const int m2 = __builtin_ctzll(cand);
                cand &= cand - 1;
                const int al = mycnt[m2] > 0u;
                const int la = mylast[m2];
                if (al < v_alive || (al == v_alive && la < v_last)) {
                  victim = m2;
                  v_alive = al;
                  v_last = la;
                }
              }
              res &= ~(1ull << victim);
              used -= w.wmib[victim];
              ++nev;
            }
            capbad |= (uint32_t)(used + need > capd);
            // timeline (Eq. 7)
            int64_t s, ls = -1;
            if (miss) {
              ls = max64(pf_bit(myfl, u) ? w.arrival[wf] : r, freet);
              const int64_t le = ls + w.load[m * D + d];
              res |= mbit;
              used += w.wmib[m];
              ++nld;
              s = max64(r, le);
            } else {
              s = max64(r, freet);
            }
            peak = (used + mx) > peak ? (used + mx) : peak;
            for (int v = u;;) {
              const int64_t f = s + w.lat[v * D + d];
              myfin[v] = f;
              if (has_sched) {
                sched.start_us[pw * N + v] = s;
                sched.finish_us[pw * N + v] = f;
                sched.load_start_us[pw * N + v] = (v == u) ? ls : -1;
              }
              s = f;
              const int c = w.chain_next[v];
              if (c < 0 || !fuse_bit(myfl, c)) break;
              v = c;
            }
            freet = s;
            mylast[m] = seq++;
          }
        }
      }
      __syncthreads();
    }

    // ---- per-plan reductions (Sec. 4 metrics) ----
    if (active) {
      atomicMin(&acc[g_me].headroom, capd - peak);
      atomicAdd(&acc[g_me].loads, nld);
      atomicAdd(&acc[g_me].evicts, nev);
      if (capbad) atomicOr(&acc[g_me].status, (uint32_t)WF_ST_CAPACITY);
      if (inel) atomicOr(&acc[g_me].status, (uint32_t)WF_ST_INELIGIBLE);
      if (has_sched) sched.peak_mib[pw * D + d_me] = peak;
    }
    __syncthreads();
    for (int g = 0; g < gcount; ++g) {
      const int64_t* fin = finish + (int64_t)g * N;
      unsigned long long* wm = wfmax + (int64_t)g * WF;
      for (int u = lane; u < N; u += 64) {
        const unsigned long long f = (unsigned long long)fin[u];
        atomicMax(&acc[g].max_finish, f);
        atomicMax(&wm[w.act_wf[u]], f);
      }
      __syncthreads();
      // nearest-rank p95: the k-th smallest completion latency, k = ceil(0.95 W)
      const int kk = (95 * WF + 99) / 100;
      for (int a = lane; a < WF; a += 64) {
        const int64_t ca = (int64_t)wm[a] - w.arrival[a];
        int lt = 0, le = 0;
        for (int b = 0; b < WF; ++b) {
          const int64_t cb = (int64_t)wm[b] - w.arrival[b];
          lt += cb < ca;
          le += cb <= ca;
        }
        if (lt < kk && kk <= le) acc[g].p95 = ca;
      }
      __syncthreads();
    }
    if (lane < gcount) {
      const PlanAcc a = acc[lane];
      wf_plan_score sc;
      if (a.status & WF_ST_INELIGIBLE) {
        sc.makespan_us = 0;
        sc.p95_us = 0;
        sc.objective = 0.0f;
        sc.status = WF_ST_INELIGIBLE;
        sc.min_headroom_mib = 0;
        sc.n_loads = 0;
        sc.n_evicts = 0;
      } else {
        const int64_t mk = N > 0 ? (int64_t)a.max_finish - w.min_arrival : 0;
        const int64_t p95 = WF > 0 ? (int64_t)a.p95 : 0;
        const float fa = (float)mk;
        const float fb = (float)p95;
        const float x = w.w_mk * fa;
        const float y = w.w_p95 * fb;
        sc.makespan_us = mk;
        sc.p95_us = p95;
        sc.objective = x + y;
        sc.status = a.status;
        sc.min_headroom_mib = a.headroom;
        sc.n_loads = (uint16_t)(a.loads > 65535u ? 65535u : a.loads);
        sc.n_evicts = (uint16_t)(a.evicts > 65535u ? 65535u : a.evicts);
      }
      scores[p0 + lane] = sc;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_score(const WindowDev& w, const ScoreLaunch& L, int64_t* scratch,
                        const int8_t* dev, const uint16_t* prio, const uint8_t* flags,
                        int64_t n_plans, wf_plan_score* scores, const wf_plan_sched* sched,
                        hipStream_t stream) {
  wf_plan_sched s{};
  if (sched) s = *sched;
  const int has = sched != nullptr;
  // allow the dynamic LDS request (no-op when it is below the default limit)
  (void)hipFuncSetAttribute(L.big ? reinterpret_cast<const void*>(&score_plans<true>)
                                  : reinterpret_cast<const void*>(&score_plans<false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, L.lds_bytes);
  if (L.big)
    hipLaunchKernelGGL(score_plans<true>, dim3(L.grid), dim3(64), L.lds_bytes, stream, w, L,
                       scratch, dev, prio, flags, n_plans, scores, s, has);
  else
    hipLaunchKernelGGL(score_plans<false>, dim3(L.grid), dim3(64), L.lds_bytes, stream, w, L,
                       scratch, dev, prio, flags, n_plans, scores, s, has);
  return hipGetLastError();
}

}  // namespace wfp
