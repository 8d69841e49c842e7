// Batched scoring of candidate physical execution plans on gfx950.
//
// A workgroup of several waves first copies the window's table image into
// LDS (shared by its waves).  Each wave then loops over groups of G plans
// (persistent grid) and, per group:
//   1. stages the G packed plan rows (device, priority, fuse/prefetch bits)
//      into its own LDS region with 16-byte loads;
//   2. counts unit heads per (device, model) -- the remaining uses that the
//      reclamation rule consults (lanes over activations);
//   3. for every topological level, per plan (lanes over activations):
//        - releases r = max(arrival, latest predecessor finish) (Eq. 2), one
//          lane per incoming edge, as an LDS atomic max on order-preserving
//          time bits;
//        - each unit head's slot in the resource order (priority, index)
//          (Eq. 10): its priority minus the level's first index when the
//          level's head priorities are distinct values in range (the common,
//          permutation case), else its rank by (priority, index);
//        - the unit record at that slot: fused-chain run time (Eq. 4),
//          chain memory maximum, model, prefetch bit, workflow;
//      then lane (g, d) = (lane / D, lane % D) walks device d of plan g over
//      the level's slots in order: reuse / reclaim / load (Eq. 5, Eq. 11)
//      and the max-plus timeline of Eq. 7;
//   4. reduces makespan, nearest-rank p95, objective and headroom.
// Residency, reclamation and memory depend only on each device's unit
// sequence, never on times, so device lanes are independent within a level;
// every predecessor sits at a lower level, so releases are final when a
// level starts.
//
// Times are relative to the window origin (earliest arrival or free time):
// uint32 when the host has proven no time of any plan can reach 2^32, else
// fp64 (every time is an integer below 2^53, so fp64 max/add are exact).
#include "kernels.h"

namespace wfp {
namespace {

template <typename TT>
struct TimeOps;

template <>
struct TimeOps<uint32_t> {
  using bits_t = uint32_t;
  __device__ static uint32_t load(const bits_t* p) { return *p; }
  __device__ static bits_t bits(uint32_t t) { return t; }
  __device__ static uint32_t tmax(uint32_t a, uint32_t b) { return a > b ? a : b; }
  __device__ static uint32_t add(uint32_t a, uint32_t d) { return a + d; }
  __device__ static int64_t i64(uint32_t t) { return (int64_t)t; }
};

template <>
struct TimeOps<double> {
  using bits_t = unsigned long long;
  __device__ static double load(const bits_t* p) { return __longlong_as_double((long long)*p); }
  __device__ static bits_t bits(double t) { return (bits_t)__double_as_longlong(t); }
  __device__ static double tmax(double a, double b) { return fmax(a, b); }
  __device__ static double add(double a, uint32_t d) { return a + (double)d; }
  __device__ static int64_t i64(double t) { return (int64_t)t; }
};

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Copy nbytes from HBM to LDS with the widest aligned accesses.
__device__ __forceinline__ void stage(unsigned char* dst, const unsigned char* src, int nbytes,
                                      int lane) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(src);
  if (((a | (uintptr_t)nbytes) & 15) == 0) {
    const uint4* s = reinterpret_cast<const uint4*>(src);
    uint4* d = reinterpret_cast<uint4*>(dst);
    for (int i = lane; i < (nbytes >> 4); i += 64) d[i] = s[i];
  } else if (((a | (uintptr_t)nbytes) & 3) == 0) {
    const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
    uint32_t* d = reinterpret_cast<uint32_t*>(dst);
    for (int i = lane; i < (nbytes >> 2); i += 64) d[i] = s[i];
  } else {
    for (int i = lane; i < nbytes; i += 64) dst[i] = src[i];
  }
}

template <typename TT, bool TAB_LDS, bool NIBBLE, bool WAVE_GLOBAL>
__global__ __launch_bounds__(512) void score_plans(ScoreParams sp,
                                                   const int8_t* __restrict__ dev_all,
                                                   const uint16_t* __restrict__ prio_all,
                                                   const uint8_t* __restrict__ flags_all, int64_t P,
                                                   wf_plan_score* __restrict__ scores,
                                                   wf_plan_sched sched, int has_sched) {
  using TO = TimeOps<TT>;
  using TB = typename TO::bits_t;
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int N = sp.N, W = sp.W, M = sp.M, D = sp.D, NB = sp.NB, G = sp.G, WMAX = sp.wmax,
            NW = sp.nwords;
  const int MH = (M + 1) >> 1;

  // ---- window tables ----
  const unsigned char* tb;
  int wave_base;
  if constexpr (TAB_LDS) {
    const uint4* src = reinterpret_cast<const uint4*>(sp.tab);
    uint4* dst = reinterpret_cast<uint4*>(lds);
    for (int i = tid; i < (sp.t.bytes >> 4); i += blockDim.x) dst[i] = src[i];
    __syncthreads();
    tb = lds;
    wave_base = sp.t.bytes;
  } else {
    tb = sp.tab;
    wave_base = 0;
  }
  const uint32_t* t_act = reinterpret_cast<const uint32_t*>(tb + sp.t.act);
  const uint16_t* t_cnext = reinterpret_cast<const uint16_t*>(tb + sp.t.cnext);
  const uint32_t* t_edge = reinterpret_cast<const uint32_t*>(tb + sp.t.edge);
  const int32_t* t_eoff = reinterpret_cast<const int32_t*>(tb + sp.t.eoff);
  const int32_t* t_loff = reinterpret_cast<const int32_t*>(tb + sp.t.loff);
  const int32_t* t_lat = reinterpret_cast<const int32_t*>(tb + sp.t.lat);
  const int32_t* t_mem = reinterpret_cast<const int32_t*>(tb + sp.t.mem);
  const int32_t* t_load = reinterpret_cast<const int32_t*>(tb + sp.t.load);
  const int32_t* t_wmib = reinterpret_cast<const int32_t*>(tb + sp.t.wmib);
  const int32_t* t_cap = reinterpret_cast<const int32_t*>(tb + sp.t.cap);
  const TB* t_arr = reinterpret_cast<const TB*>(tb + sp.t.arr);
  const unsigned long long* t_res0 = reinterpret_cast<const unsigned long long*>(tb + sp.t.res0);
  const TB* t_free0 = reinterpret_cast<const TB*>(tb + sp.t.free0);

  // ---- this wave's region (LDS, or HBM scratch for very large windows) ----
  unsigned char* wl;
  if constexpr (WAVE_GLOBAL)
    wl = sp.scratch + ((int64_t)blockIdx.x * sp.waves + wid) * (int64_t)sp.wo.bytes;
  else
    wl = lds + wave_base + wid * sp.wo.bytes;
  int8_t* s_dev = reinterpret_cast<int8_t*>(wl + sp.wo.dev);
  uint16_t* s_prio = reinterpret_cast<uint16_t*>(wl + sp.wo.prio);
  uint8_t* s_fl = reinterpret_cast<uint8_t*>(wl + sp.wo.flags);
  TB* s_fin = reinterpret_cast<TB*>(wl + sp.wo.fin);
  TB* s_rt = reinterpret_cast<TB*>(wl + sp.wo.rt);
  uint4* s_rec = reinterpret_cast<uint4*>(wl + sp.wo.rec);
  unsigned long long* s_claim = reinterpret_cast<unsigned long long*>(wl + sp.wo.claim);
  unsigned long long* s_mask = reinterpret_cast<unsigned long long*>(wl + sp.wo.mask);
  uint32_t* s_cnt = reinterpret_cast<uint32_t*>(wl + sp.wo.cnt);
  int32_t* s_last = reinterpret_cast<int32_t*>(wl + sp.wo.last);
  TB* s_wfm = reinterpret_cast<TB*>(wl + sp.wo.wfm);
  PlanAcc* s_acc = reinterpret_cast<PlanAcc*>(wl + sp.wo.acc);

  const int g_me = lane / D;
  const int d_me = lane - g_me * D;
  const int64_t n_groups = (P + G - 1) / G;
  const int64_t stride = (int64_t)gridDim.x * sp.waves;

  for (int64_t grp = (int64_t)blockIdx.x * sp.waves + wid; grp < n_groups; grp += stride) {
    const int64_t p0 = grp * G;
    const int gc = (int)((P - p0) < G ? (P - p0) : G);

    // ---- stage the group's plan rows ----
    stage(reinterpret_cast<unsigned char*>(s_dev),
          reinterpret_cast<const unsigned char*>(dev_all + p0 * N), gc * N, lane);
    stage(reinterpret_cast<unsigned char*>(s_prio),
          reinterpret_cast<const unsigned char*>(prio_all + p0 * N), gc * N * 2, lane);
    stage(s_fl, flags_all + p0 * NB, gc * NB, lane);
    for (int i = lane; i < G * D * MH; i += 64) s_cnt[i] = 0u;
    if constexpr (!NIBBLE)
      for (int i = lane; i < G * D * M; i += 64) s_last[i] = -1;
    for (int i = lane; i < G * W; i += 64) s_wfm[i] = 0;
    if (lane < G) {
      s_acc[lane].status = 0u;
      s_acc[lane].headroom = 0x7fffffff;
      s_acc[lane].loads = 0u;
      s_acc[lane].evicts = 0u;
      s_acc[lane].max_finish = 0ull;
      s_acc[lane].p95 = 0;
    }
    wave_sync();

    // ---- unit heads per (device, model): remaining uses ----
    for (int g = 0; g < gc; ++g) {
      const int8_t* pdev = s_dev + g * N;
      const uint8_t* pfl = s_fl + g * NB;
      for (int u = lane; u < N; u += 64) {
        const uint32_t a = t_act[u];
        if (((pfl[u >> 2] >> ((u & 3) << 1)) & 1) && (a & 64u)) continue;  // chain member
        const int d = pdev[u];
        if ((unsigned)d >= (unsigned)D) {
          atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
          continue;
        }
        const int m = (int)(a & 63u);
        atomicAdd(&s_cnt[(g * D + d) * MH + (m >> 1)], 1u << ((m & 1) << 4));
      }
    }
    wave_sync();

    // ---- device-lane state ----
    const bool act = g_me < gc;
    const int gme = act ? g_me : 0;
    const int64_t pw = p0 + gme;
    const int cbase = (gme * D + d_me) * MH;
    const int lbase = (gme * D + d_me) * M;
    uint64_t res = 0;
    int32_t used = 0, peak = 0, capd = 0;
    TT freet = 0;
    uint32_t nld = 0, nev = 0, capbad = 0;
    int32_t seq = 0;
    uint64_t Q = 0;  // reclamation queue, 4 bits per resident model, next victim lowest
    int qlen = 0, qdead = 0;
    if (act) {
      res = t_res0[d_me];
      capd = t_cap[d_me];
      freet = TO::load(t_free0 + d_me);
      for (int m = 0; m < M; ++m)
        if ((res >> m) & 1ull) used += t_wmib[m];
      peak = used;
      if constexpr (NIBBLE) {
        // models with no use on this device first (least recently used = by
        // id), then the ones still needed (also by id)
        for (int pass = 0; pass < 2; ++pass)
          for (int m = 0; m < M; ++m) {
            if (!((res >> m) & 1ull)) continue;
            const uint32_t c = (s_cnt[cbase + (m >> 1)] >> ((m & 1) << 4)) & 0xffffu;
            if ((c == 0u) == (pass == 0)) {
              Q |= (uint64_t)m << (4 * qlen);
              ++qlen;
            }
          }
        for (int m = 0; m < M; ++m)
          if (((res >> m) & 1ull) && ((s_cnt[cbase + (m >> 1)] >> ((m & 1) << 4)) & 0xffffu) == 0u)
            ++qdead;
      }
    }

    for (int lv = 0; lv < sp.n_levels; ++lv) {
      const int lo = t_loff[lv], hi = t_loff[lv + 1], wlv = hi - lo, nwl = (wlv + 63) >> 6;
      const int e0 = t_eoff[lv], e1 = t_eoff[lv + 1];

      for (int g = 0; g < gc; ++g) {
        TB* rt = s_rt + g * WMAX;
        uint4* rec = s_rec + g * WMAX;
        unsigned long long* cl = s_claim + g * NW;
        unsigned long long* mk = s_mask + g * D * NW;
        const TB* fin = s_fin + g * N;
        const int8_t* pdev = s_dev + g * N;
        const uint16_t* pprio = s_prio + g * N;
        const uint8_t* pfl = s_fl + g * NB;
        for (int i = lane; i < wlv; i += 64) rt[i] = 0;
        for (int i = lane; i < nwl; i += 64) cl[i] = 0ull;
        for (int i = lane; i < D * nwl; i += 64) mk[(i / nwl) * NW + (i % nwl)] = 0ull;
        wave_sync();
        // releases: latest predecessor finish (Eq. 2)
        for (int e = e0 + lane; e < e1; e += 64) {
          const uint32_t ed = t_edge[e];
          atomicMax(&rt[(int)(ed >> 16) - lo], fin[ed & 0xffffu]);
        }
        // slots in the resource order and unit records
        for (int pass = 0; pass < 2; ++pass) {
          int bad = 0;
          for (int u = lo + lane; u < hi; u += 64) {
            const uint32_t a = t_act[u];
            const int flb = pfl[u >> 2] >> ((u & 3) << 1);
            if ((flb & 1) && (a & 64u)) continue;  // chain member
            const int d = pdev[u];
            if ((unsigned)d >= (unsigned)D) continue;
            const int pu = pprio[u];
            int k = pu - lo;
            if (pass == 0) {
              if ((unsigned)k >= (unsigned)wlv) {
                bad = 1;
                continue;
              }
              const unsigned long long bit = 1ull << (k & 63);
              if (atomicOr(&cl[k >> 6], bit) & bit) {
                bad = 1;
                continue;
              }
            } else {
              k = 0;  // rank by (priority, index) among the level's heads
              for (int j = lo; j < hi; ++j) {
                const uint32_t aj = t_act[j];
                if (((pfl[j >> 2] >> ((j & 3) << 1)) & 1) && (aj & 64u)) continue;
                if ((unsigned)pdev[j] >= (unsigned)D) continue;
                const int pj = pprio[j];
                k += (pj < pu) || (pj == pu && j < u);
              }
            }
            // unit record: fused chain (Eq. 4), run time sum, memory max
            uint32_t T = 0, mx = 0;
            int inel = 0, chain = 0;
            for (int v = u;;) {
              const int32_t l = t_lat[v * D + d];
              inel |= l < 0;
              T += (uint32_t)l;
              const uint32_t mv = (uint32_t)t_mem[v * sp.mem_si + d * sp.mem_sd];
              mx = mv > mx ? mv : mx;
              const int c = t_cnext[v];
              if (c == 0xffff || !((pfl[c >> 2] >> ((c & 3) << 1)) & 1)) break;
              v = c;
              chain = 1;
            }
            if (inel) atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
            const uint32_t meta = (uint32_t)u | ((a & 63u) << 16) | ((uint32_t)((flb >> 1) & 1) << 22) |
                                  ((uint32_t)chain << 23);
            rec[k] = make_uint4(T, mx, meta, a >> 16);
            atomicOr(&mk[d * NW + (k >> 6)], 1ull << (k & 63));
            atomicMax(&rt[u - lo], t_arr[a >> 16]);
          }
          if (pass == 0) {
            if (!__any(bad)) break;
            wave_sync();
            for (int i = lane; i < D * nwl; i += 64) mk[(i / nwl) * NW + (i % nwl)] = 0ull;
          }
          wave_sync();
        }
      }
      wave_sync();

      // ---- device lanes walk their units of this level in slot order ----
      if (act) {
        const uint4* rec = s_rec + gme * WMAX;
        const TB* rt = s_rt + gme * WMAX;
        const unsigned long long* mk = s_mask + (gme * D + d_me) * NW;
        TB* fin = s_fin + gme * N;
        const uint8_t* pfl = s_fl + gme * NB;
        const int d = d_me;
        for (int j = 0; j < nwl; ++j) {
          unsigned long long bits = mk[j];
          while (bits) {
            const int k = (j << 6) + __builtin_ctzll(bits);
            bits &= bits - 1;
            const uint4 rc = rec[k];
            const int u = (int)(rc.z & 0xffffu);
            const int m = (int)((rc.z >> 16) & 63u);
            const TT r = TO::load(rt + (u - lo));
            // one remaining use of m on this device consumed
            uint32_t* cw = &s_cnt[cbase + (m >> 1)];
            const int sh = (m & 1) << 4;
            const uint32_t cword = *cw - (1u << sh);
            *cw = cword;
            const uint64_t mb = 1ull << m;
            const bool miss = !(res & mb);
            const int32_t wm = t_wmib[m];
            const int32_t mxu = (int32_t)rc.y;
            const int32_t need = (miss ? wm : 0) + mxu;
            if constexpr (NIBBLE) {
              if (!miss) {  // take m out of the queue; it re-enters as most recent
                const uint64_t x = Q ^ (0x1111111111111111ull * (uint64_t)m);
                const uint64_t z = (x - 0x1111111111111111ull) & ~x & 0x8888888888888888ull;
                const int pos = __builtin_ctzll(z) >> 2;
                const uint64_t low = (pos == 0) ? 0ull : (Q & ((1ull << (4 * pos)) - 1ull));
                Q = low | ((Q >> (4 * pos + 4)) << (4 * pos));
                --qlen;
              }
              while (used + need > capd && qlen > 0) {  // reclaim the queue head
                const int v = (int)(Q & 15ull);
                Q >>= 4;
                --qlen;
                qdead -= (qdead > 0);
                res &= ~(1ull << v);
                used -= t_wmib[v];
                ++nev;
              }
            } else {
              while (used + need > capd) {
                uint64_t cand = res & ~mb;
                if (!cand) break;
                int victim = 0, v_alive = 2, v_last = 0x7fffffff;
                while (cand) {
                  const int m2 = __builtin_ctzll(cand);
                  cand &= cand - 1;
                  const int al = ((s_cnt[cbase + (m2 >> 1)] >> ((m2 & 1) << 4)) & 0xffffu) != 0u;
                  const int la = s_last[lbase + m2];
                  if (al < v_alive || (al == v_alive && la < v_last)) {
                    victim = m2;
                    v_alive = al;
                    v_last = la;
                  }
                }
                res &= ~(1ull << victim);
                used -= t_wmib[victim];
                ++nev;
              }
            }
            capbad |= (uint32_t)(used + need > capd);
            TT s, ls = 0;
            if (miss) {
              const TT arrv = TO::load(t_arr + rc.w);
              ls = TO::tmax(((rc.z >> 22) & 1u) ? arrv : r, freet);
              const TT le = TO::add(ls, (uint32_t)t_load[m * D + d]);
              res |= mb;
              used += wm;
              ++nld;
              s = TO::tmax(r, le);
            } else {
              s = TO::tmax(r, freet);
            }
            peak = (used + mxu) > peak ? (used + mxu) : peak;
            if constexpr (NIBBLE) {
              if (((cword >> sh) & 0xffffu) == 0u) {  // last use: joins the no-use part
                const uint64_t lowm = (qdead == 0) ? 0ull : ((1ull << (4 * qdead)) - 1ull);
                Q = (Q & lowm) | ((uint64_t)m << (4 * qdead)) | ((Q & ~lowm) << 4);
                ++qdead;
              } else {
                Q |= (uint64_t)m << (4 * qlen);
              }
              ++qlen;
            } else {
              s_last[lbase + m] = seq++;
            }
            const TT f = TO::add(s, rc.x);
            freet = f;
            if (!((rc.z >> 23) & 1u)) {
              fin[u] = TO::bits(f);
              if (has_sched) {
                sched.start_us[pw * N + u] = sp.origin + TO::i64(s);
                sched.finish_us[pw * N + u] = sp.origin + TO::i64(f);
                sched.load_start_us[pw * N + u] = miss ? sp.origin + TO::i64(ls) : (int64_t)-1;
              }
            } else {
              TT t = s;
              for (int v = u;;) {
                const TT tv = TO::add(t, (uint32_t)t_lat[v * D + d]);
                fin[v] = TO::bits(tv);
                if (has_sched) {
                  sched.start_us[pw * N + v] = sp.origin + TO::i64(t);
                  sched.finish_us[pw * N + v] = sp.origin + TO::i64(tv);
                  sched.load_start_us[pw * N + v] =
                      (v == u && miss) ? sp.origin + TO::i64(ls) : (int64_t)-1;
                }
                t = tv;
                const int c = t_cnext[v];
                if (c == 0xffff || !((pfl[c >> 2] >> ((c & 3) << 1)) & 1)) break;
                v = c;
              }
            }
          }
        }
      }
      wave_sync();
    }

    // ---- per-plan reductions (Sec. 4 metrics) ----
    if (act) {
      atomicMin(&s_acc[gme].headroom, capd - peak);
      atomicAdd(&s_acc[gme].loads, nld);
      atomicAdd(&s_acc[gme].evicts, nev);
      if (capbad) atomicOr(&s_acc[gme].status, (uint32_t)WF_ST_CAPACITY);
      if (has_sched) sched.peak_mib[pw * D + d_me] = peak;
    }
    wave_sync();
    for (int g = 0; g < gc; ++g) {
      const TB* fin = s_fin + g * N;
      TB* wm = s_wfm + g * W;
      for (int u = lane; u < N; u += 64) {
        const TB f = fin[u];
        atomicMax(&s_acc[g].max_finish, (unsigned long long)f);
        atomicMax(&wm[t_act[u] >> 16], f);
      }
      wave_sync();
      // nearest-rank p95: the k-th smallest completion latency, k = ceil(0.95 W)
      const int kk = (95 * W + 99) / 100;
      for (int a = lane; a < W; a += 64) {
        const int64_t ca = TO::i64(TO::load(wm + a)) - TO::i64(TO::load(t_arr + a));
        int lt = 0, le = 0;
        for (int b = 0; b < W; ++b) {
          const int64_t cb = TO::i64(TO::load(wm + b)) - TO::i64(TO::load(t_arr + b));
          lt += cb < ca;
          le += cb <= ca;
        }
        if (lt < kk && kk <= le) s_acc[g].p95 = ca;
      }
      wave_sync();
    }
    if (lane < gc) {
      const PlanAcc a = s_acc[lane];
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
        const TT mf = TO::load(reinterpret_cast<const TB*>(&a.max_finish));
        const int64_t mk = N > 0 ? sp.origin + TO::i64(mf) - sp.min_arrival : 0;
        const int64_t p95 = W > 0 ? (int64_t)a.p95 : 0;
        const float fa = (float)mk;
        const float fb = (float)p95;
        const float x = sp.w_mk * fa;
        const float y = sp.w_p95 * fb;
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
    wave_sync();
  }
}

template <typename TT, bool TAB_LDS, bool NIBBLE, bool WAVE_GLOBAL>
hipError_t launch_variant(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                          const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                          const wf_plan_sched& s, int has, hipStream_t stream) {
  auto k = score_plans<TT, TAB_LDS, NIBBLE, WAVE_GLOBAL>;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                            hipFuncAttributeMaxDynamicSharedMemorySize, sp.lds_bytes);
  hipLaunchKernelGGL(k, dim3(sp.grid), dim3(64 * sp.waves), sp.lds_bytes, stream, sp, dev, prio,
                     flags, n_plans, scores, s, has);
  return hipGetLastError();
}

template <typename TT, bool NIBBLE>
hipError_t launch_place(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                        const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                        const wf_plan_sched& s, int has, hipStream_t stream) {
  if (sp.wave_global)
    return launch_variant<TT, false, NIBBLE, true>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
  if (sp.tab_in_lds)
    return launch_variant<TT, true, NIBBLE, false>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
  return launch_variant<TT, false, NIBBLE, false>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
}

template <typename TT>
hipError_t launch_time(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                       const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                       const wf_plan_sched& s, int has, hipStream_t stream) {
  if (sp.nibble) return launch_place<TT, true>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
  return launch_place<TT, false>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
}

}  // namespace

hipError_t launch_score(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                        const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                        const wf_plan_sched* sched, hipStream_t stream) {
  wf_plan_sched s{};
  if (sched) s = *sched;
  const int has = sched != nullptr;
  if (sp.time64) return launch_time<double>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
  return launch_time<uint32_t>(sp, dev, prio, flags, n_plans, scores, s, has, stream);
}

}  // namespace wfp
