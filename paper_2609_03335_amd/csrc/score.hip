// Batched scoring of candidate physical execution plans on gfx950.
//
// A workgroup of several waves first copies the window's table image into
// LDS (shared by its waves).  Each wave then loops over groups of G plans
// (persistent grid) and, per group:
//   1. stages the G packed device rows and flag rows into its own LDS
//      region with 16-byte loads (priorities are read once, from HBM);
//   2. counts unit heads per (device, model) -- the remaining uses that the
//      reclamation rule consults (lanes over activations);
//   3. for every topological level, per plan (lanes over activations):
//        - each unit head's slot in the resource order (priority, index)
//          (Eq. 10): its priority minus the level's first index when the
//          level's head priorities are distinct values in range (the
//          permutation case), else its rank by (priority, index);
//        - releases r = max(arrival, latest predecessor finish) (Eq. 2): one
//          lane per incoming edge, an LDS atomic max on order-preserving
//          time bits;
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

// Copy nbytes from HBM with the widest aligned accesses.
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

__device__ __forceinline__ int fuse_bit(const uint8_t* fl, int v) {
  return (fl[v >> 2] >> ((v & 3) << 1)) & 1;
}

// slot entry: activation | model << 16 | prefetch << 22 | has fused successor << 23
constexpr uint32_t kPf = 1u << 22;
constexpr uint32_t kChain = 1u << 23;

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
            NWA = sp.nwa;
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
  const uint32_t* t_alv = reinterpret_cast<const uint32_t*>(tb + sp.t.alv);
  const TB* t_aarr = reinterpret_cast<const TB*>(tb + sp.t.aarr);
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
  const uint32_t* t_sink = reinterpret_cast<const uint32_t*>(tb + sp.t.sink);

  // ---- this wave's region (LDS, or HBM scratch for very large windows) ----
  unsigned char* wl;
  if constexpr (WAVE_GLOBAL)
    wl = sp.scratch + ((int64_t)blockIdx.x * sp.waves + wid) * (int64_t)sp.wo.bytes;
  else
    wl = lds + wave_base + wid * sp.wo.bytes;
  uint8_t* s_fl = reinterpret_cast<uint8_t*>(wl + sp.wo.flags);
  uint32_t* s_rec = reinterpret_cast<uint32_t*>(wl + sp.wo.rec);
  unsigned long long* s_mask = reinterpret_cast<unsigned long long*>(wl + sp.wo.mask);
  unsigned long long* s_claim = reinterpret_cast<unsigned long long*>(wl + sp.wo.claim);
  uint32_t* s_cnt = reinterpret_cast<uint32_t*>(wl + sp.wo.cnt);
  TB* s_fin = reinterpret_cast<TB*>(wl + sp.wo.fin);
  PlanAcc* s_acc = reinterpret_cast<PlanAcc*>(wl + sp.wo.acc);
  int8_t* s_dev = reinterpret_cast<int8_t*>(wl + sp.wo.dev);
  uint16_t* s_prio = reinterpret_cast<uint16_t*>(wl + sp.wo.prio);
  TB* s_rt = reinterpret_cast<TB*>(wl + sp.wo.rt);
  uint16_t* s_stamp = reinterpret_cast<uint16_t*>(wl + sp.wo.stamp);
  TB* s_wfm = reinterpret_cast<TB*>(wl + sp.wo.wfm);

  const int g_me = lane / D;
  const int d_me = lane - g_me * D;
  const int64_t n_groups = (P + G - 1) / G;
  const int64_t stride = (int64_t)gridDim.x * sp.waves;

  for (int64_t grp = (int64_t)blockIdx.x * sp.waves + wid; grp < n_groups; grp += stride) {
    const int64_t p0 = grp * G;
    const int gc = (int)((P - p0) < G ? (P - p0) : G);

    // ---- stage the group's rows ----
    stage(reinterpret_cast<unsigned char*>(s_dev),
          reinterpret_cast<const unsigned char*>(dev_all + p0 * N), gc * N, lane);
    stage(reinterpret_cast<unsigned char*>(s_prio),
          reinterpret_cast<const unsigned char*>(prio_all + p0 * N), gc * N * 2, lane);
    stage(s_fl, flags_all + p0 * NB, gc * NB, lane);
    for (int i = lane; i < G * D * MH; i += 64) s_cnt[i] = 0u;
    for (int i = lane; i < G * D * NWA; i += 64) s_mask[i] = 0ull;
    for (int i = lane; i < G * NWA; i += 64) s_claim[i] = 0ull;
    if (lane < G) {
      s_acc[lane].status = 0u;
      s_acc[lane].headroom = 0x7fffffff;
      s_acc[lane].loads = 0u;
      s_acc[lane].evicts = 0u;
      s_acc[lane].max_finish = 0ull;
      s_acc[lane].p95 = 0;
    }
    wave_sync();

    // ---- resource order of every unit head, remaining uses per (device, model) ----
    for (int g = 0; g < gc; ++g) {
      const int8_t* pdev = s_dev + g * N;
      const uint16_t* pprio = s_prio + g * N;
      const uint8_t* pfl = s_fl + g * NB;
      uint32_t* cnt = s_cnt + g * D * MH;
      uint32_t* rec = s_rec + g * N;
      unsigned long long* mk = s_mask + g * D * NWA;
      unsigned long long* cl = s_claim + g * NWA;
      int bad = 0;
      for (int u = lane; u < N; u += 64) {
        const uint32_t a = t_act[u];
        const int fb = pfl[u >> 2] >> ((u & 3) << 1);
        if ((fb & 1) && (a & 64u)) continue;  // chain member
        const int d = pdev[u];
        if ((unsigned)d >= (unsigned)D) {
          atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
          continue;
        }
        const int m = (int)(a & 63u);
        atomicAdd(&cnt[d * MH + (m >> 1)], 1u << ((m & 1) << 4));
        // fast path: the slot is the priority when the level's head
        // priorities are distinct values in the level's index range
        const uint32_t lvw = t_alv[u];
        const int slot = (int)pprio[u];
        if ((unsigned)(slot - (int)(lvw & 0xffffu)) >= (lvw >> 16)) {
          bad = 1;
          continue;
        }
        const unsigned long long bit = 1ull << (slot & 63);
        if (atomicOr(&cl[slot >> 6], bit) & bit) {
          bad = 1;
          continue;
        }
        const int c = t_cnext[u];
        const uint32_t chain = (c != 0xffff && fuse_bit(pfl, c)) ? kChain : 0u;
        rec[slot] = (uint32_t)u | ((a & 63u) << 16) | ((uint32_t)((fb >> 1) & 1) << 22) | chain;
        atomicOr(&mk[d * NWA + (slot >> 6)], bit);
      }
      if (__any(bad)) {  // general path: rank by (priority, index) within each level
        wave_sync();
        for (int i = lane; i < D * NWA; i += 64) mk[i] = 0ull;
        wave_sync();
        for (int u = lane; u < N; u += 64) {
          const uint32_t a = t_act[u];
          const int fb = pfl[u >> 2] >> ((u & 3) << 1);
          if ((fb & 1) && (a & 64u)) continue;
          const int d = pdev[u];
          if ((unsigned)d >= (unsigned)D) continue;
          const uint32_t lvw = t_alv[u];
          const int lo = (int)(lvw & 0xffffu), hi = lo + (int)(lvw >> 16);
          const int pu = pprio[u];
          int slot = lo;
          for (int j = lo; j < hi; ++j) {
            if (fuse_bit(pfl, j) && (t_act[j] & 64u)) continue;
            if ((unsigned)pdev[j] >= (unsigned)D) continue;
            const int pj = pprio[j];
            slot += (pj < pu) || (pj == pu && j < u);
          }
          const int c = t_cnext[u];
          const uint32_t chain = (c != 0xffff && fuse_bit(pfl, c)) ? kChain : 0u;
          rec[slot] = (uint32_t)u | ((a & 63u) << 16) | ((uint32_t)((fb >> 1) & 1) << 22) | chain;
          atomicOr(&mk[d * NWA + (slot >> 6)], 1ull << (slot & 63));
        }
      }
    }
    wave_sync();

    // ---- device-lane state (the staged rows are dead from here on) ----
    for (int i = lane; i < G * W; i += 64) s_wfm[i] = 0;
    const bool act = g_me < gc;
    const int gme = act ? g_me : 0;
    const int64_t pw = p0 + gme;
    uint32_t* mycnt = s_cnt + (gme * D + d_me) * MH;
    uint16_t* mystamp = s_stamp + (gme * D + d_me) * M;
    const unsigned long long* mymask = s_mask + (gme * D + d_me) * NWA;
    const uint32_t* myrec = s_rec + gme * N;
    const TB* myrt = s_rt + gme * WMAX;
    TB* myfin = s_fin + gme * N;
    const uint8_t* myfl = s_fl + gme * NB;
    uint64_t res = 0;
    int32_t used = 0, peak = 0, capd = 0;
    TT freet = 0;
    uint32_t nld = 0, nev = 0, capbad = 0, inel = 0;
    uint32_t seq = 1;
    // reclamation queues (at most 16 models): resident models with no
    // remaining use on this device (qd) and with remaining uses (qa), each in
    // least-recently-used order (never used: by id), 4 bits per entry, next
    // victim in the low bits; a victim comes from qd first
    uint64_t qd = 0, qa = 0;
    int nd = 0, na = 0;
    if (act) {
      res = t_res0[d_me];
      capd = t_cap[d_me];
      freet = TO::load(t_free0 + d_me);
      for (uint64_t r = res; r; r &= r - 1) {
        const int m = __builtin_ctzll(r);
        used += t_wmib[m];
        if constexpr (NIBBLE) {
          if (((mycnt[m >> 1] >> ((m & 1) << 4)) & 0xffffu) == 0u) {
            qd |= (uint64_t)m << (4 * nd);
            ++nd;
          } else {
            qa |= (uint64_t)m << (4 * na);
            ++na;
          }
        } else {
          mystamp[m] = 0;
        }
      }
      peak = used;
    }

    for (int lv = 0; lv < sp.n_levels; ++lv) {
      const int lo = t_loff[lv], hi = t_loff[lv + 1], wlv = hi - lo;
      const int e0 = t_eoff[lv], e1 = t_eoff[lv + 1];
      // ---- latest predecessor finish of the level's activations (Eq. 2) ----
      if (e1 > e0) {
        for (int g = 0; g < gc; ++g) {
          TB* rt = s_rt + g * WMAX;
          for (int i = lane; i < wlv; i += 64) rt[i] = 0;
          wave_sync();
          const TB* fin = s_fin + g * N;
          for (int e = e0 + lane; e < e1; e += 64) {
            const uint32_t ed = t_edge[e];
            atomicMax(&rt[(int)(ed >> 16) - lo], fin[ed & 0xffffu]);
          }
        }
        wave_sync();
      }

      // ---- device lanes walk their units of this level in slot order ----
      if (act) {
        const int d = d_me;
        const int j0 = lo >> 6, j1 = (hi - 1) >> 6;
        for (int j = j0; j <= j1; ++j) {
          unsigned long long bits = mymask[j];
          if (j == j0) bits &= ~0ull << (lo & 63);
          if (j == j1 && (hi & 63)) bits &= (1ull << (hi & 63)) - 1ull;
          while (bits) {
            const int slot = (j << 6) + __builtin_ctzll(bits);
            bits &= bits - 1;
            const uint32_t meta = myrec[slot];
            const int u = (int)(meta & 0xffffu);
            const int m = (int)((meta >> 16) & 63u);
            const TT arrv = TO::load(t_aarr + u);
            const TT r = (e1 > e0) ? TO::tmax(TO::load(myrt + (u - lo)), arrv) : arrv;
            // run time (summed over a fused chain, Eq. 4) and memory (max)
            const int32_t l0 = t_lat[u * D + d];
            int32_t mxu = t_mem[u * sp.mem_si + d * sp.mem_sd];
            inel |= (uint32_t)(l0 < 0);
            uint32_t T = (uint32_t)l0;
            if (meta & kChain) {
              for (int v = t_cnext[u];;) {
                const int32_t lv2 = t_lat[v * D + d];
                const int32_t mv = t_mem[v * sp.mem_si + d * sp.mem_sd];
                inel |= (uint32_t)(lv2 < 0);
                T += (uint32_t)lv2;
                mxu = mv > mxu ? mv : mxu;
                const int c = t_cnext[v];
                if (c == 0xffff || !fuse_bit(myfl, c)) break;
                v = c;
              }
            }
            // one remaining use of m on this device consumed
            const int sh = (m & 1) << 4;
            const uint32_t cword = mycnt[m >> 1] - (1u << sh);
            mycnt[m >> 1] = cword;
            const bool last_use = ((cword >> sh) & 0xffffu) == 0u;
            const uint64_t mb = 1ull << m;
            const bool hit = (res & mb) != 0ull;
            const int32_t wm = t_wmib[m];
            const int32_t need = (hit ? 0 : wm) + mxu;
            // reclaim (Sec. 3.5): a copy with no remaining use first, else the
            // least recently used, else the lower model id
            if constexpr (NIBBLE) {
              if (hit) {  // m is in qa: take it out, it re-enters as most recent
                const uint64_t x = qa ^ (0x1111111111111111ull * (uint64_t)m);
                const uint64_t z = (x - 0x1111111111111111ull) & ~x & 0x8888888888888888ull;
                const int s4 = __builtin_ctzll(z) & ~3;  // 4 * position
                const uint64_t low = qa & ((1ull << s4) - 1ull);
                const uint64_t high = (s4 >= 60) ? 0ull : ((qa >> (s4 + 4)) << s4);
                qa = low | high;
                --na;
              }
              while (used + need > capd && (nd | na)) {
                int v;
                if (nd) {
                  v = (int)(qd & 15ull);
                  qd >>= 4;
                  --nd;
                } else {
                  v = (int)(qa & 15ull);
                  qa >>= 4;
                  --na;
                }
                res &= ~(1ull << v);
                used -= t_wmib[v];
                ++nev;
              }
              if (last_use) {
                qd |= (uint64_t)m << (4 * nd);
                ++nd;
              } else {
                qa |= (uint64_t)m << (4 * na);
                ++na;
              }
            } else {
              while (used + need > capd) {
                uint64_t cand = res & ~mb;
                if (!cand) break;
                int v = 0;
                uint32_t best = 0xffffffffu;
                while (cand) {
                  const int m2 = __builtin_ctzll(cand);
                  cand &= cand - 1;
                  const uint32_t alive = ((mycnt[m2 >> 1] >> ((m2 & 1) << 4)) & 0xffffu) != 0u;
                  const uint32_t key = (alive << 16) | mystamp[m2];
                  if (key < best) {
                    best = key;
                    v = m2;
                  }
                }
                res &= ~(1ull << v);
                used -= t_wmib[v];
                ++nev;
              }
              mystamp[m] = (uint16_t)seq++;
            }
            capbad |= (uint32_t)(used + need > capd);
            // timeline (Eq. 7): a load waits for the device and starts at the
            // release, or at the workflow arrival when prefetched
            const TT ls = TO::tmax((meta & kPf) ? arrv : r, freet);
            const TT le = TO::add(ls, (uint32_t)t_load[m * D + d]);
            const TT s = TO::tmax(r, hit ? freet : le);
            if (!hit) {
              res |= mb;
              used += wm;
              ++nld;
            }
            peak = (used + mxu) > peak ? (used + mxu) : peak;
            const TT f = TO::add(s, T);
            freet = f;
            if (!(meta & kChain)) {
              myfin[u] = TO::bits(f);
              if (has_sched) {
                sched.start_us[pw * N + u] = sp.origin + TO::i64(s);
                sched.finish_us[pw * N + u] = sp.origin + TO::i64(f);
                sched.load_start_us[pw * N + u] = hit ? (int64_t)-1 : sp.origin + TO::i64(ls);
              }
            } else {
              TT t = s;
              for (int v = u;;) {
                const TT tv = TO::add(t, (uint32_t)t_lat[v * D + d]);
                myfin[v] = TO::bits(tv);
                if (has_sched) {
                  sched.start_us[pw * N + v] = sp.origin + TO::i64(t);
                  sched.finish_us[pw * N + v] = sp.origin + TO::i64(tv);
                  sched.load_start_us[pw * N + v] =
                      (v == u && !hit) ? sp.origin + TO::i64(ls) : (int64_t)-1;
                }
                t = tv;
                const int c = t_cnext[v];
                if (c == 0xffff || !fuse_bit(myfl, c)) break;
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
      if (inel) atomicOr(&s_acc[gme].status, (uint32_t)WF_ST_INELIGIBLE);
      if (has_sched) sched.peak_mib[pw * D + d_me] = peak;
    }
    // a workflow's completion is the latest finish among its activations
    // without a successor in the same workflow
    for (int g = 0; g < gc; ++g) {
      const TB* fin = s_fin + g * N;
      TB* wm = s_wfm + g * W;
      for (int i = lane; i < sp.S; i += 64) {
        const uint32_t sk = t_sink[i];
        atomicMax(&wm[sk >> 16], fin[sk & 0xffffu]);
      }
    }
    wave_sync();
    // nearest-rank p95 (the ceil(0.95 W)-th smallest completion latency) and
    // the latest finish, lanes over (plan, workflow)
    const int kk = (95 * W + 99) / 100;
    for (int it = lane; it < gc * W; it += 64) {
      const int g = it / W, a = it - g * W;
      const TB* wm = s_wfm + g * W;
      const TT fa = TO::load(wm + a);
      const int64_t ca = TO::i64(fa) - TO::i64(TO::load(t_arr + a));
      int lt = 0, le = 0;
      for (int b = 0; b < W; ++b) {
        const int64_t cb = TO::i64(TO::load(wm + b)) - TO::i64(TO::load(t_arr + b));
        lt += cb < ca;
        le += cb <= ca;
      }
      if (lt < kk && kk <= le) s_acc[g].p95 = ca;
      atomicMax(&s_acc[g].max_finish, (unsigned long long)TO::bits(fa));
    }
    wave_sync();
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
