// Batched scoring of candidate physical execution plans on gfx950.
//
// A persistent grid of waves loops over groups of G plans; lane (g, d) =
// (lane / D, lane % D) owns device d of plan g.  The window's table image is
// read from LDS (one copy per workgroup) or through the cache.  Per group:
//   1. flag rows are staged into the wave's LDS region; device and priority
//      rows are read four activations per lane (or built in LDS for
//      candidates generated around an incumbent);
//   2. resource order (Eq. 10): each unit head's slot is its priority when
//      every level's head priorities are distinct values in the level's index
//      range (checked by counting heads against distinct slots), else its rank
//      by (priority, index) within the level; slot entries, per-device slot
//      masks and each (device, model)'s last slot are recorded, and the last
//      unit of each model on each device is marked;
//   3. per topological level: releases r = max(arrival, latest predecessor
//      finish) (Eq. 2) by LDS atomic max over the level's incoming edges,
//      accumulated in the finish array itself; then each device lane walks its
//      units of the level in slot order -- reuse / reclaim / load (Eq. 5,
//      Eq. 11) and the max-plus timeline of Eq. 7 -- with everything that
//      does not depend on the device's sequential state loaded a unit ahead;
//   4. makespan, nearest-rank p95, objective, headroom and counts.
// Residency, reclamation and memory depend only on each device's unit
// sequence, never on times, so device lanes are independent within a level;
// every predecessor sits at a lower level, so releases are final when a
// level starts.
//
// Times are relative to the window origin (earliest arrival or free time):
// uint32 or fp64 (every time is an integer below 2^53, so fp64 max/add are
// exact).  uint32 additions saturate; a plan with a saturated time is flagged
// (kRescore) and the host rescores its group in fp64 unless it has proven
// that no time can reach 2^32.
#pragma once

#include <type_traits>

#include "kernels.h"
#include "mutation.h"

namespace wfp {
namespace {

template <typename TT>
struct TimeOps;

template <>
struct TimeOps<uint32_t> {
  using bits_t = uint32_t;
  __device__ static uint32_t load(const bits_t* p) { return *p; }
  __device__ static uint32_t words(uint32_t lo, uint32_t) { return lo; }
  __device__ static bits_t bits(uint32_t t) { return t; }
  __device__ static uint32_t tmax(uint32_t a, uint32_t b) { return a > b ? a : b; }
  // saturating: a time that would pass 2^32 - 1 stays there, and every max
  // and sum that takes it does too, up to the device's last finish
  __device__ static uint32_t add(uint32_t a, uint32_t d) { return __builtin_elementwise_add_sat(a, d); }
  __device__ static uint32_t sub(uint32_t a, uint32_t b) { return a - b; }
  __device__ static int64_t i64(uint32_t t) { return (int64_t)t; }
};

template <>
struct TimeOps<double> {
  using bits_t = unsigned long long;
  __device__ static double load(const bits_t* p) { return __longlong_as_double((long long)*p); }
  __device__ static double words(uint32_t lo, uint32_t hi) {
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
  }
  __device__ static bits_t bits(double t) { return (bits_t)__double_as_longlong(t); }
  __device__ static double tmax(double a, double b) { return fmax(a, b); }
  __device__ static double add(double a, uint32_t d) { return a + (double)d; }
  __device__ static double sub(double a, double b) { return a - b; }
  __device__ static int64_t i64(double t) { return (int64_t)t; }
};

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Zero nbytes at a 16-byte aligned address: 16-byte stores, then the tail.
__device__ __forceinline__ void zero_bytes(unsigned char* dst, int nbytes, int lane) {
  uint4* d = reinterpret_cast<uint4*>(dst);
  const int n16 = nbytes >> 4;
  for (int i = lane; i < n16; i += 64) d[i] = make_uint4(0u, 0u, 0u, 0u);
  for (int i = (n16 << 4) + lane; i < nbytes; i += 64) dst[i] = 0;
}

// Copy nbytes with 4-byte accesses when source, destination and size allow.
__device__ __forceinline__ void copy_row(unsigned char* dst, const unsigned char* src, int nbytes,
                                         int lane) {
  if (((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | (uintptr_t)nbytes) &
       3) == 0) {
    const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
    uint32_t* d = reinterpret_cast<uint32_t*>(dst);
    for (int i = lane; i < (nbytes >> 2); i += 64) d[i] = s[i];
  } else {
    for (int i = lane; i < nbytes; i += 64) dst[i] = src[i];
  }
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

// Candidate c from the incumbent's rows held whole.
__device__ __forceinline__ void mutate(uint64_t c, const SearchArgs& sa, int N,
                                       const unsigned long long* elig, const uint32_t* alv,
                                       int8_t* rd, uint16_t* rp, uint8_t* rf) {
  FullRows rows{rd, rp, rf};
  mutate_rows(c, sa, N, elig, alv, rows);
}

// slot entry: activation | model << 16 | prefetch << 22 | has fused successor << 23 |
// last unit of its model on the device << 30 | finish written by the general
// path (a fused chain, or schedule output requested) << 31
constexpr uint32_t kPf = 1u << 22;
constexpr uint32_t kChain = 1u << 23;
constexpr uint32_t kLast = 1u << 30;
constexpr uint32_t kSlow = 1u << 31;

// What the device walk needs about one unit that does not depend on the
// device's sequential state; it is loaded one unit ahead of its use.
template <typename TT>
struct UnitPre {
  uint32_t meta;  // slot entry
  int slot;       // resource-order slot, -1 past the device's last unit
  TT arrv;        // workflow arrival
  TT rtv;         // latest predecessor finish (0 for a source)
  int32_t lat;    // head run time on the device (-1: ineligible)
  int32_t mem;    // head activation memory on the device
  int2 lw;        // model load time on the device, model weights
  uint32_t act;   // activation word (ranking-key mode only)
};

// SEARCH: plans are candidates generated around the incumbent rows dev_all,
// prio_all, flags_all ([N] each) rather than [P][N] rows read from HBM.
// PHI: each plan's ranking key (Eq. 12) is written instead of its score.
template <bool PHI>
using OutRec = std::conditional_t<PHI, wf_plan_key, wf_plan_score>;

// PLACE: 0 = per-wave regions in LDS, 1 = their per-activation arrays in HBM
// scratch, 2 = the ring of recent levels in LDS (scan reclamation, rows from
// HBM).
// (the HBM layout, PLACE 1, is bound by the latency of its per-activation
// arrays: it is built for three waves per SIMD, four-wave workgroups, three
// per CU, although that spills registers)
template <typename TT, bool TAB_LDS, int QB, int PLACE, bool SEARCH, bool PHI, bool SCHED>
__global__ __launch_bounds__(PLACE == 1 ? 256 : 512, PLACE == 1 ? 3 : 1) void score_plans(ScoreParams sp,
                                                   const int8_t* __restrict__ dev_all,
                                                   const uint16_t* __restrict__ prio_all,
                                                   const uint8_t* __restrict__ flags_all, int64_t P,
                                                   OutRec<PHI>* __restrict__ scores,
                                                   wf_plan_sched sched, int has_sched_arg,
                                                   SearchArgs sa) {
  using TO = TimeOps<TT>;
  using TB = typename TO::bits_t;
  // reclamation queue: QB bits of 4-bit model ids (QB = 0: no queue, the
  // resident set is scanned instead)
  constexpr bool NIBBLE = QB > 0;
  // QB = -1, -3: the paper's reclamation order (copies held on another
  // device, then next-use distance per reload time, then recency) over the scanned
  // resident set; QB = -2, -3: devices with batch limits (several units at
  // once, each in one of up to kMaxBatch slots)
  constexpr bool PAPER = QB == -1 || QB == -3;
  constexpr bool BATCH = QB <= -2;
  // PLACE 2: the ring of recent levels, the order built level by level, all
  // in LDS.  PLACE 4: the finishes in the ring (LDS), the order built before
  // the walk with the other per-activation arrays in HBM (the paper's order,
  // whose next use per slot needs every level's order first).
  constexpr bool RING = PLACE == 2;           // order built level by level
  constexpr bool RING_FIN = PLACE == 2 || PLACE == 4;  // finishes in the ring
  constexpr bool WAVE_GLOBAL = PLACE == 1 || PLACE == 4;
  static_assert(!RING || QB == 0 || QB == -2, "ring layout: scans");
  static_assert(PLACE != 4 || ((QB == -1 || QB == -3) && !SEARCH), "ring finishes: the paper's order");
  using QT = std::conditional_t<QB == 32, uint32_t, uint64_t>;
  constexpr QT kOnes = (QT)0x1111111111111111ull, kHigh = (QT)0x8888888888888888ull;
  constexpr int kQBits = (int)sizeof(QT) * 8;
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int N = sp.N, W = sp.W, M = sp.M, D = sp.D, NB = sp.NB, G = sp.G, NWA = sp.nwa;

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
  const uint16_t* t_cnext = reinterpret_cast<const uint16_t*>(tb + sp.t.cnext);
  const uint32_t* t_edge = reinterpret_cast<const uint32_t*>(tb + sp.t.edge);
  const int32_t* t_eoff = reinterpret_cast<const int32_t*>(tb + sp.t.eoff);
  const int32_t* t_loff = reinterpret_cast<const int32_t*>(tb + sp.t.loff);
  const uint4* t_ud = reinterpret_cast<const uint4*>(tb + sp.t.ud);
  const int2* t_lw = reinterpret_cast<const int2*>(tb + sp.t.lw);
  const int32_t* t_wmib = reinterpret_cast<const int32_t*>(tb + sp.t.wmib);  // (LDS below)
  // paper reclamation order: the workgroup's copy of every (model, device)
  // load time, read per candidate victim
  uint32_t* wg_ld = reinterpret_cast<uint32_t*>(lds + wave_base);
  if constexpr (PAPER) {
    const int2* lw = reinterpret_cast<const int2*>(tb + sp.t.lw);
    for (int i = tid; i < M * D; i += blockDim.x) wg_ld[i] = (uint32_t)lw[i].x;
    __syncthreads();
  }
  // every model's weights, read per reclamation: the workgroup's copy in LDS
  // (after the paper order's load times) when the tables stay in HBM
  if constexpr (!TAB_LDS) {
    int32_t* wg_wm = reinterpret_cast<int32_t*>(lds + wave_base + (PAPER ? ((M * D * 4 + 15) & ~15) : 0));
    for (int i = tid; i < M; i += blockDim.x) wg_wm[i] = t_wmib[i];
    __syncthreads();
    t_wmib = wg_wm;
  }
  wave_base += sp.wg_ld;
  const int32_t* t_cap = reinterpret_cast<const int32_t*>(tb + sp.t.cap);
  const TB* t_arr = reinterpret_cast<const TB*>(tb + sp.t.arr);
  const unsigned long long* t_res0 = reinterpret_cast<const unsigned long long*>(tb + sp.t.res0);
  const TB* t_free0 = reinterpret_cast<const TB*>(tb + sp.t.free0);
  const uint32_t* t_sink = reinterpret_cast<const uint32_t*>(tb + sp.t.sink);
  const unsigned long long* t_elig = reinterpret_cast<const unsigned long long*>(tb + sp.t.elig);
  const int32_t* t_batch = reinterpret_cast<const int32_t*>(tb + sp.t.batch);
  const uint16_t* t_rpos = reinterpret_cast<const uint16_t*>(tb + sp.t.rpos);
  const uint16_t* t_rsnk = reinterpret_cast<const uint16_t*>(tb + sp.t.rsnk);
  // ring layout: slot entries per plan (the widest level), finishes per plan
  // (the ring), a finish's position
  const int RW = RING ? sp.ring_w : N;
  const int FS = RING_FIN ? sp.ring_size : N;
  auto fpos = [&](int u) -> int {
    if constexpr (RING_FIN) return (int)t_rpos[u];
    else return u;
  };

  // ---- this wave's region (LDS, or HBM scratch for very large windows) ----
  // (with regions in HBM, the small per-(device, model) arrays stay in LDS:
  // big() addresses the HBM part, small() the LDS part)
  unsigned char* wl;
  unsigned char* wls;
  if constexpr (WAVE_GLOBAL) {
    wl = sp.scratch + ((int64_t)blockIdx.x * sp.waves + wid) * (int64_t)(sp.wo.bytes - sp.wo.split);
    wls = lds + wave_base + wid * sp.wo.split;
  } else {
    wl = lds + wave_base + wid * sp.wo.bytes;
    wls = wl;
  }
  auto big = [&](int off) -> unsigned char* { return wl + (WAVE_GLOBAL ? off - sp.wo.split : off); };
  auto small = [&](int off) -> unsigned char* { return wls + off; };
  uint8_t* s_fl = reinterpret_cast<uint8_t*>(big(sp.wo.flags));
  uint32_t* s_rec = reinterpret_cast<uint32_t*>(big(sp.wo.rec));
  unsigned long long* s_mask = reinterpret_cast<unsigned long long*>(big(sp.wo.mask));
  // last[] shares fin's storage in the queue modes, else it is a small array
  // (the paper order keeps no last[]; its offset is fin's)
  uint32_t* s_last = reinterpret_cast<uint32_t*>((NIBBLE || PAPER) ? big(sp.wo.last) : small(sp.wo.last));
  TB* s_fin = reinterpret_cast<TB*>(PLACE == 4 ? small(sp.wo.fin) : big(sp.wo.fin));
  PlanAcc* s_acc = reinterpret_cast<PlanAcc*>(small(sp.wo.acc));
  uint16_t* s_stamp = reinterpret_cast<uint16_t*>(small(sp.wo.stamp));
  uint16_t* s_nx = reinterpret_cast<uint16_t*>(big(sp.wo.nx));      // paper order only
  uint16_t* s_nxu = reinterpret_cast<uint16_t*>(small(sp.wo.nxu));
  unsigned long long* s_snap = reinterpret_cast<unsigned long long*>(small(sp.wo.snap));
  HState* s_hst = reinterpret_cast<HState*>(small(sp.wo.hstate));  // more than 64 devices only
  unsigned long long* s_hold = reinterpret_cast<unsigned long long*>(small(sp.wo.hold));  // replica caps
  const int32_t* t_rcap = reinterpret_cast<const int32_t*>(tb + sp.t.rcap);
  TB* s_wfm = reinterpret_cast<TB*>(PLACE == 4 ? small(sp.wo.wfm) : big(sp.wo.wfm));
  int8_t* s_rdev = reinterpret_cast<int8_t*>(big(sp.wo.rows));         // generated candidates
  uint16_t* s_rprio = reinterpret_cast<uint16_t*>(big(sp.wo.rows_prio));
  // (the ring layout keeps a candidate as the incumbent plus its changed sites)
  uint32_t* s_pat = reinterpret_cast<uint32_t*>(big(sp.wo.rows));

  const int g_me = lane / D;
  // every unit's finish goes through the general path when the schedule is
  // written out
  // SCHED: the schedule is written (known at compile time, so that the
  // instantiations without one carry none of its code or registers)
  const bool has_sched = SCHED && has_sched_arg != 0;
  const uint32_t slow0 = has_sched ? kSlow : 0u;
  const int d_me = lane - g_me * D;
  const int64_t n_groups = (P + G - 1) / G;
  const int64_t stride = (int64_t)gridDim.x * sp.waves;
  // per-device table rows of this lane's device (bound per device below)
  const uint4* ud_d = t_ud + d_me;
  const int2* lw_d = t_lw + d_me;

  // rows read four activations per lane with 4- and 8-byte loads
  const bool vec = (N & 3) == 0 && (SEARCH || ((reinterpret_cast<uintptr_t>(dev_all) & 3) == 0 &&
                                               (reinterpret_cast<uintptr_t>(prio_all) & 7) == 0));
  // one 256-activation chunk and at most eight plans per group: the next
  // group's device and priority rows are loaded while this group is walked
  constexpr int kB = 8;
  const bool pre = !SEARCH && !RING && !WAVE_GLOBAL && vec && N <= 256 && G <= kB && !sp.rescore;
  uint32_t dvp[kB];
  uint2 pvp[kB];
  auto load_rows = [&](int64_t grp_, uint32_t* dv, uint2* pv) {
    const int64_t q0 = grp_ * G;
    const int gq = (int)((P - q0) < G ? (P - q0) : G);
    const int uc = 4 * lane < N ? 4 * lane : 0;
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const int g = k < gq ? k : gq - 1;
      dv[k] = *reinterpret_cast<const uint32_t*>(dev_all + (q0 + g) * N + uc);
      pv[k] = *reinterpret_cast<const uint2*>(prio_all + (q0 + g) * N + uc);
    }
  };
  {
    const int64_t g_first = (int64_t)blockIdx.x * sp.waves + wid;
    if (pre && g_first < n_groups) load_rows(g_first, dvp, pvp);
  }

  for (int64_t grp = (int64_t)blockIdx.x * sp.waves + wid; grp < n_groups; grp += stride) {
    const int64_t p0 = grp * G;
    const int gc = (int)((P - p0) < G ? (P - p0) : G);
    if (sp.rescore) {
      // second pass: only groups holding a plan the uint32 pass flagged
      const bool flagged = lane < gc && (scores[p0 + lane].status & kRescore) != 0u;
      if (__ballot(flagged) == 0ull) continue;
    }

    // ---- stage the group's flag rows, clear the ordering state ----
    if constexpr (SEARCH && RING) {
      // every plan of the group starts as the incumbent; lane g then writes
      // candidate g's changed sites and mutates its flag row
      for (int g = 0; g < gc; ++g) copy_row(s_fl + g * NB, flags_all, NB, lane);
      wave_sync();
      if (lane < gc) {
        PatchRows rows{s_pat + lane * kPatchWords, dev_all, prio_all, s_fl + lane * NB};
        rows.p[0] = 0u;
        mutate_rows((uint64_t)(sa.first + p0 + lane), sa, N, t_elig, t_alv, rows);
      }
    } else if constexpr (SEARCH) {
      // every plan of the group starts as the incumbent, then takes its
      // candidate's mutations (one lane per plan, in order)
      for (int g = 0; g < gc; ++g) {
        copy_row(reinterpret_cast<unsigned char*>(s_rdev + g * N),
                 reinterpret_cast<const unsigned char*>(dev_all), N, lane);
        copy_row(reinterpret_cast<unsigned char*>(s_rprio + g * N),
                 reinterpret_cast<const unsigned char*>(prio_all), 2 * N, lane);
        copy_row(s_fl + g * NB, flags_all, NB, lane);
      }
      wave_sync();
      if (lane < gc)
        mutate((uint64_t)(sa.first + p0 + lane), sa, N, t_elig, t_alv, s_rdev + lane * N,
               s_rprio + lane * N, s_fl + lane * NB);
    } else {
      stage(s_fl, flags_all + p0 * NB, gc * NB, lane);
    }
    // last[] (each (device, model)'s last slot) serves the other reclamation
    // orders only
    if constexpr (!PAPER)
      zero_bytes(reinterpret_cast<unsigned char*>(s_last), G * D * M * (RING ? 2 : 4), lane);
    zero_bytes(reinterpret_cast<unsigned char*>(s_mask), G * D * NWA * 8, lane);
    if (lane < G) {
      PlanAcc a0;
      a0.status = 0u;
      a0.headroom = 0x7fffffff;
      a0.loads = 0u;
      a0.evicts = 0u;
      a0.max_finish = 0ull;
      a0.p95 = 0;
      a0.heads = 0u;
      a0.claimed = 0u;
      a0.bad = 0u;
      a0.pad = 0u;
      a0.ph_adm = 0ull;
      a0.ph_cf = 0ull;
      a0.ph_h = 0ull;
      a0.ph_pn = 0u;
      a0.ph_pad = 0u;
      s_acc[lane] = a0;
    }
    wave_sync();

    // device and priority of activation u in plan g, for the ring layout's
    // level-by-level order: the plan rows in HBM, or the incumbent's with
    // the candidate's changed sites
    auto ring_dev = [&](int g, int u) -> int {
      if constexpr (SEARCH) {
        const PatchRows rows{s_pat + g * kPatchWords, dev_all, prio_all, nullptr};
        return rows.dev(u);
      } else {
        return dev_all[(p0 + g) * N + u];
      }
    };
    auto ring_prio = [&](int g, int u) -> int {
      if constexpr (SEARCH) {
        const PatchRows rows{s_pat + g * kPatchWords, dev_all, prio_all, nullptr};
        return rows.prio(u);
      } else {
        return prio_all[(p0 + g) * N + u];
      }
    };
    if constexpr (!RING) {
      // ---- resource order (Eq. 10), first try: a unit head's slot is its
      // priority, valid when each level's head priorities are distinct values
      // in the level's index range (checked below by counting) ----
      // one activation u of plan g with device d and priority pr; cbyte is the
      // flag byte of u's chain successor
      auto order_fast = [&](int g, int u, int d, int pr, uint32_t a, uint32_t lvw, uint32_t c,
                            uint32_t fb, uint32_t cbyte, uint32_t& nh, uint32_t& nbad,
                            uint32_t& ninel) {
        const bool head = !((fb & 1u) && (a & 64u));  // not a fused chain member
        const bool okd = (unsigned)d < (unsigned)D;
        const bool inr = (unsigned)(pr - (int)(lvw & 0xffffu)) < (lvw >> 16);
        const bool chain = c != 0xffffu && ((cbyte >> ((c & 3u) << 1)) & 1u);
        ninel |= (uint32_t)(head && !okd);
        nbad |= (uint32_t)(head && okd && !inr);
        if (head && okd && inr) {
          const uint32_t m = a & 63u;
          s_rec[g * N + pr] = (uint32_t)u | (m << 16) | ((fb & 2u) << 21) |
                              (chain ? kChain | kSlow : slow0);
          atomicOr(&s_mask[(g * D + d) * NWA + (pr >> 6)], 1ull << (pr & 63));
          if constexpr (!PAPER) atomicMax(&s_last[(g * D + d) * M + (int)m], (uint32_t)pr + 1u);
          ++nh;
        }
      };
      // per-plan totals from uniform control flow, at most 4 heads per lane:
      // wave ballots instead of 64 conflicting LDS atomics
      auto order_flush4 = [&](int g, uint32_t nh, uint32_t nbad, uint32_t ninel) {
        const uint32_t tot = (uint32_t)__popcll(__ballot(nh & 1u)) +
                             2u * (uint32_t)__popcll(__ballot(nh & 2u)) +
                             4u * (uint32_t)__popcll(__ballot(nh & 4u));
        const bool any_bad = __ballot(nbad != 0u) != 0ull;
        const bool any_inel = __ballot(ninel != 0u) != 0ull;
        if (lane == 0) {
          if (any_inel) s_acc[g].status |= (uint32_t)WF_ST_INELIGIBLE;
          if (any_bad) s_acc[g].bad = 1u;
          s_acc[g].heads += tot;
        }
      };
      // device and priority rows of plan g: HBM, or the generated candidate
      auto row_dev = [&](int g) -> const int8_t* {
        if constexpr (SEARCH) return s_rdev + g * N;
        else return dev_all + (p0 + g) * N;
      };
      auto row_prio = [&](int g) -> const uint16_t* {
        if constexpr (SEARCH) return s_rprio + g * N;
        else return prio_all + (p0 + g) * N;
      };
      // the rows of plans g0 .. g0 + kB - 1 at activations uc .. uc + 3
      auto rows4 = [&](int g0, int uc, uint32_t* dv, uint2* pv) {
  #pragma unroll
        for (int k = 0; k < kB; ++k) {
          const int g = (g0 + k < gc) ? g0 + k : gc - 1;
          if (pre) {
            dv[k] = dvp[k];
            pv[k] = pvp[k];
          } else {
            dv[k] = *reinterpret_cast<const uint32_t*>(row_dev(g) + uc);
            pv[k] = *reinterpret_cast<const uint2*>(row_prio(g) + uc);
          }
        }
      };
      if (vec) {
        // four consecutive activations per lane: one 4-byte device load, one
        // 8-byte priority load and one flag byte per plan; every load of a
        // batch of plans is issued before any of it is used
        for (int base = 0; base < N; base += 256) {
          const int u0 = base + 4 * lane;
          const bool live = u0 < N;
          const int uc = live ? u0 : 0;
          const uint4 act4 = *reinterpret_cast<const uint4*>(t_act + uc);
          const uint4 alv4 = *reinterpret_cast<const uint4*>(t_alv + uc);
          const uint2 cn4 = *reinterpret_cast<const uint2*>(t_cnext + uc);
          const uint32_t cn[4] = {cn4.x & 0xffffu, cn4.x >> 16, cn4.y & 0xffffu, cn4.y >> 16};
          for (int g0 = 0; g0 < gc; g0 += kB) {
            uint32_t dv[kB], fl[kB], cb[kB][4];
            uint2 pv[kB];
            rows4(g0, uc, dv, pv);
  #pragma unroll
            for (int k = 0; k < kB; ++k) {
              const int g = (g0 + k < gc) ? g0 + k : gc - 1;
              fl[k] = s_fl[g * NB + (uc >> 2)];
  #pragma unroll
              for (int j = 0; j < 4; ++j)
                cb[k][j] = sp.has_chains ? s_fl[g * NB + ((cn[j] != 0xffffu ? cn[j] : (uint32_t)uc) >> 2)]
                                         : 0u;
            }
  #pragma unroll
            for (int k = 0; k < kB; ++k) {
              const int g = g0 + k;
              if (g >= gc) break;
              uint32_t nh = 0, nbad = 0, ninel = 0;
              if (live) {
                order_fast(g, uc, (int)(int8_t)(dv[k] & 0xffu), (int)(pv[k].x & 0xffffu), act4.x,
                           alv4.x, cn[0], fl[k], cb[k][0], nh, nbad, ninel);
                order_fast(g, uc + 1, (int)(int8_t)((dv[k] >> 8) & 0xffu), (int)(pv[k].x >> 16),
                           act4.y, alv4.y, cn[1], fl[k] >> 2, cb[k][1], nh, nbad, ninel);
                order_fast(g, uc + 2, (int)(int8_t)((dv[k] >> 16) & 0xffu), (int)(pv[k].y & 0xffffu),
                           act4.z, alv4.z, cn[2], fl[k] >> 4, cb[k][2], nh, nbad, ninel);
                order_fast(g, uc + 3, (int)(int8_t)(dv[k] >> 24), (int)(pv[k].y >> 16), act4.w,
                           alv4.w, cn[3], fl[k] >> 6, cb[k][3], nh, nbad, ninel);
              }
              order_flush4(g, nh, nbad, ninel);
            }
          }
        }
      } else {
        for (int g = 0; g < gc; ++g) {
          const int8_t* pdev = row_dev(g);
          const uint16_t* pprio = row_prio(g);
          const uint8_t* pfl = s_fl + g * NB;
          uint32_t nh = 0, nbad = 0, ninel = 0;
          for (int u = lane; u < N; u += 64) {
            const uint32_t fb = (uint32_t)pfl[u >> 2] >> ((u & 3) << 1);
            const uint32_t c = t_cnext[u];
            const uint32_t cbyte = pfl[(c != 0xffffu ? c : (uint32_t)u) >> 2];
            order_fast(g, u, pdev[u], pprio[u], t_act[u], t_alv[u], c, fb, cbyte, nh, nbad, ninel);
          }
          if (ninel) atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
          if (nbad) atomicOr(&s_acc[g].bad, 1u);
          if (nh) atomicAdd(&s_acc[g].heads, nh);
        }
      }
      wave_sync();
      // distinct slots claimed per plan: the union of its devices' masks
      for (int i = lane; i < gc * NWA; i += 64) {
        const int g = i / NWA, w = i - g * NWA;
        unsigned long long x = 0ull;
        for (int d = 0; d < D; ++d) x |= s_mask[(g * D + d) * NWA + w];
        if (x) atomicAdd(&s_acc[g].claimed, (uint32_t)__popcll(x));
      }
      wave_sync();
      // plans whose priorities are not a permutation of each level's heads'
      // index range (one lane per plan)
      uint64_t rankedm;
      {
        const PlanAcc& ag = s_acc[lane < gc ? lane : 0];  // G <= 64
        const bool rk = lane < gc && (ag.bad != 0u || ag.heads != ag.claimed);
        rankedm = __ballot(rk);
      }
      // general path: rank by (priority, index) within each level
      for (uint64_t rm = rankedm; rm; rm &= rm - 1ull) {
        const int g = __builtin_ctzll(rm);
        const int8_t* pdev = row_dev(g);
        const uint16_t* pprio = row_prio(g);
        const uint8_t* pfl = s_fl + g * NB;
        uint32_t* rec = s_rec + g * N;
        unsigned long long* mk = s_mask + g * D * NWA;
        uint32_t* lastp = s_last + g * D * M;
        for (int i = lane; i < D * NWA; i += 64) mk[i] = 0ull;
        if constexpr (!PAPER)
          for (int i = lane; i < D * M; i += 64) lastp[i] = 0u;
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
          rec[slot] = (uint32_t)u | ((a & 63u) << 16) | ((uint32_t)((fb >> 1) & 1) << 22) | chain |
                      (chain ? kSlow : slow0);
          atomicOr(&mk[d * NWA + (slot >> 6)], 1ull << (slot & 63));
          if constexpr (!PAPER) atomicMax(&lastp[d * M + (int)(a & 63u)], (uint32_t)slot + 1u);
        }
        wave_sync();
      }
      if constexpr (NIBBLE) {
        // mark each (device, model)'s last unit in its slot entry: the
        // reclamation queues need only that bit, and last[] dies here
        if (vec) {
          // plans ordered by priority: re-derive each head's (device, slot,
          // model) from its row; all loads first, then the marks
          for (int base = 0; base < N; base += 256) {
            const int u0 = base + 4 * lane;
            const bool live = u0 < N;
            const int uc = live ? u0 : 0;
            const uint4 act4 = *reinterpret_cast<const uint4*>(t_act + uc);
            const uint4 alv4 = *reinterpret_cast<const uint4*>(t_alv + uc);
            const uint32_t av[4] = {act4.x, act4.y, act4.z, act4.w};
            const uint32_t lv[4] = {alv4.x, alv4.y, alv4.z, alv4.w};
            for (int g0 = 0; g0 < gc; g0 += kB) {
              uint32_t dv[kB];
              uint2 pv[kB];
              rows4(g0, uc, dv, pv);
              uint32_t fl[kB];
  #pragma unroll
              for (int k = 0; k < kB; ++k) {
                const int g = (g0 + k < gc) ? g0 + k : gc - 1;
                fl[k] = s_fl[g * NB + (uc >> 2)];
              }
              int idx[kB][4], prs[kB][4];
              bool ok[kB][4];
              uint32_t lst[kB][4];
  #pragma unroll
              for (int k = 0; k < kB; ++k) {
                const int g = g0 + k;
                const bool plan_ok = live && g < gc && !((rankedm >> (g & 63)) & 1ull);
  #pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int d = (int)(int8_t)((dv[k] >> (8 * j)) & 0xffu);
                  const int pr = (int)(((j < 2 ? pv[k].x : pv[k].y) >> (16 * (j & 1))) & 0xffffu);
                  const uint32_t fb = fl[k] >> (2 * j);
                  const bool head = !((fb & 1u) && (av[j] & 64u));
                  const bool okd = (unsigned)d < (unsigned)D;
                  const bool inr = (unsigned)(pr - (int)(lv[j] & 0xffffu)) < (lv[j] >> 16);
                  ok[k][j] = plan_ok && head && okd && inr;
                  prs[k][j] = pr;
                  idx[k][j] = ok[k][j] ? (g * D + d) * M + (int)(av[j] & 63u) : 0;
                }
              }
  #pragma unroll
              for (int k = 0; k < kB; ++k)
  #pragma unroll
                for (int j = 0; j < 4; ++j) lst[k][j] = s_last[idx[k][j]];
  #pragma unroll
              for (int k = 0; k < kB; ++k)
  #pragma unroll
                for (int j = 0; j < 4; ++j)
                  if (ok[k][j] && lst[k][j] == (uint32_t)prs[k][j] + 1u)
                    atomicOr(&s_rec[(g0 + k) * N + prs[k][j]], kLast);
            }
          }
        }
        // ranked plans (and every plan without the vector path): by slot
        for (int g = 0; g < gc; ++g) {
          if (vec && !((rankedm >> g) & 1ull)) continue;
          uint32_t* rec = s_rec + g * N;
          const unsigned long long* mk = s_mask + g * D * NWA;
          const uint32_t* lastp = s_last + g * D * M;
          const int8_t* pdev = row_dev(g);
          for (int sl = lane; sl < N; sl += 64) {
            const uint32_t e = rec[sl];
            // entries of empty slots are stale: the activation, its device and
            // the model may be anything; only an occupied slot counts
            const int u = (int)(e & 0xffffu);
            const int d = u < N ? (int)pdev[u] : -1;
            const int m = (int)((e >> 16) & 63u);
            const bool occ = (unsigned)d < (unsigned)D && m < M &&
                             ((mk[d * NWA + (sl >> 6)] >> (sl & 63)) & 1ull);
            if (occ && lastp[d * M + m] == (uint32_t)sl + 1u) rec[sl] = e | kLast;
          }
        }
        wave_sync();
      }
    } else {
      // ring layout: the order is built level by level during the walk; here
      // only each (device, model)'s number of units (the reclamation order
      // asks whether a copy has a remaining use on its device) and the
      // plans with a unit head on no valid device
      for (int it = lane; it < gc * N; it += 64) {
        const int g = it / N, u = it - g * N;
        const uint32_t a = t_act[u];
        const uint32_t fb = (uint32_t)s_fl[g * NB + (u >> 2)] >> ((u & 3) << 1);
        if ((fb & 1u) && (a & 64u)) continue;  // a fused chain member
        const int dv = ring_dev(g, u);
        if ((unsigned)dv < (unsigned)D) {
          // 16-bit counts, two to a word (a count stays below 2^16)
          const int ci = (g * D + dv) * M + (int)(a & 63u);
          atomicAdd(&s_last[ci >> 1], 1u << ((ci & 1) << 4));
        } else {
          atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
        }
      }
      wave_sync();
    }

    if (pre && grp + stride < n_groups) load_rows(grp + stride, dvp, pvp);

    // ---- device-lane state ----
    // With more than 64 devices (one plan per wave) a lane owns two devices,
    // d_me and d_me + 64: their states take turns in registers, the other
    // one waiting in the wave's LDS region, and each level walks the first
    // device's units, then the second's (devices are independent within a
    // level).
    const int NH = D > 64 ? 2 : 1;
    const bool act_plan = g_me < gc;
    const int gme = act_plan ? g_me : 0;
    const int64_t pw = p0 + gme;
    bool act = act_plan;
    int d = d_me;
    uint32_t* mylast = s_last + (gme * D + d_me) * M;
    // ring layout: the lane's 16-bit counts of units still to walk per model
    uint16_t* mycnt = reinterpret_cast<uint16_t*>(s_last) + (gme * D + d_me) * M;
    uint16_t* mystamp = s_stamp + (gme * D + d_me) * M;
    uint16_t* mynxu = s_nxu + (gme * D + d_me) * M;  // next use of each model (device index)
    const unsigned long long* mymask = s_mask + (gme * D + d_me) * NWA;
    const uint32_t* myrec = s_rec + gme * RW;
    TB* myfin = s_fin + gme * FS;
    const uint8_t* myfl = s_fl + gme * NB;
    // the lane's h-th device (h = 0, 1) and its table rows; a lane without
    // a second device keeps in-range pointers and stays inactive
    auto bind = [&](int h) {
      d = d_me + 64 * h;
      act = act_plan && d < D;
      const int dd = d < D ? d : d_me;
      mylast = s_last + (gme * D + dd) * M;
      mycnt = reinterpret_cast<uint16_t*>(s_last) + (gme * D + dd) * M;
      mystamp = s_stamp + (gme * D + dd) * M;
      mynxu = s_nxu + (gme * D + dd) * M;
      mymask = s_mask + (gme * D + dd) * NWA;
      ud_d = t_ud + dd;
      lw_d = t_lw + dd;
    };
    uint64_t res = 0;
    int32_t used = 0, peak = 0, capd = 0;
    TT freet = 0;
    uint32_t nld = 0, nev = 0, capbad = 0, inel = 0;
    uint32_t seq = 1;
    // reclamation queue (at most 16 models), 4 bits per entry, next victim
    // in the low bits: first the nd resident models with no remaining use on
    // this device, then those still needed, each part in least-recently-used
    // order (never used: by id); nq entries in all
    QT Q = 0;
    int nd = 0, nq = 0;
    // ranking-key terms (Eq. 12) of this device lane: admitted ready units
    // per class (16 bits each), models reclaimed from the device so far, the
    // latest admitted ready completion, lifecycle overhead, timely prefetches
    using HT = std::conditional_t<std::is_same<TT, double>::value, double, unsigned long long>;
    unsigned long long ph_adm = 0ull, ph_rec = 0ull;
    TT ph_cf = 0;
    HT ph_h = 0;
    uint32_t ph_pn = 0u;
    // paper order: this unit's index among the device's units, and the
    // models resident on the plan's other devices as the level starts
    int kdev = 0;
    unsigned long long others = 0ull;
    // replica caps: the models the device holds as the level starts or loads
    // during it
    unsigned long long lv_hold = 0ull;
    // batch limits: per slot the free time, and the running unit's finish,
    // memory and model; the last first-action time (dispatch is in order)
    int nbatch = 1;
    TT bs_free[kMaxBatch], bs_fin[kMaxBatch], bdisp = 0;
    int32_t bs_mem[kMaxBatch], bs_model[kMaxBatch];
    // the idle device's state in LDS, and back
    using HT2 = HT;
    auto save = [&](int h) {
      HState& x = s_hst[h * 64 + lane];
      x.res = res;
      x.freet = (unsigned long long)TO::bits(freet);
      x.q = (unsigned long long)Q;
      x.ph_adm = ph_adm;
      x.ph_rec = ph_rec;
      x.ph_cf = (unsigned long long)TO::bits(ph_cf);
      if constexpr (std::is_same<HT2, double>::value)
        x.ph_h = (unsigned long long)__double_as_longlong(ph_h);
      else
        x.ph_h = (unsigned long long)ph_h;
      x.bdisp = (unsigned long long)TO::bits(bdisp);
#pragma unroll
      for (int k = 0; k < kMaxBatch; ++k) {
        x.bs_free[k] = (unsigned long long)TO::bits(bs_free[k]);
        x.bs_fin[k] = (unsigned long long)TO::bits(bs_fin[k]);
        x.bs_mem[k] = bs_mem[k];
        x.bs_model[k] = bs_model[k];
      }
      x.used = used;
      x.peak = peak;
      x.capd = capd;
      x.nld = nld;
      x.nev = nev;
      x.capbad = capbad;
      x.inel = inel;
      x.seq = seq;
      x.nd = nd;
      x.nq = nq;
      x.ph_pn = ph_pn;
      x.kdev = kdev;
      x.nbatch = nbatch;
    };
    auto load = [&](int h) {
      const HState& x = s_hst[h * 64 + lane];
      res = x.res;
      freet = TO::load(reinterpret_cast<const TB*>(&x.freet));
      Q = (QT)x.q;
      ph_adm = x.ph_adm;
      ph_rec = x.ph_rec;
      ph_cf = TO::load(reinterpret_cast<const TB*>(&x.ph_cf));
      if constexpr (std::is_same<HT2, double>::value)
        ph_h = __longlong_as_double((long long)x.ph_h);
      else
        ph_h = (HT2)x.ph_h;
      bdisp = TO::load(reinterpret_cast<const TB*>(&x.bdisp));
#pragma unroll
      for (int k = 0; k < kMaxBatch; ++k) {
        bs_free[k] = TO::load(reinterpret_cast<const TB*>(&x.bs_free[k]));
        bs_fin[k] = TO::load(reinterpret_cast<const TB*>(&x.bs_fin[k]));
        bs_mem[k] = x.bs_mem[k];
        bs_model[k] = x.bs_model[k];
      }
      used = x.used;
      peak = x.peak;
      capd = x.capd;
      nld = x.nld;
      nev = x.nev;
      capbad = x.capbad;
      inel = x.inel;
      seq = x.seq;
      nd = x.nd;
      nq = x.nq;
      ph_pn = x.ph_pn;
      kdev = x.kdev;
      nbatch = x.nbatch;
    };
    for (int h = 0; h < NH; ++h) {
    if (NH > 1) bind(h);
    res = 0;
    used = peak = capd = 0;
    freet = 0;
    nld = nev = capbad = inel = 0u;
    seq = 1;
    Q = 0;
    nd = nq = 0;
    ph_adm = ph_rec = 0ull;
    ph_cf = 0;
    ph_h = 0;
    ph_pn = 0u;
    kdev = 0;
    nbatch = 1;
    bdisp = 0;
#pragma unroll
    for (int k = 0; k < kMaxBatch; ++k) {
      bs_free[k] = 0;
      bs_fin[k] = 0;
      bs_mem[k] = 0;
      bs_model[k] = 0;
    }
    if (PAPER && act) {
      // one backward pass over the device's units: for each unit, the index
      // of the next unit of the device with the same model (0xffff: none);
      // what remains in mynxu is every model's first use
      for (int m = 0; m < M; ++m) mynxu[m] = 0xffff;
      int cnt = 0;
      for (int j = 0; j < NWA; ++j) cnt += __popcll(mymask[j]);
      uint16_t* mynx = s_nx + gme * N;
      for (int j = NWA - 1; j >= 0; --j) {
        for (unsigned long long bits = mymask[j]; bits;) {
          const int b = 63 - __clzll(bits);
          bits &= ~(1ull << b);
          const int sl = (j << 6) + b;
          const int m = (int)((myrec[sl] >> 16) & 63u);
          --cnt;
          mynx[sl] = mynxu[m];
          mynxu[m] = (uint16_t)cnt;
        }
      }
    }
    if (act) {
      res = t_res0[d];
      capd = t_cap[d];
      freet = TO::load(t_free0 + d);
      if constexpr (BATCH) {
        nbatch = t_batch[d];
        bdisp = freet;
#pragma unroll
        for (int k = 0; k < kMaxBatch; ++k) {
          bs_free[k] = freet;
          bs_fin[k] = freet;
        }
      }
      QT qa = 0;
      int na = 0;
      for (uint64_t r = res; r; r &= r - 1) {
        const int m = __builtin_ctzll(r);
        used += t_wmib[m];
        if constexpr (NIBBLE) {
          if (mylast[m] == 0u) {
            Q |= (QT)m << (4 * nd);
            ++nd;
          } else {
            qa |= (QT)m << (4 * na);
            ++na;
          }
        } else {
          mystamp[m] = 0;
        }
      }
      if constexpr (NIBBLE) {
        if (na) Q |= qa << (4 * nd);  // nd + na <= QB / 4, so 4 * nd < QB here
        nq = nd + na;
      }
      peak = used;
    }
    if (NH > 1) save(h);
    }
    if constexpr (NIBBLE) wave_sync();  // last[] (aliasing fin) is read above
    // every finish starts at 0: it accumulates the latest predecessor finish
    // before its level, then holds the activation's own finish
    zero_bytes(reinterpret_cast<unsigned char*>(s_fin), G * FS * (int)sizeof(TB), lane);
    zero_bytes(reinterpret_cast<unsigned char*>(s_wfm), G * W * (int)sizeof(TB), lane);
    wave_sync();

    // ring layout: fold the finishes of level L's activations without a
    // successor in their workflow into the workflow's latest finish (L
    // leaves the ring), or clear L's positions (L enters it)
    auto ring_level = [&](int L, bool clear) {
      const int loL = t_loff[L], wL = t_loff[L + 1] - loL;
      for (int it = lane; it < gc * wL; it += 64) {
        const int g = it / wL, u = loL + (it - g * wL);
        TB* f = s_fin + g * FS + (int)t_rpos[u];
        if (clear) {
          *f = (TB)0;
        } else {
          const uint32_t wf = t_rsnk[u];
          if (wf != 0xffffu) atomicMax(&s_wfm[g * W + (int)wf], *f);
        }
      }
    };
    for (int lv = 0; lv < sp.n_levels; ++lv) {
      const int lo = t_loff[lv], hi = t_loff[lv + 1];
      const int e0 = t_eoff[lv], e1 = t_eoff[lv + 1];
      if constexpr (RING_FIN) {
        // ---- the level leaving the ring ----
        const int lold = lv - sp.ring_b - 1, lnew = lv + sp.ring_a;
        if (lold >= 0) {
          if (!PHI) ring_level(lold, false);
          if (lnew < sp.n_levels) {
            wave_sync();  // the positions may be shared
            ring_level(lnew, true);
          }
        }
        if constexpr (!RING) wave_sync();
      }
      if constexpr (RING) {
        // ---- this level's resource order (Eq. 10): a head's slot is its
        // priority when the level's head priorities are distinct values in
        // its index range, else its rank by (priority, index) ----
        const int width = hi - lo, jb = lo >> 6;
        for (int i = lane; i < gc * D * NWA; i += 64) s_mask[i] = 0ull;
        if (lane < gc) s_acc[lane].bad = 0u;
        wave_sync();
        auto head_entry = [&](int g, int u, uint32_t a, uint32_t fb) -> uint32_t {
          const int c = t_cnext[u];
          const bool chain = c != 0xffff && fuse_bit(s_fl + g * NB, c);
          return (uint32_t)u | ((a & 63u) << 16) | ((fb & 2u) << 21) | (chain ? kChain | kSlow : slow0);
        };
        for (int it = lane; it < gc * width; it += 64) {
          const int g = it / width, u = lo + (it - g * width);
          const uint32_t a = t_act[u];
          const uint32_t fb = (uint32_t)s_fl[g * NB + (u >> 2)] >> ((u & 3) << 1);
          if ((fb & 1u) && (a & 64u)) continue;
          const int dv = ring_dev(g, u);
          if ((unsigned)dv >= (unsigned)D) continue;
          const int pr = ring_prio(g, u);
          if ((unsigned)(pr - lo) >= (unsigned)width) {
            s_acc[g].bad = 1u;
            continue;
          }
          s_rec[g * RW + (pr - lo)] = head_entry(g, u, a, fb);
          const unsigned long long bit = 1ull << (pr & 63);
          // a slot taken twice: the priorities are not distinct
          if (atomicOr(&s_mask[(g * D + dv) * NWA + ((pr >> 6) - jb)], bit) & bit) s_acc[g].bad = 1u;
        }
        wave_sync();
        // a slot claimed on two devices is a repeated priority as well
        for (int i = lane; i < gc * NWA; i += 64) {
          const int g = i / NWA, w = i - g * NWA;
          unsigned long long x = 0ull;
          bool dup = false;
          for (int e = 0; e < D; ++e) {
            const unsigned long long y = s_mask[(g * D + e) * NWA + w];
            dup |= (x & y) != 0ull;
            x |= y;
          }
          if (dup) s_acc[g].bad = 1u;
        }
        wave_sync();
        const uint64_t rankedm = __ballot(lane < gc && s_acc[lane < gc ? lane : 0].bad != 0u);
        for (uint64_t rm = rankedm; rm; rm &= rm - 1ull) {
          const int g = __builtin_ctzll(rm);
          const uint8_t* pfl = s_fl + g * NB;
          for (int i = lane; i < D * NWA; i += 64) s_mask[g * D * NWA + i] = 0ull;
          wave_sync();
          for (int u = lo + lane; u < hi; u += 64) {
            const uint32_t a = t_act[u];
            const uint32_t fb = (uint32_t)pfl[u >> 2] >> ((u & 3) << 1);
            if ((fb & 1u) && (a & 64u)) continue;
            const int dv = ring_dev(g, u);
            if ((unsigned)dv >= (unsigned)D) continue;
            const int pu = ring_prio(g, u);
            int slot = lo;
            for (int j = lo; j < hi; ++j) {
              if (fuse_bit(pfl, j) && (t_act[j] & 64u)) continue;
              if ((unsigned)ring_dev(g, j) >= (unsigned)D) continue;
              const int pj = ring_prio(g, j);
              slot += (pj < pu) || (pj == pu && j < u);
            }
            s_rec[g * RW + (slot - lo)] = head_entry(g, u, a, fb);
            atomicOr(&s_mask[(g * D + dv) * NWA + ((slot >> 6) - jb)], 1ull << (slot & 63));
          }
          wave_sync();
        }
      }
      // ---- latest predecessor finish of the level's activations (Eq. 2):
      // one lane per incoming edge.  A fused chain member already holds its
      // own finish, which is later than its only predecessor's ----
      if (e1 > e0) {
        const uint32_t* t_ed = RING_FIN ? reinterpret_cast<const uint32_t*>(tb + sp.t.redge) : t_edge;
        for (int e = e0 + lane; e < e1; e += 64) {
          const uint32_t ed = t_ed[e];
          const int src = (int)(ed & 0xffffu), dst = (int)(ed >> 16);
          for (int g0 = 0; g0 < gc; g0 += kB) {
            TB f[kB];
#pragma unroll
            for (int k = 0; k < kB; ++k) {
              const int g = (g0 + k < gc) ? g0 + k : gc - 1;
              f[k] = s_fin[g * FS + src];
            }
#pragma unroll
            for (int k = 0; k < kB; ++k)
              if (g0 + k < gc) atomicMax(&s_fin[(g0 + k) * FS + dst], f[k]);
          }
        }
        wave_sync();
      }

      // ---- paper order: the pool's residency as the level starts ----
      if constexpr (PAPER) {
        for (int h = 0; h < NH; ++h) {
          if (NH > 1) {
            bind(h);
            res = s_hst[h * 64 + lane].res;
          }
          if (act) s_snap[gme * D + d] = res;
        }
        wave_sync();
      }

      // ---- device lanes walk their units of this level in slot order ----
      for (int h = 0; h < NH; ++h) {
      if (NH > 1) {
        bind(h);
        load(h);
      }
      if constexpr (PAPER) {
        others = 0ull;
        if (act)
          for (int e = 0; e < D; ++e)
            if (e != d) others |= s_snap[gme * D + e];
      }
      // (the queue modes keep the resident mask only for the replica check)
      if (!NIBBLE || sp.rcap) lv_hold = res;
      if (act) {
        const int j1 = (hi - 1) >> 6;
        const unsigned long long hmask = (hi & 63) ? ((1ull << (hi & 63)) - 1ull) : ~0ull;
        // a level of at most 64 slots: this device's slots of the level as
        // one word, slot lo at bit 0
        const int width = hi - lo;
        const bool narrow = width <= 64;
        int j = lo >> 6;
        // ring layout: the level's mask words and slot entries start at 0
        const int jo = RING ? (lo >> 6) : 0, ro = RING ? lo : 0;
        unsigned long long bits, wnext = 0ull;
        if (narrow) {
          const int sh = lo & 63;
          bits = mymask[j - jo] >> sh;
          if (sh + width > 64) bits |= mymask[j + 1 - jo] << (64 - sh);  // then j + 1 <= j1
          if (width < 64) bits &= (1ull << width) - 1ull;
        } else {
          // wider: the current word's remaining bits, and the next word
          // already loaded
          bits = mymask[j - jo] & (~0ull << (lo & 63));
          if (j < j1) wnext = mymask[j + 1 - jo] & ((j + 1 == j1) ? hmask : ~0ull);
        }
        // the device's next slot in the level; -1 when there is none, -2 for
        // a trip with no unit (an exhausted word followed by an empty one)
        auto next_narrow = [&]() -> int {
          const int sl = lo + __builtin_ctzll(bits | (1ull << 63));
          const bool have = bits != 0ull;
          bits &= bits - 1ull;
          return have ? sl : -1;
        };
        auto next_wide = [&]() -> int {
          const bool adv = bits == 0ull && j < j1;
          bits = adv ? wnext : bits;
          j += adv ? 1 : 0;
          const int jn = j + 1 <= j1 ? j + 1 : j1;
          const unsigned long long wl2 = mymask[jn - jo] & ((jn == j1) ? hmask : ~0ull);
          wnext = adv ? (j < j1 ? wl2 : 0ull) : wnext;
          const int sl = (j << 6) + __builtin_ctzll(bits | (1ull << 63));
          const bool have = bits != 0ull;
          bits &= bits - 1ull;
          return have ? sl : (j < j1 ? -2 : -1);
        };
        // slot entry; without a slot a stand-in (activation lo, model 0)
        // keeps every address below in range
        auto entry = [&](int sl) -> uint32_t {
          const uint32_t keep = (uint32_t)~(sl >> 31);  // all ones for a real slot
          const uint32_t raw = myrec[(int)((uint32_t)(sl - ro) & keep)];
          return (raw & keep) | ((uint32_t)lo & ~keep);
        };
        auto fetch = [&](int sl, uint32_t meta, UnitPre<TT>& p) {
          const uint32_t u = meta & 0xffffu, m = (meta >> 16) & 63u;
          p.meta = meta;
          p.slot = sl;
          const uint4 r = ud_d[__umul24(u, (uint32_t)D)];
          p.lat = (int32_t)r.x;
          p.mem = (int32_t)r.y;
          p.arrv = TO::words(r.z, r.w);
          p.rtv = TO::load(myfin + fpos((int)u));
          p.lw = lw_d[__umul24(m, (uint32_t)D)];
          if constexpr (PHI) {
            if constexpr (std::is_same<TT, uint32_t>::value)
              p.act = r.w;
            else
              p.act = t_act[u];
          }
        };
        // one unit of the device's sequence: reuse / reclaim / load, then
        // the timeline
        // one victim among the candidate copies `cand` (not empty): the
        // paper's order, or no remaining use first, then least recently used
        // (ascending ids: equal keys keep the lower id)
        auto victim_paper = [&](uint64_t cand) -> int {
          int v = __builtin_ctzll(cand);
          uint32_t vred = (uint32_t)((others >> v) & 1ull);
          uint32_t vnu = mynxu[v];
          uint32_t vld = wg_ld[__umul24((uint32_t)v, (uint32_t)D) + (uint32_t)d];
          uint32_t vlru = mystamp[v];
          for (cand &= cand - 1; cand; cand &= cand - 1) {
            const int m2 = __builtin_ctzll(cand);
            const uint32_t red = (uint32_t)((others >> m2) & 1ull);
            const uint32_t nu = mynxu[m2];
            const uint32_t ld = wg_ld[__umul24((uint32_t)m2, (uint32_t)D) + (uint32_t)d];
            const uint32_t lru = mystamp[m2];
            if (paper_victim_before(red, nu, ld, lru, vred, vnu, vld, vlru, (uint32_t)kdev)) {
              v = m2;
              vred = red;
              vnu = nu;
              vld = ld;
              vlru = lru;
            }
          }
          return v;
        };
        auto victim_lru = [&](uint64_t cand, int slot) -> int {
          int v = 0;
          uint32_t best = 0xffffffffu;
          while (cand) {
            const int m2 = __builtin_ctzll(cand);
            cand &= cand - 1;
            // a remaining use on the device: a later slot (ring layout: a
            // unit not yet walked)
            const uint32_t alive = RING ? (uint32_t)(mycnt[m2] != 0u) : (uint32_t)(mylast[m2] > (uint32_t)slot + 1u);
            const uint32_t key = (alive << 16) | mystamp[m2];
            if (key < best) {
              best = key;
              v = m2;
            }
          }
          return v;
        };
        auto process = [&](const UnitPre<TT>& X) {
          if (X.slot >= 0) {
            const int u = (int)(X.meta & 0xffffu);
            const int m = (int)((X.meta >> 16) & 63u);
            const uint64_t mbit = 1ull << m;
            if constexpr (RING) --mycnt[m];  // units of m on the device still to walk
            // copies reclaimed for this unit (schedule output), accumulated
            // in place so that nothing stays live in registers without one
            const bool rec_on = has_sched && sched.reclaimed_models != nullptr;
            if (rec_on) sched.reclaimed_models[pw * N + u] = 0ull;
            bool hit;
            int32_t w0 = 0, w1 = 0;
            if constexpr (!NIBBLE) hit = ((res >> m) & 1ull) != 0ull;
            if constexpr (NIBBLE) {
              // the queue holds exactly the resident models: m is resident
              // when it is found among the first nq entries (in the
              // still-needed part); it is taken out and re-enters as the most
              // recent
              const uint32_t m8 = (uint32_t)m * 0x11111111u;  // m in every nibble
              QT mq = (QT)m8;
              if constexpr (QB == 64) mq |= (QT)m8 << 32;
              const QT x = Q ^ mq;
              const QT z = (x - kOnes) & ~x & kHigh;  // lowest flag: first zero nibble
              int s4;  // 4 * position
              if constexpr (QB == 64)
                s4 = __builtin_ctzll(z | (1ull << 63)) & ~3;
              else
                s4 = __builtin_ctz(z | (1u << 31)) & ~3;
              hit = z != (QT)0 && (s4 >> 2) < nq;
              const QT low = Q & (((QT)1 << s4) - (QT)1);
              const QT high = (s4 >= kQBits - 4) ? (QT)0 : ((Q >> (s4 + 4)) << s4);
              Q = hit ? (low | high) : Q;
              nq -= hit ? 1 : 0;
              // the first two victims' weights, looked up ahead of need
              w0 = t_wmib[(int)(Q & (QT)15)];
              w1 = t_wmib[(int)((Q >> 4) & (QT)15)];
            }
            const TT r = TO::tmax(X.rtv, X.arrv);
            // run time (summed over a fused chain, Eq. 4) and memory (max)
            int32_t mxu = X.mem;
            inel |= (uint32_t)(X.lat < 0);
            uint32_t T = (uint32_t)X.lat;
            if (X.meta & kChain) {
              for (int v = t_cnext[u];;) {
                const int2 lm = *reinterpret_cast<const int2*>(ud_d + __umul24((uint32_t)v, (uint32_t)D));
                const int32_t lv2 = lm.x, mv = lm.y;
                inel |= (uint32_t)(lv2 < 0);
                T += (uint32_t)lv2;
                mxu = mv > mxu ? mv : mxu;
                const int c = t_cnext[v];
                if (c == 0xffff || !fuse_bit(myfl, c)) break;
                v = c;
              }
            }
            const int32_t need = (hit ? 0 : X.lw.y) + mxu;
            // batch limits: the slot that frees first, the first action's
            // time t, and the memory and leases of the units running at t
            int ks = 0;
            TT sft = bs_free[0], t0 = 0;
            int32_t run_act = 0;
            if constexpr (BATCH) {
#pragma unroll
              for (int k = 1; k < kMaxBatch; ++k)
                if (k < nbatch && bs_free[k] < sft) {
                  ks = k;
                  sft = bs_free[k];
                }
              t0 = TO::tmax(TO::tmax((!hit && (X.meta & kPf)) ? X.arrv : r, sft), bdisp);
              for (;;) {
                uint64_t leased = 0ull;
                TT nf = 0;
                bool any = false;
                run_act = 0;
#pragma unroll
                for (int k = 0; k < kMaxBatch; ++k) {
                  const bool running = k < nbatch && bs_fin[k] > t0;
                  run_act += running ? bs_mem[k] : 0;
                  leased |= running ? (1ull << bs_model[k]) : 0ull;
                  nf = running && (!any || bs_fin[k] < nf) ? bs_fin[k] : nf;
                  any |= running;
                }
                // reclaim lease-free copies (Sec. 3.5) in the window's order
                while (used + run_act + need > capd) {
                  const uint64_t cand = res & ~mbit & ~leased;
                  if (!cand) break;
                  int v;
                  if constexpr (PAPER)
                    v = victim_paper(cand);
                  else
                    v = victim_lru(cand, X.slot);
                  res &= ~(1ull << v);
                  if constexpr (PHI) ph_rec |= 1ull << v;
                  if (rec_on) sched.reclaimed_models[pw * N + u] |= 1ull << v;
                  used -= t_wmib[v];
                  ++nev;
                }
                // fits, or no running unit left to wait for
                if (!(used + run_act + need > capd) || !any) break;
                t0 = nf;
              }
              mystamp[m] = (uint16_t)seq++;
              if constexpr (PAPER) {
                mynxu[m] = s_nx[gme * N + X.slot];
                ++kdev;
              }
            } else if constexpr (NIBBLE) {
              // reclaim (Sec. 3.5): a copy with no remaining use first, else
              // the least recently used, else the lower model id
              int t = 0;
              while (used + need > capd && nq > 0) {
                const int v = (int)(Q & (QT)15);
                if constexpr (PHI) ph_rec |= 1ull << v;
                if (rec_on) sched.reclaimed_models[pw * N + u] |= 1ull << v;
                if (sp.rcap) res &= ~(1ull << v);
                Q >>= 4;
                --nq;
                nd = nd > 0 ? nd - 1 : 0;
                int32_t wv = t ? w1 : w0;
                if (t >= 2) wv = t_wmib[v];
                used -= wv;
                ++nev;
                ++t;
              }
              // m re-enters after the no-remaining-use part when this was its
              // last unit on the device, else at the end
              const bool last_use = (X.meta & kLast) != 0u;
              const int pos = 4 * (last_use ? nd : nq);  // nq < QB / 4 here
              const QT lowm = ((QT)1 << pos) - (QT)1;
              Q = (Q & lowm) | ((QT)m << pos) | ((Q & ~lowm) << 4);
              nd += last_use ? 1 : 0;
              ++nq;
            } else if constexpr (PAPER) {
              (void)w0;
              (void)w1;
              while (used + need > capd) {
                const uint64_t cand = res & ~mbit;
                if (!cand) break;
                const int v = victim_paper(cand);
                res &= ~(1ull << v);
                if constexpr (PHI) ph_rec |= 1ull << v;
                if (rec_on) sched.reclaimed_models[pw * N + u] |= 1ull << v;
                used -= t_wmib[v];
                ++nev;
              }
              mystamp[m] = (uint16_t)seq++;
              mynxu[m] = s_nx[gme * N + X.slot];
              ++kdev;
            } else {
              (void)w0;
              (void)w1;
              while (used + need > capd) {
                const uint64_t cand = res & ~mbit;
                if (!cand) break;
                const int v = victim_lru(cand, X.slot);
                res &= ~(1ull << v);
                if constexpr (PHI) ph_rec |= 1ull << v;
                if (rec_on) sched.reclaimed_models[pw * N + u] |= 1ull << v;
                used -= t_wmib[v];
                ++nev;
              }
              mystamp[m] = (uint16_t)seq++;
            }
            const bool over = used + run_act + need > capd;
            capbad |= (uint32_t)over;
            // timeline (Eq. 7): a load waits for the device (a slot) and
            // starts at the release, or at the workflow arrival when
            // prefetched
            const TT dev_free = BATCH ? sft : freet;
            const TT ls = BATCH ? t0 : TO::tmax((X.meta & kPf) ? X.arrv : r, freet);
            const TT le = TO::add(ls, (uint32_t)X.lw.x);
            const TT s = BATCH ? (hit ? t0 : TO::tmax(r, le)) : TO::tmax(r, hit ? freet : le);
            // ready work: no predecessor, arrived by the window time
            const bool ready = PHI && ((X.act >> 7) & 1u);
            if constexpr (PHI) {
              if (!hit) {
                // a reload of a copy this plan reclaimed from the device
                if ((ph_rec >> m) & 1ull) ph_h += (HT)(uint32_t)X.lw.x;
                // a prefetch is timely when its load is done by the release
                if (!ready && (X.meta & kPf) && le <= r) ++ph_pn;
                // the delay a load adds to ready work
                if (ready) ph_h += (HT)TO::sub(s, TO::tmax(r, dev_free));
              }
            }
            if (!NIBBLE || sp.rcap) {
              res |= mbit;
              lv_hold |= mbit;
            }
            used += hit ? 0 : X.lw.y;
            nld += hit ? 0u : 1u;
            peak = (used + run_act + mxu) > peak ? (used + run_act + mxu) : peak;
            const TT f = TO::add(s, T);
            if constexpr (BATCH) {
#pragma unroll
              for (int k = 0; k < kMaxBatch; ++k) {
                const bool mine = k == ks;
                bs_free[k] = mine ? f : bs_free[k];
                bs_fin[k] = mine ? f : bs_fin[k];
                bs_mem[k] = mine ? mxu : bs_mem[k];
                bs_model[k] = mine ? m : bs_model[k];
              }
              bdisp = t0;
            }
            if constexpr (PHI) {
              if (ready && !over) {
                ph_adm += 1ull << (16u * ((X.act >> 8) & 3u));
                ph_cf = TO::tmax(ph_cf, f);
              }
            }
            freet = f;
            if (!(X.meta & kSlow)) {
              myfin[fpos(u)] = TO::bits(f);
            } else {
              TT t = s;
              for (int v = u;;) {
                const TT tv =
                    TO::add(t, ud_d[__umul24((uint32_t)v, (uint32_t)D)].x);
                myfin[fpos(v)] = TO::bits(tv);
                if (has_sched) {
                  sched.start_us[pw * N + v] = sp.origin + TO::i64(t);
                  sched.finish_us[pw * N + v] = sp.origin + TO::i64(tv);
                  sched.load_start_us[pw * N + v] =
                      (v == u && !hit) ? sp.origin + TO::i64(ls) : (int64_t)-1;
                  if (rec_on && v != u) sched.reclaimed_models[pw * N + v] = 0ull;
                }
                t = tv;
                const int c = t_cnext[v];
                if (c == 0xffff || !fuse_bit(myfl, c)) break;
                v = c;
              }
            }
          }
        };
        // two units per trip so that the prefetched unit needs no copy; one
        // copy of the loop per kind of level
        auto run = [&](auto&& next_slot) {
          UnitPre<TT> A, B;
          {
            const int sa = next_slot();
            fetch(sa, entry(sa), A);
          }
          int sb = A.slot != -1 ? next_slot() : -1;
          uint32_t mb_next = entry(sb);
          while (A.slot != -1) {
            fetch(sb, mb_next, B);
            const int sc = sb != -1 ? next_slot() : -1;
            const uint32_t mc = entry(sc);
            process(A);
            if (B.slot == -1) break;
            fetch(sc, mc, A);
            sb = sc != -1 ? next_slot() : -1;
            mb_next = entry(sb);
            process(B);
          }
        };
        if (narrow)
          run(next_narrow);
        else
          run(next_wide);
      }
      if (sp.rcap && act) s_hold[gme * D + d] = lv_hold;
      if (NH > 1) save(h);
      }
      wave_sync();
      // ---- replica caps (Sec. 3.5 scale-out): a model held or loaded in
      // this level on more devices than its cap; lanes over (plan, model) ----
      if (sp.rcap) {
        for (int it = lane; it < gc * M; it += 64) {
          const int g = it / M, m = it - g * M;
          int copies = 0;
          for (int e = 0; e < D; ++e) copies += (int)((s_hold[g * D + e] >> m) & 1ull);
          if (copies > t_rcap[m]) atomicOr(&s_acc[g].status, (uint32_t)WF_ST_REPLICA);
        }
        wave_sync();
      }
    }

    // ---- per-plan reductions (Sec. 4 metrics) ----
    for (int h = 0; h < NH; ++h) {
    if (NH > 1) {
      bind(h);
      load(h);
    }
    if (act) {
      atomicMin(&s_acc[gme].headroom, capd - peak);
      atomicAdd(&s_acc[gme].loads, nld);
      atomicAdd(&s_acc[gme].evicts, nev);
      if (capbad) atomicOr(&s_acc[gme].status, (uint32_t)WF_ST_CAPACITY);
      if constexpr (std::is_same<TT, uint32_t>::value) {
        // a saturated time ends in the device's last finish
        TT last = freet;
        if constexpr (BATCH) {
#pragma unroll
          for (int k = 0; k < kMaxBatch; ++k) last = TO::tmax(last, bs_free[k]);
        }
        if (last == 0xffffffffu) atomicOr(&s_acc[gme].status, kRescore);
      }
      if (inel) atomicOr(&s_acc[gme].status, (uint32_t)WF_ST_INELIGIBLE);
      if (has_sched) sched.peak_mib[pw * D + d] = peak;
      if constexpr (PHI) {
        if (ph_adm) {
          atomicAdd(&s_acc[gme].ph_adm, ph_adm);
          atomicMax(&s_acc[gme].ph_cf, (unsigned long long)TO::bits(ph_cf));
        }
        if (ph_pn) atomicAdd(&s_acc[gme].ph_pn, ph_pn);
        // exact: an integer below 2^53 with fp64 times
        if (ph_h) atomicAdd(&s_acc[gme].ph_h, (unsigned long long)ph_h);
      }
    }
    }
    // a workflow's completion is the latest finish among its activations
    // without a successor in the same workflow (not part of the ranking key);
    // the ring layout folded every level but its last ring_b + 1 during the
    // walk
    if constexpr (RING_FIN) {
      if (!PHI)
        for (int L = sp.n_levels - sp.ring_b - 1 > 0 ? sp.n_levels - sp.ring_b - 1 : 0; L < sp.n_levels; ++L)
          ring_level(L, false);
    }
    for (int i = lane; i < ((PHI || RING_FIN) ? 0 : sp.S); i += 64) {
      const uint32_t sk = t_sink[i];
      const int src = (int)(sk & 0xffffu), wf = (int)(sk >> 16);
      for (int g0 = 0; g0 < gc; g0 += kB) {
        TB f[kB];
#pragma unroll
        for (int k = 0; k < kB; ++k) {
          const int g = (g0 + k < gc) ? g0 + k : gc - 1;
          f[k] = s_fin[g * N + src];
        }
#pragma unroll
        for (int k = 0; k < kB; ++k)
          if (g0 + k < gc) atomicMax(&s_wfm[(g0 + k) * W + wf], f[k]);
      }
    }
    wave_sync();
    // completion latencies in place, and the latest finish
    for (int it = lane; it < (PHI ? 0 : gc * W); it += 64) {
      const int g = it / W, a = it - g * W;
      const TB fb = s_wfm[it];
      atomicMax(&s_acc[g].max_finish, (unsigned long long)fb);
      s_wfm[it] = TO::bits(TO::sub(TO::load(&fb), TO::load(t_arr + a)));
    }
    wave_sync();
    // nearest-rank p95: the ceil(0.95 W)-th smallest completion latency,
    // lanes over (plan, workflow)
    const int kk = (95 * W + 99) / 100;
    for (int it = lane; it < (PHI ? 0 : gc * W); it += 64) {
      const int g = it / W;
      const TB* cw = s_wfm + g * W;
      const TT ca = TO::load(cw + (it - g * W));
      int lt = 0, le = 0;
#pragma unroll 8
      for (int b = 0; b < W; ++b) {
        const TT cb = TO::load(cw + b);
        lt += cb < ca;
        le += cb <= ca;
      }
      if (lt < kk && kk <= le) s_acc[g].p95 = TO::i64(ca);
    }
    wave_sync();
    if (PHI && lane < gc) {
      const PlanAcc a = s_acc[lane];
      wf_plan_key k;
      k.c_ready_us = 0;
      k.h_life_us = 0;
      for (int c = 0; c < WF_MAX_CLASSES; ++c) k.admitted[c] = 0;
      k.timely_prefetch = 0;
      k.pad = 0;
      k.status = (a.status & WF_ST_INELIGIBLE) ? (uint32_t)WF_ST_INELIGIBLE : a.status;
      if (!(a.status & WF_ST_INELIGIBLE)) {
        if (a.ph_adm)
          k.c_ready_us = sp.origin + TO::i64(TO::load(reinterpret_cast<const TB*>(&a.ph_cf)));
        k.h_life_us = (int64_t)a.ph_h;
        for (int c = 0; c < WF_MAX_CLASSES; ++c)
          k.admitted[c] = (uint16_t)((a.ph_adm >> (16 * c)) & 0xffffull);
        k.timely_prefetch = (uint16_t)(a.ph_pn > 65535u ? 65535u : a.ph_pn);
      }
      reinterpret_cast<wf_plan_key*>(scores)[p0 + lane] = k;
    } else if (lane < gc) {
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
      reinterpret_cast<wf_plan_score*>(scores)[p0 + lane] = sc;
    }
    wave_sync();
  }
}

template <typename TT, bool TAB_LDS, int QB, int PLACE, bool SEARCH, bool PHI, bool SCHED>
hipError_t launch_variant(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                          const uint8_t* flags, int64_t n_plans, OutRec<PHI>* out,
                          const wf_plan_sched& s, int has, const SearchArgs& sa,
                          hipStream_t stream) {
  auto k = score_plans<TT, TAB_LDS, QB, PLACE, SEARCH, PHI, SCHED>;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                            hipFuncAttributeMaxDynamicSharedMemorySize, sp.lds_bytes);
  hipLaunchKernelGGL(k, dim3(sp.grid), dim3(64 * sp.waves), sp.lds_bytes, stream, sp, dev, prio,
                     flags, n_plans, out, s, has, sa);
  return hipGetLastError();
}

template <typename TT, int QB, bool SEARCH, bool PHI, bool SCHED>
hipError_t launch_place(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                        const uint8_t* flags, int64_t n_plans, OutRec<PHI>* out,
                        const wf_plan_sched& s, int has, const SearchArgs& sa, hipStream_t stream) {
  if constexpr ((QB == -1 || QB == -3) && !SEARCH) {
    if (sp.ring == 2)
      return launch_variant<TT, false, QB, 4, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans,
                                                                  out, s, has, sa, stream);
  }
  if constexpr (QB == 0 || QB == -2) {
    if (sp.ring)
      return launch_variant<TT, false, QB, 2, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans,
                                                                  out, s, has, sa, stream);
  }
  if (sp.wave_global)
    return launch_variant<TT, false, QB, 1, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans,
                                                                out, s, has, sa, stream);
  if (sp.tab_in_lds)
    return launch_variant<TT, true, QB, 0, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans,
                                                               out, s, has, sa, stream);
  return launch_variant<TT, false, QB, 0, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans,
                                                              out, s, has, sa, stream);
}

template <typename TT, bool SEARCH, bool PHI, bool SCHED>
hipError_t launch_time(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                       const uint8_t* flags, int64_t n_plans, OutRec<PHI>* out,
                       const wf_plan_sched& s, int has, const SearchArgs& sa, hipStream_t stream) {
  switch (sp.nibble) {
    case -1:
      return launch_place<TT, -1, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
    case -2:
      return launch_place<TT, -2, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
    case -3:
      return launch_place<TT, -3, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
    case 32:
      return launch_place<TT, 32, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
    case 64:
      return launch_place<TT, 64, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
    default:
      return launch_place<TT, 0, SEARCH, PHI, SCHED>(sp, dev, prio, flags, n_plans, out, s, has, sa, stream);
  }
}

// Plans from HBM rows, or candidates generated around an incumbent; fp64 or
// uint32 times; with or without the schedule output (rows from HBM only).
template <bool PHI>
hipError_t launch_all(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                      const uint8_t* flags, int64_t n_plans, OutRec<PHI>* out,
                      const wf_plan_sched* sched, const SearchArgs* search, hipStream_t stream) {
  wf_plan_sched s{};
  if (sched) s = *sched;
  const SearchArgs sa = search ? *search : SearchArgs{};
  if constexpr (!PHI) {
    if (sched && !search) {
      if (sp.time64)
        return launch_time<double, false, false, true>(sp, dev, prio, flags, n_plans, out, s, 1, sa, stream);
      return launch_time<uint32_t, false, false, true>(sp, dev, prio, flags, n_plans, out, s, 1, sa, stream);
    }
  }
  if (sp.time64) {
    if (search) return launch_time<double, true, PHI, false>(sp, dev, prio, flags, n_plans, out, s, 0, sa, stream);
    return launch_time<double, false, PHI, false>(sp, dev, prio, flags, n_plans, out, s, 0, sa, stream);
  }
  if (search) return launch_time<uint32_t, true, PHI, false>(sp, dev, prio, flags, n_plans, out, s, 0, sa, stream);
  return launch_time<uint32_t, false, PHI, false>(sp, dev, prio, flags, n_plans, out, s, 0, sa, stream);
}

}  // namespace
}  // namespace wfp
