// The lean scoring kernel: windows whose times fit uint32 offsets, with at
// most 16 models and at most 512 activations -- the configuration the
// throughput workload (256 activations x 1,048,576 plans) runs in.  Same
// results as the general kernel of score_kernel.h, with only the code these
// windows need: 16-bit slot entries, uint32 times, no schedule, and the
// per-unit tables of the walk in LDS.  Variants (template parameters): the
// default reclamation order on a queue of 4-bit model ids (QB = 32 or 64)
// or the paper's order over a resident mask (QB = -1); ranking keys of Eq.
// 12 instead of scores (PHI); replica caps (RCAP); batch limits (BATCH).
// With SEARCH the plans are candidates generated around an incumbent (at
// most kPatchMaxMut mutations each): a candidate is kept as the incumbent's
// rows plus the sites its mutations changed (in the finish array's storage,
// dead until the walk), and the order sweep patches the incumbent's row
// words with them, so no candidate row exists in HBM or LDS.
//
// A persistent grid of waves loops over groups of G plans; lane (g, d) =
// (lane / D, lane % D) owns device d of plan g.  Per group:
//   1. flag rows are staged into LDS; the resource order (Eq. 10) puts each
//      unit head at slot = its priority when each level's head priorities
//      are distinct values of the level's index range (checked by counting),
//      else at its rank by (priority, index) within the level; a 16-bit slot
//      entry, the device's slot mask and each (device, model)'s last slot are
//      recorded, and the last slots become flags in the slot entries;
//   2. per topological level, releases (Eq. 2) by LDS atomic max over the
//      level's incoming edges, then each device lane walks its units of the
//      level in slot order: reuse / reclaim / load (Eq. 5, Eq. 11) and the
//      max-plus timeline of Eq. 7;
//   3. makespan, nearest-rank p95, objective, headroom and counts (or the
//      ranking key).
// Memory is tracked as the excess of a unit's need over the device's free
// memory: a unit fits when its excess after reclamation is <= 0, the device's
// peak is its capacity plus the largest such excess, so the peak, the
// CAPACITY test and the headroom need one max per unit.
#include <type_traits>

#include "kernels.h"
#include "mutation.h"

namespace wfp {
namespace {

// (ranking keys: loads holds the timely prefetches P_N, max_finish and p95
// together the 64-bit count of admitted ready units per class)
struct LeanAcc {
  uint32_t status;
  int32_t headroom;
  uint32_t loads;
  uint32_t evicts;
  uint32_t max_finish;  // relative time
  uint32_t p95;         // selected completion latency
  uint32_t heads;       // unit heads given a slot by the first ordering try
  uint32_t claimed;     // distinct slots they occupy
  uint32_t bad;         // a head priority outside its level's index range
  uint32_t cf;          // ranking keys: latest admitted ready finish
  unsigned long long h_life;  // ranking keys: lifecycle overhead
};
static_assert(sizeof(LeanAcc) == 48, "LeanAcc layout");

// slot entry
constexpr uint32_t kEAct = 0x1ffu;
constexpr uint32_t kEPf = 1u << 13;
constexpr uint32_t kEChain = 1u << 14;
constexpr uint32_t kELast = 1u << 15;  // the model's last unit on the device (set before the walk)

__device__ __forceinline__ void lsync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ void zero16(unsigned char* dst, int nbytes, int lane) {
  uint4* d = reinterpret_cast<uint4*>(dst);
  const int n16 = nbytes >> 4;
  for (int i = lane; i < n16; i += 64) d[i] = make_uint4(0u, 0u, 0u, 0u);
  for (int i = (n16 << 4) + lane; i < nbytes; i += 64) dst[i] = 0;
}

__device__ __forceinline__ void stage_rows(unsigned char* dst, const unsigned char* src, int nbytes,
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

__device__ __forceinline__ uint32_t fuse_of(const uint8_t* fl, int v) {
  return ((uint32_t)fl[v >> 2] >> ((v & 3) << 1)) & 1u;
}

// uint32 time addition: saturating when the window's bound is not proven
// below 2^32 (a saturated time only grows through the max-plus steps, so it
// ends in its device's last finish, where it is detected)
template <bool CHECKED>
__device__ __forceinline__ uint32_t tadd(uint32_t a, uint32_t b) {
  if constexpr (CHECKED)
    return __builtin_elementwise_add_sat(a, b);
  else
    return a + b;
}

__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }

// PHI: each plan's ranking key (Eq. 12) is written instead of its score.
// RCAP: the window caps replicas (a resident mask beside the queue).
// BATCH: devices run up to their batch limit of units at once (plan scores
// only).  QB = -1: the paper's reclamation order over a resident mask, no
// queue (plan scores only).
// Variants built for three waves per SIMD: every queue variant (some
// registers of the key, replica-cap and batch variants spill, which costs
// less than the waves gained where LDS holds more than eight); the paper's
// order keeps two.
template <bool SEARCH, bool PHI, bool RCAP, bool BATCH, int QB>
constexpr bool lean_plain() {
  return QB > 0;
}

template <bool CHECKED, int QB, bool SEARCH, bool PHI, bool RCAP, bool BATCH>
__global__ __launch_bounds__(64 * (lean_plain<SEARCH, PHI, RCAP, BATCH, QB>() ? kLeanPlainWaves
                                                                                : kLeanWaves))
void score_lean(ScoreParams sp, LeanParams lp,
                                                  const int8_t* __restrict__ dev_all,
                                                  const uint16_t* __restrict__ prio_all,
                                                  const uint8_t* __restrict__ flags_all, int64_t P,
                                                  wf_plan_score* __restrict__ scores, SearchArgs sa) {
  using QT = std::conditional_t<QB == 32, uint32_t, uint64_t>;
  constexpr QT kOnes = (QT)0x1111111111111111ull, kHigh = (QT)0x8888888888888888ull;
  static_assert(!BATCH || (!SEARCH && !PHI && !RCAP), "batch limits: plan scores only");
  constexpr bool PAPER = QB < 0;
  static_assert(!PAPER || (!SEARCH && !PHI && !RCAP && !BATCH), "the paper's order: plan scores only");
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int N = sp.N, W = sp.W, M = sp.M, D = sp.D, NB = sp.NB, G = lp.G, NWA = sp.nwa;

  // ---- window tables: the per-unit ones in LDS, the rest through the cache ----
  {
    const uint4* src = reinterpret_cast<const uint4*>(lp.tab);
    uint4* dst = reinterpret_cast<uint4*>(lds);
    for (int i = tid; i < (lp.t.lds_bytes >> 4); i += blockDim.x) dst[i] = src[i];
  }
  __syncthreads();
  const unsigned char* tg = lp.tab;
  const int4* t_lw = reinterpret_cast<const int4*>(lds + lp.t.lw);
  const int32_t* t_wmib = reinterpret_cast<const int32_t*>(lds + lp.t.wmib);
  const uint32_t* t_aarr = reinterpret_cast<const uint32_t*>(lds + lp.t.aarr);
  const int32_t* t_rcap = reinterpret_cast<const int32_t*>(lds + lp.t.rcap);
  const int2* t_um = reinterpret_cast<const int2*>(tg + lp.t.um);
  const uint32_t* t_act = reinterpret_cast<const uint32_t*>(tg + lp.t.act);
  const uint32_t* t_alv = reinterpret_cast<const uint32_t*>(tg + lp.t.alv);
  const uint16_t* t_cnext = reinterpret_cast<const uint16_t*>(tg + lp.t.cnext);
  const uint32_t* t_edge = reinterpret_cast<const uint32_t*>(tg + lp.t.edge);
  const int32_t* t_eoff = reinterpret_cast<const int32_t*>(tg + lp.t.eoff);
  const int32_t* t_loff = reinterpret_cast<const int32_t*>(tg + lp.t.loff);
  const int32_t* t_cap = reinterpret_cast<const int32_t*>(tg + lp.t.cap);
  const uint32_t* t_arr = reinterpret_cast<const uint32_t*>(tg + lp.t.arr);
  const unsigned long long* t_res0 = reinterpret_cast<const unsigned long long*>(tg + lp.t.res0);
  const uint32_t* t_free0 = reinterpret_cast<const uint32_t*>(tg + lp.t.free0);
  const uint32_t* t_sink = reinterpret_cast<const uint32_t*>(tg + lp.t.sink);
  const int32_t* t_batch = reinterpret_cast<const int32_t*>(tg + lp.t.batch);

  // ---- this wave's LDS region ----
  unsigned char* wl = lds + lp.t.lds_bytes + lp.wo.bytes * wid;
  uint8_t* s_fl = wl + lp.wo.flags;
  uint16_t* s_rec = reinterpret_cast<uint16_t*>(wl + lp.wo.rec);
  unsigned long long* s_mask = reinterpret_cast<unsigned long long*>(wl + lp.wo.mask);
  uint32_t* s_last = reinterpret_cast<uint32_t*>(wl + lp.wo.last);
  uint32_t* s_fin = reinterpret_cast<uint32_t*>(wl + lp.wo.fin);
  uint32_t* s_wfm = reinterpret_cast<uint32_t*>(wl + lp.wo.wfm);
  LeanAcc* s_acc = reinterpret_cast<LeanAcc*>(wl + lp.wo.acc);
  uint32_t* s_pat = s_fin;  // generated candidates' changed sites (until the walk)
  uint16_t* s_hold = reinterpret_cast<uint16_t*>(wl + lp.wo.hold);  // replica caps
  // the paper's order: resident models of each device as the level starts
  // (in the replica caps' region), next use per slot
  uint16_t* s_snap = s_hold;
  uint16_t* s_nx = reinterpret_cast<uint16_t*>(wl + lp.wo.nx);
  uint8_t* s_nx8 = wl + lp.wo.nx;  // at most 256 activations: one byte, 0 for none
  const bool nx8 = N <= 256;

  const int g_me = lane / D;
  const int d_me = lane - g_me * D;
  const int64_t n_groups = (P + G - 1) / G;
  const int64_t stride = (int64_t)gridDim.x * lp.waves;
  // this lane's device rows
  const int2* um_d = t_um + d_me * N;
  const int4* lw_d = t_lw + d_me * M;

  // rows read four activations per lane with 4- and 8-byte loads
  const bool vec = (N & 3) == 0 && (reinterpret_cast<uintptr_t>(dev_all) & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(prio_all) & 7) == 0;
  // the order sweep takes four plans at a time (all their row loads issued
  // before any is used)
  constexpr int kB = 4;
  const bool pre = false;
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
    const int64_t g_first = (int64_t)blockIdx.x * lp.waves + wid;
    if (pre && g_first < n_groups) load_rows(g_first, dvp, pvp);
  }

  for (int64_t grp = (int64_t)blockIdx.x * lp.waves + wid; grp < n_groups; grp += stride) {
    const int64_t p0 = grp * G;
    const int gc = (int)((P - p0) < G ? (P - p0) : G);

    if constexpr (SEARCH) {
      // every plan starts as the incumbent; lane g then applies candidate
      // g's mutations to its changed sites and flag row
      for (int i = lane; i < gc * NB; i += 64) s_fl[i] = flags_all[i - (i / NB) * NB];
      lsync();
      if (lane < gc) {
        PatchRows rows{s_pat + lane * kPatchWords, dev_all, prio_all, s_fl + lane * NB};
        rows.p[0] = 0u;
        mutate_rows((uint64_t)(sa.first + p0 + lane), sa, N, sa.elig, t_alv, rows);
      }
    } else {
      stage_rows(s_fl, flags_all + p0 * NB, gc * NB, lane);
    }
    zero16(reinterpret_cast<unsigned char*>(s_last), G * D * M * 4, lane);
    zero16(reinterpret_cast<unsigned char*>(s_mask), G * D * NWA * 8, lane);
    if (lane < G) {
      LeanAcc a0{};
      a0.headroom = 0x7fffffff;
      s_acc[lane] = a0;
    }
    lsync();

    // device and priority of activation u in plan g
    auto rdev = [&](int g, int u) -> int {
      if constexpr (SEARCH) {
        const PatchRows rows{s_pat + g * kPatchWords, dev_all, prio_all, nullptr};
        return rows.dev(u);
      } else {
        return dev_all[(p0 + g) * N + u];
      }
    };
    auto rprio = [&](int g, int u) -> int {
      if constexpr (SEARCH) {
        const PatchRows rows{s_pat + g * kPatchWords, dev_all, prio_all, nullptr};
        const int k = rows.find(u);
        return k >= 0 ? (int)(rows.p[1 + 2 * k] >> 16) : (int)prio_all[u];
      } else {
        return prio_all[(p0 + g) * N + u];
      }
    };
    // the incumbent's row words at activations uc .. uc + 3 with candidate
    // g's changed sites written in
    auto patch4 = [&](int g, int uc, uint32_t& dv, uint2& pv) {
      const uint32_t* pp = s_pat + g * kPatchWords;
      const int n = (int)pp[0];
      for (int k = 0; k < n; ++k) {
        const uint32_t e0 = pp[1 + 2 * k];
        const uint32_t o = (e0 & 0xffffu) - (uint32_t)uc;
        if (o < 4u) {
          const uint32_t sh = o << 3, ph = (o & 1u) << 4, pr = e0 >> 16;
          dv = (dv & ~(0xffu << sh)) | ((pp[2 + 2 * k] & 0xffu) << sh);
          if (o < 2u)
            pv.x = (pv.x & ~(0xffffu << ph)) | (pr << ph);
          else
            pv.y = (pv.y & ~(0xffffu << ph)) | (pr << ph);
        }
      }
    };

    // ---- resource order (Eq. 10), first try: slot = priority ----
    auto order_one = [&](int g, int u, int d, int pr, uint32_t a, uint32_t lvw, uint32_t c,
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
        s_rec[g * N + pr] =
            (uint16_t)((uint32_t)u | (m << 9) | ((fb & 2u) << 12) | (chain ? kEChain : 0u));
        atomicOr(&s_mask[(g * D + d) * NWA + (pr >> 6)], 1ull << (pr & 63));
        atomicMax(&s_last[(g * D + d) * M + (int)m], (uint32_t)pr + 1u);
        ++nh;
      }
    };
    auto flush4 = [&](int g, uint32_t nh, uint32_t nbad, uint32_t ninel) {
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
    if (vec) {
      for (int base = 0; base < N; base += 256) {
        const int u0 = base + 4 * lane;
        const bool live = u0 < N;
        const int uc = live ? u0 : 0;
        const uint4 act4 = *reinterpret_cast<const uint4*>(t_act + uc);
        const uint4 alv4 = *reinterpret_cast<const uint4*>(t_alv + uc);
        const uint2 cn4 = *reinterpret_cast<const uint2*>(t_cnext + uc);
        // (generated candidates: the incumbent's words, the same for every plan)
        const uint32_t idv = SEARCH ? *reinterpret_cast<const uint32_t*>(dev_all + uc) : 0u;
        const uint2 ipv = SEARCH ? *reinterpret_cast<const uint2*>(prio_all + uc) : make_uint2(0u, 0u);
        const uint32_t cn[4] = {cn4.x & 0xffffu, cn4.x >> 16, cn4.y & 0xffffu, cn4.y >> 16};
        for (int g0 = 0; g0 < gc; g0 += kB) {
          uint32_t dv[kB], fl[kB], cb[kB][4];
          uint2 pv[kB];
#pragma unroll
          for (int k = 0; k < kB; ++k) {
            const int g = (g0 + k < gc) ? g0 + k : gc - 1;
            if constexpr (SEARCH) {
              dv[k] = idv;
              pv[k] = ipv;
              patch4(g, uc, dv[k], pv[k]);
            } else if (pre) {
              dv[k] = dvp[k];
              pv[k] = pvp[k];
            } else {
              dv[k] = *reinterpret_cast<const uint32_t*>(dev_all + (p0 + g) * N + uc);
              pv[k] = *reinterpret_cast<const uint2*>(prio_all + (p0 + g) * N + uc);
            }
          }
#pragma unroll
          for (int k = 0; k < kB; ++k) {
            const int g = (g0 + k < gc) ? g0 + k : gc - 1;
            fl[k] = s_fl[g * NB + (uc >> 2)];
#pragma unroll
            for (int j = 0; j < 4; ++j)
              cb[k][j] = sp.has_chains
                             ? s_fl[g * NB + ((cn[j] != 0xffffu ? cn[j] : (uint32_t)uc) >> 2)]
                             : 0u;
          }
#pragma unroll
          for (int k = 0; k < kB; ++k) {
            const int g = g0 + k;
            if (g >= gc) break;
            uint32_t nh = 0, nbad = 0, ninel = 0;
            if (live) {
              order_one(g, uc, (int)(int8_t)(dv[k] & 0xffu), (int)(pv[k].x & 0xffffu), act4.x,
                        alv4.x, cn[0], fl[k], cb[k][0], nh, nbad, ninel);
              order_one(g, uc + 1, (int)(int8_t)((dv[k] >> 8) & 0xffu), (int)(pv[k].x >> 16),
                        act4.y, alv4.y, cn[1], fl[k] >> 2, cb[k][1], nh, nbad, ninel);
              order_one(g, uc + 2, (int)(int8_t)((dv[k] >> 16) & 0xffu), (int)(pv[k].y & 0xffffu),
                        act4.z, alv4.z, cn[2], fl[k] >> 4, cb[k][2], nh, nbad, ninel);
              order_one(g, uc + 3, (int)(int8_t)(dv[k] >> 24), (int)(pv[k].y >> 16), act4.w,
                        alv4.w, cn[3], fl[k] >> 6, cb[k][3], nh, nbad, ninel);
            }
            flush4(g, nh, nbad, ninel);
          }
        }
      }
    } else {
      for (int g = 0; g < gc; ++g) {
        const uint8_t* pfl = s_fl + g * NB;
        uint32_t nh = 0, nbad = 0, ninel = 0;
        for (int u = lane; u < N; u += 64) {
          const uint32_t fb = (uint32_t)pfl[u >> 2] >> ((u & 3) << 1);
          const uint32_t c = t_cnext[u];
          const uint32_t cbyte = pfl[(c != 0xffffu ? c : (uint32_t)u) >> 2];
          order_one(g, u, rdev(g, u), rprio(g, u), t_act[u], t_alv[u], c, fb, cbyte, nh, nbad,
                    ninel);
        }
        if (ninel) atomicOr(&s_acc[g].status, (uint32_t)WF_ST_INELIGIBLE);
        if (nbad) atomicOr(&s_acc[g].bad, 1u);
        if (nh) atomicAdd(&s_acc[g].heads, nh);
      }
    }
    lsync();
    // distinct slots claimed per plan: the union of its devices' masks
    for (int i = lane; i < gc * NWA; i += 64) {
      const int g = i / NWA, w = i - g * NWA;
      unsigned long long x = 0ull;
      for (int d = 0; d < D; ++d) x |= s_mask[(g * D + d) * NWA + w];
      if (x) atomicAdd(&s_acc[g].claimed, (uint32_t)__popcll(x));
    }
    lsync();
    uint64_t rankedm;
    {
      const LeanAcc& ag = s_acc[lane < gc ? lane : 0];  // G <= 64
      rankedm = __ballot(lane < gc && (ag.bad != 0u || ag.heads != ag.claimed));
    }
    // plans whose priorities are not a permutation of each level's heads'
    // index range: rank by (priority, index) within each level
    for (uint64_t rm = rankedm; rm; rm &= rm - 1ull) {
      const int g = __builtin_ctzll(rm);
      const uint8_t* pfl = s_fl + g * NB;
      uint16_t* rec = s_rec + g * N;
      unsigned long long* mk = s_mask + g * D * NWA;
      uint32_t* lastp = s_last + g * D * M;
      for (int i = lane; i < D * NWA; i += 64) mk[i] = 0ull;
      for (int i = lane; i < D * M; i += 64) lastp[i] = 0u;
      lsync();
      for (int u = lane; u < N; u += 64) {
        const uint32_t a = t_act[u];
        const uint32_t fb = (uint32_t)pfl[u >> 2] >> ((u & 3) << 1);
        if ((fb & 1u) && (a & 64u)) continue;
        const int d = rdev(g, u);
        if ((unsigned)d >= (unsigned)D) continue;
        const uint32_t lvw = t_alv[u];
        const int lo = (int)(lvw & 0xffffu), hi = lo + (int)(lvw >> 16);
        const int pu = rprio(g, u);
        int slot = lo;
        for (int j = lo; j < hi; ++j) {
          if (fuse_of(pfl, j) && (t_act[j] & 64u)) continue;
          if ((unsigned)rdev(g, j) >= (unsigned)D) continue;
          const int pj = rprio(g, j);
          slot += (pj < pu) || (pj == pu && j < u);
        }
        const int c = t_cnext[u];
        const bool chain = c != 0xffff && fuse_of(pfl, c);
        rec[slot] = (uint16_t)((uint32_t)u | ((a & 63u) << 9) | ((fb & 2u) << 12) |
                               (chain ? kEChain : 0u));
        atomicOr(&mk[d * NWA + (slot >> 6)], 1ull << (slot & 63));
        atomicMax(&lastp[d * M + (int)(a & 63u)], (uint32_t)slot + 1u);
      }
      lsync();
    }
    if (pre && grp + stride < n_groups) load_rows(grp + stride, dvp, pvp);

    // ---- device-lane state ----
    const bool act = g_me < gc;
    const int gme = act ? g_me : 0;
    const int d = d_me;
    const uint32_t* mylast = s_last + (gme * D + d) * M;
    const unsigned long long* mymask64 = s_mask + (gme * D + d) * NWA;
    uint16_t* myrec = s_rec + gme * N;
    uint32_t* myfin = s_fin + gme * N;
    const uint8_t* myfl = s_fl + gme * NB;
    // the last unit of each model on the device gets its flag; the models
    // the device uses at all (read before the finish region is cleared)
    // (every read issued before any write: M <= 16)
    uint32_t umask = 0u;
    if (!PAPER && act) {
      uint32_t lv[16], ev[16];
#pragma unroll
      for (int m = 0; m < 16; ++m) lv[m] = m < M ? mylast[m] : 0u;
#pragma unroll
      for (int m = 0; m < 16; ++m) ev[m] = lv[m] ? (uint32_t)myrec[lv[m] - 1u] : 0u;
#pragma unroll
      for (int m = 0; m < 16; ++m)
        if (lv[m]) {
          myrec[lv[m] - 1u] = (uint16_t)(ev[m] | kELast);
          umask |= 1u << m;
        }
    }
    // reclamation queue of the resident models, 4 bits each, next victim in
    // the low bits: first the nd4 / 4 models with no remaining use on this
    // device, then those still needed, each part least recently used first
    // (never used: by id); nq4 / 4 entries in all
    QT Q = 0;
    uint32_t nq4 = 0, nd4 = 0;
    int32_t fm = 0;   // free memory: capacity - resident weights
    int32_t pe = 0;   // largest excess of a unit's need over the free memory
    uint32_t freet = 0, nld = 0, nev4 = 0, inel = 0;
    // ranking-key terms (Eq. 12) of this device lane: models reclaimed from
    // the device so far, admitted ready units per class (16 bits each), their
    // latest finish, lifecycle overhead, timely prefetches
    uint32_t ph_rec = 0u, ph_cf = 0u, ph_pn = 0u;
    // replica caps: the resident models, and those held as the level starts
    // or loaded during it (the queue holds the order, this mask the set)
    uint32_t rmask = 0u, lv_hold = 0u;
    unsigned long long ph_adm = 0ull, ph_h = 0ull;
    // batch limits: per slot the time it frees (the running unit's finish),
    // the unit's memory, and its model's bit (a lease while it runs); the
    // last dispatch time (units dispatch in order).  Slots beyond the
    // device's limit never free and hold bit 16, outside every model.
    uint32_t bs_fin[kMaxBatch], bs_lb[kMaxBatch], bdisp = 0u;
    int32_t bs_mem[kMaxBatch];
    int nbatch = 1;
#pragma unroll
    for (int k = 0; k < kMaxBatch; ++k) {
      bs_fin[k] = 0u;
      bs_lb[k] = 0u;
      bs_mem[k] = 0;
    }
    if (act) {
      const uint64_t res = t_res0[d];
      rmask = (uint32_t)res;
      const int32_t capd = t_cap[d];
      freet = t_free0[d];
      if constexpr (BATCH) {
        nbatch = t_batch[d];
        bdisp = freet;
#pragma unroll
        for (int k = 0; k < kMaxBatch; ++k) {
          bs_fin[k] = k < nbatch ? freet : 0xffffffffu;
          bs_lb[k] = k < nbatch ? 0u : 1u << 16;
        }
      }
      int32_t used = 0;
      QT qa = 0;
      uint32_t na = 0;
      for (uint64_t r = res; r; r &= r - 1) {
        const int m = __builtin_ctzll(r);
        used += t_wmib[m];
        if constexpr (!PAPER) {
          if (!((umask >> m) & 1u)) {
            Q |= (QT)m << nd4;
            nd4 += 4;
          } else {
            qa |= (QT)m << na;
            na += 4;
          }
        }
      }
      if (na) Q |= qa << nd4;  // nd4 + na <= QB here
      nq4 = nd4 + na;
      fm = capd - used;
      pe = used - capd;
    }
    // the paper's order: per model the device index of its next use (low 16
    // bits, 0xffff: none) and its last-use stamp (high 16 bits, 0: not used
    // yet), in the last-slot region; one backward pass over the device's
    // units gives every slot the next use of its model after it
    uint32_t* mypk = s_last + (gme * D + d) * M;
    uint32_t kdev = 0u, seq = 1u, others = 0u;
    if (PAPER && act) {
      for (int m = 0; m < M; ++m) mypk[m] = 0xffffu;
      int cnt = 0;
      for (int j = 0; j < NWA; ++j) cnt += __popcll(mymask64[j]);
      for (int j = NWA - 1; j >= 0; --j)
        for (unsigned long long bits = mymask64[j]; bits;) {
          const int b = 63 - __clzll(bits);
          bits &= ~(1ull << b);
          const int sl = (j << 6) + b;
          const uint32_t m = ((uint32_t)myrec[sl] >> 9) & 15u;
          --cnt;
          if (nx8)
            s_nx8[gme * N + sl] = mypk[m] == 0xffffu ? (uint8_t)0 : (uint8_t)mypk[m];
          else
            s_nx[gme * N + sl] = (uint16_t)mypk[m];
          mypk[m] = (uint32_t)cnt;
        }
      s_snap[gme * D + d] = (uint16_t)rmask;
    }

    // every finish starts at 0: it accumulates the latest predecessor finish
    // before its level, then holds the activation's own finish
    zero16(reinterpret_cast<unsigned char*>(s_fin), G * N * 4, lane);
    zero16(reinterpret_cast<unsigned char*>(s_wfm), G * W * 4, lane);
    lsync();

    for (int lv = 0; lv < sp.n_levels; ++lv) {
      const int lo = t_loff[lv], hi = t_loff[lv + 1];
      const int eb = t_eoff[lv], ee = t_eoff[lv + 1];
      // ---- latest predecessor finish of the level's activations (Eq. 2):
      // one lane per incoming edge; a fused chain member already holds its
      // own, later, finish ----
      if (ee > eb) {
        for (int e = eb + lane; e < ee; e += 64) {
          const uint32_t ed = t_edge[e];
          const int src = (int)(ed & 0xffffu), dst = (int)(ed >> 16);
          for (int g0 = 0; g0 < gc; g0 += kB) {
            uint32_t f[kB];
#pragma unroll
            for (int k = 0; k < kB; ++k) {
              const int g = (g0 + k < gc) ? g0 + k : gc - 1;
              f[k] = s_fin[g * N + src];
            }
#pragma unroll
            for (int k = 0; k < kB; ++k)
              if (g0 + k < gc) atomicMax(&s_fin[(g0 + k) * N + dst], f[k]);
          }
        }
        lsync();
      }

      // ---- device lanes walk their units of the level in slot order ----
      lv_hold = rmask;
      if (PAPER && act) {
        // models resident on the plan's other devices as the level starts
        others = 0u;
        for (int e = 0; e < D; ++e) others |= e != d ? (uint32_t)s_snap[gme * D + e] : 0u;
      }
      if (act) {
        const int j1 = (hi - 1) >> 6;
        const unsigned long long hmask = (hi & 63) ? ((1ull << (hi & 63)) - 1ull) : ~0ull;
        const int width = hi - lo;
        const bool narrow = width <= 64;
        int j = lo >> 6;
        unsigned long long bits, wnext = 0ull;
        if (narrow) {
          const int sh = lo & 63;
          bits = mymask64[j] >> sh;
          if (sh + width > 64) bits |= mymask64[j + 1] << (64 - sh);
          if (width < 64) bits &= (1ull << width) - 1ull;
        } else {
          bits = mymask64[j] & (~0ull << (lo & 63));
          if (j < j1) wnext = mymask64[j + 1] & ((j + 1 == j1) ? hmask : ~0ull);
        }
        // the device's next slot of the level; -1 when there is none, -2
        // for a trip without a unit (a finished word followed by an empty one)
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
          const unsigned long long wl2 = mymask64[jn] & ((jn == j1) ? hmask : ~0ull);
          wnext = adv ? (j < j1 ? wl2 : 0ull) : wnext;
          const int sl = (j << 6) + __builtin_ctzll(bits | (1ull << 63));
          const bool have = bits != 0ull;
          bits &= bits - 1ull;
          return have ? sl : (j < j1 ? -2 : -1);
        };
        // everything of a unit that does not depend on the device's
        // sequential state; without a slot, activation 0 and model 0 keep
        // every address in range
        struct U { int slot; uint32_t e, lst, arr, r, act; int32_t lat, mem; int4 lw; };
        auto fetch = [&](int sl, U& X) {
          X.slot = sl;
          const uint32_t e = sl >= 0 ? (uint32_t)myrec[sl] : 0u;
          X.e = e;
          const uint32_t u = e & kEAct, m = (e >> 9) & 15u;
          X.lst = !PAPER && (e & kELast) ? 1u : 0u;
          const int2 r = um_d[u];
          X.lat = r.x;
          X.mem = r.y;
          X.arr = t_aarr[u];
          X.r = umax(myfin[u], X.arr);
          X.lw = lw_d[m];
          if constexpr (PHI) X.act = t_act[u];
        };
        auto process = [&](const U& X) {
          if (X.slot < 0) return;
          const uint32_t u = X.e & kEAct;
          const uint32_t m = (X.e >> 9) & 15u;
          // run time (summed over a fused chain, Eq. 4) and memory (max)
          uint32_t T = (uint32_t)X.lat;
          int32_t mx = X.mem;
          inel |= (uint32_t)X.lat >> 31;
          if (X.e & kEChain) {
            for (int v = t_cnext[u];;) {
              const int2 lm = um_d[v];
              inel |= (uint32_t)lm.x >> 31;
              T += (uint32_t)lm.x;
              mx = lm.y > mx ? lm.y : mx;
              const int c = t_cnext[v];
              if (c == 0xffff || !fuse_of(myfl, c)) break;
              v = c;
            }
          }
          // residency: m is resident when its nibble is among the first
          // nq4 / 4 entries; a hit takes it out of the queue (it re-enters
          // below as the most recent)
          // (the paper's order: the resident mask)
          bool hit;
          if constexpr (PAPER) {
            hit = ((rmask >> m) & 1u) != 0u;
          } else {
            QT mq = (QT)(uint32_t)X.lw.z;
            if constexpr (QB == 64) mq |= mq << 32;
            const QT x = Q ^ mq;
            QT z = (x - kOnes) & ~x & kHigh;  // lowest flag: first zero nibble
            const QT valid = nq4 >= (uint32_t)QB ? ~(QT)0 : (((QT)1 << nq4) - (QT)1);
            z &= valid;
            hit = z != (QT)0;
            uint32_t s4;
            if constexpr (QB == 64)
              s4 = (uint32_t)__builtin_ctzll(z | (1ull << 63)) & ~3u;
            else
              s4 = (uint32_t)__builtin_ctz(z | (1u << 31)) & ~3u;
            const QT lowm = ((QT)1 << s4) - (QT)1;
            const QT rem = (Q & lowm) | ((Q >> 4) & ~lowm);
            Q = hit ? rem : Q;
            nq4 -= hit ? 4u : 0u;
          }
          const int32_t need = mx + (hit ? 0 : X.lw.y);
          int32_t ex;       // > 0: the unit does not fit yet
          int32_t run = 0;  // memory of the units still running (batch limits)
          int ks = 0;       // batch limits: the unit's slot, and its dispatch time
          uint32_t t0 = 0u;
          if constexpr (PAPER) {
            ex = need - fm;
            // reclaim (Sec. 3.5) in the paper's order: copies resident on
            // another device of the plan first, then the longest distance to
            // the next use per reload time, then least recently used (equal
            // keys: the lower model id)
            auto ldw = [&](int x) { return *reinterpret_cast<const int2*>(lw_d + x); };
            for (uint32_t cand = rmask & ~(1u << m); ex > 0 && cand != 0u;) {
              // a copy held on another device goes before any other: when
              // there are such copies the choice is among them; the first
              // three candidates' keys are read at once
              const uint32_t cr = cand & others;
              uint32_t sel = cr ? cr : cand;
              const int ca = __builtin_ctz(sel);
              sel &= sel - 1u;
              const int cb = sel ? __builtin_ctz(sel) : ca;
              sel &= sel - 1u;
              const int cc = sel ? __builtin_ctz(sel) : ca;
              sel &= sel - 1u;
              const uint32_t pa = mypk[ca], pb = mypk[cb], pc = mypk[cc];
              const int2 la = ldw(ca), lb = ldw(cb), lc = ldw(cc);
              int v = ca;
              uint32_t vpk = pa;
              int2 vl = la;
              // (ascending ids: equal keys keep the lower id)
              auto consider = [&](int x, uint32_t pk, int2 l) {
                if (paper_victim_before(0u, pk & 0xffffu, (uint32_t)l.x, pk >> 16, 0u, vpk & 0xffffu,
                                        (uint32_t)vl.x, vpk >> 16, kdev)) {
                  v = x;
                  vpk = pk;
                  vl = l;
                }
              };
              if (cb != ca) consider(cb, pb, lb);
              if (cc != ca) consider(cc, pc, lc);
              for (; sel; sel &= sel - 1u) {
                const int m2 = __builtin_ctz(sel);
                consider(m2, mypk[m2], ldw(m2));
              }
              cand &= ~(1u << v);
              rmask &= ~(1u << v);
              ex -= vl.y;
              nev4 += 4u;
            }
          } else if constexpr (BATCH) {
            // the slot that frees first; units dispatch in order, at the
            // release (the arrival for a prefetched load) at the earliest
            uint32_t sft = bs_fin[0];
#pragma unroll
            for (int k = 1; k < kMaxBatch; ++k)
              if (bs_fin[k] < sft) {
                ks = k;
                sft = bs_fin[k];
              }
            t0 = umax(umax((!hit && (X.e & kEPf)) ? X.arr : X.r, sft), bdisp);
            // the units running at t0: their memory, leases on their
            // models, and the first of their finishes
            uint32_t leased, nf;
            auto running_at = [&]() {
              leased = 0u;
              nf = 0xffffffffu;
              run = 0;
#pragma unroll
              for (int k = 0; k < kMaxBatch; ++k) {
                const bool r = bs_fin[k] > t0;
                run += r ? bs_mem[k] : 0;
                leased |= r ? bs_lb[k] : 0u;
                nf = r ? umin(nf, bs_fin[k]) : nf;
              }
            };
            // reclaim (Sec. 3.5) in the queue's order, passing over the
            // copies whose model holds a lease; when the unit still does not
            // fit, wait for the next running unit to finish (its lease and
            // memory end) and look again
            int32_t ex0 = need - fm;  // excess without the running units
            for (;;) {
              running_at();
              for (uint32_t p = 0u; ex0 + run > 0 && p < nq4;) {
                const uint32_t v = (uint32_t)(Q >> p) & 15u;
                const int32_t wv = t_wmib[v];
                if ((leased >> v) & 1u) {
                  p += 4u;
                  continue;
                }
                const QT lowm = ((QT)1 << p) - (QT)1;
                Q = (Q & lowm) | ((Q >> 4) & ~lowm);
                nq4 -= 4u;
                nd4 -= p < nd4 ? 4u : 0u;
                ex0 -= wv;
                nev4 += 4u;
              }
              // fits, or no running unit left to wait for
              if (ex0 + run <= 0 || (leased & 0xffffu) == 0u) break;
              t0 = nf;
            }
            ex = ex0 + run;
          } else {
            ex = need - fm;
            // reclaim (Sec. 3.5) from the queue's front: no remaining use
            // first, then least recently used, then the lower model id; the
            // first two victims branch-free, any further ones in a loop
            {
              const uint32_t q0 = (uint32_t)(Q & (QT)15), q1 = (uint32_t)((Q >> 4) & (QT)15);
              const int32_t w0 = t_wmib[q0];
              const int32_t w1 = t_wmib[q1];
              const bool c0 = ex > 0 && nq4 >= 4u;
              const int32_t ex0 = ex - w0;
              const bool c1 = c0 && ex0 > 0 && nq4 >= 8u;
              const uint32_t k4 = (c0 ? 4u : 0u) + (c1 ? 4u : 0u);
              ex = c1 ? ex0 - w1 : (c0 ? ex0 : ex);
              if constexpr (PHI) ph_rec |= (c0 ? 1u << q0 : 0u) | (c1 ? 1u << q1 : 0u);
              if constexpr (RCAP) rmask &= ~((c0 ? 1u << q0 : 0u) | (c1 ? 1u << q1 : 0u));
              Q >>= k4;
              nq4 -= k4;
              nd4 = nd4 > k4 ? nd4 - k4 : 0u;
              nev4 += k4;
              while (ex > 0 && nq4 >= 4u && c1) {
                const int v = (int)(Q & (QT)15);
                Q >>= 4;
                nq4 -= 4u;
                nd4 = nd4 > 4u ? nd4 - 4u : 0u;
                ex -= t_wmib[v];
                nev4 += 4u;
                if constexpr (PHI) ph_rec |= 1u << v;
                if constexpr (RCAP) rmask &= ~(1u << v);
              }
            }
          }
          // peak memory = capacity + the largest excess after reclamation;
          // free memory after the load: mx + run - ex
          pe = ex > pe ? ex : pe;
          fm = mx + run - ex;
          // m re-enters after the no-remaining-use part when this was its
          // last unit on the device, else at the end (the paper's order: its
          // next use and last-use stamp)
          if constexpr (PAPER) {
            uint32_t nu;
            if (nx8) {
              nu = s_nx8[gme * N + X.slot];
              nu = nu ? nu : 0xffffu;
            } else {
              nu = s_nx[gme * N + X.slot];
            }
            mypk[m] = nu | (seq << 16);
            ++seq;
            ++kdev;
          } else {
            const uint32_t pos = X.lst ? nd4 : nq4;
            const QT lowm = ((QT)1 << pos) - (QT)1;
            Q = (Q & lowm) | ((QT)m << pos) | ((Q & ~lowm) << 4);
            nd4 += X.lst ? 4u : 0u;
            nq4 += 4u;
          }
          nld += hit ? 0u : 1u;
          if constexpr (RCAP || PAPER) rmask |= 1u << m;
          if constexpr (RCAP) lv_hold |= 1u << m;
          // timeline (Eq. 7): a load waits for the device and starts at the
          // release, or at the workflow arrival when prefetched; the unit
          // starts at max(release, load end), or at max(release, device
          // free) when its model was resident
          // (batch limits: the load starts at the dispatch, a resident
          // model's unit runs at once)
          const uint32_t a0 = (X.e & kEPf) ? X.arr : X.r;
          const uint32_t ls = BATCH ? t0 : umax(a0, freet);
          const uint32_t le = tadd<CHECKED>(ls, (uint32_t)X.lw.x);
          const uint32_t s = BATCH ? (hit ? t0 : umax(X.r, le)) : umax(X.r, hit ? freet : le);
          const uint32_t fr0 = freet;
          if (!(X.e & kEChain)) {
            const uint32_t f = tadd<CHECKED>(s, T);
            myfin[u] = f;
            freet = f;
          } else {
            // members back to back on the head's device
            uint32_t t = s;
            for (int v = (int)u;;) {
              const uint32_t tv = tadd<CHECKED>(t, (uint32_t)um_d[v].x);
              myfin[v] = tv;
              t = tv;
              const int c = t_cnext[v];
              if (c == 0xffff || !fuse_of(myfl, c)) break;
              v = c;
            }
            freet = t;
          }
          if constexpr (BATCH) {
#pragma unroll
            for (int k = 0; k < kMaxBatch; ++k) {
              bs_fin[k] = k == ks ? freet : bs_fin[k];
              bs_mem[k] = k == ks ? mx : bs_mem[k];
              bs_lb[k] = k == ks ? 1u << m : bs_lb[k];
            }
            bdisp = t0;
          }
          if constexpr (PHI) {
            // ready work: no predecessor, arrived by the window time
            const bool ready = ((X.act >> 7) & 1u) != 0u;
            if (!hit) {
              // a reload of a copy this plan reclaimed from the device
              if ((ph_rec >> m) & 1u) ph_h += (uint32_t)X.lw.x;
              // a prefetch is timely when its load is done by the release
              if (!ready && (X.e & kEPf) && le <= X.r) ++ph_pn;
              // the delay a load adds to ready work
              if (ready) ph_h += s - umax(X.r, fr0);
            }
            if (ready && ex <= 0) {
              ph_adm += 1ull << (16u * ((X.act >> 8) & 3u));
              ph_cf = umax(ph_cf, freet);
            }
          }
        };
        // two units per trip so that the prefetched unit needs no copy; one
        // copy of the loop per kind of level
        auto run = [&](auto&& next_slot) {
          U A, B;
          fetch(next_slot(), A);
          while (A.slot != -1) {
            fetch(next_slot(), B);
            process(A);
            if (B.slot == -1) break;
            fetch(next_slot(), A);
            process(B);
          }
        };
        if (narrow)
          run(next_narrow);
        else
          run(next_wide);
      }
      if (RCAP && act) s_hold[gme * D + d] = (uint16_t)lv_hold;
      if (PAPER && act) s_snap[gme * D + d] = (uint16_t)rmask;
      lsync();
      // ---- replica caps (Sec. 3.5 scale-out): a model held or loaded in
      // this level on more devices than its cap; lanes over (plan, model) ----
      if constexpr (RCAP) {
        for (int it = lane; it < gc * M; it += 64) {
          const int g = it / M, m = it - g * M;
          int copies = 0;
          for (int e = 0; e < D; ++e) copies += (int)((s_hold[g * D + e] >> m) & 1u);
          if (copies > t_rcap[m]) atomicOr(&s_acc[g].status, (uint32_t)WF_ST_REPLICA);
        }
        lsync();
      }
    }

    // ---- per-plan reductions (Sec. 4 metrics) ----
    if (act) {
      if constexpr (PHI) {
        if (ph_adm) {
          atomicAdd(reinterpret_cast<unsigned long long*>(&s_acc[gme].max_finish), ph_adm);
          atomicMax(&s_acc[gme].cf, ph_cf);
        }
        if (ph_pn) atomicAdd(&s_acc[gme].loads, ph_pn);
        if (ph_h) atomicAdd(&s_acc[gme].h_life, ph_h);
      } else {
        atomicMin(&s_acc[gme].headroom, -pe);
        atomicAdd(&s_acc[gme].loads, nld);
        atomicAdd(&s_acc[gme].evicts, nev4 >> 2);
      }
      uint32_t st = pe > 0 ? (uint32_t)WF_ST_CAPACITY : 0u;
      if (inel) st |= (uint32_t)WF_ST_INELIGIBLE;
      // a saturated time ends in the device's last finish
      uint32_t last = freet;
      if constexpr (BATCH) {
#pragma unroll
        for (int k = 0; k < kMaxBatch; ++k) last = k < nbatch ? umax(last, bs_fin[k]) : last;
      }
      if (CHECKED && last == 0xffffffffu) st |= kRescore;
      if (st) atomicOr(&s_acc[gme].status, st);
    }
    // a workflow's completion is the latest finish among its activations
    // without a successor in the same workflow (not part of the ranking key)
    for (int i = lane; i < (PHI ? 0 : sp.S); i += 64) {
      const uint32_t sk = t_sink[i];
      const int src = (int)(sk & 0xffffu), wf = (int)(sk >> 16);
      for (int g0 = 0; g0 < gc; g0 += kB) {
        uint32_t f[kB];
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
    lsync();
    // completion latencies in place, and the latest finish; nearest-rank
    // p95 is the ceil(0.95 W)-th smallest latency, which for W <= 19 is the
    // largest one
    const int kk = (95 * W + 99) / 100;
    for (int it = lane; it < (PHI ? 0 : gc * W); it += 64) {
      const int g = it / W, a = it - g * W;
      const uint32_t fb = s_wfm[it];
      atomicMax(&s_acc[g].max_finish, fb);
      s_wfm[it] = fb - t_arr[a];
      if (kk == W) atomicMax(&s_acc[g].p95, fb - t_arr[a]);
    }
    lsync();
    // otherwise counting, lanes over (plan, workflow)
    for (int it = lane; it < (PHI || kk == W ? 0 : gc * W); it += 64) {
      const int g = it / W;
      const uint32_t* cw = s_wfm + g * W;
      const uint32_t ca = cw[it - g * W];
      int lt = 0, le = 0;
#pragma unroll 8
      for (int b = 0; b < W; ++b) {
        const uint32_t cb = cw[b];
        lt += cb < ca;
        le += cb <= ca;
      }
      if (lt < kk && kk <= le) s_acc[g].p95 = ca;
    }
    lsync();
    if (PHI && lane < gc) {
      const LeanAcc a = s_acc[lane];
      const unsigned long long adm = *reinterpret_cast<const unsigned long long*>(&a.max_finish);
      wf_plan_key k;
      k.c_ready_us = 0;
      k.h_life_us = 0;
      for (int c = 0; c < WF_MAX_CLASSES; ++c) k.admitted[c] = 0;
      k.timely_prefetch = 0;
      k.pad = 0;
      k.status = (a.status & WF_ST_INELIGIBLE) ? (uint32_t)WF_ST_INELIGIBLE : a.status;
      if (!(a.status & WF_ST_INELIGIBLE)) {
        if (adm) k.c_ready_us = sp.origin + (int64_t)a.cf;
        k.h_life_us = (int64_t)a.h_life;
        for (int c = 0; c < WF_MAX_CLASSES; ++c) k.admitted[c] = (uint16_t)((adm >> (16 * c)) & 0xffffull);
        k.timely_prefetch = (uint16_t)(a.loads > 65535u ? 65535u : a.loads);
      }
      reinterpret_cast<wf_plan_key*>(scores)[p0 + lane] = k;
    } else if (lane < gc) {
      const LeanAcc a = s_acc[lane];
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
        const int64_t mk = N > 0 ? sp.origin + (int64_t)a.max_finish - sp.min_arrival : 0;
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
    lsync();
  }
}

template <bool CHECKED, int QB, bool SEARCH, bool PHI, bool RCAP, bool BATCH>
hipError_t launch_lean_variant(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                               const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                               wf_plan_score* scores, const SearchArgs& sa, hipStream_t stream) {
  auto k = score_lean<CHECKED, QB, SEARCH, PHI, RCAP, BATCH>;
  LeanParams l = lp;
  if (lean_plain<SEARCH, PHI, RCAP, BATCH, QB>()) {
    // the plain variant's own launch, its grid fitted to the plans
    l.waves = lp.xwaves;
    l.lds_bytes = lp.xlds_bytes;
    const int64_t wgs = ((n_plans + lp.G - 1) / lp.G + l.waves - 1) / l.waves;
    l.grid = wgs < lp.xgrid ? (int)wgs : lp.xgrid;
  }
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                            hipFuncAttributeMaxDynamicSharedMemorySize, l.lds_bytes);
  hipLaunchKernelGGL(k, dim3(l.grid), dim3(64 * l.waves), l.lds_bytes, stream, sp, l, dev, prio,
                     flags, n_plans, scores, sa);
  return hipGetLastError();
}

template <bool CHECKED, bool SEARCH, bool PHI, bool RCAP, bool BATCH>
hipError_t launch_lean_q(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                         const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                         wf_plan_score* scores, const SearchArgs& sa, hipStream_t stream) {
  if (lp.qbits == 32)
    return launch_lean_variant<CHECKED, 32, SEARCH, PHI, RCAP, BATCH>(sp, lp, dev, prio, flags,
                                                                       n_plans, scores, sa, stream);
  return launch_lean_variant<CHECKED, 64, SEARCH, PHI, RCAP, BATCH>(sp, lp, dev, prio, flags,
                                                                     n_plans, scores, sa, stream);
}

template <bool CHECKED, bool SEARCH, bool PHI>
hipError_t launch_lean_r(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                         const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                         wf_plan_score* scores, const SearchArgs& sa, hipStream_t stream) {
  if (lp.rcap)
    return launch_lean_q<CHECKED, SEARCH, PHI, true, false>(sp, lp, dev, prio, flags, n_plans,
                                                            scores, sa, stream);
  return launch_lean_q<CHECKED, SEARCH, PHI, false, false>(sp, lp, dev, prio, flags, n_plans,
                                                           scores, sa, stream);
}

template <bool SEARCH, bool PHI>
hipError_t launch_lean_c(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                         const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                         wf_plan_score* scores, const SearchArgs& sa, hipStream_t stream) {
  if (lp.checked)
    return launch_lean_r<true, SEARCH, PHI>(sp, lp, dev, prio, flags, n_plans, scores, sa, stream);
  return launch_lean_r<false, SEARCH, PHI>(sp, lp, dev, prio, flags, n_plans, scores, sa, stream);
}

}  // namespace

hipError_t launch_score_lean(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                             const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                             void* out, const SearchArgs* search, bool keys, hipStream_t stream) {
  const SearchArgs sa = search ? *search : SearchArgs{};
  wf_plan_score* o = static_cast<wf_plan_score*>(out);
  if (lp.paper) {
    // the paper's reclamation order: plan scores only
    if (search || keys || lp.rcap || lp.batch) return hipErrorInvalidValue;
    if (lp.checked)
      return launch_lean_variant<true, -1, false, false, false, false>(sp, lp, dev, prio, flags,
                                                                       n_plans, o, sa, stream);
    return launch_lean_variant<false, -1, false, false, false, false>(sp, lp, dev, prio, flags,
                                                                      n_plans, o, sa, stream);
  }
  if (lp.batch) {
    // windows with batch limits: plan scores only
    if (search || keys || lp.rcap) return hipErrorInvalidValue;
    if (lp.checked)
      return launch_lean_q<true, false, false, false, true>(sp, lp, dev, prio, flags, n_plans, o,
                                                            sa, stream);
    return launch_lean_q<false, false, false, false, true>(sp, lp, dev, prio, flags, n_plans, o, sa,
                                                           stream);
  }
  if (search)
    return keys ? launch_lean_c<true, true>(sp, lp, dev, prio, flags, n_plans, o, sa, stream)
                : launch_lean_c<true, false>(sp, lp, dev, prio, flags, n_plans, o, sa, stream);
  return keys ? launch_lean_c<false, true>(sp, lp, dev, prio, flags, n_plans, o, sa, stream)
              : launch_lean_c<false, false>(sp, lp, dev, prio, flags, n_plans, o, sa, stream);
}

}  // namespace wfp
