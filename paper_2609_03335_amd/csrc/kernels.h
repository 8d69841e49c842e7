// Internal interface between the host library (host.hip) and the gfx950
// kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wf_plan.h"

namespace wfp {

constexpr int kMaxBatch = WF_MAX_BATCH;  // slots per device in the batch-limit modes

// The paper's reclamation preference (Sec. 3.5): whether copy x is reclaimed
// before copy y.  red: resident on another device as the level started;
// nu: device index of the next use (0xffff: none); ld: reload time; lru:
// last-use stamp (0: never used); k: the current unit's device index.
// Ratios (nu - k) / ld compare by cross-multiplication; no next use or a
// free reload is an infinite ratio.
__device__ __forceinline__ bool paper_victim_before(uint32_t redx, uint32_t nux, uint32_t ldx,
                                                    uint32_t lrux, uint32_t redy, uint32_t nuy,
                                                    uint32_t ldy, uint32_t lruy, uint32_t k) {
  // evaluated without branches: each level of the preference decides only
  // where all earlier levels tie
  const bool infx = nux == 0xffffu || ldx == 0u;
  const bool infy = nuy == 0xffffu || ldy == 0u;
  const unsigned long long a = (unsigned long long)(nux - k) * ldy;
  const unsigned long long b = (unsigned long long)(nuy - k) * ldx;
  const bool ratio_tie = infx || a == b;  // both infinite, or equal finite ratios
  const bool by_ratio = infx != infy ? infx : (!ratio_tie && a > b);
  const bool later = infx != infy || !ratio_tie ? by_ratio : lrux < lruy;
  return redx != redy ? redx > redy : later;
}

// Byte offsets of the window tables inside the table image.  The host builds
// the image once per window; the scoring kernel copies it into LDS (or reads
// it from HBM when it is too large) and uses the same offsets either way.
struct TabOffsets {
  int act;     // u32 [N]    model | fusible << 6 | ready << 7 | class << 8 | workflow << 16
               //            (ready: no predecessor and arrived by time 0; class: the
               //            workflow's priority class of the ranking key)
  int alv;     // u32 [N]    first index of the activation's level | level width << 16
  int cnext;   // u16 [N]    successor v of u when Eq. 3 holds for (u, v), else 0xffff
  int edge;    // u32 [E]    predecessor | activation << 16, grouped by activation (CSR order)
  int eoff;    // i32 [L+1]  first edge of each level
  int loff;    // i32 [L+1]  first activation of each level
  int ud;      // 16 B [N*D] per (activation, device): {run time (-1 ineligible), activation
               //            memory, arrival of the activation's workflow (relative time,
               //            low word / high word for fp64); with uint32 times the last word
               //            repeats the activation's act entry}
  int lw;      // i32x2 [M*D] {load time, model weights}
  int wmib;    // i32 [M]    model weights
  int cap;     // i32 [D]    device capacity
  int arr;     // time [W]   workflow arrival relative to the window origin
  int res0;    // u64 [D]    initial resident-model mask
  int free0;   // time [D]   initial busy-until relative to the window origin
  int sink;    // u32 [S]    activations without successor in their workflow: index | workflow << 16
  int elig;    // u64 [N][2] devices d with lat[i][d] >= 0 (bit d % 64 of word d / 64)
  int batch;   // i32 [D]    batch limit (units a device runs at once)
  int rcap;    // i32 [M]    replica cap of each model (windows with caps)
  // ring of recent levels (ScoreParams::ring): finishes are kept only for
  // the levels a unit can still reach, at ring positions
  int rpos;    // u16 [N]    ring position: activation index mod ring size
  int redge;   // u32 [E]    as edge, with ring positions instead of activation ids
  int rsnk;    // u16 [N]    workflow of an activation without successor in its
               //            workflow, else 0xffff
  int bytes;
};

// Byte offsets inside one wave's LDS region (G plans scored together).
struct WaveOffsets {
  int flags;   // u8 [G][NB]       staged fuse/prefetch rows
  int rec;     // u32 [G][N]       slot entry per resource-order slot (packed)
  int mask;    // u64 [G][D][NWA]  slots of each device's units
  int last;    // u32 [G][D][M]    1 + slot of the last unit of each (device, model), 0 = none
               //                  (until the walk: inside the finish region, after the
               //                  candidates' changed sites, where it fits); the paper's
               //                  order: next use and last-use stamp of each model;
               //                  with the in-register reclamation queues it shares storage
               //                  with fin (dead before the first finish is written)
  int fin;     // time [G][N]      latest predecessor finish, then the activation's own finish
  int acc;     // PlanAcc [G]
  int stamp;   // u16 [G*D][M]     last use of each model (general reclamation only)
               // (ring layout: rec holds [G][widest level] entries of the current
               // level, mask [G][D][NWA] its words, last the u16 count of each
               // (device, model)'s units not yet walked, fin [G][ring size])
  int rows;    // generated candidates only: int8 [G][N] devices, then u16 [G][N]
               //                  priorities at rows + rows_prio; they live in fin's
               //                  storage (after last[] when that shares it) until
               //                  the order is built
  int rows_prio;
  int wfm;     // time [G][W]      latest finish per workflow
  int nx;      // u16 [G][N]       paper reclamation order: per slot, the device index of
               //                  the next unit of the device with the same model
  int nxu;     // u16 [G*D][M]     paper order: next use of each model (device index)
  int snap;    // u64 [G][D]       paper order: resident models as the level starts
  int hstate;  // HState [2][64]   more than 64 devices: the state of each lane's idle device
  int hold;    // u64 [G][D]       replica caps: models each device held or loaded in the level
  int bytes;
  // per-wave regions in HBM: the arrays at offsets below `split` (acc, and
  // outside the queue modes last, stamp, nxu, snap: O(G D M) bytes) stay in
  // LDS, `split` bytes per wave; the others live in HBM, `bytes - split` per
  // wave, at their offset minus split.  0 when the whole region is in LDS.
  int split;
};

// With more than 64 devices each lane owns two; the state of the one not in
// registers waits in LDS (times as their bit patterns).
struct HState {
  unsigned long long res, freet, q, ph_adm, ph_rec, ph_cf, ph_h, bdisp;
  unsigned long long bs_free[kMaxBatch], bs_fin[kMaxBatch];
  int32_t bs_mem[kMaxBatch], bs_model[kMaxBatch];
  int32_t used, peak, capd;
  uint32_t nld, nev, capbad, inel, seq;
  int32_t nd, nq;
  uint32_t ph_pn;
  int32_t kdev, nbatch, pad;
};

struct ScoreParams {
  int32_t N, W, M, D, NB, S, n_levels, nwa;
  int64_t origin;             // absolute time of relative time 0
  int64_t min_arrival;        // first workflow arrival (absolute)
  float w_mk, w_p95;
  const unsigned char* tab;   // table image in HBM
  TabOffsets t;
  WaveOffsets wo;
  int G;                      // plans per wave (G * D <= 64; 1 when D > 64, each lane
                              // then owning devices lane and lane + 64)
  int waves;                  // waves per workgroup
  int tab_in_lds;             // 1: the table image is staged in LDS
  int wave_global;            // 1: per-wave regions live in HBM scratch (windows too big for LDS)
  unsigned char* scratch;     // per-wave regions when wave_global
  int lds_bytes;              // dynamic LDS per workgroup
  int wg_ld;                  // bytes of the workgroup's copies of every (model, device)
                              // load time (paper reclamation order only) and of every
                              // model's weights, after the table image when that is in
                              // LDS and before the waves' regions
  int grid;                   // workgroups (persistent)
  int time64;                 // 1: fp64 times, 0: uint32 times
  int nibble;                 // reclamation queue width in bits (32 or 64), 0: scan,
                              // -1: scan in the paper's reclamation order; -2 / -3: the
                              // same two scans with per-device batch limits
  int queue;                  // width a queue would take (32 or 64; 0: over 16 models)
  int has_chains;             // 1: some activation satisfies Eq. 3 (fused units possible)
  int rcap;                   // 1: the window caps replicas (checked per level)
  int rescore;                // 1: fp64 pass over the groups holding a plan whose uint32
                              // times saturated (status bit kRescore of the first pass)
  // ring of recent levels (deep or wide windows, scan reclamation, plan rows
  // from HBM): the slot entries and device masks of the current level only,
  // and the finishes of the levels from ring_b behind the current one (the
  // longest edge, in levels) to ring_a ahead (a fused chain's members get
  // their finish with the chain head), at positions index mod ring_size:
  // ring_size is the most activations any such span of levels holds, so
  // the live finishes never share a position
  int ring;                   // 1: the ring layout; 2: the HBM layout with the finishes in
                              // the ring (the paper's order)
  int ring_ok;                // 1: the window admits it (tables rpos, redge, rsnk built)
  int ring_size, ring_w, ring_a, ring_b;  // ring_w: the widest level
};

// Byte offsets inside one wave's LDS region of the lean kernel (lean.hip):
// G plans, lane (g, d) = (lane / D, lane % D).
struct LeanOffsets {
  int flags;   // u8 [G][NB]       staged fuse/prefetch rows
  int rec;     // u16 [G][N]       per resource-order slot: activation | model << 9 |
               //                  prefetch << 13 | fused successor << 14
  int mask;    // u64 [G][D][NWA]  slots of each device's units
  int last;    // u32 [G][D][M]    1 + slot of the last unit of each (device, model), 0 = none
               //                  (until the walk: inside the finish region, after the
               //                  candidates' changed sites, where it fits); the paper's
               //                  order: next use and last-use stamp of each model
  int fin;     // u32 [G][N]       latest predecessor finish, then the activation's own finish
  int wfm;     // u32 [G][W]       latest finish per workflow, then its completion latency
  int acc;     // LeanAcc [G]
  int hold;    // u16 [G][D]       replica caps: models each device held or loaded in the
               //                  level; the paper's order: resident models as the level starts
  int nx;      // u8 or u16 [G][N] the paper's order: per slot, the device index of the next
               //                  unit of the same model on the device (u8 for N <= 256, with
               //                  0 for none; u16 with 0xffff for none)
  int bytes;
};

// The lean kernel's window tables: one image in HBM whose first part (the
// tables the walk reads per unit, lds_bytes) every workgroup copies into
// LDS; the rest is read through the cache.
struct LeanTab {
  // LDS part
  int lw;      // i32x4 [D][M] {load time, model weights, model id in every nibble, 0}
  int wmib;    // i32 [M]
  int aarr;    // u32 [N]    arrival of the activation's workflow (relative time)
  int rcap;    // i32 [M]    replica cap of each model (windows with caps)
  int lds_bytes;
  // through the cache
  int um;      // i32x2 [D][N] {run time (-1 ineligible), activation memory} of each
               //            activation on each device
  int act;     // u32 [N]    as TabOffsets::act
  int alv;     // u32 [N]    as TabOffsets::alv
  int cnext;   // u16 [N]    as TabOffsets::cnext
  int edge;    // u32 [E]    as TabOffsets::edge
  int eoff;    // i32 [L+1]
  int loff;    // i32 [L+1]
  int cap;     // i32 [D]
  int arr;     // u32 [W]    workflow arrival (relative time)
  int res0;    // u64 [D]
  int free0;   // u32 [D]
  int sink;    // u32 [S]    as TabOffsets::sink
  int batch;   // i32 [D]    batch limit of each device
  int bytes;
};

// Launch plan of the lean kernel (scores or ranking keys of plans read from
// HBM or generated around an incumbent; uint32 times, at most 16 models, at
// most 512 activations; the default reclamation order in a 4-bit queue, or,
// for plan scores only, the paper's order over a resident mask; devices with
// batch limits for plan scores only).
struct LeanParams {
  int ok;          // 1: the window qualifies and a layout fits in LDS
  int checked;     // 1: uint32 additions saturate and flag the plan for the fp64 pass
  int qbits;       // reclamation queue width: 32 or 64; -1: no queue (the paper's order)
  int G, waves, grid, lds_bytes;
  const unsigned char* tab;  // the lean table image in HBM
  LeanTab t;
  LeanOffsets wo;  // wave regions follow the image's LDS part
  int search_ok;   // 1: it also generates candidates (their changed sites fit the
                   // finish array's storage)
  int rcap;        // 1: the window caps replicas (checked per level)
  int batch;       // 1: devices with batch limits (plan scores only)
  int paper;       // 1: the paper's reclamation order (plan scores only; qbits -1)
  // the variants with the reclamation queue are built for three waves per
  // SIMD: up to kLeanPlainWaves waves per workgroup, their own launch
  int xwaves, xgrid, xlds_bytes;
};

// Waves per workgroup of the lean kernel: the queue variants, and the
// paper's order.
constexpr int kLeanPlainWaves = 10;
constexpr int kLeanWaves = 8;

// Generated candidates kept as the incumbent plus their changed sites (the
// lean kernel, and the general kernel's ring layout): at most this many
// mutations each (at most 2 changed sites per mutation).
constexpr int kPatchMaxMut = 8;
// words of one candidate's changed sites (a count, then 4 words per mutation)
constexpr int kPatchWords = 1 + 4 * kPatchMaxMut;

struct SearchArgs;

// Scores (wf_plan_score [n]) or, with keys, ranking keys (wf_plan_key [n])
// of plans read from HBM, or (search) of candidates generated around the
// incumbent rows dev/prio/flags.
hipError_t launch_score_lean(const ScoreParams& sp, const LeanParams& lp, const int8_t* dev,
                             const uint16_t* prio, const uint8_t* flags, int64_t n_plans,
                             void* out, const SearchArgs* search, bool keys, hipStream_t stream);

// Internal status bit of a uint32-time pass: some time of the plan reached
// 2^32 - 1 (saturated), so an fp64 pass rescores it.  Never left in a record
// a call returns.
constexpr uint32_t kRescore = 1u << 31;

// Per-plan accumulators kept in LDS by the scoring kernel.
struct PlanAcc {
  uint32_t status;
  int32_t headroom;
  uint32_t loads;
  uint32_t evicts;
  unsigned long long max_finish;  // time bits
  long long p95;                  // selected completion latency (time units)
  uint32_t heads;                 // unit heads given a slot by the fast ordering path
  uint32_t claimed;               // distinct slots they occupy
  uint32_t bad;                   // a head priority outside its level's index range
  uint32_t pad;
  // ranking-key terms (Eq. 12)
  unsigned long long ph_adm;      // admitted ready units per class, 16 bits each
  unsigned long long ph_cf;       // latest admitted ready finish (time bits)
  unsigned long long ph_h;        // lifecycle overhead (time units)
  uint32_t ph_pn;                 // timely prefetches
  uint32_t ph_pad;
};

// Candidates generated around an incumbent plan instead of read from HBM.
struct SearchArgs {
  uint64_t seed;
  int32_t n_mut;
  int32_t mode;   // WF_SEARCH_UNIFORM or WF_SEARCH_RULES
  int64_t first;  // index of the first candidate
  int32_t D;
  // rule tables of the window (WF_SEARCH_RULES): each activation's best
  // binding (-1: none eligible) and the devices on which PlanPrefetch sets
  // its prefetch bit ([N][2] 64-bit masks)
  const int8_t* rule_best;
  const unsigned long long* rule_pf;
  // each activation's eligible devices ([N][2] 64-bit masks; the general
  // kernel reads its own table image's copy)
  const unsigned long long* elig;
};

// Scores plans read from dev/prio/flags ([P][N] rows), or -- with search --
// candidates first .. first+P-1 generated around the incumbent rows dev/prio/
// flags ([N] each).
hipError_t launch_score(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                        const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                        const wf_plan_sched* sched, const SearchArgs* search,
                        hipStream_t stream);

// Ranking keys (Eq. 12) of plans or generated candidates.
hipError_t launch_score_keys(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                             const uint8_t* flags, int64_t n_plans, wf_plan_key* keys,
                             const SearchArgs* search, hipStream_t stream);

// Rows of candidates first .. first+P-1 around the incumbent rows.
hipError_t launch_search_rows(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                              const uint8_t* flags, const SearchArgs& search, int64_t n,
                              int8_t* out_dev, uint16_t* out_prio, uint8_t* out_flags,
                              hipStream_t stream);

// Argmins: at most kArgminKeyBlocks partial results in `work`
// (ARGMIN_KEY_WORK_BYTES per block, owned by the context), then one block for
// the final result.
constexpr int kArgminKeyBlocks = 512;
constexpr size_t ARGMIN_KEY_WORK_BYTES = 64;

hipError_t launch_argmin(const wf_plan_score* scores, int64_t n_plans, int64_t* out_index,
                         void* work, hipStream_t stream);

// Device address of the current device's static array of kArgminKeyBlocks
// partial minima (argmin.hip), looked up on the first call for `device` (the
// current device) and kept; the argmin that allocates nothing uses it as its
// work area.
hipError_t static_scratch(int device, void** out);
hipError_t launch_argmin_keys(const wf_plan_key* keys, int64_t n_plans, int64_t* out_index,
                              void* work, hipStream_t stream);

// Prefix commit of one plan (prefix.hip): next_arrival is the earliest
// workflow arrival later than 0 (INT64_MAX when none).
hipError_t launch_prefix(const ScoreParams& sp, int64_t next_arrival, const int8_t* dev,
                         const int64_t* start, const int64_t* finish, const int64_t* load_start,
                         const uint64_t* reclaimed, uint8_t* commit, uint64_t* commit_rec,
                         int64_t* t_next, hipStream_t stream);

}  // namespace wfp
