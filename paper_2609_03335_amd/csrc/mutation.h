// Candidate plans generated around an incumbent (shared by the scoring
// kernels): Philox4x32-10 draws and the mutations they select, applied
// through an accessor of the candidate's rows, so that a kernel can keep the
// rows whole (in LDS) or as the incumbent plus the sites the mutations
// changed.
#pragma once

#include "kernels.h"

namespace wfp {

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds of the
// Philox-4x32 bijection of the counter x, the key bumped by the Weyl
// constants after every round.
__device__ __forceinline__ void philox4x32_10(uint32_t x[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t a = x[0], c = x[2];
    x[0] = __umulhi(0xCD9E8D57u, c) ^ x[1] ^ k0;
    x[1] = 0xCD9E8D57u * c;
    x[2] = __umulhi(0xD2511F53u, a) ^ x[3] ^ k1;
    x[3] = 0xD2511F53u * a;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// Turns the rows held by R (the incumbent's) into candidate c: the n_mut
// mutations drawn from Philox4x32-10 with counter (c, t) and the seed as key
// -- another eligible device for activation i, a swap of two priorities
// inside i's level, or a toggled fuse / prefetch bit of i.  With the rules
// (Algorithm 1, Sec. 3.5) the device is i's best feasible binding and the
// prefetch bit is what PlanPrefetch decides on i's current device.
// R provides dev(i), set_dev(i, d), swap_prio(i, j), toggle_flag(i, bit)
// (bit 0: fuse, 1: prefetch) and set_prefetch(i, on).
template <typename R>
__device__ __forceinline__ void mutate_rows(uint64_t c, const SearchArgs& sa, int N,
                                            const unsigned long long* elig, const uint32_t* alv,
                                            R& rows) {
  if (N <= 0) return;
  for (int t = 0; t < sa.n_mut; ++t) {
    uint32_t x[4] = {(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)t, 0u};
    philox4x32_10(x, (uint32_t)sa.seed, (uint32_t)(sa.seed >> 32));
    const int i = (int)__umulhi(x[1], (uint32_t)N);
    const uint32_t kind = x[0] >> 30;
    if (sa.mode == WF_SEARCH_RULES && (kind == 0u || kind == 3u)) {
      if (kind == 0u) {
        const int b = sa.rule_best[i];
        if (b >= 0) rows.set_dev(i, b);
      } else {
        const int d = rows.dev(i);
        if (d >= 0 && d < sa.D) rows.set_prefetch(i, ((sa.rule_pf[2 * i + (d >> 6)] >> (d & 63)) & 1ull) != 0ull);
      }
    } else if (kind == 0u) {
      unsigned long long e = elig[2 * i], e1 = elig[2 * i + 1];
      const uint32_t n0 = (uint32_t)__popcll(e), n = n0 + (uint32_t)__popcll(e1);
      if (n) {
        uint32_t k = __umulhi(x[2], n);
        int base = 0;
        if (k >= n0) {
          k -= n0;
          e = e1;
          base = 64;
        }
        for (; k; --k) e &= e - 1ull;
        rows.set_dev(i, base + __builtin_ctzll(e));
      }
    } else if (kind == 1u) {
      const uint32_t lvw = alv[i];
      rows.swap_prio(i, (int)(lvw & 0xffffu) + (int)__umulhi(x[2], lvw >> 16));
    } else {
      rows.toggle_flag(i, kind == 3u ? 1 : 0);
    }
  }
}

// Whole rows (device, priority, flag bytes of one candidate).
struct FullRows {
  int8_t* rd;
  uint16_t* rp;
  uint8_t* rf;
  __device__ __forceinline__ int dev(int i) const { return rd[i]; }
  __device__ __forceinline__ void set_dev(int i, int d) { rd[i] = (int8_t)d; }
  __device__ __forceinline__ void swap_prio(int i, int j) {
    const uint16_t pi = rp[i];
    rp[i] = rp[j];
    rp[j] = pi;
  }
  __device__ __forceinline__ void toggle_flag(int i, int bit) {
    rf[i >> 2] ^= (uint8_t)(1u << (((i & 3) << 1) + bit));
  }
  __device__ __forceinline__ void set_prefetch(int i, bool on) {
    const uint8_t b = (uint8_t)(2u << ((i & 3) << 1));
    rf[i >> 2] = on ? (uint8_t)(rf[i >> 2] | b) : (uint8_t)(rf[i >> 2] & ~b);
  }
};

// A candidate as the incumbent's rows plus the changed sites: per plan a
// count, then 2 words per site (activation | priority << 16, device).
struct PatchRows {
  uint32_t* p;             // this plan's count and sites
  const int8_t* idev;      // incumbent rows
  const uint16_t* iprio;
  uint8_t* rf;             // this plan's flag row (staged)
  __device__ __forceinline__ int find(int i) const {
    const int n = (int)p[0];
    for (int k = 0; k < n; ++k)
      if ((int)(p[1 + 2 * k] & 0xffffu) == i) return k;
    return -1;
  }
  __device__ __forceinline__ int site(int i) {
    int k = find(i);
    if (k < 0) {
      k = (int)p[0];
      p[1 + 2 * k] = (uint32_t)i | ((uint32_t)iprio[i] << 16);
      p[2 + 2 * k] = (uint32_t)(int32_t)idev[i];
      p[0] = (uint32_t)(k + 1);
    }
    return k;
  }
  __device__ __forceinline__ int dev(int i) const {
    const int k = find(i);
    return k >= 0 ? (int)(int32_t)p[2 + 2 * k] : (int)idev[i];
  }
  __device__ __forceinline__ int prio(int i) const {
    const int k = find(i);
    return k >= 0 ? (int)(p[1 + 2 * k] >> 16) : (int)iprio[i];
  }
  __device__ __forceinline__ void set_dev(int i, int d) { p[2 + 2 * site(i)] = (uint32_t)d; }
  __device__ __forceinline__ void swap_prio(int i, int j) {
    const int ki = site(i), kj = site(j);
    const uint32_t pi = p[1 + 2 * ki] >> 16, pj = p[1 + 2 * kj] >> 16;
    p[1 + 2 * ki] = (uint32_t)i | (pj << 16);
    p[1 + 2 * kj] = (uint32_t)j | (pi << 16);
  }
  __device__ __forceinline__ void toggle_flag(int i, int bit) {
    rf[i >> 2] ^= (uint8_t)(1u << (((i & 3) << 1) + bit));
  }
  __device__ __forceinline__ void set_prefetch(int i, bool on) {
    const uint8_t b = (uint8_t)(2u << ((i & 3) << 1));
    rf[i >> 2] = on ? (uint8_t)(rf[i >> 2] | b) : (uint8_t)(rf[i >> 2] & ~b);
  }
};


}  // namespace wfp
