// The prefix commit of Algorithm 1 (Prefix_t) for one selected plan: the
// next predicted event after the window time 0 (the earliest activation
// finish, load end or workflow arrival later than 0), and which grants,
// loads and reclamations of the plan begin before it.  O(N) for one plan:
// one workgroup, a block-wide minimum, then one pass of flags.
#include <cstdint>

#include "kernels.h"

namespace wfp {
namespace {

constexpr int kPrefixThreads = 1024;

__device__ __forceinline__ long long wave_min64(long long x) {
  for (int off = 32; off > 0; off >>= 1) {
    const long long o = __shfl_xor(x, off, 64);
    x = o < x ? o : x;
  }
  return x;
}

__global__ __launch_bounds__(kPrefixThreads) void prefix_commit(
    const unsigned char* __restrict__ tab, int off_act, int off_lw, int N, int D,
    long long next_arrival, const int8_t* __restrict__ dev, const int64_t* __restrict__ start,
    const int64_t* __restrict__ finish, const int64_t* __restrict__ load_start,
    const uint64_t* __restrict__ reclaimed, uint8_t* __restrict__ commit,
    uint64_t* __restrict__ commit_rec, int64_t* __restrict__ t_next) {
  __shared__ long long part[kPrefixThreads / 64];
  const uint32_t* act = reinterpret_cast<const uint32_t*>(tab + off_act);
  const int2* lw = reinterpret_cast<const int2*>(tab + off_lw);
  // events later than 0: finishes and load ends (arrivals come from the host)
  long long t = next_arrival;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const long long f = finish[i];
    if (f > 0 && f < t) t = f;
    const long long ls = load_start[i];
    const int d = dev[i];
    if (ls >= 0 && (unsigned)d < (unsigned)D) {
      const long long le = ls + lw[(int)(act[i] & 63u) * D + d].x;
      if (le > 0 && le < t) t = le;
    }
  }
  t = wave_min64(t);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = t;
  __syncthreads();
  if (threadIdx.x < 64) {
    t = threadIdx.x < (int)(blockDim.x >> 6) ? part[threadIdx.x] : (long long)INT64_MAX;
    t = wave_min64(t);
    if (threadIdx.x == 0) part[0] = t;
  }
  __syncthreads();
  t = part[0];
  if (threadIdx.x == 0) *t_next = t;
  // every action that begins before the event is committed, with the
  // reclamations before the unit's first action
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const long long s = start[i], ls = load_start[i];
    const uint32_t grant = s < t ? 1u : 0u;
    const uint32_t load = (ls >= 0 && ls < t) ? 2u : 0u;
    const long long first = ls >= 0 ? ls : s;
    commit[i] = (uint8_t)(grant | load);
    commit_rec[i] = first < t ? reclaimed[i] : 0ull;
  }
}

}  // namespace

hipError_t launch_prefix(const ScoreParams& sp, int64_t next_arrival, const int8_t* dev,
                         const int64_t* start, const int64_t* finish, const int64_t* load_start,
                         const uint64_t* reclaimed, uint8_t* commit, uint64_t* commit_rec,
                         int64_t* t_next, hipStream_t stream) {
  hipLaunchKernelGGL(prefix_commit, dim3(1), dim3(kPrefixThreads), 0, stream, sp.tab, sp.t.act,
                     sp.t.lw, sp.N, sp.D, (long long)next_arrival, dev, start, finish, load_start,
                     reclaimed, commit, commit_rec, t_next);
  return hipGetLastError();
}

}  // namespace wfp
