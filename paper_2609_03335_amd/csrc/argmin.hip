// Batch argmin over plan scores: among feasible plans (status == 0) the
// smallest objective, the lowest plan index on ties, -1 when none is
// feasible (the selection step that follows Propagate in Algorithm 1, with
// the scalar objective in place of the lexicographic key of Eq. 12).
//
// Each plan maps to a 64-bit key (order-preserving objective bits << 32 |
// plan index); infeasible plans map to ~0.  The minimum key is reduced in a
// wave with cross-lane shuffles, then across the grid with one 64-bit atomic
// min per wave into the caller's output slot, which a final single-lane
// kernel turns into the plan index.  The output slot doubles as the
// reduction cell, so the call needs no library-owned scratch.
#include "kernels.h"

namespace wfp {
namespace {

__device__ __forceinline__ unsigned long long plan_key(const wf_plan_score* s, int64_t i) {
  if (s[i].status != 0u) return ~0ull;
  uint32_t b = __float_as_uint(s[i].objective);
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);  // total order on non-NaN floats
  return ((unsigned long long)b << 32) | (unsigned long long)(uint32_t)i;
}

__device__ __forceinline__ unsigned long long wave_min(unsigned long long k) {
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long o = __shfl_xor(k, off, 64);
    k = o < k ? o : k;
  }
  return k;
}

__global__ __launch_bounds__(64) void argmin_init(unsigned long long* cell) { *cell = ~0ull; }

__global__ __launch_bounds__(256) void argmin_reduce(const wf_plan_score* __restrict__ s,
                                                     int64_t n, unsigned long long* cell) {
  unsigned long long best = ~0ull;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const unsigned long long k = plan_key(s, i);
    best = k < best ? k : best;
  }
  best = wave_min(best);
  if ((threadIdx.x & 63) == 0 && best != ~0ull) atomicMin(cell, best);
}

__global__ __launch_bounds__(64) void argmin_finish(unsigned long long* cell) {
  const unsigned long long k = *cell;
  *reinterpret_cast<int64_t*>(cell) = (k == ~0ull) ? (int64_t)-1 : (int64_t)(k & 0xffffffffull);
}

}  // namespace

hipError_t launch_argmin(const wf_plan_score* scores, int64_t n_plans, int64_t* out_index,
                         int grid, hipStream_t stream) {
  unsigned long long* cell = reinterpret_cast<unsigned long long*>(out_index);
  hipLaunchKernelGGL(argmin_init, dim3(1), dim3(1), 0, stream, cell);
  if (n_plans > 0) {
    int64_t need = (n_plans + 255) / 256;
    const int g = (int)(need < grid ? need : grid);
    hipLaunchKernelGGL(argmin_reduce, dim3(g), dim3(256), 0, stream, scores, n_plans, cell);
  }
  hipLaunchKernelGGL(argmin_finish, dim3(1), dim3(1), 0, stream, cell);
  return hipGetLastError();
}

}  // namespace wfp
