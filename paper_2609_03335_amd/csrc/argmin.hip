// Batch argmin over plan scores: among feasible plans (status == 0) the
// smallest objective, the lowest plan index on ties, -1 when none is
// feasible (the selection step that follows Propagate in Algorithm 1, with
// the scalar objective in place of the lexicographic key of Eq. 12).
//
// Each plan maps to a 64-bit key (order-preserving objective bits << 32 |
// plan index); infeasible plans map to ~0.  Each block reduces a strided
// share of the plans (wave shuffles, then LDS across its waves) to one
// partial minimum in a work area, and one final block reduces the partials
// and writes the plan index: deterministic, and without a contended atomic.
#include <mutex>

#include "kernels.h"

// Partial minima of wf_plan_argmin_noalloc: one 64-bit key per block of the
// first pass (4 KiB).  Each GPU holds its own copy for the life of the
// process; host code reaches it only through the address that
// hipGetSymbolAddress returns for that GPU (static_scratch below).
static __device__ __align__(256) unsigned long long scratch[wfp::kArgminKeyBlocks];

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

// The block's minimum of k over its 256 threads; valid in thread 0.
__device__ unsigned long long block_min(unsigned long long k) {
  k = wave_min(k);
  __shared__ unsigned long long wmin[4];
  if ((threadIdx.x & 63) == 0) wmin[threadIdx.x >> 6] = k;
  __syncthreads();
  if (threadIdx.x == 0)
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) k = wmin[w] < k ? wmin[w] : k;
  return k;
}

__global__ __launch_bounds__(256) void argmin_partial(const wf_plan_score* __restrict__ s,
                                                      int64_t n, unsigned long long* part) {
  unsigned long long best = ~0ull;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const unsigned long long k = plan_key(s, i);
    best = k < best ? k : best;
  }
  best = block_min(best);
  if (threadIdx.x == 0) part[blockIdx.x] = best;
}

__global__ __launch_bounds__(256) void argmin_final(const unsigned long long* __restrict__ part,
                                                    int nparts, int64_t* out_index) {
  unsigned long long best = ~0ull;
  for (int i = threadIdx.x; i < nparts; i += blockDim.x) best = part[i] < best ? part[i] : best;
  best = block_min(best);
  if (threadIdx.x == 0)
    *out_index = (best == ~0ull) ? (int64_t)-1 : (int64_t)(best & 0xffffffffull);
}

}  // namespace

hipError_t static_scratch(int device, void** out) {
  // looked up once per device, with that device current (the caller's
  // thread has it selected), and kept: every GPU's copy of the array has its
  // own address, and the array's name in host code is no device address
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *out = addr[device];
  return hipSuccess;
}

hipError_t launch_argmin(const wf_plan_score* scores, int64_t n_plans, int64_t* out_index,
                         void* work, hipStream_t stream) {
  unsigned long long* part = reinterpret_cast<unsigned long long*>(work);
  int blocks = 0;
  if (n_plans > 0) {
    const int64_t need = (n_plans + 255) / 256;
    blocks = (int)(need < kArgminKeyBlocks ? need : kArgminKeyBlocks);
    hipLaunchKernelGGL(argmin_partial, dim3(blocks), dim3(256), 0, stream, scores, n_plans, part);
  }
  hipLaunchKernelGGL(argmin_final, dim3(1), dim3(256), 0, stream, part, blocks, out_index);
  return hipGetLastError();
}

}  // namespace wfp

// Lexicographic argmin of ranking keys (Eq. 12): among keys with status 0,
// the smallest (-A_1, ..., -A_4, C_F, -P_N, H_life), the lowest plan index
// on ties, -1 when none is feasible.  Each block reduces a strided share of
// the keys (wave shuffles, then LDS across the block's waves) to one partial
// result in the work area; one final block reduces the partials.
namespace wfp {
namespace {

// (infeasible, packed complements of A_1..A_4, C_F, complement of P_N,
// H_life, index), compared in that order.
struct KeyBest {
  unsigned long long f, a, cf, pn, h;
  long long idx;
};

__device__ __forceinline__ bool key_less(const KeyBest& x, const KeyBest& y) {
  if (x.f != y.f) return x.f < y.f;
  if (x.a != y.a) return x.a < y.a;
  if (x.cf != y.cf) return x.cf < y.cf;
  if (x.pn != y.pn) return x.pn < y.pn;
  if (x.h != y.h) return x.h < y.h;
  return x.idx < y.idx;
}

__device__ __forceinline__ KeyBest key_none() {
  KeyBest b;
  b.f = ~0ull;
  b.a = b.cf = b.pn = b.h = ~0ull;
  b.idx = 0x7fffffffffffffffll;
  return b;
}

__device__ __forceinline__ KeyBest key_of(const wf_plan_key& k, long long i) {
  KeyBest b;
  b.f = k.status != 0u ? 1ull : 0ull;
  b.a = 0ull;
  for (int c = 0; c < WF_MAX_CLASSES; ++c)
    b.a = (b.a << 16) | (unsigned long long)(uint16_t)(0xffffu - k.admitted[c]);
  b.cf = (unsigned long long)k.c_ready_us ^ 0x8000000000000000ull;  // order of int64
  b.pn = 0xffffull - k.timely_prefetch;
  b.h = (unsigned long long)k.h_life_us ^ 0x8000000000000000ull;
  b.idx = i;
  return b;
}

__device__ __forceinline__ KeyBest key_shfl(const KeyBest& x, int off) {
  KeyBest o;
  o.f = __shfl_xor(x.f, off, 64);
  o.a = __shfl_xor(x.a, off, 64);
  o.cf = __shfl_xor(x.cf, off, 64);
  o.pn = __shfl_xor(x.pn, off, 64);
  o.h = __shfl_xor(x.h, off, 64);
  o.idx = __shfl_xor(x.idx, off, 64);
  return o;
}

// The block's best of `best` over its 256 threads; valid in thread 0.
__device__ KeyBest block_best(KeyBest best) {
  for (int off = 32; off > 0; off >>= 1) {
    const KeyBest o = key_shfl(best, off);
    if (key_less(o, best)) best = o;
  }
  __shared__ KeyBest wbest[4];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) wbest[w] = best;
  __syncthreads();
  if (threadIdx.x == 0)
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k)
      if (key_less(wbest[k], best)) best = wbest[k];
  return best;
}

__global__ __launch_bounds__(256) void argmin_key_partial(const wf_plan_key* __restrict__ keys,
                                                          int64_t n, KeyBest* __restrict__ part) {
  KeyBest best = key_none();
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const KeyBest k = key_of(keys[i], i);
    if (key_less(k, best)) best = k;
  }
  best = block_best(best);
  if (threadIdx.x == 0) part[blockIdx.x] = best;
}

__global__ __launch_bounds__(256) void argmin_key_final(const KeyBest* __restrict__ part,
                                                        int nparts, int64_t* out_index) {
  KeyBest best = key_none();
  for (int i = threadIdx.x; i < nparts; i += blockDim.x)
    if (key_less(part[i], best)) best = part[i];
  best = block_best(best);
  if (threadIdx.x == 0) *out_index = best.f == 0ull ? (int64_t)best.idx : (int64_t)-1;
}

}  // namespace

static_assert(sizeof(KeyBest) <= ARGMIN_KEY_WORK_BYTES, "work area per block");

hipError_t launch_argmin_keys(const wf_plan_key* keys, int64_t n_plans, int64_t* out_index,
                              void* work, hipStream_t stream) {
  KeyBest* part = reinterpret_cast<KeyBest*>(work);
  int blocks = 0;
  if (n_plans > 0) {
    const int64_t need = (n_plans + 255) / 256;
    blocks = (int)(need < kArgminKeyBlocks ? need : kArgminKeyBlocks);
    hipLaunchKernelGGL(argmin_key_partial, dim3(blocks), dim3(256), 0, stream, keys, n_plans, part);
  }
  hipLaunchKernelGGL(argmin_key_final, dim3(1), dim3(256), 0, stream, part, blocks, out_index);
  return hipGetLastError();
}

}  // namespace wfp
