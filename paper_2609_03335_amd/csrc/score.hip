// Batched scoring of candidate physical execution plans on gfx950: the
// scalar objective of every plan, and the rows of generated candidates.  The
// kernel itself is in score_kernel.h.
#include "score_kernel.h"

namespace wfp {
namespace {

// One workgroup per candidate: the incumbent's rows, then its mutations.
__global__ __launch_bounds__(64) void search_rows(const int8_t* __restrict__ dev,
                                                  const uint16_t* __restrict__ prio,
                                                  const uint8_t* __restrict__ flags, SearchArgs sa,
                                                  int N, const unsigned long long* elig,
                                                  const uint32_t* alv, int8_t* out_dev,
                                                  uint16_t* out_prio, uint8_t* out_flags) {
  const int64_t k = blockIdx.x;
  const int NB = (N + 3) / 4;
  int8_t* rd = out_dev + k * N;
  uint16_t* rp = out_prio + k * N;
  uint8_t* rf = out_flags + k * NB;
  for (int i = threadIdx.x; i < N; i += 64) {
    rd[i] = dev[i];
    rp[i] = prio[i];
  }
  for (int i = threadIdx.x; i < NB; i += 64) rf[i] = flags[i];
  __syncthreads();
  if (threadIdx.x == 0) mutate((uint64_t)(sa.first + k), sa, N, elig, alv, rd, rp, rf);
}

}  // namespace

hipError_t launch_score(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                        const uint8_t* flags, int64_t n_plans, wf_plan_score* scores,
                        const wf_plan_sched* sched, const SearchArgs* search,
                        hipStream_t stream) {
  return launch_all<false>(sp, dev, prio, flags, n_plans, scores, sched, search, stream);
}

hipError_t launch_search_rows(const ScoreParams& sp, const int8_t* dev, const uint16_t* prio,
                              const uint8_t* flags, const SearchArgs& search, int64_t n,
                              int8_t* out_dev, uint16_t* out_prio, uint8_t* out_flags,
                              hipStream_t stream) {
  const unsigned long long* elig =
      reinterpret_cast<const unsigned long long*>(sp.tab + sp.t.elig);
  const uint32_t* alv = reinterpret_cast<const uint32_t*>(sp.tab + sp.t.alv);
  hipLaunchKernelGGL(search_rows, dim3((unsigned)n), dim3(64), 0, stream, dev, prio, flags, search,
                     sp.N, elig, alv, out_dev, out_prio, out_flags);
  return hipGetLastError();
}

}  // namespace wfp
