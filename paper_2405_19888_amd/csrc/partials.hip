// The partial-result kernel: one launch that runs both producers of partial
// attention results side by side.
//
//   workgroups [0, n_skv)            split-KV role: every request's own tokens
//                                    (on the per-request path, prefix as well)
//   workgroups [n_skv, n_skv + n_pre) prefix-group role: each group's shared
//                                    prefix, read once for all of its members
//
// The split-KV grid is two workgroups per CU (one when each wave streams two
// heads) and the prefix-group work of the benchmark workloads is about one
// more per CU, so every workgroup is resident from the start (measured: each
// CU holds eight split-KV waves and four prefix-group waves) and the prefix
// work overlaps the own-token stream.  Both roles fit one launch shape: 256
// threads, the LDS union of both roles (about 48 KiB, three workgroups per CU)
// and a register budget of three waves per SIMD (two for the two-heads
// instance).
#include "prefix_role.h"
#include "splitkv_role.h"

namespace parrot {

constexpr int kPartialsLds = kPrefixLds > kSplitkvLds ? kPrefixLds : kSplitkvLds;

template <int DT, int D, bool APPEND, int HPW>
__device__ __forceinline__ void run_splitkv(const SplitKVArgs& a, char* lds, int wg) {
  if constexpr (HPW == 2) {
    splitkv_role<DT, D, true, APPEND, 2>(a, lds, wg);   // shared path, two heads per wave
  } else {
    if (a.with_prefix)
      splitkv_role<DT, D, false, APPEND>(a, lds, wg);   // per-request path: cached loads
    else
      splitkv_role<DT, D, true, APPEND>(a, lds, wg);    // shared path: streaming loads
  }
}

// APPEND: also write this decode step's K/V into the cache (decode with
// append).  HPW = 2: the shared path streams two adjacent heads per split-KV
// wave; twice the registers per fetched block, so that kernel runs two waves
// per SIMD.
template <int DT, int D, bool APPEND, int HPW>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(HPW == 2 ? 2 : 3)))
void k_partials(PartialsArgs a) {
  __shared__ __attribute__((aligned(1024))) char lds[kPartialsLds];
  if ((int)blockIdx.x < a.n_skv)
    run_splitkv<DT, D, APPEND, HPW>(a.skv, lds, blockIdx.x);
  else
    prefix_role<DT, D>(a.pre, lds, blockIdx.x - a.n_skv);
}

template <int DT, int D, bool APPEND>
static void launch_partials_hpw(const PartialsArgs& a, long blocks, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
  if constexpr (DT != kF32) {   // 16-bit caches only (fp32 blocks are twice the registers)
    if (a.skv.hpw == 2) {
      hipExtLaunchKernelGGL((k_partials<DT, D, APPEND, 2>), dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0, a);
      return;
    }
  }
  hipExtLaunchKernelGGL((k_partials<DT, D, APPEND, 1>), dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0, a);
}

template <int DT, int D>
static hipError_t launch_partials_t(const PartialsArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const long blocks = (long)a.n_skv + a.n_pre;
  if (blocks <= 0) return hipSuccess;
  if (a.skv.k_new)
    launch_partials_hpw<DT, D, true>(a, blocks, s, e0, e1);
  else
    launch_partials_hpw<DT, D, false>(a, blocks, s, e0, e1);
  return hipGetLastError();
}

hipError_t launch_partials(const PartialsArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0,
                           hipEvent_t e1) {
  if (a.skv.R > kMaxRequests || a.n_skv < 1 || a.skv.nwaves != a.n_skv * kSkvWaves ||
      (a.skv.hpw != 1 && a.skv.hpw != 2) || a.skv.H % a.skv.hpw != 0 ||
      (a.skv.hpw == 2 && (a.skv.with_prefix || dtype == kF32)) ||
      a.skv.nwaves / (a.skv.H / a.skv.hpw) < 1)
    return hipErrorInvalidValue;
  if (a.n_pre > 0 && (a.pre.cp > prefix_detail::kMaxChunkBlocks * kBlock || a.pre.cp % 32 != 0))
    return hipErrorInvalidValue;
  switch (dtype * 1000 + D) {
    case kF32 * 1000 + 64: return launch_partials_t<kF32, 64>(a, s, e0, e1);
    case kF32 * 1000 + 128: return launch_partials_t<kF32, 128>(a, s, e0, e1);
    case kF16 * 1000 + 64: return launch_partials_t<kF16, 64>(a, s, e0, e1);
    case kF16 * 1000 + 128: return launch_partials_t<kF16, 128>(a, s, e0, e1);
    case kBF16 * 1000 + 64: return launch_partials_t<kBF16, 64>(a, s, e0, e1);
    case kBF16 * 1000 + 128: return launch_partials_t<kBF16, 128>(a, s, e0, e1);
  }
  return hipErrorInvalidValue;
}

}  // namespace parrot
