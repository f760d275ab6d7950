// Log-sum-exp merge of the partial results of every (request, head), and the
// device-side input validator.
//
// Partials of disjoint key sets combine exactly: with base-2 log-sum-exps
// l_i and normalised outputs o_i, the union has l = log2 sum_i 2^{l_i} and
// o = sum_i 2^{l_i - l} o_i (Section 7, "Kernel Optimization": the prefix's
// interim results are amalgamated with the non-shared part).
#include "common.h"

namespace parrot {

template <int N>
PARROT_DEV float group_max(float x) {
  x = fmaxf(x, dpp_f<kDppXor1>(x));
  x = fmaxf(x, dpp_f<kDppXor2>(x));
  x = fmaxf(x, dpp_f<kDppHalfMirror>(x));
  x = fmaxf(x, dpp_f<kDppMirror>(x));
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

// One wave per (request, head); each lane owns D/64 output elements.  The
// request's slot counts come from the descriptor the split-KV workgroup 0
// wrote, so the only dependent load before the data is that descriptor.  Lane
// i then reads the log-sum-exp of slot i while the partial outputs of its
// first kBatch partials are loaded in the same round; later ones (long
// prefixes or long runs) are read batch by batch with their weights.
// kBatch: partial outputs loaded per round (registers: kBatch * D / 64 per
// lane); the small variant serves calls with at most 8 slots per sequence.
template <int DT, int D, int kBatch>
__global__ __launch_bounds__(256) void k_merge(MergeArgs a) {
  using E = Elem<DT>;
  constexpr int EPL = D / kWave;
  static_assert(kBatch <= kWave, "one batch's weights fit one lane each");
  const int lane = threadIdx.x & 63;
  const long w = (long)blockIdx.x * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (w >= (long)a.R * a.H) return;
  const int r = (int)(w / a.H);
  const int h = (int)(w % a.H);
  const int4 meta = *reinterpret_cast<const int4*>(a.merge_meta + kMetaInts * r);
  const int nlev = meta.y;                  // prefix levels of the request's chain
  const unsigned lo = (unsigned)meta.z, hi = (unsigned)meta.w;
  int np[kMaxDepth] = {(int)(lo & 0xFFFFu), (int)(lo >> 16), (int)(hi & 0xFFFFu), (int)(hi >> 16)};
#pragma unroll
  for (int l = 0; l < kMaxDepth; ++l) np[l] = l < nlev ? np[l] : 0;
  // partial i of the request: level 0's chunks, level 1's, ..., then the pieces
  const int b1 = np[0], b2 = b1 + np[1], b3 = b2 + np[2], b4 = b3 + np[3];
  const int n = b4 + meta.x;
  const size_t base = (size_t)(r * a.H + h) * a.seg;
  char* outp = (char*)a.out + ((size_t)(r * a.H + h) * D + lane * EPL) * E::kBytes;
  if (n == 0) {  // empty context: defined as out = 0, lse = -inf
#pragma unroll
    for (int e = 0; e < EPL; ++e) E::store1(outp + e * E::kBytes, 0.f);
    if (lane == 0) a.lse[r * a.H + h] = -INFINITY;
    return;
  }
  auto slot_of = [&](int i) {               // selects only, so loads unroll freely
    int sl = a.seg_pre + (i - b4);
    sl = i < b4 ? 3 * a.seg_p + (i - b3) : sl;
    sl = i < b3 ? 2 * a.seg_p + (i - b2) : sl;
    sl = i < b2 ? a.seg_p + (i - b1) : sl;
    return i < b1 ? i : sl;
  };
  // lane i holds the slot of partial i; the first 64 are broadcast by readlane
  const int slot_lane = slot_of(lane);
  auto slot_bcast = [&](int i) { return i < kWave ? __builtin_amdgcn_readlane(slot_lane, i) : slot_of(i); };
  auto load_o = [&](int i, float* v) {
    const float* src = a.o_part + (base + slot_bcast(i)) * D + lane * EPL;
    if constexpr (EPL == 2) {
      const float2 x = *reinterpret_cast<const float2*>(src);
      v[0] = x.x; v[1] = x.y;
    } else {
#pragma unroll
      for (int e = 0; e < EPL; ++e) v[e] = src[e];
    }
  };

  // first pass: every lane's lse slot and the first batch of outputs together
  const float l_lane = lane < n ? a.lse_part[base + slot_lane] : -INFINITY;
  float v[kBatch][EPL];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    // only the partials that exist: the workspace stride (kBatch follows it)
    // can be far above a sequence's partial count, and loads of repeated
    // slots would still cost the cache round trips (measured: the 32-layer
    // mixed workload's merge 11.1 -> 7.0 us)
    if (u < n) load_o(u, v[u]);
  }

  float mx = l_lane;
  for (int i = lane + kWave; i < n; i += kWave) mx = fmaxf(mx, a.lse_part[base + slot_of(i)]);
  mx = group_max<64>(mx);
  const float w_lane = lane < n ? fast_exp2(l_lane - mx) : 0.f;
  float tot = w_lane;
  for (int i = lane + kWave; i < n; i += kWave) tot += fast_exp2(a.lse_part[base + slot_of(i)] - mx);
  tot = group_sum<64>(tot);

  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    if (u < n) {
      const float wu = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w_lane), u));
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = __builtin_fmaf(wu, v[u][e], acc[e]);
    }
  }
  for (int j0 = kBatch; j0 < n; j0 += kBatch) {
    float wv[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int j = min(j0 + u, n - 1);
      load_o(j, v[u]);
      wv[u] = a.lse_part[base + slot_bcast(j)];
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (j0 + u < n) {
        const float wu = fast_exp2(wv[u] - mx);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = __builtin_fmaf(wu, v[u][e], acc[e]);
      }
    }
  }
  const float inv = 1.f / tot;
#pragma unroll
  for (int e = 0; e < EPL; ++e) E::store1(outp + e * E::kBytes, acc[e] * inv);
  if (lane == 0) a.lse[r * a.H + h] = (mx + fast_log2(tot)) * kLn2;
}

template <int DT, int D>
static hipError_t launch_merge_t(const MergeArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const long waves = (long)a.R * a.H;
  if (waves <= 0) return hipSuccess;
  const dim3 grid((unsigned)((waves + 3) / 4));
  // The 8-partial batch (fewer registers, more waves resident) whenever a
  // sequence's partials are expected to fit it: at most 8 slots, or, on the
  // shared path, at most 4 prefix chunks ahead of the own-token pieces (a run
  // of own tokens touches one or two pieces there; more take further rounds).
  // Measured on the 32-layer mixed workload (4 prefix chunks, 64 slots):
  // 5.6 us against 6.9 us with the 32-partial batch.
  if (a.seg <= 8 || (a.seg_pre > 0 && a.seg_pre <= 4))
    hipExtLaunchKernelGGL((k_merge<DT, D, 8>), grid, dim3(256), 0, s, e0, e1, 0, a);
  else
    hipExtLaunchKernelGGL((k_merge<DT, D, 64 / (D / kWave)>), grid, dim3(256), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  switch (dtype * 1000 + D) {
    case kF32 * 1000 + 64: return launch_merge_t<kF32, 64>(a, s, e0, e1);
    case kF32 * 1000 + 128: return launch_merge_t<kF32, 128>(a, s, e0, e1);
    case kF16 * 1000 + 64: return launch_merge_t<kF16, 64>(a, s, e0, e1);
    case kF16 * 1000 + 128: return launch_merge_t<kF16, 128>(a, s, e0, e1);
    case kBF16 * 1000 + 64: return launch_merge_t<kBF16, 64>(a, s, e0, e1);
    case kBF16 * 1000 + 128: return launch_merge_t<kBF16, 128>(a, s, e0, e1);
  }
  return hipErrorInvalidValue;
}

// --------------------------------------------------------------- validation
// Error codes written to result[0] (first failure wins): 1 bad group id,
// 2 bad prefix length, 3 bad suffix length, 4 empty context, 5 prefix block id
// out of the pool, 6 suffix block id out of the pool, 7 bad parent, 8 chain
// too deep; prefill rows: 9 bad row offsets, 10 too many rows for a request,
// 11 too many rows reading a group; decode: 12 more requests read a group's
// prefix than max_group_size (the prefix role sizes its query tiles from that
// bound, so readers past it would get no prefix partial).  result[1] is the
// entry index, result[2] the offending value.
PARROT_DEV void report(int* res, int code, int idx, int val) {
  if (atomicCAS(res, 0, code) == 0) { res[1] = idx; res[2] = val; }
}

__global__ __launch_bounds__(256) void k_validate(ValidateArgs a) {
  for (int g = threadIdx.x; g < a.NG; g += blockDim.x) {
    if (a.parents) {
      // parent in [-1, g): chains end; a chain of at most depth groups
      const int par = a.parents[g];
      if (par < -1 || par >= g) { report(a.result, 7, g, par); continue; }
      // walk at most depth steps (another group's parent may be invalid too)
      int n = 1;
      for (int x = par; x >= 0 && x < a.NG && n <= a.depth; x = a.parents[x]) ++n;
      if (n > a.depth) { report(a.result, 8, g, n); continue; }
    }
    const int P = a.plen[g];
    if (P < 1 || P > a.max_p) { report(a.result, 2, g, P); continue; }
    for (int b = 0; b < (P + a.B - 1) / a.B; ++b) {
      const int id = a.ptab[(long)g * a.pstride + b];
      if (id < 0 || id >= a.npblk) report(a.result, 5, g * a.pstride + b, id);
    }
  }
  for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
    const int g = a.gid[r];
    if (g < -1 || g >= a.NG) { report(a.result, 1, r, g); continue; }
    const int S = a.slen[r];
    if (S < 0 || S > a.max_s) { report(a.result, 3, r, S); continue; }
    const int P = g >= 0 ? a.plen[g] : 0;
    if (P + S < 1) report(a.result, 4, r, P + S);
    for (int b = 0; b < (S + a.B - 1) / a.B; ++b) {
      const int id = a.stab[(long)r * a.sstride + b];
      if (id < 0 || id >= a.nsblk) report(a.result, 6, r * a.sstride + b, id);
    }
  }
  if (a.qoff) {
    if (threadIdx.x == 0) {
      if (a.qoff[0] != 0) report(a.result, 9, 0, a.qoff[0]);
      if (a.qoff[a.R] != a.T) report(a.result, 9, a.R, a.qoff[a.R]);
    }
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
      const long n = (long)a.qoff[r + 1] - a.qoff[r];
      if (n < 0) { report(a.result, 9, r + 1, a.qoff[r + 1]); continue; }
      if (n > a.slen[r] || n > a.max_q) report(a.result, 10, r, (int)n);
    }
  }
  // readers of each group's prefix: its members and its descendants' members
  // (decode: one per request; prefill: the request's rows), summed in LDS for
  // 1024 groups at a time and compared with the bound the launch was sized for
  __shared__ unsigned long long cnt[1024];
  const int code = a.qoff ? 11 : 12;
  for (int g0 = 0; g0 < a.NG; g0 += 1024) {
    for (int i = threadIdx.x; i < 1024; i += blockDim.x) cnt[i] = 0;
    __syncthreads();
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
      const long n = a.qoff ? (long)a.qoff[r + 1] - a.qoff[r] : 1;
      const unsigned long long add = n > 0 ? (unsigned long long)n : 0ull;
      int x = a.gid[r];
      for (int d = 0; d < a.depth && x >= 0 && x < a.NG; ++d) {
        if (x >= g0 && x < g0 + 1024) atomicAdd(&cnt[x - g0], add);
        x = a.parents ? a.parents[x] : -1;
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 1024 && g0 + i < a.NG; i += blockDim.x)
      if (cnt[i] > (unsigned long long)a.max_grp)
        report(a.result, code, g0 + i, cnt[i] > 0x7fffffffull ? 0x7fffffff : (int)cnt[i]);
    __syncthreads();
  }
}

hipError_t launch_validate(const ValidateArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace parrot
