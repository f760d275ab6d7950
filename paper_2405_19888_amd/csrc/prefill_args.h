// Arguments of the prefill kernel, shared by the kernel and the host code.
#pragma once

#include "common.h"

namespace parrot {

// Prefill of the new rows of forked contexts.  Rows [qoff[r], qoff[r+1]) of
// q are request r's last Q_r own tokens.  Partial results use the decode
// layout with rows in place of requests: o_part [T][H][seg][D], slots
// [l*seg_p, (l+1)*seg_p) for prefix level l, [seg_pre, seg) for own-token
// chunks of co tokens; merge_meta [T][4].  The single pass (single = 1)
// writes out and lse itself and uses none of o_part, lse_part, merge_meta.
struct PrefillArgs {
  const void* q;         // [T][H][D]
  const void* pk; const void* pv;
  const void* sk; const void* sv;
  const int* ptab; const int* plen; const int* stab; const int* slen; const int* gid;
  const int* parents;    // nested groups (NULL: flat)
  const int* qoff;       // [R + 1]
  float* o_part; float* lse_part;
  int* merge_meta;
  int T, R, H, NG, depth;
  int pstride, sstride, max_p, max_s, max_q, npblk, nsblk;
  int seg, seg_p, seg_pre, seg_s;
  int cp, co;            // prefix and own chunk tokens
  int qtiles_p, qtiles_o;   // row tiles per group, per request
  int n_pre, n_own;      // prefix-chunk and own-chunk work items per head
  int meta_wgs;          // workgroups that also write the row descriptors (256 rows each)
  float scale_log2;
  int single;            // single-pass items (flat groups, one chunk each): write out, lse
  void* out; float* lse; // [T][H][D] dtype, [T][H] (single pass only)
};

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0,
                          hipEvent_t e1);

}  // namespace parrot
