// Internal declarations shared by the kernels and the C-ABI layer of
// libparrot_attn (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

namespace parrot {

// ---------------------------------------------------------------- constants
constexpr int kBlock = 16;          // tokens per KV block
constexpr int kWave = 64;           // CDNA wavefront
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Partial results live in the workspace as
//   o_part  [R][H][seg][D] float32   (normalised partial output of one piece)
//   lse_part[R][H][seg]    float32   (base-2 log-sum-exp of the piece's scaled logits)
//   merge_meta[R][4]       int32     (per request: split-KV pieces, prefix levels,
//                                     prefix-chunk slots per level, 16 bits each)
// Slots [l*seg_p, l*seg_p + seg_p) hold the prefix-group chunks of the group
// at level l of the request's chain (chunk c covers that prefix's tokens
// [c*cp, (c+1)*cp); level 0 is the outermost group, and flat groups use level
// 0 only); slots [seg_pre, seg) hold split-KV pieces, seg_pre = depth * seg_p.  The
// split-KV kernel sees every request's blocks (own tokens, preceded by its
// group's prefix on the per-request path) as one flat list ordered by
// (request, head, block) and gives each wave an equal run of it; piece p of
// sequence (r, h) is the part that the p-th wave touching that sequence owns.
struct Plan {
  int cp;                // prefix chunk tokens (prefix-group kernel)
  int depth;             // prefix levels (1 for flat groups)
  int seg_p, seg_pre, seg_s, seg; // slots per (request, head)
  int prefix_waves;      // waves per prefix-kernel workgroup (16 queries each)
  int prefix_qtiles;     // query tiles per group
  int skv_waves;         // split-KV grid, in waves
  int skv_min_q;         // blocks per split-KV wave, lower bound
  size_t o_bytes, lse_bytes, info_bytes, total_bytes;
};

constexpr int kMaxRequests = 1024;   // per call (split-KV keeps per-request data in LDS)
constexpr int kSkvWaves = 4;         // waves per split-KV workgroup
constexpr int kMaxDepth = 4;         // prefix levels of nested groups
constexpr int kMetaInts = 4;         // merge_meta ints per request

struct SplitKVArgs {
  const void* q;
  const void* pk; const void* pv;
  const void* sk; const void* sv;
  const int* ptab; const int* plen;
  const int* stab; const int* slen;
  const int* gid;
  const int* parents;    // nested groups (NULL: flat)
  const void* k_new;     // this step's token per (request, head), or NULL
  const void* v_new;
  void* app_k; void* app_v;   // pools the new token is written to (suffix pools)
  float* o_part; float* lse_part;
  int* merge_meta;       // written by split-KV workgroup 0 for the merge
  int R, H, NG;
  int pstride, sstride;
  int max_p, max_s;
  int npblk, nsblk;
  int seg, seg_pre, cp;
  int depth;             // prefix levels walked for the merge descriptor
  int with_prefix;       // 1: each sequence is the group prefix, then the own tokens
  int nwaves;            // waves launched
  int min_q;             // blocks per wave >= min_q
  int hpw;               // heads per split-KV wave: 1, or 2 (shared path, H even)
  float scale_log2;      // sm_scale * log2(e)
};

struct PrefixArgs {
  const void* q;
  const void* pk; const void* pv;
  const int* ptab; const int* plen; const int* gid;
  const int* parents;    // nested groups (NULL: flat)
  int depth;             // prefix levels (1: flat)
  float* o_part; float* lse_part;
  int R, H, NG;
  int pstride, max_p, npblk;
  int seg, seg_p, cp;
  int qtiles;            // query tiles per group (grid factor)
  float scale_log2;
};

struct MergeArgs {
  const float* o_part; const float* lse_part;
  const int* merge_meta;
  void* out; float* lse;
  int R, H;
  int seg, seg_p, seg_pre;   // slots per sequence, per prefix level, before the pieces
};

struct ValidateArgs {
  const int* ptab; const int* plen; const int* stab; const int* slen; const int* gid;
  const int* parents;    // nested groups (NULL: flat)
  int depth;             // prefix levels allowed (nested)
  int* result;           // [0] = error code, [1] = index, [2] = value
  int R, NG, B;
  int pstride, sstride, max_p, max_s, npblk, nsblk;
  const int* qoff;       // prefill row offsets [R + 1] (NULL: decode)
  int T, max_q, max_grp; // prefill rows, rows per request, rows per group
};

// dtype codes follow parrot_dtype
enum Dtype { kF32 = 0, kF16 = 1, kBF16 = 2 };

// Both producers of partial results in one launch: n_skv split-KV workgroups
// followed by n_pre prefix-group workgroups (none on the per-request path).
struct PartialsArgs {
  SplitKVArgs skv;
  PrefixArgs pre;
  int n_skv, n_pre;
};

// Each launcher attaches the optional (start, stop) timing events to its kernel.
// a.skv.k_new != NULL selects the kernel that also appends this step's token
hipError_t launch_partials(const PartialsArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_merge(const MergeArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_validate(const ValidateArgs& a, hipStream_t s);

// ------------------------------------------------------------ device helpers
#if defined(__HIP_DEVICE_COMPILE__)
#define PARROT_DEV __device__ __forceinline__
#else
#define PARROT_DEV __device__ inline
#endif

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// DPP lane moves inside rows of 16 lanes (bound_ctrl: out-of-row reads give 0,
// never used here because every control below stays inside its row).
template <int CTRL>
PARROT_DEV float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7-i within each 8
constexpr int kDppMirror = 0x140;     // lane i <-> 15-i within each 16

// Sum over aligned groups of N lanes (N = 4, 8, 16, 32, 64); every lane of the
// group receives the total.
template <int N>
PARROT_DEV float group_sum(float x) {
  static_assert(N == 4 || N == 8 || N == 16 || N == 32 || N == 64, "group size");
  x += dpp_f<kDppXor1>(x);
  x += dpp_f<kDppXor2>(x);
  if constexpr (N >= 8) x += dpp_f<kDppHalfMirror>(x);
  if constexpr (N >= 16) x += dpp_f<kDppMirror>(x);
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

// Workgroup barrier for kernels that manage their own memory counters: this
// wave's LDS operations complete (lgkmcnt 0), then s_barrier.  No hardware
// fence and no wait on vector-memory loads, so direct-to-LDS loads issued
// earlier stay in flight (a __syncthreads() would wait for every global load
// still in flight: on gfx9 loads and stores share one counter); the empty asm
// statements keep the compiler from moving memory accesses across the barrier.
PARROT_DEV void lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt and expcnt untouched
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// 16-byte direct-to-LDS load (global_load_lds_dwordx4): lane l's 16 bytes
// from `src` land at LDS byte address lds_base + 16 * l.  lds_base must be
// wave-uniform.  Written as inline assembly so that the compiler does not
// attach its own (conservative) waits for these loads: the caller owns the
// vmcnt accounting, must have no other vector-memory loads outstanding where
// it waits, and must drain its loads (wait_vmcnt<0>) before the wave ends.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is clobbered on purpose
PARROT_DEV void lds_dma16(const void* src, unsigned lds_base) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off"
      :
      : "s"(lds_base), "v"(src)
      : "memory", "m0");
}
// The same load in the instruction's scalar-base form: a wave-uniform 64-bit
// base plus a per-lane 32-bit byte offset (lane l reads base + voff).
PARROT_DEV void lds_dma16_sbase(const void* base, unsigned voff, unsigned lds_base) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2"
      :
      : "s"(lds_base), "v"(voff), "s"(base)
      : "memory", "m0");
}
#pragma clang diagnostic pop

PARROT_DEV unsigned lds_addr(const void* p) {
  return (unsigned)(size_t)((__attribute__((address_space(3))) const char*)p);
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14).
template <int N>
PARROT_DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// max(x[l], x[l ^ 16]) and max(x[l], x[l ^ 32]) with the gfx950 lane-swap
// instructions (VALU, no trip through the LDS crossbar): the two outputs of a
// self-swap hold x[l] and x[l ^ 16] (resp. x[l ^ 32]) in some order.
PARROT_DEV float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
PARROT_DEV float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
PARROT_DEV float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
PARROT_DEV float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

PARROT_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
PARROT_DEV float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// 16-byte global load (kept as a plain vector load so the compiler emits
// global_load_dwordx4).
PARROT_DEV u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
// Wave-uniform read of a read-only int through the constant address space,
// which the compiler turns into a scalar load.  Scalar loads are counted by
// lgkmcnt, so waiting for such a value (a block-table entry that the next KV
// addresses depend on) does not also wait for the vector loads in flight.
PARROT_DEV int ld_uniform(const int* p) {
  typedef __attribute__((address_space(4))) const int const_int;
  return *reinterpret_cast<const_int*>(reinterpret_cast<uintptr_t>(p));
}
// Streaming 16-byte load (nontemporal hint) for KV data read once per call:
// on this GPU it sustains about 10 % more read bandwidth than a cached load.
PARROT_DEV u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Reinterpret one 32-bit word as a pair of 16-bit floats.  The word is taken
// by value on purpose: this compiler's __builtin_bit_cast applied directly to an
// ext-vector element such as v.y reads element 0 instead.
PARROT_DEV f16x2 as_f16x2(unsigned u) { return __builtin_bit_cast(f16x2, u); }
PARROT_DEV bf16x2 as_bf16x2(unsigned u) { return __builtin_bit_cast(bf16x2, u); }

// Element traits: conversion of the 16 bytes a lane loads into floats, and the
// dot product of those bytes with the lane's query slice.
template <int DT> struct Elem;

template <> struct Elem<kF32> {
  static constexpr int kBytes = 4;
  static constexpr int kPerLoad = 4;
  PARROT_DEV static void to_f32(const u32x4& v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  PARROT_DEV static float dot(const u32x4& k, const u32x4& q) {
    float f[4], g[4];
    to_f32(k, f); to_f32(q, g);
    float s = f[0] * g[0];
    s = __builtin_fmaf(f[1], g[1], s);
    s = __builtin_fmaf(f[2], g[2], s);
    return __builtin_fmaf(f[3], g[3], s);
  }
  PARROT_DEV static void store1(void* p, float x) { *reinterpret_cast<float*>(p) = x; }
};

template <> struct Elem<kF16> {
  static constexpr int kBytes = 2;
  static constexpr int kPerLoad = 8;
  PARROT_DEV static void to_f32(const u32x4& v, float* f) {
    const unsigned w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f16x2 h = as_f16x2(w[i]);
      f[2 * i] = (float)h.x;
      f[2 * i + 1] = (float)h.y;
    }
  }
  PARROT_DEV static float dot(const u32x4& k, const u32x4& q) {
    float s = __builtin_amdgcn_fdot2(as_f16x2(k.x), as_f16x2(q.x), 0.0f, false);
    s = __builtin_amdgcn_fdot2(as_f16x2(k.y), as_f16x2(q.y), s, false);
    s = __builtin_amdgcn_fdot2(as_f16x2(k.z), as_f16x2(q.z), s, false);
    return __builtin_amdgcn_fdot2(as_f16x2(k.w), as_f16x2(q.w), s, false);
  }
  PARROT_DEV static void store1(void* p, float x) { *reinterpret_cast<_Float16*>(p) = (_Float16)x; }
};

template <> struct Elem<kBF16> {
  static constexpr int kBytes = 2;
  static constexpr int kPerLoad = 8;
  PARROT_DEV static void to_f32(const u32x4& v, float* f) {
    const unsigned w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  PARROT_DEV static float dot(const u32x4& k, const u32x4& q) {
    float s = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.x), as_bf16x2(q.x), 0.0f, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.y), as_bf16x2(q.y), s, false);
    s = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.z), as_bf16x2(q.z), s, false);
    return __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.w), as_bf16x2(q.w), s, false);
  }
  PARROT_DEV static void store1(void* p, float x) { *reinterpret_cast<__bf16*>(p) = (__bf16)x; }
};

// Clamp helpers: device contents are trusted, but indices are clamped so that
// a bad value can never move an access outside the buffers.
PARROT_DEV int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

}  // namespace parrot
