// Measurement aids.  The read-bandwidth ceiling of the device (the roofline of
// the bandwidth-bound decode kernels; Section 8.3 of the paper notes that
// token generation is bound by memory bandwidth), and the matrix-core issue
// ceiling with a given share of vector instructions (the roofline of the
// MFMA-bound prefill tile, whose softmax interleaves vector work with its
// products).  Every 16-byte piece of a
// buffer is read once with a nontemporal global_load_dwordx4, the way the
// split-KV role streams KV blocks; the values are folded with XOR and each
// wave adds its fold to one word, so no load can be dropped.
#include "ceiling.h"
#include "common.h"

namespace parrot {

PARROT_DEV unsigned fold(const u32x4& v) { return v.x ^ v.y ^ v.z ^ v.w; }

PARROT_DEV void publish(unsigned acc, unsigned* sink) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) atomicXor(sink, acc);
}

// Grid-stride order: thread t of the grid reads pieces t, t + T, t + 2T, ...
// (T = all threads), UNROLL of them per iteration, so consecutive lanes read
// consecutive pieces (1 KiB per wave instruction) and each thread keeps
// UNROLL loads in flight.
template <int UNROLL>
__global__ __launch_bounds__(256) void k_read_grid_stride(const u32x4* __restrict__ src, size_t n16,
                                                           unsigned* sink) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  unsigned acc = 0;
  for (; i + (UNROLL - 1) * stride < n16; i += UNROLL * stride) {
    u32x4 v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= fold(v[u]);
  }
  for (; i < n16; i += stride) acc ^= fold(__builtin_nontemporal_load(src + i));
  publish(acc, sink);
}

// Span order: the buffer's whole 1 KiB rows (64 pieces) are cut into one
// contiguous span per wave, which the wave reads front to back, UNROLL rows in
// flight (the access order of a KV stream); the pieces after the last whole
// row are read by the first wave.
template <int UNROLL>
__global__ __launch_bounds__(256) void k_read_spans(const u32x4* __restrict__ src, size_t n16,
                                                     unsigned* sink) {
  const int lane = threadIdx.x & 63;
  const size_t waves = (size_t)gridDim.x * (blockDim.x >> 6);
  const size_t w = (size_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const size_t rows = n16 / kWave;
  const size_t per = (rows + waves - 1) / waves;
  const size_t r0 = w * per < rows ? w * per : rows;
  const size_t r1 = r0 + per < rows ? r0 + per : rows;
  unsigned acc = 0;
  size_t r = r0;
  for (; r + UNROLL <= r1; r += UNROLL) {
    u32x4 v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + (r + u) * kWave + lane);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= fold(v[u]);
  }
  for (; r < r1; ++r) acc ^= fold(__builtin_nontemporal_load(src + r * kWave + lane));
  if (w == 0 && rows * kWave + lane < n16) acc ^= fold(__builtin_nontemporal_load(src + rows * kWave + lane));
  publish(acc, sink);
}

// The optional (e0, e1) events are attached to the launch itself, as the
// decode kernels' are.
template <int UNROLL>
static void launch_read(const u32x4* p, size_t n16, unsigned* sink, int workgroups, bool spans,
                        hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((unsigned)workgroups), block(256);
  if (spans)
    hipExtLaunchKernelGGL(k_read_spans<UNROLL>, grid, block, 0, s, e0, e1, 0, p, n16, sink);
  else
    hipExtLaunchKernelGGL(k_read_grid_stride<UNROLL>, grid, block, 0, s, e0, e1, 0, p, n16, sink);
}

hipError_t launch_read_ceiling(const void* src, size_t bytes, unsigned* sink, int workgroups,
                               int unroll, bool spans, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const size_t n16 = bytes / 16;
  const u32x4* p = reinterpret_cast<const u32x4*>(src);
  switch (unroll) {
    case 4: launch_read<4>(p, n16, sink, workgroups, spans, s, e0, e1); break;
    case 8: launch_read<8>(p, n16, sink, workgroups, spans, s, e0, e1); break;
    case 16: launch_read<16>(p, n16, sink, workgroups, spans, s, e0, e1); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Matrix-core issue probe: registers only.  Each iteration issues eight
// independent v_mfma_f32_16x16x32_f16 (eight accumulator chains) and, spread
// evenly between them, VX4 / 4 vector instructions per MFMA (four v_exp_f32
// per iteration, the rest v_fmac_f32 on independent registers).  The instructions are inline
// assembly in the written order, so the compiler neither drops nor regroups
// them; every result is folded into the sink at the end.  A kernel whose
// softmax issues about VX4 / 4 vector instructions per MFMA cannot beat this
// rate.
#define PARROT_PROBE_MFMA(c) \
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b))
#define PARROT_PROBE_EXP(x) asm volatile("v_exp_f32 %0, %0" : "+v"(x))
#define PARROT_PROBE_FMA(x) asm volatile("v_fmac_f32 %0, %0, %1" : "+v"(x) : "v"(k))

template <int VX4>
__global__ __launch_bounds__(256) void k_mfma_issue(int iters, unsigned* sink) {
  constexpr int NV = VX4 * 2;                         // vector instructions per iteration
  static_assert(NV == 0 || (NV >= 8 && NV <= 32), "vector share");
  const int lane = threadIdx.x & 63;
  f16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) { a[i] = (_Float16)(0.001f * (lane + i)); b[i] = (_Float16)(0.001f * (lane - i)); }
  f32x4 c[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) c[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float e[4], f[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = -0.001f * (lane + j);
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = 0.001f * (lane - j);
  const float k = 0.5f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      PARROT_PROBE_MFMA(c[j]);
      // after MFMA j: NV / 8 vector instructions (one more on the first NV % 8
      // slots), the even slots' first one an exp
      constexpr int base = NV / 8, extra = NV % 8;
      const int n = base + (j < extra ? 1 : 0);
#pragma unroll
      for (int u = 0; u < 5; ++u) {
        if (u < n) {
          if (u == 0 && j % 2 == 0) PARROT_PROBE_EXP(e[j / 2]);
          else PARROT_PROBE_FMA(f[(j + u) % 8]);
        }
      }
    }
  }
  // the last MFMA results are read by plain vector code below: let them land
  // (the accumulators are operands, so no read of them moves above the wait)
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+v"(c[0]), "+v"(c[1]), "+v"(c[2]), "+v"(c[3]), "+v"(c[4]), "+v"(c[5]), "+v"(c[6]), "+v"(c[7]));
  unsigned acc = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    acc ^= __float_as_uint(c[j][0]) ^ __float_as_uint(c[j][1]) ^ __float_as_uint(c[j][2]) ^ __float_as_uint(c[j][3]);
#pragma unroll
  for (int j = 0; j < 4; ++j) acc ^= __float_as_uint(e[j]);
#pragma unroll
  for (int j = 0; j < 8; ++j) acc ^= __float_as_uint(f[j]);
  publish(acc, sink);
}
#undef PARROT_PROBE_MFMA
#undef PARROT_PROBE_EXP
#undef PARROT_PROBE_FMA

hipError_t launch_mfma_issue(unsigned* sink, int workgroups, int iters, int vx4, hipStream_t s,
                             hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((unsigned)workgroups), block(256);
  switch (vx4) {
    case 0: hipExtLaunchKernelGGL(k_mfma_issue<0>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    case 8: hipExtLaunchKernelGGL(k_mfma_issue<8>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    case 10: hipExtLaunchKernelGGL(k_mfma_issue<10>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    case 11: hipExtLaunchKernelGGL(k_mfma_issue<11>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    case 12: hipExtLaunchKernelGGL(k_mfma_issue<12>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    case 16: hipExtLaunchKernelGGL(k_mfma_issue<16>, grid, block, 0, s, e0, e1, 0, iters, sink); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace parrot
