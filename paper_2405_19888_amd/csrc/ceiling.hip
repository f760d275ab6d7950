// Read-bandwidth ceiling of the device (a measurement aid for the roofline of
// the bandwidth-bound decode kernels; Section 8.3 of the paper notes that
// token generation is bound by memory bandwidth).  Every 16-byte piece of a
// buffer is read once with a nontemporal global_load_dwordx4, the way the
// split-KV role streams KV blocks; the values are folded with XOR and each
// wave adds its fold to one word, so no load can be dropped.
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

}  // namespace parrot
