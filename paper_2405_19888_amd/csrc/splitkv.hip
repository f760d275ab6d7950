// Split-KV decode attention over paged K/V (the non-shared tokens of each
// request; with the prefix slots enabled it is also the per-request baseline).
//
// One wavefront owns one work item (request r, head h, chunk c).  A chunk is a
// run of whole 16-token blocks.  A token row is D*elt bytes, read as
// D*elt/16 lanes x 16 bytes, so every load instruction of the wave covers a
// contiguous 1 KiB of the block (fully coalesced 128-bit loads).  Each group
// of lanes that shares a token computes its slice of q.k, the slices are summed
// with DPP row operations, and every token group keeps its own online-softmax
// state; the groups are combined once at the end of the chunk.  The chunk's
// normalised output and its base-2 log-sum-exp go to the workspace.
#include "common.h"

namespace parrot {

template <int DT, int D>
__global__ __launch_bounds__(256) void k_splitkv(SplitKVArgs a) {
  using E = Elem<DT>;
  constexpr int ROW_B = D * E::kBytes;        // bytes per token row
  constexpr int LPT = ROW_B / 16;             // lanes per token
  constexpr int TPI = kWave / LPT;            // tokens per load instruction
  constexpr int IPB = kBlock / TPI;           // load instructions per block
  constexpr int EPL = E::kPerLoad;            // elements per lane load
  static_assert(TPI * ROW_B == 1024, "one instruction covers 1 KiB");

  const int lane = threadIdx.x & 63;
  const long wave = (long)blockIdx.x * (blockDim.x >> 6) +
                    __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int H = a.H;
  if (wave >= (long)a.R * a.nc * H) return;
  const int h = (int)(wave % H);
  const long rest = wave / H;
  const int c = a.first_c + (int)(rest % a.nc);
  const int r = (int)(rest / a.nc);

  // resolve the chunk to a token range of one paged sequence
  int t0, t1, nblk;
  const int* tbl;
  const char* kpool;
  const char* vpool;
  if (c < a.seg_p) {
    const int g = a.gid[r];
    if (g < 0 || g >= a.NG) return;
    const int P = clampi(a.plen[g], 0, a.max_p);
    t0 = c * a.cp;
    if (t0 >= P) return;
    t1 = min(P, t0 + a.cp);
    tbl = a.ptab + (long)g * a.pstride;
    kpool = (const char*)a.pk; vpool = (const char*)a.pv; nblk = a.npblk;
  } else {
    const int S = clampi(a.slen[r], 0, a.max_s);
    t0 = (c - a.seg_p) * a.cs;
    if (t0 >= S) return;
    t1 = min(S, t0 + a.cs);
    tbl = a.stab + (long)r * a.sstride;
    kpool = (const char*)a.sk; vpool = (const char*)a.sv; nblk = a.nsblk;
  }

  const int sub = lane % LPT;                 // which 16-byte slice of the row
  const int tg = lane / LPT;                  // token group
  const u32x4 qf = ld16((const char*)a.q + ((size_t)(r * H + h) * D + sub * EPL) * E::kBytes);
  const size_t blk_stride = (size_t)H * kBlock * ROW_B;
  const size_t head_off = (size_t)h * kBlock * ROW_B + (size_t)lane * 16;

  float m = -INFINITY, l = 0.f;
  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.f;

  const int b0 = t0 / kBlock, b1 = (t1 + kBlock - 1) / kBlock;
  u32x4 kc[IPB], vc[IPB], kn[IPB], vn[IPB];
  {
    const int blk = clampi(tbl[b0], 0, nblk - 1);
    const char* kb = kpool + blk * blk_stride + head_off;
    const char* vb = vpool + blk * blk_stride + head_off;
#pragma unroll
    for (int i = 0; i < IPB; ++i) { kc[i] = ld16(kb + i * 1024); vc[i] = ld16(vb + i * 1024); }
  }
  for (int b = b0; b < b1; ++b) {
    if (b + 1 < b1) {
      const int blk = clampi(tbl[b + 1], 0, nblk - 1);
      const char* kb = kpool + blk * blk_stride + head_off;
      const char* vb = vpool + blk * blk_stride + head_off;
#pragma unroll
      for (int i = 0; i < IPB; ++i) { kn[i] = ld16(kb + i * 1024); vn[i] = ld16(vb + i * 1024); }
    }
    float s[IPB];
#pragma unroll
    for (int i = 0; i < IPB; ++i) s[i] = group_sum<LPT>(E::dot(kc[i], qf)) * a.scale_log2;
    if (b * kBlock + kBlock > t1) {           // partly filled block: mask the tail
#pragma unroll
      for (int i = 0; i < IPB; ++i) {
        if (b * kBlock + i * TPI + tg >= t1) {
          s[i] = -INFINITY;
          vc[i] = u32x4{0u, 0u, 0u, 0u};      // 0 * NaN would poison the sum
        }
      }
    }
    float bm = s[0];
#pragma unroll
    for (int i = 1; i < IPB; ++i) bm = fmaxf(bm, s[i]);
    const float mn = fmaxf(m, bm);
    const float mref = (mn == -INFINITY) ? 0.f : mn;
    const float alpha = fast_exp2(m - mref);
    float psum = 0.f;
    float p[IPB];
#pragma unroll
    for (int i = 0; i < IPB; ++i) { p[i] = fast_exp2(s[i] - mref); psum += p[i]; }
    l = l * alpha + psum;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] *= alpha;
#pragma unroll
    for (int i = 0; i < IPB; ++i) {
      float v[EPL];
      E::to_f32(vc[i], v);
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = __builtin_fmaf(p[i], v[e], acc[e]);
    }
    m = mn;
#pragma unroll
    for (int i = 0; i < IPB; ++i) { kc[i] = kn[i]; vc[i] = vn[i]; }
  }

  // combine the token groups that share a row slice
#pragma unroll
  for (int off = LPT; off < kWave; off <<= 1) {
    const float mo = __shfl_xor(m, off);
    const float lo = __shfl_xor(l, off);
    const float mn = fmaxf(m, mo);
    const float mref = (mn == -INFINITY) ? 0.f : mn;
    const float sa = fast_exp2(m - mref), sb = fast_exp2(mo - mref);
    l = l * sa + lo * sb;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = acc[e] * sa + __shfl_xor(acc[e], off) * sb;
    m = mn;
  }
  if (tg == 0) {
    const size_t slot = (size_t)(r * H + h) * a.seg + c;
    const float inv = 1.f / l;
    float* o = a.o_part + slot * D + sub * EPL;
#pragma unroll
    for (int e = 0; e < EPL; e += 4)
      *reinterpret_cast<f32x4*>(o + e) = f32x4{acc[e] * inv, acc[e + 1] * inv, acc[e + 2] * inv, acc[e + 3] * inv};
    if (lane == 0) a.lse_part[slot] = m + fast_log2(l);
  }
}

template <int DT, int D>
static hipError_t launch_splitkv_t(const SplitKVArgs& a, hipStream_t s) {
  const long waves = (long)a.R * a.nc * a.H;
  if (waves <= 0) return hipSuccess;
  const long blocks = (waves + 3) / 4;
  hipLaunchKernelGGL((k_splitkv<DT, D>), dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_splitkv(const SplitKVArgs& a, int dtype, int D, hipStream_t s) {
  switch (dtype * 1000 + D) {
    case kF32 * 1000 + 64: return launch_splitkv_t<kF32, 64>(a, s);
    case kF32 * 1000 + 128: return launch_splitkv_t<kF32, 128>(a, s);
    case kF16 * 1000 + 64: return launch_splitkv_t<kF16, 64>(a, s);
    case kF16 * 1000 + 128: return launch_splitkv_t<kF16, 128>(a, s);
    case kBF16 * 1000 + 64: return launch_splitkv_t<kBF16, 64>(a, s);
    case kBF16 * 1000 + 128: return launch_splitkv_t<kBF16, 128>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace parrot
