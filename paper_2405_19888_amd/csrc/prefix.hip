// Prefix-group decode attention on MFMA (gfx950).
//
// One workgroup owns (group g, head h, prefix chunk c, query tile qt).  The
// chunk's K and V blocks are staged through LDS in 16 KiB tiles per tensor,
// double-buffered, so the shared prefix is read from HBM once per group
// (Section 6, "Kernel Optimization": prefix KV tiles are loaded to on-chip
// memory once and reused by every request of the group).  Each wave owns 16 of
// the group's queries and computes, per 16-token block,
//   S^T = K * Q^T   (16 tokens x 16 queries; v_mfma_f32_16x16x32_{f16,bf16})
//   O^T += V^T * P^T (D x 16 queries; v_mfma_f32_16x16x16{f16,bf16_1k})
// with an online softmax in fp32.  Computing the transposed products keeps
// every per-query quantity (running max, sum, output rows) in the lanes that
// own that query, so the softmax needs no lane shuffles besides the block max.
// V^T operands come straight from the row-major LDS tile through
// ds_read_b64_tr_b16.  fp32 inputs use v_mfma_f32_16x16x4f32 with the same
// tiling.  Each member's partial result (normalised output, base-2
// log-sum-exp) is written to its own workspace slot.
#include "common.h"

namespace parrot {

namespace {

constexpr int kTileBytes = 16384;   // per tensor per stage

typedef __attribute__((address_space(3))) char lds_char;

PARROT_DEV u32x4 lds_ld16(const char* p) { return *reinterpret_cast<const u32x4*>(p); }

template <int DT> struct Mfma;

template <> struct Mfma<kF16> {
  PARROT_DEV static f32x4 qk(const u32x4& a, const u32x4& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
  PARROT_DEV static unsigned long long pack_p(const float* p) {
    f16x4 h = {(_Float16)p[0], (_Float16)p[1], (_Float16)p[2], (_Float16)p[3]};
    return __builtin_bit_cast(unsigned long long, h);
  }
  PARROT_DEV static unsigned long long tr_read(const char* lds_ptr) {
    typedef __attribute__((address_space(3))) f16x4 lds_v4;
    typedef __fp16 fp16x4_ __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) fp16x4_ lds_fp16x4;
    fp16x4_ v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_fp16x4*)(lds_char*)lds_ptr);
    return __builtin_bit_cast(unsigned long long, v);
  }
  PARROT_DEV static f32x4 pv(unsigned long long a, unsigned long long b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a), __builtin_bit_cast(f16x4, b), c, 0, 0, 0);
  }
};

template <> struct Mfma<kBF16> {
  PARROT_DEV static f32x4 qk(const u32x4& a, const u32x4& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  PARROT_DEV static unsigned long long pack_p(const float* p) {
    bf16x4 h = {(__bf16)p[0], (__bf16)p[1], (__bf16)p[2], (__bf16)p[3]};
    return __builtin_bit_cast(unsigned long long, h);
  }
  PARROT_DEV static unsigned long long tr_read(const char* lds_ptr) {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds_char*)lds_ptr);
    return __builtin_bit_cast(unsigned long long, v);
  }
  PARROT_DEV static f32x4 pv(unsigned long long a, unsigned long long b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a), __builtin_bit_cast(i16x4, b), c, 0, 0, 0);
  }
};

}  // namespace

template <int DT, int D>
__global__ __launch_bounds__(512) void k_prefix(PrefixArgs a) {
  using E = Elem<DT>;
  constexpr int ROW_B = D * E::kBytes;
  constexpr int BLK_B = kBlock * ROW_B;               // one block of one head
  constexpr int TILE_BLK = kTileBytes / BLK_B;        // blocks per stage
  constexpr int CHUNKS = 2 * kTileBytes / 16;         // 16-byte pieces per stage (K and V)
  constexpr int MAX_PER_THREAD = CHUNKS / 256;        // workgroups have >= 4 waves
  constexpr int DT16 = D / 16;                        // 16-wide d tiles
  static_assert(TILE_BLK >= 1, "tile holds a block");

  __shared__ __attribute__((aligned(16))) char smem[2][2][kTileBytes];
  __shared__ int members[128];
  __shared__ int s_count;

  const int nthreads = blockDim.x;
  const int nwaves = nthreads >> 6;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  int wg = blockIdx.x;
  const int H = a.H;
  const int h = wg % H; wg /= H;
  const int c = wg % a.seg_p; wg /= a.seg_p;
  const int qt = wg % a.qtiles;
  const int g = wg / a.qtiles;
  if (g >= a.NG) return;
  const int P = clampi(a.plen[g], 0, a.max_p);
  const int t0 = c * a.cp;
  if (t0 >= P) return;
  const int t1 = min(P, t0 + a.cp);
  const int qbase = qt * nwaves * 16;

  // members of group g, in request order; this tile takes [qbase, qbase + 16*nwaves)
  if (wave == 0) {
    int count = 0;
    for (int base = 0; base < a.R; base += kWave) {
      const int r = base + lane;
      const bool is = r < a.R && a.gid[r] == g;
      const unsigned long long mask = __ballot(is);
      const int pos = count + __popcll(mask & ((1ull << lane) - 1ull));
      if (is && pos >= qbase && pos < qbase + nwaves * 16) members[pos - qbase] = r;
      count += __popcll(mask);
    }
    if (lane == 0) s_count = count;
  }
  __syncthreads();
  const int nq = min(s_count - qbase, nwaves * 16);
  if (nq <= 0) return;                                 // uniform over the workgroup

  const int qi = wave * 16 + (lane & 15);              // this lane's query column
  const bool has_q = wave * 16 < nq;                   // wave-uniform
  const bool q_ok = qi < nq;
  const int rq = q_ok ? members[qi] : 0;

  // query operand (B of S^T = K Q^T): lane holds query lane%16, k-slice lane/16
  constexpr int KS = (DT == kF32) ? D / 4 : D / 32;   // MFMA k-steps over D
  u32x4 qf16[(DT == kF32) ? 1 : KS];
  float qf32[(DT == kF32) ? KS : 1];
  {
    const char* qrow = (const char*)a.q + (size_t)(rq * H + h) * ROW_B;
    if constexpr (DT == kF32) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf32[ks] = q_ok ? reinterpret_cast<const float*>(qrow)[4 * ks + (lane >> 4)] : 0.f;
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf16[ks] = q_ok ? ld16(qrow + (32 * ks + 8 * (lane >> 4)) * 2) : u32x4{0u, 0u, 0u, 0u};
    }
  }

  const int b0 = t0 / kBlock;
  const int nb = (t1 - t0 + kBlock - 1) / kBlock;
  const int nstages = (nb + TILE_BLK - 1) / TILE_BLK;
  const int* tbl = a.ptab + (long)g * a.pstride;
  const size_t blk_stride = (size_t)H * BLK_B;
  const size_t head_off = (size_t)h * BLK_B;
  const char* kpool = (const char*)a.pk;
  const char* vpool = (const char*)a.pv;

  // cooperative stage load: piece e in [0, CHUNKS): tensor e / (CHUNKS/2),
  // block (e % (CHUNKS/2)) / (BLK_B/16), 16-byte offset inside that block
  u32x4 stage_regs[MAX_PER_THREAD];
  auto load_stage = [&](int st) {
#pragma unroll
    for (int j = 0; j < MAX_PER_THREAD; ++j) {
      const int e = tid + j * nthreads;
      stage_regs[j] = u32x4{0u, 0u, 0u, 0u};
      if (e < CHUNKS) {
        const int tensor = e / (CHUNKS / 2);
        const int w = e % (CHUNKS / 2);
        const int bl = w / (BLK_B / 16);
        const int off = w % (BLK_B / 16);
        const int b = st * TILE_BLK + bl;              // block index within the chunk
        const int tok = (b0 + b) * kBlock + (off * 16) / ROW_B;
        if (b < nb && tok < t1) {
          const int blk = clampi(tbl[b0 + b], 0, a.npblk - 1);
          const char* src = (tensor ? vpool : kpool) + blk * blk_stride + head_off + off * 16;
          stage_regs[j] = ld16(src);
        }
      }
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int j = 0; j < MAX_PER_THREAD; ++j) {
      const int e = tid + j * nthreads;
      if (e < CHUNKS) {
        const int tensor = e / (CHUNKS / 2);
        const int w = e % (CHUNKS / 2);
        *reinterpret_cast<u32x4*>(&smem[buf][tensor][w * 16]) = stage_regs[j];
      }
    }
  };

  float m = -INFINITY, lsum = 0.f;
  f32x4 o[DT16];
#pragma unroll
  for (int i = 0; i < DT16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_stage(0);
  store_stage(0);
  __syncthreads();
  for (int st = 0; st < nstages; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstages) load_stage(st + 1);
    if (has_q) {
      const char* ktile = smem[buf][0];
      const char* vtile = smem[buf][1];
      const int nbl = min(TILE_BLK, nb - st * TILE_BLK);
      for (int bl = 0; bl < nbl; ++bl) {
        const char* kb = ktile + bl * BLK_B;
        const char* vb = vtile + bl * BLK_B;
        // S^T[token 4*(lane/16)+i][query lane%16]
        f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
        if constexpr (DT == kF32) {
          const float* kf = reinterpret_cast<const float*>(kb + (lane & 15) * ROW_B);
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            s4 = __builtin_amdgcn_mfma_f32_16x16x4f32(kf[4 * ks + (lane >> 4)], qf32[ks], s4, 0, 0, 0);
        } else {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            s4 = Mfma<DT>::qk(lds_ld16(kb + (lane & 15) * ROW_B + (32 * ks + 8 * (lane >> 4)) * 2), qf16[ks], s4);
        }
        const int tok_base = (b0 + st * TILE_BLK + bl) * kBlock + 4 * (lane >> 4);
        float s[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) s[i] = (tok_base + i < t1) ? s4[i] * a.scale_log2 : -INFINITY;
        float bm = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
        bm = fmaxf(bm, __shfl_xor(bm, 16));
        bm = fmaxf(bm, __shfl_xor(bm, 32));
        const float mn = fmaxf(m, bm);                 // finite: the block has a token
        const float alpha = fast_exp2(m - mn);
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = fast_exp2(s[i] - mn);
        lsum = lsum * alpha + (p[0] + p[1]) + (p[2] + p[3]);
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) o[dt] *= alpha;
        if constexpr (DT == kF32) {
          // O^T[d][q] += V^T[d][t] P^T[t][q] with k index kk <-> token 4*kk + kt
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) {
            const float* vrow = reinterpret_cast<const float*>(vb + (4 * (lane >> 4) + kt) * ROW_B);
#pragma unroll
            for (int dt = 0; dt < DT16; ++dt)
              o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vrow[dt * 16 + (lane & 15)], p[kt], o[dt], 0, 0, 0);
          }
        } else {
          const unsigned long long pb = Mfma<DT>::pack_p(p);
          // lane k of 16-lane group G reads V[4G + k/4][dt*16 + 4*(k%4) .. +3]
          const char* vsrc = vb + (4 * (lane >> 4) + ((lane & 15) >> 2)) * ROW_B + 4 * (lane & 3) * 2;
#pragma unroll
          for (int dt = 0; dt < DT16; ++dt)
            o[dt] = Mfma<DT>::pv(Mfma<DT>::tr_read(vsrc + dt * 32), pb, o[dt]);
        }
        m = mn;
      }
    }
    if (st + 1 < nstages) store_stage(buf ^ 1);
    __syncthreads();
  }

  if (!has_q) return;
  float lt = lsum + __shfl_xor(lsum, 16);
  lt += __shfl_xor(lt, 32);
  if (q_ok) {
    const size_t slot = (size_t)(rq * H + h) * a.seg + c;
    const float inv = 1.f / lt;
    float* dst = a.o_part + slot * D + 4 * (lane >> 4);
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) *reinterpret_cast<f32x4*>(dst + dt * 16) = o[dt] * inv;
    if (lane < 16) a.lse_part[slot] = m + fast_log2(lt);
  }
}

template <int DT, int D>
static hipError_t launch_prefix_t(const PrefixArgs& a, int waves, hipStream_t s) {
  const long blocks = (long)a.NG * a.seg_p * a.H * a.qtiles;
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_prefix<DT, D>), dim3((unsigned)blocks), dim3(64 * waves), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_prefix(const PrefixArgs& a, int dtype, int D, int waves, hipStream_t s) {
  if (waves < 4 || waves > 8) return hipErrorInvalidValue;
  switch (dtype * 1000 + D) {
    case kF32 * 1000 + 64: return launch_prefix_t<kF32, 64>(a, waves, s);
    case kF32 * 1000 + 128: return launch_prefix_t<kF32, 128>(a, waves, s);
    case kF16 * 1000 + 64: return launch_prefix_t<kF16, 64>(a, waves, s);
    case kF16 * 1000 + 128: return launch_prefix_t<kF16, 128>(a, waves, s);
    case kBF16 * 1000 + 64: return launch_prefix_t<kBF16, 64>(a, waves, s);
    case kBF16 * 1000 + 128: return launch_prefix_t<kBF16, 128>(a, waves, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace parrot
