// Prefix-group decode attention on MFMA (gfx950).
//
// One workgroup owns (group g, head h, prefix chunk c, query tile qt).  The
// chunk's K and V blocks pass through LDS in 16 KiB stages (K and V together),
// so the shared prefix is read from HBM once per group (Section 7, "Kernel
// Optimization": prefix KV tiles are loaded to on-chip memory once and reused
// by every request of the group).  Stages are fetched with direct-to-LDS loads
// (global_load_lds_dwordx4) into a ring of three stage buffers, two stages
// ahead of the one being computed; the wait for a stage is an explicit vmcnt,
// so the loads need no registers and stay in flight across the barriers.
//
// Each wave owns 16 of the group's queries and computes, per 16-token block,
//   S^T  = K Q^T    (16 tokens x 16 queries; v_mfma_f32_16x16x32_{f16,bf16})
//   O^T += V^T P^T  (D x 16 queries; v_mfma_f32_16x16x16{f16,bf16_1k})
// with an online softmax in fp32.  Computing the transposed products keeps the
// per-query running max, sum and output rows in the lanes that own the query,
// so only the block max crosses lanes (lane-swap instructions, no LDS trip).
// V^T operands come straight from the row-major LDS tile through
// ds_read_b64_tr_b16.  fp32 inputs use v_mfma_f32_16x16x4f32 with the same
// tiling.
//
// LDS rows are swizzled: 16-byte granule j of token row t is stored at granule
// j ^ f(t), f(t) = ((t & 3) << 1) | ((t >> 2) & 1).  Eight consecutive rows then
// hit eight distinct granules (conflict-free 128-bit K reads by 16 lanes of
// different tokens), and four consecutive rows hit four distinct granule pairs
// (conflict-free transposed V reads).  The swizzle is applied on the global
// side: each lane of a direct-to-LDS load fetches the granule that belongs at
// its fixed LDS slot.
#pragma once

#include <cfloat>

#include "common.h"

namespace parrot {

namespace prefix_detail {

constexpr int kTensorStage = 8192;   // bytes of K (and of V) per stage
constexpr int kStageBytes = 2 * kTensorStage;
constexpr int kStageChunks = kStageBytes / 1024;  // 1 KiB per direct-to-LDS instruction
constexpr int kRing = 3;             // stage buffers in LDS (kRing - 1 stages in flight)
constexpr int kMaxChunkBlocks = 64;  // prefix chunk <= 1024 tokens


typedef __attribute__((address_space(3))) char lds_char;

PARROT_DEV int swz(int t) { return ((t & 3) << 1) | ((t >> 2) & 1); }

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
    typedef __fp16 fp16x4_ __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) fp16x4_ lds_fp16x4;
    fp16x4_ v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_fp16x4*)(lds_char*)lds_ptr);
    return __builtin_bit_cast(unsigned long long, v);
  }
  PARROT_DEV static f32x4 pv(unsigned long long a, unsigned long long b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a), __builtin_bit_cast(f16x4, b), c, 0, 0, 0);
  }
  // acc plus the four probabilities packed in w, as rounded (dot2 with (1, 1)
  // adds two packed halves into fp32 exactly)
  PARROT_DEV static float sum_p(unsigned long long w, float acc) {
    const f16x2 one = {(_Float16)1.f, (_Float16)1.f};
    acc = __builtin_amdgcn_fdot2(as_f16x2((unsigned)w), one, acc, false);
    return __builtin_amdgcn_fdot2(as_f16x2((unsigned)(w >> 32)), one, acc, false);
  }
  // k = 32 over two blocks: operand halves (lo, hi) hold block A and block B
  PARROT_DEV static f32x4 pv2(unsigned long long alo, unsigned long long ahi, unsigned long long blo,
                               unsigned long long bhi, f32x4 c) {
    const u32x4 a = {(unsigned)alo, (unsigned)(alo >> 32), (unsigned)ahi, (unsigned)(ahi >> 32)};
    const u32x4 b = {(unsigned)blo, (unsigned)(blo >> 32), (unsigned)bhi, (unsigned)(bhi >> 32)};
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
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
  PARROT_DEV static float sum_p(unsigned long long w, float acc) {
    const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
    acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2((unsigned)w), one, acc, false);
    return __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2((unsigned)(w >> 32)), one, acc, false);
  }
  PARROT_DEV static f32x4 pv2(unsigned long long alo, unsigned long long ahi, unsigned long long blo,
                               unsigned long long bhi, f32x4 c) {
    const u32x4 a = {(unsigned)alo, (unsigned)(alo >> 32), (unsigned)ahi, (unsigned)(ahi >> 32)};
    const u32x4 b = {(unsigned)blo, (unsigned)(blo >> 32), (unsigned)bhi, (unsigned)(bhi >> 32)};
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};

}  // namespace prefix_detail

constexpr int kPrefixWaves = 4;   // 16 queries per wave, 64 per workgroup
#ifndef PARROT_PREFIX_VT_AHEAD
#define PARROT_PREFIX_VT_AHEAD 4
#endif
// d tiles whose V^T fragments a decode prefix tile reads ahead of its scores
constexpr int kVtAhead = PARROT_PREFIX_VT_AHEAD;
#ifndef PARROT_PREFIX_RING
#define PARROT_PREFIX_RING 3
#endif
// Stage buffers of the decode prefix role's ring (kDecodeRing - 1 stages in
// flight per workgroup).
constexpr int kDecodeRing = PARROT_PREFIX_RING;
static_assert(kDecodeRing >= 3 && kDecodeRing <= 8, "decode prefix ring depth");
// LDS bytes of a query tile of up to `rows` rows whose key range spans up to
// `blocks` blocks: the stage ring, the tile's query rows, the key block ids, a
// count, and the rows' last visible key (causal tiles).
constexpr int tile_lds_bytes(int blocks, int rows = kPrefixWaves * 16, int ring = prefix_detail::kRing) {
  return ring * prefix_detail::kStageBytes + (2 * rows + blocks + 4) * 4;
}
constexpr int kPrefixLds = tile_lds_bytes(prefix_detail::kMaxChunkBlocks, kPrefixWaves * 16, kDecodeRing);

// LDS views shared by the tile's set-up code and the tile cores.
struct TileLds {
  char (*smem)[prefix_detail::kStageBytes];   // [ring][kStageBytes]
  int* rows;                                  // [rows] query row of each tile column
  int* tbl;                                   // [blocks] key blocks, clamped
  int* count;                                 // set-up scratch
  int* lim;                                   // [rows] last visible key token (causal)
  PARROT_DEV explicit TileLds(char* lds, int blocks = prefix_detail::kMaxChunkBlocks,
                              int nrows = kPrefixWaves * 16, int ring = prefix_detail::kRing)
      : smem(reinterpret_cast<char (*)[prefix_detail::kStageBytes]>(lds)),
        rows(reinterpret_cast<int*>(lds + ring * prefix_detail::kStageBytes)),
        tbl(rows + nrows),
        count(tbl + blocks),
        lim(count + 4) {}
};

// One query tile against one range of a paged key sequence.
struct TileJob {
  const void* q;                  // [rows][H][D]
  const void* pk; const void* pv; // pools of the key sequence
  int npool;                      // blocks in those pools
  int H, h;
  int t0, t1;                     // key tokens [t0, t1); t0 a multiple of 16
  float* o_part; float* lse_part; // partial results [rows][H][seg][D], [rows][H][seg]
  int seg, slot;                  // slots per (row, head); this tile's slot
  float scale_log2;
  int lim_min;                    // causal tiles: the smallest row limit (tl.lim)
};

// The attention core of a query tile: up to 64 query rows (tl.rows, nq of
// them) against key tokens [t0, t1) whose blocks are in tl.tbl; with CAUSAL,
// row i sees only keys up to tl.lim[i].  Rows and blocks must be in LDS and
// visible to every wave.  Writes one partial result (normalised output and
// base-2 log-sum-exp; a row that sees no key gets 0 and -inf) per row.  RING:
// stage buffers of tl.smem (RING - 1 stages in flight).
template <int DT, int D, bool CAUSAL, int RING = prefix_detail::kRing>
__device__ __forceinline__ void tile_core(const TileJob& j, const TileLds& tl, int nq);

// One workgroup of the prefix role; `wg` is the role-local workgroup index.
template <int DT, int D>
__device__ __forceinline__ void prefix_role(const PrefixArgs& a, char* lds, int wg) {
  using namespace prefix_detail;
  constexpr int W = kPrefixWaves;
  const TileLds tl(lds, kMaxChunkBlocks, W * 16, kDecodeRing);
  int* members = tl.rows;
  int* s_tbl = tl.tbl;
  int& s_count = tl.count[0];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  const int H = a.H;
  const int h = wg % H; wg /= H;
  const int c = wg % a.seg_p; wg /= a.seg_p;
  const int qt = wg % a.qtiles;
  const int g = wg / a.qtiles;
  if (g >= a.NG) return;
  const int P = clampi(a.plen[g], 0, a.max_p);
  // level of g: its number of ancestors (at most depth - 1)
  int lvl = 0;
  if (a.parents) {
    int x = a.parents[g];
    while (x >= 0 && x < a.NG && lvl < a.depth - 1) {
      ++lvl;
      x = a.parents[x];
    }
  }
  const int t0 = c * a.cp;
  if (t0 >= P) return;
  const int t1 = min(P, t0 + a.cp);
  const int qbase = qt * W * 16;
  const int b0 = t0 / kBlock;
  const int nb = (t1 - t0 + kBlock - 1) / kBlock;     // <= cp / 16 <= kMaxChunkBlocks
  const int* tbl = a.ptab + (long)g * a.pstride;

  // members of group g in request order (this tile takes [qbase, qbase + 16 W));
  // the chunk's block ids, clamped into the pool
  if (wave == 0) {
    int count = 0;
    for (int base = 0; base < a.R; base += kWave) {
      const int r = base + lane;
      // r reads g's prefix when g is r's group or one of its ancestors
      bool is = false;
      if (r < a.R) {
        int x = a.gid[r];
        for (int d = 0; d < a.depth && x >= 0 && x < a.NG; ++d) {
          if (x == g) { is = true; break; }
          x = a.parents ? a.parents[x] : -1;
        }
      }
      const unsigned long long mask = __ballot(is);
      const int pos = count + __popcll(mask & ((1ull << lane) - 1ull));
      if (is && pos >= qbase && pos < qbase + W * 16) members[pos - qbase] = r;
      count += __popcll(mask);
    }
    if (lane == 0) s_count = count;
  } else if (wave == 1) {
    for (int i = lane; i < nb; i += kWave) s_tbl[i] = clampi(tbl[b0 + i], 0, a.npblk - 1);
  }
  __syncthreads();
  const int nq = min(s_count - qbase, W * 16);
  if (nq <= 0) return;                                 // uniform over the workgroup
  TileJob job;
  job.q = a.q; job.pk = a.pk; job.pv = a.pv; job.npool = a.npblk; job.H = H; job.h = h;
  job.t0 = t0; job.t1 = t1; job.o_part = a.o_part; job.lse_part = a.lse_part;
  job.seg = a.seg; job.slot = lvl * a.seg_p + c; job.scale_log2 = a.scale_log2;
  tile_core<DT, D, false, kDecodeRing>(job, tl, nq);
}

template <int DT, int D, bool CAUSAL, int RING>
__device__ __forceinline__ void tile_core(const TileJob& a, const TileLds& tl, int nq) {
  using namespace prefix_detail;
  constexpr int W = kPrefixWaves;
  using E = Elem<DT>;
  constexpr int ROW_B = D * E::kBytes;
  constexpr int GRAN = ROW_B / 16;                    // 16-byte granules per row
  constexpr int BLK_B = kBlock * ROW_B;               // one block of one head
  constexpr int STAGE_BLK = kTensorStage / BLK_B;     // blocks per stage
  constexpr int DT16 = D / 16;                        // 16-wide d tiles
  constexpr int KS = (DT == kF32) ? D / 4 : D / 32;   // MFMA k-steps over D
  constexpr int PER_WAVE = kStageChunks / W;          // direct-to-LDS loads per wave per stage
  static_assert(STAGE_BLK >= 1 && GRAN >= 8, "stage holds a block; swizzle fits a row");
  static_assert(kStageChunks % W == 0, "stage chunks split evenly over waves");

  auto smem = tl.smem;
  const int* members = tl.rows;
  const int* s_tbl = tl.tbl;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int H = a.H, h = a.h, t1 = a.t1;
  const int b0 = a.t0 / kBlock;
  const int nb = (a.t1 - a.t0 + kBlock - 1) / kBlock;

  const int qi = wave * 16 + (lane & 15);              // this lane's query column
  const bool has_q = wave * 16 < nq;                   // wave-uniform
  const bool q_ok = qi < nq;
  const int rq = q_ok ? members[qi] : 0;

  // 16-bit caches keep a lazy reference max, as the prefill tile does: the
  // reference mref (scaled log2 units) moves only when some lane's raw logits
  // exceed thr = (mref + kLazy) / scale, so the probabilities stay below
  // 2^kLazy and most pairs need no cross-lane max and no rescale.  lsr sums
  // the probabilities as rounded for the PV products and normalises the
  // output; lsum (unrounded) gives the lse.  A negative scale flips the sign
  // of q (exact), so the test runs on |scale|; a zero scale is taken as 1e-30.
  constexpr float kLazy = 8.f;
  const float scale = fmaxf(fabsf(a.scale_log2), 1e-30f);
  const float inv_scale = 1.f / scale;
  const unsigned qsign = a.scale_log2 < 0.f ? 0x80008000u : 0u;

  // query operand (B of S^T = K Q^T): lane holds query lane%16, k-slice lane/16
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
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 v = q_ok ? ld16(qrow + (32 * ks + 8 * (lane >> 4)) * 2) : u32x4{0u, 0u, 0u, 0u};
        qf16[ks] = v ^ u32x4{qsign, qsign, qsign, qsign};
      }
    }
  }
  // Direct-to-LDS stage loads.  Wave w issues chunks w, w + W, ... of each
  // stage; lane l of a chunk writes LDS bytes [16 l, 16 l + 16) of that chunk,
  // i.e. block bl, token row t, granule slot pos, and fetches the global
  // granule pos ^ f(t) of that row.
  const size_t blk_stride = (size_t)H * BLK_B;
  int c_bl[PER_WAVE];
  unsigned c_src[PER_WAVE];
  bool c_v[PER_WAVE];
#pragma unroll
  for (int j = 0; j < PER_WAVE; ++j) {
    const int q = wave + j * W;                        // chunk index in the stage
    const int off = (q % (kStageChunks / 2)) * 1024 + lane * 16;   // byte in the tensor stage
    c_v[j] = q >= kStageChunks / 2;
    c_bl[j] = off / BLK_B;
    const int t = (off % BLK_B) / ROW_B;
    const int pos = (off % ROW_B) / 16;
    c_src[j] = (unsigned)(h * BLK_B + t * ROW_B + ((pos ^ swz(t)) << 4));
  }
  const int nstages = (nb + STAGE_BLK - 1) / STAGE_BLK;
  const int last = nstages - 1;
  // Block ids of a stage (wave-uniform: a chunk lies inside one block) are read
  // from the LDS table one stage before its loads are issued, so issuing waits
  // on nothing; each load takes the block's base in scalar registers and the
  // lane's offset in a vector register.
  int tb[PER_WAVE];
  auto table = [&](int st) {
#pragma unroll
    for (int j = 0; j < PER_WAVE; ++j) tb[j] = s_tbl[min(st * STAGE_BLK + c_bl[j], nb - 1)];   // past the chunk: re-read, unused
  };
  auto issue = [&](int buf) {
#pragma unroll
    for (int j = 0; j < PER_WAVE; ++j) {
      // block ids are clamped when the table is filled; clamping again here
      // keeps every load inside the pool whatever the LDS table holds
      const unsigned blk = min((unsigned)__builtin_amdgcn_readfirstlane(tb[j]), (unsigned)(a.npool - 1));
      const char* base = (const char*)(c_v[j] ? a.pv : a.pk) + (size_t)blk * blk_stride;
      lds_dma16_sbase(base, c_src[j], lds_addr(&smem[buf][(wave + j * W) * 1024]));
    }
  };

  float m = -INFINITY, lsum = 0.f;          // fp32 caches: running max, sum
  float mref = -FLT_MAX, thr = -INFINITY, lsr = 0.f;   // 16-bit caches (lsum shared)
  f32x4 o[DT16];
#pragma unroll
  for (int i = 0; i < DT16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  // lane-constant parts of the LDS read addresses
  const int kt_row = lane & 15;                               // K: token row of this lane
  const int vt_row = 4 * (lane >> 4) + ((lane & 15) >> 2);    // V^T: token row (16-bit types)
  const int vt_half = 8 * (lane & 1);
  const int vt_pair = (lane & 3) >> 1;

  // S^T of one block into s4 (16 tokens x 16 queries)
  auto scores = [&](const char* kb) {
    f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
    if constexpr (DT == kF32) {
      const char* krow = kb + kt_row * ROW_B + 4 * (lane >> 4);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const float kv = *reinterpret_cast<const float*>(krow + ((ks ^ swz(kt_row)) << 4));
        s4 = __builtin_amdgcn_mfma_f32_16x16x4f32(kv, qf32[ks], s4, 0, 0, 0);
      }
    } else {
      const char* krow = kb + kt_row * ROW_B;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 kv = *reinterpret_cast<const u32x4*>(krow + (((4 * ks + (lane >> 4)) ^ swz(kt_row)) << 4));
        s4 = Mfma<DT>::qk(kv, qf16[ks], s4);
      }
    }
    return s4;
  };
  // masked, scaled logits of the lane's 4 tokens of block `blk` (chunk-relative)
  const int lim = CAUSAL ? (q_ok ? tl.lim[qi] : -1) : 0;
  auto logits = [&](const f32x4& s4, int blk, float* s) {
    const int tok_base = (b0 + blk) * kBlock + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool vis = (tok_base + i < t1) && (!CAUSAL || tok_base + i <= lim);
      s[i] = vis ? s4[i] * a.scale_log2 : -INFINITY;
    }
  };
  // online-softmax update with n logits per lane; returns the probabilities
  auto update = [&](float* s, float* p, int n) {
    float bm = s[0];
    for (int i = 1; i < n; ++i) bm = fmaxf(bm, s[i]);
    bm = max_xor32(max_xor16(bm));
    const float mn = fmaxf(m, bm);                   // -inf only for a causal row that sees nothing yet
    const float mref = (CAUSAL && mn == -INFINITY) ? 0.f : mn;
    const float alpha = fast_exp2(m - mref);
    float ps = 0.f;
    for (int i = 0; i < n; ++i) { p[i] = fast_exp2(s[i] - mref); ps += p[i]; }
    lsum = lsum * alpha + ps;
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) o[dt] *= alpha;
    m = mn;
  };

  // 16-bit caches: mask the logits of tokens past the range end (and, for a
  // causal tile, past each row's limit); x[i] holds token tok0 + 16 (i / 4) +
  // 4 (lane / 16) + i % 4
  auto mask16 = [&](float* x, int n, int tok0) {
    const int tlane = tok0 + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < n; ++i) {
      const int tok = tlane + (i >> 2) * kBlock + (i & 3);
      const bool vis = tok < t1 && (!CAUSAL || tok <= lim);
      x[i] = vis ? x[i] : -INFINITY;
    }
  };
  // lazy reference test (rare branch: move the reference, rescale the state),
  // then the probabilities and their unrounded sum
  auto lazy16 = [&](const float* x, float* p, int n) {
    float lm = x[0];
#pragma unroll
    for (int i = 1; i < n; ++i) lm = fmaxf(lm, x[i]);
    if (__builtin_amdgcn_ballot_w64(lm > thr) != 0) {
      const float mn = fmaxf(mref, max_xor32(max_xor16(lm)) * scale);
      const float alpha = fast_exp2(mref - mn);      // 0 after -FLT_MAX, 1 if unmoved
      lsum *= alpha;
      lsr *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT16; ++dt) o[dt] *= alpha;
      mref = mn;
      thr = (mn + kLazy) * inv_scale;
    }
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < n; ++i) { p[i] = fast_exp2(__builtin_fmaf(x[i], scale, -mref)); ps += p[i]; }
    lsum += ps;
  };

  auto compute = [&](int st, int buf) {
    const int nbl = min(STAGE_BLK, nb - st * STAGE_BLK);
    int bl = 0;
    if constexpr (DT != kF32) {
      // two blocks per softmax update and per k = 32 PV product
      for (; bl + 1 < nbl; bl += 2) {
        const char* kbA = &smem[buf][bl * BLK_B];
        const char* vbA = &smem[buf][kTensorStage + bl * BLK_B];
        const int tok0 = (b0 + st * STAGE_BLK + bl) * kBlock;
        const char* vrowA = vbA + vt_row * ROW_B + vt_half;
        // V^T fragments of the first kVtAhead d tiles, read before the scores
        // so that their LDS round trip overlaps the QK^T products and softmax
        unsigned long long vt[kVtAhead > 0 ? kVtAhead : 1][2];
#pragma unroll
        for (int dt = 0; dt < kVtAhead; ++dt) {
          const int off = ((2 * dt + vt_pair) ^ swz(vt_row)) << 4;
          vt[dt][0] = Mfma<DT>::tr_read(vrowA + off);
          vt[dt][1] = Mfma<DT>::tr_read(vrowA + BLK_B + off);
        }
        const f32x4 sA = scores(kbA);
        const f32x4 sB = scores(kbA + BLK_B);
        float x[8], p[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { x[i] = sA[i]; x[4 + i] = sB[i]; }
        if (CAUSAL || tok0 + 2 * kBlock > t1) mask16(x, 8, tok0);
        lazy16(x, p, 8);
        const unsigned long long pA = Mfma<DT>::pack_p(p), pB = Mfma<DT>::pack_p(p + 4);
        lsr = Mfma<DT>::sum_p(pB, Mfma<DT>::sum_p(pA, lsr));
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) {
          if (dt < kVtAhead) {
            const int r = dt < kVtAhead ? dt : 0;      // in range in the untaken branch too
            o[dt] = Mfma<DT>::pv2(vt[r][0], vt[r][1], pA, pB, o[dt]);
          } else {
            const int off = ((2 * dt + vt_pair) ^ swz(vt_row)) << 4;
            o[dt] = Mfma<DT>::pv2(Mfma<DT>::tr_read(vrowA + off), Mfma<DT>::tr_read(vrowA + BLK_B + off),
                                  pA, pB, o[dt]);
          }
        }
      }
    }
    for (; bl < nbl; ++bl) {
      const char* kb = &smem[buf][bl * BLK_B];
      const char* vb = &smem[buf][kTensorStage + bl * BLK_B];
      float s[4], p[4];
      if constexpr (DT == kF32) {
        logits(scores(kb), st * STAGE_BLK + bl, s);
        update(s, p, 4);
      } else {
        const f32x4 s4 = scores(kb);
        const int tok0 = (b0 + st * STAGE_BLK + bl) * kBlock;
#pragma unroll
        for (int i = 0; i < 4; ++i) s[i] = s4[i];
        if (CAUSAL || tok0 + kBlock > t1) mask16(s, 4, tok0);
        lazy16(s, p, 4);
      }
      if constexpr (DT == kF32) {
        // O^T[d][q] += V^T[d][t] P^T[t][q] with k index kk <-> token 4*kk + kt
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const int row = 4 * (lane >> 4) + kt;
          const char* vrow = vb + row * ROW_B + 4 * (lane & 3);
#pragma unroll
          for (int dt = 0; dt < DT16; ++dt) {
            const float vv = *reinterpret_cast<const float*>(vrow + (((4 * dt + ((lane & 15) >> 2)) ^ swz(row)) << 4));
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vv, p[kt], o[dt], 0, 0, 0);
          }
        }
      } else {
        const unsigned long long pb = Mfma<DT>::pack_p(p);
        lsr = Mfma<DT>::sum_p(pb, lsr);
        // lane k of 16-lane group G reads V[4G + k/4][dt*16 + 4*(k%4) .. +3]
        const char* vrow = vb + vt_row * ROW_B + vt_half;
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt)
          o[dt] = Mfma<DT>::pv(Mfma<DT>::tr_read(vrow + (((2 * dt + vt_pair) ^ swz(vt_row)) << 4)), pb, o[dt]);
      }
    }
  };

  // Ring of RING stage buffers, RING - 1 stages in flight while one is
  // computed.  At iteration st the wave's loads for st are the oldest outstanding ones,
  // so vmcnt((RING - 2) * PER_WAVE) means st has landed; the barrier then
  // makes every wave's part visible and guarantees every wave is done with
  // buffer (st - 1) % RING, which stage st + RING - 1 overwrites.
  static_assert((RING - 2) * PER_WAVE < 64, "vmcnt range");
#pragma unroll
  for (int i = 0; i < RING - 1; ++i) {
    table(min(i, last));
    issue(i);
  }
  table(min(RING - 1, last));
  // The compiler tracks the query loads but not the direct-to-LDS loads; make
  // it wait for the queries here, once, instead of at their first use inside
  // the loop (where its wait would also drain the stage ring every iteration).
  // This wait covers the prologue stages too: one round trip for both.
  if constexpr (DT == kF32) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : : "v"(qf32[ks]));
  } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : : "v"(qf16[ks]));
  }
  wait_vmcnt<0>();
  for (int st = 0; st < nstages; ++st) {
    const int buf = st % RING;
    wait_vmcnt<(RING - 2) * PER_WAVE>();
    lds_sync();
    if (st == last && (t1 & (kBlock - 1)) != 0) {
      // zero the V rows past the end of the chunk's last, partly filled block
      // (their probabilities are 0, but 0 * NaN would poison the product)
      const int bl = (nb - 1) - st * STAGE_BLK;
      const int first = t1 & (kBlock - 1);
      char* vb = &smem[buf][kTensorStage + bl * BLK_B];
      for (int i = tid; i < (kBlock - first) * GRAN; i += W * 64) {
        const int t = first + i / GRAN;
        *reinterpret_cast<u32x4*>(vb + t * ROW_B + ((i % GRAN) << 4)) = u32x4{0u, 0u, 0u, 0u};
      }
      lds_sync();
    }
    issue((st + RING - 1) % RING);
    table(min(st + RING, last));
    if (has_q) compute(st, buf);
  }
  wait_vmcnt<0>();   // the re-read stages issued by the last iterations

  if (!has_q) return;
  float lt = sum_xor16(lsum);
  lt = sum_xor32(lt);
  // the output is normalised by the sum of the weights the products used
  float lw = lt;
  if constexpr (DT != kF32) lw = sum_xor32(sum_xor16(lsr));
  const float mfin = DT == kF32 ? m : mref;
  if (q_ok) {
    const size_t slot = (size_t)(rq * H + h) * a.seg + a.slot;
    const float inv = (CAUSAL && lw == 0.f) ? 0.f : 1.f / lw;
    float* dst = a.o_part + slot * D + 4 * (lane >> 4);
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) *reinterpret_cast<f32x4*>(dst + dt * 16) = o[dt] * inv;
    if (lane < 16) a.lse_part[slot] = (CAUSAL && lt == 0.f) ? -INFINITY : mfin + fast_log2(lt);
  }
}

}  // namespace parrot
