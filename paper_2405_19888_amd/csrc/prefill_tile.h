// The prefill query tile on MFMA (gfx950, fp16 / bf16 caches): 128 query rows
// against one range of a paged key sequence (a partial result per row), or
// against a prefix and then each row's own tokens (the output itself).
//
// Decode's prefix tile (tile_core) gives each wave 16 queries: enough to make
// a bandwidth-bound prefix stream cheap, but a prefill tile is bound by the
// matrix cores, and with 16 queries per wave the LDS reads of K and V, the
// online softmax and the per-stage bookkeeping cost more than the MFMAs.  Here
// each wave owns kWideSets (2) 16-query column sets that share every K and V
// fragment read from LDS, so one K read feeds kWideSets QK^T MFMAs and one
// transposed V read feeds kWideSets PV MFMAs.  The rest follows tile_core:
//   * K/V stages of 16 KiB (K and V of 32 tokens for D = 128, 64 for D = 64)
//     fill a ring of three LDS buffers through direct-to-LDS loads, two stages
//     ahead; the loads take a scalar base (pool + block * stride) and a
//     per-lane offset, and each stage's two block ids are read from LDS one
//     stage before they are needed, so issuing a stage waits on nothing;
//   * S^T = K Q^T and O^T += V^T P^T on v_mfma_f32_16x16x32_{f16,bf16} over
//     XOR-swizzled LDS rows (swz_wide below), V^T read with ds_read_b64_tr_b16;
//   * online softmax in fp32 with a lazily moved reference: the exponentials
//     use a reference max that is raised only when a row's max exceeds it by
//     more than 8 (log2 units), so the accumulators are rescaled a few times
//     per row instead of at every step, and probabilities stay below 2^8
//     (exact enough in fp16 / bf16, whose relative precision does not depend
//     on magnitude);
//   * masking (the end of the key range, the causal diagonal) only in the
//     stages that need it.
#pragma once

#include <cfloat>
#include <type_traits>

#include "prefill_shape.h"
#include "prefix_role.h"

namespace parrot {

// LDS row swizzle of the wide tile: 16-byte granule j of token row t sits at
// granule j ^ f(t).  The LDS serves 256 bytes per pass (64 banks), i.e. 16
// lanes of a 16-byte K read (16 token rows, one logical granule) or 32 lanes of
// an 8-byte transposed V read (8 token rows, two adjacent granules).  f spreads
// both over all 64 banks: for 256-byte rows (D = 128) f is a bijection of the
// 16 rows whose values differ above bit 0 within rows 0-7 and within rows
// 8-15; for 128-byte rows (D = 64) two rows share a 256-byte span, and f is a
// bijection within each row parity with the same property.
template <int GRAN>
PARROT_DEV int swz_wide(int t) {
  if constexpr (GRAN == 16) return ((t & 7) << 1) | ((t >> 3) & 1);
  else return (t & 6) | ((t >> 3) & 1);
}

constexpr int kWideRing = prefix_detail::kRing;   // stage buffers (two stages in flight)

// Tile kinds: one pass whose rows get a partial result each (a prefix chunk,
// or a causal chunk of one request's own tokens), or the single pass of a
// tile that sees the whole context of its rows and writes their output.
enum WideKind { kWidePrefix = 0, kWideOwn = 1, kWideSingle = 2 };

// The single-pass tile's own-token passes and its output.  The tile's rows
// come from one or more requests, in runs of consecutive rows; after the
// prefix range of the TileJob (none when it is empty), each run's rows see the
// own tokens of their request up to their positions (held in the LDS limit
// array), and every other row of the tile sees none of those tokens.
struct WideSingle {
  const void* sk; const void* sv;   // own-token pools
  const int* stab;                  // [requests][sstride] own-token block tables
  int sstride, nsblk;
  const int2* runs;                 // LDS [nruns]: (request, first tile row), row order
  int nruns;
  void* out; float* lse;            // [rows][H][D] dtype, [rows][H] natural-log lse
};

template <int DT>
PARROT_DEV void store4(void* p, const f32x4& v) {
  if constexpr (DT == kF16) {
    const f16x4 x = {(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
    *reinterpret_cast<f16x4*>(p) = x;
  } else {
    const bf16x4 x = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
    *reinterpret_cast<bf16x4*>(p) = x;
  }
}

// Two probabilities rounded to the cache type, packed as the PV MFMA reads them.
template <int DT>
PARROT_DEV unsigned pack2(float a, float b) {
  if constexpr (DT == kF16) {
    const f16x2 x = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(unsigned, x);
  } else {
    const bf16x2 x = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(unsigned, x);
  }
}

// acc plus the two packed probabilities of `w` (a dot2 with (1, 1) adds two
// packed halves into fp32 exactly).
template <int DT>
PARROT_DEV float add_pair(unsigned w, float acc) {
  if constexpr (DT == kF16) {
    const f16x2 one = {(_Float16)1.f, (_Float16)1.f};
    return __builtin_amdgcn_fdot2(as_f16x2(w), one, acc, false);
  } else {
    const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
    return __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(w), one, acc, false);
  }
}

// LDS reads at a byte address held in a register plus a compile-time offset
// (one instruction with an immediate offset).
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
PARROT_DEV u32x4 lds_read16(unsigned addr, int off) {
  return *reinterpret_cast<const lds_u32x4*>((prefix_detail::lds_char*)addr + off);
}
template <int DT>
PARROT_DEV unsigned long long lds_read_tr(unsigned addr, int off) {
  if constexpr (DT == kF16) {
    typedef __fp16 fp16x4_ __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) fp16x4_ lds_fp16x4;
    fp16x4_ v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_fp16x4*)((prefix_detail::lds_char*)addr + off));
    return __builtin_bit_cast(unsigned long long, v);
  } else {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)((prefix_detail::lds_char*)addr + off));
    return __builtin_bit_cast(unsigned long long, v);
  }
}

template <int DT, int D, int KIND>
__device__ __forceinline__ void wide_tile_impl(const TileJob& a, const TileLds& tl, int nq,
                                               const WideSingle& sg) {
  using namespace prefix_detail;
  static_assert(DT == kF16 || DT == kBF16, "16-bit caches only");
  constexpr int W = kPrefixWaves;
  constexpr int ROW_B = D * 2;
  constexpr int GRAN = ROW_B / 16;                    // 16-byte granules per row
  constexpr int BLK_B = kBlock * ROW_B;               // one block of one head
  constexpr int STAGE_BLK = kTensorStage / BLK_B;     // blocks per stage (2 or 4)
  constexpr int STAGE_TOK = STAGE_BLK * kBlock;
  constexpr int DT16 = D / 16;                        // 16-wide d tiles
  constexpr int KS = D / 32;                          // MFMA k-steps over D
  constexpr int PER_WAVE = kStageChunks / W;          // direct-to-LDS loads per wave per stage
  constexpr float kLazy = 8.f;                        // reference-max slack, log2 units
  static_assert(STAGE_BLK % 2 == 0 && (GRAN == 8 || GRAN == 16), "stages hold block pairs; swizzle fits a row");
  static_assert(STAGE_TOK % 32 == 0, "stages hold whole pairs");

  auto smem = tl.smem;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int H = a.H, h = a.h;
  // a negative scale flips the sign of q (exact), so that the raw logit max
  // times |scale| is the scaled max; a zero scale is taken as 1e-30, which
  // leaves every finite logit at 0 (to within 1e-22) and a masked one at -inf
  const float scale = fmaxf(fabsf(a.scale_log2), 1e-30f);
  const float inv_scale = 1.f / scale;   // any rounding of it only shifts the lazy threshold
  const unsigned qsign = a.scale_log2 < 0.f ? 0x80008000u : 0u;

  constexpr int NS = kWideSets;
  constexpr int WROWS = 16 * NS;                      // tile rows per wave
  int qi[NS], lim[NS];
  bool q_ok[NS];
  u32x4 qf[NS][KS];
#pragma unroll
  for (int c = 0; c < NS; ++c) {
    qi[c] = wave * WROWS + c * 16 + (lane & 15);
    q_ok[c] = qi[c] < nq;
    const int rq = q_ok[c] ? tl.rows[qi[c]] : 0;
    lim[c] = KIND == kWideOwn ? (q_ok[c] ? tl.lim[qi[c]] : -1) : 0;
    const char* qrow = (const char*)a.q + (size_t)(rq * H + h) * ROW_B;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 v = q_ok[c] ? ld16(qrow + (32 * ks + 8 * (lane >> 4)) * 2) : u32x4{0u, 0u, 0u, 0u};
      qf[c][ks] = v ^ u32x4{qsign, qsign, qsign, qsign};
    }
  }
  const bool has_q = wave * WROWS < nq;               // wave-uniform (the wave's last sets may
                                                      // be empty: they run on zero queries)

  // Direct-to-LDS stage loads: wave w issues chunks w, w + W, ... (1 KiB each);
  // lane l of a chunk fills LDS bytes [16 l, 16 l + 16) of it, i.e. block
  // c_bl of the stage, token row t, granule slot pos, from the global granule
  // pos ^ f(t) of that row.
  const size_t blk_stride = (size_t)H * BLK_B;
  int c_bl[PER_WAVE];
  unsigned c_off[PER_WAVE];
  bool c_v[PER_WAVE];
#pragma unroll
  for (int j = 0; j < PER_WAVE; ++j) {
    const int q = wave + j * W;
    const int off = (q % (kStageChunks / 2)) * 1024 + lane * 16;
    c_v[j] = q >= kStageChunks / 2;
    c_bl[j] = off / BLK_B;
    const int t = (off % BLK_B) / ROW_B;
    const int pos = (off % ROW_B) / 16;
    c_off[j] = (unsigned)(h * BLK_B + t * ROW_B + ((pos ^ swz_wide<GRAN>(t)) << 4));
  }

  // reference max of the exponentials, running sum of the probabilities, and
  // of the probabilities as rounded for the PV products.  Before a row's
  // first visible key its reference is -FLT_MAX, finite: every finite logit
  // moves it, and exp2(logit * scale - reference) needs no guard (a masked
  // logit, -inf, gives 0)
  float mref[NS], thr[NS], lsum[NS], lsr[NS];
  f32x4 o[NS][DT16];
#pragma unroll
  for (int c = 0; c < NS; ++c) {
    mref[c] = -FLT_MAX; lsum[c] = 0.f; lsr[c] = 0.f;
    thr[c] = -INFINITY;                 // a row's first finite logit moves its reference
  }
#pragma unroll
  for (int c = 0; c < NS; ++c)
#pragma unroll
    for (int i = 0; i < DT16; ++i) o[c][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int kt_row = lane & 15;                               // K: token row of this lane
  const int vt_row = 4 * (lane >> 4) + ((lane & 15) >> 2);    // V^T: token row
  const int vt_half = 8 * (lane & 1);
  const int vt_pair = (lane & 3) >> 1;
  // LDS byte addresses of this lane's K fragment (k-step ks) and V^T fragment
  // (d tile dt) in block 0 of ring buffer 0; buffers and blocks add
  // compile-time offsets.  Kept opaque, so the compiler holds one register
  // per fragment and every read is one instruction with an immediate offset.
  unsigned ka[KS], va[DT16];
  {
    const unsigned base = lds_addr(&smem[0][0]);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      ka[ks] = base + kt_row * ROW_B + (((4 * ks + (lane >> 4)) ^ swz_wide<GRAN>(kt_row)) << 4);
      asm volatile("" : "+v"(ka[ks]));
    }
#pragma unroll
    for (int dt = 0; dt < DT16; ++dt) {
      va[dt] = base + kTensorStage + vt_row * ROW_B + vt_half +
               (((2 * dt + vt_pair) ^ swz_wide<GRAN>(vt_row)) << 4);
      asm volatile("" : "+v"(va[dt]));
    }
  }

  // One pass over key tokens [t0, t1) (t0 a multiple of 16) of the pools
  // pk / pv, whose block ids the LDS table holds from t0 / 16 on.  Causal
  // passes cut row c of each set after key lim[c]; keys before lim_min + 1
  // need no cut.  `active`: the wave has rows the pass serves (wave-uniform);
  // `cut_all`: the wave also holds rows the pass must not touch, so every
  // pair takes the masking path.
  auto pass = [&](auto causal_c, const void* pk, const void* pv, int npool, int t0, int t1,
                  int lim_min, bool active, bool cut_all) {
    constexpr bool CAUSAL = decltype(causal_c)::value;
    const int b0 = t0 / kBlock;
    const int nb = (t1 - t0 + kBlock - 1) / kBlock;
    const int nstages = (nb + STAGE_BLK - 1) / STAGE_BLK;
    const int last = nstages - 1;
    auto table = [&](int st, int* tb) {
#pragma unroll
      for (int j = 0; j < PER_WAVE; ++j) tb[j] = tl.tbl[min(st * STAGE_BLK + c_bl[j], nb - 1)];
    };
    auto issue = [&](const int* tb, int buf) {
#pragma unroll
      for (int j = 0; j < PER_WAVE; ++j) {
        // block ids are clamped when the table is filled; clamping again here
        // keeps every load inside the pool whatever the LDS table holds
        const unsigned blk = min((unsigned)__builtin_amdgcn_readfirstlane(tb[j]), (unsigned)(npool - 1));
        const char* base = (const char*)(c_v[j] ? pv : pk) + (size_t)blk * blk_stride;
        lds_dma16_sbase(base, c_off[j], lds_addr(&smem[buf][(wave + j * W) * 1024]));
      }
    };

    // one pair of blocks (32 tokens) of stage buffer `buf`, first block `bl`;
    // `tok0` is the pair's first key token; `masked` selects the masking path
    auto pair = [&](int buf, int bl, int tok0, bool masked) {
      const int kb = buf * kStageBytes + bl * BLK_B;       // K of the pair's first block
      // K fragments feed the QK^T MFMAs of both sets; the V^T fragments are
      // read next to their PV MFMAs, two d tiles (four reads) per wait, so each
      // LDS round trip is covered by four MFMAs instead of two.  Reading them
      // all ahead (or all K ahead, or the first V^T reads above the softmax)
      // needs more registers than three waves per SIMD leave: the compiler
      // spills, or the third wave is lost; either was slower (measured).
      u32x4 kf[2][KS];
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[b][ks] = lds_read16(ka[ks], kb + b * BLK_B);
      f32x4 s[NS][2];
#pragma unroll
      for (int c = 0; c < NS; ++c)
#pragma unroll
        for (int b = 0; b < 2; ++b) s[c][b] = f32x4{0.f, 0.f, 0.f, 0.f};
      // four accumulator chains, each MFMA four issues after the one it adds to
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int c = 0; c < NS; ++c) s[c][b] = Mfma<DT>::qk(kf[b][ks], qf[c][ks], s[c][b]);

      unsigned pw[NS][4];
#pragma unroll
      for (int c = 0; c < NS; ++c) {
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { x[i] = s[c][0][i]; x[4 + i] = s[c][1][i]; }
        if (masked) {
          // token tok0 + 4 (lane / 16) + 16 (i / 4) + i % 4 is visible below `bound`
          const int rel = (CAUSAL ? min(t1, lim[c] + 1) : t1) - tok0 - 4 * (lane >> 4);
#pragma unroll
          for (int i = 0; i < 8; ++i) x[i] = (i >> 2) * kBlock + (i & 3) < rel ? x[i] : -INFINITY;
        }
        // The row's reference only has to move when some lane's own logits
        // exceed it by more than kLazy, i.e. exceed thr = (mref + kLazy) /
        // scale in logit units: that test needs no cross-lane max, and the
        // cross-lane max is taken only in the (rare) branch that moves it.
        // (scale > 0: the scaled max of a masked lane stays -inf, no NaN)
        // (grouped as v_max3 takes them: four instructions for eight values)
        const float lm = fmaxf(fmaxf(fmaxf(fmaxf(x[0], x[1]), x[2]), fmaxf(fmaxf(x[3], x[4]), x[5])),
                               fmaxf(x[6], x[7]));
        if (__builtin_amdgcn_ballot_w64(lm > thr[c]) != 0) {
          const float mn = fmaxf(mref[c], max_xor32(max_xor16(lm)) * scale);
          const float alpha = fast_exp2(mref[c] - mn);      // 0 after -FLT_MAX, 1 if unmoved
          lsum[c] *= alpha;
          lsr[c] *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT16; ++dt) o[c][dt] *= alpha;
          mref[c] = mn;
          thr[c] = (mn + kLazy) * inv_scale;
        }
        float p[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) p[i] = fast_exp2(__builtin_fmaf(x[i], scale, -mref[c]));   // masked: 0
        lsum[c] += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
        // lsr: the probabilities as the PV MFMA reads them (rounded to the
        // cache type).  Dividing the products by this sum makes the output a
        // weighted mean of the values with exactly the weights the products
        // used, so the rounding of a dominant weight cancels (with the lazy
        // reference a dominant weight is rarely 1); the lse keeps the sum of
        // the unrounded probabilities.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pw[c][i] = pack2<DT>(p[2 * i], p[2 * i + 1]);
          lsr[c] = add_pair<DT>(pw[c][i], lsr[c]);
        }
      }
      const int vb = buf * kStageBytes + bl * BLK_B;       // V^T of the pair's first block
      static_assert(DT16 % 2 == 0, "d tiles are read in pairs");
#pragma unroll
      for (int dt = 0; dt < DT16; dt += 2) {
        unsigned long long vt[2][2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          vt[u][0] = lds_read_tr<DT>(va[dt + u], vb);
          vt[u][1] = lds_read_tr<DT>(va[dt + u], vb + BLK_B);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int c = 0; c < NS; ++c) {
            const unsigned long long b0 = pw[c][0] | ((unsigned long long)pw[c][1] << 32);
            const unsigned long long b1 = pw[c][2] | ((unsigned long long)pw[c][3] << 32);
            o[c][dt + u] = Mfma<DT>::pv2(vt[u][0], vt[u][1], b0, b1, o[c][dt + u]);
          }
      }
    };

    // Ring of kRing stage buffers, kRing - 1 stages in flight (see tile_core).
    int tb[PER_WAVE];
#pragma unroll
    for (int i = 0; i < kRing - 1; ++i) {
      table(min(i, last), tb);
      issue(tb, i);
    }
    table(min(kRing - 1, last), tb);
#pragma unroll
    for (int c = 0; c < NS; ++c)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) asm volatile("" : : "v"(qf[c][ks]));
    wait_vmcnt<0>();
    const int full_end = CAUSAL ? min(t1, lim_min + 1) : t1;   // keys before it need no mask
    // one stage; `bufc` carries the ring buffer as a constant, so that every LDS
    // address of the stage is a lane constant plus an immediate offset
    auto step = [&](int st, auto bufc) {
      constexpr int buf = decltype(bufc)::value;
      wait_vmcnt<(kRing - 2) * PER_WAVE>();
      lds_sync();
      if (st == last && (t1 & (kBlock - 1)) != 0) {
        // zero the V rows past the end of the range's last, partly filled block
        // (their probabilities are 0, but 0 * NaN would poison the product); when
        // that block opens a pair, the pair's second slot holds a second copy of
        // it (loads past the range re-read the last block): zero that one too
        const int bl = (nb - 1) - st * STAGE_BLK;
        const int first = t1 & (kBlock - 1);
        const int copies = (bl & 1) ? 1 : 2;
        const int per = (kBlock - first) * GRAN;
        for (int i = tid; i < copies * per; i += W * 64) {
          const int cp = i / per, k = i % per;
          char* vz = &smem[buf][kTensorStage + (bl + cp) * BLK_B];
          const int t = first + k / GRAN;
          *reinterpret_cast<u32x4*>(vz + t * ROW_B + ((k % GRAN) << 4)) = u32x4{0u, 0u, 0u, 0u};
        }
        lds_sync();
      }
      issue(tb, (st + kRing - 1) % kRing);
      table(min(st + kRing, last), tb);
      if (active) {
        const int tok_st = (b0 + st * STAGE_BLK) * kBlock;
        const int nbl = min(STAGE_BLK, nb - st * STAGE_BLK);
#pragma unroll
        for (int bl = 0; bl < STAGE_BLK; bl += 2) {
          if (bl < nbl) {
            // a pair whose second block lies past the range reads a zeroed or
            // stale buffer slot; its tokens are masked
            const int tok0 = tok_st + bl * kBlock;
            pair(buf, bl, tok0, cut_all || tok0 + 2 * kBlock > full_end);
          }
        }
      }
    };
    static_assert(kRing == 3, "the stage loop is unrolled over the ring");
    for (int st = 0; st < nstages; st += kRing) {
      step(st, std::integral_constant<int, 0>{});
      if (st + 1 < nstages) step(st + 1, std::integral_constant<int, 1>{});
      if (st + 2 < nstages) step(st + 2, std::integral_constant<int, 2>{});
    }
    wait_vmcnt<0>();   // the re-read stages issued by the last iterations
  };

  if constexpr (KIND == kWideSingle) {
    if (a.t1 > a.t0)
      pass(std::false_type{}, a.pk, a.pv, a.npool, a.t0, a.t1, 0, has_q, false);
    for (int k = 0; k < sg.nruns; ++k) {
      // run k: tile rows [lo, hi) of one request, own positions tl.lim[lo..hi)
      const int2 run = sg.runs[k];
      const int lo = run.y, hi = k + 1 < sg.nruns ? sg.runs[k + 1].y : nq;
      const int t1 = tl.lim[hi - 1] + 1;               // keys 0 .. the last row's position
      const int nb = (t1 + kBlock - 1) / kBlock;
      __syncthreads();                                 // the previous pass is done with the LDS
      const int* tbl = sg.stab + (long)run.x * sg.sstride;
      for (int i = tid; i < nb; i += W * 64) tl.tbl[i] = clampi(tbl[i], 0, sg.nsblk - 1);
#pragma unroll
      for (int c = 0; c < NS; ++c) lim[c] = q_ok[c] && qi[c] >= lo && qi[c] < hi ? tl.lim[qi[c]] : -1;
      __syncthreads();
      const int w0 = wave * WROWS, w1 = min(w0 + WROWS, nq);
      pass(std::true_type{}, sg.sk, sg.sv, sg.nsblk, 0, t1, tl.lim[lo], w0 < hi && w1 > lo,
           w0 < lo || w1 > hi);
    }
  } else {
    pass(std::integral_constant<bool, KIND == kWideOwn>{}, a.pk, a.pv, a.npool, a.t0, a.t1,
         a.lim_min, has_q, false);
  }

  if (!has_q) return;
#pragma unroll
  for (int c = 0; c < NS; ++c) {
    const float lt = sum_xor32(sum_xor16(lsum[c]));
    const float ltr = sum_xor32(sum_xor16(lsr[c]));
    if (q_ok[c]) {
      const int rq = tl.rows[qi[c]];
      const bool empty = lt == 0.f;                   // a causal row that saw no key
      const float inv = ltr > 0.f ? 1.f / ltr : 0.f;
      if constexpr (KIND == kWideSingle) {
        char* dst = (char*)sg.out + ((size_t)(rq * H + h) * D + 4 * (lane >> 4)) * 2;
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) store4<DT>(dst + dt * 32, o[c][dt] * inv);
        if (lane < 16) sg.lse[rq * H + h] = empty ? -INFINITY : (mref[c] + fast_log2(lt)) * kLn2;
      } else {
        const size_t slot = (size_t)(rq * H + h) * a.seg + a.slot;
        float* dst = a.o_part + slot * D + 4 * (lane >> 4);
#pragma unroll
        for (int dt = 0; dt < DT16; ++dt) *reinterpret_cast<f32x4*>(dst + dt * 16) = o[c][dt] * inv;
        if (lane < 16) a.lse_part[slot] = empty ? -INFINITY : mref[c] + fast_log2(lt);
      }
    }
  }
}

// One pass, partial results: a prefix chunk (CAUSAL false) or a causal chunk
// of one request's own tokens (row limits in the LDS limit array).
template <int DT, int D, bool CAUSAL>
__device__ __forceinline__ void wide_tile(const TileJob& a, const TileLds& tl, int nq) {
  wide_tile_impl<DT, D, CAUSAL ? kWideOwn : kWidePrefix>(a, tl, nq, WideSingle{});
}

// The whole context of the tile's rows: the TileJob's prefix range, then each
// run's own tokens; writes the output and lse of every row.
template <int DT, int D>
__device__ __forceinline__ void wide_tile_single(const TileJob& a, const TileLds& tl, int nq,
                                                 const WideSingle& sg) {
  wide_tile_impl<DT, D, kWideSingle>(a, tl, nq, sg);
}

}  // namespace parrot
