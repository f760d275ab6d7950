// Prefill of forked contexts: the new rows of each request against its
// group's shared prefix (and the prefixes of the group's ancestors) and,
// causally, against its own tokens (Section 7: Fill with a parent context
// fills only the new tokens on top of the parent's KV cache).
//
// Split plan: the work splits the same way as decode, with many query rows
// per request:
//
//   prefix items (g, chunk c, head h, row tile qt): the rows of every request
//     that reads g's prefix, stacked in request order, one tile of rows at a
//     time, against chunk c of the prefix.  No mask: every prefix token
//     precedes every row.  The chunk is streamed once per tile of rows drawn
//     from all of the group's members (once for the whole group when its rows
//     fit one tile).
//   own items (r, chunk k, head h, row tile t): one tile of consecutive rows
//     of request r against its own tokens [k*co, (k+1)*co), each row cut
//     after its own position.
//
// Tiles hold 128 rows on fp16 / bf16 caches (wide_tile) and 64 on fp32 caches
// (decode's tile_core); both run QK^T and PV on MFMA over LDS-staged 16-token
// blocks and write one partial result per (row, head, item); the decode merge
// kernel then combines them per row, reading the row descriptors that the
// first workgroups write.
//
// Single pass (16-bit caches, flat groups, prefix and own tokens within one
// chunk each; the host decides): no partial results and no merge.  A group
// tile (g, head h, row tile qt) takes the same stacked rows as a prefix item,
// sees the whole prefix and then, run by run, each of its requests' own
// tokens up to its rows' positions, and writes the rows' output; tiles of
// ungrouped requests see only their own tokens.
//
// Work items are placed per XCD (workgroup b runs on XCD b mod 8): XCD x takes
// every item of heads x, x + 8, ..., one head after another (split plan: a
// head's own items after the next head's prefix items), prefix items before
// own items and row tiles fastest.  Each XCD then holds the same share of the
// work, and the workgroups that run together on it read the same head's key
// chunk, which stays in that XCD's L2.
#include "prefill_args.h"
#include "prefill_tile.h"

namespace parrot {

constexpr int kPrefillMaxBlocks = 512;                       // chunk <= 8192 tokens
// query rows per tile: the wide tile for 16-bit caches, decode's tile for fp32
template <int DT> constexpr int kTileRows = DT == kF32 ? kPrefixWaves * 16 : kWideRows;
template <int DT> constexpr int kTileRing = DT == kF32 ? prefix_detail::kRing : kWideRing;
constexpr int kPrefillTileLds = tile_lds_bytes(kPrefillMaxBlocks, kWideRows, kWideRing);
// single-pass tiles also keep their runs of rows per request after the tile's view
constexpr int kPrefillLds = kPrefillTileLds + kWideRows * (int)sizeof(int2);
constexpr int kPrefillLdsF32 = tile_lds_bytes(kPrefillMaxBlocks);

// The one LDS view of a prefill tile: its stage ring, rows, block table and
// limits laid out for the tile core that DT selects (both item kinds use it).
template <int DT>
PARROT_DEV TileLds prefill_lds(char* lds) {
  return TileLds(lds, kPrefillMaxBlocks, kTileRows<DT>, kTileRing<DT>);
}
// The single-pass tile's runs: (request, first tile row) per run of rows.
PARROT_DEV int2* prefill_runs(char* lds) { return reinterpret_cast<int2*>(lds + kPrefillTileLds); }
static_assert(kPrefillTileLds % 8 == 0, "runs are 8-byte aligned");
constexpr int kXcds = 8;                                     // workgroups go round-robin over XCDs


struct ReqRows { int start, count, S; };

// Rows of request r, clamped so that every row index stays in [0, T) and a
// request has at most min(S_r, max_q) rows (the launch covers no more).
PARROT_DEV ReqRows req_rows(const PrefillArgs& a, int r) {
  const int S = clampi(a.slen[r], 0, a.max_s);
  const int start = clampi(a.qoff[r], 0, a.T);
  const long n = (long)a.qoff[r + 1] - (long)a.qoff[r];
  const int cap = min(min(S, a.max_q), a.T - start);
  return {start, (int)(n < 0 ? 0 : (n > cap ? cap : n)), S};
}

// Row descriptor for the merge: own-chunk slots and the prefix chunks per
// level of the row's chain (the decode descriptor, per row).  Rows that no
// request holds get an empty descriptor (output 0, lse -inf).
PARROT_DEV void write_row_meta(const PrefillArgs& a, int t) {
  int lo = 0, hi = a.R - 1, r = -1;          // last request with qoff[r] <= t
  while (lo <= hi) {
    const int mid = (lo + hi) >> 1;
    if (a.qoff[mid] <= t) { r = mid; lo = mid + 1; } else { hi = mid - 1; }
  }
  int4 m = {0, 0, 0, 0};
  if (r >= 0) {
    const ReqRows rw = req_rows(a, r);
    if (t >= rw.start && t < rw.start + rw.count) {
      const int pos = rw.S - rw.count + (t - rw.start);
      int np[kMaxDepth] = {0, 0, 0, 0};
      int chain[kMaxDepth];
      int nlev = 0;
      int x = a.gid[r];
      while (x >= 0 && x < a.NG && nlev < a.depth) {
        chain[nlev++] = x;
        x = a.parents ? a.parents[x] : -1;
      }
      // at most seg_p chunks per level (none when no prefix items run, as
      // when max_group_rows is 0), so the merge never reads past the row's slots
#pragma unroll
      for (int i = 0; i < kMaxDepth; ++i)
        if (i < nlev) np[nlev - 1 - i] = min((clampi(a.plen[chain[i]], 0, a.max_p) + a.cp - 1) / a.cp, a.seg_p);
      m = int4{pos / a.co + 1, nlev, (int)((unsigned)np[0] | ((unsigned)np[1] << 16)),
               (int)((unsigned)np[2] | ((unsigned)np[3] << 16))};
    }
  }
  *reinterpret_cast<int4*>(a.merge_meta + kMetaInts * t) = m;
}

// Prefix item: chunk c of group g's prefix for row tile qt of the rows that
// read it, head h.
template <int DT, int D>
__device__ __forceinline__ void prefill_prefix_item(const PrefillArgs& a, char* lds, int h, int item) {
  const int qt = item % a.qtiles_p; item /= a.qtiles_p;
  const int c = item % a.seg_p;
  const int g = item / a.seg_p;
  if (g >= a.NG) return;
  const int P = clampi(a.plen[g], 0, a.max_p);
  const int t0 = c * a.cp;
  if (t0 >= P) return;
  const int t1 = min(P, t0 + a.cp);
  int lvl = 0;                                         // ancestors of g (< depth)
  if (a.parents) {
    int x = a.parents[g];
    while (x >= 0 && x < a.NG && lvl < a.depth - 1) { ++lvl; x = a.parents[x]; }
  }
  constexpr int ROWS = kTileRows<DT>;
  const TileLds tl = prefill_lds<DT>(lds);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const long qbase = (long)qt * ROWS;
  const int b0 = t0 / kBlock, nb = (t1 - t0 + kBlock - 1) / kBlock;
  if (wave == 0) {
    // rows of the requests that read g's prefix, in request order; this tile
    // takes rows [qbase, qbase + ROWS) of that list
    long base = 0;
    for (int b = 0; b < a.R && base < qbase + ROWS; b += kWave) {
      const int r = b + lane;
      bool reads = false;
      if (r < a.R) {
        int x = a.gid[r];
        for (int d = 0; d < a.depth && x >= 0 && x < a.NG; ++d) {
          if (x == g) { reads = true; break; }
          x = a.parents ? a.parents[x] : -1;
        }
      }
      ReqRows rw = {0, 0, 0};
      if (reads) rw = req_rows(a, r);
      long inc = rw.count;                             // inclusive scan over lanes
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const long v = __shfl_up(inc, d);
        if (lane >= d) inc += v;
      }
      const long first = base + inc - rw.count;
      const long lo = first > qbase ? first : qbase;
      const long hi = min(first + rw.count, qbase + ROWS);
      for (long x = lo; x < hi; ++x) tl.rows[x - qbase] = rw.start + (int)(x - first);
      base += __shfl(inc, kWave - 1);
    }
    if (lane == 0) *tl.count = (int)(base - qbase > ROWS ? ROWS : (base - qbase < 0 ? 0 : base - qbase));
  } else if (wave == 1) {
    const int* tbl = a.ptab + (long)g * a.pstride;
    for (int i = lane; i < nb; i += kWave) tl.tbl[i] = clampi(tbl[b0 + i], 0, a.npblk - 1);
  }
  __syncthreads();
  const int nq = *tl.count;
  if (nq <= 0) return;                                 // uniform over the workgroup
  TileJob j;
  j.q = a.q; j.pk = a.pk; j.pv = a.pv; j.npool = a.npblk; j.H = a.H; j.h = h;
  j.t0 = t0; j.t1 = t1; j.o_part = a.o_part; j.lse_part = a.lse_part;
  j.seg = a.seg; j.slot = lvl * a.seg_p + c; j.scale_log2 = a.scale_log2; j.lim_min = 0;
  if constexpr (DT == kF32)
    tile_core<DT, D, false>(j, tl, nq);
  else
    wide_tile<DT, D, false>(j, tl, nq);
}

// Own item: own tokens [k*co, (k+1)*co) of request r for its row tile t,
// head h; row i of the tile sees own tokens up to its position.
template <int DT, int D>
__device__ __forceinline__ void prefill_own_item(const PrefillArgs& a, char* lds, int h, int item) {
  const int t = item % a.qtiles_o; item /= a.qtiles_o;
  const int k = item % a.seg_s;
  const int r = item / a.seg_s;
  if (r >= a.R) return;
  constexpr int ROWS = kTileRows<DT>;
  const ReqRows rw = req_rows(a, r);
  const int row0 = t * ROWS;
  if (row0 >= rw.count) return;
  const int nq = min(ROWS, rw.count - row0);
  const int pos0 = rw.S - rw.count + row0;             // position of the tile's first row
  const int t0 = k * a.co;
  if (t0 > pos0 + nq - 1) return;
  const int t1 = min(min(rw.S, t0 + a.co), pos0 + nq);
  const TileLds tl = prefill_lds<DT>(lds);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b0 = t0 / kBlock, nb = (t1 - t0 + kBlock - 1) / kBlock;
  if (wave == 0) {
    for (int i = lane; i < nq; i += kWave) {
      tl.rows[i] = rw.start + row0 + i;
      tl.lim[i] = pos0 + i;
    }
  } else if (wave == 1) {
    const int* tbl = a.stab + (long)r * a.sstride;
    for (int i = lane; i < nb; i += kWave) tl.tbl[i] = clampi(tbl[b0 + i], 0, a.nsblk - 1);
  }
  __syncthreads();
  TileJob j;
  j.q = a.q; j.pk = a.sk; j.pv = a.sv; j.npool = a.nsblk; j.H = a.H; j.h = h;
  j.t0 = t0; j.t1 = t1; j.o_part = a.o_part; j.lse_part = a.lse_part;
  j.seg = a.seg; j.slot = a.seg_pre + k; j.scale_log2 = a.scale_log2; j.lim_min = pos0;
  if constexpr (DT == kF32)
    tile_core<DT, D, true>(j, tl, nq);
  else
    wide_tile<DT, D, true>(j, tl, nq);
}

// Single-pass group tile (g, row tile qt, head h) of flat groups: rows of the
// requests in group g, stacked as for the prefix items, against the whole
// prefix and then each run's own tokens; writes the rows' output.
template <int DT, int D>
__device__ __forceinline__ void prefill_single_group_item(const PrefillArgs& a, char* lds, int h,
                                                          int item) {
  const int qt = item % a.qtiles_p;
  const int g = item / a.qtiles_p;
  if (g >= a.NG) return;
  const int P = clampi(a.plen[g], 0, a.max_p);
  constexpr int ROWS = kWideRows;
  const TileLds tl = prefill_lds<DT>(lds);
  int2* runs = prefill_runs(lds);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const long qbase = (long)qt * ROWS;
  const int nb = (P + kBlock - 1) / kBlock;
  if (wave == 0) {
    // rows of g's members in request order: this tile takes rows [qbase,
    // qbase + ROWS) of that list, with their own positions and one run per
    // request that has rows in it
    long base = 0;
    int nruns = 0;
    for (int b = 0; b < a.R && base < qbase + ROWS; b += kWave) {
      const int r = b + lane;
      ReqRows rw = {0, 0, 0};
      if (r < a.R && a.gid[r] == g) rw = req_rows(a, r);
      long inc = rw.count;                             // inclusive scan over lanes
#pragma unroll
      for (int d = 1; d < kWave; d <<= 1) {
        const long v = __shfl_up(inc, d);
        if (lane >= d) inc += v;
      }
      const long first = base + inc - rw.count;
      const long lo = first > qbase ? first : qbase;
      const long hi = min(first + rw.count, qbase + ROWS);
      for (long x = lo; x < hi; ++x) {
        tl.rows[x - qbase] = rw.start + (int)(x - first);
        tl.lim[x - qbase] = rw.S - rw.count + (int)(x - first);
      }
      const unsigned long long has = __builtin_amdgcn_ballot_w64(hi > lo);
      if (hi > lo) {
        const int k = nruns + __builtin_popcountll(has & ((1ull << lane) - 1ull));
        runs[k] = int2{r, (int)(lo - qbase)};
      }
      nruns += __builtin_popcountll(has);
      base += __shfl(inc, kWave - 1);
    }
    if (lane == 0) {
      tl.count[0] = (int)(base - qbase > ROWS ? ROWS : (base - qbase < 0 ? 0 : base - qbase));
      tl.count[1] = nruns;
    }
  } else if (wave == 1) {
    const int* tbl = a.ptab + (long)g * a.pstride;
    for (int i = lane; i < nb; i += kWave) tl.tbl[i] = clampi(tbl[i], 0, a.npblk - 1);
  }
  __syncthreads();
  const int nq = tl.count[0];
  if (nq <= 0) return;                                 // uniform over the workgroup
  TileJob j;
  j.q = a.q; j.pk = a.pk; j.pv = a.pv; j.npool = a.npblk; j.H = a.H; j.h = h;
  j.t0 = 0; j.t1 = P; j.o_part = nullptr; j.lse_part = nullptr;
  j.seg = 0; j.slot = 0; j.scale_log2 = a.scale_log2; j.lim_min = 0;
  const WideSingle sg{a.sk, a.sv, a.stab, a.sstride, a.nsblk, runs, tl.count[1], a.out, a.lse};
  wide_tile_single<DT, D>(j, tl, nq, sg);
}

// Single-pass own tile (request r, row tile t, head h) of a request outside
// the groups: its rows against its own tokens, causal; writes their output.
// Grouped requests' rows belong to their group's tiles.
template <int DT, int D>
__device__ __forceinline__ void prefill_single_own_item(const PrefillArgs& a, char* lds, int h,
                                                        int item) {
  const int t = item % a.qtiles_o;
  const int r = item / a.qtiles_o;
  if (r >= a.R) return;
  const int g = a.gid[r];
  if (g >= 0 && g < a.NG) return;
  constexpr int ROWS = kWideRows;
  const ReqRows rw = req_rows(a, r);
  const int row0 = t * ROWS;
  if (row0 >= rw.count) return;
  const int nq = min(ROWS, rw.count - row0);
  const int pos0 = rw.S - rw.count + row0;             // position of the tile's first row
  const TileLds tl = prefill_lds<DT>(lds);
  int2* runs = prefill_runs(lds);
  const int tid = threadIdx.x;
  if (tid < nq) {
    tl.rows[tid] = rw.start + row0 + tid;
    tl.lim[tid] = pos0 + tid;
  }
  if (tid == 0) runs[0] = int2{r, 0};
  __syncthreads();
  TileJob j;
  j.q = a.q; j.pk = a.sk; j.pv = a.sv; j.npool = a.nsblk; j.H = a.H; j.h = h;
  j.t0 = 0; j.t1 = 0; j.o_part = nullptr; j.lse_part = nullptr;  // no prefix range
  j.seg = 0; j.slot = 0; j.scale_log2 = a.scale_log2; j.lim_min = 0;
  const WideSingle sg{a.sk, a.sv, a.stab, a.sstride, a.nsblk, runs, 1, a.out, a.lse};
  wide_tile_single<DT, D>(j, tl, nq, sg);
}

// Occupancy: three waves per SIMD (three workgroups per CU: 3 x 51 KiB of
// LDS, at most 168 registers per lane), for either tile core.
// SINGLE: single-pass items (16-bit caches); otherwise prefix and own items
// with partial results and row descriptors for the merge.
template <int DT, int D, bool SINGLE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
void k_prefill(PrefillArgs a) {
  static_assert(!SINGLE || DT != kF32, "single-pass tiles are the 16-bit wide tiles");
  __shared__ __attribute__((aligned(1024))) char lds[DT == kF32 ? kPrefillLdsF32 : kPrefillLds];
  static_assert(sizeof(lds) >= tile_lds_bytes(kPrefillMaxBlocks, kTileRows<DT>, kTileRing<DT>),
                "the LDS array holds the tile's layout");
  const int bid = blockIdx.x;
  if (!SINGLE && bid < a.meta_wgs) {
    const int t = bid * 256 + (int)threadIdx.x;
    if (t < a.T) write_row_meta(a, t);
  }
  // XCD x takes heads x, x + 8, ... (J of them); l is its workgroup index
  const int x = bid % kXcds, l = bid / kXcds;
  if constexpr (SINGLE) {
    // head after head: head x + 8 (l / per), item l % per of that head
    const int per = a.n_pre + a.n_own;                 // items per head
    const int j = l / per, item = l % per;
    const int h = x + kXcds * j;
    if (h >= a.H) return;
    if (item < a.n_pre)
      prefill_single_group_item<DT, D>(a, lds, h, item);
    else
      prefill_single_own_item<DT, D>(a, lds, h, item - a.n_pre);
  } else {
    // prefix items of head 0, then of head 1 with the own items of head 0,
    // and so on: the own-token streams (bandwidth-bound) of one head run
    // beside the prefix tiles (MFMA-bound) of the next, and each head's
    // prefix items still run together (its prefix chunk stays in the L2)
    const int J = (a.H - x + kXcds - 1) / kXcds;
    int rem = l, j = -1, own = 0;
    for (int k = 0; k <= J; ++k) {
      if (k < J) {
        if (rem < a.n_pre) { j = k; break; }
        rem -= a.n_pre;
      }
      if (k >= 1) {
        if (rem < a.n_own) { j = k - 1; own = 1; break; }
        rem -= a.n_own;
      }
    }
    if (j < 0) return;
    const int h = x + kXcds * j;
    if (own)
      prefill_own_item<DT, D>(a, lds, h, rem);
    else
      prefill_prefix_item<DT, D>(a, lds, h, rem);
  }
}

template <int DT, int D>
static hipError_t launch_prefill_t(const PrefillArgs& a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const long items = (long)kXcds * ((a.H + kXcds - 1) / kXcds) * ((long)a.n_pre + a.n_own);
  const long blocks = items > a.meta_wgs ? items : a.meta_wgs;
  if (blocks <= 0) return hipSuccess;
  if constexpr (DT != kF32) {
    if (a.single) {
      hipExtLaunchKernelGGL((k_prefill<DT, D, true>), dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0, a);
      return hipGetLastError();
    }
  }
  hipExtLaunchKernelGGL((k_prefill<DT, D, false>), dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int D, hipStream_t s, hipEvent_t e0,
                          hipEvent_t e1) {
  if (a.R < 1 || a.T < 1 || a.H < 1 || a.seg_s < 1 || a.qtiles_o < 1)
    return hipErrorInvalidValue;
  if (a.cp % 32 != 0 || a.co % 32 != 0 || a.cp > kPrefillMaxBlocks * kBlock ||
      a.co > kPrefillMaxBlocks * kBlock || a.cp < 32 || a.co < 32)
    return hipErrorInvalidValue;
  if (a.single && (dtype == kF32 || a.parents || a.depth != 1 || !a.out || !a.lse))
    return hipErrorInvalidValue;
  if (a.meta_wgs != (a.single ? 0 : (a.T + 255) / 256) || a.n_pre < 0 || a.n_own < 1 ||
      (long)kXcds * ((a.H + kXcds - 1) / kXcds) * ((long)a.n_pre + a.n_own) > 0x7fffffffL)
    return hipErrorInvalidValue;
  switch (dtype * 1000 + D) {
    case kF32 * 1000 + 64: return launch_prefill_t<kF32, 64>(a, s, e0, e1);
    case kF32 * 1000 + 128: return launch_prefill_t<kF32, 128>(a, s, e0, e1);
    case kF16 * 1000 + 64: return launch_prefill_t<kF16, 64>(a, s, e0, e1);
    case kF16 * 1000 + 128: return launch_prefill_t<kF16, 128>(a, s, e0, e1);
    case kBF16 * 1000 + 64: return launch_prefill_t<kBF16, 64>(a, s, e0, e1);
    case kBF16 * 1000 + 128: return launch_prefill_t<kBF16, 128>(a, s, e0, e1);
  }
  return hipErrorInvalidValue;
}

}  // namespace parrot
