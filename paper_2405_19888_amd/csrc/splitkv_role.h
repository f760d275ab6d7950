// Split-KV decode attention over paged K/V: the non-shared tokens of every
// request (and, on the per-request path, its group's prefix as well).
//
// Work layout.  Each request owns a row of 16-token block columns (its own
// tokens; on the per-request path its group's prefix blocks first).  The rows
// are laid end to end into one flat column list, which is cut into equal runs
// of Q columns ("column groups").  Wave (g, h) reduces head h over column
// group g, so every wave streams the same number of bytes, and the H waves of
// a group walk the same physical blocks at the same time, reading all heads
// of a 16-token block (one contiguous region of H token blocks per tensor)
// together.  With HPW = 2 a wave reduces the adjacent heads h, h + 1 (H / 2
// waves per group): one contiguous piece of two heads per block and tensor.
// The role's grid is a fixed number of 4-wave workgroups per CU, so the
// per-CU load is even too.  A run
// may cross request boundaries: the wave then emits one partial result
// (normalised output and base-2 log-sum-exp) per (request, head) piece.
//
// Per block, a token row is D*elt bytes read as D*elt/16 lanes x 16 bytes, so
// each load instruction covers a contiguous 1 KiB of the block (coalesced
// 128-bit loads).  Each group of lanes that shares a token computes its slice
// of q.k, the slices are summed with DPP row operations, and every token group
// keeps its own online-softmax state; the groups are combined at the end of a
// piece.  One block is reduced while the next one's loads are in flight; the
// loop is unrolled by two with ping-pong registers and every load inside it is
// unconditional, so the compiler's memory-wait counts stay exact.
#pragma once

#include "common.h"

namespace parrot {

#ifndef PARROT_SPLITKV_STREAM_SCALAR_TABLE
#define PARROT_SPLITKV_STREAM_SCALAR_TABLE 0
#endif
// Streaming path: block-table entries as scalar loads (the next block's loads
// then issue while the current block is in flight) instead of vector loads.
constexpr bool kStreamScalarTable = PARROT_SPLITKV_STREAM_SCALAR_TABLE != 0;

// LDS bytes the split-KV role needs: six per-request arrays and a total.
constexpr int kSplitkvLds = (6 * kMaxRequests + 4) * 4;

// One workgroup of the split-KV role; `wg` is the role-local workgroup index
// and a.nwaves = 4 x (number of split-KV workgroups).
//
// Load policy, chosen per path by measurement on MI355X:
//  * STREAM (the shared path: every KV block is read once per call): K/V use
//    a nontemporal hint, and a block's table entry is an ordinary vector
//    load.  Waiting for that entry also waits for the previous block, so
//    about one block per wave is in flight; with the HBM already saturated
//    this runs slightly faster than keeping two blocks in flight.
//  * per-request path (each member re-reads its group's prefix, mostly from
//    the caches): cached K/V loads, and table entries as scalar loads so the
//    next block's K/V loads can issue while the current block is in flight.
//
// APPEND: the last own token of every request with S_r >= 1 is this decode
// step's token.  Its K/V are taken from k_new / v_new instead of the pool, and
// the lanes that hold it write it into the pool slot (stab[r][(S_r-1)/16],
// (S_r-1)%16) while the block is reduced, so the cache holds it for later
// steps.  The lane that writes a 16-byte piece is the lane that would have
// read it, and no other wave reads that (block, head) in the call.
template <int DT, int D, bool STREAM, bool APPEND = false, int HPW = 1>
__device__ __forceinline__ void splitkv_role(const SplitKVArgs& a, char* lds, int wg) {
  static_assert(HPW == 1 || HPW == 2, "one or two heads per wave");
  using E = Elem<DT>;
  constexpr int ROW_B = D * E::kBytes;        // bytes per token row
  constexpr int LPT = ROW_B / 16;             // lanes per token
  constexpr int TPI = kWave / LPT;            // tokens per load instruction
  constexpr int IPB = kBlock / TPI;           // load instructions per block
  constexpr int EPL = E::kPerLoad;            // elements per lane load
  constexpr int BLK_B = kBlock * ROW_B;
  static_assert(TPI * ROW_B == 1024, "one instruction covers 1 KiB");

  // per-request data: first flat block per head-sequence, blocks per
  // sequence, leading prefix blocks, group, prefix and own token counts
  int* s_excl = reinterpret_cast<int*>(lds);
  int* s_cnt = s_excl + kMaxRequests;
  int* s_nbp = s_cnt + kMaxRequests;
  int* s_g = s_nbp + kMaxRequests;
  int* s_plen = s_g + kMaxRequests;
  int* s_slen = s_plen + kMaxRequests;
  int& s_total = s_slen[kMaxRequests];

  const int lane = threadIdx.x & 63;
  const int wave_in_wg = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int R = a.R, H = a.H;

  if (wave_in_wg == 0) {
    // Every request's own length (and, on the per-request path, its group and
    // prefix length) is loaded before the scan: one memory round trip (two on
    // the per-request path) instead of one per 64 requests.  Addresses are
    // clamped into [0, R) so every load is unconditional.
    constexpr int kIt = kMaxRequests / kWave;
    int s_in[kIt], g_in[kIt], p_in[kIt];
#pragma unroll
    for (int i = 0; i < kIt; ++i) s_in[i] = a.slen[min(i * kWave + lane, R - 1)];
    if (a.with_prefix) {
#pragma unroll
      for (int i = 0; i < kIt; ++i) {
        const int g = a.gid[min(i * kWave + lane, R - 1)];
        g_in[i] = (g >= 0 && g < a.NG) ? g : -1;
      }
#pragma unroll
      for (int i = 0; i < kIt; ++i) p_in[i] = 0;
      if (a.NG > 0) {                        // no prefix lengths exist without groups
#pragma unroll
        for (int i = 0; i < kIt; ++i) p_in[i] = a.plen[g_in[i] >= 0 ? g_in[i] : 0];
      }
    }
    int carry = 0;
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
      const int base = i * kWave;
      if (base >= R) break;
      const int r = base + lane;
      const bool valid = r < R;
      const int S = valid ? clampi(s_in[i], 0, a.max_s) : 0;
      int g = -1, P = 0;
      if (a.with_prefix && valid) {
        g = g_in[i];
        P = g >= 0 ? clampi(p_in[i], 0, a.max_p) : 0;
      }
      const int nbp = (P + kBlock - 1) / kBlock;
      const int cnt = nbp + (S + kBlock - 1) / kBlock;
      int incl = cnt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
      }
      if (valid) {
        s_excl[r] = carry + incl - cnt; s_cnt[r] = cnt; s_nbp[r] = nbp;
        s_g[r] = g; s_plen[r] = P; s_slen[r] = S;
      }
      carry += __shfl(incl, kWave - 1);
    }
    if (lane == 0) s_total = carry;
  }
  __syncthreads();
  const int C = s_total;                                      // flat block columns
  const int HG = H / HPW;                                     // head groups (H % HPW == 0)
  const int G = a.nwaves / HG;                                // column groups
  const int Qg = (C + G - 1) / G;
  const int Q = Qg > a.min_q ? Qg : a.min_q;                  // columns per group
  if (wg == 0) {
    // Merge descriptor of each request: how many prefix-chunk slots (shared
    // path: chunks of its group's prefix) and how many split-KV pieces (the
    // column groups its run of columns touches) hold its partial results.
    // With nested groups, the request's chain is walked from its own group
    // outwards (at most depth groups); level l counts from the outermost.
    for (int rr = threadIdx.x; rr < R; rr += blockDim.x) {
      int np[kMaxDepth] = {0, 0, 0, 0};
      int nlev = 0;
      if (!a.with_prefix) {
        int chain[kMaxDepth];
        int x = a.gid[rr];
        while (x >= 0 && x < a.NG && nlev < a.depth) {
          chain[nlev++] = x;
          x = a.parents ? a.parents[x] : -1;
        }
#pragma unroll
        for (int i = 0; i < kMaxDepth; ++i)
          if (i < nlev) np[nlev - 1 - i] = (clampi(a.plen[chain[i]], 0, a.max_p) + a.cp - 1) / a.cp;
      }
      const int first = s_excl[rr], n = s_cnt[rr];
      const int ns = n > 0 ? (first + n - 1) / Q - first / Q + 1 : 0;
      *reinterpret_cast<int4*>(a.merge_meta + kMetaInts * rr) =
          make_int4(ns, nlev, (int)((unsigned)np[0] | ((unsigned)np[1] << 16)),
                    (int)((unsigned)np[2] | ((unsigned)np[3] << 16)));
    }
  }
  const int w = wg * kSkvWaves + wave_in_wg;
  const int grp = w / HG;
  const int h = (w % HG) * HPW;               // first head of the wave (HPW adjacent heads)
  const int c0 = grp * Q;
  if (grp >= G || c0 >= C) return;
  const int nblk_run = (C - c0 < Q) ? (C - c0) : Q;

  // the request holding column c0: the last request whose first column is <= c0
  int r = 0;
  for (int base = 0; base < R; base += kWave) {
    const int rr = base + lane;
    const unsigned long long mask = __ballot(rr < R && s_excl[rr] <= c0);
    const int n = __popcll(mask);
    if (n > 0) r = base + n - 1;
    if (n < kWave) break;
  }
  int cnt = s_cnt[r];
  if (cnt <= 0) return;                       // unreachable for consistent data
  int b = c0 - s_excl[r];

  const int sub = lane % LPT;                 // which 16-byte slice of the row
  const int tg = lane / LPT;                  // token group
  const size_t blk_stride = (size_t)H * BLK_B;

  // One fetched block: K and V slices of the wave's heads (adjacent in the
  // pool, so HPW * 4 KiB contiguous per tensor), the matching query slices,
  // and the metadata needed to reduce it and to close its piece.
  struct Blk {
    u32x4 k[HPW * IPB], v[HPW * IPB], q[HPW];
    int ntok;      // valid tokens in the block
    int seq;       // r * H + h (first head)
    int piece_end; // last block of its sequence
    int app;       // APPEND: piece (of a head's IPB loads) holding this lane's share of the new token, else -1
    size_t app_off;  // APPEND: pool byte offset of that piece for the first head
  };
  auto fetch = [&](Blk& B) {
    const int nbp = s_nbp[r];
    const char* kp;
    const char* vp;
    int entry, nblk, ntok;
    if (b < nbp) {
      entry = (STREAM && !kStreamScalarTable) ? a.ptab[(long)s_g[r] * a.pstride + b]
                                              : ld_uniform(a.ptab + (long)s_g[r] * a.pstride + b);
      kp = (const char*)a.pk; vp = (const char*)a.pv; nblk = a.npblk;
      ntok = s_plen[r] - b * kBlock;
    } else {
      const int bs = b - nbp;
      entry = (STREAM && !kStreamScalarTable) ? a.stab[(long)r * a.sstride + bs]
                                              : ld_uniform(a.stab + (long)r * a.sstride + bs);
      kp = (const char*)a.sk; vp = (const char*)a.sv; nblk = a.nsblk;
      ntok = s_slen[r] - bs * kBlock;
    }
    const int blk = clampi(entry, 0, nblk - 1);
    const size_t off = blk * blk_stride + (size_t)h * BLK_B + (size_t)lane * 16;
    if constexpr (APPEND) {
      // the own tokens' last block holds the new token at slot (S - 1) % 16
      B.app = -1;
      if (b >= nbp && b == cnt - 1) {
        const int last = (s_slen[r] - 1) % kBlock;
        if (tg == last % TPI) B.app = last / TPI;
      }
      B.app_off = off + (size_t)(B.app < 0 ? 0 : B.app) * 1024;   // first head's piece
#pragma unroll
      for (int i = 0; i < HPW * IPB; ++i) {
        // load i is piece i % IPB of head h + i / IPB; the new token's pieces
        // come from k_new / v_new
        const size_t noff = ((size_t)(r * H + h + i / IPB) * D) * E::kBytes + (size_t)sub * 16;
        const bool nw = (i % IPB) == B.app;
        const char* ks = nw ? (const char*)a.k_new + noff : kp + off + i * 1024;
        const char* vs = nw ? (const char*)a.v_new + noff : vp + off + i * 1024;
        B.k[i] = STREAM ? ld16_stream(ks) : ld16(ks);
        B.v[i] = STREAM ? ld16_stream(vs) : ld16(vs);
      }
    } else {
#pragma unroll
      for (int i = 0; i < HPW * IPB; ++i) {
        B.k[i] = STREAM ? ld16_stream(kp + off + i * 1024) : ld16(kp + off + i * 1024);
        B.v[i] = STREAM ? ld16_stream(vp + off + i * 1024) : ld16(vp + off + i * 1024);
      }
    }
#pragma unroll
    for (int u = 0; u < HPW; ++u)
      B.q[u] = ld16((const char*)a.q + ((size_t)(r * H + h + u) * D + sub * EPL) * E::kBytes);
    B.ntok = ntok < kBlock ? ntok : kBlock;
    B.seq = r * H + h;
    B.piece_end = (b == cnt - 1);
    // advance the cursor to the next column (same head)
    if (++b == cnt) {
      b = 0;
      do { ++r; } while (r < R && s_cnt[r] == 0);
      cnt = r < R ? s_cnt[r] : 1;
    }
  };

  float m[HPW], l[HPW];
  float acc[HPW][EPL];
#pragma unroll
  for (int u = 0; u < HPW; ++u) {
    m[u] = -INFINITY; l[u] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[u][e] = 0.f;
  }

  // close the current piece of sequences seq .. seq + HPW - 1 (the wave's
  // heads): combine the token groups, write the normalised output and
  // log-sum-exp, reset the state
  auto close_piece = [&](int seq) {
    const int piece = grp - s_excl[seq / H] / Q;
#pragma unroll
    for (int u = 0; u < HPW; ++u) {
#pragma unroll
      for (int off = LPT; off < kWave; off <<= 1) {
        const float mo = __shfl_xor(m[u], off);
        const float lo = __shfl_xor(l[u], off);
        const float mn = fmaxf(m[u], mo);
        const float mref = (mn == -INFINITY) ? 0.f : mn;
        const float sa = fast_exp2(m[u] - mref), sb = fast_exp2(mo - mref);
        l[u] = l[u] * sa + lo * sb;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[u][e] = acc[u][e] * sa + __shfl_xor(acc[u][e], off) * sb;
        m[u] = mn;
      }
      if (tg == 0) {
        const size_t slot = (size_t)(seq + u) * a.seg + a.seg_pre + piece;
        const float inv = 1.f / l[u];
        float* o = a.o_part + slot * D + sub * EPL;
#pragma unroll
        for (int e = 0; e < EPL; e += 4)
          *reinterpret_cast<f32x4*>(o + e) = f32x4{acc[u][e] * inv, acc[u][e + 1] * inv,
                                                   acc[u][e + 2] * inv, acc[u][e + 3] * inv};
        if (lane == 0) a.lse_part[slot] = m[u] + fast_log2(l[u]);
      }
      m[u] = -INFINITY; l[u] = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[u][e] = 0.f;
    }
  };

  auto reduce = [&](Blk& B, bool run_end) {
    if constexpr (APPEND) {
      if (B.app >= 0) {                        // write this step's token into the cache
#pragma unroll
        for (int u = 0; u < HPW; ++u)
#pragma unroll
          for (int i = 0; i < IPB; ++i) {
            if (i == B.app) {
              const size_t wo = B.app_off + (size_t)u * BLK_B;       // head h + u
              *reinterpret_cast<u32x4*>((char*)a.app_k + wo) = B.k[u * IPB + i];
              *reinterpret_cast<u32x4*>((char*)a.app_v + wo) = B.v[u * IPB + i];
            }
          }
      }
    }
#pragma unroll
    for (int u = 0; u < HPW; ++u) {
      u32x4* bk = B.k + u * IPB;
      u32x4* bv = B.v + u * IPB;
      float s[IPB];
#pragma unroll
      for (int i = 0; i < IPB; ++i) s[i] = group_sum<LPT>(E::dot(bk[i], B.q[u])) * a.scale_log2;
      if (B.ntok < kBlock) {                  // partly filled block: mask the tail
#pragma unroll
        for (int i = 0; i < IPB; ++i) {
          if (i * TPI + tg >= B.ntok) {
            s[i] = -INFINITY;
            bv[i] = u32x4{0u, 0u, 0u, 0u};    // 0 * NaN would poison the sum
          }
        }
      }
      float bm = s[0];
#pragma unroll
      for (int i = 1; i < IPB; ++i) bm = fmaxf(bm, s[i]);
      const float mn = fmaxf(m[u], bm);
      const float mref = (mn == -INFINITY) ? 0.f : mn;
      const float alpha = fast_exp2(m[u] - mref);
      float psum = 0.f;
      float p[IPB];
#pragma unroll
      for (int i = 0; i < IPB; ++i) { p[i] = fast_exp2(s[i] - mref); psum += p[i]; }
      l[u] = l[u] * alpha + psum;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[u][e] *= alpha;
#pragma unroll
      for (int i = 0; i < IPB; ++i) {
        float v[EPL];
        E::to_f32(bv[i], v);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[u][e] = __builtin_fmaf(p[i], v[e], acc[u][e]);
      }
      m[u] = mn;
    }
    if (B.piece_end || run_end) close_piece(B.seq);
  };

  Blk A, Bb;
  fetch(A);
  for (int i = 0;; i += 2) {
    if (i + 1 >= nblk_run) { reduce(A, true); break; }
    fetch(Bb);
    reduce(A, false);
    if (i + 2 >= nblk_run) { reduce(Bb, true); break; }
    fetch(A);
    reduce(Bb, false);
  }
}

}  // namespace parrot
