// C ABI of libparrot_attn: argument checks, work sizing and kernel launches.
// Everything here runs on host scalars; no call reads device memory except
// parrot_validate_inputs, which synchronises on purpose.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <mutex>
#include <string>

#include "parrot_attn.h"
#include "ceiling.h"
#include "common.h"
#include "errors.h"
#include "prefill_args.h"
#include "prefill_shape.h"

namespace {

thread_local std::string g_err;

parrot_status fail(parrot_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

}  // namespace

namespace parrot {

parrot_status set_error(parrot_status s, const char* fmt, ...) {
  if (s == PARROT_OK) {
    g_err.clear();
    return s;
  }
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

}  // namespace parrot

namespace {

long ceil_div(long a, long b) { return (a + b - 1) / b; }

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

// Chunk sizes and slot counts.  Chunks are whole 16-token blocks.  A prefix
// chunk is one prefix-group workgroup's work (see prefix_chunk below).
#ifndef PARROT_PREFIX_CHUNK
#define PARROT_PREFIX_CHUNK 256
#endif
#ifndef PARROT_SPLITKV_WGS_PER_CU
#define PARROT_SPLITKV_WGS_PER_CU 2     // split-KV workgroups (4 waves each) per CU
#endif
#ifndef PARROT_SPLITKV_MIN_BLOCKS
#define PARROT_SPLITKV_MIN_BLOCKS 2
#endif
#ifndef PARROT_SPLITKV_HPW
#define PARROT_SPLITKV_HPW 2            // heads per split-KV wave on the shared path (1 or 2)
#endif
#ifndef PARROT_SPLITKV_WGS_PER_CU_HPW2
#define PARROT_SPLITKV_WGS_PER_CU_HPW2 1
#endif
constexpr int kPrefixChunk = PARROT_PREFIX_CHUNK;
constexpr int kPrefixChunkMax = 1024;   // the prefix role's table stage holds 64 blocks
constexpr int kSplitkvWgsPerCu = PARROT_SPLITKV_WGS_PER_CU;
constexpr int kSplitkvMinBlocks = PARROT_SPLITKV_MIN_BLOCKS;
constexpr int kSplitkvHpw = PARROT_SPLITKV_HPW;
constexpr int kSplitkvWgsPerCuHpw2 = PARROT_SPLITKV_WGS_PER_CU_HPW2;

// Compute units of the current device (cached per device; no device sync).
int num_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// Heads per split-KV wave on the shared path.  Two adjacent heads give each
// wave one contiguous 8 KiB piece per tensor and block instead of 4 KiB: a read
// probe over random 128 KiB blocks reaches 7.0 TB/s with 8 KiB pieces at four
// waves per CU against 6.7 TB/s with 4 KiB pieces at eight (the same bytes in
// flight), and the own-token stream ran 2-3.5 % faster on the 32-layer mixed,
// system-prompt and map-reduce workloads.  Its kernel runs two waves per SIMD
// (twice the registers per fetched block), which leaves fewer slots for the
// prefix workgroups once the own-token stream drains, so it is taken when the
// prefix tokens (bound: groups x max_prefix_len) are at most half the own
// tokens (bound: requests x max_suffix_len): at a 16384-token prefix over 32
// requests it was 2.3 % slower.  Even head counts and 16-bit caches only (an
// fp32 block is twice the registers).  Decode with append takes the same
// layout as the plain call, so the two give the same bits.
int splitkv_hpw(const parrot_problem* p, bool shared) {
  if (kSplitkvHpw != 2 || !shared || p->num_heads % 2 != 0 || p->dtype == PARROT_DTYPE_F32) return 1;
  const double prefix_tokens = (double)p->num_groups * p->max_prefix_len;
  const double own_tokens = (double)p->num_requests * p->max_suffix_len;
  return 2.0 * prefix_tokens <= own_tokens ? 2 : 1;
}

// Split-KV workgroups of a decode launch: a fixed number per CU, and at least
// one wave per head group.
long splitkv_workgroups(int heads, int hpw = 1) {
  long n = (long)num_cus() * (hpw == 2 ? kSplitkvWgsPerCuHpw2 : kSplitkvWgsPerCu);
  const long hg = heads / hpw;
  if (n * parrot::kSkvWaves < hg) n = ceil_div(hg, parrot::kSkvWaves);
  return n;
}

// Column groups of the split-KV role (waves per head group).
long splitkv_groups(int heads, int hpw) {
  return splitkv_workgroups(heads, hpw) * parrot::kSkvWaves / (heads / hpw);
}

// Prefix chunk length.  One prefix-group workgroup streams one chunk of one
// head for up to 64 members, about two 16 KiB stages in flight, so its run time
// grows with the chunk; every chunk also costs each member one partial result
// written and merged.  With n(c) = max_prefix_len * groups * heads * query
// tiles / c workgroups for chunk c (an upper bound: the host only knows the
// maximum prefix length), measured on MI355X:
//  * n(1024) <= CUs: the smallest c in {256, 512, 1024} with n(c) <= CUs; all
//    prefix workgroups then run alongside the own-token stream from the start;
//  * CUs < n(1024) <= 2 CUs: c = 512, so that the workgroups that start late
//    (once the own-token stream drains) are short;
//  * otherwise c = 1024 (many rounds anyway; fewest partial results).
// The smallest chunk is 256 tokens, unless the own-token stream is too short to
// cover a 256-token chunk: a chunk costs about one memory round trip (taken as
// 1.5 us) per 32-token stage, and the stream about its bytes at 5 TB/s, so the
// chunk then shrinks to the stages the stream covers (down to one stage: 32
// tokens).  Measured: a 4-request, 128-token fp32 group (own tokens ~100)
// 16.3 -> 10.7 us per call; the benchmark workloads keep their chunks.
// `any_stream`: the chunk for the shortest own-token stream (the smallest the
// rule can give for these prefix sizes), which sizes the workspace so that it
// does not shrink when requests or own tokens are added.
int prefix_chunk(const parrot_problem* p, int qtiles, bool any_stream = false) {
  if (p->num_groups <= 0) return kPrefixChunk;
  const double work = (double)p->max_prefix_len * p->num_groups * p->num_heads * qtiles;
  const double cus = num_cus();
  const double elt = p->dtype == PARROT_DTYPE_F32 ? 4.0 : 2.0;
  const double own_bytes = (double)p->num_requests * p->max_suffix_len * 2.0 * p->num_heads * p->head_dim * elt;
  const double stream_stages = any_stream ? 0.0 : own_bytes / 5e12 / 1.5e-6;
  int cp = kPrefixChunk;
  while (cp > 32 && cp / 32 > stream_stages) cp /= 2;
  if (work / kPrefixChunkMax <= cus) {
    while (cp < kPrefixChunkMax && work / cp > cus) cp *= 2;
  } else if (work / kPrefixChunkMax <= 2 * cus) {
    cp = std::max(cp, kPrefixChunkMax / 2);
  } else {
    cp = std::max(cp, kPrefixChunkMax);
  }
  return cp;
}

parrot_status check_problem(const parrot_problem* p, parrot::Plan* pl) {
  if (!p) return fail(PARROT_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (p->num_requests < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_requests %d < 0", p->num_requests);
  if (p->num_heads < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_heads %d < 1", p->num_heads);
  if (p->num_groups < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_groups %d < 0", p->num_groups);
  if (p->dtype != PARROT_DTYPE_F32 && p->dtype != PARROT_DTYPE_F16 && p->dtype != PARROT_DTYPE_BF16)
    return fail(PARROT_ERR_UNSUPPORTED, "dtype %d is not f32, f16 or bf16", (int)p->dtype);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(PARROT_ERR_UNSUPPORTED, "head_dim %d (built for 64 and 128)", p->head_dim);
  if (p->block_size != parrot::kBlock)
    return fail(PARROT_ERR_UNSUPPORTED, "block_size %d (built for 16)", p->block_size);
  if (!std::isfinite(p->sm_scale)) return fail(PARROT_ERR_INVALID_ARGUMENT, "sm_scale is not finite");
  if (p->max_suffix_len < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "max_suffix_len %d < 0", p->max_suffix_len);
  if (p->max_prefix_len < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "max_prefix_len %d < 0", p->max_prefix_len);
  const int B = p->block_size;
  if (p->num_groups > 0) {
    if (p->max_prefix_len < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "max_prefix_len must be >= 1 when num_groups > 0");
    if (p->max_group_size < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "max_group_size must be >= 1 when num_groups > 0");
    if (p->max_group_size > p->num_requests && p->num_requests > 0)
      return fail(PARROT_ERR_INVALID_ARGUMENT, "max_group_size %d > num_requests %d", p->max_group_size, p->num_requests);
    if (p->prefix_table_stride < ceil_div(p->max_prefix_len, B))
      return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix_table_stride %d < ceil(max_prefix_len / block_size) = %ld",
                  p->prefix_table_stride, ceil_div(p->max_prefix_len, B));
    if (p->num_prefix_blocks < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_prefix_blocks must be >= 1 when num_groups > 0");
  }
  if (p->suffix_table_stride < ceil_div(p->max_suffix_len, B) || p->suffix_table_stride < 0)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "suffix_table_stride %d < ceil(max_suffix_len / block_size) = %ld",
                p->suffix_table_stride, ceil_div(p->max_suffix_len, B));
  if (p->num_suffix_blocks < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_suffix_blocks must be >= 1");
  if (p->num_requests > 0 && p->num_groups == 0 && p->max_suffix_len == 0)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "no request can have a non-empty context (no groups, max_suffix_len 0)");

  if (p->max_prefix_depth < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "max_prefix_depth %d < 0", p->max_prefix_depth);
  if (p->max_prefix_depth > parrot::kMaxDepth)
    return fail(PARROT_ERR_UNSUPPORTED, "max_prefix_depth %d > %d", p->max_prefix_depth, parrot::kMaxDepth);
  pl->depth = p->num_groups > 0 ? std::max(1, (int)p->max_prefix_depth) : 0;
  const long mg = p->num_groups > 0 ? p->max_group_size : 1;
  pl->prefix_waves = 4;
  pl->prefix_qtiles = (int)ceil_div(mg, 16 * pl->prefix_waves);
  pl->cp = prefix_chunk(p, pl->prefix_qtiles);
  pl->skv_min_q = kSplitkvMinBlocks;
  // slots: shared path = prefix chunks + split-KV pieces of the own tokens;
  // per-request path = split-KV pieces of prefix + own tokens.  One stride
  // serves both.  A sequence of n block columns touches at most
  // ceil(n / min_q) + 1 runs of the flat column list, and never more than the
  // G column groups the role has (its piece index is its group minus the
  // group of its first column).
  const long nbp_max = p->num_groups > 0 ? ceil_div(p->max_prefix_len, B) : 0;
  const long nbs_max = ceil_div(p->max_suffix_len, B);
  // the shared path streams one or two heads per wave, the per-request path
  // one; a bound on the pieces covers either
  const long groups = splitkv_groups(p->num_heads, 1);
  const long groups_shared = std::max(groups, splitkv_groups(p->num_heads, splitkv_hpw(p, true)));
  const long pieces_shared = nbs_max > 0 ? std::min(ceil_div(nbs_max, pl->skv_min_q) + 1, groups_shared) : 0;
  const long pieces_naive = std::min(ceil_div(nbp_max + nbs_max, pl->skv_min_q) + 1, groups);
  pl->seg_p = p->num_groups > 0 ? (int)ceil_div(p->max_prefix_len, pl->cp) : 0;
  if (pl->seg_p > 0xFFFF)
    return fail(PARROT_ERR_UNSUPPORTED, "max_prefix_len %d needs %d prefix chunks (at most 65535)",
                p->max_prefix_len, pl->seg_p);
  pl->seg_pre = pl->depth * pl->seg_p;
  pl->seg_s = (int)pieces_shared;
  const long seg = std::max<long>(pl->seg_pre + pieces_shared, pieces_naive);
  pl->seg = (int)seg;
  pl->skv_waves = 0;   // set at launch from the device's CU count
  // the workspace holds the slots of the smallest prefix chunk any own-token
  // stream could select (at least this call's): its size never drops when
  // num_requests or max_suffix_len grow
  const long seg_p_ws = p->num_groups > 0 ? ceil_div(p->max_prefix_len, prefix_chunk(p, pl->prefix_qtiles, true)) : 0;
  const long seg_ws = std::max<long>(std::max<long>(pl->depth * seg_p_ws + pieces_shared, pieces_naive), seg);

  const double slots = (double)p->num_requests * p->num_heads * seg_ws;
  const double flat = (double)p->num_requests * (double)(nbp_max + nbs_max);
  const double grid_b = (double)p->num_groups * pl->seg_p * p->num_heads * pl->prefix_qtiles;
  if (flat > 2e9 || grid_b > 2e9 || slots * p->head_dim * 4.0 > 9e18)
    return fail(PARROT_ERR_UNSUPPORTED, "problem too large for one launch (%.3g blocks)", flat);
  const size_t n_slots = (size_t)p->num_requests * p->num_heads * seg_ws;
  auto align256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  pl->o_bytes = align256(n_slots * p->head_dim * sizeof(float));
  pl->lse_bytes = align256(n_slots * sizeof(float));
  pl->info_bytes = align256((size_t)p->num_requests * parrot::kMetaInts * sizeof(int32_t));
  pl->total_bytes = p->num_requests > 0 ? pl->o_bytes + pl->lse_bytes + pl->info_bytes : 0;
  return PARROT_OK;
}

// The workspace layout of one shared-path call sized for that call alone: the
// prefix chunks of this call's chunk size and its split-KV pieces, with no
// slots reserved for the per-request path or for smaller chunks (used where
// the workspace is the library's own fixed array and is laid out afresh on
// every call).
void exact_shared_layout(const parrot_problem* p, parrot::Plan* pl) {
  pl->seg = pl->seg_pre + pl->seg_s;
  const size_t n_slots = (size_t)p->num_requests * p->num_heads * pl->seg;
  auto align256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  pl->o_bytes = align256(n_slots * p->head_dim * sizeof(float));
  pl->lse_bytes = align256(n_slots * sizeof(float));
  pl->info_bytes = align256((size_t)p->num_requests * parrot::kMetaInts * sizeof(int32_t));
  pl->total_bytes = p->num_requests > 0 ? pl->o_bytes + pl->lse_bytes + pl->info_bytes : 0;
}

hipEvent_t ev(void* p) { return reinterpret_cast<hipEvent_t>(p); }

parrot_status hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(PARROT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return PARROT_OK;
}

parrot_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(PARROT_ERR_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return PARROT_OK;
}

#define PARROT_TRY(x) do { parrot_status _s = (x); if (_s != PARROT_OK) return _s; } while (0)

// shared: prefix-group role for the prefixes (else the split-KV role reads
// them per request); parents: nested groups (shared path only; NULL = flat).
// k_new / v_new (both or neither): append this step's token to the suffix
// pools (which are then written) while attending.
parrot_status decode(bool shared, const parrot_problem* p, const void* q, const void* prefix_k,
                     const void* prefix_v, const void* suffix_k, const void* suffix_v,
                     const int32_t* ptab, const int32_t* plen, const int32_t* parents,
                     const int32_t* stab, const int32_t* slen, const int32_t* gid, void* out,
                     float* lse, void* workspace, size_t workspace_bytes, void* stream,
                     const parrot_trace* trace, const void* k_new = nullptr,
                     const void* v_new = nullptr, bool exact = false) {
  parrot::Plan pl;
  PARROT_TRY(check_problem(p, &pl));
  if (exact) exact_shared_layout(p, &pl);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const parrot_trace none = {nullptr, nullptr, nullptr, nullptr};
  const parrot_trace& tr = trace ? *trace : none;
  if (p->num_requests == 0) {
    g_err.clear();
    return PARROT_OK;
  }
  struct { const void* ptr; const char* name; size_t align; } req[] = {
      {q, "q", 16}, {suffix_k, "suffix_k", 16}, {suffix_v, "suffix_v", 16},
      {stab, "suffix_block_tables", 4}, {slen, "suffix_lens", 4}, {gid, "group_ids", 4},
      {out, "out", 16}, {lse, "lse", 4}, {workspace, "workspace", 256}};
  for (auto& r : req) {
    if (!r.ptr) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", r.name);
    if (!aligned(r.ptr, r.align)) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", r.name, r.align);
  }
  if (p->num_groups > 0) {
    struct { const void* ptr; const char* name; size_t align; } preq[] = {
        {prefix_k, "prefix_k", 16}, {prefix_v, "prefix_v", 16},
        {ptab, "prefix_block_tables", 4}, {plen, "prefix_lens", 4}};
    for (auto& r : preq) {
      if (!r.ptr) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", r.name);
      if (!aligned(r.ptr, r.align)) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", r.name, r.align);
    }
  }
  if (k_new || v_new) {
    struct { const void* ptr; const char* name; } areq[] = {{k_new, "k_new"}, {v_new, "v_new"}};
    for (auto& r : areq) {
      if (!r.ptr) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", r.name);
      if (!aligned(r.ptr, 16)) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", r.name);
    }
  }
  if (workspace_bytes < pl.total_bytes)
    return fail(PARROT_ERR_WORKSPACE_TOO_SMALL, "workspace is %zu bytes, need %zu", workspace_bytes, pl.total_bytes);

  float* o_part = reinterpret_cast<float*>(workspace);
  float* lse_part = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + pl.o_bytes);
  int* merge_meta = reinterpret_cast<int*>(reinterpret_cast<char*>(workspace) + pl.o_bytes + pl.lse_bytes);
  const float scale_log2 = p->sm_scale * parrot::kLog2e;
  const int D = p->head_dim, dt = (int)p->dtype;

  const bool run_prefix = shared && p->num_groups > 0 && pl.seg_p > 0;
  {
    parrot::PartialsArgs pa{};
    parrot::SplitKVArgs& a = pa.skv;
    a.q = q; a.pk = prefix_k; a.pv = prefix_v; a.sk = suffix_k; a.sv = suffix_v;
    a.ptab = ptab; a.plen = plen; a.stab = stab; a.slen = slen; a.gid = gid;
    a.parents = shared ? parents : nullptr;
    a.depth = parents ? pl.depth : 1;
    a.k_new = k_new; a.v_new = v_new;
    a.app_k = const_cast<void*>(suffix_k); a.app_v = const_cast<void*>(suffix_v);
    a.o_part = o_part; a.lse_part = lse_part; a.merge_meta = merge_meta;
    a.R = p->num_requests; a.H = p->num_heads; a.NG = p->num_groups;
    a.pstride = p->prefix_table_stride; a.sstride = p->suffix_table_stride;
    a.max_p = p->max_prefix_len; a.max_s = p->max_suffix_len;
    a.npblk = p->num_groups > 0 ? p->num_prefix_blocks : 1; a.nsblk = p->num_suffix_blocks;
    a.seg = pl.seg; a.seg_pre = shared ? pl.seg_pre : 0; a.cp = pl.cp;
    a.with_prefix = shared ? 0 : 1;
    // a fixed grid of split-KV workgroups per CU, at least one wave per head group
    a.hpw = splitkv_hpw(p, shared);
    pa.n_skv = (int)splitkv_workgroups(a.H, a.hpw);
    a.nwaves = pa.n_skv * parrot::kSkvWaves;
    a.min_q = pl.skv_min_q;
    a.scale_log2 = scale_log2;
    if (run_prefix) {
      parrot::PrefixArgs& b = pa.pre;
      b.q = q; b.pk = prefix_k; b.pv = prefix_v; b.ptab = ptab; b.plen = plen; b.gid = gid;
      b.parents = parents;
      b.depth = parents ? pl.depth : 1;
      b.o_part = o_part; b.lse_part = lse_part;
      b.R = p->num_requests; b.H = p->num_heads; b.NG = p->num_groups;
      b.pstride = p->prefix_table_stride; b.max_p = p->max_prefix_len; b.npblk = p->num_prefix_blocks;
      b.seg = pl.seg; b.seg_p = pl.seg_p; b.cp = pl.cp; b.qtiles = pl.prefix_qtiles;
      b.scale_log2 = scale_log2;
      pa.n_pre = p->num_groups * pl.seg_p * p->num_heads * pl.prefix_qtiles;
    }
    // The split-KV role holds its per-request scan in LDS for up to
    // kMaxRequests requests, so a larger batch is streamed in slices of that
    // many requests, one launch each (every per-request pointer moved to the
    // slice); the prefix-group role covers every request in the first launch,
    // and one merge follows.  The trace brackets all of them.
    const int R = p->num_requests, H = p->num_heads;
    const size_t elt = p->dtype == PARROT_DTYPE_F32 ? 4 : 2;
    for (int r0 = 0; r0 < R; r0 += parrot::kMaxRequests) {
      const int rn = std::min(parrot::kMaxRequests, R - r0);
      parrot::PartialsArgs slice = pa;
      parrot::SplitKVArgs& c = slice.skv;
      const size_t rows = (size_t)r0 * H;
      c.q = static_cast<const char*>(q) + rows * D * elt;
      c.stab = stab + (size_t)r0 * p->suffix_table_stride;
      c.slen = slen + r0;
      c.gid = gid + r0;
      if (k_new) {
        c.k_new = static_cast<const char*>(k_new) + rows * D * elt;
        c.v_new = static_cast<const char*>(v_new) + rows * D * elt;
      }
      c.o_part = o_part + rows * pl.seg * D;
      c.lse_part = lse_part + rows * pl.seg;
      c.merge_meta = merge_meta + (size_t)r0 * parrot::kMetaInts;
      c.R = rn;
      if (r0 > 0) slice.n_pre = 0;
      const bool first = r0 == 0, last = r0 + rn == R;
      PARROT_TRY(launched(parrot::launch_partials(slice, dt, D, s,
                                                  first ? ev(tr.partials_start) : nullptr,
                                                  last ? ev(tr.partials_stop) : nullptr),
                          "partials kernel"));
    }
  }
  {
    parrot::MergeArgs a{};
    a.o_part = o_part; a.lse_part = lse_part; a.merge_meta = merge_meta;
    a.out = out; a.lse = lse;
    a.R = p->num_requests; a.H = p->num_heads;
    a.seg = pl.seg; a.seg_p = pl.seg_p; a.seg_pre = shared ? pl.seg_pre : 0;
    PARROT_TRY(launched(parrot::launch_merge(a, dt, D, s, ev(tr.merge_start), ev(tr.merge_stop)),
                        "merge kernel"));
  }
  g_err.clear();
  return PARROT_OK;
}

}  // namespace

extern "C" {

size_t parrot_workspace_bytes(const parrot_problem* p) {
  parrot::Plan pl;
  if (check_problem(p, &pl) != PARROT_OK) return (size_t)-1;
  g_err.clear();
  return pl.total_bytes;
}

parrot_status parrot_shared_prefix_decode(
    const parrot_problem* p, const void* q, const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v, const int32_t* prefix_block_tables,
    const int32_t* prefix_lens, const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, void* out, float* lse, void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace) {
  return decode(true, p, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
                prefix_lens, nullptr, suffix_block_tables, suffix_lens, group_ids, out, lse,
                workspace, workspace_bytes, stream, trace);
}

parrot_status parrot_per_request_decode(
    const parrot_problem* p, const void* q, const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v, const int32_t* prefix_block_tables,
    const int32_t* prefix_lens, const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, void* out, float* lse, void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace) {
  return decode(false, p, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
                prefix_lens, nullptr, suffix_block_tables, suffix_lens, group_ids, out, lse,
                workspace, workspace_bytes, stream, trace);
}

parrot_status parrot_shared_prefix_decode_append(
    const parrot_problem* p, const void* q, const void* k_new, const void* v_new,
    const void* prefix_k, const void* prefix_v, void* suffix_k, void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens, const int32_t* group_ids,
    void* out, float* lse, void* workspace, size_t workspace_bytes, void* stream,
    const parrot_trace* trace) {
  if (p && p->num_requests > 0 && (!k_new || !v_new))
    return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", k_new ? "v_new" : "k_new");
  return decode(true, p, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
                prefix_lens, nullptr, suffix_block_tables, suffix_lens, group_ids, out, lse,
                workspace, workspace_bytes, stream, trace, k_new, v_new);
}

parrot_status parrot_nested_prefix_decode(
    const parrot_problem* p, const void* q, const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v, const int32_t* prefix_block_tables,
    const int32_t* prefix_lens, const int32_t* prefix_parents, const int32_t* suffix_block_tables,
    const int32_t* suffix_lens, const int32_t* group_ids, void* out, float* lse, void* workspace,
    size_t workspace_bytes, void* stream, const parrot_trace* trace) {
  if (p && p->num_requests > 0 && p->num_groups > 0) {
    if (!prefix_parents) return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix_parents is NULL");
    if (!aligned(prefix_parents, 4)) return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix_parents is not 4-byte aligned");
  }
  return decode(true, p, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
                prefix_lens, p && p->num_groups > 0 ? prefix_parents : nullptr,
                suffix_block_tables, suffix_lens, group_ids, out, lse, workspace,
                workspace_bytes, stream, trace);
}

}  // extern "C"

// ------------------------------------------------------ allocation-free decode
// The partial-result workspace of parrot_shared_prefix_decode_noalloc: one
// fixed array per device, held from the library's load on that device until
// the process ends.  Every call lays its partial results out afresh and
// writes each slot before the merge reads it, so nothing in it has to start
// at zero; calls that overlap on one device share it and race.
static __device__ __align__(256) char scratch[PARROT_STATIC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on the current device, looked up once per
// device with that device current.  The array's name in host code is only a
// host-side handle; kernels get this address.
parrot_status static_scratch(void** out) {
  static std::atomic<void*> addr[64];
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(PARROT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(PARROT_ERR_UNSUPPORTED, "device %d (at most 64 devices)", dev);
  void* ptr = addr[dev].load(std::memory_order_acquire);
  if (!ptr) {
    std::lock_guard<std::mutex> lock(mu);
    ptr = addr[dev].load(std::memory_order_relaxed);
    if (!ptr) {
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ptr)
        return fail(PARROT_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      addr[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return PARROT_OK;
}

}  // namespace

extern "C" {

parrot_status parrot_shared_prefix_decode_noalloc(
    const parrot_problem* p, const void* q, const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v, const int32_t* prefix_block_tables,
    const int32_t* prefix_lens, const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, void* out, float* lse, void* stream, const parrot_trace* trace) {
  parrot::Plan pl;
  PARROT_TRY(check_problem(p, &pl));
  if (p->num_requests == 0) {
    g_err.clear();
    return PARROT_OK;
  }
  exact_shared_layout(p, &pl);
  if (pl.total_bytes > (size_t)PARROT_STATIC_SCRATCH_BYTES)
    return fail(PARROT_ERR_WORKSPACE_TOO_SMALL,
                "this call needs %zu bytes of partial results; the library's fixed array holds %zu "
                "(use parrot_shared_prefix_decode with a workspace)",
                pl.total_bytes, (size_t)PARROT_STATIC_SCRATCH_BYTES);
  void* ws = nullptr;
  PARROT_TRY(static_scratch(&ws));
  return decode(true, p, q, prefix_k, prefix_v, suffix_k, suffix_v, prefix_block_tables,
                prefix_lens, nullptr, suffix_block_tables, suffix_lens, group_ids, out, lse, ws,
                (size_t)PARROT_STATIC_SCRATCH_BYTES, stream, trace, nullptr, nullptr, true);
}

}  // extern "C"

namespace {

// ------------------------------------------------------------------ prefill
constexpr int kPrefillChunkMax = 8192;   // the prefill tile's table holds 512 blocks
constexpr int kPrefillChunkMin = 256;

struct PrefillPlan {
  int depth, cp, co, seg_p, seg_pre, seg_s, seg, qtiles_p, qtiles_o;
  long n_pre, n_own;
  bool single;   // single-pass items: no partial results, no merge
  size_t o_bytes, lse_bytes, info_bytes, total_bytes;
};

// The single-pass prefill runs when the groups are flat, the caches 16-bit and
// the prefix and own ranges each fit one chunk of the split plan.
// PARROT_PREFILL_SINGLE_PASS=0 turns it off; =1 takes it whenever the ranges
// fit the tile's block table (8192 tokens), even where the split plan would
// cut them into chunks to fill the device (for tests and tuning).
// Any other value (or none) leaves the choice to the plan.
int single_pass_setting() {
  const char* e = std::getenv("PARROT_PREFILL_SINGLE_PASS");
  if (e && e[0] == '0' && e[1] == 0) return 0;
  if (e && e[0] == '1' && e[1] == 0) return 1;
  return -1;
}

// Chunk of a key range of at most `len` tokens: the whole range up to 8192
// tokens (fewest partial results), halved while the items of that chunk size
// (`items_per_chunk` per chunk) would not fill every CU with the three
// workgroups it holds.
int prefill_chunk(long len, double items_per_chunk) {
  int c = kPrefillChunkMax;
  while (c > kPrefillChunkMin && c / 2 >= len) c /= 2;
  const double cus = num_cus();
  while (c > kPrefillChunkMin && items_per_chunk * (double)ceil_div(len, c) < 3 * cus) c /= 2;
  return c;
}

parrot_status check_prefill(const parrot_problem* p, const parrot_prefill_rows* rows, bool nested,
                            PrefillPlan* pl) {
  if (!p) return fail(PARROT_ERR_INVALID_ARGUMENT, "problem is NULL");
  if (!rows) return fail(PARROT_ERR_INVALID_ARGUMENT, "rows is NULL");
  // the decode checks, with the group bound that prefill replaces by rows
  parrot_problem d = *p;
  if (d.num_groups > 0) d.max_group_size = d.num_requests > 0 ? 1 : d.max_group_size;
  parrot::Plan dpl;
  PARROT_TRY(check_problem(&d, &dpl));
  *pl = PrefillPlan{};
  const long T = rows->num_query_rows;
  if (T < 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_query_rows %ld < 0", T);
  if (T == 0) return PARROT_OK;
  if (p->num_requests == 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "num_query_rows %ld > 0 with no requests", T);
  const int mq = rows->max_query_rows;
  if (mq < 1 || mq > p->max_suffix_len)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "max_query_rows %d not in [1, max_suffix_len = %d]", mq,
                p->max_suffix_len);
  if ((long)p->num_requests * mq < T)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "num_query_rows %ld > num_requests * max_query_rows", T);
  const int mg = p->num_groups > 0 ? rows->max_group_rows : 0;
  if (mg < 0 || mg > T)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "max_group_rows %d not in [0, num_query_rows]", mg);
  if (T * p->num_heads > 0x7fffffffL)
    return fail(PARROT_ERR_UNSUPPORTED, "num_query_rows * num_heads > 2^31 - 1");
  const int H = p->num_heads;
  pl->depth = p->num_groups > 0 ? (nested ? std::max(1, (int)p->max_prefix_depth) : 1) : 0;
  const int rows_per_tile = p->dtype == PARROT_DTYPE_F32 ? 64 : parrot::kWideRows;   // the kernel's tile height
  pl->qtiles_p = (int)ceil_div(mg, rows_per_tile);
  pl->qtiles_o = (int)ceil_div(mq, rows_per_tile);
  if (p->num_groups > 0 && pl->qtiles_p > 0) {
    pl->cp = prefill_chunk(p->max_prefix_len, (double)p->num_groups * H * pl->qtiles_p);
    pl->seg_p = (int)ceil_div(p->max_prefix_len, pl->cp);
  } else {
    pl->cp = kPrefillChunkMin;
    pl->seg_p = 0;
  }
  if (pl->seg_p > 0xFFFF)
    return fail(PARROT_ERR_UNSUPPORTED, "max_prefix_len %d needs %d prefix chunks (at most 65535)",
                p->max_prefix_len, pl->seg_p);
  pl->co = prefill_chunk(p->max_suffix_len, (double)p->num_requests * H * pl->qtiles_o);
  pl->seg_s = (int)ceil_div(p->max_suffix_len, pl->co);
  pl->seg_pre = pl->depth * pl->seg_p;
  pl->seg = pl->seg_pre + pl->seg_s;
  // work items per head (the grid holds them for every head, 8 heads apart
  // per XCD)
  pl->n_pre = (long)p->num_groups * pl->seg_p * pl->qtiles_p;
  pl->n_own = (long)p->num_requests * pl->seg_s * pl->qtiles_o;
  const int setting = single_pass_setting();
  const bool fits = p->max_prefix_len <= kPrefillChunkMax && p->max_suffix_len <= kPrefillChunkMax;
  pl->single = p->dtype != PARROT_DTYPE_F32 && !nested && fits &&
               (setting == 1 || (setting == -1 && pl->seg_p <= 1 && pl->seg_s == 1));
  if (pl->single) {   // one item per group tile (whole prefix), one per own tile
    pl->n_pre = pl->seg_p > 0 ? (long)p->num_groups * pl->qtiles_p : 0;
    pl->n_own = (long)p->num_requests * pl->qtiles_o;
  }
  const long grid = 8L * ceil_div(H, 8) * (pl->n_pre + pl->n_own);
  if (grid > 0x7fffffffL)
    return fail(PARROT_ERR_UNSUPPORTED, "prefill needs %ld workgroups (at most 2^31 - 1)", grid);
  const size_t n_slots = (size_t)T * H * pl->seg;
  auto align256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  pl->o_bytes = align256(n_slots * p->head_dim * sizeof(float));
  pl->lse_bytes = align256(n_slots * sizeof(float));
  pl->info_bytes = align256((size_t)T * parrot::kMetaInts * sizeof(int32_t));
  pl->total_bytes = pl->o_bytes + pl->lse_bytes + pl->info_bytes;
  return PARROT_OK;
}

parrot_status prefill(const parrot_problem* p, const parrot_prefill_rows* rows, const void* q,
                      const int32_t* qoff, const void* prefix_k, const void* prefix_v,
                      const void* suffix_k, const void* suffix_v, const int32_t* ptab,
                      const int32_t* plen, const int32_t* parents, const int32_t* stab,
                      const int32_t* slen, const int32_t* gid, void* out, float* lse,
                      void* workspace, size_t workspace_bytes, void* stream,
                      const parrot_trace* trace) {
  PrefillPlan pl;
  PARROT_TRY(check_prefill(p, rows, parents != nullptr, &pl));
  if (rows->num_query_rows == 0) {
    g_err.clear();
    return PARROT_OK;
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const parrot_trace none = {nullptr, nullptr, nullptr, nullptr};
  const parrot_trace& tr = trace ? *trace : none;
  struct { const void* ptr; const char* name; size_t align; } req[] = {
      {q, "q", 16}, {qoff, "query_offsets", 4}, {suffix_k, "suffix_k", 16},
      {suffix_v, "suffix_v", 16}, {stab, "suffix_block_tables", 4}, {slen, "suffix_lens", 4},
      {gid, "group_ids", 4}, {out, "out", 16}, {lse, "lse", 4}, {workspace, "workspace", 256}};
  for (auto& r : req) {
    if (!r.ptr) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", r.name);
    if (!aligned(r.ptr, r.align)) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", r.name, r.align);
  }
  if (p->num_groups > 0) {
    struct { const void* ptr; const char* name; size_t align; } preq[] = {
        {prefix_k, "prefix_k", 16}, {prefix_v, "prefix_v", 16},
        {ptab, "prefix_block_tables", 4}, {plen, "prefix_lens", 4}};
    for (auto& r : preq) {
      if (!r.ptr) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is NULL", r.name);
      if (!aligned(r.ptr, r.align)) return fail(PARROT_ERR_INVALID_ARGUMENT, "%s is not %zu-byte aligned", r.name, r.align);
    }
    if (parents && !aligned(parents, 4)) return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix_parents is not 4-byte aligned");
  }
  if (workspace_bytes < pl.total_bytes)
    return fail(PARROT_ERR_WORKSPACE_TOO_SMALL, "workspace is %zu bytes, need %zu", workspace_bytes, pl.total_bytes);

  float* o_part = reinterpret_cast<float*>(workspace);
  float* lse_part = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + pl.o_bytes);
  int* merge_meta = reinterpret_cast<int*>(reinterpret_cast<char*>(workspace) + pl.o_bytes + pl.lse_bytes);
  const int T = rows->num_query_rows;
  {
    parrot::PrefillArgs a{};
    a.q = q; a.pk = prefix_k; a.pv = prefix_v; a.sk = suffix_k; a.sv = suffix_v;
    a.ptab = ptab; a.plen = plen; a.stab = stab; a.slen = slen; a.gid = gid;
    a.parents = p->num_groups > 0 ? parents : nullptr; a.qoff = qoff;
    a.o_part = o_part; a.lse_part = lse_part; a.merge_meta = merge_meta;
    a.T = T; a.R = p->num_requests; a.H = p->num_heads; a.NG = p->num_groups;
    a.depth = std::max(1, pl.depth);
    a.pstride = p->prefix_table_stride; a.sstride = p->suffix_table_stride;
    a.max_p = p->max_prefix_len; a.max_s = p->max_suffix_len; a.max_q = rows->max_query_rows;
    a.npblk = p->num_groups > 0 ? p->num_prefix_blocks : 1; a.nsblk = p->num_suffix_blocks;
    a.seg = pl.seg; a.seg_p = pl.seg_p; a.seg_pre = pl.seg_pre; a.seg_s = pl.seg_s;
    a.cp = pl.cp; a.co = pl.co; a.qtiles_p = pl.qtiles_p; a.qtiles_o = pl.qtiles_o;
    a.n_pre = (int)pl.n_pre; a.n_own = (int)pl.n_own;
    a.meta_wgs = pl.single ? 0 : (T + 255) / 256;
    a.scale_log2 = p->sm_scale * parrot::kLog2e;
    a.single = pl.single ? 1 : 0;
    a.out = out; a.lse = lse;
    PARROT_TRY(launched(parrot::launch_prefill(a, (int)p->dtype, p->head_dim, s, ev(tr.partials_start),
                                               ev(tr.partials_stop)),
                        "prefill kernel"));
  }
  if (pl.single) {
    // no merge: its trace events, if asked for, bracket nothing
    if (tr.merge_start) PARROT_TRY(hip_ok(hipEventRecord(ev(tr.merge_start), s), "hipEventRecord"));
    if (tr.merge_stop) PARROT_TRY(hip_ok(hipEventRecord(ev(tr.merge_stop), s), "hipEventRecord"));
  } else {
    parrot::MergeArgs a{};
    a.o_part = o_part; a.lse_part = lse_part; a.merge_meta = merge_meta;
    a.out = out; a.lse = lse;
    a.R = T; a.H = p->num_heads;
    a.seg = pl.seg; a.seg_p = pl.seg_p; a.seg_pre = pl.seg_pre;
    PARROT_TRY(launched(parrot::launch_merge(a, (int)p->dtype, p->head_dim, s, ev(tr.merge_start),
                                             ev(tr.merge_stop)),
                        "merge kernel"));
  }
  g_err.clear();
  return PARROT_OK;
}

}  // namespace

extern "C" {

size_t parrot_prefill_workspace_bytes(const parrot_problem* p, const parrot_prefill_rows* rows) {
  PrefillPlan pl;
  // sized for nested groups (depth max_prefix_depth): enough for flat calls too
  if (check_prefill(p, rows, true, &pl) != PARROT_OK) return (size_t)-1;
  g_err.clear();
  return pl.total_bytes;
}

int parrot_prefill_single_pass(const parrot_problem* p, const parrot_prefill_rows* rows, int nested) {
  PrefillPlan pl;
  if (check_prefill(p, rows, nested != 0, &pl) != PARROT_OK) return -1;
  g_err.clear();
  return pl.single ? 1 : 0;
}

parrot_status parrot_shared_prefix_prefill(
    const parrot_problem* p, const parrot_prefill_rows* rows, const void* q,
    const int32_t* query_offsets, const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v, const int32_t* prefix_block_tables,
    const int32_t* prefix_lens, const int32_t* prefix_parents,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens, const int32_t* group_ids,
    void* out, float* lse, void* workspace, size_t workspace_bytes, void* stream,
    const parrot_trace* trace) {
  return prefill(p, rows, q, query_offsets, prefix_k, prefix_v, suffix_k, suffix_v,
                 prefix_block_tables, prefix_lens, prefix_parents, suffix_block_tables,
                 suffix_lens, group_ids, out, lse, workspace, workspace_bytes, stream, trace);
}

}  // extern "C"

namespace {

parrot_status validate(const parrot_problem* p, const int32_t* prefix_block_tables,
                       const int32_t* prefix_lens, const int32_t* prefix_parents,
                       const int32_t* suffix_block_tables, const int32_t* suffix_lens,
                       const int32_t* group_ids, int32_t* scratch, void* stream,
                       const parrot_prefill_rows* rows = nullptr,
                       const int32_t* query_offsets = nullptr) {
  parrot::Plan pl;
  if (rows) {
    PrefillPlan fp;
    PARROT_TRY(check_prefill(p, rows, prefix_parents != nullptr, &fp));
    if (!query_offsets || !aligned(query_offsets, 4))
      return fail(PARROT_ERR_INVALID_ARGUMENT, "query_offsets is NULL or misaligned");
  } else {
    PARROT_TRY(check_problem(p, &pl));
  }
  if (p->num_requests == 0) { g_err.clear(); return PARROT_OK; }
  if (!scratch || !aligned(scratch, 4)) return fail(PARROT_ERR_INVALID_ARGUMENT, "scratch is NULL or misaligned");
  if (!suffix_block_tables || !suffix_lens || !group_ids)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "suffix tables, suffix lengths and group ids are required");
  if (p->num_groups > 0 && (!prefix_block_tables || !prefix_lens))
    return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix tables and lengths are required when num_groups > 0");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemsetAsync(scratch, 0, 3 * sizeof(int32_t), s);
  if (e != hipSuccess) return fail(PARROT_ERR_HIP, "hipMemsetAsync: %s", hipGetErrorString(e));
  parrot::ValidateArgs a{};
  a.ptab = prefix_block_tables; a.plen = prefix_lens; a.stab = suffix_block_tables;
  a.slen = suffix_lens; a.gid = group_ids; a.result = scratch;
  a.parents = p->num_groups > 0 ? prefix_parents : nullptr;
  a.depth = std::max(1, (int)p->max_prefix_depth);
  a.R = p->num_requests; a.NG = p->num_groups; a.B = p->block_size;
  a.pstride = p->prefix_table_stride; a.sstride = p->suffix_table_stride;
  a.max_p = p->max_prefix_len; a.max_s = p->max_suffix_len;
  a.npblk = p->num_prefix_blocks; a.nsblk = p->num_suffix_blocks;
  if (rows) {
    a.qoff = query_offsets; a.T = rows->num_query_rows;
    a.max_q = rows->max_query_rows; a.max_grp = rows->max_group_rows;
  } else {
    a.max_grp = p->max_group_size;
  }
  PARROT_TRY(launched(parrot::launch_validate(a, s), "validation kernel"));
  int32_t res[3] = {0, 0, 0};
  e = hipMemcpyAsync(res, scratch, sizeof res, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(PARROT_ERR_HIP, "reading validation result: %s", hipGetErrorString(e));
  static const char* what[] = {"", "group id out of [-1, num_groups)", "prefix length out of [1, max_prefix_len]",
                               "suffix length out of [0, max_suffix_len]", "empty context (prefix + suffix = 0)",
                               "prefix block id out of [0, num_prefix_blocks)",
                               "suffix block id out of [0, num_suffix_blocks)",
                               "prefix parent not in [-1, group)",
                               "prefix chain deeper than max_prefix_depth",
                               "query_offsets not 0 = offsets[0] <= ... <= offsets[R] = num_query_rows",
                               "query rows of a request > min(suffix length, max_query_rows)",
                               "rows reading a group's prefix > max_group_rows",
                               "requests reading a group's prefix > max_group_size"};
  constexpr int kCodes = (int)(sizeof what / sizeof what[0]) - 1;
  if (res[0] != 0)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "%s at entry %d (value %d)",
                (res[0] > 0 && res[0] <= kCodes) ? what[res[0]] : "unknown", res[1], res[2]);
  g_err.clear();
  return PARROT_OK;
}

}  // namespace

extern "C" {

parrot_status parrot_validate_inputs(const parrot_problem* p, const int32_t* prefix_block_tables,
                                     const int32_t* prefix_lens, const int32_t* suffix_block_tables,
                                     const int32_t* suffix_lens, const int32_t* group_ids,
                                     int32_t* scratch, void* stream) {
  return validate(p, prefix_block_tables, prefix_lens, nullptr, suffix_block_tables, suffix_lens,
                  group_ids, scratch, stream);
}

parrot_status parrot_validate_nested_inputs(const parrot_problem* p, const int32_t* prefix_block_tables,
                                            const int32_t* prefix_lens, const int32_t* prefix_parents,
                                            const int32_t* suffix_block_tables,
                                            const int32_t* suffix_lens, const int32_t* group_ids,
                                            int32_t* scratch, void* stream) {
  if (p && p->num_requests > 0 && p->num_groups > 0 && !prefix_parents)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "prefix_parents is NULL");
  return validate(p, prefix_block_tables, prefix_lens, prefix_parents, suffix_block_tables,
                  suffix_lens, group_ids, scratch, stream);
}

parrot_status parrot_validate_prefill_inputs(const parrot_problem* p, const parrot_prefill_rows* rows,
                                             const int32_t* query_offsets,
                                             const int32_t* prefix_block_tables,
                                             const int32_t* prefix_lens, const int32_t* prefix_parents,
                                             const int32_t* suffix_block_tables,
                                             const int32_t* suffix_lens, const int32_t* group_ids,
                                             int32_t* scratch, void* stream) {
  if (!rows) return fail(PARROT_ERR_INVALID_ARGUMENT, "rows is NULL");
  return validate(p, prefix_block_tables, prefix_lens, prefix_parents, suffix_block_tables,
                  suffix_lens, group_ids, scratch, stream, rows, query_offsets);
}

parrot_status parrot_hbm_read_ceiling(const void* src, size_t bytes, uint32_t* sink,
                                      int32_t workgroups, int32_t loads_per_thread,
                                      int32_t wave_spans, void* stream,
                                      const parrot_trace* trace) {
  if (!src || !sink) return fail(PARROT_ERR_INVALID_ARGUMENT, "src and sink must not be NULL");
  if (!aligned(src, 16) || !aligned(sink, 4))
    return fail(PARROT_ERR_INVALID_ARGUMENT, "src must be 16-byte and sink 4-byte aligned");
  if (bytes % 16 != 0) return fail(PARROT_ERR_INVALID_ARGUMENT, "bytes %zu is not a multiple of 16", bytes);
  if (workgroups < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "workgroups %d < 1", workgroups);
  if (loads_per_thread != 4 && loads_per_thread != 8 && loads_per_thread != 16)
    return fail(PARROT_ERR_UNSUPPORTED, "loads_per_thread %d (built for 4, 8 and 16)", loads_per_thread);
  if (wave_spans != 0 && wave_spans != 1)
    return fail(PARROT_ERR_INVALID_ARGUMENT, "wave_spans %d is not 0 or 1", wave_spans);
  PARROT_TRY(launched(parrot::launch_read_ceiling(src, bytes, sink, workgroups, loads_per_thread,
                                                  wave_spans != 0,
                                                  reinterpret_cast<hipStream_t>(stream),
                                                  trace ? ev(trace->partials_start) : nullptr,
                                                  trace ? ev(trace->partials_stop) : nullptr),
                      "read-ceiling kernel"));
  g_err.clear();
  return PARROT_OK;
}

parrot_status parrot_mfma_issue_ceiling(uint32_t* sink, int32_t workgroups, int32_t iters,
                                        int32_t valu_x4, void* stream, const parrot_trace* trace) {
  if (!sink) return fail(PARROT_ERR_INVALID_ARGUMENT, "sink must not be NULL");
  if (!aligned(sink, 4)) return fail(PARROT_ERR_INVALID_ARGUMENT, "sink must be 4-byte aligned");
  if (workgroups < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "workgroups %d < 1", workgroups);
  if (iters < 1) return fail(PARROT_ERR_INVALID_ARGUMENT, "iters %d < 1", iters);
  if (valu_x4 != 0 && valu_x4 != 8 && valu_x4 != 10 && valu_x4 != 11 && valu_x4 != 12 && valu_x4 != 16)
    return fail(PARROT_ERR_UNSUPPORTED, "valu_x4 %d (built for 0, 8, 10, 11, 12 and 16)", valu_x4);
  PARROT_TRY(launched(parrot::launch_mfma_issue(sink, workgroups, iters, valu_x4,
                                                reinterpret_cast<hipStream_t>(stream),
                                                trace ? ev(trace->partials_start) : nullptr,
                                                trace ? ev(trace->partials_stop) : nullptr),
                      "matrix-core issue kernel"));
  g_err.clear();
  return PARROT_OK;
}

const char* parrot_last_error(void) { return g_err.c_str(); }

int parrot_abi_version(void) { return PARROT_ABI_VERSION; }

}  // extern "C"
