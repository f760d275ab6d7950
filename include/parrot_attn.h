/*
 * libparrot_attn -- shared-prefix decode attention for AMD MI355X (gfx950).
 *
 * One decode iteration of one attention layer for a batch of requests, where
 * requests forked from a common parent context share that context's prompt
 * prefix (Section 5.3, "Sharing Prompt Prefix"; Section 7, the engine's
 * Fill/Generate with parent_context_id).  The shared prefix's keys and values
 * are read once per group, not once per request: a prefix stage computes
 * interim results (running max and exp-sum, here kept as an output vector and
 * a log-sum-exp) for every member of the group, a non-shared stage does the
 * same for each request's own tokens, and a merge joins them into the final
 * attention output (Section 7, "Kernel Optimization").
 *
 * Result (per request r and head h; the paper defers the formula to the
 * FlashAttention and PagedAttention work it builds on):
 *   keys/values j = 0..N-1 are group g's P prefix tokens followed by r's S
 *   own tokens (g = group_ids[r], P = prefix_lens[g] or 0 when g = -1,
 *   S = suffix_lens[r], N = P + S >= 1),
 *   s_j = sm_scale * <q[r,h,:], K_j>,  lse[r,h] = ln sum_j exp(s_j),
 *   out[r,h,:] = sum_j exp(s_j - lse[r,h]) * V_j.
 *
 * Paged KV layout (Section 7: KV cache in non-contiguous blocks located
 * through a per-request page table): a K or V pool is
 *   [num_blocks][H][B][D] elements of `dtype`, row-major,
 * and token t of a sequence with block-table row `tbl` is
 *   pool[tbl[t / B]][h][t % B][:].
 * A request's suffix starts at slot 0 of its own first block; the last block
 * of a prefix or suffix may be partly filled (slots past the length are never
 * read into a result, whatever they hold).
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns all
 *     memory and the stream.  The library allocates nothing and keeps no
 *     pointer after returning.  Calls are reentrant; concurrent calls need
 *     distinct workspaces and outputs.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *     and the call returns without synchronising.  Outputs are valid once the
 *     stream reaches the end of the call's work.
 *   - Every argument check runs before the first launch, so a call that
 *     returns an error other than PARROT_ERR_HIP enqueued nothing.
 *   - Device-side contents (lengths, group ids, block ids) are trusted: values
 *     outside the bounds stated in parrot_problem give unspecified results,
 *     but the kernels clamp every index so no access leaves the buffers whose
 *     sizes the problem describes.  parrot_validate_inputs checks them.
 *   - On error, parrot_last_error() returns a message for the calling thread.
 */
#ifndef PARROT_ATTN_H
#define PARROT_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PARROT_ABI_VERSION 8

typedef enum {
  PARROT_OK = 0,
  PARROT_ERR_INVALID_ARGUMENT = 1,   /* bad scalar, NULL or misaligned pointer */
  PARROT_ERR_UNSUPPORTED = 2,        /* head_dim, block_size or dtype not built */
  PARROT_ERR_WORKSPACE_TOO_SMALL = 3,
  PARROT_ERR_HIP = 4                 /* a HIP call failed (launch, event, sync) */
} parrot_status;

typedef enum {
  PARROT_DTYPE_F32 = 0,
  PARROT_DTYPE_F16 = 1,
  PARROT_DTYPE_BF16 = 2
} parrot_dtype;

/* Problem description: host scalars only.  Sizing and validation never read
 * device memory. */
typedef struct {
  int32_t num_requests;        /* R >= 0; R = 0 is a no-op */
  int32_t num_heads;           /* H >= 1; query heads = KV heads (multi-head) */
  int32_t head_dim;            /* D: 64 or 128 */
  int32_t block_size;          /* B: 16 tokens per KV block */
  int32_t num_groups;          /* NG >= 0 prefix groups */
  int32_t max_group_size;      /* >= members of any group; >= 1 when NG > 0 */
  int32_t max_prefix_len;      /* >= prefix_lens[g] for all g; >= 1 when NG > 0 */
  int32_t max_suffix_len;      /* >= suffix_lens[r] for all r; >= 0 */
  int32_t prefix_table_stride; /* entries per prefix table row, >= ceil(max_prefix_len / B) */
  int32_t suffix_table_stride; /* entries per suffix table row, >= ceil(max_suffix_len / B) */
  int32_t num_prefix_blocks;   /* blocks in the prefix pools (>= 1 when NG > 0) */
  int32_t num_suffix_blocks;   /* blocks in the suffix pools (>= 1) */
  parrot_dtype dtype;          /* element type of q, the KV pools and out */
  float sm_scale;              /* logits are sm_scale * q.k; finite */
  int32_t max_prefix_depth;    /* nested groups: >= the longest chain of groups,
                                  in [0, 4] (0 and 1 mean flat groups); sizes the
                                  workspace.  With nested groups, max_group_size
                                  bounds the requests that read any one group's
                                  prefix (its members and its descendants'). */
} parrot_problem;

/* Optional timing hooks: hipEvent_t handles (each may be NULL), created by the
 * caller with timing enabled.  Each kernel of a call is launched with its pair
 * attached (hipExtLaunchKernel start/stop events), so the events carry that
 * kernel's own start and end time instead of adding marker work to the
 * stream.  Attaching events still costs a few microseconds of stream time per
 * kernel, so time throughput on calls without them. */
typedef struct {
  void* partials_start;  /* the partial-result kernel (split-KV + prefix-group roles;
                            for prefill, the prefill kernel) */
  void* partials_stop;
  void* merge_start;     /* the log-sum-exp merge kernel (a prefill call on the single
                            pass has none: both events are recorded back to back) */
  void* merge_stop;
} parrot_trace;

/* Bytes of device workspace either decode entry point needs for `p`
 * (0 when R = 0).  The prefix chunk, and with it the workspace size, depends
 * on the compute-unit count of the current HIP device, so ask with the device
 * current that the calls will run on (a call with a smaller workspace fails
 * with PARROT_ERR_WORKSPACE_TOO_SMALL).  The size never decreases when
 * num_requests or max_suffix_len grow, so a workspace sized for the largest
 * batch serves every smaller one with the other fields unchanged.  Returns
 * (size_t)-1 if `p` is invalid; the reason is then in parrot_last_error(). */
size_t parrot_workspace_bytes(const parrot_problem* p);

/*
 * Shared-prefix decode attention (Section 5.3; Section 7, "Kernel
 * Optimization").  Two kernels run on `stream` in order:
 *   1. the partial-result kernel, with two kinds of workgroups side by side:
 *      - prefix-group: for each (group, head, prefix chunk) the chunk's K/V
 *        tiles are staged in LDS once and all members' queries are computed
 *        against them on MFMA with an online softmax; one partial result per
 *        member is written to the workspace;
 *      - split-KV: each request's own tokens, split into equal runs of
 *        16-token blocks over a fixed grid, with 128-bit coalesced streaming
 *        loads; one partial per (request, head) piece;
 *   2. the merge kernel: log-sum-exp combination of all partials of (r, h).
 *
 *   q                    [R][H][D] dtype, 16-byte aligned
 *   prefix_k, prefix_v   [num_prefix_blocks][H][B][D] dtype, 16-byte aligned
 *                        (may be NULL when NG = 0)
 *   suffix_k, suffix_v   [num_suffix_blocks][H][B][D] dtype, 16-byte aligned;
 *                        may be the same pools as prefix_k / prefix_v
 *   prefix_block_tables  int32 [NG][prefix_table_stride]
 *   prefix_lens          int32 [NG], each in [1, max_prefix_len]
 *   suffix_block_tables  int32 [R][suffix_table_stride]
 *   suffix_lens          int32 [R], each in [0, max_suffix_len]
 *   group_ids            int32 [R], -1 (no shared prefix) or in [0, NG);
 *                        every request needs P + S >= 1
 *   out                  [R][H][D] dtype (written, round-to-nearest-even)
 *   lse                  float32 [R][H] natural-log log-sum-exp of the logits
 *   workspace            >= parrot_workspace_bytes(p) bytes, 256-byte aligned;
 *                        contents on entry are ignored
 *   trace                optional (host) timing hooks, may be NULL
 */
parrot_status parrot_shared_prefix_decode(
    const parrot_problem* p,
    const void* q,
    const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * parrot_shared_prefix_decode without a workspace argument.  The partial
 * results go to a fixed array inside the library, PARROT_STATIC_SCRATCH_BYTES
 * (64 MiB) per device, which each device the library runs on holds until the
 * process ends.  The call allocates nothing (no hipMalloc, no library
 * allocation); the caller still owns q, the pools, the tables, out and lse.
 * A call whose partial results need more than the array holds (about
 * R * H * (prefix chunks + split-KV pieces) * (D + 1) * 4 bytes, so larger
 * batches) returns PARROT_ERR_WORKSPACE_TOO_SMALL before any launch.  Calls
 * that overlap on one device share the array and race: serialise them (one
 * stream, or events).  The array keeps the last call's contents; every call
 * writes each partial result before reading it, so it needs no clearing.
 * Results equal parrot_shared_prefix_decode's on the same inputs.  Other
 * arguments as parrot_shared_prefix_decode.
 */
#define PARROT_STATIC_SCRATCH_BYTES (64u << 20)
parrot_status parrot_shared_prefix_decode_noalloc(
    const parrot_problem* p,
    const void* q,
    const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* stream, const parrot_trace* trace);

/*
 * Per-request decode attention over the same inputs without sharing: every
 * request reads its group's prefix blocks itself, as a paged-attention
 * decode kernel does (the baseline the paper compares against in Section 8.3).
 * Same arguments, same results up to rounding; the partial-result kernel runs
 * its split-KV role only, over prefix and own tokens.
 */
parrot_status parrot_per_request_decode(
    const parrot_problem* p,
    const void* q,
    const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace);

/*
 * Shared-prefix decode attention that first appends this step's token (the
 * engine's Generate step, Section 7: each iteration fills one more token into
 * every request's context).  For every request with suffix_lens[r] >= 1, the
 * token at own position S_r - 1 is the new one: its keys and values are read
 * from
 *   k_new, v_new         [R][H][D] dtype, 16-byte aligned
 * and written into the suffix pools at slot
 * suffix_block_tables[r][(S_r - 1) / B], offset (S_r - 1) % B (whatever that
 * slot held before is ignored).  Requests with S_r = 0 append nothing.  The
 * result equals writing the new tokens first and then calling
 * parrot_shared_prefix_decode.  The written slot must belong to the request
 * alone: not to another request's blocks nor to any group's prefix (the pools
 * themselves may be the same tensors).  Other arguments as
 * parrot_shared_prefix_decode.
 */
parrot_status parrot_shared_prefix_decode_append(
    const parrot_problem* p,
    const void* q, const void* k_new, const void* v_new,
    const void* prefix_k, const void* prefix_v,
    void* suffix_k, void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace);

/*
 * Nested shared-prefix decode attention: several levels of shared prefixes
 * (Section 5.3: a prompt's prefix hash is taken after every semantic variable,
 * so one prompt can share a system prompt with many requests and a longer
 * prefix with fewer; Section 7: contexts fork from forked contexts through
 * parent_context_id).  Groups form a forest given by
 *   prefix_parents       int32 [NG]: the group whose prefix precedes group g's,
 *                        or -1; always lower than g, so chains end; a chain
 *                        holds at most max_prefix_depth groups.
 * A request of group g attends to the prefixes of g's ancestors, outermost
 * first, then g's prefix, then its own tokens.  Every group's prefix is read
 * once per call, for all requests below it.  Other arguments as
 * parrot_shared_prefix_decode (requests may belong to any group of a chain,
 * or to none); with every parent -1 the result is that of
 * parrot_shared_prefix_decode.
 */
parrot_status parrot_nested_prefix_decode(
    const parrot_problem* p,
    const void* q,
    const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* prefix_parents,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace);

/*
 * Checks the device-side contents against `p` (a debugging aid; it
 * synchronises `stream`): group ids in [-1, NG), prefix lengths in
 * [1, max_prefix_len], suffix lengths in [0, max_suffix_len], P + S >= 1,
 * every block id a length reaches in [0, pool size), and no group's prefix
 * read by more than max_group_size requests (the decode launch sizes its
 * prefix query tiles from that bound).  Returns
 * PARROT_ERR_INVALID_ARGUMENT with a message naming the first bad entry.
 * `scratch` is >= 64 bytes of device memory, 4-byte aligned.
 */
parrot_status parrot_validate_inputs(
    const parrot_problem* p,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, int32_t* scratch, void* stream);

/* parrot_validate_inputs for nested groups: also checks that every parent is
 * in [-1, g) and that no chain holds more than max_prefix_depth groups. */
parrot_status parrot_validate_nested_inputs(
    const parrot_problem* p,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* prefix_parents,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, int32_t* scratch, void* stream);

/*
 * Prefill of forked contexts (Section 7: Fill with a parent_context_id fills a
 * new context's prompt tokens on top of its parent's KV cache, so the parent's
 * tokens -- the group's shared prefix -- are not computed again; Section 5.3
 * for the sharing).  For each request r, its last Q_r own tokens are new:
 *   query_offsets        int32 [R + 1]: rows [query_offsets[r],
 *                        query_offsets[r+1]) of q belong to r, so
 *                        Q_r = query_offsets[r+1] - query_offsets[r], with
 *                        query_offsets[0] = 0, query_offsets[R] = T and
 *                        0 <= Q_r <= min(suffix_lens[r], max_query_rows).
 * Row query_offsets[r] + j is own position p = S_r - Q_r + j; it attends to
 * the prefixes of r's group chain (as parrot_nested_prefix_decode; one group
 * when prefix_parents is NULL) and then to r's own tokens 0..p (causal).  The
 * keys and values of all own tokens, the new ones included, must already be
 * in the suffix pools (the caller writes them, as for any layer's prefill).
 * Q_r < S_r continues a prompt whose first own tokens are cached (chunked
 * prefill).  Per row and head the result is the decode formula over those
 * keys.
 *
 * Rows are computed in tiles of 128 (fp16 / bf16 caches) or 64 (fp32) on
 * MFMA, with K/V staged in LDS.  Two plans, chosen per call:
 *   single pass (flat groups, 16-bit caches, prefix and own lengths that fit
 *     one chunk of 8192 tokens and enough tiles to fill the device): one
 *     kernel; a tile of the rows of a group's members (all requests reading
 *     the prefix, stacked) sees the whole prefix and then, request by
 *     request, its rows' own tokens up to their positions; ungrouped
 *     requests' tiles see their own tokens; the output is written directly
 *     and the workspace is not used;
 *   split: prefix items (stacked rows against one prefix chunk) and own
 *     items (one request's rows against one chunk of its own tokens, per-row
 *     causal limit) write partial results to the workspace, then the merge
 *     kernel combines them per (row, head).
 * parrot_prefill_single_pass tells which one a call takes.  The environment
 * variable PARROT_PREFILL_SINGLE_PASS=0 forces the split plan; =1 takes the
 * single pass wherever the groups are flat, the caches 16-bit and the lengths
 * at most 8192 (even when the split plan would cut them into chunks to fill
 * the device); other values leave the choice to the plan.  Both plans give
 * the same results to rounding.
 *
 *   rows                 (host) row counts; see parrot_prefill_rows
 *   q                    [T][H][D] dtype, 16-byte aligned
 *   prefix_parents       int32 [NG] as parrot_nested_prefix_decode, or NULL
 *                        for flat groups
 *   out                  [T][H][D] dtype;  lse  float32 [T][H]
 *   workspace            >= parrot_prefill_workspace_bytes(p, rows) bytes,
 *                        256-byte aligned
 * Other arguments as parrot_shared_prefix_decode.  `p->max_group_size` is not
 * used (rows->max_group_rows takes its place).  Rows of a call whose offsets
 * break the rules above get unspecified values but every access stays in
 * bounds; parrot_validate_prefill_inputs checks them.
 */
typedef struct {
  int32_t num_query_rows;   /* T = query_offsets[R] >= 0; T = 0 is a no-op */
  int32_t max_query_rows;   /* >= every Q_r; >= 1 when T > 0 */
  int32_t max_group_rows;   /* >= the rows that read any one group's prefix (the
                               rows of its members and, with nested groups, of
                               its descendants' members) */
} parrot_prefill_rows;

/* Bytes of workspace parrot_shared_prefix_prefill needs (0 when T = 0);
 * depends on the current device's compute-unit count like
 * parrot_workspace_bytes.  (size_t)-1 if the arguments are invalid. */
size_t parrot_prefill_workspace_bytes(const parrot_problem* p, const parrot_prefill_rows* rows);

/* 1 when parrot_shared_prefix_prefill takes the single pass for these
 * arguments on the current device, 0 when it takes the split plan, -1 if the
 * arguments are invalid.  `nested` is nonzero when prefix_parents will be
 * non-NULL (nested groups always take the split plan). */
int parrot_prefill_single_pass(const parrot_problem* p, const parrot_prefill_rows* rows, int nested);

parrot_status parrot_shared_prefix_prefill(
    const parrot_problem* p, const parrot_prefill_rows* rows,
    const void* q, const int32_t* query_offsets,
    const void* prefix_k, const void* prefix_v,
    const void* suffix_k, const void* suffix_v,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* prefix_parents,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids,
    void* out, float* lse,
    void* workspace, size_t workspace_bytes,
    void* stream, const parrot_trace* trace);

/* parrot_validate_inputs (with the parent checks when prefix_parents is not
 * NULL) plus the row offsets: query_offsets[0] = 0, non-decreasing,
 * query_offsets[R] = T, every Q_r <= min(S_r, max_query_rows), and at most
 * max_group_rows rows reading any one group. */
parrot_status parrot_validate_prefill_inputs(
    const parrot_problem* p, const parrot_prefill_rows* rows, const int32_t* query_offsets,
    const int32_t* prefix_block_tables, const int32_t* prefix_lens,
    const int32_t* prefix_parents,
    const int32_t* suffix_block_tables, const int32_t* suffix_lens,
    const int32_t* group_ids, int32_t* scratch, void* stream);

/*
 * Measurement aid: the device's attainable HBM read bandwidth, the ceiling of
 * the bandwidth-bound decode kernels (Section 8.3: token generation is bound
 * by memory bandwidth).  Reads every byte of
 *   src                  device buffer of `bytes` bytes (a multiple of 16),
 *                        16-byte aligned; size it well above the 256 MB
 *                        Infinity Cache so the reads come from HBM
 * once, with 16-byte nontemporal loads (as the split-KV role streams KV
 * blocks), `loads_per_thread` (4, 8 or 16) in flight per thread, over
 * `workgroups` workgroups of 256 threads, and XOR-folds the data into
 *   sink                 one uint32 of device memory (read-modify-written)
 * so that no load can be dropped.  wave_spans = 0: grid-stride order
 * (consecutive lanes of the whole grid read consecutive 16-byte pieces);
 * 1: the buffer is cut into one contiguous span per wave, read front to back
 * 1 KiB per instruction (the order of a KV stream).  Enqueued on `stream`;
 * the caller times it (bytes / elapsed is the read bandwidth), optionally with
 *   trace                (host) NULL, or timing hooks whose partials pair is
 *                        attached to the probe's launch (the merge pair is
 *                        unused), so the probe is timed exactly as the decode
 *                        kernels are.
 * Errors: NULL or misaligned pointers, a size that is not a multiple of 16,
 * workgroups < 1 or wave_spans not 0 or 1 give PARROT_ERR_INVALID_ARGUMENT,
 * another loads_per_thread PARROT_ERR_UNSUPPORTED; nothing is enqueued then.
 */
parrot_status parrot_hbm_read_ceiling(const void* src, size_t bytes, uint32_t* sink,
                                      int32_t workgroups, int32_t loads_per_thread,
                                      int32_t wave_spans, void* stream,
                                      const parrot_trace* trace);

/*
 * Measurement aid: the matrix cores' issue rate on this device with a given
 * share of vector instructions between the products, the attainable ceiling
 * of an MFMA kernel whose softmax interleaves vector work with its matrix
 * products (the prefill tile; Section 7, Fill with a parent context).  Each
 * of `workgroups` workgroups of 256 threads runs `iters` iterations of eight
 * independent v_mfma_f32_16x16x32_f16 per wave (8 x 16384 flop) with
 * valu_x4 / 4 vector instructions per MFMA issued between them (four
 * v_exp_f32 per iteration, the rest v_fmac_f32; valu_x4 in {0, 8, 10, 11, 12,
 * 16}), registers only, and XOR-folds the results into
 *   sink                 one uint32 of device memory (read-modify-written)
 * so that nothing is dropped.  Enqueued on `stream`; flops / elapsed is the
 * rate; `trace` (host, may be NULL) attaches its partials pair to the launch.
 * Errors: a NULL or misaligned sink, workgroups < 1 or iters < 1 give
 * PARROT_ERR_INVALID_ARGUMENT, another valu_x4 PARROT_ERR_UNSUPPORTED;
 * nothing is enqueued then.
 */
parrot_status parrot_mfma_issue_ceiling(uint32_t* sink, int32_t workgroups, int32_t iters,
                                        int32_t valu_x4, void* stream, const parrot_trace* trace);

/* Message for the last failed call on this thread ("" if none).  Valid until
 * the next call of this library on the same thread. */
const char* parrot_last_error(void);

/* PARROT_ABI_VERSION of the built library. */
int parrot_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PARROT_ATTN_H */
