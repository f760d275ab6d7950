/*
 * parrot_context -- host-side context store that produces the inputs of the
 * shared-prefix decode kernels (part of libparrot_attn; host memory only).
 *
 * A prompt is a token sequence with positions where a semantic variable ends
 * (Section 4.2, "Prompt structure-based analysis": a prefix hash is taken
 * after every semantic variable, so one prompt offers several shareable
 * prefixes).  The store keeps every such prefix it has seen in a trie keyed by
 * the hash of the segment that extends its parent prefix, with the segment's
 * tokens kept to confirm a hash hit (Section 5.3: a key-value store from
 * prefix hash to the requests that share it).  Each trie node owns the paged
 * KV blocks of its segment; a context (one request, Section 7's
 * Fill / Generate / FreeContext) owns the blocks of its tokens after its last
 * cached prefix and holds a reference on every node of its path.  A node is
 * released when no context references it.
 *
 * For a batch of contexts the store emits exactly the arrays
 * parrot_nested_prefix_decode and parrot_shared_prefix_prefill take: one group
 * per trie node on the batch's paths (parents numbered below children), each
 * group's prefix table, and each context's group, own-token table and
 * own-token count.
 *
 * The store is not thread-safe: one thread owns it.  All pointers are HOST
 * pointers.  Block ids are in [0, num_blocks) of the caller's KV pools.
 */
#ifndef PARROT_CONTEXT_H
#define PARROT_CONTEXT_H

#include <stdint.h>

#include "parrot_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct parrot_context_store parrot_context_store;

/* A store over `num_blocks` KV blocks of `block_size` tokens (block_size >= 1,
 * num_blocks >= 0).  Returns NULL on bad arguments or allocation failure. */
parrot_context_store* parrot_store_create(int32_t block_size, int32_t num_blocks);
void parrot_store_destroy(parrot_context_store* st);

/* Fill: register a prompt.  tokens[0..n) are its token ids (n >= 1);
 * boundaries[0..nb) are strictly increasing positions in [1, n] that end a
 * semantic variable.  Each prefix tokens[0..boundaries[k]) is looked up in the
 * trie and reused when cached, else created (its segment gets new blocks).
 * Tokens after the last boundary are the context's own tokens, in new private
 * blocks.  Returns the new context id (>= 0); -1 when the free blocks do not
 * suffice (nothing is changed then); -2 on bad arguments. */
int32_t parrot_store_fill(parrot_context_store* st, const int32_t* tokens, int32_t n,
                          const int32_t* boundaries, int32_t nb);

/* Generate: append one own token to a context (a new block every block_size
 * tokens).  PARROT_ERR_WORKSPACE_TOO_SMALL when no block is free. */
parrot_status parrot_store_append(parrot_context_store* st, int32_t ctx, int32_t token);

/* FreeContext: release the context's own blocks and its references. */
parrot_status parrot_store_free(parrot_context_store* st, int32_t ctx);

int32_t parrot_store_free_blocks(const parrot_context_store* st);
int32_t parrot_store_num_prefixes(const parrot_context_store* st);   /* cached trie nodes */
/* Tokens of a context: cached prefix tokens of its path and own tokens
 * (-1 for an unknown context). */
int32_t parrot_store_prefix_tokens(const parrot_context_store* st, int32_t ctx);
int32_t parrot_store_own_tokens(const parrot_context_store* st, int32_t ctx);

/* Sizes of the arrays parrot_store_build_batch fills for contexts ctxs[0..R). */
typedef struct {
  int32_t num_groups;           /* trie nodes on the contexts' paths */
  int32_t max_group_size;       /* contexts reading any one node */
  int32_t max_prefix_len;       /* longest node segment */
  int32_t max_suffix_len;       /* most own tokens */
  int32_t max_prefix_depth;     /* longest path */
  int32_t prefix_table_stride;  /* blocks of the longest segment (>= 1) */
  int32_t suffix_table_stride;  /* blocks of the most own tokens (>= 1) */
} parrot_batch_shape;

parrot_status parrot_store_batch_shape(const parrot_context_store* st, const int32_t* ctxs,
                                       int32_t R, parrot_batch_shape* shape);

/* Fill the batch arrays (sizes from parrot_store_batch_shape with the same
 * contexts): group_ids[R], suffix_lens[R], suffix_tables[R][suffix_table_stride],
 * prefix_lens[NG], prefix_parents[NG], prefix_tables[NG][prefix_table_stride].
 * Unused table entries are set to `pad_block`.  Groups are numbered in
 * breadth-first order of the trie, so every parent is below its children. */
parrot_status parrot_store_build_batch(const parrot_context_store* st, const int32_t* ctxs,
                                       int32_t R, int32_t pad_block, int32_t* group_ids,
                                       int32_t* suffix_lens, int32_t* suffix_tables,
                                       int32_t* prefix_lens, int32_t* prefix_parents,
                                       int32_t* prefix_tables);

#ifdef __cplusplus
}
#endif

#endif /* PARROT_CONTEXT_H */
