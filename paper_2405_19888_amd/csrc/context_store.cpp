// Host-side context store: a trie of cached prompt prefixes (split where a
// semantic variable ends), paged KV block allocation with reference counts,
// and the batch arrays of parrot_nested_prefix_decode.  Host code only.
#include <algorithm>
#include <cstdint>
#include <unordered_map>
#include <vector>

#include "parrot_context.h"
#include "errors.h"

namespace {

// FNV-1a over the segment's token ids, seeded with the parent's hash, so a
// node's hash covers its whole prefix.
uint64_t segment_hash(uint64_t seed, const int32_t* t, int32_t n) {
  uint64_t h = seed ^ 0xcbf29ce484222325ull;
  for (int32_t i = 0; i < n; ++i) {
    uint32_t x = static_cast<uint32_t>(t[i]);
    for (int b = 0; b < 4; ++b) {
      h ^= (x >> (8 * b)) & 0xffu;
      h *= 0x100000001b3ull;
    }
  }
  return h;
}

struct Node {
  int32_t parent = -1;             // node id, -1 for a child of the root
  int32_t depth = 0;               // 1 for a child of the root
  uint64_t hash = 0;               // hash of the whole prefix
  std::vector<int32_t> tokens;     // this node's segment
  std::vector<int32_t> blocks;     // KV blocks of the segment
  int32_t refs = 0;                // contexts whose path holds this node
  bool live = false;
};

struct Context {
  bool live = false;
  int32_t node = -1;               // deepest cached prefix, -1 for none
  int32_t own = 0;                 // own tokens
  std::vector<int32_t> blocks;     // blocks of the own tokens
};

}  // namespace

struct parrot_context_store {
  int32_t B = 16;
  std::vector<int32_t> free_list;                 // free block ids (stack)
  std::vector<Node> nodes;
  std::vector<int32_t> free_nodes;
  std::vector<Context> ctxs;
  std::vector<int32_t> free_ctxs;
  // (parent node + 1, hash of the prefix) -> child node
  std::unordered_map<uint64_t, std::vector<int32_t>> children;
  int32_t live_nodes = 0;

  static uint64_t key(int32_t parent, uint64_t h) {
    return h ^ (0x9e3779b97f4a7c15ull * static_cast<uint64_t>(parent + 1));
  }
  int32_t blocks_for(int64_t tokens) const { return static_cast<int32_t>((tokens + B - 1) / B); }

  int32_t find_child(int32_t parent, uint64_t h, const int32_t* t, int32_t n) const {
    auto it = children.find(key(parent, h));
    if (it == children.end()) return -1;
    for (int32_t c : it->second) {
      const Node& nd = nodes[c];
      if (nd.live && nd.parent == parent && nd.hash == h &&
          nd.tokens.size() == static_cast<size_t>(n) && std::equal(nd.tokens.begin(), nd.tokens.end(), t))
        return c;
    }
    return -1;
  }
  int32_t take_block() {
    int32_t b = free_list.back();
    free_list.pop_back();
    return b;
  }
  void release_node(int32_t id) {
    Node& nd = nodes[id];
    for (int32_t b : nd.blocks) free_list.push_back(b);
    auto it = children.find(key(nd.parent, nd.hash));
    if (it != children.end()) {
      auto& v = it->second;
      v.erase(std::remove(v.begin(), v.end(), id), v.end());
      if (v.empty()) children.erase(it);
    }
    nd = Node();
    free_nodes.push_back(id);
    --live_nodes;
  }
  const Context* context(int32_t c) const {
    return (c >= 0 && c < static_cast<int32_t>(ctxs.size()) && ctxs[c].live) ? &ctxs[c] : nullptr;
  }
};

extern "C" {

parrot_context_store* parrot_store_create(int32_t block_size, int32_t num_blocks) {
  if (block_size < 1 || num_blocks < 0) return nullptr;
  auto* st = new (std::nothrow) parrot_context_store();
  if (!st) return nullptr;
  st->B = block_size;
  st->free_list.resize(num_blocks);
  // hand out low block ids first
  for (int32_t i = 0; i < num_blocks; ++i) st->free_list[i] = num_blocks - 1 - i;
  return st;
}

void parrot_store_destroy(parrot_context_store* st) { delete st; }

int32_t parrot_store_fill(parrot_context_store* st, const int32_t* tokens, int32_t n,
                          const int32_t* boundaries, int32_t nb) {
  if (!st || !tokens || n < 1 || nb < 0 || (nb > 0 && !boundaries)) return -2;
  for (int32_t k = 0; k < nb; ++k) {
    const int32_t lo = k ? boundaries[k - 1] : 0;
    if (boundaries[k] <= lo || boundaries[k] > n) return -2;
  }
  // walk the trie as far as the prefixes are cached, then count new blocks
  int32_t node = -1, k = 0, pos = 0;
  uint64_t h = 0;
  std::vector<uint64_t> hashes(nb);
  for (; k < nb; ++k) {
    const int32_t len = boundaries[k] - pos;
    const uint64_t hk = segment_hash(h, tokens + pos, len);
    const int32_t c = st->find_child(node, hk, tokens + pos, len);
    if (c < 0) break;
    node = c;
    h = hk;
    pos = boundaries[k];
  }
  int64_t need = 0;
  {
    uint64_t hh = h;
    int32_t p = pos;
    for (int32_t j = k; j < nb; ++j) {
      hashes[j] = segment_hash(hh, tokens + p, boundaries[j] - p);
      hh = hashes[j];
      need += st->blocks_for(boundaries[j] - p);
      p = boundaries[j];
    }
  }
  const int32_t own = n - (nb ? boundaries[nb - 1] : 0);
  need += st->blocks_for(own);
  if (need > static_cast<int64_t>(st->free_list.size())) return -1;

  // create the missing prefixes
  for (; k < nb; ++k) {
    int32_t id;
    if (!st->free_nodes.empty()) { id = st->free_nodes.back(); st->free_nodes.pop_back(); }
    else { id = static_cast<int32_t>(st->nodes.size()); st->nodes.emplace_back(); }
    Node& nd = st->nodes[id];
    nd.parent = node;
    nd.depth = node >= 0 ? st->nodes[node].depth + 1 : 1;
    nd.hash = hashes[k];
    nd.tokens.assign(tokens + pos, tokens + boundaries[k]);
    const int32_t nbk = st->blocks_for(boundaries[k] - pos);
    for (int32_t i = 0; i < nbk; ++i) nd.blocks.push_back(st->take_block());
    nd.live = true;
    st->children[parrot_context_store::key(node, nd.hash)].push_back(id);
    ++st->live_nodes;
    node = id;
    pos = boundaries[k];
  }
  // the context: references on its path, own blocks
  int32_t cid;
  if (!st->free_ctxs.empty()) { cid = st->free_ctxs.back(); st->free_ctxs.pop_back(); }
  else { cid = static_cast<int32_t>(st->ctxs.size()); st->ctxs.emplace_back(); }
  Context& c = st->ctxs[cid];
  c = Context();
  c.live = true;
  c.node = node;
  c.own = own;
  for (int32_t i = 0, nbo = st->blocks_for(own); i < nbo; ++i) c.blocks.push_back(st->take_block());
  for (int32_t x = node; x >= 0; x = st->nodes[x].parent) ++st->nodes[x].refs;
  return cid;
}

parrot_status parrot_store_append(parrot_context_store* st, int32_t ctx, int32_t token) {
  (void)token;   // the store tracks blocks; the token's KV is written by the decode step
  if (!st || !st->context(ctx)) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "unknown context %d", ctx);
  Context& c = st->ctxs[ctx];
  if (c.own % st->B == 0) {
    if (st->free_list.empty())
      return parrot::set_error(PARROT_ERR_WORKSPACE_TOO_SMALL, "no free KV block for context %d", ctx);
    c.blocks.push_back(st->take_block());
  }
  ++c.own;
  return parrot::set_error(PARROT_OK, "");
}

parrot_status parrot_store_free(parrot_context_store* st, int32_t ctx) {
  if (!st || !st->context(ctx)) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "unknown context %d", ctx);
  Context& c = st->ctxs[ctx];
  for (int32_t b : c.blocks) st->free_list.push_back(b);
  for (int32_t x = c.node; x >= 0;) {
    const int32_t parent = st->nodes[x].parent;
    if (--st->nodes[x].refs == 0) st->release_node(x);
    x = parent;
  }
  c = Context();
  st->free_ctxs.push_back(ctx);
  return parrot::set_error(PARROT_OK, "");
}

int32_t parrot_store_free_blocks(const parrot_context_store* st) {
  return st ? static_cast<int32_t>(st->free_list.size()) : -1;
}

int32_t parrot_store_num_prefixes(const parrot_context_store* st) { return st ? st->live_nodes : -1; }

int32_t parrot_store_prefix_tokens(const parrot_context_store* st, int32_t ctx) {
  const Context* c = st ? st->context(ctx) : nullptr;
  if (!c) return -1;
  int64_t n = 0;
  for (int32_t x = c->node; x >= 0; x = st->nodes[x].parent) n += st->nodes[x].tokens.size();
  return static_cast<int32_t>(n);
}

int32_t parrot_store_own_tokens(const parrot_context_store* st, int32_t ctx) {
  const Context* c = st ? st->context(ctx) : nullptr;
  return c ? c->own : -1;
}

}  // extern "C"

namespace {

// The batch's groups: every node on the listed contexts' paths, breadth-first
// (by depth, then by node id), so a parent is numbered below its children.
parrot_status batch_groups(const parrot_context_store* st, const int32_t* ctxs, int32_t R,
                           std::vector<int32_t>* order, std::unordered_map<int32_t, int32_t>* index,
                           std::vector<int32_t>* readers) {
  if (!st) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "store is NULL");
  if (R < 0 || (R > 0 && !ctxs)) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "bad context list");
  std::unordered_map<int32_t, int32_t> count;
  for (int32_t i = 0; i < R; ++i) {
    const Context* c = st->context(ctxs[i]);
    if (!c) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "unknown context %d", ctxs[i]);
    for (int32_t x = c->node; x >= 0; x = st->nodes[x].parent) ++count[x];
  }
  order->clear();
  for (auto& kv : count) order->push_back(kv.first);
  std::sort(order->begin(), order->end(), [&](int32_t a, int32_t b) {
    const int32_t da = st->nodes[a].depth, db = st->nodes[b].depth;
    return da != db ? da < db : a < b;
  });
  index->clear();
  readers->assign(order->size(), 0);
  for (size_t g = 0; g < order->size(); ++g) {
    (*index)[(*order)[g]] = static_cast<int32_t>(g);
    (*readers)[g] = count[(*order)[g]];
  }
  return PARROT_OK;
}

}  // namespace

extern "C" {

parrot_status parrot_store_batch_shape(const parrot_context_store* st, const int32_t* ctxs,
                                       int32_t R, parrot_batch_shape* shape) {
  if (!shape) return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "shape is NULL");
  std::vector<int32_t> order, readers;
  std::unordered_map<int32_t, int32_t> index;
  parrot_status s = batch_groups(st, ctxs, R, &order, &index, &readers);
  if (s != PARROT_OK) return s;
  parrot_batch_shape sh{};
  sh.num_groups = static_cast<int32_t>(order.size());
  for (size_t g = 0; g < order.size(); ++g) {
    const Node& nd = st->nodes[order[g]];
    sh.max_group_size = std::max(sh.max_group_size, readers[g]);
    sh.max_prefix_len = std::max(sh.max_prefix_len, static_cast<int32_t>(nd.tokens.size()));
    sh.max_prefix_depth = std::max(sh.max_prefix_depth, nd.depth);
  }
  for (int32_t i = 0; i < R; ++i) sh.max_suffix_len = std::max(sh.max_suffix_len, st->ctxs[ctxs[i]].own);
  sh.prefix_table_stride = std::max(1, st->blocks_for(sh.max_prefix_len));
  sh.suffix_table_stride = std::max(1, st->blocks_for(sh.max_suffix_len));
  *shape = sh;
  return parrot::set_error(PARROT_OK, "");
}

parrot_status parrot_store_build_batch(const parrot_context_store* st, const int32_t* ctxs,
                                       int32_t R, int32_t pad_block, int32_t* group_ids,
                                       int32_t* suffix_lens, int32_t* suffix_tables,
                                       int32_t* prefix_lens, int32_t* prefix_parents,
                                       int32_t* prefix_tables) {
  parrot_batch_shape sh;
  parrot_status s = parrot_store_batch_shape(st, ctxs, R, &sh);
  if (s != PARROT_OK) return s;
  if (R > 0 && (!group_ids || !suffix_lens || !suffix_tables))
    return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "request arrays are NULL");
  if (sh.num_groups > 0 && (!prefix_lens || !prefix_parents || !prefix_tables))
    return parrot::set_error(PARROT_ERR_INVALID_ARGUMENT, "group arrays are NULL");
  std::vector<int32_t> order, readers;
  std::unordered_map<int32_t, int32_t> index;
  batch_groups(st, ctxs, R, &order, &index, &readers);
  for (size_t g = 0; g < order.size(); ++g) {
    const Node& nd = st->nodes[order[g]];
    prefix_lens[g] = static_cast<int32_t>(nd.tokens.size());
    prefix_parents[g] = nd.parent >= 0 ? index.at(nd.parent) : -1;
    int32_t* row = prefix_tables + g * static_cast<size_t>(sh.prefix_table_stride);
    for (int32_t j = 0; j < sh.prefix_table_stride; ++j)
      row[j] = j < static_cast<int32_t>(nd.blocks.size()) ? nd.blocks[j] : pad_block;
  }
  for (int32_t i = 0; i < R; ++i) {
    const Context& c = st->ctxs[ctxs[i]];
    group_ids[i] = c.node >= 0 ? index.at(c.node) : -1;
    suffix_lens[i] = c.own;
    int32_t* row = suffix_tables + i * static_cast<size_t>(sh.suffix_table_stride);
    for (int32_t j = 0; j < sh.suffix_table_stride; ++j)
      row[j] = j < static_cast<int32_t>(c.blocks.size()) ? c.blocks[j] : pad_block;
  }
  return parrot::set_error(PARROT_OK, "");
}

}  // extern "C"
