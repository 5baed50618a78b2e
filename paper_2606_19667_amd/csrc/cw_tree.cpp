// Knowledge tree and evidence orderings (host half of libcw).
//
// Paper Sec. 3.2: a trie whose root-to-node paths are the document orders of
// recently served requests. Sec. 3.3 (Eq. 1, Algorithm 1): the greedy walk that
// orders a retrieved set so its leading documents follow a cached path, and the
// exhaustive argmax it approximates. Sec. 3.4: recency stands in for residency
// (a node is cached when an order served within the last `window` insertions
// passed through it) and the optional feedback marks a path stale when the
// engine did not actually reuse it. Sec. 4 and Table `baselines`: retrieval
// order, lexicographic sorting and a recency heuristic as baselines.
//
// Layout: nodes live in one flat array (index 0 is the root); a child is found
// through an open-addressing index keyed by (parent, document), and each node
// also lists its children (first child, next sibling) for walks that visit
// every child of a node. Every
// `window` insertions the nodes that left the window are dropped and both
// arrays are rebuilt, which keeps the tree at O(window * k) nodes. A node is
// always created after its parent and compaction keeps the order, so a
// parent's index is below its children's.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "cw_internal.h"

namespace {

constexpr int32_t kMaxDocs = 4096;       // documents per call
constexpr int64_t kNever = std::numeric_limits<int64_t>::min();

// splitmix64's output mix (Steele, Lea and Flood, OOPSLA 2014).
inline uint64_t mix64(uint64_t x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ULL;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebULL;
  x ^= x >> 31;
  return x;
}

struct Node {
  int64_t doc;
  int64_t last;    // clock of the latest insertion through this node
  int64_t stale;   // clock of the latest stale mark, kNever if none
  int32_t parent;
  int32_t first_child = -1;    // children of a node form a singly linked list
  int32_t next_sibling = -1;
};

// (parent, doc) -> node index; linear probing, capacity a power of two kept
// at least twice the number of entries. Entries are never removed one by one:
// the whole index is rebuilt on compaction.
struct ChildIndex {
  std::vector<int64_t> doc;
  std::vector<int32_t> parent;
  std::vector<int32_t> node;   // -1 = empty slot
  uint64_t mask = 0;
  size_t count = 0;

  void reset(size_t min_entries) {
    size_t cap = 16;
    while (cap < 2 * min_entries + 2) cap <<= 1;
    doc.assign(cap, 0);
    parent.assign(cap, 0);
    node.assign(cap, -1);
    mask = cap - 1;
    count = 0;
  }
  static uint64_t key(int32_t p, int64_t d) { return mix64(uint64_t(d) * 0x9E3779B97F4A7C15ULL ^ uint64_t(uint32_t(p))); }
  int32_t find(int32_t p, int64_t d) const {
    for (uint64_t i = key(p, d) & mask;; i = (i + 1) & mask) {
      if (node[i] < 0) return -1;
      if (parent[i] == p && doc[i] == d) return node[i];
    }
  }
  // The pair must be absent; the caller keeps 2 * (count + 1) <= capacity.
  void put(int32_t p, int64_t d, int32_t n) {
    uint64_t i = key(p, d) & mask;
    while (node[i] >= 0) i = (i + 1) & mask;
    doc[i] = d;
    parent[i] = p;
    node[i] = n;
    ++count;
  }
};

// doc -> clock of its latest insertion (for the recency baseline).
struct DocClock {
  std::vector<int64_t> doc;
  std::vector<int64_t> when;   // kNever = empty slot
  uint64_t mask = 0;
  size_t count = 0;

  void reset(size_t min_entries) {
    size_t cap = 16;
    while (cap < 2 * min_entries + 2) cap <<= 1;
    doc.assign(cap, 0);
    when.assign(cap, kNever);
    mask = cap - 1;
    count = 0;
  }
  int64_t get(int64_t d) const {
    for (uint64_t i = mix64(uint64_t(d)) & mask;; i = (i + 1) & mask) {
      if (when[i] == kNever) return kNever;
      if (doc[i] == d) return when[i];
    }
  }
  void set(int64_t d, int64_t t) {
    if (2 * (count + 1) > doc.size()) grow();
    uint64_t i = mix64(uint64_t(d)) & mask;
    while (when[i] != kNever && doc[i] != d) i = (i + 1) & mask;
    if (when[i] == kNever) ++count;
    doc[i] = d;
    when[i] = t;
  }
  void grow() {
    std::vector<int64_t> od = std::move(doc), ow = std::move(when);
    reset(2 * count + 8);
    for (size_t i = 0; i < od.size(); ++i)
      if (ow[i] != kNever) set(od[i], ow[i]);
  }
};

}  // namespace

struct cw_tree {
  int64_t window = 1;
  int64_t clock = 0;
  std::vector<Node> nodes;   // nodes[0] is the root
  ChildIndex kids;
  DocClock docs;

  bool cached(int32_t n) const {
    const Node& x = nodes[size_t(n)];
    return x.last > clock - window && x.stale < x.last;
  }
  // The child of node p for document d, or -1.
  int32_t child(int32_t p, int64_t d) const { return kids.find(p, d); }

  void reserve_child() {
    if (2 * (kids.count + 1) <= kids.node.size()) return;
    rebuild_index(2 * kids.count + 8);
  }
  void rebuild_index(size_t min_entries) {
    kids.reset(min_entries);
    for (size_t i = 1; i < nodes.size(); ++i) kids.put(nodes[i].parent, nodes[i].doc, int32_t(i));
  }
  // Appends node c (already in `nodes`, parent set) to its parent's child list.
  void link_child(int32_t c) {
    Node& p = nodes[size_t(nodes[size_t(c)].parent)];
    nodes[size_t(c)].next_sibling = p.first_child;
    p.first_child = c;
  }
  // Drops every node that left the window (its subtree left with it: a
  // child's insertion clock never exceeds its parent's) and old document clocks.
  void prune() {
    std::vector<int32_t> remap(nodes.size(), -1);
    std::vector<Node> kept;
    kept.reserve(nodes.size());
    remap[0] = 0;
    kept.push_back(nodes[0]);
    for (size_t i = 1; i < nodes.size(); ++i) {
      const Node& x = nodes[i];
      if (x.last <= clock - window) continue;
      Node y = x;
      y.parent = remap[size_t(x.parent)];
      remap[i] = int32_t(kept.size());
      kept.push_back(y);
    }
    nodes.swap(kept);
    for (Node& x : nodes) x.first_child = x.next_sibling = -1;
    for (size_t i = 1; i < nodes.size(); ++i) link_child(int32_t(i));
    rebuild_index(nodes.size());
    DocClock fresh;
    fresh.reset(docs.count);
    for (size_t i = 0; i < docs.doc.size(); ++i)
      if (docs.when[i] != kNever && docs.when[i] > clock - window) fresh.set(docs.doc[i], docs.when[i]);
    docs = std::move(fresh);
  }
};

namespace {

cw_status check_docs(const char* what, const int64_t* docs, int32_t k, std::vector<int64_t>* sorted_out) {
  if (k < 0 || k > kMaxDocs)
    return cw::fail(CW_EINVAL, std::string(what) + ": document count must be in [0, 4096]");
  if (k > 0 && !docs) return cw::fail(CW_EINVAL, std::string(what) + ": documents pointer is NULL");
  sorted_out->assign(docs, docs + k);
  std::sort(sorted_out->begin(), sorted_out->end());
  if (std::adjacent_find(sorted_out->begin(), sorted_out->end()) != sorted_out->end())
    return cw::fail(CW_EINVAL, std::string(what) + ": documents must be distinct");
  return CW_OK;
}

// l(O, T): leading documents of `order` along cached nodes; counts lookups.
int32_t walk(const cw_tree* t, const int64_t* order, int32_t k, int32_t* probes) {
  int32_t node = 0, n = 0;
  while (n < k) {
    ++*probes;
    const int32_t c = t->child(node, order[n]);
    if (c < 0 || !t->cached(c)) break;
    node = c;
    ++n;
  }
  return n;
}

// Greedy order (Sec. 3.3, Algorithm 1), by what each level selects: among the
// cached children of the current node whose document is in the retrieved set
// and not yet placed, the one of lowest retrieval rank; the run ends at a node
// with no such child and the unplaced documents follow in retrieval rank.
// The children are visited through the node's child list; a rank table sorted
// by document ID maps a child's document to its rank. *probes gets the child
// lookups a scan in retrieval rank would make for the same choices: at a level
// that places rank j, one per unplaced rank <= j; at the level that finds
// nothing (when documents remain), one per unplaced document.
int32_t greedy(const cw_tree* t, const int64_t* docs, int32_t k, int64_t* out, int32_t* probes) {
  std::vector<std::pair<int64_t, int32_t>> by_doc(static_cast<size_t>(k));
  for (int32_t j = 0; j < k; ++j) by_doc[size_t(j)] = {docs[j], j};
  std::sort(by_doc.begin(), by_doc.end());
  auto rank_of = [&](int64_t d) -> int32_t {
    auto it = std::lower_bound(by_doc.begin(), by_doc.end(), std::make_pair(d, int32_t(-1)));
    return (it != by_doc.end() && it->first == d) ? it->second : -1;
  };
  std::vector<char> placed(static_cast<size_t>(k), 0);
  int32_t node = 0, depth = 0;
  while (depth < k) {
    int32_t best = k, best_node = -1;
    for (int32_t c = t->nodes[size_t(node)].first_child; c >= 0; c = t->nodes[size_t(c)].next_sibling) {
      if (!t->cached(c)) continue;
      const int32_t j = rank_of(t->nodes[size_t(c)].doc);
      if (j >= 0 && j < best && !placed[size_t(j)]) {
        best = j;
        best_node = c;
      }
    }
    int32_t scanned = 0;   // unplaced ranks up to the pick (all of them when none)
    for (int32_t j = 0; j < k && j <= best; ++j) scanned += placed[size_t(j)] ? 0 : 1;
    *probes += scanned;
    if (best_node < 0) break;
    placed[size_t(best)] = 1;
    out[depth++] = docs[best];
    node = best_node;
  }
  int32_t n = depth;
  for (int32_t j = 0; j < k; ++j)
    if (!placed[size_t(j)]) out[n++] = docs[j];
  return depth;
}

// Eq. 1 argmax. Every permutation's reusable run is a cached path of distinct
// documents of D from the root, so the search is a depth-first walk over those
// paths instead of over k! orders. Children are tried in retrieval rank, and a
// run replaces the best only when strictly deeper, so among equally deep runs
// the first in lexicographic order of retrieval ranks wins.
struct Exhaustive {
  const cw_tree* t;
  const int64_t* docs;
  int32_t k;
  int32_t* probes;
  std::vector<char> used;
  std::vector<int32_t> path, best;

  void dfs(int32_t node) {
    if (path.size() > best.size()) best = path;
    for (int32_t j = 0; j < k; ++j) {
      if (used[size_t(j)]) continue;
      ++*probes;
      const int32_t c = t->child(node, docs[j]);
      if (c < 0 || !t->cached(c)) continue;
      used[size_t(j)] = 1;
      path.push_back(j);
      dfs(c);
      path.pop_back();
      used[size_t(j)] = 0;
    }
  }
};

int32_t exhaustive(const cw_tree* t, const int64_t* docs, int32_t k, int64_t* out, int32_t* probes) {
  Exhaustive e{t, docs, k, probes, std::vector<char>(size_t(k), 0), {}, {}};
  e.path.reserve(size_t(k));
  e.dfs(0);
  std::vector<char> taken(size_t(k), 0);
  int32_t n = 0;
  for (int32_t j : e.best) {
    out[n++] = docs[j];
    taken[size_t(j)] = 1;
  }
  for (int32_t j = 0; j < k; ++j)
    if (!taken[size_t(j)]) out[n++] = docs[j];
  return int32_t(e.best.size());
}

// Recency heuristic: documents served within the window first, latest first
// (ties in retrieval rank), then the others in retrieval rank.
void recency(const cw_tree* t, const int64_t* docs, int32_t k, int64_t* out) {
  std::vector<std::pair<int64_t, int32_t>> key(static_cast<size_t>(k));
  for (int32_t j = 0; j < k; ++j) {
    const int64_t w = t->docs.get(docs[j]);
    key[size_t(j)] = {w > t->clock - t->window ? -w : std::numeric_limits<int64_t>::max(), j};
  }
  std::sort(key.begin(), key.end());
  for (int32_t j = 0; j < k; ++j) out[j] = docs[key[size_t(j)].second];
}

}  // namespace

extern "C" cw_status cw_tree_create(int32_t window, cw_tree** out) {
  if (!out) return cw::fail(CW_EINVAL, "tree_create: out is NULL");
  *out = nullptr;
  if (window < 1) return cw::fail(CW_EINVAL, "tree_create: window must be >= 1");
  cw_tree* t = new (std::nothrow) cw_tree;
  if (!t) return cw::fail(CW_ENOSPC, "tree_create: out of host memory");
  t->window = window;
  t->nodes.push_back(Node{0, std::numeric_limits<int64_t>::max(), kNever, -1});
  t->kids.reset(64);
  t->docs.reset(64);
  *out = t;
  return cw::ok();
}

extern "C" void cw_tree_destroy(cw_tree* tree) { delete tree; }

extern "C" int64_t cw_tree_num_nodes(const cw_tree* tree) {
  return tree ? int64_t(tree->nodes.size()) - 1 : -1;
}

extern "C" cw_status cw_tree_insert(cw_tree* tree, const int64_t* order, int32_t k) {
  if (!tree) return cw::fail(CW_EINVAL, "tree_insert: tree is NULL");
  std::vector<int64_t> s;
  cw_status st = check_docs("tree_insert", order, k, &s);
  if (st != CW_OK) return st;
  const int64_t now = ++tree->clock;
  int32_t node = 0;
  for (int32_t j = 0; j < k; ++j) {
    int32_t c = tree->child(node, order[j]);
    if (c < 0) {
      tree->reserve_child();
      c = int32_t(tree->nodes.size());
      tree->nodes.push_back(Node{order[j], now, kNever, node});
      tree->link_child(c);
      tree->kids.put(node, order[j], c);
    }
    tree->nodes[size_t(c)].last = now;
    tree->docs.set(order[j], now);
    node = c;
  }
  if (now % tree->window == 0) tree->prune();
  return cw::ok();
}

extern "C" cw_status cw_tree_mark_stale(cw_tree* tree, const int64_t* order, int32_t k,
                                        int32_t observed_depth) {
  if (!tree) return cw::fail(CW_EINVAL, "tree_mark_stale: tree is NULL");
  std::vector<int64_t> s;
  cw_status st = check_docs("tree_mark_stale", order, k, &s);
  if (st != CW_OK) return st;
  if (observed_depth < 0 || observed_depth > k)
    return cw::fail(CW_EINVAL, "tree_mark_stale: observed_depth must be in [0, k]");
  int32_t node = 0;
  for (int32_t j = 0; j < k; ++j) {
    const int32_t c = tree->child(node, order[j]);
    if (c < 0) break;
    if (j >= observed_depth) tree->nodes[size_t(c)].stale = tree->clock;
    node = c;
  }
  return cw::ok();
}

extern "C" cw_status cw_tree_order(const cw_tree* tree, int32_t strategy, const int64_t* docs, int32_t k,
                                   int64_t* out_order, int32_t* out_depth, int32_t* out_probes) {
  if (!tree) return cw::fail(CW_EINVAL, "tree_order: tree is NULL");
  if (k > 0 && !out_order) return cw::fail(CW_EINVAL, "tree_order: out_order is NULL");
  std::vector<int64_t> s;
  cw_status st = check_docs("tree_order", docs, k, &s);
  if (st != CW_OK) return st;
  int32_t probes = 0, depth = 0;
  switch (strategy) {
    case CW_ORDER_RETRIEVAL:
      std::copy(docs, docs + k, out_order);
      depth = walk(tree, out_order, k, &probes);
      break;
    case CW_ORDER_SORTED:
      std::copy(s.begin(), s.end(), out_order);
      depth = walk(tree, out_order, k, &probes);
      break;
    case CW_ORDER_RECENCY:
      recency(tree, docs, k, out_order);
      depth = walk(tree, out_order, k, &probes);
      break;
    case CW_ORDER_GREEDY:
      depth = greedy(tree, docs, k, out_order, &probes);
      break;
    case CW_ORDER_EXHAUSTIVE:
      depth = exhaustive(tree, docs, k, out_order, &probes);
      break;
    default:
      return cw::fail(CW_EINVAL, "tree_order: unknown strategy");
  }
  if (out_depth) *out_depth = depth;
  if (out_probes) *out_probes = probes;
  return cw::ok();
}
