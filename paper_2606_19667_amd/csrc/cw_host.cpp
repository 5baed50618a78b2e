// Host half of libcw: status reporting, chained block hashes, the block pool
// with prefix lookup, batch scheduling, and the attention tile planner.
//
// Paper Sec. 2.1 (with Fig. 1): KV memory lives in fixed-size token blocks;
// each block is hashed together with its prefix history and a new prompt
// reuses the longest leading run of stored blocks. Sec. 3.4: residency and
// eviction belong to the engine. The hash function is not named in the paper;
// this library uses XXH64 keyed by the previous block's hash.

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>
#include <string>
#include <unordered_map>
#include <vector>

#include "cw_internal.h"

static_assert(__BYTE_ORDER__ == __ORDER_LITTLE_ENDIAN__, "token bytes are hashed in host order");

namespace {
thread_local std::string g_last_error;
}

namespace cw {

cw_status fail(cw_status status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

cw_status ok() {
  g_last_error.clear();
  return CW_OK;
}

cw_status check_batch(const int32_t* cu, const int32_t* plen, int32_t batch, int32_t block_size,
                      int32_t bt_stride, int64_t* total_rows) {
  if (batch < 1) return fail(CW_EINVAL, "batch must be >= 1");
  if (!cu || !plen) return fail(CW_EINVAL, "cu_suffix_host and prefix_len_host are required");
  if (block_size < 1) return fail(CW_EINVAL, "block_size must be >= 1");
  if (bt_stride < 1) return fail(CW_EINVAL, "bt_stride must be >= 1");
  if (cu[0] != 0) return fail(CW_EINVAL, "cu_suffix[0] must be 0");
  for (int32_t r = 0; r < batch; ++r) {
    if (cu[r + 1] < cu[r]) return fail(CW_EINVAL, "cu_suffix must be non-decreasing");
    if (plen[r] < 0 || plen[r] % block_size != 0)
      return fail(CW_EINVAL, "prefix_len[" + std::to_string(r) + "] = " + std::to_string(plen[r]) +
                                 " is not a non-negative multiple of the block size");
    const int64_t L = int64_t(plen[r]) + (cu[r + 1] - cu[r]);
    const int64_t nb = (L + block_size - 1) / block_size;
    if (nb > bt_stride)
      return fail(CW_EINVAL, "request " + std::to_string(r) + " needs " + std::to_string(nb) +
                                 " blocks but bt_stride is " + std::to_string(bt_stride));
  }
  if (total_rows) *total_rows = cu[batch];
  return CW_OK;
}

int64_t count_tiles(const int32_t* cu, int32_t batch, int32_t hkv, int32_t per_tile) {
  int64_t n = 0;
  for (int32_t r = 0; r < batch; ++r) n += (int64_t(cu[r + 1] - cu[r]) + per_tile - 1) / per_tile;
  return n * hkv;
}

}  // namespace cw

using cw::fail;

extern "C" int32_t cw_abi_version(void) { return CW_ABI_VERSION; }

extern "C" const char* cw_last_error(void) { return g_last_error.c_str(); }

// ---------------------------------------------------------------------------
// XXH64 (the published xxHash 64-bit algorithm: four accumulator lanes over
// 32-byte stripes, 8/4/1-byte tails, final avalanche).
// ---------------------------------------------------------------------------
namespace {
constexpr uint64_t kP1 = 0x9E3779B185EBCA87ULL;
constexpr uint64_t kP2 = 0xC2B2AE3D27D4EB4FULL;
constexpr uint64_t kP3 = 0x165667B19E3779F9ULL;
constexpr uint64_t kP4 = 0x85EBCA77C2B2AE63ULL;
constexpr uint64_t kP5 = 0x27D4EB2F165667C5ULL;

inline uint64_t rotl64(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }
inline uint64_t rd64(const uint8_t* p) { uint64_t v; std::memcpy(&v, p, 8); return v; }
inline uint32_t rd32(const uint8_t* p) { uint32_t v; std::memcpy(&v, p, 4); return v; }
inline uint64_t xround(uint64_t acc, uint64_t lane) { return rotl64(acc + lane * kP2, 31) * kP1; }
inline uint64_t xmerge(uint64_t acc, uint64_t v) { return (acc ^ xround(0, v)) * kP1 + kP4; }

uint64_t xxh64(const uint8_t* p, size_t n, uint64_t seed) {
  const uint8_t* end = p + n;
  uint64_t acc;
  if (n >= 32) {
    uint64_t v1 = seed + kP1 + kP2, v2 = seed + kP2, v3 = seed, v4 = seed - kP1;
    for (; p + 32 <= end; p += 32) {
      v1 = xround(v1, rd64(p));
      v2 = xround(v2, rd64(p + 8));
      v3 = xround(v3, rd64(p + 16));
      v4 = xround(v4, rd64(p + 24));
    }
    acc = rotl64(v1, 1) + rotl64(v2, 7) + rotl64(v3, 12) + rotl64(v4, 18);
    acc = xmerge(acc, v1);
    acc = xmerge(acc, v2);
    acc = xmerge(acc, v3);
    acc = xmerge(acc, v4);
  } else {
    acc = seed + kP5;
  }
  acc += n;
  for (; p + 8 <= end; p += 8) acc = rotl64(acc ^ xround(0, rd64(p)), 27) * kP1 + kP4;
  if (p + 4 <= end) {
    acc = rotl64(acc ^ (uint64_t(rd32(p)) * kP1), 23) * kP2 + kP3;
    p += 4;
  }
  for (; p < end; ++p) acc = rotl64(acc ^ (uint64_t(*p) * kP5), 11) * kP1;
  acc ^= acc >> 33;
  acc *= kP2;
  acc ^= acc >> 29;
  acc *= kP3;
  acc ^= acc >> 32;
  return acc;
}

void chain_hashes(const int32_t* tokens, int64_t n_tokens, int32_t bs, uint64_t* out) {
  uint64_t h = 0;
  const int64_t nb = n_tokens / bs;
  for (int64_t b = 0; b < nb; ++b) {
    h = xxh64(reinterpret_cast<const uint8_t*>(tokens + b * bs), size_t(bs) * 4, h);
    out[b] = h;
  }
}
}  // namespace

extern "C" cw_status cw_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block_size,
                                     uint64_t* out_hashes) {
  if (n_tokens < 0) return fail(CW_EINVAL, "n_tokens must be >= 0");
  if (block_size < 1) return fail(CW_EINVAL, "block_size must be >= 1");
  if (n_tokens / block_size > 0 && (!tokens || !out_hashes))
    return fail(CW_EINVAL, "tokens and out_hashes are required");
  chain_hashes(tokens, n_tokens, block_size, out_hashes);
  return cw::ok();
}

// ---------------------------------------------------------------------------
// Block pool. The free queue is a doubly linked list threaded through
// prev/next (index n is the sentinel). Unlinking leaves a node's own links in
// place, so an undo log replayed in reverse can relink nodes exactly. Stored
// hashes live in a flat open-addressing index, so a pool is a handful of
// arrays and cloning one is a few memory copies.
// ---------------------------------------------------------------------------
namespace {

// Map from stored block hash to block ID: linear probing, backward-shift
// deletion, capacity a power of two >= 2 * num_blocks (each block stores at
// most one hash, so the load factor stays <= 1/2).
struct HashIndex {
  std::vector<uint64_t> key;
  std::vector<int32_t> val;  // -1 marks an empty slot
  uint64_t mask = 0;
  int shift = 64;

  void init(int32_t nblocks) {
    size_t cap = 16;
    int lg = 4;
    while (cap < 2 * size_t(nblocks)) {
      cap <<= 1;
      ++lg;
    }
    key.assign(cap, 0);
    val.assign(cap, -1);
    mask = cap - 1;
    shift = 64 - lg;
  }
  size_t home(uint64_t k) const { return size_t((k * 0x9E3779B97F4A7C15ULL) >> shift); }
  int32_t find(uint64_t k) const {
    for (size_t i = home(k);; i = (i + 1) & mask) {
      if (val[i] < 0) return -1;
      if (key[i] == k) return val[i];
    }
  }
  // Caller guarantees k is absent.
  void insert(uint64_t k, int32_t v) {
    size_t i = home(k);
    while (val[i] >= 0) i = (i + 1) & mask;
    key[i] = k;
    val[i] = v;
  }
  void erase(uint64_t k) {
    size_t i = home(k);
    while (true) {
      if (val[i] < 0) return;
      if (key[i] == k) break;
      i = (i + 1) & mask;
    }
    size_t j = i;
    while (true) {
      j = (j + 1) & mask;
      if (val[j] < 0) break;
      const size_t h = home(key[j]);
      if (((j - h) & mask) >= ((j - i) & mask)) {  // entry j may move back into the hole
        key[i] = key[j];
        val[i] = val[j];
        i = j;
      }
    }
    val[i] = -1;
  }
};

}  // namespace

struct cw_pool {
  int32_t n = 0;
  std::vector<int32_t> ref;
  std::vector<uint64_t> hash;
  std::vector<uint8_t> has_hash;
  std::vector<int32_t> prev, next;
  int32_t nfree = 0;
  HashIndex table;

  void unlink(int32_t b) {
    next[prev[b]] = next[b];
    prev[next[b]] = prev[b];
    --nfree;
  }
  void relink(int32_t b) {  // inverse of the most recent unlink(b)
    next[prev[b]] = b;
    prev[next[b]] = b;
    ++nfree;
  }
  void push_back(int32_t b) {
    const int32_t s = n;
    prev[b] = prev[s];
    next[b] = s;
    next[prev[s]] = b;
    prev[s] = b;
    ++nfree;
  }
  int32_t front() const { return next[n]; }
};

namespace {

// Mutations made by a multi-step call, undone in reverse on failure.
struct UndoLog {
  enum Kind : uint8_t { kAcquireFree, kAcquireHeld, kAlloc, kCommit };
  struct Entry {
    Kind kind;
    uint8_t had_hash;
    int32_t block;
    uint64_t hash;
  };
  std::vector<Entry> entries;

  void rollback(cw_pool* p) {
    for (auto it = entries.rbegin(); it != entries.rend(); ++it) {
      const int32_t b = it->block;
      switch (it->kind) {
        case kAcquireFree:
          p->ref[b] = 0;
          p->relink(b);
          break;
        case kAcquireHeld:
          p->ref[b] -= 1;
          break;
        case kAlloc:
          p->ref[b] = 0;
          p->relink(b);
          if (it->had_hash) {
            p->has_hash[b] = 1;
            p->hash[b] = it->hash;
            p->table.insert(it->hash, b);
          }
          break;
        case kCommit:
          p->table.erase(it->hash);
          p->has_hash[b] = 0;
          break;
      }
    }
    entries.clear();
  }
};

void acquire(cw_pool* p, int32_t b, UndoLog* log) {
  if (p->ref[b] == 0) {
    p->unlink(b);
    if (log) log->entries.push_back({UndoLog::kAcquireFree, 0, b, 0});
  } else if (log) {
    log->entries.push_back({UndoLog::kAcquireHeld, 0, b, 0});
  }
  p->ref[b] += 1;
}

int32_t match(cw_pool* p, const uint64_t* hashes, int32_t n, int32_t max_match, int32_t* out,
              UndoLog* log) {
  int32_t depth = 0;
  const int32_t lim = std::min(n, std::max(0, max_match));
  while (depth < lim) {
    const int32_t b = p->table.find(hashes[depth]);
    if (b < 0) break;
    out[depth++] = b;
  }
  for (int32_t i = 0; i < depth; ++i) acquire(p, out[i], log);
  return depth;
}

// Caller has checked nfree >= count.
void alloc_n(cw_pool* p, int32_t count, int32_t* out, UndoLog* log) {
  for (int32_t i = 0; i < count; ++i) {
    const int32_t b = p->front();
    p->unlink(b);
    const uint8_t had = p->has_hash[b];
    const uint64_t old = p->hash[b];
    if (had) {
      p->table.erase(old);
      p->has_hash[b] = 0;
    }
    p->ref[b] = 1;
    if (log) log->entries.push_back({UndoLog::kAlloc, had, b, old});
    out[i] = b;
  }
}

// Caller has validated the (hash, block) pairs.
void commit_n(cw_pool* p, const uint64_t* hashes, const int32_t* ids, int32_t n, UndoLog* log) {
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = ids[i];
    if (p->has_hash[b]) continue;
    if (p->table.find(hashes[i]) >= 0) continue;
    p->table.insert(hashes[i], b);
    p->has_hash[b] = 1;
    p->hash[b] = hashes[i];
    if (log) log->entries.push_back({UndoLog::kCommit, 0, b, hashes[i]});
  }
}

// Per-thread scratch indexed by block ID for validating one call's arguments.
struct Scratch {
  std::vector<int32_t> count;
  std::vector<uint64_t> hash;
  std::vector<int32_t> touched;
  void fit(int32_t n) {
    if (int32_t(count.size()) < n) {
      count.resize(size_t(n), 0);
      hash.resize(size_t(n), 0);
    }
    touched.clear();
  }
  void reset() {
    for (int32_t b : touched) count[size_t(b)] = 0;
    touched.clear();
  }
};
thread_local Scratch g_scratch;

cw_status check_commit(const cw_pool* p, const uint64_t* hashes, const int32_t* ids, int32_t n) {
  Scratch& sc = g_scratch;
  sc.fit(p->n);
  cw_status st = CW_OK;
  for (int32_t i = 0; i < n && st == CW_OK; ++i) {
    const int32_t b = ids[i];
    if (b < 0 || b >= p->n) {
      st = fail(CW_EINVAL, "commit: block ID out of range");
    } else if (p->ref[b] == 0) {
      st = fail(CW_EINVAL, "commit: block " + std::to_string(b) + " is not held");
    } else if (p->has_hash[b] && p->hash[b] != hashes[i]) {
      st = fail(CW_EINVAL, "commit: block " + std::to_string(b) + " already holds another hash");
    } else if (sc.count[size_t(b)] && sc.hash[size_t(b)] != hashes[i]) {
      st = fail(CW_EINVAL, "commit: block " + std::to_string(b) + " listed with two hashes");
    } else if (!sc.count[size_t(b)]) {
      sc.count[size_t(b)] = 1;
      sc.hash[size_t(b)] = hashes[i];
      sc.touched.push_back(b);
    }
  }
  sc.reset();
  return st;
}

cw_status check_release(const cw_pool* p, const int32_t* ids, int32_t n) {
  Scratch& sc = g_scratch;
  sc.fit(p->n);
  cw_status st = CW_OK;
  for (int32_t i = 0; i < n && st == CW_OK; ++i) {
    const int32_t b = ids[i];
    if (b < 0 || b >= p->n) {
      st = fail(CW_EINVAL, "release: block ID out of range");
    } else {
      if (sc.count[size_t(b)]++ == 0) sc.touched.push_back(b);
      if (sc.count[size_t(b)] > p->ref[b])
        st = fail(CW_EINVAL, "release: block " + std::to_string(b) + " is not held that often");
    }
  }
  sc.reset();
  return st;
}

void release_n(cw_pool* p, const int32_t* ids, int32_t n) {
  for (int32_t i = n - 1; i >= 0; --i) {
    const int32_t b = ids[i];
    if (--p->ref[b] == 0) p->push_back(b);
  }
}

}  // namespace

extern "C" cw_status cw_pool_create(int32_t num_blocks, const int32_t* free_order, cw_pool** out) {
  if (!out) return fail(CW_EINVAL, "out is required");
  *out = nullptr;
  if (num_blocks < 1) return fail(CW_EINVAL, "num_blocks must be >= 1");
  std::vector<int32_t> order(num_blocks);
  if (free_order) {
    std::vector<uint8_t> seen(num_blocks, 0);
    for (int32_t i = 0; i < num_blocks; ++i) {
      const int32_t b = free_order[i];
      if (b < 0 || b >= num_blocks || seen[b]) return fail(CW_EINVAL, "free_order is not a permutation");
      seen[b] = 1;
      order[i] = b;
    }
  } else {
    std::iota(order.begin(), order.end(), 0);
  }
  auto* p = new cw_pool();
  p->n = num_blocks;
  p->ref.assign(num_blocks, 0);
  p->hash.assign(num_blocks, 0);
  p->has_hash.assign(num_blocks, 0);
  p->prev.assign(num_blocks + 1, num_blocks);
  p->next.assign(num_blocks + 1, num_blocks);
  p->table.init(num_blocks);
  for (int32_t b : order) p->push_back(b);
  *out = p;
  return cw::ok();
}

extern "C" void cw_pool_destroy(cw_pool* pool) { delete pool; }

extern "C" cw_status cw_pool_clone(const cw_pool* pool, cw_pool** out) {
  if (!pool || !out) return fail(CW_EINVAL, "pool and out are required");
  *out = new cw_pool(*pool);
  return cw::ok();
}

extern "C" int32_t cw_pool_num_free(const cw_pool* pool) { return pool ? pool->nfree : -1; }

extern "C" cw_status cw_prefix_match(cw_pool* pool, const uint64_t* hashes, int32_t n_hashes,
                                     int32_t max_match, int32_t* out_block_ids, int32_t* out_depth) {
  if (!pool || !out_depth) return fail(CW_EINVAL, "pool and out_depth are required");
  if (n_hashes < 0) return fail(CW_EINVAL, "n_hashes must be >= 0");
  if (n_hashes > 0 && (!hashes || !out_block_ids))
    return fail(CW_EINVAL, "hashes and out_block_ids are required");
  *out_depth = match(pool, hashes, n_hashes, max_match, out_block_ids, nullptr);
  return cw::ok();
}

extern "C" cw_status cw_pool_alloc(cw_pool* pool, int32_t n, int32_t* out_block_ids) {
  if (!pool) return fail(CW_EINVAL, "pool is required");
  if (n < 0) return fail(CW_EINVAL, "n must be >= 0");
  if (n > 0 && !out_block_ids) return fail(CW_EINVAL, "out_block_ids is required");
  if (n > pool->nfree)
    return fail(CW_ENOSPC, "pool exhausted: " + std::to_string(n) + " blocks requested, " +
                               std::to_string(pool->nfree) + " free");
  alloc_n(pool, n, out_block_ids, nullptr);
  return cw::ok();
}

extern "C" cw_status cw_pool_commit(cw_pool* pool, const uint64_t* hashes, const int32_t* block_ids,
                                    int32_t n) {
  if (!pool) return fail(CW_EINVAL, "pool is required");
  if (n < 0) return fail(CW_EINVAL, "n must be >= 0");
  if (n > 0 && (!hashes || !block_ids)) return fail(CW_EINVAL, "hashes and block_ids are required");
  cw_status st = check_commit(pool, hashes, block_ids, n);
  if (st != CW_OK) return st;
  commit_n(pool, hashes, block_ids, n, nullptr);
  return cw::ok();
}

extern "C" cw_status cw_pool_release(cw_pool* pool, const int32_t* block_ids, int32_t n) {
  if (!pool) return fail(CW_EINVAL, "pool is required");
  if (n < 0) return fail(CW_EINVAL, "n must be >= 0");
  if (n > 0 && !block_ids) return fail(CW_EINVAL, "block_ids is required");
  cw_status st = check_release(pool, block_ids, n);
  if (st != CW_OK) return st;
  release_n(pool, block_ids, n);
  return cw::ok();
}

extern "C" cw_status cw_schedule_batch(cw_pool* pool, const int32_t* tokens, const int64_t* cu_tokens,
                                       int32_t batch, int32_t block_size, int32_t bt_stride,
                                       int32_t* out_block_table, int32_t* out_prefix_len,
                                       int32_t* out_cu_suffix) {
  if (!pool || !tokens || !cu_tokens || !out_block_table || !out_prefix_len || !out_cu_suffix)
    return fail(CW_EINVAL, "a required pointer is NULL");
  if (batch < 1) return fail(CW_EINVAL, "batch must be >= 1");
  if (block_size < 1 || bt_stride < 1) return fail(CW_EINVAL, "block_size and bt_stride must be >= 1");
  if (cu_tokens[0] != 0) return fail(CW_EINVAL, "cu_tokens[0] must be 0");
  int64_t total_suffix = 0;
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t L = cu_tokens[r + 1] - cu_tokens[r];
    if (L < 1) return fail(CW_EINVAL, "request " + std::to_string(r) + " has an empty prompt");
    if ((L + block_size - 1) / block_size > bt_stride)
      return fail(CW_EINVAL, "request " + std::to_string(r) + " does not fit bt_stride");
  }
  UndoLog log;
  std::vector<uint64_t> hashes;
  out_cu_suffix[0] = 0;
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t L = cu_tokens[r + 1] - cu_tokens[r];
    const int64_t nfull = L / block_size;
    const int64_t nblocks = (L + block_size - 1) / block_size;
    hashes.resize(size_t(nfull));
    chain_hashes(tokens + cu_tokens[r], L, block_size, hashes.data());
    int32_t* row = out_block_table + int64_t(r) * bt_stride;
    const int32_t cap = int32_t((L - 1) / block_size);
    const int32_t depth = match(pool, hashes.data(), int32_t(nfull), cap, row, &log);
    const int32_t fresh = int32_t(nblocks - depth);
    if (fresh > pool->nfree) {
      log.rollback(pool);
      return fail(CW_ENOSPC, "pool exhausted while scheduling request " + std::to_string(r));
    }
    alloc_n(pool, fresh, row + depth, &log);
    commit_n(pool, hashes.data() + depth, row + depth, int32_t(nfull - depth), &log);
    for (int64_t i = nblocks; i < bt_stride; ++i) row[i] = -1;
    out_prefix_len[r] = depth * block_size;
    total_suffix += L - int64_t(depth) * block_size;
    if (total_suffix > INT32_MAX) {
      log.rollback(pool);
      return fail(CW_EINVAL, "total suffix rows exceed INT32_MAX");
    }
    out_cu_suffix[r + 1] = int32_t(total_suffix);
  }
  return cw::ok();
}

extern "C" cw_status cw_release_batch(cw_pool* pool, const int32_t* block_table, int32_t bt_stride,
                                      const int32_t* prefix_len, const int32_t* cu_suffix,
                                      int32_t batch, int32_t block_size) {
  if (!pool || !block_table) return fail(CW_EINVAL, "pool and block_table are required");
  cw_status st = cw::check_batch(cu_suffix, prefix_len, batch, block_size, bt_stride, nullptr);
  if (st != CW_OK) return st;
  std::vector<int32_t> ids;
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t L = int64_t(prefix_len[r]) + (cu_suffix[r + 1] - cu_suffix[r]);
    const int64_t nb = (L + block_size - 1) / block_size;
    ids.insert(ids.end(), block_table + int64_t(r) * bt_stride, block_table + int64_t(r) * bt_stride + nb);
  }
  st = check_release(pool, ids.data(), int32_t(ids.size()));
  if (st != CW_OK) return st;
  // Per request, so each request's tail is reused before its head.
  size_t off = 0;
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t L = int64_t(prefix_len[r]) + (cu_suffix[r + 1] - cu_suffix[r]);
    const int32_t nb = int32_t((L + block_size - 1) / block_size);
    release_n(pool, ids.data() + off, nb);
    off += nb;
  }
  return cw::ok();
}

// ---------------------------------------------------------------------------
// Attention planner. A tile is (request, KV head, first suffix row): 256
// packed (query head, row) pairs whose keys run from 0 to the last row's
// position; its key range is cut into num_splits runs of whole 64-key steps
// (one run when not splitting), and each run is one plan entry. The attention
// grid is persistent, one workgroup per CU; workgroup w runs entries w,
// w + grid, w + 2 grid, ... of its queue.
//
// With enough (request, KV head) pairs and 256 queues, the pairs are first
// spread over the eight L2 partitions (queue w runs on partition w % 8) by
// total work, so that every tile re-reading a pair's K/V does so from that
// partition's L2; the entries of a partition then fill its 32 queues in
// rounds of one entry per queue in pair order (see rounds()), so that the
// tiles running together share their K/V. Otherwise queues are filled
// longest-processing-time first (each entry, heaviest first, goes to the
// queue with the least work so far), so that they end together.
// ---------------------------------------------------------------------------
namespace {

cw_status plan_args(const int32_t* cu, const int32_t* plen, int32_t batch, int32_t hq, int32_t hkv,
                    int32_t d, int32_t splits) {
  if (!cu || !plen) return fail(CW_EINVAL, "cu_suffix_host and prefix_len_host are required");
  if (batch < 1) return fail(CW_EINVAL, "batch must be >= 1");
  if (hq < 1 || hkv < 1 || hq % hkv != 0)
    return fail(CW_EINVAL, "num_q_heads must be a positive multiple of num_kv_heads");
  if (hq / hkv > cw::kMaxGroup) return fail(CW_EUNSUPPORTED, "more than 128 query heads per KV head");
  if (d != 64 && d != 128) return fail(CW_EUNSUPPORTED, "head_dim must be 64 or 128");
  if (splits < 1 || splits > cw::kMaxSplits) return fail(CW_EINVAL, "num_splits must be in [1, 64]");
  if (cu[0] != 0) return fail(CW_EINVAL, "cu_suffix[0] must be 0");
  for (int32_t r = 0; r < batch; ++r) {
    if (cu[r + 1] < cu[r]) return fail(CW_EINVAL, "cu_suffix must be non-decreasing");
    if (plen[r] < 0) return fail(CW_EINVAL, "prefix_len must be >= 0");
    if (int64_t(plen[r]) + (cu[r + 1] - cu[r]) > INT32_MAX - cw::kKvTile)
      return fail(CW_EUNSUPPORTED, "prompt too long");
  }
  return CW_OK;
}

struct Entry {
  int32_t f[cw::kEntFields];
  int64_t cost;
  int32_t pair;
};

// Work of an entry in 64-key steps, plus a step's worth for its start and end.
constexpr int64_t kEntryOverhead = 1;

std::vector<Entry> plan_entries(const int32_t* cu, const int32_t* plen, int32_t batch, int32_t hq, int32_t hkv,
                                int32_t splits) {
  const int32_t per = cw::tile_positions(hq / hkv);
  std::vector<Entry> out;
  for (int32_t r = 0; r < batch; ++r) {
    const int32_t S = cu[r + 1] - cu[r], P = plen[r];
    for (int32_t row0 = 0; row0 < S; row0 += per) {
      const int32_t nvalid = std::min(per, S - row0);
      const int32_t n = int32_t((int64_t(P) + row0 + nvalid + cw::kKvTile - 1) / cw::kKvTile);
      for (int32_t g = 0; g < hkv; ++g)
        for (int32_t s = 0; s < splits; ++s) {
          Entry e;
          // run s: steps n s / splits .. n (s + 1) / splits - 1, so that the
          // runs differ by at most one step and none is empty while n >= splits
          const int32_t kb = int32_t(int64_t(n) * s / splits), ke = int32_t(int64_t(n) * (s + 1) / splits);
          // steps whose keys every row of the entry sees (key 64 k + 63 <= P + row0)
          const int32_t nfull = std::max(0, std::min(ke - kb, (P + row0 + 1) / cw::kKvTile - kb));
          const int32_t f[cw::kEntFields] = {r, g, row0, nvalid, cu[r], P, P + S, kb, ke, s, nfull, cu[r] + row0};
          std::copy(f, f + cw::kEntFields, e.f);
          // (an empty run still writes its part and passes an entry switch:
          // with cost 0, longest-first placement would stack every empty run
          // on the least-loaded queue)
          e.cost = (ke - kb) + kEntryOverhead;
          e.pair = r * hkv + g;
          out.push_back(e);
        }
    }
  }
  return out;
}

// Queue of every entry and the queue count.
struct Queues {
  int32_t grid = 0;
  int32_t len = 0;                       // entries of the longest queue
  std::vector<std::vector<int32_t>> q;   // entry indices per queue, in run order
};

// Longest processing time first over `n` queues.
void lpt(const std::vector<Entry>& ents, std::vector<int32_t> idx, const std::vector<int32_t>& queues,
         std::vector<std::vector<int32_t>>* q) {
  std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) { return ents[size_t(a)].cost > ents[size_t(b)].cost; });
  std::vector<int64_t> load(queues.size(), 0);
  for (int32_t i : idx) {
    size_t x = 0;
    for (size_t k = 1; k < queues.size(); ++k)
      if (load[k] < load[x]) x = k;
    load[x] += ents[size_t(i)].cost;
    (*q)[size_t(queues[x])].push_back(i);
  }
}

// Rounds over the queues of one L2 partition: the entries, ordered by
// (request, KV head) pair, split run and first row, are cut into rounds of one
// entry per queue, and within a round the heaviest entry goes to the queue
// with the least work so far. The queues run a round at about the same time,
// so the tiles that run together on the partition come from one or two pairs
// and read the same K/V blocks out of its L2. The last three rounds' worth of
// entries go longest first to the least-loaded queue, so that the queues end
// together.
void rounds(const std::vector<Entry>& ents, std::vector<int32_t> idx, const std::vector<int32_t>& queues,
            std::vector<std::vector<int32_t>>* q) {
  std::stable_sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) {
    const Entry& x = ents[size_t(a)];
    const Entry& y = ents[size_t(b)];
    if (x.pair != y.pair) return x.pair < y.pair;
    if (x.f[cw::kEntSplit] != y.f[cw::kEntSplit]) return x.f[cw::kEntSplit] < y.f[cw::kEntSplit];
    return x.f[cw::kEntRow0] < y.f[cw::kEntRow0];
  });
  const size_t nq = queues.size();
  std::vector<int64_t> load(nq, 0);
  std::vector<size_t> order(nq);
  // the last kTail rounds' entries are placed longest first instead, which
  // evens out the queues' ends
  constexpr size_t kTail = 3;
  const size_t n_rounds = idx.size() > kTail * nq ? (idx.size() - kTail * nq) / nq : 0;
  for (size_t r0 = 0; r0 < n_rounds * nq; r0 += nq) {
    std::vector<int32_t> round(idx.begin() + std::ptrdiff_t(r0), idx.begin() + std::ptrdiff_t(r0 + nq));
    std::stable_sort(round.begin(), round.end(),
                     [&](int32_t a, int32_t b) { return ents[size_t(a)].cost > ents[size_t(b)].cost; });
    std::iota(order.begin(), order.end(), size_t(0));
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return load[a] < load[b]; });
    for (size_t k = 0; k < round.size(); ++k) {
      load[order[k]] += ents[size_t(round[k])].cost;
      (*q)[size_t(queues[order[k]])].push_back(round[k]);
    }
  }
  std::vector<int32_t> tail(idx.begin() + std::ptrdiff_t(n_rounds * nq), idx.end());
  std::stable_sort(tail.begin(), tail.end(),
                   [&](int32_t a, int32_t b) { return ents[size_t(a)].cost > ents[size_t(b)].cost; });
  for (int32_t i : tail) {
    size_t x = 0;
    for (size_t k = 1; k < nq; ++k)
      if (load[k] < load[x]) x = k;
    load[x] += ents[size_t(i)].cost;
    (*q)[size_t(queues[x])].push_back(i);
  }
}

Queues plan_queues(const std::vector<Entry>& ents, int32_t batch, int32_t hkv) {
  Queues qs;
  qs.grid = int32_t(std::min<size_t>(ents.size(), cw::kNumCu));
  if (qs.grid == 0) return qs;
  qs.q.assign(size_t(qs.grid), {});
  std::vector<int32_t> all(ents.size());
  std::iota(all.begin(), all.end(), 0);
  const int64_t npairs = int64_t(batch) * hkv;
  bool grouped = false;
  if (qs.grid == cw::kNumCu && npairs >= 4 * cw::kNumXcd) {
    // pairs to partitions by total work, heaviest pair first
    std::vector<int64_t> pair_cost(size_t(npairs), 0);
    for (const Entry& e : ents) pair_cost[size_t(e.pair)] += e.cost;
    std::vector<int32_t> order(static_cast<size_t>(npairs));
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int32_t a, int32_t b) { return pair_cost[size_t(a)] > pair_cost[size_t(b)]; });
    std::vector<int8_t> part(size_t(npairs), 0);
    int64_t load[cw::kNumXcd] = {0};
    int64_t total = 0;
    for (int32_t pr : order) {
      int x = 0;
      for (int i = 1; i < cw::kNumXcd; ++i)
        if (load[i] < load[x]) x = i;
      part[size_t(pr)] = int8_t(x);
      load[x] += pair_cost[size_t(pr)];
      total += pair_cost[size_t(pr)];
    }
    const int64_t max_load = *std::max_element(load, load + cw::kNumXcd);
    if (max_load * cw::kNumXcd <= total + total / 50) {   // within 2% of even
      grouped = true;
      for (int x = 0; x < cw::kNumXcd; ++x) {
        std::vector<int32_t> idx, queues;
        for (int32_t i : all)
          if (part[size_t(ents[size_t(i)].pair)] == x) idx.push_back(i);
        for (int32_t w = x; w < qs.grid; w += cw::kNumXcd) queues.push_back(w);
        rounds(ents, idx, queues, &qs.q);
      }
    }
  }
  if (!grouped) {
    std::vector<int32_t> queues(size_t(qs.grid));
    std::iota(queues.begin(), queues.end(), 0);
    lpt(ents, all, queues, &qs.q);
  }
  for (const auto& v : qs.q) qs.len = std::max<int32_t>(qs.len, int32_t(v.size()));
  return qs;
}

}  // namespace

namespace cw {
uint64_t batch_fingerprint(const int32_t* cu, const int32_t* plen, int32_t batch, int32_t hq, int32_t hkv,
                           int32_t d, int32_t splits) {
  // FNV-1a over the little-endian words of the description, then a final mix
  uint64_t h = 0xcbf29ce484222325ULL;
  auto add = [&](uint32_t w) {
    for (int i = 0; i < 4; ++i) {
      h ^= (w >> (8 * i)) & 0xFFu;
      h *= 0x100000001b3ULL;
    }
  };
  add(uint32_t(batch));
  add(uint32_t(hq));
  add(uint32_t(hkv));
  add(uint32_t(d));
  add(uint32_t(splits));
  for (int32_t r = 0; r <= batch; ++r) add(uint32_t(cu[r]));
  for (int32_t r = 0; r < batch; ++r) add(uint32_t(plen[r]));
  h ^= h >> 33;
  h *= 0xff51afd7ed558ccdULL;
  h ^= h >> 33;
  return h;
}
}  // namespace cw

namespace {

// Entries and queues of a plan, and the words of its header and entries.
struct PlanLayout {
  std::vector<Entry> ents;
  Queues qs;
  int64_t padded = 0;   // queue slots (grid x longest queue)
  int64_t words = 0;    // header + entries
};

PlanLayout plan_layout(const int32_t* cu, const int32_t* plen, int32_t batch, int32_t hq, int32_t hkv,
                       int32_t splits) {
  PlanLayout pl;
  pl.ents = plan_entries(cu, plen, batch, hq, hkv, splits);
  pl.qs = plan_queues(pl.ents, batch, hkv);
  pl.padded = int64_t(pl.qs.grid) * pl.qs.len;
  pl.words = cw::kPlanHeaderWords + cw::kPlanEntryWords * pl.padded;
  return pl;
}

// Writes the header and the entries (queue slot i of workgroup w at entry
// index i * grid + w) of a plan with fingerprint fp.
void write_plan(const PlanLayout& pl, const int32_t* cu, int32_t batch, int32_t hq, int32_t hkv, int32_t d,
                int32_t splits, uint64_t fp, int32_t* plan_host) {
  const uint32_t lo = uint32_t(fp), hi = uint32_t(fp >> 32);
  const Queues& qs = pl.qs;
  int64_t work = 0;
  for (const Entry& e : pl.ents) work += e.cost;
  std::fill(plan_host, plan_host + pl.words, 0);
  int32_t* h = plan_host;
  h[cw::kHdrMagic] = cw::kPlanMagic;
  h[cw::kHdrEntries] = int32_t(pl.padded);
  h[cw::kHdrFpLo] = int32_t(lo);
  h[cw::kHdrFpHi] = int32_t(hi);
  h[cw::kHdrGrid] = qs.grid;
  h[cw::kHdrSplits] = splits;
  h[cw::kHdrBatch] = batch;
  h[cw::kHdrHq] = hq;
  h[cw::kHdrHkv] = hkv;
  h[cw::kHdrD] = d;
  h[cw::kHdrRows] = cu[batch];
  h[cw::kHdrQueueLen] = qs.len;
  h[cw::kHdrWork] = int32_t(std::min<int64_t>(work, INT32_MAX));
  int32_t* body = plan_host + cw::kPlanHeaderWords;
  for (int32_t w = 0; w < qs.grid; ++w)
    for (int32_t i = 0; i < qs.len; ++i) {
      int32_t* out = body + (int64_t(i) * qs.grid + w) * cw::kPlanEntryWords;
      if (i < int32_t(qs.q[size_t(w)].size())) {
        const Entry& e = pl.ents[size_t(qs.q[size_t(w)][size_t(i)])];
        std::copy(e.f, e.f + cw::kEntFields, out);
      } else {
        out[cw::kEntR] = -1;   // end of this queue
      }
      out[cw::kEntCheck] = int32_t(cw::entry_tag(lo, hi, uint32_t(int64_t(i) * qs.grid + w)));
    }
}

}  // namespace

extern "C" int64_t cw_suffix_prefill_plan_words(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                                int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                                int32_t head_dim, int32_t num_splits) {
  cw_status st = plan_args(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, head_dim, num_splits);
  if (st != CW_OK) return st;
  const PlanLayout pl = plan_layout(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, num_splits);
  cw::ok();
  return pl.words;
}

extern "C" cw_status cw_suffix_prefill_plan(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                            int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                            int32_t head_dim, int32_t num_splits, int32_t* plan_host,
                                            int64_t plan_words) {
  cw_status st = plan_args(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, head_dim, num_splits);
  if (st != CW_OK) return st;
  const PlanLayout pl = plan_layout(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, num_splits);
  if (pl.padded > INT32_MAX / cw::kPlanEntryWords) return fail(CW_EUNSUPPORTED, "too many plan entries");
  if (!plan_host || plan_words < pl.words)
    return fail(CW_EINVAL, "plan buffer too small: need " + std::to_string(pl.words) + " words");
  const uint64_t fp = cw::batch_fingerprint(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads,
                                            head_dim, num_splits);
  write_plan(pl, cu_suffix_host, batch, num_q_heads, num_kv_heads, head_dim, num_splits, fp, plan_host);
  return cw::ok();
}

namespace cw {
uint64_t append_fingerprint(const int32_t* cu, const int32_t* plen, const int32_t* bt, int32_t bt_stride,
                            int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t num_blocks) {
  uint64_t h = batch_fingerprint(cu, plen, batch, hq, hkv, d, 1) ^ 0x9E3779B97F4A7C15ULL;
  auto add = [&](uint32_t w) {
    for (int i = 0; i < 4; ++i) {
      h ^= (w >> (8 * i)) & 0xFFu;
      h *= 0x100000001b3ULL;
    }
  };
  add(uint32_t(num_blocks));
  add(uint32_t(bt_stride));
  for (int32_t r = 0; r < batch; ++r) {
    const int64_t nb = (int64_t(plen[r]) + cu[r + 1] - cu[r] + kBlockSize - 1) / kBlockSize;
    for (int64_t j = 0; j < nb; ++j) add(uint32_t(bt[int64_t(r) * bt_stride + j]));
  }
  h ^= h >> 33;
  h *= 0xc4ceb9fe1a85ec53ULL;
  h ^= h >> 33;
  return h;
}
}  // namespace cw

namespace {

// Checks of the fused plan's arguments beyond plan_args (one split).
cw_status append_plan_args(const int32_t* cu, const int32_t* plen, const int32_t* bt, int32_t bt_stride,
                           int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t num_blocks) {
  cw_status st = plan_args(cu, plen, batch, hq, hkv, d, 1);
  if (st != CW_OK) return st;
  if (!bt) return fail(CW_EINVAL, "block_table_host is required");
  if (num_blocks < 1) return fail(CW_EINVAL, "num_blocks must be >= 1");
  if (num_blocks > cw::kMaxAppendBlocks) return fail(CW_EUNSUPPORTED, "num_blocks must be below 2^27");
  int64_t rows = 0;
  return cw::check_batch(cu, plen, batch, cw::kBlockSize, bt_stride, &rows);
}

int64_t append_table_words(int32_t batch, int32_t bt_stride) { return int64_t(batch) * bt_stride * 2; }

// The fused plan's table (layout in cw_internal.h). With cw_kv_append run
// before the attention call, a request reads its own suffix blocks after the
// append, and a prefix block that is some request's full suffix block of this
// batch (a block committed earlier in the same schedule) also holds the rows
// appended into it: both are read from those rows of k_new / v_new instead,
// so that the fused call computes what the two calls in sequence compute
// while nothing in it reads a block it writes. Refused: a suffix block named
// twice (the two appends would race) and a prefix block that is a partial
// suffix block (its bytes would be part appended rows, part older content).
cw_status build_append_table(const int32_t* cu, const int32_t* plen, const int32_t* bt, int32_t bt_stride,
                             int32_t batch, int32_t num_blocks, int32_t* table) {
  constexpr int32_t bs = cw::kBlockSize;
  std::unordered_map<int32_t, int32_t> fresh;   // suffix block -> first row (-1: partial block)
  for (int32_t r = 0; r < batch; ++r) {
    const int32_t P = plen[r], L = P + (cu[r + 1] - cu[r]);
    for (int32_t j = P / bs; j < (L + bs - 1) / bs; ++j) {
      const int32_t id = bt[int64_t(r) * bt_stride + j];
      if (id < 0 || id >= num_blocks) continue;
      const int32_t row = (j + 1) * bs <= L ? cu[r] + (j * bs - P) : -1;
      if (!fresh.emplace(id, row).second)
        return fail(CW_EINVAL, "block " + std::to_string(id) + " is named by two suffix blocks of the batch");
    }
  }
  std::fill(table, table + append_table_words(batch, bt_stride), -1);
  for (int32_t r = 0; r < batch; ++r) {
    const int32_t P = plen[r], L = P + (cu[r + 1] - cu[r]);
    for (int32_t j = 0; j < (L + bs - 1) / bs; ++j) {
      const int32_t id = bt[int64_t(r) * bt_stride + j];
      int32_t* t = table + (int64_t(r) * bt_stride + j) * 2;
      const bool in_pool = id >= 0 && id < num_blocks;
      if (j >= P / bs) {   // a suffix block of r: its rows, and the append target
        if (in_pool) {
          t[0] = cw::append_src_rows(cu[r] + (j * bs - P));
          t[1] = id;
        }
        continue;
      }
      if (!in_pool) continue;   // no block: zeros
      const auto it = fresh.find(id);
      if (it == fresh.end()) {
        t[0] = cw::append_src_block(id);
      } else if (it->second >= 0) {
        t[0] = cw::append_src_rows(it->second);
      } else {
        return fail(CW_EUNSUPPORTED, "a prefix block of request " + std::to_string(r) +
                                         " is the partial last block of a suffix in the same batch");
      }
    }
  }
  return CW_OK;
}

}  // namespace

extern "C" int64_t cw_suffix_prefill_append_plan_words(const int32_t* cu_suffix_host,
                                                       const int32_t* prefix_len_host, int32_t bt_stride,
                                                       int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                                       int32_t head_dim) {
  cw_status st = plan_args(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, head_dim, 1);
  if (st != CW_OK) return st;
  if (bt_stride < 1) return fail(CW_EINVAL, "bt_stride must be >= 1");
  const PlanLayout pl = plan_layout(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, 1);
  cw::ok();
  return pl.words + append_table_words(batch, bt_stride);
}

extern "C" cw_status cw_suffix_prefill_append_plan(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                                   const int32_t* block_table_host, int32_t bt_stride,
                                                   int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                                   int32_t head_dim, int32_t num_blocks, int32_t* plan_host,
                                                   int64_t plan_words) {
  cw_status st = append_plan_args(cu_suffix_host, prefix_len_host, block_table_host, bt_stride, batch, num_q_heads,
                                  num_kv_heads, head_dim, num_blocks);
  if (st != CW_OK) return st;
  const PlanLayout pl = plan_layout(cu_suffix_host, prefix_len_host, batch, num_q_heads, num_kv_heads, 1);
  if (pl.padded > INT32_MAX / cw::kPlanEntryWords) return fail(CW_EUNSUPPORTED, "too many plan entries");
  const int64_t need = pl.words + append_table_words(batch, bt_stride);
  if (need > INT32_MAX) return fail(CW_EUNSUPPORTED, "plan too large");
  if (!plan_host || plan_words < need)
    return fail(CW_EINVAL, "plan buffer too small: need " + std::to_string(need) + " words");
  st = build_append_table(cu_suffix_host, prefix_len_host, block_table_host, bt_stride, batch, num_blocks,
                          plan_host + pl.words);
  if (st != CW_OK) return st;
  const uint64_t fp = cw::append_fingerprint(cu_suffix_host, prefix_len_host, block_table_host, bt_stride, batch,
                                             num_q_heads, num_kv_heads, head_dim, num_blocks);
  write_plan(pl, cu_suffix_host, batch, num_q_heads, num_kv_heads, head_dim, 1, fp, plan_host);
  plan_host[cw::kHdrTable] = int32_t(pl.words);
  plan_host[cw::kHdrTableStride] = bt_stride;
  plan_host[cw::kHdrNumBlocks] = num_blocks;
  return cw::ok();
}

// Validates a plan's header against the batch description of a device call;
// sets the launch grid and split count.
namespace cw {
cw_status check_plan_header(const char* what, const int32_t* plan_host, const int32_t* cu, const int32_t* plen,
                            int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t* grid, int32_t* splits,
                            uint32_t* fp_lo, uint32_t* fp_hi, int32_t* num_entries, const int32_t* append_bt,
                            int32_t bt_stride, int32_t num_blocks) {
  const std::string w(what);
  if (!plan_host) return fail(CW_EINVAL, w + ": plan_host is required");
  if (plan_host[kHdrMagic] != kPlanMagic) return fail(CW_EINVAL, w + ": plan_host is not a plan of this library");
  const int32_t s = plan_host[kHdrSplits];
  if (s < 1 || s > kMaxSplits) return fail(CW_EINVAL, w + ": plan has an invalid split count");
  if (!append_bt && plan_host[kHdrTable] != 0)
    return fail(CW_EINVAL, w + ": the plan carries an append table (cw_suffix_prefill_append_plan): "
                               "use cw_suffix_prefill_append_attn");
  if (append_bt && plan_host[kHdrTable] == 0)
    return fail(CW_EINVAL, w + ": the plan has no append table: build it with cw_suffix_prefill_append_plan");
  const uint64_t fp = append_bt ? append_fingerprint(cu, plen, append_bt, bt_stride, batch, hq, hkv, d, num_blocks)
                                : batch_fingerprint(cu, plen, batch, hq, hkv, d, s);
  if (uint32_t(plan_host[kHdrFpLo]) != uint32_t(fp) || uint32_t(plan_host[kHdrFpHi]) != uint32_t(fp >> 32) ||
      plan_host[kHdrBatch] != batch || plan_host[kHdrHq] != hq || plan_host[kHdrHkv] != hkv || plan_host[kHdrD] != d)
    return fail(CW_EINVAL, w + ": the plan was built for another batch (cu_suffix, prefix_len, heads or head_dim differ)");
  const int32_t g = plan_host[kHdrGrid], len = plan_host[kHdrQueueLen], n = plan_host[kHdrEntries];
  if (g < 0 || g > kNumCu || len < 0 || int64_t(g) * len != n)
    return fail(CW_EINVAL, w + ": plan header is inconsistent");
  if (append_bt && (s != 1 || plan_host[kHdrTableStride] != bt_stride || plan_host[kHdrNumBlocks] != num_blocks ||
                    int64_t(plan_host[kHdrTable]) != kPlanHeaderWords + int64_t(kPlanEntryWords) * n))
    return fail(CW_EINVAL, w + ": plan header is inconsistent");
  *grid = g;
  *splits = s;
  *fp_lo = uint32_t(fp);
  *fp_hi = uint32_t(fp >> 32);
  *num_entries = n;
  return CW_OK;
}
}  // namespace cw
