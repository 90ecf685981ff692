// Host-side allocator of KV blocks.  The shared affix cache lives in
// reserved shared blocks and every request's anchors and request-specific
// positions in private blocks (Section 4.1); peak KV use is counted in whole
// blocks, which is why a single request can hold more than a plain cache
// (the block-granularity overhead discussed with Table 4).
//
// Block ids are 0 .. capacity-1.  alloc hands out the lowest free ids in
// ascending order (deterministic layouts: a fresh pool's first allocation is
// 0, 1, 2, ...); free returns them.  The pool keeps the number of blocks in
// use and its peak since creation or the last reset.

#include <set>
#include <vector>

#include "acache.h"

struct acache_block_pool {
  int32_t capacity = 0;
  int32_t in_use = 0;
  int32_t peak = 0;
  std::set<int32_t> free_ids;     // ascending
  std::vector<uint8_t> taken;     // taken[id] != 0 while allocated
};

extern "C" {

acache_status acache_block_pool_create(int32_t capacity, acache_block_pool** pool) {
  if (!pool) return ACACHE_ERR_NULL;
  *pool = nullptr;
  if (capacity < 0) return ACACHE_ERR_SHAPE;
  auto* p = new acache_block_pool;
  p->capacity = capacity;
  p->taken.assign((size_t)capacity, 0);
  for (int32_t i = 0; i < capacity; ++i) p->free_ids.insert(p->free_ids.end(), i);
  *pool = p;
  return ACACHE_OK;
}

acache_status acache_block_pool_destroy(acache_block_pool* pool) {
  delete pool;
  return ACACHE_OK;
}

acache_status acache_block_pool_alloc(acache_block_pool* pool, int32_t n, int32_t* ids) {
  if (!pool) return ACACHE_ERR_NULL;
  if (n < 0) return ACACHE_ERR_SHAPE;
  if (n == 0) return ACACHE_OK;
  if (!ids) return ACACHE_ERR_NULL;
  if ((size_t)n > pool->free_ids.size()) return ACACHE_ERR_SPACE;
  auto it = pool->free_ids.begin();
  for (int32_t i = 0; i < n; ++i) {
    ids[i] = *it;
    pool->taken[(size_t)*it] = 1;
    it = pool->free_ids.erase(it);
  }
  pool->in_use += n;
  if (pool->in_use > pool->peak) pool->peak = pool->in_use;
  return ACACHE_OK;
}

acache_status acache_block_pool_free(acache_block_pool* pool, int32_t n, const int32_t* ids) {
  if (!pool) return ACACHE_ERR_NULL;
  if (n < 0) return ACACHE_ERR_SHAPE;
  if (n == 0) return ACACHE_OK;
  if (!ids) return ACACHE_ERR_NULL;
  // validate the whole list first: an invalid call changes nothing
  std::set<int32_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t id = ids[i];
    if (id < 0 || id >= pool->capacity || !pool->taken[(size_t)id] || !seen.insert(id).second)
      return ACACHE_ERR_SHAPE;
  }
  for (int32_t i = 0; i < n; ++i) {
    pool->taken[(size_t)ids[i]] = 0;
    pool->free_ids.insert(ids[i]);
  }
  pool->in_use -= n;
  return ACACHE_OK;
}

acache_status acache_block_pool_stats(const acache_block_pool* pool, int32_t* capacity, int32_t* in_use,
                                      int32_t* peak) {
  if (!pool) return ACACHE_ERR_NULL;
  if (capacity) *capacity = pool->capacity;
  if (in_use) *in_use = pool->in_use;
  if (peak) *peak = pool->peak;
  return ACACHE_OK;
}

acache_status acache_block_pool_reset_peak(acache_block_pool* pool) {
  if (!pool) return ACACHE_ERR_NULL;
  pool->peak = pool->in_use;
  return ACACHE_OK;
}

}  // extern "C"
