// Block-id pool with the elastic gate, and the one-step-ahead toggle
// controller (the paper, Section 3: "Two handles, one virtual range" gates
// the top elastic block-id range so those blocks are only handed out while
// the elastic slice is committed; "Controller": the scheduler knows whether
// the next step is decode-only or contains a prefill, the elastic slice is
// committed during decode-only phases and decommitted at the boundary before
// a prefill, with hysteresis; committing grows the usable block count, and
// decommitting first drains the elastic blocks, syncs, then unmaps).
//
// Host-only code: nothing here touches the device except through the
// kvpool_* calls the controller makes.

#include <algorithm>
#include <new>
#include <vector>

#include "abi_internal.hpp"
#include "kvattn.h"

using kvattn::clear_error;
using kvattn::set_error;

struct kvblocks {
  int num_base = 0;
  int num_elastic = 0;
  bool admitted = false;
  std::vector<int32_t> free_base;     // stacks: back() is handed out next
  std::vector<int32_t> free_elastic;
  std::vector<uint8_t> live;          // per id: allocated and not yet freed
  int live_elastic = 0;
};

struct kvctl {
  kvpool* pool = nullptr;             // NULL: the state machine without a device
  kvblocks* blocks = nullptr;
  int hysteresis = 1;
  int streak = 0;                     // consecutive decode-only steps announced
  bool committed = false;
  int commits = 0, decommits = 0;
};

namespace {

bool is_elastic(const kvblocks* b, int32_t id) { return id >= b->num_base; }

}  // namespace

extern "C" int kvblocks_create(int num_base_blocks, int num_elastic_blocks, kvblocks** out) {
  clear_error();
  if (!out) return set_error(KV_ERR_INVALID, "kvblocks_create: out is NULL");
  *out = nullptr;
  if (num_base_blocks < 0 || num_elastic_blocks < 0 ||
      (long long)num_base_blocks + num_elastic_blocks > 0x7fffffffLL ||
      num_base_blocks + num_elastic_blocks == 0)
    return set_error(KV_ERR_INVALID, "kvblocks_create: %d base + %d elastic blocks",
                     num_base_blocks, num_elastic_blocks);
  kvblocks* b = new (std::nothrow) kvblocks;
  if (!b) return set_error(KV_ERR_OOM, "kvblocks_create: host allocation failed");
  b->num_base = num_base_blocks;
  b->num_elastic = num_elastic_blocks;
  b->live.assign((size_t)num_base_blocks + num_elastic_blocks, 0);
  // lowest ids first: the stacks hold ids in descending order
  b->free_base.resize(num_base_blocks);
  for (int i = 0; i < num_base_blocks; ++i) b->free_base[i] = num_base_blocks - 1 - i;
  b->free_elastic.resize(num_elastic_blocks);
  for (int i = 0; i < num_elastic_blocks; ++i)
    b->free_elastic[i] = num_base_blocks + num_elastic_blocks - 1 - i;
  *out = b;
  return KV_OK;
}

extern "C" void kvblocks_destroy(kvblocks* b) { delete b; }

extern "C" int kvblocks_num_free(const kvblocks* b) {
  if (!b) return set_error(KV_ERR_INVALID, "kvblocks_num_free: NULL pool");
  return (int)b->free_base.size() + (b->admitted ? (int)b->free_elastic.size() : 0);
}

extern "C" int kvblocks_num_admitted(const kvblocks* b) {
  if (!b) return set_error(KV_ERR_INVALID, "kvblocks_num_admitted: NULL pool");
  return b->num_base + (b->admitted ? b->num_elastic : 0);
}

extern "C" int kvblocks_live_elastic(const kvblocks* b) {
  if (!b) return set_error(KV_ERR_INVALID, "kvblocks_live_elastic: NULL pool");
  return b->live_elastic;
}

extern "C" int kvblocks_is_admitted(const kvblocks* b) {
  if (!b) return set_error(KV_ERR_INVALID, "kvblocks_is_admitted: NULL pool");
  return b->admitted ? 1 : 0;
}

extern "C" int kvblocks_set_elastic(kvblocks* b, int admit) {
  clear_error();
  if (!b) return set_error(KV_ERR_INVALID, "kvblocks_set_elastic: NULL pool");
  b->admitted = admit != 0;
  return KV_OK;
}

extern "C" int kvblocks_alloc(kvblocks* b, int n, int32_t* ids) {
  clear_error();
  if (!b || n < 0 || (n > 0 && !ids))
    return set_error(KV_ERR_INVALID, "kvblocks_alloc: bad arguments");
  const size_t avail = b->free_base.size() + (b->admitted ? b->free_elastic.size() : 0);
  if ((size_t)n > avail)
    return set_error(KV_ERR_OOM, "kvblocks_alloc: %d blocks asked, %zu free", n, avail);
  for (int i = 0; i < n; ++i) {
    std::vector<int32_t>& src = b->free_base.empty() ? b->free_elastic : b->free_base;
    const int32_t id = src.back();
    src.pop_back();
    b->live[id] = 1;
    if (is_elastic(b, id)) ++b->live_elastic;
    ids[i] = id;
  }
  return KV_OK;
}

extern "C" int kvblocks_free(kvblocks* b, int n, const int32_t* ids) {
  clear_error();
  if (!b || n < 0 || (n > 0 && !ids))
    return set_error(KV_ERR_INVALID, "kvblocks_free: bad arguments");
  const int total = b->num_base + b->num_elastic;
  // validate everything first: a bad call changes nothing
  std::vector<int32_t> seen(ids, ids + n);
  std::sort(seen.begin(), seen.end());
  for (int i = 0; i < n; ++i) {
    if (seen[i] < 0 || seen[i] >= total || !b->live[seen[i]])
      return set_error(KV_ERR_INVALID, "kvblocks_free: id %d is not allocated", seen[i]);
    if (i && seen[i] == seen[i - 1])
      return set_error(KV_ERR_INVALID, "kvblocks_free: id %d freed twice", seen[i]);
  }
  for (int i = 0; i < n; ++i) {
    const int32_t id = ids[i];
    b->live[id] = 0;
    if (is_elastic(b, id)) {
      --b->live_elastic;
      b->free_elastic.push_back(id);
    } else {
      b->free_base.push_back(id);
    }
  }
  return KV_OK;
}

extern "C" int kvblocks_plan_drain(kvblocks* b, int capacity, int32_t* from, int32_t* to,
                                   int* n) {
  clear_error();
  if (!b || !n || capacity < 0 || (capacity > 0 && (!from || !to)))
    return set_error(KV_ERR_INVALID, "kvblocks_plan_drain: bad arguments");
  *n = 0;
  const int need = b->live_elastic;
  if (need > capacity)
    return set_error(KV_ERR_INVALID, "kvblocks_plan_drain: %d live elastic blocks, room for %d",
                     need, capacity);
  if ((size_t)need > b->free_base.size())
    return set_error(KV_ERR_OOM, "kvblocks_plan_drain: %d live elastic blocks, %zu free base",
                     need, b->free_base.size());
  int k = 0;
  for (int id = b->num_base; id < b->num_base + b->num_elastic; ++id) {
    if (!b->live[id]) continue;
    const int32_t dst = b->free_base.back();
    b->free_base.pop_back();
    b->live[dst] = 1;
    from[k] = id;
    to[k] = dst;
    ++k;
  }
  *n = k;
  return KV_OK;
}

extern "C" int kvctl_create(kvpool* pool, kvblocks* blocks, int hysteresis_steps, kvctl** out) {
  clear_error();
  if (!out) return set_error(KV_ERR_INVALID, "kvctl_create: out is NULL");
  *out = nullptr;
  if (!blocks || hysteresis_steps < 1)
    return set_error(KV_ERR_INVALID, "kvctl_create: need a block pool and hysteresis >= 1");
  kvctl* c = new (std::nothrow) kvctl;
  if (!c) return set_error(KV_ERR_OOM, "kvctl_create: host allocation failed");
  c->pool = pool;
  c->blocks = blocks;
  c->hysteresis = hysteresis_steps;
  if (pool) {
    const int st = kvpool_is_committed(pool);
    if (st < 0) {
      delete c;
      return set_error(KV_ERR_INVALID, "kvctl_create: bad pool");
    }
    c->committed = st == 1;
  } else {
    c->committed = blocks->admitted;
  }
  blocks->admitted = c->committed;
  *out = c;
  return KV_OK;
}

extern "C" void kvctl_destroy(kvctl* c) { delete c; }

extern "C" int kvctl_is_committed(const kvctl* c) {
  if (!c) return set_error(KV_ERR_INVALID, "kvctl_is_committed: NULL controller");
  return c->committed ? 1 : 0;
}

extern "C" int kvctl_would_commit(const kvctl* c, int next_has_prefill) {
  if (!c) return set_error(KV_ERR_INVALID, "kvctl_would_commit: NULL controller");
  return (!next_has_prefill && !c->committed && c->streak + 1 >= c->hysteresis) ? 1 : 0;
}

extern "C" int kvctl_counts(const kvctl* c, int* commits, int* decommits) {
  if (!c) return set_error(KV_ERR_INVALID, "kvctl_counts: NULL controller");
  if (commits) *commits = c->commits;
  if (decommits) *decommits = c->decommits;
  return KV_OK;
}

extern "C" int kvctl_before_step(kvctl* c, int next_has_prefill, int* action, double* ms) {
  clear_error();
  if (!c) return set_error(KV_ERR_INVALID, "kvctl_before_step: NULL controller");
  if (action) *action = KVCTL_NONE;
  if (ms) *ms = 0.0;
  if (next_has_prefill) {
    c->streak = 0;
    if (!c->committed) return KV_OK;
    if (c->blocks->live_elastic > 0)
      return set_error(KV_ERR_STATE,
                       "kvctl_before_step: %d elastic blocks still live; drain them before "
                       "the prefill step", c->blocks->live_elastic);
    c->blocks->admitted = false;
    if (c->pool) {
      const int rc = kvpool_decommit_elastic(c->pool, ms);
      if (rc != KV_OK) {
        // The pool's state decides: a failed device sync leaves it committed,
        // while a failed unmap or release has already dropped the elastic
        // handles. Elastic ids are admitted only over mapped memory.
        c->committed = kvpool_is_committed(c->pool) == 1;
        c->blocks->admitted = c->committed;
        if (!c->committed) ++c->decommits;
        return rc;
      }
    }
    c->committed = false;
    ++c->decommits;
    if (action) *action = KVCTL_DECOMMIT;
    return KV_OK;
  }
  ++c->streak;
  if (c->committed || c->streak < c->hysteresis) return KV_OK;
  if (c->pool) {
    const int rc = kvpool_commit_elastic(c->pool, ms);
    if (rc != KV_OK) {
      c->streak = 0;    // try again only after another hysteresis window
      return rc;
    }
  }
  c->committed = true;
  c->blocks->admitted = true;
  ++c->commits;
  if (action) *action = KVCTL_COMMIT;
  return KV_OK;
}
