// Randomized check of the block-id pool and the toggle controller against a
// plain model, built with the address and undefined-behaviour sanitizers.
// Host code only: the elastic pool is a stub whose commit and decommit can be
// made to fail the ways the real one can (commit out of memory; decommit with
// a failed device sync, which leaves it committed; decommit with a failed
// unmap, which leaves it decommitted). Exits 0 when every invariant held.

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "abi_internal.hpp"
#include "kvattn.h"

// ---- stubs for what blockpool.cpp links against ----
struct kvpool {
  int committed = 0;
  int fail_commit = 0;     // next commit fails with KV_ERR_OOM
  int fail_decommit = 0;   // next decommit: 1 sync fails (stays committed), 2 unmap fails
};

extern "C" int kvpool_is_committed(const kvpool* p) { return p ? p->committed : -1; }
extern "C" int kvpool_commit_elastic(kvpool* p, double* ms) {
  if (ms) *ms = 0.0;
  if (p->committed) return KV_OK;
  if (p->fail_commit) {
    p->fail_commit = 0;
    return KV_ERR_OOM;
  }
  p->committed = 1;
  return KV_OK;
}
extern "C" int kvpool_decommit_elastic(kvpool* p, double* ms) {
  if (ms) *ms = 0.0;
  if (!p->committed) return KV_OK;
  const int mode = p->fail_decommit;
  p->fail_decommit = 0;
  if (mode == 1) return KV_ERR_HIP;
  p->committed = 0;
  return mode == 2 ? KV_ERR_HIP : KV_OK;
}
namespace kvattn {
int set_error(int code, const char*, ...) { return code; }
void clear_error() {}
}  // namespace kvattn

#define CHECK(cond)                                                       \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "step %d: check failed: %s\n", step, #cond);   \
      std::_Exit(1);                                                      \
    }                                                                     \
  } while (0)

int main(int argc, char** argv) {
  const int steps = argc > 1 ? std::atoi(argv[1]) : 20000;
  const unsigned seed = argc > 2 ? (unsigned)std::atoi(argv[2]) : 7u;
  const int nb = 96, ne = 32, total = nb + ne;
  std::mt19937 rng(seed);
  auto pick = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };

  kvblocks* b = nullptr;
  kvpool pool;
  kvctl* c = nullptr;
  int step = -1;
  CHECK(kvblocks_create(nb, ne, &b) == KV_OK);
  CHECK(kvctl_create(&pool, b, 3, &c) == KV_OK);

  std::vector<std::vector<int32_t>> seqs;   // the model: ids held per sequence
  std::set<int32_t> live;
  int refusals = 0, failed_commits = 0, failed_syncs = 0, failed_unmaps = 0;
  for (step = 0; step < steps; ++step) {
    const int op = pick(0, 9);
    if (op <= 2) {                                   // a sequence asks for blocks
      const int n = pick(1, 12);
      std::vector<int32_t> ids(n, -1);
      const int avail = kvblocks_num_free(b);
      const int rc = kvblocks_alloc(b, n, ids.data());
      if (n > avail) {
        CHECK(rc == KV_ERR_OOM);
      } else {
        CHECK(rc == KV_OK);
        for (int32_t id : ids) {
          CHECK(id >= 0 && id < total);
          CHECK(live.insert(id).second);              // never handed out twice
          CHECK(id < nb || kvblocks_is_admitted(b));  // elastic only while admitted
        }
        seqs.push_back(ids);
      }
    } else if (op <= 5 && !seqs.empty()) {           // a sequence finishes
      const size_t k = (size_t)pick(0, (int)seqs.size() - 1);
      CHECK(kvblocks_free(b, (int)seqs[k].size(), seqs[k].data()) == KV_OK);
      for (int32_t id : seqs[k]) live.erase(id);
      seqs.erase(seqs.begin() + (long)k);
    } else if (op == 6 && !seqs.empty()) {           // bad frees change nothing
      const int before = kvblocks_num_free(b);
      std::vector<int32_t> twice = {seqs[0][0], seqs[0][0]};
      CHECK(kvblocks_free(b, 2, twice.data()) == KV_ERR_INVALID);
      int32_t out_of_range = total + pick(0, 5);
      CHECK(kvblocks_free(b, 1, &out_of_range) == KV_ERR_INVALID);
      CHECK(kvblocks_num_free(b) == before);
    } else if (op == 7) {                            // drain by migration
      std::vector<int32_t> from(ne), to(ne);
      int n = -1;
      const int rc = kvblocks_plan_drain(b, ne, from.data(), to.data(), &n);
      if (rc == KV_OK) {
        for (int i = 0; i < n; ++i) {
          CHECK(from[i] >= nb && to[i] < nb);
          CHECK(live.count(from[i]) && live.insert(to[i]).second);
          for (auto& s : seqs) std::replace(s.begin(), s.end(), from[i], to[i]);
        }
        CHECK(kvblocks_free(b, n, from.data()) == KV_OK);
        for (int i = 0; i < n; ++i) live.erase(from[i]);
        CHECK(kvblocks_live_elastic(b) == 0);
      } else {
        CHECK(rc == KV_ERR_OOM);
      }
    } else {                                         // the scheduler's next step
      const int prefill = pick(0, 3) == 0;
      if (pick(0, 7) == 0) pool.fail_commit = 1;
      if (pick(0, 7) == 0) pool.fail_decommit = pick(1, 2);
      const int fail_commit = pool.fail_commit, fail_decommit = pool.fail_decommit;
      const int live_el = kvblocks_live_elastic(b);
      const int was = kvctl_is_committed(c);
      int action = -1;
      const int rc = kvctl_before_step(c, prefill, &action, nullptr);
      if (prefill && was && live_el > 0) {
        CHECK(rc == KV_ERR_STATE && kvctl_is_committed(c) == 1);
        ++refusals;
      } else if (prefill && was) {
        // a failed sync leaves the pool committed, a failed unmap decommitted
        CHECK(rc == (fail_decommit ? KV_ERR_HIP : KV_OK));
        CHECK(kvctl_is_committed(c) == (fail_decommit == 1 ? 1 : 0));
        failed_syncs += fail_decommit == 1;
        failed_unmaps += fail_decommit == 2;
      } else if (!prefill && !was && rc != KV_OK) {
        CHECK(rc == KV_ERR_OOM && fail_commit && kvctl_is_committed(c) == 0);
        ++failed_commits;
      } else {
        CHECK(rc == KV_OK);
      }
      if (rc == KV_OK && action == KVCTL_DECOMMIT) CHECK(was && !kvctl_is_committed(c));
      if (rc == KV_OK && action == KVCTL_COMMIT) CHECK(!was && kvctl_is_committed(c));
      pool.fail_commit = 0;
      pool.fail_decommit = 0;
    }
    // invariants after every operation
    int live_elastic = 0;
    for (int32_t id : live) live_elastic += id >= nb;
    CHECK(kvblocks_live_elastic(b) == live_elastic);
    const int admitted = kvblocks_is_admitted(b);
    CHECK(kvblocks_num_free(b) ==
          (nb - (int)live.size() + live_elastic) + (admitted ? ne - live_elastic : 0));
    CHECK(kvctl_is_committed(c) == pool.committed);
    CHECK(admitted == pool.committed);
  }
  int commits = 0, decommits = 0;
  CHECK(kvctl_counts(c, &commits, &decommits) == KV_OK);
  std::printf("ok: %d steps, %d commits, %d decommits, %d refusals with live elastic ids, "
              "%d failed commits, %d failed syncs, %d failed unmaps\n", steps, commits,
              decommits, refusals, failed_commits, failed_syncs, failed_unmaps);
  if (commits < 10 || decommits < 10 || refusals < 1 || failed_commits < 1 || failed_syncs < 1 ||
      failed_unmaps < 1) {
    std::fprintf(stderr, "the run did not reach every path\n");
    return 1;
  }
  kvctl_destroy(c);
  kvblocks_destroy(b);
  return 0;
}
