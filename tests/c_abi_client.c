/* A C99 caller of the library's C ABI, built and run by test_host.py. It uses
 * only entry points that need no GPU: the version, workspace sizing, argument
 * checks that fail before any launch (with their message), the host block
 * pool and the toggle controller without a physical pool. Prints one line per
 * check and exits non-zero on the first failure. */
#include <stdio.h>
#include <string.h>

#include "kvattn.h"
#include "kvattn_probes.h"

static int failed = 0;

static void check(int ok, const char* what) {
  printf("%s %s\n", ok ? "ok" : "FAIL", what);
  if (!ok) failed = 1;
}

int main(void) {
  check(kvattn_abi_version() == 1, "abi version");
  check(kvattn_probe_mfma_threads() == 512, "matrix probe workgroup size");
  check(kvattn_probe_read_blocks_waves(256, 8, 4096) == 8192, "read probe grid");
  check(kvattn_probe_mfma(NULL, NULL, 1, 1, NULL) == KV_ERR_INVALID, "matrix probe refuses a null output");

  /* workspace: at least the (m, l, o) partials of every split */
  {
    const int split = kvattn_decode_split_tokens(4096);
    const size_t need = kvattn_decode_workspace_bytes(256, 32, 128, 4096);
    const size_t splits = (size_t)((4096 + split - 1) / split);
    check(split > 0 && need >= (size_t)256 * 32 * splits * (128 + 2) * 4, "decode workspace");
    check(kvattn_decode_workspace_bytes(-1, 32, 128, 4096) == 0, "decode workspace of a bad shape");
  }

  /* a null query with sequences to decode is rejected before any launch */
  {
    char buf[16];
    const int rc = kvattn_decode(NULL, buf, 10, (const int32_t*)buf, (const int32_t*)buf, buf,
                                 4, 32, 8, 128, 16, 4, 64, 0.088f, KV_BF16, buf, 1 << 20, NULL);
    check(rc == KV_ERR_INVALID, "decode rejects a null query");
    check(strncmp(kv_last_error(), "kvattn_decode", 13) == 0, "error message names the call");
  }

  /* the host block pool: base ids first, elastic ids only while admitted */
  {
    kvblocks* b = NULL;
    int32_t ids[6];
    check(kvblocks_create(4, 2, &b) == KV_OK && b != NULL, "kvblocks_create");
    check(kvblocks_num_free(b) == 4, "elastic ids not admitted at first");
    check(kvblocks_alloc(b, 5, ids) == KV_ERR_OOM, "no more than the admitted ids");
    check(kvblocks_set_elastic(b, 1) == KV_OK && kvblocks_num_free(b) == 6, "admit the elastic ids");
    check(kvblocks_alloc(b, 5, ids) == KV_OK, "allocate five");
    {
      int base_first = 1, k;
      for (k = 0; k < 4; ++k) base_first &= ids[k] < 4;
      check(base_first && ids[4] >= 4 && kvblocks_live_elastic(b) == 1, "base ids first");
    }
    check(kvblocks_free(b, 2, ids) == KV_OK && kvblocks_free(b, 1, ids) == KV_ERR_INVALID,
          "double free rejected");
    {
      int32_t from[4], to[4];
      int n = 0;
      check(kvblocks_plan_drain(b, 4, from, to, &n) == KV_OK && n == 1 && from[0] == ids[4] &&
                to[0] < 4, "drain plan moves the elastic id to a base id");
    }

    /* the controller over the block pool alone: commit after the hysteresis
     * steps of decode, decommit before a prefill */
    {
      kvctl* c = NULL;
      int action = -1, commits = 0, decommits = 0;
      kvblocks* b2 = NULL;
      double ms = 0.0;
      check(kvblocks_create(8, 4, &b2) == KV_OK, "second block pool");
      check(kvctl_create(NULL, b2, 2, &c) == KV_OK && c != NULL, "kvctl_create without a pool");
      check(kvctl_before_step(c, 0, &action, &ms) == KV_OK && action == KVCTL_NONE, "decode step 1");
      check(kvctl_before_step(c, 0, &action, &ms) == KV_OK && action == KVCTL_COMMIT &&
                kvctl_is_committed(c) && kvblocks_is_admitted(b2), "commit after two decode steps");
      check(kvctl_before_step(c, 1, &action, &ms) == KV_OK && action == KVCTL_DECOMMIT &&
                !kvctl_is_committed(c) && !kvblocks_is_admitted(b2), "decommit before a prefill");
      check(kvctl_counts(c, &commits, &decommits) == KV_OK && commits == 1 && decommits == 1,
            "toggle counts");
      kvctl_destroy(c);
      kvblocks_destroy(b2);
    }
    kvblocks_destroy(b);
  }
  printf("%s\n", failed ? "FAILED" : "ALL OK");
  return failed;
}
