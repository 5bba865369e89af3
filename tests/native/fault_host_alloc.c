/* Forced host-allocation failure under AddressSanitizer with leak checking:
 * with BOOST_FAULT_HOST_ALLOC set, creating a KV pool on a plan-only context
 * fails with BOOST_ENOMEM and leaves no object behind; without it the same
 * call succeeds.  Built and run by tests/test_fault_cpu.py against the
 * host-sanitizer build of the library; LeakSanitizer reports any allocation
 * the failed calls did not release. */
#include <stdio.h>
#include <stdlib.h>

#include "boost_cap.h"

int main(void) {
  boost_ctx* ctx = NULL;
  if (boost_init(-1, &ctx) != BOOST_OK) return 2;
  boost_kv_cfg cfg = {1, 8, 128, 16, 100000, 4, BOOST_KV_LPP, 32, 64, 256, 0};
  boost_kv_pool* p = NULL;
  setenv("BOOST_FAULT_HOST_ALLOC", "1", 1);
  for (int i = 0; i < 3; ++i) {
    int rc = boost_kv_pool_create(ctx, &cfg, &p);
    if (rc != BOOST_ENOMEM || p) {
      printf("expected ENOMEM and no pool, got %d\n", rc);
      return 3;
    }
  }
  unsetenv("BOOST_FAULT_HOST_ALLOC");
  if (boost_kv_pool_create(ctx, &cfg, &p) != BOOST_OK || !p) return 4;
  boost_kv_pool_destroy(p);
  boost_shutdown(ctx);
  printf("fault-injection ok\n");
  return 0;
}
