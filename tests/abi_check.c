/* Host-only use of the C ABI from plain C: compiles against the public
 * header (as C99 and as C++), links against the built library and prints
 * the results of the host-side queries and of calls that must fail host
 * validation (no GPU work is enqueued by any call here). */
#include <stdio.h>
#include <stdint.h>

#include "sketchwalk.h"

int main(void) {
  int32_t cu[3] = {0, 100, 400};
  int64_t nb = 0, nm = 0;
  int32_t max_b = 0, kmax = 0;
  int rc;
  printf("version %d\n", sw_abi_version());
  rc = sw_layout(2, cu, 64, &nb, &nm, &max_b);
  printf("layout %d %lld %lld %d\n", rc, (long long)nb, (long long)nm, (int)max_b);
  rc = sw_select_max_count(2, cu, 64, 0, 20, SW_FORCE_FIRST | SW_FORCE_LAST, &kmax);
  printf("max_count %d %d\n", rc, (int)kmax);
  printf("sketch_ws %lld\n", (long long)sw_sketch_workspace_bytes(32, 8, 128, 2, cu, 64));
  printf("walk_ws %lld %lld\n", (long long)sw_walk_workspace_bytes(SW_WALK_MATPOW, 2, cu, 64),
         (long long)sw_walk_workspace_bytes(SW_WALK_POWER, 2, cu, 64));
  printf("state_bytes %lld\n", (long long)sw_decode_state_bytes(16, 128, 64, 1028));
  printf("step_ws %lld\n", (long long)sw_decode_step_workspace_bytes(16, 32, 8, 128));
  /* an unknown walk variant: rejected before any pointer is used */
  rc = sw_walk_update_variant(7, NULL, NULL, 8, 1.0, 2, cu, 64, NULL, NULL, NULL, 0, NULL);
  printf("bad_variant %d %s\n", rc, sw_last_error());
  /* more than SW_MAX_BLOCKS blocks in a sequence */
  {
    int32_t big[2] = {0, (SW_MAX_BLOCKS + 1) * 16};
    rc = sw_walk_update(NULL, NULL, 8, 1, big, 16, NULL, NULL, NULL);
    printf("too_many_blocks %d\n", rc);
  }
  return 0;
}
