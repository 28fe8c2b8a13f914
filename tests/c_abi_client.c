/*
 * A C99 client of libfastvr: include/fastvr.h compiles as C and the host-side
 * paths of the C ABI work from C without a GPU (version, status strings, tile
 * placement, argument validation before any HIP call).  Built and run by
 * tests/test_abi.py; prints "ok" and exits 0 on success, else the failed check.
 */
#include <stdio.h>
#include <string.h>

#include "fastvr.h"

#define CHECK(cond)                                        \
  do {                                                     \
    if (!(cond)) {                                         \
      printf("failed: %s (line %d)\n", #cond, __LINE__);   \
      return 1;                                            \
    }                                                      \
  } while (0)

int main(void) {
  int64_t n_tiles = 0, tile_len = 0;
  fastvr_status s;
  CHECK(fastvr_abi_version() == FASTVR_ABI_VERSION);
  CHECK(strcmp(fastvr_status_string(FASTVR_OK), "FASTVR_OK") == 0);
  /* the 1080p latent width 120 with 64-wide tiles overlapping by 16: 3 tiles */
  CHECK(fastvr_tile_axis(120, 64, 16, &n_tiles, &tile_len) == FASTVR_OK);
  CHECK(n_tiles == 3 && tile_len == 64);
  /* a NULL q with a non-empty problem is rejected on the host, with a message */
  s = fastvr_chunk_attn_fwd(NULL, NULL, NULL, NULL, NULL, 1, 2, 64, 64, 64, 16, 0, -1, 0.125f, NULL);
  CHECK(s == FASTVR_ERR_INVALID_ARGUMENT);
  CHECK(strlen(fastvr_last_error()) > 0);
  /* a tile placement on an empty axis is rejected */
  s = fastvr_tile_axis(0, 64, 16, &n_tiles, &tile_len);
  CHECK(s == FASTVR_ERR_INVALID_ARGUMENT);
  /* an empty problem is a successful no-op */
  s = fastvr_one_step_update(NULL, NULL, NULL, 0, 0.5f, 0, NULL);
  CHECK(s == FASTVR_OK);
  printf("ok\n");
  return 0;
}
