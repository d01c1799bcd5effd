/* A plain C99 client of the library, built by the CPU test suite with
 * -std=c99 -pedantic -Werror: the header must be valid C, and the host entry
 * points must link and work from C.  Encodes the 2 x 3 matrix
 *     1   0   2
 *     0  -0  -1
 * with tile height 2 (one tile), checks the size plan, the header counts and
 * the column maxima, decodes it back (the -0 is not stored) and checks two status strings.
 * Exit status 0 on success, otherwise the number of the failed check. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "celty.h"

int main(void) {
  const uint16_t W[6] = {0x3C00u, 0x0000u, 0x4000u, 0x0000u, 0x8000u, 0xBC00u};
  const uint16_t want[6] = {0x3C00u, 0x0000u, 0x4000u, 0x0000u, 0x0000u, 0xBC00u};
  const uint8_t want_mask[6] = {1, 0, 1, 0, 0, 1};
  int64_t G = 0, nnz = 0, pad = 0;
  uint32_t gptr[4], runs[2];
  uint16_t values[16] __attribute__((aligned(16)));
  uint16_t colmax[4] __attribute__((aligned(4)));
  uint16_t Wd[6];
  uint8_t md[6];
  celty_rlc_csc enc;

  if (celty_encode_plan(W, 3, NULL, 3, 2, 3, 2, CELTY_LAYOUT_RLC, &G, &nnz, &pad) != CELTY_OK) return 1;
  /* column 0 holds one value, column 1 none (-0 is dropped), column 2 two:
     two 8-entry groups, three stored values, no padding */
  if (G != 2 || nnz != 3 || pad != 0) return 2;
  if (celty_encode(W, 3, NULL, 3, 2, 3, 2, CELTY_LAYOUT_RLC, gptr, values, runs, colmax, G, &enc, 1) != CELTY_OK)
    return 3;
  if (enc.version != CELTY_FORMAT_VERSION || enc.T != 1 || enc.n_groups != 2 || enc.max_abs != 2.0f) return 4;
  /* column maxima: |1|, nothing stored (+0), |-1| and 2 -> 2 */
  if (colmax[0] != 0x3C00u || colmax[1] != 0x0000u || colmax[2] != 0x4000u || enc.colmax != colmax) return 10;
  if (gptr[0] != 0 || gptr[1] != 1 || gptr[2] != 1 || gptr[3] != 2) return 5;
  if (celty_decode(&enc, Wd, md) != CELTY_OK) return 6;
  if (memcmp(Wd, want, sizeof want) != 0 || memcmp(md, want_mask, sizeof want_mask) != 0) return 7;
  if (celty_encode_plan(NULL, 3, NULL, 3, 2, 3, 2, CELTY_LAYOUT_RLC, &G, &nnz, &pad) != CELTY_EINVAL) return 8;
  if (strstr(celty_status_string(CELTY_EFORMAT), "RLC-CSC") == NULL) return 9;
  printf("c abi client: ok (%s)\n", celty_status_string(CELTY_OK));
  return 0;
}
