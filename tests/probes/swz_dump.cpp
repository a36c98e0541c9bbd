// Prints the chunk swizzle of the matrix kernels' LDS tiles (host build of
// mfma_tiles.h): one line per head dimension, the XOR mask of rows 0..15.
#include "../../paper_2609_32704_amd/csrc/mfma_tiles.h"
#include <stdio.h>
int main() {
  printf("128");
  for (int r = 0; r < 16; ++r) printf(" %d", cowa::swz<16>(r));
  printf("\n64");
  for (int r = 0; r < 16; ++r) printf(" %d", cowa::swz<8>(r));
  printf("\n");
  return 0;
}
