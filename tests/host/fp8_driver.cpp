// Host driver for the FP8 E4M3 encoder of the HIP path: reads float32 bit
// patterns from stdin and prints the encoded bytes.
#include <cstdio>
#include <cstdint>
#include <cstring>
#include "../../paper_2607_06519_amd/csrc/fp8.h"

int main() {
  unsigned u;
  while (scanf("%u", &u) == 1) {
    float f;
    memcpy(&f, &u, 4);
    printf("%u\n", (unsigned)fdkv::f32_to_e4m3(f));
  }
  return 0;
}
