// Host driver for the DCT-II(4) butterfly of the HIP path: reads four
// float32 bit patterns per line and prints the bit patterns of Z_1, Z_2, Z_3.
#include <cstdio>
#include <cstdint>
#include <cstring>
#include "../../paper_2607_06519_amd/csrc/dct4.h"

int main() {
  unsigned u[4];
  while (scanf("%u %u %u %u", &u[0], &u[1], &u[2], &u[3]) == 4) {
    float x[4], z[3];
    for (int i = 0; i < 4; ++i) memcpy(&x[i], &u[i], 4);
    fdkv::dct4_high(x[0], x[1], x[2], x[3], z[0], z[1], z[2]);
    unsigned o[3];
    for (int i = 0; i < 3; ++i) memcpy(&o[i], &z[i], 4);
    printf("%u %u %u\n", o[0], o[1], o[2]);
  }
  return 0;
}
