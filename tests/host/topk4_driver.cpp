// Host driver for the streaming top-k of blocks of four: reads rows of 3D
// keys in code order (channel-major, frequency j = 1..3 minor), runs the
// selection residual_select4 runs per lane (groups of 16 channels of one
// frequency absorbed into the top-RS list, then the selection pass in code
// order), and prints the selected positions 3c + j - 1.
#include <cstdio>
#include <cstdint>
#include <vector>
#include "../../paper_2607_06519_amd/csrc/topk_net.h"

template <int D, int RS>
static void run_rows(int k, int n) {
  std::vector<uint32_t> key(3 * D);
  for (int r = 0; r < n; ++r) {
    for (int i = 0; i < 3 * D; ++i) {
      unsigned v;
      if (scanf("%u", &v) != 1) return;
      key[i] = v;
    }
    uint32_t R[RS];
    for (int i = 0; i < RS; ++i) R[i] = 0u;
    for (int ch = 0; ch < D / 16; ++ch)
      for (int j = 0; j < 3; ++j) {
        uint32_t g[16];
        for (int c = 0; c < 16; ++c) g[c] = key[(16 * ch + c) * 3 + j];
        fdkv::net::absorb16<RS>(R, g);
      }
    int need_eq;
    const uint32_t tau = fdkv::net::list_threshold<RS>(R, k, &need_eq);
    int eq = 0, s = 0;
    for (int i = 0; i < 3 * D; ++i) {
      const bool take = key[i] > tau || (key[i] == tau && eq < need_eq);
      eq += key[i] == tau ? 1 : 0;
      if (take) {
        printf("%d ", i);
        ++s;
      }
    }
    printf("\n");
  }
}

int main() {
  int D, RS, k, n;
  if (scanf("%d %d %d %d", &D, &RS, &k, &n) != 4) return 2;
  if (D == 64 && RS == 16) run_rows<64, 16>(k, n);
  else if (D == 64 && RS == 32) run_rows<64, 32>(k, n);
  else if (D == 64 && RS == 64) run_rows<64, 64>(k, n);
  else if (D == 128 && RS == 16) run_rows<128, 16>(k, n);
  else if (D == 128 && RS == 32) run_rows<128, 32>(k, n);
  else if (D == 128 && RS == 64) run_rows<128, 64>(k, n);
  else if (D == 128 && RS == 128) run_rows<128, 128>(k, n);
  else return 3;
  return 0;
}
