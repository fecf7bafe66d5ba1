// Host driver for the register top-k network of the HIP path: reads rows of
// keys from stdin and prints the selected channels (ascending), so that the
// CPU tests can compare the network with an independent sort.
#include <cstdio>
#include <cstdint>
#include <vector>
#include "../../paper_2607_06519_amd/csrc/topk_net.h"

// keep = 0: kth_largest (destroys its copy of the keys); keep = 1:
// kth_largest_keep (leaves the keys, list size GS)
template <int D, int GS>
static void run_rows(int k, int n, int keep) {
  std::vector<uint32_t> key(D), work(D);
  for (int r = 0; r < n; ++r) {
    for (int c = 0; c < D; ++c) {
      unsigned v;
      if (scanf("%u", &v) != 1) return;
      key[c] = v;
      work[c] = v;
    }
    const uint32_t tau = keep ? fdkv::net::kth_largest_keep<D, GS>(key.data(), k)
                              : fdkv::net::kth_largest<D, GS>(work.data(), k);
    uint32_t mask[D / 32];
    fdkv::net::select_mask<D>(key.data(), tau, k, mask);
    for (int s = 0; s < k; ++s) printf("%d ", fdkv::net::pop_lowest<D>(mask));
    printf("\n");
  }
}

int main() {
  int D, GS, k, n, keep;
  if (scanf("%d %d %d %d %d", &D, &GS, &k, &n, &keep) != 5) return 2;
  if (D == 64 && GS == 8) run_rows<64, 8>(k, n, keep);
  else if (D == 64 && GS == 16) run_rows<64, 16>(k, n, keep);
  else if (D == 64 && GS == 64) run_rows<64, 64>(k, n, keep);
  else if (D == 128 && GS == 8) run_rows<128, 8>(k, n, keep);
  else if (D == 128 && GS == 16) run_rows<128, 16>(k, n, keep);
  else if (D == 128 && GS == 128) run_rows<128, 128>(k, n, keep);
  else return 3;
  return 0;
}
