// Host build of the routing order used by the HIP kernels (xhc_device.h):
// route_select (the multi-kernel path) and the 16-lane rank of the
// single-pass kernel, run on the CPU over logit patterns read from stdin.
//
// Input, one token per line: m k z_0 .. z_15, each z as the hex bits of an
// fp32 value.  Output, one line per token: the k stream indices chosen by
// route_select, then the k chosen from the ranks (slot m + rank for
// candidates with rank < k - m; fixed slots 0..m-1), then the 16 - m ranks
// of the candidates.
#include <cstdio>
#include <cstring>

#include "xhc_device.h"

int main() {
  int m = 0, k = 0;
  while (std::scanf("%d %d", &m, &k) == 2) {
    float z[16];
    for (int i = 0; i < 16; ++i) {
      unsigned u = 0;
      if (std::scanf("%x", &u) != 1) return 2;
      std::memcpy(&z[i], &u, 4);
    }
    int32_t sel[xhc::kMaxK];
    float zsel[xhc::kMaxK];
    xhc::route_select<16>(z, 16, m, k, sel, zsel);
    int32_t key[16];
    for (int i = 0; i < 16; ++i) key[i] = xhc::logit_key(z[i]);
    int32_t fused[xhc::kMaxK];
    for (int j = 0; j < k; ++j) fused[j] = -1;
    int rank[16];
    for (int lane = 0; lane < 16; ++lane) {
      rank[lane] = xhc::route_rank16([&](int r) { return key[(lane - r) & 15]; }, key[lane], lane, m);
      if (lane < m) fused[lane] = lane;
      else if (rank[lane] < k - m) fused[m + rank[lane]] = lane;
    }
    for (int j = 0; j < k; ++j) std::printf("%d ", sel[j]);
    for (int j = 0; j < k; ++j) std::printf("%d ", fused[j]);
    for (int i = m; i < 16; ++i) std::printf("%d ", rank[i]);
    std::printf("\n");
  }
  return 0;
}
