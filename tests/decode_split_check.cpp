// Prints the decode launch shape chosen by choose_decode_split for each case
// read from stdin: "nbq nft heads n_cu bits" per line -> "S_q S_f".
#include <cstdio>

#include "decode_split.h"

int main() {
  long long nbq, nft, heads, n_cu;
  int bits;
  while (std::scanf("%lld %lld %lld %lld %d", &nbq, &nft, &heads, &n_cu, &bits) == 5) {
    const hyq::DecodeShape d = hyq::choose_decode_split(
        nbq, nft, heads, n_cu, 4, bits == 4 ? 4 : 2, 2LL * 64 * 128 * bits / 8, 2LL * 64 * 128 * 2);
    std::printf("%d %d\n", d.S_q, d.S_f);
  }
  return 0;
}
