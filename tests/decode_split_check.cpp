// Prints the decode launch shape the decode kernel uses (decode_shape_for)
// for each case read from stdin: "nbq nft heads n_cu bits" per line ->
// "S_q S_f".
#include <cstdio>

#include "decode_split.h"

int main() {
  long long nbq, nft, heads, n_cu;
  int bits;
  while (std::scanf("%lld %lld %lld %lld %d", &nbq, &nft, &heads, &n_cu, &bits) == 5) {
    const hyq::DecodeShape d = hyq::decode_shape_for(nbq, nft, heads, n_cu, bits);
    std::printf("%d %d\n", d.S_q, d.S_f);
  }
  return 0;
}
