// Second-opinion Philox4x32-10: PyTorch ATen's header-only philox_engine,
// compiled from source.  Reads "seed stream offset" triples on stdin and
// prints the first four 32-bit outputs of philox_engine(seed, stream, offset),
// i.e. one Philox block for key = seed and counter = (offset lo, offset hi,
// stream lo, stream hi).
#include <ATen/core/PhiloxRNGEngine.h>
#include <cinttypes>
#include <cstdio>

int main() {
  unsigned long long seed, stream, offset;
  while (std::scanf("%llu %llu %llu", &seed, &stream, &offset) == 3) {
    at::philox_engine e(seed, stream, offset);
    for (int i = 0; i < 4; ++i) std::printf("%u%c", e(), i == 3 ? '\n' : ' ');
  }
  return 0;
}
