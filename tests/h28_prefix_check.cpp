// Host build of the library's 28-point column routine (quant_device.h):
// its shared partial sums must equal the in-order sums of the definition
// (acc = +-z[0], then acc +-= z[a] for a = 1..27 with the signs of H28) bit
// for bit, for every column and both column halves, on seeded inputs that
// span wide exponent ranges.  Prints the mismatch counts; exit status 1 if
// any.
#include "quant_device.h"

#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>

using dptq::qd::h28_column;
using dptq::qd::kH28;

template <int B0, int NB>
long check(std::mt19937& g, int iters) {
  long bad = 0;
  std::uniform_real_distribution<float> u(-1.f, 1.f);
  std::uniform_int_distribution<int> e(-40, 40);
  for (int it = 0; it < iters; ++it) {
    const int spread = (it % 5) * 10 + 1;
    float z[28];
    for (int a = 0; a < 28; ++a) z[a] = std::ldexp(u(g), e(g) % spread);
    float got[NB];
    h28_column<B0, NB>(z, [&](int b, float v) { got[b] = v; });
    for (int b = 0; b < NB; ++b) {
      volatile float acc = kH28.e[0][B0 + b] > 0 ? z[0] : -z[0];
      for (int a = 1; a < 28; ++a) acc = kH28.e[a][B0 + b] > 0 ? acc + z[a] : acc - z[a];
      const float want = acc;
      if (std::memcmp(&want, &got[b], sizeof(float)) != 0) ++bad;
    }
  }
  return bad;
}

int main() {
  std::mt19937 g(2024);
  const long all = check<0, 28>(g, 400000);
  const long lo = check<0, 14>(g, 200000);
  const long hi = check<14, 14>(g, 200000);
  std::printf("mismatches: 28 columns %ld, columns 0-13 %ld, columns 14-27 %ld\n", all, lo, hi);
  return (all || lo || hi) ? 1 : 0;
}
