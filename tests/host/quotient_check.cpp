// Host-side check of the kernels' scale/quotient arithmetic (quant_math.hpp):
// for every bf16 pair (x, amax) with |x| <= amax in the chosen amax set, the
// kernels' quotient (block reciprocal + Markstein correction, with the 2^64
// pre-scaling for tiny blocks) must equal the IEEE fp32 division x / scale
// bit for bit, except that
//   * quotients below 2^-11 only need to stay below 2^-11: every value under
//     2^-10 rounds to an E4M3 zero, so a last-bit difference there (it occurs
//     when x is an fp32 subnormal and the correction step is not exact)
//     cannot change a code, and
//   * a zero result may lose its sign (the kernels OR the input sign back).
// Usage: quotient_check [stride]   (stride 1 = every amax; prints mismatches)
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "quant_math.hpp"

using namespace fp8rl::qmath;

static float f_of(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }
static uint32_t u_of(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }

int main(int argc, char** argv) {
  const int stride = argc > 1 ? std::atoi(argv[1]) : 1;
  long long pairs = 0, bad = 0;
  for (uint32_t a16 = 1; a16 < 0x7F80; ++a16) {
    const bool special = a16 < 0x0100 || (a16 & 0x7F) == 0 || (a16 & 0x7F) == 0x7F || a16 > 0x7F00 ||
                         (a16 >= 0x0C00 && a16 <= 0x0E00);
    if (!special && (a16 % stride) != 0) continue;
    const BlockScale bs = block_scale(a16);
    const float scale = f_of(a16 << 16) / 448.0f;   // IEEE division on the host
    if (u_of(scale) != u_of(bs.scale)) { std::printf("scale mismatch amax=%04x\n", a16); ++bad; }
    for (uint32_t m = 0; m <= a16; ++m) {
      for (uint32_t sgn = 0; sgn < 2; ++sgn) {
        const uint32_t h = m | (sgn << 15);
        float x = f_of(h << 16);
        const volatile float ref = x / scale;
        float xk = bs.prescaled ? x * kPrescale : x;
        const float got = quotient(xk, bs.s, bs.r);
        ++pairs;
        bool ok;
        if (std::fabs(ref) < 0x1p-11f)
          ok = std::fabs(got) < 0x1p-11f;
        else if (ref == 0.0f)
          ok = got == 0.0f;
        else
          ok = u_of(got) == u_of(ref);
        if (!ok) {
          if (bad < 20) std::printf("mismatch amax=%04x x=%04x got %08x want %08x\n", a16, h, u_of(got), u_of((float)ref));
          ++bad;
        }
      }
    }
  }
  std::printf("pairs %lld mismatches %lld\n", pairs, bad);
  return bad ? 1 : 0;
}
