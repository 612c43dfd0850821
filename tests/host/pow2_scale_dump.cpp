// Prints, for every 15-bit bf16 magnitude pattern, the power-of-two block scale
// and multiplier of the kernels' quant_math.hpp (compiled for the host):
// "amax16 scale_bits r_bits" per line.
#include <stdio.h>

#include "quant_math.hpp"

int main() {
  for (uint32_t a = 0; a < 0x7F80u; ++a) {
    const fp8rl::qmath::BlockScale b = fp8rl::qmath::block_scale_pow2(a);
    printf("%u %u %u\n", a, fp8rl::qmath::as_uint(b.scale), fp8rl::qmath::as_uint(b.r));
  }
  return 0;
}
