// Reads fp64 values (16 hex digits of their bits, one per line) and prints, per value, the bits of
// f32_round_odd(value) as 8 hex digits: the kernels' fp64 -> bf16 rounding is this float rounded
// to nearest-even bf16 by the hardware.  tests/test_round_odd.py drives it.
#include <cstdio>
#include <cstring>

#include "kparams.hpp"

int main() {
    unsigned long long bits;
    while (std::scanf("%llx", &bits) == 1) {
        double d;
        std::memcpy(&d, &bits, sizeof d);
        const float f = leyline::f32_round_odd(d);
        unsigned int u;
        std::memcpy(&u, &f, sizeof u);
        std::printf("%08x\n", u);
    }
    return 0;
}
