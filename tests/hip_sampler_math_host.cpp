// Host build of the HIP path's sampler arithmetic (paper_2505_17218_amd/csrc/sampler_math.h),
// so CPU tests can compare it bit for bit with the oracle.  Reads lines from stdin:
//   log <hex float bits>       -> hex bits of own_log
//   gumbel <hex u32>           -> hex bits of gumbel_from_bits
//   philox <c0> <c1> <c2> <c3> <k0> <k1>   (hex) -> four hex words
#include <cstdio>
#include <cstring>
#include "sampler_math.h"

int main() {
    char op[16];
    while (scanf("%15s", op) == 1) {
        if (!strcmp(op, "log")) {
            unsigned b;
            if (scanf("%x", &b) != 1) return 2;
            printf("%08x\n", dash::f_bits(dash::own_log(dash::bits_f(b))));
        } else if (!strcmp(op, "gumbel")) {
            unsigned x;
            if (scanf("%x", &x) != 1) return 2;
            printf("%08x\n", dash::f_bits(dash::gumbel_from_bits(x)));
        } else if (!strcmp(op, "philox")) {
            unsigned c[4], k[2];
            if (scanf("%x %x %x %x %x %x", &c[0], &c[1], &c[2], &c[3], &k[0], &k[1]) != 6) return 2;
            dash::U4 r = dash::philox4x32_10(dash::U4{c[0], c[1], c[2], c[3]}, k[0], k[1]);
            printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
        } else {
            return 3;
        }
    }
    return 0;
}
