// Independent Philox4x32-10 reference for the oracle's pin test: runs the
// ten-round function of rocRAND's header-only engine on the host. Reads lines
// "c0 c1 c2 c3 k0 k1" (decimal) from stdin and prints the four output words.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

struct philox_probe : rocrand_device::philox4x32_10_engine {
    uint4 run(uint4 c, uint2 k) { return ten_rounds(c, k); }
};

int main() {
    philox_probe p;
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        uint4 c = {c0, c1, c2, c3};
        uint2 k = {k0, k1};
        uint4 o = p.run(c, k);
        std::printf("%u %u %u %u\n", o.x, o.y, o.z, o.w);
    }
    return 0;
}
