// Independent Philox4x32-10 reference: rocRAND's source header, host side.
// Reads lines "c0 c1 c2 c3 k0 k1" (hex) and prints the 4 output words (hex).
// rocRAND seeds the key with the 64-bit seed (lo, hi); the counter is set
// through the engine state before calling its ten-round function.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdint>
struct probe_engine : rocrand_device::philox4x32_10_engine {
    uint4 run(uint4 ctr, uint2 key) { return this->ten_rounds(ctr, key); }
};
int main() {
    unsigned c0, c1, c2, c3, k0, k1;
    probe_engine e;
    while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        uint4 ctr = make_uint4(c0, c1, c2, c3);
        uint2 key = make_uint2(k0, k1);
        uint4 o = e.run(ctr, key);
        std::printf("%08x %08x %08x %08x\n", o.x, o.y, o.z, o.w);
    }
    return 0;
}
