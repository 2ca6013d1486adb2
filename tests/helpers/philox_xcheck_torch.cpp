// Independent Philox4x32-10 reference: PyTorch's source header (compiled here).
// Reads lines "c0 c1 c2 c3 k0 k1" (hex) and prints the 4 output words (hex).
// torch's engine: key = seed (lo, hi); counter = (offset lo, offset hi,
// subsequence lo, subsequence hi); operator() returns words 0..3 in order.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
#include <cstdint>
int main() {
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%x %x %x %x %x %x", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        uint64_t seed = ((uint64_t)k1 << 32) | k0;
        uint64_t offset = ((uint64_t)c1 << 32) | c0;
        uint64_t subseq = ((uint64_t)c3 << 32) | c2;
        at::Philox4_32 eng(seed, subseq, offset);
        unsigned o0 = eng(), o1 = eng(), o2 = eng(), o3 = eng();
        std::printf("%08x %08x %08x %08x\n", o0, o1, o2, o3);
    }
    return 0;
}
