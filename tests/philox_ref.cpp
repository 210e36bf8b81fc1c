// Calls PyTorch's Philox4x32-10 engine for (counter, key) pairs read from stdin.
// philox_engine(seed, subsequence, offset) uses counter = (offset, subsequence) and
// key = seed; four calls return the four words of one block.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
int main() {
    unsigned c0, c1, c2, c3, k0, k1;
    while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
        at::philox_engine e((static_cast<uint64_t>(k1) << 32) | k0, (static_cast<uint64_t>(c3) << 32) | c2,
                            (static_cast<uint64_t>(c1) << 32) | c0);
        unsigned a = e(), b = e(), c = e(), d = e();
        std::printf("%u %u %u %u\n", a, b, c, d);
    }
    return 0;
}
