// Prints Philox4x32-10 words from rocRAND's header-only engine, run on the
// host, as an outside implementation to check the oracle's Philox against.
// Usage: rocrand_philox_dump seed subsequence offset  -> four hex words
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>

int main(int argc, char** argv)
{
    if (argc != 4) return 2;
    unsigned long long seed = strtoull(argv[1], nullptr, 0);
    unsigned long long sub = strtoull(argv[2], nullptr, 0);
    unsigned long long off = strtoull(argv[3], nullptr, 0);
    rocrand_device::philox4x32_10_engine e(seed, sub, off);
    uint4 v = e.next4();
    std::printf("%08x %08x %08x %08x\n", v.x, v.y, v.z, v.w);
    return 0;
}
