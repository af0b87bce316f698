// Independent Philox4x32-10 stream for pinning the oracle's generator: the
// rocRAND device engine, compiled for the host only.  Prints, for the seed
// subsequence and offset (in 32-bit outputs) given on the command line, the
// first n 4-word blocks that rocrand4() returns, one block per line in hex.
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_kernel.h>

int main(int argc, char** argv)
{
    if (argc != 5) {
        std::fprintf(stderr, "usage: %s seed subsequence offset n\n", argv[0]);
        return 2;
    }
    const unsigned long long seed = std::strtoull(argv[1], nullptr, 0);
    const unsigned long long subseq = std::strtoull(argv[2], nullptr, 0);
    const unsigned long long offset = std::strtoull(argv[3], nullptr, 0);
    const int n = std::atoi(argv[4]);
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, subseq, offset, &st);
    for (int i = 0; i < n; ++i) {
        const uint4 x = rocrand4(&st);
        std::printf("%08x %08x %08x %08x\n", x.x, x.y, x.z, x.w);
    }
    return 0;
}
