// Independent Philox4x32-10 reference for the oracle's pin tests: rocRAND's
// header-only engine, compiled for and run on the host CPU.
//
// usage: philox_rocrand_ref SEED SUBSEQ Q0 NQ   -> NQ lines of 4 hex words,
// the counter blocks Q0 .. Q0+NQ-1 of subsequence SUBSEQ under SEED.
// rocRAND's engine keys with (seed lo, seed hi) and starts from counter
// (0, 0, subseq lo, subseq hi); skipping 4*Q outputs adds Q to words 0..1.
#include <cstdio>
#include <cstdlib>
#include <rocrand/rocrand_philox4x32_10.h>

int main(int argc, char** argv) {
    if (argc != 5) { std::fprintf(stderr, "usage: %s seed subseq q0 nq\n", argv[0]); return 2; }
    unsigned long long seed = std::strtoull(argv[1], nullptr, 0);
    unsigned long long sub  = std::strtoull(argv[2], nullptr, 0);
    unsigned long long q0   = std::strtoull(argv[3], nullptr, 0);
    long long nq            = std::strtoll(argv[4], nullptr, 0);
    rocrand_device::philox4x32_10_engine eng(seed, sub, 4ull * q0);
    for (long long q = 0; q < nq; ++q) {
        unsigned int w0 = eng(), w1 = eng(), w2 = eng(), w3 = eng();
        std::printf("%08x %08x %08x %08x\n", w0, w1, w2, w3);
    }
    return 0;
}
