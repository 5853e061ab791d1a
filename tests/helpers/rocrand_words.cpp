// Test helper: prints Philox4x32-10 words from rocRAND's header-only engine, an
// implementation independent of the oracle.  The engine's documented semantics
// (seed -> key, subsequence -> upper counter words, offset -> words skipped) make
// word number `offset` of subsequence `sid` the noise word of absolute element
// index `offset`.
// usage: rocrand_words SEED SID OFFSET COUNT   (decimal; prints COUNT hex words)
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>
int main(int argc, char** argv) {
    if (argc != 5) return 2;
    unsigned long long seed = strtoull(argv[1], 0, 10), sid = strtoull(argv[2], 0, 10);
    unsigned long long off = strtoull(argv[3], 0, 10), n = strtoull(argv[4], 0, 10);
    rocrand_device::philox4x32_10_engine e(seed, sid, off);
    for (unsigned long long i = 0; i < n; ++i) printf("%08x\n", e());
    return 0;
}
