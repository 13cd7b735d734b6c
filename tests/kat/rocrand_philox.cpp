// Test-only helper: exposes rocRAND's own Philox4x32-10 engine (host side of
// its header API) so the oracle's Philox can be checked against an
// implementation it shares nothing with.  Built by the project build step;
// loaded only by the test suite.
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_philox4x32_10.h>
#include <stdint.h>

extern "C" void kat_rocrand_philox(uint64_t seed, uint64_t ctr_low64, uint64_t ctr_high64,
                                   uint32_t out[4])
{
    rocrand_state_philox4x32_10 state;
    // subsequence selects counter words 2..3; the skip (in 32-bit outputs,
    // four per block) selects counter words 0..1.  The skip is applied in
    // pieces so that 4 * ctr_low64 never overflows 64 bits.
    rocrand_init(seed, ctr_high64, 0ull, &state);
    const unsigned long long low62 = ctr_low64 & ((1ull << 62) - 1ull);
    skipahead(low62 * 4ull, &state);
    for (unsigned long long q = 0; q < (ctr_low64 >> 62); ++q) {
        skipahead(1ull << 63, &state);  // 2^62 blocks in two halves
        skipahead(1ull << 63, &state);
    }
    uint4 r = rocrand4(&state);
    out[0] = r.x;
    out[1] = r.y;
    out[2] = r.z;
    out[3] = r.w;
}
