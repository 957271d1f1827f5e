// Test-only pin: exposes rocRAND's header implementation of Philox4x32-10
// (a library routine, independent of both the oracle and the HIP kernels) so
// the oracle's Philox can be checked against it on arbitrary counters/keys.
#include <rocrand/rocrand_philox4x32_10.h>
#include <stdint.h>

namespace {
struct ExposedPhilox : rocrand_device::philox4x32_10_engine {
    uint4 rounds(uint4 counter, uint2 key) { return ten_rounds(counter, key); }
};
}  // namespace

extern "C" void pin_philox4x32_10(uint64_t n, const uint32_t* ctr, const uint32_t* key,
                                  uint32_t* out) {
    ExposedPhilox e;
    for (uint64_t i = 0; i < n; ++i) {
        uint4 c = {ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]};
        uint2 k = {key[2 * i], key[2 * i + 1]};
        uint4 r = e.rounds(c, k);
        out[4 * i] = r.x;
        out[4 * i + 1] = r.y;
        out[4 * i + 2] = r.z;
        out[4 * i + 3] = r.w;
    }
}
