// Test-only shim: exposes rocRAND's host-callable Philox4x32-10 bijection
// (an independent, open-source implementation of the SC'11 generator) so the
// oracle's own Philox can be checked against it.  Built by the test suite.
#include <cstdint>
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_philox4x32_10.h>

namespace {
struct ExposedPhilox : rocrand_device::philox4x32_10_engine {
  uint4 bijection(uint4 counter, uint2 key) { return this->ten_rounds(counter, key); }
};
}  // namespace

extern "C" void shim_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out, int n) {
  ExposedPhilox eng;
  for (int i = 0; i < n; ++i) {
    uint4 c{ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]};
    uint2 k{key[2 * i], key[2 * i + 1]};
    uint4 r = eng.bijection(c, k);
    out[4 * i] = r.x; out[4 * i + 1] = r.y; out[4 * i + 2] = r.z; out[4 * i + 3] = r.w;
  }
}
