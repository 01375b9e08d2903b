// Test-only cross-check: the v-th 32-bit output of rocRAND's open-source
// philox4x32_10 engine (rocrand/rocrand_philox4x32_10.h, host side) seeded with r,
// subsequence 0; the engine's offset counts 32-bit outputs.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdint>

extern "C" void rocrand_stream_word(const uint32_t* v, const uint64_t* r, int64_t n,
                                    uint32_t* out) {
  for (int64_t i = 0; i < n; ++i) {
    rocrand_device::philox4x32_10_engine engine(r[i], 0, v[i]);
    out[i] = engine.next();
  }
}
