// Test-only cross-check: the v-th 32-bit output of PyTorch's open-source Philox
// engine (ATen/core/PhiloxRNGEngine.h) seeded with r, subsequence 0.  The engine's
// offset counts 128-bit blocks, so it starts at block floor(v/4) and the
// (v mod 4 + 1)-th draw is the wanted word.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdint>

extern "C" void aten_stream_word(const uint32_t* v, const uint64_t* r, int64_t n,
                                 uint32_t* out) {
  for (int64_t i = 0; i < n; ++i) {
    at::philox_engine engine(r[i], 0, v[i] / 4u);
    uint32_t word = 0;
    for (uint32_t j = 0; j <= v[i] % 4u; ++j) word = engine();
    out[i] = word;
  }
}
