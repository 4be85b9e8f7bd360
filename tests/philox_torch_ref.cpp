// Philox4x32-10 blocks computed by PyTorch's header-only engine (ATen/core/PhiloxRNGEngine.h),
// an implementation of the SC'11 generator written independently of the oracle's. Built on
// the host by the oracle tests and compared with the oracle bit for bit.
//
// The engine is keyed by a 64-bit seed (key words: low, high) and starts at the counter
// (offset low, offset high, subsequence low, subsequence high); its first four outputs are
// the four words of that counter's block.
#include <ATen/core/PhiloxRNGEngine.h>

#include <cstdint>

extern "C" void torch_philox_blocks(int64_t n, const uint32_t* ctr, const uint32_t* key,
                                    uint32_t* out) {
  const uint64_t seed = (uint64_t)key[0] | ((uint64_t)key[1] << 32);
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t* c = ctr + 4 * i;
    const uint64_t offset = (uint64_t)c[0] | ((uint64_t)c[1] << 32);
    const uint64_t subsequence = (uint64_t)c[2] | ((uint64_t)c[3] << 32);
    at::philox_engine e(seed, subsequence, offset);
    for (int j = 0; j < 4; ++j) out[4 * i + j] = e();
  }
}
