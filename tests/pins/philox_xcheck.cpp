// Host-only helper for the oracle's Philox pin: the word streams of two
// independent published Philox4x32-10 engines, rocRAND's device/host engine
// header and ATen's CPU Philox engine header, in the oracle's stream layout
// (element w = output lane w mod 4 of block w / 4, counter words 2-3 zero).
// Nothing here is shared with the oracle or the product.
#include <cstdint>
#include <rocrand/rocrand_philox4x32_10.h>
#include <ATen/core/PhiloxRNGEngine.h>

extern "C" {

// rocRAND engine at subsequence 0, skipping `offset` 32-bit words.
void xc_rocrand_words(uint64_t seed, uint64_t offset, uint64_t n, uint32_t* out)
{
    rocrand_device::philox4x32_10_engine eng(seed, 0, offset);
    for (uint64_t i = 0; i < n; ++i)
        out[i] = eng.next();
}

// ATen engine: its offset counts 128-bit blocks, so start at block offset/4
// and drop the first offset%4 words.
void xc_aten_words(uint64_t seed, uint64_t offset, uint64_t n, uint32_t* out)
{
    at::Philox4_32 eng(seed, 0, offset / 4);
    for (uint64_t i = 0; i < offset % 4; ++i)
        (void)eng();
    for (uint64_t i = 0; i < n; ++i)
        out[i] = eng();
}

}
