// Reference Philox4x32-10 blocks for the oracle's pins, from rocRAND's
// header implementation (test infrastructure; independent of oracle/ and of
// the GPU library).
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdint>

namespace {
struct Engine : rocrand_device::philox4x32_10_engine {
    uint4 block(uint4 c, uint2 k) { return this->ten_rounds(c, k); }
};
}  // namespace

// count blocks: counter words ctr[4i..4i+3], key words key[2i..2i+1] -> out[4i..4i+3]
extern "C" void ref_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out, int64_t count) {
    Engine e;
    for (int64_t i = 0; i < count; ++i) {
        const uint4 r = e.block(uint4{ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]},
                                uint2{key[2 * i], key[2 * i + 1]});
        out[4 * i] = r.x;
        out[4 * i + 1] = r.y;
        out[4 * i + 2] = r.z;
        out[4 * i + 3] = r.w;
    }
}
