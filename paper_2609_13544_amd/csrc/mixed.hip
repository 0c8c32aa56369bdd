// Pass 1 of the error signature for mixed-precision pairs (Section III-C:
// an FP32 golden output against the same operation run in FP16 or FP64):
// one instantiation of the chunk pass per accepted golden/test combination.
#include "sig_chunk.h"

namespace peat {

hipError_t launch_sig_mixed_kind(const SigParams &p, int kind, int64_t n, hipStream_t s) {
    static_assert(kKindTypes[3][1] == PEAT_F64 && kKindTypes[9][0] == PEAT_BF16, "kind table order");
    switch (kind) {
        case 3: return launch_kind<PEAT_F32, PEAT_F64>(p, n, s);
        case 4: return launch_kind<PEAT_F32, PEAT_F16>(p, n, s);
        case 5: return launch_kind<PEAT_F32, PEAT_BF16>(p, n, s);
        case 6: return launch_kind<PEAT_F16, PEAT_F32>(p, n, s);
        case 7: return launch_kind<PEAT_BF16, PEAT_F32>(p, n, s);
        case 8: return launch_kind<PEAT_F16, PEAT_F64>(p, n, s);
        case 9: return launch_kind<PEAT_BF16, PEAT_F64>(p, n, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace peat
