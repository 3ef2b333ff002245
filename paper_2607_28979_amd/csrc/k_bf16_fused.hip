// Host side of the fused kernel: shape support and dispatch to the
// per-shape instantiations (k_bf16_fused_inst.hip, built once per shape).
#include "k_bf16_fused_kernel.h"

namespace mot {

#define MOT_DECL(a, b) \
    hipError_t launch_fused_##a##_##b(const Problem& p, const UnitTab& ut, bool routed, hipStream_t stream);
MOT_DECL(128, 128) MOT_DECL(128, 256) MOT_DECL(128, 512)
MOT_DECL(256, 128) MOT_DECL(256, 256) MOT_DECL(256, 512)
MOT_DECL(512, 128) MOT_DECL(512, 256) MOT_DECL(512, 512)
#undef MOT_DECL

namespace {

hipError_t launch_shape(const Problem& p, const UnitTab& ut, bool routed, hipStream_t stream) {
    if (ut.n == 0 || p.n_tok == 0) return hipSuccess;
    const int key = p.d_in * 1000 + p.d_out;
    switch (key) {
        case 128128: return launch_fused_128_128(p, ut, routed, stream);
        case 128256: return launch_fused_128_256(p, ut, routed, stream);
        case 128512: return launch_fused_128_512(p, ut, routed, stream);
        case 256128: return launch_fused_256_128(p, ut, routed, stream);
        case 256256: return launch_fused_256_256(p, ut, routed, stream);
        case 256512: return launch_fused_256_512(p, ut, routed, stream);
        case 512128: return launch_fused_512_128(p, ut, routed, stream);
        case 512256: return launch_fused_512_256(p, ut, routed, stream);
        case 512512: return launch_fused_512_512(p, ut, routed, stream);
        default: return hipErrorNotSupported;
    }
}

}  // namespace

bool fused_supported(const Problem& p) {
    const bool din = p.d_in == 128 || p.d_in == 256 || p.d_in == 512;
    const bool dout = p.d_out == 128 || p.d_out == 256 || p.d_out == 512;
    return din && dout && p.hidden % 64 == 0 && p.E * p.hidden >= 64 && p.E <= MOT_MAX_EXPERTS;
}

int fused_tile_rows(const Problem& p) {
    switch (p.d_in * 1000 + p.d_out) {
        case 128128: return Cfg<128, 128>::BM;
        case 128256: return Cfg<128, 256>::BM;
        case 128512: return Cfg<128, 512>::BM;
        case 256128: return Cfg<256, 128>::BM;
        case 256256: return Cfg<256, 256>::BM;
        case 256512: return Cfg<256, 512>::BM;
        case 512128: return Cfg<512, 128>::BM;
        case 512256: return Cfg<512, 256>::BM;
        case 512512: return Cfg<512, 512>::BM;
        default: return 0;
    }
}

hipError_t launch_bf16_fused(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    return launch_shape(p, ut, false, stream);
}

hipError_t launch_bf16_fused_routed(const Problem& p, const UnitTab& ut, hipStream_t stream) {
    return launch_shape(p, ut, true, stream);
}

}  // namespace mot
