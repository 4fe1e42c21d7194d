// Attention-logit kernels with the stage-2 residual correction (the kernel
// template is in isoq_scores.h): m = 64 or 128 sign bits at the decoding
// widths up to 192, 64 at d = 256 and 512; group sizes 1 (static LDS) or any
// (dynamic LDS).
#include "isoq_scores.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, bool F16, int QM>
ScoreKernel entry_qjl(int group)
{
    using S = ScoreShape<D, BITS, QM>;
    if (group == 1 && kStaticLds<D, BITS, 1, QM>)
        return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, 1, QM>), 0};
    return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, 0, QM>),
            sizeof(float) * (size_t)S::lds_floats(group)};
}

template <int VAR, int D, int BITS, bool F16>
ScoreKernel pick_m(int group, int m)
{
    if (m == 64)
        return entry_qjl<VAR, D, BITS, F16, 64>(group);
    if constexpr (D <= 192) {
        if (m == 128)
            return entry_qjl<VAR, D, BITS, F16, 128>(group);
    }
    return {nullptr, 0};
}

template <int VAR, int D>
ScoreKernel pick_bits(int bits, bool f16, int group, int m)
{
    switch (bits) {
    case 2: return f16 ? pick_m<VAR, D, 2, true>(group, m) : pick_m<VAR, D, 2, false>(group, m);
    case 3: return f16 ? pick_m<VAR, D, 3, true>(group, m) : pick_m<VAR, D, 3, false>(group, m);
    case 4: return f16 ? pick_m<VAR, D, 4, true>(group, m) : pick_m<VAR, D, 4, false>(group, m);
    }
    return {nullptr, 0};
}

template <int VAR>
ScoreKernel pick_d(int d, int bits, bool f16, int group, int m)
{
    switch (d) {
    case 64: return pick_bits<VAR, 64>(bits, f16, group, m);
    case 80: return pick_bits<VAR, 80>(bits, f16, group, m);
    case 96: return pick_bits<VAR, 96>(bits, f16, group, m);
    case 128: return pick_bits<VAR, 128>(bits, f16, group, m);
    case 160: return pick_bits<VAR, 160>(bits, f16, group, m);
    case 192: return pick_bits<VAR, 192>(bits, f16, group, m);
    case 256: return pick_bits<VAR, 256>(bits, f16, group, m);
    case 512: return pick_bits<VAR, 512>(bits, f16, group, m);
    }
    return {nullptr, 0};
}

}  // namespace

ScoreKernel score_qjl_kernel_for(int variant, int d, int bits, bool f16, int group, int m)
{
    switch (variant) {
    case VAR_FULL: return pick_d<VAR_FULL>(d, bits, f16, group, m);
    case VAR_FAST: return pick_d<VAR_FAST>(d, bits, f16, group, m);
    case VAR_PLANAR2D: return pick_d<VAR_PLANAR2D>(d, bits, f16, group, m);
    }
    return {nullptr, 0};
}

}  // namespace isoq
