// Compile-time dispatch of the attention-logit kernels without the stage-2
// sketch over width, bits, query type and group size (the kernel template is
// in isoq_scores.h), shared by the translation units that instantiate it for
// the rotation variants (isoq_scores.hip, isoq_scores_8d.hip).
#pragma once

#include "isoq_scores.h"

namespace isoq {
namespace {

template <int VAR, int D, int BITS, bool F16, int GT>
ScoreKernel entry(int group)
{
    using S = ScoreShape<D, BITS, 0>;
    if constexpr (kStaticLds<D, BITS, GT, 0>)
        return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, GT, 0>), 0};
    return {reinterpret_cast<const void *>(&score_kernel<VAR, D, BITS, F16, 0, 0>),
            sizeof(float) * (size_t)S::lds_floats(group)};
}

template <int VAR, int D, int BITS, bool F16>
ScoreKernel pick_group(int group)
{
    switch (group) {
    case 1: return entry<VAR, D, BITS, F16, 1>(group);
    case 4: return entry<VAR, D, BITS, F16, 4>(group);
    }
    return entry<VAR, D, BITS, F16, 0>(group);
}

template <int VAR, int D, int BITS>
ScoreKernel pick_dtype(bool f16, int group)
{
    return f16 ? pick_group<VAR, D, BITS, true>(group) : pick_group<VAR, D, BITS, false>(group);
}

template <int VAR, int D>
ScoreKernel pick_bits(int bits, bool f16, int group)
{
    switch (bits) {
    case 2: return pick_dtype<VAR, D, 2>(f16, group);
    case 3: return pick_dtype<VAR, D, 3>(f16, group);
    case 4: return pick_dtype<VAR, D, 4>(f16, group);
    }
    return {nullptr, 0};
}

template <int VAR>
ScoreKernel pick_d(int d, int bits, bool f16, int group)
{
    switch (d) {
    case 64: return pick_bits<VAR, 64>(bits, f16, group);
    case 80: return pick_bits<VAR, 80>(bits, f16, group);
    case 96: return pick_bits<VAR, 96>(bits, f16, group);
    case 128: return pick_bits<VAR, 128>(bits, f16, group);
    case 160: return pick_bits<VAR, 160>(bits, f16, group);
    case 192: return pick_bits<VAR, 192>(bits, f16, group);
    case 256: return pick_bits<VAR, 256>(bits, f16, group);
    case 512: return pick_bits<VAR, 512>(bits, f16, group);
    }
    return {nullptr, 0};
}

}  // namespace
}  // namespace isoq
