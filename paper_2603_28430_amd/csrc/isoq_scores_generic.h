// Attention logits at key widths without a tuned logit kernel (any d from 1
// to 1024 outside {64, 80, 96, 128, 160, 192, 256, 512}): the shape of the
// padded record the width-generic kernel reads, and its dispatch.  Host code
// includes this header; the kernel is in isoq_scores_generic.hip.
#pragma once

#include "isoq_internal.h"

namespace isoq {

// The padded layout of Sec. 5.1's zero padding, as the generic stage-1
// kernels store it: `slots` rotation slots of SW coordinates (4, or 8 for
// 8-D blocks), record bytes `rec`, parameter floats per set `set_stride`.
struct GenScoreShape {
    int32_t d;
    int32_t slots;
    int32_t rec;
    int32_t rec_lp;      // the cache layout's pieces: 1 << rec_lp bytes, or records whole (< 0)
    int64_t set_stride;
};

// Kernel (args: SArgs, GenScoreShape; grid (query head, chunk of
// kScoreChunk positions, sequence), 256 threads, dynamic LDS
// generic_score_lds(slots, variant) bytes) or nullptr.
const void *generic_score_kernel_for(int variant, int bits, bool f16);

inline size_t generic_score_lds(int slots, int variant)
{
    return sizeof(float) * (16 + (size_t)slots * (variant == VAR_BLOCK8 ? 8 : 4));
}

}  // namespace isoq
