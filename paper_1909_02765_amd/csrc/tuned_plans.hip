// The measured plan tables: for shapes the offline sweep timed on MI355X
// (tune.py), the fastest (kernel variant, split count), one table per
// (weight layout, epilogue) pair: OIHW or prepacked weights (the kernels load
// these differently, so the fastest variant can differ), and the plain
// convolution or the fused ReLU + 2x2 max-pool epilogue (a plan whose tiles
// pool in the workgroup saves the second kernel the others need).  Entries name the variant, so the
// tables survive changes to the variant list; an entry whose variant no
// longer exists, or no longer accepts the shape, is ignored.
#include <cstring>

#include "internal.h"

namespace ilpm {
namespace {

struct TunedEntry {
    int c_in, h, w, c_out, k, stride, pad;
    const char *variant;
    int splits;
};

const TunedEntry kTuned[] = {
#include "tuned_plans.inc"
};

const TunedEntry kTunedPrepacked[] = {
#include "tuned_plans_prepacked.inc"
};

const TunedEntry kTunedPooled[] = {
#include "tuned_plans_pooled.inc"
};

const TunedEntry kTunedPooledPrepacked[] = {
#include "tuned_plans_pooled_prepacked.inc"
};

template <size_t N>
bool lookup(const TunedEntry (&table)[N], const ConvShape &s, ilpm_plan *p)
{
    for (const TunedEntry &e : table) {
        if (e.c_in != s.c_in || e.h != s.h || e.w != s.w || e.c_out != s.c_out || e.k != s.k ||
            e.stride != s.stride || e.pad != s.pad)
            continue;
        for (int v = 0; v < igemm_num_variants(); ++v)
            if (std::strcmp(igemm_variant_name(v), e.variant) == 0) return igemm_make_plan(s, v, e.splits, p);
        for (int v = 0; v < direct_num_variants(); ++v)
            if (std::strcmp(direct_variant_name(v), e.variant) == 0) return direct_make_plan(s, v, p);
        return false;
    }
    return false;
}

}  // namespace

bool tuned_plan(const ConvShape &s, ilpm_plan *p, bool prepacked, bool pooled)
{
    if (pooled) return prepacked ? lookup(kTunedPooledPrepacked, s, p) : lookup(kTunedPooled, s, p);
    return prepacked ? lookup(kTunedPrepacked, s, p) : lookup(kTuned, s, p);
}

}  // namespace ilpm
