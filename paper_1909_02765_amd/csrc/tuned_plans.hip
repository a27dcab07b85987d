// The measured plan table: for shapes the offline sweep timed on MI355X
// (tune.py), the fastest (kernel variant, split count).  Entries name the
// variant, so the table survives changes to the variant list; an entry whose
// variant no longer exists, or no longer accepts the shape, is ignored.
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

}  // namespace

bool tuned_plan(const ConvShape &s, ilpm_plan *p)
{
    for (const TunedEntry &e : kTuned) {
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

}  // namespace ilpm
