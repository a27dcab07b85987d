// Matrix-core kernel variants, part 1 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part1(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 16, 2, 0, false, true>>("k3s1_t14x14_co64_cc16_pf"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 8, 2, 0, false, true>>("k3s1_t14x14_co64_pf"),
    make_variant<Cfg<3, 1, 14, 14, 2, 1, 2, 1, 8>>("k3s1_t14x14_co32_k2"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 4>>("k3s1_t14x14_co64_cc4"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 4>>("k3s1_t7x7_co64_cc4"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
