// Matrix-core kernel variants, part 2 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part2(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 8>>("k3s1_t7x7_co64"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 8, 2, 0, true>>("k3s1_t7x7_co64_wl"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 16>>("k3s1_t7x7_co64_cc16"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 4, 1, 16>>("k3s1_t7x7_co64_k4"),
    make_variant<Cfg<3, 1, 8, 32, 2, 2, 1, 2, 8>>("k3s1_t8x32_co64"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 64>>("k3s1_t4x4_co16_k4"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
