// Matrix-core kernel variants, part 5 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part5(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 2, 7, 7, 4, 1, 1, 1, 8>>("k3s2_t7x7_co64"),
    make_variant<Cfg<3, 2, 7, 7, 4, 1, 1, 1, 16>>("k3s2_t7x7_co64_cc16"),
    make_variant<Cfg<3, 2, 7, 7, 4, 1, 4, 1, 16>>("k3s2_t7x7_co64_k4"),
    make_variant<Cfg<3, 2, 4, 4, 1, 1, 4, 1, 64>>("k3s2_t4x4_co16_k4"),
    make_variant<Cfg<3, 2, 4, 4, 1, 1, 4, 1, 16, 3, 8, true>>("k3s2_t4x4_co16_k4_cc16_s8_wl"),
    make_variant<Cfg<1, 1, 7, 7, 4, 1, 1, 1, 16>>("k1s1_t7x7_co64"),
    make_variant<Cfg<3, 1, 7, 7, 1, 1, 4, 1, 16, 3, 4, true>>("k3s1_t7x7_co16_k4_s4_wl"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
