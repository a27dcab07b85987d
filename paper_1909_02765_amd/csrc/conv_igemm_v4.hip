// Matrix-core kernel variants, part 4 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part4(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 32, 3, 8, true>>("k3s1_t4x4_co16_k4_cc32_s8_wl"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 2, 16, 3, 8, true>>("k3s1_t4x4_co32_k4_cc16_s8_wl"),
    make_variant<Cfg<3, 1, 8, 8, 1, 1, 4, 1, 16, 3, 4, true>>("k3s1_t8x8_co16_k4_cc16_s4_wl"),
    make_variant<Cfg<3, 1, 8, 8, 1, 1, 4, 1, 16, 3, 8, true>>("k3s1_t8x8_co16_k4_cc16_s8_wl"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 4, 3, 4>>("k3s1_t7x7_co64_cc4_s4"),
    make_variant<Cfg<3, 1, 7, 7, 4, 1, 1, 1, 4, 3, 8>>("k3s1_t7x7_co64_cc4_s8"),
    make_variant<Cfg<3, 1, 7, 7, 2, 1, 2, 1, 16, 3, 8>>("k3s1_t7x7_co32_k2_s8"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
