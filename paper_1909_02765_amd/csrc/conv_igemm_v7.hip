// Matrix-core kernel variants, part 7 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part7(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<5, 1, 4, 4, 1, 1, 4, 1, 32>>("k5s1_t4x4_co16_k4"),
    make_variant<Cfg<5, 1, 4, 4, 1, 1, 4, 1, 16, 3, 8, true>>("k5s1_t4x4_co16_k4_cc16_s8_wl"),
    make_variant<Cfg<5, 1, 8, 8, 1, 1, 4, 1, 16, 3, 4, true>>("k5s1_t8x8_co16_k4_cc16_s4_wl"),
    make_variant<Cfg<5, 1, 4, 4, 1, 1, 4, 1, 16, 3, 16, true>>("k5s1_t4x4_co16_k4_cc16_s16_wl"),
    make_variant<Cfg<3, 1, 14, 14, 1, 1, 4, 1, 16>>("k3s1_t14x14_co16_k4"),
    make_variant<Cfg<3, 1, 7, 7, 1, 1, 4, 1, 16>>("k3s1_t7x7_co16_k4"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
