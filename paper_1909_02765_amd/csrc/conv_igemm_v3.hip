// Matrix-core kernel variants, part 3 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part3(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 32>>("k3s1_t4x4_co16_k4_cc32"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 2, 32>>("k3s1_t4x4_co32_k4"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 4, 16>>("k3s1_t4x4_co64_k4"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 16, 3, 4, true>>("k3s1_t4x4_co16_k4_cc16_s4_wl"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 16, 3, 8, true>>("k3s1_t4x4_co16_k4_cc16_s8_wl"),
    make_variant<Cfg<3, 1, 4, 4, 1, 1, 4, 1, 16, 3, 16, true>>("k3s1_t4x4_co16_k4_cc16_s16_wl"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
