// Matrix-core kernel variants, part 6 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part6(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<1, 1, 7, 7, 4, 1, 4, 1, 32>>("k1s1_t7x7_co64_k4"),
    make_variant<Cfg<1, 1, 14, 14, 4, 1, 1, 1, 16>>("k1s1_t14x14_co64"),
    make_variant<Cfg<1, 1, 4, 4, 1, 1, 4, 1, 64>>("k1s1_t4x4_co16_k4"),
    make_variant<Cfg<5, 1, 7, 7, 4, 1, 1, 1, 4>>("k5s1_t7x7_co64"),
    make_variant<Cfg<5, 1, 7, 7, 4, 1, 1, 1, 8>>("k5s1_t7x7_co64_cc8"),
    make_variant<Cfg<5, 1, 7, 7, 4, 1, 2, 1, 8>>("k5s1_t7x7_co64_k2"),
    make_variant<Cfg<3, 1, 7, 7, 2, 1, 2, 1, 16>>("k3s1_t7x7_co32_k2"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
