// Matrix-core kernel variants, part 0 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part0(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 14, 14, 2, 1, 2, 2, 8>>("k3s1_t14x14_co64_k2"),
    make_variant<Cfg<3, 1, 14, 14, 2, 1, 2, 2, 16>>("k3s1_t14x14_co64_k2_cc16"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 8>>("k3s1_t14x14_co64"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 2, 1, 8>>("k3s1_t14x14_co64_w8"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 2, 1, 16>>("k3s1_t14x14_co64_w8_cc16"),
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 16>>("k3s1_t14x14_co64_cc16"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
