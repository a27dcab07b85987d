// Matrix-core kernel variants, part 9 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel): layers with large outputs,
// with their output stores at device scope.
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part9(const Variant **table)
{
    //                                         KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Sc1Out<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 16, 2, 0, false, true>>>("k3s1_t14x14_co64_cc16_pf_sc1"),
    make_variant<Sc1Out<Cfg<3, 1, 14, 14, 4, 1, 1, 1, 4>>>("k3s1_t14x14_co64_cc4_sc1"),
    make_variant<Sc1Out<Cfg<3, 1, 14, 14, 2, 1, 2, 1, 8>>>("k3s1_t14x14_co32_k2_sc1"),
    make_variant<Sc1Out<Cfg<3, 1, 14, 14, 1, 1, 4, 1, 16>>>("k3s1_t14x14_co16_k4_sc1"),
    make_variant<Sc1Out<Cfg<3, 1, 7, 7, 1, 1, 4, 1, 16>>>("k3s1_t7x7_co16_k4_sc1"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
