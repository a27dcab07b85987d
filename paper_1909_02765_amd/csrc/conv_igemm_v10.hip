// Matrix-core kernel variants, part 10 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel): 14x14 tiles, 32 output
// channels, the input channels split over two waves, with 16-channel stages
// (half the stage boundaries of the 8-channel form: VGG conv2_2, 128->128 at
// 112^2, 31.7 -> 30.6 us with device-scope stores; 32-channel stages and the
// same change for four-wave splits measured slower).
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part10(const Variant **table)
{
    //                                         KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 14, 14, 2, 1, 2, 1, 16>>("k3s1_t14x14_co32_k2_cc16"),
    make_variant<Sc1Out<Cfg<3, 1, 14, 14, 2, 1, 2, 1, 16>>>("k3s1_t14x14_co32_k2_cc16_sc1"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
