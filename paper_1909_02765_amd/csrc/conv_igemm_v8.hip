// Matrix-core kernel variants, part 8 of the table (the templates are in
// conv_igemm.h; the parts compile in parallel).  This part is built with the
// compiler's default accumulator register form instead of the VGPR form the
// other parts use: in the VGPR form, the prepacked-weight, in-workgroup
// pooled instantiation of this variant computed wrong values (rows 1-3 of
// its second output-channel block in the tile's last pixel blocks) where the
// default form is bit for bit right.
#include "conv_igemm.h"

namespace ilpm {
namespace ig {

int variants_part8(const Variant **table)
{
    //                                  KS S  TH  TW NWC NWP NWK MA CC
    static const Variant t[] = {
    make_variant<Cfg<3, 1, 14, 14, 4, 1, 1, 2, 8>>("k3s1_t14x14_co128"),
    };
    *table = t;
    return (int)(sizeof(t) / sizeof(t[0]));
}

}  // namespace ig
}  // namespace ilpm
