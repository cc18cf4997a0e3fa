// variants_f16.hip - the FP16 -> FP32 kernel table (see variants.hpp).
#include "variants.hpp"

namespace mpg {

const Variant kF16[] = {VARIANT_LIST(F16)};
static_assert(sizeof(kF16) / sizeof(kF16[0]) == kNumF16, "variant count out of date in variants.hpp");

}  // namespace mpg
