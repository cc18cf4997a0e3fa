// variants_s8.hip - the INT8 -> INT32 kernel table (see variants.hpp).
#include "variants.hpp"

namespace mpg {

const Variant kS8[] = {VARIANT_LIST(S8)};
static_assert(sizeof(kS8) / sizeof(kS8[0]) == kNumS8, "variant count out of date in variants.hpp");

}  // namespace mpg
