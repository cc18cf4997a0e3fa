// variants_s4.hip - the INT4 -> INT32 kernel table (see variants.hpp).
#include "variants.hpp"

namespace mpg {

// INT4 also runs on the FP6 matrix cores: converted by a pre-pass into a
// workspace (f6_gemm.hpp, wide_f6.hpp; "k" is k per stage) or inside the GEMM
// (wide_i4.hpp).
const Variant kS4[] = {VARIANT_LIST(S4),
                             fp6<F6_256x256_w8_s3>("fp6pipe256x256_w2x4_k128_s3"),
                             fp6<F6_256x256_w8_s2>("fp6pipe256x256_w2x4_k128_s2"),
                             fp6<F6_256x256_w4_s3>("fp6pipe256x256_w2x2_k128_s3"),
                             fp6<F6_256x256_w8t_s3>("fp6pipe256x256_w4x2_k128_s3"),
                             fp6<F6_256x128_w4_s4>("fp6pipe256x128_w2x2_k128_s4"),
                             fp6<F6_128x128_w4_s4>("fp6pipe128x128_w2x2_k128_s4"),
                             fp6<F6_128x128_w4_s6>("fp6pipe128x128_w2x2_k128_s6"),
                             fp6<F6_128x128_w4_k256_s3>("fp6pipe128x128_w2x2_k256_s3"),
                             fp6wide("fp6wide256x256_w2x2_k128_s3"),
                             // conversion inside the GEMM (no workspace); "k": K multiple
                             i4wide("e2m3wide256x256_w2x2_k256"),
                             i4wide<CP_SC0>("e2m3wide256x256_w2x2_k256_sc0"),
                             i4wide<CP_SC1>("e2m3wide256x256_w2x2_k256_sc1"),
                             i4wide<CP_NT>("e2m3wide256x256_w2x2_k256_nt"),
                             fp6wide<CP_SC0>("fp6wide256x256_w2x2_k128_s3_sc0"),
                             fp6wide<CP_SC1>("fp6wide256x256_w2x2_k128_s3_sc1"),
                             fp6wide<CP_NT>("fp6wide256x256_w2x2_k128_s3_nt"),
                             fp6wide_sk("fp6wide256x256_w2x2_k128_s3_sk")};
static_assert(sizeof(kS4) / sizeof(kS4[0]) == kNumS4, "variant count out of date in variants.hpp");

}  // namespace mpg
