// tposeb.hip - kernels for B stored K x N row-major (tposeb_gemm.hpp).
#include "variants.hpp"
#include "tposeb_gemm.hpp"

namespace mpg {

// Kernel for dtype (F16, S8 or S4) on the 8-wave 256 x 256 tile, or null.
const void *tposeb_kernel(int dtype) {
    typedef void (*fn_t)(const uint8_t *, const uint8_t *, void *, int, int, int, int, int, EpiParams);
    static const fn_t f16 = &tiled_gemm_tb<F16, T256x256_w8_s2>;
    static const fn_t s8 = &tiled_gemm_tb<S8, T256x256_w8_s2>;
    static const fn_t s4 = &tiled_gemm_tb<S4, T256x256_w8_s2>;
    return dtype == F16 ? reinterpret_cast<const void *>(f16)
                        : (dtype == S8 ? reinterpret_cast<const void *>(s8)
                                       : (dtype == S4 ? reinterpret_cast<const void *>(s4) : nullptr));
}

}  // namespace mpg
