// Batched banded LU, 16 lanes per matrix and one column per lane, for
// kl + 1 = 1..8 (getrf_g16.hpp).
#include "getrf_g16.hpp"

namespace bandlu {

WinKernel win_kernel_g16_c1_h1_8(int H) {
    static constexpr WinKernel table[8] = {
        &getrf_g16_kernel<1>, &getrf_g16_kernel<2>, &getrf_g16_kernel<3>, &getrf_g16_kernel<4>,
        &getrf_g16_kernel<5>, &getrf_g16_kernel<6>, &getrf_g16_kernel<7>, &getrf_g16_kernel<8>};
    return (H >= 1 && H <= 8) ? table[H - 1] : nullptr;
}

}  // namespace bandlu
