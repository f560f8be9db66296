// Lean window kernel with the forward solve fused into it, instantiated for
// 1 column(s) per lane and kl + 1 = 2..7 (one file per width keeps compiles
// parallel).
#include "getrf_lean64.hpp"

namespace bandlu {

WinKernel lean64_fwd_kernel_c1(int H) {
    static constexpr WinKernel table[] = {
        &getrf_lean64_kernel<2, 1, true>, &getrf_lean64_kernel<3, 1, true>,
        &getrf_lean64_kernel<4, 1, true>, &getrf_lean64_kernel<5, 1, true>,
        &getrf_lean64_kernel<6, 1, true>, &getrf_lean64_kernel<7, 1, true>};
    return (H >= 2 && H <= 7) ? table[H - 2] : nullptr;
}

}  // namespace bandlu
