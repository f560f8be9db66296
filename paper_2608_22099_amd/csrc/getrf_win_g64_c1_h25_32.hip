// Register-window banded LU instantiated for 64 lanes per matrix, 1 column(s)
// per lane and kl + 1 = 25..32 (one file per range keeps compiles parallel).
#include "getrf_win64.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c1_h25_32(int H) {
    static constexpr auto table = Win64Range<1, 25, 32>::make(
        std::make_integer_sequence<int, 32 - 25 + 1>{});
    return (H >= 25 && H <= 32) ? table[H - 25] : nullptr;
}

}  // namespace bandlu
