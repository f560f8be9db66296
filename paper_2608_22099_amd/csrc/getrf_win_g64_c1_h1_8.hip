// Register-window banded LU instantiated for 64 lanes per matrix, 1 column(s)
// per lane and kl + 1 = 1..8 (one file per range keeps compiles parallel).
#include "getrf_win64.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c1_h1_8(int H) {
    static constexpr auto table = Win64Range<1, 1, 8>::make(
        std::make_integer_sequence<int, 8 - 1 + 1>{});
    return (H >= 1 && H <= 8) ? table[H - 1] : nullptr;
}

}  // namespace bandlu
