// Register-window banded LU instantiated for 64 lanes per matrix, 1 column(s)
// per lane and kl + 1 = 17..24 (one file per range keeps compiles parallel).
#include "getrf_win64.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c1_h17_24(int H) {
    static constexpr auto table = Win64Range<1, 17, 24>::make(
        std::make_integer_sequence<int, 24 - 17 + 1>{});
    return (H >= 17 && H <= 24) ? table[H - 17] : nullptr;
}

}  // namespace bandlu
