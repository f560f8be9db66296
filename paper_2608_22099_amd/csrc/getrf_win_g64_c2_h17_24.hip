// Register-window banded LU instantiated for 64 lanes per matrix, 2 column(s)
// per lane and kl + 1 = 17..24 (one file per range keeps compiles parallel).
#include "getrf_window.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c2_h17_24(int H) {
    static constexpr auto table = WinRange<64, 2, 17, 24>::make(
        std::make_integer_sequence<int, 24 - 17 + 1>{});
    return (H >= 17 && H <= 24) ? table[H - 17] : nullptr;
}

}  // namespace bandlu
