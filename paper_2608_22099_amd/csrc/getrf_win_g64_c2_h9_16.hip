// Register-window banded LU instantiated for 64 lanes per matrix, 2 column(s)
// per lane and kl + 1 = 9..16 (one file per range keeps compiles parallel).
#include "getrf_win64.hpp"

namespace bandlu {

WinKernel win_kernel_g64_c2_h9_16(int H) {
    static constexpr auto table = Win64Range<2, 9, 16>::make(
        std::make_integer_sequence<int, 16 - 9 + 1>{});
    return (H >= 9 && H <= 16) ? table[H - 9] : nullptr;
}

}  // namespace bandlu
