// Two-wavefront banded LU (getrf_split.hpp) instantiated for 1 column(s) per
// lane and kl + 1 = 2..16 (one file per range keeps compiles parallel).
#include "getrf_split.hpp"

namespace bandlu {

WinKernel split_kernel_c1_h2_16(int H) {
    static constexpr auto table = SplitRange<1, 2, 16>::make(std::make_integer_sequence<int, 16 - 2 + 1>{});
    return (H >= 2 && H <= 16) ? table[H - 2] : nullptr;
}

}  // namespace bandlu
