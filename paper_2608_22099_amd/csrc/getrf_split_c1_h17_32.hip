// Two-wavefront banded LU (getrf_split.hpp) instantiated for 1 column(s) per
// lane and kl + 1 = 17..32 (one file per range keeps compiles parallel).
#include "getrf_split.hpp"

namespace bandlu {

WinKernel split_kernel_c1_h17_32(int H) {
    static constexpr auto table = SplitRange<1, 17, 32>::make(std::make_integer_sequence<int, 32 - 17 + 1>{});
    return (H >= 17 && H <= 32) ? table[H - 17] : nullptr;
}

}  // namespace bandlu
