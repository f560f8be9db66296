// Diagonal-pivot banded LU (getrf_diag.hpp) instantiated for ku = 1..8 (one
// file per range keeps compiles parallel).
#include "getrf_diag.hpp"

namespace bandlu {

WinKernel diag_kernel_ku1_8(int KU) {
    static constexpr auto table = DiagRange<1, 8>::make(std::make_integer_sequence<int, 8 - 1 + 1>{});
    return (KU >= 1 && KU <= 8) ? table[KU - 1] : nullptr;
}

}  // namespace bandlu
